// Non-GEMM kernels of the packed MLP step on gfx950: the linear head with the
// loss and its gradient, column sweeps for bias gradients, the packed AdamW
// update, validation scoring and greedy ensemble selection.
//
// Reductions use wave64 shuffles and fixed-order LDS trees so that every
// result is bit-reproducible run to run (no float atomics anywhere).
#include <math.h>

#include "pack_internal.h"
#include "philox.h"

namespace tabpack {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float ld_act(const __bf16* p, int64_t i) { return (float)p[i]; }
__device__ __forceinline__ float ld_act(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ void st_act(__bf16* p, int64_t i, float v) { p[i] = (__bf16)v; }
__device__ __forceinline__ void st_act(float* p, int64_t i, float v) { p[i] = v; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Fixed-order sum over a 256-thread block (4 waves); result valid in thread 0.
__device__ __forceinline__ double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) r = ((sh[0] + sh[1]) + (sh[2] + sh[3]));
  return r;
}

constexpr double kClip = 1e-15;

// Per-row validation loss of a candidate value p against target y (fp64):
// squared error, binary CE, or CE of the true-class probability.
__device__ __forceinline__ double row_score(Task task, double p, const void* y, int64_t i) {
  if (task == Task::REG) {
    const double d = p - (double)static_cast<const float*>(y)[i];
    return d * d;
  }
  if (task == Task::BIN) {
    const double t = (double)static_cast<const float*>(y)[i];
    const double q = fmin(fmax(p, kClip), 1.0 - kClip);
    return -t * log(q) - (1.0 - t) * log1p(-q);
  }
  return -log(fmin(fmax(p, kClip), 1.0));
}

__device__ __forceinline__ double finish_score(Task task, double sum, int64_t n) {
  double s = sum / (double)n;
  if (task == Task::REG) s = sqrt(s);
  return isfinite(s) ? s : INFINITY;
}

// ------------------------------------------------------------------- head --
// One wave per (member, row): Y = H_L[row] . W_out^T + b_out, then either the
// training loss and dLoss/dY of the row, or the eval prediction.
template <typename T, bool EVAL>
__global__ __launch_bounds__(256) void head_fwd_kernel(Task task, const T* H, const float* theta,
                                                       const MemberDev* mem, int Bp, int d_out,
                                                       const void* y, const int32_t* idx, int B,
                                                       int rows_valid, int64_t row_base, int64_t Nv,
                                                       float* dY, float* rowloss, float* pred) {
  const int k = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= Bp) return;
  const MemberDev md = mem[k];
  const T* h = H + md.act_off + (int64_t)row * md.dp;
  const float* Wo = theta + md.w_out_off;
  float acc[kMaxOut];
#pragma unroll
  for (int o = 0; o < kMaxOut; ++o) acc[o] = 0.0f;
  for (int c = lane; c < md.dp; c += 64) {
    const float hv = ld_act(h, c);
#pragma unroll
    for (int o = 0; o < kMaxOut; ++o)
      if (o < d_out) acc[o] += hv * Wo[(int64_t)o * md.dp + c];
  }
  float z[kMaxOut];
#pragma unroll
  for (int o = 0; o < kMaxOut; ++o) z[o] = (o < d_out) ? wave_sum(acc[o]) + theta[md.b_out_off + o] : 0.0f;
  if (lane != 0) return;

  const bool valid = EVAL ? row < rows_valid : row < B;
  int64_t src = 0;
  if (valid) src = EVAL ? row_base + row : (int64_t)idx[(int64_t)k * B + row];
  if (EVAL) {
    if (!valid) return;
    float p;
    if (task == Task::REG) {
      p = z[0];
    } else if (task == Task::BIN) {
      p = 1.0f / (1.0f + expf(-z[0]));
    } else {
      const int lab = min(max(static_cast<const int32_t*>(y)[src], 0), d_out - 1);
      float mx = z[0];
      for (int o = 1; o < d_out; ++o) mx = fmaxf(mx, z[o]);
      float se = 0.0f;
      for (int o = 0; o < d_out; ++o) se += expf(z[o] - mx);
      p = expf(z[lab] - mx) / se;
    }
    pred[(int64_t)k * Nv + row_base + row] = p;
    return;
  }
  float* dy = dY + ((int64_t)k * Bp + row) * d_out;
  if (!valid) {
    for (int o = 0; o < d_out; ++o) dy[o] = 0.0f;
    rowloss[(int64_t)k * Bp + row] = 0.0f;
    return;
  }
  const float invB = 1.0f / (float)B;
  float loss;
  if (task == Task::REG) {
    const float d = z[0] - static_cast<const float*>(y)[src];
    loss = d * d;
    dy[0] = 2.0f * d * invB;
  } else if (task == Task::BIN) {
    const float t = static_cast<const float*>(y)[src];
    const float x = z[0];
    loss = fmaxf(x, 0.0f) - x * t + log1pf(expf(-fabsf(x)));
    dy[0] = (1.0f / (1.0f + expf(-x)) - t) * invB;
  } else {
    const int lab = min(max(static_cast<const int32_t*>(y)[src], 0), d_out - 1);
    float mx = z[0];
    for (int o = 1; o < d_out; ++o) mx = fmaxf(mx, z[o]);
    float se = 0.0f;
    for (int o = 0; o < d_out; ++o) se += expf(z[o] - mx);
    const float lse = mx + logf(se);
    loss = lse - z[lab];
    for (int o = 0; o < d_out; ++o) dy[o] = (expf(z[o] - lse) - (o == lab ? 1.0f : 0.0f)) * invB;
  }
  rowloss[(int64_t)k * Bp + row] = loss;
}

// Per-member batch-mean loss and head-bias gradient (fixed-order fp64 sums).
__global__ __launch_bounds__(256) void loss_reduce_kernel(const float* rowloss, const float* dY,
                                                          const MemberDev* mem, int Bp, int B,
                                                          int d_out, float* grad, float* loss_out) {
  __shared__ double sh[4];
  const int k = blockIdx.x;
  double s = 0.0;
  for (int r = threadIdx.x; r < B; r += 256) s += (double)rowloss[(int64_t)k * Bp + r];
  s = block_sum_d(s, sh);
  if (threadIdx.x == 0) loss_out[k] = (float)(s / (double)B);
  for (int o = 0; o < d_out; ++o) {
    double g = 0.0;
    for (int r = threadIdx.x; r < B; r += 256) g += (double)dY[((int64_t)k * Bp + r) * d_out + o];
    g = block_sum_d(g, sh);
    if (threadIdx.x == 0) grad[mem[k].b_out_off + o] = (float)g;
  }
}

// Column sweep of the head backward for 64 columns of one member:
//   dH_L = dY W_out, dZ_L = dH_L * [H_L > 0] * s_k, dW_out = dY^T H_L, db_L = sum_rows dZ_L.
template <typename T>
__global__ __launch_bounds__(256) void head_bwd_kernel(const T* H, const float* theta,
                                                       const MemberDev* mem, const ColTile* tiles,
                                                       int Bp, int d_out, const float* dY, T* dZ,
                                                       float* grad) {
  __shared__ float shw[4][kMaxOut + 1][64];
  const ColTile ct = tiles[blockIdx.x];
  const MemberDev md = mem[ct.member];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int c = ct.c0 + tx;
  const bool valid = c < md.dp;
  float wo[kMaxOut], accw[kMaxOut];
#pragma unroll
  for (int o = 0; o < kMaxOut; ++o) {
    wo[o] = (valid && o < d_out) ? theta[md.w_out_off + (int64_t)o * md.dp + c] : 0.0f;
    accw[o] = 0.0f;
  }
  float accb = 0.0f;
  const T* h = H + md.act_off;
  T* dz = dZ + md.act_off;
  const float* dyk = dY + (int64_t)ct.member * Bp * d_out;
  for (int b = ty; b < Bp; b += 4) {
    float dy[kMaxOut];
#pragma unroll
    for (int o = 0; o < kMaxOut; ++o) dy[o] = (o < d_out) ? dyk[(int64_t)b * d_out + o] : 0.0f;
    const float hv = valid ? ld_act(h, (int64_t)b * md.dp + c) : 0.0f;
    float dh = 0.0f;
#pragma unroll
    for (int o = 0; o < kMaxOut; ++o) {
      dh += dy[o] * wo[o];
      accw[o] += dy[o] * hv;
    }
    const float g = hv > 0.0f ? dh * md.drop_s : 0.0f;
    if (valid) st_act(dz, (int64_t)b * md.dp + c, g);
    accb += g;
  }
#pragma unroll
  for (int o = 0; o < kMaxOut; ++o) shw[ty][o][tx] = accw[o];
  shw[ty][kMaxOut][tx] = accb;
  __syncthreads();
  if (ty == 0 && valid) {
    for (int o = 0; o < d_out; ++o)
      grad[md.w_out_off + (int64_t)o * md.dp + c] =
          (shw[0][o][tx] + shw[1][o][tx]) + (shw[2][o][tx] + shw[3][o][tx]);
    grad[md.b_last_off + c] =
        (shw[0][kMaxOut][tx] + shw[1][kMaxOut][tx]) + (shw[2][kMaxOut][tx] + shw[3][kMaxOut][tx]);
  }
}

// db_l[c] = sum of the per-row-block column partials written by the dX epilogue,
// in a fixed order; 64 columns of one member per workgroup.
__global__ __launch_bounds__(64) void bias_from_partials_kernel(const float* part, const MemberDev* mem,
                                                                const ColTile* tiles, int nparts,
                                                                const int64_t* bias_off, float* grad) {
  const ColTile ct = tiles[blockIdx.x];
  const MemberDev md = mem[ct.member];
  const int c = ct.c0 + threadIdx.x;
  if (c >= md.dp) return;
  const float* p = part + md.act_off / kPartRows;
  float s = 0.0f;
  for (int r = 0; r < nparts; ++r) s += p[(int64_t)r * md.dp + c];
  grad[bias_off[ct.member] + c] = s;
}

// ----------------------------------------------------------------- gather --
// H_0 of member k, row r: the feature row X[idx[k * B + r]] (or X[row_base + r]
// for contiguous rows) in the GEMM precision, zero-padded to Pin columns; rows
// r >= rows_valid are zero.  One wave per row, float4 reads.
template <typename T>
__global__ __launch_bounds__(256) void gather_kernel(const float* X, int d_in, int Pin, const int32_t* idx,
                                                     int B, int64_t row_base, int rows_valid, int Bp, T* H0) {
  const int k = blockIdx.y;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= Bp) return;
  T* dst = H0 + ((int64_t)k * Bp + r) * Pin;
  const bool valid = r < rows_valid;
  const int64_t src = valid ? (idx ? (int64_t)idx[(int64_t)k * B + r] : row_base + r) : 0;
  const float* x = X + src * d_in;
  const bool vec = (d_in % 4 == 0) && ((reinterpret_cast<uintptr_t>(X) & 15) == 0);
  for (int c = lane * 4; c < Pin; c += 256) {
    float v[4];
    if (valid && vec && c + 4 <= d_in) {
      const f32x4 q = *reinterpret_cast<const f32x4*>(x + c);
      v[0] = q[0], v[1] = q[1], v[2] = q[2], v[3] = q[3];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (valid && c + e < d_in) ? x[c + e] : 0.0f;
    }
    if constexpr (sizeof(T) == 2) {
      const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[1]) << 16);
      const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[3]) << 16);
      *reinterpret_cast<u32x2*>(dst + c) = u32x2{lo, hi};
    } else {
      *reinterpret_cast<f32x4*>(dst + c) = f32x4{v[0], v[1], v[2], v[3]};
    }
  }
}

// ------------------------------------------------------------------ AdamW --
// One wave per 256-element chunk of the packed parameter buffer; every chunk
// belongs to one member and is all-weight or all-bias, so (lr_k, wd_k) and the
// decay switch are wave-uniform.  float4 loads/stores, 30 bytes per element
// with the bf16 shadow.
template <bool SHADOW>
__global__ __launch_bounds__(256) void adamw_kernel(float* theta, const float* grad, float* m,
                                                    float* v, uint16_t* shadow,
                                                    const uint32_t* chunk_tab, const MemberDev* mem,
                                                    int64_t nchunks, float bc1, float bc2_sqrt,
                                                    float beta1, float beta2, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  for (int64_t c = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); c < nchunks; c += nw) {
    const uint32_t e = chunk_tab[c];
    const MemberDev md = mem[e & 0x7FFFFFFFu];
    const float decay = (e >> 31) ? 1.0f : 1.0f - md.lr * md.wd;
    const float step = md.lr / bc1;
    const int64_t i = c * kChunk + lane * 4;
    f32x4 th = *reinterpret_cast<const f32x4*>(theta + i);
    const f32x4 g = *reinterpret_cast<const f32x4*>(grad + i);
    f32x4 mm = *reinterpret_cast<const f32x4*>(m + i);
    f32x4 vv = *reinterpret_cast<const f32x4*>(v + i);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      th[q] *= decay;
      mm[q] = beta1 * mm[q] + (1.0f - beta1) * g[q];
      vv[q] = beta2 * vv[q] + (1.0f - beta2) * g[q] * g[q];
      th[q] -= step * mm[q] / (sqrtf(vv[q]) / bc2_sqrt + eps);
    }
    *reinterpret_cast<f32x4*>(theta + i) = th;
    *reinterpret_cast<f32x4*>(m + i) = mm;
    *reinterpret_cast<f32x4*>(v + i) = vv;
    if (SHADOW) {
      uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[0]) |
                    ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[1]) << 16);
      uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[2]) |
                    ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[3]) << 16);
      *reinterpret_cast<u32x2*>(shadow + i) = u32x2{lo, hi};
    }
  }
}

__global__ void to_shadow_kernel(const float* theta, uint16_t* shadow, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    shadow[i] = __builtin_bit_cast(uint16_t, (__bf16)theta[i]);
}

// ------------------------------------------------------------ eval scores --
__global__ __launch_bounds__(256) void eval_score_kernel(Task task, const float* pred,
                                                         const void* yv, int64_t Nv,
                                                         double* score_out) {
  __shared__ double sh[4];
  const int k = blockIdx.x;
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < Nv; i += 256) s += row_score(task, (double)pred[k * Nv + i], yv, i);
  s = block_sum_d(s, sh);
  if (threadIdx.x == 0) score_out[k] = finish_score(task, s, Nv);
}

__global__ void dropout_mask_kernel(uint32_t key0, uint32_t key1, uint32_t step, int layer,
                                    int member, uint32_t t, int B, int width, uint8_t* out) {
  const int64_t n = (int64_t)B * width;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / width), c = (int)(i % width);
    const Words4 w = philox4x32_10((uint32_t)r >> 2, (uint32_t)c,
                                   ((uint32_t)member << 8) | (uint32_t)layer, step, key0, key1);
    const uint32_t wq[4] = {w.w0, w.w1, w.w2, w.w3};
    out[i] = wq[r & 3] >= t ? 1 : 0;
  }
}

// --------------------------------------------------------- greedy select --
// state[0] = ensemble size n, state[1] = stopped flag, state[2] = this
// iteration's pick (-1 if none).  sum[i] = running fp64 sum of the picked
// candidates' values on row i.
constexpr int kSelRows = 1024;  // rows per workgroup of the candidate sweep

__global__ __launch_bounds__(256) void select_partial_kernel(Task task, const float* cand,
                                                             const void* yv, int64_t Nv,
                                                             const double* sum, const int32_t* state,
                                                             double* partial, int nblk) {
  __shared__ double sh[4];
  if (state[1]) return;
  const int c = blockIdx.y;
  const double cnt = (double)(state[0] + 1);
  const int64_t r0 = (int64_t)blockIdx.x * kSelRows;
  const int64_t r1 = r0 + kSelRows < Nv ? r0 + kSelRows : Nv;
  double s = 0.0;
  for (int64_t i = r0 + threadIdx.x; i < r1; i += 256)
    s += row_score(task, (sum[i] + (double)cand[(int64_t)c * Nv + i]) / cnt, yv, i);
  s = block_sum_d(s, sh);
  if (threadIdx.x == 0) partial[(int64_t)c * nblk + blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void select_pick_kernel(Task task, int C, int64_t Nv, int m_ens,
                                                          const double* partial, int nblk,
                                                          int32_t* state, double* best,
                                                          int32_t* sel) {
  __shared__ double shs[256];
  __shared__ int shi[256];
  if (state[1]) {
    if (threadIdx.x == 0) state[2] = -1;
    return;
  }
  const int n = state[0];
  double bs = INFINITY;
  int bi = 0x7FFFFFFF;
  for (int c = threadIdx.x; c < C; c += 256) {
    bool taken = false;
    for (int j = 0; j < n; ++j) taken |= (sel[j] == c);
    double tot = 0.0;
    for (int b = 0; b < nblk; ++b) tot += partial[(int64_t)c * nblk + b];
    const double s = taken ? INFINITY : finish_score(task, tot, Nv);
    if (s < bs || (s == bs && c < bi)) {
      bs = s;
      bi = c;
    }
  }
  shs[threadIdx.x] = bs;
  shi[threadIdx.x] = bi;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (threadIdx.x < w) {
      const double s2 = shs[threadIdx.x + w];
      const int i2 = shi[threadIdx.x + w];
      if (s2 < shs[threadIdx.x] || (s2 == shs[threadIdx.x] && i2 < shi[threadIdx.x])) {
        shs[threadIdx.x] = s2;
        shi[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double s = shs[0];
    const int c = shi[0];
    if (!(s < INFINITY) || c >= C || (n > 0 && !(s < *best))) {
      state[1] = 1;
      state[2] = -1;
    } else {
      sel[n] = c;
      state[0] = n + 1;
      state[2] = c;
      *best = s;
      if (n + 1 >= m_ens || n + 1 >= C) state[1] = 1;
    }
  }
}

__global__ void select_update_kernel(const float* cand, int64_t Nv, const int32_t* state, double* sum) {
  const int c = state[2];
  if (c < 0) return;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < Nv;
       i += (int64_t)gridDim.x * blockDim.x)
    sum[i] += (double)cand[(int64_t)c * Nv + i];
}

__global__ void select_init_kernel(double* sum, int64_t Nv, int32_t* state, double* best) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < Nv;
       i += (int64_t)gridDim.x * blockDim.x)
    sum[i] = 0.0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    state[0] = 0;
    state[1] = 0;
    state[2] = -1;
    *best = INFINITY;
  }
}

__global__ void select_final_kernel(const int32_t* state, const double* best, int32_t* n_sel,
                                    double* score) {
  *n_sel = state[0];
  *score = *best;
}

inline int grid_for(int64_t n, int per) {
  int64_t g = (n + per - 1) / per;
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (int)g;
}

}  // namespace

int select_blocks(int64_t Nv) { return (int)((Nv + kSelRows - 1) / kSelRows); }

hipError_t launch_head_fwd(Prec prec, Task task, bool eval, const void* H, const float* theta,
                           const MemberDev* mem, int K, int Bp, int d_out, const void* y,
                           const int32_t* idx, int B, int rows_valid, int64_t row_base, int64_t Nv,
                           float* dY, float* rowloss, float* pred, hipStream_t s) {
  const dim3 grid((Bp + 3) / 4, K);
  if (prec == Prec::BF16) {
    if (eval)
      hipLaunchKernelGGL((head_fwd_kernel<__bf16, true>), grid, dim3(256), 0, s, task,
                         static_cast<const __bf16*>(H), theta, mem, Bp, d_out, y, idx, B, rows_valid,
                         row_base, Nv, dY, rowloss, pred);
    else
      hipLaunchKernelGGL((head_fwd_kernel<__bf16, false>), grid, dim3(256), 0, s, task,
                         static_cast<const __bf16*>(H), theta, mem, Bp, d_out, y, idx, B, rows_valid,
                         row_base, Nv, dY, rowloss, pred);
  } else {
    if (eval)
      hipLaunchKernelGGL((head_fwd_kernel<float, true>), grid, dim3(256), 0, s, task,
                         static_cast<const float*>(H), theta, mem, Bp, d_out, y, idx, B, rows_valid,
                         row_base, Nv, dY, rowloss, pred);
    else
      hipLaunchKernelGGL((head_fwd_kernel<float, false>), grid, dim3(256), 0, s, task,
                         static_cast<const float*>(H), theta, mem, Bp, d_out, y, idx, B, rows_valid,
                         row_base, Nv, dY, rowloss, pred);
  }
  return hipGetLastError();
}

hipError_t launch_loss_reduce(const float* rowloss, const float* dY, const MemberDev* mem, int K,
                              int Bp, int B, int d_out, float* grad, float* loss_out, hipStream_t s) {
  hipLaunchKernelGGL(loss_reduce_kernel, dim3(K), dim3(256), 0, s, rowloss, dY, mem, Bp, B, d_out,
                     grad, loss_out);
  return hipGetLastError();
}

hipError_t launch_head_bwd(Prec prec, const void* H, const float* theta, const MemberDev* mem,
                           const ColTile* tiles, int ntiles, int Bp, int d_out, const float* dY,
                           void* dZ, float* grad, hipStream_t s) {
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((head_bwd_kernel<__bf16>), dim3(ntiles), dim3(256), 0, s,
                       static_cast<const __bf16*>(H), theta, mem, tiles, Bp, d_out, dY,
                       static_cast<__bf16*>(dZ), grad);
  else
    hipLaunchKernelGGL((head_bwd_kernel<float>), dim3(ntiles), dim3(256), 0, s,
                       static_cast<const float*>(H), theta, mem, tiles, Bp, d_out, dY,
                       static_cast<float*>(dZ), grad);
  return hipGetLastError();
}

hipError_t launch_bias_from_partials(const float* part, const MemberDev* mem, const ColTile* tiles,
                                     int ntiles, int nparts, const int64_t* bias_off, float* grad,
                                     hipStream_t s) {
  hipLaunchKernelGGL(bias_from_partials_kernel, dim3(ntiles), dim3(64), 0, s, part, mem, tiles, nparts,
                     bias_off, grad);
  return hipGetLastError();
}

hipError_t launch_gather(Prec prec, const float* X, int d_in, int Pin, const int32_t* idx, int B,
                         int64_t row_base, int rows_valid, int members, int Bp, void* H0, hipStream_t s) {
  const dim3 grid((Bp + 3) / 4, members);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((gather_kernel<__bf16>), grid, dim3(256), 0, s, X, d_in, Pin, idx, B, row_base,
                       rows_valid, Bp, static_cast<__bf16*>(H0));
  else
    hipLaunchKernelGGL((gather_kernel<float>), grid, dim3(256), 0, s, X, d_in, Pin, idx, B, row_base,
                       rows_valid, Bp, static_cast<float*>(H0));
  return hipGetLastError();
}

hipError_t launch_adamw(Prec prec, float* theta, const float* grad, float* m, float* v,
                        uint16_t* shadow, const uint32_t* chunk_tab, const MemberDev* mem,
                        int64_t nchunks, float bc1, float bc2_sqrt, float beta1, float beta2,
                        float eps, hipStream_t s) {
  const int grid = grid_for(nchunks, 4);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((adamw_kernel<true>), dim3(grid), dim3(256), 0, s, theta, grad, m, v, shadow,
                       chunk_tab, mem, nchunks, bc1, bc2_sqrt, beta1, beta2, eps);
  else
    hipLaunchKernelGGL((adamw_kernel<false>), dim3(grid), dim3(256), 0, s, theta, grad, m, v, shadow,
                       chunk_tab, mem, nchunks, bc1, bc2_sqrt, beta1, beta2, eps);
  return hipGetLastError();
}

hipError_t launch_to_shadow(const float* theta, uint16_t* shadow, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(to_shadow_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, theta, shadow, n);
  return hipGetLastError();
}

hipError_t launch_eval_score(Task task, const float* pred, const void* yv, int K, int64_t Nv,
                             double* score_out, hipStream_t s) {
  hipLaunchKernelGGL(eval_score_kernel, dim3(K), dim3(256), 0, s, task, pred, yv, Nv, score_out);
  return hipGetLastError();
}

hipError_t launch_dropout_mask(uint32_t key0, uint32_t key1, uint32_t step, int layer, int member,
                               uint32_t t, int B, int width, uint8_t* out, hipStream_t s) {
  hipLaunchKernelGGL(dropout_mask_kernel, dim3(grid_for((int64_t)B * width, 256)), dim3(256), 0, s,
                     key0, key1, step, layer, member, t, B, width, out);
  return hipGetLastError();
}

hipError_t launch_select_init(double* sum, int64_t Nv, int32_t* state, double* best,
                              int32_t* n_sel_out, double* score_out, hipStream_t s) {
  (void)n_sel_out;
  (void)score_out;
  hipLaunchKernelGGL(select_init_kernel, dim3(grid_for(Nv, 256)), dim3(256), 0, s, sum, Nv, state, best);
  return hipGetLastError();
}

hipError_t launch_select_iter(Task task, const float* cand, const void* yv, int C, int64_t Nv,
                              int m_ens, double* sum, double* partial, int nblk, int32_t* state,
                              double* best, int32_t* sel_out, hipStream_t s) {
  hipLaunchKernelGGL(select_partial_kernel, dim3(nblk, C), dim3(256), 0, s, task, cand, yv, Nv, sum,
                     state, partial, nblk);
  hipLaunchKernelGGL(select_pick_kernel, dim3(1), dim3(256), 0, s, task, C, Nv, m_ens, partial, nblk,
                     state, best, sel_out);
  hipLaunchKernelGGL(select_update_kernel, dim3(grid_for(Nv, 256)), dim3(256), 0, s, cand, Nv, state,
                     sum);
  return hipGetLastError();
}

hipError_t launch_select_final(const int32_t* state, const double* best, int32_t* n_sel_out,
                               double* score_out, hipStream_t s) {
  hipLaunchKernelGGL(select_final_kernel, dim3(1), dim3(1), 0, s, state, best, n_sel_out, score_out);
  return hipGetLastError();
}

}  // namespace tabpack
