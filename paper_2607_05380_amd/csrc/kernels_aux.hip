// Non-GEMM kernels of the packed MLP step on gfx950: the linear head with the
// loss and its gradient, column sweeps for bias gradients, the packed AdamW
// update, validation scoring and greedy ensemble selection.
//
// Reductions use wave64 shuffles and fixed-order LDS trees so that every
// result is bit-reproducible run to run (no float atomics anywhere).
#include <math.h>

#include "pack_internal.h"
#include "adamw.h"
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
// 8 consecutive activations (one 16-byte bf16 vector, two fp32 vectors).
template <typename T>
struct Vec8;
template <>
struct Vec8<__bf16> {
  __device__ static void load(const __bf16* p, float (&x)[8]) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static void store(__bf16* p, const float (&x)[8]) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[2 * i]) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[2 * i + 1]) << 16);
    *reinterpret_cast<uint4*>(p) = uint4{w[0], w[1], w[2], w[3]};
  }
};
template <>
struct Vec8<float> {
  __device__ static void load(const float* p, float (&x)[8]) {
    const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
  __device__ static void store(float* p, const float (&x)[8]) {
    *reinterpret_cast<float4*>(p) = float4{x[0], x[1], x[2], x[3]};
    *reinterpret_cast<float4*>(p + 4) = float4{x[4], x[5], x[6], x[7]};
  }
};

// Y = H_L[row] . W_out^T + b_out for 8 rows per wave (8 lanes per row, each
// lane a 16-byte column vector per step), then, by MODE: the training loss and
// dLoss/dY of the row (kHeadTrain); the score-ready eval value (kHeadEval:
// output, P(class 1) or P(true class)) at pred[k * Nv + row_base + row]; or
// all d_out prediction values (kHeadPredict: outputs, P(class 1) or the softmax
// probabilities) at pred[((blockIdx.y * Nv) + row_base + row) * d_out + o].
// D >= d_out is the output count rounded up to a power of two.  H is the start
// of the activation buffers; member k reads its last hidden layer at H + h_last.
template <typename T, int MODE, int D>
__global__ __launch_bounds__(256) void head_fwd_kernel(Task task, const T* H, const float* theta,
                                                       const MemberDev* mem, int Bp, int d_out,
                                                       const void* y, const int32_t* idx, int B,
                                                       int rows_valid, int64_t row_base, int64_t Nv,
                                                       float* dY, float* rowloss, float* pred,
                                                       const int32_t* members) {
  const int k = members ? members[blockIdx.y] : (int)blockIdx.y;
  const int lane = threadIdx.x & 63, sub = lane & 7;
  const int row = blockIdx.x * 32 + (threadIdx.x >> 3);
  if (row >= Bp) return;  // Bp is a multiple of 32: whole 8-lane groups leave together
  const MemberDev md = mem[k];
  const T* h = H + md.h_last + (int64_t)row * md.dp;
  const float* Wo = theta + md.w_out_off;
  float acc[D];
#pragma unroll
  for (int o = 0; o < D; ++o) acc[o] = 0.0f;
  // unrolled so that several rows' loads are in flight at once (the loop is
  // latency-bound otherwise: one 16-byte load per lane per iteration)
#pragma unroll 4
  for (int c = sub * 8; c < md.dp; c += 64) {
    float x[8];
    Vec8<T>::load(h + c, x);
#pragma unroll
    for (int o = 0; o < D; ++o) {
      if (o >= d_out) break;
      const float4 w0 = *reinterpret_cast<const float4*>(Wo + (int64_t)o * md.dp + c);
      const float4 w1 = *reinterpret_cast<const float4*>(Wo + (int64_t)o * md.dp + c + 4);
      acc[o] += ((x[0] * w0.x + x[1] * w0.y) + (x[2] * w0.z + x[3] * w0.w)) +
                ((x[4] * w1.x + x[5] * w1.y) + (x[6] * w1.z + x[7] * w1.w));
    }
  }
  float z[kMaxOut];
#pragma unroll
  for (int o = 0; o < kMaxOut; ++o) z[o] = 0.0f;
#pragma unroll
  for (int o = 0; o < D; ++o) {
    float v = acc[o];
    v += __shfl_xor(v, 1, 64);
    v += __shfl_xor(v, 2, 64);
    v += __shfl_xor(v, 4, 64);
    if (o < d_out) z[o] = v + theta[md.b_out_off + o];
  }
  if (sub != 0) return;

  constexpr bool EVAL = MODE != kHeadTrain;
  const bool valid = EVAL ? row < rows_valid : row < B;
  int64_t src = 0;
  if (valid) src = EVAL ? row_base + row : (int64_t)idx[(int64_t)k * B + row];
  if constexpr (MODE == kHeadPredict) {
    if (!valid) return;
    float* out = pred + ((int64_t)blockIdx.y * Nv + row_base + row) * d_out;
    if (task == Task::REG) {
      for (int o = 0; o < d_out; ++o) out[o] = z[o];
    } else if (task == Task::BIN) {
      out[0] = 1.0f / (1.0f + expf(-z[0]));
    } else {
      float mx = z[0];
      for (int o = 1; o < d_out; ++o) mx = fmaxf(mx, z[o]);
      float se = 0.0f;
      for (int o = 0; o < d_out; ++o) se += expf(z[o] - mx);
      for (int o = 0; o < d_out; ++o) out[o] = expf(z[o] - mx) / se;
    }
    return;
  }
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

// CPT consecutive activations of one row.
template <typename T, int CPT>
struct VecN;
template <typename T>
struct VecN<T, 8> {
  __device__ static void load(const T* p, float (&x)[8]) { Vec8<T>::load(p, x); }
  __device__ static void store(T* p, const float (&x)[8]) { Vec8<T>::store(p, x); }
};
template <>
struct VecN<__bf16, 4> {
  __device__ static void load(const __bf16* p, float (&x)[4]) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    x[0] = __uint_as_float(u.x << 16);
    x[1] = __uint_as_float(u.x & 0xFFFF0000u);
    x[2] = __uint_as_float(u.y << 16);
    x[3] = __uint_as_float(u.y & 0xFFFF0000u);
  }
  __device__ static void store(__bf16* p, const float (&x)[4]) {
    const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[0]) |
                        ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[1]) << 16);
    const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[2]) |
                        ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[3]) << 16);
    *reinterpret_cast<uint2*>(p) = uint2{lo, hi};
  }
};
template <>
struct VecN<float, 4> {
  __device__ static void load(const float* p, float (&x)[4]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  }
  __device__ static void store(float* p, const float (&x)[4]) {
    *reinterpret_cast<float4*>(p) = float4{x[0], x[1], x[2], x[3]};
  }
};

// Head backward over one (member, 32*CPT columns, RB rows) block:
//   dH_L = dY W_out, dZ_L = dH_L * [H_L > 0] * s_k (written out),
//   and this row block's partial sums of dW_out = dY^T H_L and db_L = sum dZ_L,
//   reduced over the block's 8 row slots in a fixed order and stored to part
//   (part[(rb * (d_out + 1) + o) * dp + c]; o = d_out holds db_L).
//   H and dZ are the starts of the activation buffers and of the dZ pair; a
//   member's L is its own depth (H + h_last, dZ + dz_last).
template <typename T, int D, int CPT>
__global__ __launch_bounds__(256) void head_bwd_kernel(const T* H, const float* theta, const MemberDev* mem,
                                                       const HeadTile* tiles, int Bp, int d_out, int RB,
                                                       const float* dY, T* dZ, float* part) {
  __shared__ float red[8][32 * CPT];
  const HeadTile ht = tiles[blockIdx.x];
  const MemberDev md = mem[ht.member];
  const int cv = threadIdx.x & 31, slot = threadIdx.x >> 5;
  const int c = ht.c0 + cv * CPT;
  const bool valid = c < md.dp;
  float wo[D][CPT], accw[D][CPT], accb[CPT];
#pragma unroll
  for (int o = 0; o < D; ++o)
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      wo[o][j] = (valid && o < d_out) ? theta[md.w_out_off + (int64_t)o * md.dp + c + j] : 0.0f;
      accw[o][j] = 0.0f;
    }
#pragma unroll
  for (int j = 0; j < CPT; ++j) accb[j] = 0.0f;
  const T* h = H + md.h_last;
  T* dz = dZ + md.dz_last;
  const float* dyk = dY + (int64_t)ht.member * Bp * d_out;
  const int r1 = min(ht.r0 + RB, Bp);
  // unrolled so that several rows' loads are in flight at once
#pragma unroll 4
  for (int r = ht.r0 + slot; r < r1; r += 8) {
    float dy[D];
#pragma unroll
    for (int o = 0; o < D; ++o) dy[o] = o < d_out ? dyk[(int64_t)r * d_out + o] : 0.0f;
    if (!valid) continue;
    float hv[CPT], g[CPT];
    VecN<T, CPT>::load(h + (int64_t)r * md.dp + c, hv);
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      float dh = 0.0f;
#pragma unroll
      for (int o = 0; o < D; ++o) {
        dh += dy[o] * wo[o][j];
        accw[o][j] += dy[o] * hv[j];
      }
      g[j] = hv[j] > 0.0f ? dh * md.drop_s : 0.0f;
      accb[j] += g[j];
    }
    VecN<T, CPT>::store(dz + (int64_t)r * md.dp + c, g);
  }
  // fixed-order reduction over the 8 row slots, one quantity at a time
  float* pk = part + (int64_t)(Bp / RB) * (d_out + 1) * (md.act_off / Bp);
  const int rb = ht.r0 / RB;
  for (int o = 0; o <= d_out; ++o) {
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      float v = accb[j];  // o == d_out: the bias partial
#pragma unroll
      for (int oo = 0; oo < D; ++oo)
        if (oo == o && o < d_out) v = accw[oo][j];
      red[slot][cv * CPT + j] = v;
    }
    __syncthreads();
    const int cc = threadIdx.x;  // one column of the block per thread
    if (cc < 32 * CPT && ht.c0 + cc < md.dp) {
      const float v = ((red[0][cc] + red[1][cc]) + (red[2][cc] + red[3][cc])) +
                      ((red[4][cc] + red[5][cc]) + (red[6][cc] + red[7][cc]));
      pk[((int64_t)rb * (d_out + 1) + o) * md.dp + ht.c0 + cc] = v;
    }
    __syncthreads();
  }
}

// sum over i < ceil(n / step) of term(i), added in order of i; the terms are
// fetched 8 at a time before they are added, so their loads overlap
template <typename V, typename F>
__device__ __forceinline__ V sum_in_order(int n, int step, F term) {
  const int m = n <= 0 ? 0 : (n + step - 1) / step;
  V s = 0;
  int i = 0;
  for (; i + 8 <= m; i += 8) {
    V v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = term(i + u);
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; i < m; ++i) s += term(i);
  return s;
}

// The gradient sums of a member group, one wave per ColTile (fixed orders):
//   part >= 0: db_{part+1}[c] = sum over the 64-row blocks of the dX
//     epilogue's column partials (bias layer part at colpart + part * part_stride);
//   kSumHead:  dW_out[o][c] and db_L[c] = sums over the head backward's row blocks;
//   kSumLoss:  the batch-mean loss of the member (fp64 over its B rows) and
//     db_out[o] = sum of dY over the rows (fp64).
__global__ __launch_bounds__(256) void grad_sums_kernel(const float* colpart, int64_t part_stride,
                                                        const float* headpart, int RB, const float* rowloss,
                                                        const float* dY, const MemberDev* mem, const ColTile* tiles,
                                                        int ntiles, int Bp, int B, int d_out,
                                                        const int64_t* bias_off, int K, float* grad,
                                                        float* loss_out) {
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= ntiles) return;
  const ColTile ct = tiles[w];
  const MemberDev md = mem[ct.member];
  const int lane = threadIdx.x & 63;
  if (ct.part == kSumLoss) {
    const int64_t r0 = (int64_t)ct.member * Bp;
    const double s =
        wave_sum_d(sum_in_order<double>(B - lane, 64, [&](int i) { return (double)rowloss[r0 + lane + 64 * i]; }));
    if (lane == 0) loss_out[ct.member] = (float)(s / (double)B);
    for (int o = 0; o < d_out; ++o) {
      const double g = wave_sum_d(
          sum_in_order<double>(B - lane, 64, [&](int i) { return (double)dY[(r0 + lane + 64 * i) * d_out + o]; }));
      if (lane == 0) grad[md.b_out_off + o] = (float)g;
    }
    return;
  }
  const int c = ct.c0 + lane;
  if (c >= md.dp) return;
  if (ct.part == kSumHead) {
    const int nrb = Bp / RB;
    const float* pk = headpart + (int64_t)nrb * (d_out + 1) * (md.act_off / Bp);
    for (int o = 0; o <= d_out; ++o) {
      const float v =
          sum_in_order<float>(nrb, 1, [&](int rb) { return pk[((int64_t)rb * (d_out + 1) + o) * md.dp + c]; });
      if (o < d_out)
        grad[md.w_out_off + (int64_t)o * md.dp + c] = v;
      else
        grad[md.b_last_off + c] = v;
    }
    return;
  }
  const float* p = colpart + ct.part * part_stride + md.act_off / kPartRows;
  grad[bias_off[(int64_t)ct.part * K + ct.member] + c] =
      sum_in_order<float>(Bp / kPartRows, 1, [&](int r) { return p[(int64_t)r * md.dp + c]; });
}

// ----------------------------------------------------------------- gather --
// H_0 of member k, row r: the feature row X[idx[k * B + r]] (or X[row_base + r]
// for contiguous rows) in the GEMM precision, zero-padded to Pin columns; rows
// r >= rows_valid are zero.  One wave per row, float4 reads.
template <typename T>
__global__ __launch_bounds__(256) void gather_kernel(const float* X, int d_in, int Pin, const int32_t* idx,
                                                     int B, int64_t row_base, int rows_valid, int Bp, T* H0,
                                                     const int32_t* members) {
  const int k = members ? members[blockIdx.y] : (int)blockIdx.y;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= Bp) return;
  T* dst = H0 + ((int64_t)k * Bp + r) * Pin;
  const bool valid = r < rows_valid;
  const int64_t src = valid ? (idx ? (int64_t)idx[(int64_t)k * B + r] : row_base + r) : 0;
  const float* x = X + src * d_in;
  const bool vec = (d_in % 4 == 0) && ((reinterpret_cast<uintptr_t>(X) & 15) == 0);
  // 1024 columns per round: the lane's four 16-byte loads are all issued
  // before any store; X rows are read once, so the loads bypass the caches
  for (int c0 = 0; c0 < Pin; c0 += 1024) {
    float v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + u * 256 + lane * 4;
      if (valid && vec && c + 4 <= d_in) {
        const f32x4 q = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(x + c));
        v[u][0] = q[0], v[u][1] = q[1], v[u][2] = q[2], v[u][3] = q[3];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[u][e] = (valid && c + e < d_in) ? x[c + e] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + u * 256 + lane * 4;
      if (c >= Pin) continue;
      if constexpr (sizeof(T) == 2) {
        const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[u][0]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[u][1]) << 16);
        const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[u][2]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[u][3]) << 16);
        *reinterpret_cast<u32x2*>(dst + c) = u32x2{lo, hi};
      } else {
        *reinterpret_cast<f32x4*>(dst + c) = f32x4{v[u][0], v[u][1], v[u][2], v[u][3]};
      }
    }
  }
}

// -------------------------------------------------------------- idx check --
// The batch indices come from the caller: every entry outside [0, N) is
// replaced by row 0 in the copy the step's kernels read, and flags bit 0 of
// the status word, so that no kernel ever reads outside X or y.  The flag
// store is predicated on a per-lane condition (a plain vector store; every
// writer stores the same value).
__global__ __launch_bounds__(256) void idx_check_kernel(const int32_t* __restrict__ idx, int64_t n, int64_t N,
                                                        int32_t* __restrict__ out, uint32_t* status) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int32_t v = idx[i];
  const bool bad = v < 0 || (int64_t)v >= N;
  out[i] = bad ? 0 : v;
  if (bad) status[0] = 1u;
}

// ----------------------------------------------------------- stream copy --
// dst <- src in 16-byte vectors with non-temporal loads and stores (the
// access pattern of the optimizer epilogues): a kernel of known HBM traffic
// for calibrating hardware byte counters and the achievable streaming rate.
// Each thread keeps four vectors in flight.
__global__ __launch_bounds__(256) void stream_copy_kernel(const f32x4* __restrict__ src, f32x4* __restrict__ dst,
                                                          int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    f32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
  }
  for (; i < n; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// ------------------------------------------------------------------ AdamW --
// One wave per 256-element chunk of the packed parameter buffer; every chunk
// belongs to one member and is all-weight or all-bias, so (lr_k, wd_k) and the
// decay switch are wave-uniform.  float4 loads/stores, 30 bytes per element
// with the bf16 shadow.
template <bool SHADOW>
__global__ __launch_bounds__(256) void adamw_kernel(float* theta, const float* grad, float* m,
                                                    float* v, uint16_t* shadow,
                                                    const uint32_t* chunk_tab, const uint32_t* list,
                                                    const MemberDev* mem, int64_t nchunks, AdamConst ac) {
  const int lane = threadIdx.x & 63;
  const int64_t nw = (int64_t)gridDim.x * 4;
  const int64_t w0 = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int64_t w = w0; w < nchunks; w += nw) {
    const int64_t c = list ? (int64_t)list[w] : w;
    const uint32_t e = chunk_tab[c];
    const MemberDev md = mem[e & 0x7FFFFFFFu];
    const float decay = (e >> 31) ? 1.0f : 1.0f - md.lr * md.wd;
    const float step = md.lr / ac.bc1;
    const int64_t i = c * kChunk + lane * 4;
    f32x4 th = *reinterpret_cast<const f32x4*>(theta + i);
    const f32x4 g = *reinterpret_cast<const f32x4*>(grad + i);
    f32x4 mm = *reinterpret_cast<const f32x4*>(m + i);
    f32x4 vv = *reinterpret_cast<const f32x4*>(v + i);
    adamw_vec4(th, g, mm, vv, decay, step, ac);
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

// xb row r = X row r in bf16, zero-padded from d_in to Pin columns: one
// thread per 8 output columns (one 16-byte store).
__global__ __launch_bounds__(256) void rows_to_bf16_kernel(const float* X, int64_t N, int d_in, int Pin,
                                                           __bf16* xb) {
  const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int vpr = Pin / 8;
  if (v >= N * vpr) return;
  const int64_t r = v / vpr;
  const int c0 = (int)(v - r * vpr) * 8;
  const float* x = X + r * d_in;
  uint32_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = c0 + 2 * q;
    const float a = c < d_in ? x[c] : 0.0f, b = c + 1 < d_in ? x[c + 1] : 0.0f;
    w[q] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)a) | ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)b) << 16);
  }
  *reinterpret_cast<uint4*>(xb + r * Pin + c0) = uint4{w[0], w[1], w[2], w[3]};
}

__global__ void to_shadow_kernel(const float* theta, uint16_t* shadow, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    shadow[i] = __builtin_bit_cast(uint16_t, (__bf16)theta[i]);
}

// ------------------------------------------------------------ eval scores --
__global__ __launch_bounds__(256) void eval_score_kernel(Task task, const float* pred,
                                                         const void* yv, int64_t Nv,
                                                         double* score_out, const int32_t* members) {
  __shared__ double sh[4];
  const int k = members ? members[blockIdx.x] : (int)blockIdx.x;
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < Nv; i += 256) s += row_score(task, (double)pred[k * Nv + i], yv, i);
  s = block_sum_d(s, sh);
  if (threadIdx.x == 0) score_out[k] = finish_score(task, s, Nv);
}

// Keep word of a dropout mask: bit r is set iff row 32*rb + r of column c is
// kept, i.e. the 16-bit half (r & 1) of word ((r >> 1) & 3) of Philox block
// (4 rb + r / 8, c, c2, step) is >= t: one block decides 8 rows, four blocks a
// word.  The training path (dropout_words_kernel -> forward epilogue) and the
// test hook below both go through this function.
__device__ __forceinline__ uint32_t keep_word(uint32_t key0, uint32_t key1, uint32_t step, uint32_t c2, int rb,
                                              int c, uint32_t t) {
  uint32_t w = 0;
#pragma unroll 2
  for (int b = 0; b < 4; ++b) {
    const Words4 x = philox4x32_10((uint32_t)(rb * 4 + b), (uint32_t)c, c2, step, key0, key1);
    const uint32_t q[4] = {x.w0, x.w1, x.w2, x.w3};
#pragma unroll
    for (int i = 0; i < 4; ++i)  // rows 8 b + 2 i (low half) and 8 b + 2 i + 1 (high half)
      w |= (((uint32_t)((q[i] & 0xFFFFu) >= t)) | ((uint32_t)((q[i] >> 16) >= t) << 1)) << (8 * b + 2 * i);
  }
  return w;
}

// Keep words of every hidden layer of every member for one training step:
// word (rb, c) of layer l, member k at out[(l-1)*A32 + act_off/32 + rb*dp + c].
// Rows >= rows_valid and columns >= width get 0 (the epilogue zeroes them).
__global__ __launch_bounds__(256) void dropout_words_kernel(uint32_t key0, uint32_t key1, uint32_t step,
                                                            const MemberDev* mem, int Bp, int rows_valid,
                                                            int64_t A32, uint32_t* out, const int32_t* members) {
  const int k = members ? members[blockIdx.y] : (int)blockIdx.y, l = blockIdx.z + 1;
  const MemberDev md = mem[k];
  if (l > md.depth) return;  // the member has no layer l
  const int64_t nw = (int64_t)(Bp / 32) * md.dp;
  const int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (w >= nw) return;
  const int rb = (int)(w / md.dp), c = (int)(w % md.dp);
  uint32_t word = 0;
  if (rb * 32 < rows_valid && c < md.width)
    word = md.drop_t == 0u ? ~0u : keep_word(key0, key1, step, ((uint32_t)k << 8) | (uint32_t)l, rb, c, md.drop_t);
  out[(int64_t)(l - 1) * A32 + md.act_off / 32 + w] = word;
}

// Test hook: the keep mask of one (layer, member) as bytes [B, width].
__global__ void dropout_mask_kernel(uint32_t key0, uint32_t key1, uint32_t step, int layer,
                                    int member, uint32_t t, int B, int width, uint8_t* out) {
  const int64_t n = (int64_t)((B + 31) / 32) * width;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int rb = (int)(i / width), c = (int)(i % width);
    const uint32_t w = keep_word(key0, key1, step, ((uint32_t)member << 8) | (uint32_t)layer, rb, c, t);
    for (int r = 0; r < 32 && rb * 32 + r < B; ++r) out[(int64_t)(rb * 32 + r) * width + c] = (w >> r) & 1;
  }
}

// --------------------------------------------------------- greedy select --
// state[0] = ensemble size n, state[1] = stopped flag, state[2] = this
// iteration's pick (-1 if none).  sum[i] = running fp64 sum of the picked
// candidates' values on row i.
constexpr int kSelRows = 1024;  // rows per workgroup of the candidate sweep

// Candidate sweep of one greedy iteration: workgroup (rb, c) sums candidate c's
// per-row scores of the extended ensemble (sum + q_c) / (n + 1) over rows
// 1024 rb .. 1024 rb + 1023 in a fixed order into partial[c * nblk + rb].
// (Measured alternatives: 4 candidates per workgroup with every load issued
// up front, 20 us per sweep of 96 x 70,000 against 16.5 us for this one.)
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

// Pick of one greedy iteration, one 1024-thread workgroup: wave w takes the
// candidates c = w, w + 16, ... in batches of kPickBatch whose partial loads are
// all issued before any is summed (lane-strided over the row blocks, then a
// fixed shuffle tree: the same order for every candidate); the already picked
// candidates are marked in an LDS bit set (C <= 65535).
constexpr int kPickWaves = 16, kPickBatch = 8;
__global__ __launch_bounds__(1024) void select_pick_kernel(Task task, int C, int64_t Nv, int m_ens,
                                                           const double* partial, int nblk,
                                                           int32_t* state, double* best,
                                                           int32_t* sel) {
  __shared__ double wbs[kPickWaves];
  __shared__ int wbi[kPickWaves];
  __shared__ uint32_t taken_bits[2048];
  if (state[1]) {
    if (threadIdx.x == 0) state[2] = -1;
    return;
  }
  const int n = state[0];
  for (int j = threadIdx.x; j < 2048; j += 1024) taken_bits[j] = 0u;
  __syncthreads();
  for (int j = threadIdx.x; j < n; j += 1024) {
    const int c = sel[j];
    atomicOr(&taken_bits[c >> 5], 1u << (c & 31));
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double bs = INFINITY;
  int bi = 0x7FFFFFFF;
  for (int c0 = w; c0 < C; c0 += kPickWaves * kPickBatch) {
    double tot[kPickBatch];
#pragma unroll
    for (int u = 0; u < kPickBatch; ++u) {
      const int c = c0 + u * kPickWaves;
      tot[u] = 0.0;
      if (c < C)
        for (int b = lane; b < nblk; b += 64) tot[u] += partial[(int64_t)c * nblk + b];
    }
#pragma unroll
    for (int u = 0; u < kPickBatch; ++u) {
      const int c = c0 + u * kPickWaves;
      const double t = wave_sum_d(tot[u]);
      if (c >= C) continue;
      const bool taken = (taken_bits[c >> 5] >> (c & 31)) & 1u;
      const double sc = taken ? INFINITY : finish_score(task, t, Nv);
      if (sc < bs || (sc == bs && c < bi)) {
        bs = sc;
        bi = c;
      }
    }
  }
  if (lane == 0) {
    wbs[w] = bs;
    wbi[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = wbs[0];
    int c = wbi[0];
    for (int k = 1; k < kPickWaves; ++k)
      if (wbs[k] < s || (wbs[k] == s && wbi[k] < c)) {
        s = wbs[k];
        c = wbi[k];
      }
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

// Ensemble prediction of one row chunk: out[(row_base + r) * d_out + o] is the
// mean over the n member predictions part[(i * Bp + r) * d_out + o], summed in
// member order in fp64.
__global__ __launch_bounds__(256) void ensemble_mean_kernel(const float* part, int n, int Bp, int rows, int d_out,
                                                            int64_t row_base, float* out) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)rows * d_out) return;
  const int64_t stride = (int64_t)Bp * d_out;
  double s = 0.0;
  for (int i = 0; i < n; ++i) s += (double)part[i * stride + e];
  out[row_base * d_out + e] = (float)(s / n);
}

inline int grid_for(int64_t n, int per) {
  int64_t g = (n + per - 1) / per;
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (int)g;
}

}  // namespace

int select_blocks(int64_t Nv) { return (int)((Nv + kSelRows - 1) / kSelRows); }

namespace {
template <typename T, int MODE, int D>
void head_fwd_t(dim3 grid, hipStream_t s, Task task, const void* H, const float* theta, const MemberDev* mem,
                int Bp, int d_out, const void* y, const int32_t* idx, int B, int rows_valid, int64_t row_base,
                int64_t Nv, float* dY, float* rowloss, float* pred, const int32_t* members) {
  hipLaunchKernelGGL((head_fwd_kernel<T, MODE, D>), grid, dim3(256), 0, s, task, static_cast<const T*>(H), theta,
                     mem, Bp, d_out, y, idx, B, rows_valid, row_base, Nv, dY, rowloss, pred, members);
}

template <typename T, int MODE>
void head_fwd_d(int d_out, dim3 grid, hipStream_t s, Task task, const void* H, const float* theta,
                const MemberDev* mem, int Bp, const void* y, const int32_t* idx, int B, int rows_valid,
                int64_t row_base, int64_t Nv, float* dY, float* rowloss, float* pred, const int32_t* members) {
#define TABPACK_HEAD_FWD(DD)                                                                                   \
  head_fwd_t<T, MODE, DD>(grid, s, task, H, theta, mem, Bp, d_out, y, idx, B, rows_valid, row_base, Nv, dY, \
                          rowloss, pred, members)
  if (d_out <= 1) TABPACK_HEAD_FWD(1);
  else if (d_out <= 2) TABPACK_HEAD_FWD(2);
  else if (d_out <= 4) TABPACK_HEAD_FWD(4);
  else if (d_out <= 8) TABPACK_HEAD_FWD(8);
  else TABPACK_HEAD_FWD(16);
#undef TABPACK_HEAD_FWD
}

}  // namespace

hipError_t launch_head_fwd(Prec prec, Task task, int mode, const void* H, const float* theta,
                           const MemberDev* mem, int K, int Bp, int d_out, const void* y,
                           const int32_t* idx, int B, int rows_valid, int64_t row_base, int64_t Nv,
                           float* dY, float* rowloss, float* pred, const int32_t* members, hipStream_t s) {
  if (Bp % 32 != 0 || d_out < 1 || d_out > kMaxOut || mode < kHeadTrain || mode > kHeadPredict)
    return hipErrorInvalidValue;
  if (K <= 0) return hipSuccess;
  const dim3 grid(Bp / 32, K);
#define TABPACK_HEAD_FWD_MODE(TT, MM)                                                                         \
  head_fwd_d<TT, MM>(d_out, grid, s, task, H, theta, mem, Bp, y, idx, B, rows_valid, row_base, Nv, dY, rowloss, \
                     pred, members)
  if (prec == Prec::BF16) {
    if (mode == kHeadTrain) TABPACK_HEAD_FWD_MODE(__bf16, kHeadTrain);
    else if (mode == kHeadEval) TABPACK_HEAD_FWD_MODE(__bf16, kHeadEval);
    else TABPACK_HEAD_FWD_MODE(__bf16, kHeadPredict);
  } else {
    if (mode == kHeadTrain) TABPACK_HEAD_FWD_MODE(float, kHeadTrain);
    else if (mode == kHeadEval) TABPACK_HEAD_FWD_MODE(float, kHeadEval);
    else TABPACK_HEAD_FWD_MODE(float, kHeadPredict);
  }
#undef TABPACK_HEAD_FWD_MODE
  return hipGetLastError();
}

namespace {
template <typename T>
void head_bwd_d(int d_out, int ntiles, hipStream_t s, const void* H, const float* theta, const MemberDev* mem,
                const HeadTile* tiles, int Bp, int RB, const float* dY, void* dZ, float* part) {
#define TABPACK_HEAD_BWD(DD, CC)                                                                             \
  hipLaunchKernelGGL((head_bwd_kernel<T, DD, CC>), dim3(ntiles), dim3(256), 0, s, static_cast<const T*>(H), \
                     theta, mem, tiles, Bp, d_out, RB, dY, static_cast<T*>(dZ), part)
  if (d_out <= 1) TABPACK_HEAD_BWD(1, 8);
  else if (d_out <= 2) TABPACK_HEAD_BWD(2, 8);
  else if (d_out <= 4) TABPACK_HEAD_BWD(4, 8);
  else if (d_out <= 8) TABPACK_HEAD_BWD(8, 4);
  else TABPACK_HEAD_BWD(16, 4);
#undef TABPACK_HEAD_BWD
}
}  // namespace

int head_bwd_cols(int d_out) { return d_out <= 4 ? 256 : 128; }


hipError_t launch_head_bwd(Prec prec, const void* H, const float* theta, const MemberDev* mem,
                           const HeadTile* tiles, int ntiles, int Bp, int RB, int d_out, const float* dY,
                           void* dZ, float* part, hipStream_t s) {
  if (RB <= 0 || Bp % RB != 0 || d_out < 1 || d_out > kMaxOut) return hipErrorInvalidValue;
  if (ntiles <= 0) return hipSuccess;
  if (prec == Prec::BF16)
    head_bwd_d<__bf16>(d_out, ntiles, s, H, theta, mem, tiles, Bp, RB, dY, dZ, part);
  else
    head_bwd_d<float>(d_out, ntiles, s, H, theta, mem, tiles, Bp, RB, dY, dZ, part);
  return hipGetLastError();
}


hipError_t launch_grad_sums(const float* colpart, int64_t part_stride, const float* headpart, int RB,
                            const float* rowloss, const float* dY, const MemberDev* mem, const ColTile* tiles,
                            int ntiles, int Bp, int B, int d_out, const int64_t* bias_off, int K, float* grad,
                            float* loss_out, hipStream_t s) {
  if (RB <= 0 || Bp % RB != 0 || Bp % kPartRows != 0) return hipErrorInvalidValue;
  if (ntiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(grad_sums_kernel, dim3((ntiles + 3) / 4), dim3(256), 0, s, colpart, part_stride, headpart, RB,
                     rowloss, dY, mem, tiles, ntiles, Bp, B, d_out, bias_off, K, grad, loss_out);
  return hipGetLastError();
}

hipError_t launch_gather(Prec prec, const float* X, int d_in, int Pin, const int32_t* idx, int B,
                         int64_t row_base, int rows_valid, int members, int Bp, void* H0,
                         const int32_t* member_ids, hipStream_t s) {
  if (members <= 0) return hipSuccess;
  const dim3 grid((Bp + 3) / 4, members);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((gather_kernel<__bf16>), grid, dim3(256), 0, s, X, d_in, Pin, idx, B, row_base,
                       rows_valid, Bp, static_cast<__bf16*>(H0), member_ids);
  else
    hipLaunchKernelGGL((gather_kernel<float>), grid, dim3(256), 0, s, X, d_in, Pin, idx, B, row_base,
                       rows_valid, Bp, static_cast<float*>(H0), member_ids);
  return hipGetLastError();
}

hipError_t launch_idx_check(const int32_t* idx, int64_t n, int64_t N, int32_t* out, uint32_t* status,
                            hipStream_t s) {
  hipLaunchKernelGGL(idx_check_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, idx, n, N, out, status);
  return hipGetLastError();
}

hipError_t launch_stream_copy(const void* src, void* dst, int64_t n16, hipStream_t s) {
  // eight workgroups per CU, each thread streaming 16 bytes x 4 per round
  const int64_t blocks = std::min<int64_t>(grid_for(n16, 256), 256 * 8);
  hipLaunchKernelGGL(stream_copy_kernel, dim3(blocks), dim3(256), 0, s, static_cast<const f32x4*>(src),
                     static_cast<f32x4*>(dst), n16);
  return hipGetLastError();
}

hipError_t launch_adamw(Prec prec, float* theta, const float* grad, float* m, float* v,
                        uint16_t* shadow, const uint32_t* chunk_tab, const uint32_t* list,
                        const MemberDev* mem, int64_t nchunks, const AdamConst& ac, hipStream_t s) {
  if (nchunks <= 0) return hipSuccess;
  const int grid = grid_for(nchunks, 4);
  (void)prec;
  if (shadow)
    hipLaunchKernelGGL((adamw_kernel<true>), dim3(grid), dim3(256), 0, s, theta, grad, m, v, shadow,
                       chunk_tab, list, mem, nchunks, ac);
  else
    hipLaunchKernelGGL((adamw_kernel<false>), dim3(grid), dim3(256), 0, s, theta, grad, m, v, shadow,
                       chunk_tab, list, mem, nchunks, ac);
  return hipGetLastError();
}

hipError_t launch_ensemble_mean(const float* part, int n, int Bp, int rows, int d_out, int64_t row_base,
                                float* out, hipStream_t s) {
  if (n <= 0 || rows <= 0) return hipSuccess;
  const int64_t ne = (int64_t)rows * d_out;
  hipLaunchKernelGGL(ensemble_mean_kernel, dim3((unsigned)((ne + 255) / 256)), dim3(256), 0, s, part, n, Bp, rows,
                     d_out, row_base, out);
  return hipGetLastError();
}

hipError_t launch_rows_to_bf16(const float* X, int64_t N, int d_in, int Pin, void* xb, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (Pin % 8 || Pin < d_in) return hipErrorInvalidValue;
  const int64_t nv = N * (Pin / 8);
  hipLaunchKernelGGL(rows_to_bf16_kernel, dim3((unsigned)((nv + 255) / 256)), dim3(256), 0, s, X, N, d_in, Pin,
                     static_cast<__bf16*>(xb));
  return hipGetLastError();
}

hipError_t launch_to_shadow(const float* theta, uint16_t* shadow, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(to_shadow_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, theta, shadow, n);
  return hipGetLastError();
}

hipError_t launch_eval_score(Task task, const float* pred, const void* yv, int K, int64_t Nv,
                             double* score_out, const int32_t* members, hipStream_t s) {
  if (K <= 0) return hipSuccess;
  hipLaunchKernelGGL(eval_score_kernel, dim3(K), dim3(256), 0, s, task, pred, yv, Nv, score_out, members);
  return hipGetLastError();
}

hipError_t launch_dropout_mask(uint32_t key0, uint32_t key1, uint32_t step, int layer, int member,
                               uint32_t t, int B, int width, uint8_t* out, hipStream_t s) {
  hipLaunchKernelGGL(dropout_mask_kernel, dim3(grid_for((int64_t)((B + 31) / 32) * width, 256)), dim3(256), 0, s,
                     key0, key1, step, layer, member, t, B, width, out);
  return hipGetLastError();
}

hipError_t launch_dropout_words(uint32_t key0, uint32_t key1, uint32_t step, const MemberDev* mem, int K, int L,
                                int max_dp, int Bp, int rows_valid, int64_t A32, uint32_t* out,
                                const int32_t* members, hipStream_t s) {
  if (K <= 0) return hipSuccess;
  const int64_t nw = (int64_t)(Bp / 32) * max_dp;
  hipLaunchKernelGGL(dropout_words_kernel, dim3((unsigned)((nw + 255) / 256), K, L), dim3(256), 0, s, key0, key1, step,
                     mem, Bp, rows_valid, A32, out, members);
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
  hipLaunchKernelGGL(select_pick_kernel, dim3(1), dim3(1024), 0, s, task, C, Nv, m_ens, partial, nblk,
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
