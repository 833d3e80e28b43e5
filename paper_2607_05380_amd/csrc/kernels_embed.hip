// Periodic feature embeddings of the members (the paper's App. "Feature
// Embeddings"): feature x_i of a row becomes d_emb values
//   E[i d_emb]     = alpha_i0 x_i + beta_i0
//   E[i d_emb + j] = alpha_ij cos(w_i,j-1 x_i + b_i,j-1) + beta_ij   (j >= 1)
// and the first layer reads the row's d_in * d_emb values.  Each member has its
// own d_emb and parameters, so its embedded batch E [Bp, p_in] is written per
// step (GEMM precision) and read by the first-layer forward and weight-gradient
// GEMMs; the backward pass reduces dE [Bp, p_in] (fp32, from the first layer's
// data-gradient GEMM) over the rows into the parameters' gradients.
#include "pack_internal.h"

namespace tabpack {
namespace {

constexpr int kEmbRows = 64;  // rows per forward workgroup (the padded batch is a multiple)

template <typename T>
__device__ __forceinline__ T to_gemm(float x);
template <>
__device__ __forceinline__ __bf16 to_gemm<__bf16>(float x) {
  return (__bf16)x;
}
template <>
__device__ __forceinline__ float to_gemm<float>(float x) {
  return x;
}

// cos and sin of a phase phi (radians) for the bf16 packs: the hardware's
// v_cos_f32 / v_sin_f32 take revolutions, so t = phi / (2 pi) is reduced to
// [-1/2, 1/2] by subtracting the nearest integer first.  The error (about 1e-6
// absolute for phases up to a few hundred radians, most of it the rounding of
// t) is far below the bf16 rounding of the embedded values.  fp32 packs use
// cosf / sincosf.
__device__ __forceinline__ float revolutions(float phi) {
  const float t = phi * 0.15915494309189535f;
  return t - rintf(t);
}
template <bool FAST>
__device__ __forceinline__ float cos_of(float phi) {
  if constexpr (FAST)
    return __builtin_amdgcn_cosf(revolutions(phi));
  else
    return cosf(phi);
}
template <bool FAST>
__device__ __forceinline__ void sincos_of(float phi, float* sn, float* cs) {
  if constexpr (FAST) {
    const float t = revolutions(phi);
    *sn = __builtin_amdgcn_sinf(t);
    *cs = __builtin_amdgcn_cosf(t);
  } else {
    sincosf(phi, sn, cs);
  }
}

// Parameters of embedding column col (< d_in d_emb) of a member: feature i,
// position j, alpha, beta and (j >= 1) w, b.
struct EmbCol {
  int i, j;
  float a, be, w, b;
};
__device__ __forceinline__ EmbCol emb_col(const MemberDev& md, const float* theta, int col) {
  EmbCol e;
  e.i = col / md.d_emb;
  e.j = col - e.i * md.d_emb;
  e.a = theta[md.e_a + col];
  e.be = theta[md.e_be + col];
  e.w = e.b = 0.0f;
  if (e.j > 0) {
    const int64_t wi = (int64_t)e.i * (md.d_emb - 1) + e.j - 1;
    e.w = theta[md.e_w + wi];
    e.b = theta[md.e_b + wi];
  }
  return e;
}

// The features a workgroup's 256 columns starting at c0 read, [i0, i0 + nf):
// at most 255 / d_emb + 2 of them (d_emb >= 2).
constexpr int kEmbFeat = 130;
struct FeatRange {
  int i0, nf;
};
__device__ __forceinline__ FeatRange feat_range(int c0, int d_emb, int d_in) {
  const int i0 = c0 / d_emb;
  return FeatRange{i0, min(d_in - 1, (c0 + 255) / d_emb) - i0 + 1};
}

// xs[r][f] = x of feature i0 + f in row r of the chunk (zero for rows whose
// xrow is negative).
__device__ __forceinline__ void stage_features(const float* X, const int64_t* xrow, int nrows, FeatRange fr,
                                               float (*xs)[kEmbFeat]) {
  for (int e = threadIdx.x; e < nrows * fr.nf; e += 256) {
    const int r = e / fr.nf, f = e - r * fr.nf;
    const int64_t xo = xrow[r];
    xs[r][f] = xo >= 0 ? X[xo + fr.i0 + f] : 0.0f;
  }
}

// One workgroup per (256 columns, member, kEmbRows rows): the chunk's feature
// values are staged in LDS, each thread keeps its column's parameters in
// registers and writes the column down the rows (a row's 256 columns are one
// contiguous store per workgroup).
template <typename T, bool FAST>
__global__ __launch_bounds__(256) void embed_fwd_kernel(const float* X, int d_in, const int32_t* idx, int B,
                                                        int64_t row_base, int rows_valid, const MemberDev* mem,
                                                        const int32_t* members, const float* theta, T* E) {
  __shared__ int64_t xrow[kEmbRows];
  __shared__ float xs[kEmbRows][kEmbFeat];
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  const int c0 = blockIdx.x * 256;
  if (c0 >= md.p_in) return;  // uniform: past this member's columns
  const int r0 = blockIdx.z * kEmbRows;
  if (threadIdx.x < kEmbRows) {
    const int r = r0 + threadIdx.x;
    xrow[threadIdx.x] = r < rows_valid ? (idx ? (int64_t)idx[(int64_t)k * B + r] : row_base + r) * d_in : -1;
  }
  __syncthreads();
  const FeatRange fr = feat_range(min(c0, d_in * md.d_emb - 1), md.d_emb, d_in);
  stage_features(X, xrow, kEmbRows, fr, xs);
  __syncthreads();
  const int col = c0 + threadIdx.x;
  if (col >= md.p_in) return;
  const bool on = col < d_in * md.d_emb;  // else a padding column: zeros
  EmbCol e{0, 0, 0.0f, 0.0f, 0.0f, 0.0f};
  if (on) e = emb_col(md, theta, col);
  const int f = on ? e.i - fr.i0 : 0;
  T* out = E + md.e_act + (int64_t)r0 * md.p_in + col;
#pragma unroll 8
  for (int rr = 0; rr < kEmbRows; ++rr) {
    float v = 0.0f;
    if (on && xrow[rr] >= 0) {
      const float x = xs[rr][f];
      v = e.j == 0 ? e.a * x + e.be : e.a * cos_of<FAST>(e.w * x + e.b) + e.be;
    }
    out[(int64_t)rr * md.p_in] = to_gemm<T>(v);
  }
}

// One workgroup per (256 columns, member): each thread sums its column's four
// gradient terms over the batch rows in row order (fp32), reading dE one row of
// 256 columns at a time; the rows' data indices go through LDS 256 at a time.
// (Staging the feature values in LDS as the forward does, 64 rows per chunk,
// measured twice as slow: three barriers per chunk expose every load.)
template <bool FAST>
__global__ __launch_bounds__(256) void embed_bwd_kernel(const float* X, int d_in, const int32_t* idx, int B,
                                                        const MemberDev* mem, const int32_t* members,
                                                        const float* theta, const float* dE, float* grad) {
  __shared__ int64_t xrow[256];
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  if ((int)blockIdx.x * 256 >= md.p_in) return;  // uniform
  const int col = blockIdx.x * 256 + threadIdx.x;
  const bool on = col < d_in * md.d_emb;
  EmbCol e{0, 0, 0.0f, 0.0f, 0.0f, 0.0f};
  if (on) e = emb_col(md, theta, col);
  const float* de = dE + md.e_act + (on ? col : 0);
  float ga = 0.0f, gbe = 0.0f, gw = 0.0f, gb = 0.0f;
  for (int rc = 0; rc < B; rc += 256) {
    const int n = min(256, B - rc);
    __syncthreads();  // the previous chunk's indices are no longer read
    if ((int)threadIdx.x < n) xrow[threadIdx.x] = (int64_t)idx[(int64_t)k * B + rc + threadIdx.x] * d_in;
    __syncthreads();
    if (!on) continue;
#pragma unroll 8
    for (int rr = 0; rr < n; ++rr) {
      const float x = X[xrow[rr] + e.i];
      const float g = de[(int64_t)(rc + rr) * md.p_in];
      gbe += g;
      if (e.j == 0) {
        ga += g * x;
      } else {
        float sn, cs;
        sincos_of<FAST>(e.w * x + e.b, &sn, &cs);
        ga += g * cs;
        const float t = -g * e.a * sn;
        gb += t;
        gw += t * x;
      }
    }
  }
  if (!on) return;
  grad[md.e_a + col] = ga;
  grad[md.e_be + col] = gbe;
  if (e.j > 0) {
    const int64_t wi = (int64_t)e.i * (md.d_emb - 1) + e.j - 1;
    grad[md.e_w + wi] = gw;
    grad[md.e_b + wi] = gb;
  }
}

}  // namespace

hipError_t launch_embed_fwd(Prec prec, const float* X, int d_in, const int32_t* idx, int B, int64_t row_base,
                            int rows_valid, int Bp, const MemberDev* mem, const int32_t* members, int nmembers,
                            int max_pin, const float* theta, void* E, hipStream_t s) {
  if (nmembers <= 0 || max_pin <= 0) return hipSuccess;
  if (Bp % kEmbRows) return hipErrorInvalidValue;
  const dim3 grid((max_pin + 255) / 256, nmembers, Bp / kEmbRows);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((embed_fwd_kernel<__bf16, true>), grid, dim3(256), 0, s, X, d_in, idx, B, row_base,
                       rows_valid, mem, members, theta, static_cast<__bf16*>(E));
  else
    hipLaunchKernelGGL((embed_fwd_kernel<float, false>), grid, dim3(256), 0, s, X, d_in, idx, B, row_base,
                       rows_valid, mem, members, theta, static_cast<float*>(E));
  return hipGetLastError();
}

hipError_t launch_embed_bwd(Prec prec, const float* X, int d_in, const int32_t* idx, int B, const MemberDev* mem,
                            const int32_t* members, int nmembers, int max_pin, const float* theta, const float* dE,
                            float* grad, hipStream_t s) {
  if (nmembers <= 0 || max_pin <= 0) return hipSuccess;
  const dim3 grid((max_pin + 255) / 256, nmembers);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((embed_bwd_kernel<true>), grid, dim3(256), 0, s, X, d_in, idx, B, mem, members, theta, dE,
                       grad);
  else
    hipLaunchKernelGGL((embed_bwd_kernel<false>), grid, dim3(256), 0, s, X, d_in, idx, B, mem, members, theta, dE,
                       grad);
  return hipGetLastError();
}

}  // namespace tabpack
