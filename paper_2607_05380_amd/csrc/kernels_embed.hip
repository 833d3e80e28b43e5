// Periodic feature embeddings of the members (the paper's App. "Feature
// Embeddings"): feature x_i of a row becomes d_emb values
//   E[i d_emb]     = alpha_i0 x_i + beta_i0
//   E[i d_emb + j] = alpha_ij cos(w_i,j-1 x_i + b_i,j-1) + beta_ij   (j >= 1)
// and the first layer reads the row's d_in * d_emb values.  Each member has its
// own d_emb and parameters, so its embedded batch E [Bp, p_in] is written per
// step (GEMM precision) and read by the first-layer forward and weight-gradient
// GEMMs.  In the backward pass the first layer's data-gradient GEMM reduces
// dE = dZ_1 W_1 in its epilogue (fp32 accumulators) into per-64-row-block sums
// of the four gradient terms; embed_grad_kernel adds the blocks.
#include "emb_trig.h"
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
      v = e.j == 0 ? e.a * x + e.be : e.a * emb_cos<FAST>(e.w * x + e.b) + e.be;
    }
    out[(int64_t)rr * md.p_in] = to_gemm<T>(v);
  }
}

// The embedding parameters' gradients from the first layer's data-gradient
// GEMM: its epilogue leaves, per member, column and 64-row block pb, the four
// sums over the block's rows (alpha, beta, w, b terms) at
// part[e_act / 16 + (pb * 4 + q) * p_in + col]; here they are added over the
// blocks in block order.  One thread per (column, member).
__global__ __launch_bounds__(256) void embed_grad_kernel(int d_in, int nblk, const MemberDev* mem,
                                                         const int32_t* members, const float* part, float* grad) {
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= d_in * md.d_emb) return;
  const float* p = part + md.e_act / 16 + col;
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int pb = 0; pb < nblk; ++pb)
#pragma unroll
    for (int q = 0; q < 4; ++q) s[q] += p[(int64_t)(pb * 4 + q) * md.p_in];
  grad[md.e_a + col] = s[0];
  grad[md.e_be + col] = s[1];
  const int i = col / md.d_emb, j = col - i * md.d_emb;
  if (j > 0) {
    const int64_t wi = (int64_t)i * (md.d_emb - 1) + j - 1;
    grad[md.e_w + wi] = s[2];
    grad[md.e_b + wi] = s[3];
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

hipError_t launch_embed_grad(int d_in, int Bp, const MemberDev* mem, const int32_t* members, int nmembers,
                             int max_pin, const float* part, float* grad, hipStream_t s) {
  if (nmembers <= 0 || max_pin <= 0) return hipSuccess;
  if (Bp % 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_grad_kernel, dim3((max_pin + 255) / 256, nmembers), dim3(256), 0, s, d_in, Bp / 64, mem,
                     members, part, grad);
  return hipGetLastError();
}

}  // namespace tabpack
