// Periodic feature embeddings of the members (the paper's App. "Feature
// Embeddings"): feature x_i of a row becomes d_emb values
//   E[i d_emb]     = alpha_i0 x_i + beta_i0
//   E[i d_emb + j] = alpha_ij cos(w_i,j-1 x_i + b_i,j-1) + beta_ij   (j >= 1)
// and the first layer reads the row's d_in * d_emb values.  Each member has its
// own d_emb and parameters.  In the packed layout feature i owns the columns
// i dp .. i dp + dp - 1 of W_1 (dp = d_emb rounded up to 8; the last dp -
// d_emb are zero padding).  E is never stored: the first layer's forward and
// weight-gradient GEMMs produce it in their operand paths from the data rows
// and a per-member column table, built here from the parameters at the start
// of every step.  In the backward pass the first layer's data-gradient GEMM
// reduces dE = dZ_1 W_1 in its epilogue (fp32 accumulators) into
// per-64-row-block sums of the four gradient terms; embed_grad_kernel adds the
// blocks.
#include "pack_internal.h"

namespace tabpack {
namespace {

// Embedding column col of a member: feature i owns columns i dp .. i dp +
// dp - 1 (dp = d_emb rounded up to 8), position j = col - i dp; j >= d_emb is
// zero padding.  The parameters: alpha, beta [d_in, d_emb] and (j >= 1) w, b
// [d_in, d_emb - 1].
struct EmbCol {
  int i, j;
  bool real;
  float a, be, w, b;
};
__device__ __forceinline__ int emb_dp(int d_emb) { return (d_emb + 7) & ~7; }
__device__ __forceinline__ EmbCol emb_col(const MemberDev& md, const float* theta, int d_in, int col) {
  EmbCol e;
  const int dp = emb_dp(md.d_emb);
  e.i = col / dp;
  e.j = col - e.i * dp;
  e.real = e.i < d_in && e.j < md.d_emb;
  e.a = e.be = e.w = e.b = 0.0f;
  if (e.real) {
    const int64_t ai = (int64_t)e.i * md.d_emb + e.j;
    e.a = theta[md.e_a + ai];
    e.be = theta[md.e_be + ai];
    if (e.j > 0) {
      const int64_t wi = (int64_t)e.i * (md.d_emb - 1) + e.j - 1;
      e.w = theta[md.e_w + wi];
      e.b = theta[md.e_b + wi];
    }
  }
  return e;
}

// Column tables of the members' embeddings for the first-layer GEMMs that
// produce E in their operand paths: one thread per (column, member); entry c
// holds {w, b, alpha, beta} of column c (w = b = 0 at j = 0; zeros in the
// padding).  FAST (bf16 packs): w and b divided by 2 pi, so that w x + b is
// the phase in revolutions.
template <bool FAST>
__global__ __launch_bounds__(256) void embed_table_kernel(int d_in, const MemberDev* mem, const int32_t* members,
                                                          const float* theta, float4* tab) {
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= md.p_in) return;
  const EmbCol e = emb_col(md, theta, d_in, col);  // zeros in the padding
  constexpr float kInv2Pi = 0.15915494309189535f;
  tab[md.e_tab + col] = FAST ? make_float4(e.w * kInv2Pi, e.b * kInv2Pi, e.a, e.be) : make_float4(e.w, e.b, e.a, e.be);
}

// The embedding parameters' gradients from the first layer's data-gradient
// GEMM: its epilogue leaves, per member, real column and 64-row block pb, the
// four sums over the block's rows (alpha, beta, w, b terms) at
// part[e_act / 16 + (pb * 4 + q) * p_in + col]; here they are added over the
// blocks in block order.  One thread per (column, member).
__global__ __launch_bounds__(256) void embed_grad_kernel(int d_in, int nblk, const MemberDev* mem,
                                                         const int32_t* members, const float* part, float* grad) {
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= md.p_in) return;
  const int dp = emb_dp(md.d_emb), i = col / dp, j = col - i * dp;
  if (i >= d_in || j >= md.d_emb) return;  // padding column
  const float* p = part + md.e_act / 16 + col;
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int pb = 0; pb < nblk; ++pb)
#pragma unroll
    for (int q = 0; q < 4; ++q) s[q] += p[(int64_t)(pb * 4 + q) * md.p_in];
  const int64_t ai = (int64_t)i * md.d_emb + j;
  grad[md.e_a + ai] = s[0];
  grad[md.e_be + ai] = s[1];
  if (j > 0) {
    const int64_t wi = (int64_t)i * (md.d_emb - 1) + j - 1;
    grad[md.e_w + wi] = s[2];
    grad[md.e_b + wi] = s[3];
  }
}

}  // namespace

hipError_t launch_embed_table(Prec prec, int d_in, const MemberDev* mem, const int32_t* members, int nmembers,
                              int max_pin, const float* theta, float4* tab, hipStream_t s) {
  if (nmembers <= 0 || max_pin <= 0) return hipSuccess;
  const dim3 grid((max_pin + 255) / 256, nmembers);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL(embed_table_kernel<true>, grid, dim3(256), 0, s, d_in, mem, members, theta, tab);
  else
    hipLaunchKernelGGL(embed_table_kernel<false>, grid, dim3(256), 0, s, d_in, mem, members, theta, tab);
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
