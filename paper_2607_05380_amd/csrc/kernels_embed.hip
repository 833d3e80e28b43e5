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

// One workgroup per (row, member); threads stride over the row's columns.
template <typename T>
__global__ __launch_bounds__(256) void embed_fwd_kernel(const float* X, int d_in, const int32_t* idx, int B,
                                                        int64_t row_base, int rows_valid, const MemberDev* mem,
                                                        const int32_t* members, const float* theta, T* E) {
  const int r = blockIdx.x;
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  T* out = E + md.e_act + (int64_t)r * md.p_in;
  const int ncol = d_in * md.d_emb;
  const bool valid = r < rows_valid;
  const float* xr = nullptr;
  if (valid) xr = X + (idx ? (int64_t)idx[(int64_t)k * B + r] : row_base + r) * d_in;
  for (int col = threadIdx.x; col < md.p_in; col += 256) {
    float v = 0.0f;
    if (valid && col < ncol) {
      const int i = col / md.d_emb, j = col - i * md.d_emb;
      const float x = xr[i];
      const float a = theta[md.e_a + col], be = theta[md.e_be + col];
      if (j == 0) {
        v = a * x + be;
      } else {
        const int64_t wi = (int64_t)i * (md.d_emb - 1) + j - 1;
        v = a * cosf(theta[md.e_w + wi] * x + theta[md.e_b + wi]) + be;
      }
    }
    out[col] = to_gemm<T>(v);
  }
}

// One workgroup per (feature i, member): thread t takes embedding column
// j = t % 32 (j < d_emb) over the rows r = t / 32 + 8 m, accumulating the four
// gradient sums in fp32; the 8 row groups are then added in a fixed order.
__global__ __launch_bounds__(256) void embed_bwd_kernel(const float* X, int d_in, const int32_t* idx, int B,
                                                        const MemberDev* mem, const int32_t* members,
                                                        const float* theta, const float* dE, float* grad) {
  __shared__ float red[4][8][32];
  const int i = blockIdx.x;
  const int k = members[blockIdx.y];
  const MemberDev md = mem[k];
  const int j = threadIdx.x & 31, rg = threadIdx.x >> 5;
  const bool on = j < md.d_emb;
  const int col = i * md.d_emb + j;
  float ga = 0.0f, gbe = 0.0f, gw = 0.0f, gb = 0.0f;
  if (on) {
    const float* de = dE + md.e_act + col;
    float w = 0.0f, bb = 0.0f, alpha = theta[md.e_a + col];
    if (j > 0) {
      w = theta[md.e_w + (int64_t)i * (md.d_emb - 1) + j - 1];
      bb = theta[md.e_b + (int64_t)i * (md.d_emb - 1) + j - 1];
    }
    for (int r = rg; r < B; r += 8) {
      const float x = X[(int64_t)idx[(int64_t)k * B + r] * d_in + i];
      const float g = de[(int64_t)r * md.p_in];
      gbe += g;
      if (j == 0) {
        ga += g * x;
      } else {
        float sn, cs;
        sincosf(w * x + bb, &sn, &cs);
        ga += g * cs;
        const float t = -g * alpha * sn;
        gb += t;
        gw += t * x;
      }
    }
  }
  red[0][rg][j] = ga;
  red[1][rg][j] = gbe;
  red[2][rg][j] = gw;
  red[3][rg][j] = gb;
  __syncthreads();
  if (rg == 0 && on) {
    float s[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      s[q] = ((red[q][0][j] + red[q][1][j]) + (red[q][2][j] + red[q][3][j])) +
             ((red[q][4][j] + red[q][5][j]) + (red[q][6][j] + red[q][7][j]));
    grad[md.e_a + col] = s[0];
    grad[md.e_be + col] = s[1];
    if (j > 0) {
      const int64_t wi = (int64_t)i * (md.d_emb - 1) + j - 1;
      grad[md.e_w + wi] = s[2];
      grad[md.e_b + wi] = s[3];
    }
  }
}

}  // namespace

hipError_t launch_embed_fwd(Prec prec, const float* X, int d_in, const int32_t* idx, int B, int64_t row_base,
                            int rows_valid, int Bp, const MemberDev* mem, const int32_t* members, int nmembers,
                            int max_pin, const float* theta, void* E, hipStream_t s) {
  (void)max_pin;
  if (nmembers <= 0) return hipSuccess;
  const dim3 grid(Bp, nmembers);
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((embed_fwd_kernel<__bf16>), grid, dim3(256), 0, s, X, d_in, idx, B, row_base, rows_valid, mem,
                       members, theta, static_cast<__bf16*>(E));
  else
    hipLaunchKernelGGL((embed_fwd_kernel<float>), grid, dim3(256), 0, s, X, d_in, idx, B, row_base, rows_valid, mem,
                       members, theta, static_cast<float*>(E));
  return hipGetLastError();
}

hipError_t launch_embed_bwd(const float* X, int d_in, const int32_t* idx, int B, const MemberDev* mem,
                            const int32_t* members, int nmembers, const float* theta, const float* dE, float* grad,
                            hipStream_t s) {
  if (nmembers <= 0) return hipSuccess;
  hipLaunchKernelGGL(embed_bwd_kernel, dim3(d_in, nmembers), dim3(256), 0, s, X, d_in, idx, B, mem, members, theta,
                     dE, grad);
  return hipGetLastError();
}

}  // namespace tabpack
