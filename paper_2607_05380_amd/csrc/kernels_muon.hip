// Muon for the hidden weights of every member (the paper trains the main
// rectangular weights of the backbone's linear layers with Muon and every other
// parameter with AdamW; Muon: Jordan et al., 2024).  Per weight W [rows, cols]
// with gradient G:
//   B <- mu B + G;  U = G + mu B (Nesterov) or U = B
//   X = U / (||U||_F + 1e-7), as U^T when the true rows exceed the true columns
//   steps x: A = X X^T;  B' = b A + c A A;  X = a X + B' X   (grouped GEMMs, EPI_NS)
//   W <- W (1 - lr wd) - lr max(1, rows/cols)^(1/2) X  (transposed back)
// The kernels here are the elementwise stages around the grouped GEMMs; each
// works on 64 x 64 blocks of a weight (MuonTile), padding included: padded
// rows and columns of G, B and W are zero, so they stay zero through the
// iteration and the update.
#include "pack_internal.h"

namespace tabpack {
namespace {

constexpr int kMT = 64;  // rows and columns of a MuonTile

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <typename T>
__device__ __forceinline__ T to_t(float x);
template <>
__device__ __forceinline__ __bf16 to_t<__bf16>(float x) {
  return (__bf16)x;
}
template <>
__device__ __forceinline__ float to_t<float>(float x) {
  return x;
}
__device__ __forceinline__ float from_t(__bf16 x) { return (float)x; }
__device__ __forceinline__ float from_t(float x) { return x; }

// Momentum update and the squared norm of U per tile.  Thread t owns column
// c0 + t % 64 of rows r0 + t / 64 + 4 i (i < 16): every access is a run of 64
// consecutive floats.  part[tile] = sum of u^2 over the tile (fixed order).
__global__ __launch_bounds__(256) void muon_prep_kernel(const MuonMat* mats, const MuonTile* tiles,
                                                        const float* grad, float* buf, float mu, int nesterov,
                                                        double* part) {
  __shared__ double sh[4];
  const MuonTile t = tiles[blockIdx.x];
  const MuonMat m = mats[t.mat];
  const int c = t.c0 + (threadIdx.x & 63);
  double s = 0.0;
  if (c < m.Cp) {
#pragma unroll 4
    for (int i = 0; i < kMT / 4; ++i) {
      const int r = t.r0 + (threadIdx.x >> 6) + 4 * i;
      if (r >= m.R) break;
      const int64_t e = m.woff + (int64_t)r * m.Cp + c;
      const float g = grad[e];
      const float b = mu * buf[e] + g;
      buf[e] = b;
      const float u = nesterov ? g + mu * b : b;
      s += (double)u * (double)u;
    }
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

// inv[k] = 1 / (||U_k|| + 1e-7) from the tile partials of matrix k, in tile order.
__global__ void muon_norm_kernel(const int32_t* tile0, int nmats, const double* part, float* inv) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= nmats) return;
  double s = 0.0;
  for (int i = tile0[k]; i < tile0[k + 1]; ++i) s += part[i];
  inv[k] = (float)(1.0 / (sqrt(s) + 1e-7));
}

// X0 = U / (||U|| + 1e-7) in the GEMM precision, [S, L] row-major: U itself
// (S = rows), or U^T for tall weights, transposed through LDS so that reads
// and writes both run along rows.
template <typename T>
__global__ __launch_bounds__(256) void muon_convert_kernel(const MuonMat* mats, const MuonTile* tiles,
                                                           const float* grad, const float* buf, float mu,
                                                           int nesterov, const float* inv, T* X) {
  __shared__ float tr[kMT][kMT + 1];
  const MuonTile t = tiles[blockIdx.x];
  const MuonMat m = mats[t.mat];
  const float sc = inv[t.mat];
  const int cl = threadIdx.x & 63;
#pragma unroll 4
  for (int i = 0; i < kMT / 4; ++i) {
    const int rl = (threadIdx.x >> 6) + 4 * i;
    const int r = t.r0 + rl, c = t.c0 + cl;
    float x = 0.0f;
    if (r < m.R && c < m.Cp) {
      const int64_t e = m.woff + (int64_t)r * m.Cp + c;
      const float g = grad[e], b = buf[e];
      x = (nesterov ? g + mu * b : b) * sc;
      if (!m.tall) X[m.xoff + (int64_t)r * m.Cp + c] = to_t<T>(x);
    }
    tr[rl][cl] = x;
  }
  if (!m.tall) return;  // uniform
  __syncthreads();
  // X[c, r] = U[r, c]: thread owns row c0 + 4 i + t / 64 of X, column r0 + t % 64
#pragma unroll 4
  for (int i = 0; i < kMT / 4; ++i) {
    const int cl2 = (threadIdx.x >> 6) + 4 * i, rl2 = threadIdx.x & 63;
    const int r = t.r0 + rl2, c = t.c0 + cl2;
    if (r < m.R && c < m.Cp) X[m.xoff + (int64_t)c * m.R + r] = to_t<T>(tr[rl2][cl2]);
  }
}

// W <- W (1 - lr wd) - lr scale O with O read from X (transposed back for tall
// weights); the bf16 copy of W for the GEMMs is written beside it.
template <typename T>
__global__ __launch_bounds__(256) void muon_update_kernel(const MuonMat* mats, const MuonTile* tiles, float* theta,
                                                          uint16_t* shadow, const T* X) {
  __shared__ float tr[kMT][kMT + 1];
  const MuonTile t = tiles[blockIdx.x];
  const MuonMat m = mats[t.mat];
  if (m.tall) {
#pragma unroll 4
    for (int i = 0; i < kMT / 4; ++i) {
      const int cl2 = (threadIdx.x >> 6) + 4 * i, rl2 = threadIdx.x & 63;
      const int r = t.r0 + rl2, c = t.c0 + cl2;
      tr[rl2][cl2] = (r < m.R && c < m.Cp) ? from_t(X[m.xoff + (int64_t)c * m.R + r]) : 0.0f;
    }
    __syncthreads();
  }
  const float decay = m.decay, step = m.step;
  const int cl = threadIdx.x & 63;
#pragma unroll 4
  for (int i = 0; i < kMT / 4; ++i) {
    const int rl = (threadIdx.x >> 6) + 4 * i;
    const int r = t.r0 + rl, c = t.c0 + cl;
    if (r >= m.R || c >= m.Cp) continue;
    const int64_t e = m.woff + (int64_t)r * m.Cp + c;
    const float o = m.tall ? tr[rl][cl] : from_t(X[m.xoff + (int64_t)r * m.Cp + c]);
    float w;
    {
#pragma clang fp contract(off)
      w = theta[e] * decay - step * o;
    }
    theta[e] = w;
    if (shadow) shadow[e] = __builtin_bit_cast(uint16_t, (__bf16)w);
  }
}

}  // namespace

hipError_t launch_muon_prep(const MuonMat* mats, const MuonTile* tiles, int ntiles, const float* grad, float* buf,
                            float mu, int nesterov, double* part, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(muon_prep_kernel, dim3(ntiles), dim3(256), 0, s, mats, tiles, grad, buf, mu, nesterov, part);
  return hipGetLastError();
}

hipError_t launch_muon_norm(const int32_t* tile0, int nmats, const double* part, float* inv, hipStream_t s) {
  if (nmats <= 0) return hipSuccess;
  hipLaunchKernelGGL(muon_norm_kernel, dim3((nmats + 63) / 64), dim3(64), 0, s, tile0, nmats, part, inv);
  return hipGetLastError();
}

hipError_t launch_muon_convert(Prec prec, const MuonMat* mats, const MuonTile* tiles, int ntiles, const float* grad,
                               const float* buf, float mu, int nesterov, const float* inv, void* X, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((muon_convert_kernel<__bf16>), dim3(ntiles), dim3(256), 0, s, mats, tiles, grad, buf, mu,
                       nesterov, inv, static_cast<__bf16*>(X));
  else
    hipLaunchKernelGGL((muon_convert_kernel<float>), dim3(ntiles), dim3(256), 0, s, mats, tiles, grad, buf, mu,
                       nesterov, inv, static_cast<float*>(X));
  return hipGetLastError();
}

hipError_t launch_muon_update(Prec prec, const MuonMat* mats, const MuonTile* tiles, int ntiles, float* theta,
                              uint16_t* shadow, const void* X, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  if (prec == Prec::BF16)
    hipLaunchKernelGGL((muon_update_kernel<__bf16>), dim3(ntiles), dim3(256), 0, s, mats, tiles, theta, shadow,
                       static_cast<const __bf16*>(X));
  else
    hipLaunchKernelGGL((muon_update_kernel<float>), dim3(ntiles), dim3(256), 0, s, mats, tiles, theta, shadow,
                       static_cast<const float*>(X));
  return hipGetLastError();
}

}  // namespace tabpack
