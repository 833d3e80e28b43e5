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

typedef float f32x4v __attribute__((ext_vector_type(4)));
// 4 consecutive elements of X (8 bytes in bf16, 16 in fp32)
__device__ __forceinline__ void store4(__bf16* p, f32x4v x) {
  const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[0]) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[1]) << 16);
  const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[2]) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x[3]) << 16);
  *reinterpret_cast<uint2*>(p) = uint2{lo, hi};
}
__device__ __forceinline__ void store4(float* p, f32x4v x) { *reinterpret_cast<f32x4v*>(p) = x; }
__device__ __forceinline__ f32x4v load4(const __bf16* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return f32x4v{__builtin_bit_cast(float, u.x << 16), __builtin_bit_cast(float, u.x & 0xffff0000u),
                __builtin_bit_cast(float, u.y << 16), __builtin_bit_cast(float, u.y & 0xffff0000u)};
}
__device__ __forceinline__ f32x4v load4(const float* p) { return *reinterpret_cast<const f32x4v*>(p); }

typedef f32x4v f32x4;

// Thread t of a tile owns the 4 columns c0 + 4 (t % 16) .. + 3 of rows
// r0 + t / 16 + 16 i (i < 4): every access moves 16 bytes of a row (the padded
// column counts are multiples of 8, the weights start on 256-element
// boundaries).
constexpr int kTPR = kMT / 4;         // threads per tile row
constexpr int kRPP = 256 / kTPR;      // rows per pass

// Momentum update and the squared norm of U per tile: part[tile] = sum of u^2
// over the tile, in a fixed order.
__global__ __launch_bounds__(256) void muon_prep_kernel(const MuonMat* mats, const MuonTile* tiles,
                                                        const float* grad, float* buf, float mu, int nesterov,
                                                        double* part) {
  __shared__ double sh[4];
  const MuonTile t = tiles[blockIdx.x];
  const MuonMat m = mats[t.mat];
  const int c = t.c0 + 4 * (threadIdx.x % kTPR);
  double s = 0.0;
  if (c < m.Cp) {
#pragma unroll
    for (int i = 0; i < kMT / kRPP; ++i) {
      const int r = t.r0 + threadIdx.x / kTPR + kRPP * i;
      if (r >= m.R) break;
      const int64_t e = m.woff + (int64_t)r * m.Cp + c;
      const f32x4 g = *reinterpret_cast<const f32x4*>(grad + e);
      f32x4 b = *reinterpret_cast<const f32x4*>(buf + e);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        b[q] = mu * b[q] + g[q];
        const float u = nesterov ? g[q] + mu * b[q] : b[q];
        s += (double)u * (double)u;
      }
      *reinterpret_cast<f32x4*>(buf + e) = b;
    }
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

// inv[k] = 1 / (||U_k|| + 1e-7): one wave per matrix sums its tile partials
// lane-strided, then in a fixed shuffle tree.
__global__ __launch_bounds__(256) void muon_norm_kernel(const int32_t* tile0, int nmats, const double* part,
                                                        float* inv) {
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (k >= nmats) return;  // wave-uniform
  double s = 0.0;
  for (int i = tile0[k] + lane; i < tile0[k + 1]; i += 64) s += part[i];
  s = wave_sum(s);
  if (lane == 0) inv[k] = (float)(1.0 / (sqrt(s) + 1e-7));
}

// X0 = U / (||U|| + 1e-7) in the GEMM precision, [S, L] row-major: U itself
// (S = rows), or U^T for tall weights, transposed through LDS so that reads
// and writes both move 4 elements of a row.
template <typename T>
__global__ __launch_bounds__(256) void muon_convert_kernel(const MuonMat* mats, const MuonTile* tiles,
                                                           const float* grad, const float* buf, float mu,
                                                           int nesterov, const float* inv, T* X) {
  __shared__ float tr[kMT][kMT + 1];
  const MuonTile t = tiles[blockIdx.x];
  const MuonMat m = mats[t.mat];
  const float sc = inv[t.mat];
  const int cl = 4 * (threadIdx.x % kTPR);
#pragma unroll
  for (int i = 0; i < kMT / kRPP; ++i) {
    const int rl = threadIdx.x / kTPR + kRPP * i;
    const int r = t.r0 + rl, c = t.c0 + cl;
    f32x4 x = {0.0f, 0.0f, 0.0f, 0.0f};
    if (r < m.R && c < m.Cp) {
      const int64_t e = m.woff + (int64_t)r * m.Cp + c;
      const f32x4 g = *reinterpret_cast<const f32x4*>(grad + e);
      const f32x4 b = *reinterpret_cast<const f32x4*>(buf + e);
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = (nesterov ? g[q] + mu * b[q] : b[q]) * sc;
      if (!m.tall) store4(X + m.xoff + (int64_t)r * m.Cp + c, x);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) tr[rl][cl + q] = x[q];
  }
  if (!m.tall) return;  // uniform
  __syncthreads();
  // X[c, r .. r + 3] = U[r .. r + 3, c]
#pragma unroll
  for (int i = 0; i < kMT / kRPP; ++i) {
    const int cl2 = threadIdx.x / kTPR + kRPP * i, rl2 = 4 * (threadIdx.x % kTPR);
    const int r = t.r0 + rl2, c = t.c0 + cl2;
    if (r < m.R && c < m.Cp) {
      const f32x4 x = {tr[rl2][cl2], tr[rl2 + 1][cl2], tr[rl2 + 2][cl2], tr[rl2 + 3][cl2]};
      store4(X + m.xoff + (int64_t)c * m.R + r, x);
    }
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
#pragma unroll
    for (int i = 0; i < kMT / kRPP; ++i) {
      const int cl2 = threadIdx.x / kTPR + kRPP * i, rl2 = 4 * (threadIdx.x % kTPR);
      const int r = t.r0 + rl2, c = t.c0 + cl2;
      f32x4 o = {0.0f, 0.0f, 0.0f, 0.0f};
      if (r < m.R && c < m.Cp) o = load4(X + m.xoff + (int64_t)c * m.R + r);
#pragma unroll
      for (int q = 0; q < 4; ++q) tr[rl2 + q][cl2] = o[q];
    }
    __syncthreads();
  }
  const float decay = m.decay, step = m.step;
  const int cl = 4 * (threadIdx.x % kTPR);
#pragma unroll
  for (int i = 0; i < kMT / kRPP; ++i) {
    const int rl = threadIdx.x / kTPR + kRPP * i;
    const int r = t.r0 + rl, c = t.c0 + cl;
    if (r >= m.R || c >= m.Cp) continue;
    const int64_t e = m.woff + (int64_t)r * m.Cp + c;
    const f32x4 o = m.tall ? f32x4{tr[rl][cl], tr[rl][cl + 1], tr[rl][cl + 2], tr[rl][cl + 3]}
                           : load4(X + m.xoff + (int64_t)r * m.Cp + c);
    f32x4 w = *reinterpret_cast<const f32x4*>(theta + e);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma clang fp contract(off)
      w[q] = w[q] * decay - step * o[q];
    }
    *reinterpret_cast<f32x4*>(theta + e) = w;
    if (shadow) {
      const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[1]) << 16);
      const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[3]) << 16);
      *reinterpret_cast<uint2*>(shadow + e) = uint2{lo, hi};
    }
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
  hipLaunchKernelGGL(muon_norm_kernel, dim3((nmats + 3) / 4), dim3(256), 0, s, tile0, nmats, part, inv);
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
