// cos and sin of an embedding phase phi (radians), shared by the embedding
// kernels and the first layer's data-gradient epilogue.  FAST (bf16 packs):
// the hardware's v_cos_f32 / v_sin_f32 take revolutions, so t = phi / (2 pi)
// is reduced to [-1/2, 1/2] by subtracting the nearest integer first; the
// error (about 1e-6 absolute for phases up to a few hundred radians, most of
// it the rounding of t) is far below the bf16 rounding of the embedded
// values.  Otherwise (fp32 packs) cosf / sincosf.
#pragma once

#include <hip/hip_runtime.h>

namespace tabpack {

__device__ __forceinline__ float emb_revolutions(float phi) {
  const float t = phi * 0.15915494309189535f;
  return t - rintf(t);
}
template <bool FAST>
__device__ __forceinline__ float emb_cos(float phi) {
  if constexpr (FAST)
    return __builtin_amdgcn_cosf(emb_revolutions(phi));
  else
    return cosf(phi);
}
template <bool FAST>
__device__ __forceinline__ void emb_sincos(float phi, float* sn, float* cs) {
  if constexpr (FAST) {
    const float t = emb_revolutions(phi);
    *sn = __builtin_amdgcn_sinf(t);
    *cs = __builtin_amdgcn_cosf(t);
  } else {
    sincosf(phi, sn, cs);
  }
}

}  // namespace tabpack
