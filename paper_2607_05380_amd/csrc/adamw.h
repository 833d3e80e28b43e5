// adamw.h -- the per-parameter AdamW update shared by the optimizer kernel and
// the fused weight-gradient epilogue (torch.optim.AdamW semantics: decoupled
// decay applied to the parameter first, then the bias-corrected Adam step with
// eps added after the square root of the corrected second moment).
#pragma once

#include "pack_internal.h"

namespace tabpack {

// Contraction into fused multiply-adds is off: the optimizer runs inside
// several kernels (the weight-gradient GEMM's epilogues of each tile shape and
// the standalone kernel), and every one of them must round each operation the
// same way for results not to depend on the tile shape.
__device__ __forceinline__ void adamw_elem(float& th, float g, float& m, float& v, float decay, float step,
                                           const AdamConst& c) {
#pragma clang fp contract(off)
  th *= decay;
  m = c.beta1 * m + c.omb1 * g;
  v = c.beta2 * v + c.omb2 * g * g;
  th -= step * m / (sqrtf(v) / c.bc2_sqrt + c.eps);
}

// Four consecutive parameters held in vector registers.
template <typename V4>
__device__ __forceinline__ void adamw_vec4(V4& th, const V4& g, V4& m, V4& v, float decay, float step,
                                           const AdamConst& c) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float t = th[q], mm = m[q], vv = v[q];
    adamw_elem(t, g[q], mm, vv, decay, step, c);
    th[q] = t;
    m[q] = mm;
    v[q] = vv;
  }
}

}  // namespace tabpack
