// Grouped ragged GEMM for the packed MLP step on gfx950 (CDNA4).
//
// One launch covers one GEMM kind of one layer for all K members: the host
// planner emits a list of 128x128 output tiles (member, m0, n0) over each
// member's own, q-padded extents, so members of different widths share a
// launch without padding to the widest member (the paper's packing grows
// every member to the maximum width and uses a batched matmul, Section 3.3;
// here only the tile quantum is wasted).
//
// Per workgroup: 256 threads = 4 wave64s in a 2x2 grid, each wave owning a
// 64x64 sub-tile as 2x2 MFMA 32x32 blocks (bf16: v_mfma_f32_32x32x16_bf16,
// fp32: v_mfma_f32_32x32x2_f32), fp32 accumulation.  Operand tiles are staged
// through LDS (double-buffered, one barrier per K step) in a depth-contiguous
// [row][16-byte vectors] layout; operands stored rows-contiguous in HBM are
// transposed in registers while being written to LDS, and the first layer
// gathers its member's fp32 feature rows straight from X (no materialised
// batch).  Epilogues are fused:
//   EPI_FWD       bias + ReLU + inverted dropout (Philox4x32-10 per member) -> H
//   EPI_FWD_EVAL  bias + ReLU -> H
//   EPI_DX        dH * [H_prev > 0] * s_k  -> dZ_prev  (ReLU' and dropout' from H)
//   EPI_DW        fp32 store of the weight gradient tile
// Every output element is owned by exactly one workgroup and reduced over the
// full depth in a fixed order: no atomics, bit-reproducible.
#include "pack_internal.h"
#include "philox.h"

namespace tabpack {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int NT = 256;       // threads per workgroup
constexpr int TM = 128;       // tile rows (GEMM M)
constexpr int TN = 128;       // tile cols (GEMM N)
constexpr int KV = 4;         // 16-byte vectors per LDS row per K step
constexpr int PITCH = KV * 16 + 16;  // LDS row pitch in bytes (one vector of padding)

template <typename T>
struct Elem;
template <>
struct Elem<__bf16> {
  static constexpr int VE = 8;  // elements per 16 bytes
};
template <>
struct Elem<float> {
  static constexpr int VE = 4;
};

__device__ __forceinline__ uint32_t bf16_bits(float f) {
  __bf16 b = (__bf16)f;  // round to nearest even (v_cvt_pk_bf16_f32)
  return (uint32_t)__builtin_bit_cast(uint16_t, b);
}

__device__ __forceinline__ float to_float(__bf16 x) { return (float)x; }
__device__ __forceinline__ float to_float(float x) { return x; }

template <typename T>
__device__ __forceinline__ T from_float(float f);
template <>
__device__ __forceinline__ __bf16 from_float<__bf16>(float f) {
  return (__bf16)f;
}
template <>
__device__ __forceinline__ float from_float<float>(float f) {
  return f;
}

// Pack VE fp32 values (one 16-byte LDS vector worth of T) into 4 dwords.
template <typename T>
__device__ __forceinline__ u32x4 pack_vec(const float* f);
template <>
__device__ __forceinline__ u32x4 pack_vec<__bf16>(const float* f) {
  u32x4 r;
  r[0] = bf16_bits(f[0]) | (bf16_bits(f[1]) << 16);
  r[1] = bf16_bits(f[2]) | (bf16_bits(f[3]) << 16);
  r[2] = bf16_bits(f[4]) | (bf16_bits(f[5]) << 16);
  r[3] = bf16_bits(f[6]) | (bf16_bits(f[7]) << 16);
  return r;
}
template <>
__device__ __forceinline__ u32x4 pack_vec<float>(const float* f) {
  u32x4 r;
  r[0] = __float_as_uint(f[0]);
  r[1] = __float_as_uint(f[1]);
  r[2] = __float_as_uint(f[2]);
  r[3] = __float_as_uint(f[3]);
  return r;
}

__device__ __forceinline__ int64_t gather_row(const GemmArgs& a, int member, int r) {
  return a.idx ? (int64_t)a.idx[(int64_t)member * a.idx_stride + r] : a.row_base + r;
}

// ---------------------------------------------------------------- loaders --
// Each loader moves one R x (KV*VE) operand tile per K step: load() issues the
// global reads for depth offset k0 into registers, store() writes them to LDS.

// Depth-contiguous operand stored as T.
template <typename T, int R>
struct LoadKmaj {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int NV = R * KV / NT;
  u32x4 reg[NV];
  const T* ptr[NV];
  bool ok[NV];
  int kv[NV];
  int r[NV];
  __device__ void init(const T* P, int64_t ld, int row0, int rbound, int tid) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = tid + i * NT;
      r[i] = v / KV;
      kv[i] = v % KV;
      ok[i] = row0 + r[i] < rbound;
      ptr[i] = P + (int64_t)(row0 + r[i]) * ld + kv[i] * VE;
    }
  }
  __device__ void load(int k0, int kd) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const bool in = ok[i] && (k0 + kv[i] * VE < kd);
      reg[i] = in ? *reinterpret_cast<const u32x4*>(ptr[i] + k0) : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ void store(char* lds) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) *reinterpret_cast<u32x4*>(lds + r[i] * PITCH + kv[i] * 16) = reg[i];
  }
};

// Rows-contiguous operand stored as T: each thread reads 2 depth rows of VE
// consecutive tile rows and writes VE LDS rows of 2 depth values.
template <typename T, int R>
struct LoadRmaj {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int RB = R / VE;
  static_assert(RB * (KV * VE / 2) == NT, "one 2 x VE block per thread");
  u32x4 reg[2];
  const T* ptr;
  int64_t ld;
  int rb, kp;
  bool ok;
  __device__ void init(const T* P, int64_t ld_, int row0, int rbound, int tid) {
    rb = tid % RB;
    kp = tid / RB;
    ld = ld_;
    ok = row0 + rb * VE < rbound;
    ptr = P + row0 + rb * VE;
  }
  __device__ void load(int k0, int kd) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int k = k0 + 2 * kp + j;
      reg[j] = (ok && k < kd) ? *reinterpret_cast<const u32x4*>(ptr + (int64_t)k * ld)
                              : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ void store(char* lds) const {
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t a = reg[0][e >> 1], b = reg[1][e >> 1];
        const uint32_t w = (e & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
        *reinterpret_cast<uint32_t*>(lds + (rb * 8 + e) * PITCH + kp * 4) = w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        *reinterpret_cast<u32x2*>(lds + (rb * 4 + e) * PITCH + kp * 8) = u32x2{reg[0][e], reg[1][e]};
    }
  }
};

// Gathered fp32 feature rows, depth (feature) contiguous; converted to T.
template <typename T, int R>
struct LoadXgk {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int NV = R * KV / NT;
  float f[NV][VE];
  const float* ptr[NV];
  bool ok[NV];
  int kv[NV];
  int r[NV];
  int d_in;
  bool vec;
  __device__ void init(const GemmArgs& a, int member, int row0, int tid) {
    d_in = a.d_in;
    vec = (a.d_in % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.X) & 15) == 0);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = tid + i * NT;
      r[i] = v / KV;
      kv[i] = v % KV;
      const int br = row0 + r[i];
      ok[i] = br < a.rows_valid;
      const int64_t src = ok[i] ? gather_row(a, member, br) : 0;
      ptr[i] = a.X + src * a.d_in + kv[i] * VE;
    }
  }
  __device__ void load(int k0, int) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int kk = k0 + kv[i] * VE;
      if (ok[i] && vec && kk + VE <= d_in) {
#pragma unroll
        for (int q = 0; q < VE / 4; ++q) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(ptr[i] + k0 + 4 * q);
          f[i][4 * q + 0] = x[0];
          f[i][4 * q + 1] = x[1];
          f[i][4 * q + 2] = x[2];
          f[i][4 * q + 3] = x[3];
        }
      } else {
#pragma unroll
        for (int e = 0; e < VE; ++e) f[i][e] = (ok[i] && kk + e < d_in) ? ptr[i][k0 + e] : 0.0f;
      }
    }
  }
  __device__ void store(char* lds) const {
#pragma unroll
    for (int i = 0; i < NV; ++i)
      *reinterpret_cast<u32x4*>(lds + r[i] * PITCH + kv[i] * 16) = pack_vec<T>(f[i]);
  }
};

// Gathered fp32 feature rows used transposed: tile rows are features, depth is
// the batch row.  Each thread reads 2 batch rows x VE features.
template <typename T, int R>
struct LoadXgr {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int RB = R / VE;
  static_assert(RB * (KV * VE / 2) == NT, "one 2 x VE block per thread");
  float f[2][VE];
  const float* X;
  const int32_t* idx;
  int64_t row_base;
  int d_in, rows_valid;
  int rb, kp, f0;
  bool vec;
  __device__ void init(const GemmArgs& args, int member, int row0, int tid) {
    X = args.X;
    idx = args.idx ? args.idx + (int64_t)member * args.idx_stride : nullptr;
    row_base = args.row_base;
    d_in = args.d_in;
    rows_valid = args.rows_valid;
    rb = tid % RB;
    kp = tid / RB;
    f0 = row0 + rb * VE;
    vec = (args.d_in % 4 == 0) && ((reinterpret_cast<uintptr_t>(args.X) & 15) == 0);
  }
  __device__ void load(int k0, int) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int br = k0 + 2 * kp + j;
      const bool okr = br < rows_valid;
      const int64_t src = okr ? (idx ? (int64_t)idx[br] : row_base + br) : 0;
      const float* p = X + src * d_in + f0;
      if (okr && vec && f0 + VE <= d_in) {
#pragma unroll
        for (int q = 0; q < VE / 4; ++q) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(p + 4 * q);
          f[j][4 * q + 0] = x[0];
          f[j][4 * q + 1] = x[1];
          f[j][4 * q + 2] = x[2];
          f[j][4 * q + 3] = x[3];
        }
      } else {
#pragma unroll
        for (int e = 0; e < VE; ++e) f[j][e] = (okr && f0 + e < d_in) ? p[e] : 0.0f;
      }
    }
  }
  __device__ void store(char* lds) const {
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      if constexpr (sizeof(T) == 2) {
        *reinterpret_cast<uint32_t*>(lds + (rb * 8 + e) * PITCH + kp * 4) =
            bf16_bits(f[0][e]) | (bf16_bits(f[1][e]) << 16);
      } else {
        *reinterpret_cast<u32x2*>(lds + (rb * 4 + e) * PITCH + kp * 8) =
            u32x2{__float_as_uint(f[0][e]), __float_as_uint(f[1][e])};
      }
    }
  }
};

template <typename T, int KIND, int R>
struct LoaderFor;
template <typename T, int R>
struct LoaderFor<T, OP_KMAJ, R> {
  using type = LoadKmaj<T, R>;
};
template <typename T, int R>
struct LoaderFor<T, OP_RMAJ, R> {
  using type = LoadRmaj<T, R>;
};
template <typename T, int R>
struct LoaderFor<T, OP_XGK, R> {
  using type = LoadXgk<T, R>;
};
template <typename T, int R>
struct LoaderFor<T, OP_XGR, R> {
  using type = LoadXgr<T, R>;
};

template <typename L, int KIND, typename T>
__device__ __forceinline__ void loader_init(L& ld, const GemmArgs& a, const GemmDesc& d,
                                            const void* P, int64_t lp, int row0, int rbound,
                                            int tid) {
  if constexpr (KIND == OP_XGK || KIND == OP_XGR)
    ld.init(a, d.member, row0, tid);
  else
    ld.init(static_cast<const T*>(P), lp, row0, rbound, tid);
}

// ------------------------------------------------------------------- MFMA --
template <typename T>
__device__ __forceinline__ void mma_step(const char* As, const char* Bs, f32x16 (&acc)[2][2],
                                         int wm, int wn, int lane) {
  const int rl = lane & 31;
  const int hv = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < KV / 2; ++ks) {
    const int vo = (2 * ks + hv) * 16;
    if constexpr (sizeof(T) == 2) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + i * 32 + rl) * PITCH + vo);
        b[i] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + i * 32 + rl) * PITCH + vo);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    } else {
      f32x4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = *reinterpret_cast<const f32x4*>(As + (wm * 64 + i * 32 + rl) * PITCH + vo);
        b[i] = *reinterpret_cast<const f32x4*>(Bs + (wn * 64 + i * 32 + rl) * PITCH + vo);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
  }
}

// --------------------------------------------------------------- epilogue --
// Accumulator register r of a 32x32 block held by lane l is element
// (row 8*(r/4) + 4*(l/32) + r%4, col l%32): each lane owns 4 runs of 4
// consecutive rows of one column, so one Philox block (4 words) serves a run.
template <typename T, int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, const GemmDesc& d, const Tile& t,
                                         f32x16 (&acc)[2][2], int wm, int wn, int lane) {
  const int hv = lane >> 5;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = t.n0 + wn * 64 + j * 32 + (lane & 31);
    if (col >= d.N) continue;
    if constexpr (EPI == EPI_DW) {
      float* C = static_cast<float*>(d.C);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = t.m0 + wm * 64 + i * 32 + 8 * g + 4 * hv;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (row + q < d.M) C[(int64_t)(row + q) * d.ldc + col] = acc[i][j][4 * g + q];
        }
    } else if constexpr (EPI == EPI_DX) {
      T* C = static_cast<T*>(d.C);
      const T* Hp = static_cast<const T*>(d.Haux);
      float cs = 0.0f;  // column sum over this wave's 64 rows (this lane's 32 of them)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = t.m0 + wm * 64 + i * 32 + 8 * g + 4 * hv;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int64_t o = (int64_t)(row + q) * d.ldc + col;
            const float hp = to_float(Hp[o]);
            const float dz = hp > 0.0f ? acc[i][j][4 * g + q] * d.drop_s : 0.0f;
            cs += dz;
            C[o] = from_float<T>(dz);
          }
        }
      // lanes l and l^32 hold the two interleaved halves of the same column
      cs += __shfl_xor(cs, 32, 64);
      if (hv == 0) d.colpart[(int64_t)(t.m0 / 64 + wm) * d.N + col] = cs;
    } else {
      T* C = static_cast<T*>(d.C);
      const float bias = d.bias[col];
      const bool colok = col < d.width;
      const bool drop = (EPI == EPI_FWD) && d.drop_t != 0u;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = t.m0 + wm * 64 + i * 32 + 8 * g + 4 * hv;
          Words4 w{0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
          if (drop)
            w = philox4x32_10((uint32_t)row >> 2, (uint32_t)col,
                              ((uint32_t)d.member << 8) | (uint32_t)a.layer, a.step, a.key0,
                              a.key1);
          const uint32_t wq[4] = {w.w0, w.w1, w.w2, w.w3};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float h = fmaxf(acc[i][j][4 * g + q] + bias, 0.0f);
            if (EPI == EPI_FWD) h = (wq[q] >= d.drop_t) ? h * d.drop_s : 0.0f;
            if (!colok || row + q >= a.rows_valid) h = 0.0f;
            C[(int64_t)(row + q) * d.ldc + col] = from_float<T>(h);
          }
        }
    }
  }
}

// ----------------------------------------------------------------- kernel --
template <typename T, int AK, int BK_, int EPI>
__global__ __launch_bounds__(NT) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2][(TM + TN) * PITCH];
  const Tile t = a.tiles[blockIdx.x];
  const GemmDesc d = a.descs[t.desc];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int BKE = KV * Elem<T>::VE;  // depth per K step

  typename LoaderFor<T, AK, TM>::type la;
  typename LoaderFor<T, BK_, TN>::type lb;
  loader_init<decltype(la), AK, T>(la, a, d, d.A, d.lda, t.m0, d.M, tid);
  loader_init<decltype(lb), BK_, T>(lb, a, d, d.B, d.ldb, t.n0, d.N, tid);

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (d.Kd + BKE - 1) / BKE;
  la.load(0, d.Kd);
  lb.load(0, d.Kd);
  la.store(smem[0]);
  lb.store(smem[0] + TM * PITCH);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load((kt + 1) * BKE, d.Kd);
      lb.load((kt + 1) * BKE, d.Kd);
    }
    mma_step<T>(smem[cur], smem[cur] + TM * PITCH, acc, wm, wn, lane);
    if (more) {
      la.store(smem[cur ^ 1]);
      lb.store(smem[cur ^ 1] + TM * PITCH);
    }
    __syncthreads();
  }
  epilogue<T, EPI>(a, d, t, acc, wm, wn, lane);
}

template <typename T, int AK, int BK_, int EPI>
hipError_t launch_t(const GemmArgs& args, hipStream_t s) {
  if (args.ntiles <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<T, AK, BK_, EPI>), dim3(args.ntiles), dim3(NT), 0, s, args);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_prec(OpKind ak, OpKind bk, EpiKind e, const GemmArgs& args, hipStream_t s) {
  if (ak == OP_XGK && bk == OP_KMAJ && e == EPI_FWD) return launch_t<T, OP_XGK, OP_KMAJ, EPI_FWD>(args, s);
  if (ak == OP_XGK && bk == OP_KMAJ && e == EPI_FWD_EVAL)
    return launch_t<T, OP_XGK, OP_KMAJ, EPI_FWD_EVAL>(args, s);
  if (ak == OP_KMAJ && bk == OP_KMAJ && e == EPI_FWD) return launch_t<T, OP_KMAJ, OP_KMAJ, EPI_FWD>(args, s);
  if (ak == OP_KMAJ && bk == OP_KMAJ && e == EPI_FWD_EVAL)
    return launch_t<T, OP_KMAJ, OP_KMAJ, EPI_FWD_EVAL>(args, s);
  if (ak == OP_KMAJ && bk == OP_RMAJ && e == EPI_DX) return launch_t<T, OP_KMAJ, OP_RMAJ, EPI_DX>(args, s);
  if (ak == OP_RMAJ && bk == OP_RMAJ && e == EPI_DW) return launch_t<T, OP_RMAJ, OP_RMAJ, EPI_DW>(args, s);
  if (ak == OP_RMAJ && bk == OP_XGR && e == EPI_DW) return launch_t<T, OP_RMAJ, OP_XGR, EPI_DW>(args, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(Prec prec, OpKind a, OpKind b, EpiKind e, const GemmArgs& args, hipStream_t s) {
  return prec == Prec::BF16 ? launch_prec<__bf16>(a, b, e, args, s) : launch_prec<float>(a, b, e, args, s);
}

}  // namespace tabpack
