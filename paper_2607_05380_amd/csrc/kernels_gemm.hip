// Grouped ragged GEMM for the packed MLP step on gfx950 (CDNA4).
//
// One launch covers one GEMM kind of one layer for all K members: the host
// planner emits a list of output tiles (member, m0, n0, shape) over each
// member's own q-padded extents, so members of different widths share a launch
// without padding to the widest member (the paper's packing grows every member
// to the maximum width and uses a batched matmul, Section 3.3).
//
// Workgroup: 256 threads = 4 wave64s in a 2 x 2 grid.  Tile shapes (uniform
// per workgroup; one launch runs one tile set, chosen by the host):
//   small 128 x 128: each wave owns 64 x 64 = 2 x 2 MFMA 32x32 blocks; 64 KB
//         of LDS, two workgroups per CU.  The default for every GEMM.
//   tall  256 x 128 (waves 128 x 64), two workgroups per CU, with small tiles
//         on a member's row edge.
//   big   256 x 256 (waves 128 x 128), one workgroup per CU, with small tiles
//         on a member's edges.
// The small tile is bound by the bytes in flight per CU rather than by LDS or
// MFMA throughput: each workgroup has one 64-deep K step (32 KB) in flight
// while it computes the previous one, against a direct-load latency of about
// 1800 cycles.  Measured per 64-deep step and workgroup pair: about 1800
// cycles for 1024 cycles of MFMA per SIMD.
// MFMA: v_mfma_f32_32x32x16_bf16 (fp32 mode: v_mfma_f32_32x32x2_f32), fp32
// accumulators.  A wave whose sub-tile lies wholly outside the member's
// extents skips its MFMAs.
//
// Staging: per K step each operand tile goes HBM -> LDS in NS stages with one
// barrier per step; the loads of the next steps are in flight during the MFMAs
// of the current one.  bf16 uses direct-to-LDS loads (global_load_lds_dwordx4,
// no staging registers); fp32 stages through registers with raw buffer loads
// and runs small tiles only.  Inside a K step a wave reads the fragments of
// 16-deep step ks + 2 while the MFMAs of step ks run.
// LDS layouts:
//   depth-contiguous operands (element (r, k) at P[r * ld + k]), bf16:
//     row-major, the 16-byte chunks of a row XOR-swizzled by row (see
//     kmaj16_off); fragments are conflict-free 16-byte reads and each quad of
//     a direct load reads one aligned 64-byte piece of one row.
//     fp32: [row][8 x 16 B], vector s of row r in slot s ^ (r & 7) ^ ((r >> 3) & 7).
//   rows-contiguous operands (element (r, k) at P[k * ld + r]), bf16: stored as
//     loaded, [depth row][R], the 32-byte chunk c of depth row k at c ^ 2(k & 3);
//     fragments come from two ds_read_b64_tr_b16 each.  Within a 16-lane group
//     that instruction hands lane i the element i % 4 of the 8 bytes addressed
//     by lane 4j + i / 4 as its j-th value, so lane (s, group g) addressing
//     depth row 8h + s/4 (+4) at rows 16(g & 1) + 4(s & 3) receives rows
//     16(g & 1) + s at depths 8h..8h+3 (+4) -- exactly an MFMA operand.  These
//     8-byte reads run at half the byte rate of 16-byte reads (measured
//     ~130 vs ~255 B/clk per CU).
//   rows-contiguous operands, fp32: transposed in registers into the first layout.
//
// Fused epilogues:
//   EPI_FWD       bias + ReLU + inverted dropout (Philox4x32-10 per member) -> H
//   EPI_FWD_EVAL  bias + ReLU -> H
//   EPI_DX        dH * [H_prev > 0] * s_k -> dZ_prev, plus column sums of the
//                 unrounded values per 64-row block (bias-gradient partials)
//   EPI_DW        fp32 store of the weight-gradient tile, or AdamW applied to
//                 the weights it covers (small tiles: the whole tile staged in
//                 LDS and streamed by the workgroup)
//   EPI_NS        alpha * Y + beta * acc -> C in the GEMM precision (the
//                 products of the Newton-Schulz iteration of the Muon optimizer)
//   EPI_DE        the embedded first layer's dE = dZ_1 W_1 reduced over each
//                 64-row block into the four embedding-gradient sums per column
//                 (dE itself is never stored)
// Every output element is owned by exactly one workgroup and reduced over the
// full depth in a fixed order: no atomics, bit-reproducible.
#include <algorithm>
#include <type_traits>

#include "adamw.h"
#include "pack_internal.h"

namespace tabpack {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int NT = 256;                 // threads per workgroup (2 x 2 waves)
constexpr int KV = 8;                   // 16-byte vectors of depth per row per K step
constexpr int ROW = KV * 16;            // 128 bytes of depth per row per K step
// Big-tile bf16 pipeline: kBigNs stages of kBigKs 16-deep steps of both
// 256-row operand tiles (the fp32 big path is not used: fp32 runs small tiles).
#ifndef TABPACK_BIG_KS
#define TABPACK_BIG_KS 4
#endif
#ifndef TABPACK_BIG_NS
#define TABPACK_BIG_NS 2
#endif
constexpr int kBigKs = TABPACK_BIG_KS, kBigNs = TABPACK_BIG_NS;
constexpr int kLdsBig = kBigNs * 2 * 256 * 32 * kBigKs > 2 * 2 * 256 * ROW ? kBigNs * 2 * 256 * 32 * kBigKs
                                                                          : 2 * 2 * 256 * ROW;
static_assert(kLdsBig <= 160 * 1024, "one big-tile workgroup per CU");
// Small-tile bf16 pipeline: kSmallNs stages of kSmallKs 16-deep MFMA steps.
#ifndef TABPACK_SMALL_KS
#define TABPACK_SMALL_KS 4
#endif
#ifndef TABPACK_SMALL_NS
#define TABPACK_SMALL_NS 2
#endif
constexpr int kSmallKs = TABPACK_SMALL_KS, kSmallNs = TABPACK_SMALL_NS;
constexpr int kStageBytes = 4 * 32 * (2 * 128 + 32);  // epilogue staging of the 4 waves of a small tile
constexpr int kLdsSmallBf16 =
    kSmallNs * 2 * 128 * 32 * kSmallKs > kStageBytes ? kSmallNs * 2 * 128 * 32 * kSmallKs : kStageBytes;
constexpr int kLdsSmallF32 = 2 * 2 * 128 * ROW;  // two register-staged 32-deep fp32 stages
constexpr int kLdsSmall = kLdsSmallBf16 > kLdsSmallF32 ? kLdsSmallBf16 : kLdsSmallF32;
// workgroups (waves per SIMD) per CU for the small kernel: as many as the
// 160 KB of LDS hold, at most 3 (the register budget of 3 waves per SIMD)
constexpr int wpe_for(int lds) { return 160 * 1024 / lds >= 3 ? 3 : (160 * 1024 / lds >= 2 ? 2 : 1); }
constexpr int kSmallWpeBf16 = wpe_for(kLdsSmallBf16), kSmallWpeF32 = wpe_for(kLdsSmallF32);
constexpr int kSmallWpe = kSmallWpeBf16;
// Tall-tile bf16 pipeline: kTallNs stages of kTallKs 16-deep steps of the
// 256-row and 128-row operand tiles; the small edge tiles of the same launch
// keep the small pipeline.  Both must fit two workgroups per CU.
#ifndef TABPACK_TALL_KS
#define TABPACK_TALL_KS 2
#endif
#ifndef TABPACK_TALL_NS
#define TABPACK_TALL_NS 3
#endif
constexpr int kTallKs = TABPACK_TALL_KS, kTallNs = TABPACK_TALL_NS;
constexpr int kLdsTallBf16 = kTallNs * (256 + 128) * 32 * kTallKs;
constexpr int kLdsTall = kLdsTallBf16 > kLdsSmallBf16 ? kLdsTallBf16 : kLdsSmallBf16;
static_assert(kLdsTall <= 80 * 1024, "two tall-tile workgroups per CU");
// LDS table of the batch rows' row numbers in the data copy for the weight
// gradient of the first layer (bf16 kernels of EPI_DW only)
template <typename T, int EPI>
constexpr int XMapBytes = EPI == EPI_DW ? kMapRows * 4 : 0;
static_assert((kLdsSmallBf16 + kMapRows * 4) * kSmallWpeBf16 <= 160 * 1024, "small weight-gradient occupancy");
static_assert(kLdsBig + kMapRows * 4 <= 160 * 1024, "one big-tile workgroup per CU");

template <int SH>
struct Shape;
template <>
struct Shape<kShapeBig> {
  static constexpr int MB = 4, NB = 4, TM = 256, TN = 256;
  static constexpr int STAGE = 32 * (NB * 128 + 32);  // epilogue staging bytes per wave
};
template <>
struct Shape<kShapeSmall> {
  static constexpr int MB = 2, NB = 2, TM = 128, TN = 128;
  static constexpr int STAGE = 32 * (NB * 128 + 32);
};
template <>
struct Shape<kShapeTall> {
  static constexpr int MB = 4, NB = 2, TM = 256, TN = 128;
  static constexpr int STAGE = 32 * (NB * 128 + 32);
};
template <>
struct Shape<kShapeWide> {
  static constexpr int MB = 2, NB = 2, TM = 128, TN = 256;
  static constexpr int STAGE = 32 * (NB * 128 + 32);
};
template <>
struct Shape<kShapeTall8> {
  static constexpr int MB = 2, NB = 2, TM = 256, TN = 128;
  static constexpr int STAGE = 32 * (NB * 128 + 32);
};

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

// depth-contiguous layout: byte offset of 16-byte vector `slot` of row `row`
__device__ __forceinline__ int kmaj_off(int row, int slot) {
  return row * ROW + ((slot ^ (row & 7) ^ ((row >> 3) & 7)) << 4);
}

// depth-contiguous bf16 layout used with direct-to-LDS loads, for K steps of
// KS 16-deep MFMA steps: row-major, 32*KS bytes (CPR = 2*KS 16-byte chunks) of
// depth per row, chunk c of row r stored at chunk position c ^ f(r) with
// f(r) = (r / (16/CPR)) % CPR.  The 16 rows read by a quarter-wave's 16-byte
// fragment loads then cover all 64 banks, and each quad of lanes of a direct
// load fills one aligned 64-byte piece of one row, i.e. it reads one aligned
// 64-byte piece of one global row (in permuted order): one cache-line lookup
// per quad.
template <int KS>
__device__ __forceinline__ int kmaj_f(int row) {
  constexpr int CPR = 2 * KS;
  return (row / (16 / CPR)) & (CPR - 1);
}
template <int KS>
__device__ __forceinline__ int kmaj16_off(int row, int c) {
  return row * (32 * KS) + ((c ^ kmaj_f<KS>(row)) << 4);
}

// rows-contiguous bf16 layout (R rows): byte offset of element `col` of depth row k
template <int R>
__device__ __forceinline__ int rmaj_off(int k, int col) {
  return k * (R * 2) + ((((col >> 4) ^ ((k & 3) << 1))) << 5) + ((col & 15) << 1);
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

// ------------------------------------------------------------------ waits --
// vmcnt <= N, every other counter at its maximum (gfx9 s_waitcnt encoding),
// plus lgkmcnt(0) when LDS is set.
template <int N, bool LDS>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | ((LDS ? 0 : 15) << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without a memory fence: the waits that make data visible
// are explicit around it, and the empty asm statements keep the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Global-memory views of pointers taken from the descriptor tables.  The
// compiler cannot infer their address space and would use flat accesses,
// which also count against the LDS counter: every LDS wait of the epilogue
// would then wait for the global stores before it too.
#define TABPACK_GLOBAL __attribute__((address_space(1)))
template <typename V>
__device__ __forceinline__ TABPACK_GLOBAL V* glob(V* p) {
  return (TABPACK_GLOBAL V*)p;
}
template <typename V>
__device__ __forceinline__ const TABPACK_GLOBAL V* glob(const V* p) {
  return (const TABPACK_GLOBAL V*)p;
}

// ---------------------------------------------------------------- loaders --
// A loader moves one R x 128-byte-depth operand tile per K step: load() issues
// raw buffer loads for depth offset k0 into registers, store() writes them to
// LDS.  An element outside the operand (row beyond the member's extent, depth
// beyond K) gets an offset past the buffer's range, which the hardware returns
// as zero -- no branch and no select on the data, so the loads stay in flight
// across the MFMAs of the current step.
constexpr uint32_t kOob = 0x80000000u;   // an offset outside every operand buffer
constexpr int kRsrcWord3 = 0x00020000;   // gfx9 raw buffer descriptor: 32-bit data format, no swizzle

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)(bytes < kOob ? bytes : kOob - 16),
                                           kRsrcWord3);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}

// Depth-contiguous operand (T), element (r, k) at P[r * ld + k] -> depth-contiguous LDS.
template <typename T, int R>
struct LoadKmaj {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int NV = R * KV / NT;
  u32x4 reg[NV];
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t off[NV];  // byte offset of this thread's vector at depth 0, or kOob
  int slot;
  __device__ void init(const T* P, int64_t ld, int row0, int rbound, int, int tid) {
    rsrc = make_rsrc(P, (int64_t)rbound * ld * (int64_t)sizeof(T));
    slot = tid % KV;  // NT is a multiple of KV: every vector of a thread has this slot
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int r = (tid + i * NT) / KV;
      off[i] = row0 + r < rbound ? (uint32_t)(((int64_t)(row0 + r) * ld + slot * VE) * sizeof(T)) : kOob;
    }
  }
  __device__ void load(int k0, int kd, int) {
    const bool kin = k0 + slot * VE < kd;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      reg[i] = buf_load16(rsrc, (kin && off[i] != kOob) ? off[i] + k0 * (uint32_t)sizeof(T) : kOob);
  }
  __device__ void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int v = tid + i * NT;
      *reinterpret_cast<u32x4*>(lds + kmaj_off(v / KV, v % KV)) = reg[i];
    }
  }
};

// Rows-contiguous fp32 operand: 4 x 4 blocks transposed in registers into the
// depth-contiguous LDS layout.
template <int R>
struct LoadRmajF32 {
  static constexpr int RB = R / 4;              // row blocks
  static constexpr int NBLK = RB * KV;          // blocks per tile
  static constexpr int PER = NBLK / NT;
  u32x4 reg[PER][4];
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t off[PER];
  int64_t ldb;
  __device__ void init(const float* P, int64_t ld, int row0, int rbound, int kd, int tid) {
    ldb = ld * 4;
    rsrc = make_rsrc(P, (int64_t)kd * ldb);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = tid + p * NT;
      const int rb = b % RB, kb = b / RB;
      off[p] = row0 + rb * 4 < rbound ? (uint32_t)(kb * 4 * ldb + (int64_t)(row0 + rb * 4) * 4) : kOob;
    }
  }
  __device__ void load(int k0, int kd, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int kb = (tid + p * NT) / RB;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool in = off[p] != kOob && k0 + kb * 4 + e < kd;
        reg[p][e] = buf_load16(rsrc, in ? off[p] + (uint32_t)((k0 + e) * ldb) : kOob);
      }
    }
  }
  __device__ void store(char* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int b = tid + p * NT;
      const int rb = b % RB, kb = b / RB;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4 o{reg[p][0][i], reg[p][1][i], reg[p][2][i], reg[p][3][i]};
        *reinterpret_cast<u32x4*>(lds + kmaj_off(rb * 4 + i, kb)) = o;
      }
    }
  }
};

// Direct-to-LDS loaders (bf16): buffer_load_dwordx4 ... lds writes lane i's 16
// bytes at the instruction's LDS base + 16 i, so each wave fills whole 1 KB
// chunks of the LDS tile and every lane fetches the global vector that belongs
// at its position in the swizzled layout.  Nothing is staged in registers.
// A lane's byte offset (the per-lane part of the address) is fixed for the
// whole tile; the K position moves in the scalar offset, so a K step costs no
// vector instructions.  A lane whose row lies outside the operand has an
// offset past the buffer's range and reads zeros; depth beyond K can only
// occur in the last K step, which checks it per lane.
typedef void __attribute__((address_space(3)))* lptr_t;
typedef __attribute__((address_space(3))) int32_t lds_i32;

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lptr_t)lds, 16, voff, soff, 0, 0);
}

// Depth-contiguous bf16 operand -> swizzled row-major LDS layout.  Each
// instruction fills BR = 32/KS whole rows (1 KB); wave w issues blocks
// w*PER .. w*PER+PER-1.  Lane i lands at row (i / CPR) of the block, chunk
// position i % CPR, so it fetches the row's chunk (i % CPR) ^ f(row).  f of a
// block's rows depends only on the block's parity.
template <int R, int KS>
struct DmaKmaj {
  static constexpr int CPR = 2 * KS;           // 16-byte chunks per row
  static constexpr int BR = 64 / CPR;          // rows per 1 KB block
  static constexpr int PER = R / BR / 4;       // blocks per wave
  static_assert(PER % 2 == 0, "block parity follows p");
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t voff[PER];  // byte offset (depth 0) of this lane's vector in block p, or kOob
  int kofs[2];         // depth offset (elements) of this lane's vector per block parity
  int wave;
  // rows != nullptr: row r < nrows of the operand is row rows[r] of P (src_rows
  // rows), rows >= nrows read as zero
  __device__ void init(const __bf16* P, int64_t ld, int row0, int rbound, int, int wave_, int lane,
                       const int32_t* rows = nullptr, int nrows = 0, int64_t src_rows = 0) {
    rsrc = make_rsrc(P, (rows ? src_rows : (int64_t)rbound) * ld * 2);
    wave = wave_;
    const int r = lane / CPR;
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int row = (wave * PER + par) * BR + r;
      kofs[par] = ((lane % CPR) ^ kmaj_f<KS>(row)) * 8;
    }
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int row = row0 + (wave * PER + p) * BR + r;
      if (rows)
        voff[p] = row < nrows ? (uint32_t)(((int64_t)rows[row] * ld + kofs[p & 1]) * 2) : kOob;
      else
        voff[p] = row < rbound ? (uint32_t)(((int64_t)row * ld + kofs[p & 1]) * 2) : kOob;
    }
  }
  __device__ void issue(char* lds, int k0, int kd) const {
    const uint32_t soff = (uint32_t)k0 * 2u;
    if (k0 + 16 * KS <= kd) {
#pragma unroll
      for (int p = 0; p < PER; ++p) dma16(rsrc, lds + (wave * PER + p) * 1024, voff[p], soff);
    } else {
      const bool kin0 = k0 + kofs[0] < kd, kin1 = k0 + kofs[1] < kd;
#pragma unroll
      for (int p = 0; p < PER; ++p)
        dma16(rsrc, lds + (wave * PER + p) * 1024, ((p & 1) ? kin1 : kin0) ? voff[p] : kOob, soff);
    }
  }
};

// Rows-contiguous bf16 operand -> rows-contiguous LDS layout (16*KS depth rows x R).
template <int R, int KS>
struct DmaRmaj {
  static constexpr int RBYTES = 2 * R;                      // bytes per depth row in LDS
  static constexpr int PER = 16 * KS * RBYTES / 1024 / 4;   // chunks per wave
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t ldb;        // bytes per depth row in HBM
  uint32_t voff[PER];  // byte offset (depth 0) of the vector this lane fetches for chunk p, or kOob
  int krow[PER];       // its depth row inside a K step
  int wave;
  // map != nullptr: depth row k < nmap is row map[k] (an LDS table) of P
  // (src_rows rows), depth rows >= nmap read as zero
  const lds_i32* map;
  int nmap;
  __device__ void init(const __bf16* P, int64_t ld, int row0, int rbound, int kd, int wave_, int lane,
                       const lds_i32* map_ = nullptr, int nmap_ = 0, int64_t src_rows = 0) {
    rsrc = make_rsrc(P, (map_ ? src_rows : (int64_t)kd) * ld * 2);
    wave = wave_;
    ldb = (uint32_t)(ld * 2);
    map = map_;
    nmap = nmap_;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int pos = (wave * PER + p) * 1024 + lane * 16;
      const int k = pos / RBYTES, b = pos % RBYTES;
      const int chunk = (b >> 5) ^ ((k & 3) << 1);
      const int col = chunk * 16 + ((b >> 4) & 1) * 8;
      krow[p] = k;
      const int64_t dep = map_ ? 0 : k * (int64_t)ldb;
      voff[p] = row0 + col < rbound ? (uint32_t)(dep + (int64_t)(row0 + col) * 2) : kOob;
    }
  }
  __device__ void issue(char* lds, int k0, int kd) const {
    if (map) {  // wave-uniform
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int k = k0 + krow[p];
        const uint32_t o = k < nmap && voff[p] != kOob ? (uint32_t)map[k] * ldb + voff[p] : kOob;
        dma16(rsrc, lds + (wave * PER + p) * 1024, o, 0);
      }
      return;
    }
    const uint32_t soff = (uint32_t)k0 * ldb;
    if (k0 + 16 * KS <= kd) {
#pragma unroll
      for (int p = 0; p < PER; ++p) dma16(rsrc, lds + (wave * PER + p) * 1024, voff[p], soff);
    } else {
#pragma unroll
      for (int p = 0; p < PER; ++p)
        dma16(rsrc, lds + (wave * PER + p) * 1024, k0 + krow[p] < kd ? voff[p] : kOob, soff);
    }
  }
};

// The embedded first-layer input E (App. "Feature Embeddings": feature x_i of
// a row gives alpha_i0 x_i + beta_i0 and, for j >= 1, alpha_ij cos(w x_i + b)
// + beta_ij) is never stored: the first layer's forward GEMM produces it as its
// A operand and the weight-gradient GEMM as its B operand, from the data rows
// and the member's column table.  Feature i owns the columns i dp .. i dp +
// dp - 1 (dp = d_emb rounded up to 8; the columns j >= d_emb are zero
// padding), so every 16-byte chunk of a row (8 bf16 or 4 fp32 columns, at a
// multiple of 8 or 4) belongs to one feature.  Table entry c = {w, b, alpha,
// beta} of column c (w = b = 0 at j = 0; zeros in the padding; bf16 packs
// hold w and b in revolutions).

// The value of one element: x is the row's value of the column's feature;
// MAYBE_J0: the column may be a feature's first (j = 0, flagged by j0).
template <bool FAST, bool MAYBE_J0>
__device__ __forceinline__ float emb_value(const f32x4& tv, float x, bool j0) {
  float g;
  if constexpr (FAST)
    g = __builtin_amdgcn_cosf(__builtin_amdgcn_fractf(fmaf(tv[0], x, tv[1])));
  else
    g = cosf(fmaf(tv[0], x, tv[1]));
  if constexpr (MAYBE_J0) {
    // computed for the element either way (the compiler would otherwise
    // branch around the cosine): the choice below stays a select
    asm volatile("" : "+v"(g));
    g = j0 ? x : g;
  }
  return fmaf(tv[2], g, tv[3]);
}

// 16 bytes of the operand in the GEMM precision from 16 / sizeof(T) values
template <typename T>
__device__ __forceinline__ u32x4 emb_pack(const float* v) {
  if constexpr (sizeof(T) == 2) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v[2 * q], v[2 * q + 1]}, bf16x2));
    return o;
  } else {
    return u32x4{__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                 __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])};
  }
}

struct EmbMember {
  __amdgpu_buffer_rsrc_t tab;  // the member's column table, p_in entries
  int dp, d_in1;
  uint32_t magic;              // ceil(2^32 / dp): feature of column c = umulhi(c, magic)
  __device__ void init(const GemmArgs& a, const GemmDesc& d) {
    const MemberDev& md = a.emb_mem[d.member];
    dp = (md.d_emb + 7) & ~7;
    d_in1 = a.emb_d_in - 1;
    magic = (uint32_t)((0x100000000ull + (uint64_t)dp - 1) / (uint64_t)dp);
    tab = make_rsrc(a.emb_tab + md.e_tab, (int64_t)md.p_in * 16);
  }
  __device__ f32x4 entry(int c) const { return __builtin_bit_cast(f32x4, buf_load16(tab, (uint32_t)c * 16u)); }
  // the feature of column c (clamped: columns past the table read zeros)
  __device__ int feature(int c) const { return min((int)__umulhi((uint32_t)c, magic), d_in1); }
  __device__ bool first(int c) const { return c == (int)__umulhi((uint32_t)c, magic) * dp; }  // j = 0
};

// A operand of the forward (rows: the tile's TM batch rows, depth-contiguous
// LDS layout): per K step, lane l of wave w produces chunk l / 8 of rows
// l % 8 + 8 w + (NTH / 8) i (i < 8 TM / NTH, NTH threads), so the 8 lanes of
// a lane group share a chunk and its table entries.  bf16: the K step's 64 table entries reach LDS with
// one direct load of wave 0 (two steps ahead, beside the W_1 stage), and each
// lane group reads its 8 from there (one address per group: no bank
// conflicts); the rows' x are loaded into registers two steps ahead.  fp32:
// each thread loads its chunk's entries itself.  Rows outside the batch read
// data row 0 (finite values; the epilogue zeroes those rows).
template <typename T, int TM = 128, int NTH = NT>
struct EmbRowsProducer {
  static constexpr int VE = 16 / sizeof(T);  // columns per chunk
  static constexpr int NR = TM * 8 / NTH;    // rows per thread
  static constexpr int RS = NTH / 8;         // row stride between a thread's rows
  EmbMember em;
  const float* xrow[NR];  // the rows' feature 0
  int slot, rl0, lane, wave;
  f32x4 tv[VE];           // the table entries of the step being produced
  float x[2][NR];         // the rows' x, two K steps in flight (register set = step & 1)
  __device__ void init(const GemmArgs& a, const GemmDesc& d, const Tile& t, int tid) {
    em.init(a, d);
    lane = tid % 64;
    wave = tid / 64;
    slot = lane / 8;
    rl0 = lane % 8 + 8 * wave;
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int r = t.m0 + rl0 + RS * i;
      const int64_t row =
          r < a.rows_valid ? (a.emb_idx ? (int64_t)a.emb_idx[(int64_t)d.member * a.rows_valid + r] : a.emb_row_base + r)
                           : 0;
      xrow[i] = a.emb_x + row * a.emb_d_in;
    }
  }
  // bf16: the 64 entries of the step at k0 into tlds (wave 0; lane l: entry k0 + l)
  __device__ void issue_tab(char* tlds, int k0) const {
    if (wave == 0) dma16(em.tab, tlds, (uint32_t)lane * 16u, (uint32_t)k0 * 16u);
  }
  __device__ void read_tab(const char* tlds) {
#pragma unroll
    for (int e = 0; e < VE; ++e) tv[e] = *reinterpret_cast<const f32x4*>(tlds + (slot * VE + e) * 16);
  }
  template <int S>
  __device__ void load_x(int k0) {
    const int f = em.feature(k0 + slot * VE);
#pragma unroll
    for (int i = 0; i < NR; ++i) x[S][i] = *glob(xrow[i] + f);
  }
  // fp32: entries and x of the step at k0 (register set 0)
  __device__ void load(int k0) {
    const int c = k0 + slot * VE;
#pragma unroll
    for (int e = 0; e < VE; ++e) tv[e] = em.entry(c + e);
    load_x<0>(k0);
  }
  // the chunk of the step at k0 from set S; off(row, slot): its byte offset in the A stage
  template <int S, typename Off>
  __device__ void store(char* lds, int k0, Off off) const {
    const bool j0 = em.first(k0 + slot * VE);
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      float v[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e)
        v[e] = e == 0 ? emb_value<sizeof(T) == 2, true>(tv[e], x[S][i], j0)
                      : emb_value<sizeof(T) == 2, false>(tv[e], x[S][i], false);
      *reinterpret_cast<u32x4*>(lds + off(rl0 + RS * i, slot)) = emb_pack<T>(v);
    }
  }
};

// B operand of the weight gradient (columns: the tile's 128 embedding
// columns, depth: batch rows).  The columns, their table entries and feature
// are fixed for the tile; per K step each thread fetches the x of its depth
// rows (data rows from the LDS map of the batch indices; rows past the batch
// read another batch row, whose products meet zero gradient rows).
//   bf16: chunk tid % 16 (8 columns) of depth rows tid / 16 + 16 i (i < 4),
//         into the rows-contiguous layout (rmaj_off);
//   fp32: column tid % 128 at depth rows 16 (tid / 128) .. + 15, four 16-byte
//         depth vectors into the depth-contiguous layout (kmaj_off).
template <typename T>
struct EmbColsProducer {
  static constexpr bool FAST = sizeof(T) == 2;
  static constexpr int NC = FAST ? 8 : 1;    // columns per thread
  static constexpr int NK = FAST ? 4 : 16;   // depth rows per thread per K step
  EmbMember em;
  f32x4 tv[NC];
  bool j0;
  int f;                        // the columns' feature
  int col, kr0;                 // the thread's first column (tile-relative), first depth row
  const float* X;
  int d_in;
  const lds_i32* map;
  int nmap;
  float x[FAST ? 2 : 1][NK];    // bf16: two K steps in flight (register sets S = step & 1)
  __device__ void init(const GemmArgs& a, const GemmDesc& d, const Tile& t, int tid, const lds_i32* map_,
                       int nmap_) {
    em.init(a, d);
    X = a.emb_x;
    d_in = a.emb_d_in;
    map = map_;
    nmap = nmap_;
    col = FAST ? (tid % 16) * 8 : tid % 128;
    kr0 = FAST ? tid / 16 : (tid / 128) * 16;
    const int c = t.n0 + col;
#pragma unroll
    for (int e = 0; e < NC; ++e) tv[e] = em.entry(c + e);
    f = em.feature(c);
    j0 = em.first(c);
  }
  __device__ int krow(int i) const { return FAST ? kr0 + 16 * i : kr0 + i; }
  template <int S>
  __device__ void load(int k0) {
#pragma unroll
    for (int i = 0; i < NK; ++i)  // rows past the batch read the batch's last row (any data row serves)
      x[S][i] = *glob(X + (int64_t)map[min(k0 + krow(i), nmap - 1)] * d_in + f);
  }
  template <int S>
  __device__ void store(char* lds) const {
    if constexpr (FAST) {
#pragma unroll
      for (int i = 0; i < NK; ++i) {
        float v[NC];
#pragma unroll
        for (int e = 0; e < NC; ++e)
          v[e] = e == 0 ? emb_value<true, true>(tv[e], x[S][i], j0) : emb_value<true, false>(tv[e], x[S][i], false);
        *reinterpret_cast<u32x4*>(lds + rmaj_off<128>(krow(i), col)) = emb_pack<T>(v);
      }
    } else {
#pragma unroll
      for (int s = 0; s < NK / 4; ++s) {
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = emb_value<false, true>(tv[0], x[S][4 * s + q], j0);
        *reinterpret_cast<u32x4*>(lds + kmaj_off(col, kr0 / 4 + s)) = emb_pack<T>(v);
      }
    }
  }
};

template <typename T, int KIND, int R, int KS>
struct LoaderFor;
template <int R, int KS>
struct LoaderFor<__bf16, OP_KMAJ, R, KS> {
  using type = DmaKmaj<R, KS>;
  static constexpr bool tr = false;  // fragments read from the depth-contiguous layout
  static constexpr bool dma = true;
};
template <int R, int KS>
struct LoaderFor<__bf16, OP_RMAJ, R, KS> {
  using type = DmaRmaj<R, KS>;
  static constexpr bool tr = true;   // fragments read with ds_read_b64_tr_b16
  static constexpr bool dma = true;
};
template <int R, int KS>
struct LoaderFor<float, OP_KMAJ, R, KS> {
  using type = LoadKmaj<float, R>;
  static constexpr bool tr = false;
  static constexpr bool dma = false;
};
template <int R, int KS>
struct LoaderFor<float, OP_RMAJ, R, KS> {
  using type = LoadRmajF32<R>;
  static constexpr bool tr = false;
  static constexpr bool dma = false;
};

// ------------------------------------------------------------- fragments --
// 8 bf16 of depth 16*ks + 8*h .. +7 (h = lane / 32) of operand row
// row_block + lane % 32, from the rows-contiguous layout.
template <int R>
__device__ __forceinline__ bf16x8 frag_tr(const char* lds, int row_block, int ks, int lane) {
  const int s = lane & 15, g = lane >> 4;
  const int k = 16 * ks + 8 * (g >> 1) + (s >> 2);
  const int col = row_block + 16 * (g & 1) + 4 * (s & 3);
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds + rmaj_off<R>(k, col)));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds + rmaj_off<R>(k + 4, col)));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], b[0], b[1]});
}

// The same fragment through inline assembly.  The compiler cannot prove that
// a transposing read of one stage does not alias the direct-to-LDS loads just
// issued into the other, and would wait for those loads before every read;
// through assembly the read is invisible to it, so the caller waits for the
// result itself (an explicit lgkmcnt before the first use).
template <int R>
__device__ __forceinline__ u32x2 ds_tr16_b64(const char* p) {
  typedef __attribute__((address_space(3))) const char* lds_cptr;
  const uint32_t a = (uint32_t)(uintptr_t)(lds_cptr)p;
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(a));
  return r;
}
template <int R>
__device__ __forceinline__ bf16x8 frag_tr_asm(const char* lds, int row_block, int ks, int lane) {
  const int s = lane & 15, g = lane >> 4;
  const int k = 16 * ks + 8 * (g >> 1) + (s >> 2);
  const int col = row_block + 16 * (g & 1) + 4 * (s & 3);
  const u32x2 a = ds_tr16_b64<R>(lds + rmaj_off<R>(k, col));
  const u32x2 b = ds_tr16_b64<R>(lds + rmaj_off<R>(k + 4, col));
  return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], b[0], b[1]});
}

template <int KS>
__device__ __forceinline__ bf16x8 frag_kmaj_asm(const char* lds, int row_block, int ks, int lane) {
  typedef __attribute__((address_space(3))) const char* lds_cptr;
  const uint32_t a = (uint32_t)(uintptr_t)(lds_cptr)(lds + kmaj16_off<KS>(row_block + (lane & 31), 2 * ks + (lane >> 5)));
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(a));
  return __builtin_bit_cast(bf16x8, r);
}

template <int KS>
__device__ __forceinline__ bf16x8 frag_kmaj_bf16(const char* lds, int row_block, int ks, int lane) {
  return *reinterpret_cast<const bf16x8*>(lds + kmaj16_off<KS>(row_block + (lane & 31), 2 * ks + (lane >> 5)));
}

template <bool TR, int R, int KS>
__device__ __forceinline__ bf16x8 frag_bf16(const char* lds, int row_block, int ks, int lane) {
  if constexpr (TR)
    return frag_tr<R>(lds, row_block, ks, lane);
  else
    return frag_kmaj_bf16<KS>(lds, row_block, ks, lane);
}

// ------------------------------------------------------------------- MFMA --
// One K step (128 bytes of depth) for this wave's MB x NB blocks.  Blocks
// outside the member's extents hold zeros and are computed anyway: the loop
// stays free of branches so LDS reads and MFMAs overlap.
template <typename T, int SH, bool TRA, bool TRB, int KS>
__device__ __forceinline__ void mma_step(const char* As, const char* Bs,
                                         f32x16 (&acc)[Shape<SH>::MB][Shape<SH>::NB], int wm, int wn,
                                         int lane) {
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB, TM = Shape<SH>::TM, TN = Shape<SH>::TN;
  if constexpr (sizeof(T) == 2 && SH != kShapeBig) {
    // Small and tall tiles: the fragments of 16-deep step ks + 2 are read
    // while the MFMAs of step ks run.  The scheduling barriers pin that order
    // (left alone, the scheduler reuses one set of fragment registers and
    // waits for the LDS before every 16-deep step).  Fragment reads go
    // through assembly, so the wait for a step's fragments is explicit: every
    // LDS read issued after them may still be in flight.
    constexpr int NRD = (TRA ? 2 * MB : MB) + (TRB ? 2 * NB : NB);  // LDS reads per 16-deep step
    bf16x8 a[KS][MB], b[KS][NB];
    auto rd = [&](int ks) {
#pragma unroll
      for (int i = 0; i < MB; ++i) {
        if constexpr (TRA)
          a[ks][i] = frag_tr_asm<TM>(As, wm * MB * 32 + i * 32, ks, lane);
        else
          a[ks][i] = frag_kmaj_asm<KS>(As, wm * MB * 32 + i * 32, ks, lane);
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        if constexpr (TRB)
          b[ks][j] = frag_tr_asm<TN>(Bs, wn * NB * 32 + j * 32, ks, lane);
        else
          b[ks][j] = frag_kmaj_asm<KS>(Bs, wn * NB * 32 + j * 32, ks, lane);
      }
    };
    rd(0);
    if constexpr (KS > 1) rd(1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 2 < KS) rd(ks + 2);
      {
        const int later = (ks + 1 < KS ? NRD : 0) + (ks + 2 < KS ? NRD : 0);
        __builtin_amdgcn_sched_barrier(0);
        if (later >= 15)
          __builtin_amdgcn_s_waitcnt(0xcf7f);  // lgkmcnt(15)
        else if (later >= 12)
          __builtin_amdgcn_s_waitcnt(0xcc7f);  // lgkmcnt(12)
        else if (later >= 8)
          __builtin_amdgcn_s_waitcnt(0xc87f);  // lgkmcnt(8)
        else if (later >= 6)
          __builtin_amdgcn_s_waitcnt(0xc67f);  // lgkmcnt(6)
        else if (later >= 4)
          __builtin_amdgcn_s_waitcnt(0xc47f);  // lgkmcnt(4)
        else
          __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][i], b[ks][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else if constexpr (sizeof(T) == 2) {
    // Big tiles: fragments of the next 16-deep step are read while the MFMAs
    // of this one run; the loop stays rolled (a full unroll hoists every step's
    // reads and does not fit beside 256 accumulators).  The last step re-reads
    // step 0, which is harmless.
    bf16x8 a[MB], b[NB];
#pragma unroll
    for (int i = 0; i < MB; ++i) a[i] = frag_bf16<TRA, TM, KS>(As, wm * MB * 32 + i * 32, 0, lane);
#pragma unroll
    for (int j = 0; j < NB; ++j) b[j] = frag_bf16<TRB, TN, KS>(Bs, wn * NB * 32 + j * 32, 0, lane);
#pragma unroll 1
    for (int ks = 0; ks < KS; ++ks) {
      const int kn = (ks + 1) & (KS - 1);
      bf16x8 na[MB], nb[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) na[i] = frag_bf16<TRA, TM, KS>(As, wm * MB * 32 + i * 32, kn, lane);
#pragma unroll
      for (int j = 0; j < NB; ++j) nb[j] = frag_bf16<TRB, TN, KS>(Bs, wn * NB * 32 + j * 32, kn, lane);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = na[i];
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j] = nb[j];
    }
  } else {
    const int rl = lane & 31, hv = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < KV / 2; ++ks) {
      f32x4 a[MB], b[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i)
        a[i] = *reinterpret_cast<const f32x4*>(As + kmaj_off(wm * MB * 32 + i * 32 + rl, 2 * ks + hv));
#pragma unroll
      for (int j = 0; j < NB; ++j)
        b[j] = *reinterpret_cast<const f32x4*>(Bs + kmaj_off(wn * NB * 32 + j * 32 + rl, 2 * ks + hv));
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
  }
}

// --------------------------------------------------------------- epilogue --
// Accumulator register r of a 32x32 block held by lane l is element
// (row 8*(r/4) + 4*(l/32) + r%4, col l%32): each lane owns 16 of the 32 rows
// of one column, i.e. half of the bits of one (32-row block, column) keep or
// mask word.
//
// Results leave through LDS: each wave stages one 32-row block of its
// 32 x (32*NB) output at a time in a private region of 32 * (NB*128 + 32)
// bytes (row stride padded so the two half-waves' column writes fall on
// disjoint banks; the operand buffers are free by then), then reads it back as
// 16-byte row vectors and stores whole row segments: a store instruction
// covers full 256- or 512-byte row pieces instead of 64-byte column strips.

template <typename OT, int NB>
struct Stage {
  static constexpr int ES = sizeof(OT);
  static constexpr int ROWS = 32;                                // rows per pass
  static constexpr int GP = ROWS / 8;                            // row runs (g values) per pass
  static constexpr int NPASS = 32 / ROWS;
  static constexpr int RS = NB * 32 * ES + (ES == 2 ? 16 : 32);  // padded row stride (bytes)
  static constexpr int VPR = NB * 32 * ES / 16;                  // 16-byte vectors per row
  static constexpr int PER_LANE = ROWS * VPR / 64;
  static constexpr int BYTES = 32 * (NB * 128 + 32);
  static_assert(ROWS * RS <= BYTES, "stage region");
};

// Makes the staged block written by every lane of the wave visible to the
// reads that follow (LDS executes one wave's operations in order; this keeps
// the compiler from moving them across each other).
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// g: the row run relative to the pass (0 .. GP-1)
template <typename OT, int NB>
__device__ __forceinline__ void stage_put(char* stage, int j, int g, int q, int lane, OT v) {
  using S = Stage<OT, NB>;
  *reinterpret_cast<OT*>(stage + (8 * g + 4 * (lane >> 5) + q) * S::RS + (32 * j + (lane & 31)) * S::ES) = v;
}

// Stores the staged rows: rows row0.., columns col0.. of C (ld in elements);
// rows >= M and vectors starting at or beyond N are skipped (N is a multiple
// of the vector width).
template <typename OT, int NB>
__device__ __forceinline__ void stage_flush(const char* stage, OT* C, int64_t ld, int row0, int col0, int M, int N,
                                            int lane) {
  using S = Stage<OT, NB>;
  constexpr int VE = 16 / S::ES;
#pragma unroll
  for (int it = 0; it < S::PER_LANE; ++it) {
    const int v = it * 64 + lane;
    const int r = v / S::VPR, c = v % S::VPR;
    const u32x4 x = *reinterpret_cast<const u32x4*>(stage + r * S::RS + c * 16);
    const int row = row0 + r, col = col0 + c * VE;
    if (row < M && col < N) *glob(reinterpret_cast<u32x4*>(C + (int64_t)row * ld + col)) = x;
  }
}

// Rows of alpha * Y + beta * acc from the staged fp32 accumulators: each lane
// takes 4 consecutive columns of a row (Y read as 4 elements), rounds once to
// OT and stores them; rows >= M and columns >= N are skipped (N is a multiple
// of 4).
template <typename OT, int NB>
__device__ __forceinline__ void stage_flush_ns(const char* stage, OT* C, int64_t ldc, const OT* Y, int64_t ldy,
                                               float alpha, float beta, int row0, int col0, int M, int N,
                                               int lane) {
  using S = Stage<float, NB>;
#pragma unroll
  for (int it = 0; it < S::PER_LANE; ++it) {
    const int v = it * 64 + lane;
    const int r = v / S::VPR, c = v % S::VPR;
    const f32x4 x = *reinterpret_cast<const f32x4*>(stage + r * S::RS + c * 16);
    const int row = row0 + r, col = col0 + c * 4;
    if (row >= M || col >= N) continue;
    float o[4] = {beta * x[0], beta * x[1], beta * x[2], beta * x[3]};
    if (Y) {
      const OT* yp = Y + (int64_t)row * ldy + col;
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = alpha * to_float(yp[q]) + o[q];
    }
    OT* cp = C + (int64_t)row * ldc + col;
    if constexpr (sizeof(OT) == 2) {
      const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[1]) << 16);
      const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[3]) << 16);
      *glob(reinterpret_cast<u32x2*>(cp)) = u32x2{lo, hi};
    } else {
      *glob(reinterpret_cast<f32x4*>(cp)) = f32x4{o[0], o[1], o[2], o[3]};
    }
  }
}

// The transpose of the staged block, for symmetric results: staged column c
// (C column col0 + c) becomes C row col0 + c, whose elements row0 .. row0 + 31
// each lane writes 4 at a time (Y read at the same transposed positions).
template <typename OT, int NB>
__device__ __forceinline__ void stage_flush_ns_mirror(const char* stage, OT* C, int64_t ldc, const OT* Y,
                                                      int64_t ldy, float alpha, float beta, int row0, int col0,
                                                      int M, int N, int lane) {
  using S = Stage<float, NB>;
  constexpr int CV = 32 / 4;  // 4-row vectors per staged column
#pragma unroll
  for (int it = 0; it < NB * 32 * CV / 64; ++it) {
    const int v = it * 64 + lane;
    const int c = v / CV, r = (v % CV) * 4;
    const int orow = col0 + c, ocol = row0 + r;
    if (orow >= M || ocol >= N) continue;
    float o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = beta * *reinterpret_cast<const float*>(stage + (r + q) * S::RS + c * 4);
    if (Y) {
      const OT* yp = Y + (int64_t)orow * ldy + ocol;
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = alpha * to_float(yp[q]) + o[q];
    }
    OT* cp = C + (int64_t)orow * ldc + ocol;
    if constexpr (sizeof(OT) == 2) {
      const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[1]) << 16);
      const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)o[3]) << 16);
      *glob(reinterpret_cast<u32x2*>(cp)) = u32x2{lo, hi};
    } else {
      *glob(reinterpret_cast<f32x4*>(cp)) = f32x4{o[0], o[1], o[2], o[3]};
    }
  }
}

// The last Newton-Schulz iteration's rows with the Muon update fused: the new
// X = alpha Y + beta (staged block), rounded to OT as it would be stored,
// replaces the staged values; then each weight element w it orthogonalises
// becomes w decay - step x (no contraction, as in the separate update), read
// row-wise or, for tall weights (W = X^T), column-wise from the stage.
template <typename OT, int NB>
__device__ __forceinline__ void stage_update_ns(const GemmArgs& a, const GemmDesc& d, char* stage, int row0, int col0,
                                                int lane) {
  using S = Stage<float, NB>;
  const OT* Y = static_cast<const OT*>(d.Y);
#pragma unroll
  for (int it = 0; it < S::PER_LANE; ++it) {
    const int v = it * 64 + lane;
    const int r = v / S::VPR, c = v % S::VPR;
    const int row = row0 + r, col = col0 + c * 4;
    if (row >= d.M || col >= d.N) continue;
    f32x4& x = *reinterpret_cast<f32x4*>(stage + r * S::RS + c * 16);
    const f32x4 xv = x;
    float o[4] = {a.ns_beta * xv[0], a.ns_beta * xv[1], a.ns_beta * xv[2], a.ns_beta * xv[3]};
    if (Y) {
      const OT* yp = Y + (int64_t)row * d.ldy + col;
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = a.ns_alpha * to_float(yp[q]) + o[q];
    }
    x = f32x4{to_float(from_float<OT>(o[0])), to_float(from_float<OT>(o[1])), to_float(from_float<OT>(o[2])),
              to_float(from_float<OT>(o[3]))};
  }
  wave_sync_lds();
  const float decay = d.ns_decay, step = d.ns_step;
  auto update = [&](int64_t e, const f32x4& x) {
    float* tp = a.ns_theta + d.poff + e;
    f32x4 w = *glob(reinterpret_cast<const f32x4*>(tp));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma clang fp contract(off)
      w[q] = w[q] * decay - step * x[q];
    }
    *glob(reinterpret_cast<f32x4*>(tp)) = w;
    if (a.ns_shadow) {
      const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[0]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[1]) << 16);
      const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[2]) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)w[3]) << 16);
      *glob(reinterpret_cast<u32x2*>(a.ns_shadow + d.poff + e)) = u32x2{lo, hi};
    }
  };
  if (!d.ns_tall) {  // W row = X row: the row-wise vectors above
#pragma unroll
    for (int it = 0; it < S::PER_LANE; ++it) {
      const int v = it * 64 + lane;
      const int r = v / S::VPR, c = v % S::VPR;
      const int row = row0 + r, col = col0 + c * 4;
      if (row >= d.M || col >= d.N) continue;
      update((int64_t)row * d.N + col, *reinterpret_cast<const f32x4*>(stage + r * S::RS + c * 16));
    }
  } else {  // W row = X column: 4 consecutive staged rows of one staged column
    constexpr int CV = 32 / 4;
#pragma unroll
    for (int it = 0; it < NB * 32 * CV / 64; ++it) {
      const int v = it * 64 + lane;
      const int c = v / CV, r = (v % CV) * 4;
      const int wrow = col0 + c, wcol = row0 + r;
      if (wrow >= d.N || wcol >= d.M) continue;
      f32x4 x;
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = *reinterpret_cast<const float*>(stage + (r + q) * S::RS + c * 4);
      update((int64_t)wrow * d.M + wcol, x);
    }
  }
}

// Weight-gradient rows with the optimizer fused: each staged vector holds the
// gradients of 4 consecutive weights, which are updated in place (theta, both
// moments, the bf16 shadow); the gradient itself is stored only on request.
// The optimizer state of all the lane's vectors is loaded before any update so
// the loads' latencies overlap.
template <int NB, int MB>
__device__ __forceinline__ void stage_flush_adamw(const GemmArgs& a, const GemmDesc& d, const char* stage, int row0,
                                                  int col0, int lane) {
  using S = Stage<float, NB>;
  // vectors whose optimizer state is loaded before any of them is updated:
  // all of the lane's 8 beside the small tile's 64 accumulators, 4 at a time
  // beside the 128 or 256 of the tall and big tiles
  constexpr int G = MB * NB <= 4 ? S::PER_LANE : 4;
  static_assert(S::PER_LANE % G == 0, "whole groups");
  const AdamConst ac = a.adam;
  const float decay = 1.0f - d.lr * d.wd;
  const float step = d.lr / ac.bc1;
#pragma unroll 1
  for (int it0 = 0; it0 < S::PER_LANE; it0 += G) {
    f32x4 g[G], th[G], m[G], vv[G];
    int64_t e[G];
    bool ok[G];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const int v = (it0 + u) * 64 + lane;
      const int r = v / S::VPR, c = v % S::VPR;
      const int row = row0 + r, col = col0 + c * 4;
      ok[u] = row < d.opt_rows && col < d.N;
      g[u] = *reinterpret_cast<const f32x4*>(stage + r * S::RS + c * 16);
      e[u] = (int64_t)row * d.ldc + col;
      if (ok[u]) {  // the optimizer state streams: non-temporal, so it does not evict GEMM operands
        th[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a.theta + d.poff + e[u]));
        m[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a.am + d.poff + e[u]));
        vv[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(a.av + d.poff + e[u]));
      }
    }
#pragma unroll
    for (int u = 0; u < G; ++u) {
      if (!ok[u]) continue;
      if (a.keep_grad) *glob(reinterpret_cast<f32x4*>(static_cast<float*>(d.C) + e[u])) = g[u];
      adamw_vec4(th[u], g[u], m[u], vv[u], decay, step, ac);
      __builtin_nontemporal_store(th[u], reinterpret_cast<f32x4*>(a.theta + d.poff + e[u]));
      __builtin_nontemporal_store(m[u], reinterpret_cast<f32x4*>(a.am + d.poff + e[u]));
      __builtin_nontemporal_store(vv[u], reinterpret_cast<f32x4*>(a.av + d.poff + e[u]));
      if (a.shadow) {  // read by the next forward and dX GEMMs: a normal store
        const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[u][0]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[u][1]) << 16);
        const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[u][2]) |
                            ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)th[u][3]) << 16);
        *reinterpret_cast<u32x2*>(a.shadow + d.poff + e[u]) = u32x2{lo, hi};
      }
    }
  }
}

// Weight-gradient tile of the small shape with the optimizer fused, done by
// the whole workgroup: the 128 x 128 fp32 gradient tile is staged in LDS (it
// fills the 64 KB the operand stages used), then the 256 threads stream the
// optimizer over it in row-contiguous 16-byte vectors, 16 per thread, with the
// optimizer state of kAdamAhead vectors in flight ahead of the one being
// updated, so the update of one vector never waits for the stores of the one
// before.  LDS layout: element (r, c) at r * 512 + 16 ((c / 4) ^ 8 ((r / 4) & 1))
// + 4 (c % 4): the two half-waves of an accumulator write (rows 4 apart) fall
// on disjoint banks, and each 16-byte vector stays contiguous.
// Vectors in flight: 8 (210 VGPRs) measured 0.8% faster per training step than
// 4; 16 exceeds the register budget of two workgroups per CU and spills.
#ifndef TABPACK_ADAM_AHEAD
#define TABPACK_ADAM_AHEAD 8
#endif
constexpr int kAdamAhead = TABPACK_ADAM_AHEAD;
__device__ __forceinline__ int dwt_off(int r, int c) {
  return r * 512 + ((((c >> 2) ^ (((r >> 2) & 1) << 3))) << 4) + ((c & 3) << 2);
}

// rows of the gradient tile staged per pass: the whole tile when the small
// kernel's LDS holds it, else halves (every kernel has at least that much LDS)
constexpr int kDwPassRows = kLdsSmallBf16 >= 128 * 512 ? 128 : 64;

__device__ __forceinline__ void dw_adamw_small(const GemmArgs& a, const GemmDesc& d, const Tile& t,
                                               f32x16 (&acc)[2][2], int wm, int wn, int lane, int tid, char* lds0) {
  constexpr int NPASS = 128 / kDwPassRows;
  constexpr int NV = kDwPassRows / 8;  // vectors per thread per pass
  const int hv = lane >> 5;
  const AdamConst ac = a.adam;
  const float decay = 1.0f - d.lr * d.wd;
  const float step = d.lr / ac.bc1;
  // the rows that hold weights (the padding rows stay zero: not loaded, not written)
  const int mrows = min(d.opt_rows - t.m0, 128), ncols = min(d.N - t.n0, 128);
  // vector u of this thread in a pass: row 8 u + tid / 32 of the pass, columns 4 (tid % 32) .. +3
  const int r0 = tid >> 5, c = (tid & 31) * 4;
  const bool colok = c < ncols;
  const int64_t estep = 8 * d.ldc;
  float* th_p = a.theta + d.poff;
  float* m_p = a.am + d.poff;
  float* v_p = a.av + d.poff;
  f32x4 th[kAdamAhead], m[kAdamAhead], vv[kAdamAhead];
#pragma unroll 1
  for (int pass = 0; pass < NPASS; ++pass) {
    const int prow0 = pass * kDwPassRows;  // first tile row of this pass
    const int64_t e0 = (int64_t)(t.m0 + prow0 + r0) * d.ldc + t.n0 + c;  // element offset of vector 0
    auto ok = [&](int u) { return colok && prow0 + 8 * u + r0 < mrows; };
    auto load = [&](int u) {
      const int64_t e = e0 + u * estep;
      if (ok(u)) {
        th[u % kAdamAhead] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(th_p + e));
        m[u % kAdamAhead] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(m_p + e));
        vv[u % kAdamAhead] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(v_p + e));
      }
    };
    if (pass > 0) {
      wait_vm<63, true>();
      bar();  // every thread is done reading the previous pass
    }
    // the first vectors' optimizer state is requested before the gradient
    // tile is staged, so its latency overlaps the staging and the barrier
#pragma unroll
    for (int u = 0; u < kAdamAhead; ++u) load(u);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm * 64 + 32 * i + 8 * (r >> 2) + 4 * hv + (r & 3) - prow0;
          const int col = wn * 64 + 32 * j + (lane & 31);
          if (row >= 0 && row < kDwPassRows) *reinterpret_cast<float*>(lds0 + dwt_off(row, col)) = acc[i][j][r];
        }
    wait_vm<63, true>();  // this wave's LDS writes are done (the state loads may still be in flight)
    bar();
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int b = u % kAdamAhead;
      const int64_t e = e0 + u * estep;
      const bool in = ok(u);
      f32x4 g = *reinterpret_cast<const f32x4*>(lds0 + dwt_off(8 * u + r0, c));
      f32x4 t_ = th[b], m_ = m[b], v_ = vv[b];
      if (u + kAdamAhead < NV) load(u + kAdamAhead);
      if (in) {
        if (a.keep_grad) *glob(reinterpret_cast<f32x4*>(static_cast<float*>(d.C) + e)) = g;
        adamw_vec4(t_, g, m_, v_, decay, step, ac);
        __builtin_nontemporal_store(t_, reinterpret_cast<f32x4*>(th_p + e));
        __builtin_nontemporal_store(m_, reinterpret_cast<f32x4*>(m_p + e));
        __builtin_nontemporal_store(v_, reinterpret_cast<f32x4*>(v_p + e));
        if (a.shadow) {
          const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)t_[0]) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)t_[1]) << 16);
          const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)t_[2]) |
                              ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)t_[3]) << 16);
          *reinterpret_cast<u32x2*>(a.shadow + d.poff + e) = u32x2{lo, hi};
        }
      }
    }
  }
}

// Small per-lane inputs of the epilogue, loaded when a tile starts so that
// their latency hides behind the main loop: the dropout keep words (forward),
// the bias (forward), the keep/ReLU mask words of the previous layer (dX).
// Word (i, j) covers rows 32*i .. 32*i+31 of the wave's block, column
// lane%32 of block j.
template <int SH>
struct EpiPre {
  uint32_t w[Shape<SH>::MB][Shape<SH>::NB];
  float bias[Shape<SH>::NB];
};

template <int EPI, int SH>
__device__ __forceinline__ void epi_prefetch(const GemmDesc& d, const Tile& t, int wm, int wn, int lane,
                                             EpiPre<SH>& pre) {
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB;
  const int colL = t.n0 + wn * NB * 32 + (lane & 31);
  const int rb0 = (t.m0 + wm * MB * 32) / 32;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const bool colin = colL + 32 * j < d.N;
    pre.bias[j] = 0.0f;
    if constexpr (EPI == EPI_FWD || EPI == EPI_FWD_EVAL)
      if (colin) pre.bias[j] = *glob(d.bias + colL + 32 * j);
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const bool in = colin && (rb0 + i) * 32 < d.M;
      pre.w[i][j] = EPI == EPI_DX ? 0u : ~0u;
      if constexpr (EPI == EPI_FWD) {
        if (d.drop_t != 0u && in) pre.w[i][j] = *glob(d.keepw + (int64_t)(rb0 + i) * d.N + colL + 32 * j);
      } else if constexpr (EPI == EPI_DX) {
        if (in) pre.w[i][j] = *glob(d.mask + (int64_t)(rb0 + i) * d.N + colL + 32 * j);
      }
    }
  }
}

template <typename T, int EPI, int SH>
__device__ __forceinline__ void epilogue(const GemmArgs& a, const GemmDesc& d, const Tile& t,
                                         f32x16 (&acc)[Shape<SH>::MB][Shape<SH>::NB], int wm, int wn, int lane,
                                         int mv, int nv, char* stage, const EpiPre<SH>& pre) {
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB;
  const int hv = lane >> 5;
  const int col0 = t.n0 + wn * NB * 32;  // the wave's first column
  const int row0 = t.m0 + wm * MB * 32;  // the wave's first row
  const int colL = col0 + (lane & 31);   // this lane's column in block j: colL + 32 j
  bool colin[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) colin[j] = j < nv && colL + 32 * j < d.N;
  if constexpr (EPI == EPI_DW) {
    using S = Stage<float, NB>;
    float* C = static_cast<float*>(d.C);
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      if (i >= mv) continue;
#pragma unroll
      for (int p = 0; p < S::NPASS; ++p) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int g = 0; g < S::GP; ++g)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              stage_put<float, NB>(stage, j, g, q, lane, acc[i][j][4 * (p * S::GP + g) + q]);
        wave_sync_lds();
        if (a.theta)
          stage_flush_adamw<NB, MB>(a, d, stage, row0 + 32 * i + S::ROWS * p, col0, lane);
        else
          stage_flush<float, NB>(stage, C, d.ldc, row0 + 32 * i + S::ROWS * p, col0, d.M, d.N, lane);
        wave_sync_lds();
      }
    }
  } else if constexpr (EPI == EPI_NS) {
    using S = Stage<float, NB>;
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      if (i >= mv) continue;
#pragma unroll
      for (int p = 0; p < S::NPASS; ++p) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int g = 0; g < S::GP; ++g)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              stage_put<float, NB>(stage, j, g, q, lane, acc[i][j][4 * (p * S::GP + g) + q]);
        wave_sync_lds();
        if (a.ns_theta) {  // uniform: the last iteration applies the Muon update instead of storing X
          stage_update_ns<T, NB>(a, d, stage, row0 + 32 * i + S::ROWS * p, col0, lane);
        } else {
          stage_flush_ns<T, NB>(stage, static_cast<T*>(d.C), d.ldc, static_cast<const T*>(d.Y), d.ldy, a.ns_alpha,
                                a.ns_beta, row0 + 32 * i + S::ROWS * p, col0, d.M, d.N, lane);
          if (a.ns_sym && t.m0 < t.n0)  // uniform: a tile above the diagonal also writes its mirror image
            stage_flush_ns_mirror<T, NB>(stage, static_cast<T*>(d.C), d.ldc, static_cast<const T*>(d.Y), d.ldy,
                                         a.ns_alpha, a.ns_beta, row0 + 32 * i + S::ROWS * p, col0, d.M, d.N, lane);
        }
        wave_sync_lds();
      }
    }
  } else if constexpr (EPI == EPI_DX) {
    // dZ = dH * [H_prev > 0] * s; the keep/ReLU decisions of the forward pass
    // come as mask words (bit r of word (row/32, col) = row 32*(row/32) + r).
    // Column sums of dZ per 64-row half go to colpart (bias-gradient
    // partials, reduced by a later kernel).
    using S = Stage<T, NB>;
    T* C = static_cast<T*>(d.C);
    float cs[NB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      const int rb = row0 + 32 * i;
      if ((i & 1) == 0) {
#pragma unroll
        for (int j = 0; j < NB; ++j) cs[j] = 0.0f;
      }
      const uint32_t(&mw)[NB] = pre.w[i];
#pragma unroll
      for (int p = 0; p < S::NPASS; ++p) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int g = 0; g < S::GP; ++g)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int gg = p * S::GP + g;
              const float dz =
                  ((mw[j] >> (8 * gg + 4 * hv + q)) & 1) ? acc[i][j][4 * gg + q] * d.drop_s : 0.0f;
              cs[j] += dz;
              stage_put<T, NB>(stage, j, g, q, lane, from_float<T>(dz));
            }
        wave_sync_lds();
        stage_flush<T, NB>(stage, C, d.ldc, rb + S::ROWS * p, col0, d.M, d.N, lane);
        wave_sync_lds();
      }
      if (i & 1) {
        const int hb = row0 + 32 * (i - 1);  // first row of this 64-row half
        const int64_t prow = (int64_t)(hb / kPartRows) * d.N;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          // lanes l and l^32 hold the two interleaved row halves of one column
          const float c = cs[j] + __shfl_xor(cs[j], 32, 64);
          if (hv == 0 && colin[j] && hb < d.M) *glob(d.colpart + prow + colL + 32 * j) = c;
        }
      }
    }
  } else {
    using S = Stage<T, NB>;
    T* C = static_cast<T*>(d.C);
    const float(&bias)[NB] = pre.bias;
    const float s_keep = (EPI == EPI_FWD) ? d.drop_s : 1.0f;
#pragma unroll
    for (int i = 0; i < MB; ++i) {
      if (i >= mv) continue;
      const int rb = row0 + 32 * i;
      // one word per column decides which of the block's rows keep their
      // value: bit r is set when row rb + r is kept by dropout, exists in the
      // batch, and the column lies in the member's true width.  Shifted by
      // 4 hv, bit 8 g + q is this lane's element (g, q).
      const int nrow = a.rows_valid - rb;
      const uint32_t rowmask = nrow >= 32 ? ~0u : (nrow <= 0 ? 0u : (1u << nrow) - 1u);
      uint32_t kw[NB], mw[NB];
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const uint32_t w = (EPI == EPI_FWD ? pre.w[i][j] : ~0u) & rowmask;
        kw[j] = colL + 32 * j < d.width ? w >> (4 * hv) : 0u;
        mw[j] = 0u;
      }
#pragma unroll
      for (int p = 0; p < S::NPASS; ++p) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int g = 0; g < S::GP; ++g)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int gg = p * S::GP + g;
              const int b = 8 * gg + q;
              float h = fmaxf(acc[i][j][4 * gg + q] + bias[j], 0.0f);
              if constexpr (EPI == EPI_FWD) h *= s_keep;
              h = ((kw[j] >> b) & 1u) ? h : 0.0f;
              const T hs = from_float<T>(h);
              // H > 0 (h >= 0, so only a zero of either sign has a zero magnitude)
              if constexpr (sizeof(T) == 2)
                mw[j] |= (uint32_t)((__builtin_bit_cast(uint16_t, hs) & 0x7fffu) != 0u) << b;
              else
                mw[j] |= (uint32_t)((__builtin_bit_cast(uint32_t, hs) & 0x7fffffffu) != 0u) << b;
              stage_put<T, NB>(stage, j, g, q, lane, hs);
            }
        wave_sync_lds();
        stage_flush<T, NB>(stage, C, d.ldc, rb + S::ROWS * p, col0, d.M, d.N, lane);
        wave_sync_lds();
      }
      if constexpr (EPI == EPI_FWD) {
        // mask words for the backward pass: the two half-waves hold
        // complementary bits of the same (32-row block, column) word
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const uint32_t mine = mw[j] << (4 * hv);
          const uint32_t w = mine | (uint32_t)__shfl_xor((int)mine, 32, 64);
          if (hv == 0 && colin[j] && rb < d.M) *glob(d.mask + (int64_t)(rb >> 5) * d.N + colL + 32 * j) = w;
        }
      }
    }
  }
}

// ------------------------------------------------------------------- tile --
// Waits until at most `newer` K steps (of PS direct loads per wave each) are
// still in flight and this wave's LDS reads are done.
template <int PS, int NS>
__device__ __forceinline__ void wait_stage(int newer) {
  static_assert(NS >= 2 && NS <= 8 && (NS - 2) * PS < 64, "vmcnt holds the newer steps' loads");
  switch (newer < NS - 2 ? (newer < 0 ? 0 : newer) : NS - 2) {
    case 0: wait_vm<0, true>(); break;
    case 1: wait_vm<(NS > 2 ? PS : 0), true>(); break;
    case 2: wait_vm<(NS > 3 ? 2 * PS : 0), true>(); break;
    case 3: wait_vm<(NS > 4 ? 3 * PS : 0), true>(); break;
    case 4: wait_vm<(NS > 5 ? 4 * PS : 0), true>(); break;
    case 5: wait_vm<(NS > 6 ? 5 * PS : 0), true>(); break;
    default: wait_vm<(NS > 7 ? 6 * PS : 0), true>(); break;
  }
}

// One output tile over the member's whole depth.  bf16 operands stream into
// LDS with direct loads in NS stages of KS 16-deep MFMA steps: NS-1 K steps are
// in flight while one is computed.  fp32 operands go through registers with
// two stages.
// EPI_DE: the tile's block of dE = dZ_1 W_1 (rows: batch rows, columns: the
// embedded inputs i d_emb + j) reduced into the embedding parameters' gradient
// terms.  The x values of the tile's rows and features are staged in LDS
// first (the operand buffers are free); each lane then walks the 16 rows it
// holds of each 32 x 32 block, the lanes l and l + 32 holding the other rows
// of the same column are added, and each wave writes its 64-row block's four
// sums per column.  Batch rows >= rows_valid are left out.
constexpr int kDeFeat = 18;  // features of 128 columns: at most 127 / 8 + 2 (8 or more columns per feature)
template <typename T, int SH>
__device__ __forceinline__ void epilogue_de(const GemmArgs& a, const GemmDesc& d, const Tile& t,
                                            f32x16 (&acc)[Shape<SH>::MB][Shape<SH>::NB], int wm, int wn,
                                            int lane, int tid, char* lds0) {
  static_assert(SH == kShapeSmall, "dE tiles are small tiles");
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB, TM = Shape<SH>::TM;
  constexpr bool FAST = sizeof(T) == 2;
  const MemberDev& md = a.emb_mem[d.member];
  // feature i owns columns i dp .. i dp + dp - 1, the last dp - d_emb of them zero padding
  const int d_emb = md.d_emb, dp = (d_emb + 7) & ~7, d_in = a.emb_d_in, ncol = d_in * dp;
  int64_t* rowoff = reinterpret_cast<int64_t*>(lds0);                    // [TM]
  float(*xs)[kDeFeat] = reinterpret_cast<float(*)[kDeFeat]>(lds0 + TM * 8);  // [TM][kDeFeat]
  const int i0 = min(t.n0, ncol - 1) / dp;
  const int nf = min(d_in - 1, (min(t.n0 + TM, ncol) - 1) / dp) - i0 + 1;
  if (tid < TM) {
    const int r = t.m0 + tid;
    rowoff[tid] = r < a.rows_valid ? (int64_t)a.emb_idx[(int64_t)d.member * a.rows_valid + r] * d_in : -1;
  }
  __syncthreads();
  for (int e = tid; e < TM * nf; e += NT) {
    const int r = e / nf, f = e - r * nf;
    const int64_t xo = rowoff[r];
    xs[r][f] = xo >= 0 ? a.emb_x[xo + i0 + f] : 0.0f;
  }
  __syncthreads();
  const int hv = lane >> 5;
  float* part = static_cast<float*>(d.C) + (int64_t)((t.m0 >> 6) + wm) * 4 * d.ldc;
  const bool all_rows = t.m0 + TM <= a.rows_valid;  // uniform
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int col = t.n0 + wn * NB * 32 + 32 * j + (lane & 31);
    const int fi = col / dp, fj = col - fi * dp;
    const int f = min(fi - i0, nf - 1);  // padding columns past the last feature read a staged one
    const bool on = col < ncol && fj < d_emb, j0 = fj == 0;
    // the column's table entry {w, b, alpha, beta} (bf16 packs: w, b in revolutions; zeros in the
    // padding), as the producers of E use it
    const f32x4 te = on ? __builtin_bit_cast(f32x4, a.emb_tab[md.e_tab + col]) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // s0 = sum g f (f = x at j = 0, else cos), s1 = sum g, u = sum g sin, v = sum g sin x; the w and b
    // terms are -alpha v and -alpha u (unused at j = 0), every element computed the same way
    float s0 = 0.0f, s1 = 0.0f, u = 0.0f, v = 0.0f;
    // ALL: every row of the tile is a batch row (the common case: a loop without the row test)
    auto sums = [&](auto ALL) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wm * MB * 32 + 32 * i + 8 * (r >> 2) + 4 * hv + (r & 3);
        float g = acc[i][j][r];
        if constexpr (!ALL.value)
          if (t.m0 + rl >= a.rows_valid) g = 0.0f;
        const float x = xs[rl][f];
        float sn, cs;
        if constexpr (FAST) {
          const float rev = __builtin_amdgcn_fractf(fmaf(te[0], x, te[1]));
          sn = __builtin_amdgcn_sinf(rev);
          cs = __builtin_amdgcn_cosf(rev);
        } else {
          sincosf(fmaf(te[0], x, te[1]), &sn, &cs);
        }
        s1 += g;
        s0 = fmaf(g, j0 ? x : cs, s0);
        const float gs = g * sn;
        u += gs;
        v = fmaf(gs, x, v);
      }
    };
    if (all_rows)
      sums(std::true_type{});
    else
      sums(std::false_type{});
    s0 += __shfl_xor(s0, 32, 64);
    s1 += __shfl_xor(s1, 32, 64);
    u += __shfl_xor(u, 32, 64);
    v += __shfl_xor(v, 32, 64);
    if (on && hv == 0) {
      part[col] = s0;
      part[d.ldc + col] = s1;
      part[2 * d.ldc + col] = -te[2] * v;
      part[3 * d.ldc + col] = -te[2] * u;
    }
  }
}

template <typename T, int AK, int BK_, int EPI, int SH, int KS, int NS>
__device__ __forceinline__ void run_tile(const GemmArgs& a, const GemmDesc& d, const Tile& t, char* lds0, int tid,
                                         int wave, char* xmap = nullptr) {
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB, TM = Shape<SH>::TM, TN = Shape<SH>::TN;
  using LA = LoaderFor<T, AK, TM, KS>;
  using LB = LoaderFor<T, BK_, TN, KS>;
  const int lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  // this wave's 32-blocks inside the member's extents (wave-uniform); a wave
  // with none skips its MFMAs but still takes part in loads and barriers
  const int mrem = d.M - (t.m0 + wm * MB * 32), nrem = d.N - (t.n0 + wn * NB * 32);
  const int mv = mrem <= 0 ? 0 : (mrem >= MB * 32 ? MB : (mrem + 31) / 32);
  const int nv = nrem <= 0 ? 0 : (nrem >= NB * 32 ? NB : (nrem + 31) / 32);
  const bool compute = mv > 0 && nv > 0;

  typename LA::type la;
  typename LB::type lb;

  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  EpiPre<SH> pre;
  epi_prefetch<EPI, SH>(d, t, wm, wn, lane, pre);

  if constexpr (LA::dma) {
    static_assert(LB::dma, "both operands staged the same way");
    constexpr int BKE = 16 * KS;                      // depth (elements) per K step
    constexpr int TA = TM * 32 * KS, TB = TN * 32 * KS;  // operand tile bytes per K step
    constexpr int PS = LA::type::PER + LB::type::PER;  // direct loads per wave per K step
    const int nk = (d.Kd + BKE - 1) / BKE;
    if constexpr (AK == OP_KMAJ && (EPI == EPI_FWD || EPI == EPI_FWD_EVAL))
      la.init(static_cast<const T*>(d.A), d.lda, t.m0, d.M, d.Kd, wave, lane, d.xrows, d.xrows_n, d.xsrc_rows);
    else
      la.init(static_cast<const T*>(d.A), d.lda, t.m0, d.M, d.Kd, wave, lane);
    if constexpr (BK_ == OP_RMAJ && EPI == EPI_DW) {
      if (d.xrows) {  // the batch rows' row numbers, for every K step's loads (one table per tile)
        lds_i32* m = (lds_i32*)xmap;
        for (int i = tid; i < d.xrows_n; i += NT) m[i] = d.xrows[i];
        __syncthreads();
        lb.init(static_cast<const T*>(d.B), d.ldb, t.n0, d.N, d.Kd, wave, lane, m, d.xrows_n, d.xsrc_rows);
      } else {
        lb.init(static_cast<const T*>(d.B), d.ldb, t.n0, d.N, d.Kd, wave, lane);
      }
    } else {
      lb.init(static_cast<const T*>(d.B), d.ldb, t.n0, d.N, d.Kd, wave, lane);
    }
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
      if (s < nk) {
        char* b = lds0 + s * (TA + TB);
        la.issue(b, s * BKE, d.Kd);
        lb.issue(b + TA, s * BKE, d.Kd);
      }
    for (int kt = 0; kt < nk; ++kt) {
      // step kt has landed in every wave's share and every wave is done with
      // the buffer the next load overwrites (it held step kt-1)
      wait_stage<PS, NS>(min(NS - 2, nk - 1 - kt));
      bar();
      if (kt + NS - 1 < nk) {
        char* b = lds0 + ((kt + NS - 1) % NS) * (TA + TB);
        la.issue(b, (kt + NS - 1) * BKE, d.Kd);
        lb.issue(b + TA, (kt + NS - 1) * BKE, d.Kd);
      }
      char* cur = lds0 + (kt % NS) * (TA + TB);
      if (compute) mma_step<T, SH, LA::tr, LB::tr, KS>(cur, cur + TA, acc, wm, wn, lane);
    }
    wait_vm<0, true>();
    bar();  // the epilogue stages results in the operand buffers
  } else {
    constexpr int BKE = KV * Elem<T>::VE;
    constexpr int TA = TM * ROW, TB = TN * ROW;
    char* lds1 = lds0 + TA + TB;
    const int nk = (d.Kd + BKE - 1) / BKE;
    la.init(static_cast<const T*>(d.A), d.lda, t.m0, d.M, d.Kd, tid);
    lb.init(static_cast<const T*>(d.B), d.ldb, t.n0, d.N, d.Kd, tid);
    la.load(0, d.Kd, tid);
    lb.load(0, d.Kd, tid);
    la.store(lds0, tid);
    lb.store(lds0 + TA, tid);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      char* cur = (kt & 1) ? lds1 : lds0;
      char* nxt = (kt & 1) ? lds0 : lds1;
      const bool more = kt + 1 < nk;
      if (more) {
        la.load((kt + 1) * BKE, d.Kd, tid);
        lb.load((kt + 1) * BKE, d.Kd, tid);
      }
      if (compute) mma_step<T, SH, LA::tr, LB::tr, KS>(cur, cur + TA, acc, wm, wn, lane);
      if (more) {
        la.store(nxt, tid);
        lb.store(nxt + TA, tid);
      }
      __syncthreads();
    }
  }
  if constexpr (EPI == EPI_DW && SH == kShapeSmall && sizeof(T) == 2) {
    if (a.theta) {  // uniform: the whole workgroup takes the staged-tile path
      dw_adamw_small(a, d, t, acc, wm, wn, lane, tid, lds0);
      return;
    }
  }
  if constexpr (EPI == EPI_DE)
    epilogue_de<T, SH>(a, d, t, acc, wm, wn, lane, tid, lds0);
  else
    epilogue<T, EPI, SH>(a, d, t, acc, wm, wn, lane, mv, nv, lds0 + wave * Shape<SH>::STAGE, pre);
}

// Output tiles of the embedded first layer (small tiles): the forward, whose A
// operand (E) EmbRowsProducer produces, and the weight gradient, whose B
// operand (E) EmbColsProducer produces; the other operand streams as in
// run_tile.  bf16: two stages of 64-deep steps; at step kt the producer's
// loads and the other operand's direct loads for step kt + 1 are issued, the
// MFMAs of step kt run, then the producer writes step kt + 1 into the other
// stage (its loads have landed by then).  fp32: the register-staged two-stage
// loop of run_tile with the producer as one of the loaders.
template <int EPI, int SH>
__device__ __forceinline__ void tile_extents(const GemmDesc& d, const Tile& t, int wm, int wn, int& mv, int& nv) {
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB;
  const int mrem = d.M - (t.m0 + wm * MB * 32), nrem = d.N - (t.n0 + wn * NB * 32);
  mv = mrem <= 0 ? 0 : (mrem >= MB * 32 ? MB : (mrem + 31) / 32);
  nv = nrem <= 0 ? 0 : (nrem >= NB * 32 ? NB : (nrem + 31) / 32);
}

// SH: small tiles (4 waves in 2 x 2) or, for the forward in bf16, wide tiles
// (8 waves in 2 x 4: twice the output columns per produced A element) and
// tall 8-wave tiles (4 x 2) for a last strip of at most 128 columns
template <typename T, int AK, int BK_, int EPI, int SH = kShapeSmall>
__device__ __forceinline__ void run_tile_emb(const GemmArgs& a, const GemmDesc& d, const Tile& t, char* lds0, int tid,
                                             int wave, char* xmap) {
  constexpr bool FWD = AK == OP_EMB;  // else the weight gradient (B produced)
  static_assert(FWD ? BK_ == OP_KMAJ : (AK == OP_RMAJ && BK_ == OP_EMB && EPI == EPI_DW), "embedded operand");
  constexpr bool WIDE = SH == kShapeWide, W8 = WIDE || SH == kShapeTall8;
  static_assert(SH == kShapeSmall || (W8 && FWD && sizeof(T) == 2), "8-wave tiles: the bf16 forward");
  constexpr int NW = W8 ? 8 : 4;  // waves
  constexpr int MB = Shape<SH>::MB, NB = Shape<SH>::NB, TM = Shape<SH>::TM, TN = Shape<SH>::TN;
  const int lane = tid & 63;
  const int wm = WIDE ? wave >> 2 : wave >> 1, wn = WIDE ? wave & 3 : wave & 1;
  int mv, nv;
  tile_extents<EPI, SH>(d, t, wm, wn, mv, nv);
  const bool compute = mv > 0 && nv > 0;
  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  EpiPre<SH> pre;
  epi_prefetch<EPI, SH>(d, t, wm, wn, lane, pre);
  // the producer (A or B) and the streamed operand (B = W_1, or A = dZ_1)
  std::conditional_t<FWD, EmbRowsProducer<T, TM, 64 * NW>, EmbColsProducer<T>> ep;
  if constexpr (FWD) {
    ep.init(a, d, t, tid);
  } else {  // the batch rows' data rows, for every K step's x loads (one table per tile)
    lds_i32* m = (lds_i32*)xmap;
    for (int i = tid; i < d.xrows_n; i += NT) m[i] = d.xrows[i];
    __syncthreads();
    ep.init(a, d, t, tid, m, d.xrows_n);
  }
  if constexpr (sizeof(T) == 2) {
    constexpr int KS = kSmallKs;
    static_assert(KS == 4 && kSmallNs == 2, "the producers fill 64-deep steps of two stages");
    // 8-wave tiles: waves 4 h .. 4 h + 3 load B rows h TN / 2 .. (h + 1) TN / 2 - 1
    constexpr int BR = W8 ? TN / 2 : TN;
    using LS = std::conditional_t<FWD, DmaKmaj<BR, KS>, DmaRmaj<TM, KS>>;
    constexpr int BKE = 16 * KS, TA = TM * 32 * KS, TB = TN * 32 * KS;
    static_assert(!W8 || TA + TB == (128 + 256) * 32 * KS, "8-wave tiles share one LDS layout");
    const int bh = W8 ? wave >> 2 : 0;  // B half of the wave (8-wave tiles)
    LS ls;
    if constexpr (FWD)
      ls.init(static_cast<const T*>(d.B), d.ldb, t.n0 + BR * bh, d.N, d.Kd, wave & 3, lane);
    else
      ls.init(static_cast<const T*>(d.A), d.lda, t.m0, d.M, d.Kd, wave, lane);
    const int nk = (d.Kd + BKE - 1) / BKE;
    // stage k: the produced operand at prod(b), the streamed one at strm(b)
    auto prod = [](char* b) { return FWD ? b : b + TA; };
    auto strm = [&](char* b) { return FWD ? b + TA + bh * (BR * 32 * KS) : b; };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    // forward: the table entries of step s in tab(s & 1), after both stages
    auto tab = [&](int s) { return lds0 + 2 * (TA + TB) + (s & 1) * 1024; };
    // the producer's loads of step s (register set s & 1; the forward's table two steps ahead too)
    auto load = [&](int s, auto S) {
      if constexpr (FWD) {
        ep.template load_x<S.value>(s * BKE);
        ep.issue_tab(tab(s), s * BKE);
      } else {
        ep.template load<S.value>(s * BKE);
      }
    };
    auto store = [&](int s, auto S, char* b) {
      if constexpr (FWD) {
        ep.read_tab(tab(s));
        ep.template store<S.value>(prod(b), s * BKE, [](int row, int sl) { return kmaj16_off<KS>(row, sl); });
      } else {
        ep.template store<S.value>(prod(b));
      }
    };
    // The producer's loads run two K steps ahead (register set = step & 1), so
    // their latency hides behind a whole step, as the direct loads' does.
    // Memory operations keep their program order around the direct loads
    // (empty asm statements); the wait at the top of a step covers both.
    load(0, S0{});
    load(min(1, nk - 1), S1{});
    asm volatile("" ::: "memory");
    ls.issue(strm(lds0), 0, d.Kd);
    asm volatile("" ::: "memory");
    if constexpr (FWD) {  // step 0's table entries
      wait_vm<0, true>();
      bar();
    }
    store(0, S0{}, lds0);
    // step kt: the loads of step kt + 2 (set kt & 1, clamped to the last
    // step, so the body has no conditional memory operations), the direct
    // loads of step kt + 1, the MFMAs of step kt, then step kt + 1 produced
    // from set S = (kt + 1) & 1
    auto step = [&](int kt, auto S) {
      wait_vm<0, true>();  // step kt's direct loads, the producer's loads and LDS writes are done
      bar();
      char* cur = lds0 + (kt & 1) * (TA + TB);
      char* nxt = lds0 + ((kt + 1) & 1) * (TA + TB);
      load(min(kt + 2, nk - 1), std::integral_constant<int, 1 - S.value>{});
      asm volatile("" ::: "memory");
      ls.issue(strm(nxt), (kt + 1) * BKE, d.Kd);
      asm volatile("" ::: "memory");
      if (compute) mma_step<T, SH, !FWD, !FWD, KS>(cur, cur + TA, acc, wm, wn, lane);
      store(kt + 1, S, nxt);
    };
    for (int kt = 0; kt + 1 < nk;) {
      step(kt, S1{});
      if (++kt + 1 >= nk) break;
      step(kt, S0{});
      ++kt;
    }
    wait_vm<0, true>();
    bar();
    if (compute) {
      char* cur = lds0 + ((nk - 1) & 1) * (TA + TB);
      mma_step<T, SH, !FWD, !FWD, KS>(cur, cur + TA, acc, wm, wn, lane);
    }
    wait_vm<0, true>();
    bar();  // the epilogue stages results in the operand buffers
  } else {
    constexpr int BKE = KV * Elem<T>::VE;
    constexpr int TA = TM * ROW, TB = TN * ROW;
    std::conditional_t<FWD, LoadKmaj<T, TN>, LoadRmajF32<TM>> ls;
    if constexpr (FWD)
      ls.init(static_cast<const T*>(d.B), d.ldb, t.n0, d.N, d.Kd, tid);
    else
      ls.init(static_cast<const T*>(d.A), d.lda, t.m0, d.M, d.Kd, tid);
    char* lds1 = lds0 + TA + TB;
    const int nk = (d.Kd + BKE - 1) / BKE;
    auto load = [&](int k0) {
      if constexpr (FWD)
        ep.load(k0);
      else
        ep.template load<0>(k0);
    };
    auto store = [&](char* b, int k0) {
      if constexpr (FWD) {
        ep.template store<0>(b, k0, [](int row, int sl) { return kmaj_off(row, sl); });
        ls.store(b + TA, tid);
      } else {
        ls.store(b, tid);
        ep.template store<0>(b + TA);
      }
    };
    load(0);
    ls.load(0, d.Kd, tid);
    store(lds0, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      char* cur = (kt & 1) ? lds1 : lds0;
      char* nxt = (kt & 1) ? lds0 : lds1;
      const bool more = kt + 1 < nk;
      if (more) {
        load((kt + 1) * BKE);
        ls.load((kt + 1) * BKE, d.Kd, tid);
      }
      if (compute) mma_step<T, SH, false, false, 4>(cur, cur + TA, acc, wm, wn, lane);
      if (more) store(nxt, (kt + 1) * BKE);
      __syncthreads();
    }
  }
  if constexpr (EPI == EPI_DW && sizeof(T) == 2) {
    if (a.theta) {  // uniform: the whole workgroup takes the staged-tile path
      dw_adamw_small(a, d, t, acc, wm, wn, lane, tid, lds0);
      return;
    }
  }
  epilogue<T, EPI, SH>(a, d, t, acc, wm, wn, lane, mv, nv, lds0 + wave * Shape<SH>::STAGE, pre);
}

// ----------------------------------------------------------------- kernel --
// Launches whose tiles include the big shape: 256x256 tiles with two 64-deep
// stages (128 KB of LDS), one workgroup (one wave per SIMD) per CU.
template <typename T, int AK, int BK_, int EPI>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1))) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBig + XMapBytes<T, EPI>];
  const Tile t = a.tiles[blockIdx.x];
  const GemmDesc d = a.descs[t.desc];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  if (t.shape == kShapeBig) {
    run_tile<T, AK, BK_, EPI, kShapeBig, kBigKs, kBigNs>(a, d, t, smem, tid, wave, smem + kLdsBig);
    return;
  }
  run_tile<T, AK, BK_, EPI, kShapeSmall, 4, 2>(a, d, t, smem, tid, wave, smem + kLdsBig);
}

// Launches of small tiles only: 64 KB of LDS, two workgroups per CU, so one
// workgroup's epilogue overlaps the other's MFMA loop.  bf16: kSmallNs stages
// of kSmallKs 16-deep steps; fp32: two register-staged stages.
template <typename T, int AK, int BK_, int EPI>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(
    sizeof(T) == 2 ? kSmallWpeBf16 : kSmallWpeF32, sizeof(T) == 2 ? kSmallWpeBf16 : kSmallWpeF32))) void
gemm_kernel_small(GemmArgs a) {
  constexpr int kOps = sizeof(T) == 2 ? kLdsSmallBf16 : kLdsSmallF32;
  // + the embedded forward's two 1 KB stages of column-table entries (bf16)
  constexpr int kTab = AK == OP_EMB && sizeof(T) == 2 ? 2048 : 0;
  static_assert(kTab == 0 || kLdsSmallBf16 == 2 * 2 * 128 * 32 * kSmallKs, "table stages follow the operand stages");
  __shared__ __attribute__((aligned(16))) char smem[kOps + kTab + XMapBytes<T, EPI>];
  const Tile t = a.tiles[blockIdx.x];
  const GemmDesc d = a.descs[t.desc];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if constexpr (AK == OP_EMB || BK_ == OP_EMB)
    run_tile_emb<T, AK, BK_, EPI>(a, d, t, smem, tid, wave, smem + kOps + kTab);
  else if constexpr (sizeof(T) == 2)
    run_tile<T, AK, BK_, EPI, kShapeSmall, kSmallKs, kSmallNs>(a, d, t, smem, tid, wave, smem + kOps);
  else
    run_tile<T, AK, BK_, EPI, kShapeSmall, 4, 2>(a, d, t, smem, tid, wave);
}

// The embedded first layer's bf16 forward on wide tiles (128 x 256; a last
// strip of at most 128 columns on tall 256 x 128 tiles): one workgroup of 8
// waves per CU (two stages of 48 KB: 16 KB of produced E and 32 KB of W_1, or
// the reverse; two 1 KB stages of column-table entries).
template <int EPI>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_kernel_emb_wide(GemmArgs a) {
  constexpr int kOps = 2 * (128 + 256) * 32 * kSmallKs;
  static_assert(8 * Shape<kShapeWide>::STAGE <= kOps, "epilogue staging of 8 waves");
  __shared__ __attribute__((aligned(16))) char smem[kOps + 2048];
  const Tile t = a.tiles[blockIdx.x];
  const GemmDesc d = a.descs[t.desc];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (t.shape == kShapeWide)
    run_tile_emb<__bf16, OP_EMB, OP_KMAJ, EPI, kShapeWide>(a, d, t, smem, tid, wave, nullptr);
  else
    run_tile_emb<__bf16, OP_EMB, OP_KMAJ, EPI, kShapeTall8>(a, d, t, smem, tid, wave, nullptr);
}

// Launches of tall tiles (256 x 128) with small edge tiles, bf16 only: two
// workgroups per CU, each with kTallNs stages of the tall pipeline.
template <int AK, int BK_, int EPI>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_kernel_tall(GemmArgs a) {
  static_assert(kLdsTall + XMapBytes<__bf16, EPI> <= 80 * 1024, "two tall-tile workgroups per CU");
  __shared__ __attribute__((aligned(16))) char smem[kLdsTall + XMapBytes<__bf16, EPI>];
  const Tile t = a.tiles[blockIdx.x];
  const GemmDesc d = a.descs[t.desc];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (t.shape == kShapeTall) {
    run_tile<__bf16, AK, BK_, EPI, kShapeTall, kTallKs, kTallNs>(a, d, t, smem, tid, wave, smem + kLdsTall);
    return;
  }
  run_tile<__bf16, AK, BK_, EPI, kShapeSmall, kSmallKs, kSmallNs>(a, d, t, smem, tid, wave, smem + kLdsTall);
}

template <typename T, int AK, int BK_, int EPI>
hipError_t launch_t(const GemmArgs& args, hipStream_t s) {
  if (args.ntiles <= 0) return hipSuccess;
  if constexpr (sizeof(T) == 4) {  // fp32 operands: small tiles only
    if (args.tile_set != TILES_SMALL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_kernel_small<T, AK, BK_, EPI>), dim3(args.ntiles), dim3(NT), 0, s, args);
  } else {
    switch (args.tile_set) {
      case TILES_SMALL:
        hipLaunchKernelGGL((gemm_kernel_small<T, AK, BK_, EPI>), dim3(args.ntiles), dim3(NT), 0, s, args);
        break;
      case TILES_TALL:
        hipLaunchKernelGGL((gemm_kernel_tall<AK, BK_, EPI>), dim3(args.ntiles), dim3(NT), 0, s, args);
        break;
      case TILES_BIG:
        hipLaunchKernelGGL((gemm_kernel<T, AK, BK_, EPI>), dim3(args.ntiles), dim3(NT), 0, s, args);
        break;
      default:
        return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

template <typename T, int AK, int BK_, int EPI>
hipError_t launch_small(const GemmArgs& args, hipStream_t s) {
  if (args.ntiles <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel_small<T, AK, BK_, EPI>), dim3(args.ntiles), dim3(NT), 0, s, args);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_prec(OpKind ak, OpKind bk, EpiKind e, const GemmArgs& args, hipStream_t s) {
  if (ak == OP_KMAJ && bk == OP_KMAJ && e == EPI_FWD) return launch_t<T, OP_KMAJ, OP_KMAJ, EPI_FWD>(args, s);
  if (ak == OP_KMAJ && bk == OP_KMAJ && e == EPI_FWD_EVAL)
    return launch_t<T, OP_KMAJ, OP_KMAJ, EPI_FWD_EVAL>(args, s);
  if (ak == OP_KMAJ && bk == OP_RMAJ && e == EPI_DX) return launch_t<T, OP_KMAJ, OP_RMAJ, EPI_DX>(args, s);
  if (ak == OP_RMAJ && bk == OP_RMAJ && e == EPI_DW) return launch_t<T, OP_RMAJ, OP_RMAJ, EPI_DW>(args, s);
  if (ak == OP_EMB || bk == OP_EMB) {  // the embedded first layer: small tiles (the bf16 forward: or wide)
    if (!args.emb_tab || !args.emb_x || !args.emb_mem) return hipErrorInvalidValue;
    if (args.tile_set == TILES_WIDE) {
      if constexpr (sizeof(T) == 2) {
        if (ak == OP_EMB && bk == OP_KMAJ && (e == EPI_FWD || e == EPI_FWD_EVAL)) {
          if (args.ntiles <= 0) return hipSuccess;
          if (e == EPI_FWD)
            hipLaunchKernelGGL(gemm_kernel_emb_wide<EPI_FWD>, dim3(args.ntiles), dim3(512), 0, s, args);
          else
            hipLaunchKernelGGL(gemm_kernel_emb_wide<EPI_FWD_EVAL>, dim3(args.ntiles), dim3(512), 0, s, args);
          return hipGetLastError();
        }
      }
      return hipErrorInvalidValue;
    }
    if (args.tile_set != TILES_SMALL) return hipErrorInvalidValue;
    if (ak == OP_EMB && bk == OP_KMAJ && e == EPI_FWD) return launch_small<T, OP_EMB, OP_KMAJ, EPI_FWD>(args, s);
    if (ak == OP_EMB && bk == OP_KMAJ && e == EPI_FWD_EVAL)
      return launch_small<T, OP_EMB, OP_KMAJ, EPI_FWD_EVAL>(args, s);
    if (ak == OP_RMAJ && bk == OP_EMB && e == EPI_DW) return launch_small<T, OP_RMAJ, OP_EMB, EPI_DW>(args, s);
    return hipErrorInvalidValue;
  }
  if (ak == OP_KMAJ && bk == OP_RMAJ && e == EPI_DE) {  // the embedding's dE reduction: small tiles only
    if (args.tile_set != TILES_SMALL) return hipErrorInvalidValue;
    return launch_small<T, OP_KMAJ, OP_RMAJ, EPI_DE>(args, s);
  }
  if (e == EPI_NS) {  // Newton-Schulz products
    if (ak == OP_KMAJ && bk == OP_KMAJ) return launch_t<T, OP_KMAJ, OP_KMAJ, EPI_NS>(args, s);
    if (ak == OP_KMAJ && bk == OP_RMAJ) return launch_t<T, OP_KMAJ, OP_RMAJ, EPI_NS>(args, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(Prec prec, OpKind a, OpKind b, EpiKind e, const GemmArgs& args, hipStream_t s) {
  return prec == Prec::BF16 ? launch_prec<__bf16>(a, b, e, args, s) : launch_prec<float>(a, b, e, args, s);
}

}  // namespace tabpack
