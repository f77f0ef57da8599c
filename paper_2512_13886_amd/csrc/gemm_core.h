// MFMA main loop of a 128x128 output tile of C = A B^T, both operands stored
// row-major with the contraction index contiguous ("NT"): A row r and B row c
// each hold the K values of one dot product. This is the layout of both hot
// contractions: the batched H-product Y[b][n] = sum_k Z[b][k] H[n][k] (H is
// symmetric) and the Hessian block H[i][j] = sum_t XT[i][t] XT[j][t].
//
// Work split: WGM x WGN waves, each owning a (BM / WGM) x (BN / WGN) sub-tile
// as blocks of 16x16 MFMA outputs (4 floats per lane each), times KSPLIT
// groups of such waves that share the tile and take disjoint K slices of
// every stage (their partial sums are added when the tile is staged for the
// epilogue). K advances in stages of SRB = 128 or 256 bytes per row (32 or 64
// fp32, 64 or 128 bf16 values).
//
// Operands move HBM/L2 -> LDS with gfx950's direct loads
// (global_load_lds_dwordx4): no registers are spent on prefetch and the loads
// of stage s + 1 are issued right after the barrier that frees their buffer,
// ahead of the LDS reads and MFMAs of stage s (enforced with scheduling
// groups). One wave's direct load writes 1 KiB of LDS contiguously (lane l at
// byte 16 l), i.e. 1024 / SRB tile rows; to keep the fragment reads free of
// bank conflicts without padding, the 16-byte segment g of tile row r is
// stored at physical segment g ^ (r % (SRB / 16)), and each lane fetches from
// global memory the logical segment that belongs at its physical slot. The
// stage buffers are distinct LDS arrays and the stage loop is unrolled by
// their count, so that no LDS read shares an object with an in-flight direct
// load and the compiler adds no wait for it.
//
// Fragment layout (v_mfma_f32_16x16x4_f32 and v_mfma_f32_16x16x32_bf16): lane
// l supplies row (l % 16) of a 16-row block and the K group (l / 16). One
// 16-byte LDS read gives a lane 4 consecutive fp32 values or 8 consecutive
// bf16 values of its row. For fp32 the 4 values feed 4 MFMAs (K = 4 each,
// lane group g contributing K index 4g + e at MFMA e); for bf16 they feed one
// MFMA with K = 32. A and B use the same K permutation, so every product pair
// meets exactly once. Output element (lane, e) of a 16x16 block is
// row 4 * (lane / 16) + e, column lane % 16.
#pragma once

#include <type_traits>

#include "common.h"

namespace optima {

// Stage width of the 4-wave 128 x 128 configuration.
constexpr int kStageRowBytes = 128;

template <int MB, int NB>
__device__ inline void mfma_f32_blocks(f4 (&acc)[MB][NB], const uint4 (&a)[MB], const uint4 (&b)[NB]) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
#pragma unroll
      for (int ni = 0; ni < NB; ++ni) {
        const unsigned av = e == 0 ? a[mi].x : e == 1 ? a[mi].y : e == 2 ? a[mi].z : a[mi].w;
        const unsigned bv = e == 0 ? b[ni].x : e == 1 ? b[ni].y : e == 2 ? b[ni].z : b[ni].w;
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(av), __uint_as_float(bv),
                                                           acc[mi][ni], 0, 0, 0);
      }
}

template <int MB, int NB>
__device__ inline void mfma_bf16_blocks(f4 (&acc)[MB][NB], const uint4 (&a)[MB], const uint4 (&b)[NB]) {
#pragma unroll
  for (int mi = 0; mi < MB; ++mi)
#pragma unroll
    for (int ni = 0; ni < NB; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          __builtin_bit_cast(bf16x8, a[mi]), __builtin_bit_cast(bf16x8, b[ni]), acc[mi][ni], 0, 0, 0);
}

struct Bf16Tag {};

// fp32 emulated by bf16 MFMAs: every value v is stored as two bf16 planes,
// hi = rne(v) and lo = rne(v - hi), and a product a*b is formed as
// a_hi b_hi + a_hi b_lo + a_lo b_hi (the dropped terms are below 2^-16 |a b|).
struct Bf16x3Tag {};

__device__ inline uint32_t bf16_rne_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ inline float bf16_bits_value(uint32_t h) { return __uint_as_float(h << 16); }

// Plane layout of a row of dp values: for every block of 32 consecutive
// columns, 64 bytes of hi plane then 64 bytes of lo plane. A row therefore
// takes 4 dp bytes, like fp32, and each 128-byte piece of a K stage holds 32
// columns of both planes.
__device__ inline void store_split(uint16_t* row_planes, int n, float v) {
  const uint32_t hi = bf16_rne_bits(v);
  const uint32_t lo = bf16_rne_bits(v - bf16_bits_value(hi));
  uint16_t* b = row_planes + (n >> 5) * 64 + (n & 31);
  b[0] = uint16_t(hi);
  b[32] = uint16_t(lo);
}

// Tile configuration: a BM x BN output tile per workgroup, WGM x WGN x KSPLIT
// waves, each owning a (BM / WGM) x (BN / WGN) sub-tile of 16x16 blocks and
// 1 / KSPLIT of every stage's K, NBUF LDS stage buffers (prefetch distance
// NBUF - 1 stages) and SRB bytes per row and stage.
template <int BM_, int BN_, int WGM_, int WGN_, int NBUF_, int KSPLIT_ = 1, int SRB_ = 128>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, NBUF = NBUF_;
  static constexpr int KSPLIT = KSPLIT_, SRB = SRB_;
  static constexpr int kTileWaves = WGM * WGN;     // waves per K group
  static constexpr int kWaves = kTileWaves * KSPLIT;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int MB = BM / WGM / 16;  // 16-row blocks per wave
  static constexpr int NB = BN / WGN / 16;  // 16-column blocks per wave
  static constexpr int kSegs = SRB / 16;    // 16-byte segments per row and stage
  static constexpr int kRowsPerLoad = 1024 / SRB;
  static constexpr int kLoadsA = BM / kRowsPerLoad / kWaves;  // 1-KiB wave loads per stage
  static constexpr int kLoadsB = BN / kRowsPerLoad / kWaves;
  static constexpr int kLoads = kLoadsA + kLoadsB;
  static constexpr int kBufBytes = (BM + BN) * SRB;
  // 64-byte chunks (4 segments: 16 fp32 or 32 bf16 K values per row) per
  // stage, and per wave.
  static constexpr int kChunks = SRB / 64;
  static constexpr int kWaveChunks = kChunks / KSPLIT;
  static_assert(SRB == 128 || SRB == 256, "stage width");
  static_assert(BM % (kRowsPerLoad * kWaves) == 0 && BN % (kRowsPerLoad * kWaves) == 0,
                "load rounds");
  static_assert(NBUF == 2 || NBUF == 3, "stage buffers");
  static_assert(kWaveChunks >= 2 && kWaveChunks % 2 == 0, "K slice of a wave");
};

// The 128 x 128 tile with 4 waves of 64 x 64 and two 128-byte stage buffers.
using Tile128 = TileCfg<128, 128, 2, 2, 2>;

// Rows of the tile that this thread's direct loads fetch: A round i covers
// A tile row load_row<Cfg>(i), B round i covers B tile row load_row<Cfg>(i);
// the byte offset of the fetched 16-byte segment within the row's stage is
// load_seg_bytes<Cfg>(i).
template <typename Cfg>
__device__ inline int load_row(int i) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  return (i * Cfg::kWaves + wave) * Cfg::kRowsPerLoad + lane / Cfg::kSegs;
}
template <typename Cfg>
__device__ inline int load_seg_bytes(int i) {
  const int lane = threadIdx.x & 63;
  return ((lane % Cfg::kSegs) ^ (load_row<Cfg>(i) % Cfg::kSegs)) * 16;
}

template <typename Cfg>
struct Operands {
  const char* a[Cfg::kLoadsA];
  const char* b[Cfg::kLoadsB];
};

template <typename Cfg>
__device__ inline void issue_stage(const Operands<Cfg>& src, int s, char* buf) {
  const size_t o = size_t(s) * Cfg::SRB;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsA; ++i)
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(src.a[i] + o),
        (__attribute__((address_space(3))) void*)(buf + (i * Cfg::kWaves + wave) * 1024), 16, 0, 0);
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsB; ++i)
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(src.b[i] + o),
        (__attribute__((address_space(3))) void*)(buf + Cfg::BM * Cfg::SRB +
                                                  (i * Cfg::kWaves + wave) * 1024),
        16, 0, 0);
}

// 16 bytes of logical segment `seg` of tile row r (A rows first, then B).
template <typename Cfg>
__device__ inline uint4 lds_frag(const char* buf, int r, int seg) {
  return *reinterpret_cast<const uint4*>(buf + r * Cfg::SRB + ((seg ^ (r % Cfg::kSegs)) * 16));
}

// This wave's K group (which slice of every stage it multiplies).
template <typename Cfg>
__device__ inline int k_group() {
  return (threadIdx.x >> 6) / Cfg::kTileWaves;
}

template <typename Cfg, typename T>
__device__ inline void compute_stage(f4 (&acc)[Cfg::MB][Cfg::NB], const char* buf) {
  constexpr int MB = Cfg::MB, NB = Cfg::NB;
  const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) % Cfg::kTileWaves;
  const int ra = (wave / Cfg::WGN) * MB * 16 + (lane & 15);
  const int rb = Cfg::BM + (wave % Cfg::WGN) * NB * 16 + (lane & 15);
  const int g = lane >> 4;
  const int c0 = k_group<Cfg>() * Cfg::kWaveChunks;  // first 64-byte chunk of this wave
  if constexpr (std::is_same<T, Bf16x3Tag>::value) {
    // A pair of chunks is one 32-column block: segments 0-3 hold its hi
    // plane, 4-7 its lo plane. Per output block hi*hi, hi*lo, lo*hi (one
    // 16x16x32 bf16 MFMA each).
    static_assert(Cfg::kWaveChunks == 2, "one plane block per wave and stage");
    const int sg = 4 * c0;
    uint4 a0[MB], a1[MB], b0[NB], b1[NB];
#pragma unroll
    for (int mi = 0; mi < MB; ++mi) a0[mi] = lds_frag<Cfg>(buf, ra + mi * 16, sg + g);
#pragma unroll
    for (int ni = 0; ni < NB; ++ni) b0[ni] = lds_frag<Cfg>(buf, rb + ni * 16, sg + g);
    mfma_bf16_blocks<MB, NB>(acc, a0, b0);
#pragma unroll
    for (int ni = 0; ni < NB; ++ni) b1[ni] = lds_frag<Cfg>(buf, rb + ni * 16, sg + 4 + g);
    mfma_bf16_blocks<MB, NB>(acc, a0, b1);
#pragma unroll
    for (int mi = 0; mi < MB; ++mi) a1[mi] = lds_frag<Cfg>(buf, ra + mi * 16, sg + 4 + g);
    mfma_bf16_blocks<MB, NB>(acc, a1, b0);
    __builtin_amdgcn_sched_group_barrier(0x020, Cfg::kLoads, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, MB + NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, MB * NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, MB * NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, MB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, MB * NB, 0);
  } else {
    static_assert(Cfg::kWaveChunks == 2, "two chunks per wave and stage");
    constexpr int kMfmaPerChunk = std::is_same<T, float>::value ? 4 * MB * NB : MB * NB;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      uint4 a[MB], b[NB];
#pragma unroll
      for (int mi = 0; mi < MB; ++mi) a[mi] = lds_frag<Cfg>(buf, ra + mi * 16, 4 * (c0 + c) + g);
#pragma unroll
      for (int ni = 0; ni < NB; ++ni) b[ni] = lds_frag<Cfg>(buf, rb + ni * 16, 4 * (c0 + c) + g);
      if constexpr (std::is_same<T, float>::value)
        mfma_f32_blocks<MB, NB>(acc, a, b);
      else
        mfma_bf16_blocks<MB, NB>(acc, a, b);
    }
    __builtin_amdgcn_sched_group_barrier(0x020, Cfg::kLoads, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, MB + NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, kMfmaPerChunk, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, MB + NB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, kMfmaPerChunk, 0);
  }
}

// s_waitcnt vmcnt(n) (0 <= n < 64), leaving expcnt and lgkmcnt unwaited.
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// Barrier of a ring of LDS stage buffers fed by direct loads: this wave's
// loads other than its N most recent have landed and its LDS reads are
// complete, then all waves meet. It is a bare s_barrier: the workgroup fence
// of __syncthreads makes the compiler wait for every direct load in flight
// (they write LDS), which would leave only the newest stage loading during
// each compute. The empty asm statements keep the compiler from moving
// memory accesses across.
template <int N>
__device__ inline void ring_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70);  // vmcnt(N) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// src.a[i] / src.b[i]: address of the 16-byte segment this thread fetches in
// A / B tile row load_row<Cfg>(i) at the first stage (row start +
// load_seg_bytes<Cfg>(i)); stage s adds s * Cfg::SRB. All addresses must be
// 16-byte aligned. lds0..lds2 (lds2 only with NBUF == 3) must be distinct
// __shared__ arrays of Cfg::kBufBytes declared by the kernel: the loop is
// unrolled by NBUF so that no LDS read names an array with an in-flight load.
template <typename Cfg, typename T>
__device__ inline void gemm_tile_mainloop(f4 (&acc)[Cfg::MB][Cfg::NB], const Operands<Cfg>& src,
                                          int n, char* lds0, char* lds1, char* lds2) {
#pragma unroll
  for (int mi = 0; mi < Cfg::MB; ++mi)
#pragma unroll
    for (int ni = 0; ni < Cfg::NB; ++ni) acc[mi][ni] = f4{0.f, 0.f, 0.f, 0.f};
  if (n <= 0) return;
  auto cl = [n](int s) { return s < n ? s : n - 1; };

  if constexpr (Cfg::NBUF == 2) {
    issue_stage<Cfg>(src, 0, lds0);
    int s = 0;
    for (; s + 1 < n; s += 2) {
      wait_vmcnt<0>();
      __syncthreads();
      issue_stage<Cfg>(src, s + 1, lds1);
      compute_stage<Cfg, T>(acc, lds0);
      wait_vmcnt<0>();
      __syncthreads();
      issue_stage<Cfg>(src, cl(s + 2), lds0);
      compute_stage<Cfg, T>(acc, lds1);
    }
    if (s < n) {  // odd count: the last stage is in lds0
      wait_vmcnt<0>();
      __syncthreads();
      compute_stage<Cfg, T>(acc, lds0);
    }
  } else {
    issue_stage<Cfg>(src, 0, lds0);
    issue_stage<Cfg>(src, cl(1), lds1);
    int s = 0;
    for (; s + 2 < n; s += 3) {
      ring_barrier<Cfg::kLoads>();  // stage s landed, stage s + 1 may still fly
      issue_stage<Cfg>(src, s + 2, lds2);
      compute_stage<Cfg, T>(acc, lds0);
      ring_barrier<Cfg::kLoads>();
      issue_stage<Cfg>(src, cl(s + 3), lds0);
      compute_stage<Cfg, T>(acc, lds1);
      ring_barrier<Cfg::kLoads>();
      issue_stage<Cfg>(src, cl(s + 4), lds1);
      compute_stage<Cfg, T>(acc, lds2);
    }
    if (s < n) {  // one or two stages left, in lds0 and lds1
      wait_vmcnt<Cfg::kLoads>();
      __syncthreads();
      compute_stage<Cfg, T>(acc, lds0);
      if (s + 1 < n) {
        wait_vmcnt<0>();
        __syncthreads();
        compute_stage<Cfg, T>(acc, lds1);
      }
    }
  }
  // No direct load may still be writing LDS when the workgroup moves on.
  wait_vmcnt<0>();
  __syncthreads();
}

// ---------------------------------------------------------------------------
// 2:4-sparse A operand on v_smfmac_f32_16x16x64_bf16
// ---------------------------------------------------------------------------
// When every group of 4 consecutive K values of every A row has at most 2
// nonzeros (a 2:4 pruning mask applied to the multiplied vectors), A is kept
// compressed: per group 2 stored values, the entries at 2 positions p0 < p1
// that cover the group's nonzeros (padded with the lowest free positions),
// and per stored value its 2-bit position. One sparse MFMA multiplies a
// 16 x 64 block of A (16 x 32 stored values) by a dense 64 x 16 block of B,
// in the time of a dense 16 x 16 x 32 one, so it skips the products with
// the zeros.
//
// Operand layout of the instruction (checked on gfx950 against a reference
// product for every lane and value slot): lane l supplies A row l % 16 and
// the 8 stored values of logical K [16 g, 16 g + 16), g = l / 16, two per
// group of 4 in group order; bits 2 i..2 i + 1 of its 16-bit index give the
// position of stored value i within its group. Lane l supplies B column
// l % 16 at K [8 g, 8 g + 8) (values 0-7) and [32 + 8 g, 32 + 8 g + 8)
// (values 8-15). The result has the layout of the dense 16 x 16 MFMA.
//
// Storage of A: per row and 64-column block of K, 128 bytes: the 32 stored
// hi values (64 B), then the 32 stored lo values; lane group g's 16 bytes
// sit at byte 16 g of each plane. Indices: per row and block four 16-bit
// words (8 bytes), word g for lane group g.
//
// Work split: a 256 x 128 output tile per workgroup of 8 waves (4 x 2, each
// 64 x 64). The operand loads from L2, not the MFMAs, bound these products
// (about 25 bytes per clock and CU were measured for both the direct loads
// and plain 16-byte loads), so the tile is the largest whose double-
// buffered stages fit the LDS: per 64-column stage the stored A rows
// (256 x 128 B), their index words (256 x 8 B) and the split planes of B
// (128 x 256 B), 66 KiB, all fetched once per workgroup by direct loads.
// The index words come stage-major (one stage's words of consecutive tile
// rows are contiguous): with 8 bytes per row in a row-major array each
// stage's 2 KiB would touch 256 cache lines, as many as the A rows.
// That is 64 algorithmic flops per loaded byte, twice the dense bf16x3
// 128 x 128 tile's 32.
struct SpTile {
  static constexpr int BM = 256, BN = 128, WGM = 4, WGN = 2, KSPLIT = 1;
  static constexpr int kTileWaves = 8, kWaves = 8, kThreads = 512;
  static constexpr int MB = 4, NB = 4;
  static constexpr int kKPerStage = 64;
  static constexpr int kARowBytes = 128;  // stored A bytes per row and stage
  static constexpr int kBRowBytes = 256;  // B bytes per row and stage (both planes)
  static constexpr int kASegs = kARowBytes / 16, kBSegs = kBRowBytes / 16;
  static constexpr int kLoadsA = BM * kARowBytes / 1024 / kWaves;  // 1-KiB wave loads
  static constexpr int kLoadsB = BN * kBRowBytes / 1024 / kWaves;
  static constexpr int kIdxOff = BM * kARowBytes + BN * kBRowBytes;  // index words
  static constexpr int kBufBytes = kIdxOff + BM * 8;
  static_assert(BM * 8 == kWaves * 256, "one 4-byte-per-lane index load per wave");
};

struct SpOperands {
  const char* a[SpTile::kLoadsA];  // A segment of this thread's direct loads at stage 0
  const char* b[SpTile::kLoadsB];  // B segment of this thread's direct loads at stage 0
  const char* ai;                  // its 4 bytes of index words at stage 0
  int64_t ai_stage;                // bytes from one stage's index words to the next
};

// Tile rows fetched by this thread's direct loads and the byte offset of the
// fetched 16-byte segment in the row's stage. A rows take 128 bytes (8
// segments, physical segment g ^ (r % 8)), B rows 256 bytes (16 segments,
// g ^ (r % 16)); index row r takes 8 bytes, 2 lanes per row.
__device__ inline int sp_a_row(int i) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  return (i * SpTile::kWaves + wave) * (1024 / SpTile::kARowBytes) + lane / SpTile::kASegs;
}
__device__ inline int sp_a_seg_bytes(int i) {
  const int lane = threadIdx.x & 63;
  return ((lane % SpTile::kASegs) ^ (sp_a_row(i) % SpTile::kASegs)) * 16;
}
__device__ inline int sp_b_row(int i) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  return (i * SpTile::kWaves + wave) * (1024 / SpTile::kBRowBytes) + lane / SpTile::kBSegs;
}
__device__ inline int sp_b_seg_bytes(int i) {
  const int lane = threadIdx.x & 63;
  return ((lane % SpTile::kBSegs) ^ (sp_b_row(i) % SpTile::kBSegs)) * 16;
}
__device__ inline int sp_idx_row() { return (threadIdx.x >> 6) * 32 + (threadIdx.x & 63) / 2; }
__device__ inline int sp_idx_bytes() { return (threadIdx.x & 1) * 4; }

__device__ inline void sp_issue_stage(const SpOperands& src, int s, char* buf) {
  const int wave = threadIdx.x >> 6;
  const size_t oa = size_t(s) * SpTile::kARowBytes, ob = size_t(s) * SpTile::kBRowBytes;
#pragma unroll
  for (int i = 0; i < SpTile::kLoadsA; ++i)
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(src.a[i] + oa),
        (__attribute__((address_space(3))) void*)(buf + (i * SpTile::kWaves + wave) * 1024), 16,
        0, 0);
#pragma unroll
  for (int i = 0; i < SpTile::kLoadsB; ++i)
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(src.b[i] + ob),
        (__attribute__((address_space(3))) void*)(buf + SpTile::BM * SpTile::kARowBytes +
                                                  (i * SpTile::kWaves + wave) * 1024),
        16, 0, 0);
  __builtin_amdgcn_global_load_lds(
      (const __attribute__((address_space(1))) void*)(src.ai + s * src.ai_stage),
      (__attribute__((address_space(3))) void*)(buf + SpTile::kIdxOff + wave * 256), 4, 0, 0);
}

// Fragment reads load ext-vector values straight from the stage buffer: a
// 16-byte struct load would be split and re-merged by the backend, which
// drops the LDS alias scope and makes every such read wait for the direct
// loads in flight.
__device__ inline bf16x8 sp_a_frag(const char* buf, int r, int seg) {
  return *reinterpret_cast<const bf16x8*>(buf + r * SpTile::kARowBytes +
                                          ((seg ^ (r & (SpTile::kASegs - 1))) * 16));
}
__device__ inline bf16x8 sp_b_frag16(const char* buf, int r, int seg) {
  return *reinterpret_cast<const bf16x8*>(buf + SpTile::BM * SpTile::kARowBytes +
                                          r * SpTile::kBRowBytes +
                                          ((seg ^ (r & (SpTile::kBSegs - 1))) * 16));
}
__device__ inline bf16x16 sp_b_pair(bf16x8 k0, bf16x8 k1) {
  return __builtin_shufflevector(k0, k1, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
}

// Byte offsets within a stage buffer of this lane's fragment reads for the
// first 16-row block of its A and B rows: the A hi and lo segments, the
// index words and the four B segments (hi planes of K [0, 32) and [32, 64),
// then the lo planes). Row block mi of A adds mi * 2048 and block ni of B
// adds ni * 4096, which leaves the swizzles unchanged.
struct SpFragOffsets {
  uint32_t ah, al, ix, b0, b1, b2, b3;
};
__device__ inline SpFragOffsets sp_frag_offsets() {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ra = (wave / SpTile::WGN) * SpTile::MB * 16 + (lane & 15);
  const int rb = (wave % SpTile::WGN) * SpTile::NB * 16 + (lane & 15);
  const int g = lane >> 4, sa = ra & (SpTile::kASegs - 1), sb = rb & (SpTile::kBSegs - 1);
  const uint32_t a0 = ra * SpTile::kARowBytes;
  const uint32_t b = SpTile::BM * SpTile::kARowBytes + rb * SpTile::kBRowBytes;
  return {a0 + ((g ^ sa) * 16u),        a0 + (((4 + g) ^ sa) * 16u),
          uint32_t(SpTile::kIdxOff + ra * 8 + 2 * g),
          b + ((g ^ sb) * 16u),         b + (((8 + g) ^ sb) * 16u),
          b + (((4 + g) ^ sb) * 16u),   b + (((12 + g) ^ sb) * 16u)};
}

__device__ inline void sp_compute_stage(f4 (&acc)[SpTile::MB][SpTile::NB], const char* buf) {
  constexpr int MB = SpTile::MB, NB = SpTile::NB;
  // The empty asm statement makes the offsets opaque at every stage, so the
  // compiler keeps these seven values in registers and folds each read's
  // constant part (row block, buffer) into the read's offset field, instead
  // of hoisting one address register per read out of the loop.
  SpFragOffsets o = sp_frag_offsets();
  asm volatile("" : "+v"(o.ah), "+v"(o.al), "+v"(o.ix), "+v"(o.b0), "+v"(o.b1), "+v"(o.b2),
               "+v"(o.b3));
  bf16x8 ah[MB], al[MB];
  int ix[MB];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
    ah[mi] = *reinterpret_cast<const bf16x8*>(buf + o.ah + mi * 16 * SpTile::kARowBytes);
    al[mi] = *reinterpret_cast<const bf16x8*>(buf + o.al + mi * 16 * SpTile::kARowBytes);
    ix[mi] = *reinterpret_cast<const uint16_t*>(buf + o.ix + mi * 16 * 8);
  }
  // B row segments: hi planes of K [0, 32) at 0-3 and [32, 64) at 8-11, lo
  // planes at 4-7 and 12-15. Consecutive MFMAs use different accumulators.
#pragma unroll
  for (int ni = 0; ni < NB; ++ni) {
    const char* bb = buf + ni * 16 * SpTile::kBRowBytes;
    const bf16x16 bh = sp_b_pair(*reinterpret_cast<const bf16x8*>(bb + o.b0),
                                 *reinterpret_cast<const bf16x8*>(bb + o.b1));
    const bf16x16 bl = sp_b_pair(*reinterpret_cast<const bf16x8*>(bb + o.b2),
                                 *reinterpret_cast<const bf16x8*>(bb + o.b3));
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
      acc[mi][ni] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(ah[mi],
                                                              bh, acc[mi][ni], ix[mi], 0, 0);
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
      acc[mi][ni] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(ah[mi],
                                                              bl, acc[mi][ni], ix[mi], 0, 0);
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
      acc[mi][ni] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(al[mi],
                                                              bh, acc[mi][ni], ix[mi], 0, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x020, SpTile::kLoadsA + SpTile::kLoadsB + 1, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, 3 * MB + 8, 0);
#pragma unroll
  for (int ni = 0; ni < NB - 2; ++ni) {
    __builtin_amdgcn_sched_group_barrier(0x008, 3 * MB, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 6 * MB, 0);
}

// Stage barrier of the sparse loop: this wave's direct loads and LDS reads
// are complete, then all waves meet. The empty asm statements keep the
// compiler from moving memory accesses across the barrier.
__device__ inline void sp_stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0 | 0x70);  // vmcnt(0) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Stages per iteration of the sparse main loop's unrolled body. The compiler
// lets part of a stage's MFMAs run past the next stage barrier (they then
// overlap the wait for the slowest wave), but not past the loop's back edge:
// bodies of 8 stages measured about 1 % faster per fused launch than bodies of
// 2 or 4, and bodies of 16 slower.
constexpr int kSpUnroll = 8;

// n stages (of 64 K values) of the sparse product, starting at the stage the
// operand addresses point to; lds0 / lds1 are distinct __shared__ arrays of
// SpTile::kBufBytes. The loads of stage s + 1 run during the compute of
// stage s; stage s is in lds0 when s is even. (An L2 prefetch touch of stage
// s + 2 was measured to cost more in load requests than it saved in latency.)
__device__ inline void gemm_sparse_mainloop(f4 (&acc)[SpTile::MB][SpTile::NB],
                                            const SpOperands& src, int n, char* lds0,
                                            char* lds1) {
#pragma unroll
  for (int mi = 0; mi < SpTile::MB; ++mi)
#pragma unroll
    for (int ni = 0; ni < SpTile::NB; ++ni) acc[mi][ni] = f4{0.f, 0.f, 0.f, 0.f};
  if (n <= 0) return;
  sp_issue_stage(src, 0, lds0);
  int s = 0;
  for (; s + kSpUnroll <= n; s += kSpUnroll) {
#pragma unroll
    for (int u = 0; u < kSpUnroll; u += 2) {
      sp_stage_barrier();
      sp_issue_stage(src, s + u + 1, lds1);
      sp_compute_stage(acc, lds0);
      sp_stage_barrier();
      if (u + 2 < kSpUnroll) {
        sp_issue_stage(src, s + u + 2, lds0);
      } else if (s + kSpUnroll < n) {
        sp_issue_stage(src, s + kSpUnroll, lds0);
      }
      sp_compute_stage(acc, lds1);
    }
  }
  for (; s + 1 < n; s += 2) {  // the stages left over, two at a time
    sp_stage_barrier();
    sp_issue_stage(src, s + 1, lds1);
    sp_compute_stage(acc, lds0);
    sp_stage_barrier();
    if (s + 2 < n) sp_issue_stage(src, s + 2, lds0);
    sp_compute_stage(acc, lds1);
  }
  if (s < n) {  // odd count: the last stage is in lds0
    sp_stage_barrier();
    sp_compute_stage(acc, lds0);
  }
  // No direct load may still be writing LDS when the workgroup moves on.
  wait_vmcnt<0>();
  __syncthreads();
}

// Epilogue staging of the 256 x 128 accumulator tile through the stage
// buffers: tile rows 64 q .. 64 q + 63 go to region q (lds0, lds0 + 32 KiB,
// lds1, lds1 + 32 KiB), 512 bytes per row, 16-byte column chunk c of row r at
// physical chunk c ^ (r & 31) (conflict-free as in stage_tile).
__device__ inline char* sp_stage_region(char* lds0, char* lds1, int r) {
  const int q = r >> 6;
  return (q < 2 ? lds0 : lds1) + (q & 1) * 32768 + (r & 63) * 512;
}
__device__ inline void sp_stage_tile(const f4 (&acc)[SpTile::MB][SpTile::NB], char* lds0,
                                     char* lds1) {
  static_assert(SpTile::kBufBytes >= 2 * 64 * 512, "stage buffers too small for the tile");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / SpTile::WGN, wn = wave % SpTile::WGN;
#pragma unroll
  for (int mi = 0; mi < SpTile::MB; ++mi)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = wm * SpTile::MB * 16 + mi * 16 + 4 * (lane >> 4) + e;
      char* row = sp_stage_region(lds0, lds1, r);
#pragma unroll
      for (int ni = 0; ni < SpTile::NB; ++ni) {
        const int col = wn * SpTile::NB * 16 + ni * 16 + (lane & 15);
        *reinterpret_cast<float*>(row + ((col >> 2) ^ (r & 31)) * 16 + (col & 3) * 4) =
            acc[mi][ni][e];
      }
    }
}
__device__ inline float4 sp_staged_chunk(char* lds0, char* lds1, int r, int c) {
  return *reinterpret_cast<const float4*>(sp_stage_region(lds0, lds1, r) + ((c ^ (r & 31)) * 16));
}

// Epilogue staging of a 128 x 128 fp32 accumulator tile through the (then
// idle) stage buffers: tile rows 0-63 go to buf0 and 64-127 to buf1, 512
// bytes per row, 16-byte column chunk c of row r at physical chunk
// c ^ (r & 31). Both the MFMA-layout writes (16 lanes per row, four rows
// 4 apart) and the row-chunk reads are free of bank conflicts. With K groups
// the first group writes and the others add their partial sums in group
// order. After a barrier every thread can read 16-byte chunks of 4
// consecutive columns.
template <typename Cfg>
__device__ inline void stage_tile(const f4 (&acc)[Cfg::MB][Cfg::NB], char* buf0, char* buf1) {
  static_assert(Cfg::BM == 128 && Cfg::BN == 128, "staging covers 128 x 128 tiles");
  static_assert(Cfg::kBufBytes >= 64 * 512, "stage buffers too small for the tile");
  const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) % Cfg::kTileWaves;
  const int wm = wave / Cfg::WGN, wn = wave % Cfg::WGN;
  const int kg = k_group<Cfg>();
#pragma unroll
  for (int grp = 0; grp < Cfg::KSPLIT; ++grp) {
    if (grp > 0) __syncthreads();
    if (kg != grp) continue;
#pragma unroll
    for (int mi = 0; mi < Cfg::MB; ++mi)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = wm * Cfg::MB * 16 + mi * 16 + 4 * (lane >> 4) + e;
        char* row = (r < 64 ? buf0 : buf1) + (r & 63) * 512;
#pragma unroll
        for (int ni = 0; ni < Cfg::NB; ++ni) {
          const int col = wn * Cfg::NB * 16 + ni * 16 + (lane & 15);
          const int ch = (col >> 2) ^ (r & 31);
          float* q = reinterpret_cast<float*>(row + ch * 16 + (col & 3) * 4);
          *q = grp == 0 ? acc[mi][ni][e] : *q + acc[mi][ni][e];
        }
      }
  }
}

__device__ inline float4 staged_chunk(const char* buf0, const char* buf1, int r, int c) {
  const char* row = (r < 64 ? buf0 : buf1) + (r & 63) * 512;
  return *reinterpret_cast<const float4*>(row + ((c ^ (r & 31)) * 16));
}

// Output coordinates of accumulator element (mi, ni, e) of this thread,
// relative to the tile origin (configurations without K groups).
template <typename Cfg>
__device__ inline int acc_row(int mi, int e) {
  static_assert(Cfg::KSPLIT == 1, "K groups hold partial sums");
  const int lane = threadIdx.x & 63, wm = (threadIdx.x >> 6) / Cfg::WGN;
  return wm * Cfg::MB * 16 + mi * 16 + 4 * (lane >> 4) + e;
}
template <typename Cfg>
__device__ inline int acc_col(int ni) {
  static_assert(Cfg::KSPLIT == 1, "K groups hold partial sums");
  const int lane = threadIdx.x & 63, wn = (threadIdx.x >> 6) % Cfg::WGN;
  return wn * Cfg::NB * 16 + ni * 16 + (lane & 15);
}

// Maps a linear workgroup index to an output tile so that the workgroups that
// the dispatcher sends to one XCD (index modulo 8) cover a compact block of
// tiles, and within an XCD consecutive workgroups sweep groups of 8 tile rows
// (shared B tiles stay in that XCD's L2).
__device__ inline void tile_of_block(int bid, int nwg, int tiles_m, int tiles_n, int* tm, int* tn) {
  int lin = bid;
  if ((nwg & 7) == 0) lin = (bid & 7) * (nwg >> 3) + (bid >> 3);
  const int group = 8 * tiles_n;
  const int g = lin / group;
  const int first_m = g * 8;
  const int gm = min(8, tiles_m - first_m);
  const int in = lin - g * group;
  *tm = first_m + in % gm;
  *tn = in / gm;
}

}  // namespace optima
