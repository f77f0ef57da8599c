// MFMA main loop of a 128x128 output tile of C = A B^T, both operands stored
// row-major with the contraction index contiguous ("NT"): A row r and B row c
// each hold the K values of one dot product. This is the layout of both hot
// contractions: the batched H-product Y[b][n] = sum_k Z[b][k] H[n][k] (H is
// symmetric) and the Hessian block H[i][j] = sum_t XT[i][t] XT[j][t].
//
// Work split: 256 threads = 4 waves in a 2x2 grid, each wave owning a 64x64
// sub-tile as 4x4 blocks of 16x16 MFMA outputs (16 accumulators of 4 floats).
// K advances in stages of 128 bytes per row (32 fp32 or 64 bf16 values).
//
// Operands move HBM/L2 -> LDS with gfx950's direct loads
// (global_load_lds_dwordx4): no registers are spent on prefetch and the loads
// of stage s + 1 are issued right after the barrier that frees their buffer,
// ahead of the LDS reads and MFMAs of stage s (enforced with scheduling
// groups). One wave's direct load writes 1 KiB of LDS contiguously (lane l at
// byte 16 l), i.e. 8 tile rows of 128 bytes; to keep the fragment reads free
// of bank conflicts without padding, the 16-byte segment g of tile row r is
// stored at physical segment g ^ (r & 7), and each lane fetches from global
// memory the logical segment that belongs at its physical slot. The two stage
// buffers are distinct LDS arrays and the stage loop is unrolled by two, so
// that no LDS read shares an object with an in-flight direct load and the
// compiler adds no wait for it.
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

#include "common.h"

namespace optima {

constexpr int kStageRowBytes = 128;
constexpr int kStageBufBytes = 2 * kTile * kStageRowBytes;  // A and B tiles, 32 KiB

template <typename T>
struct MfmaOp;

template <>
struct MfmaOp<float> {
  __device__ static inline void run(f4 (&acc)[4][4], const uint4 (&a)[4], const uint4 (&b)[4]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const unsigned av = e == 0 ? a[mi].x : e == 1 ? a[mi].y : e == 2 ? a[mi].z : a[mi].w;
          const unsigned bv = e == 0 ? b[ni].x : e == 1 ? b[ni].y : e == 2 ? b[ni].z : b[ni].w;
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x4f32(
              __uint_as_float(av), __uint_as_float(bv), acc[mi][ni], 0, 0, 0);
        }
      }
    }
  }
};

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
// takes 4 dp bytes, like fp32, and each 128-byte K stage of the GEMM core
// holds 32 columns of both planes.
__device__ inline void store_split(uint16_t* row_planes, int n, float v) {
  const uint32_t hi = bf16_rne_bits(v);
  const uint32_t lo = bf16_rne_bits(v - bf16_bits_value(hi));
  uint16_t* b = row_planes + (n >> 5) * 64 + (n & 31);
  b[0] = uint16_t(hi);
  b[32] = uint16_t(lo);
}

template <>
struct MfmaOp<Bf16Tag> {
  __device__ static inline void run(f4 (&acc)[4][4], const uint4 (&a)[4], const uint4 (&b)[4]) {
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, a[mi]), __builtin_bit_cast(bf16x8, b[ni]),
            acc[mi][ni], 0, 0, 0);
      }
    }
  }
};

// Rows of the tile that this thread's direct loads fetch: round i (0..3)
// covers tile row load_row(i); the byte offset of the fetched 16-byte segment
// within the row's 128-byte stage is load_seg_bytes().
__device__ inline int load_row(int i) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  return (i * 4 + wave) * 8 + (lane >> 3);
}
__device__ inline int load_seg_bytes() {
  const int lane = threadIdx.x & 63;
  return ((lane & 7) ^ (lane >> 3)) * 16;
}

template <typename T>
struct StageShape;
template <>
struct StageShape<float> {
  static constexpr int kMfmaPerChunk = 64;
};
template <>
struct StageShape<Bf16Tag> {
  static constexpr int kMfmaPerChunk = 16;
};

__device__ inline void issue_stage(const char* const (&a_src)[4], const char* const (&b_src)[4],
                                   int s, char* buf) {
  const size_t o = size_t(s) * kStageRowBytes;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    char* d = buf + (i * 4 + wave) * 1024;
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(a_src[i] + o),
        (__attribute__((address_space(3))) void*)d, 16, 0, 0);
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(b_src[i] + o),
        (__attribute__((address_space(3))) void*)(d + kTile * kStageRowBytes), 16, 0, 0);
  }
}

template <typename T>
__device__ inline void compute_stage(f4 (&acc)[4][4], const char* buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1, g = lane >> 4;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    uint4 a[4], b[4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
      const int r = wm * 64 + mi * 16 + (lane & 15);
      a[mi] = *reinterpret_cast<const uint4*>(buf + r * kStageRowBytes + (((4 * c + g) ^ (r & 7)) * 16));
    }
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
      const int r = wn * 64 + ni * 16 + (lane & 15);
      b[ni] = *reinterpret_cast<const uint4*>(buf + kTile * kStageRowBytes + r * kStageRowBytes +
                                             (((4 * c + g) ^ (r & 7)) * 16));
    }
    MfmaOp<T>::run(acc, a, b);
  }
  // Order within the stage: the 8 direct loads issued just before, then per
  // chunk its 8 LDS reads and its MFMAs.
  __builtin_amdgcn_sched_group_barrier(0x020, 8, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, StageShape<T>::kMfmaPerChunk, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, StageShape<T>::kMfmaPerChunk, 0);
}

// Split-bf16 stage: segments 0-3 of a row hold the hi plane of 32 K values,
// segments 4-7 the lo plane; per 16x16 block the stage runs hi*hi, then
// hi*lo and lo*hi, each a v_mfma_f32_16x16x32_bf16.
template <>
__device__ inline void compute_stage<Bf16x3Tag>(f4 (&acc)[4][4], const char* buf) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1, g = lane >> 4;
  uint4 a0[4], b0[4], a1[4], b1[4];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int r = wm * 64 + mi * 16 + (lane & 15);
    a0[mi] = *reinterpret_cast<const uint4*>(buf + r * kStageRowBytes + ((g ^ (r & 7)) * 16));
  }
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const int r = wn * 64 + ni * 16 + (lane & 15);
    b0[ni] = *reinterpret_cast<const uint4*>(buf + kTile * kStageRowBytes + r * kStageRowBytes +
                                             ((g ^ (r & 7)) * 16));
  }
  MfmaOp<Bf16Tag>::run(acc, a0, b0);
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int r = wm * 64 + mi * 16 + (lane & 15);
    a1[mi] = *reinterpret_cast<const uint4*>(buf + r * kStageRowBytes + (((4 + g) ^ (r & 7)) * 16));
  }
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const int r = wn * 64 + ni * 16 + (lane & 15);
    b1[ni] = *reinterpret_cast<const uint4*>(buf + kTile * kStageRowBytes + r * kStageRowBytes +
                                             (((4 + g) ^ (r & 7)) * 16));
  }
  MfmaOp<Bf16Tag>::run(acc, a0, b1);
  MfmaOp<Bf16Tag>::run(acc, a1, b0);
  __builtin_amdgcn_sched_group_barrier(0x020, 8, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);
}

// s_waitcnt vmcnt(0), leaving expcnt and lgkmcnt unwaited.
__device__ inline void wait_direct_loads() { __builtin_amdgcn_s_waitcnt(0xF70); }

// a_src[i] / b_src[i]: address of the 16-byte segment this thread fetches in
// tile row load_row(i) at the first stage (row start + load_seg_bytes());
// stage s adds s * kStageRowBytes. All addresses must be 16-byte aligned.
template <typename T>
__device__ inline void gemm_tile_mainloop(f4 (&acc)[4][4], const char* const (&a_src)[4],
                                          const char* const (&b_src)[4], int n_stages) {
  __shared__ __attribute__((aligned(1024))) char lds0[kStageBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[kStageBufBytes];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f4{0.f, 0.f, 0.f, 0.f};
  if (n_stages <= 0) return;

  issue_stage(a_src, b_src, 0, lds0);
  int s = 0;
  for (; s + 1 < n_stages; s += 2) {
    wait_direct_loads();
    __syncthreads();
    issue_stage(a_src, b_src, s + 1, lds1);
    compute_stage<T>(acc, lds0);
    wait_direct_loads();
    __syncthreads();
    issue_stage(a_src, b_src, s + 2 < n_stages ? s + 2 : n_stages - 1, lds0);
    compute_stage<T>(acc, lds1);
  }
  if (s < n_stages) {  // odd count: the last stage is in lds0
    wait_direct_loads();
    __syncthreads();
    compute_stage<T>(acc, lds0);
  }
  // No direct load may still be writing LDS when the workgroup moves on.
  wait_direct_loads();
  __syncthreads();
}

// Output coordinates of accumulator element (mi, ni, e) of this thread,
// relative to the tile origin.
__device__ inline int acc_row(int mi, int e) {
  const int lane = threadIdx.x & 63, wm = (threadIdx.x >> 6) >> 1;
  return wm * 64 + mi * 16 + 4 * (lane >> 4) + e;
}
__device__ inline int acc_col(int ni) {
  const int lane = threadIdx.x & 63, wn = (threadIdx.x >> 6) & 1;
  return wn * 64 + ni * 16 + (lane & 15);
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
