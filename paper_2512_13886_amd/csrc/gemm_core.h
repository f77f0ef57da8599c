// MFMA main loop of a 128x128 output tile of C = A B^T, both operands stored
// row-major with the contraction index contiguous ("NT"): A row r and B row c
// each hold the K values of one dot product. This is the layout of both hot
// contractions: the batched H-product Y[b][n] = sum_k Z[b][k] H[n][k] (H is
// symmetric) and the Hessian block H[i][j] = sum_t XT[i][t] XT[j][t].
//
// Work split: 256 threads = 4 waves in a 2x2 grid, each wave owning a 64x64
// sub-tile as 4x4 blocks of 16x16 MFMA outputs (16 accumulators of 4 floats).
// K advances in stages of 128 bytes per row (32 fp32 or 64 bf16 values):
// every thread fetches 4 A and 4 B 16-byte vectors of the next stage into
// registers while the waves run the MFMAs of the current stage out of LDS;
// two LDS stage buffers need one barrier per stage. LDS rows are padded by 16
// bytes so that the 16-byte fragment reads of 16 consecutive rows fall in
// distinct banks.
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
constexpr int kLdsRowBytes = kStageRowBytes + 16;
constexpr int kStageBytes = 2 * kTile * kLdsRowBytes;  // A and B tiles
constexpr int kGemmLdsBytes = 2 * kStageBytes;         // double buffered

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

// a_src[i] / b_src[i]: byte address of this thread's 16-byte vector in load
// row (threadIdx.x / 8 + 32 i) at the first stage; stage s adds
// s * kStageRowBytes. All addresses must be 16-byte aligned. The prefetch
// of stage s + 1 is unconditional (the last stage re-reads itself) so that
// the prefetch registers never leave the register file.
template <typename T>
__device__ inline void gemm_tile_mainloop(f4 (&acc)[4][4], const char* const (&a_src)[4],
                                          const char* const (&b_src)[4], int n_stages,
                                          char* lds) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int seg = tid & 7, rq = tid >> 3;

#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f4{0.f, 0.f, 0.f, 0.f};
  if (n_stages <= 0) return;

  const int st_off = rq * kLdsRowBytes + seg * 16;
  const int frag_a = (wm * 64 + (lane & 15)) * kLdsRowBytes + (lane >> 4) * 16;
  const int frag_b = kTile * kLdsRowBytes + (wn * 64 + (lane & 15)) * kLdsRowBytes + (lane >> 4) * 16;

  uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
#define OPTIMA_GLOAD(S)                                                        \
  {                                                                            \
    const size_t o_ = size_t(S) * kStageRowBytes;                              \
    ra0 = *reinterpret_cast<const uint4*>(a_src[0] + o_);                      \
    ra1 = *reinterpret_cast<const uint4*>(a_src[1] + o_);                      \
    ra2 = *reinterpret_cast<const uint4*>(a_src[2] + o_);                      \
    ra3 = *reinterpret_cast<const uint4*>(a_src[3] + o_);                      \
    rb0 = *reinterpret_cast<const uint4*>(b_src[0] + o_);                      \
    rb1 = *reinterpret_cast<const uint4*>(b_src[1] + o_);                      \
    rb2 = *reinterpret_cast<const uint4*>(b_src[2] + o_);                      \
    rb3 = *reinterpret_cast<const uint4*>(b_src[3] + o_);                      \
  }
#define OPTIMA_LSTORE(BUF)                                                     \
  {                                                                            \
    char* As_ = lds + (BUF) * kStageBytes + st_off;                            \
    char* Bs_ = As_ + kTile * kLdsRowBytes;                                    \
    *reinterpret_cast<uint4*>(As_ + 0 * 32 * kLdsRowBytes) = ra0;              \
    *reinterpret_cast<uint4*>(As_ + 1 * 32 * kLdsRowBytes) = ra1;              \
    *reinterpret_cast<uint4*>(As_ + 2 * 32 * kLdsRowBytes) = ra2;              \
    *reinterpret_cast<uint4*>(As_ + 3 * 32 * kLdsRowBytes) = ra3;              \
    *reinterpret_cast<uint4*>(Bs_ + 0 * 32 * kLdsRowBytes) = rb0;              \
    *reinterpret_cast<uint4*>(Bs_ + 1 * 32 * kLdsRowBytes) = rb1;              \
    *reinterpret_cast<uint4*>(Bs_ + 2 * 32 * kLdsRowBytes) = rb2;              \
    *reinterpret_cast<uint4*>(Bs_ + 3 * 32 * kLdsRowBytes) = rb3;              \
  }

  OPTIMA_GLOAD(0);
  OPTIMA_LSTORE(0);
  __syncthreads();

  for (int s = 0; s < n_stages; ++s) {
    const int sn = s + 1 < n_stages ? s + 1 : s;
    OPTIMA_GLOAD(sn);
    const char* base = lds + (s & 1) * kStageBytes;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      uint4 a[4], b[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        a[mi] = *reinterpret_cast<const uint4*>(base + frag_a + mi * 16 * kLdsRowBytes + c * 64);
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
        b[ni] = *reinterpret_cast<const uint4*>(base + frag_b + ni * 16 * kLdsRowBytes + c * 64);
      MfmaOp<T>::run(acc, a, b);
    }
    if (s + 1 < n_stages) OPTIMA_LSTORE((s + 1) & 1);
    __syncthreads();
  }
#undef OPTIMA_GLOAD
#undef OPTIMA_LSTORE
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
