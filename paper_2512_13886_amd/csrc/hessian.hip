// Layer Hessian H = X^T X (Section 3.4 "Hessian calculation") and damping.
//
// The tokens arrive row-major, X[t][i]. Both MFMA operands of X^T X need the
// token index contiguous, so each slab of up to kMaxSlab tokens is first
// transposed into XT[i][t] (features padded to the 128-wide tile, tokens
// padded with zeros to a whole 128-byte stage). The product then runs on the
// lower-triangular 128x128 tiles only, each tile's slab of tokens split into
// `splits` contiguous ranges so that small layers still fill the GPU. Every
// (tile, split) workgroup adds its partial sum into a private fp32 buffer, so
// no atomics are involved and the result is deterministic. A final pass sums
// the partials in split order, adds the incoming H when accumulating, and
// writes each lower-triangle value to both (i, j) and (j, i): H comes out
// exactly symmetric.
//
// bf16 tokens use v_mfma_f32_16x16x32_bf16 (the bf16 x bf16 products are exact
// in fp32); fp32 tokens use v_mfma_f32_16x16x4_f32.
//
// bf16 tokens with d a multiple of 256 (every transformer width here) take a
// direct path instead: no transpose. Token rows go from X straight into LDS
// and the MFMA operands are gathered from there with gfx950's transposing LDS
// read, on 256 x 256 lower-triangular tiles; the whole token range is one
// launch, split along the tokens so that the tiles fill all CUs evenly.
#include "common.h"
#include "gemm_core.h"

namespace optima {
namespace {

constexpr int64_t kMaxSlab = 65536;

struct HessPlan {
  int64_t dp, esz, kse, slab, tiles;
  int splits;
  size_t xt_elems, part_elems;
};

HessPlan plan(int64_t n_tok, int64_t d, int dtype) {
  HessPlan p{};
  p.dp = round_up(d, kTile);
  p.esz = dtype == OPTIMA_DTYPE_BF16 ? 2 : 4;
  p.kse = kStageRowBytes / p.esz;  // tokens per 128-byte stage
  p.slab = std::min<int64_t>(round_up(std::max<int64_t>(n_tok, 1), p.kse), kMaxSlab);
  const int64_t T = p.dp / kTile;
  p.tiles = T * (T + 1) / 2;
  const int64_t stages = p.slab / p.kse;
  p.splits = int(std::max<int64_t>(1, std::min<int64_t>({ceil_div(2048, p.tiles), 64, stages})));
  p.xt_elems = size_t(p.dp) * size_t(p.slab);
  p.part_elems = size_t(p.splits) * size_t(p.dp) * size_t(p.dp);
  return p;
}

template <typename T>
__global__ void __launch_bounds__(kThreads) k_transpose(const T* X, int64_t d, int64_t t0,
                                                        int64_t rows, int64_t cols_pad, int64_t dp,
                                                        T* XT) {
  __shared__ T tile[64][65];
  const int64_t tt0 = int64_t(blockIdx.x) * 64;  // token within the slab
  const int64_t f0 = int64_t(blockIdx.y) * 64;   // feature
  for (int e = threadIdx.x; e < 64 * 64; e += kThreads) {
    const int r = e >> 6, c = e & 63;
    const int64_t tt = tt0 + r, f = f0 + c;
    T v{};
    if (tt < rows && f < d) v = X[(t0 + tt) * d + f];
    tile[r][c] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += kThreads) {
    const int r = e >> 6, c = e & 63;  // r: feature, c: token
    const int64_t f = f0 + r, tt = tt0 + c;
    if (f < dp && tt < cols_pad) XT[f * cols_pad + tt] = tile[c][r];
  }
}

// Lower-triangular tile index -> (ti, tj), ti >= tj.
__device__ inline void tri_tile(int idx, int* ti, int* tj) {
  int i = int((sqrtf(8.f * float(idx) + 1.f) - 1.f) * 0.5f);
  while ((i + 1) * (i + 2) / 2 <= idx) ++i;
  while (i * (i + 1) / 2 > idx) --i;
  *ti = i;
  *tj = idx - i * (i + 1) / 2;
}

template <typename T>
__global__ void __launch_bounds__(kThreads) k_syrk(const char* XT, int64_t pitch_bytes,
                                                   int stages, int splits, int64_t dp,
                                                   float* part, int first) {
  __shared__ __attribute__((aligned(1024))) char lds0[Tile128::kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[Tile128::kBufBytes];
  const int tile = blockIdx.x / splits;
  const int sp = blockIdx.x - tile * splits;
  int ti, tj;
  tri_tile(tile, &ti, &tj);
  const int s0 = int(int64_t(stages) * sp / splits);
  const int s1 = int(int64_t(stages) * (sp + 1) / splits);
  using Cfg = Tile128;
  Operands<Cfg> src;
  const int64_t k_off = int64_t(s0) * Cfg::SRB;
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsA; ++i)
    src.a[i] = XT + (int64_t(ti) * kTile + load_row<Cfg>(i)) * pitch_bytes + k_off +
               load_seg_bytes<Cfg>(i);
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsB; ++i)
    src.b[i] = XT + (int64_t(tj) * kTile + load_row<Cfg>(i)) * pitch_bytes + k_off +
               load_seg_bytes<Cfg>(i);
  f4 acc[Cfg::MB][Cfg::NB];
  gemm_tile_mainloop<Cfg, T>(acc, src, s1 - s0, lds0, lds1, nullptr);
  float* P = part + size_t(sp) * size_t(dp) * size_t(dp);
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t i = int64_t(ti) * kTile + acc_row<Cfg>(mi, e);
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int64_t j = int64_t(tj) * kTile + acc_col<Cfg>(ni);
        float* q = P + i * dp + j;
        *q = first ? acc[mi][ni][e] : *q + acc[mi][ni][e];
      }
    }
}

// Sums the split partials of the 64x64 block (bi, bj), bi >= bj, into H and
// mirrors it to the upper triangle.
__global__ void __launch_bounds__(kThreads) k_hess_reduce(const float* part, int splits, int64_t dp,
                                                          int64_t d, float* H, int accumulate) {
  __shared__ float tile[64][65];
  int bi, bj;
  tri_tile(blockIdx.x, &bi, &bj);
  for (int e = threadIdx.x; e < 64 * 64; e += kThreads) {
    const int r = e >> 6, c = e & 63;
    const int64_t i = int64_t(bi) * 64 + r, j = int64_t(bj) * 64 + c;
    float v = 0.f;
    if (i < d && j < d && (bi > bj || r >= c)) {
      for (int s = 0; s < splits; ++s) v += part[size_t(s) * dp * dp + i * dp + j];
      if (accumulate) v = H[i * d + j] + v;
      H[i * d + j] = v;
    }
    tile[r][c] = v;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += kThreads) {
    const int r = e >> 6, c = e & 63;  // output row bj*64 + r, column bi*64 + c
    const int64_t i = int64_t(bj) * 64 + r, j = int64_t(bi) * 64 + c;
    if (i < d && j < d && (bi > bj || c > r)) H[i * d + j] = tile[c][r];
  }
}

// The same for d % 4 == 0 with 16-byte chunks of 4 columns: thread t takes
// chunks t, t + 256, t + 512 and t + 768 of the block and adds the splits
// of all four in split order, so 16 loads are in flight per step. The sums
// are those of k_hess_reduce, bit for bit.
__global__ void __launch_bounds__(kThreads) k_hess_reduce4(const float* part, int splits, int64_t dp,
                                                           int64_t d, float* H, int accumulate) {
  static_assert(kThreads == 256, "four chunks per thread cover the 64 x 64 block");
  __shared__ float tile[64][65];
  int bi, bj;
  tri_tile(blockIdx.x, &bi, &bj);
  float4 v[4];
  int64_t off[4];
  bool in[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int ch = threadIdx.x + kThreads * q, r = ch >> 4, c = 4 * (ch & 15);
    const int64_t i = int64_t(bi) * 64 + r, j = int64_t(bj) * 64 + c;
    in[q] = i < d && j < d;  // d % 4 == 0: chunks are all in or all out
    off[q] = in[q] ? i * dp + j : 0;
    v[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const size_t plane = size_t(dp) * size_t(dp);
#pragma unroll 2
  for (int sp = 0; sp < splits; ++sp) {
    const float* P = part + size_t(sp) * plane;
    float4 t[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) t[q] = *reinterpret_cast<const float4*>(P + off[q]);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[q].x += t[q].x;
      v[q].y += t[q].y;
      v[q].z += t[q].z;
      v[q].w += t[q].w;
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int ch = threadIdx.x + kThreads * q, r = ch >> 4, c = 4 * (ch & 15);
    const int64_t i = int64_t(bi) * 64 + r, j = int64_t(bj) * 64 + c;
    float e[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
    if (in[q]) {
      float* h = H + i * d + j;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const bool lower = bi > bj || r >= c + k;
        if (!lower) e[k] = 0.f;
        else if (accumulate) e[k] = h[k] + e[k];
      }
      if (bi > bj) {
        *reinterpret_cast<float4*>(h) = make_float4(e[0], e[1], e[2], e[3]);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (r >= c + k) h[k] = e[k];
      }
    } else {
      e[0] = e[1] = e[2] = e[3] = 0.f;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) tile[r][c + k] = e[k];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += kThreads) {
    const int r = e >> 6, c = e & 63;  // output row bj*64 + r, column bi*64 + c
    const int64_t i = int64_t(bj) * 64 + r, j = int64_t(bi) * 64 + c;
    if (i < d && j < d && (bi > bj || c > r)) H[i * d + j] = tile[c][r];
  }
}

// Shared diagonal preconditioning: D_i = diag(H)_i^(-1/2) (computed in fp64,
// 1 where the diagonal is not positive and finite).
__global__ void __launch_bounds__(kThreads) k_jacobi_d(const float* H, int64_t d, float* D) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i >= d) return;
  const double h = H[i * d + i];
  D[i] = (h > 0.0 && isfinite(h)) ? float(1.0 / sqrt(h)) : 1.f;
}

// H_ij <- H_ij (D_i D_j): the factor is the same product for (i, j) and
// (j, i), so an exactly symmetric H stays exactly symmetric.
__global__ void __launch_bounds__(kThreads) k_jacobi_scale(float* H, int64_t d, const float* D) {
  const int64_t total = d * d;
  for (int64_t e = int64_t(blockIdx.x) * kThreads + threadIdx.x; e < total;
       e += int64_t(gridDim.x) * kThreads) {
    const int64_t i = e / d, j = e - i * d;
    H[e] = H[e] * (D[i] * D[j]);
  }
}

__global__ void __launch_bounds__(1024) k_damp(float* H, int64_t d, float rel, float* lambda_out) {
  __shared__ double red[16];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < d; i += 1024) s += double(H[i * d + i]);
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  double tr = 0.0;
  for (int w = 0; w < 16; ++w) tr += red[w];
  const double lam = double(rel) * tr / double(d);
  if (threadIdx.x == 0) *lambda_out = isfinite(lam) ? float(lam) : __builtin_nanf("");
  if (!isfinite(lam)) return;
  for (int64_t i = threadIdx.x; i < d; i += 1024) H[i * d + i] = float(double(H[i * d + i]) + lam);
}

// ---------------------------------------------------------------------------
// Direct path (bf16, d % 256 == 0)
// ---------------------------------------------------------------------------
//
// Workgroup: one 256 x 256 output tile (ti, tj), ti >= tj, over a contiguous
// range of 64-token stages; 8 waves in a 4 x 2 grid, each wave owning 64 x
// 128 outputs (4 x 8 blocks of 16 x 16). The stages stream through a ring of
// four LDS buffers of 32 tokens each, so that while one buffer is read the
// loads of the next three are in flight. Buffer: block A holds
// X[t][256 ti + 0..255] and block B X[t][256 tj + 0..255] for its 32 tokens,
// one 512-byte row per token, written by direct loads (one wave load = 1 KiB
// = 2 token rows). Within a row the 16-byte segment g sits at physical
// segment g ^ swz(row), which keeps both the loads' writes and the
// transposing reads free of bank conflicts.
//
// Operands: ds_read_b64_tr_b16 treats the eight-byte reads of each 16-lane
// group as a 4 x 16 matrix of 16-bit values (lane j supplies row j / 4,
// columns 4 (j % 4) .. 4 (j % 4) + 3) and returns column i to lane i. Lanes
// j of group g address token row 8 g + 4 h + j / 4 and features
// f + 4 (j % 4): lane i then holds tokens 8 g + 4 h + 0..3 of feature f + i,
// and the reads for h = 0 and h = 1 together give the 8 consecutive tokens
// that a 16x16x32 bf16 MFMA takes from lane (g, i), for both operands. The
// output block (lane, e) is then H[f_a + 4 g + e][f_b + i] as in the NT core.
namespace dt {
constexpr int kRows = 64;                   // tokens per stage (unit of the token splits)
constexpr int kBufRows = 32;                // tokens per ring buffer (one MFMA K step)
constexpr int kRing = 4;                    // ring buffers
constexpr int kBlock = 256;                 // features per operand block (tile side)
constexpr int kRowBytes = 2 * kBlock;       // 512
constexpr int kBlockBytes = kBufRows * kRowBytes;
constexpr int kBufBytes = 2 * kBlockBytes;  // 32 KiB per ring buffer
constexpr int kMaxSplits = 64;
constexpr int kCus = 256;                   // MI355X compute units (sizing only)

// Wave layout of the 256 x 256 tile: WAVES / 2 x 2 waves; with 8 waves each
// owns 64 x 128 outputs and two waves share each SIMD. (Four waves of
// 128 x 128 read a third fewer LDS bytes per MFMA, but with one wave per SIMD
// nothing hides the LDS and load latency: measured 1.5 times slower.)
template <int WAVES>
struct Cfg {
  static constexpr int kWaves = WAVES;
  static constexpr int kThreads = 64 * WAVES;
  static constexpr int WGN = 2, WGM = WAVES / WGN;
  static constexpr int kMB = kBlock / WGM / 16, kNB = kBlock / WGN / 16;
  static constexpr int kLoads = kBlockBytes / 1024 / WAVES;  // wave loads per block per thread
  static constexpr int kBufLoads = 2 * kLoads;                // per buffer (blocks A and B)
};

// Physical XOR of the 16-byte segment index for token row r of a stage:
// flips segment bits 1-3 by (r & 3) and bit 3 of r.
__device__ inline int swz(int r) { return 2 * ((r & 3) | (((r >> 3) & 1) << 2)); }

typedef short v4s __attribute__((ext_vector_type(4)));

__device__ inline uint2 tr_read(const char* p) {
  const v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s*)(p));
  return __builtin_bit_cast(uint2, v);
}

// Direct loads of one ring buffer. Round i of this thread fetches token row
// row0 + 2 WAVES i (row0 = 2 wave + lane / 32) at physical segment lane % 32;
// `a` / `b` point at that row's A / B block for round 0 without the segment
// offset, seg[i & 1] is the logical segment's byte offset for the round.
template <typename C>
__device__ inline void issue(const char* a, const char* b, int64_t round_bytes, const int (&seg)[2],
                             char* buf) {
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < C::kLoads; ++i)
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(a + i * round_bytes + seg[i & 1]),
        (__attribute__((address_space(3))) void*)(buf + (i * C::kWaves + wave) * 1024), 16, 0, 0);
#pragma unroll
  for (int i = 0; i < C::kLoads; ++i)
    __builtin_amdgcn_global_load_lds(
        (const __attribute__((address_space(1))) void*)(b + i * round_bytes + seg[i & 1]),
        (__attribute__((address_space(3))) void*)(buf + kBlockBytes + (i * C::kWaves + wave) * 1024),
        16, 0, 0);
}

// Operand fragments of the 32 tokens in ring buffer `buf`.
template <typename C>
__device__ inline void read_frags(const char* buf, uint4 (&a)[C::kMB], uint4 (&b)[C::kNB]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int g = lane >> 4, j = lane & 15;
  // Token row 8 g + 4 h + j / 4 has (row & 3) = j / 4 and bit 3 of the row
  // equal to g & 1, so its swizzle depends on the lane only.
  const int sw = 2 * ((j >> 2) | ((g & 1) << 2));
  const int intra = 8 * (j & 1);
  const int seg_lane = (j & 3) >> 1;
  const char* A0 = buf + (8 * g + (j >> 2)) * kRowBytes;
  const char* A1 = A0 + 4 * kRowBytes;
#pragma unroll
  for (int mi = 0; mi < C::kMB; ++mi) {
    const int o = (((((wm * C::kMB + mi) * 16) >> 3) + seg_lane) ^ sw) * 16 + intra;
    const uint2 lo = tr_read(A0 + o), hi = tr_read(A1 + o);
    a[mi] = make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
#pragma unroll
  for (int ni = 0; ni < C::kNB; ++ni) {
    const int o = (((((wn * C::kNB + ni) * 16) >> 3) + seg_lane) ^ sw) * 16 + intra;
    const uint2 lo = tr_read(A0 + kBlockBytes + o), hi = tr_read(A1 + kBlockBytes + o);
    b[ni] = make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
}

template <typename C>
__device__ inline void mfma_step(f4 (&acc)[C::kMB][C::kNB], const uint4 (&a)[C::kMB],
                                 const uint4 (&b)[C::kNB]) {
#pragma unroll
  for (int mi = 0; mi < C::kMB; ++mi)
#pragma unroll
    for (int ni = 0; ni < C::kNB; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          __builtin_bit_cast(bf16x8, a[mi]), __builtin_bit_cast(bf16x8, b[ni]), acc[mi][ni], 0, 0,
          0);
}

template <typename C>
__device__ inline void compute(f4 (&acc)[C::kMB][C::kNB], const char* buf) {
  constexpr int kReads = 2 * (C::kMB + C::kNB), kMfma = C::kMB * C::kNB;
  uint4 a[C::kMB], b[C::kNB];
  read_frags<C>(buf, a, b);
  mfma_step<C>(acc, a, b);
  __builtin_amdgcn_sched_group_barrier(0x020, C::kBufLoads, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
  __builtin_amdgcn_sched_group_barrier(0x008, kMfma, 0);
}

// One step of the ring: buffer `cur` holds the next 32 tokens once this
// wave's loads other than the two most recent buffers' have landed and every
// wave has arrived (so every wave is also done reading `nxt`, read one step
// earlier); then the loads of the buffer three ahead go to `nxt` and `cur` is
// consumed.
template <typename C>
__device__ inline void ring_step(f4 (&acc)[C::kMB][C::kNB], const char* a, const char* b,
                                 int64_t round_bytes, const int (&seg)[2], char* cur, char* nxt) {
  ring_barrier<2 * C::kBufLoads>();
  issue<C>(a, b, round_bytes, seg, nxt);
  compute<C>(acc, cur);
}

}  // namespace dt

// Lower-triangle tile (ti >= tj) of position idx in an order that keeps
// nearby positions on few feature blocks: the triangle of nt blocks is cut
// into super-tiles of 4 x 4 blocks, taken row by row (SI >= SJ), and each
// super-tile's tiles row by row. 32 consecutive positions touch 8 to 12
// blocks instead of nearly all of them.
__device__ inline void grouped_tri_tile(int idx, int nt, int* ti, int* tj) {
  constexpr int G = 4;
  const int ns = (nt + G - 1) / G;
  *ti = 0;
  *tj = 0;
  for (int SI = 0; SI < ns; ++SI)
    for (int SJ = 0; SJ <= SI; ++SJ) {
      const int i0 = G * SI, i1 = min(i0 + G, nt), j0 = G * SJ, j1 = min(j0 + G, nt);
      const int w = j1 - j0, m = i1 - i0;
      const int cnt = SI != SJ ? m * w : m * (m + 1) / 2;
      if (idx < cnt) {
        if (SI != SJ) {
          *ti = i0 + idx / w;
          *tj = j0 + idx % w;
        } else {
          int r = 0;
          while (idx > r) idx -= ++r;
          *ti = i0 + r;
          *tj = j0 + idx;
        }
        return;
      }
      idx -= cnt;
    }
}

// X: [n_rows][d] bf16 with n_rows >= stages * 64. The work units are the
// (split, tile) pairs of the triangle of d / 256 blocks; split sp covers
// stages [stages sp / splits, stages (sp + 1) / splits). The dispatcher
// sends workgroup b to XCD b % 8, so XCD x runs workgroups x, x + 8, ... in
// that order. XCD x owns the x-th eighth of the tiles in grouped_tri_tile
// order (a few feature blocks) for every split, and runs them split by
// split. Its 32 resident workgroups then share one or two token ranges and
// few blocks, which its L2 fetches once for all of them; and all eight XCDs
// move through the tokens together, so the device-wide cache serves one
// XCD's misses to the others. The grid is 8 times the largest XCD share;
// workgroups beyond their XCD's share exit at once.
// Writes (first) or adds the tile's partial sum into part[sp] ([d][d] fp32).
template <int WAVES>
__global__ void __launch_bounds__(64 * WAVES) k_syrk_direct(const uint16_t* X, int64_t d,
                                                            int stages, int splits, float* part,
                                                            int first) {
  using namespace dt;
  using C = Cfg<WAVES>;
  __shared__ __attribute__((aligned(1024))) char lds0[kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds2[kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds3[kBufBytes];
  static_assert(kRing == 4 && kRows == 2 * kBufRows, "the loop below is written for this ring");
  const int nt = int(d / kBlock);
  const int n_tiles = nt * (nt + 1) / 2;
  const int x = blockIdx.x & 7, l = blockIdx.x >> 3;
  const int t0 = int(int64_t(n_tiles) * x / 8), tx = int(int64_t(n_tiles) * (x + 1) / 8) - t0;
  if (int64_t(l) >= int64_t(tx) * splits) return;
  const int sp = l / tx;
  int ti, tj;
  grouped_tri_tile(t0 + l % tx, nt, &ti, &tj);
  const int s0 = int(int64_t(stages) * sp / splits);
  const int s1 = int(int64_t(stages) * (sp + 1) / splits);
  const int n = s1 - s0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = 2 * wave + (lane >> 5);
  const int seg[2] = {((lane & 31) ^ swz(row)) * 16, ((lane & 31) ^ swz(row + 2 * WAVES)) * 16};
  const int64_t row_bytes = d * 2;
  const char* xb = reinterpret_cast<const char*>(X) + (int64_t(s0) * kRows + row) * row_bytes;
  const char* a = xb + int64_t(ti) * kBlock * 2;
  const char* b = xb + int64_t(tj) * kBlock * 2;
  const int64_t round_bytes = 2 * WAVES * row_bytes;
  const int64_t buf_bytes = kBufRows * row_bytes;

  f4 acc[C::kMB][C::kNB];
#pragma unroll
  for (int mi = 0; mi < C::kMB; ++mi)
#pragma unroll
    for (int ni = 0; ni < C::kNB; ++ni) acc[mi][ni] = f4{0.f, 0.f, 0.f, 0.f};
  if (n > 0) {
    // nb = 2 n buffers of 32 tokens. Loads past the last buffer repeat it
    // (into buffers nobody reads again) so that every step waits for the
    // same count; they are drained before the epilogue.
    const int nb = 2 * n;
    auto at = [nb, buf_bytes](const char* p, int q) { return p + (q < nb ? q : nb - 1) * buf_bytes; };
    issue<C>(a, b, round_bytes, seg, lds0);
    issue<C>(at(a, 1), at(b, 1), round_bytes, seg, lds1);
    issue<C>(at(a, 2), at(b, 2), round_bytes, seg, lds2);
    int q = 0;
    for (; q + 4 <= nb; q += 4) {
      ring_step<C>(acc, at(a, q + 3), at(b, q + 3), round_bytes, seg, lds0, lds3);
      ring_step<C>(acc, at(a, q + 4), at(b, q + 4), round_bytes, seg, lds1, lds0);
      ring_step<C>(acc, at(a, q + 5), at(b, q + 5), round_bytes, seg, lds2, lds1);
      ring_step<C>(acc, at(a, q + 6), at(b, q + 6), round_bytes, seg, lds3, lds2);
    }
    if (q < nb) {
      ring_step<C>(acc, at(a, q + 3), at(b, q + 3), round_bytes, seg, lds0, lds3);
      ring_step<C>(acc, at(a, q + 4), at(b, q + 4), round_bytes, seg, lds1, lds0);
    }
    wait_vmcnt<0>();
    __syncthreads();
  }
  float* P = part + size_t(sp) * size_t(d) * size_t(d);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
#pragma unroll
  for (int mi = 0; mi < C::kMB; ++mi)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t i = int64_t(ti) * kBlock + (wm * C::kMB + mi) * 16 + 4 * (lane >> 4) + e;
#pragma unroll
      for (int ni = 0; ni < C::kNB; ++ni) {
        const int64_t jj = int64_t(tj) * kBlock + (wn * C::kNB + ni) * 16 + (lane & 15);
        float* q = P + i * d + jj;
        *q = first ? acc[mi][ni][e] : *q + acc[mi][ni][e];
      }
    }
}

// Copies `rows` (< 64) token rows starting at t0 into a zero-padded 64-row
// buffer so that the direct path never loads past the end of X.
__global__ void __launch_bounds__(kThreads) k_tail_rows(const uint16_t* X, int64_t d, int64_t t0,
                                                        int rows, uint16_t* out) {
  const int64_t total = int64_t(dt::kRows) * d;
  for (int64_t e = int64_t(blockIdx.x) * kThreads + threadIdx.x; e < total;
       e += int64_t(gridDim.x) * kThreads) {
    const int64_t r = e / d;
    out[e] = r < rows ? X[(t0 + r) * d + (e - r * d)] : uint16_t(0);
  }
}

constexpr int kDirectWaves = 8;  // the layout of k_syrk_direct that the library launches

struct DirectPlan {
  int64_t tiles;
  int full_stages, tail_rows, splits;
  size_t part_elems;
};

// Grid of k_syrk_direct over `tiles` tiles and `splits` splits: 8 times the
// largest XCD share (ceil(tiles / 8) tiles, every split).
unsigned direct_grid(int64_t tiles, int splits) {
  return unsigned(8 * ceil_div(tiles, int64_t(8)) * splits);
}

bool direct_ok(int64_t d, int dtype) {
  return dtype == OPTIMA_DTYPE_BF16 && d % dt::kBlock == 0;
}

DirectPlan direct_plan(int64_t n_tok, int64_t d) {
  DirectPlan p{};
  const int64_t nt = d / dt::kBlock;
  p.tiles = nt * (nt + 1) / 2;
  p.full_stages = int(n_tok / dt::kRows);
  p.tail_rows = int(n_tok % dt::kRows);
  // Splits along the tokens: the fewest rounds of workgroups per CU relative
  // to the work, with 1% per split for the partial sums; at most 4 GiB of
  // partials. Each XCD (an eighth of the CUs) runs the largest eighth of the
  // tiles for every split.
  int best = 1;
  double best_cost = 1e30;
  const int max_s = std::max(1, std::min(dt::kMaxSplits, p.full_stages));
  for (int S = 1; S <= max_s; ++S) {
    if (S > 1 && double(S) * double(d) * double(d) * 4.0 > double(int64_t(1) << 32)) break;
    const double rounds = double(ceil_div(ceil_div(p.tiles, int64_t(8)) * S, dt::kCus / 8));
    const double c = rounds / S * (1.0 + 0.01 * S);
    if (c < best_cost - 1e-12) {
      best = S;
      best_cost = c;
    }
  }
  p.splits = best;
  p.part_elems = size_t(p.splits) * size_t(d) * size_t(d);  // one [d][d] partial per split
  return p;
}

// Sums the split partials (pitch dp) into H (pitch d), both triangles.
optima_status reduce_partials(const float* part, int splits, int64_t dp, int64_t d, float* H,
                              int accumulate, hipStream_t s) {
  const int64_t B = ceil_div(d, 64);
  const dim3 grid(unsigned(B * (B + 1) / 2));
  if (d % 4 == 0)
    hipLaunchKernelGGL(k_hess_reduce4, grid, dim3(kThreads), 0, s, part, splits, dp, d, H,
                       accumulate);
  else
    hipLaunchKernelGGL(k_hess_reduce, grid, dim3(kThreads), 0, s, part, splits, dp, d, H,
                       accumulate);
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

}  // namespace

size_t hessian_workspace_bytes(int64_t n_tok, int64_t d, int dtype) {
  Carver c(nullptr);
  if (direct_ok(d, dtype)) {
    const DirectPlan p = direct_plan(n_tok, d);
    c.take<float>(p.part_elems);
    c.take<uint16_t>(size_t(dt::kRows) * size_t(d));
    return c.bytes();
  }
  const HessPlan p = plan(n_tok, d, dtype);
  c.take<char>(p.xt_elems * p.esz);
  c.take<float>(p.part_elems);
  return c.bytes();
}

optima_status hessian_accumulate(const void* X, int dtype, int64_t n_tok, int64_t d, float* H,
                                 int accumulate, void* ws, hipStream_t s) {
  if (n_tok == 0) {
    if (!accumulate) OPTIMA_HIP_TRY(hipMemsetAsync(H, 0, size_t(d) * size_t(d) * sizeof(float), s));
    return OPTIMA_OK;
  }
  if (direct_ok(d, dtype) && aligned16(X)) {
    const DirectPlan p = direct_plan(n_tok, d);
    Carver c(ws);
    float* part = c.take<float>(p.part_elems);
    uint16_t* tail = c.take<uint16_t>(size_t(dt::kRows) * size_t(d));
    const uint16_t* Xb = static_cast<const uint16_t*>(X);
    int splits = p.splits;
    if (p.full_stages > 0) {
      hipLaunchKernelGGL(k_syrk_direct<kDirectWaves>, dim3(direct_grid(p.tiles, splits)),
                         dim3(64 * kDirectWaves), 0, s, Xb, d, p.full_stages, splits, part, 1);
      OPTIMA_LAUNCH_CHECK();
    } else {
      splits = 1;
    }
    if (p.tail_rows > 0) {
      hipLaunchKernelGGL(k_tail_rows, dim3(256), dim3(kThreads), 0, s, Xb, d,
                         int64_t(p.full_stages) * dt::kRows, p.tail_rows, tail);
      OPTIMA_LAUNCH_CHECK();
      hipLaunchKernelGGL(k_syrk_direct<kDirectWaves>, dim3(direct_grid(p.tiles, 1)),
                         dim3(64 * kDirectWaves), 0, s, tail, d, 1, 1, part,
                         p.full_stages > 0 ? 0 : 1);
      OPTIMA_LAUNCH_CHECK();
    }
    return reduce_partials(part, splits, d, d, H, accumulate, s);
  }
  const HessPlan p = plan(n_tok, d, dtype);
  Carver c(ws);
  char* XT = c.take<char>(p.xt_elems * p.esz);
  float* part = c.take<float>(p.part_elems);
  int first = 1;
  for (int64_t t0 = 0; t0 < n_tok; t0 += p.slab) {
    const int64_t rows = std::min<int64_t>(p.slab, n_tok - t0);
    const int stages = int(ceil_div(rows, p.kse));
    const int64_t cols = int64_t(stages) * p.kse;
    const dim3 tg(unsigned(ceil_div(cols, 64)), unsigned(ceil_div(p.dp, 64)));
    if (dtype == OPTIMA_DTYPE_BF16) {
      hipLaunchKernelGGL(k_transpose<uint16_t>, tg, dim3(kThreads), 0, s,
                         static_cast<const uint16_t*>(X), d, t0, rows, p.slab, p.dp,
                         reinterpret_cast<uint16_t*>(XT));
    } else {
      hipLaunchKernelGGL(k_transpose<float>, tg, dim3(kThreads), 0, s,
                         static_cast<const float*>(X), d, t0, rows, p.slab, p.dp,
                         reinterpret_cast<float*>(XT));
    }
    OPTIMA_LAUNCH_CHECK();
    const dim3 sg(unsigned(p.tiles * p.splits));
    const int64_t pitch = p.slab * p.esz;
    if (dtype == OPTIMA_DTYPE_BF16) {
      hipLaunchKernelGGL(k_syrk<Bf16Tag>, sg, dim3(kThreads), 0, s, XT, pitch, stages, p.splits,
                         p.dp, part, first);
    } else {
      hipLaunchKernelGGL(k_syrk<float>, sg, dim3(kThreads), 0, s, XT, pitch, stages, p.splits,
                         p.dp, part, first);
    }
    OPTIMA_LAUNCH_CHECK();
    first = 0;
  }
  return reduce_partials(part, p.splits, p.dp, d, H, accumulate, s);
}

optima_status hessian_jacobi(float* H, int64_t d, float* D, hipStream_t s) {
  hipLaunchKernelGGL(k_jacobi_d, dim3(unsigned(ceil_div(d, kThreads))), dim3(kThreads), 0, s, H, d,
                     D);
  OPTIMA_LAUNCH_CHECK();
  const int64_t blocks = std::min<int64_t>(8192, ceil_div(d * d, kThreads));
  hipLaunchKernelGGL(k_jacobi_scale, dim3(unsigned(blocks)), dim3(kThreads), 0, s, H, d, D);
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

optima_status hessian_damp(float* H, int64_t d, float rel, float* lambda_out, hipStream_t s) {
  hipLaunchKernelGGL(k_damp, dim3(1), dim3(1024), 0, s, H, d, rel, lambda_out);
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

}  // namespace optima
