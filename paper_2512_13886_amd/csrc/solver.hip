// Batched column-QP solve (Eq. (6)) by restarted accelerated PDHG on gfx950.
//
// Per column j the state is x (two ping-pong buffers: the H-product reads one
// while the fused update writes the other), the average x_ag, and the
// maintained products Hx = H x, Hx_ag = H x_ag, Hw0 = H w0. All are fp32
// [n_cols][dp] with dp = d rounded up to the 128-wide tile; padding entries
// are zero and stay zero (they behave as pruned). With the products kept,
// one iteration needs a single product with H:
//   update   g = 2((1-a) Hx_ag + a Hx - Hw0), x' = sel(m, x - eta g, 0),
//            x_ag' = (1-a) x_ag + a x'
//   product  Hx' = H x', Hx_ag' = (1-a) Hx_ag + a Hx'
// (H x_md = (1-a) Hx_ag + a Hx by linearity, so the gradient needs no second
// product). The product kernel runs the next iteration's update in its
// epilogue, element by element, so between checks each iteration is one
// launch. Columns that terminate leave the active list; the products then run
// over the active rows only.
//
// Solves whose iteration products run on the 2:4-sparse MFMA pack every
// per-column vector after the initial check. Group g (columns 4g..4g+3) has
// two stored positions p0 < p1, its kept columns padded with the lowest
// pruned ones; slot 2g + t holds the entry at position p_t. An iteration
// never needs the entries at pruned positions: x and x_ag are zero there and
// the gradient there is discarded. So the update moves half the bytes. A
// slot whose position is pruned holds x = x_ag = +0 throughout. The checks
// take f on the kept entries as
//   f(x) = f(x0) + (x - x0)^T (H x + H x0 - 2 H w0)
// (x - x0 vanishes off the kept set), with g0 = H x0 - H w0 packed into the
// second half of Hx_ag's row.
#include <atomic>

#include "common.h"
#include "readback.h"
#include "gemm_core.h"

namespace optima {
namespace {

// kPlainAdd: out1 = H x + out2 (the setup product H w0 = H x0 + H p of a
// sparse solve, p = w0 - x0 the pruned part).
enum GemmMode { kPlain = 0, kPlain2 = 1, kStore = 2, kFused = 3, kPlainAdd = 4 };
// kPrecSparse: bf16x3 with the multiplied vectors stored 2:4-compressed (the
// iteration products of a solve whose mask keeps at most 2 of every 4).
enum Prec { kPrecF32 = OPTIMA_PREC_FP32, kPrecBf16x3 = OPTIMA_PREC_BF16X3, kPrecSparse = 2 };

struct ProductArgs {
  const float* A;      // rows of the multiplied vectors, pitch dp
  const float* B;      // H, [dp][dp] (pitch dp)
  const int* rows;     // active list (row r of the launch is column rows[r]); NULL = identity
  int n_rows;
  int dp;
  int d;
  float* out1;         // kPlain/kPlain2/kPlainAdd: destination; kStore: Hx
  float* out2;         // kPlain2: second destination; kPlainAdd: the addend
  float* HA;           // Hx_ag (kStore, kFused)
  const float* HW0;    // kFused
  const float* Xin;    // kFused: x of the current iteration (same as A)
  float* Xout;         // kFused: x of the next iteration
  float* XA;           // kFused: x_ag
  const uint8_t* mask; // [n_cols][d]
  const int* kbase;    // iterations since restart, per column, at the last check
  int s;               // iterations since the last check before this product
  const float* Lp;     // step constant L
  const uint16_t* Ap;  // kPrecBf16x3: split planes of A (same rows as A);
                       // kPrecSparse: their 2:4-compressed form
  const uint16_t* Aidx;  // kPrecSparse: index words of the compressed rows
  const uint16_t* AidxS;  // the same for rows 0..n_rows-1 of this product, stage-major
                          // (k_idx_stage_major): the 2:4 tile kernel reads these
  int idx_pitch;          // rows per stage of AidxS
  const uint16_t* Bp;  // kPrecBf16x3, kPrecSparse: split planes of H
  uint16_t* XoutP;     // kFused: split (or compressed) planes of the next x
  const uint8_t* slot; // kPrecSparse: stored positions and keep flags per group (slot_code)
};

struct RowCoef {
  float alpha, alpha1, eta1;
};

template <int MODE>
__device__ inline RowCoef row_coef(const ProductArgs& p, int j, float L) {
  RowCoef c{0.f, 0.f, 0.f};
  if (MODE == kFused || MODE == kStore) {
    const float k = float(p.kbase[j] + p.s);
    c.alpha = 2.f / (k + 2.f);
    c.alpha1 = 2.f / (k + 3.f);
    c.eta1 = (k + 2.f) / (2.f * L);
  }
  return c;
}

__device__ inline float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ inline void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ inline float2 ld2(const float* p) { return *reinterpret_cast<const float2*>(p); }
__device__ inline void st2(float* p, float2 v) { *reinterpret_cast<float2*>(p) = v; }

// Keep flags of columns n..n+3 (n a multiple of 4) of mask row j.
__device__ inline void mask4(const uint8_t* mask, int d, int j, int n, bool (&keep)[4]) {
  const uint8_t* m = mask + size_t(j) * d + n;
  if ((d & 3) == 0 && n + 3 < d) {
    const uchar4 v = *reinterpret_cast<const uchar4*>(m);
    keep[0] = v.x != 0;
    keep[1] = v.y != 0;
    keep[2] = v.z != 0;
    keep[3] = v.w != 0;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) keep[e] = n + e < d && m[e] != 0;
  }
}

// Split planes of 4 consecutive values at column n (a multiple of 4) of a
// plane-layout row: two 8-byte stores.
__device__ inline void store_split4(uint16_t* row_planes, int n, const float (&v)[4]) {
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hi[e] = bf16_rne_bits(v[e]);
    lo[e] = bf16_rne_bits(v[e] - bf16_bits_value(hi[e]));
  }
  uint16_t* b = row_planes + (n >> 5) * 64 + (n & 31);
  *reinterpret_cast<uint2*>(b) = make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16));
  *reinterpret_cast<uint2*>(b + 32) = make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16));
}

// 2:4-compressed storage of a group of 4 (the layout of the sparse product):
// the group is stored at two positions p0 < p1, its kept positions padded
// with the lowest free ones. kSparsePairs packs p0 | p1 << 2 for each 4-bit
// keep pattern (patterns keeping 3 or 4 never reach a sparse solve).
constexpr uint64_t sparse_pair_table() {
  uint64_t t = 0;
  for (int k = 0; k < 16; ++k) {
    int q[2] = {0, 0}, c = 0;
    for (int e = 0; e < 4; ++e)
      if (((k >> e) & 1) && c < 2) q[c++] = e;
    for (int e = 0; e < 4; ++e)
      if (!((k >> e) & 1) && c < 2) q[c++] = e;
    const int p0 = q[0] < q[1] ? q[0] : q[1], p1 = q[0] < q[1] ? q[1] : q[0];
    t |= uint64_t(p0 | (p1 << 2)) << (4 * k);
  }
  return t;
}
constexpr uint64_t kSparsePairs = sparse_pair_table();

__device__ inline uint32_t sparse_pair_code(const bool (&keep)[4]) {
  const int k = int(keep[0]) | (int(keep[1]) << 1) | (int(keep[2]) << 2) | (int(keep[3]) << 3);
  return uint32_t(kSparsePairs >> (4 * k)) & 15u;
}

// Slot code of a group: its stored positions p0 < p1 and whether each is
// kept, packed as p0 | p1 << 2 | kept(p0) << 4 | kept(p1) << 5.
struct SlotCode {
  int p0, p1;
  bool k0, k1;
};
__device__ inline uint32_t slot_code_bits(const bool (&keep)[4]) {
  const uint32_t code = sparse_pair_code(keep);
  const int p0 = int(code & 3u), p1 = int(code >> 2);
  bool k0 = keep[0], k1 = keep[0];
#pragma unroll
  for (int e = 1; e < 4; ++e) {
    k0 = e == p0 ? keep[e] : k0;
    k1 = e == p1 ? keep[e] : k1;
  }
  return code | (uint32_t(k0) << 4) | (uint32_t(k1) << 5);
}
__device__ inline SlotCode slot_code(uint32_t c) {
  return SlotCode{int(c & 3u), int((c >> 2) & 3u), (c & 16u) != 0, (c & 32u) != 0};
}
// The values at positions p0 and p1 of a group of 4.
__device__ inline float2 pick_pair(const float (&v)[4], const SlotCode& c) {
  float a = v[0], b = v[0];
#pragma unroll
  for (int e = 1; e < 4; ++e) {
    a = e == c.p0 ? v[e] : a;
    b = e == c.p1 ? v[e] : b;
  }
  return make_float2(a, b);
}

// Compressed planes of group g of a row (dp / 2 stored values per plane,
// 2 dp bytes per row; per 64 columns 32 hi values, then 32 lo): the values a
// and b at its two stored positions, hi and lo.
__device__ inline void store_pair_planes(uint16_t* row, int g, float a, float b) {
  const uint32_t ha = bf16_rne_bits(a), hb = bf16_rne_bits(b);
  const uint32_t la = bf16_rne_bits(a - bf16_bits_value(ha)), lb = bf16_rne_bits(b - bf16_bits_value(hb));
  uint16_t* blk = row + (g >> 4) * 64 + (g & 15) * 2;
  *reinterpret_cast<uint32_t*>(blk) = ha | (hb << 16);
  *reinterpret_cast<uint32_t*>(blk + 32) = la | (lb << 16);
}

// What the packed update of the group at column n (a multiple of 4) of
// column j reads besides the product: its slot code and the packed state.
// Kernels that know j before their product is done load it early.
struct PackedIn {
  uint32_t code;
  float2 ha, hw, xi, xa;
};
template <int MODE>
__device__ inline PackedIn load_packed(const ProductArgs& p, int j, int n) {
  PackedIn in{};
  const int g = n >> 2;
  const size_t o = size_t(j) * p.dp + 2 * g;
  in.code = p.slot[size_t(j) * (p.dp >> 2) + g];
  in.ha = ld2(p.HA + o);
  if (MODE == kFused) {
    in.hw = ld2(p.HW0 + o);
    in.xi = ld2(p.Xin + o);
    in.xa = ld2(p.XA + o);
  }
  return in;
}

// Stores that other workgroups of the same cooperative launch read: relaxed
// agent-scope atomics (sc1), which the L2s of all XCDs see without the cache
// write-back and invalidation that a release/acquire fence costs.
__device__ inline void store_u32_agent(void* q, uint32_t v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(q), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void store_f4_agent(float* q, float4 v) {
  uint64_t* w = reinterpret_cast<uint64_t*>(q);
  __hip_atomic_store(w, (uint64_t(__float_as_uint(v.y)) << 32) | __float_as_uint(v.x),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(w + 1, (uint64_t(__float_as_uint(v.w)) << 32) | __float_as_uint(v.z),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Loads of what other workgroups of the launch wrote (the same scope).
__device__ inline uint4 load_u4_agent(const void* q) {
  const uint64_t* w = reinterpret_cast<const uint64_t*>(q);
  const uint64_t a = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t b = __hip_atomic_load(w + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_uint4(uint32_t(a), uint32_t(a >> 32), uint32_t(b), uint32_t(b >> 32));
}

// Consumes y = (H x)[j][n..n+3] for column j (n a multiple of 4); the
// iteration products of a sparse solve update the packed vectors. COHERENT:
// the planes of the next x are stored with agent-scope atomics (the
// cooperative few-column launch, where every workgroup reads them).
template <int MODE, bool COHERENT = false>
__device__ inline void finish_packed(const ProductArgs& p, int j, int n, float4 y4,
                                     const RowCoef& c, const PackedIn& in) {
  const int g = n >> 2;
  const size_t o = size_t(j) * p.dp + 2 * g;
  const SlotCode sc = slot_code(in.code);
  const float yv[4] = {y4.x, y4.y, y4.z, y4.w};
  const float2 y2 = pick_pair(yv, sc);
  const float y[2] = {y2.x, y2.y};
  const bool keep[2] = {sc.k0, sc.k1};
  const float hav[2] = {in.ha.x, in.ha.y};
  if (MODE == kStore) {
    float ha[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) ha[e] = (1.f - c.alpha) * hav[e] + c.alpha * y[e];
    st2(p.HA + o, make_float2(ha[0], ha[1]));
    st2(p.out1 + o, y2);
  } else {
    const float hwv[2] = {in.hw.x, in.hw.y};
    const float xiv[2] = {in.xi.x, in.xi.y}, xav[2] = {in.xa.x, in.xa.y};
    float ha[2], xn[2], xa[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      ha[e] = (1.f - c.alpha) * hav[e] + c.alpha * y[e];
      const float gr = 2.f * ((1.f - c.alpha1) * ha[e] + c.alpha1 * y[e] - hwv[e]);
      xn[e] = keep[e] ? xiv[e] - c.eta1 * gr : 0.f;
      xa[e] = (1.f - c.alpha1) * xav[e] + c.alpha1 * xn[e];
    }
    st2(p.XA + o, make_float2(xa[0], xa[1]));
    st2(p.HA + o, make_float2(ha[0], ha[1]));
    st2(p.Xout + o, make_float2(xn[0], xn[1]));
    if (COHERENT) {
      const uint32_t ha_ = bf16_rne_bits(xn[0]), hb_ = bf16_rne_bits(xn[1]);
      const uint32_t la_ = bf16_rne_bits(xn[0] - bf16_bits_value(ha_));
      const uint32_t lb_ = bf16_rne_bits(xn[1] - bf16_bits_value(hb_));
      uint16_t* blk = p.XoutP + size_t(j) * p.dp + (g >> 4) * 64 + (g & 15) * 2;
      store_u32_agent(blk, ha_ | (hb_ << 16));
      store_u32_agent(blk + 32, la_ | (lb_ << 16));
    } else {
      store_pair_planes(p.XoutP + size_t(j) * p.dp, g, xn[0], xn[1]);
    }
  }
}

template <int MODE>
__device__ inline void epilogue_packed(const ProductArgs& p, int j, int n, float4 y4,
                                       const RowCoef& c) {
  finish_packed<MODE>(p, j, n, y4, c, load_packed<MODE>(p, j, n));
}

// What the dense update of columns n..n+3 (n a multiple of 4) of column j
// reads besides the product (kStore, kFused).
struct Dense4In {
  float4 ha, hw, xi, xa;
  bool keep[4];
};
template <int MODE>
__device__ inline Dense4In load_dense4(const ProductArgs& p, int j, int n) {
  Dense4In in{};
  const size_t o = size_t(j) * p.dp + n;
  in.ha = ld4(p.HA + o);
  if (MODE == kFused) {
    in.hw = ld4(p.HW0 + o);
    in.xi = ld4(p.Xin + o);
    in.xa = ld4(p.XA + o);
    mask4(p.mask, p.d, j, n, in.keep);
  }
  return in;
}

// The dense update of columns n..n+3 of column j from y = (H x)[j][n..n+3].
// COHERENT: the next x is stored with agent-scope atomics (the cooperative
// few-column launch, where every workgroup reads it).
template <int MODE, int PREC, bool COHERENT = false>
__device__ inline void finish_dense4(const ProductArgs& p, int j, int n, float4 y4,
                                     const RowCoef& c, const Dense4In& in) {
  const size_t o = size_t(j) * p.dp + n;
  if (MODE == kStore) {
    float4 ha = in.ha;
    ha.x = (1.f - c.alpha) * ha.x + c.alpha * y4.x;
    ha.y = (1.f - c.alpha) * ha.y + c.alpha * y4.y;
    ha.z = (1.f - c.alpha) * ha.z + c.alpha * y4.z;
    ha.w = (1.f - c.alpha) * ha.w + c.alpha * y4.w;
    st4(p.HA + o, ha);
    st4(p.out1 + o, y4);
  } else {  // kFused: finish this iteration's products, run the next update
    const float y[4] = {y4.x, y4.y, y4.z, y4.w};
    const float hav[4] = {in.ha.x, in.ha.y, in.ha.z, in.ha.w};
    const float hwv[4] = {in.hw.x, in.hw.y, in.hw.z, in.hw.w};
    const float xiv[4] = {in.xi.x, in.xi.y, in.xi.z, in.xi.w};
    const float xav[4] = {in.xa.x, in.xa.y, in.xa.z, in.xa.w};
    float ha[4], xn[4], xa[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ha[e] = (1.f - c.alpha) * hav[e] + c.alpha * y[e];
      const float g = 2.f * ((1.f - c.alpha1) * ha[e] + c.alpha1 * y[e] - hwv[e]);
      xn[e] = in.keep[e] ? xiv[e] - c.eta1 * g : 0.f;
      xa[e] = (1.f - c.alpha1) * xav[e] + c.alpha1 * xn[e];
    }
    st4(p.XA + o, make_float4(xa[0], xa[1], xa[2], xa[3]));
    st4(p.HA + o, make_float4(ha[0], ha[1], ha[2], ha[3]));
    if (COHERENT)
      store_f4_agent(p.Xout + o, make_float4(xn[0], xn[1], xn[2], xn[3]));
    else
      st4(p.Xout + o, make_float4(xn[0], xn[1], xn[2], xn[3]));
    if (PREC == kPrecBf16x3) store_split4(p.XoutP + size_t(j) * p.dp * 2, n, xn);
  }
}

template <int MODE, int PREC>
__device__ inline void epilogue4(const ProductArgs& p, int j, int n, float4 y4, const RowCoef& c) {
  if (PREC == kPrecSparse && (MODE == kFused || MODE == kStore)) {
    epilogue_packed<MODE>(p, j, n, y4, c);
    return;
  }
  const size_t o = size_t(j) * p.dp + n;
  if (MODE == kPlain) {
    st4(p.out1 + o, y4);
  } else if (MODE == kPlain2) {
    st4(p.out1 + o, y4);
    st4(p.out2 + o, y4);
  } else if (MODE == kPlainAdd) {
    const float4 a = ld4(p.out2 + o);
    st4(p.out1 + o, make_float4(a.x + y4.x, a.y + y4.y, a.z + y4.z, a.w + y4.w));
  } else {
    finish_dense4<MODE, PREC>(p, j, n, y4, c, load_dense4<MODE>(p, j, n));
  }
}

// The products of `splits` contiguous K ranges of one output tile; with
// splits == 1 the tile is finished in place, otherwise each range writes its
// partial sum to part[split][launch row][n] and k_split_epilogue adds them.
// The accumulators pass through LDS so that the epilogue works on 16-byte
// chunks of 4 consecutive columns (full-width loads and stores).
// Four waves per workgroup and 64 KiB of LDS let two workgroups share a CU,
// so one workgroup's memory-bound fused update overlaps the other's MFMA main
// loop (eight-wave tiles that fill a CU alone leave that update exposed).
using ProductTile = Tile128;

template <int MODE, int PREC>
__global__ void __launch_bounds__(ProductTile::kThreads) k_product(ProductArgs p, int splits,
                                                                   float* part) {
  using Cfg = ProductTile;
  __shared__ __attribute__((aligned(1024))) char lds0[Cfg::kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[Cfg::kBufBytes];
  const int tiles_m = (p.n_rows + kTile - 1) / kTile;
  const int tiles_n = p.dp / kTile;
  const int n_tiles = tiles_m * tiles_n;
  const int lin = blockIdx.x % n_tiles;
  const int sp = blockIdx.x / n_tiles;
  int tm, tn;
  tile_of_block(lin, n_tiles, tiles_m, tiles_n, &tm, &tn);
  const int m0 = tm * kTile, n0 = tn * kTile;
  const int stages = p.dp * 4 / Cfg::SRB;
  const int s0 = int(int64_t(stages) * sp / splits);
  const int s1 = int(int64_t(stages) * (sp + 1) / splits);

  Operands<Cfg> src;
  const size_t k_off = size_t(s0) * Cfg::SRB;
  // Both layouts take 4 dp bytes per row.
  const char* a_base = PREC == kPrecBf16x3 ? reinterpret_cast<const char*>(p.Ap)
                                           : reinterpret_cast<const char*>(p.A);
  const char* b_base = PREC == kPrecBf16x3 ? reinterpret_cast<const char*>(p.Bp)
                                           : reinterpret_cast<const char*>(p.B);
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsA; ++i) {
    int r = m0 + load_row<Cfg>(i);
    r = r < p.n_rows ? r : p.n_rows - 1;
    const int j = p.rows ? p.rows[r] : r;
    src.a[i] = a_base + size_t(j) * p.dp * 4 + k_off + load_seg_bytes<Cfg>(i);
  }
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsB; ++i)
    src.b[i] = b_base + size_t(n0 + load_row<Cfg>(i)) * p.dp * 4 + k_off + load_seg_bytes<Cfg>(i);
  f4 acc[Cfg::MB][Cfg::NB];
  if (PREC == kPrecBf16x3)
    gemm_tile_mainloop<Cfg, Bf16x3Tag>(acc, src, s1 - s0, lds0, lds1, nullptr);
  else
    gemm_tile_mainloop<Cfg, float>(acc, src, s1 - s0, lds0, lds1, nullptr);

  stage_tile<Cfg>(acc, lds0, lds1);
  __syncthreads();
  const float L = (MODE == kFused || MODE == kStore) ? *p.Lp : 0.f;
  float* P = part + size_t(sp) * size_t(tiles_m) * kTile * size_t(p.dp);
#pragma unroll 4
  for (int q = 0; q < kTile * kTile / 4 / Cfg::kThreads; ++q) {
    const int c = threadIdx.x + Cfg::kThreads * q;  // 16-byte chunk of the tile
    const int r = c >> 5, ch = c & 31;
    const int rg = m0 + r;
    if (rg >= p.n_rows) continue;
    const float4 y = staged_chunk(lds0, lds1, r, ch);
    const int n = n0 + 4 * ch;
    if (splits > 1) {
      st4(P + size_t(rg) * p.dp + n, y);
      continue;
    }
    const int j = p.rows ? p.rows[rg] : rg;
    epilogue4<MODE, PREC>(p, j, n, y, row_coef<MODE>(p, j, L));
  }
}

// The dense products on 256 x 128 tiles of 8 waves, one workgroup per CU,
// for long contractions or large batches (wide_tile_path): a quarter fewer
// operand bytes per flop than the 128 x 128 tile, whose loads from L2 bound
// it there. Three
// 48 KiB stage buffers keep two stages loading during each stage's MFMAs.
// The 128 KiB accumulator tile is staged for the epilogue through them (see
// wide_stage_row). Split ranges, partial sums and the epilogue work as in
// k_product, with partial rows padded to the 256-row tile.
using WideTile = TileCfg<256, 128, 4, 2, 3>;
constexpr int kWideMinDim = 8192;    // with batches of at least kWideMinRows columns
constexpr int kWideMinRows = 256;
constexpr int kWideMidDim = 4096;    // with batches of at least kWideMidRows columns
constexpr int kWideMidRows = 4096;

// Where the wide tile beats the 128 x 128 tile, whose two workgroups per CU
// overlap one's update epilogue with the other's main loop. At d = 4096 the
// two tie at 4096 columns; the wide tile is 7 % faster over the 7600 to
// 14336 columns of the gate/up solves and 8 % slower at 1024.
inline bool wide_tile_path(int64_t dp, int64_t n_rows) {
  return (dp >= kWideMinDim && n_rows >= kWideMinRows) ||
         (dp >= kWideMidDim && n_rows >= kWideMidRows);
}

// Epilogue staging of the wide tile's 256 x 128 fp32 accumulators: tile rows
// 32 q .. 32 q + 31 take 16 KiB region q, the (q / 3)-th 16 KiB of buffer
// q % 3, 512 bytes per row; 16-byte column chunk c of row r sits at physical
// chunk c ^ (r & 31), which keeps the MFMA-layout writes and the row-chunk
// reads free of bank conflicts.
__device__ inline char* wide_stage_row(char* lds0, char* lds1, char* lds2, int r) {
  const int q = r >> 5;
  char* buf = q % 3 == 0 ? lds0 : (q % 3 == 1 ? lds1 : lds2);
  return buf + (q / 3) * 16384 + (r & 31) * 512;
}
__device__ inline void wide_stage_tile(const f4 (&acc)[WideTile::MB][WideTile::NB], char* lds0,
                                       char* lds1, char* lds2) {
  static_assert(WideTile::BM == 256 && WideTile::BN == 128, "staging covers 256 x 128 tiles");
  static_assert(WideTile::kBufBytes >= 3 * 16384, "three 16 KiB regions per stage buffer");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WideTile::WGN, wn = wave % WideTile::WGN;
#pragma unroll
  for (int mi = 0; mi < WideTile::MB; ++mi)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = wm * WideTile::MB * 16 + mi * 16 + 4 * (lane >> 4) + e;
      char* row = wide_stage_row(lds0, lds1, lds2, r);
#pragma unroll
      for (int ni = 0; ni < WideTile::NB; ++ni) {
        const int col = wn * WideTile::NB * 16 + ni * 16 + (lane & 15);
        *reinterpret_cast<float*>(row + ((col >> 2) ^ (r & 31)) * 16 + (col & 3) * 4) =
            acc[mi][ni][e];
      }
    }
}

template <int MODE, int PREC>
__global__ void __launch_bounds__(WideTile::kThreads) k_product_wide(ProductArgs p, int splits,
                                                                     float* part) {
  using Cfg = WideTile;
  static_assert(Cfg::NBUF == 3, "three stage buffers");
  __shared__ __attribute__((aligned(1024))) char lds0[Cfg::kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[Cfg::kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds2[Cfg::kBufBytes];
  const int tiles_m = (p.n_rows + Cfg::BM - 1) / Cfg::BM;
  const int tiles_n = p.dp / Cfg::BN;
  const int n_tiles = tiles_m * tiles_n;
  const int lin = blockIdx.x % n_tiles;
  const int sp = blockIdx.x / n_tiles;
  int tm, tn;
  tile_of_block(lin, n_tiles, tiles_m, tiles_n, &tm, &tn);
  const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
  const int stages = p.dp * 4 / Cfg::SRB;
  const int s0 = int(int64_t(stages) * sp / splits);
  const int s1 = int(int64_t(stages) * (sp + 1) / splits);

  Operands<Cfg> src;
  const size_t k_off = size_t(s0) * Cfg::SRB;
  const char* a_base = PREC == kPrecBf16x3 ? reinterpret_cast<const char*>(p.Ap)
                                           : reinterpret_cast<const char*>(p.A);
  const char* b_base = PREC == kPrecBf16x3 ? reinterpret_cast<const char*>(p.Bp)
                                           : reinterpret_cast<const char*>(p.B);
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsA; ++i) {
    int r = m0 + load_row<Cfg>(i);
    r = r < p.n_rows ? r : p.n_rows - 1;
    const int j = p.rows ? p.rows[r] : r;
    src.a[i] = a_base + size_t(j) * p.dp * 4 + k_off + load_seg_bytes<Cfg>(i);
  }
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsB; ++i)
    src.b[i] = b_base + size_t(n0 + load_row<Cfg>(i)) * p.dp * 4 + k_off + load_seg_bytes<Cfg>(i);
  f4 acc[Cfg::MB][Cfg::NB];
  if (PREC == kPrecBf16x3)
    gemm_tile_mainloop<Cfg, Bf16x3Tag>(acc, src, s1 - s0, lds0, lds1, lds2);
  else
    gemm_tile_mainloop<Cfg, float>(acc, src, s1 - s0, lds0, lds1, lds2);

  wide_stage_tile(acc, lds0, lds1, lds2);
  __syncthreads();
  const float L = (MODE == kFused || MODE == kStore) ? *p.Lp : 0.f;
  float* P = part + size_t(sp) * size_t(tiles_m) * Cfg::BM * size_t(p.dp);
  constexpr int kChunks = Cfg::BM * Cfg::BN / 4;
#pragma unroll 4
  for (int q = 0; q < kChunks / Cfg::kThreads; ++q) {
    const int c = threadIdx.x + Cfg::kThreads * q;  // 16-byte chunk of the tile
    const int r = c >> 5, ch = c & 31;
    const int rg = m0 + r;
    if (rg >= p.n_rows) continue;
    const float4 y = *reinterpret_cast<const float4*>(wide_stage_row(lds0, lds1, lds2, r) +
                                                       ((ch ^ (r & 31)) * 16));
    const int n = n0 + 4 * ch;
    if (splits > 1) {
      st4(P + size_t(rg) * p.dp + n, y);
      continue;
    }
    const int j = p.rows ? p.rows[rg] : rg;
    epilogue4<MODE, PREC>(p, j, n, y, row_coef<MODE>(p, j, L));
  }
}

#ifdef OPTIMA_PHASE_STAMPS
// Instrumented builds only (build.py phases): clock stamps (the 100 MHz
// counter of wall_clock64) of the phases of the two kernels that run the
// iteration products of a sparse solve, read back by optima_phase_stamps.
// Each workgroup of k_product_sparse records its start, the end of its main
// loop and its end; four workgroups of k_few_persistent record each
// iteration's start, the end of its product, of the reduction, of the update
// and of the barrier. Thread 0 writes them with ordinary stores.
constexpr int kTileStampSlots = 1 << 16;
constexpr int kCoopStampBlocks = 4, kCoopStampIters = 256;
__device__ uint64_t g_tile_stamps[kTileStampSlots][4];
__device__ unsigned g_tile_stamp_count;
__device__ uint64_t g_coop_stamps[kCoopStampBlocks][kCoopStampIters][6];

__device__ inline void tile_stamp(uint64_t t0, uint64_t t1, int mode, int n_rows) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint64_t t2 = wall_clock64();
    const unsigned slot = atomicAdd(&g_tile_stamp_count, 1u);
    if (slot < unsigned(kTileStampSlots)) {
      g_tile_stamps[slot][0] = t0;
      g_tile_stamps[slot][1] = t1;
      g_tile_stamps[slot][2] = t2;
      g_tile_stamps[slot][3] = uint64_t(blockIdx.x) | (uint64_t(mode) << 32) |
                               (uint64_t(n_rows) << 40);
    }
  }
}
__device__ inline int coop_stamp_block() {
  const unsigned b = blockIdx.x, n = gridDim.x;
  return b == 0 ? 0 : b == n / 3 ? 1 : b == 2 * n / 3 ? 2 : b == n - 1 ? 3 : -1;
}
#endif

// The iteration products with x 2:4-compressed (kPrecSparse): 256 x 128
// tiles of 8 waves on the sparse MFMA, one workgroup per CU (132 KiB of
// LDS). Split ranges, partial sums and the epilogue work as in k_product,
// with partial rows padded to the 256-row tile.
template <int MODE>
__global__ void __launch_bounds__(SpTile::kThreads) k_product_sparse(ProductArgs p, int splits,
                                                                     float* part) {
  __shared__ __attribute__((aligned(1024))) char lds0[SpTile::kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[SpTile::kBufBytes];
  const int tiles_m = (p.n_rows + SpTile::BM - 1) / SpTile::BM;
  const int tiles_n = p.dp / SpTile::BN;
  const int n_tiles = tiles_m * tiles_n;
  const int lin = blockIdx.x % n_tiles;
  const int sp = blockIdx.x / n_tiles;
  int tm, tn;
  tile_of_block(lin, n_tiles, tiles_m, tiles_n, &tm, &tn);
  const int m0 = tm * SpTile::BM, n0 = tn * SpTile::BN;
  const int stages = p.dp / SpTile::kKPerStage;
  const int s0 = int(int64_t(stages) * sp / splits);
  const int s1 = int(int64_t(stages) * (sp + 1) / splits);

  auto col_of = [&](int r) {
    r = m0 + r;
    r = r < p.n_rows ? r : p.n_rows - 1;
    return p.rows ? p.rows[r] : r;
  };
  SpOperands src;
  const char* ap = reinterpret_cast<const char*>(p.Ap);
#pragma unroll
  for (int i = 0; i < SpTile::kLoadsA; ++i)
    src.a[i] = ap + size_t(col_of(sp_a_row(i))) * p.dp * 2 + size_t(s0) * SpTile::kARowBytes +
               sp_a_seg_bytes(i);
#pragma unroll
  for (int i = 0; i < SpTile::kLoadsB; ++i)
    src.b[i] = reinterpret_cast<const char*>(p.Bp) + size_t(n0 + sp_b_row(i)) * p.dp * 4 +
               size_t(s0) * SpTile::kBRowBytes + sp_b_seg_bytes(i);
  src.ai = reinterpret_cast<const char*>(p.AidxS) +
           (size_t(s0) * size_t(p.idx_pitch) + size_t(m0 + sp_idx_row())) * 8 + sp_idx_bytes();
  src.ai_stage = int64_t(p.idx_pitch) * 8;
  f4 acc[SpTile::MB][SpTile::NB];
#ifdef OPTIMA_PHASE_STAMPS
  const uint64_t stamp0 = wall_clock64();
#endif
  gemm_sparse_mainloop(acc, src, s1 - s0, lds0, lds1);
#ifdef OPTIMA_PHASE_STAMPS
  const uint64_t stamp1 = wall_clock64();
#endif

  sp_stage_tile(acc, lds0, lds1);
  __syncthreads();
  const float L = (MODE == kFused || MODE == kStore) ? *p.Lp : 0.f;
  float* P = part + size_t(sp) * size_t(tiles_m) * SpTile::BM * size_t(p.dp);
  constexpr int kChunks = SpTile::BM * SpTile::BN / 4;
#pragma unroll 4
  for (int q = 0; q < kChunks / SpTile::kThreads; ++q) {
    const int c = threadIdx.x + SpTile::kThreads * q;  // 16-byte chunk of the tile
    const int r = c >> 5, ch = c & 31;
    const int rg = m0 + r;
    if (rg >= p.n_rows) continue;
    const float4 y = sp_staged_chunk(lds0, lds1, r, ch);
    const int n = n0 + 4 * ch;
    if (splits > 1) {
      st4(P + size_t(rg) * p.dp + n, y);
      continue;
    }
    const int j = p.rows ? p.rows[rg] : rg;
    epilogue4<MODE, kPrecSparse>(p, j, n, y, row_coef<MODE>(p, j, L));
  }
#ifdef OPTIMA_PHASE_STAMPS
  tile_stamp(stamp0, stamp1, MODE, p.n_rows);
#endif
}

// The iteration products when at most kSkinnyRows columns are still active
// (the last columns of a paper-mode solve). H is streamed once from HBM as
// its split planes: each workgroup takes 16 rows and its 8 waves split the
// contraction into 8 ranges. A wave computes the 16 x 16 block (active
// vectors padded to 16) x (H rows) over its range on
// v_mfma_f32_16x16x32_bf16 as hi*hi + hi*lo + lo*hi, the bf16x3 products of
// the MFMA tiles; it splits the active vectors' fp32 values into hi =
// rne(v) and lo = rne(v - hi) as it loads them. Loads of 8 K steps are in
// flight at a time. The eight partial blocks are added in wave order, then
// the product epilogue runs with the solve's plane layout. fp32 solves keep
// the fp32 MFMA tiles.
constexpr int kSkinnyRows = 8;
constexpr int kSkinnyHRows = 16;     // H rows per workgroup
constexpr int kSkinnyWaves = 8;      // contraction ranges per workgroup
constexpr int kSkinnyBatch = 8;      // K steps of 32 whose loads are in flight together

__device__ inline uint32_t split_pair_hi(float a, float b, uint32_t& lo) {
  const uint32_t ha = bf16_rne_bits(a), hb = bf16_rne_bits(b);
  const uint32_t la = bf16_rne_bits(a - bf16_bits_value(ha));
  const uint32_t lb = bf16_rne_bits(b - bf16_bits_value(hb));
  lo = la | (lb << 16);
  return ha | (hb << 16);
}

// hi and lo bf16 planes of 8 consecutive fp32 values.
__device__ inline void split8(float4 v0, float4 v1, bf16x8& hi, bf16x8& lo) {
  uint4 h, l;
  h.x = split_pair_hi(v0.x, v0.y, l.x);
  h.y = split_pair_hi(v0.z, v0.w, l.y);
  h.z = split_pair_hi(v1.x, v1.y, l.z);
  h.w = split_pair_hi(v1.z, v1.w, l.w);
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

template <int MODE, int PREC>
__global__ void __launch_bounds__(64 * kSkinnyWaves) k_product_skinny(ProductArgs p) {
  static_assert(PREC == kPrecBf16x3, "split-plane bf16x3 products only");
  __shared__ float red[kSkinnyWaves][kSkinnyHRows][kSkinnyHRows + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kSkinnyHRows;
  const int nr = p.n_rows;
  const int r = lane & 15, g = lane >> 4;
  // This lane's A row (active vector r; lanes of rows r >= nr read column
  // rows[0] and zero what they read) and B row (the planes of H row n0 + r:
  // per 32 columns 64 bytes of hi, then of lo).
  const bool has_x = r < nr;
  const float* xrow = p.A + size_t(p.rows ? p.rows[has_x ? r : 0] : (has_x ? r : 0)) * p.dp;
  const char* hrow = reinterpret_cast<const char*>(p.Bp) + size_t(n0 + r) * p.dp * 4 + 16 * g;
  // The update's inputs do not depend on the product: their loads go out
  // first and land while H streams in.
  const int t = threadIdx.x;
  const bool upd = t < 4 * nr;
  const int jv = upd ? (p.rows ? p.rows[t >> 2] : (t >> 2)) : 0;
  const int nv = n0 + 4 * (t & 3);
  Dense4In din{};
  if (upd) din = load_dense4<MODE>(p, jv, nv);
  const RowCoef cv = upd ? row_coef<MODE>(p, jv, *p.Lp) : RowCoef{};
  const int steps = p.dp / 32, per = steps / kSkinnyWaves;  // dp % 256 == 0
  const int s0 = wave * per, s1 = s0 + per;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  auto mma = [&](uint4 bh4, uint4 bl4, float4 x0, float4 x1) {
    bf16x8 ah, al;
    split8(x0, x1, ah, al);
    if (!has_x) ah = al = bf16x8{};
    const bf16x8 bh = __builtin_bit_cast(bf16x8, bh4), bl = __builtin_bit_cast(bf16x8, bl4);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
  };
  int st = s0;
  for (; st + kSkinnyBatch <= s1; st += kSkinnyBatch) {
    uint4 hh[kSkinnyBatch], hl[kSkinnyBatch];
    float4 xv[kSkinnyBatch][2];
#pragma unroll
    for (int b = 0; b < kSkinnyBatch; ++b) {
      hh[b] = *reinterpret_cast<const uint4*>(hrow + size_t(st + b) * 128);
      hl[b] = *reinterpret_cast<const uint4*>(hrow + size_t(st + b) * 128 + 64);
      const int k = (st + b) * 32 + 8 * g;
      xv[b][0] = ld4(xrow + k);
      xv[b][1] = ld4(xrow + k + 4);
    }
    // Keep the scheduler from sinking the loads toward their uses: all of
    // the batch's loads go out before the first MFMA waits for data.
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int b = 0; b < kSkinnyBatch; ++b) mma(hh[b], hl[b], xv[b][0], xv[b][1]);
  }
  for (; st < s1; ++st) {
    const int k = st * 32 + 8 * g;
    mma(*reinterpret_cast<const uint4*>(hrow + size_t(st) * 128),
        *reinterpret_cast<const uint4*>(hrow + size_t(st) * 128 + 64), ld4(xrow + k),
        ld4(xrow + k + 4));
  }
  // Output (lane, e): vector 4 g + e, H row n0 + r (the dense 16 x 16 layout).
#pragma unroll
  for (int e = 0; e < 4; ++e) red[wave][4 * g + e][r] = acc[e];
  __syncthreads();
  if (upd) {
    const int v = t >> 2, q = t & 3;
    float y[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float a = red[0][v][4 * q + e];
#pragma unroll
      for (int w = 1; w < kSkinnyWaves; ++w) a += red[w][v][4 * q + e];
      y[e] = a;
    }
    finish_dense4<MODE, PREC>(p, jv, nv, make_float4(y[0], y[1], y[2], y[3]), cv, din);
  }
}

// The same for sparse solves: the A operand is x's compressed planes and
// index words, as in k_product_sparse, on v_smfmac_f32_16x16x64_bf16 (hi*hi,
// hi*lo, lo*hi), one 64-column step per instruction. Each lane reads its 16
// bytes of hi and of lo (the 8 stored values of columns 16 g .. 16 g + 15
// of its vector), its 2-byte index word, and H's hi and lo planes of
// columns 8 g .. 8 g + 7 and 32 + 8 g .. 32 + 8 g + 7. The 8 waves take
// contiguous step ranges of near-equal length.
constexpr int kSkinnySparseBatch = 4;  // 64-column steps whose loads are in flight together

template <int MODE>
__global__ void __launch_bounds__(64 * kSkinnyWaves) k_product_skinny_sparse(ProductArgs p) {
  __shared__ float red[kSkinnyWaves][kSkinnyHRows][kSkinnyHRows + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kSkinnyHRows;
  const int nr = p.n_rows;
  const int r = lane & 15, g = lane >> 4;
  const bool has_x = r < nr;
  const int jx = p.rows ? p.rows[has_x ? r : 0] : (has_x ? r : 0);
  // Per 64 columns: x's planes take 128 bytes (64 hi, 64 lo), its index
  // words 8 bytes, H's planes 256 bytes (hi, lo of the first 32 columns,
  // then of the next 32).
  const char* arow = reinterpret_cast<const char*>(p.Ap) + size_t(jx) * p.dp * 2 + 16 * g;
  const char* irow = reinterpret_cast<const char*>(p.Aidx) + size_t(jx) * (p.dp / 8) + 2 * g;
  const char* hrow = reinterpret_cast<const char*>(p.Bp) + size_t(n0 + r) * p.dp * 4 + 16 * g;
  // The update's inputs do not depend on the product: their loads go out
  // first and land while H streams in.
  const int t = threadIdx.x;
  const bool upd = t < 4 * nr;
  const int jv = upd ? (p.rows ? p.rows[t >> 2] : (t >> 2)) : 0;
  const int nv = n0 + 4 * (t & 3);
  PackedIn pin{};
  if (upd) pin = load_packed<MODE>(p, jv, nv);
  const RowCoef cv = upd ? row_coef<MODE>(p, jv, *p.Lp) : RowCoef{};
  const int steps = p.dp / 64;
  const int s0 = steps * wave / kSkinnyWaves, s1 = steps * (wave + 1) / kSkinnyWaves;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  auto mma = [&](uint4 ah4, uint4 al4, int ix, uint4 h0, uint4 l0, uint4 h1, uint4 l1) {
    bf16x8 ah = __builtin_bit_cast(bf16x8, ah4), al = __builtin_bit_cast(bf16x8, al4);
    if (!has_x) ah = al = bf16x8{};
    const bf16x16 bh = sp_b_pair(__builtin_bit_cast(bf16x8, h0), __builtin_bit_cast(bf16x8, h1));
    const bf16x16 bl = sp_b_pair(__builtin_bit_cast(bf16x8, l0), __builtin_bit_cast(bf16x8, l1));
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(ah, bh, acc, ix, 0, 0);
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(ah, bl, acc, ix, 0, 0);
    acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(al, bh, acc, ix, 0, 0);
  };
  auto ld16 = [](const char* q) { return *reinterpret_cast<const uint4*>(q); };
  int st = s0;
  for (; st + kSkinnySparseBatch <= s1; st += kSkinnySparseBatch) {
    uint4 ah[kSkinnySparseBatch], al[kSkinnySparseBatch], h0[kSkinnySparseBatch],
        l0[kSkinnySparseBatch], h1[kSkinnySparseBatch], l1[kSkinnySparseBatch];
    int ix[kSkinnySparseBatch];
#pragma unroll
    for (int b = 0; b < kSkinnySparseBatch; ++b) {
      const char* a = arow + size_t(st + b) * 128;
      const char* h = hrow + size_t(st + b) * 256;
      ah[b] = ld16(a);
      al[b] = ld16(a + 64);
      ix[b] = *reinterpret_cast<const uint16_t*>(irow + size_t(st + b) * 8);
      h0[b] = ld16(h);
      l0[b] = ld16(h + 64);
      h1[b] = ld16(h + 128);
      l1[b] = ld16(h + 192);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int b = 0; b < kSkinnySparseBatch; ++b) mma(ah[b], al[b], ix[b], h0[b], l0[b], h1[b], l1[b]);
  }
  for (; st < s1; ++st) {
    const char* a = arow + size_t(st) * 128;
    const char* h = hrow + size_t(st) * 256;
    mma(ld16(a), ld16(a + 64), *reinterpret_cast<const uint16_t*>(irow + size_t(st) * 8), ld16(h),
        ld16(h + 64), ld16(h + 128), ld16(h + 192));
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) red[wave][4 * g + e][r] = acc[e];
  __syncthreads();
  if (upd) {
    const int v = t >> 2, q = t & 3;
    float y[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float a = red[0][v][4 * q + e];
#pragma unroll
      for (int w = 1; w < kSkinnyWaves; ++w) a += red[w][v][4 * q + e];
      y[e] = a;
    }
    finish_packed<MODE>(p, jv, nv, make_float4(y[0], y[1], y[2], y[3]), cv, pin);
  }
}

// All iterations of a block (the iterations between two checks) with at most
// kSkinnyRows active columns in one cooperative launch. Each workgroup owns
// the 16 rows of H that the few-column kernels give it, and keeps their
// split planes in registers for the whole block (16 rows x 4 dp bytes over
// 512 lanes: 128 registers a lane at dp = 4096), so H is read from HBM once
// per block instead of once per iteration. An iteration is the few-column
// product (the same instructions and summation order as
// k_product_skinny[_sparse]) and its update epilogue; the workgroups then
// meet at a grid barrier before the next iteration reads the x just written.
// The barrier's arrival counters live in the solver workspace; a wait that
// exceeds kBarrierPolls sets a flag that the host turns into an error, so
// every wave always reaches the end of the kernel.
constexpr int kPersistMaxDp = 4096;
constexpr int kPersistBatch = 4;  // steps whose x loads are in flight together
constexpr unsigned kBarrierPolls = 1u << 20;
constexpr int kDirectScopeSc1 = 16;  // cache-policy bits of an agent-scope (sc1) buffer access
constexpr int kXsPitch = 2 * kPersistMaxDp + 16;  // LDS bytes per staged x row (sparse)
// Arrival counters of the grid barrier: kBarGroups group counters and one
// top counter, kBarStride words (128 bytes) apart. Four groups measured
// fastest: one counter for all 256 workgroups made every arrival wait its
// turn at one address (4.0 us a barrier against 2.4 us).
constexpr int kBarGroups = 4;
constexpr int kBarStride = 32;
constexpr int kBarWords = (kBarGroups + 1) * kBarStride;

struct PersistArgs {
  ProductArgs p;      // rows, n_rows, dp, d, HA, HW0, XA, mask, kbase, Lp, Bp, Aidx, slot, out1
  float* X[2];        // x of the iterations, ping-pong
  uint16_t* XP[2];    // their split (or compressed) planes
  uint32_t x_bytes;   // bytes of each X[] and XP[] buffer the launch may address (< 2^31)
  int cur;            // index of the first iteration's x
  int n_iter;         // iterations of the block; the last one stores H x in out1
  unsigned* arrivals; // kBarWords words, zero at the launch (grid_arrive)
  int* timeout;       // set to 1 when a barrier wait gives up
};

// Grid barrier k (k = 1, 2, ...) of the cooperative launch, in two halves so
// that loads the next iteration needs can go out between them. Everything
// that crosses workgroups (the next x) is written and read with agent-scope
// accesses, so the barrier only has to order them: each thread's stores are
// complete (vmcnt) before its workgroup arrives.
//
// Arrival: workgroup b adds 1 to the counter of group b % G (G = min(4,
// gridDim.x)); the counters only grow, so group g is complete for barrier k
// at k times its size, and the workgroup whose add completes it adds 1 to
// the top counter. Every workgroup reaches barrier k before any leaves it,
// so no add of barrier k + 1 can be counted early. A workgroup leaves once
// the top counter reaches k G. A wait that runs out of polls raises the
// time-out flag; from then on every barrier of the launch returns at once,
// so the launch ends quickly and the host reports the error.
__device__ inline void grid_arrive(unsigned* bar, unsigned k, int* timeout) {
  wait_vmcnt<0>();
  __syncthreads();
  if (threadIdx.x == 0 &&
      __hip_atomic_load(timeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
    const unsigned G = min(unsigned(kBarGroups), gridDim.x);
    const unsigned grp = blockIdx.x % G;
    const unsigned size = gridDim.x / G + (grp < gridDim.x % G ? 1u : 0u);
    const unsigned old = __hip_atomic_fetch_add(bar + grp * kBarStride, 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1u == k * size)
      __hip_atomic_fetch_add(bar + kBarGroups * kBarStride, 1u, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}
__device__ inline void grid_wait(const unsigned* bar, unsigned k, int* timeout) {
  if (threadIdx.x == 0 &&
      __hip_atomic_load(timeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
    const unsigned* top = bar + kBarGroups * kBarStride;
    const unsigned target = k * min(unsigned(kBarGroups), gridDim.x);
    unsigned seen = __hip_atomic_load(top, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    unsigned polls = 0;
    while (seen < target) {
      if (++polls >= kBarrierPolls ||
          __hip_atomic_load(timeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
        __hip_atomic_store(timeout, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      seen = __hip_atomic_load(top, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
}

// Raw buffer over `bytes` from `base`; loads through it with the sc1 policy
// are agent-scope (see store_u32_agent), 16 bytes at a time.
__device__ inline __amdgpu_buffer_rsrc_t agent_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), 0x00020000);
}
__device__ inline uint4 load16_agent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, kDirectScopeSc1);
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <int PREC>
__global__ void __launch_bounds__(64 * kSkinnyWaves) k_few_persistent(PersistArgs a) {
  constexpr bool kSparse = PREC == kPrecSparse;
  constexpr int kStepCols = kSparse ? 64 : 32;         // contraction columns per step
  constexpr int kMaxSteps = kPersistMaxDp / kStepCols / kSkinnyWaves;  // per wave
  constexpr int kHVec = kSparse ? 4 : 2;               // 16-byte H pieces per step
  __shared__ float red[kSkinnyWaves][kSkinnyHRows][kSkinnyHRows + 1];
  // Sparse: the compressed planes of the active x rows, staged once per
  // iteration (rows kXsPitch bytes apart, which keeps the fragment reads of
  // 16 rows on distinct banks).
  __shared__ __attribute__((aligned(16))) char xs[kSparse ? kSkinnyRows * kXsPitch : 16];
  // Sparse: the active rows' index words (dp / 8 bytes each), constant for
  // the launch, copied once.
  __shared__ __attribute__((aligned(16))) uint32_t ids[kSparse ? kSkinnyRows * kPersistMaxDp / 32 : 4];
  ProductArgs p = a.p;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kSkinnyHRows;
  const int nr = p.n_rows;
  const int r = lane & 15, g = lane >> 4;
  const bool has_x = r < nr;
  const int jx = p.rows ? p.rows[has_x ? r : 0] : (has_x ? r : 0);
  const int t = threadIdx.x;
  const bool upd = t < 4 * nr;
  const int jv = upd ? (p.rows ? p.rows[t >> 2] : (t >> 2)) : 0;
  const int nv = n0 + 4 * (t & 3);
  const int steps = p.dp / kStepCols;
  const int s0 = steps * wave / kSkinnyWaves, s1 = steps * (wave + 1) / kSkinnyWaves;

  // This lane's pieces of H row n0 + r for the wave's steps.
  const char* hrow = reinterpret_cast<const char*>(p.Bp) + size_t(n0 + r) * p.dp * 4 + 16 * g;
  uint4 hreg[kMaxSteps][kHVec];
#pragma unroll
  for (int k = 0; k < kMaxSteps; ++k)
#pragma unroll
    for (int v = 0; v < kHVec; ++v)
      hreg[k][v] = s0 + k < s1 ? *reinterpret_cast<const uint4*>(
                                     hrow + size_t(s0 + k) * (kStepCols * 4) + 64 * v)
                               : make_uint4(0u, 0u, 0u, 0u);

  if constexpr (kSparse) {
    const int words = p.dp / 32;  // 4-byte words of one row's index words
    for (int e = threadIdx.x; e < nr * words; e += blockDim.x) {
      const int k = e / words, w = e - k * words;
      const int jk = p.rows ? p.rows[k] : k;
      ids[k * (kPersistMaxDp / 32) + w] =
          reinterpret_cast<const uint32_t*>(p.Aidx)[size_t(jk) * words + w];
    }
    __syncthreads();
  }
  const float L = *p.Lp;
  int cur = a.cur;
  p.Xin = a.X[cur];
  PackedIn pin{};
  Dense4In din{};
  if (upd) {
    if constexpr (kSparse) pin = load_packed<kFused>(p, jv, nv);
    else din = load_dense4<kFused>(p, jv, nv);
  }
#ifdef OPTIMA_PHASE_STAMPS
  const int stamp_b = coop_stamp_block();
  uint64_t st[6];
#endif
  for (int i = 0; i < a.n_iter; ++i) {
    const bool last = i == a.n_iter - 1;
#ifdef OPTIMA_PHASE_STAMPS
    st[0] = wall_clock64();
#endif
    p.s = i;
    p.Xin = a.X[cur];
    p.Xout = a.X[cur ^ 1];
    p.XoutP = a.XP[cur ^ 1];
    const RowCoef cv = upd ? row_coef<kFused>(p, jv, L) : RowCoef{};
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (kSparse) {
      // The active rows' planes (dp * 2 bytes each) into LDS by agent-scope
      // direct loads, all in flight at once: wave w fetches the w-th KiB of
      // every row, lanes past the row's end fetch its last 16 bytes again.
      const int row_bytes = p.dp * 2;
      const int off = min(wave * 1024 + lane * 16, row_bytes - 16);
      const char* xplanes = reinterpret_cast<const char*>(a.XP[cur]);
      for (int k = 0; k < nr; ++k) {
        const int jk = p.rows ? p.rows[k] : k;
        __builtin_amdgcn_global_load_lds(
            (const __attribute__((address_space(1))) void*)(xplanes + size_t(jk) * row_bytes + off),
            (__attribute__((address_space(3))) void*)(xs + k * kXsPitch + wave * 1024), 16, 0,
            kDirectScopeSc1);
      }
      wait_vmcnt<0>();
      __syncthreads();
      const char* xrow = xs + (has_x ? r : 0) * kXsPitch + 16 * g;
      const char* irow = reinterpret_cast<const char*>(ids) + (has_x ? r : 0) * (kPersistMaxDp / 8) + 2 * g;
#pragma unroll
      for (int b = 0; b < kMaxSteps; b += kPersistBatch) {
        uint4 ah[kPersistBatch], al[kPersistBatch];
        int ix[kPersistBatch];
#pragma unroll
        for (int k = 0; k < kPersistBatch; ++k) {
          if (s0 + b + k < s1) {
            const char* q = xrow + (s0 + b + k) * 128;
            ah[k] = *reinterpret_cast<const uint4*>(q);
            al[k] = *reinterpret_cast<const uint4*>(q + 64);
            ix[k] = *reinterpret_cast<const uint16_t*>(irow + (s0 + b + k) * 8);
          }
        }
#pragma unroll
        for (int k = 0; k < kPersistBatch; ++k) {
          if (s0 + b + k < s1) {
            bf16x8 xh = __builtin_bit_cast(bf16x8, ah[k]), xl = __builtin_bit_cast(bf16x8, al[k]);
            if (!has_x) xh = xl = bf16x8{};
            const bf16x16 bh = sp_b_pair(__builtin_bit_cast(bf16x8, hreg[b + k][0]),
                                         __builtin_bit_cast(bf16x8, hreg[b + k][2]));
            const bf16x16 bl = sp_b_pair(__builtin_bit_cast(bf16x8, hreg[b + k][1]),
                                         __builtin_bit_cast(bf16x8, hreg[b + k][3]));
            acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(xh, bh, acc, ix[k], 0, 0);
            acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(xh, bl, acc, ix[k], 0, 0);
            acc = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(xl, bh, acc, ix[k], 0, 0);
          }
        }
      }
    } else {
      const __amdgpu_buffer_rsrc_t xr = agent_rsrc(a.X[cur], a.x_bytes);
      const uint32_t xrow = uint32_t(jx) * uint32_t(p.dp) * 4u + 32u * g;
#pragma unroll
      for (int b = 0; b < kMaxSteps; b += kPersistBatch) {
        uint4 x0[kPersistBatch], x1[kPersistBatch];
#pragma unroll
        for (int k = 0; k < kPersistBatch; ++k) {
          if (s0 + b + k < s1) {
            const uint32_t q = xrow + uint32_t(s0 + b + k) * 128u;
            x0[k] = load16_agent(xr, q);
            x1[k] = load16_agent(xr, q + 16u);
          }
        }
#pragma unroll
        for (int k = 0; k < kPersistBatch; ++k) {
          if (s0 + b + k < s1) {
            bf16x8 xh, xl;
            split8(make_float4(__uint_as_float(x0[k].x), __uint_as_float(x0[k].y),
                               __uint_as_float(x0[k].z), __uint_as_float(x0[k].w)),
                   make_float4(__uint_as_float(x1[k].x), __uint_as_float(x1[k].y),
                               __uint_as_float(x1[k].z), __uint_as_float(x1[k].w)),
                   xh, xl);
            if (!has_x) xh = xl = bf16x8{};
            const bf16x8 bh = __builtin_bit_cast(bf16x8, hreg[b + k][0]);
            const bf16x8 bl = __builtin_bit_cast(bf16x8, hreg[b + k][1]);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, bh, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, bl, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl, bh, acc, 0, 0, 0);
          }
        }
      }
    }
#ifdef OPTIMA_PHASE_STAMPS
    st[1] = wall_clock64();
#endif
#pragma unroll
    for (int e = 0; e < 4; ++e) red[wave][4 * g + e][r] = acc[e];
    __syncthreads();
#ifdef OPTIMA_PHASE_STAMPS
    st[2] = wall_clock64();
#endif
    if (upd) {
      const int v = t >> 2, q = t & 3;
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float sum = red[0][v][4 * q + e];
#pragma unroll
        for (int w = 1; w < kSkinnyWaves; ++w) sum += red[w][v][4 * q + e];
        y[e] = sum;
      }
      const float4 y4 = make_float4(y[0], y[1], y[2], y[3]);
      if constexpr (kSparse) {
        if (last)
          finish_packed<kStore>(p, jv, nv, y4, cv, pin);
        else
          finish_packed<kFused, true>(p, jv, nv, y4, cv, pin);
      } else {
        if (last)
          finish_dense4<kStore, kPrecBf16x3>(p, jv, nv, y4, cv, din);
        else
          finish_dense4<kFused, kPrecBf16x3, true>(p, jv, nv, y4, cv, din);
      }
    }
    if (!last) {
      // The next iteration's update inputs are this thread's own stores of
      // this iteration: their loads go out while the barrier waits.
      cur ^= 1;
      p.Xin = a.X[cur];
#ifdef OPTIMA_PHASE_STAMPS
      st[3] = wall_clock64();
#endif
      grid_arrive(a.arrivals, unsigned(i + 1), a.timeout);
      if (upd) {
        if constexpr (kSparse) pin = load_packed<kFused>(p, jv, nv);
        else din = load_dense4<kFused>(p, jv, nv);
      }
      grid_wait(a.arrivals, unsigned(i + 1), a.timeout);
#ifdef OPTIMA_PHASE_STAMPS
      st[4] = wall_clock64();
      if (stamp_b >= 0 && threadIdx.x == 0 && i < kCoopStampIters) {
        for (int e = 0; e < 5; ++e) g_coop_stamps[stamp_b][i][e] = st[e];
        g_coop_stamps[stamp_b][i][5] = uint64_t(a.n_iter);
      }
#endif
    }
  }
}

// Sums the split partials in split order and applies the product epilogue.
template <int MODE, int PREC>
__global__ void __launch_bounds__(kThreads) k_split_epilogue(ProductArgs p, int splits,
                                                             int rows_pad, const float* part) {
  const int r = blockIdx.x;
  if (r >= p.n_rows) return;
  const int j = p.rows ? p.rows[r] : r;
  const size_t split_stride = size_t(rows_pad) * size_t(p.dp);
  const RowCoef c = row_coef<MODE>(p, j, (MODE == kFused || MODE == kStore) ? *p.Lp : 0.f);
  for (int n = 4 * (blockIdx.y * kThreads + threadIdx.x); n < p.dp; n += 4 * gridDim.y * kThreads) {
    const float* q = part + size_t(r) * p.dp + n;
    float4 y = ld4(q);
    for (int sp = 1; sp < splits; ++sp) {
      const float4 t = ld4(q + sp * split_stride);
      y.x += t.x;
      y.y += t.y;
      y.z += t.z;
      y.w += t.w;
    }
    epilogue4<MODE, PREC>(p, j, n, y, c);
  }
}

// Iteration update from the stored products (first iteration after a check).
// With `sparse` the vectors are packed and slot gives each group's code.
__global__ void __launch_bounds__(kThreads) k_update(const int* rows, int n_rows, int dp, int d,
                                                     const float* X, float* Xout, float* XA,
                                                     const float* HX, const float* HA,
                                                     const float* HW0, const uint8_t* mask,
                                                     const int* kbase, const float* Lp,
                                                     uint16_t* XoutP, int sparse,
                                                     const uint8_t* slot) {
  const int r = blockIdx.x;
  if (r >= n_rows) return;
  const int j = rows ? rows[r] : r;
  const float k = float(kbase[j]);
  const float alpha = 2.f / (k + 2.f);
  const float eta = (k + 1.f) / (2.f * *Lp);
  const size_t base = size_t(j) * dp;
  if (sparse) {
    const int groups = dp / 4;
    for (int g = blockIdx.y * kThreads + threadIdx.x; g < groups; g += gridDim.y * kThreads) {
      const size_t o = base + 2 * g;
      const SlotCode c = slot_code(slot[size_t(j) * groups + g]);
      const float2 ha2 = ld2(HA + o), hx2 = ld2(HX + o), hw2 = ld2(HW0 + o), x2 = ld2(X + o),
                   xa2 = ld2(XA + o);
      const float hav[2] = {ha2.x, ha2.y}, hxv[2] = {hx2.x, hx2.y}, hwv[2] = {hw2.x, hw2.y};
      const float xv[2] = {x2.x, x2.y}, xav[2] = {xa2.x, xa2.y};
      const bool keep[2] = {c.k0, c.k1};
      float xn[2], xa[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float gr = 2.f * ((1.f - alpha) * hav[e] + alpha * hxv[e] - hwv[e]);
        xn[e] = keep[e] ? xv[e] - eta * gr : 0.f;
        xa[e] = (1.f - alpha) * xav[e] + alpha * xn[e];
      }
      st2(XA + o, make_float2(xa[0], xa[1]));
      st2(Xout + o, make_float2(xn[0], xn[1]));
      store_pair_planes(XoutP + base, g, xn[0], xn[1]);
    }
    return;
  }
  for (int n = 4 * (blockIdx.y * kThreads + threadIdx.x); n < dp; n += 4 * gridDim.y * kThreads) {
    const size_t o = base + n;
    const float4 ha4 = ld4(HA + o), hx4 = ld4(HX + o), hw4 = ld4(HW0 + o), x4 = ld4(X + o),
                 xa4 = ld4(XA + o);
    const float hav[4] = {ha4.x, ha4.y, ha4.z, ha4.w}, hxv[4] = {hx4.x, hx4.y, hx4.z, hx4.w};
    const float hwv[4] = {hw4.x, hw4.y, hw4.z, hw4.w}, xv[4] = {x4.x, x4.y, x4.z, x4.w};
    const float xav[4] = {xa4.x, xa4.y, xa4.z, xa4.w};
    bool keep[4];
    mask4(mask, d, j, n, keep);
    float xn[4], xa[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float g = 2.f * ((1.f - alpha) * hav[e] + alpha * hxv[e] - hwv[e]);
      xn[e] = keep[e] ? xv[e] - eta * g : 0.f;
      xa[e] = (1.f - alpha) * xav[e] + alpha * xn[e];
    }
    st4(XA + o, make_float4(xa[0], xa[1], xa[2], xa[3]));
    st4(Xout + o, make_float4(xn[0], xn[1], xn[2], xn[3]));
    if (XoutP) store_split4(XoutP + base * 2, n, xn);
  }
}

// Packs the state of the active columns of a sparse solve after the initial
// check: x (X, in place) and x_ag (XA) from x0, Hx (HX, in place) and Hx_ag
// (HA) from H x0, Hw0 (HW0, in place), and g0 = H x0 - H w0 into the second
// half of HA's row. Slot 2g + t comes from position 4g + p_t >= 2g + t, so
// in place a write never lands beyond its source. Chunks of kThreads groups
// go in order with a barrier between a chunk's reads and its writes: chunk c
// reads positions from 4 kThreads c on and writes slots below
// 2 kThreads (c + 1), so only the chunk's own reads can be overwritten.
__global__ void __launch_bounds__(kThreads) k_pack(const int* rows, int n_rows, int dp,
                                                   const uint8_t* slot, float* X, float* XA,
                                                   float* HX, float* HA, float* HW0) {
  const int r = blockIdx.x;
  if (r >= n_rows) return;
  const int j = rows ? rows[r] : r;
  const size_t base = size_t(j) * dp;
  const int groups = dp / 4;
  for (int c0 = 0; c0 < groups; c0 += kThreads) {
    const int g = c0 + threadIdx.x;
    const bool on = g < groups;
    float2 x = make_float2(0.f, 0.f), hx = x, hw = x;
    if (on) {
      const SlotCode c = slot_code(slot[size_t(j) * groups + g]);
      const float4 x4 = ld4(X + base + 4 * g), h4 = ld4(HX + base + 4 * g),
                   w4 = ld4(HW0 + base + 4 * g);
      const float xv[4] = {x4.x, x4.y, x4.z, x4.w}, hv[4] = {h4.x, h4.y, h4.z, h4.w},
                  wv[4] = {w4.x, w4.y, w4.z, w4.w};
      x = pick_pair(xv, c);
      hx = pick_pair(hv, c);
      hw = pick_pair(wv, c);
    }
    __syncthreads();
    if (on) {
      const size_t o = base + 2 * g;
      st2(X + o, x);
      st2(XA + o, x);
      st2(HX + o, hx);
      st2(HA + o, hx);
      st2(HW0 + o, hw);
      st2(HA + base + dp / 2 + 2 * g, make_float2(hx.x - hw.x, hx.y - hw.y));
    }
  }
}

// Copies W0 into padded rows and forms the start point x = x_ag = sel(m, w0, 0).
// Padded copy of the anchors (divided by the column scaling D when given),
// the start point sel(mask, w0, +0), its average and split planes.
__global__ void __launch_bounds__(kThreads) k_prep(const float* W0, const uint8_t* mask, int n_cols,
                                                   int d, int dp, float* W0P, float* X, float* XA,
                                                   uint16_t* XP, uint16_t* WP,
                                                   const float* scale, int* flags) {
  const int j = blockIdx.x;
  const size_t base = size_t(j) * dp;
  bool bad = false;
  for (int n = blockIdx.y * kThreads + threadIdx.x; n < dp; n += gridDim.y * kThreads) {
    float w = 0.f;
    bool keep = false;
    if (n < d) {
      w = W0[size_t(j) * d + n];
      keep = mask[size_t(j) * d + n] != 0;
      bad |= !isfinite(w);
      if (scale) {
        const float sc = scale[n];
        bad |= !(sc > 0.f) || !isfinite(sc);
        w = w / sc;
      }
    }
    W0P[base + n] = w;
    const float x = keep ? w : 0.f;
    X[base + n] = x;
    XA[base + n] = x;
    if (XP) store_split(XP + base * 2, n, x);
    if (WP) store_split(WP + base * 2, n, w);
  }
  if (bad) atomicOr(flags, 1);
}

// k_prep for a solve that may run on the sparse products, one thread per
// group of 4 columns. k_sparse_index has already set flags[1] and flags[2].
// When both are clear, the setup products run on the sparse kernel and need
// only x0 and the compressed planes of x0 (kept pairs, into XP) and of the
// pruned part p = w0 - x0 (pruned pairs, into WP): nothing else is written.
// Otherwise everything k_prep writes is written.
__global__ void __launch_bounds__(kThreads) k_prep_sparse(const float* W0, const uint8_t* mask,
                                                          int d, int dp, float* W0P, float* X,
                                                          float* XA, uint16_t* XP, uint16_t* WP,
                                                          const float* scale, int* flags) {
  const int j = blockIdx.x;
  const size_t base = size_t(j) * dp;
  const bool compressed = flags[1] == 0 && flags[2] == 0;  // uniform
  bool bad = false;
  for (int g = blockIdx.y * kThreads + threadIdx.x; 4 * g < dp; g += gridDim.y * kThreads) {
    const int n = 4 * g;
    bool keep[4], pruned[4];
    mask4(mask, d, j, n, keep);
    float w[4], x[4], pv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      w[e] = 0.f;
      if (n + e < d) {
        w[e] = W0[size_t(j) * d + n + e];
        bad |= !isfinite(w[e]);
        if (scale) {
          const float sc = scale[n + e];
          bad |= !(sc > 0.f) || !isfinite(sc);
          w[e] = w[e] / sc;
        }
      }
      pruned[e] = !keep[e] && n + e < d;
      x[e] = keep[e] ? w[e] : 0.f;
      pv[e] = pruned[e] ? w[e] : 0.f;
    }
    st4(X + base + n, make_float4(x[0], x[1], x[2], x[3]));
    if (compressed) {
      const uint32_t c0 = sparse_pair_code(keep), c1 = sparse_pair_code(pruned);
      const float2 a = pick_pair(x, SlotCode{int(c0 & 3u), int(c0 >> 2), true, true});
      const float2 b = pick_pair(pv, SlotCode{int(c1 & 3u), int(c1 >> 2), true, true});
      store_pair_planes(XP + base, g, a.x, a.y);
      store_pair_planes(WP + base, g, b.x, b.y);
    } else {
      st4(W0P + base + n, make_float4(w[0], w[1], w[2], w[3]));
      st4(XA + base + n, make_float4(x[0], x[1], x[2], x[3]));
      store_split4(XP + base * 2, n, x);
      store_split4(WP + base * 2, n, w);
    }
  }
  if (bad) atomicOr(flags, 1);
}

// Split planes of H (row pitch 4 dp bytes), built once per solve.
// With `flags`, it also sets flags[0] = 1 if H holds a NaN or Inf (the scan
// of k_scan_pad_h, for an H that needs no padding).
__global__ void __launch_bounds__(kThreads) k_split_h(const float* Hm, int dp, uint16_t* HP,
                                                      int* flags) {
  const int i = blockIdx.x;
  bool bad = false;
  for (int n = blockIdx.y * kThreads + threadIdx.x; n < dp; n += gridDim.y * kThreads) {
    const float v = Hm[size_t(i) * dp + n];
    bad |= !isfinite(v);
    store_split(HP + size_t(i) * dp * 2, n, v);
  }
  if (flags && bad) atomicOr(flags, 1);
}

// Index words of the 2:4-compressed layout, one thread per row, 64-column
// block and lane group (dp / 16 words per row; word w covers columns
// 16 w .. 16 w + 15 of the row), the slot codes of those 4 groups (dp / 4
// bytes per row), and flags[1] = 1 if some group of 4 keeps more than 2
// (the mask then has no compressed form). idx2 gets the index words of the
// pruned columns below d, and flags[2] = 1 if some group prunes more than 2
// of them (the pruned part of w0 then has no compressed form).
__global__ void __launch_bounds__(kThreads) k_sparse_index(const uint8_t* mask, int n_cols, int d,
                                                           int dp, uint16_t* idx, uint8_t* slot,
                                                           uint16_t* idx2, int* flags) {
  const int words = dp / 16;
  const int64_t t = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (t >= int64_t(n_cols) * words) return;
  const int j = int(t / words), w = int(t % words);
  uint32_t word = 0, codes = 0, word2 = 0;
  bool bad = false, bad2 = false;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int n = 16 * w + 4 * q;
    bool keep[4], pruned[4];
    mask4(mask, d, j, n, keep);
#pragma unroll
    for (int e = 0; e < 4; ++e) pruned[e] = !keep[e] && n + e < d;
    bad |= int(keep[0]) + int(keep[1]) + int(keep[2]) + int(keep[3]) > 2;
    bad2 |= int(pruned[0]) + int(pruned[1]) + int(pruned[2]) + int(pruned[3]) > 2;
    word |= sparse_pair_code(keep) << (4 * q);
    codes |= slot_code_bits(keep) << (8 * q);
    word2 |= sparse_pair_code(pruned) << (4 * q);
  }
  idx[size_t(j) * words + w] = uint16_t(word);
  idx2[size_t(j) * words + w] = uint16_t(word2);
  *reinterpret_cast<uint32_t*>(slot + size_t(j) * (dp / 4) + 4 * w) = codes;
  if (bad) atomicOr(flags + 1, 1);
  if (bad2) atomicOr(flags + 2, 1);
}


// Zero-padded copy of H (used when d is not a multiple of the tile) with a
// finiteness scan; with hp == nullptr it only scans.
__global__ void __launch_bounds__(kThreads) k_scan_pad_h(const float* H, int d, int dp, float* hp,
                                                         int* flags) {
  bool bad = false;
  const size_t total = size_t(dp) * dp;
  const size_t stride = size_t(gridDim.x) * kThreads;
  for (size_t e = size_t(blockIdx.x) * kThreads + threadIdx.x; e < total; e += stride) {
    const int i = int(e / dp), jj = int(e % dp);
    float v = 0.f;
    if (i < d && jj < d) {
      v = H[size_t(i) * d + jj];
      bad |= !isfinite(v);
    }
    if (hp) hp[e] = v;
  }
  if (bad) atomicOr(flags, 1);
}

__global__ void k_step_constant(const float* lambda_max, float step_safety, float* Lp, int* flags) {
  const float lm = *lambda_max;
  if (!(lm > 0.f) || !isfinite(lm)) {
    atomicOr(flags, 2);
    *Lp = 1.f;
    return;
  }
  *Lp = float(2.0 * double(lm) * (1.0 + double(step_safety)));
}

struct ColState {
  int* kbase;         // iterations since restart as of the last check
  int* restarts;
  int* done;
  double* kkt_restart;
  double* kkt_prev;
  double* f_anchor;
  double* c_norm;     // ||2 H w0||_2
  double* w0hw0;      // w0^T H w0
  double* f_start;    // f(x0)
};

struct CheckArgs {
  const int* rows;
  int n_rows;
  int dp, d;
  float* X;            // current x
  uint16_t* XP;        // its split planes (kPrecBf16x3), else NULL
  int packed;          // sparse solve after the initial check: packed vectors,
                       // XP holds the 2:4-compressed planes
  const uint8_t* slot; // slot codes (packed)
  float* XA;
  float* HX;
  float* HA;
  const float* HW0;
  const float* W0;     // [n_cols][d]
  const uint8_t* mask;
  const float* scale;  // column scaling D of a preconditioned H, or NULL
  ColState st;
  int n_block;         // iterations run since the last check
  int64_t t;           // total iterations run
  int initial;         // first check at the start point
  int final_check;     // t == max_iters
  optima_solver_opts o;
  float* W_out;
  optima_solve_stats stats;
};

// One workgroup per active column: scores x and x_ag, picks the candidate,
// then terminates the column or applies an accepted restart.
__global__ void __launch_bounds__(kThreads) k_check(CheckArgs a) {
  __shared__ double red[kThreads / 64];
  __shared__ int decision;  // bit 0: terminate, bit 1: restart, bit 2: candidate is x
  const int r = blockIdx.x;
  if (r >= a.n_rows) return;
  const int j = a.rows ? a.rows[r] : r;
  const size_t base = size_t(j) * a.dp;

  // With a column scaling D the iterates live in y = D^-1 w; r_d and ||2 H w0||
  // are taken with the gradient in the original coordinates (divided by D),
  // gap, f and z^T H z are the same in both.
  double rdx = 0, gpx = 0, fx = 0, qx = 0, rda = 0, gpa = 0, fa = 0, qa = 0, cn = 0, wq = 0;
  const int groups = a.dp / 4;
  const uint8_t* sl = a.packed ? a.slot + size_t(j) * groups : nullptr;
  // Packed: sums over the stored slots; f is accumulated as
  // (z - x0)^T (H z - H w0 + g0) and f(x0) is added after the reduction.
  for (int g = threadIdx.x; a.packed && g < groups; g += kThreads) {
    const SlotCode c = slot_code(sl[g]);
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const size_t o = base + 2 * g + t;
      const bool keep = t ? c.k1 : c.k0;
      const int n = 4 * g + (t ? c.p1 : c.p0);
      float x0f = 0.f;
      double inv = 1.0;
      if (keep) {
        x0f = a.W0[size_t(j) * a.d + n];
        if (a.scale) {
          x0f = x0f / a.scale[n];
          inv = 1.0 / double(a.scale[n]);
        }
      }
      const double x0 = x0f, hw = a.HW0[o], g0 = a.HA[base + a.dp / 2 + 2 * g + t];
      const double x = a.X[o], hx = a.HX[o];
      const double gx = 2.0 * (hx - hw);
      rdx += keep ? (gx * inv) * (gx * inv) : 0.0;
      gpx += x * gx;
      fx += (x - x0) * ((hx - hw) + g0);
      qx += x * hx;
      const double xa = a.XA[o], ha = a.HA[o];
      const double ga = 2.0 * (ha - hw);
      rda += keep ? (ga * inv) * (ga * inv) : 0.0;
      gpa += xa * ga;
      fa += (xa - x0) * ((ha - hw) + g0);
      qa += xa * ha;
    }
  }
  for (int n = threadIdx.x; !a.packed && n < a.d; n += kThreads) {
    const size_t o = base + n;
    const double hw = a.HW0[o];
    const double inv = a.scale ? 1.0 / double(a.scale[n]) : 1.0;
    const double w0 = double(a.W0[size_t(j) * a.d + n]) * inv;
    const bool keep = a.mask[size_t(j) * a.d + n] != 0;
    const double x = a.X[o], hx = a.HX[o];
    const double gx = 2.0 * (hx - hw);
    rdx += keep ? (gx * inv) * (gx * inv) : 0.0;
    gpx += x * gx;
    fx += (x - w0) * (hx - hw);
    qx += x * hx;
    if (a.initial) {
      cn += 4.0 * (hw * inv) * (hw * inv);
      wq += w0 * hw;
    } else {
      const double xa = a.XA[o], ha = a.HA[o];
      const double ga = 2.0 * (ha - hw);
      rda += keep ? (ga * inv) * (ga * inv) : 0.0;
      gpa += xa * ga;
      fa += (xa - w0) * (ha - hw);
      qa += xa * ha;
    }
  }
  rdx = block_sum(rdx, red);
  gpx = block_sum(gpx, red);
  fx = block_sum(fx, red);
  qx = block_sum(qx, red);
  if (a.initial) {
    cn = block_sum(cn, red);
    wq = block_sum(wq, red);
  } else {
    rda = block_sum(rda, red);
    gpa = block_sum(gpa, red);
    fa = block_sum(fa, red);
    qa = block_sum(qa, red);
  }

  if (threadIdx.x == 0) {
    const optima_solver_opts& o = a.o;
    const ColState& st = a.st;
    double c_norm, w0hw0;
    if (a.initial) {
      c_norm = sqrt(cn);
      w0hw0 = wq;
      st.c_norm[j] = c_norm;
      st.w0hw0[j] = w0hw0;
    } else {
      c_norm = st.c_norm[j];
      w0hw0 = st.w0hw0[j];
      if (a.packed) {
        fx += st.f_start[j];
        fa += st.f_start[j];
      }
    }
    const double rd_x = sqrt(rdx), gap_x = fabs(gpx), kkt_x = sqrt(rd_x * rd_x + gap_x * gap_x);
    double rd_c = rd_x, gap_c = gap_x, kkt_c = kkt_x, f_c = fx, q_c = qx;
    bool cand_x = true;
    if (!a.initial) {
      const double rd_a = sqrt(rda), gap_a = fabs(gpa), kkt_a = sqrt(rd_a * rd_a + gap_a * gap_a);
      cand_x = kkt_x < kkt_a;  // ties go to the average
      if (!cand_x) {
        rd_c = rd_a;
        gap_c = gap_a;
        kkt_c = kkt_a;
        f_c = fa;
        q_c = qa;
      }
    }
    const double P = f_c, D = -q_c + w0hw0;
    const bool conv = rd_c <= double(o.eps_abs) + double(o.eps_rel) * c_norm &&
                      gap_c <= double(o.eps_abs) + double(o.eps_rel) * (fabs(P) + fabs(D));
    int dec = cand_x ? 4 : 0;
    if (a.initial) {
      if (a.stats.f_initial) a.stats.f_initial[j] = float(fx);
      st.f_start[j] = fx;
      st.kkt_restart[j] = kkt_x;
      st.kkt_prev[j] = kkt_x;
      st.f_anchor[j] = fx;
      st.kbase[j] = 0;
      st.restarts[j] = 0;
      if ((conv && !o.fixed_iters) || a.final_check) dec |= 1;
    } else {
      const bool stop = (conv && !o.fixed_iters) || a.final_check;
      if (stop) {
        dec |= 1;
      } else {
        const double k = double(st.kbase[j] + a.n_block);
        const bool cond = kkt_c <= double(o.beta_sufficient) * st.kkt_restart[j] ||
                          (kkt_c <= double(o.beta_necessary) * st.kkt_restart[j] &&
                           kkt_c > st.kkt_prev[j]) ||
                          k >= double(o.beta_artificial) * double(a.t);
        if (o.restarts && cond && f_c <= st.f_anchor[j]) {
          dec |= 2;
          st.kbase[j] = 0;
          st.kkt_restart[j] = kkt_c;
          st.f_anchor[j] = f_c;
          st.restarts[j] += 1;
        } else {
          st.kbase[j] = int(k);
        }
        st.kkt_prev[j] = kkt_c;
      }
    }
    if (dec & 1) {
      st.done[j] = 1;
      if (a.stats.iters) a.stats.iters[j] = int(a.t);
      if (a.stats.restarts) a.stats.restarts[j] = st.restarts[j];
      if (a.stats.converged) a.stats.converged[j] = conv ? 1 : 0;
      if (a.stats.f_final) a.stats.f_final[j] = float(f_c);
      if (a.stats.kkt_final) a.stats.kkt_final[j] = float(kkt_c);
    }
    decision = dec;
  }
  __syncthreads();
  const int dec = decision;
  if (dec & 1) {
    const float* src = (dec & 4) ? a.X : a.XA;
    for (int n = threadIdx.x; n < a.d; n += kThreads) {
      float v;
      if (a.packed) {  // +0 at pruned positions
        const SlotCode c = slot_code(sl[n >> 2]);
        const int e = n & 3;
        v = c.k0 && e == c.p0 ? src[base + 2 * (n >> 2)]
            : c.k1 && e == c.p1 ? src[base + 2 * (n >> 2) + 1]
                                : 0.f;
      } else {
        v = src[base + n];
      }
      a.W_out[size_t(j) * a.d + n] = a.scale ? v * a.scale[n] : v;
    }
  } else if (dec & 2) {
    float* xd = (dec & 4) ? a.XA : a.X;
    float* hd = (dec & 4) ? a.HA : a.HX;
    const float* xs = (dec & 4) ? a.X : a.XA;
    const float* hs = (dec & 4) ? a.HX : a.HA;
    const int len = a.packed ? a.dp / 2 : a.dp;
    for (int n = threadIdx.x; n < len; n += kThreads) {
      xd[base + n] = xs[base + n];
      hd[base + n] = hs[base + n];
      if (!(dec & 4) && a.XP && !a.packed) store_split(a.XP + base * 2, n, xs[base + n]);
    }
    if (!(dec & 4) && a.XP && a.packed)
      for (int g = threadIdx.x; g < groups; g += kThreads)
        store_pair_planes(a.XP + base, g, xs[base + 2 * g], xs[base + 2 * g + 1]);
  }
}

// ---------------------------------------------------------------------------
// Conjugate gradients on the unconstrained form (OPTIMA_METHOD_CG)
// ---------------------------------------------------------------------------
// With the pruned entries fixed at zero, Eq. (6) is unconstrained in the kept
// entries K and its optimum solves H_KK x_K = (H w0)_K (Eq. (11) written for
// w). Per column: r = P (H w0 - H x0), p = r; each iteration q = H p (one
// batched product), alpha = r.r / p.q_K, x += alpha p, r -= alpha q_K,
// beta = r'.r' / r.r, p = r' + beta p. Entries outside K stay exactly 0 in
// x, r and p. Buffers: x = X0, r = XA, p = X1 (split planes XP0), q = HA,
// r.r per column in st.kkt_prev (fp64).
struct CgArgs {
  const int* rows;
  int n_rows;
  int dp, d;
  float* X;
  float* R;
  float* P;
  uint16_t* PP;      // split planes of p (kPrecBf16x3), else NULL
  const float* Q;    // H p
  const float* HX;   // H x0 (initialisation)
  const float* HW0;
  const uint8_t* mask;
  double* rr;
};

__global__ void __launch_bounds__(kThreads) k_cg_init(CgArgs a) {
  __shared__ double red[kThreads / 64];
  const int r = blockIdx.x;
  if (r >= a.n_rows) return;
  const int j = a.rows ? a.rows[r] : r;
  const size_t base = size_t(j) * a.dp;
  double s = 0.0;
  for (int n = threadIdx.x; n < a.dp; n += kThreads) {
    const bool keep = n < a.d && a.mask[size_t(j) * a.d + n] != 0;
    const float v = keep ? a.HW0[base + n] - a.HX[base + n] : 0.f;
    a.R[base + n] = v;
    a.P[base + n] = v;
    if (a.PP) store_split(a.PP + base * 2, n, v);
    s += double(v) * double(v);
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) a.rr[j] = s;
}

// One CG iteration of one active column (one workgroup per column).
__global__ void __launch_bounds__(kThreads) k_cg_step(CgArgs a) {
  __shared__ double red[kThreads / 64];
  const int r = blockIdx.x;
  if (r >= a.n_rows) return;
  const int j = a.rows ? a.rows[r] : r;
  const size_t base = size_t(j) * a.dp;
  const uint8_t* m = a.mask + size_t(j) * a.d;
  double pq = 0.0;
  for (int n = threadIdx.x; n < a.d; n += kThreads)
    if (m[n]) pq += double(a.P[base + n]) * double(a.Q[base + n]);
  pq = block_sum(pq, red);
  const double rr = a.rr[j];
  const float alpha = float(rr > 0.0 && pq > 0.0 ? rr / pq : 0.0);
  double rr2 = 0.0;
  for (int n = threadIdx.x; n < a.d; n += kThreads) {
    if (!m[n]) continue;
    const size_t o = base + n;
    a.X[o] = a.X[o] + alpha * a.P[o];
    const float rn = a.R[o] - alpha * a.Q[o];
    a.R[o] = rn;
    rr2 += double(rn) * double(rn);
  }
  rr2 = block_sum(rr2, red);
  const float beta = float(rr > 0.0 ? rr2 / rr : 0.0);
  for (int n = threadIdx.x; n < a.d; n += kThreads) {
    if (!m[n]) continue;
    const size_t o = base + n;
    const float pn = a.R[o] + beta * a.P[o];
    a.P[o] = pn;
    if (a.PP) store_split(a.PP + base * 2, n, pn);
  }
  if (threadIdx.x == 0) a.rr[j] = rr2;
}

// Termination test of the CG iterate with the rAPDHG rule. With x = 0 off K:
// g_K = -2 r_K, so r_d = 2 ||r_K||, gap = 2 |x.r|, x^T H x = x.Hw0 - x.r and
// f(x) = w0^T H w0 - x.Hw0 - x.r (sums over K).
struct CgCheckArgs {
  const int* rows;
  int n_rows;
  int dp, d;
  const float* X;
  const float* R;
  const float* HW0;
  const uint8_t* mask;
  const float* scale;
  ColState st;
  int64_t t;
  int final_check;
  optima_solver_opts o;
  float* W_out;
  optima_solve_stats stats;
};

__global__ void __launch_bounds__(kThreads) k_cg_check(CgCheckArgs a) {
  __shared__ double red[kThreads / 64];
  __shared__ int stop;
  const int r = blockIdx.x;
  if (r >= a.n_rows) return;
  const int j = a.rows ? a.rows[r] : r;
  const size_t base = size_t(j) * a.dp;
  const uint8_t* m = a.mask + size_t(j) * a.d;
  double rr = 0.0, xr = 0.0, xh = 0.0;
  for (int n = threadIdx.x; n < a.d; n += kThreads) {
    if (!m[n]) continue;
    const double x = a.X[base + n], rv = a.R[base + n];
    const double ro = a.scale ? rv / double(a.scale[n]) : rv;  // original coordinates
    rr += ro * ro;
    xr += x * rv;
    xh += x * double(a.HW0[base + n]);
  }
  rr = block_sum(rr, red);
  xr = block_sum(xr, red);
  xh = block_sum(xh, red);
  if (threadIdx.x == 0) {
    const optima_solver_opts& o = a.o;
    const double rd = 2.0 * sqrt(rr), gap = 2.0 * fabs(xr);
    const double w0hw0 = a.st.w0hw0[j];
    const double f = w0hw0 - xh - xr, D = w0hw0 - (xh - xr);
    const bool conv = rd <= double(o.eps_abs) + double(o.eps_rel) * a.st.c_norm[j] &&
                      gap <= double(o.eps_abs) + double(o.eps_rel) * (fabs(f) + fabs(D));
    const bool st_ = (conv && !o.fixed_iters) || a.final_check;
    if (st_) {
      a.st.done[j] = 1;
      if (a.stats.iters) a.stats.iters[j] = int(a.t);
      if (a.stats.restarts) a.stats.restarts[j] = 0;
      if (a.stats.converged) a.stats.converged[j] = conv ? 1 : 0;
      if (a.stats.f_final) a.stats.f_final[j] = float(f);
      if (a.stats.kkt_final) a.stats.kkt_final[j] = float(sqrt(rd * rd + gap * gap));
    }
    stop = st_ ? 1 : 0;
  }
  __syncthreads();
  if (stop)
    for (int n = threadIdx.x; n < a.d; n += kThreads)
      a.W_out[size_t(j) * a.d + n] = a.scale ? a.X[base + n] * a.scale[n] : a.X[base + n];
}

// Stable compaction of the active list: keeps the columns not yet done.
__global__ void __launch_bounds__(1024) k_compact(const int* rows_in, int n_in, const int* done,
                                                  int* rows_out, int* n_out) {
  __shared__ int scan[1024];
  __shared__ int carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int b = 0; b < n_in; b += 1024) {
    const int r = b + threadIdx.x;
    int j = 0, keep = 0;
    if (r < n_in) {
      j = rows_in ? rows_in[r] : r;
      keep = done[j] ? 0 : 1;
    }
    scan[threadIdx.x] = keep;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
      const int v = threadIdx.x >= o ? scan[threadIdx.x - o] : 0;
      __syncthreads();
      scan[threadIdx.x] += v;
      __syncthreads();
    }
    if (keep) rows_out[carry + scan[threadIdx.x] - 1] = j;
    __syncthreads();
    if (threadIdx.x == 1023) carry += scan[1023];
    __syncthreads();
  }
  if (threadIdx.x == 0) *n_out = carry;
}

// Stage-major copy of the index words that the 2:4 tile product reads for
// rows 0..n_pad-1: entry (s, r), at out + 4 (s pitch + r), holds the 8 bytes
// of stage s of column rows[min(r, n_rows - 1)] (the tile kernel's padded
// rows repeat the last row). One thread per entry, r fastest.
__global__ void __launch_bounds__(kThreads) k_idx_stage_major(const uint16_t* idx, const int* rows,
                                                              int n_rows, int n_pad, int stages,
                                                              int pitch, uint16_t* out) {
  const int64_t e = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (e >= int64_t(stages) * n_pad) return;
  const int st = int(e / n_pad), r = int(e - int64_t(st) * n_pad);
  const int rr = r < n_rows ? r : n_rows - 1;
  const int j = rows ? rows[rr] : rr;
  *reinterpret_cast<uint2*>(out + (size_t(st) * pitch + r) * 4) =
      *reinterpret_cast<const uint2*>(idx + (size_t(j) * stages + st) * 4);
}

// Split-K limits: at most kMaxSplits ranges, and at most kMaxSplitTiles
// (tile, range) pairs, which bounds the partial-sum buffer to 128 MiB.
constexpr int kMaxSplits = 16;
constexpr int kMaxSplitTiles = 2048;

struct Layout {
  int64_t dp;
  bool pad_h;
  size_t part_elems;
  float* part;
  float *X0, *X1, *XA, *HX, *HA, *HW0, *Hp, *L;
  uint16_t *XP0, *XP1, *HP;  // split planes for kPrecBf16x3
  uint16_t* XIDX;            // index words of the 2:4-compressed x planes
  uint16_t* XIDX2;           // index words of the pruned part of w0
  uint16_t* XIDXS;           // stage-major copy for one product's rows (k_idx_stage_major)
  int idx_pitch;             // its rows per stage: n_cols rounded up to the 2:4 tile
  uint8_t* SLOT;             // slot codes of the packed vectors, dp / 4 per column
  int *rows0, *rows1, *n_active, *flags;
  unsigned* bar;             // grid barrier of k_few_persistent: arrival counters
  ColState st;
};

Layout carve(void* ws, int64_t d, int64_t n_cols, size_t* bytes) {
  Layout l{};
  l.dp = round_up(d, kTile);
  l.pad_h = (d % kTile) != 0;
  Carver c(ws);
  const size_t vec = size_t(n_cols) * size_t(l.dp);
  l.X0 = c.take<float>(vec);
  l.X1 = c.take<float>(vec);
  l.XA = c.take<float>(vec);
  l.HX = c.take<float>(vec);
  l.HA = c.take<float>(vec);
  l.HW0 = c.take<float>(vec);
  l.Hp = l.pad_h ? c.take<float>(size_t(l.dp) * size_t(l.dp)) : nullptr;
  l.part_elems = std::min<size_t>(size_t(kMaxSplitTiles) * kTile * kTile,
                                  size_t(kMaxSplits) * size_t(round_up(n_cols, kTile)) * size_t(l.dp));
  l.part = c.take<float>(l.part_elems);
  l.XP0 = c.take<uint16_t>(2 * vec);
  l.XP1 = c.take<uint16_t>(2 * vec);
  l.HP = c.take<uint16_t>(2 * size_t(l.dp) * size_t(l.dp));
  l.XIDX = c.take<uint16_t>(size_t(n_cols) * size_t(l.dp / 16));
  l.XIDX2 = c.take<uint16_t>(size_t(n_cols) * size_t(l.dp / 16));
  l.idx_pitch = int(round_up(n_cols, SpTile::BM));
  l.XIDXS = c.take<uint16_t>(size_t(l.idx_pitch) * size_t(l.dp / 16));
  l.SLOT = c.take<uint8_t>(size_t(n_cols) * size_t(l.dp / 4));
  l.rows0 = c.take<int>(n_cols);
  l.rows1 = c.take<int>(n_cols);
  l.st.kbase = c.take<int>(n_cols);
  l.st.restarts = c.take<int>(n_cols);
  l.st.done = c.take<int>(n_cols);
  l.st.kkt_restart = c.take<double>(n_cols);
  l.st.kkt_prev = c.take<double>(n_cols);
  l.st.f_anchor = c.take<double>(n_cols);
  l.st.c_norm = c.take<double>(n_cols);
  l.st.w0hw0 = c.take<double>(n_cols);
  l.st.f_start = c.take<double>(n_cols);
  l.n_active = c.take<int>(4);
  l.flags = c.take<int>(4);
  l.bar = c.take<unsigned>(kBarWords);
  l.L = c.take<float>(4);
  if (bytes) *bytes = c.bytes();
  return l;
}

// CU count of the current device, queried once per device. Calls from
// several host threads may race to fill an entry; they store the same value.
int device_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Number of K ranges for a product over `tiles` output tiles: splitting pays
// when the tiles leave CUs idle or unevenly loaded. The model counts the
// workgroups the busiest CU runs (relative to its share of the total work),
// rates a CU with a single workgroup at 60% (one wave per SIMD cannot hide
// the stage barriers), and charges 3% per extra range for the partial sums.
int choose_splits(int tiles, int stages, int tiles_m, int dp, size_t part_cap) {
  const int n_cu = device_cu_count();
  if (tiles >= 4 * n_cu) return 1;
  auto cost = [&](int S) {
    const int per_cu = int(ceil_div(int64_t(tiles) * S, n_cu));
    const double eff = per_cu >= 2 ? 1.0 : 0.6;
    return double(per_cu) / S / eff * (1.0 + 0.03 * (S - 1));
  };
  int best = 1;
  double best_cost = cost(1);
  for (int S = 2; S <= kMaxSplits && S <= stages; ++S) {
    if (int64_t(tiles) * S > kMaxSplitTiles) break;
    if (size_t(S) * size_t(tiles_m) * kTile * size_t(dp) > part_cap) break;
    const double c = cost(S);
    if (c < best_cost - 1e-9) {
      best = S;
      best_cost = c;
    }
  }
  return best;
}

// Number of K ranges for a tile that fills a CU with one workgroup: the
// fewest CU rounds per unit of work, charging 5% per extra range for the
// partial sums and their epilogue.
int choose_splits_one_per_cu(int tiles, int stages, int rows_pad, int dp, size_t part_cap) {
  const int n_cu = device_cu_count();
  auto cost = [&](int S) {
    return double(ceil_div(int64_t(tiles) * S, n_cu)) / S * (1.0 + 0.05 * (S - 1));
  };
  int best = 1;
  double best_cost = cost(1);
  for (int S = 2; S <= kMaxSplits && S <= stages; ++S) {
    if (int64_t(tiles) * S > kMaxSplitTiles) break;
    if (size_t(S) * size_t(rows_pad) * size_t(dp) > part_cap) break;
    const double c = cost(S);
    if (c < best_cost - 1e-9) {
      best = S;
      best_cost = c;
    }
  }
  return best;
}

// Whether the iteration products (kFused / kStore) of n_rows active columns
// run the few-column kernels.
bool few_column_path(int prec, int n_rows, int dp) {
  if (n_rows > kSkinnyRows) return false;
  if (prec == kPrecSparse) return true;
  return prec == kPrecBf16x3 && dp % (32 * kSkinnyWaves) == 0;
}

// Whether a block of few-column iterations can run as one cooperative launch
// of k_few_persistent on the current device: cooperative launches are
// supported and all dp / 16 workgroups fit on the device at once. Queried
// once per device and precision.
bool persistent_fits(int prec, int dp) {
  static std::atomic<int> cache[64][2];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
  const int slot = prec == kPrecSparse ? 0 : 1;
  int blocks_per_cu = cache[dev][slot].load(std::memory_order_relaxed);
  if (blocks_per_cu == 0) {
    int coop = 0, n = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess)
      coop = 0;
    hipError_t e = prec == kPrecSparse
                       ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                             &n, k_few_persistent<kPrecSparse>, 64 * kSkinnyWaves, 0)
                       : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                             &n, k_few_persistent<kPrecBf16x3>, 64 * kSkinnyWaves, 0);
    if (e != hipSuccess) (void)hipGetLastError();
    blocks_per_cu = coop && e == hipSuccess && n > 0 ? n : -1;
    cache[dev][slot].store(blocks_per_cu, std::memory_order_relaxed);
  }
  if (blocks_per_cu < 0) return false;
  return int64_t(dp / kSkinnyHRows) <= int64_t(blocks_per_cu) * device_cu_count();
}

bool persistent_path(int prec, int n_rows, int dp) {
  if (!few_column_path(prec, n_rows, dp) || dp > kPersistMaxDp) return false;
  if (prec != kPrecSparse && (prec != kPrecBf16x3 || dp % (32 * kSkinnyWaves) != 0)) return false;
  return persistent_fits(prec, dp);
}

// One cooperative launch for the n iterations of a block; false (nothing
// launched) when the runtime refuses the cooperative launch.
bool launch_persistent(const PersistArgs& a, int prec, hipStream_t s) {
  PersistArgs arg = a;
  void* params[] = {&arg};
  const dim3 grid(unsigned(a.p.dp / kSkinnyHRows)), block(64 * kSkinnyWaves);
  const hipError_t e =
      prec == kPrecSparse
          ? hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&k_few_persistent<kPrecSparse>),
                                       grid, block, params, 0, s)
          : hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&k_few_persistent<kPrecBf16x3>),
                                       grid, block, params, 0, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return true;
}

template <int MODE, int PREC>
optima_status launch_product(const ProductArgs& p, const Layout& l, hipStream_t s) {
  if constexpr ((MODE == kFused || MODE == kStore) && PREC == kPrecSparse) {
    if (few_column_path(PREC, p.n_rows, p.dp)) {
      hipLaunchKernelGGL((k_product_skinny_sparse<MODE>), dim3(unsigned(p.dp / kSkinnyHRows)),
                         dim3(64 * kSkinnyWaves), 0, s, p);
      OPTIMA_LAUNCH_CHECK();
      return OPTIMA_OK;
    }
  }
  if constexpr ((MODE == kFused || MODE == kStore) && PREC == kPrecBf16x3) {
    if (few_column_path(PREC, p.n_rows, p.dp)) {
      hipLaunchKernelGGL((k_product_skinny<MODE, PREC>), dim3(unsigned(p.dp / kSkinnyHRows)),
                         dim3(64 * kSkinnyWaves), 0, s, p);
      OPTIMA_LAUNCH_CHECK();
      return OPTIMA_OK;
    }
  }
  if constexpr (PREC == kPrecBf16x3) {
    if (wide_tile_path(p.dp, p.n_rows)) {
      const int tiles_m = int(ceil_div(p.n_rows, WideTile::BM));
      const int tiles_n = p.dp / WideTile::BN;
      const int rows_pad = tiles_m * WideTile::BM;
      const int S = choose_splits_one_per_cu(tiles_m * tiles_n, p.dp * 4 / WideTile::SRB,
                                             rows_pad, p.dp, l.part_elems);
      hipLaunchKernelGGL((k_product_wide<MODE, PREC>), dim3(tiles_m * tiles_n * S),
                         dim3(WideTile::kThreads), 0, s, p, S, l.part);
      OPTIMA_LAUNCH_CHECK();
      if (S > 1) {
        const dim3 g(unsigned(p.n_rows), unsigned(ceil_div(p.dp, 4 * kThreads)));
        hipLaunchKernelGGL((k_split_epilogue<MODE, PREC>), g, dim3(kThreads), 0, s, p, S,
                           rows_pad, static_cast<const float*>(l.part));
        OPTIMA_LAUNCH_CHECK();
      }
      return OPTIMA_OK;
    }
  }
  const bool sparse = PREC == kPrecSparse;
  const int bm = sparse ? SpTile::BM : kTile;
  const int tiles_m = int(ceil_div(p.n_rows, bm));
  const int tiles_n = p.dp / kTile;
  const int stages = sparse ? p.dp / SpTile::kKPerStage : p.dp * 4 / ProductTile::SRB;
  const int rows_pad = tiles_m * bm;
  const int S = sparse ? choose_splits_one_per_cu(tiles_m * tiles_n, stages, rows_pad, p.dp,
                                                  l.part_elems)
                       : choose_splits(tiles_m * tiles_n, stages, tiles_m, p.dp, l.part_elems);
  if constexpr (PREC == kPrecSparse)
    hipLaunchKernelGGL((k_product_sparse<MODE>), dim3(tiles_m * tiles_n * S),
                       dim3(SpTile::kThreads), 0, s, p, S, l.part);
  else
    hipLaunchKernelGGL((k_product<MODE, PREC>), dim3(tiles_m * tiles_n * S),
                       dim3(ProductTile::kThreads), 0, s, p, S, l.part);
  OPTIMA_LAUNCH_CHECK();
  if (S > 1) {
    const dim3 g(unsigned(p.n_rows), unsigned(ceil_div(p.dp, 4 * kThreads)));
    hipLaunchKernelGGL((k_split_epilogue<MODE, PREC>), g, dim3(kThreads), 0, s, p, S, rows_pad,
                       static_cast<const float*>(l.part));
    OPTIMA_LAUNCH_CHECK();
  }
  return OPTIMA_OK;
}

// Before a run of 2:4 tile products over rows 0..n_rows-1 (column rows[r],
// or r without a list): their index words from `idx` in the stage-major
// order that k_product_sparse reads.
optima_status stage_major_idx(const uint16_t* idx, const int* rows, int n_rows, const Layout& l,
                              ProductArgs& p, hipStream_t s) {
  p.AidxS = l.XIDXS;
  p.idx_pitch = l.idx_pitch;
  if (n_rows <= 0) return OPTIMA_OK;
  const int stages = int(l.dp / SpTile::kKPerStage);
  const int n_pad = int(round_up(n_rows, SpTile::BM));
  const int64_t entries = int64_t(stages) * n_pad;
  hipLaunchKernelGGL(k_idx_stage_major, dim3(unsigned(ceil_div(entries, kThreads))),
                     dim3(kThreads), 0, s, idx, rows, n_rows, n_pad, stages, l.idx_pitch,
                     l.XIDXS);
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

template <int MODE>
optima_status launch_product(const ProductArgs& p, const Layout& l, int prec, hipStream_t s) {
  if (prec == kPrecSparse) return launch_product<MODE, kPrecSparse>(p, l, s);
  return prec == kPrecBf16x3 ? launch_product<MODE, kPrecBf16x3>(p, l, s)
                             : launch_product<MODE, kPrecF32>(p, l, s);
}


// The CG iteration loop (after setup, the initial check and compaction).
optima_status cg_loop(const Layout& l, ProductArgs p, int dp, int di, const uint8_t* mask,
                      const optima_solver_opts& o, float* W_out,
                      const optima_solve_stats& stats, optima_solve_info& inf, hipEvent_t* ev,
                      bool timed, int n_act, hipStream_t s) {
  const bool split = o.precision == kPrecBf16x3;
  CgArgs cg{};
  cg.dp = dp;
  cg.d = di;
  cg.X = l.X0;
  cg.R = l.XA;
  cg.P = l.X1;
  cg.PP = split ? l.XP0 : nullptr;
  cg.Q = l.HA;
  cg.HX = l.HX;
  cg.HW0 = l.HW0;
  cg.mask = mask;
  cg.rr = l.st.kkt_prev;
  CgCheckArgs ck{};
  ck.dp = dp;
  ck.d = di;
  ck.X = l.X0;
  ck.R = l.XA;
  ck.HW0 = l.HW0;
  ck.mask = mask;
  ck.scale = o.col_scale;
  ck.st = l.st;
  ck.o = o;
  ck.W_out = W_out;
  ck.stats = stats;
  p.A = l.X1;
  p.Ap = l.XP0;
  p.out1 = l.HA;
  int* rows = l.rows0;
  int* rows_next = l.rows1;
  int64_t t = 0;
  const int64_t ce = o.check_every;
  while (t < o.max_iters && n_act > 0) {
    const int64_t t_next = std::min<int64_t>((t / ce + 1) * ce, o.max_iters);
    const int n = int(t_next - t);
    p.rows = rows;
    p.n_rows = n_act;
    cg.rows = rows;
    cg.n_rows = n_act;
    if (timed) OPTIMA_HIP_TRY(hipEventRecord(ev[0], s));
    for (int i = 0; i < n; ++i) {
      if (auto e = launch_product<kPlain>(p, l, o.precision, s)) return e;
      hipLaunchKernelGGL(k_cg_step, dim3(unsigned(n_act)), dim3(kThreads), 0, s, cg);
      OPTIMA_LAUNCH_CHECK();
    }
    if (timed) OPTIMA_HIP_TRY(hipEventRecord(ev[1], s));
    inf.gemm_calls += n;
    inf.row_products += int64_t(n) * n_act;
    inf.timed_launches += n;
    inf.timed_row_products += int64_t(n) * n_act;
    t = t_next;
    ck.rows = rows;
    ck.n_rows = n_act;
    ck.t = t;
    ck.final_check = t == o.max_iters;
    hipLaunchKernelGGL(k_cg_check, dim3(unsigned(n_act)), dim3(kThreads), 0, s, ck);
    OPTIMA_LAUNCH_CHECK();
    inf.checks += 1;
    hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, rows, n_act, l.st.done, rows_next,
                       l.n_active);
    OPTIMA_LAUNCH_CHECK();
    std::swap(rows, rows_next);
    OPTIMA_HIP_TRY(read_back(&n_act, l.n_active, sizeof(int), s));
    if (timed) {
      float ms = 0.f;
      OPTIMA_HIP_TRY(hipEventElapsedTime(&ms, ev[0], ev[1]));
      inf.timed_product_ms += ms;
    }
  }
  inf.iterations = t;
  return OPTIMA_OK;
}

}  // namespace

size_t qp_workspace_bytes(int64_t d, int64_t n_cols) {
  size_t b = 0;
  carve(nullptr, d, n_cols, &b);
  return b;
}

optima_status qp_solve(const float* H, int64_t d, const float* lambda_max, const float* W0,
                       const uint8_t* mask, int64_t n_cols, const optima_solver_opts& o,
                       void* ws, float* W_out, const optima_solve_stats& stats,
                       optima_solve_info* info, hipStream_t s) {
  size_t need = 0;
  Layout l = carve(ws, d, n_cols, &need);
  const int dp = int(l.dp), di = int(d), nc = int(n_cols);
  optima_solve_info inf{};

  OPTIMA_HIP_TRY(hipMemsetAsync(l.flags, 0, 4 * sizeof(int), s));
  OPTIMA_HIP_TRY(hipMemsetAsync(l.bar, 0, kBarWords * sizeof(unsigned), s));
  OPTIMA_HIP_TRY(hipMemsetAsync(l.n_active, 0, 4 * sizeof(int), s));
  OPTIMA_HIP_TRY(hipMemsetAsync(l.st.done, 0, size_t(nc) * sizeof(int), s));
  const float* Hm = H;
  const bool split = o.precision == kPrecBf16x3;
  // The finiteness scan of H: a pass of its own when H needs padding or no
  // split planes are built, else part of the split (k_split_h).
  const bool scan_in_split = split && !l.pad_h;
  if (!scan_in_split) {
    const int blocks = int(std::min<int64_t>(4096, ceil_div(int64_t(dp) * dp, kThreads)));
    hipLaunchKernelGGL(k_scan_pad_h, dim3(blocks), dim3(kThreads), 0, s, H, di, dp, l.Hp, l.flags);
    OPTIMA_LAUNCH_CHECK();
    if (l.pad_h) Hm = l.Hp;
  }
  const bool use_cg = o.method == OPTIMA_METHOD_CG;
  if (!use_cg) {  // CG needs no step size
    hipLaunchKernelGGL(k_step_constant, dim3(1), dim3(1), 0, s, lambda_max, o.step_safety, l.L,
                       l.flags);
    OPTIMA_LAUNCH_CHECK();
  }
  const dim3 vec_grid(unsigned(nc), unsigned(ceil_div(dp, 4 * kThreads)));
  // The rAPDHG iteration products skip the pruned entries on the 2:4 sparse
  // MFMA when every group of 4 of every mask row keeps at most 2. The index
  // words come first: k_prep_sparse reads the flags they set.
  const bool try_sparse = split && !use_cg && o.sparse;
  if (try_sparse) {
    const int64_t words = int64_t(nc) * (dp / 16);
    hipLaunchKernelGGL(k_sparse_index, dim3(unsigned(ceil_div(words, kThreads))), dim3(kThreads),
                       0, s, mask, nc, di, dp, l.XIDX, l.SLOT, l.XIDX2, l.flags);
    OPTIMA_LAUNCH_CHECK();
    // x0, and either the compressed planes of x0 and of p = w0 - x0 or
    // everything k_prep writes (see k_prep_sparse).
    const dim3 g_grid(unsigned(nc), unsigned(ceil_div(dp / 4, kThreads)));
    hipLaunchKernelGGL(k_prep_sparse, g_grid, dim3(kThreads), 0, s, W0, mask, di, dp, l.HX, l.X0,
                       l.XA, l.XP0, l.XP1, o.col_scale, l.flags);
  } else {
    // W0 padded copy goes to HX first; Hw0 = H w0, then Hx = Hx_ag = H x0.
    // Split planes: x0 into XP0, W0 into XP1 (free until the first update).
    hipLaunchKernelGGL(k_prep, vec_grid, dim3(kThreads), 0, s, W0, mask, nc, di, dp, l.HX, l.X0,
                       l.XA, split ? l.XP0 : nullptr, split ? l.XP1 : nullptr, o.col_scale,
                       l.flags);
  }
  OPTIMA_LAUNCH_CHECK();
  if (split) {
    hipLaunchKernelGGL(k_split_h, dim3(unsigned(dp), unsigned(ceil_div(dp, 4 * kThreads))),
                       dim3(kThreads), 0, s, Hm, dp, l.HP, scan_in_split ? l.flags : nullptr);
    OPTIMA_LAUNCH_CHECK();
  }
  int flags[3] = {0, 0, 0};
  OPTIMA_HIP_TRY(read_back(flags, l.flags, 3 * sizeof(int), s));
  if (flags[0]) return OPTIMA_E_NONFINITE;
  const bool sparse = try_sparse && !flags[1];
  const int iprec = sparse ? int(kPrecSparse) : o.precision;
  inf.sparse_products = sparse ? 1 : 0;

  ProductArgs p{};
  p.B = Hm;
  p.dp = dp;
  p.d = di;
  p.mask = mask;
  p.kbase = l.st.kbase;
  p.Lp = l.L;
  p.rows = nullptr;
  p.n_rows = nc;
  p.Bp = l.HP;
  p.Aidx = l.XIDX;
  p.slot = l.SLOT;
  if (sparse && !flags[2]) {
    // Both setup operands are 2:4-compressible: H x0 on the kept pairs and
    // H w0 = H x0 + H p with p = w0 - x0 on the pruned pairs, both on the
    // sparse MFMA (k_prep_sparse wrote their compressed planes). Where w0 is
    // zero off the mask, H p is exactly zero and H w0 equals H x0 bit for
    // bit.
    p.A = l.X0;
    p.Ap = l.XP0;
    p.Aidx = l.XIDX;
    p.out1 = l.HX;
    p.out2 = l.HA;
    if (auto e = stage_major_idx(l.XIDX, nullptr, nc, l, p, s)) return e;
    if (auto e = launch_product<kPlain2>(p, l, kPrecSparse, s)) return e;
    p.Ap = l.XP1;
    p.Aidx = l.XIDX2;
    p.out1 = l.HW0;
    p.out2 = l.HX;
    if (auto e = stage_major_idx(l.XIDX2, nullptr, nc, l, p, s)) return e;
    if (auto e = launch_product<kPlainAdd>(p, l, kPrecSparse, s)) return e;
    p.Aidx = l.XIDX;
  } else {
    // The setup products use the solve's precision too: H w0 and H x0 then
    // agree bit for bit wherever w0 and x0 do (all-kept columns start at
    // their optimum with a zero gradient).
    p.A = l.HX;
    p.Ap = l.XP1;
    p.out1 = l.HW0;
    if (auto e = launch_product<kPlain>(p, l, o.precision, s)) return e;
    p.A = l.X0;
    p.Ap = l.XP0;
    p.out1 = l.HX;
    p.out2 = l.HA;
    if (auto e = launch_product<kPlain2>(p, l, o.precision, s)) return e;
  }
  inf.gemm_calls += 2;
  inf.row_products += 2 * int64_t(nc);

  CheckArgs ca{};
  ca.dp = dp;
  ca.d = di;
  ca.XA = l.XA;
  ca.HX = l.HX;
  ca.HA = l.HA;
  ca.HW0 = l.HW0;
  ca.W0 = W0;
  ca.mask = mask;
  ca.scale = o.col_scale;
  ca.packed = 0;
  ca.slot = l.SLOT;
  ca.st = l.st;
  ca.o = o;
  ca.W_out = W_out;
  ca.stats = stats;

  // Initial check at the start point.
  ca.rows = nullptr;
  ca.n_rows = nc;
  ca.X = l.X0;
  ca.initial = 1;
  ca.final_check = o.max_iters == 0;
  ca.t = 0;
  ca.n_block = 0;
  hipLaunchKernelGGL(k_check, dim3(nc), dim3(kThreads), 0, s, ca);
  OPTIMA_LAUNCH_CHECK();
  inf.checks += 1;
  if (use_cg) {
    CgArgs ci{};
    ci.rows = nullptr;
    ci.n_rows = nc;
    ci.dp = dp;
    ci.d = di;
    ci.R = l.XA;
    ci.P = l.X1;
    ci.PP = split ? l.XP0 : nullptr;
    ci.HX = l.HX;
    ci.HW0 = l.HW0;
    ci.mask = mask;
    ci.rr = l.st.kkt_prev;
    hipLaunchKernelGGL(k_cg_init, dim3(unsigned(nc)), dim3(kThreads), 0, s, ci);
    OPTIMA_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, (const int*)nullptr, nc, l.st.done,
                     l.rows0, l.n_active);
  OPTIMA_LAUNCH_CHECK();
  int n_act = 0;
  OPTIMA_HIP_TRY(read_back(&n_act, l.n_active, sizeof(int), s));
  if (sparse && n_act > 0) {
    hipLaunchKernelGGL(k_pack, dim3(unsigned(n_act)), dim3(kThreads), 0, s, l.rows0, n_act, dp,
                       l.SLOT, l.X0, l.XA, l.HX, l.HA, l.HW0);
    OPTIMA_LAUNCH_CHECK();
    ca.packed = 1;
  }

  // Optional timing of the iteration loop's product launches.
  hipEvent_t ev[2] = {nullptr, nullptr};
  if (info) {
    OPTIMA_HIP_TRY(hipEventCreate(&ev[0]));
    if (hipEventCreate(&ev[1]) != hipSuccess) {
      (void)hipEventDestroy(ev[0]);
      return OPTIMA_E_HIP;
    }
  }
  struct EventGuard {
    hipEvent_t* e;
    ~EventGuard() {
      if (e[0]) (void)hipEventDestroy(e[0]);
      if (e[1]) (void)hipEventDestroy(e[1]);
    }
  } guard{ev};

  if (use_cg) {
    const optima_status e = cg_loop(l, p, dp, di, mask, o, W_out, stats, inf, ev, info != nullptr,
                                    n_act, s);
    if (e) return e;
    if (info) *info = inf;
    return OPTIMA_OK;
  }

  int* rows = l.rows0;
  int* rows_next = l.rows1;
  float* xbuf[2] = {l.X0, l.X1};
  uint16_t* xpl[2] = {l.XP0, l.XP1};
  int cur = 0;
  int64_t t = 0;
  const int64_t ce = o.check_every;
  while (t < o.max_iters && n_act > 0) {
    const int64_t t_next = std::min<int64_t>((t / ce + 1) * ce, o.max_iters);
    const int n = int(t_next - t);
    const dim3 ug(unsigned(n_act), unsigned(ceil_div(dp, 4 * kThreads)));
    hipLaunchKernelGGL(k_update, ug, dim3(kThreads), 0, s, rows, n_act, dp, di, xbuf[cur],
                       xbuf[cur ^ 1], l.XA, l.HX, l.HA, l.HW0, mask, l.st.kbase, l.L,
                       split ? xpl[cur ^ 1] : nullptr, sparse ? 1 : 0, l.SLOT);
    OPTIMA_LAUNCH_CHECK();
    cur ^= 1;
    p.rows = rows;
    p.n_rows = n_act;
    p.HA = l.HA;
    p.HW0 = l.HW0;
    p.XA = l.XA;
    if (iprec == kPrecSparse && !few_column_path(iprec, n_act, dp))
      if (auto e = stage_major_idx(l.XIDX, rows, n_act, l, p, s)) return e;
    if (info) OPTIMA_HIP_TRY(hipEventRecord(ev[0], s));
    bool persisted = false;
    if (o.cooperative && persistent_path(iprec, n_act, dp) &&
        size_t(nc) * size_t(dp) * 4 < (size_t(1) << 31)) {
      PersistArgs pa{};
      pa.p = p;
      pa.p.out1 = l.HX;
      pa.X[0] = xbuf[0];
      pa.X[1] = xbuf[1];
      pa.XP[0] = xpl[0];
      pa.XP[1] = xpl[1];
      pa.x_bytes = uint32_t(size_t(nc) * size_t(dp) * 4);
      pa.cur = cur;
      pa.n_iter = n;
      pa.arrivals = l.bar;
      pa.timeout = l.n_active + 1;
      OPTIMA_HIP_TRY(hipMemsetAsync(l.bar, 0, kBarWords * sizeof(unsigned), s));
      persisted = launch_persistent(pa, iprec, s);
      if (persisted) {
        cur ^= (n - 1) & 1;
        inf.persistent_launches += 1;
      }
    }
    if (!persisted) {
      for (int i = 0; i + 1 < n; ++i) {
        p.A = xbuf[cur];
        p.Ap = xpl[cur];
        p.Xin = xbuf[cur];
        p.Xout = xbuf[cur ^ 1];
        p.XoutP = xpl[cur ^ 1];
        p.s = i;
        if (auto e = launch_product<kFused>(p, l, iprec, s)) return e;
        cur ^= 1;
      }
      p.A = xbuf[cur];
      p.Ap = xpl[cur];
      p.out1 = l.HX;
      p.s = n - 1;
      if (auto e = launch_product<kStore>(p, l, iprec, s)) return e;
    }
    if (info) OPTIMA_HIP_TRY(hipEventRecord(ev[1], s));
    inf.gemm_calls += n;
    inf.row_products += int64_t(n) * n_act;
    inf.timed_launches += n;
    inf.timed_row_products += int64_t(n) * n_act;
    const bool few = few_column_path(iprec, n_act, dp);  // this block's launches
    const int act_block = n_act;
    t = t_next;

    ca.rows = rows;
    ca.n_rows = n_act;
    ca.X = xbuf[cur];
    ca.XP = split ? xpl[cur] : nullptr;
    ca.initial = 0;
    ca.final_check = t == o.max_iters;
    ca.t = t;
    ca.n_block = n;
    hipLaunchKernelGGL(k_check, dim3(n_act), dim3(kThreads), 0, s, ca);
    OPTIMA_LAUNCH_CHECK();
    inf.checks += 1;
    hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, rows, n_act, l.st.done, rows_next,
                       l.n_active);
    OPTIMA_LAUNCH_CHECK();
    std::swap(rows, rows_next);
    int act_timeout[2] = {0, 0};
    OPTIMA_HIP_TRY(read_back(act_timeout, l.n_active, 2 * sizeof(int), s));
    n_act = act_timeout[0];
    if (act_timeout[1]) return OPTIMA_E_HIP;  // a grid barrier wait gave up
    if (info) {
      float ms = 0.f;
      OPTIMA_HIP_TRY(hipEventElapsedTime(&ms, ev[0], ev[1]));
      inf.timed_product_ms += ms;
      if (few) {
        inf.few_launches += n;
        inf.few_row_products += int64_t(n) * act_block;
        inf.few_product_ms += ms;
      }
    }
  }
  inf.iterations = t;
  if (info) *info = inf;
  return OPTIMA_OK;
}

#ifdef OPTIMA_PHASE_STAMPS
// Copies the stamps into host memory (tile: up to max_tile rows of 4
// uint64; coop: 4 x 256 x 6 uint64), clears the tile count and returns the
// number of tile stamps recorded since the last call (< 0: HIP error).
extern "C" int optima_phase_stamps(uint64_t* tile, int max_tile, uint64_t* coop) {
  unsigned n = 0;
  if (hipDeviceSynchronize() != hipSuccess) return -1;
  if (hipMemcpyFromSymbol(&n, HIP_SYMBOL(g_tile_stamp_count), sizeof(n)) != hipSuccess) return -1;
  const size_t rows = std::min<size_t>(std::min<size_t>(n, kTileStampSlots), size_t(std::max(max_tile, 0)));
  if (rows && hipMemcpyFromSymbol(tile, HIP_SYMBOL(g_tile_stamps), rows * 4 * sizeof(uint64_t)) != hipSuccess)
    return -1;
  if (coop && hipMemcpyFromSymbol(coop, HIP_SYMBOL(g_coop_stamps), sizeof(g_coop_stamps)) != hipSuccess)
    return -1;
  const unsigned zero = 0;
  if (hipMemcpyToSymbol(HIP_SYMBOL(g_tile_stamp_count), &zero, sizeof(zero)) != hipSuccess) return -1;
  return int(std::min<size_t>(n, kTileStampSlots));
}
#endif

}  // namespace optima
