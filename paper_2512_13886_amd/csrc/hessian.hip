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
  const int64_t k_off = int64_t(s0) * kStageRowBytes + load_seg_bytes();
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsA; ++i)
    src.a[i] = XT + (int64_t(ti) * kTile + load_row<Cfg>(i)) * pitch_bytes + k_off;
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsB; ++i)
    src.b[i] = XT + (int64_t(tj) * kTile + load_row<Cfg>(i)) * pitch_bytes + k_off;
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

}  // namespace

size_t hessian_workspace_bytes(int64_t n_tok, int64_t d, int dtype) {
  const HessPlan p = plan(n_tok, d, dtype);
  Carver c(nullptr);
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
  const int64_t B = ceil_div(d, 64);
  hipLaunchKernelGGL(k_hess_reduce, dim3(unsigned(B * (B + 1) / 2)), dim3(kThreads), 0, s, part,
                     p.splits, p.dp, d, H, accumulate);
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

optima_status hessian_damp(float* H, int64_t d, float rel, float* lambda_out, hipStream_t s) {
  hipLaunchKernelGGL(k_damp, dim3(1), dim3(1024), 0, s, H, d, rel, lambda_out);
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

}  // namespace optima
