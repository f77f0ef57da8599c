// Forward pass of a linear layer on the calibration tokens, for the layer
// loop of Algorithm 1: its outputs y = L(x) feed the next layer's Hessian and
// the update X <- L(X) that follows the pruning of L. It also forms the
// squared output error between two weight sets. The relative layer-wise
// error of Section 4 is a ratio of such errors, each against the dense
// layer's outputs.
//
// Z = X W^T with X [n_tok][d_in] bf16 (calibration activations) and W fp32
// rounded to bf16 (round to nearest even, the weights a bf16 model stores),
// on v_mfma_f32_16x16x32_bf16 with fp32 accumulation: the 128 x 128 tile of
// the GEMM core with token rows as A and weight rows as B (both contiguous in
// d_in). Epilogue per 4 consecutive outputs: the squared difference to a
// reference Z (fp64 partial sums), the activation and the store.
#include "common.h"
#include "readback.h"
#include "gemm_core.h"

namespace optima {
namespace {

// bf16 copy of W with rows padded by zeros to rows_pad; flags[0] = 1 if W
// holds a NaN or Inf.
__global__ void __launch_bounds__(kThreads) k_weights_bf16(const float* W, int64_t d_out,
                                                           int64_t d_in, uint16_t* Wb,
                                                           int* flags) {
  const int64_t r = blockIdx.x;
  bool bad = false;
  for (int64_t k = threadIdx.x; k < d_in; k += kThreads) {
    float v = 0.f;
    if (r < d_out) {
      v = W[r * d_in + k];
      bad |= !isfinite(v);
    }
    Wb[r * d_in + k] = uint16_t(bf16_rne_bits(v));
  }
  if (bad) atomicOr(flags, 1);
}

__device__ inline float act_apply(int act, float z) {
  return act == OPTIMA_ACT_SILU ? z / (1.f + expf(-z)) : z;
}

// One 128 x 128 tile of Z per workgroup (tokens x outputs). A y_dtype other
// than BF16 or F32 stores nothing; err_part[blockIdx.x] receives the tile's sum of (Z - Y_ref)^2.
__global__ void __launch_bounds__(Tile128::kThreads) k_forward(const char* X, int64_t n_tok,
                                                               int64_t d_in, const uint16_t* Wb,
                                                               int64_t d_out, int act,
                                                               void* Y, int y_dtype,
                                                               const float* Y_ref,
                                                               double* err_part) {
  using Cfg = Tile128;
  __shared__ __attribute__((aligned(1024))) char lds0[Cfg::kBufBytes];
  __shared__ __attribute__((aligned(1024))) char lds1[Cfg::kBufBytes];
  __shared__ double red[Cfg::kThreads / 64];
  const int tiles_m = int((n_tok + kTile - 1) / kTile);
  const int tiles_n = int((d_out + kTile - 1) / kTile);
  int tm, tn;
  tile_of_block(blockIdx.x, tiles_m * tiles_n, tiles_m, tiles_n, &tm, &tn);
  const int64_t m0 = int64_t(tm) * kTile, n0 = int64_t(tn) * kTile;
  const int64_t pitch = d_in * 2;  // bytes per row of X and of Wb
  Operands<Cfg> src;
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsA; ++i) {
    int64_t t = m0 + load_row<Cfg>(i);
    t = t < n_tok ? t : n_tok - 1;
    src.a[i] = X + t * pitch + load_seg_bytes<Cfg>(i);
  }
  const char* wb = reinterpret_cast<const char*>(Wb);
#pragma unroll
  for (int i = 0; i < Cfg::kLoadsB; ++i)
    src.b[i] = wb + (n0 + load_row<Cfg>(i)) * pitch + load_seg_bytes<Cfg>(i);
  f4 acc[Cfg::MB][Cfg::NB];
  gemm_tile_mainloop<Cfg, Bf16Tag>(acc, src, int(pitch / Cfg::SRB), lds0, lds1, nullptr);
  stage_tile<Cfg>(acc, lds0, lds1);
  __syncthreads();

  double e = 0.0;
#pragma unroll 4
  for (int q = 0; q < kTile * kTile / 4 / Cfg::kThreads; ++q) {
    const int c = threadIdx.x + Cfg::kThreads * q;  // 16-byte chunk of the tile
    const int r = c >> 5, ch = c & 31;
    const int64_t t = m0 + r, n = n0 + 4 * ch;
    if (t >= n_tok || n >= d_out) continue;  // d_out % 4 == 0: chunks are all in or all out
    const float4 z = staged_chunk(lds0, lds1, r, ch);
    const size_t o = size_t(t) * size_t(d_out) + size_t(n);
    if (Y_ref) {
      const float4 y = *reinterpret_cast<const float4*>(Y_ref + o);
      const double a = double(z.x) - y.x, b = double(z.y) - y.y, cc = double(z.z) - y.z,
                   d = double(z.w) - y.w;
      e += a * a + b * b + cc * cc + d * d;
    }
    if (y_dtype == OPTIMA_DTYPE_F32) {
      *reinterpret_cast<float4*>(static_cast<float*>(Y) + o) =
          make_float4(act_apply(act, z.x), act_apply(act, z.y), act_apply(act, z.z),
                      act_apply(act, z.w));
    } else if (y_dtype == OPTIMA_DTYPE_BF16) {
      const uint32_t b0 = bf16_rne_bits(act_apply(act, z.x)), b1 = bf16_rne_bits(act_apply(act, z.y));
      const uint32_t b2 = bf16_rne_bits(act_apply(act, z.z)), b3 = bf16_rne_bits(act_apply(act, z.w));
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(Y) + o) =
          make_uint2(b0 | (b1 << 16), b2 | (b3 << 16));
    }
  }
  if (err_part) {
    e = block_sum(e, red);
    if (threadIdx.x == 0) err_part[blockIdx.x] = e;
  }
}

// err_out = sum of the n per-tile partials, in a fixed order.
__global__ void __launch_bounds__(kThreads) k_err_reduce(const double* part, int n,
                                                         double* err_out) {
  __shared__ double red[kThreads / 64];
  double s = 0.0;
  for (int i = threadIdx.x; i < n; i += kThreads) s += part[i];
  s = block_sum(s, red);
  if (threadIdx.x == 0) *err_out = s;
}

struct FwdLayout {
  uint16_t* Wb;
  double* part;
  int* flags;
};

FwdLayout carve_forward(void* ws, int64_t n_tok, int64_t d_in, int64_t d_out, size_t* bytes) {
  Carver c(ws);
  FwdLayout l{};
  const int64_t rows_pad = round_up(d_out, kTile);
  l.Wb = c.take<uint16_t>(size_t(rows_pad) * size_t(d_in));
  l.part = c.take<double>(size_t(ceil_div(n_tok, kTile) * ceil_div(d_out, kTile)));
  l.flags = c.take<int>(4);
  if (bytes) *bytes = c.bytes();
  return l;
}

}  // namespace

size_t linear_forward_workspace_bytes(int64_t n_tok, int64_t d_in, int64_t d_out) {
  size_t b = 0;
  carve_forward(nullptr, n_tok, d_in, d_out, &b);
  return b;
}

optima_status linear_forward(const void* X, int64_t n_tok, int64_t d_in, const float* W,
                             int64_t d_out, int act, void* Y, int y_dtype, const float* Y_ref,
                             double* err_out, void* ws, hipStream_t s) {
  FwdLayout l = carve_forward(ws, n_tok, d_in, d_out, nullptr);
  const int64_t rows_pad = round_up(d_out, kTile);
  OPTIMA_HIP_TRY(hipMemsetAsync(l.flags, 0, sizeof(int), s));
  hipLaunchKernelGGL(k_weights_bf16, dim3(unsigned(rows_pad)), dim3(kThreads), 0, s, W, d_out,
                     d_in, l.Wb, l.flags);
  OPTIMA_LAUNCH_CHECK();
  int flag = 0;
  OPTIMA_HIP_TRY(read_back(&flag, l.flags, sizeof(int), s));
  if (flag) return OPTIMA_E_NONFINITE;
  if (n_tok == 0) {
    if (err_out) OPTIMA_HIP_TRY(hipMemsetAsync(err_out, 0, sizeof(double), s));
    return OPTIMA_OK;
  }
  const int tiles = int(ceil_div(n_tok, kTile) * ceil_div(d_out, kTile));
  hipLaunchKernelGGL(k_forward, dim3(unsigned(tiles)), dim3(Tile128::kThreads), 0, s,
                     static_cast<const char*>(X), n_tok, d_in, l.Wb, d_out, act, Y,
                     Y ? y_dtype : -1, err_out ? Y_ref : nullptr, err_out ? l.part : nullptr);
  OPTIMA_LAUNCH_CHECK();
  if (err_out) {
    hipLaunchKernelGGL(k_err_reduce, dim3(1), dim3(kThreads), 0, s, l.part, tiles, err_out);
    OPTIMA_LAUNCH_CHECK();
  }
  return OPTIMA_OK;
}

}  // namespace optima
