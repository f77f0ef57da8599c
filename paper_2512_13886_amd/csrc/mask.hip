// Wanda mask selection on the device: the mask that the weight update starts
// from (Algorithm 1 takes M from a selector; the configurations use Wanda's
// saliency, cited in Section 2, with the 2:4 pattern of Section 4).
//
// score[j][i] = W0[j][i]^2 * c[i] in fp64 (the square of |W0| sqrt(c): same
// order; the square of an fp32 weight is exact in fp64 and the product is
// rounded once, so every IEEE implementation gets the same bits). Scores are
// compared through an order-preserving 64-bit key: NaN lowest, -0 == +0.
//
// Unstructured: one workgroup per row finds the keep-th largest key T by an
// 8-pass radix select (8-bit digits, most significant first, LDS histogram),
// then keeps every key > T and, in index order, as many keys == T as are still
// needed. 2:4: one thread per group of 4 ranks its scores.
#include "common.h"

namespace optima {
namespace {

constexpr int kMaskThreads = 256;

__device__ inline double col_value(const void* c, int dtype, int64_t stride, int64_t i) {
  return dtype == OPTIMA_DTYPE_F64 ? static_cast<const double*>(c)[i * stride]
                                   : double(static_cast<const float*>(c)[i * stride]);
}

__device__ inline uint64_t mask_key(float w, double c) {
  const double wd = double(w);
  double s = (wd * wd) * c;
  if (s != s) return 0;       // NaN ranks below everything
  if (s == 0.0) s = 0.0;      // -0 ranks with +0
  const uint64_t b = static_cast<uint64_t>(__double_as_longlong(s));
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__global__ void __launch_bounds__(kMaskThreads) k_mask_topk(const float* W0, int64_t d,
                                                            const void* c, int c_dtype,
                                                            int64_t c_stride, int64_t keep,
                                                            uint8_t* mask) {
  __shared__ unsigned hist[256];
  __shared__ uint64_t s_prefix;
  __shared__ int64_t s_need;
  __shared__ int64_t scan[kMaskThreads];
  const int64_t j = blockIdx.x;
  const float* w = W0 + j * d;
  uint8_t* m = mask + j * d;
  const int tid = threadIdx.x;
  if (keep <= 0 || keep >= d) {
    const uint8_t v = keep > 0 ? 1 : 0;
    for (int64_t i = tid; i < d; i += kMaskThreads) m[i] = v;
    return;
  }
  uint64_t prefix = 0, pmask = 0;
  int64_t need = keep;  // keys still to take at or below the current prefix
  for (int pass = 7; pass >= 0; --pass) {
    const int shift = 8 * pass;
    hist[tid] = 0;
    __syncthreads();
    for (int64_t i = tid; i < d; i += kMaskThreads) {
      const uint64_t k = mask_key(w[i], col_value(c, c_dtype, c_stride, i));
      if ((k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      int64_t above = 0;
      int b = 255;
      for (; b > 0; --b) {
        if (above + hist[b] >= need) break;
        above += hist[b];
      }
      s_prefix = prefix | (uint64_t(b) << shift);
      s_need = need - above;
    }
    __syncthreads();
    prefix = s_prefix;
    need = s_need;
    pmask |= uint64_t(255) << shift;
  }
  // prefix is now the keep-th largest key T; `need` keys equal to T are kept,
  // the ones with the lowest indices. Each thread takes a contiguous range.
  const int64_t chunk = (d + kMaskThreads - 1) / kMaskThreads;
  const int64_t lo = tid * chunk < d ? tid * chunk : d;
  const int64_t hi = lo + chunk < d ? lo + chunk : d;
  int64_t eq = 0;
  for (int64_t i = lo; i < hi; ++i)
    eq += mask_key(w[i], col_value(c, c_dtype, c_stride, i)) == prefix;
  scan[tid] = eq;
  __syncthreads();
  if (tid == 0) {  // exclusive scan in thread order
    int64_t run = 0;
    for (int t = 0; t < kMaskThreads; ++t) {
      const int64_t v = scan[t];
      scan[t] = run;
      run += v;
    }
  }
  __syncthreads();
  int64_t rank = scan[tid];
  for (int64_t i = lo; i < hi; ++i) {
    const uint64_t k = mask_key(w[i], col_value(c, c_dtype, c_stride, i));
    uint8_t v = k > prefix ? 1 : 0;
    if (k == prefix) v = rank++ < need ? 1 : 0;
    m[i] = v;
  }
}

__global__ void __launch_bounds__(kMaskThreads) k_mask_2to4(const float* W0, int64_t n_groups,
                                                            int64_t d, const void* c, int c_dtype,
                                                            int64_t c_stride, uint8_t* mask) {
  const int64_t g = int64_t(blockIdx.x) * kMaskThreads + threadIdx.x;
  if (g >= n_groups) return;
  const int64_t e0 = g * 4;             // flat element index of the group
  const int64_t i0 = e0 % d;            // its feature index (d % 4 == 0)
  uint64_t k[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) k[q] = mask_key(W0[e0 + q], col_value(c, c_dtype, c_stride, i0 + q));
  uint32_t out = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int beaten = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) beaten += (k[r] > k[q]) || (k[r] == k[q] && r < q);
    out |= uint32_t(beaten < 2) << (8 * q);
  }
  *reinterpret_cast<uint32_t*>(mask + e0) = out;
}

}  // namespace

optima_status wanda_mask(const float* W0, int64_t n_cols, int64_t d, const void* col_sq,
                         int col_dtype, int64_t col_stride, int pattern, double sparsity,
                         uint8_t* mask, hipStream_t s) {
  if (n_cols == 0) return OPTIMA_OK;
  if (pattern == OPTIMA_MASK_2TO4) {
    const int64_t groups = n_cols * d / 4;
    hipLaunchKernelGGL(k_mask_2to4, dim3(unsigned(ceil_div(groups, kMaskThreads))),
                       dim3(kMaskThreads), 0, s, W0, groups, d, col_sq, col_dtype, col_stride,
                       mask);
  } else {
    const int64_t keep = d - int64_t(floor(sparsity * double(d)));
    hipLaunchKernelGGL(k_mask_topk, dim3(unsigned(n_cols)), dim3(kMaskThreads), 0, s, W0, d,
                       col_sq, col_dtype, col_stride, keep, mask);
  }
  OPTIMA_LAUNCH_CHECK();
  return OPTIMA_OK;
}

}  // namespace optima
