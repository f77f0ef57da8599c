// Largest eigenvalue of the damped Hessian by power iteration; it sets the
// solver's step constant L = 2 lambda_max (1 + safety). Each iteration is one
// HBM-bound pass over H (a GEMV with one wave per row, 16-byte loads) and a
// one-workgroup pass that forms the Rayleigh quotient and the next norm.
#include "common.h"

namespace optima {
namespace {

struct PowState {
  double norm2_0;     // ||v0||^2
  double rho[2];      // rho of iteration i kept in slot i & 1 (written by iteration i + 1)
  int conv;
  int iters;
};

constexpr int kRowsPerWave = 2;
constexpr int kRowsPerBlock = (kThreads / 64) * kRowsPerWave;

// Power iteration i (1-based): y_i = H v_{i-1} / ||v_{i-1}|| with one wave per
// row. Every workgroup first sums the partials (||y||^2, v.y) that all
// workgroups of iteration i - 1 left in part[(i-1) & 1], in the same fixed
// order, so all of them get bit-identical values of ||y_{i-1}|| and
// rho_{i-1} = v_{i-2}^T H v_{i-2} (unit v) and take the same convergence
// decision; workgroup 0 records it. No workgroup waits for another: the
// kernel boundary orders the iterations.
template <bool VEC4>
__global__ void __launch_bounds__(kThreads) k_power_iter(const float* H, int64_t d, const float* vin,
                                                         float* y, double2* part, int nblk,
                                                         PowState* st, int it, float tol,
                                                         float* lambda_out) {
  if (st->conv) return;
  __shared__ double ra[kThreads], rb[kThreads];
  __shared__ double sn[kRowsPerBlock], sd[kRowsPerBlock];
  double norm2;
  if (it == 1) {
    norm2 = st->norm2_0;
  } else {
    const double2* prev = part + size_t((it - 1) & 1) * nblk;
    double a = 0.0, b = 0.0;
    for (int i = threadIdx.x; i < nblk; i += kThreads) {
      const double2 q = prev[i];
      a += q.x;
      b += q.y;
    }
    ra[threadIdx.x] = a;
    rb[threadIdx.x] = b;
    __syncthreads();
    for (int o = kThreads / 2; o > 0; o >>= 1) {
      if (threadIdx.x < o) {
        ra[threadIdx.x] += ra[threadIdx.x + o];
        rb[threadIdx.x] += rb[threadIdx.x + o];
      }
      __syncthreads();
    }
    norm2 = ra[0];
    const double rho = rb[0];
    const bool done = norm2 == 0.0 ||
                      (it > 2 && fabs(rho - st->rho[(it - 2) & 1]) <= double(tol) * fabs(rho));
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      st->rho[(it - 1) & 1] = rho;
      *lambda_out = norm2 == 0.0 ? 0.f : float(rho);
      st->iters = it - 1;
      if (done) st->conv = 1;
    }
    if (done) return;
  }
  const double inv = 1.0 / sqrt(norm2);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < kRowsPerWave; ++q) {
    const int lr = w * kRowsPerWave + q;
    const int64_t row = int64_t(blockIdx.x) * kRowsPerBlock + lr;
    double n2 = 0.0, dt = 0.0;
    if (row < d) {
      const float* h = H + row * d;
      float acc0 = 0.f, acc1 = 0.f;
      if (VEC4) {
        const int64_t n4 = d >> 2;
        const float4* h4 = reinterpret_cast<const float4*>(h);
        const float4* v4 = reinterpret_cast<const float4*>(vin);
        int64_t k = lane;
        for (; k + 64 < n4; k += 128) {
          const float4 a = h4[k], b = v4[k], c = h4[k + 64], e = v4[k + 64];
          acc0 += a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
          acc1 += c.x * e.x + c.y * e.y + c.z * e.z + c.w * e.w;
        }
        for (; k < n4; k += 64) {
          const float4 a = h4[k], b = v4[k];
          acc0 += a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
        }
      } else {
        for (int64_t k = lane; k < d; k += 64) acc0 += h[k] * vin[k];
      }
      float acc = acc0 + acc1;
      for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
      const float yr = float(double(acc) * inv);
      if (lane == 0) {
        y[row] = yr;
        n2 = double(yr) * double(yr);
        dt = double(vin[row]) * inv * double(yr);
      }
    }
    if (lane == 0) {
      sn[lr] = n2;
      sd[lr] = dt;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double a = 0.0, b = 0.0;
    for (int i = 0; i < kRowsPerBlock; ++i) {
      a += sn[i];
      b += sd[i];
    }
    part[size_t(it & 1) * nblk + blockIdx.x] = make_double2(a, b);
  }
}

// Closes the last iteration when max_iters ran out before convergence.
__global__ void __launch_bounds__(kThreads) k_power_close(const double2* part, int nblk,
                                                          PowState* st, int it,
                                                          float* lambda_out) {
  if (st->conv) return;
  __shared__ double ra[kThreads], rb[kThreads];
  const double2* prev = part + size_t(it & 1) * nblk;
  double a = 0.0, b = 0.0;
  for (int i = threadIdx.x; i < nblk; i += kThreads) {
    a += prev[i].x;
    b += prev[i].y;
  }
  ra[threadIdx.x] = a;
  rb[threadIdx.x] = b;
  __syncthreads();
  for (int o = kThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      ra[threadIdx.x] += ra[threadIdx.x + o];
      rb[threadIdx.x] += rb[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *lambda_out = ra[0] == 0.0 ? 0.f : float(rb[0]);
    st->iters = it;
  }
}

__global__ void __launch_bounds__(1024) k_power_init(const float* v0, int64_t d, float* v,
                                                     PowState* st, float* lambda_out) {
  __shared__ double red[16];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < d; i += 1024) {
    const float x = v0[i];
    v[i] = x;
    s += double(x) * double(x);
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < 16; ++w) t += red[w];
    st->norm2_0 = t;
    st->rho[0] = st->rho[1] = 0.0;
    st->conv = t > 0.0 ? 0 : 1;
    st->iters = 0;
    *lambda_out = 0.f;
  }
}

__global__ void k_copy_iters(const PowState* st, int32_t* iters) { *iters = st->iters; }

}  // namespace

size_t spectral_norm_workspace_bytes(int64_t d) {
  Carver c(nullptr);
  c.take<float>(size_t(d));
  c.take<float>(size_t(d));
  c.take<double2>(2 * size_t(ceil_div(d, kRowsPerBlock)));
  c.take<PowState>(1);
  return c.bytes();
}

optima_status spectral_norm(const float* H, int64_t d, const float* v0, int max_iters, float tol,
                            void* ws, float* lambda_max, int32_t* iters, hipStream_t s) {
  Carver c(ws);
  float* buf[2] = {c.take<float>(size_t(d)), c.take<float>(size_t(d))};
  const int nblk = int(ceil_div(d, kRowsPerBlock));
  double2* part = c.take<double2>(2 * size_t(nblk));
  PowState* st = c.take<PowState>(1);
  hipLaunchKernelGGL(k_power_init, dim3(1), dim3(1024), 0, s, v0, d, buf[0], st, lambda_max);
  OPTIMA_LAUNCH_CHECK();
  const bool vec4 = (d % 4) == 0 && aligned16(H);
  constexpr int kPoll = 32;
  for (int it = 1; it <= max_iters; ++it) {
    const float* vin = buf[(it - 1) & 1];
    float* y = buf[it & 1];
    if (vec4)
      hipLaunchKernelGGL(k_power_iter<true>, dim3(unsigned(nblk)), dim3(kThreads), 0, s, H, d, vin,
                         y, part, nblk, st, it, tol, lambda_max);
    else
      hipLaunchKernelGGL(k_power_iter<false>, dim3(unsigned(nblk)), dim3(kThreads), 0, s, H, d,
                         vin, y, part, nblk, st, it, tol, lambda_max);
    OPTIMA_LAUNCH_CHECK();
    if (it % kPoll == 0 && it < max_iters) {
      int conv = 0;
      OPTIMA_HIP_TRY(hipMemcpyAsync(&conv, &st->conv, sizeof(int), hipMemcpyDeviceToHost, s));
      OPTIMA_HIP_TRY(hipStreamSynchronize(s));
      if (conv) break;
    }
  }
  // Iteration i's rho is formed at the start of iteration i + 1; one more
  // (row-free) pass closes the final iteration.
  hipLaunchKernelGGL(k_power_close, dim3(1), dim3(kThreads), 0, s, part, nblk, st, max_iters,
                     lambda_max);
  OPTIMA_LAUNCH_CHECK();
  if (iters) {
    hipLaunchKernelGGL(k_copy_iters, dim3(1), dim3(1), 0, s, st, iters);
    OPTIMA_LAUNCH_CHECK();
  }
  OPTIMA_HIP_TRY(hipStreamSynchronize(s));
  return OPTIMA_OK;
}

}  // namespace optima
