// Largest eigenvalue of the damped Hessian; it sets the solver's step constant
// L = 2 lambda_max (1 + safety).
//
// block == 1: power iteration. Each iteration is one HBM-bound pass over H (a
// GEMV with one wave per row, 16-byte loads); the next launch reduces the
// Rayleigh quotient and the norm.
//
// block = b in [2, 16]: subspace iteration with Rayleigh-Ritz. With Y_{i-1}
// the previous block (b vectors, fp32) and R_{i-1} the Cholesky factor of its
// Gram matrix (Y_{i-1}^T Y_{i-1} = R^T R, so Q_i = Y_{i-1} R^-1 is an
// orthonormal basis of its span), pass i computes
//     Y_i = (H Y_{i-1}) R_{i-1}^-1  (= H Q_i)
// on v_mfma_f32_16x16x4_f32 in one read of H, and per workgroup the fp64
// partial sums over its rows of G = Y_i^T Y_i, T = Q_i^T Y_i and
// S = Q_i^T Q_i. A one-workgroup finish sums the partials in a fixed order
// and forms the Ritz values of span(Q_i) as the eigenvalues of
// L_S^-1 T L_S^-T (S = L_S L_S^T; exact even if Q_i is not quite
// orthonormal). The largest one comes from repeated squaring of that b x b
// matrix: after m squarings (trace-normalised) M is proportional to C^(2^m),
// and trace(C M) / trace(M) is within (b - 1) / (e 2^m) relative of
// lambda_max(C) for positive semi-definite C. The finish then factors G for
// the next pass. Directions whose Cholesky pivot falls below 1e-14 of their
// diagonal are numerically dependent and are dropped (their rows and columns
// of the factor's inverse are zero).
//
// Lanczos (optima_spectral_lanczos): the largest Ritz value of the Krylov
// space of one start vector, from the tridiagonal matrix of the symmetric
// Lanczos recurrence with full reorthogonalisation; one HBM-bound GEMV over H
// per step plus small latency-bound kernels (described with them below).
#include "common.h"
#include <mutex>

#include "readback.h"

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

// h . v over d entries by one wave (16-byte loads when VEC4: d % 4 == 0 and
// both rows 16-byte aligned); every lane returns the sum.
template <bool VEC4>
__device__ inline float row_dot(const float* h, const float* v, int64_t d, int lane) {
  float acc0 = 0.f, acc1 = 0.f;
  if (VEC4) {
    const int64_t n4 = d >> 2;
    const float4* h4 = reinterpret_cast<const float4*>(h);
    const float4* v4 = reinterpret_cast<const float4*>(v);
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
    for (int64_t k = lane; k < d; k += 64) acc0 += h[k] * v[k];
  }
  float acc = acc0 + acc1;
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  return acc;
}

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
      const float acc = row_dot<VEC4>(H + row * d, vin, d, lane);
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

// ---------------------------------------------------------------------------
// Subspace iteration (block >= 2)
// ---------------------------------------------------------------------------

constexpr int kMaxBlock = 16;
constexpr int kSubRows = 16;                 // rows of H per workgroup
constexpr int kSubThreads = 512;             // 8 waves: 8 slices of K
constexpr int kGram = kMaxBlock * kMaxBlock;
constexpr int kPart = 3 * kGram;             // G, T, S partials per workgroup
constexpr int kSquarings = 32;
// The squarings stop once no entry of the trace-normalised M moves by more
// than this: M is then the projector onto the top eigenvector, or the next
// eigenvalue is within this relative distance of the top one.
constexpr double kSquareTol = 1e-14;
constexpr double kDropRel = 1e-14;
constexpr int kPitch = kMaxBlock + 1;

struct SubState {
  double theta;  // largest Ritz value of the last pass
  int conv;
  int iters;
};

// Lower Cholesky factor L (A = L L^T) of the leading b x b block of A, which
// is overwritten. Run by all threads of a 256-thread workgroup; thread t owns
// entry (t / 16, t % 16). A pivot not above kDropRel times the column's
// original diagonal (or NaN) drops the direction: its column of L stays 0.
// Step j updates the trailing block straight from column j of A,
// A[i][k] -= A[i][j] A[k][j] / p (= L[i][j] L[k][j]), so that one barrier
// per column suffices and the square root stays off the dependent chain.
__device__ void chol_drop(double (*A)[kPitch], double (*L)[kPitch], double* diag0, int b) {
  const int t = threadIdx.x, i = t >> 4, k = t & 15;
  if (t < kMaxBlock) diag0[t] = A[t][t];
  L[i][k] = 0.0;
  __syncthreads();
  for (int j = 0; j < b; ++j) {
    const double p = A[j][j];
    const bool keep = p > kDropRel * diag0[j];
    if (keep) {
      const double aij = A[i][j];
      if (i > j && k > j && i < b && k < b) A[i][k] -= aij * (A[k][j] / p);
      if (k == j && i >= j && i < b) L[i][j] = i == j ? sqrt(p) : aij / sqrt(p);
    }
    __syncthreads();
  }
}

// X = L^-1 for a lower-triangular L whose zero diagonal entries mark dropped
// directions (their rows and columns of X are 0). Thread c < 16 forms
// column c by forward substitution with the column in registers; the 16
// pivot reciprocals are formed first, in parallel.
__device__ void inv_lower(double (*L)[kPitch], double (*X)[kPitch], int b) {
  const int c = threadIdx.x;
  __shared__ double rpiv[kMaxBlock];
  if (c < kMaxBlock) rpiv[c] = L[c][c] != 0.0 ? 1.0 / L[c][c] : 0.0;
  __syncthreads();
  if (c < kMaxBlock) {
    double xc[kMaxBlock];
#pragma unroll
    for (int i = 0; i < kMaxBlock; ++i) {
      double s = i == c ? 1.0 : 0.0;
#pragma unroll
      for (int k = 0; k < i; ++k) s -= k >= c ? L[i][k] * xc[k] : 0.0;
      xc[i] = (i >= c && i < b && c < b) ? s * rpiv[i] : 0.0;
    }
#pragma unroll
    for (int i = 0; i < kMaxBlock; ++i) X[i][c] = xc[i];
  }
  __syncthreads();
}

// Pass i >= 1 (see the file comment); workgroup blk covers rows
// [16 blk, 16 blk + 16) of the padded row range [0, dpp).
template <bool VEC4>
__global__ void __launch_bounds__(kSubThreads) k_subspace_pass(const float* H, int64_t d,
                                                               int64_t dpp, const float* Yprev,
                                                               float* Ycur, const double* Rinv,
                                                               double* part, SubState* st) {
  if (st->conv) return;
  constexpr int kSlices = kSubThreads / 64;
  __shared__ float red[kSlices][256];
  __shared__ double Rs[kGram];
  __shared__ double Zs[kSubRows][kPitch], Ys[kSubRows][kPitch], Qs[kSubRows][kPitch];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int ks = w;
  const int64_t r0 = int64_t(blockIdx.x) * kSubRows;
  for (int i = tid; i < kGram; i += kSubThreads) Rs[i] = Rinv[i];

  // Z = H Y_{i-1}^T for this workgroup's rows. MFMA lane l supplies row
  // (l % 16) of H and vector (l % 16) of Y at contraction indices
  // 16 c + 4 (l / 16) + {0..3}: four MFMAs per 16-wide chunk c of K, each
  // fed by one 16-byte load per operand. Wave w takes the chunks c = w
  // (mod 8).
  const int64_t row = r0 + (lane & 15);
  const bool row_ok = row < d;
  const float* hrow = H + (row_ok ? row : 0) * d;
  const float* yrow = Yprev + int64_t(lane & 15) * dpp + 4 * (lane >> 4);
  const int kq = 4 * (lane >> 4);
  const int64_t nch = dpp / 16;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  auto load_a = [&](int64_t c) {
    const int64_t k = c * 16 + kq;
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
    if (VEC4) {
      if (row_ok && k < d) a = *reinterpret_cast<const float4*>(hrow + k);
    } else if (row_ok) {
      if (k < d) a.x = hrow[k];
      if (k + 1 < d) a.y = hrow[k + 1];
      if (k + 2 < d) a.z = hrow[k + 2];
      if (k + 3 < d) a.w = hrow[k + 3];
    }
    return a;
  };
  auto mfma4 = [&](float4 a, float4 y) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, y.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, y.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, y.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, y.w, acc, 0, 0, 0);
  };
  int64_t c = ks;
  for (; c + 7 * kSlices < nch; c += 8 * kSlices) {  // eight 16-byte loads per operand in flight
    float4 a[8], y[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      a[u] = load_a(c + kSlices * u);
      y[u] = *reinterpret_cast<const float4*>(yrow + (c + kSlices * u) * 16);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) mfma4(a[u], y[u]);
  }
  for (; c + 3 * kSlices < nch; c += 4 * kSlices) {
    float4 a[4], y[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      a[u] = load_a(c + kSlices * u);
      y[u] = *reinterpret_cast<const float4*>(yrow + (c + kSlices * u) * 16);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) mfma4(a[u], y[u]);
  }
  for (; c < nch; c += kSlices) mfma4(load_a(c), *reinterpret_cast<const float4*>(yrow + c * 16));
#pragma unroll
  for (int e = 0; e < 4; ++e) red[w][e * 64 + lane] = acc[e];
  __syncthreads();
  // Sum the K slices in a fixed order. MFMA output (lane, e) is row
  // 4 (lane / 16) + e, vector lane % 16 of the 16 x 16 tile.
  if (tid < 256) {
    const int ln = tid & 63, e = tid >> 6;
    double z = 0.0;
    for (int q = 0; q < kSlices; ++q) z += double(red[q][e * 64 + ln]);
    Zs[4 * (ln >> 4) + e][ln & 15] = z;
  }
  __syncthreads();
  // Y_i = Z R^-1 (stored in fp32), Q_i = Y_{i-1} R^-1 for these rows.
  if (tid < kSubRows * kMaxBlock) {
    const int r = tid >> 4, a = tid & 15;
    double yn = 0.0, q = 0.0;
    for (int k = 0; k < kMaxBlock; ++k) {
      yn += Zs[r][k] * Rs[k * kMaxBlock + a];
      q += double(Yprev[int64_t(k) * dpp + r0 + r]) * Rs[k * kMaxBlock + a];
    }
    const float yf = float(yn);
    Ycur[int64_t(a) * dpp + r0 + r] = yf;
    Ys[r][a] = double(yf);
    Qs[r][a] = q;
  }
  __syncthreads();
  if (tid < kGram) {
    const int a = tid >> 4, b2 = tid & 15;
    double g = 0.0, tt = 0.0, ss = 0.0;
    for (int r = 0; r < kSubRows; ++r) {
      g += Ys[r][a] * Ys[r][b2];
      tt += Qs[r][a] * Ys[r][b2];
      ss += Qs[r][a] * Qs[r][b2];
    }
    double* P = part + size_t(blockIdx.x) * kPart;
    P[tid] = g;
    P[kGram + tid] = tt;
    P[2 * kGram + tid] = ss;
  }
}

// Y_0 = the caller's start vectors (zero-padded to 16 x dpp) and the partial
// Gram sums of Y_0 over this workgroup's rows.
__global__ void __launch_bounds__(kSubThreads) k_subspace_init(const float* V0, int b, int64_t d,
                                                               int64_t dpp, float* Y0,
                                                               double* part, SubState* st) {
  __shared__ double Ys[kSubRows][kPitch];
  const int tid = threadIdx.x, r = tid >> 4, a = tid & 15;
  const int64_t row = int64_t(blockIdx.x) * kSubRows + r;
  if (r < kSubRows) {
    const float v = (a < b && row < d) ? V0[int64_t(a) * d + row] : 0.f;
    Y0[int64_t(a) * dpp + row] = v;
    Ys[r][a] = double(v);
  }
  if (blockIdx.x == 0 && tid == 0) {
    st->theta = 0.0;
    st->conv = 0;
    st->iters = 0;
  }
  __syncthreads();
  if (tid < kGram) {
    const int i = tid >> 4, j = tid & 15;
    double g = 0.0;
    for (int q = 0; q < kSubRows; ++q) g += Ys[q][i] * Ys[q][j];
    double* P = part + size_t(blockIdx.x) * kPart;
    P[tid] = g;
    P[kGram + tid] = 0.0;
    P[2 * kGram + tid] = 0.0;
  }
}

// Sums the per-workgroup partials of G, T and S (kPart entries each row of
// `part`, nblk rows) into tot[kPart]: workgroup b takes 32 entries, its 8
// thread groups sum 8 contiguous ranges of rows, then the 8 range sums are
// added in order (a fixed order: deterministic).
constexpr int kRedEntries = 32, kRedSegs = 8;
__global__ void __launch_bounds__(256) k_subspace_reduce(const double* part, int nblk,
                                                         double* tot, const SubState* st) {
  if (st->conv) return;
  __shared__ double seg[kRedSegs][kRedEntries];
  const int el = threadIdx.x % kRedEntries, sg = threadIdx.x / kRedEntries;
  const int e = blockIdx.x * kRedEntries + el;
  const int per = (nblk + kRedSegs - 1) / kRedSegs;
  const int k0 = sg * per, k1 = min(nblk, k0 + per);
  double a = 0.0;
#pragma unroll 8
  for (int k = k0; k < k1; ++k) a += part[size_t(k) * kPart + e];  // eight loads in flight
  seg[sg][el] = a;
  __syncthreads();
  if (sg == 0) {
    double t = 0.0;
    for (int q = 0; q < kRedSegs; ++q) t += seg[q][el];
    tot[e] = t;
  }
}

// Finish of pass `it` (0: the start block only). One workgroup of 256.
__global__ void __launch_bounds__(256) k_subspace_finish(const double* tot, int b, int it,
                                                         float tol, double* Rinv, SubState* st,
                                                         float* lambda_out) {
  if (st->conv) return;
  __shared__ double G[kMaxBlock][kPitch], T[kMaxBlock][kPitch], S[kMaxBlock][kPitch];
  __shared__ double L[kMaxBlock][kPitch], X[kMaxBlock][kPitch], W[kMaxBlock][kPitch];
  __shared__ double M[kMaxBlock][kPitch];
  __shared__ double diag0[kMaxBlock], rowsum[kMaxBlock];
  __shared__ int bad;
  const int t = threadIdx.x, i = t >> 4, j = t & 15;
  if (t == 0) bad = 0;
  __syncthreads();
  {
    const double g = tot[t], tt = tot[kGram + t], ss = tot[2 * kGram + t];
    G[i][j] = g;
    T[i][j] = tt;
    S[i][j] = ss;
    if (!isfinite(g) || !isfinite(tt) || !isfinite(ss)) bad = 1;
  }
  __syncthreads();
  if (bad) {
    if (t == 0) {
      *lambda_out = __builtin_nanf("");
      st->iters = it;
      st->conv = 1;
    }
    return;
  }
  if (it >= 1) {
    // C = L_S^-1 T L_S^-T, symmetrised.
    chol_drop(S, L, diag0, b);
    inv_lower(L, X, b);
    double w = 0.0;
    for (int k = 0; k < kMaxBlock; ++k) w += X[i][k] * T[k][j];
    W[i][j] = w;
    __syncthreads();
    double cij = 0.0, cji = 0.0;
    for (int k = 0; k < kMaxBlock; ++k) {
      cij += W[i][k] * X[j][k];
      cji += W[j][k] * X[i][k];
    }
    const double cs = 0.5 * (cij + cji);
    __syncthreads();
    T[i][j] = cs;  // T now holds C
    __syncthreads();
    double tr = 0.0;
    for (int k = 0; k < kMaxBlock; ++k) tr += T[k][k];
    double theta = 0.0;
    if (tr > 0.0) {
      M[i][j] = cs / tr;
      __syncthreads();
      for (int q = 0; q < kSquarings; ++q) {
        double m2 = 0.0;
        for (int k = 0; k < kMaxBlock; ++k) m2 += M[i][k] * M[k][j];
        W[i][j] = m2;
        __syncthreads();
        double tr2 = 0.0;
        for (int k = 0; k < kMaxBlock; ++k) tr2 += W[k][k];
        const double mn = m2 / tr2;
        const bool moved = !(fabs(mn - M[i][j]) <= kSquareTol);
        M[i][j] = mn;
        if (!__syncthreads_or(moved)) break;
      }
      if (t < kMaxBlock) {
        double rs = 0.0;
        for (int k = 0; k < kMaxBlock; ++k) rs += T[t][k] * M[t][k];
        rowsum[t] = rs;
      }
      __syncthreads();
      double num = 0.0, den = 0.0;
      for (int k = 0; k < kMaxBlock; ++k) {
        num += rowsum[k];
        den += M[k][k];
      }
      theta = num / den;
    }
    const bool done = theta == 0.0 ||
                      (it >= 2 && fabs(theta - st->theta) <= double(tol) * fabs(theta));
    __syncthreads();
    if (t == 0) {
      st->theta = theta;
      st->iters = it;
      *lambda_out = float(theta);
      if (done) st->conv = 1;
    }
    if (done) return;
  }
  // Factor of the next pass: G = R^T R with R = L_G^T, so R^-1 = (L_G^-1)^T.
  chol_drop(G, L, diag0, b);
  inv_lower(L, X, b);
  Rinv[i * kMaxBlock + j] = X[j][i];
}

__global__ void k_copy_sub_iters(const SubState* st, int32_t* iters) { *iters = st->iters; }

// ---------------------------------------------------------------------------
// Lanczos
// ---------------------------------------------------------------------------
//
// Step j (0-based) of the symmetric Lanczos process with full
// reorthogonalisation, six launches:
//   k_lz_matvec  q_j = w / ||w|| (w: the previous step's residual, or v0),
//                y = H q_j (one wave per row, HBM-bound), and per workgroup
//                the partial sums of q_i . y, i <= j;
//   k_lz_coef    c_i = q_i . y (fixed-order sums of those partials);
//   k_lz_orth    w = y - sum_i c_i q_i, and partial sums of q_i . w;
//   k_lz_coef    c'_i = q_i . w;
//   k_lz_orth    w <- w - sum_i c'_i q_i, and partial sums of ||w||^2;
//   k_lz_finish  alpha_j = c_j + c'_j, beta_j = ||w||, and the largest
//                eigenvalue of T = tridiag(beta; alpha; beta) by Sturm-count
//                multisection in fp64; the stopping test.
// In exact arithmetic c_i vanishes for i < j - 1, c_(j-1) = beta_(j-1) and
// c_j = alpha_j: the two passes are the three-term recurrence followed by one
// more Gram-Schmidt pass over the whole basis, in classical form. The basis
// is kept in fp32 (pitch dp), every sum in fp64. A set `conv` makes every
// later launch return at once.

constexpr int kLzMax = OPTIMA_LANCZOS_MAX_STEPS;
constexpr int kLzRows = 64;                 // rows per workgroup of k_lz_orth
constexpr int kLzFinThreads = 512;          // multisection points per round
constexpr double kLzBreakdown = 1e-6;       // beta_j <= this * theta_j: K_j invariant
constexpr double kLzWidth = 1e-12;          // relative width that ends the multisection
constexpr int kLzRounds = 8;
constexpr double kLzGeoSpan = 44.0;         // first round: offsets W 2^-44 .. W

struct LzState {
  double alpha[kLzMax];
  double beta[kLzMax];
  double c[2][kLzMax];  // coefficients of the two Gram-Schmidt passes
  double inv;           // 1 / ||w|| of the vector that becomes q_j
  double theta;         // largest Ritz value after the last finished step
  double theta_lo;      // a value not above it (the final bracket's lower end)
  int conv;
  int steps;
};

// w = v0, inv = 1 / ||v0||. A zero start vector ends at once with 0; a
// non-finite one with NaN.
__global__ void __launch_bounds__(1024) k_lz_init(const float* v0, int64_t d, float* w,
                                                  LzState* st, float* lambda_out) {
  __shared__ double red[16];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < d; i += 1024) {
    const float x = v0[i];
    w[i] = x;
    s += double(x) * double(x);
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int k = 0; k < 16; ++k) t += red[k];
    const bool ok = t > 0.0 && isfinite(t);
    st->inv = ok ? 1.0 / sqrt(t) : 0.0;
    st->theta = 0.0;
    st->theta_lo = -INFINITY;
    st->conv = ok ? 0 : 1;
    st->steps = 0;
    *lambda_out = isfinite(t) ? 0.f : __builtin_nanf("");
  }
}

template <bool VEC4>
__global__ void __launch_bounds__(kThreads) k_lz_matvec(const float* H, int64_t d, int64_t dp,
                                                        const float* w, float* Q, int j, float* y,
                                                        double* part, int nblk, LzState* st) {
  if (st->conv) return;
  __shared__ float ys[kRowsPerBlock], qs[kRowsPerBlock];
  const double inv = st->inv;
  float* qj = Q + int64_t(j) * dp;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < kRowsPerWave; ++q) {
    const int lr = wv * kRowsPerWave + q;
    const int64_t row = int64_t(blockIdx.x) * kRowsPerBlock + lr;
    float yr = 0.f, qr = 0.f;
    if (row < d) {
      yr = float(double(row_dot<VEC4>(H + row * d, w, d, lane)) * inv);
      qr = float(double(w[row]) * inv);
      if (lane == 0) {
        y[row] = yr;
        qj[row] = qr;
      }
    }
    if (lane == 0) {
      ys[lr] = yr;
      qs[lr] = qr;
    }
  }
  __syncthreads();
  const int64_t r0 = int64_t(blockIdx.x) * kRowsPerBlock;
  for (int i = threadIdx.x; i <= j; i += kThreads) {
    double sum = 0.0;
    for (int r = 0; r < kRowsPerBlock && r0 + r < d; ++r) {
      const float qv = i == j ? qs[r] : Q[int64_t(i) * dp + r0 + r];
      sum += double(qv) * double(ys[r]);
    }
    part[int64_t(i) * nblk + blockIdx.x] = sum;
  }
}

// c[pass][i] = sum over blocks of part[i][*] in a fixed order, one wave per i.
__global__ void __launch_bounds__(kThreads) k_lz_coef(const double* part, int nblk, int j,
                                                      int pass, LzState* st) {
  if (st->conv) return;
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (i > j) return;
  const double* p = part + int64_t(i) * nblk;
  double s0 = 0.0, s1 = 0.0;
  int b = lane;
  for (; b + 64 < nblk; b += 128) {
    s0 += p[b];
    s1 += p[b + 64];
  }
  if (b < nblk) s0 += p[b];
  double s = s0 + s1;
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if (lane == 0) st->c[pass][i] = s;
}

// One Gram-Schmidt pass over kLzRows rows: w = src - sum_{i<=j} c[pass]_i q_i
// (wave v takes the terms i = v mod 4, summed in LDS in a fixed order). Pass
// 0 then leaves the partial sums of q_i . w in part[i][block]; pass 1 the
// partial ||w||^2 in norm_part[block].
__global__ void __launch_bounds__(kThreads) k_lz_orth(const float* Q, int64_t d, int64_t dp,
                                                      int j, int pass, const float* src,
                                                      float* w, double* part, int nblk,
                                                      double* norm_part, LzState* st) {
  if (st->conv) return;
  constexpr int kW = kThreads / 64;
  __shared__ double sum[kW][kLzRows];
  __shared__ float ws[kLzRows];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t r0 = int64_t(blockIdx.x) * kLzRows, r = r0 + lane;
  const bool in = r < d;
  const double* c = st->c[pass];
  double acc = 0.0;
  if (in)
    for (int i = wv; i <= j; i += kW) acc += c[i] * double(Q[int64_t(i) * dp + r]);
  sum[wv][lane] = acc;
  __syncthreads();
  if (wv == 0) {
    float wr = 0.f;
    if (in) {
      const double t = ((sum[0][lane] + sum[1][lane]) + sum[2][lane]) + sum[3][lane];
      wr = float(double(src[r]) - t);
      w[r] = wr;
    }
    ws[lane] = wr;
  }
  __syncthreads();
  if (pass == 0) {
    for (int i = wv; i <= j; i += kW) {
      double s = in ? double(Q[int64_t(i) * dp + r]) * double(ws[lane]) : 0.0;
      for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
      if (lane == 0) part[int64_t(i) * nblk + blockIdx.x] = s;
    }
  } else if (wv == 0) {
    double s = double(ws[lane]) * double(ws[lane]);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (lane == 0) norm_part[blockIdx.x] = s;
  }
}

// Number of eigenvalues of the n x n tridiagonal matrix below x, from the
// signs of the LDL^T pivots of T - x I (Sturm count). ab[k] holds (a_k,
// b_(k-1)^2), b_(-1)^2 = 0. Pivots smaller than pivmin in magnitude become
// -pivmin. Each pivot's reciprocal is the hardware estimate refined by one
// Newton step (error a few ulps); the count tolerates relative errors of
// that size in the pivots, since they amount to a tiny perturbation of T.
__device__ inline int lz_count_below(const double2* ab, int n, double x, double pivmin) {
  double p = 1.0;  // the pivot before the first one: b_(-1)^2 / p adds nothing
  int cnt = 0;
  for (int k = 0; k < n; ++k) {
    const double2 e = ab[k];
    double r = __builtin_amdgcn_rcp(p);
    r = fma(r, fma(-p, r, 1.0), r);
    p = fma(-e.y, r, e.x - x);
    if (fabs(p) < pivmin) p = -pivmin;
    cnt += p < 0.0;
  }
  return cnt;
}

// Multisection point t of round `round` in [lo, hi]: the first round spaces
// the offsets from lo geometrically (W 2^-44 .. W, W = hi - lo), since the
// top Ritz value moves little from one step to the next; later rounds
// uniformly.
__device__ inline double lz_point(double lo, double hi, int round, int t) {
  if (round == 0)
    return t == kLzFinThreads - 1
               ? hi
               : lo + (hi - lo) * exp2(-kLzGeoSpan * (1.0 - double(t + 1) / kLzFinThreads));
  return lo + (hi - lo) / double(kLzFinThreads + 1) * double(t + 1);
}

// alpha_j, beta_j, theta_j = lambda_max(T_(j+1)) and the stopping decision:
// stop when |theta_j - theta_(j-1)| <= tol theta_j, when beta_j <=
// kLzBreakdown theta_j, or after n_max steps. One workgroup; the largest
// eigenvalue of T to a relative width of kLzWidth.
__global__ void __launch_bounds__(kLzFinThreads) k_lz_finish(const double* norm_part, int nblk,
                                                             int j, int n_max, float tol,
                                                             LzState* st, float* lambda_out) {
  if (st->conv) return;
  constexpr int kW = kLzFinThreads / 64;
  __shared__ double2 ab[kLzMax];
  __shared__ double rs[kW], ramax[kW], rgmax[kW], rbmax[kW];
  __shared__ int rbad[kW];
  __shared__ double lo_s, hi_s;
  __shared__ int first_all;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, n = j + 1;
  const double alpha = st->c[0][j] + st->c[1][j];
  // ||w||^2, and per row of T its diagonal and Gershgorin bound.
  double s = 0.0;
  for (int k = t; k < nblk; k += kLzFinThreads) s += norm_part[k];
  double am = -INFINITY, gm = -INFINITY, bm = 0.0;
  int bad = 0;
  if (t < n) {
    const double a = t == j ? alpha : st->alpha[t];
    const double bl = t > 0 ? st->beta[t - 1] : 0.0, br = t < j ? st->beta[t] : 0.0;
    ab[t] = make_double2(a, bl * bl);
    am = a;
    gm = a + fabs(bl) + fabs(br);
    bm = br * br;
    bad = !(isfinite(a) && isfinite(bl));
  }
  for (int o = 32; o > 0; o >>= 1) {
    s += __shfl_xor(s, o, 64);
    am = fmax(am, __shfl_xor(am, o, 64));
    gm = fmax(gm, __shfl_xor(gm, o, 64));
    bm = fmax(bm, __shfl_xor(bm, o, 64));
    bad |= __shfl_xor(bad, o, 64);
  }
  if (lane == 0) {
    rs[wv] = s;
    ramax[wv] = am;
    rgmax[wv] = gm;
    rbmax[wv] = bm;
    rbad[wv] = bad;
  }
  __syncthreads();
  double beta2 = 0.0, amax = -INFINITY, gmax = -INFINITY, bmax = 0.0;
  for (int k = 0; k < kW; ++k) {
    beta2 += rs[k];
    amax = fmax(amax, ramax[k]);
    gmax = fmax(gmax, rgmax[k]);
    bmax = fmax(bmax, rbmax[k]);
    bad |= rbad[k];
  }
  const bool finite = !bad && isfinite(beta2);
  double theta;
  if (!finite) {
    theta = __builtin_nan("");
  } else {
    // lambda_max(T) lies in [max(a_k, theta_lo of the previous step),
    // Gershgorin bound]: a diagonal entry is a Rayleigh quotient, and T_j
    // contains T_(j-1) as a leading block (Cauchy interlacing).
    const double pivmin = 1e-290 * fmax(1.0, bmax);
    if (t == 0) {
      lo_s = fmax(amax, st->theta_lo);
      hi_s = gmax + fmax(fabs(gmax) * 1e-14, 1e-300);
    }
    __syncthreads();
    for (int round = 0; round < kLzRounds; ++round) {
      const double lo = lo_s, hi = hi_s;
      if (hi - lo <= kLzWidth * fmax(fabs(lo), fabs(hi))) break;
      const double x = lz_point(lo, hi, round, t);
      if (t == 0) first_all = kLzFinThreads;
      __syncthreads();
      // count(x_t) is non-decreasing in t; the top eigenvalue lies between the
      // last point with fewer than n eigenvalues below it and the first with n.
      if (lz_count_below(ab, n, x, pivmin) == n) atomicMin(&first_all, t);
      __syncthreads();
      if (t == 0) {
        const int f = first_all;
        lo_s = f == 0 ? lo : lz_point(lo, hi, round, f - 1);
        hi_s = f == kLzFinThreads ? hi : lz_point(lo, hi, round, f);
      }
      __syncthreads();
    }
    theta = 0.5 * (lo_s + hi_s);
  }
  if (t == 0) {
    const double beta = sqrt(beta2);
    const bool done = !finite || n >= n_max ||
                      (j >= 1 && fabs(theta - st->theta) <= double(tol) * fabs(theta)) ||
                      beta <= kLzBreakdown * fabs(theta);
    st->alpha[j] = alpha;
    st->beta[j] = beta;
    st->theta = theta;
    st->theta_lo = finite ? lo_s : -INFINITY;
    st->steps = n;
    st->inv = done ? 0.0 : 1.0 / beta;
    *lambda_out = float(theta);
    if (done) st->conv = 1;
  }
}

__global__ void k_copy_lz_steps(const LzState* st, int32_t* steps) { *steps = st->steps; }

}  // namespace

size_t spectral_norm_workspace_bytes(int64_t d, int block) {
  Carver c(nullptr);
  if (block == 1) {
    c.take<float>(size_t(d));
    c.take<float>(size_t(d));
    c.take<double2>(2 * size_t(ceil_div(d, kRowsPerBlock)));
    c.take<PowState>(1);
  } else {
    const int64_t dpp = round_up(d, kSubRows);
    c.take<float>(size_t(kMaxBlock) * size_t(dpp));
    c.take<float>(size_t(kMaxBlock) * size_t(dpp));
    c.take<double>(size_t(dpp / kSubRows) * kPart);
    c.take<double>(kPart);
    c.take<double>(kGram);
    c.take<SubState>(1);
  }
  return c.bytes();
}

namespace {

optima_status power_iteration(const float* H, int64_t d, const float* v0, int max_iters, float tol,
                              void* ws, float* lambda_max, int32_t* iters, bool plain_waits,
                              hipStream_t s) {
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
      OPTIMA_HIP_TRY(plain_waits ? read_back_plain(&conv, &st->conv, sizeof(int), s)
                                 : read_back(&conv, &st->conv, sizeof(int), s));
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
  OPTIMA_HIP_TRY(plain_waits ? wait_stream_plain(s) : wait_stream(s));
  return OPTIMA_OK;
}

optima_status subspace_iteration(const float* H, int64_t d, const float* V0, int b,
                                 int max_iters, float tol, void* ws, float* lambda_max,
                                 int32_t* iters, bool plain_waits, hipStream_t s) {
  const int64_t dpp = round_up(d, kSubRows);
  const int nblk = int(dpp / kSubRows);
  Carver c(ws);
  float* Y[2] = {c.take<float>(size_t(kMaxBlock) * size_t(dpp)),
                 c.take<float>(size_t(kMaxBlock) * size_t(dpp))};
  double* part = c.take<double>(size_t(nblk) * kPart);
  double* tot = c.take<double>(kPart);
  double* Rinv = c.take<double>(kGram);
  SubState* st = c.take<SubState>(1);
  const dim3 rg(unsigned(kPart / kRedEntries));
  hipLaunchKernelGGL(k_subspace_init, dim3(unsigned(nblk)), dim3(kSubThreads), 0, s, V0, b, d,
                     dpp, Y[0], part, st);
  OPTIMA_LAUNCH_CHECK();
  hipLaunchKernelGGL(k_subspace_reduce, rg, dim3(256), 0, s, part, nblk, tot, st);
  OPTIMA_LAUNCH_CHECK();
  hipLaunchKernelGGL(k_subspace_finish, dim3(1), dim3(256), 0, s, tot, b, 0, tol, Rinv, st,
                     lambda_max);
  OPTIMA_LAUNCH_CHECK();
  const bool vec4 = (d % 4) == 0 && aligned16(H);
  constexpr int kPoll = 4;
  for (int it = 1; it <= max_iters; ++it) {
    if (vec4)
      hipLaunchKernelGGL(k_subspace_pass<true>, dim3(unsigned(nblk)), dim3(kSubThreads), 0, s, H,
                         d, dpp, Y[(it - 1) & 1], Y[it & 1], Rinv, part, st);
    else
      hipLaunchKernelGGL(k_subspace_pass<false>, dim3(unsigned(nblk)), dim3(kSubThreads), 0, s, H,
                         d, dpp, Y[(it - 1) & 1], Y[it & 1], Rinv, part, st);
    OPTIMA_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_subspace_reduce, rg, dim3(256), 0, s, part, nblk, tot, st);
    OPTIMA_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_subspace_finish, dim3(1), dim3(256), 0, s, tot, b, it, tol, Rinv, st,
                       lambda_max);
    OPTIMA_LAUNCH_CHECK();
    if (it % kPoll == 0 && it < max_iters) {
      int conv = 0;
      OPTIMA_HIP_TRY(plain_waits ? read_back_plain(&conv, &st->conv, sizeof(int), s)
                                 : read_back(&conv, &st->conv, sizeof(int), s));
      if (conv) break;
    }
  }
  if (iters) {
    hipLaunchKernelGGL(k_copy_sub_iters, dim3(1), dim3(1), 0, s, st, iters);
    OPTIMA_LAUNCH_CHECK();
  }
  OPTIMA_HIP_TRY(plain_waits ? wait_stream_plain(s) : wait_stream(s));
  return OPTIMA_OK;
}

// Workspace of the Lanczos process for at most m steps: the basis (m rows of
// pitch dp), y, w, the partial sums of both passes and of the norm, state.
struct LzLayout {
  float *Q, *y, *w;
  double *part1, *part2, *norm_part;
  LzState* st;
  int64_t dp;
  int nblk1, nblk2;
};

LzLayout lz_layout(void* ws, int64_t d, int m, size_t* bytes) {
  Carver c(ws);
  LzLayout l{};
  l.dp = round_up(d, 64);
  l.nblk1 = int(ceil_div(d, kRowsPerBlock));
  l.nblk2 = int(ceil_div(d, kLzRows));
  l.Q = c.take<float>(size_t(m) * size_t(l.dp));
  l.y = c.take<float>(size_t(l.dp));
  l.w = c.take<float>(size_t(l.dp));
  l.part1 = c.take<double>(size_t(m) * size_t(l.nblk1));
  l.part2 = c.take<double>(size_t(m) * size_t(l.nblk2));
  l.norm_part = c.take<double>(size_t(l.nblk2));
  l.st = c.take<LzState>(1);
  if (bytes) *bytes = c.bytes();
  return l;
}

}  // namespace

optima_status spectral_norm(const float* H, int64_t d, const float* V0, int block, int max_iters,
                            float tol, void* ws, float* lambda_max, int32_t* iters,
                            hipStream_t s) {
  if (block == 1)
    return power_iteration(H, d, V0, max_iters, tol, ws, lambda_max, iters, false, s);
  return subspace_iteration(H, d, V0, block, max_iters, tol, ws, lambda_max, iters, false, s);
}

// ---------------------------------------------------------------------------
// The spectral norm without allocation: the work buffer is `scratch`, a
// fixed array of the library's code object (one copy per device, kept until
// the process ends), and the host waits land in host stack memory.
// ---------------------------------------------------------------------------
namespace {

// Covers spectral_norm_workspace_bytes(d, block) for every d <=
// OPTIMA_SPECTRAL_NOALLOC_MAX_DIM and block <= kMaxBlock: two blocks of 16
// fp32 vectors (2 MiB at d = 16384), the fp64 partial Gram sums of 16-row
// slabs (6 MiB) and a few KiB of sums and state.
constexpr size_t kScratchBytes = OPTIMA_SPECTRAL_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes == (size_t(8) << 20) + (size_t(64) << 10), "scratch size");
constexpr int kScratchDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

// Device address of `scratch` per device. In host code the array's name is
// only a host-side stand-in for the symbol; its device address comes from
// hipGetSymbolAddress, looked up once per device with that device current.
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices];

hipError_t scratch_for(hipStream_t s, void** out) {
  int dev = 0;
  hipError_t e = hipStreamGetDevice(s, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

optima_status spectral_norm_noalloc(const float* H, int64_t d, const float* V0, int block,
                                    int max_iters, float tol, float* lambda_max, int32_t* iters,
                                    hipStream_t s) {
  if (d > OPTIMA_SPECTRAL_NOALLOC_MAX_DIM ||
      spectral_norm_workspace_bytes(d, block) > kScratchBytes)
    return OPTIMA_E_WORKSPACE;
  void* ws = nullptr;
  OPTIMA_HIP_TRY(scratch_for(s, &ws));
  // The iterations initialise every piece of the buffer they read, so the
  // contents left by an earlier call need no clearing.
  if (block == 1)
    return power_iteration(H, d, V0, max_iters, tol, ws, lambda_max, iters, true, s);
  return subspace_iteration(H, d, V0, block, max_iters, tol, ws, lambda_max, iters, true, s);
}

size_t spectral_lanczos_workspace_bytes(int64_t d, int max_steps) {
  size_t bytes = 0;
  lz_layout(nullptr, d, int(std::min<int64_t>(max_steps, d)), &bytes);
  return bytes;
}

optima_status spectral_lanczos(const float* H, int64_t d, const float* v0, int max_steps,
                               float tol, void* ws, float* lambda_max, int32_t* steps,
                               hipStream_t s) {
  const int m = int(std::min<int64_t>(max_steps, d));
  const LzLayout l = lz_layout(ws, d, m, nullptr);
  hipLaunchKernelGGL(k_lz_init, dim3(1), dim3(1024), 0, s, v0, d, l.w, l.st, lambda_max);
  OPTIMA_LAUNCH_CHECK();
  const bool vec4 = (d % 4) == 0 && aligned16(H);
  constexpr int kPoll = 8;
  for (int j = 0; j < m; ++j) {
    if (vec4)
      hipLaunchKernelGGL(k_lz_matvec<true>, dim3(unsigned(l.nblk1)), dim3(kThreads), 0, s, H, d,
                         l.dp, l.w, l.Q, j, l.y, l.part1, l.nblk1, l.st);
    else
      hipLaunchKernelGGL(k_lz_matvec<false>, dim3(unsigned(l.nblk1)), dim3(kThreads), 0, s, H, d,
                         l.dp, l.w, l.Q, j, l.y, l.part1, l.nblk1, l.st);
    OPTIMA_LAUNCH_CHECK();
    const dim3 cg(unsigned(ceil_div(j + 1, kThreads / 64)));
    hipLaunchKernelGGL(k_lz_coef, cg, dim3(kThreads), 0, s, l.part1, l.nblk1, j, 0, l.st);
    OPTIMA_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_lz_orth, dim3(unsigned(l.nblk2)), dim3(kThreads), 0, s, l.Q, d, l.dp, j,
                       0, l.y, l.w, l.part2, l.nblk2, l.norm_part, l.st);
    OPTIMA_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_lz_coef, cg, dim3(kThreads), 0, s, l.part2, l.nblk2, j, 1, l.st);
    OPTIMA_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_lz_orth, dim3(unsigned(l.nblk2)), dim3(kThreads), 0, s, l.Q, d, l.dp, j,
                       1, l.w, l.w, l.part2, l.nblk2, l.norm_part, l.st);
    OPTIMA_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_lz_finish, dim3(1), dim3(kLzFinThreads), 0, s, l.norm_part, l.nblk2, j,
                       m, tol, l.st, lambda_max);
    OPTIMA_LAUNCH_CHECK();
    if ((j + 1) % kPoll == 0 && j + 1 < m) {
      int conv = 0;
      OPTIMA_HIP_TRY(read_back(&conv, &l.st->conv, sizeof(int), s));
      if (conv) break;
    }
  }
  if (steps) {
    hipLaunchKernelGGL(k_copy_lz_steps, dim3(1), dim3(1), 0, s, l.st, steps);
    OPTIMA_LAUNCH_CHECK();
  }
  OPTIMA_HIP_TRY(wait_stream(s));
  return OPTIMA_OK;
}

}  // namespace optima
