// Joint scale solve of the scale update (paper eq. (6), App. E.2): one
// wavefront per row.
//
// The G x G Gram matrix (upper triangle from the Gram kernel, symmetrised by
// construction) and the right-hand side r_a = c_a^T (W H)_a are held in LDS in
// fp64 and factored by a right-looking Cholesky.  The stabilised branch of
// App. E.2 (add lambda I and factor again) is taken when an entry is not
// finite, a pivot is not positive, or the smallest pivot is at most
// r_cond * max(largest diagonal, 2^-23).  Every Cholesky pivot is a Schur
// complement and bounded below by the smallest eigenvalue, and the largest
// diagonal bounds the largest eigenvalue from below, so this test only fires
// where the paper's eigenvalue test fires.  A second failure leaves the row's
// scales unchanged and is counted.
#include "jarq_internal.h"

namespace jarq {

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ double wave_min(double x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmin(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ double wave_max(double x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmax(x, __shfl_xor(x, off));
  return x;
}

// In-place Cholesky of the lower triangle of A (G x G, leading dimension LD).
// Returns the smallest pivot before the square root (<= 0 or NaN on failure).
__device__ double chol_lower(double* A, int G, int LD, int lane) {
  double minpiv = INFINITY;
  for (int k = 0; k < G; ++k) {
    const double piv = A[k * LD + k];
    minpiv = fmin(minpiv, piv);
    if (!(piv > 0.0) || !isfinite(piv)) return piv > 0.0 ? NAN : piv;
    const double d = sqrt(piv);
    __syncthreads();
    if (lane == 0) A[k * LD + k] = d;
    for (int i = k + 1 + lane; i < G; i += 64) A[i * LD + k] /= d;
    __syncthreads();
    for (int i = k + 1 + lane; i < G; i += 64) {
      const double lik = A[i * LD + k];
      for (int j = k + 1; j <= i; ++j) A[i * LD + j] -= lik * A[j * LD + k];
    }
    __syncthreads();
  }
  return minpiv;
}

__global__ __launch_bounds__(64) void solve_kernel(int rows, int cols, int g,
                                                   const float* __restrict__ gram,
                                                   const float* __restrict__ wh,
                                                   const uint8_t* __restrict__ codes,
                                                   const int32_t* __restrict__ zeros,
                                                   float* __restrict__ scales,
                                                   const uint8_t* __restrict__ active,
                                                   Counters* __restrict__ cnt,
                                                   Flags* __restrict__ flags, float lam,
                                                   float rcond) {
  const int G = cols / g;
  const int LD = G + 1;
  const int row = blockIdx.x;
  const int lane = threadIdx.x;
  if (row >= rows) return;
  if (active != nullptr && !active[row]) return;
  extern __shared__ double sm[];
  double* A = sm;              // G x LD: lower = factor, strict upper = original
  double* diag = A + G * LD;   // original diagonal
  double* r = diag + G;        // right-hand side, then the solution
  const float* gr = gram + (size_t)row * G * G;
  bool finite = true;
  double dmax = 0.0;
  for (int e = lane; e < G * G; e += 64) {
    const int i = e / G, h = e % G;
    const float v = (h >= i) ? gr[i * G + h] : gr[h * G + i];
    finite &= isfinite(v);
    A[i * LD + h] = (double)v;
    if (i == h) {
      diag[i] = (double)v;
      dmax = fmax(dmax, (double)v);
    }
  }
  // r_a = sum over the group of c * (W H)
  for (int a = lane; a < G; a += 64) {
    const int z = zeros[(size_t)row * G + a];
    const float* whp = wh + (size_t)row * cols + (size_t)a * g;
    const uint8_t* qp = codes + (size_t)row * cols + (size_t)a * g;
    double s = 0.0;
    for (int c = 0; c < g; c += 4) {
      const f32x4 w4 = *(const f32x4*)(whp + c);
      const uint32_t q4 = *(const uint32_t*)(qp + c);
#pragma unroll
      for (int i = 0; i < 4; ++i) s += (double)((int)((q4 >> (8 * i)) & 0xffu) - z) * (double)w4[i];
    }
    r[a] = s;
    finite &= isfinite(s);
  }
  const bool all_finite = __all(finite);
  dmax = wave_max(dmax);
  __syncthreads();

  bool ridge = !all_finite;
  double minpiv = 0.0;
  if (!ridge) {
    minpiv = chol_lower(A, G, LD, lane);
    ridge = !(minpiv > (double)rcond * fmax(dmax, (double)kFp32Eps)) || !isfinite(minpiv);
  }
  if (ridge) {
    __syncthreads();
    for (int e = lane; e < G * G; e += 64) {
      const int i = e / G, h = e % G;
      if (h < i) A[i * LD + h] = A[h * LD + i];
      if (h == i) A[i * LD + i] = diag[i] + (double)lam;
    }
    __syncthreads();
    minpiv = chol_lower(A, G, LD, lane);
    if (!(minpiv > 0.0) || !isfinite(minpiv)) {
      if (lane == 0) {
        atomicAdd(&cnt->solve_failed, 1u);
        atomicAdd(&flags->solve_failed, 1);
        atomicAdd(&cnt->ridge_rows, 1u);
      }
      return;  // keep the previous scales of this row
    }
    if (lane == 0) atomicAdd(&cnt->ridge_rows, 1u);
  }
  __syncthreads();
  // Forward substitution L y = r, then L^T s = y (right-looking, lanes over rows).
  for (int k = 0; k < G; ++k) {
    if (lane == 0) r[k] /= A[k * LD + k];
    __syncthreads();
    const double yk = r[k];
    for (int i = k + 1 + lane; i < G; i += 64) r[i] -= A[i * LD + k] * yk;
    __syncthreads();
  }
  for (int k = G - 1; k >= 0; --k) {
    if (lane == 0) r[k] /= A[k * LD + k];
    __syncthreads();
    const double sk = r[k];
    for (int i = lane; i < k; i += 64) r[i] -= A[k * LD + i] * sk;
    __syncthreads();
  }
  for (int a = lane; a < G; a += 64) scales[(size_t)row * G + a] = (float)r[a];
}

hipError_t launch_solve(hipStream_t st, int rows, int cols, int g, const float* gram,
                        const float* wh, const uint8_t* codes, const int32_t* zeros,
                        float* scales, const uint8_t* active, Counters* cnt, Flags* flags,
                        float lam, float rcond) {
  const int G = cols / g;
  const size_t lds = ((size_t)G * (G + 1) + 2 * (size_t)G) * sizeof(double);
  hipError_t e = hipFuncSetAttribute((const void*)solve_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(solve_kernel, dim3(rows), dim3(64), lds, st, rows, cols, g, gram, wh, codes,
                     zeros, scales, active, cnt, flags, lam, rcond);
  return hipGetLastError();
}

}  // namespace jarq
