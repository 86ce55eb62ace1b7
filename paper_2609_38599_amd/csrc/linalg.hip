// Dense fp64 kernels of the per-layer set-up: a blocked Cholesky factorization
// and the matrix products it and the GPTQ-style host are built from.
//
// Cholesky (right-looking, 64-column blocks): for each diagonal block,
// factor it in LDS and invert its factor (one work-group), scale the panel
// below by the inverse transpose, and subtract the panel's outer product from
// the lower triangle of the trailing matrix.  Everything is fp64; the MI355X
// runs fp64 vector FMAs at the rate of its fp64 matrix cores, so the products
// are register-blocked vector code.
#include "jarq_internal.h"

namespace jarq {

namespace {
constexpr int LT = 64;   // output tile edge of the products, and the Cholesky block size
constexpr int LK = 16;   // k-step of the products
constexpr int LP = LT + 4;
}  // namespace

// C[i][j] (+)= alpha sum_{k in slice z} A[i][k] B(j, k) for i < M, j < N, with
// B(j, k) = B[j][k] (B row-major over j) or, when BK, B[k][j] (row-major over k),
// the k range split into slices of `kslice` (slice z = blockIdx.z writes
// C + z * cz).  LOWER: only j <= i is computed and written (tiles wholly above
// the diagonal exit at once).  A work-group reads rows i0..i0+63 of A and
// j0..j0+63 of B for its own k range before it writes its tile, so A may
// alias C when N <= 64 and the tile's k range is all of K (the panel step).
template <bool LOWER, bool BK>
__global__ __launch_bounds__(256) void gemm_nt_f64_kernel(int M, int N, int K, int kslice,
                                                          double alpha, const double* A,
                                                          long long lda, const double* B,
                                                          long long ldb, double* C,
                                                          long long ldc, long long cz,
                                                          int accumulate) {
  const int i0 = blockIdx.y * LT, j0 = blockIdx.x * LT;
  if (LOWER && j0 > i0 + LT - 1) return;
  __shared__ double as[LK][LP];
  __shared__ double bs[LK][LP];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int k_begin = blockIdx.z * kslice;
  const int k_end = min(K, k_begin + kslice);
  C += (long long)blockIdx.z * cz;
  double acc[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[u][v] = 0.0;
  // Loads: thread t takes row t / 4 of the tile and 4 consecutive k at 4 (t % 4).
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  for (int k0 = k_begin; k0 < k_end; k0 += LK) {
    double ra[4], rb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = k0 + lk + u;
      const bool kin = k < k_end;
      ra[u] = (kin && i0 + lr < M) ? A[(long long)(i0 + lr) * lda + k] : 0.0;
      if (BK) {
        // thread t: k row t / 16, four consecutive j at 4 (t % 16)
        const int kb = k0 + (tid >> 4), jb = j0 + (tid & 15) * 4 + u;
        rb[u] = (kb < k_end && jb < N) ? B[(long long)kb * ldb + jb] : 0.0;
      } else {
        rb[u] = (kin && j0 + lr < N) ? B[(long long)(j0 + lr) * ldb + k] : 0.0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      as[lk + u][lr] = ra[u];
      if (BK)
        bs[tid >> 4][(tid & 15) * 4 + u] = rb[u];
      else
        bs[lk + u][lr] = rb[u];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < LK; ++k) {
      double a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] = as[k][ty * 4 + u];
#pragma unroll
      for (int v = 0; v < 4; ++v) b[v] = bs[k][tx * 4 + v];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fma(a[u], b[v], acc[u][v]);
    }
  }
  // All reads of A and B by this work-group are done before any write.
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = i0 + ty * 4 + u;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int j = j0 + tx * 4 + v;
      if (i < M && j < N && (!LOWER || j <= i)) {
        double* c = C + (long long)i * ldc + j;
        *c = accumulate ? fma(alpha, acc[u][v], *c) : alpha * acc[u][v];
      }
    }
  }
}

static hipError_t launch_gemm_f64(hipStream_t st, bool lower, bool bk, int M, int N, int K,
                                  int kslice, double alpha, const double* A, long long lda,
                                  const double* B, long long ldb, double* C, long long ldc,
                                  long long cz, bool accumulate) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (kslice <= 0) kslice = K > 0 ? K : 1;
  const int nz = K > 0 ? (K + kslice - 1) / kslice : 1;
  dim3 grid((N + LT - 1) / LT, (M + LT - 1) / LT, nz);
  if (lower)
    hipLaunchKernelGGL((gemm_nt_f64_kernel<true, false>), grid, dim3(256), 0, st, M, N, K, kslice,
                       alpha, A, lda, B, ldb, C, ldc, cz, (int)accumulate);
  else if (bk)
    hipLaunchKernelGGL((gemm_nt_f64_kernel<false, true>), grid, dim3(256), 0, st, M, N, K, kslice,
                       alpha, A, lda, B, ldb, C, ldc, cz, (int)accumulate);
  else
    hipLaunchKernelGGL((gemm_nt_f64_kernel<false, false>), grid, dim3(256), 0, st, M, N, K, kslice,
                       alpha, A, lda, B, ldb, C, ldc, cz, (int)accumulate);
  return hipGetLastError();
}

hipError_t launch_gemm_nt_f64(hipStream_t st, bool lower, int M, int N, int K, int kslice,
                              double alpha, const double* A, long long lda, const double* B,
                              long long ldb, double* C, long long ldc, long long cz,
                              bool accumulate) {
  return launch_gemm_f64(st, lower, false, M, N, K, kslice, alpha, A, lda, B, ldb, C, ldc, cz,
                         accumulate);
}

hipError_t launch_gemm_nn_f64_sliced(hipStream_t st, int M, int N, int K, int kslice,
                                     double alpha, const double* A, long long lda,
                                     const double* B, long long ldb, double* C, long long ldc,
                                     long long cz) {
  return launch_gemm_f64(st, false, true, M, N, K, kslice, alpha, A, lda, B, ldb, C, ldc, cz,
                         false);
}

hipError_t launch_gemm_nn_f64(hipStream_t st, int M, int N, int K, double alpha, const double* A,
                              long long lda, const double* B, long long ldb, double* C,
                              long long ldc, bool accumulate) {
  return launch_gemm_f64(st, false, true, M, N, K, K, alpha, A, lda, B, ldb, C, ldc, 0,
                         accumulate);
}

// Factor the nb x nb diagonal block at A (leading dimension lda, lower part
// read and written) as L L^T, and write L^{-1} (lower, zeros above) to
// Linv [64][64].  A pivot that is not positive and finite sets *flag and is
// replaced by 1 so that the factorization runs to its end.
__global__ __launch_bounds__(256) void potrf_diag_kernel(double* __restrict__ A, long long lda,
                                                         int nb, double* __restrict__ Linv,
                                                         int* __restrict__ flag) {
  __shared__ double L[LT][LT + 1];
  __shared__ double X[LT][LT + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < LT * LT; e += 256) {
    const int i = e / LT, j = e % LT;
    L[i][j] = (i < nb && j <= i) ? A[(long long)i * lda + j] : 0.0;
  }
  __syncthreads();
  // Trailing updates on a 16 x 16 thread grid: thread (ty, tx) owns rows
  // ty + 16 a and columns tx + 16 b of the block (no index division).
  const int tx = tid & 15, ty = tid >> 4;
  for (int j = 0; j < nb; ++j) {
    double piv = L[j][j];
    const bool bad = !(piv > 0.0) || !isfinite(piv);
    const double dj = bad ? 1.0 : sqrt(piv);
    __syncthreads();  // every thread has read L[j][j]
    if (tid == 0) {
      L[j][j] = dj;
      if (bad) *flag = 1;
    }
    if (tid > j && tid < nb) L[tid][j] /= dj;
    __syncthreads();
#pragma unroll
    for (int a = 0; a < LT / 16; ++a) {
      const int i = ty + 16 * a;
      if (i > j && i < nb) {
        const double lij = L[i][j];
#pragma unroll
        for (int b = 0; b < LT / 16; ++b) {
          const int k = tx + 16 * b;
          if (k > j && k <= i) L[i][k] = fma(-lij, L[k][j], L[i][k]);
        }
      }
    }
    __syncthreads();
  }
  for (int e = tid; e < nb * nb; e += 256) {
    const int i = e / nb, j = e % nb;
    if (j <= i) A[(long long)i * lda + j] = L[i][j];
  }
  // L^{-1} row by row: X[i][i] = 1 / L[i][i] and, for c < i,
  // X[i][c] = -(sum_{t=c}^{i-1} L[i][t] X[t][c]) / L[i][i].  Thread 4 c + q
  // takes column c and every fourth t from c + q; the four partial sums are
  // added across the four adjacent lanes.
  {
    const int c = tid >> 2, q = tid & 3;
    if (q == 0 && c < nb) X[c][c] = 1.0 / L[c][c];
    __syncthreads();
    for (int i = 1; i < nb; ++i) {
      double s = 0.0;
      if (c < i)
        for (int t = c + q; t < i; t += 4) s = fma(L[i][t], X[t][c], s);
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      if (c < i && q == 0) X[i][c] = -s / L[i][i];
      __syncthreads();
    }
  }
  for (int e = tid; e < LT * LT; e += 256) {
    const int i = e / LT, j = e % LT;
    Linv[e] = (i < nb && j < nb && j <= i) ? X[i][j] : 0.0;
  }
}

// In-place lower Cholesky factor of A [d][d] (leading dimension lda; the
// strict upper part is neither read nor written).  Linv: 64 x 64 fp64 scratch,
// or, with keep_inverses, one 64 x 64 block per diagonal block (block b at
// Linv + 4096 b holds the inverse of the factor's diagonal block b).  *flag is
// set when a pivot is not positive (the caller clears it first).
hipError_t launch_potrf_f64(hipStream_t st, double* A, int d, long long lda, double* Linv_base,
                            int* flag, bool keep_inverses) {
  for (int k0 = 0; k0 < d; k0 += LT) {
    const int nb = min(LT, d - k0);
    double* Linv = keep_inverses ? Linv_base + (long long)(k0 / LT) * LT * LT : Linv_base;
    double* akk = A + (long long)k0 * lda + k0;
    hipLaunchKernelGGL(potrf_diag_kernel, dim3(1), dim3(256), 0, st, akk, lda, nb, Linv, flag);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int rest = d - k0 - nb;
    if (rest <= 0) break;
    double* panel = A + (long long)(k0 + nb) * lda + k0;
    // panel = panel L_kk^{-T}: row i of the panel times row j of L_kk^{-1}
    e = launch_gemm_nt_f64(st, false, rest, nb, nb, nb, 1.0, panel, lda, Linv, LT, panel, lda, 0,
                           false);
    if (e != hipSuccess) return e;
    // trailing lower triangle -= panel panel^T
    double* trail = A + (long long)(k0 + nb) * lda + (k0 + nb);
    e = launch_gemm_nt_f64(st, true, rest, rest, nb, nb, -1.0, panel, lda, panel, lda, trail, lda,
                           0, true);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Lower part of H in fp64: C[i][j] = H[i][j], or with reverse the Hessian
// with its channel order reversed, C[i][j] = H[d-1-i][d-1-j].
__global__ __launch_bounds__(256) void copy_lower_kernel(const float* __restrict__ H, int d,
                                                         int reverse, double* __restrict__ C) {
  const long long n = (long long)d * d;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256) {
    const int i = (int)(e / d), j = (int)(e % d);
    if (j <= i)
      C[e] = (double)(reverse ? H[(long long)(d - 1 - i) * d + (d - 1 - j)] : H[e]);
  }
}

// M[k][t] = C[d-1-t][d-1-k] for t <= k (reflection about the anti-diagonal,
// which maps a lower triangle onto a lower triangle), 32 x 32 tiles through LDS.
__global__ __launch_bounds__(256) void antitranspose_lower_kernel(const double* __restrict__ C,
                                                                  int d, double* __restrict__ M) {
  __shared__ double tile[32][33];
  const int k0 = blockIdx.y * 32, t0 = blockIdx.x * 32;
  if (t0 > k0 + 31) return;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // ty < 8
  // The source block holds rows d-1-t and columns d-1-k: read row r = d-1-(t0+31-a)
  // for a = 0..31 with consecutive columns.
  for (int a = ty; a < 32; a += 8) {
    const int t = t0 + 31 - a, k = k0 + 31 - tx;
    if (t < d && k < d && t <= k) tile[a][tx] = C[(long long)(d - 1 - t) * d + (d - 1 - k)];
  }
  __syncthreads();
  for (int a = ty; a < 32; a += 8) {
    const int k = k0 + a, t = t0 + tx;
    if (k < d && t < d && t <= k) M[(long long)k * d + t] = tile[31 - tx][31 - a];
  }
}

hipError_t launch_copy_lower(hipStream_t st, const float* H, int d, bool reverse, double* C) {
  const long long n = (long long)d * d;
  const long long blocks = (n + 255) / 256 < 16384 ? (n + 255) / 256 : 16384;
  hipLaunchKernelGGL(copy_lower_kernel, dim3((unsigned)blocks), dim3(256), 0, st, H, d,
                     (int)reverse, C);
  return hipGetLastError();
}

hipError_t launch_antitranspose_lower(hipStream_t st, const double* C, int d, double* M) {
  const int nt = (d + 31) / 32;
  hipLaunchKernelGGL(antitranspose_lower_kernel, dim3(nt, nt), dim3(256), 0, st, C, d, M);
  return hipGetLastError();
}

}  // namespace jarq
