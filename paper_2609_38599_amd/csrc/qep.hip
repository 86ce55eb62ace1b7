// Propagation-corrected target (App. E.5, eqs. (mu-target) and (w-corr)).
// Mixing the full-precision response into the target, Y(mu) = (1 - mu) X W +
// mu X~ W, makes the refinement problem the main one with W replaced by
//   W_corr = W + (1 - mu) H^{-1} X~^T (X - X~) W        (columns = output channels),
// H = X~^T X~ + nu^2 I.  With rows as output channels (this library's layout)
// and D = X~^T (X - X~):   W_corr = W + (1 - mu) (W D^T) H^{-1}.
//
// On the GPU, in fp64: T = W D^T (one product), H = L L^T (blocked Cholesky,
// keeping the inverse of every 64 x 64 diagonal block), then T H^{-1} by two
// blocked triangular solves over 64-column blocks of T, in place:
//   forward   Y L^T = T:  Y_k = (T_k - Y_{<k} L_{k,<k}^T) L_kk^{-T},
//   backward  Z L   = Y:  Z_k = (Y_k - Z_{>k} L_{>k,k}) L_kk^{-1},
// and W_corr = W + (1 - mu) Z rounded once to fp32.
#include "jarq_internal.h"

namespace jarq {

namespace {
constexpr int QB = 64;
constexpr int kMaxSlices = 8;   // k-slices of the off-diagonal updates of the solves
size_t al(size_t x) { return (x + 255) & ~size_t(255); }
// k-slice length for a K-long update: at most kMaxSlices slices, 16-aligned
int slice_of(int K) {
  const int s = (K + kMaxSlices - 1) / kMaxSlices;
  return ((s + 15) / 16) * 16;
}
}  // namespace

size_t qep_workspace_bytes(int rows, int cols) {
  const size_t R = rows, C = cols, nb = (C + QB - 1) / QB;
  return al(C * C * 8) + al(nb * QB * QB * 8) + al(R * C * 8) + al(R * C * 8) + al(4) +
         al((size_t)kMaxSlices * R * QB * 8);
}

// T[r][c] += sum_z P[z][r][c] (z in order) for the nb columns of one block.
__global__ __launch_bounds__(256) void add_slices_kernel(double* __restrict__ T, long long ldt,
                                                         int rows, int nb,
                                                         const double* __restrict__ P, int nz,
                                                         long long pz) {
  const long long n = (long long)rows * nb;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256) {
    const long long r = e / nb;
    const int c = (int)(e % nb);
    double s = T[r * ldt + c];
    for (int z = 0; z < nz; ++z) s += P[z * pz + r * nb + c];
    T[r * ldt + c] = s;
  }
}

__global__ __launch_bounds__(256) void to_f64_kernel(const float* __restrict__ x, long long n,
                                                     double* __restrict__ y) {
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256)
    y[e] = (double)x[e];
}

__global__ __launch_bounds__(256) void qep_finish_kernel(const double* __restrict__ W,
                                                         const double* __restrict__ Z,
                                                         long long n, double c,
                                                         float* __restrict__ out) {
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256)
    out[e] = (float)(W[e] + c * Z[e]);
}

static unsigned grid_for(long long n) {
  const long long b = (n + 255) / 256;
  return (unsigned)(b < 16384 ? b : 16384);
}

hipError_t launch_qep_correct(hipStream_t st, int rows, int cols, const float* W, const float* H,
                              const double* D, double mu, float* Wcorr, char* ws,
                              int** flag_out) {
  const size_t R = rows, C = cols, nblk = (C + QB - 1) / QB;
  double* L = (double*)ws;
  double* Linv = (double*)(ws + al(C * C * 8));
  double* W64 = (double*)((char*)Linv + al(nblk * QB * QB * 8));
  double* T = (double*)((char*)W64 + al(R * C * 8));
  int* flag = (int*)((char*)T + al(R * C * 8));
  double* P = (double*)((char*)flag + al(4));   // [kMaxSlices][rows][nb] partial updates
  const long long pz = (long long)rows * QB;
  *flag_out = flag;
  const long long n = (long long)rows * cols;
  const long long d = cols;
  hipError_t e = launch_zero_bytes(st, flag, sizeof(int));
  if (e != hipSuccess) return e;
  e = launch_copy_lower(st, H, cols, false, L);
  if (e != hipSuccess) return e;
  e = launch_potrf_f64(st, L, cols, d, Linv, flag, true);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(to_f64_kernel, dim3(grid_for(n)), dim3(256), 0, st, W, n, W64);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // T[r][a] = sum_b W[r][b] D[a][b]
  e = launch_gemm_nt_f64(st, false, rows, cols, cols, cols, 1.0, W64, d, D, d, T, d, 0, false);
  if (e != hipSuccess) return e;
  // forward: Y L^T = T
  for (int k0 = 0; k0 < cols; k0 += QB) {
    const int nb = min(QB, cols - k0);
    if (k0 > 0) {
      // T_k -= Y_{<k} L_{k,<k}^T, the k range split into slices summed in order
      const int ks = slice_of(k0);
      e = launch_gemm_nt_f64(st, false, rows, nb, k0, ks, -1.0, T, d, L + (long long)k0 * d, d,
                             P, nb, pz, false);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(add_slices_kernel, dim3(grid_for((long long)rows * nb)), dim3(256), 0, st,
                         T + k0, d, rows, nb, P, (k0 + ks - 1) / ks, pz);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    e = launch_gemm_nt_f64(st, false, rows, nb, nb, nb, 1.0, T + k0, d,
                           Linv + (long long)(k0 / QB) * QB * QB, QB, T + k0, d, 0, false);
    if (e != hipSuccess) return e;
  }
  // backward: Z L = Y
  for (int k0 = (int)((nblk - 1) * QB); k0 >= 0; k0 -= QB) {
    const int nb = min(QB, cols - k0);
    const int rest = cols - k0 - nb;
    if (rest > 0) {
      // T_k -= Z_{>k} L_{>k,k}, sliced as in the forward pass
      const int ks = slice_of(rest);
      e = launch_gemm_nn_f64_sliced(st, rows, nb, rest, ks, -1.0, T + k0 + nb, d,
                                    L + (long long)(k0 + nb) * d + k0, d, P, nb, pz);
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(add_slices_kernel, dim3(grid_for((long long)rows * nb)), dim3(256), 0, st,
                         T + k0, d, rows, nb, P, (rest + ks - 1) / ks, pz);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    e = launch_gemm_nn_f64(st, rows, nb, nb, 1.0, T + k0, d,
                           Linv + (long long)(k0 / QB) * QB * QB, QB, T + k0, d, false);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(qep_finish_kernel, dim3(grid_for(n)), dim3(256), 0, st, W64, T, n, 1.0 - mu,
                     Wcorr);
  return hipGetLastError();
}

}  // namespace jarq
