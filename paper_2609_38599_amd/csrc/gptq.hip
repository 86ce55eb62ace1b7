// GPTQ-style host on the GPU: the starting state (S0, Q0, Z) from sequential
// error compensation (App. A.1 names GPTQ as a host; its recursion is the
// nearest-plane relation of App. G.7), columns in their natural order, the
// grid of each group fixed at its first column from the compensated weights by
// the min/max rule of the RTN host.
//
// Formulation without any inverse.  Let M be the lower-triangular matrix with
// M^T M = H; with J the order-reversing permutation, J H J = C C^T (C lower,
// the ordinary Cholesky factor) and M = J C^T J.  With e = w - what (original
// weights minus quantized ones), GPTQ's update rule is equivalent to
//   column k is rounded from  w_k + (sum_{i<k} M_ki e_i) / M_kk,
// and the compensated weights of a whole group G at its first column are
//   w_G + M_GG^{-1} (M_GP e_P),   P = the columns before G
// (the group's block of the triangular system restricted to the prefix).  The
// product M_GP e_P for every row is one fp64 matrix product per group (split
// over k into partial slices, summed in a fixed order); the triangular parts
// run per row, one row per thread.
#include "jarq_internal.h"

namespace jarq {

namespace {
constexpr int kGptqKSlice = 512;   // k-slice of the per-group products
}

size_t gptq_workspace_bytes(int rows, int cols, int g) {
  const size_t R = rows, C = cols;
  const int kmax = cols - g;
  const size_t ns = kmax > 0 ? (size_t)((kmax + kGptqKSlice - 1) / kGptqKSlice) : 1;
  auto a = [](size_t x) { return (x + 255) & ~size_t(255); };
  return a(C * C * 8) + a(C * C * 8) + a(R * C * 8) + a(ns * R * g * 8) + a(64 * 64 * 8) + a(4);
}

// One row per thread; dynamic LDS: cs [g][64] (c = M_GP e_P) and es [g][64]
// (first y = M_GG^{-1} c, then the group's errors e).
template <int G_SIZE>
__global__ __launch_bounds__(64) void gptq_group_kernel(int rows, int cols, int bits, int grp,
                                                        const float* __restrict__ W,
                                                        const double* __restrict__ M,
                                                        const double* __restrict__ comp,
                                                        int nsplit, double* __restrict__ E,
                                                        uint8_t* __restrict__ codes,
                                                        float* __restrict__ scales,
                                                        int32_t* __restrict__ zeros) {
  constexpr int g = G_SIZE;
  extern __shared__ double gsm[];
  double* cs = gsm;
  double* es = gsm + g * 64;
  const int tid = threadIdx.x;
  const int r = blockIdx.x * 64 + tid;
  const bool live = r < rows;
  const int rr = live ? r : rows - 1;
  const int b0 = grp * g;
  const int G = cols / g;
  const double qmax = (double)((1 << bits) - 1);
  const double* Mg = M + (long long)b0 * cols + b0;   // M_GG: Mg[m * cols + n], n <= m
  const float* w = W + (long long)rr * cols + b0;
  const long long cstride = (long long)rows * g;

  // y = M_GG^{-1} c and the group's grid from w + y (0 forced into the range).
  double lo = 0.0, hi = 0.0;
  for (int m = 0; m < g; ++m) {
    double c = 0.0;
    for (int z = 0; z < nsplit; ++z) c += comp[z * cstride + (long long)rr * g + m];
    cs[m * 64 + tid] = c;
    double s = c;
    for (int n = 0; n < m; ++n) s = fma(-Mg[(long long)m * cols + n], es[n * 64 + tid], s);
    const double y = s / Mg[(long long)m * cols + m];
    es[m * 64 + tid] = y;
    const double v = (double)w[m] + y;
    lo = fmin(lo, v);
    hi = fmax(hi, v);
  }
  const double s = hi > lo ? (hi - lo) / qmax : 1.0;
  const float s32 = (float)s;
  const double s64 = (double)s32;
  const double zp = fmin(fmax(rint(-lo / s64), 0.0), qmax);

  // Columns in order: round w_k + (c_k + sum_{n<k} M_kn e_n) / M_kk.
  uint8_t* q_out = codes + (long long)rr * cols + b0;
  double* e_out = E + (long long)rr * cols + b0;
  for (int m = 0; m < g; ++m) {
    double t = cs[m * 64 + tid];
    for (int n = 0; n < m; ++n) t = fma(Mg[(long long)m * cols + n], es[n * 64 + tid], t);
    const double wk = (double)w[m];
    const double x = wk + t / Mg[(long long)m * cols + m];
    const double q = fmin(fmax(rint(x / s64) + zp, 0.0), qmax);
    const double e = wk - s64 * (q - zp);
    es[m * 64 + tid] = e;
    if (live) {
      e_out[m] = e;
      q_out[m] = (uint8_t)q;
    }
  }
  if (live) {
    scales[(long long)r * G + grp] = s32;
    zeros[(long long)r * G + grp] = (int32_t)zp;
  }
}

template <int G_SIZE>
static hipError_t launch_gptq_group_t(hipStream_t st, int rows, int cols, int bits, int grp,
                                      const float* W, const double* M, const double* comp,
                                      int nsplit, double* E, uint8_t* codes, float* scales,
                                      int32_t* zeros) {
  const size_t lds = (size_t)2 * G_SIZE * 64 * sizeof(double);
  hipError_t e = hipFuncSetAttribute((const void*)gptq_group_kernel<G_SIZE>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(gptq_group_kernel<G_SIZE>, dim3((rows + 63) / 64), dim3(64), lds, st, rows,
                     cols, bits, grp, W, M, comp, nsplit, E, codes, scales, zeros);
  return hipGetLastError();
}

// The whole host: factor the reversed Hessian, form M, then group by group the
// product M_GP e_P and the per-row triangular passes.  Returns the HIP error
// of the first failed launch; *flag (device) is set when H is not positive
// definite.
hipError_t launch_gptq(hipStream_t st, int rows, int cols, int g, int bits, const float* W,
                       const float* H, char* ws, uint8_t* codes, float* scales, int32_t* zeros,
                       int** flag_out) {
  auto a = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t CC = (size_t)cols * cols * 8;
  double* Cf = (double*)ws;
  double* M = (double*)(ws + a(CC));
  double* E = (double*)(ws + 2 * a(CC));
  double* comp = (double*)(ws + 2 * a(CC) + a((size_t)rows * cols * 8));
  const int kmax = cols - g;
  const size_t ns = kmax > 0 ? (size_t)((kmax + kGptqKSlice - 1) / kGptqKSlice) : 1;
  double* Linv = (double*)((char*)comp + a(ns * rows * g * 8));
  int* flag = (int*)((char*)Linv + a(64 * 64 * 8));
  *flag_out = flag;
  hipError_t e = launch_zero_bytes(st, flag, sizeof(int));
  if (e != hipSuccess) return e;
  e = launch_copy_lower(st, H, cols, true, Cf);
  if (e != hipSuccess) return e;
  e = launch_potrf_f64(st, Cf, cols, cols, Linv, flag, false);
  if (e != hipSuccess) return e;
  e = launch_antitranspose_lower(st, Cf, cols, M);
  if (e != hipSuccess) return e;
  const int G = cols / g;
  for (int grp = 0; grp < G; ++grp) {
    const int b0 = grp * g;
    const int nsplit = b0 > 0 ? (b0 + kGptqKSlice - 1) / kGptqKSlice : 0;
    if (b0 > 0) {
      // comp[z][r][m] = sum_{t in slice z} E[r][t] M[b0 + m][t]
      e = launch_gemm_nt_f64(st, false, rows, g, b0, kGptqKSlice, 1.0, E, cols,
                             M + (long long)b0 * cols, cols, comp, g, (long long)rows * g, false);
      if (e != hipSuccess) return e;
    }
    switch (g) {
      case 32: e = launch_gptq_group_t<32>(st, rows, cols, bits, grp, W, M, comp, nsplit, E, codes, scales, zeros); break;
      case 64: e = launch_gptq_group_t<64>(st, rows, cols, bits, grp, W, M, comp, nsplit, E, codes, scales, zeros); break;
      case 128: e = launch_gptq_group_t<128>(st, rows, cols, bits, grp, W, M, comp, nsplit, E, codes, scales, zeros); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace jarq
