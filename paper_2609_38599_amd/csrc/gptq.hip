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
// run per row, sixteen lanes per row.
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

// Sixteen lanes per row (16 rows per 256-thread work-group): lane j owns the
// group positions n = j + 16 t (t = 0 .. g/16 - 1) and keeps their values in
// registers.  Each of the g sequential steps m forms sum_{n<m} M_mn v_n as
// per-lane partial sums reduced over the row's lanes; the owner of m takes
// the step.  Pass 1: y = M_GG^{-1} c and the group's grid from w + y (0 forced
// into the range); pass 2: the columns in order, each rounded from
// w_m + (c_m + sum_{n<m} M_mn e_n) / M_mm.
template <int G_SIZE>
__global__ __launch_bounds__(256) void gptq_group_kernel(int rows, int cols, int bits, int grp,
                                                         const float* __restrict__ W,
                                                         const double* __restrict__ M,
                                                         const double* __restrict__ comp,
                                                         int nsplit, double* __restrict__ E,
                                                         uint8_t* __restrict__ codes,
                                                         float* __restrict__ scales,
                                                         int32_t* __restrict__ zeros) {
  constexpr int g = G_SIZE;
  constexpr int NT = g / 16;
  const int j = threadIdx.x & 15;
  const int r = blockIdx.x * 16 + (threadIdx.x >> 4);
  const bool live = r < rows;
  const int rr = live ? r : rows - 1;
  const int b0 = grp * g;
  const int G = cols / g;
  const double qmax = (double)((1 << bits) - 1);
  const double* Mg = M + (long long)b0 * cols + b0;   // M_GG: Mg[m * cols + n], n <= m
  const float* w = W + (long long)rr * cols + b0;
  const long long cstride = (long long)rows * g;
  double cl[NT], wl[NT], vl[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int n = j + 16 * t;
    double c = 0.0;
    for (int z = 0; z < nsplit; ++z) c += comp[z * cstride + (long long)rr * g + n];
    cl[t] = c;
    wl[t] = (double)w[n];
    vl[t] = 0.0;
  }
  // Row m of M_GG at this lane's positions, loaded one step ahead into the
  // buffer of the other step parity (no register copies: a copy would wait
  // for the loads in flight).  The last step reloads row g - 1 (in bounds).
  double ma[NT], mb[NT];
  auto load_row = [&](int m, double (&dst)[NT]) __attribute__((always_inline)) {
    const double* mrow = Mg + (long long)(m < g ? m : g - 1) * cols + j;
#pragma unroll
    for (int t2 = 0; t2 < NT; ++t2) dst[t2] = mrow[16 * t2];
  };
  // sum_{n < m} M_mn v_n over the row's lanes (positions of earlier blocks, and
  // of block t those before m), with mrow = row m at this lane's positions
  auto row_dot = [&](int t, int i, const double (&mrow)[NT]) __attribute__((always_inline)) {
    double part = 0.0;
#pragma unroll
    for (int t2 = 0; t2 < NT; ++t2)
      if (t2 < t) part = fma(mrow[t2], vl[t2], part);
    if (j < i) part = fma(mrow[t], vl[t], part);
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) part += __shfl_xor(part, off);
    return part;
  };

  // pass 1: y = M_GG^{-1} c, grid from w + y
  double lo = 0.0, hi = 0.0;
  auto step1 = [&](int t, int i, const double (&mrow)[NT]) __attribute__((always_inline)) {
    const double part = row_dot(t, i, mrow);
    if (j == i) {
      const double y = (cl[t] - part) / mrow[t];   // the owner's mrow[t] is M_mm
      vl[t] = y;
      const double v = wl[t] + y;
      lo = fmin(lo, v);
      hi = fmax(hi, v);
    }
  };
  load_row(0, ma);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    for (int i = 0; i < 16; i += 2) {
      load_row(16 * t + i + 1, mb);
      step1(t, i, ma);
      load_row(16 * t + i + 2, ma);
      step1(t, i + 1, mb);
    }
  }
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) {
    lo = fmin(lo, __shfl_xor(lo, off));
    hi = fmax(hi, __shfl_xor(hi, off));
  }
  const double s = hi > lo ? (hi - lo) / qmax : 1.0;
  const float s32 = (float)s;
  const double s64 = (double)s32;
  const double zp = fmin(fmax(rint(-lo / s64), 0.0), qmax);

  // pass 2: the columns in order (vl now takes the errors e = w - s (q - z))
  uint8_t ql[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) ql[t] = 0;
  auto step2 = [&](int t, int i, const double (&mrow)[NT]) __attribute__((always_inline)) {
    const double part = row_dot(t, i, mrow);
    if (j == i) {
      const double x = wl[t] + (cl[t] + part) / mrow[t];
      const double q = fmin(fmax(rint(x / s64) + zp, 0.0), qmax);
      vl[t] = wl[t] - s64 * (q - zp);
      ql[t] = (uint8_t)q;
    }
  };
  load_row(0, ma);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    for (int i = 0; i < 16; i += 2) {
      load_row(16 * t + i + 1, mb);
      step2(t, i, ma);
      load_row(16 * t + i + 2, ma);
      step2(t, i + 1, mb);
    }
  }
  if (live) {
    uint8_t* q_out = codes + (long long)r * cols + b0;
    double* e_out = E + (long long)r * cols + b0;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      q_out[j + 16 * t] = ql[t];
      e_out[j + 16 * t] = vl[t];
    }
    if (j == 0) {
      scales[(long long)r * G + grp] = s32;
      zeros[(long long)r * G + grp] = (int32_t)zp;
    }
  }
}

template <int G_SIZE>
static hipError_t launch_gptq_group_t(hipStream_t st, int rows, int cols, int bits, int grp,
                                      const float* W, const double* M, const double* comp,
                                      int nsplit, double* E, uint8_t* codes, float* scales,
                                      int32_t* zeros) {
  hipLaunchKernelGGL(gptq_group_kernel<G_SIZE>, dim3((rows + 15) / 16), dim3(256), 0, st, rows,
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
