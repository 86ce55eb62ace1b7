// Per-layer factors of the diagonal Hessian blocks (paper eq. (9)).
//
// The paper factors each group block of the design, A_i = U_i R_i (thin QR,
// no column permutation).  Only R_i enters the code update, and
// R_i^T R_i = A_i^T A_i = H_ii, so R_i is the upper Cholesky factor of H_ii
// (the Babai proposal does not depend on the row signs of R_i).  One work-group
// factors one g x g block in LDS in fp64, inverts the lower factor L_i = R_i^T
// column by column, and writes the fp32 forms the sweep kernels read (and
// keeps L_i^{-1} in fp64 in place of L_i):
//   rinv  row n = row n of L_i^{-1}       (u = R_i^{-T} he = L_i^{-1} he)
//   rcol  column l, chunk c, lane j, w: R_i(m, l) / R_i(m, m) for m < l, 0
//         for m >= l, with m = j + 16 (W c + w), W = min(4, g / 16) (column l
//         of R_i above the diagonal with each row scaled by its inverse
//         diagonal, cut into chunks of W positions per lane and laid out
//         lane-contiguous, as the 16 lanes of a row own positions j + 16 t
//         and read one chunk each with one W-float access); only the chunks
//         a back-substitution step reads are kept (RcolLayout)
//   rdinv 1 / R_i(l, l),  rdsq R_i(l, l)^2,  rmat R_i (row-major).
#include "jarq_internal.h"

namespace jarq {

template <int G_SIZE>
__global__ __launch_bounds__(256) void chol_groups_kernel(const float* __restrict__ H, int cols,
                                                          double* __restrict__ lfac,
                                                          float* __restrict__ rinv,
                                                          float* __restrict__ rcol,
                                                          float* __restrict__ rdinv,
                                                          float* __restrict__ rdsq,
                                                          float* __restrict__ rmat,
                                                          Flags* __restrict__ flags) {
  constexpr int g = G_SIZE;
  constexpr int LD = g + 1;
  constexpr int NT = g / 16;
  extern __shared__ double A[];  // g x LD
  __shared__ int fail;
  const int blk = blockIdx.x;
  const int tid = threadIdx.x;
  const float* Hb = H + (size_t)blk * g * cols + (size_t)blk * g;
  for (int e = tid; e < g * g; e += blockDim.x) {
    const int r = e / g, c = e % g;
    A[r * LD + c] = (double)Hb[(size_t)r * cols + c];
  }
  if (tid == 0) fail = 0;
  __syncthreads();
  // Right-looking Cholesky H_ii = L L^T on the lower triangle.
  for (int k = 0; k < g; ++k) {
    if (tid == 0) {
      double piv = A[k * LD + k];
      if (!(piv > 0.0) || !isfinite(piv)) {
        fail = 1;
        piv = 1.0;
      }
      A[k * LD + k] = sqrt(piv);
    }
    __syncthreads();
    const double d = A[k * LD + k];
    for (int i = k + 1 + tid; i < g; i += blockDim.x) A[i * LD + k] /= d;
    __syncthreads();
    const int n = g - k - 1;
    for (int e = tid; e < n * n; e += blockDim.x) {
      const int i = k + 1 + e / n, j = k + 1 + e % n;
      if (j <= i) A[i * LD + j] -= A[i * LD + k] * A[j * LD + k];
    }
    __syncthreads();
  }
  double* Lb = lfac + (size_t)blk * g * g;
  for (int e = tid; e < g * g; e += blockDim.x) {
    const int r = e / g, c = e % g;
    Lb[e] = (c <= r) ? A[r * LD + c] : 0.0;
  }
  __syncthreads();
  // Column j of L^{-1}: Linv(i, j) = (delta_ij - sum_{j<=k<i} L(i,k) Linv(k,j)) / L(i,i).
  // Thread j owns column j of A, which now receives L^{-1}; L is read back from lfac.
  if (tid < g) {
    const int j = tid;
    for (int i = 0; i < g; ++i) {
      double v = 0.0;
      if (i >= j) {
        double acc = (i == j) ? 1.0 : 0.0;
        for (int k = j; k < i; ++k) acc -= Lb[i * g + k] * A[k * LD + j];
        v = acc / Lb[i * g + i];
      }
      A[i * LD + j] = v;
    }
  }
  __syncthreads();
  float* rinv_b = rinv + (size_t)blk * g * g;
  float* rcol_b = rcol + (size_t)blk * g * g;
  for (int e = tid; e < g * g; e += blockDim.x) {
    const int r = e / g, c = e % g;
    rinv_b[e] = (float)A[r * LD + c];
    // column l, chunk c, lane j, w for e = ((l NC + c) 16 + j) W + w:
    // R(m, l) / R(m, m), m = j + 16 (W c + w), R = L^T; kept where the back
    // substitution reads it (c < RcolLayout<g>::chunks(l))
    using RL = RcolLayout<g>;
    constexpr int W = RL::W;
    const int l = e / (16 * NT);
    const int rem = e % (16 * NT);
    const int j = (rem / W) % 16;
    const int cc = rem / (16 * W);
    const int t = cc * W + rem % W;
    const int m = j + 16 * t;
    if (cc < RL::chunks(l))
      rcol_b[RL::offset(l) + (cc * 16 + j) * W + rem % W] =
          (float)(m < l ? Lb[l * g + m] / Lb[m * g + m] : 0.0);
  }
  // R_i = L_i^T in fp32, row m: rmat[m][n] = L_i(n, m) (zero below the diagonal).
  float* rmat_b = rmat + (size_t)blk * g * g;
  for (int e = tid; e < g * g; e += blockDim.x) {
    const int m = e / g, n = e % g;
    rmat_b[e] = (float)(n >= m ? Lb[n * g + m] : 0.0);
  }
  for (int l = tid; l < g; l += blockDim.x) {
    const double d = Lb[l * g + l];
    rdinv[(size_t)blk * g + l] = (float)(1.0 / d);
    rdsq[(size_t)blk * g + l] = (float)(d * d);
  }
  __syncthreads();  // every read of L is done
  // Keep L_i^{-1} in fp64 (it replaces L_i in lfac) for M = blockdiag(L^{-1}) H.
  for (int e = tid; e < g * g; e += blockDim.x) Lb[e] = A[(e / g) * LD + e % g];
  if (tid == 0 && fail) atomicAdd(&flags->not_spd, 1);
}

template <int G_SIZE>
static hipError_t launch_chol_t(hipStream_t st, int cols, const float* H, char* ws,
                                const Layout& lay) {
  const int G = cols / G_SIZE;
  const size_t lds = (size_t)G_SIZE * (G_SIZE + 1) * sizeof(double);
  static std::atomic<unsigned long long> lds_set{0};
  hipError_t e = allow_dynamic_lds((const void*)chol_groups_kernel<G_SIZE>, lds, lds_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chol_groups_kernel<G_SIZE>, dim3(G), dim3(256), lds, st, H, cols,
                     (double*)(ws + lay.lfac), (float*)(ws + lay.rinv), (float*)(ws + lay.rcol),
                     (float*)(ws + lay.rdinv), (float*)(ws + lay.rdsq), (float*)(ws + lay.rmat),
                     (Flags*)(ws + lay.flags));
  return hipGetLastError();
}

// R_i rows as two fp16 terms for the objective's products: row c scaled by
// 2^t_c (its largest entry in [2^13, 2^14)), hi = fp16(x), lo = fp16(x - hi).
// One wavefront per row (g <= 128: two entries per lane).
__global__ __launch_bounds__(256) void split_r_kernel(const float* __restrict__ rmat, int nrows,
                                                      int g, _Float16* __restrict__ hi,
                                                      _Float16* __restrict__ lo,
                                                      float* __restrict__ row_inv) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= nrows) return;
  const float* x = rmat + (size_t)r * g;
  const float a = lane < g ? x[lane] : 0.f;
  const float b = lane + 64 < g ? x[lane + 64] : 0.f;
  float m = fmaxf(fabsf(a), fabsf(b));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  const int t = (m > 0.f && isfinite(m)) ? 13 - ilogbf(m) : 0;
  if (lane == 0) row_inv[r] = ldexpf(1.f, -t);
  if (lane < g) {
    const float v = ldexpf(a, t);
    const _Float16 h = (_Float16)v;
    hi[(size_t)r * g + lane] = h;
    lo[(size_t)r * g + lane] = (_Float16)(v - (float)h);
  }
  if (lane + 64 < g) {
    const float v = ldexpf(b, t);
    const _Float16 h = (_Float16)v;
    hi[(size_t)r * g + lane + 64] = h;
    lo[(size_t)r * g + lane + 64] = (_Float16)(v - (float)h);
  }
}

hipError_t launch_split_r(hipStream_t st, int cols, int g, char* ws, const Layout& lay) {
  if (g > 128) return hipErrorInvalidValue;
  const int nrows = cols;  // G groups of g rows
  hipLaunchKernelGGL(split_r_kernel, dim3((nrows + 3) / 4), dim3(256), 0, st,
                     (const float*)(ws + lay.rmat), nrows, g, (_Float16*)(ws + lay.rph),
                     (_Float16*)(ws + lay.rpl), (float*)(ws + lay.rrow));
  return hipGetLastError();
}

hipError_t launch_chol_groups(hipStream_t st, int cols, int g, const float* H, char* ws,
                              const Layout& lay) {
  switch (g) {
    case 32: return launch_chol_t<32>(st, cols, H, ws, lay);
    case 64: return launch_chol_t<64>(st, cols, H, ws, lay);
    case 128: return launch_chol_t<128>(st, cols, H, ws, lay);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jarq
