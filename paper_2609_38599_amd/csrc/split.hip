// Two-term fp16 representations for the matrix-core contractions.
//
// gfx950 has no xf32 matrix instruction; its fp16 matrix rate is 16x the fp32
// one.  A fp32 value x scaled by a power of two 2^t is written as
// hi = fp16(x 2^t), lo = fp16(x 2^t - hi), which carries 22 significant bits.
// Products of such planes accumulate in fp32 on the matrix cores.
//   H:  one scale for the whole matrix, chosen so max |H| 2^t lies in [2^13, 2^14).
//   M = blockdiag(L_i^{-1}) H (the code update's coordinates, eq. (10)): one
//       scale per row of M, same rule.
//   W: one scale per row, same rule (for the layer's fixed W M^T and W_i L_i).
// Small-integer operands (codes minus zero points, code changes) are exact in fp16.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ void atomic_max_abs(float* dst, float v) {
  // |v| >= 0: IEEE ordering of non-negative floats equals their bit ordering.
  atomicMax((unsigned int*)dst, __float_as_uint(fabsf(v)));
}

__global__ void absmax_kernel(const float* __restrict__ x, size_t n, float* __restrict__ out) {
  float m = 0.f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    m = fmaxf(m, fabsf(x[i]));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((threadIdx.x & 63) == 0) atomic_max_abs(out, m);
}

__device__ __forceinline__ int pow2_exponent(float amax) {
  // t with amax * 2^t in [2^13, 2^14); 0 for an all-zero or nonfinite input.
  if (!(amax > 0.f) || !isfinite(amax)) return 0;
  return 13 - ilogbf(amax);
}

__global__ void split_h_kernel(const float* __restrict__ H, size_t n,
                               const float* __restrict__ amax, _Float16* __restrict__ hi,
                               _Float16* __restrict__ lo, float* __restrict__ inv_scale) {
  const int t = pow2_exponent(*amax);
  if (blockIdx.x == 0 && threadIdx.x == 0) *inv_scale = ldexpf(1.f, -t);
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const float x = ldexpf(H[i], t);
    const _Float16 h = (_Float16)x;
    hi[i] = h;
    lo[i] = (_Float16)(x - (float)h);
  }
}

hipError_t launch_split_h(hipStream_t st, int cols, const float* H, char* ws, const Layout& lay) {
  const size_t n = (size_t)cols * cols;
  float* amax = (float*)(ws + lay.hscale) + 1;
  hipError_t e = launch_zero_bytes(st, amax, sizeof(float));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(absmax_kernel, dim3(1024), dim3(256), 0, st, H, n, amax);
  hipLaunchKernelGGL(split_h_kernel, dim3(2048), dim3(256), 0, st, H, n, amax,
                     (_Float16*)(ws + lay.hhi), (_Float16*)(ws + lay.hlo),
                     (float*)(ws + lay.hscale));
  return hipGetLastError();
}

// M = blockdiag(L_i^{-1}) H.  Row n of M (group i = n / g, local index nl) is
// sum_{m <= nl} L_i^{-1}(nl, m) H(i g + m, :): the residual product with M in
// place of H gives u = L_i^{-1} (H e)_i for every group at once, and its
// blocks M(i-block, h-block) = L_i^{-1} H_ih carry a code change of group h
// into u_i.  Formed in fp64 from the fp64 inverse, rounded to fp32 into a
// temporary, with each row's maximum; then split with one scale per row.
// Work-group: the g rows of group i for 256 columns, thread = column.
template <int G_SIZE>
__global__ __launch_bounds__(256) void form_m_kernel(const float* __restrict__ H, int cols,
                                                     const double* __restrict__ linv,
                                                     float* __restrict__ mtmp,
                                                     float* __restrict__ rowmax) {
  constexpr int g = G_SIZE;
  const int i = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  __shared__ double li[g * g];
  const double* Li = linv + (size_t)i * g * g;
  for (int e = threadIdx.x; e < g * g; e += 256) li[e] = Li[e];
  __syncthreads();
  const bool cin = c < cols;
  float hc[g];
#pragma unroll
  for (int m = 0; m < g; ++m) hc[m] = cin ? H[(size_t)(i * g + m) * cols + c] : 0.f;
  for (int nl = 0; nl < g; ++nl) {
    double acc = 0.0;
#pragma unroll
    for (int m = 0; m < g; ++m)
      if (m <= nl) acc = fma(li[nl * g + m], (double)hc[m], acc);
    const float v = (float)acc;
    float mx = fabsf(v);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if (cin) mtmp[(size_t)(i * g + nl) * cols + c] = v;
    if ((threadIdx.x & 63) == 0) atomic_max_abs(rowmax + i * g + nl, mx);
  }
}

__global__ void split_rows_kernel(const float* __restrict__ x, int cols, int nrows,
                                  const float* __restrict__ rowmax, _Float16* __restrict__ hi,
                                  _Float16* __restrict__ lo, float* __restrict__ row_inv) {
  const size_t n = (size_t)nrows * cols;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / cols);
    const int t = pow2_exponent(rowmax[r]);
    if (e % cols == 0) row_inv[r] = ldexpf(1.f, -t);
    const float v = ldexpf(x[e], t);
    const _Float16 h = (_Float16)v;
    hi[e] = h;
    lo[e] = (_Float16)(v - (float)h);
  }
}

template <int G_SIZE>
static hipError_t launch_split_m_t(hipStream_t st, int cols, const float* H, char* ws,
                                   const Layout& lay) {
  // The H planes (written afterwards by launch_split_h) serve as the fp32
  // temporary: together they span cols * cols * 4 bytes.
  float* mtmp = (float*)(ws + lay.hhi);
  float* rowmax = (float*)(ws + lay.mmax);
  hipError_t e = launch_zero_bytes(st, rowmax, (size_t)cols * sizeof(float));
  if (e != hipSuccess) return e;
  dim3 grid((cols + 255) / 256, cols / G_SIZE);
  hipLaunchKernelGGL(form_m_kernel<G_SIZE>, grid, dim3(256), 0, st, H, cols,
                     (const double*)(ws + lay.lfac), mtmp, rowmax);
  hipLaunchKernelGGL(split_rows_kernel, dim3(2048), dim3(256), 0, st, mtmp, cols, cols, rowmax,
                     (_Float16*)(ws + lay.mhi), (_Float16*)(ws + lay.mlo),
                     (float*)(ws + lay.mrow));
  return hipGetLastError();
}

hipError_t launch_split_m(hipStream_t st, int cols, int g, const float* H, char* ws,
                          const Layout& lay) {
  switch (g) {
    case 32: return launch_split_m_t<32>(st, cols, H, ws, lay);
    case 64: return launch_split_m_t<64>(st, cols, H, ws, lay);
    case 128: return launch_split_m_t<128>(st, cols, H, ws, lay);
    default: return hipErrorInvalidValue;
  }
}

// W as two fp16 planes for the layer's constant products (T = W M^T and
// RW = W_i L_i, formed once by jarq_prepare): one work-group per row, the
// row maximum, then the planes and the row's inverse scale 2^-t.  Each thread
// keeps its NCH chunks of four weights in registers between the two passes
// (rows of at most 1024 NCH columns), so W is read once.
template <int NCH>
__global__ __launch_bounds__(256) void split_w_kernel(int cols, const float* __restrict__ W,
                                                      _Float16* __restrict__ whi,
                                                      _Float16* __restrict__ wlo,
                                                      float* __restrict__ wrow_inv) {
  const int row = blockIdx.x;
  __shared__ float red[4];
  const float* wr = W + (size_t)row * cols;
  f32x4 wv[NCH];
  float m = 0.f;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < cols) {
      wv[k] = *(const f32x4*)(wr + c);
#pragma unroll
      for (int i = 0; i < 4; ++i) m = fmaxf(m, fabsf(wv[k][i]));
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const int t = pow2_exponent(m);
  if (threadIdx.x == 0) wrow_inv[row] = ldexpf(1.f, -t);
  _Float16* hr = whi + (size_t)row * cols;
  _Float16* lr = wlo + (size_t)row * cols;
  typedef _Float16 h4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < cols) {
      h4 hv, lv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = ldexpf(wv[k][i], t);
        const _Float16 h = (_Float16)e;
        hv[i] = h;
        lv[i] = (_Float16)(e - (float)h);
      }
      *(h4*)(hr + c) = hv;
      *(h4*)(lr + c) = lv;
    }
  }
}

hipError_t launch_split_w(hipStream_t st, int rows, int cols, const float* W, _Float16* whi,
                          _Float16* wlo, float* wrow_inv) {
  if (rows <= 0) return hipSuccess;
  if (cols <= 4096)
    hipLaunchKernelGGL(split_w_kernel<4>, dim3(rows), dim3(256), 0, st, cols, W, whi, wlo, wrow_inv);
  else if (cols <= 12288)
    hipLaunchKernelGGL(split_w_kernel<12>, dim3(rows), dim3(256), 0, st, cols, W, whi, wlo, wrow_inv);
  else if (cols <= 16384)   // the most a layer can have: 128 groups of at most 128
    hipLaunchKernelGGL(split_w_kernel<16>, dim3(rows), dim3(256), 0, st, cols, W, whi, wlo, wrow_inv);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// cz = q - z as fp16 (exact: codes and zero points are small integers), by
// layer row; 16 codes per thread and step.
__global__ void codes_cz_kernel(int rows, int cols, int g, const uint8_t* __restrict__ codes,
                                const int32_t* __restrict__ zeros, _Float16* __restrict__ cz) {
  const int G = cols / g;
  const size_t chunks = (size_t)rows * cols / 16;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < chunks;
       e += (size_t)gridDim.x * blockDim.x) {
    const size_t off = e * 16;
    const int r = (int)(off / cols), c = (int)(off % cols);
    const uint4 q = *(const uint4*)(codes + off);
    const float z = (float)zeros[(size_t)r * G + c / g];
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    f16x8 h0, h1;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      h0[b] = (_Float16)((float)((w[b >> 2] >> (8 * (b & 3))) & 0xffu) - z);
      h1[b] = (_Float16)((float)((w[2 + (b >> 2)] >> (8 * (b & 3))) & 0xffu) - z);
    }
    *(f16x8*)(cz + off) = h0;
    *(f16x8*)(cz + off + 8) = h1;
  }
}

hipError_t launch_codes_cz(hipStream_t st, int rows, int cols, int g, const uint8_t* codes,
                           const int32_t* zeros, _Float16* cz) {
  if (rows <= 0 || cols % 16 != 0) return rows <= 0 ? hipSuccess : hipErrorInvalidValue;
  hipLaunchKernelGGL(codes_cz_kernel, dim3(2048), dim3(256), 0, st, rows, cols, g, codes, zeros,
                     cz);
  return hipGetLastError();
}

}  // namespace jarq
