// C = A H on fp32 matrix cores, for the per-layer W H of the scale
// right-hand sides (prepare) and for the stand-alone objective (jarq_objective,
// from H (w - what) of every row; paper Sec. 3.3.2 and eq. (7)); the sweep's
// own residual product runs on fp16 matrix cores (sgemm.hip).
//
// A = W (per-layer WH for the scale right-hand sides) or A = E = W - What with
// What = s_i (q - z_i) formed on the fly from the codes, scales and zero points
// (eq. (1)).  With kObj the epilogue also writes, per row and 64-column slice,
// sum_c A(row, c) C(row, c) in fp64: for A = E these partials sum to
// L_j = e_j^T H e_j, the objective right after the scale update (App. E.2).
//
// Tiling: 128 x 128 output tile per 256-thread work-group, 2 x 2 waves of
// 64 x 64, each a 2 x 2 grid of v_mfma_f32_32x32x2f32 accumulators.  H is
// symmetric, so the B operand B(k, n) = H(k, n) is read as H(n, k): every lane
// loads four consecutive k of one A row and one H row (16-byte loads); MFMA
// step t of a chunk of 8 takes k = k0 + 4 * (lane / 32) + t, the same
// permutation for A and B.
#include "jarq_internal.h"

namespace jarq {

namespace {

__device__ __forceinline__ f32x4 load_a4(const float* __restrict__ W,
                                         const uint8_t* __restrict__ codes,
                                         const float* __restrict__ scales,
                                         const int32_t* __restrict__ zeros, int row, int rows,
                                         int k, int cols, int g, int G, bool quant) {
  if (row >= rows) return f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 w = *(const f32x4*)(W + (size_t)row * cols + k);
  if (!quant) return w;
  const uint32_t q4 = *(const uint32_t*)(codes + (size_t)row * cols + k);
  const int grp = k / g;
  const float s = scales[(size_t)row * G + grp];
  const int z = zeros[(size_t)row * G + grp];
  w.x -= s * (float)((int)(q4 & 0xffu) - z);
  w.y -= s * (float)((int)((q4 >> 8) & 0xffu) - z);
  w.z -= s * (float)((int)((q4 >> 16) & 0xffu) - z);
  w.w -= s * (float)((int)(q4 >> 24) - z);
  return w;
}

__device__ __forceinline__ f32x4 load_h4(const float* __restrict__ H, int n, int cols, int k) {
  if (n >= cols) return f32x4{0.f, 0.f, 0.f, 0.f};
  return *(const f32x4*)(H + (size_t)n * cols + k);
}

__device__ __forceinline__ float elem_a(const float* __restrict__ W,
                                        const uint8_t* __restrict__ codes,
                                        const float* __restrict__ scales,
                                        const int32_t* __restrict__ zeros, int row, int col,
                                        int cols, int g, int G, bool quant) {
  float w = W[(size_t)row * cols + col];
  if (!quant) return w;
  const int grp = col / g;
  const float s = scales[(size_t)row * G + grp];
  const int z = zeros[(size_t)row * G + grp];
  return w - s * (float)((int)codes[(size_t)row * cols + col] - z);
}

}  // namespace

template <bool kQuant, bool kObj, bool kStore>
__global__ __launch_bounds__(256, 2) void gemm_ah_kernel(int rows, int cols, int g,
                                                         const float* __restrict__ W,
                                                         const uint8_t* __restrict__ codes,
                                                         const float* __restrict__ scales,
                                                         const int32_t* __restrict__ zeros,
                                                         const float* __restrict__ H,
                                                         float* __restrict__ C,
                                                         double* __restrict__ objpart) {
  const int G = cols / g;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lm = lane & 31, kh = lane >> 5;
  const int m0 = blockIdx.y * 128 + wm * 64;
  const int n0 = blockIdx.x * 128 + wn * 64;
  const int ra0 = m0 + lm, ra1 = m0 + 32 + lm;
  const int cb0 = n0 + lm, cb1 = n0 + 32 + lm;

  f32x16 acc00 = {}, acc01 = {}, acc10 = {}, acc11 = {};

  f32x4 a0 = load_a4(W, codes, scales, zeros, ra0, rows, 4 * kh, cols, g, G, kQuant);
  f32x4 a1 = load_a4(W, codes, scales, zeros, ra1, rows, 4 * kh, cols, g, G, kQuant);
  f32x4 b0 = load_h4(H, cb0, cols, 4 * kh);
  f32x4 b1 = load_h4(H, cb1, cols, 4 * kh);
  for (int k0 = 0; k0 < cols; k0 += 8) {
    const int kn = k0 + 8 + 4 * kh;
    f32x4 na0, na1, nb0, nb1;
    const bool more = (k0 + 8) < cols;
    if (more) {
      na0 = load_a4(W, codes, scales, zeros, ra0, rows, kn, cols, g, G, kQuant);
      na1 = load_a4(W, codes, scales, zeros, ra1, rows, kn, cols, g, G, kQuant);
      nb0 = load_h4(H, cb0, cols, kn);
      nb1 = load_h4(H, cb1, cols, kn);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      acc00 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[t], b0[t], acc00, 0, 0, 0);
      acc01 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[t], b1[t], acc01, 0, 0, 0);
      acc10 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[t], b0[t], acc10, 0, 0, 0);
      acc11 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[t], b1[t], acc11, 0, 0, 0);
    }
    if (more) {
      a0 = na0;
      a1 = na1;
      b0 = nb0;
      b1 = nb1;
    }
  }

  // Accumulator layout of a 32x32 block: element v of lane l is
  // (row 8 * (v / 4) + 4 * (l / 32) + v % 4, column l % 32).
  const f32x16* accs[2][2] = {{&acc00, &acc01}, {&acc10, &acc11}};
  const int nt = (cols + kObjTile - 1) / kObjTile;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    double part[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) part[v] = 0.0;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int col = n0 + nb * 32 + lm;
      const f32x16 a = *accs[mb][nb];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + mb * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
        if (row < rows && col < cols) {
          if (kStore) C[(size_t)row * cols + col] = a[v];
          if (kObj) {
            const float e = elem_a(W, codes, scales, zeros, row, col, cols, g, G, kQuant);
            part[v] += (double)e * (double)a[v];
          }
        }
      }
    }
    if (kObj) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        double x = part[v];
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) x += __shfl_xor(x, off);
        part[v] = x;
      }
      if (lm == 0) {
        const int slice = n0 / kObjTile;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + mb * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
          if (row < rows && slice < nt) objpart[(size_t)row * nt + slice] = part[v];
        }
      }
    }
  }
}

hipError_t launch_gemm_ah(hipStream_t st, int rows, int cols, int g, bool quant,
                          const float* W, const uint8_t* codes, const float* scales,
                          const int32_t* zeros, const float* H, float* C, double* objpart) {
  dim3 grid((cols + 127) / 128, (rows + 127) / 128);
  dim3 block(256);
  const bool obj = objpart != nullptr;
  const bool store = C != nullptr;
  if (quant) {
    if (obj && store)
      hipLaunchKernelGGL((gemm_ah_kernel<true, true, true>), grid, block, 0, st, rows, cols, g, W,
                         codes, scales, zeros, H, C, objpart);
    else if (obj)
      hipLaunchKernelGGL((gemm_ah_kernel<true, true, false>), grid, block, 0, st, rows, cols, g,
                         W, codes, scales, zeros, H, C, objpart);
    else
      hipLaunchKernelGGL((gemm_ah_kernel<true, false, true>), grid, block, 0, st, rows, cols, g,
                         W, codes, scales, zeros, H, C, objpart);
  } else {
    if (obj)
      hipLaunchKernelGGL((gemm_ah_kernel<false, true, true>), grid, block, 0, st, rows, cols, g,
                         W, codes, scales, zeros, H, C, objpart);
    else
      hipLaunchKernelGGL((gemm_ah_kernel<false, false, true>), grid, block, 0, st, rows, cols, g,
                         W, codes, scales, zeros, H, C, objpart);
  }
  return hipGetLastError();
}

}  // namespace jarq
