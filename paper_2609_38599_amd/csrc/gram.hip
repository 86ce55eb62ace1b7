// Grouped Gram matrices of the scale update (paper eqs. (5)-(6)).
//
// For row j with c_i = q_i - z_i 1 (exact small integers), entry (a, h) of
// B_j^T B_j is c_a^T H_ah c_h (B_j has columns A_i c_i and H = A^T A).  The
// matrix is symmetric, so only h >= a is formed.  A work-group takes a tile of
// 64 rows and a pair of row-groups {p, G-1-p} (so every work-group walks G+1
// blocks); for each block h it forms T = H(a-group, h-group) C(rows, h-group)^T
// with v_mfma_f32_32x32x2f32 (M = the g weights of group a, N = 32 rows,
// K = the g weights of group h) and reduces T against c_a per row in fp64.
#include "jarq_internal.h"

namespace jarq {

template <int G_SIZE>
__global__ __launch_bounds__(256) void gram_kernel(int rows, int cols,
                                                   const float* __restrict__ H,
                                                   const uint8_t* __restrict__ codes,
                                                   const int32_t* __restrict__ zeros,
                                                   float* __restrict__ gram) {
  constexpr int g = G_SIZE;
  constexpr int NAB = g / 32;              // 32-weight blocks of the a-group
  constexpr int PAIRS = NAB * 2;           // (a-block, 32-row block) pairs per tile
  constexpr int PPW = PAIRS >= 4 ? PAIRS / 4 : 1;  // pairs per wave
  const int G = cols / g;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int lm = lane & 31, kh = lane >> 5;
  const int r0 = blockIdx.x * 64;
  const int p = blockIdx.y;
  __shared__ double red[NAB][64];

  int ab[PPW], jb[PPW];
  bool live[PPW];
#pragma unroll
  for (int q = 0; q < PPW; ++q) {
    const int pair = (PAIRS >= 4) ? wave * PPW + q : wave;
    live[q] = pair < PAIRS;
    ab[q] = live[q] ? pair / 2 : 0;
    jb[q] = live[q] ? pair % 2 : 0;
  }

  for (int side = 0; side < 2; ++side) {
    const int ga = side == 0 ? p : G - 1 - p;
    if (side == 1 && ga == p) break;
    // c_a values this lane needs in the reduction: rows jb*32+lm, weights
    // ab*32 + 8*jj + 4*kh + i (the accumulator rows it holds).
    float ca[PPW][16];
#pragma unroll
    for (int q = 0; q < PPW; ++q) {
      const int row = r0 + jb[q] * 32 + lm;
      const bool ok = live[q] && row < rows;
      const int z = ok ? zeros[(size_t)row * G + ga] : 0;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        uint32_t q4 = 0;
        if (ok) q4 = *(const uint32_t*)(codes + (size_t)row * cols + ga * g + ab[q] * 32 + 8 * jj + 4 * kh);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          ca[q][4 * jj + i] = ok ? (float)((int)((q4 >> (8 * i)) & 0xffu) - z) : 0.f;
      }
    }
    for (int h = ga; h < G; ++h) {
      f32x16 acc[PPW];
#pragma unroll
      for (int q = 0; q < PPW; ++q) acc[q] = f32x16{};
      int zh[PPW];
      bool okr[PPW];
#pragma unroll
      for (int q = 0; q < PPW; ++q) {
        const int row = r0 + jb[q] * 32 + lm;
        okr[q] = live[q] && row < rows;
        zh[q] = okr[q] ? zeros[(size_t)row * G + h] : 0;
      }
      for (int k0 = 0; k0 < g; k0 += 8) {
        const int kk = k0 + 4 * kh;
#pragma unroll
        for (int q = 0; q < PPW; ++q) {
          const int arow = ga * g + ab[q] * 32 + lm;
          const f32x4 a4 = *(const f32x4*)(H + (size_t)arow * cols + h * g + kk);
          const int row = r0 + jb[q] * 32 + lm;
          uint32_t q4 = 0;
          if (okr[q]) q4 = *(const uint32_t*)(codes + (size_t)row * cols + h * g + kk);
          f32x4 b4;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            b4[i] = okr[q] ? (float)((int)((q4 >> (8 * i)) & 0xffu) - zh[q]) : 0.f;
#pragma unroll
          for (int t = 0; t < 4; ++t)
            acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[t], b4[t], acc[q], 0, 0, 0);
        }
      }
      // acc element v of lane l: T(a = ab*32 + 8*(v/4) + 4*kh + v%4, row = jb*32 + l%32).
#pragma unroll
      for (int q = 0; q < PPW; ++q) {
        double s = 0.0;
#pragma unroll
        for (int v = 0; v < 16; ++v) s += (double)ca[q][v] * (double)acc[q][v];
        s += __shfl_xor(s, 32);
        if (live[q] && kh == 0) red[ab[q]][jb[q] * 32 + lm] = s;
      }
      __syncthreads();
      if (threadIdx.x < 64) {
        double s = 0.0;
#pragma unroll
        for (int a = 0; a < NAB; ++a) s += red[a][threadIdx.x];
        const int row = r0 + threadIdx.x;
        if (row < rows) gram[((size_t)row * G + ga) * G + h] = (float)s;
      }
      __syncthreads();
    }
  }
}

hipError_t launch_gram(hipStream_t st, int rows, int cols, int g, const float* H,
                       const uint8_t* codes, const int32_t* zeros, float* gram) {
  const int G = cols / g;
  dim3 grid((rows + 63) / 64, (G + 1) / 2);
  switch (g) {
    case 32:
      hipLaunchKernelGGL(gram_kernel<32>, grid, dim3(256), 0, st, rows, cols, H, codes, zeros, gram);
      break;
    case 64:
      hipLaunchKernelGGL(gram_kernel<64>, grid, dim3(256), 0, st, rows, cols, H, codes, zeros, gram);
      break;
    case 128:
      hipLaunchKernelGGL(gram_kernel<128>, grid, dim3(256), 0, st, rows, cols, H, codes, zeros, gram);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace jarq
