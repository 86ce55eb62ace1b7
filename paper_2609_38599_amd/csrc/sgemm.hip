// Residual product P = E H of the sweep on fp16 matrix cores (paper Sec. 3.3.2:
// the conditional residual of eq. (7) needs (H e)_i for every row and group).
//
// E and H arrive as two-term fp16 planes (split.hip) with power-of-two scales:
// E = (Eh + El) re_m, H = (Hh + Hl) rh.  The product keeps the three terms
// above 2^-22 relative, P = (Eh Hh + Eh Hl + El Hh) re_m rh, accumulated in fp32
// by v_mfma_f32_32x32x16_f16 — fp32-class accuracy at 3/16 of the fp32 matrix
// work.  With kObj the epilogue writes, per row and 64-column slice,
// sum_c E(row, c) P(row, c) in fp64; summed over slices that is L_j, the
// objective right after the scale update (App. E.2).
//
// Tiling: 256 x 128 output tile per 256-thread work-group, 2 x 2 waves of
// 128 x 64 (4 x 2 accumulators of 32 x 32), K in steps of 32 staged through
// LDS with double buffering (both planes of both operands, 120 KB).  H is
// symmetric, so B(k, n) = H(n, k): both operands are read along k with 16-byte
// loads, and each lane's MFMA fragment is 8 consecutive k of one row.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

namespace {
constexpr int BM = 256, BN = 128, BK = 32, PADK = BK + 8;  // row stride 80 B: no bank conflicts
constexpr int A_PLANE = BM * PADK, B_PLANE = BN * PADK;
constexpr int STAGE = 2 * A_PLANE + 2 * B_PLANE;  // halves per stage
}  // namespace

template <bool kObj>
__global__ __launch_bounds__(256, 1) void split_gemm_kernel(
    int M, int N, int K, const _Float16* __restrict__ Ah, const _Float16* __restrict__ Al,
    const float* __restrict__ arow_inv, const _Float16* __restrict__ Bh,
    const _Float16* __restrict__ Bl, const float* __restrict__ b_inv, float* __restrict__ C,
    double* __restrict__ objpart) {
  extern __shared__ _Float16 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lm = lane & 31, kh = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;

  // global -> LDS chunk assignment (16-byte chunks, 4 per 32-wide k row)
  const int crow = tid >> 2;   // 0..63
  const int ckc = tid & 3;     // k chunk
  f16x8 ra[8], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = crow + 64 * (i & 3);
      const _Float16* src = (i < 4 ? Ah : Al);
      const int gm = m0 + row;
      ra[i] = gm < M ? *(const f16x8*)(src + (size_t)gm * K + k0 + ckc * 8) : f16x8{};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = crow + 64 * (i & 1);
      const _Float16* src = (i < 2 ? Bh : Bl);
      const int gn = n0 + row;
      rb[i] = gn < N ? *(const f16x8*)(src + (size_t)gn * K + k0 + ckc * 8) : f16x8{};
    }
  };
  auto lstore = [&](int st) {
    _Float16* base = lds + st * STAGE;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = crow + 64 * (i & 3);
      *(f16x8*)(base + (i >> 2) * A_PLANE + row * PADK + ckc * 8) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = crow + 64 * (i & 1);
      *(f16x8*)(base + 2 * A_PLANE + (i >> 1) * B_PLANE + row * PADK + ckc * 8) = rb[i];
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  const int nk = K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const _Float16* base = lds + st * STAGE;
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      const int kk = ks + 8 * kh;
      f16x8 ah[4], al[4], bh[2], bl[2];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int r = wm * 128 + a * 32 + lm;
        ah[a] = *(const f16x8*)(base + r * PADK + kk);
        al[a] = *(const f16x8*)(base + A_PLANE + r * PADK + kk);
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int r = wn * 64 + b * 32 + lm;
        bh[b] = *(const f16x8*)(base + 2 * A_PLANE + r * PADK + kk);
        bl[b] = *(const f16x8*)(base + 2 * A_PLANE + B_PLANE + r * PADK + kk);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[a], bh[b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[a], bl[b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[a], bh[b], acc[a][b], 0, 0, 0);
        }
    }
    if (kt + 1 < nk) lstore(st ^ 1);
    __syncthreads();
  }

  // Epilogue.  Accumulator element v of lane l in a 32x32 block:
  // (row 8 * (v / 4) + 4 * (l / 32) + v % 4, column l % 32).
  const float bs = *b_inv;
  const int nt = (N + kObjTile - 1) / kObjTile;
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    double part[16];
    float rsc[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = m0 + wm * 128 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
      rsc[v] = row < M ? arow_inv[row] : 0.f;
      part[v] = 0.0;
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = n0 + wn * 64 + b * 32 + lm;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 128 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
        if (row < M && col < N) {
          const float p = acc[a][b][v] * (rsc[v] * bs);
          C[(size_t)row * N + col] = p;
          if (kObj) {
            const size_t ix = (size_t)row * K + col;
            const float e = ((float)Ah[ix] + (float)Al[ix]) * rsc[v];
            part[v] += (double)e * (double)p;
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
        const int slice = (n0 + wn * 64) / kObjTile;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wm * 128 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
          if (row < M && slice < nt) objpart[(size_t)row * nt + slice] = part[v];
        }
      }
    }
  }
}

hipError_t launch_split_gemm(hipStream_t st, int rows, int cols, const char* ws,
                             const Layout& lay, float* C, double* objpart) {
  const size_t lds = (size_t)2 * STAGE * sizeof(_Float16);
  const void* fn = objpart != nullptr ? (const void*)split_gemm_kernel<true>
                                      : (const void*)split_gemm_kernel<false>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid((cols + BN - 1) / BN, (rows + BM - 1) / BM);
  const _Float16* ah = (const _Float16*)(ws + lay.ehi);
  const _Float16* al = (const _Float16*)(ws + lay.elo);
  const _Float16* bh = (const _Float16*)(ws + lay.hhi);
  const _Float16* bl = (const _Float16*)(ws + lay.hlo);
  const float* ar = (const float*)(ws + lay.erow);
  const float* bi = (const float*)(ws + lay.hscale);
  if (objpart != nullptr)
    hipLaunchKernelGGL(split_gemm_kernel<true>, grid, dim3(256), lds, st, rows, cols, cols, ah, al,
                       ar, bh, bl, bi, C, objpart);
  else
    hipLaunchKernelGGL(split_gemm_kernel<false>, grid, dim3(256), lds, st, rows, cols, cols, ah, al,
                       ar, bh, bl, bi, C, objpart);
  return hipGetLastError();
}

}  // namespace jarq
