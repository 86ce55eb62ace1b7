// Gauss-Seidel residual update between panels of groups (paper eq. (7)).
//
// The code update visits the groups of a row in order; group i must see the
// accepted changes of every earlier group.  Groups are processed in panels of
// consecutive groups: inside a panel the Babai kernel corrects its own later
// groups, and once a panel is done this kernel folds its accepted changes into
// the residual product of every later column, for all rows at once:
//   P(:, c) -= sum_{h in panel} s_h (dq_h H(h-block, c))       for c >= panel end,
// with dq_h the exact integer code changes (fp16) and H read as its two fp16
// planes (v_mfma_f32_32x32x16_f16, two products); the per-row, per-group scale
// s_h is applied to each group's partial sum in fp32.  H is symmetric, so
// B(k, n) = H(n, k) is read along k.
//
// Tiling: 128 x 128 output tile per 256-thread work-group, 2 x 2 waves of
// 64 x 64, K (the panel's columns) in steps of 32 staged through LDS with
// double buffering.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

namespace {
constexpr int BM = 128, BN = 128, BK = 32, PADK = BK + 8;
constexpr int A_TILE = BM * PADK, B_TILE = BN * PADK;
constexpr int STAGE = A_TILE + 2 * B_TILE;  // halves per stage
constexpr int MAX_PANEL_GROUPS = 16;
}  // namespace

__global__ __launch_bounds__(256, 2) void panel_update_kernel(
    int rows, int cols, int g, int c0, int c1, const _Float16* __restrict__ dq,
    const _Float16* __restrict__ Hh, const _Float16* __restrict__ Hl,
    const float* __restrict__ h_inv, const float* __restrict__ scales, float* __restrict__ P) {
  extern __shared__ _Float16 lds[];
  __shared__ float sc_s[BM][MAX_PANEL_GROUPS];
  const int G = cols / g;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lm = lane & 31, kh = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int n0 = c1 + blockIdx.x * BN;
  const int h0 = c0 / g;
  const int ng = (c1 - c0) / g;
  const float hinv = *h_inv;

  for (int e = tid; e < BM * ng; e += 256) {
    const int r = e / ng, h = e % ng;
    const int gr = m0 + r;
    sc_s[r][h] = gr < rows ? scales[(size_t)gr * G + h0 + h] * hinv : 0.f;
  }

  // global -> LDS chunks of 16 bytes: A 128 rows x 4 chunks, B 2 planes x 128 rows x 4 chunks
  const int crow = tid >> 2;   // 0..63
  const int ckc = tid & 3;
  f16x8 ra[2], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int gm = m0 + crow + 64 * i;
      ra[i] = gm < rows ? *(const f16x8*)(dq + (size_t)gm * cols + k0 + ckc * 8) : f16x8{};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int gn = n0 + crow + 64 * (i & 1);
      const _Float16* src = (i < 2 ? Hh : Hl);
      rb[i] = gn < cols ? *(const f16x8*)(src + (size_t)gn * cols + k0 + ckc * 8) : f16x8{};
    }
  };
  auto lstore = [&](int st) {
    _Float16* base = lds + st * STAGE;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      *(f16x8*)(base + (crow + 64 * i) * PADK + ckc * 8) = ra[i];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *(f16x8*)(base + A_TILE + (i >> 1) * B_TILE + (crow + 64 * (i & 1)) * PADK + ckc * 8) = rb[i];
  };

  f32x16 acc[2][2], seg[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      acc[a][b] = f32x16{};
      seg[a][b] = f32x16{};
    }

  const int nk = (c1 - c0) / BK;
  const int steps_per_group = g / BK;
  gload(c0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) gload(c0 + (kt + 1) * BK);
    const _Float16* base = lds + st * STAGE;
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      const int kk = ks + 8 * kh;
      f16x8 af[2], bh[2], bl[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) af[a] = *(const f16x8*)(base + (wm * 64 + a * 32 + lm) * PADK + kk);
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int r = wn * 64 + b * 32 + lm;
        bh[b] = *(const f16x8*)(base + A_TILE + r * PADK + kk);
        bl[b] = *(const f16x8*)(base + A_TILE + B_TILE + r * PADK + kk);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          seg[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[a], bh[b], seg[a][b], 0, 0, 0);
          seg[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[a], bl[b], seg[a][b], 0, 0, 0);
        }
    }
    if ((kt + 1) % steps_per_group == 0) {
      // end of group h: acc += s_h (per row) * seg
      const int h = kt / steps_per_group;
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float sv = sc_s[wm * 64 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4)][h];
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            acc[a][b][v] = fmaf(seg[a][b][v], sv, acc[a][b][v]);
            seg[a][b][v] = 0.f;
          }
        }
    }
    if (kt + 1 < nk) lstore(st ^ 1);
    __syncthreads();
  }
  // Accumulator element v of lane l in a 32x32 block:
  // (row 8 * (v / 4) + 4 * (l / 32) + v % 4, column l % 32).
  // All loads of P are issued before any store: the compiler cannot prove the
  // addresses distinct and would otherwise serialise 64 round trips to memory.
  float pold[2][2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = n0 + wn * 64 + b * 32 + lm;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 64 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
        pold[a][b][v] = (row < rows && col < cols) ? P[(size_t)row * cols + col] : 0.f;
      }
    }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = n0 + wn * 64 + b * 32 + lm;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * 64 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
        if (row < rows && col < cols) P[(size_t)row * cols + col] = pold[a][b][v] - acc[a][b][v];
      }
    }
}

int panel_groups(int g) { return 512 / g < MAX_PANEL_GROUPS ? 512 / g : MAX_PANEL_GROUPS; }

hipError_t launch_panel_update(hipStream_t st, int rows, int cols, int g, int c0, int c1,
                               const char* ws, const Layout& lay, const float* scales, float* P) {
  if (c1 >= cols) return hipSuccess;
  const size_t lds = (size_t)2 * STAGE * sizeof(_Float16);
  hipError_t e = hipFuncSetAttribute((const void*)panel_update_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid((cols - c1 + BN - 1) / BN, (rows + BM - 1) / BM);
  hipLaunchKernelGGL(panel_update_kernel, grid, dim3(256), lds, st, rows, cols, g, c0, c1,
                     (const _Float16*)(ws + lay.dq), (const _Float16*)(ws + lay.hhi),
                     (const _Float16*)(ws + lay.hlo), (const float*)(ws + lay.hscale), scales, P);
  return hipGetLastError();
}

}  // namespace jarq
