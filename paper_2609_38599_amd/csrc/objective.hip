// Row objective right after the scale update (App. E.2): per row j and group
// i, (R_i e_i) . U_i = e_i^T (H e)_i from the residual product U = E M^T;
// summed over the groups that is L_j.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// Per row j and group i: (R_i e_i) . U_i = e_i^T L_i L_i^{-1} (H e)_i, summed
// in fp64.  V = E_i L_i (V(j, c) = sum_k E(j, k) R_i(c, k)) on fp16 matrix
// cores (v_mfma_f32_16x16x32_f16) against the two-term planes of the rows of
// R_i.  With e = w - s (q - z) (eq. (1)), V = RW - s C_i L_i: RW = W_i L_i is
// fixed for the layer (kMode 1 forms it once, from the two-term planes of W:
// three products, written out), and the per-sweep part takes the exact codes
// minus zero points (cz) as A: two products, then V = RW - s (cz R_i^T) and
// the dot with U (kMode 2).  R_i(c, k) = 0 for k < c, so output columns c
// only take the 32-wide k-chunks from 32 floor(c / 32) on; only those are
// staged in LDS (rows packed, padded by 8 halves).  Work-group: 64
// kDotRowBlocks rows x one group; each wave takes kDotRowBlocks blocks of 16
// consecutive rows.  Rows of cz, RW, W and the scales are layer rows
// (through the row map), U and the partials are by position.
constexpr int kDotRowBlocks = 4;   // 16-row blocks per wave

template <int G_SIZE, int kMode>
__global__ __launch_bounds__(256) void group_dot_kernel(int rows, int cols,
                                                        const _Float16* __restrict__ Ah,
                                                        const _Float16* __restrict__ Al,
                                                        const float* __restrict__ arow_inv,
                                                        const _Float16* __restrict__ rph,
                                                        const _Float16* __restrict__ rpl,
                                                        const float* __restrict__ rrow,
                                                        const float* __restrict__ scales,
                                                        float* __restrict__ RW,
                                                        const float* __restrict__ U,
                                                        double* __restrict__ objpart,
                                                        const int32_t* __restrict__ rowmap,
                                                        const int* __restrict__ n_dev) {
  if (n_dev != nullptr) rows = *n_dev;
  if (blockIdx.x * (64 * kDotRowBlocks) >= rows) return;  // uniform: nothing to do here
  constexpr int g = G_SIZE;
  constexpr int NKC = g / 32;   // 32-wide k-chunks
  constexpr int NMB = g / 16;   // 16-column output blocks
  constexpr int NB32 = g / 32;  // 32-row bands of R_i
  // packed rows: band b (rows 32 b .. 32 b + 31) keeps columns 32 b .. g - 1
  constexpr int PLANE = 32 * (NB32 * (g + 8) - 16 * NB32 * (NB32 - 1));
  auto roff = [](int c) {
    const int b = c >> 5;
    return 32 * (b * (g + 8) - 16 * b * (b - 1)) + (c & 31) * (g - 32 * b + 8);
  };
  __shared__ __attribute__((aligned(16))) _Float16 rs_h[PLANE];
  __shared__ __attribute__((aligned(16))) _Float16 rs_l[PLANE];
  const int G = cols / g;
  const int i = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int mr = lane & 15, kq = lane >> 4;
  {
    // all of this thread's pieces are requested before any is stored
    const _Float16* Rh = rph + (size_t)i * g * g;
    const _Float16* Rl = rpl + (size_t)i * g * g;
    constexpr int NE = (g * g / 8 + 255) / 256;
    f16x8 th[NE], tl[NE];
#pragma unroll
    for (int u = 0; u < NE; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int c = e / (g / 8), k0 = 8 * (e % (g / 8));
      if (e < g * g / 8 && k0 >= 32 * (c >> 5)) {
        th[u] = *(const f16x8*)(Rh + (size_t)c * g + k0);
        tl[u] = *(const f16x8*)(Rl + (size_t)c * g + k0);
      }
    }
#pragma unroll
    for (int u = 0; u < NE; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int c = e / (g / 8), k0 = 8 * (e % (g / 8));
      const int kb = 32 * (c >> 5);
      if (e < g * g / 8 && k0 >= kb) {
        *(f16x8*)(rs_h + roff(c) + k0 - kb) = th[u];
        *(f16x8*)(rs_l + roff(c) + k0 - kb) = tl[u];
      }
    }
  }
  __syncthreads();
  const float* rsc = rrow + (size_t)i * g;
  for (int rb = 0; rb < kDotRowBlocks; ++rb) {
    const int r0 = blockIdx.x * (64 * kDotRowBlocks) + wave * (16 * kDotRowBlocks) + rb * 16;
    if (r0 >= rows) break;
    // A fragments: row r0 + mr, k = 32 kc + 8 kq .. + 7; rows past the edge
    // read row 0 and reach only outputs that are never stored.  Mode 1 reads
    // the W planes by position (all rows), mode 2 cz by layer row.
    const int arow = r0 + mr < rows ? r0 + mr : 0;
    const size_t ab = (size_t)(kMode == 2 ? map_row(rowmap, arow) : arow) * cols +
                      (size_t)i * g + 8 * kq;
    f16x8 ah[NKC], al[NKC];
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      ah[kc] = *(const f16x8*)(Ah + ab + kc * 32);
      if constexpr (kMode == 1) al[kc] = *(const f16x8*)(Al + ab + kc * 32);
    }
    // this lane's four output rows (position and layer row) and scales
    int prow[4], lrow[4];
    float sj[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = r0 + 4 * kq + v;
      prow[v] = row < rows ? row : 0;
      lrow[v] = kMode == 2 ? map_row(rowmap, prow[v]) : prow[v];
      sj[v] = kMode == 2 ? scales[(size_t)lrow[v] * G + i] : 0.f;
    }
    double part[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      const int c = mb * 16 + mr;   // this lane's column of V (and of its B fragment)
      float u[4], rw[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if constexpr (kMode == 2) {
          u[v] = U[(size_t)prow[v] * cols + (size_t)i * g + c];
          rw[v] = RW[(size_t)lrow[v] * cols + (size_t)i * g + c];
        }
      }
      const float cs = rsc[c];
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        if (kc < mb / 2) continue;  // chunk left of the diagonal: zero
        // B(k, c) = R_i(c, k), k = 32 kc + 8 kq .. + 7
        const int at = roff(c) + (kc - mb / 2) * 32 + 8 * kq;
        const f16x8 bh = *(const f16x8*)(rs_h + at);
        const f16x8 bl = *(const f16x8*)(rs_l + at);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[kc], bh, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[kc], bl, acc, 0, 0, 0);
        if constexpr (kMode == 1)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[kc], bh, acc, 0, 0, 0);
      }
      // element v of lane l: (row 4 (l / 16) + v, column l % 16) of the block
      if constexpr (kMode == 1) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = r0 + 4 * kq + v;
          if (row < rows) RW[(size_t)row * cols + (size_t)i * g + c] = acc[v] * cs * arow_inv[row];
        }
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          part[v] = fma((double)(rw[v] - sj[v] * (acc[v] * cs)), (double)u[v], part[v]);
      }
    }
    if constexpr (kMode == 2) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        double x = part[v];
#pragma unroll
        for (int off = 8; off >= 1; off >>= 1) x += __shfl_xor(x, off);
        const int row = r0 + 4 * kq + v;
        if (mr == 0 && row < rows) objpart[(size_t)row * G + i] = x;
      }
    }
  }
}

// Operands: A planes ah / al with row scales arow (mode 1: W's planes; mode
// 2: cz, al and arow unused).
template <int G_SIZE, int kMode>
static hipError_t launch_group_dot_t(hipStream_t st, int rows, int cols, const char* ws,
                                     const Layout& lay, const _Float16* ah, const _Float16* al,
                                     const float* arow, const float* scales, const float* U,
                                     double* objpart, const int32_t* rowmap, const int* n_dev) {
  dim3 grid((rows + 64 * kDotRowBlocks - 1) / (64 * kDotRowBlocks), cols / G_SIZE);
  hipLaunchKernelGGL((group_dot_kernel<G_SIZE, kMode>), grid, dim3(256), 0, st, rows, cols, ah,
                     al, arow, (const _Float16*)(ws + lay.rph), (const _Float16*)(ws + lay.rpl),
                     (const float*)(ws + lay.rrow), scales, (float*)(ws + lay.rw), U, objpart,
                     rowmap, n_dev);
  return hipGetLastError();
}

template <int kMode>
static hipError_t launch_group_dot(hipStream_t st, int rows, int cols, int g, const char* ws,
                                   const Layout& lay, const _Float16* ah, const _Float16* al,
                                   const float* arow, const float* scales, const float* U,
                                   double* objpart, const int32_t* rowmap, const int* n_dev) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  switch (g) {
    case 32:
      return launch_group_dot_t<32, kMode>(st, rows, cols, ws, lay, ah, al, arow, scales, U,
                                           objpart, rowmap, n_dev);
    case 64:
      return launch_group_dot_t<64, kMode>(st, rows, cols, ws, lay, ah, al, arow, scales, U,
                                           objpart, rowmap, n_dev);
    case 128:
      return launch_group_dot_t<128, kMode>(st, rows, cols, ws, lay, ah, al, arow, scales, U,
                                            objpart, rowmap, n_dev);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_group_objective(hipStream_t st, int rows, int cols, int g, const char* ws,
                                  const Layout& lay, const float* scales, const float* U,
                                  double* objpart, const int32_t* rowmap, const int* n_dev) {
  return launch_group_dot<2>(st, rows, cols, g, ws, lay, (const _Float16*)(ws + lay.cz), nullptr,
                             nullptr, scales, U, objpart, rowmap, n_dev);
}

hipError_t launch_rw_product(hipStream_t st, int rows, int cols, int g, const char* ws,
                             const Layout& lay, const _Float16* whi, const _Float16* wlo,
                             const float* wrow_inv) {
  return launch_group_dot<1>(st, rows, cols, g, ws, lay, whi, wlo, wrow_inv, nullptr, nullptr,
                             nullptr, nullptr, nullptr);
}

}  // namespace jarq
