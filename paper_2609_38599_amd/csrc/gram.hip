// Grouped Gram matrices of the scale update (paper eqs. (5)-(6)).
//
// For row j with c_i = q_i - z_i 1 (exact small integers), entry (a, h) of
// B_j^T B_j is c_a^T H_ah c_h (B_j has columns A_i c_i and H = A^T A).  The
// matrix is symmetric, so only h >= a is formed.  A work-group takes a tile of
// 128 rows and a pair of row-groups {p, G-1-p} (so every work-group walks G+1
// blocks); for each block h it forms T = H(a-group, h-group) C(rows, h-group)^T
// on fp16 matrix cores (v_mfma_f32_32x32x16_f16, M = the g weights of group a,
// N = 32 rows, K = the g weights of group h) with H as its two fp16 planes and
// the codes exact in fp16, then reduces T against c_a for every row.
//
// Waves split the a-group into 32-weight blocks and the tile's rows; each H
// fragment is used for all of a wave's rows.  The codes of block h are staged
// in LDS as fp16 once per work-group (bit trick: the fp16 with bits
// 0x6400 | q is 1024 + q) and the next block's codes are fetched while the
// current block runs on the matrix cores.  Two work-groups share a CU (LDS and
// registers sized for it), so one's staging, reduction and H loads overlap
// the other's matrix work.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

namespace {
constexpr int RT = 128;  // rows per work-group

// Four codes (one byte each) -> four fp16 values q - z, exactly.
__device__ __forceinline__ void codes_to_f16(uint32_t q4, f16x2 zz, f16x2* out) {
  // 0x64qq as fp16 is 1024 + q
  const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, q4, 0x07010700u);  // [q1, 0x64, q0, 0x64]
  const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, q4, 0x07030702u);  // [q3, 0x64, q2, 0x64]
  out[0] = __builtin_bit_cast(f16x2, lo) - zz;
  out[1] = __builtin_bit_cast(f16x2, hi) - zz;
}
}  // namespace

template <int G_SIZE>
__global__ __launch_bounds__(256, 2) void gram_kernel(int rows, int cols,
                                                      const _Float16* __restrict__ Hh,
                                                      const _Float16* __restrict__ Hl,
                                                      const float* __restrict__ h_inv,
                                                      const uint8_t* __restrict__ codes,
                                                      const int32_t* __restrict__ zeros,
                                                      float* __restrict__ gram,
                                                      const int32_t* __restrict__ rowmap) {
  constexpr int g = G_SIZE;
  constexpr int NAB = g / 32;            // 32-weight blocks of an a-group
  constexpr int WPA = 4 / NAB;           // waves sharing an a-block
  constexpr int RW = RT / WPA;           // rows per wave
  constexpr int JB = RW / 32;            // 32-row blocks per wave
  constexpr int KS = g / 16;             // k-steps of one block
  constexpr int LDC = g + 8;             // fp16 row stride of staged code tiles
  const int G = cols / g;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int tid = threadIdx.x;
  const int lm = lane & 31, kh = lane >> 5;
  const int ab = wave % NAB;
  const int rbase = (wave / NAB) * RW;
  const int r0 = blockIdx.x * RT;
  const int p = blockIdx.y;
  const float hinv = *h_inv;

  extern __shared__ _Float16 sm[];
  _Float16* ch_s = sm;                  // RT x LDC: c of block h
  _Float16* ca_s = ch_s + RT * LDC;     // RT x LDC: c of the a-group
  double* red = (double*)(ca_s + RT * LDC);  // NAB x RT

  // Stage the codes of column block `blk` of the tile as fp16 (c = q - z):
  // threads 2t and 2t + 1 own the two halves of row t of the tile.
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr int TPR = 256 / RT;          // threads per staged row
  constexpr int CPT = g / TPR;           // codes per thread
  u32x4 stq[CPT / 16];
  int stz = 0;
  const int trow = tid / TPR, tpart = tid % TPR;
  const int srow = r0 + trow;
  // Tile rows are positions of the sweep (Gram output) holding layer rows
  // (codes, zero points).  Positions past the edge load position 0
  // (unconditional loads, so that none is waited for here): each row's Gram
  // entries depend on that row only, and those past the edge are never stored.
  const int lrow = map_row(rowmap, srow < rows ? srow : 0);
  auto fetch_codes = [&](int blk) {
    const u32x4* src = (const u32x4*)(codes + (size_t)lrow * cols + (size_t)blk * g + tpart * CPT);
#pragma unroll
    for (int i = 0; i < CPT / 16; ++i) stq[i] = src[i];
    stz = zeros[(size_t)lrow * G + blk];
  };
  auto store_codes = [&](_Float16* dst) {
    const _Float16 zb = (_Float16)(1024 + stz);
    const f16x2 zz = f16x2{zb, zb};
    _Float16* drow = dst + trow * LDC + tpart * CPT;
#pragma unroll
    for (int i = 0; i < CPT / 16; ++i) {
      f16x2 v[8];
#pragma unroll
      for (int w = 0; w < 4; ++w) codes_to_f16(stq[i][w], zz, v + 2 * w);
      *(f16x8*)(drow + i * 16) = f16x8{v[0][0], v[0][1], v[1][0], v[1][1], v[2][0], v[2][1], v[3][0], v[3][1]};
      *(f16x8*)(drow + i * 16 + 8) = f16x8{v[4][0], v[4][1], v[5][0], v[5][1], v[6][0], v[6][1], v[7][0], v[7][1]};
    }
  };
  // H fragments of block (a-group ga, column block h) for this wave's a-block.
  f16x8 hf[2][KS];
  auto fetch_h = [&](int ga, int h) {
    const size_t rowoff = (size_t)(ga * g + ab * 32 + lm) * cols + (size_t)h * g + 8 * kh;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      hf[0][ks] = *(const f16x8*)(Hh + rowoff + ks * 16);
      hf[1][ks] = *(const f16x8*)(Hl + rowoff + ks * 16);
    }
  };

  float outv[32];
#pragma unroll
  for (int q = 0; q < 32; ++q) outv[q] = 0.f;
  for (int side = 0; side < 2; ++side) {
    const int ga = side == 0 ? p : G - 1 - p;
    if (side == 1 && ga == p) break;
    lds_barrier();
    fetch_codes(ga);
    store_codes(ca_s);
    fetch_codes(ga);     // block h = ga comes first
    for (int h = ga; h < G; ++h) {
      lds_barrier();   // previous block's reads of ch_s are done
      store_codes(ch_s);
      // H fragments of this block (their latency is covered by the other
      // work-group on the CU), codes of the next one
      fetch_h(ga, h);
      if (h + 1 < G) fetch_codes(h + 1);
      lds_barrier();
      f32x16 acc[JB];
#pragma unroll
      for (int b = 0; b < JB; ++b) acc[b] = f32x16{};
      // Code fragments of k-slice ks + 1 are read while slice ks is on the
      // matrix cores (LDS latency off the critical path).
      f16x8 cf[2][JB];
#pragma unroll
      for (int b = 0; b < JB; ++b)
        cf[0][b] = *(const f16x8*)(ch_s + (rbase + b * 32 + lm) * LDC + 8 * kh);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 1 < KS) {
#pragma unroll
          for (int b = 0; b < JB; ++b)
            cf[(ks + 1) & 1][b] =
                *(const f16x8*)(ch_s + (rbase + b * 32 + lm) * LDC + (ks + 1) * 16 + 8 * kh);
        }
#pragma unroll
        for (int b = 0; b < JB; ++b) {
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hf[0][ks], cf[ks & 1][b], acc[b], 0, 0, 0);
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(hf[1][ks], cf[ks & 1][b], acc[b], 0, 0, 0);
        }
      }
      // acc element v of lane l: T(a = ab*32 + 8*(v/4) + 4*kh + v%4, row = rbase + b*32 + l%32).
#pragma unroll
      for (int b = 0; b < JB; ++b) {
        const int rr = rbase + b * 32 + lm;
        float s = 0.f;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
          const f16x4 c4 = *(const f16x4*)(ca_s + rr * LDC + ab * 32 + 8 * jj + 4 * kh);
#pragma unroll
          for (int i = 0; i < 4; ++i) s = fmaf((float)c4[i], acc[b][4 * jj + i], s);
        }
        double d = (double)s;
        d += __shfl_xor(d, 32);
        if (kh == 0) red[ab * RT + rr] = d;
      }
      lds_barrier();
      if (tid < RT) {
        // Thread tid owns row r0 + tid: keep its entries (ga, h) for up to 32
        // consecutive h in registers and store them as one contiguous run.
        const int rr = tid;
        double s = 0.0;
#pragma unroll
        for (int a = 0; a < NAB; ++a) s += red[a * RT + rr];
        const float val = (float)(s * (double)hinv);
        const int j = (h - ga) & 31;
#pragma unroll
        for (int q = 0; q < 32; ++q) outv[q] = q == j ? val : outv[q];
        const int row = r0 + rr;
        if ((j == 31 || h == G - 1) && row < rows) {
          float* dst = gram + ((size_t)row * G + ga) * G + (h - j);
#pragma unroll
          for (int q = 0; q < 32; ++q)
            if (q <= j) dst[q] = outv[q];
        }
      }
    }
  }
}

template <int G_SIZE>
static hipError_t launch_gram_t(hipStream_t st, int rows, int cols, const char* ws,
                                const Layout& lay, const uint8_t* codes, const int32_t* zeros,
                                float* gram, const int32_t* rowmap) {
  constexpr int g = G_SIZE;
  const int G = cols / g;
  const size_t lds = (size_t)2 * RT * (g + 8) * sizeof(_Float16) + (size_t)(g / 32) * RT * sizeof(double);
  hipError_t e = hipFuncSetAttribute((const void*)gram_kernel<g>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid((rows + RT - 1) / RT, (G + 1) / 2);
  hipLaunchKernelGGL(gram_kernel<g>, grid, dim3(256), lds, st, rows, cols,
                     (const _Float16*)(ws + lay.hhi), (const _Float16*)(ws + lay.hlo),
                     (const float*)(ws + lay.hscale), codes, zeros, gram, rowmap);
  return hipGetLastError();
}

hipError_t launch_gram(hipStream_t st, int rows, int cols, int g, const char* ws,
                       const Layout& lay, const uint8_t* codes, const int32_t* zeros,
                       float* gram, const int32_t* rowmap) {
  switch (g) {
    case 32: return launch_gram_t<32>(st, rows, cols, ws, lay, codes, zeros, gram, rowmap);
    case 64: return launch_gram_t<64>(st, rows, cols, ws, lay, codes, zeros, gram, rowmap);
    case 128: return launch_gram_t<128>(st, rows, cols, ws, lay, codes, zeros, gram, rowmap);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jarq
