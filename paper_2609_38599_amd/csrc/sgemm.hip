// Split-precision products on fp16 matrix cores for the residual product of
// the sweep (paper Sec. 3.3.2: the conditional residual of eq. (7) needs
// (H e)_i for every row and group, used in the coordinates of eq. (10)).
// split3_kernel (three products of two-term planes of both operands) forms
// the layer's fixed T = W M^T once per layer; resid_kernel (further below)
// forms every sweep's U = T - What M^T with the exact q - z as one operand.
//
// Operands arrive as two-term fp16 planes with power-of-two scales (split.hip):
// A = (Ah + Al) ra_m per row m, B(k, n) = Bt(n, k) with Bt = (Bh + Bl) rb_n per
// row n.  The product keeps the three terms above 2^-22 relative,
// A B = (Ah Bh + Ah Bl + Al Bh) ra_m rb_n, accumulated in fp32 by
// v_mfma_f32_32x32x16_f16 — fp32-class accuracy at 3/16 of the fp32 matrix
// work.  With Bt = M = blockdiag(L_i^{-1}) H the product E M^T has in group
// i's columns of row j L_i^{-1} (H e_j)_i, the u of eq. (10) before division
// by the scale.
//
// Epilogues: store C = A B, or subtract, C -= A B.  The objective that
// follows the residual product is in objective.hip.
//
// Tiling: 256 x BN output tile per 512-thread work-group, 2 x 4 waves of
// 128 x BN/4 (two waves per SIMD, so one wave's waits are covered by the
// other's matrix work), K in steps of 32.  Both planes of both operands go
// straight from global memory to LDS (global_load_lds_dwordx4, no register
// staging) into one of two stages (128 KB for BN = 256); the eight loads of
// the next stage are spread over the first four fragment blocks of the
// current one.  Fragment reads are software-pipelined one block ahead (see
// compute).  One work-group per CU.  Tiles are ordered so that
// each XCD (work-groups are dealt to the 8 XCDs round-robin) works on a
// compact block of tiles that share A row-tiles and B column-tiles in its L2.
#include <hip/hip_ext.h>

#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

namespace {
constexpr int BM = 256, BK = 32;

// Tile of work-group wid; false when wid has none (the grid may be sized for
// more rows than the sweep has).
__device__ __forceinline__ bool tile_of(int wid, int nbm, int nbn, int& tm, int& tn) {
  const int total = nbm * nbn;
  const int q = total / 8, r = total % 8;
  const int x = wid % 8, loc = wid / 8;
  if (loc >= q + (x < r ? 1 : 0)) return false;  // this XCD's share is taken
  const int id = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + loc;
  constexpr int GM = 4;  // tile-rows per band
  const int band = id / (GM * nbn);
  const int first = band * GM;
  const int gsz = min(nbm - first, GM);
  const int within = id - band * GM * nbn;
  tm = first + within % gsz;
  tn = within / gsz;
  return true;
}

// LDS holds each plane tile as rows of 32 halves (four 16-byte chunks); chunk
// c of row r sits at position c ^ swz(r).  A fragment read (lane = row, two
// chunks across the wave halves) serves 16 consecutive rows per clock, and
// the 64-byte rows share 256-byte bank lines four at a time: rows r, r + 4,
// r + 8 and r + 12 take distinct positions.
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

// One 16-byte direct global -> LDS load per lane (lane L writes lds + 16 L bytes).
// A plain device function: the builtin and the LDS address space exist on the
// device side only.
__device__ __forceinline__ void dma16(const _Float16* src, _Float16* lds) {
  __builtin_amdgcn_global_load_lds((const void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}
}  // namespace

template <int BN, int kMode>
__global__ __launch_bounds__(512, 1) void split3_kernel(
    int M, int N, int K, int lda, int ldb, int ldc, const _Float16* __restrict__ Ah,
    const _Float16* __restrict__ Al, const float* __restrict__ arow_inv,
    const _Float16* __restrict__ Bh, const _Float16* __restrict__ Bl,
    const float* __restrict__ bcol_inv, float* __restrict__ C, const int* __restrict__ m_dev) {
  if (m_dev != nullptr) M = *m_dev;
  constexpr int WN = BN / 4;   // wave tile columns
  constexpr int NB = WN / 32;  // 32-column blocks per wave
  constexpr int A_PLANE = BM * BK, B_PLANE = BN * BK;  // halves
  constexpr int STAGE = 2 * A_PLANE + 2 * B_PLANE;
  // Two stages in two distinct arrays, so that the compiler can tell which
  // one an outstanding direct-to-LDS load writes.
  __shared__ __attribute__((aligned(1024))) _Float16 buf0[STAGE];
  __shared__ __attribute__((aligned(1024))) _Float16 buf1[STAGE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int lm = lane & 31, kh = lane >> 5;
  const int nbm = (M + BM - 1) / BM, nbn = (N + BN - 1) / BN;
  int tm, tn;
  if (M <= 0 || !tile_of(blockIdx.x, nbm, nbn, tm, tn)) return;  // uniform across the work-group
  const int m0 = tm * BM, n0 = tn * BN;

  // Direct global -> LDS loads, 16 bytes per lane: one instruction fills 1 KB
  // of LDS (16 rows of a plane tile).  Wave w fills the 1 KB pieces w, w + 4,
  // ...; lane L of a piece holds row 16 j + L / 4 at chunk position L % 4, i.e.
  // chunk (L % 4) ^ swz(row).  Rows past the edge read row 0 instead: their
  // products only reach output rows and columns that are never stored.
  // Element offsets are 32-bit (operands stay below 2^31 elements).
  constexpr int APW = A_PLANE / 512 / 8;  // 1 KB pieces per wave per A plane
  constexpr int BPW = B_PLANE / 512 / 8;
  unsigned aoff[APW], boff[BPW];
#pragma unroll
  for (int i = 0; i < APW; ++i) {
    const int r = 16 * (wave + 8 * i) + (lane >> 2);
    const int gm = m0 + r;
    aoff[i] = (unsigned)(gm < M ? gm : 0) * (unsigned)lda + (unsigned)(((lane & 3) ^ swz(r)) * 8);
  }
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int r = 16 * (wave + 8 * i) + (lane >> 2);
    const int gn = n0 + r;
    boff[i] = (unsigned)(gn < N ? gn : 0) * (unsigned)ldb + (unsigned)(((lane & 3) ^ swz(r)) * 8);
  }
  // Load j of the eight direct loads of a stage: j = 0..3 the A planes
  // (hi, lo of piece 0, then of piece 1), j = 4..7 the B planes.
  auto issue_one = [&](int j, int k0, _Float16* stage) {
    static_assert(APW == 2 && BPW == 2, "eight loads per stage");
    const int i = (j >> 1) & 1;
    if (j < 4) {
      _Float16* dst = stage + (wave + 8 * i) * 512;
      if (j & 1) dma16(Al + k0 + aoff[i], dst + A_PLANE); else dma16(Ah + k0 + aoff[i], dst);
    } else {
      _Float16* dst = stage + 2 * A_PLANE + (wave + 8 * i) * 512;
      if (j & 1) dma16(Bl + k0 + boff[i], dst + B_PLANE); else dma16(Bh + k0 + boff[i], dst);
    }
  };
  auto issue = [&](int k0, _Float16* stage) {
#pragma unroll
    for (int i = 0; i < APW; ++i) {
      _Float16* dst = stage + (wave + 8 * i) * 512;
      dma16(Ah + k0 + aoff[i], dst);
      dma16(Al + k0 + aoff[i], dst + A_PLANE);
    }
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      _Float16* dst = stage + 2 * A_PLANE + (wave + 8 * i) * 512;
      dma16(Bh + k0 + boff[i], dst);
      dma16(Bl + k0 + boff[i], dst + B_PLANE);
    }
  };

  f32x16 acc[4][NB];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = f32x16{};

  // Fragment reads are inline asm, paired with explicit waits whose operands
  // are the fragments they guard (the compiler neither sees when the data
  // arrives nor can move a use above its wait).  The reads also carry no
  // dependence on the direct loads, so no drain of those is inserted: every
  // stage is complete before the barrier that precedes its reads.
  auto lds_rd = [&](const _Float16* plane, int r, int ks) {
    const int c = (ks >> 3) + kh;
    const uint32_t ad = (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)(
        plane + r * BK + ((c ^ swz(r)) << 3));
    f16x8 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(ad));
    return v;
  };
  // One k-step on stage `base` as eight blocks s (k-slice s / 4, A row block
  // s % 4).  Block s first issues the reads for block s + 1 (block 1 also those
  // of the second k-slice's B fragments) and two of the next stage's direct
  // loads (into `stn` at k0n; none if k0n < 0), then waits only for the reads
  // issued before this block (LDS returns in order) and runs its 6 products,
  // so the reads of block s + 1 overlap them.
  auto compute = [&](const _Float16* base, int k0n, _Float16* stn) {
    f16x8 bh[2][NB], bl[2][NB], ah[2], al[2];
    auto loadB = [&](int ks, f16x8 (&h)[NB], f16x8 (&l)[NB]) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int r = wn * WN + b * 32 + lm;
        h[b] = lds_rd(base + 2 * A_PLANE, r, ks);
        l[b] = lds_rd(base + 2 * A_PLANE + B_PLANE, r, ks);
      }
    };
    auto loadA = [&](int ks, int a, f16x8& h, f16x8& l) {
      const int r = wm * 128 + a * 32 + lm;
      h = lds_rd(base, r, ks);
      l = lds_rd(base + A_PLANE, r, ks);
    };
    loadB(0, bh[0], bl[0]);
    loadA(0, 0, ah[0], al[0]);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int ksl = s >> 2, a = s & 3, c = s & 1;
      if (s + 1 < 8) loadA(((s + 1) >> 2) * 16, (s + 1) & 3, ah[c ^ 1], al[c ^ 1]);
      if (s == 1) loadB(16, bh[1], bl[1]);
      if (k0n >= 0 && s < 4) {
        issue_one(2 * s, k0n, stn);
        issue_one(2 * s + 1, k0n, stn);
      }
      static_assert(NB == 2, "wait operands list two B fragments");
#define JARQ_WAIT_OPS \
  "+v"(ah[c]), "+v"(al[c]), "+v"(bh[ksl][0]), "+v"(bh[ksl][1]), "+v"(bl[ksl][0]), "+v"(bl[ksl][1])
      if (s == 7)
        asm volatile("s_waitcnt lgkmcnt(0)" : JARQ_WAIT_OPS);
      else if (s == 1)
        asm volatile("s_waitcnt lgkmcnt(6)" : JARQ_WAIT_OPS);
      else
        asm volatile("s_waitcnt lgkmcnt(2)" : JARQ_WAIT_OPS);
#undef JARQ_WAIT_OPS
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[c], bh[ksl][b], acc[a][b], 0, 0, 0);
        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[c], bl[ksl][b], acc[a][b], 0, 0, 0);
        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[c], bh[ksl][b], acc[a][b], 0, 0, 0);
      }
    }
  };

  // Double buffering: the loads of step k + 1 fly while step k computes; the
  // barrier at the end of a step (which waits for this thread's outstanding
  // loads) makes the next stage visible and frees the one just read.
  const int nk = K / BK;
  issue(0, buf0);
  __syncthreads();
  int kt = 0;
  for (; kt + 2 <= nk; kt += 2) {
    compute(buf0, (kt + 1) * BK, buf1);
    __syncthreads();
    compute(buf1, kt + 2 < nk ? (kt + 2) * BK : -1, buf0);
    __syncthreads();
  }
  if (kt < nk) compute(buf0, -1, buf1);  // odd step count: the last step sits in buf0

  // Epilogue.  Accumulator element v of lane l in a 32x32 block:
  // (row 8 * (v / 4) + 4 * (l / 32) + v % 4, column l % 32).
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int rb0 = m0 + wm * 128 + a * 32 + 4 * kh;  // row of element v: rb0 + 8 (v / 4) + v % 4
    // Unconditional loads from clamped addresses (a load under a branch is
    // waited for inside the branch); out-of-range elements are never stored.
    float rsc[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) rsc[v] = arow_inv[min(rb0 + 8 * (v / 4) + (v % 4), M - 1)];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int col = n0 + wn * WN + b * 32 + lm;
      const float cs = bcol_inv[min(col, N - 1)];
      if (kMode == 1) {
        // All loads of the block before its stores: the compiler cannot prove
        // the addresses distinct and would otherwise serialise the round trips.
        float old[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = rb0 + 8 * (v / 4) + (v % 4);
          old[v] = C[(size_t)min(row, M - 1) * ldc + min(col, N - 1)];
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = rb0 + 8 * (v / 4) + (v % 4);
          if (row < M && col < N)
            C[(size_t)row * ldc + col] = old[v] - acc[a][b][v] * (rsc[v] * cs);
        }
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = rb0 + 8 * (v / 4) + (v % 4);
          if (row < M && col < N) C[(size_t)row * ldc + col] = acc[a][b][v] * (rsc[v] * cs);
        }
      }
    }
  }
}

template <int BN, int kMode>
static hipError_t launch_split3_t(hipStream_t st, int M, int N, int K, int lda, int ldb,
                                  int ldc, const _Float16* ah, const _Float16* al,
                                  const float* arow, const _Float16* bh, const _Float16* bl,
                                  const float* bcol, float* C, const int* m_dev) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % BK != 0) return hipErrorInvalidValue;
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  hipLaunchKernelGGL((split3_kernel<BN, kMode>), dim3(tiles), dim3(512), 0, st, M, N, K, lda, ldb,
                     ldc, ah, al, arow, bh, bl, bcol, C, m_dev);
  return hipGetLastError();
}

// T = W M^T for the layer, all rows (jarq_prepare): W's two fp16 planes
// against M's, three products.
hipError_t launch_wm_product(hipStream_t st, int rows, int cols, const char* ws,
                             const Layout& lay, const _Float16* whi, const _Float16* wlo,
                             const float* wrow_inv) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const _Float16* bh = (const _Float16*)(ws + lay.mhi);
  const _Float16* bl = (const _Float16*)(ws + lay.mlo);
  const float* bc = (const float*)(ws + lay.mrow);
  return launch_split3_t<256, 0>(st, rows, cols, cols, cols, cols, cols, whi, wlo, wrow_inv, bh,
                                 bl, bc, (float*)(ws + lay.tm), nullptr);
}

// ---- residual product from the exact codes ----
//
// With E = W - What and What(j, k) = s(j, i) (q(j, k) - z(j, i)) for k in group
// i (eq. (1)), U = E M^T = T - What M^T with T = W M^T fixed for the layer
// (formed once by jarq_prepare with split3_kernel).  The codes minus
// zero points are small integers, exact in fp16 (the cz plane), so
//   (What M^T)(j, n) = 2^-t_n sum_i s(j, i) sum_{k in i} cz(j, k) (Mh + Ml)(n, k)
// needs two products per k-slice instead of three; each group's partial sum
// (seg, exact products accumulated in fp32 on the matrix cores) is scaled by
// its row's s and added to the running sum in fp32 when the group ends.
//
// Tiling: 256 x 128 output tile per 512-thread work-group, 4 x 2 waves of
// 64 x 64 (two 32 x 32 blocks each way: the accumulators and the group's
// partial sums both fit next to the fragments at two waves per SIMD), K in
// steps of 64 (32 when g = 32) straight from global memory into two LDS
// stages by direct loads.  A stage row holds CPR 16-byte chunks; chunk c of
// tile row r sits at position c ^ rswz(r).  A 16-byte read serves 16 lanes
// (256 bytes, all 64 banks) per clock, and the lanes of a fragment read are
// 16 consecutive rows at one chunk: with 128-byte rows, two rows share each
// 256-byte bank line, so row r's position must differ from every other row
// of the 16 with the same parity (rswz = (r / 2) mod 8); with 64-byte rows,
// four rows share a line and (r / 4) mod 4 separates the rows of each
// residue mod 4.  Fragment reads run one k-slice ahead of the products.  Rows
// of cz, the scales and T are the layer's rows (gathered through the row
// map); U is stored by position.
namespace {
constexpr int RBM = 256, RBN = 128;
template <int CPR>
__device__ __forceinline__ int rswz(int r) {
  if constexpr (CPR == 8) return (r >> 1) & 7;
  return (r >> 2) & 3;
}
}  // namespace

template <int G_SIZE>
__global__ __launch_bounds__(512, 1) void resid_kernel(
    int M, int N, int K, const _Float16* __restrict__ Cz, const float* __restrict__ scales,
    const _Float16* __restrict__ Bh, const _Float16* __restrict__ Bl,
    const float* __restrict__ bcol_inv, const float* __restrict__ T, float* __restrict__ U,
    const int32_t* __restrict__ rowmap, const int* __restrict__ m_dev) {
  if (m_dev != nullptr) M = *m_dev;
  constexpr int g = G_SIZE;
  constexpr int RBK = g >= 64 ? 64 : 32;                 // k per stage
  constexpr int KQ = RBK / 16;                           // k-slices per stage
  constexpr int CPR = RBK / 8;                           // 16-byte chunks per stage row
  constexpr int RPP = 64 / CPR;                          // rows per 1 KB piece
  constexpr int SPG = g / RBK;                           // stages per group
  constexpr int A_PLANE = RBM * RBK, B_PLANE = RBN * RBK;  // halves
  constexpr int APW = RBM / RPP / 8, BPW = RBN / RPP / 8;  // pieces per wave per plane
  constexpr int STAGE = A_PLANE + 2 * B_PLANE;
  __shared__ __attribute__((aligned(1024))) _Float16 buf0[STAGE];
  __shared__ __attribute__((aligned(1024))) _Float16 buf1[STAGE];
  __shared__ __attribute__((aligned(16))) float sc_s[2][RBM];  // s of the tile's rows, current / next group
  __shared__ int lr_s[RBM];                                     // layer row of each tile row
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lm = lane & 31, kh = lane >> 5;
  const int G = K / g;
  const int nbm = (M + RBM - 1) / RBM, nbn = (N + RBN - 1) / RBN;
  int tm, tn;
  if (M <= 0 || !tile_of(blockIdx.x, nbm, nbn, tm, tn)) return;  // uniform across the work-group
  const int m0 = tm * RBM, n0 = tn * RBN;
  // Tile rows past the edge take the tile's first row: their products only
  // reach outputs that are never stored.
  if (tid < RBM) lr_s[tid] = map_row(rowmap, m0 + (m0 + tid < M ? tid : 0));
  __syncthreads();

  // Direct loads, 16 bytes per lane, one 1 KB piece (RPP rows) per
  // instruction: wave w fills pieces w, w + 8, ... of each plane; lane L holds
  // row RPP j + L / CPR at position L % CPR, i.e. chunk (L % CPR) ^ rswz(row).
  unsigned aoff[APW], boff[BPW];
#pragma unroll
  for (int i = 0; i < APW; ++i) {
    const int r = RPP * (wave + 8 * i) + lane / CPR;
    aoff[i] = (unsigned)lr_s[r] * (unsigned)K + (unsigned)(((lane % CPR) ^ rswz<CPR>(r)) * 8);
  }
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int r = RPP * (wave + 8 * i) + lane / CPR;
    const int gn = n0 + r;
    boff[i] = (unsigned)(gn < N ? gn : 0) * (unsigned)K + (unsigned)(((lane % CPR) ^ rswz<CPR>(r)) * 8);
  }
  // load j (0 .. NDMA - 1) of a stage's direct loads: the cz pieces first,
  // then the M pieces, high and low plane in turn
  constexpr int NDMA = APW + 2 * BPW;
  auto issue_one = [&](int j, int k0, _Float16* stage) {
    if (j < APW) {
      dma16(Cz + k0 + aoff[j], stage + (wave + 8 * j) * 512);
    } else {
      const int i = (j - APW) >> 1;
      if (((j - APW) & 1) == 0)
        dma16(Bh + k0 + boff[i], stage + A_PLANE + (wave + 8 * i) * 512);
      else
        dma16(Bl + k0 + boff[i], stage + A_PLANE + B_PLANE + (wave + 8 * i) * 512);
    }
  };
  auto issue = [&](int k0, _Float16* stage) {
#pragma unroll
    for (int j = 0; j < NDMA; ++j) issue_one(j, k0, stage);
  };
  // the tile's scales of group i into sc_s[i & 1] (threads 0..RBM-1)
  auto stage_scales = [&](int i) {
    if (tid < RBM) sc_s[i & 1][tid] = scales[(size_t)lr_s[tid] * G + i];
  };

  f32x16 acc[2][2], seg[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  auto lds_rd = [&](const _Float16* plane, int r, int q) {
    const int c = 2 * q + kh;  // k-slice q: chunks 2 q (lanes 0-31) and 2 q + 1
    const uint32_t ad = (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)(
        plane + r * RBK + ((c ^ rswz<CPR>(r)) << 3));
    f16x8 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(ad));
    return v;
  };
  // One stage (KQ k-slices of 16) on `base`; `first`: the stage opens a group
  // (its products start the partial sums from zero).  The six reads of slice
  // q + 1 are issued before the wait for slice q (LDS returns in order), and
  // the next stage's direct loads (into `stn` at k0n; none if k0n < 0) are
  // spread over the slices.
  auto compute = [&](const _Float16* base, bool first, int k0n, _Float16* stn) {
    f16x8 af[2][2], bh[2][2], bl[2][2];  // [slot][block]
    auto rd = [&](int q, int sl) {
#pragma unroll
      for (int a = 0; a < 2; ++a) af[sl][a] = lds_rd(base, wm * 64 + a * 32 + lm, q);
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        bh[sl][b] = lds_rd(base + A_PLANE, wn * 64 + b * 32 + lm, q);
        bl[sl][b] = lds_rd(base + A_PLANE + B_PLANE, wn * 64 + b * 32 + lm, q);
      }
    };
    rd(0, 0);
#pragma unroll
    for (int q = 0; q < KQ; ++q) {
      const int sl = q & 1;
      if (k0n >= 0) {
#pragma unroll
        for (int j = q * NDMA / KQ; j < (q + 1) * NDMA / KQ; ++j) issue_one(j, k0n, stn);
      }
      if (q + 1 < KQ) {
        rd(q + 1, sl ^ 1);
        if (sl == 0)
          asm volatile("s_waitcnt lgkmcnt(6)"
                       : "+v"(af[0][0]), "+v"(af[0][1]), "+v"(bh[0][0]), "+v"(bh[0][1]),
                         "+v"(bl[0][0]), "+v"(bl[0][1]));
        else
          asm volatile("s_waitcnt lgkmcnt(6)"
                       : "+v"(af[1][0]), "+v"(af[1][1]), "+v"(bh[1][0]), "+v"(bh[1][1]),
                         "+v"(bl[1][0]), "+v"(bl[1][1]));
      } else {
        if (sl == 0)
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(af[0][0]), "+v"(af[0][1]), "+v"(bh[0][0]), "+v"(bh[0][1]),
                         "+v"(bl[0][0]), "+v"(bl[0][1]));
        else
          asm volatile("s_waitcnt lgkmcnt(0)"
                       : "+v"(af[1][0]), "+v"(af[1][1]), "+v"(bh[1][0]), "+v"(bh[1][1]),
                         "+v"(bl[1][0]), "+v"(bl[1][1]));
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const f32x16 c0 = (first && q == 0) ? f32x16{} : seg[a][b];
          seg[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[sl][a], bh[sl][b], c0, 0, 0, 0);
          seg[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[sl][a], bl[sl][b], seg[a][b], 0, 0, 0);
        }
    }
  };
  // acc += s (per row) * seg at the end of group i; element v of a block is
  // row 8 (v / 4) + 4 (lane / 32) + v % 4
  auto fold = [&](int i) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const f32x4 s4 = *(const f32x4*)&sc_s[i & 1][wm * 64 + a * 32 + 8 * v4 + 4 * kh];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int u = 0; u < 4; ++u)
            acc[a][b][4 * v4 + u] = fmaf(seg[a][b][4 * v4 + u], s4[u], acc[a][b][4 * v4 + u]);
      }
    }
  };

  // Double buffering: the loads of stage k + 1 fly while stage k computes;
  // the barrier at the end of a stage (which waits for this thread's
  // outstanding loads) makes the next stage visible and frees the one just
  // read.  The scales of group i + 1 are staged during group i (their buffer
  // was last read by group i - 1's fold, before a barrier).
  const int nk = K / RBK;
  stage_scales(0);
  issue(0, buf0);
  __syncthreads();
  for (int i = 0; i < G; ++i) {
    if (i + 1 < G) stage_scales(i + 1);
#pragma unroll
    for (int ks = 0; ks < SPG; ++ks) {  // unrolled: whether a stage opens its group is known
      const int kt = i * SPG + ks;
      _Float16* cur = (kt & 1) ? buf1 : buf0;
      _Float16* nxt = (kt & 1) ? buf0 : buf1;
      compute(cur, ks == 0, kt + 1 < nk ? (kt + 1) * RBK : -1, nxt);
      if (ks == SPG - 1) fold(i);
      __syncthreads();
    }
  }

  // Epilogue: U = T - acc 2^-t_n.  Accumulator element v of lane l in a
  // 32 x 32 block: (row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32).
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int tb = wm * 64 + a * 32 + 4 * kh;  // tile row of element v: tb + 8 (v / 4) + v % 4
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = n0 + wn * 64 + b * 32 + lm;
      const int colc = min(col, N - 1);
      const float cs = bcol_inv[colc];
      float tv[16];
#pragma unroll
      for (int v = 0; v < 16; ++v)
        tv[v] = T[(size_t)lr_s[tb + 8 * (v / 4) + (v % 4)] * N + colc];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + tb + 8 * (v / 4) + (v % 4);
        if (row < M && col < N) U[(size_t)row * N + col] = tv[v] - acc[a][b][v] * cs;
      }
    }
  }
}

template <int G_SIZE>
static hipError_t launch_resid_t(hipStream_t st, int rows, int cols, const char* ws,
                                 const Layout& lay, const float* scales, float* U,
                                 const int32_t* rowmap, const int* n_dev, hipEvent_t ev_start,
                                 hipEvent_t ev_stop) {
  const int tiles = ((rows + RBM - 1) / RBM) * ((cols + RBN - 1) / RBN);
  if (ev_start != nullptr || ev_stop != nullptr) {
    // timed: the events take the dispatch's own timestamps
    hipExtLaunchKernelGGL((resid_kernel<G_SIZE>), dim3(tiles), dim3(512), 0, st, ev_start,
                          ev_stop, 0u, rows, cols, cols, (const _Float16*)(ws + lay.cz), scales,
                          (const _Float16*)(ws + lay.mhi), (const _Float16*)(ws + lay.mlo),
                          (const float*)(ws + lay.mrow), (const float*)(ws + lay.tm), U, rowmap,
                          n_dev);
  } else {
    hipLaunchKernelGGL((resid_kernel<G_SIZE>), dim3(tiles), dim3(512), 0, st, rows, cols, cols,
                       (const _Float16*)(ws + lay.cz), scales, (const _Float16*)(ws + lay.mhi),
                       (const _Float16*)(ws + lay.mlo), (const float*)(ws + lay.mrow),
                       (const float*)(ws + lay.tm), U, rowmap, n_dev);
  }
  return hipGetLastError();
}

hipError_t launch_resid(hipStream_t st, int rows, int cols, int g, const char* ws,
                        const Layout& lay, const float* scales, float* U, const int32_t* rowmap,
                        const int* n_dev, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (rows <= 0 || cols <= 0) {  // nothing to launch: the events still mark the spot
    hipError_t e = hipSuccess;
    if (ev_start != nullptr) e = hipEventRecord(ev_start, st);
    if (e == hipSuccess && ev_stop != nullptr) e = hipEventRecord(ev_stop, st);
    return e;
  }
  if (cols % BK != 0) return hipErrorInvalidValue;
  switch (g) {
    case 32:
      return launch_resid_t<32>(st, rows, cols, ws, lay, scales, U, rowmap, n_dev, ev_start, ev_stop);
    case 64:
      return launch_resid_t<64>(st, rows, cols, ws, lay, scales, U, rowmap, n_dev, ev_start, ev_stop);
    case 128:
      return launch_resid_t<128>(st, rows, cols, ws, lay, scales, U, rowmap, n_dev, ev_start,
                                 ev_stop);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jarq
