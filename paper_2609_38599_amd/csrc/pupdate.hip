// Gauss-Seidel update between panels of groups (paper eq. (7), in the
// coordinates of eq. (10)).
//
// The code update visits the groups of a row in order; group i must see the
// accepted changes of every earlier group.  Groups are processed in panels of
// consecutive groups: inside a panel the Babai kernel corrects its own later
// groups, and once a panel is done this kernel folds its accepted changes into
// U = E M^T (M = blockdiag(L_i^{-1}) H) for every later column, all rows at once:
//   U(:, c) -= sum_{h in panel} s_h (dq_h M(c, h-block)^T)       for c >= panel end,
// with dq_h the exact integer code changes (fp16) and M read as its two fp16
// planes (v_mfma_f32_32x32x16_f16, two products); the per-row, per-group scale
// s_h is applied to each group's partial sum in fp32 and the per-column scale
// of M at the end.  B(k, c) = M(c, k) is read along k.
//
// Tiling: 128 x 128 output tile per 256-thread work-group, 2 x 2 waves of
// 64 x 64, K (the panel's columns) in steps of 32 moved straight from global
// memory into a three-stage LDS ring (global_load_lds_dwordx4); two
// work-groups per CU.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

namespace {
constexpr int BM = 128, BN = 128, BK = 32;
constexpr int A_TILE = BM * BK, B_TILE = BN * BK;  // halves
constexpr int STAGE = A_TILE + 2 * B_TILE;
constexpr int DMA_PER_WAVE = STAGE / 512 / 4;     // 1 KB pieces per wave per stage

// Chunk c (16 bytes) of row r of a staged tile sits at position c ^ swz(r).
// A fragment read serves 16 consecutive rows at one chunk per clock, and the
// 64-byte rows share 256-byte bank lines four at a time: rows r, r + 4,
// r + 8, r + 12 need distinct positions.  (r >> 2) & 3 gives them (no
// conflict cycles in the counters; ((r >> 1) + (r >> 3)) & 3 left every
// fragment read 2-way conflicted.)
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

__device__ __forceinline__ void dma16(const _Float16* src, _Float16* lds) {
  __builtin_amdgcn_global_load_lds((const void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Wait until at most n of this wave's vector-memory operations are in flight
// (other counters untouched), then meet the other waves.  The empty asm
// statements keep the compiler from moving LDS accesses across the barrier.
// LDS reads issued as instructions of their own: the compiler does not treat
// them as reads that an outstanding direct-to-LDS load might feed, so it adds
// no wait for those loads; the kernel's own waits (every stage is complete
// before the barrier that precedes its reads) keep them correct.  The caller
// waits for the results with JARQ_LDS_WAIT(...), whose operands are the values the
// wait guards: the compiler cannot see that a read's result arrives later, so
// every use must depend on the wait itself, not only on the read.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}
__device__ __forceinline__ f16x8 lds_read16(uint32_t a) {
  f16x8 r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(a));
  return r;
}
__device__ __forceinline__ f32x4 lds_read16f(uint32_t a) {
  f32x4 r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(a));
  return r;
}
// Operands: "+v"(value) for each value the wait guards.
#define JARQ_LDS_WAIT(...) asm volatile("s_waitcnt lgkmcnt(0)" : __VA_ARGS__ : : "memory")

template <int N>
__device__ __forceinline__ void wait_vm_and_barrier() {
  static_assert(N < 16, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
}  // namespace

__global__ __launch_bounds__(256, 2) void panel_update_kernel(
    int rows, int cols, int g, int c0, int c1, const _Float16* __restrict__ dq,
    const _Float16* __restrict__ Mh, const _Float16* __restrict__ Ml,
    const float* __restrict__ bcol_inv, const float* __restrict__ scales,
    const int32_t* __restrict__ plist, const uint32_t* __restrict__ pcount, int list_cap,
    float* __restrict__ P, const int32_t* __restrict__ rowmap) {
  // Three stages in three distinct arrays: the loads of steps k + 1 and k + 2
  // fly while step k computes.
  __shared__ __attribute__((aligned(1024))) _Float16 buf0[STAGE];
  __shared__ __attribute__((aligned(1024))) _Float16 buf1[STAGE];
  __shared__ __attribute__((aligned(1024))) _Float16 buf2[STAGE];
  __shared__ __attribute__((aligned(16))) float sc_s[kMaxPanelGroups][BM];
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

  // Only rows that accepted a change in the panel need an update: the code
  // update listed them in kSubLists sub-lists (plist, pcount); this
  // work-group takes positions m0 .. m0 + BM - 1 of their concatenation, and
  // work-groups past the end have nothing to do.
  int pre[kSubLists + 1];  // exclusive prefix sums of the sub-list lengths (uniform)
  pre[0] = 0;
#pragma unroll
  for (int s = 0; s < kSubLists; ++s) pre[s + 1] = pre[s] + (int)pcount[s * kCtrStride];
  const int total = pre[kSubLists];
  if (m0 >= total) return;  // uniform across the work-group
  const int nvalid = min(BM, total - m0);
  // The list lives in the third stage, which is first loaded after every
  // use of it (set-up, behind the loop's first barrier); a separate array
  // would push the work-group past half of the LDS (one per CU).
  int* rl_s = (int*)buf2;
  if (tid < BM) {
    // position m lies in the last sub-list that starts at or before it
    const int m = m0 + (tid < nvalid ? tid : 0);
    int s = 0;
#pragma unroll
    for (int q = 1; q < kSubLists; ++q) s = pre[q] <= m ? q : s;
    rl_s[tid] = plist[(size_t)s * list_cap + (m - pre[s])];
  }
  __syncthreads();
  // Tile row t is row rl_s[t] for t < nvalid; later tile rows repeat a valid row
  // and are never stored.
  auto row_of = [&](int t) { return rl_s[t < nvalid ? t : 0]; };

  // Rows of this lane's accumulator elements (element v of a 32x32 block is
  // row 8 (v / 4) + 4 (lane / 32) + v % 4), kept for the epilogue.
  int erow[2][16];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int v = 0; v < 16; ++v) erow[a][v] = row_of(wm * 64 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4));


  // Piece j (1 KB = 16 rows of one plane tile) of a stage goes to wave j % 4;
  // lane L holds row 16 (j % 8) + L / 4, chunk (L % 4) ^ swz(row).  Pieces
  // 0-7: dq rows, 8-15: M high plane rows, 16-23: M low plane rows.  Rows past
  // the edge read row 0: their products reach no stored output.
  unsigned off[DMA_PER_WAVE];
  const _Float16* base[DMA_PER_WAVE];
#pragma unroll
  for (int q = 0; q < DMA_PER_WAVE; ++q) {
    const int j = wave + 4 * q;
    const int r = 16 * (j % 8) + (lane >> 2);
    const int chunk = (lane & 3) ^ swz(r);
    if (j < 8) {
      off[q] = (unsigned)row_of(r) * (unsigned)cols + (unsigned)(chunk * 8);
      base[q] = dq;
    } else {
      const int gn = n0 + r;
      off[q] = (unsigned)(gn < cols ? gn : 0) * (unsigned)cols + (unsigned)(chunk * 8);
      base[q] = j < 16 ? Mh : Ml;
    }
  }
  auto issue = [&](int k0, _Float16* stage) {
#pragma unroll
    for (int q = 0; q < DMA_PER_WAVE; ++q) {
      const int j = wave + 4 * q;
      dma16(base[q] + k0 + off[q], stage + j * 512);
    }
  };
  auto frag = [&](const _Float16* tile, int r, int ks) {
    const int c = (ks >> 3) + kh;
    return lds_read16(lds_addr(tile + r * BK + ((c ^ swz(r)) << 3)));
  };

  f32x16 acc[2][2], seg[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      acc[a][b] = f32x16{};
      seg[a][b] = f32x16{};
    }
  const int steps_per_group = g / BK;
  auto compute = [&](const _Float16* st, int kt) {
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      f16x8 af[2], bh[2], bl[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) af[a] = frag(st, wm * 64 + a * 32 + lm, ks);
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int r = wn * 64 + b * 32 + lm;
        bh[b] = frag(st + A_TILE, r, ks);
        bl[b] = frag(st + A_TILE + B_TILE, r, ks);
      }
      JARQ_LDS_WAIT("+v"(af[0]), "+v"(af[1]), "+v"(bh[0]), "+v"(bh[1]), "+v"(bl[0]),
                    "+v"(bl[1]));
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
      f32x4 s4[2][4];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4)   // rows 8 v4 + 4 (lane / 32) + 0..3 of block a
          s4[a][v4] = lds_read16f(lds_addr(&sc_s[h][wm * 64 + a * 32 + 8 * v4 + 4 * kh]));
      JARQ_LDS_WAIT("+v"(s4[0][0]), "+v"(s4[0][1]), "+v"(s4[0][2]), "+v"(s4[0][3]),
                    "+v"(s4[1][0]), "+v"(s4[1][1]), "+v"(s4[1][2]), "+v"(s4[1][3]));
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const f32x4 q = s4[a][v / 4];
          const float sv = (v % 4 == 0) ? q.x : (v % 4 == 1) ? q.y : (v % 4 == 2) ? q.z : q.w;
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            acc[a][b][v] = fmaf(seg[a][b][v], sv, acc[a][b][v]);
            seg[a][b][v] = 0.f;
          }
        }
    }
  };

  // Step k reads stage k % 3.  Before it: this wave's loads of step k are done
  // (only the loads of step k + 1, issued later, may still fly: at most one
  // stage's worth outstanding, since vector-memory loads complete in order),
  // then all waves meet, which also frees the stage read at step k - 1 for the
  // loads of step k + 2.
  const int nk = (c1 - c0) / BK;  // >= 1
  // The tile rows' scales of the panel's groups into sc_s (the list holds
  // positions; scales are by layer row).  The first two stages' direct loads
  // go out first and every scale load right behind them, so both are in
  // flight together (one round trip where the scales used to be waited for
  // before the stages were issued); the row-map loads, where rows are
  // compacted, precede the stages.  Thread e of the BM x ng entries takes e,
  // e + 256, ... (past the end: the last entry again, loaded and not stored).
  constexpr int SCV = kMaxPanelGroups * BM / 256;
  // one straight-line copy per form of the row map, so that the compiler's
  // waits count exactly the loads each copy issues
  auto stage_first = [&](auto&& layer_row) __attribute__((always_inline)) {
    int lrow[SCV];
    float scv[SCV];
#pragma unroll
    for (int u = 0; u < SCV; ++u) {
      const int e = min(tid + 256 * u, BM * ng - 1);
      lrow[u] = layer_row(row_of(e / ng));
    }
    issue(c0, buf0);
    if (nk > 1) issue(c0 + BK, buf1);
#pragma unroll
    for (int u = 0; u < SCV; ++u) {
      const int e = min(tid + 256 * u, BM * ng - 1);
      scv[u] = scales[(size_t)lrow[u] * G + h0 + e % ng];
    }
#pragma unroll
    for (int u = 0; u < SCV; ++u) {
      const int e = tid + 256 * u;
      if (e < BM * ng) sc_s[e % ng][e / ng] = scv[u];
    }
  };
  if (rowmap != nullptr)
    stage_first([&](int p) { return (int)rowmap[p]; });
  else
    stage_first([](int p) { return p; });
  lds_barrier();  // sc_s; the stages' direct loads are waited for in the loop
  for (int kt = 0; kt < nk; kt += 3) {
    if (kt + 1 < nk) wait_vm_and_barrier<DMA_PER_WAVE>(); else wait_vm_and_barrier<0>();
    if (kt + 2 < nk) issue(c0 + (kt + 2) * BK, buf2);
    compute(buf0, kt);
    if (kt + 1 >= nk) break;
    if (kt + 2 < nk) wait_vm_and_barrier<DMA_PER_WAVE>(); else wait_vm_and_barrier<0>();
    if (kt + 3 < nk) issue(c0 + (kt + 3) * BK, buf0);
    compute(buf1, kt + 1);
    if (kt + 2 >= nk) break;
    if (kt + 3 < nk) wait_vm_and_barrier<DMA_PER_WAVE>(); else wait_vm_and_barrier<0>();
    if (kt + 4 < nk) issue(c0 + (kt + 4) * BK, buf1);
    compute(buf2, kt + 2);
  }

  // Accumulator element v of lane l in a 32x32 block:
  // (row 8 * (v / 4) + 4 * (l / 32) + v % 4, column l % 32).
  // Per 32-row block a: all loads of P (unconditional, from a clamped
  // address) are issued first and every loaded value is taken into its
  // register (the empty asm statements) before the first store.  With loads
  // still in flight at a store under a branch, the compiler waited for every
  // outstanding memory operation, the stores before it included, at each
  // store (one write round trip after another); holding all 64 values at
  // once spills registers.
  float csv[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) csv[b] = bcol_inv[min(n0 + wn * 64 + b * 32 + lm, cols - 1)];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    float pold[2][16];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = min(n0 + wn * 64 + b * 32 + lm, cols - 1);
#pragma unroll
      for (int v = 0; v < 16; ++v) pold[b][v] = P[(size_t)erow[a][v] * cols + col];
    }
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) asm volatile("" : "+v"(pold[b][v]));
    if (a == 0) asm volatile("" : "+v"(csv[0]), "+v"(csv[1]));
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int col = n0 + wn * 64 + b * 32 + lm;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int t = wm * 64 + a * 32 + 8 * (v / 4) + 4 * kh + (v % 4);
        if (t < nvalid && col < cols)
          P[(size_t)erow[a][v] * cols + col] = pold[b][v] - acc[a][b][v] * csv[b];
      }
    }
  }
}

int panel_groups(int g) { return panel_groups_of(g); }

hipError_t launch_panel_update(hipStream_t st, int rows, int cols, int g, int c0, int c1,
                               const char* ws, const Layout& lay, const float* scales, float* P,
                               const int32_t* rowmap) {
  if (c1 >= cols) return hipSuccess;
  if ((c1 - c0) % BK != 0 || (c1 - c0) / g > kMaxPanelGroups) return hipErrorInvalidValue;
  dim3 grid((cols - c1 + BN - 1) / BN, (rows + BM - 1) / BM);
  hipLaunchKernelGGL(panel_update_kernel, grid, dim3(256), 0, st, rows, cols, g, c0, c1,
                     (const _Float16*)(ws + lay.dq), (const _Float16*)(ws + lay.mhi),
                     (const _Float16*)(ws + lay.mlo), (const float*)(ws + lay.mrow), scales,
                     (const int32_t*)(ws + lay.plist),
                     (const uint32_t*)(ws + lay.pcount) +
                         (size_t)(c0 / (g * panel_groups_of(g))) * kSubLists * kCtrStride,
                     sublist_cap(rows), P, rowmap);
  return hipGetLastError();
}

}  // namespace jarq
