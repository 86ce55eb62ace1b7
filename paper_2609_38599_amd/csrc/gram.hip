// Grouped Gram matrices of the scale update (paper eqs. (5)-(6)).
//
// For row j with c_i = q_i - z_i 1 (exact small integers), entry (a, h) of
// B_j^T B_j is c_a^T H_ah c_h (B_j has columns A_i c_i and H = A^T A).  The
// matrix is symmetric, so only h >= a is formed, always the same way: T =
// H(a-group, h-group) C(rows, h-group)^T on fp16 matrix cores
// (v_mfma_f32_32x32x16_f16, M = the g weights of group a, N = 32 rows, K = the
// g weights of group h) with H as its two fp16 planes and the codes exact in
// fp16, then T reduced against c_a for every row (block_entries below).
//
// Full build: a work-group takes a tile of 128 rows and a pair of row-groups
// {p, G-1-p} (so every work-group walks G+1 blocks).
//
// Incremental build: entry (a, h) depends on the codes of groups a and h
// only, so after a code update only the entries of groups whose codes changed
// need forming.  The code update lists, per group x, the rows whose group x
// it changed (in any order), and a work-group takes a tile of
// 128 listed rows of one x and forms the G entries of row and column x of
// their matrices, (a, x) for a < x and (x, h) for h >= x, with the same
// block_entries arithmetic, so every entry is bit-identical to the full
// build's.  An entry of two changed groups is formed twice, to the same bits.
// The build chooses the incremental form when the last code update left a
// complete set of matrices and the listed work is smaller (gram_use_lists);
// every work-group of both kernels reaches the same choice.
//
// Waves split the a-group into 32-weight blocks and the tile's rows; each H
// fragment is used for all of a wave's rows.  Codes are staged in LDS as fp16
// (bit trick: the fp16 with bits 0x6400 | q is 1024 + q) and the next block's
// codes are fetched while the current block runs on the matrix cores.  Two
// work-groups share a CU (LDS and registers sized for it), so one's staging,
// reduction and H loads overlap the other's matrix work.
//
// The matrices are stored by layer row: a row's matrix survives the sweeps in
// which it is not rebuilt, whatever its position in the sweep's row list.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

namespace {
constexpr int RT = 128;  // rows per work-group
constexpr int kMaxGramGroups = 128;  // the most groups a layer may have

// Four codes (one byte each) -> four fp16 values q - z, exactly.
__device__ __forceinline__ void codes_to_f16(uint32_t q4, f16x2 zz, f16x2* out) {
  // 0x64qq as fp16 is 1024 + q
  const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, q4, 0x07010700u);  // [q1, 0x64, q0, 0x64]
  const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, q4, 0x07030702u);  // [q3, 0x64, q2, 0x64]
  out[0] = __builtin_bit_cast(f16x2, lo) - zz;
  out[1] = __builtin_bit_cast(f16x2, hi) - zz;
}

// Whether this sweep's build uses the row lists: the matrices of the last
// sweep are complete (ctl->valid) and the listed tiles walk clearly fewer
// blocks than the full build (tiles of 128 rows x G blocks per changed group,
// against pairs of a-groups x (G + 1) blocks per tile of the n rows; a listed
// block costs more, its work-group stages the codes of two groups).
// Evaluated by whole wavefronts: lane l reads the lengths of the lists of
// groups l and l + 64 (a layer has at most 128 groups), and a reduction over
// the lanes gives every lane the same answer.
__device__ __forceinline__ int list_length(const int32_t* gpre, int x) {
  return gpre[x * (kSubLists + 1) + kSubLists];
}
__device__ __forceinline__ bool gram_use_lists(const GramCtl* ctl, const int32_t* gpre, int G,
                                               int n) {
  if (ctl == nullptr || ctl->valid == 0) return false;
  const int lane = threadIdx.x & 63;
  int tiles = 0;
  if (lane < G) tiles += (list_length(gpre, lane) + RT - 1) / RT;
  if (lane + 64 < G) tiles += (list_length(gpre, lane + 64) + RT - 1) / RT;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) tiles += __shfl_xor(tiles, off);
  const long long listed = tiles;
  const long long full = (long long)((n + RT - 1) / RT) * ((G + 1) / 2) * (G + 1);
  return 3 * listed * G < 2 * full;
}
}  // namespace

// ---- pieces shared by both builds (so every entry has one arithmetic) ----

template <int G_SIZE>
struct GramShape {
  static constexpr int g = G_SIZE;
  static constexpr int NAB = g / 32;       // 32-weight blocks of an a-group
  static constexpr int WPA = 4 / NAB;      // waves sharing an a-block
  static constexpr int RW = RT / WPA;      // rows per wave
  static constexpr int JB = RW / 32;       // 32-row blocks per wave
  static constexpr int KS = g / 16;        // k-steps of one block
  static constexpr int LDC = g + 8;        // fp16 row stride of staged code tiles
  static constexpr int TPR = 256 / RT;     // threads per staged row
  static constexpr int CPT = g / TPR;      // codes per thread
  static constexpr size_t lds_bytes() {
    return (size_t)2 * RT * LDC * sizeof(_Float16) + (size_t)NAB * RT * sizeof(double);
  }
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Codes of column block `blk` of layer row lrow (this thread's part: codes
// tpart * CPT .. + CPT of the group) and the group's zero point.
template <int G_SIZE>
struct CodeStage {
  u32x4 q[GramShape<G_SIZE>::CPT / 16];
  int z;
  __device__ __forceinline__ void fetch(const uint8_t* __restrict__ codes,
                                        const int32_t* __restrict__ zeros, int lrow, int blk,
                                        int cols, int G, int tpart) {
    constexpr int g = G_SIZE, CPT = GramShape<G_SIZE>::CPT;
    const u32x4* src = (const u32x4*)(codes + (size_t)lrow * cols + (size_t)blk * g + tpart * CPT);
#pragma unroll
    for (int i = 0; i < CPT / 16; ++i) q[i] = src[i];
    z = zeros[(size_t)lrow * G + blk];
  }
  // as fp16 c = q - z into row trow of a staged tile
  __device__ __forceinline__ void store(_Float16* dst, int trow, int tpart) const {
    constexpr int CPT = GramShape<G_SIZE>::CPT, LDC = GramShape<G_SIZE>::LDC;
    const _Float16 zb = (_Float16)(1024 + z);
    const f16x2 zz = f16x2{zb, zb};
    _Float16* drow = dst + trow * LDC + tpart * CPT;
#pragma unroll
    for (int i = 0; i < CPT / 16; ++i) {
      f16x2 v[8];
#pragma unroll
      for (int w = 0; w < 4; ++w) codes_to_f16(q[i][w], zz, v + 2 * w);
      *(f16x8*)(drow + i * 16) = f16x8{v[0][0], v[0][1], v[1][0], v[1][1], v[2][0], v[2][1], v[3][0], v[3][1]};
      *(f16x8*)(drow + i * 16 + 8) = f16x8{v[4][0], v[4][1], v[5][0], v[5][1], v[6][0], v[6][1], v[7][0], v[7][1]};
    }
  }
};

// H fragments of block (a-group ga, column block h) for this wave's a-block.
template <int G_SIZE>
__device__ __forceinline__ void fetch_h(f16x8 (&hf)[2][GramShape<G_SIZE>::KS],
                                        const _Float16* __restrict__ Hh,
                                        const _Float16* __restrict__ Hl, int ga, int h, int cols,
                                        int lane, int wave) {
  using S = GramShape<G_SIZE>;
  const int lm = lane & 31, kh = lane >> 5, ab = wave % S::NAB;
  const size_t rowoff = (size_t)(ga * S::g + ab * 32 + lm) * cols + (size_t)h * S::g + 8 * kh;
#pragma unroll
  for (int ks = 0; ks < S::KS; ++ks) {
    hf[0][ks] = *(const f16x8*)(Hh + rowoff + ks * 16);
    hf[1][ks] = *(const f16x8*)(Hl + rowoff + ks * 16);
  }
}

// Entries (ga, h) of the tile's rows from the staged codes of h (ch_s), of ga
// (ca_s) and the H fragments in hf: the products, the reduction against c_a
// over this wave's 32 a-weights (fp32, then fp64 across the wave halves) into
// red.  The entry of tile row t is then entry_value(red, t).
template <int G_SIZE>
__device__ __forceinline__ void block_entries(const _Float16* ca_s, const _Float16* ch_s,
                                              const f16x8 (&hf)[2][GramShape<G_SIZE>::KS],
                                              double* red, int lane, int wave) {
  using S = GramShape<G_SIZE>;
  constexpr int JB = S::JB, KS = S::KS, LDC = S::LDC;
  const int lm = lane & 31, kh = lane >> 5;
  const int ab = wave % S::NAB;
  const int rbase = (wave / S::NAB) * S::RW;
  f32x16 acc[JB];
#pragma unroll
  for (int b = 0; b < JB; ++b) acc[b] = f32x16{};
  // Code fragments of k-slice ks + 1 are read while slice ks is on the matrix
  // cores (LDS latency off the critical path).
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
}

template <int G_SIZE>
__device__ __forceinline__ float entry_value(const double* red, int t, float hinv) {
  double s = 0.0;
#pragma unroll
  for (int a = 0; a < GramShape<G_SIZE>::NAB; ++a) s += red[a * RT + t];
  return (float)(s * (double)hinv);
}

// ---- full build: 128 positions x a pair of a-groups per work-group ----
template <int G_SIZE>
__global__ __launch_bounds__(256, 2) void gram_kernel(int rows, int cols,
                                                      const _Float16* __restrict__ Hh,
                                                      const _Float16* __restrict__ Hl,
                                                      const float* __restrict__ h_inv,
                                                      const uint8_t* __restrict__ codes,
                                                      const int32_t* __restrict__ zeros,
                                                      float* __restrict__ gram,
                                                      const int32_t* __restrict__ rowmap,
                                                      const int* __restrict__ n_dev,
                                                      GramCtl* __restrict__ ctl,
                                                      const int32_t* __restrict__ gpre) {
  using S = GramShape<G_SIZE>;
  const int G = cols / S::g;
  const int n = n_dev != nullptr ? *n_dev : rows;
  // every work-group takes the same branch (same counts, same n)
  const bool lists = gram_use_lists(ctl, gpre, G, n);
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0 && ctl != nullptr)
    ctl->listed = lists ? 1 : 0;
  if (lists) return;
  const int r0 = blockIdx.x * RT;
  if (r0 >= n) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tid = threadIdx.x;
  const float hinv = *h_inv;
  extern __shared__ _Float16 sm[];
  _Float16* ch_s = sm;                        // RT x LDC: c of block h
  _Float16* ca_s = ch_s + RT * S::LDC;        // RT x LDC: c of the a-group
  double* red = (double*)(ca_s + RT * S::LDC);  // NAB x RT
  // Layer row of tile row t (positions past the end repeat the tile's first:
  // unconditional loads, never stored).
  auto layer_row = [&](int t) { return map_row(rowmap, r0 + (r0 + t < n ? t : 0)); };
  const int trow = tid / S::TPR, tpart = tid % S::TPR;
  const int lrow = layer_row(trow);
  CodeStage<G_SIZE> st;
  f16x8 hf[2][S::KS];
  const int p = blockIdx.y;
  // Thread tid < RT owns tile row tid: it keeps its entries (ga, h) for up to
  // 32 consecutive h in registers and stores them as one contiguous run.
  float* grow_out = gram + (size_t)layer_row(tid < RT ? tid : 0) * G * G;
  float outv[32];
#pragma unroll
  for (int q = 0; q < 32; ++q) outv[q] = 0.f;
  for (int side = 0; side < 2; ++side) {
    const int ga = side == 0 ? p : G - 1 - p;
    if (side == 1 && ga == p) break;
    lds_barrier();
    st.fetch(codes, zeros, lrow, ga, cols, G, tpart);
    st.store(ca_s, trow, tpart);
    st.fetch(codes, zeros, lrow, ga, cols, G, tpart);  // block h = ga comes first
    for (int h = ga; h < G; ++h) {
      lds_barrier();  // previous block's reads of ch_s are done
      st.store(ch_s, trow, tpart);
      // H fragments of this block (their latency is covered by the other
      // work-group on the CU), codes of the next one
      fetch_h<G_SIZE>(hf, Hh, Hl, ga, h, cols, lane, wave);
      if (h + 1 < G) st.fetch(codes, zeros, lrow, h + 1, cols, G, tpart);
      lds_barrier();
      block_entries<G_SIZE>(ca_s, ch_s, hf, red, lane, wave);
      lds_barrier();
      if (tid < RT) {
        const float val = entry_value<G_SIZE>(red, tid, hinv);
        const int j = (h - ga) & 31;
#pragma unroll
        for (int q = 0; q < 32; ++q) outv[q] = q == j ? val : outv[q];
        if ((j == 31 || h == G - 1) && r0 + tid < n) {
          float* dst = grow_out + (size_t)ga * G + (h - j);
#pragma unroll
          for (int q = 0; q < 32; ++q)
            if (q <= j) dst[q] = outv[q];
        }
      }
    }
  }
}

// ---- incremental build: persistent work-groups over (x, tile, chunk) ----
// Item (x, c, t): tile t (128 rows) of the list of group x, blocks b in chunk
// c (`chunk` consecutive blocks); block b forms entry (b, x) for b < x and
// (x, b) for b >= x.  The codes of x stay staged while the chunk runs.  Items
// are numbered with the tile fastest, and each round of the grid deals a
// contiguous range of items to each XCD (work-groups go to the 8 XCDs in
// turn), so the tiles that read the same H blocks share that XCD's L2.  A
// work-group's blocks run one after another, each behind its own H loads, so
// the launch lasts as long as the busiest work-group's blocks: the chunk (4,
// 2 or 1 blocks) is the one that gives the fewest blocks to the busiest
// work-group, rounds x chunk with rounds = ceil(items / grid), the larger
// chunk on a tie (fewer stagings of the codes of x).
constexpr int kChunk = 4;

template <int G_SIZE>
__global__ __launch_bounds__(256, 2) void gram_listed_kernel(
    int rows, int cols, const _Float16* __restrict__ Hh, const _Float16* __restrict__ Hl,
    const float* __restrict__ h_inv, const uint8_t* __restrict__ codes,
    const int32_t* __restrict__ zeros, float* __restrict__ gram, const int* __restrict__ n_dev,
    const GramCtl* __restrict__ ctl, const int32_t* __restrict__ glist,
    const int32_t* __restrict__ gpre, int list_cap) {
  using S = GramShape<G_SIZE>;
  const int G = cols / S::g;
  const int n = n_dev != nullptr ? *n_dev : rows;
  if (!gram_use_lists(ctl, gpre, G, n)) return;  // uniform
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tid = threadIdx.x;
  const float hinv = *h_inv;
  extern __shared__ _Float16 sm[];
  _Float16* cx_s = sm;                        // RT x LDC: c of group x
  _Float16* cb_s = cx_s + RT * S::LDC;        // RT x LDC: c of block b
  double* red = (double*)(cb_s + RT * S::LDC);  // NAB x RT
  // first_s[x]: first item of group x's list (an exclusive scan of the tile
  // counts over the groups, Hillis-Steele over 128 + 1 entries, times the
  // chunks per tile)
  __shared__ int first_s[kMaxGramGroups + 1];
  __shared__ int scan_s[kMaxGramGroups];
  if (tid < kMaxGramGroups)
    scan_s[tid] = tid < G ? (list_length(gpre, tid) + RT - 1) / RT : 0;
  __syncthreads();
  for (int w = 1; w < kMaxGramGroups; w <<= 1) {
    const int v = (tid < kMaxGramGroups && tid >= w) ? scan_s[tid - w] : 0;
    __syncthreads();
    if (tid < kMaxGramGroups) scan_s[tid] += v;
    __syncthreads();
  }
  const int tiles_all = scan_s[kMaxGramGroups - 1];  // same in every work-group
  const int grid = (int)gridDim.x;
  int chunk = kChunk;
  {
    int best = ((tiles_all * ((G + kChunk - 1) / kChunk) + grid - 1) / grid) * kChunk;
    for (int c = kChunk / 2; c >= 1; c /= 2) {
      const int busiest = ((tiles_all * ((G + c - 1) / c) + grid - 1) / grid) * c;
      if (busiest < best) {
        best = busiest;
        chunk = c;
      }
    }
  }
  const int nch = (G + chunk - 1) / chunk;
  if (tid <= kMaxGramGroups) first_s[tid] = tid == 0 ? 0 : scan_s[tid - 1] * nch;
  __syncthreads();
  const int items = first_s[G];
  const int trow = tid / S::TPR, tpart = tid % S::TPR;
  CodeStage<G_SIZE> st, stx;
  f16x8 hf[2][S::KS];
  // Item geometry; the codes of x and of the item's first block are fetched
  // one item ahead (during the previous item's last block).
  struct Item {
    int x, b0, b1, r0, ntile, lrow, orow;
  };
  // Layer row at position k of group x's list (the concatenation of its
  // sub-lists): k lies in the last sub-list that starts at or before it.
  auto list_row = [&](int x, int k) {
    const int32_t* pr = gpre + x * (kSubLists + 1);
    int s = 0;
#pragma unroll
    for (int q = 1; q < kSubLists; ++q) s = pr[q] <= k ? q : s;
    return glist[((size_t)x * kSubLists + s) * list_cap + (k - pr[s])];
  };
  auto locate = [&](int item) {
    Item it;
    // the last x with first_s[x] <= item (binary search; empty lists share
    // their first item with the next list)
    int lo = 0, hi = G - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (first_s[mid] <= item) lo = mid; else hi = mid - 1;
    }
    const int x = lo;
    const int local = item - first_s[x];
    const int len = list_length(gpre, x);
    const int tiles = (len + RT - 1) / RT;
    const int c = local / tiles, t = local - c * tiles;
    it.x = x;
    it.r0 = t * RT;
    it.ntile = len;
    it.lrow = list_row(x, it.r0 + (it.r0 + trow < len ? trow : 0));
    // the output row of thread tid < RT
    it.orow = list_row(x, it.r0 + (tid < RT && it.r0 + tid < len ? tid : 0));
    it.b0 = c * chunk;
    it.b1 = min(it.b0 + chunk, G);
    return it;
  };
  // Position of this work-group in its round.  Work-groups go to the 8 XCDs
  // in turn, two per CU: the first half of the positions takes the first
  // per_xcd / 2 work-groups of every XCD (one per CU), XCD-major, the second
  // half the others, so a short last round spreads over every XCD, one
  // work-group per CU, while runs of consecutive items (tiles that read the
  // same H blocks) still share an XCD's L2.
  const int per_xcd = gridDim.x / 8;
  const int wg = (int)blockIdx.x, local = wg / 8;
  int slot;
  if (per_xcd % 2 == 0) {
    const int half = per_xcd / 2;
    slot = (local / half) * (int)(gridDim.x / 2) + (wg % 8) * half + local % half;
  } else {
    slot = (wg % 8) * per_xcd + local;
  }
  int item = slot;
  if (item >= items) return;  // uniform
  Item it = locate(item);
  stx.fetch(codes, zeros, it.lrow, it.x, cols, G, tpart);
  st.fetch(codes, zeros, it.lrow, it.b0, cols, G, tpart);
  // Each entry is stored one block late, after the next block's loads have
  // been issued: loads and stores retire in order, so a store issued before
  // them would hold up the wait for those loads.
  float* pend_at = nullptr;
  float pend_v = 0.f;
  while (true) {
    const int x = it.x;
    const bool store = tid < RT && it.r0 + tid < it.ntile;
    float* grow_out = gram + (size_t)it.orow * G * G;
    const int next = item + gridDim.x;
    Item nt = it;
    lds_barrier();  // the previous item's reads are done
    stx.store(cx_s, trow, tpart);
    for (int b = it.b0; b < it.b1; ++b) {
      const int ga = b < x ? b : x, h = b < x ? x : b;
      if (b > it.b0) lds_barrier();  // previous block's reads of cb_s are done
      st.store(cb_s, trow, tpart);
      fetch_h<G_SIZE>(hf, Hh, Hl, ga, h, cols, lane, wave);
      if (b + 1 < it.b1) {
        st.fetch(codes, zeros, it.lrow, b + 1, cols, G, tpart);
      } else if (next < items) {
        nt = locate(next);
        stx.fetch(codes, zeros, nt.lrow, nt.x, cols, G, tpart);
        st.fetch(codes, zeros, nt.lrow, nt.b0, cols, G, tpart);
      }
      if (pend_at != nullptr) *pend_at = pend_v;
      lds_barrier();
      // (a, h) codes: (b, x) left of the diagonal block, (x, b) from it on
      block_entries<G_SIZE>(b < x ? cb_s : cx_s, b < x ? cx_s : cb_s, hf, red, lane, wave);
      lds_barrier();
      pend_at = store ? grow_out + (size_t)ga * G + h : nullptr;
      if (store) pend_v = entry_value<G_SIZE>(red, tid, hinv);
    }
    if (next >= items) break;
    item = next;
    it = nt;
  }
  if (pend_at != nullptr) *pend_at = pend_v;
}

template <int G_SIZE>
static hipError_t launch_gram_t(hipStream_t st, int rows, int cols, const char* ws,
                                const Layout& lay, const uint8_t* codes, const int32_t* zeros,
                                float* gram, const int32_t* rowmap, const int* n_dev,
                                bool incremental) {
  constexpr int g = G_SIZE;
  const int G = cols / g;
  const size_t lds = GramShape<g>::lds_bytes();
  GramCtl* ctl = incremental ? (GramCtl*)(ws + lay.gctl) : nullptr;
  const int32_t* glist = (const int32_t*)(ws + lay.glist);
  const int32_t* gpre = (const int32_t*)(ws + lay.gpre);
  static std::atomic<unsigned long long> full_set{0}, listed_set{0};
  hipError_t e = allow_dynamic_lds((const void*)gram_kernel<g>, lds, full_set);
  if (e == hipSuccess && incremental)
    e = allow_dynamic_lds((const void*)gram_listed_kernel<g>, lds, listed_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((gram_kernel<g>), dim3((rows + RT - 1) / RT, (G + 1) / 2), dim3(256), lds,
                     st, rows, cols, (const _Float16*)(ws + lay.hhi),
                     (const _Float16*)(ws + lay.hlo), (const float*)(ws + lay.hscale), codes,
                     zeros, gram, rowmap, n_dev, ctl, gpre);
  if (incremental) {
    // two resident work-groups per CU, each looping over the listed items
    int dev = 0, ncu = 256;
    if (hipGetDevice(&dev) == hipSuccess)
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    const int wgs = (2 * ncu) >= 8 ? ((2 * ncu) & ~7) : 8;  // a multiple of the 8 XCDs
    hipLaunchKernelGGL((gram_listed_kernel<g>), dim3(wgs), dim3(256), lds, st, rows, cols,
                       (const _Float16*)(ws + lay.hhi), (const _Float16*)(ws + lay.hlo),
                       (const float*)(ws + lay.hscale), codes, zeros, gram, n_dev, ctl, glist,
                       gpre, sublist_cap(rows));
  }
  return hipGetLastError();
}

hipError_t launch_gram(hipStream_t st, int rows, int cols, int g, const char* ws,
                       const Layout& lay, const uint8_t* codes, const int32_t* zeros,
                       float* gram, const int32_t* rowmap, const int* n_dev, bool incremental) {
  switch (g) {
    case 32:
      return launch_gram_t<32>(st, rows, cols, ws, lay, codes, zeros, gram, rowmap, n_dev, incremental);
    case 64:
      return launch_gram_t<64>(st, rows, cols, ws, lay, codes, zeros, gram, rowmap, n_dev, incremental);
    case 128:
      return launch_gram_t<128>(st, rows, cols, ws, lay, codes, zeros, gram, rowmap, n_dev, incremental);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jarq
