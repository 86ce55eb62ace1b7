// Gauss-Seidel code update with bounded Babai proposals (paper Sec. 3.3.2,
// eqs. (7)-(10), acceptance on eq. (8), small-scale skip of App. E.2).
//
// For row j and group i, with e = w - what at the latest codes (new codes for
// groups h < i, previous ones for h >= i; all at the new scales), let
// he = (H e)_i and u = R_i^{-T} he / s_i.  Changing the group's codes by the
// integer vector d changes F_j by s_i^2 (||u - R_i d||^2 - ||u||^2), so the
// proposal of eq. (10) is the nearest-plane back substitution
//   x_l = q_l + (u_l - sum_{m>l} R_i(l,m) d_m) / R_i(l,l),  l = g-1..0,
//   q_l^cand = clip(rint(x_l), 0, 2^b - 1),  d_l = q_l^cand - q_l,
// and it is kept iff it changes a code and the change of F is finite and
// negative.  (This is eq. (10) with v = u + R_i(q - z): v - R_i(q^cand - z) =
// u - R_i d.)  The change is evaluated from the code changes themselves,
//   dF / s_i^2 = ||u - R_i d||^2 - ||u||^2 = sum_l R_i(l,l)^2 a_l (a_l - 2 u_l / R_i(l,l)),
// a_l = (R_i d)_l / R_i(l,l), whose terms vanish exactly where no change
// reaches, so its rounding scales with the change rather than with ||u||^2.
//
// One 512-thread work-group owns 16 rows and visits the groups of one panel
// [i0, i1) in order; P holds U = E M^T (M = blockdiag(L_i^{-1}) H) with the
// changes of earlier panels already folded in (pupdate.hip), so its group-i
// columns are L_i^{-1} (H e)_i for codes as they were when the panel began.
// Waves 0-3 run the back substitution of group i while waves 4-7 prepare
// group i + 1:
//   correction: u_{i+1} s_{i+1} = P_{i+1} - sum_{i0<=h<=i} s_h dq_h M(i+1, h)^T,
//     dq_h the accepted code changes of the panel's earlier groups (exact in
//     fp16, zero elsewhere) and the block M(i+1, h) = L_{i+1}^{-1} H_{i+1,h}
//     read as two fp16 terms: two v_mfma_f32_16x16x32_f16 per k-slice.  Blocks
//     in which no row of the tile accepted are skipped; the block of group i
//     itself waits for its decision, the others are applied meanwhile.
//   R~ = R_{i+1} with unit diagonal, staged into LDS by direct loads.
// Back substitution: 16 lanes per row, lane j owns positions j + 16 t and keeps
// y_l = u_l / R(l,l) - sum of R~(l, m) d_m over the positions m > l decided so
// far (R~ = R with rows scaled by 1/R(m,m), staged without its unit diagonal);
// at step l the owner's change d_l = clip(rint(y_l)) is broadcast within the
// row (DPP row broadcast) and every lane subtracts R~(m, l) d_l from its y_m,
// m < l.  A position's y is final once it is decided, so d_l is taken again
// from the final y after the last step (nothing is recorded per step), and
// u_l / R(l,l) - y_l + d_l = a_l above.  No branches and no LDS round trip on
// the dependency chain.  The accept test then reduces over the
// row's lanes with DPP.  Decisions stay in LDS: codes and dq of the panel are
// written once, with 16-byte stores, after its last group.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Load / store at base + byte offset.  With a wave-uniform base and a 32-bit
// offset the access takes the scalar-base form (SGPR pair + one offset VGPR):
// no 64-bit per-lane addresses to keep live.
template <typename T>
__device__ __forceinline__ T ld_at(const T* base, uint32_t byte_off) {
  return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + byte_off);
}
template <typename T>
__device__ __forceinline__ void st_at(T* base, uint32_t byte_off, T v) {
  *reinterpret_cast<T*>(reinterpret_cast<char*>(base) + byte_off) = v;
}

// One 16-byte direct global -> LDS load per lane (lane L writes lds + 16 L
// bytes; lds is the same for the whole wave).
__device__ __forceinline__ void dma16(const float* src, float* lds) {
  __builtin_amdgcn_global_load_lds((const void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

// Per lane and position l = j + 16 t of the row: y = u~_l - sum_m R~(l, m) d_m
// over the positions m > l already decided, and the bounds -q_l, 2^b - 1 - q_l
// of the code change taken at l.
template <int NT>
struct ChainState {
  float y[NT];
  float lo[NT];
  float hi[NT];
};

// Sum over each row of 16 lanes, in every lane of the row (xor 1 and 2 within
// quads, then the half-row and row mirrors); every lane adds the same two
// operands in each round, so all lanes hold the same bits.
__device__ __forceinline__ float row_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xf, 0xf, false));
  return v;
}
__device__ __forceinline__ int row_sum(int v) {
  v += __builtin_amdgcn_mov_dpp(v, 0xB1, 0xf, 0xf, false);
  v += __builtin_amdgcn_mov_dpp(v, 0x4E, 0xf, 0xf, false);
  v += __builtin_amdgcn_mov_dpp(v, 0x141, 0xf, 0xf, false);
  v += __builtin_amdgcn_mov_dpp(v, 0x140, 0xf, 0xf, false);
  return v;
}

// Compile-time loop: Unroll<K, N>::run(f) calls f(IntC<k>) for k = K .. N - 1.
template <int V>
struct IntC {
  static constexpr int value = V;
};
template <int K, int N>
struct Unroll {
  template <typename F>
  static __device__ __forceinline__ void run(F&& f) {
    if constexpr (K < N) {
      f(IntC<K>{});
      Unroll<K + 1, N>::run(f);
    }
  }
};

// Value of lane JL of each row of 16 lanes, in every lane of that row.
template <int JL>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + JL, 0xf, 0xf, false));
}

// R~ column l as seen by lane j: the NT values R~(j + 16 t, l), t < NT, in
// chunks of W = min(4, NT) (the layout of the staged columns:
// [l][chunk][lane][W], so the 16 lanes of a row read consecutive bytes).
// Only t <= l / 16 can be nonzero and only those are read, one float at a
// time (adjacent ones merge into one wide access; a wide access with unused
// parts would let the compiler reuse their registers while it is in flight).
template <int NT>
struct RCol {
  static constexpr int W = NT < 4 ? NT : 4;
  float v[NT];
};

template <int L, int NT>
__device__ __forceinline__ RCol<NT> load_rcol(const float* __restrict__ rc, int cj) {
  constexpr int W = RCol<NT>::W;
  RCol<NT> r;
  if constexpr (L >= 0) {
    constexpr int base = RcolLayout<16 * NT>::offset(L);
#pragma unroll
    for (int t = 0; t <= (L >> 4); ++t) r.v[t] = rc[base + ((t / W) * 16 + cj) * W + t % W];
  }
  return r;
}

// One step of the back substitution; the R~ columns of the next four steps are
// in flight (loaded ahead so that LDS latency stays off the chain).  The change
// at position L is the rounded y clipped to the code range (clip(round(q + y))
// - q, up to the rounding of exact ties).
template <int L, int NT>
struct ChainStep {
  static __device__ __forceinline__ void run(ChainState<NT>& s, const float* __restrict__ rc,
                                             int cj, const RCol<NT>& c0, const RCol<NT>& c1,
                                             const RCol<NT>& c2, const RCol<NT>& c3) {
    constexpr int TL = L >> 4;
    constexpr int JL = L & 15;
    const RCol<NT> c4 = load_rcol<L - 4, NT>(rc, cj);
    const float dv = __builtin_amdgcn_fmed3f(rintf(s.y[TL]), s.lo[TL], s.hi[TL]);
    const float db = row_bcast<JL>(dv);
#pragma unroll
    for (int t = 0; t <= TL; ++t) s.y[t] = fmaf(-c0.v[t], db, s.y[t]);
    // Keep the scheduler from hoisting far-away work (register pressure).
    if (JL == 0) __builtin_amdgcn_sched_barrier(0);
    ChainStep<L - 1, NT>::run(s, rc, cj, c1, c2, c3, c4);
  }
};

template <int NT>
struct ChainStep<-1, NT> {
  static __device__ __forceinline__ void run(ChainState<NT>&, const float* __restrict__, int,
                                             const RCol<NT>&, const RCol<NT>&, const RCol<NT>&,
                                             const RCol<NT>&) {}
};

template <int G_SIZE>
__global__ __launch_bounds__(512, 1) void babai_kernel(
    int rows, int cols, int bits, int i0, int i1, const float* __restrict__ P,
    const _Float16* __restrict__ Mh, const _Float16* __restrict__ Ml,
    const float* __restrict__ mrow_inv, const float* __restrict__ rcol,
    const float* __restrict__ rdinv,
    const float* __restrict__ rdsq, uint8_t* __restrict__ codes,
    const float* __restrict__ scales, const uint8_t* __restrict__ active,
    _Float16* __restrict__ dq, int32_t* __restrict__ plist, uint32_t* __restrict__ pcount,
    uint8_t* __restrict__ cand_out,
    uint8_t* __restrict__ dec_out, Counters* __restrict__ cnt,
    const int32_t* __restrict__ rowmap, const int* __restrict__ n_dev,
    int32_t* __restrict__ glist, uint32_t* __restrict__ gcount, int list_cap,
    _Float16* __restrict__ cz, const float* __restrict__ wh, double* __restrict__ rhs) {
  if (n_dev != nullptr) rows = *n_dev;
  if ((int)blockIdx.x * 16 >= rows) return;  // the whole work-group: no row here
  constexpr int g = G_SIZE;
  constexpr int RT = 16;                 // rows per work-group
  constexpr int NT = g / 16;             // positions per lane in the back substitution
  constexpr int NBLK = g / 16;           // 16-column blocks of a group
  constexpr int BPW = NBLK >= 4 ? NBLK / 4 : 1;  // column blocks per prep wave
  constexpr int KS = g / 32;             // fp16 k-slices of one group block
  constexpr int LDH = g + 4;
  constexpr int PG = panel_groups_of(g);
  constexpr int PW = PG * g;             // panel width
  // dqp_s row stride: 16 bytes past the panel width, so that the 16 rows a
  // fragment read serves start in 16 distinct 16-byte bank groups (a stride
  // of PW halves would put all 16 in one)
  constexpr int PWS = PW + 8;
  constexpr int RC_FLOATS = RcolLayout<g>::total;  // the staged part of a group's R~
  static_assert(RC_FLOATS % 1024 == 0, "R~ staged in 1 KB pieces, four per preparation lane set");
  constexpr int RC_PER_THREAD = RC_FLOATS / (256 * 4);  // f32x4 copies per prep thread to stage R~
  const int G = cols / g;
  const float qmax = (float)((1 << bits) - 1);

  // R~ columns [l][j][t] of two groups in two distinct arrays (written by
  // direct global -> LDS loads while the other one is read).
  __shared__ __attribute__((aligned(1024))) float rc0_s[RC_FLOATS];
  __shared__ __attribute__((aligned(1024))) float rc1_s[RC_FLOATS];
  __shared__ float u_s[RT * LDH];                    // u s of the current group
  __shared__ __attribute__((aligned(16))) _Float16 dqp_s[RT * PWS];  // accepted changes in the panel
  __shared__ int tacc_s[PG];                         // any row of the tile accepted group
  __shared__ int cnt_s[4];                           // accepted, changed, skipped, blocks
  __shared__ int racc_s[RT];                         // bit i - i0: the row accepted group i

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r0 = blockIdx.x * RT;
  const bool chain_wave = wave < 4;

  // back-substitution role (waves 0-3): 16 lanes per row
  const int crow = (wave & 3) * 4 + (lane >> 4);
  const int cj = lane & 15;
  // Tile rows are positions of the sweep (P, dq, the panel row list); the
  // layer row of position p (codes, scales, flags) is map_row(rowmap, p).
  const int grow = r0 + crow;
  const bool row_in = grow < rows;
  const int crid = map_row(rowmap, row_in ? grow : 0);
  const bool row_act = row_in && (active == nullptr || active[crid] != 0);
  // preparation role (waves 4-7): matrix-core lanes, A row / B column = lane & 15,
  // k slice = lane >> 4, output rows 4 (lane >> 4) + v
  const int pw = wave - 4;
  const int ptid = tid - 256;
  const int mr = lane & 15;
  const int kq = lane >> 4;
  const bool prep_live = !chain_wave && pw * BPW < NBLK;

  if (tid < PG) tacc_s[tid] = 0;
  if (tid < 4) cnt_s[tid] = 0;
  if (tid < RT) racc_s[tid] = 0;

  // Bases of this work-group's 16 positions (wave-uniform); offsets from them
  // fit in 32 bits (16 rows of at most 2^26 columns).
  const float* __restrict__ P_t = P + (size_t)r0 * cols;
  _Float16* __restrict__ dq_t = dq + (size_t)r0 * cols;
  // Local position of a lane, or position 0 past the edge (loads stay
  // unconditional; such values are never used).
  auto lrow = [&](int lr) { return (uint32_t)(r0 + lr < rows ? lr : 0); };
  const uint32_t ucols = (uint32_t)cols;

  // ---- preparation: u s = L^{-1} (H e) of the next group, this wave's columns ----
  // u of the group being prepared, and of the one after it (loaded a
  // position early: it does not depend on this panel's decisions)
  f32x4 ua0[BPW], ua1[BPW];
  // R~ of group i into dst: 1 KB pieces, piece j by prep wave j % 4 (lane L
  // copies bytes 16 L .. 16 L + 15 of the piece).  Complete once the issuing
  // wave has passed its next barrier.
  auto stage_rcol = [&](int i, float* dst) {
    const float* src = rcol + (size_t)i * g * g;
#pragma unroll
    for (int q = 0; q < RC_PER_THREAD; ++q) {
      const int j = pw + 4 * q;
      dma16((const float*)((const char*)src + (uint32_t)((j * 256 + lane * 4) * 4)), dst + j * 256);
    }
  };
  // u of group i as the residual product left it (U = E M^T, changes of
  // earlier panels already folded in), this wave's columns.
  auto u_from_p = [&](int i, f32x4 (&ut)[BPW]) {
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
      const int n = (pw * BPW + b) * 16 + mr;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        ut[b][v] = ld_at(P_t, (lrow(4 * kq + v) * ucols + (uint32_t)(i * g + n)) * 4u);
    }
  };
  // Fragments of M(i-block, h-block) = L_i^{-1} H_ih for this wave's columns,
  // and the factors s_h (per row) and 2^-t of M's rows (per column).
  struct TFrag {
    f16x8 bh[BPW][KS], bl[BPW][KS];
    float sh[4];
    float cs[BPW];
  };
  // scales of the layer rows of this lane's 4 output rows (preparation role)
  const float* sc_rows[4];
#pragma unroll
  for (int v = 0; v < 4; ++v)
    sc_rows[v] = scales + (size_t)map_row(rowmap, r0 + (int)lrow(4 * kq + v)) * G;
  auto load_t = [&](int i, int h, TFrag& f) {
    // rows i g .. i g + g - 1 of M (uniform bases), this lane's row n within
    const _Float16* mh_i = Mh + (size_t)i * g * cols;
    const _Float16* ml_i = Ml + (size_t)i * g * cols;
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
      const int n = (pw * BPW + b) * 16 + mr;
      const uint32_t trow = ((uint32_t)n * ucols + (uint32_t)(h * g + 8 * kq)) * 2u;
#pragma unroll
      for (int kc = 0; kc < KS; ++kc) {
        f.bh[b][kc] = ld_at((const f16x8*)mh_i, trow + kc * 64);
        f.bl[b][kc] = ld_at((const f16x8*)ml_i, trow + kc * 64);
      }
      f.cs[b] = ld_at(mrow_inv + i * g, (uint32_t)(n * 4));
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) f.sh[v] = sc_rows[v][h];
  };
  // uacc -= s_h dq_h M(i-block, h-block)^T (dq_h exact in fp16, M as two fp16
  // terms).  dq_h is zero in every row of the tile unless one of them accepted
  // group h: then the product can be skipped (may_skip) or computed anyway,
  // which keeps the fragment loads ahead of their use (a use under a branch
  // drags the loads into it).
  auto apply_t = [&](int h, const TFrag& f, bool may_skip, f32x4 (&uacc)[BPW]) {
    const bool any = tacc_s[h - i0] != 0;
    if (may_skip && !any) return;
    if (ptid == 0 && any) cnt_s[3] += 1;
    f16x8 a[KS];
#pragma unroll
    for (int kc = 0; kc < KS; ++kc)
      a[kc] = *(const f16x8*)(dqp_s + mr * PWS + (h - i0) * g + kc * 32 + 8 * kq);
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
      f32x4 seg = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < KS; ++kc) {
        seg = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[kc], f.bh[b][kc], seg, 0, 0, 0);
        seg = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[kc], f.bl[b][kc], seg, 0, 0, 0);
      }
      // 16x16 accumulator: element v of lane l is (row 4 * (l / 16) + v, column l % 16);
      // rows past the edge carry zero changes.
#pragma unroll
      for (int v = 0; v < 4; ++v) uacc[b][v] = fmaf(-seg[v], f.sh[v] * f.cs[b], uacc[b][v]);
    }
  };
  auto write_u = [&](const f32x4 (&uacc)[BPW]) {
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
      const int c = (pw * BPW + b) * 16 + mr;
#pragma unroll
      for (int v = 0; v < 4; ++v) u_s[(4 * kq + v) * LDH + c] = uacc[b][v];
    }
  };

  // Chain role: codes, scale and diagonal factors of the next group are
  // fetched during the current one (they do not change in between).
  // Loads are unconditional (rows past the edge read row 0) so that none of
  // them waits for its data here; row_in is applied where they are used.
  uint32_t nq[NT];
  float nrdinv[NT], nrdsq[NT], ns = 0.f;
  const uint8_t* __restrict__ codes_c = codes + (size_t)crid * cols;  // this lane's row
  const float* __restrict__ scales_c = scales + (size_t)crid * G;
  auto chain_prefetch = [&](int i) {
    const uint32_t cb = (uint32_t)(i * g + cj);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      nq[t] = ld_at(codes_c, cb + 16 * t);
      nrdinv[t] = ld_at(rdinv + i * g, (uint32_t)((cj + 16 * t) * 4));
      nrdsq[t] = ld_at(rdsq + i * g, (uint32_t)((cj + 16 * t) * 4));
    }
    ns = scales_c[i];
  };
  // ---- epilogue items: 16 columns of one row of the panel, item c = row
  // c / per_row, columns 16 (c % per_row) onwards.  The preparation threads
  // take them all (items ptid and ptid + 256; a panel is at most 512 columns
  // wide) and load the old codes, cz and scale-system right-hand sides during
  // the panel's last back substitution, which they do not take part in.
  const int per_row = (i1 - i0) * g / 16;
  const int n_items = RT * per_row;
  static_assert(RT * (PG * g / 16) <= 512, "two epilogue items per preparation thread");
  u32x4 e_qw[2];
  f16x8 e_c0[2], e_c1[2];
  double e_rhs[2];
  int e_lrow[2];  // layer rows of the two items (both row-map loads go out first)
  auto epi_load = [&]() {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int r = (ptid + 256 * u) / per_row;
      e_lrow[u] = map_row(rowmap, r0 + r < rows ? r0 + r : r0);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = ptid + 256 * u;
      const int r = c / per_row;
      const int k = (c - r * per_row) * 16;
      if (c < n_items && r0 + r < rows) {
        const size_t lrow_r = (size_t)e_lrow[u];
        const uint32_t oq = (uint32_t)(i0 * g + k);
        e_qw[u] = ld_at((const u32x4*)(codes + lrow_r * cols), oq);
        e_c0[u] = ld_at((const f16x8*)(cz + lrow_r * cols), 2 * oq);
        e_c1[u] = ld_at((const f16x8*)(cz + lrow_r * cols), 2 * oq + 16);
        if (k % g == 0) e_rhs[u] = rhs[lrow_r * G + (size_t)(i0 + k / g)];
      }
    }
  };

  // The two roles run separate loops with the same barriers (two per group),
  // so neither role's loop-carried registers are live in the other's code.
  // Barriers inside the loops are on LDS only: global loads stay in flight
  // across them.
  if (chain_wave) {
    chain_prefetch(i0);
    // The loads of group i0's codes, scale and diagonal factors go out before
    // the barrier and stay in flight behind the preparation role's staging
    // (the pointers handed to the empty statement keep the compiler from
    // sinking them below it).
    asm volatile("" ::"v"(codes_c), "v"(scales_c), "s"(rdinv), "s"(rdsq) : "memory");
    int acc_bits = 0;  // bit i - i0: this row accepted group i
    lds_barrier();  // u and R~ of group i0 staged
    for (int i = i0; i < i1; ++i) {
      // ---- back substitution of group i, 16 lanes per row ----
      const bool has_next = i + 1 < i1;
      const float* rc_i = (i & 1) ? rc1_s : rc0_s;
      const float s = row_in ? ns : 0.f;
      float rdsq_i[NT], qold[NT];
      ChainState<NT> cs;
      float ut[NT];
      const bool skip = !(fabsf(s) > kFp32Eps);
      const bool do_row = row_act && !skip;
      const float inv_s = do_row ? 1.f / s : 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int l = cj + 16 * t;
        ut[t] = u_s[crow * LDH + l] * inv_s * nrdinv[t];
        rdsq_i[t] = nrdsq[t];
        const float q = row_in ? (float)nq[t] : 0.f;
        qold[t] = q;
        cs.y[t] = ut[t];
        cs.lo[t] = -q;
        cs.hi[t] = qmax - q;
      }
      if (has_next) chain_prefetch(i + 1);
      ChainStep<g - 1, NT>::run(cs, rc_i, cj, load_rcol<g - 1, NT>(rc_i, cj),
                                load_rcol<g - 2, NT>(rc_i, cj), load_rcol<g - 3, NT>(rc_i, cj),
                                load_rcol<g - 4, NT>(rc_i, cj));
      // d_l again from the final y_l (unchanged since its step), a_l =
      // sum_{m >= l} R~(l, m) d_m = u~_l - y_l + d_l (unit diagonal of R~);
      // the change of F divided by s_i^2 is sum_l R(l, l)^2 a_l (a_l - 2 u~_l).
      float dF = 0.f;
      int changed = 0;
      float dd[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        dd[t] = __builtin_amdgcn_fmed3f(rintf(cs.y[t]), cs.lo[t], cs.hi[t]);
        const float a = (ut[t] - cs.y[t]) + dd[t];
        dF = fmaf(rdsq_i[t] * a, a - 2.f * ut[t], dF);
        changed += dd[t] != 0.f;
      }
      dF = row_sum(dF);
      changed = row_sum(changed);
      // A proposal equal to the current codes changes F by exactly 0, which the
      // strict test rejects; NaN changes (non-finite u) give a NaN dF.
      const bool accept = do_row && changed > 0 && isfinite(dF) && (dF < 0.f);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int l = cj + 16 * t;
        dqp_s[crow * PWS + (i - i0) * g + l] = accept ? (_Float16)dd[t] : (_Float16)0.f;
      }
      if (cand_out != nullptr && row_in) {
        const size_t cbase = (size_t)crid * cols + (size_t)i * g;
#pragma unroll
        for (int t = 0; t < NT; ++t)
          cand_out[cbase + cj + 16 * t] =
              (uint8_t)(do_row ? fminf(fmaxf(qold[t] + dd[t], 0.f), qmax) : qold[t]);
      }
      acc_bits |= accept ? 1 << (i - i0) : 0;
      if (row_in && cj == 0) {
        if (dec_out != nullptr) {
          uint8_t dd = !row_act ? kDecStopped : (skip ? kDecSkip : (accept ? kDecAccept : kDecReject));
          dec_out[(size_t)crid * G + i] = dd;
        }
        if (accept) {
          tacc_s[i - i0] = 1;
          atomicAdd(&cnt_s[0], 1);
          atomicAdd(&cnt_s[1], changed);
        }
        if (row_act && skip) atomicAdd(&cnt_s[2], 1);
      }
      lds_barrier();  // group i decided: its changes are in dqp_s, tacc_s
      lds_barrier();  // u and R~ of group i + 1 ready
    }
    if (row_in && cj == 0) racc_s[crow] = acc_bits;
  } else {
    // Group i0 + p stages group i0 + p + 1 and applies the changes of groups
    // i0 .. i0 + p to it.  Each position p has its own body, so the
    // fragment buffers alternate without copies (a copy would wait for the
    // loads in flight) and the R~ buffer is known at compile time (i0 is
    // even: group i0 + p + 1 goes to rc1_s for even p).
    static_assert(PG % 2 == 0, "panels hold an even number of groups");
    stage_rcol(i0, rc0_s);
    if (prep_live) {
      u_from_p(i0, ua1);
      write_u(ua1);
    }
    // R~ of group i0 (direct loads) has landed once this wave's vector memory
    // counter is zero; u of group i0 + 1 then stays in flight across the
    // barrier.
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    if (prep_live && i0 + 1 < i1) u_from_p(i0 + 1, ua0);
    lds_barrier();  // u and R~ of group i0 staged
    auto prep_at = [&](auto pc) {
      constexpr int p = decltype(pc)::value;
      const int i = i0 + p;
      TFrag fa, fb;
      // u of group i + 1 is in ua[p % 2] (loaded one position earlier); the
      // load of group i + 2's goes out now
      f32x4 (&uc)[BPW] = (p % 2 == 0) ? ua0 : ua1;
      f32x4 (&un)[BPW] = (p % 2 == 0) ? ua1 : ua0;
      if (prep_live) {
        if (i + 2 < i1) u_from_p(i + 2, un);
        // block h = i0 + k sits in fa for even k, fb for odd k; the next
        // block loads while the current one is applied, and the last one,
        // M(i + 1, i), stays in flight across the barrier.  A block of an
        // earlier group that no row of the tile accepted (decided before this
        // position) is neither loaded nor applied.
        auto wanted = [&](int k) { return k == p || tacc_s[k] != 0; };
        if (wanted(0)) load_t(i + 1, i0, fa);
        Unroll<0, p>::run([&](auto kc) {
          constexpr int k = decltype(kc)::value;
          if constexpr (k % 2 == 0) {
            if (wanted(k + 1)) load_t(i + 1, i0 + k + 1, fb);
            apply_t(i0 + k, fa, true, uc);
          } else {
            if (wanted(k + 1)) load_t(i + 1, i0 + k + 1, fa);
            apply_t(i0 + k, fb, true, uc);
          }
        });
      }
      // R~ (i + 1) last: LDS reads issued after a direct load to LDS wait for
      // it (the compiler cannot tell the buffers apart), and it has the rest
      // of the back substitution of group i to land.
      if constexpr (p % 2 == 0)
        stage_rcol(i + 1, rc1_s);
      else
        stage_rcol(i + 1, rc0_s);
      lds_barrier();  // group i decided: its changes are in dqp_s, tacc_s
      if (prep_live) {
        if constexpr (p % 2 == 0)
          apply_t(i, fa, true, uc);
        else
          apply_t(i, fb, true, uc);
        write_u(uc);
      }
      // The direct loads of R~ (i + 1) are complete once this wave's vector
      // memory counter is zero.
      __builtin_amdgcn_s_waitcnt(kVmcnt0);
      lds_barrier();  // u and R~ of group i + 1 ready
    };
    // straight-line over the positions (no loop to hoist addresses out of)
    Unroll<0, PG - 1>::run([&](auto pc) {
      if (i0 + decltype(pc)::value + 1 < i1) prep_at(pc);
    });
    // last group of the panel: nothing to prepare; the epilogue's loads go out
    epi_load();
    // Taken into registers here, where these waves only wait for the back
    // substitution (the compiler would otherwise wait for them in the
    // epilogue, behind its stores).
#pragma unroll
    for (int u = 0; u < 2; ++u)
      asm volatile("" : "+v"(e_qw[u]), "+v"(e_c0[u]), "+v"(e_c1[u]), "+v"(e_rhs[u]), "+v"(e_lrow[u]));
    if (i1 > i0) {
      lds_barrier();
      lds_barrier();
    }
  }

  __syncthreads();  // racc_s
  // ---- rows that accepted a change: appended to the panel's row list (the
  // panel update folds in only these rows; their order there is immaterial),
  // this work-group's sub-list
  const int sub = (int)blockIdx.x % kSubLists;
  if (wave == 0) {
    const bool f = lane < RT && racc_s[lane] != 0;
    const unsigned long long m = __ballot(f);
    uint32_t base = 0;
    if (lane == 0 && m != 0) base = atomicAdd(&pcount[sub * kCtrStride], (uint32_t)__popcll(m));
    base = __shfl(base, 0);
    if (f)
      plist[(size_t)sub * list_cap + base + (uint32_t)__popcll(m & ((1ull << lane) - 1))] = r0 + lane;
  } else if (wave == 1 && glist != nullptr) {
    // ---- and, per group of the panel, to that group's list of changed rows
    // (the next sweep forms the Gram entries of only those): lane p reserves
    // room for group i0 + p, every lane r then writes row r's entries
    const int ng = i1 - i0;
    int mask = 0;  // rows of the tile that accepted group i0 + lane
    if (lane < ng) {
#pragma unroll
      for (int r = 0; r < RT; ++r) mask |= ((racc_s[r] >> lane) & 1) << r;
    }
    uint32_t base = 0;
    if (lane < ng && mask != 0)
      base = atomicAdd(&gcount[((size_t)(i0 + lane) * kSubLists + sub) * kCtrStride],
                       (uint32_t)__popc(mask));
    if (lane < RT && r0 + lane < rows) {
      const int bits = racc_s[lane];
      const int lrow_r = map_row(rowmap, r0 + lane);
      for (int p = 0; p < ng; ++p) {
        const int mp = __shfl(mask, p);
        const uint32_t bp = __shfl(base, p);
        if ((bits >> p) & 1)
          glist[((size_t)(i0 + p) * kSubLists + sub) * list_cap + bp +
                (uint32_t)__popc(mp & ((1 << lane) - 1))] = lrow_r;
      }
    } else {
      for (int p = 0; p < ng; ++p) {  // the shuffles need every lane
        (void)__shfl(mask, p);
        (void)__shfl(base, p);
      }
    }
  }

  // ---- codes += accepted changes, cz (q - z as fp16) likewise, and dq =
  // accepted changes, over the panel's columns: 16 columns per item (16-byte
  // code, 2 x 16-byte cz and dq accesses), by the preparation threads.  The
  // scale systems' right-hand sides follow the codes: r_i += d_i^T (W H)_i,
  // summed in fp64 over the g / 16 consecutive threads of a group.  dqp_s is
  // complete since the last barrier.
  if (!chain_wave) {
    // the changes of both items and, where a code changes, their (W H) first:
    // no load waits behind a store
    f16x8 d0[2], d1[2];
    bool any[2];
    f32x4 w4[2][4];  // (W H) of the 16 columns, only where a code changes
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = ptid + 256 * u;
      const int r = c / per_row;
      const int k = (c - r * per_row) * 16;
      const bool live = c < n_items && r0 + r < rows;
      const int rr = live ? r : 0;
      const int kk = live ? k : 0;
      d0[u] = *(const f16x8*)(dqp_s + rr * PWS + kk);
      d1[u] = *(const f16x8*)(dqp_s + rr * PWS + kk + 8);
      any[u] = false;
#pragma unroll
      for (int b = 0; b < 8; ++b)
        any[u] |= (d0[u][b] != (_Float16)0.f) | (d1[u][b] != (_Float16)0.f);
      any[u] = any[u] && live;
      if (any[u]) {
        const float* whp = wh + (size_t)e_lrow[u] * cols + (uint32_t)(i0 * g + k);
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4) w4[u][b4] = *(const f32x4*)(whp + 4 * b4);
      }
    }
    // then the right-hand side increments d^T (W H) (summed over the g / 16
    // threads of a group), then every store
    double part[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      part[u] = 0.0;
      if (any[u]) {
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int b = 4 * b4 + e;
            part[u] = fma((double)(b < 8 ? d0[u][b] : d1[u][b - 8]), (double)w4[u][b4][e], part[u]);
          }
      }
      if (__ballot(any[u]) != 0) {  // waves without a change skip the reduction
#pragma unroll
        for (int off = 1; off < g / 16; off <<= 1) part[u] += __shfl_xor(part[u], off);
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = ptid + 256 * u;
      const int r = c / per_row;
      const int k = (c - r * per_row) * 16;
      if (c < n_items && r0 + r < rows) {
        const uint32_t o = (uint32_t)r * ucols + (uint32_t)(i0 * g + k);
        const size_t lrow_r = (size_t)e_lrow[u];
        uint8_t* codes_r = codes + lrow_r * cols;
        _Float16* cz_r = cz + lrow_r * cols;
        const uint32_t oq = (uint32_t)(i0 * g + k);
        uint32_t w[4] = {e_qw[u][0], e_qw[u][1], e_qw[u][2], e_qw[u][3]};
        // Byte b of word b / 4 gains d_b; new codes stay in [0, 2^bits - 1],
        // so the word-wide add never carries into a neighbouring byte.
#pragma unroll
        for (int b = 0; b < 16; ++b) {
          const int dv = (int)(b < 8 ? d0[u][b] : d1[u][b - 8]);
          w[b >> 2] += (uint32_t)dv << (8 * (b & 3));
        }
        st_at((uint4*)codes_r, oq, make_uint4(w[0], w[1], w[2], w[3]));
        st_at((f16x8*)cz_r, 2 * oq, e_c0[u] + d0[u]);  // small integers: exact
        st_at((f16x8*)cz_r, 2 * oq + 16, e_c1[u] + d1[u]);
        st_at((f16x8*)dq_t, 2 * o, d0[u]);
        st_at((f16x8*)dq_t, 2 * o + 16, d1[u]);
        if (k % g == 0 && part[u] != 0.0) rhs[lrow_r * G + (size_t)(i0 + k / g)] = e_rhs[u] + part[u];
      }
    }
  }
  if (tid == 0) {
    Counters* c = cnt + sub;
    if (cnt_s[0]) atomicAdd(&c->accepted, (unsigned long long)cnt_s[0]);
    if (cnt_s[1]) atomicAdd(&c->changed, (unsigned long long)cnt_s[1]);
    if (cnt_s[2]) atomicAdd(&c->skipped, (unsigned long long)cnt_s[2]);
    if (cnt_s[3]) atomicAdd(&c->corr_blocks, (unsigned long long)cnt_s[3]);
  }
}

template <int G_SIZE>
static hipError_t launch_babai_t(hipStream_t st, int rows, int cols, int bits, int i0, int i1,
                                 const float* P, const char* ws, const Layout& lay,
                                 uint8_t* codes, const float* scales, const uint8_t* active,
                                 uint8_t* cand, uint8_t* decision, Counters* cnt,
                                 const int32_t* rowmap, const int* n_dev, int32_t* glist,
                                 uint32_t* gcount, int list_cap) {
  constexpr int g = G_SIZE;
  constexpr int PG = panel_groups_of(g);
  if (i1 - i0 > PG || i0 % PG != 0) return hipErrorInvalidValue;
  if (i1 <= i0) return hipSuccess;
  // 32-bit offsets: 16 rows of fp32 and g rows of fp16 M from a uniform base
  if ((size_t)cols * 64 >= (size_t(1) << 32) || (size_t)cols * g * 2 >= (size_t(1) << 32))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(babai_kernel<g>, dim3((rows + 15) / 16), dim3(512), 0, st, rows, cols, bits,
                     i0, i1, P, (const _Float16*)(ws + lay.mhi), (const _Float16*)(ws + lay.mlo),
                     (const float*)(ws + lay.mrow), (const float*)(ws + lay.rcol),
                     (const float*)(ws + lay.rdinv),
                     (const float*)(ws + lay.rdsq), codes, scales, active,
                     (_Float16*)(ws + lay.dq), (int32_t*)(ws + lay.plist),
                     (uint32_t*)(ws + lay.pcount) + (size_t)(i0 / PG) * kSubLists * kCtrStride,
                     cand, decision, cnt, rowmap, n_dev, glist, gcount, list_cap,
                     (_Float16*)(ws + lay.cz), (const float*)(ws + lay.wh), (double*)(ws + lay.rhs));
  return hipGetLastError();
}

hipError_t launch_babai(hipStream_t st, int rows, int cols, int g, int bits, int i0, int i1,
                        const float* P,
                        const char* ws, const Layout& lay, uint8_t* codes, const float* scales,
                        const int32_t* zeros, const uint8_t* active, uint8_t* cand,
                        uint8_t* decision, Counters* cnt, const int32_t* rowmap, const int* n_dev,
                        int32_t* glist, uint32_t* gcount, int list_cap) {
  (void)zeros;
  switch (g) {
    case 32:
      return launch_babai_t<32>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, active,
                                cand, decision, cnt, rowmap, n_dev, glist, gcount, list_cap);
    case 64:
      return launch_babai_t<64>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, active,
                                cand, decision, cnt, rowmap, n_dev, glist, gcount, list_cap);
    case 128:
      return launch_babai_t<128>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, active,
                                 cand, decision, cnt, rowmap, n_dev, glist, gcount, list_cap);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace jarq
