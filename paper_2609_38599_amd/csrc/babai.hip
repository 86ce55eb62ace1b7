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
// One 256-thread work-group owns 16 rows and visits the groups of one panel
// [i0, i1) in order; P already holds the changes of earlier panels (folded in
// by pupdate.hip).  Per group:
//   1. correction: he = P_i - sum_{i0<=h<i} s_h (dq_h H_hi), dq_h the accepted
//      code changes of earlier groups of the panel (exact in fp16, zero elsewhere).  H is read as its two fp16 planes, so each block
//      is two v_mfma_f32_16x16x32_f16 products per k-slice, scaled by s_h per
//      row.  Blocks in which no row of the tile accepted are skipped.
//   2. u = he L_i^{-T} / s_i (L_i^{-1} = R_i^{-T}) on fp32 matrix cores.
//   3. back substitution: 16 lanes per row, lane j owns positions j + 16 t and
//      keeps base_l = q_l + u_l / R(l,l) and acc_l = sum_{m>l} R(l,m) d_m / R(l,l)
//      (after the last step acc_l = a_l above);
//      at step l every lane evaluates its candidate, the owner's change d_l is
//      broadcast within the row (DPP row broadcast) and each lane folds
//      R(m, l) / R(m, m) d_l into its own acc_m.  No branches, no LDS round trip
//      on the dependency chain.
//   4. accept test per row, in-place code update, dq_i, trace and counters.
#include "jarq_internal.h"

namespace jarq {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// One 16-byte direct global -> LDS load per lane (lane L writes lds + 16 L
// bytes; lds is the same for the whole wave).
__device__ __forceinline__ void dma16(const float* src, float* lds) {
  __builtin_amdgcn_global_load_lds((const void*)src,
                                   (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

template <int NT>
struct ChainState {
  float base[NT];
  float acc[NT];
  float qold[NT];
  float qc[NT];
};

template <int JL>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + JL, 0xf, 0xf, false));
}

// R~ column l as seen by lane j: the NT values R~(j + 16 t, l), t < NT.  Only
// t <= l / 16 can be nonzero.
template <int NT>
struct RCol {
  f32x4 v[(NT + 3) / 4];
};

template <int L, int NT>
__device__ __forceinline__ RCol<NT> load_rcol(const float* __restrict__ rc, int cj) {
  RCol<NT> r;
  if (L >= 0) {
    const float* p = rc + (L * 16 + cj) * NT;
#pragma unroll
    for (int c = 0; c * 4 <= (L >> 4); ++c) r.v[c] = *(const f32x4*)(p + 4 * c);
  }
  return r;
}

// One step of the back substitution; the R~ columns of the next two steps are
// already in flight (loaded two steps ahead so LDS latency stays off the chain).
template <int L, int NT>
struct ChainStep {
  static __device__ __forceinline__ void run(ChainState<NT>& s, const float* __restrict__ rc,
                                             int cj, float qmax, const RCol<NT>& cur,
                                             const RCol<NT>& nxt) {
    constexpr int TL = L >> 4;
    constexpr int JL = L & 15;
    const RCol<NT> nn = load_rcol<L - 2, NT>(rc, cj);
    const float xv = s.base[TL] - s.acc[TL];
    const float qv = fminf(fmaxf(rintf(xv), 0.f), qmax);
    s.qc[TL] = cj == JL ? qv : s.qc[TL];
    const float db = row_bcast<JL>(qv - s.qold[TL]);
#pragma unroll
    for (int c = 0; c * 4 <= TL; ++c)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (4 * c + q <= TL) s.acc[4 * c + q] = fmaf(cur.v[c][q], db, s.acc[4 * c + q]);
    // Keep the scheduler from hoisting far-away work (register pressure).
    if (JL == 0) __builtin_amdgcn_sched_barrier(0);
    ChainStep<L - 1, NT>::run(s, rc, cj, qmax, nxt, nn);
  }
};

template <int NT>
struct ChainStep<-1, NT> {
  static __device__ __forceinline__ void run(ChainState<NT>&, const float* __restrict__, int,
                                             float, const RCol<NT>&, const RCol<NT>&) {}
};

template <int G_SIZE>
__global__ __launch_bounds__(512, 1) void babai_kernel(
    int rows, int cols, int bits, int i0, int i1, const float* __restrict__ P,
    const _Float16* __restrict__ Mh, const _Float16* __restrict__ Ml,
    const float* __restrict__ mrow_inv, const float* __restrict__ rcol,
    const float* __restrict__ rdinv,
    const float* __restrict__ rdsq, uint8_t* __restrict__ codes,
    const float* __restrict__ scales, const uint8_t* __restrict__ active,
    _Float16* __restrict__ dq, uint8_t* __restrict__ rowflag, uint8_t* __restrict__ cand_out,
    uint8_t* __restrict__ dec_out, Counters* __restrict__ cnt) {
  constexpr int g = G_SIZE;
  constexpr int RT = 16;                 // rows per work-group
  constexpr int NT = g / 16;             // positions per lane in the back substitution
  constexpr int NBLK = g / 16;           // 16-column blocks of a group
  constexpr int BPW = NBLK >= 4 ? NBLK / 4 : 1;  // column blocks per prep wave
  constexpr int KS = g / 32;             // fp16 k-slices of one group block
  constexpr int LDH = g + 4;
  constexpr int PG = panel_groups_of(g);
  constexpr int PW = PG * g;             // panel width
  constexpr int RC_PER_THREAD = g * g / (256 * 4);  // f32x4 copies per prep thread to stage R~
  const int G = cols / g;
  const float qmax = (float)((1 << bits) - 1);

  // R~ columns [l][j][t] of two groups in two distinct arrays (written by
  // direct global -> LDS loads while the other one is read).
  __shared__ __attribute__((aligned(1024))) float rc0_s[g * g];
  __shared__ __attribute__((aligned(1024))) float rc1_s[g * g];
  __shared__ float u_s[RT * LDH];                    // u s of the current group
  __shared__ __attribute__((aligned(16))) _Float16 dqp_s[RT * PW];  // accepted changes in the panel
  __shared__ int tacc_s[PG];                         // any row of the tile accepted group
  __shared__ int cnt_s[4];                           // accepted, changed, skipped, blocks

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r0 = blockIdx.x * RT;
  const bool chain_wave = wave < 4;

  // back-substitution role (waves 0-3): 16 lanes per row
  const int crow = (wave & 3) * 4 + (lane >> 4);
  const int cj = lane & 15;
  const int grow = r0 + crow;
  const bool row_in = grow < rows;
  const bool row_act = row_in && (active == nullptr || active[grow] != 0);
  // preparation role (waves 4-7): matrix-core lanes, A row / B column = lane & 15,
  // k slice = lane >> 4, output rows 4 (lane >> 4) + v
  const int pw = wave - 4;
  const int ptid = tid - 256;
  const int mr = lane & 15;
  const int kq = lane >> 4;
  const bool prep_live = !chain_wave && pw * BPW < NBLK;

  if (tid < PG) tacc_s[tid] = 0;
  if (tid < 4) cnt_s[tid] = 0;

  // ---- preparation: u s = L^{-1} (H e) of the next group, this wave's columns ----
  f32x4 uacc[BPW];
  // R~ of group i into dst: 1 KB pieces, piece j by prep wave j % 4 (lane L
  // copies bytes 16 L .. 16 L + 15 of the piece).  Complete once the issuing
  // wave has passed its next barrier.
  auto stage_rcol = [&](int i, float* dst) {
    const float* src = rcol + (size_t)i * g * g;
#pragma unroll
    for (int q = 0; q < RC_PER_THREAD; ++q) {
      const int j = pw + 4 * q;
      dma16(src + j * 256 + lane * 4, dst + j * 256);
    }
  };
  // u of group i as the residual product left it (U = E M^T, changes of
  // earlier panels already folded in), this wave's columns.
  auto u_from_p = [&](int i) {
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
      const int n = (pw * BPW + b) * 16 + mr;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int gr = r0 + 4 * kq + v;
        // rows past the edge read row 0 (unconditional load); never used
        uacc[b][v] = P[(size_t)(gr < rows ? gr : 0) * cols + (size_t)i * g + n];
      }
    }
  };
  // Fragments of M(i-block, h-block) = L_i^{-1} H_ih for this wave's columns,
  // and the factors s_h (per row) and 2^-t of M's rows (per column).
  struct TFrag {
    f16x8 bh[BPW][KS], bl[BPW][KS];
    float sh[4];
    float cs[BPW];
  };
  auto load_t = [&](int i, int h, TFrag& f) {
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
      const int n = i * g + (pw * BPW + b) * 16 + mr;
      const size_t trow = (size_t)n * cols + (size_t)h * g + 8 * kq;
#pragma unroll
      for (int kc = 0; kc < KS; ++kc) {
        f.bh[b][kc] = *(const f16x8*)(Mh + trow + kc * 32);
        f.bl[b][kc] = *(const f16x8*)(Ml + trow + kc * 32);
      }
      f.cs[b] = mrow_inv[n];
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int gr = r0 + 4 * kq + v;
      f.sh[v] = scales[(size_t)(gr < rows ? gr : 0) * G + h];
    }
  };
  // uacc -= s_h dq_h M(i-block, h-block)^T (dq_h exact in fp16, M as two fp16 terms).
  auto apply_t = [&](int h, const TFrag& f) {
    if (tacc_s[h - i0] == 0) return;
    if (ptid == 0) cnt_s[3] += 1;
    f16x8 a[KS];
#pragma unroll
    for (int kc = 0; kc < KS; ++kc)
      a[kc] = *(const f16x8*)(dqp_s + mr * PW + (h - i0) * g + kc * 32 + 8 * kq);
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
  auto write_u = [&]() {
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
  const int srow = row_in ? grow : 0;
  auto chain_prefetch = [&](int i) {
    const size_t cb = (size_t)srow * cols + (size_t)i * g;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int l = cj + 16 * t;
      nq[t] = codes[cb + l];
      nrdinv[t] = rdinv[(size_t)i * g + l];
      nrdsq[t] = rdsq[(size_t)i * g + l];
    }
    ns = scales[(size_t)srow * G + i];
  };
  if (chain_wave) chain_prefetch(i0);
  bool any_acc = false;  // chain role: this row accepted a change in the panel

  if (!chain_wave) {
    stage_rcol(i0, (i0 & 1) ? rc1_s : rc0_s);
    if (prep_live) {
      u_from_p(i0);
      write_u();
    }
  }
  __syncthreads();

  for (int i = i0; i < i1; ++i) {
    const bool has_next = i + 1 < i1;
    TFrag tnext;
    if (chain_wave) {
      // ---- back substitution of group i, 16 lanes per row ----
      const float* rc_i = (i & 1) ? rc1_s : rc0_s;
      const float s = row_in ? ns : 0.f;
      float rdsq_i[NT];
      ChainState<NT> cs;
      float ut[NT];
      const bool skip = !(fabsf(s) > kFp32Eps);
      const bool do_row = row_act && !skip;
      const float inv_s = do_row ? 1.f / s : 0.f;
      const size_t cbase = (size_t)grow * cols + (size_t)i * g;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int l = cj + 16 * t;
        ut[t] = u_s[crow * LDH + l] * inv_s * nrdinv[t];
        rdsq_i[t] = nrdsq[t];
        const float q = row_in ? (float)nq[t] : 0.f;
        cs.qold[t] = q;
        cs.qc[t] = q;
        cs.base[t] = q + ut[t];
        cs.acc[t] = 0.f;
      }
      if (has_next) chain_prefetch(i + 1);
      ChainStep<g - 1, NT>::run(cs, rc_i, cj, qmax, load_rcol<g - 1, NT>(rc_i, cj),
                                load_rcol<g - 2, NT>(rc_i, cj));
      float dF = 0.f;  // change of F divided by s_i^2
      int changed = 0;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const float a = cs.acc[t];
        dF = fmaf(rdsq_i[t] * a, a - 2.f * ut[t], dF);
        changed += cs.qc[t] != cs.qold[t];
      }
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) {
        dF += __shfl_xor(dF, off);
        changed += __shfl_xor(changed, off);
      }
      // A proposal equal to the current codes changes F by exactly 0, which the
      // strict test rejects.
      const bool accept = do_row && changed > 0 && isfinite(dF) && (dF < 0.f);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int l = cj + 16 * t;
        const _Float16 d = accept ? (_Float16)(cs.qc[t] - cs.qold[t]) : (_Float16)0.f;
        dqp_s[crow * PW + (i - i0) * g + l] = d;
        if (row_in) {
          if (accept) codes[cbase + l] = (uint8_t)cs.qc[t];
          dq[cbase + l] = d;
          if (cand_out != nullptr) cand_out[cbase + l] = (uint8_t)(do_row ? cs.qc[t] : cs.qold[t]);
        }
      }
      any_acc |= accept;
      if (row_in && cj == 0) {
        if (dec_out != nullptr) {
          uint8_t dd = !row_act ? kDecStopped : (skip ? kDecSkip : (accept ? kDecAccept : kDecReject));
          dec_out[(size_t)grow * G + i] = dd;
        }
        if (accept) {
          tacc_s[i - i0] = 1;
          atomicAdd(&cnt_s[0], 1);
          atomicAdd(&cnt_s[1], changed);
        }
        if (row_act && skip) atomicAdd(&cnt_s[2], 1);
      }
    } else if (has_next) {
      // ---- meanwhile: everything of group i + 1 that does not wait for group i ----
      stage_rcol(i + 1, ((i + 1) & 1) ? rc1_s : rc0_s);
      if (prep_live) {
        u_from_p(i + 1);
        // Fragments of the next block load while the current one is applied;
        // the last load, T(i + 1, i), stays in flight across the barrier.
        load_t(i + 1, i0, tnext);
        for (int h = i0; h < i; ++h) {
          const TFrag f = tnext;
          load_t(i + 1, h + 1, tnext);
          apply_t(h, f);
        }
      }
    }
    __syncthreads();  // group i decided: its changes are in dqp_s, tacc_s
    if (has_next && prep_live) {
      apply_t(i, tnext);
      write_u();
    }
    __syncthreads();  // u and R~ of group i + 1 ready
  }
  if (chain_wave && row_in && cj == 0) rowflag[grow] = any_acc ? 1 : 0;
  if (tid == 0) {
    if (cnt_s[0]) atomicAdd(&cnt->accepted, (unsigned long long)cnt_s[0]);
    if (cnt_s[1]) atomicAdd(&cnt->changed, (unsigned long long)cnt_s[1]);
    if (cnt_s[2]) atomicAdd(&cnt->skipped, (unsigned long long)cnt_s[2]);
    if (cnt_s[3]) atomicAdd(&cnt->corr_blocks, (unsigned long long)cnt_s[3]);
  }
}

template <int G_SIZE>
static hipError_t launch_babai_t(hipStream_t st, int rows, int cols, int bits, int i0, int i1,
                                 const float* P, const char* ws, const Layout& lay,
                                 uint8_t* codes, const float* scales, const uint8_t* active,
                                 uint8_t* cand, uint8_t* decision, Counters* cnt) {
  constexpr int g = G_SIZE;
  constexpr int PG = panel_groups_of(g);
  if (i1 - i0 > PG || i0 % PG != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(babai_kernel<g>, dim3((rows + 15) / 16), dim3(512), 0, st, rows, cols, bits,
                     i0, i1, P, (const _Float16*)(ws + lay.mhi), (const _Float16*)(ws + lay.mlo),
                     (const float*)(ws + lay.mrow), (const float*)(ws + lay.rcol),
                     (const float*)(ws + lay.rdinv),
                     (const float*)(ws + lay.rdsq), codes, scales, active,
                     (_Float16*)(ws + lay.dq), (uint8_t*)(ws + lay.rowflag), cand, decision, cnt);
  return hipGetLastError();
}

hipError_t launch_babai(hipStream_t st, int rows, int cols, int g, int bits, int i0, int i1,
                        const float* P,
                        const char* ws, const Layout& lay, uint8_t* codes, const float* scales,
                        const int32_t* zeros, const uint8_t* active, uint8_t* cand,
                        uint8_t* decision, Counters* cnt) {
  (void)zeros;
  switch (g) {
    case 32:
      return launch_babai_t<32>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, active,
                                cand, decision, cnt);
    case 64:
      return launch_babai_t<64>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, active,
                                cand, decision, cnt);
    case 128:
      return launch_babai_t<128>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, active,
                                 cand, decision, cnt);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace jarq
