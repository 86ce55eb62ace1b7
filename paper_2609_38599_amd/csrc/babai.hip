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
__global__ __launch_bounds__(256, 1) void babai_kernel(
    int rows, int cols, int bits, int i0, int i1, const float* __restrict__ P,
    const _Float16* __restrict__ Hh,
    const _Float16* __restrict__ Hl, const float* __restrict__ h_inv,
    const float* __restrict__ rinv, const float* __restrict__ rcol,
    const float* __restrict__ rdinv, const float* __restrict__ rdsq, uint8_t* __restrict__ codes,
    const float* __restrict__ scales, const int32_t* __restrict__ zeros,
    const uint8_t* __restrict__ active, _Float16* __restrict__ dq,
    uint8_t* __restrict__ cand_out, uint8_t* __restrict__ dec_out, Counters* __restrict__ cnt) {
  constexpr int g = G_SIZE;
  constexpr int RT = 16;                 // rows per work-group
  constexpr int NT = g / 16;             // positions per lane in the back substitution
  constexpr int NBLK = g / 16;           // 16-column blocks of a group
  constexpr int BPW = NBLK >= 4 ? NBLK / 4 : 1;  // column blocks per wave
  constexpr int KS = g / 32;             // fp16 k-slices of one group block
  constexpr int LDH = g + 4;
  constexpr int RC_PER_THREAD = g * g / (256 * 4);  // f32x4 loads to stage R~ columns
  const int G = cols / g;
  const float qmax = (float)((1 << bits) - 1);

  extern __shared__ float smem[];
  float* rc_s = smem;                    // g * g   R~ columns, [l][j][t]
  float* he_s = rc_s + g * g;            // RT x LDH
  float* u_s = he_s + RT * LDH;          // RT x LDH
  int* tacc_s = (int*)(u_s + RT * LDH);  // G       any row of the tile accepted group h
  int* cnt_s = tacc_s + G;               // 4       accepted, changed, skipped, correction blocks

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r0 = blockIdx.x * RT;

  // back-substitution role
  const int crow = wave * 4 + (lane >> 4);
  const int cj = lane & 15;
  const int grow = r0 + crow;
  const bool row_in = grow < rows;
  const bool row_act = row_in && (active == nullptr || active[grow] != 0);
  // matrix-core role: A row / B column = lane & 15, k slice = lane >> 4
  const int mr = lane & 15;
  const int kq = lane >> 4;
  const int arow = r0 + mr;
  const bool arow_in = arow < rows;
  const bool wave_live = wave * BPW < NBLK;
  const float hinv = *h_inv;

  for (int h = tid; h < G; h += 256) tacc_s[h] = 0;
  if (tid < 4) cnt_s[tid] = 0;

  for (int i = i0; i < i1; ++i) {
    __syncthreads();  // previous group's dq stores and LDS reuse
    {
      const float* src = rcol + (size_t)i * g * g;
#pragma unroll
      for (int q = 0; q < RC_PER_THREAD; ++q)
        *(f32x4*)(rc_s + (tid + 256 * q) * 4) = *(const f32x4*)(src + (tid + 256 * q) * 4);
    }
    // Loads that do not depend on the correction, issued before it.
    f32x4 rv[BPW][g / 16];
    float pv[BPW][4];
    if (wave_live) {
      const float* rinv_i = rinv + (size_t)i * g * g;
#pragma unroll
      for (int b = 0; b < BPW; ++b) {
        const int n = (wave * BPW + b) * 16 + mr;
#pragma unroll
        for (int kc = 0; kc < g / 16; ++kc)
          rv[b][kc] = *(const f32x4*)(rinv_i + (size_t)n * g + kc * 16 + 4 * kq);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int gr = r0 + 4 * kq + v;
          pv[b][v] = gr < rows ? P[(size_t)gr * cols + i * g + n] : 0.f;
        }
      }
    }
    // 1. correction and he
    if (wave_live) {
      f32x4 acc[BPW];
#pragma unroll
      for (int b = 0; b < BPW; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int h = i0; h < i; ++h) {
        if (tacc_s[h] == 0) continue;
        if (tid == 0) cnt_s[3] += 1;
        f16x8 a[KS], bh[BPW][KS], bl[BPW][KS];
#pragma unroll
        for (int kc = 0; kc < KS; ++kc)
          a[kc] = arow_in ? *(const f16x8*)(dq + (size_t)arow * cols + h * g + kc * 32 + 8 * kq)
                          : f16x8{};
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          const size_t hrow =
              (size_t)(i * g + (wave * BPW + b) * 16 + mr) * cols + (size_t)h * g + 8 * kq;
#pragma unroll
          for (int kc = 0; kc < KS; ++kc) {
            bh[b][kc] = *(const f16x8*)(Hh + hrow + kc * 32);
            bl[b][kc] = *(const f16x8*)(Hl + hrow + kc * 32);
          }
        }
        float sh[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int gr = r0 + 4 * kq + v;
          sh[v] = gr < rows ? scales[(size_t)gr * G + h] * hinv : 0.f;
        }
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          f32x4 seg = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kc = 0; kc < KS; ++kc) {
            seg = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[kc], bh[b][kc], seg, 0, 0, 0);
            seg = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[kc], bl[b][kc], seg, 0, 0, 0);
          }
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[b][v] = fmaf(seg[v], sh[v], acc[b][v]);
        }
      }
      // 16x16 accumulator: element v of lane l is (row 4 * (l / 16) + v, column l % 16).
#pragma unroll
      for (int b = 0; b < BPW; ++b) {
        const int c = (wave * BPW + b) * 16 + mr;
#pragma unroll
        for (int v = 0; v < 4; ++v) he_s[(4 * kq + v) * LDH + c] = pv[b][v] - acc[b][v];
      }
    }
    __syncthreads();
    // 2. u (before division by the scale) = he L^{-T}
    if (wave_live) {
      f32x4 acc[BPW];
#pragma unroll
      for (int b = 0; b < BPW; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < g / 16; ++kc) {
        const f32x4 a4 = *(const f32x4*)(he_s + mr * LDH + kc * 16 + 4 * kq);
#pragma unroll
        for (int b = 0; b < BPW; ++b)
#pragma unroll
          for (int t = 0; t < 4; ++t)
            acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[t], rv[b][kc][t], acc[b], 0, 0, 0);
      }
#pragma unroll
      for (int b = 0; b < BPW; ++b) {
        const int c = (wave * BPW + b) * 16 + mr;
#pragma unroll
        for (int v = 0; v < 4; ++v) u_s[(4 * kq + v) * LDH + c] = acc[b][v];
      }
    }
    __syncthreads();
    // 3. back substitution, 16 lanes per row
    float s = 0.f;
    if (row_in) s = scales[(size_t)grow * G + i];
    const bool skip = !(fabsf(s) > kFp32Eps);
    const bool do_row = row_act && !skip;
    const float inv_s = do_row ? 1.f / s : 0.f;
    ChainState<NT> cs;
    float ut[NT];
    const size_t cbase = (size_t)grow * cols + (size_t)i * g;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int l = cj + 16 * t;
      ut[t] = u_s[crow * LDH + l] * inv_s * rdinv[(size_t)i * g + l];
      const float q = row_in ? (float)codes[cbase + l] : 0.f;
      cs.qold[t] = q;
      cs.qc[t] = q;
      cs.base[t] = q + ut[t];
      cs.acc[t] = 0.f;
    }
    ChainStep<g - 1, NT>::run(cs, rc_s, cj, qmax, load_rcol<g - 1, NT>(rc_s, cj),
                              load_rcol<g - 2, NT>(rc_s, cj));
    float dF = 0.f;  // change of F divided by s_i^2
    int changed = 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float a = cs.acc[t];
      dF = fmaf(rdsq[(size_t)i * g + cj + 16 * t] * a, a - 2.f * ut[t], dF);
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
    // 4. outputs
    if (row_in) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int l = cj + 16 * t;
        if (accept) codes[cbase + l] = (uint8_t)cs.qc[t];
        dq[cbase + l] = accept ? (_Float16)(cs.qc[t] - cs.qold[t]) : (_Float16)0.f;
        if (cand_out != nullptr) cand_out[cbase + l] = (uint8_t)(do_row ? cs.qc[t] : cs.qold[t]);
      }
    }
    if (row_in && cj == 0) {
      if (dec_out != nullptr) {
        uint8_t d = !row_act ? kDecStopped : (skip ? kDecSkip : (accept ? kDecAccept : kDecReject));
        dec_out[(size_t)grow * G + i] = d;
      }
      if (accept) {
        tacc_s[i] = 1;
        atomicAdd(&cnt_s[0], 1);
        atomicAdd(&cnt_s[1], changed);
      }
      if (row_act && skip) atomicAdd(&cnt_s[2], 1);
    }
  }
  __syncthreads();
  if (tid == 0) {
    if (cnt_s[0]) atomicAdd(&cnt->accepted, (unsigned long long)cnt_s[0]);
    if (cnt_s[1]) atomicAdd(&cnt->changed, (unsigned long long)cnt_s[1]);
    if (cnt_s[2]) atomicAdd(&cnt->skipped, (unsigned long long)cnt_s[2]);
    if (cnt_s[3]) atomicAdd(&cnt->corr_blocks, (unsigned long long)cnt_s[3]);
  }
}

template <int G_SIZE>
static hipError_t launch_babai_t(hipStream_t st, int rows, int cols, int bits, int i0, int i1,
                                 const float* P,
                                 const char* ws, const Layout& lay, uint8_t* codes,
                                 const float* scales, const int32_t* zeros,
                                 const uint8_t* active, uint8_t* cand, uint8_t* decision,
                                 Counters* cnt) {
  constexpr int g = G_SIZE;
  const int G = cols / g;
  const size_t lds =
      ((size_t)g * g + 2 * 16 * (g + 4)) * sizeof(float) + ((size_t)G + 4) * sizeof(int);
  hipError_t e = hipFuncSetAttribute((const void*)babai_kernel<g>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(babai_kernel<g>, dim3((rows + 15) / 16), dim3(256), lds, st, rows, cols, bits,
                     i0, i1, P, (const _Float16*)(ws + lay.hhi), (const _Float16*)(ws + lay.hlo),
                     (const float*)(ws + lay.hscale), (const float*)(ws + lay.rinv),
                     (const float*)(ws + lay.rcol), (const float*)(ws + lay.rdinv),
                     (const float*)(ws + lay.rdsq), codes, scales, zeros, active,
                     (_Float16*)(ws + lay.dq), cand, decision, cnt);
  return hipGetLastError();
}

hipError_t launch_babai(hipStream_t st, int rows, int cols, int g, int bits, int i0, int i1,
                        const float* P,
                        const char* ws, const Layout& lay, uint8_t* codes, const float* scales,
                        const int32_t* zeros, const uint8_t* active, uint8_t* cand,
                        uint8_t* decision, Counters* cnt) {
  switch (g) {
    case 32:
      return launch_babai_t<32>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, zeros, active,
                                cand, decision, cnt);
    case 64:
      return launch_babai_t<64>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, zeros, active,
                                cand, decision, cnt);
    case 128:
      return launch_babai_t<128>(st, rows, cols, bits, i0, i1, P, ws, lay, codes, scales, zeros, active,
                                 cand, decision, cnt);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace jarq
