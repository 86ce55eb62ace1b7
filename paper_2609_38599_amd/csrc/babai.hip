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
// and it is kept iff ||u - R_i d||^2 = sum_l R_i(l,l)^2 (x_l - q_l^cand)^2 is
// finite and smaller than ||u||^2.  (This is eq. (10) with v = u + R_i(q - z):
// v - R_i(q^cand - z) = u - R_i d.)
//
// One 256-thread work-group owns 16 rows and visits the groups in order.
// Per group:
//   1. correction: he = P_i - sum_{h<i} D_h H_hi, where P = E H from the
//      start of the sweep and D_h = s_h (q_h^new - q_h^old) holds the accepted
//      changes of earlier groups (zero elsewhere); blocks h in which no row of
//      the tile accepted are skipped.  v_mfma_f32_16x16x4f32, M = 16 rows.
//   2. u = he L_i^{-T} / s_i with L_i^{-1} = R_i^{-T} (v_mfma_f32_16x16x4f32).
//   3. back substitution: 16 lanes per row, lane j owns positions j + 16 t;
//      the owner of position l rounds, the change d_l is broadcast to the
//      row's 16 lanes, and each lane folds R_i(m, l) d_l into its own m < l.
//      R_i is staged in LDS per group.
//   4. accept test per row, in-place code update, D_i, trace and counters.
#include "jarq_internal.h"

namespace jarq {

template <int G_SIZE>
__global__ __launch_bounds__(256, 1) void babai_kernel(
    int rows, int cols, int bits, const float* __restrict__ P, const float* __restrict__ H,
    const float* __restrict__ rinv, const float* __restrict__ rcol,
    const float* __restrict__ rdinv, const float* __restrict__ rdsq, uint8_t* __restrict__ codes,
    const float* __restrict__ scales, const int32_t* __restrict__ zeros,
    const uint8_t* __restrict__ active, float* __restrict__ dlt, uint8_t* __restrict__ cand_out,
    uint8_t* __restrict__ dec_out, Counters* __restrict__ cnt) {
  constexpr int g = G_SIZE;
  constexpr int RT = 16;                 // rows per work-group
  constexpr int NT = g / 16;             // positions per lane in the back substitution
  constexpr int NBLK = g / 16;           // 16-column blocks of a group
  constexpr int BPW = NBLK >= 4 ? NBLK / 4 : 1;  // column blocks per wave
  constexpr int LDH = g + 4;
  const int G = cols / g;
  const float qmax = (float)((1 << bits) - 1);

  extern __shared__ float smem[];
  float* rc_s = smem;                    // g * g   R_i columns, [l][j][t]
  float* he_s = rc_s + g * g;            // RT x LDH
  float* u_s = he_s + RT * LDH;          // RT x LDH
  float* di_s = u_s + RT * LDH;          // g       1 / R(l,l)
  float* dq_s = di_s + g;                // g       R(l,l)^2
  int* tacc_s = (int*)(dq_s + g);        // G       any row of the tile accepted group h
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
  // matrix-core role: A row / B column = lane & 15, k quarter = lane >> 4
  const int mr = lane & 15;
  const int kq = lane >> 4;
  const int arow = r0 + mr;
  const bool arow_in = arow < rows;

  for (int h = tid; h < G; h += 256) tacc_s[h] = 0;
  if (tid < 4) cnt_s[tid] = 0;

  for (int i = 0; i < G; ++i) {
    __syncthreads();  // previous group's D stores, LDS reuse
    {
      const float* src = rcol + (size_t)i * g * g;
      for (int e = tid * 4; e < g * g; e += 256 * 4) *(f32x4*)(rc_s + e) = *(const f32x4*)(src + e);
      for (int e = tid; e < g; e += 256) {
        di_s[e] = rdinv[(size_t)i * g + e];
        dq_s[e] = rdsq[(size_t)i * g + e];
      }
    }
    // 1. correction and he
    {
      f32x4 acc[BPW];
#pragma unroll
      for (int b = 0; b < BPW; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
      const bool wave_live = wave * BPW < NBLK;
      if (wave_live) {
        for (int h = 0; h < i; ++h) {
          if (tacc_s[h] == 0) continue;
          if (tid == 0) cnt_s[3] += 1;
          for (int k0 = h * g; k0 < (h + 1) * g; k0 += 16) {
            const int kk = k0 + 4 * kq;
            const f32x4 a4 = arow_in ? *(const f32x4*)(dlt + (size_t)arow * cols + kk)
                                     : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int b = 0; b < BPW; ++b) {
              const int ncol = i * g + (wave * BPW + b) * 16 + mr;
              const f32x4 b4 = *(const f32x4*)(H + (size_t)ncol * cols + kk);
#pragma unroll
              for (int t = 0; t < 4; ++t)
                acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[t], b4[t], acc[b], 0, 0, 0);
            }
          }
        }
        // 16x16 accumulator: element v of lane l is (row 4 * (l / 16) + v, column l % 16).
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          const int c = (wave * BPW + b) * 16 + mr;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int rr = 4 * kq + v;
            const int gr = r0 + rr;
            const float pv = gr < rows ? P[(size_t)gr * cols + i * g + c] : 0.f;
            he_s[rr * LDH + c] = pv - acc[b][v];
          }
        }
      }
    }
    __syncthreads();
    // 2. u (before division by the scale) = he L^{-T}
    if (wave * BPW < NBLK) {
      f32x4 acc[BPW];
#pragma unroll
      for (int b = 0; b < BPW; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
      const float* rinv_i = rinv + (size_t)i * g * g;
      for (int k0 = 0; k0 < g; k0 += 16) {
        const int kk = k0 + 4 * kq;
        const f32x4 a4 = *(const f32x4*)(he_s + mr * LDH + kk);
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          const int n = (wave * BPW + b) * 16 + mr;
          const f32x4 b4 = *(const f32x4*)(rinv_i + (size_t)n * g + kk);
#pragma unroll
          for (int t = 0; t < 4; ++t)
            acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[t], b4[t], acc[b], 0, 0, 0);
        }
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
    int z = 0;
    if (row_in) {
      s = scales[(size_t)grow * G + i];
      z = zeros[(size_t)grow * G + i];
    }
    const bool skip = !(fabsf(s) > kFp32Eps);
    const bool do_row = row_act && !skip;
    float u[NT], acc[NT], xr[NT];
    int qold[NT], qc[NT];
    const size_t cbase = (size_t)grow * cols + (size_t)i * g;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int l = cj + 16 * t;
      u[t] = do_row ? u_s[crow * LDH + l] / s : 0.f;
      qold[t] = row_in ? (int)codes[cbase + l] : 0;
      qc[t] = qold[t];
      acc[t] = 0.f;
      xr[t] = 0.f;
    }
    float rsum = 0.f;
#pragma unroll
    for (int l = g - 1; l >= 0; --l) {
      const int tl = l >> 4;
      const int jl = l & 15;
      const float xv = (float)qold[tl] + (u[tl] - acc[tl]) * di_s[l];
      const float qv = fminf(fmaxf(rintf(xv), 0.f), qmax);
      const float dv = qv - (float)qold[tl];
      if (cj == jl) {
        xr[tl] = xv;
        qc[tl] = (int)qv;
        const float ex = xv - qv;
        rsum += dq_s[l] * ex * ex;
      }
      const float db = __shfl(dv, (lane & 48) | jl);
      const float* rl = rc_s + (l * 16 + cj) * NT;
#pragma unroll
      for (int t = 0; t <= tl; ++t) acc[t] += rl[t] * db;
    }
    float unorm = 0.f;
    int changed = 0;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      unorm += u[t] * u[t];
      changed += qc[t] != qold[t];
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) {
      unorm += __shfl_xor(unorm, off);
      rsum += __shfl_xor(rsum, off);
      changed += __shfl_xor(changed, off);
    }
    // A proposal equal to the current codes changes F by exactly 0, which the
    // strict test rejects whatever the rounding of the two norms.
    const bool accept = do_row && changed > 0 && isfinite(rsum) && (rsum < unorm);
    // 4. outputs
    if (row_in) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int l = cj + 16 * t;
        const int dq = qc[t] - qold[t];
        if (accept) codes[cbase + l] = (uint8_t)qc[t];
        dlt[cbase + l] = accept ? s * (float)dq : 0.f;
        if (cand_out != nullptr) cand_out[cbase + l] = (uint8_t)(do_row ? qc[t] : qold[t]);
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
static hipError_t launch_babai_t(hipStream_t st, int rows, int cols, int bits, const float* P,
                                 const float* H, const char* ws, const Layout& lay,
                                 uint8_t* codes, const float* scales, const int32_t* zeros,
                                 const uint8_t* active, float* dlt, uint8_t* cand,
                                 uint8_t* decision, Counters* cnt) {
  constexpr int g = G_SIZE;
  const int G = cols / g;
  const size_t lds = ((size_t)g * g + 2 * 16 * (g + 4) + 2 * g) * sizeof(float) +
                     ((size_t)G + 4) * sizeof(int);
  hipError_t e = hipFuncSetAttribute((const void*)babai_kernel<g>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(babai_kernel<g>, dim3((rows + 15) / 16), dim3(256), lds, st, rows, cols, bits,
                     P, H, (const float*)(ws + lay.rinv), (const float*)(ws + lay.rcol),
                     (const float*)(ws + lay.rdinv), (const float*)(ws + lay.rdsq), codes, scales,
                     zeros, active, dlt, cand, decision, cnt);
  return hipGetLastError();
}

hipError_t launch_babai(hipStream_t st, int rows, int cols, int g, int bits, const float* P,
                        const float* H, const char* ws, const Layout& lay, uint8_t* codes,
                        const float* scales, const int32_t* zeros, const uint8_t* active,
                        float* dlt, uint8_t* cand, uint8_t* decision, Counters* cnt) {
  switch (g) {
    case 32:
      return launch_babai_t<32>(st, rows, cols, bits, P, H, ws, lay, codes, scales, zeros, active,
                                dlt, cand, decision, cnt);
    case 64:
      return launch_babai_t<64>(st, rows, cols, bits, P, H, ws, lay, codes, scales, zeros, active,
                                dlt, cand, decision, cnt);
    case 128:
      return launch_babai_t<128>(st, rows, cols, bits, P, H, ws, lay, codes, scales, zeros, active,
                                 dlt, cand, decision, cnt);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace jarq
