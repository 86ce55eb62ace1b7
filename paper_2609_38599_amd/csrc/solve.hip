// Joint scale solve of the scale update (paper eq. (6), App. E.2), in fp64.
//
// The G x G Gram matrix (upper triangle from the Gram kernel, symmetrised by
// construction) and the right-hand side r_a = c_a^T (W H)_a are factored by a
// right-looking Cholesky.  Three kernels:
//   solve_reg_kernel (G <= 32): lane i of a row holds row i of the matrix in
//     registers, two rows per wavefront; the column of each step is exchanged
//     through LDS, the forward substitution runs inside the factorisation, the
//     backward one reads L transposed through LDS.
//   solve_tile_kernel (32 < G <= 108): one row per wavefront, the lower
//     triangle in 4 x 4 register tiles spread over the lanes (see there).
//   solve_col_kernel (108 < G <= 128): the matrix in LDS, column-major, one
//     row per work-group of 128 lanes.
// The stabilised branch of
// App. E.2 (add lambda I and factor again) is taken when an entry is not
// finite, a pivot is not positive, the smallest pivot is at most
// r_cond * max(largest diagonal, 2^-23), or the smallest eigenvalue is at
// most t = r_cond * max(||A||_F, 2^-23).  Every Cholesky pivot is a Schur
// complement and bounded below by the smallest eigenvalue, and the largest
// diagonal bounds the largest eigenvalue from below, so the pivot test only
// fires where the paper's eigenvalue test fires; it can miss a nearly
// singular matrix whose pivots all stay large, which the last test catches.
// ||A||_F bounds the largest eigenvalue from above, so the last test fires
// wherever the paper's does, and beyond it only where the smallest
// eigenvalue lies in (r_cond lambda_max, t].  It is settled cheaply where it
// clearly does not fire: with L's comparison matrix C (|diagonal|, minus
// |off-diagonal|), C^{-1} >= |L^{-1}| entrywise, so x = C^{-1} 1 (solved
// beside the forward substitution) gives ||L^{-1}||_inf <= max x and
// lambda_min = 1 / ||L^{-1}||_2^2 >= 1 / (G (max x)^2).  Only where that
// bound is not above t is A - t I factored: it is positive definite exactly
// when lambda_min > t.  A second failure after lambda I leaves the row's
// scales unchanged and is counted.
#include "jarq_internal.h"

namespace jarq {

// Right-hand sides of the scale systems, r_i = c_i^T (W H)_i for group i of a
// row (eq. (6)), in fp64.  They depend on the row's codes of group i only, so
// the sweep keeps them in `cache` ([layer rows][G]): the first scale solve of
// a run (ctl->valid == 0, or no ctl) forms them from W H and the codes and
// stores them; later ones read them, the code update having added
// d^T (W H)_i for every change d it made since.
struct RhsSrc {
  const float* wh;
  const uint8_t* codes;
  const int32_t* zeros;
  double* cache;
  const GramCtl* ctl;
};

template <int g>
__device__ __forceinline__ double rhs_entry(const RhsSrc& rs, int grow, int i, int cols, int G) {
  const float* whp = rs.wh + (size_t)grow * cols + (size_t)i * g;
  const uint8_t* qp = rs.codes + (size_t)grow * cols + (size_t)i * g;
  const double z = (double)rs.zeros[(size_t)grow * G + i];
  double r = 0.0;
  constexpr int CH = g < 32 ? g : 32;  // columns per batch of loads
#pragma unroll
  for (int c0 = 0; c0 < g; c0 += CH) {
    uint4 qv[CH / 16];
    f32x4 wv[CH / 4];
#pragma unroll
    for (int u = 0; u < CH / 16; ++u) qv[u] = *(const uint4*)(qp + c0 + 16 * u);
#pragma unroll
    for (int u = 0; u < CH / 4; ++u) wv[u] = *(const f32x4*)(whp + c0 + 4 * u);
#pragma unroll
    for (int u = 0; u < CH / 4; ++u) {
      const uint32_t w32 = (u & 3) == 0 ? qv[u / 4].x : (u & 3) == 1 ? qv[u / 4].y
                           : (u & 3) == 2 ? qv[u / 4].z : qv[u / 4].w;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        r = fma((double)((w32 >> (8 * e)) & 0xffu) - z, (double)wv[u][e], r);
    }
  }
  return r;
}

// r_i of layer row grow; `store`: this lane owns the entry (stores it when it
// forms it).
template <int g>
__device__ __forceinline__ double rhs_of(const RhsSrc& rs, int grow, int i, int cols, int G,
                                         bool store) {
  const bool cached = rs.ctl != nullptr && rs.ctl->valid != 0;
  if (cached) return rs.cache[(size_t)grow * G + i];
  const double r = rhs_entry<g>(rs, grow, i, cols, G);
  if (store) rs.cache[(size_t)grow * G + i] = r;
  return r;
}

// 1 / sqrt(x) in fp64: the hardware estimate (about 23 bits) and two Newton
// steps y <- y (3/2 - x y^2 / 2), each of which doubles the correct bits.
__device__ __forceinline__ double rsqrt_f64(double x) {
  double y = __builtin_amdgcn_rsq(x);
  const double h = 0.5 * x;
#pragma unroll
  for (int it = 0; it < 2; ++it) y *= fma(-h * y, y, 1.5);
  return y;
}

template <int GM, int GS>
__global__ __launch_bounds__(64, 2) void solve_reg_kernel(int rows, int cols,
                                                       const float* __restrict__ gram,
                                                       const RhsSrc rs,
                                                       float* __restrict__ scales,
                                                       const uint8_t* __restrict__ active,
                                                       Counters* __restrict__ cnt,
                                                       Flags* __restrict__ flags, float lam,
                                                       float rcond, int accept,
                                                       const int32_t* __restrict__ rowmap,
                                                       const int* __restrict__ n_dev) {
  constexpr int RPW = 64 / GM;  // rows per wavefront
  if (n_dev != nullptr) rows = *n_dev;
  if ((int)blockIdx.x * RPW >= rows) return;  // the whole wavefront: no row here
  constexpr int g = GS;
  const int G = cols / g;
  const int lane = threadIdx.x;
  const int slot = lane / GM;
  const int i = lane % GM;      // this lane's row of the G x G system
  // position `row` of the sweep (Gram matrices) holds layer row `grow`
  // (everything else)
  const int row = blockIdx.x * RPW + slot;
  const bool row_ok = row < rows;
  const bool live = i < G;
  const int rr = row_ok ? row : 0;  // loads stay unconditional: positions past the edge read 0
  const int grow = map_row(rowmap, rr);
  const bool act = row_ok && (active == nullptr || active[grow] != 0);
  const int ic = live ? i : G - 1;

  // column exchange of the factorisation steps and the transposed factor
  // (col_rt: r and the comparison system's x side by side, one access each)
  __shared__ double col_a[RPW][GM], col_r[RPW][GM];
  __shared__ double2 col_rt[RPW][GM];
  __shared__ double lt[RPW][GM][GM + 1];

  // ---- right-hand side r_i = sum over group i of (q - z) (W H) ----
  double r0 = rhs_of<g>(rs, grow, ic, cols, G, live && row_ok);
  if (!live) r0 = 0.0;

  // ---- row i of the Gram matrix (entry (i, j) stored at (min, max)) ----
  double A[GM];
  double diag = 0.0, sq = 0.0;  // A_ii; sum of squares of row i
  bool finite = isfinite(r0);
  const float* gr = gram + (size_t)grow * G * G;  // stored by layer row
  auto load_rows = [&](double shift) __attribute__((always_inline)) {
    sq = 0.0;
#pragma unroll
    for (int j = 0; j < GM; ++j) {
      const bool in = live && j < G;
      const int idx = in ? (j <= i ? j * G + i : i * G + j) : 0;
      const float v = gr[idx];
      if (in) finite &= isfinite(v);
      if (j == i) diag = in ? (double)v : 1.0;
      if (in) sq = fma((double)v, (double)v, sq);
      A[j] = in ? (double)v + (j == i ? shift : 0.0) : (j == i ? 1.0 : 0.0);
    }
  };
  load_rows(0.0);

  // ---- factorisation A = L L^T with the forward substitution L y = r ----
  // Step k: lane k's pivot and r_k reach every lane of the row through LDS
  // (one wavefront: its LDS accesses complete in order, so no barrier); the
  // trailing update A_ij -= A_ik A_jk / A_kk and r_i -= A_ik r_k / A_kk run in
  // every lane (entries above the diagonal are never read).  Afterwards lane
  // i holds L(i, 0..i), y_i and 1 / L(i, i).  The comparison system C x = 1
  // runs along the same way (|l_ik| x_k added where l_ik y_k is subtracted);
  // lane i ends with x_i.
  double r, dinv = 0.0, minpiv, xc;
  bool pivots_ok;
  auto factor = [&]() __attribute__((always_inline)) {
    r = r0;
    xc = 1.0;
    minpiv = INFINITY;
    pivots_ok = true;
#pragma unroll
    for (int k = 0; k < GM; ++k) {
      if (k < G) {
        col_a[slot][i] = A[k];
        col_rt[slot][i] = double2{r, xc};
        const double piv = col_a[slot][k];
        const double2 rt = col_rt[slot][k];
        const double rk = rt.x, tk = rt.y;
        pivots_ok &= piv > 0.0 && isfinite(piv);
        minpiv = fmin(minpiv, piv);
        const double rs = rsqrt_f64(piv);
        const double li = A[k] * (rs * rs);
#pragma unroll
        for (int j = k + 1; j < GM; ++j) A[j] = fma(-li, col_a[slot][j], A[j]);
        r = i > k ? fma(-li, rk, r) : (i == k ? rk * rs : r);
        xc = i > k ? fma(fabs(li), tk, xc) : (i == k ? tk * rs : xc);
        A[k] *= rs;
        if (i == k) dinv = rs;
      }
    }
  };
  factor();
  double dmax = live ? diag : 0.0, fro = live ? sq : 0.0;
  double xm = live ? (xc == xc ? xc : INFINITY) : 0.0;  // a NaN bound clears nothing
#pragma unroll
  for (int off = GM / 2; off >= 1; off >>= 1) {
    dmax = fmax(dmax, __shfl_xor(dmax, off));
    fro += __shfl_xor(fro, off);
    xm = fmax(xm, __shfl_xor(xm, off));
  }
  const double tshift = (double)rcond * fmax(sqrt(fro), (double)kFp32Eps);
  const unsigned long long bad = __ballot(!finite);
  const unsigned long long slot_mask = GM == 64 ? ~0ull : (((1ull << GM) - 1) << (slot * GM));
  const bool all_finite = (bad & slot_mask) == 0;
  bool ridge = !all_finite || !pivots_ok ||
               !(minpiv > (double)rcond * fmax(dmax, (double)kFp32Eps));
  // lambda_min >= 1 / (G (max x)^2); where that does not clear t, factor A - t I
  const bool unsure = !ridge && !((double)G * xm * xm * tshift < 1.0);
  if (__any(unsure)) {
    load_rows(unsure ? -tshift : 0.0);
    factor();
    ridge = ridge || (unsure && !(pivots_ok && minpiv > 0.0));
  }
  // A + lam I for the rows that need it; the other rows of the wavefront
  // factor A again (the same arithmetic, so the same factor)
  bool failed = false;
  if (__any(ridge || unsure)) {
    load_rows(ridge ? (double)lam : 0.0);
    factor();
    failed = ridge && !(pivots_ok && minpiv > 0.0);
  }

  // ---- backward substitution L^T s = y: L transposed through LDS ----
#pragma unroll
  for (int j = 0; j < GM; ++j) lt[slot][i][j] = A[j];
#pragma unroll
  for (int k = GM - 1; k >= 0; --k) {
    if (k < G) {
      col_r[slot][i] = r * dinv;
      const double sk = col_r[slot][k];
      const double lkj = lt[slot][k][i];
      r = i < k ? fma(-lkj, sk, r) : (i == k ? sk : r);
    }
  }

  // Ridge acceptance (the remark of App. G.5, optional): a ridge solution is
  // kept only when it does not increase F_j.  At fixed codes
  // F_j(s) = const + s^T G s - 2 r^T s, so the change needs the Gram matrix
  // (reloaded: A holds the factor) and r only.
  bool keep_old = false;
  if (accept && __any(ridge && !failed)) {
    const double s_new = live ? r : 0.0;
    const double s_old = live ? (double)scales[(size_t)grow * G + i] : 0.0;
    load_rows(0.0);
    col_a[slot][i] = s_new;
    col_r[slot][i] = s_old;
    double tn = 0.0, to = 0.0;
#pragma unroll
    for (int j = 0; j < GM; ++j) {
      tn = fma(A[j], col_a[slot][j], tn);
      to = fma(A[j], col_r[slot][j], to);
    }
    double dq = live ? (s_new * tn - 2.0 * r0 * s_new) - (s_old * to - 2.0 * r0 * s_old) : 0.0;
#pragma unroll
    for (int off = GM / 2; off >= 1; off >>= 1) dq += __shfl_xor(dq, off);
    keep_old = ridge && !failed && dq > 0.0;
  }

  if (act && live && !failed && !keep_old) scales[(size_t)grow * G + i] = (float)r;
  if (act && i == 0) {
    if (ridge) atomicAdd(&cnt->ridge_rows, 1u);
    if (failed) {
      atomicAdd(&cnt->solve_failed, 1u);
      atomicAdd(&flags->solve_failed, 1);
    }
  }
}

// G in (32, 128]: one row per work-group of 64 or 128 threads; lane i owns
// row i of the system, which sits in LDS column-major (element (a, b) at
// b * LD + a), so a lane's own accesses are contiguous across lanes and step
// k's column (a, k) is a broadcast read.  Column k is left unscaled and
// 1 / sqrt(pivot k) is kept per k: L(a, k) = A(a, k) rk_s[k].  One barrier
// per step (the trailing update writes columns > k only).
template <int GS>
__global__ __launch_bounds__(128) void solve_col_kernel(int rows, int cols,
                                                        const float* __restrict__ gram,
                                                        const RhsSrc rs,
                                                        float* __restrict__ scales,
                                                        const uint8_t* __restrict__ active,
                                                        Counters* __restrict__ cnt,
                                                        Flags* __restrict__ flags, float lam,
                                                        float rcond, int accept,
                                                        const int32_t* __restrict__ rowmap,
                                                        const int* __restrict__ n_dev) {
  constexpr int g = GS;
  const int G = cols / g;
  const int LD = G | 1;  // odd stride (in doubles): rows of a column spread over banks
  const int row = blockIdx.x;  // position of the sweep; layer row grow
  const int i = threadIdx.x;
  const int nthr = blockDim.x;
  if (n_dev != nullptr) rows = *n_dev;
  if (row >= rows) return;
  const int grow = map_row(rowmap, row);
  if (active != nullptr && !active[grow]) return;
  const bool live = i < G;
  const int ic = live ? i : G - 1;
  extern __shared__ double sm[];
  double* A = sm;               // G columns of LD
  double* r_s = A + (size_t)G * LD;  // broadcast slot of r / s
  double* rk_s = r_s + G;       // 1 / sqrt(pivot k)
  double* red = rk_s + G;       // two wavefronts' partial max / flags
  double* x_s = red + 2;        // broadcast slot of the comparison system

  // right-hand side r_i = sum over group i of (q - z) (W H)
  const double r0 = rhs_of<g>(rs, grow, ic, cols, G, live);

  const float* gr = gram + (size_t)grow * G * G;  // stored by layer row
  double diag = 0.0, sq = 0.0;  // A_ii; sum of squares of row i
  bool finite = !live || isfinite(r0);
  // column-major copy of the system (+ shift on the diagonal); entry (i, j)
  // of the Gram matrix is stored at (min, max)
  // (batches of 8: loads first, from clamped indices, then the LDS stores)
  auto load = [&](double shift) __attribute__((always_inline)) {
    sq = 0.0;
    if (live) {
      for (int j0 = 0; j0 < G; j0 += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = min(j0 + u, G - 1);
          v[u] = gr[j <= i ? j * G + i : i * G + j];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + u;
          if (j < G) {
            finite &= isfinite(v[u]);
            if (j == i) diag = (double)v[u];
            sq = fma((double)v[u], (double)v[u], sq);
            A[(size_t)j * LD + i] = (double)v[u] + (j == i ? shift : 0.0);
          }
        }
      }
    }
  };
  // Right-looking factorisation with the forward substitution; returns in r
  // this lane's y_i, and in xc its x_i of the comparison system C x = 1.
  // Pivot k is read by every lane from LDS.
  double r = 0.0, xc = 1.0, minpiv = INFINITY;
  bool pivots_ok = true;
  auto factor = [&]() __attribute__((always_inline)) {
    r = r0;
    xc = 1.0;
    minpiv = INFINITY;
    pivots_ok = true;
    if (live) {
      r_s[i] = r;
      x_s[i] = xc;
    }
    __syncthreads();
    for (int k = 0; k < G; ++k) {
      const double piv = A[(size_t)k * LD + k];
      const double rk = r_s[k];
      const double xk = x_s[k];
      pivots_ok &= piv > 0.0 && isfinite(piv);
      minpiv = fmin(minpiv, piv);
      const double rs = rsqrt_f64(piv);
      if (live && i > k) {
        const double li = A[(size_t)k * LD + i] * (rs * rs);
        // A(i, j) -= A(i, k) A(j, k) / A(k, k) for k < j <= i, 8 at a time:
        // reads first (clamped), then the writes
        for (int j0 = k + 1; j0 <= i; j0 += 8) {
          double cv[8], av[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int j = min(j0 + u, i);
            cv[u] = A[(size_t)k * LD + j];
            av[u] = A[(size_t)j * LD + i];
          }
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (j0 + u <= i) A[(size_t)(j0 + u) * LD + i] = fma(-li, cv[u], av[u]);
        }
        r = fma(-li, rk, r);
        r_s[i] = r;
        xc = fma(fabs(li), xk, xc);
        x_s[i] = xc;
      }
      if (i == k) {
        r = rk * rs;
        xc = xk * rs;
        rk_s[k] = rs;
      }
      __syncthreads();
    }
  };
  auto slot_max = [&](double v) {  // over the work-group's live lanes
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off));
    if ((i & 63) == 0) red[i >> 6] = v;
    __syncthreads();
    v = red[0];
    if (nthr > 64) v = fmax(v, red[1]);
    __syncthreads();
    return v;
  };
  auto all_true = [&](bool b) {
    const bool w = __all(b);
    if ((i & 63) == 0) red[i >> 6] = w ? 1.0 : 0.0;
    __syncthreads();
    bool res = red[0] != 0.0 && (nthr <= 64 || red[1] != 0.0);
    __syncthreads();
    return res;
  };

  auto slot_sum = [&](double v) {  // over the work-group's lanes
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    if ((i & 63) == 0) red[i >> 6] = v;
    __syncthreads();
    v = red[0];
    if (nthr > 64) v += red[1];
    __syncthreads();
    return v;
  };

  load(0.0);
  const double dmax = slot_max(live ? diag : 0.0);
  const double tshift = (double)rcond * fmax(sqrt(slot_sum(live ? sq : 0.0)), (double)kFp32Eps);
  const bool all_finite = all_true(finite);
  factor();
  bool ridge = !all_finite || !pivots_ok ||
               !(minpiv > (double)rcond * fmax(dmax, (double)kFp32Eps));
  // lambda_min >= 1 / (G (max x)^2); where that does not clear t, factor
  // A - t I and then A again (a NaN bound clears nothing)
  const double xm = slot_max(live ? (xc == xc ? xc : INFINITY) : 0.0);
  if (!ridge && !((double)G * xm * xm * tshift < 1.0)) {  // uniform
    __syncthreads();
    load(-tshift);
    factor();
    ridge = !(pivots_ok && minpiv > 0.0);
    if (!ridge) {
      __syncthreads();
      load(0.0);
      factor();
    }
  }
  bool failed = false;
  if (ridge) {  // uniform: every lane saw the same pivots
    __syncthreads();
    load((double)lam);
    factor();
    failed = !(pivots_ok && minpiv > 0.0);
  }

  // backward substitution L^T s = y: L(k, j) = A(k, j) rk_s[j] for j < k
  for (int k = G - 1; k >= 0; --k) {
    if (i == k) {
      r *= rk_s[k];
      r_s[k] = r;
    }
    __syncthreads();
    if (live && i < k) r = fma(-A[(size_t)i * LD + k] * rk_s[i], r_s[k], r);
  }

  // Ridge acceptance (optional), as in solve_reg_kernel; the Gram matrix is
  // read again from global memory (A holds the factor).
  bool keep_old = false;
  if (accept && ridge && !failed) {  // uniform across the work-group
    const double s_new = live ? r : 0.0;
    const double s_old = live ? (double)scales[(size_t)grow * G + i] : 0.0;
    __syncthreads();  // the backward substitution's reads of r_s are done
    if (live) {
      r_s[i] = s_new;
      rk_s[i] = s_old;
    }
    __syncthreads();
    double tn = 0.0, to = 0.0;
    if (live) {
      for (int j0 = 0; j0 < G; j0 += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = min(j0 + u, G - 1);
          v[u] = gr[j <= i ? j * G + i : i * G + j];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (j0 + u < G) {
            tn = fma((double)v[u], r_s[j0 + u], tn);
            to = fma((double)v[u], rk_s[j0 + u], to);
          }
      }
    }
    double dq = live ? (s_new * tn - 2.0 * r0 * s_new) - (s_old * to - 2.0 * r0 * s_old) : 0.0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) dq += __shfl_xor(dq, off);
    if ((i & 63) == 0) red[i >> 6] = dq;
    __syncthreads();
    dq = nthr > 64 ? red[0] + red[1] : red[0];
    keep_old = dq > 0.0;
  }

  if (live && !failed && !keep_old) scales[(size_t)grow * G + i] = (float)r;
  if (i == 0) {
    if (ridge) atomicAdd(&cnt->ridge_rows, 1u);
    if (failed) {
      atomicAdd(&cnt->solve_failed, 1u);
      atomicAdd(&flags->solve_failed, 1);
    }
  }
}

// One wavefront per row for every G up to 108: the lower triangle of the
// G x G system in 4 x 4 tiles held in registers, tile t (numbered column by
// column: tiles of column-block 0 first) in lane t % 64, slot t / 64.  Step k
// of the right-looking factorisation publishes column k of the Schur
// complement in LDS (the lanes holding it write it; a barrier, which for one
// wavefront only orders the accesses, precedes every read), every lane forms
// 1/sqrt(pivot) from it itself (same bits everywhere) and scales what it
// reads, and every tile with columns right of k subtracts l_rk l_ck from its
// entries.  Tiles of finished column blocks drop out (the slot is skipped once
// every lane's tile in it is finished).  The forward substitution L y = r runs
// along (r_i in lane i % 64, slot i / 64; y_k broadcast by a cross-lane
// shuffle), and the published columns stay in LDS (packed column-major lower
// triangle) for the backward one.
// f(IntC<0>), ..., f(IntC<3>): a loop of four steps with a static index
template <int V>
struct StepC {
  static constexpr int value = V;
};
template <typename F>
__device__ __forceinline__ void Unroll4(F&& f) {
  f(StepC<0>{});
  f(StepC<1>{});
  f(StepC<2>{});
  f(StepC<3>{});
}

template <int TPL, int GS>
__global__ __launch_bounds__(64) void solve_tile_kernel(int rows, int cols,
                                                        const float* __restrict__ gram,
                                                        const RhsSrc rs,
                                                        float* __restrict__ scales,
                                                        const uint8_t* __restrict__ active,
                                                        Counters* __restrict__ cnt,
                                                        Flags* __restrict__ flags, float lam,
                                                        float rcond, int accept,
                                                        const int32_t* __restrict__ rowmap,
                                                        const int* __restrict__ n_dev) {
  constexpr int g = GS;
  const int G = cols / g;
  if (n_dev != nullptr) rows = *n_dev;
  const int row = blockIdx.x;  // position of the sweep; layer row grow
  if (row >= rows) return;
  const int grow = map_row(rowmap, row);
  if (active != nullptr && !active[grow]) return;
  const int lane = threadIdx.x;
  const int T = (G + 3) >> 2;            // tile rows (and columns)
  const int NT = T * (T + 1) / 2;        // tiles of the lower triangle
  extern __shared__ double sm[];
  double* colbuf = sm;                         // column k of L: rows k .. G - 1
  double* rsb = colbuf + G * (G + 1) / 2;      // ridge acceptance: previous scales
  double* vb = rsb + G;                        // ridge acceptance: new scales
  auto cstart = [&](int k) { return k * G - k * (k - 1) / 2; };

  // ---- right-hand side r_i = sum over group i of (q - z) (W H), i = lane, lane + 64 ----
  double r0[2] = {0.0, 0.0};
  bool finite = true;
#pragma unroll
  for (int sl = 0; sl < 2; ++sl) {
    const int i = lane + 64 * sl;
    if (i < G) {
      r0[sl] = rhs_of<g>(rs, grow, i, cols, G, true);
      finite &= isfinite(r0[sl]);
    }
  }

  // ---- this lane's tiles ----
  double ta[TPL][4][4];
  int ttr[TPL], ttc[TPL];
  bool tvalid[TPL];
#pragma unroll
  for (int m = 0; m < TPL; ++m) {
    int id = lane + 64 * m, tc = 0;
    tvalid[m] = id < NT;
    while (tc < T && id >= T - tc) {  // column-block tc holds T - tc tiles
      id -= T - tc;
      ++tc;
    }
    ttc[m] = tc;
    ttr[m] = tc + id;
  }
  // last step at which slot m still has columns to update, over the wavefront
  int kend[TPL];
#pragma unroll
  for (int m = 0; m < TPL; ++m) {
    int e = tvalid[m] ? 4 * ttc[m] + 3 : -1;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) e = max(e, __shfl_xor(e, off));
    kend[m] = e;
  }
  const float* gr = gram + (size_t)grow * G * G;  // upper triangle, stored by layer row
  double diag = 0.0, sq = 0.0;  // largest diagonal; sum of squares (both triangles)
  auto load = [&](double shift) __attribute__((always_inline)) {
    sq = 0.0;
#pragma unroll
    for (int m = 0; m < TPL; ++m) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int r = 4 * ttr[m] + a, c = 4 * ttc[m] + b;
          const bool in = tvalid[m] && r < G && c <= r;
          const float v = in ? gr[(size_t)c * G + r] : 0.f;
          if (in) finite &= isfinite(v);
          if (in && r == c) diag = fmax(diag, (double)v);
          sq = fma((r == c ? 1.0 : 2.0) * (double)v, (double)v, sq);
          ta[m][a][b] = (double)v + (in && r == c ? shift : 0.0);
        }
      }
      // one tile's loads in flight at a time (registers)
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // The column published at step k is the Schur complement's column k
  // (unscaled); every lane forms 1/sqrt(pivot) from it, and reads scale by it.
  // The comparison system C x = 1 runs beside the forward substitution (xx).
  double rr[2], xx[2], rs_own[2] = {0.0, 0.0}, minpiv = INFINITY;
  bool pivots_ok = true;
  auto factor = [&]() __attribute__((always_inline)) {
    rr[0] = r0[0];
    rr[1] = r0[1];
    xx[0] = 1.0;
    xx[1] = 1.0;
    minpiv = INFINITY;
    pivots_ok = true;
    for (int kc = 0; kc < T; ++kc) {
      // four steps per column block, unrolled: the tile column j is static
      Unroll4([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        const int k = 4 * kc + j;
        if (k >= G) return;  // uniform
        // column k of the packed store, indexed by row: colk[r] for r >= k
        double* colk = colbuf + (cstart(k) - k);
        // publish column k (rows k .. G - 1) from the tiles of column-block kc
#pragma unroll
        for (int m = 0; m < TPL; ++m) {
          if (tvalid[m] && ttc[m] == kc) {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
              const int r = 4 * ttr[m] + a;
              if (r >= k && r < G) colk[4 * ttr[m] + a] = ta[m][a][j];
            }
          }
        }
        __syncthreads();  // one wavefront: orders the LDS writes before the reads
        const double piv = colk[k];
        pivots_ok &= piv > 0.0 && isfinite(piv);
        minpiv = fmin(minpiv, piv);
        const double rs = rsqrt_f64(piv);
        const double rs2 = rs * rs;
        // forward substitution: y_k = r_k / l_kk, r_i -= l_ik y_k for i > k
        const double yk = __shfl(k >> 6 ? rr[1] : rr[0], k & 63) * rs;
        const double xk = __shfl(k >> 6 ? xx[1] : xx[0], k & 63) * rs;
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) {
          const int i = lane + 64 * sl;
          if (i > k && i < G) {
            const double lik = colk[i] * rs;
            rr[sl] = fma(-lik, yk, rr[sl]);
            xx[sl] = fma(fabs(lik), xk, xx[sl]);
          }
          if (i == k) {
            rr[sl] = yk;
            xx[sl] = xk;
            rs_own[sl] = rs;
          }
        }
        // Trailing update of the tiles with columns right of k, unmasked:
        // an entry (r, c) with r > k and c > k (r, c < G) reads its column
        // values from column k; every other entry of a tile is finished or
        // padding, is never read again, and may take any value.  Rows below
        // k and past G read inside the allocation (column k - 1's tail, the
        // scratch after the last column).
#pragma unroll
        for (int m = 0; m < TPL; ++m) {
          if (k < kend[m]) {
            const double* pr = colk + 4 * ttr[m];
            const double* pc = colk + 4 * ttc[m];
            double lr[4], lc[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) lr[a] = pr[a] * rs2;
#pragma unroll
            for (int b = 0; b < 4; ++b) lc[b] = pc[b];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
              for (int b = 0; b < 4; ++b) ta[m][a][b] = fma(-lr[a], lc[b], ta[m][a][b]);
          }
          // one tile's column values live at a time (registers)
          __builtin_amdgcn_sched_barrier(0);
        }
      });
    }
  };

  load(0.0);
  double dmax = diag, fro = sq;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    dmax = fmax(dmax, __shfl_xor(dmax, off));
    fro += __shfl_xor(fro, off);
  }
  const double tshift = (double)rcond * fmax(sqrt(fro), (double)kFp32Eps);
  const bool all_finite = __all(finite);
  factor();
  bool ridge = !all_finite || !pivots_ok ||
               !(minpiv > (double)rcond * fmax(dmax, (double)kFp32Eps));
  // lambda_min >= 1 / (G (max x)^2); where that does not clear t, factor
  // A - t I and then A again (a NaN bound clears nothing)
  double xm = 0.0;
#pragma unroll
  for (int sl = 0; sl < 2; ++sl)
    if (lane + 64 * sl < G) xm = fmax(xm, xx[sl] == xx[sl] ? xx[sl] : INFINITY);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) xm = fmax(xm, __shfl_xor(xm, off));
  if (!ridge && !((double)G * xm * xm * tshift < 1.0)) {  // uniform
    __syncthreads();  // the last step's reads are done before the columns are rewritten
    load(-tshift);
    factor();
    ridge = !(pivots_ok && minpiv > 0.0);
    if (!ridge) {
      __syncthreads();
      load(0.0);
      factor();
    }
  }
  bool failed = false;
  if (ridge) {  // uniform: every lane saw the same pivots
    __syncthreads();  // the last step's reads are done before the columns are rewritten
    load((double)lam);
    factor();
    failed = !(pivots_ok && minpiv > 0.0);
  }

  // ---- backward substitution L^T s = y: s_k = y_k / l_kk, y_i -= l_ki s_k ----
  // l_ki = (column i as published) / sqrt(pivot i); lane i keeps 1/sqrt(pivot i).
  for (int k = G - 1; k >= 0; --k) {
    const double sk = __shfl(k >> 6 ? rr[1] * rs_own[1] : rr[0] * rs_own[0], k & 63);
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      const int i = lane + 64 * sl;
      if (i < k) rr[sl] = fma(-(colbuf[cstart(i) + k - i] * rs_own[sl]), sk, rr[sl]);
      if (i == k) rr[sl] = sk;
    }
  }

  // Ridge acceptance (optional; the remark of App. G.5): keep the ridge
  // solution only when it does not increase F_j, from the Gram matrix
  // (reloaded: the tiles hold the factor) and the right-hand side:
  // dq = s'^T G s' - s^T G s - 2 r^T (s' - s).
  bool keep_old = false;
  if (accept && ridge && !failed) {  // uniform
    double s_old[2];
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      const int i = lane + 64 * sl;
      s_old[sl] = i < G ? (double)scales[(size_t)grow * G + i] : 0.0;
      if (i < G) {
        vb[i] = rr[sl];       // s' (new)
        rsb[i] = s_old[sl];   // s (previous)
      }
    }
    __syncthreads();  // the writes before every lane's reads
    load(0.0);
    double dq = 0.0;
#pragma unroll
    for (int m = 0; m < TPL; ++m) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int r = 4 * ttr[m] + a, c = 4 * ttc[m] + b;
          if (tvalid[m] && r < G && c <= r) {
            const double w = r == c ? 1.0 : 2.0;
            dq += w * ta[m][a][b] * (vb[r] * vb[c] - rsb[r] * rsb[c]);
          }
        }
      }
    }
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
      if (lane + 64 * sl < G) dq -= 2.0 * r0[sl] * (rr[sl] - s_old[sl]);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) dq += __shfl_xor(dq, off);
    keep_old = dq > 0.0;
  }

  if (!failed && !keep_old) {
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      const int i = lane + 64 * sl;
      if (i < G) scales[(size_t)grow * G + i] = (float)rr[sl];
    }
  }
  if (lane == 0) {
    if (ridge) atomicAdd(&cnt->ridge_rows, 1u);
    if (failed) {
      atomicAdd(&cnt->solve_failed, 1u);
      atomicAdd(&flags->solve_failed, 1);
    }
  }
}

template <int TPL, int GS>
static hipError_t launch_solve_tile(hipStream_t st, int rows, int cols, const float* gram,
                                    const RhsSrc& rs,
                                    float* scales, const uint8_t* active, Counters* cnt,
                                    Flags* flags, float lam, float rcond, int accept,
                                    const int32_t* rowmap, const int* n_dev) {
  const int G = cols / GS;
  const size_t lds = ((size_t)G * (G + 1) / 2 + 2 * (size_t)G) * sizeof(double);
  // the most any system of this tile count needs (T (T + 1) / 2 <= 64 TPL tiles of 4)
  constexpr int kGmax = TPL == 1 ? 40 : TPL == 2 ? 60 : TPL == 3 ? 76 : TPL == 4 ? 88 : 108;
  static std::atomic<unsigned long long> lds_set{0};
  hipError_t e = allow_dynamic_lds((const void*)solve_tile_kernel<TPL, GS>,
                                   ((size_t)kGmax * (kGmax + 1) / 2 + 2 * kGmax) * sizeof(double),
                                   lds_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((solve_tile_kernel<TPL, GS>), dim3(rows), dim3(64), lds, st, rows, cols,
                     gram, rs, scales, active, cnt, flags, lam, rcond, accept,
                     rowmap, n_dev);
  return hipGetLastError();
}

template <int GS>
static hipError_t launch_solve_col(hipStream_t st, int rows, int cols, const float* gram,
                                   const RhsSrc& rs,
                                   float* scales, const uint8_t* active, Counters* cnt,
                                   Flags* flags, float lam, float rcond, int accept,
                                   const int32_t* rowmap, const int* n_dev) {
  const int G = cols / GS;
  const int LD = G | 1;
  const size_t lds = ((size_t)G * LD + 3 * (size_t)G + 2) * sizeof(double);
  static std::atomic<unsigned long long> lds_set{0};
  // the widest layer: G = 128 (odd stride 129)
  hipError_t e = allow_dynamic_lds((const void*)solve_col_kernel<GS>,
                                   ((size_t)128 * 129 + 3 * 128 + 2) * sizeof(double), lds_set);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((solve_col_kernel<GS>), dim3(rows), dim3(G <= 64 ? 64 : 128), lds, st, rows,
                     cols, gram, rs, scales, active, cnt, flags, lam, rcond, accept, rowmap, n_dev);
  return hipGetLastError();
}

template <int GM, int GS>
static hipError_t launch_solve_reg(hipStream_t st, int rows, int cols, const float* gram,
                                   const RhsSrc& rs,
                                   float* scales, const uint8_t* active, Counters* cnt,
                                   Flags* flags, float lam, float rcond, int accept,
                                   const int32_t* rowmap, const int* n_dev) {
  constexpr int RPW = 64 / GM;
  hipLaunchKernelGGL((solve_reg_kernel<GM, GS>), dim3((rows + RPW - 1) / RPW), dim3(64), 0, st,
                     rows, cols, gram, rs, scales, active, cnt, flags, lam, rcond, accept, rowmap, n_dev);
  return hipGetLastError();
}

hipError_t launch_solve(hipStream_t st, int rows, int cols, int g, const float* gram,
                        const float* wh, const uint8_t* codes, const int32_t* zeros,
                        double* rhs_cache, const GramCtl* rctl,
                        float* scales, const uint8_t* active, Counters* cnt, Flags* flags,
                        float lam, float rcond, int accept, const int32_t* rowmap,
                        const int* n_dev) {
  const int G = cols / g;
  const int T = (G + 3) / 4, NT = T * (T + 1) / 2;  // 4 x 4 tiles of the lower triangle
  const RhsSrc rs{wh, codes, zeros, rhs_cache, rctl};
#define JARQ_SOLVE_TILE(TPL)                                                                     \
  switch (g) {                                                                                   \
    case 32: return launch_solve_tile<TPL, 32>(st, rows, cols, gram, rs, scales,   \
                                               active, cnt, flags, lam, rcond, accept, rowmap,   \
                                               n_dev);                                           \
    case 64: return launch_solve_tile<TPL, 64>(st, rows, cols, gram, rs, scales,   \
                                               active, cnt, flags, lam, rcond, accept, rowmap,   \
                                               n_dev);                                           \
    case 128: return launch_solve_tile<TPL, 128>(st, rows, cols, gram, rs, scales, \
                                                 active, cnt, flags, lam, rcond, accept, rowmap, \
                                                 n_dev);                                         \
    default: return hipErrorInvalidValue;                                                        \
  }
  if (G <= 32) {  // two systems per wavefront, a row of the system per lane
    switch (g) {
      case 32: return launch_solve_reg<32, 32>(st, rows, cols, gram, rs, scales,
                                               active, cnt, flags, lam, rcond, accept, rowmap,
                                               n_dev);
      case 64: return launch_solve_reg<32, 64>(st, rows, cols, gram, rs, scales,
                                               active, cnt, flags, lam, rcond, accept, rowmap,
                                               n_dev);
      case 128: return launch_solve_reg<32, 128>(st, rows, cols, gram, rs, scales,
                                                 active, cnt, flags, lam, rcond, accept, rowmap,
                                                 n_dev);
      default: return hipErrorInvalidValue;
    }
  }
  if (NT <= 128) { JARQ_SOLVE_TILE(2) }
  if (NT <= 192) { JARQ_SOLVE_TILE(3) }
  if (NT <= 256) { JARQ_SOLVE_TILE(4) }
  if (NT <= 384) { JARQ_SOLVE_TILE(6) }
#undef JARQ_SOLVE_TILE
  if (G <= 128) {  // the widest layers: the system in LDS, one work-group per row
    switch (g) {
      case 32: return launch_solve_col<32>(st, rows, cols, gram, rs, scales, active,
                                           cnt, flags, lam, rcond, accept, rowmap, n_dev);
      case 64: return launch_solve_col<64>(st, rows, cols, gram, rs, scales, active,
                                           cnt, flags, lam, rcond, accept, rowmap, n_dev);
      case 128: return launch_solve_col<128>(st, rows, cols, gram, rs, scales,
                                             active, cnt, flags, lam, rcond, accept, rowmap, n_dev);
      default: break;
    }
  }
  return hipErrorInvalidValue;  // G > 128 is rejected by the API
}

}  // namespace jarq
