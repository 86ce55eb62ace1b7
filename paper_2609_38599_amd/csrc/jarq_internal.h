// Internal declarations shared by the HIP translation units of libjarq.
// Nothing here is part of the public ABI (include/jarq.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

namespace jarq {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kFp32Eps = 1.1920928955078125e-07f;  // 2^-23, App. E.2 "FP32 machine epsilon"
constexpr int kObjTile = 64;                           // columns per objective partial

// Per-group outcome of the code update.
enum : uint8_t { kDecReject = 0, kDecAccept = 1, kDecSkip = 2, kDecStopped = 3 };

// Device-side counters of one sweep.  Integer atomics only, so totals do not
// depend on scheduling.
// Counts of one sweep.  The workspace holds kSubLists copies, one cache line
// each: work-group b of the code update adds into copy b % kSubLists (a
// single copy would serialise every work-group's atomics); the sweep record
// sums them.
struct Counters {
  unsigned long long accepted;
  unsigned long long changed;
  unsigned long long skipped;
  unsigned long long corr_blocks;  // 16-row x g x g correction products executed
  unsigned int ridge_rows;
  unsigned int solve_failed;
  unsigned int active_rows;
  unsigned int pad;
  unsigned char line_pad[80];      // one 128-byte line per copy
};

// Row lists that every work-group of a launch appends to are split into
// kSubLists sub-lists: work-group b appends to sub-list b % kSubLists, whose
// counter sits kCtrStride words (one cache line) away from the next one's.
// A list is the concatenation of its sub-lists; each sub-list has room for
// sublist_cap(rows) entries.
constexpr int kSubLists = 16;
constexpr int kCtrStride = 32;
__host__ __device__ inline int sublist_cap(int rows) {
  const int tiles = (rows + 15) / 16;
  return 16 * ((tiles + kSubLists - 1) / kSubLists);
}

// One recorded sweep.
struct SweepRecord {
  double objective_after_scales;
  unsigned long long accepted;
  unsigned long long changed;
  unsigned long long skipped;
  unsigned long long corr_blocks;
  unsigned int ridge_rows;
  unsigned int solve_failed;
  unsigned int active_rows;   // rows that ran the code update
  unsigned int started_rows;  // rows the sweep started with
  unsigned int gram_listed;   // the Gram matrices were rebuilt from the row lists
  unsigned int pad;
};

// State of the incremental Gram build (gram.hip).
struct GramCtl {
  int valid;   // every active row's matrix matches its codes before the last code update
  int listed;  // the last build used the row lists
  int pad[2];
};

// Rows a sweep works on, kept on the device when early stopping is on.
struct SweepCtl {
  int n;        // rows active at the start of the sweep (the list in rowmap)
  int started;  // sweeps that started with at least one row
  int pad[2];
};

// Status words written by device checks and read by the host.
struct Flags {
  int not_spd;         // blocks H_ii that failed Cholesky
  int bad_codes;       // codes > 2^b - 1
  int bad_zeros;       // |z| > 1024
  int solve_failed;    // rows whose scale solve failed after the ridge (all sweeps)
  int pad[4];
};

// hipFuncSetAttribute(MaxDynamicSharedMemorySize, bytes) once per kernel and
// device (bit d of `done` for device d < 64): the attribute belongs to the
// function, and setting it again on every launch costs host time that the GPU
// spends idle between short kernels.  `bytes` is the most any launch of the
// kernel asks for.
inline hipError_t allow_dynamic_lds(const void* fn, size_t bytes,
                                    std::atomic<unsigned long long>& done) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
  const unsigned long long bit = (dev >= 0 && dev < 64) ? 1ull << dev : 0ull;
  if (bit != 0 && (done.load(std::memory_order_acquire) & bit) != 0) return hipSuccess;
  const hipError_t e =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e == hipSuccess && bit != 0) done.fetch_or(bit, std::memory_order_release);
  return e;
}

// Offsets (bytes) of the workspace regions for one problem size.
struct Layout {
  size_t lfac;      // [G][g][g] f64: L_i^{-1} (holds L_i while it is factored)
  size_t rinv;      // [G][g][g] f32: row n = row n of L_i^{-1} = column n of R_i^{-1}
  size_t rcol;      // [G][g][g/(16 W)][16][W] f32: R~_i columns in lane chunks (W = min(4, g/16))
  size_t rdinv;     // [G][g] f32: 1 / R_i(l,l)
  size_t rdsq;      // [G][g] f32: R_i(l,l)^2
  size_t hhi;       // [cols][cols] f16: H 2^t, high term
  size_t hlo;       // [cols][cols] f16: H 2^t, low term
  size_t hscale;    // f32[2]: 2^-t, max |H|
  size_t rmat;      // [G][g][g] f32: R_i = L_i^T, row-major
  size_t rph;       // [G][g][g] f16: R_i row c scaled by 2^t_c, high term
  size_t rpl;       // [G][g][g] f16: low term
  size_t rrow;      // [G][g] f32: 2^-t_c of the R rows
  size_t mhi;       // [cols][cols] f16: M = blockdiag(L_i^{-1}) H, row n scaled by 2^t_n, high term
  size_t mlo;       // [cols][cols] f16: low term
  size_t mrow;      // [cols] f32: 2^-t_n
  size_t mmax;      // [cols] f32: row maxima of M (prep scratch)
  size_t wrow;      // [rows] f32: 2^-t_row of W's fp16 planes (prepare; the planes
                    // themselves occupy p's memory until the first sweep)
  size_t wh;        // [rows][cols] f32: W H
  size_t tm;        // [rows][cols] f32: T = W M^T (the residual product of W alone)
  size_t rw;        // [rows][cols] f32: W_i L_i per group (the objective's part of W alone)
  size_t cz;        // [rows][cols] f16: q - z, exact, by layer row (kept with the codes)
  size_t gram;      // [rows][G][G] f32: upper triangle of B^T B
  size_t rhs;       // [rows][G] f64: the scale systems' right-hand sides c_i^T (W H)_i
  size_t p;         // [rows][cols] f32: (W - What) H
  size_t dq;        // [rows][cols] f16: q_new - q_old of accepted groups, 0 elsewhere
  size_t plist;     // [kSubLists][cap] i32: rows that accepted a change in the last panel (any order)
  size_t pcount;    // [panels][kSubLists] u32 kCtrStride apart: lengths of the sub-lists
  size_t objpart;   // [rows][ceil(cols/64)] f64: partial row objectives
  size_t lcur;      // [rows] f64
  size_t lprev;     // [rows] f64
  size_t active;    // [rows] u8
  size_t stopat;    // [rows] i32: iteration at which the row stopped, 0 while it has not
  size_t glist;     // [G][kSubLists][cap] i32: rows that changed group i (incremental Gram build)
  size_t gcount;    // [G][kSubLists] u32 kCtrStride apart: lengths of the sub-lists
  size_t gpre;      // [G][kSubLists + 1] i32: their exclusive prefix sums (last: list length)
  size_t gctl;      // GramCtl
  size_t sctl;      // SweepCtl
  size_t rowmap;    // [rows] i32: row of each position of the sweep (rows still active, ascending)
  size_t counters;  // Counters
  size_t hist;      // [64] SweepRecord
  size_t flags;     // Flags
  size_t total;
};

Layout make_layout(int rows, int cols, int g);

// ---- launchers (each returns hipGetLastError() of its launches) ----

hipError_t launch_chol_groups(hipStream_t st, int cols, int g, const float* H, char* ws,
                              const Layout& lay);
// R_i rows as two fp16 terms with per-row power-of-two scales (rph, rpl, rrow).
hipError_t launch_split_r(hipStream_t st, int cols, int g, char* ws, const Layout& lay);

// C = A H with A = W (quant == false) or A = W - What (quant == true).  When
// objpart is non-null, objpart[row][col/64] receives sum over the 64-column
// slice of A(row, c) * C(row, c) in fp64.  C may be null (objective only).
hipError_t launch_gemm_ah(hipStream_t st, int rows, int cols, int g, bool quant,
                          const float* W, const uint8_t* codes, const float* scales,
                          const int32_t* zeros, const float* H, float* C, double* objpart);

hipError_t launch_split_h(hipStream_t st, int cols, const float* H, char* ws, const Layout& lay);
// M = blockdiag(L_i^{-1}) H as two fp16 planes with per-row scales (after
// launch_chol_groups; uses the H planes as scratch, so call launch_split_h after).
hipError_t launch_split_m(hipStream_t st, int cols, int g, const float* H, char* ws,
                          const Layout& lay);

// The layer's constant parts of the per-sweep products (jarq_prepare), from
// W as two fp16 planes (whi, wlo with row scales 2^-t in wrow, all rows):
// T = W M^T into lay.tm (three products, sgemm.hip) and RW = W_i L_i per
// group into lay.rw (objective.hip).
hipError_t launch_split_w(hipStream_t st, int rows, int cols, const float* W, _Float16* whi,
                          _Float16* wlo, float* wrow_inv);
hipError_t launch_wm_product(hipStream_t st, int rows, int cols, const char* ws,
                             const Layout& lay, const _Float16* whi, const _Float16* wlo,
                             const float* wrow_inv);
hipError_t launch_rw_product(hipStream_t st, int rows, int cols, int g, const char* ws,
                             const Layout& lay, const _Float16* whi, const _Float16* wlo,
                             const float* wrow_inv);
// cz = q - z as fp16 for all rows (kept in step with the codes by the code update).
hipError_t launch_codes_cz(hipStream_t st, int rows, int cols, int g, const uint8_t* codes,
                           const int32_t* zeros, _Float16* cz);
// U = T - What M^T from the exact codes (cz) and the scales, layer rows
// through rowmap, U by position (sgemm.hip).  ev_start / ev_stop (nullable):
// events that take the kernel's own start and end times (no marker of their
// own in the stream).
hipError_t launch_resid(hipStream_t st, int rows, int cols, int g, const char* ws,
                        const Layout& lay, const float* scales, float* U, const int32_t* rowmap,
                        const int* n_dev, hipEvent_t ev_start = nullptr,
                        hipEvent_t ev_stop = nullptr);
// Per position and group, (R_i e_i) . U_i = e_i^T (H e)_i (fp64) into
// objpart[position][group], from RW, cz and the scales (layer rows via rowmap).
hipError_t launch_group_objective(hipStream_t st, int rows, int cols, int g, const char* ws,
                                  const Layout& lay, const float* scales, const float* U,
                                  double* objpart, const int32_t* rowmap, const int* n_dev);

// Row counts on the device: every per-row kernel of a sweep takes the number
// of positions n as `rows` (the most it may be, which sizes the grid) and,
// when n_dev is not null, reads the current n from *n_dev; work-groups past it
// return at once.

// Upper triangles of the grouped Gram matrices from the fp16 planes of H,
// stored by layer row.  incremental: build from the rows listed per changed
// group when that is cheaper and the matrices of the last sweep are complete
// (the code update lists the rows it changed per group in glist / gcount;
// GramCtl in the workspace).
hipError_t launch_gram(hipStream_t st, int rows, int cols, int g, const char* ws,
                       const Layout& lay, const uint8_t* codes, const int32_t* zeros,
                       float* gram, const int32_t* rowmap, const int* n_dev, bool incremental);

// The scale solves.  Right-hand sides come from rhs_cache ([layer rows][G]
// fp64) when rctl says the matrices and right-hand sides of the last sweep
// are complete (rctl->valid), else from W H and the codes (then stored there).
hipError_t launch_solve(hipStream_t st, int rows, int cols, int g, const float* gram,
                        const float* wh, const uint8_t* codes, const int32_t* zeros,
                        double* rhs_cache, const GramCtl* rctl,
                        float* scales, const uint8_t* active, Counters* cnt, Flags* flags,
                        float lam, float rcond, int accept, const int32_t* rowmap,
                        const int* n_dev);

// Code update of the groups [i0, i1) (one panel).  The positions of the rows
// that accepted a change go to the panel's row list (plist, pcount).  With
// glist not null, every row whose group i the update changed is appended (as
// its layer row, in any order) to group i's list (glist, gcount); the
// counters are zeroed before the sweep's first panel.  list_cap =
// sublist_cap(rows of the layer).
hipError_t launch_babai(hipStream_t st, int rows, int cols, int g, int bits, int i0, int i1,
                        const float* P, const char* ws, const Layout& lay, uint8_t* codes,
                        const float* scales, const int32_t* zeros, const uint8_t* active,
                        uint8_t* cand, uint8_t* decision, Counters* cnt, const int32_t* rowmap,
                        const int* n_dev, int32_t* glist, uint32_t* gcount, int list_cap);

// Work-group barrier for LDS only: waits for this wave's LDS operations,
// not for its outstanding global loads (a __syncthreads would, which drains
// any prefetch in flight).  The empty asm statements keep the compiler from
// moving memory accesses across it.
constexpr int kVmcnt0 = 0x0F70;  // s_waitcnt operand: vmcnt(0), lgkmcnt and expcnt at their maximum

__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maximum
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Early stopping shrinks the set of rows a sweep works on.  Per-sweep
// intermediates (U, objective partials, dq, the panel row lists) are indexed
// by position p < n in the sweep's row list; the layer's state (W, codes,
// q - z, scales, zeros, W H, the cached scale right-hand sides, the Gram
// matrices, which persist across sweeps, and the stopping state) by row.  The
// list is null while every row takes part (position = row).
__device__ __forceinline__ int map_row(const int32_t* rowmap, int p) {
  return rowmap != nullptr ? rowmap[p] : p;
}

// rowmap[0 .. n) = the rows with active[r] != 0, ascending, and sctl->n = n
// (one work-group).
hipError_t launch_compact_rows(hipStream_t st, int rows, const uint8_t* active, int32_t* rowmap,
                               SweepCtl* sctl);

// Groups per panel of the code update (512 columns, at most 16 groups).
// R~ columns of a group for the back substitution (written by chol.hip, read
// by babai.hip).  The 16 lanes of a row own positions j + 16 t, t < NT = g /
// 16, and read a column in chunks of W = min(4, NT) positions per lane, one
// W-float access each (chunk c: t = W c .. W c + W - 1, lane-contiguous, 16 W
// floats).  Step l reads only t <= l / 16, so column l keeps its first
// (l / 16) / W + 1 chunks; columns follow one another.  With B = 16 W, column
// l in band b = l / B has b + 1 chunks and starts at
// 16 W (B b (b - 1) / 2 + b (l - B b) + l) floats.
template <int g>
struct RcolLayout {
  static constexpr int NT = g / 16;
  static constexpr int W = NT < 4 ? NT : 4;
  static constexpr int B = 16 * W;
  __host__ __device__ static constexpr int chunks(int l) { return l / B + 1; }
  __host__ __device__ static constexpr int offset(int l) {
    return 16 * W * (B * (l / B) * (l / B - 1) / 2 + (l / B) * (l - B * (l / B)) + l);
  }
  static constexpr int total = 16 * W * (B * (g / B) * (g / B - 1) / 2 + g);
};

constexpr int kMaxPanelGroups = 16;
constexpr int panel_groups_of(int g) { return 512 / g < kMaxPanelGroups ? 512 / g : kMaxPanelGroups; }
int panel_groups(int g);

// P(:, c1:) -= the accepted changes of the groups in columns [c0, c1) (the
// panel's rows listed by the code update in the panel's plist / pcount
// sub-lists; rows = the layer's rows).
hipError_t launch_panel_update(hipStream_t st, int rows, int cols, int g, int c0, int c1,
                               const char* ws, const Layout& lay, const float* scales, float* P,
                               const int32_t* rowmap);

hipError_t launch_row_objective(hipStream_t st, int rows, int nt, const double* objpart,
                                double* out);

// Also zeroes the counters zero_ctr[t * kCtrStride], t < nzero, and likewise
// zero_ctr2 (the code update's list counters) before any row is handled.
// A row that stops gets stopat[row] = sweep.
hipError_t launch_stop_check(hipStream_t st, int rows, int nt, const double* objpart,
                             double* lcur, double* lprev, uint8_t* active, int32_t* stopat,
                             int sweep, float tau, const int32_t* rowmap, uint32_t* zero_ctr,
                             int nzero, uint32_t* zero_ctr2, int nzero2, const int* n_dev);

hipError_t launch_fill_u8(hipStream_t st, uint8_t* p, size_t n, uint8_t v);
hipError_t launch_zero_bytes(hipStream_t st, void* p, size_t n);

// Also: gram->valid = 1 (every active row's matrix now exists),
// sctl->started counted, gpre = the prefix sums of the Gram row sub-lists.
hipError_t launch_record_sweep(hipStream_t st, int rows, const double* lcur,
                               const uint8_t* active, Counters* cnt, SweepRecord* rec,
                               SweepCtl* sctl, GramCtl* gctl, const uint32_t* gcount,
                               int32_t* gpre, int G);

hipError_t launch_validate(hipStream_t st, int rows, int cols, int g, int bits,
                           const uint8_t* codes, const int32_t* zeros, Flags* flags);

// Per-layer set-up from calibration inputs and the round-to-nearest host.
hipError_t launch_hessian_update(hipStream_t st, const float* X, int m, int d, double alpha,
                                 double* Hacc);
hipError_t launch_hessian_update_bf16(hipStream_t st, const void* X, int m, int d, double alpha,
                                      double* Hacc);
hipError_t launch_hessian_finalize(hipStream_t st, const double* Hacc, int d, double damp,
                                   double nu2, float* H);
hipError_t launch_rtn(hipStream_t st, const float* W, int rows, int cols, int g, int bits,
                      uint8_t* codes, float* scales, int32_t* zeros);

// Dense fp64 building blocks (linalg.hip).
hipError_t launch_gemm_nt_f64(hipStream_t st, bool lower, int M, int N, int K, int kslice,
                              double alpha, const double* A, long long lda, const double* B,
                              long long ldb, double* C, long long ldc, long long cz,
                              bool accumulate);
// C_z = alpha A B over k-slice z (B k-major [K][N]), slice z stored at C + z cz.
hipError_t launch_gemm_nn_f64_sliced(hipStream_t st, int M, int N, int K, int kslice,
                                     double alpha, const double* A, long long lda,
                                     const double* B, long long ldb, double* C, long long ldc,
                                     long long cz);
hipError_t launch_gemm_nn_f64(hipStream_t st, int M, int N, int K, double alpha, const double* A,
                              long long lda, const double* B, long long ldb, double* C,
                              long long ldc, bool accumulate);
hipError_t launch_potrf_f64(hipStream_t st, double* A, int d, long long lda, double* Linv,
                            int* flag, bool keep_inverses);
hipError_t launch_copy_lower(hipStream_t st, const float* H, int d, bool reverse, double* C);
hipError_t launch_antitranspose_lower(hipStream_t st, const double* C, int d, double* M);

// Propagation-corrected target (setup.hip, qep.hip).
hipError_t launch_cross_update(hipStream_t st, const float* Xq, const float* X, int m, int d,
                               double alpha, double* Dacc);
size_t qep_workspace_bytes(int rows, int cols);
hipError_t launch_qep_correct(hipStream_t st, int rows, int cols, const float* W, const float* H,
                              const double* D, double mu, float* Wcorr, char* ws, int** flag_out);

// After refinement (post.hip).
hipError_t launch_canonicalize(hipStream_t st, int rows, int cols, int g, int bits,
                               uint8_t* codes, float* scales, int32_t* zeros);
hipError_t launch_dequantize(hipStream_t st, int rows, int cols, int g, const uint8_t* codes,
                             const float* scales, const int32_t* zeros, const int32_t* perm,
                             int dtype, void* out);
hipError_t launch_pack(hipStream_t st, int rows, int cols, int bits, const uint8_t* codes,
                       uint32_t* packed);
hipError_t launch_unpack(hipStream_t st, int rows, int cols, int bits, const uint32_t* packed,
                         uint8_t* codes);
hipError_t launch_act_order(hipStream_t st, const float* H, int d, int32_t* perm);
hipError_t launch_permute(hipStream_t st, int rows, int d, const int32_t* perm, const float* W,
                          const float* H, float* Wp, float* Hp);

// GPTQ-style host (gptq.hip).
size_t gptq_workspace_bytes(int rows, int cols, int g);
hipError_t launch_gptq(hipStream_t st, int rows, int cols, int g, int bits, const float* W,
                       const float* H, char* ws, uint8_t* codes, float* scales, int32_t* zeros,
                       int** flag_out);

}  // namespace jarq
