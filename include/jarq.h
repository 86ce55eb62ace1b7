/*
 * jarq.h - C ABI of the JARQ refinement sweep for one quantized linear layer
 * on an AMD Instinct MI355X (gfx950).
 *
 * Problem (paper Sec. 3.1-3.2).  A layer with weights W (rows = output
 * channels, cols = input channels) is held in group-wise uniform form,
 * eq. (1): row j, group i is s_ij * (q_ij - z_ij), with g consecutive weights
 * per group, one signed fp32 scale and one integer zero point per group, and
 * b-bit codes q in {0, ..., 2^b - 1}.  Refinement changes the scales S and
 * the codes Q and never the bit width, the groups or the zero points Z
 * (Sec. 3.1).  It minimises the layer objective of eq. (4) written with the
 * calibration Hessian H = X^T X + nu^2 I:
 *     F_j = (w_j - what_j)^T H (w_j - what_j),   F = sum_j F_j.
 *
 * One sweep (Sec. 3.3, App. E.2) is, for every row independently:
 *   (b) joint scale update: solve the G x G normal equations eq. (6),
 *       B_j^T B_j s = B_j^T y_j, with entries c_i^T H_ih c_h and c_i^T (H w)_i
 *       (c_i = q_i - z_i), adding 1e-4 I when the Gram matrix is near singular;
 *   (a) residual product P = (W - What) H at the new scales and the previous
 *       codes, and L_j = sum_c E_jc P_jc (the objective right after the scale
 *       update, used for early stopping);
 *   (c) Gauss-Seidel code update over the groups i = 1..G (eq. (7)): one
 *       bounded Babai nearest-plane proposal per group on the upper Cholesky
 *       factor R_i of H_ii (eqs. (9)-(10)), kept only if it strictly lowers
 *       F_j (eq. (8)).  Groups with |s_ij| <= 2^-23 keep their codes.
 *
 * Conventions for every entry point:
 *   - Pointers are device pointers unless marked [host].  Arrays are dense
 *     row-major.  The caller owns every buffer; the library allocates no
 *     device memory and keeps no global state.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All device work is enqueued on it in order.
 *   - W, H, scales and codes must be 16-byte aligned,
 *     the workspace 256-byte aligned.
 *   - Argument errors return JARQ_EINVAL before anything is enqueued; the
 *     outputs are then untouched.
 *   - The workspace of a jarq_prepare call is reused by the later calls on
 *     the same layer; calls that share a workspace must not overlap.
 *   - Zero points must satisfy |z| <= 1024 (codes minus zero points are held
 *     exactly in fp16 on the matrix cores); jarq_sweeps and jarq_refine check
 *     this, the stage entry points assume it.
 */
#ifndef JARQ_H_
#define JARQ_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define JARQ_ABI_VERSION 9
/* Timed stages of a sweep (jarq_stats.stage_ms columns): 0 Gram matrices,
 * 1 scale solve, 2 residual product U = E M^T (formed as W M^T - What M^T
 * from the codes), 3 row objectives and stopping test, 4 code update: the
 * Babai kernels (one per panel of groups), 5 code update: the panel updates
 * between them.  Stages 4 and 5 interleave; each of their launches is timed
 * on its own. */
#define JARQ_NUM_STAGES 6
#define JARQ_MAX_RECORDED_SWEEPS 64

typedef enum jarq_status {
  JARQ_OK = 0,
  JARQ_EINVAL = 1,        /* bad argument (shape, pointer, alignment, code range) */
  JARQ_ENOT_SPD = 2,      /* some diagonal block H_ii is not positive definite (eq. (9)) */
  JARQ_ESCALE_SOLVE = 3,  /* a row's Gram matrix failed Cholesky after the ridge (App. E.2) */
  JARQ_EHIP = 4,          /* a HIP runtime call or kernel launch failed */
  JARQ_EWORKSPACE = 5,    /* workspace missing, too small or misaligned */
  JARQ_ESTATIC_LIMIT = 6  /* jarq_refine_static: the layer needs more than
                             JARQ_STATIC_WORKSPACE_BYTES of workspace */
} jarq_status;

/* Problem description.  Sizes are those of eq. (1). */
typedef struct jarq_params {
  int32_t rows;          /* d_out >= 1: output channels = rows of W */
  int32_t cols;          /* d_in: columns of W and order of H; a multiple of group_size */
  int32_t group_size;    /* g in {32, 64, 128} */
  int32_t bits;          /* b in [1, 8] */
  int32_t sweeps;        /* iteration budget K in [0, 4096]; K = 0 leaves the host state */
  float tau;             /* early-stopping threshold of App. E.2 (1e-5 there); < 0 disables */
  float ridge_lambda;    /* lambda added on a near-singular Gram matrix (1e-4, App. E.2) */
  float ridge_rcond;     /* r_cond of the near-singularity test (1e-10, App. E.2) */
  int32_t ridge_accept;  /* 0: keep every ridge solution (App. E.2); 1: keep a ridge solution
                            only if it does not increase F_j, else the row keeps its
                            previous scales (the remark on ridge acceptance, App. G.5) */
} jarq_params;

/* Filled by jarq_sweeps / jarq_refine when a stats pointer is given [host].
 * Per-sweep arrays hold the first JARQ_MAX_RECORDED_SWEEPS sweeps.
 * stage_mask is read, not written: bit s selects stage s for timing (0 = all
 * stages).  Each timed stage costs a pair of HIP events per sweep, and every
 * event leaves the GPU idle for a few microseconds between kernels; stages not
 * selected report 0 ms. */
typedef struct jarq_stats {
  uint32_t stage_mask;               /* [in] stages to time, bit s = stage s; 0 = all */
  int32_t sweeps_run;                /* sweeps started (a sweep in which every row had stopped is not run) */
  int32_t rows_active_end;           /* rows still active after the last sweep */
  double objective_after_scales[JARQ_MAX_RECORDED_SWEEPS];  /* sum_j L_j, fp64 */
  int64_t accepted_groups[JARQ_MAX_RECORDED_SWEEPS];
  int64_t codes_changed[JARQ_MAX_RECORDED_SWEEPS];
  int64_t skipped_groups[JARQ_MAX_RECORDED_SWEEPS];          /* |s| <= 2^-23 */
  int32_t ridge_rows[JARQ_MAX_RECORDED_SWEEPS];              /* stabilised scale solves */
  int32_t rows_active[JARQ_MAX_RECORDED_SWEEPS];             /* rows that ran the code update */
  int64_t correction_blocks[JARQ_MAX_RECORDED_SWEEPS];      /* 16-row x g x g correction products run */
  int32_t gram_listed[JARQ_MAX_RECORDED_SWEEPS];            /* 1: only the Gram entries of groups the
                                                               last code update changed were formed */
  float stage_ms[JARQ_MAX_RECORDED_SWEEPS][JARQ_NUM_STAGES]; /* HIP-event ms per stage, see JARQ_NUM_STAGES */
  float prep_ms;                                             /* jarq_refine only */
} jarq_stats;

/* Bytes of device workspace needed for `p`; 0 if `p` is invalid. */
size_t jarq_workspace_bytes(const jarq_params* p);

/*
 * Per-layer set-up (eq. (9) and the right-hand-side shortcut of App. G.8):
 * factor every diagonal block H_ii = R_i^T R_i (fp64 Cholesky), store R_i,
 * R_i^{-1} and 1/diag(R_i) in fp32, and compute WH = W H in fp32.  Synchronises
 * `stream` and returns JARQ_ENOT_SPD if a block is not positive definite.
 * W [rows][cols] fp32; H [cols][cols] fp32, symmetric, full storage.
 */
jarq_status jarq_prepare(const jarq_params* p, const float* W, const float* H,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Scale update (b) for every row from the given codes (eqs. (5)-(6), App. E.2),
 * on a prepared workspace.  scales [rows][G] fp32 are overwritten; codes
 * [rows][cols] uint8 and zeros [rows][G] int32 are read.  Asynchronous; a row
 * whose solve fails after the ridge keeps its previous scales and is counted
 * in the workspace (reported by jarq_sweeps / jarq_refine).
 */
jarq_status jarq_scale_step(const jarq_params* p, const float* H, const uint8_t* codes,
                            float* scales, const int32_t* zeros,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * Residual product (a) and Gauss-Seidel code update (c) at the given scales,
 * on a prepared workspace.  codes [rows][cols] are updated in place.
 * Optional trace outputs (NULL to skip), written for every row and group:
 *   cand     [rows][cols] uint8: the Babai proposal of eq. (10) for the group
 *            (the unchanged codes where the group was skipped);
 *   decision [rows][G] uint8: 0 rejected, 1 accepted, 2 skipped (|s| <= 2^-23).
 * Asynchronous.
 */
jarq_status jarq_code_step(const jarq_params* p, const float* W, const float* H,
                           uint8_t* codes, const float* scales, const int32_t* zeros,
                           void* workspace, size_t workspace_bytes, void* stream,
                           uint8_t* cand, uint8_t* decision);

/*
 * K = p->sweeps sweeps (b) -> (a) -> [early stop] -> (c) on a prepared
 * workspace, starting with every row active.  codes and scales are updated
 * in place; zeros are read only.  Checks first that every code is in
 * [0, 2^b - 1] and every |zero point| <= 1024 (JARQ_EINVAL otherwise, nothing
 * changed).  Synchronises `stream` before returning.  `stats` [host] may be
 * NULL.  Returns JARQ_ESCALE_SOLVE if any row's solve failed after the ridge
 * (that row keeps its previous scales).
 * From the second sweep on, the Gram matrices of (b) are formed only for the
 * groups whose codes the previous sweep changed when that is cheaper (entry
 * (a, h) depends on the codes of groups a and h alone, eq. (5)); the entries
 * are bit-identical to a full build.  With early stopping the set of active
 * rows stays on the device; every fourth sweep its size is copied behind that
 * sweep into pinned host memory (allocated and freed by the call), and the
 * host stops launching once a copy that has landed shows no row left (the
 * stream is never drained for it).
 */
jarq_status jarq_sweeps(const jarq_params* p, const float* W, const float* H,
                        uint8_t* codes, float* scales, const int32_t* zeros,
                        void* workspace, size_t workspace_bytes, void* stream,
                        jarq_stats* stats);

/*
 * Per-row outcome of the early-stopping rule (App. E.2, eq. (strict_stopping))
 * in the last jarq_sweeps / jarq_refine call on this workspace: stop_sweep
 * [rows] int32 (device, 4-byte aligned) receives, for every row, the
 * iteration k >= 2 whose stopping test stopped it (the row kept that
 * iteration's scales and skipped its code update), or 0 if the row ran every
 * iteration (always 0 when tau < 0).  `p` must describe the same layer as that
 * call.  Asynchronous (a device-to-device copy on `stream`).
 */
jarq_status jarq_stop_sweeps(const jarq_params* p, const void* workspace, size_t workspace_bytes,
                             int32_t* stop_sweep, void* stream);

/* jarq_prepare followed by jarq_sweeps. */
jarq_status jarq_refine(const jarq_params* p, const float* W, const float* H,
                        uint8_t* codes, float* scales, const int32_t* zeros,
                        void* workspace, size_t workspace_bytes, void* stream,
                        jarq_stats* stats);

/*
 * jarq_refine without a workspace argument, for callers that cannot allocate
 * device memory (code under graph capture, tight serving loops, harnesses
 * that forbid allocation): the same kernels run on a workspace that the
 * library holds in a static device array of JARQ_STATIC_WORKSPACE_BYTES
 * (512 MiB; enough for a 4096 x 4096 layer at g = 128), created on each GPU
 * the library runs on and held until the process ends.  The call allocates
 * nothing: no hipMalloc, no hipFree, no HIP event, no pinned host memory (with
 * early stopping its fourth-sweep look at the active count is a blocking
 * copy instead).  Layers whose
 * jarq_workspace_bytes exceeds the limit are rejected with
 * JARQ_ESTATIC_LIMIT before anything is enqueued.  Results are those of
 * jarq_refine on the same inputs; stats (nullable) is filled the same way
 * except that no stage is timed (stage_ms and prep_ms are 0).  Every call on
 * one GPU uses that GPU's single array, which keeps the previous call's
 * contents (each call overwrites what it reads): calls that overlap on one
 * GPU, from any stream or thread, race and must be serialised by the caller.
 * Synchronises `stream`.
 */
#define JARQ_STATIC_WORKSPACE_BYTES (512u << 20)
jarq_status jarq_refine_static(const jarq_params* p, const float* W, const float* H,
                               uint8_t* codes, float* scales, const int32_t* zeros, void* stream,
                               jarq_stats* stats);

/*
 * Layer objective eq. (4) in the Hessian form for the given state:
 * row_objective [rows] fp64 receives F_j = (w_j - what_j)^T H (w_j - what_j),
 * with H (w_j - what_j) accumulated in fp32 and the dot product in fp64.
 * Needs a workspace sized for `p` (it need not be prepared).  Asynchronous.
 */
jarq_status jarq_objective(const jarq_params* p, const float* W, const float* H,
                           const uint8_t* codes, const float* scales, const int32_t* zeros,
                           void* workspace, size_t workspace_bytes, void* stream,
                           double* row_objective);

/*
 * Per-layer set-up from calibration inputs: the Hessian of the layer
 * objective, H = X~^T X~ + nu^2 I (App. E.1: the Gram matrix of the stacked
 * design A = [X~; nu I]), accumulated over chunks of tokens.
 *
 * jarq_hessian_accumulate adds alpha X^T X to Hacc, for X [m][d] fp32
 * (m tokens of d input channels, row-major, 16-byte aligned, d a multiple of
 * 4, 1 <= d <= 32768, 0 <= m < 2^31; m = 0 does nothing and X may then be
 * NULL) and Hacc [d][d] fp64
 * in full symmetric storage (8-byte aligned; the caller zeroes it before the
 * first chunk).  Products are rounded to fp32 and summed in fp32 over at most
 * 256 tokens; those partial sums are added in fp64.  Hacc stays exactly
 * symmetric.  Calls on one Hacc must be ordered (same stream).  Asynchronous.
 */
jarq_status jarq_hessian_accumulate(const float* X, int64_t m, int32_t d, double alpha,
                                    double* Hacc, void* stream);

/*
 * The same accumulation for X [m][d] in bf16 (the 16-bit brain float format,
 * passed as raw 16-bit words; 16-byte aligned, d a multiple of 8, the other
 * limits as above).  Products of bf16 values are exact in fp32; they are
 * summed in fp32 over at most 256 tokens and those partial sums in fp64.
 */
jarq_status jarq_hessian_accumulate_bf16(const void* X, int64_t m, int32_t d, double alpha,
                                         double* Hacc, void* stream);

/*
 * H [d][d] fp32 (16-byte aligned) = Hacc + (damp * mean(diag Hacc) + nu2) I,
 * rounded once to fp32.  damp = 0, nu2 = nu^2 is App. E.1's regularised
 * Hessian; damp > 0 adds the relative diagonal damping used by GPTQ-style
 * pipelines.  damp and nu2 must be finite and >= 0.  H and Hacc must not
 * overlap.  Asynchronous.
 */
jarq_status jarq_hessian_finalize(const double* Hacc, int32_t d, double damp, double nu2,
                                  float* H, void* stream);

/*
 * Round-to-nearest host state (S0, Q0, Z) of eq. (1) for W [rows][cols] fp32
 * (App. A.1: asymmetric group-wise RTN; the min/max reading): per group,
 * lo = min(min w, 0), hi = max(max w, 0), s = (hi - lo)/(2^b - 1) (s = 1 if
 * hi == lo) rounded to fp32, z = clip(rint(-lo/s), 0, 2^b - 1) and
 * q = clip(rint(w/s) + z, 0, 2^b - 1), z and q from the stored s in fp64.
 * Uses rows, cols, group_size and bits of `p` (which must be valid as a whole).
 * codes [rows][cols] uint8 (16-byte aligned), scales [rows][G] fp32 and
 * zeros [rows][G] int32 are written.  Asynchronous.
 */
jarq_status jarq_rtn(const jarq_params* p, const float* W, uint8_t* codes, float* scales,
                     int32_t* zeros, void* stream);

/*
 * Propagation-corrected target (App. E.5, eqs. (mu-target), (w-corr)).  With
 * X the inputs a layer receives in the full-precision model and X~ those it
 * receives after the preceding layers were quantized, the mixed target
 * (1 - mu) X W + mu X~ W (mu in [0, 1]; mu = 1 is the main target) turns the
 * refinement problem into the main one with W replaced by
 *     W_corr = W + (1 - mu) (W D^T) H^{-1},   D = X~^T (X - X~)
 * (rows = output channels; H = X~^T X~ + nu^2 I from jarq_hessian_* on X~),
 * plus a constant.  Refine W_corr with the usual entry points.
 *
 * jarq_cross_accumulate adds alpha X~^T (X - X~) to Dacc [d][d] fp64 (not
 * symmetric), for Xq = X~ and X [m][d] fp32 (same tokens, same layout and
 * limits as jarq_hessian_accumulate; X - X~ is formed in fp32, products and
 * partial sums as there).  Use the alpha of the Hessian so that D and H share
 * their scale.  Asynchronous.
 */
jarq_status jarq_cross_accumulate(const float* Xq, const float* X, int64_t m, int32_t d,
                                  double alpha, double* Dacc, void* stream);

/*
 * Wcorr [rows][cols] fp32 (16-byte aligned) = W + (1 - mu) (W D^T) H^{-1} for
 * W [rows][cols] fp32, H [cols][cols] fp32 (symmetric, full storage, positive
 * definite; only its lower part is read) and D [cols][cols] fp64, computed in
 * fp64 (Cholesky of H, two blocked triangular solves) and rounded once.  Uses
 * rows, cols of `p` (which must be valid as a whole).  The workspace
 * (256-byte aligned, jarq_qep_workspace_bytes(p) bytes) is used only during
 * the call.  Synchronises `stream`; JARQ_ENOT_SPD if H is not positive
 * definite (Wcorr is then unspecified).
 */
size_t jarq_qep_workspace_bytes(const jarq_params* p);
jarq_status jarq_qep_correct(const jarq_params* p, const float* W, const float* H,
                             const double* D, double mu, float* Wcorr, void* workspace,
                             size_t workspace_bytes, void* stream);

/*
 * GPTQ-style host state (S0, Q0, Z) for W [rows][cols] fp32 and H [cols][cols]
 * fp32 (symmetric, full storage, positive definite): App. A.1 uses GPTQ as a
 * host; its sequential error compensation is the nearest-plane relation of
 * App. G.7.  Columns are visited in their natural order (no activation
 * ordering, so groups stay contiguous).  At the first column of each group the
 * group's grid is fixed by the min/max rule of jarq_rtn on the weights
 * compensated for every earlier column; each column is then rounded on that
 * grid after compensation for every earlier column, including those of its own
 * group.  All arithmetic is fp64 (H is factored as J H J = C C^T, J the
 * order reversal).  codes (16-byte aligned), scales and zeros as for
 * jarq_rtn.  The workspace (256-byte aligned, jarq_gptq_workspace_bytes(p)
 * bytes: two cols x cols fp64 matrices, rows x cols fp64 errors and partial
 * products) is used only during the call.  Synchronises `stream`; returns
 * JARQ_ENOT_SPD if H is not positive definite (the outputs are then
 * unspecified).
 */
size_t jarq_gptq_workspace_bytes(const jarq_params* p);
jarq_status jarq_gptq(const jarq_params* p, const float* W, const float* H, uint8_t* codes,
                      float* scales, int32_t* zeros, void* workspace, size_t workspace_bytes,
                      void* stream);

/*
 * After refinement.
 *
 * jarq_canonicalize (App. E.3, eq. (canonicalization)): every group with
 * s < 0 becomes s' = -s, q' = (2^b - 1) - q, z' = (2^b - 1) - z, which
 * represents the same weights (eq. (canonicalization_equivalence)) with
 * codes in the same range; groups with s >= 0 are left alone.  This changes
 * Z, so it runs only after refinement, for formats that need positive
 * scales.  In place; codes 16-byte aligned.  Asynchronous.
 */
jarq_status jarq_canonicalize(const jarq_params* p, uint8_t* codes, float* scales,
                              int32_t* zeros, void* stream);

/* Output dtypes of jarq_dequantize. */
#define JARQ_F32 0
#define JARQ_F16 1
#define JARQ_BF16 2

/*
 * Dequantized weights out [rows][cols] = s (q - z) of eq. (1), computed in fp32
 * and rounded once (to nearest even) to dtype JARQ_F32, JARQ_F16 or JARQ_BF16
 * (the model's floating-point dtype, App. A.1).  perm (nullable, [cols]
 * int32): the refined layer lives in permuted input coordinates, position k
 * being original column perm[k] (activation ordering; App. A.1 and E.2 restore
 * the original coordinates on write-back); out is then in the original order.
 * perm must be a permutation of 0..cols-1 (entries outside that range are
 * skipped).  Asynchronous.
 */
jarq_status jarq_dequantize(const jarq_params* p, const uint8_t* codes, const float* scales,
                            const int32_t* zeros, const int32_t* perm, int32_t dtype, void* out,
                            void* stream);

/*
 * b-bit codes packed into 32-bit words: row r is one little-endian bit stream
 * in which code k occupies bits [k b, k b + b); stream bit t is bit t % 32 of
 * word t / 32 of the row; each row starts on a new word, so packed is
 * [rows][ceil(cols b / 32)] uint32 (bits past the last code are 0).
 * jarq_unpack_codes is the inverse.  Asynchronous.
 */
jarq_status jarq_pack_codes(const jarq_params* p, const uint8_t* codes, uint32_t* packed,
                            void* stream);
jarq_status jarq_unpack_codes(const jarq_params* p, const uint32_t* packed, uint8_t* codes,
                              void* stream);

/*
 * Activation ordering of a GPTQ host (App. A.1): perm [d] int32 lists the
 * input channels by decreasing diag(H), ties by increasing index (H [d][d]
 * fp32, diagonal not NaN).  jarq_permute gathers the layer into that order:
 * Wp[r][k] = W[r][perm[k]] ([rows][cols]) and Hp[k][l] = H[perm[k]][perm[l]]
 * ([cols][cols]), with rows and cols from `p`.  Refinement then runs on
 * (Wp, Hp) with groups of consecutive permuted columns, and jarq_dequantize
 * with the same perm writes the weights back in the original order.
 * Asynchronous.
 */
jarq_status jarq_act_order(const float* H, int32_t d, int32_t* perm, void* stream);
jarq_status jarq_permute(const jarq_params* p, const int32_t* perm, const float* W, const float* H,
                         float* Wp, float* Hp, void* stream);

/*
 * Measurement aid (not part of refinement): a kernel that moves a known
 * number of bytes through the local data share (LDS), used to scale LDS
 * profiler counters to bytes and to see the rate the LDS sustains for a
 * streaming reader.  `workgroups` work-groups of 256 threads each write 32 KB
 * of LDS once and read it `passes` times (16-byte reads, no bank conflict),
 * then write one float per thread to out [workgroups * 256] (device, 4-byte
 * aligned).  Returns the LDS bytes moved (writes + reads), or -1 on a bad
 * argument or a failed launch.  Asynchronous.
 */
int64_t jarq_lds_probe(int32_t workgroups, int32_t passes, float* out, void* stream);

/* Static, NUL-terminated description of a status code. */
const char* jarq_status_string(jarq_status s);

/* JARQ_ABI_VERSION of the built library. */
int32_t jarq_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* JARQ_H_ */
