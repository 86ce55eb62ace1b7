// C ABI of libjarq (declared in include/jarq.h): argument checks, workspace
// layout, and the stream-ordered sequence of kernels of one refinement run.
#include <math.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "jarq.h"
#include "jarq_internal.h"

namespace jarq {

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
// Panels of the code update (each has kSubLists row counters).
static int pcount_words(int cols, int g) {
  const int pg = panel_groups_of(g);
  return (cols / g + pg - 1) / pg;
}

Layout make_layout(int rows, int cols, int g) {
  Layout L{};
  const size_t R = (size_t)rows, C = (size_t)cols, G = (size_t)(cols / g), gg = (size_t)g * g;
  const size_t nt = (C + kObjTile - 1) / kObjTile;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  L.lfac = take(G * gg * sizeof(double));
  L.rinv = take(G * gg * sizeof(float));
  L.rcol = take(G * gg * sizeof(float));
  L.rdinv = take(G * g * sizeof(float));
  L.rdsq = take(G * g * sizeof(float));
  L.hhi = take(C * C * 2);
  L.hlo = take(C * C * 2);
  L.hscale = take(2 * sizeof(float));
  L.rmat = take(G * gg * sizeof(float));
  L.rph = take(G * gg * 2);
  L.rpl = take(G * gg * 2);
  L.rrow = take(G * g * sizeof(float));
  L.mhi = take(C * C * 2);
  L.mlo = take(C * C * 2);
  L.mrow = take(C * sizeof(float));
  L.mmax = take(C * sizeof(float));
  L.wrow = take(R * sizeof(float));
  L.wh = take(R * C * sizeof(float));
  L.tm = take(R * C * sizeof(float));
  L.rw = take(R * C * sizeof(float));
  L.cz = take(R * C * 2);
  L.gram = take(R * G * G * sizeof(float));
  L.rhs = take(R * G * sizeof(double));
  L.p = take(R * C * sizeof(float));
  L.dq = take(R * C * 2);
  const size_t cap = (size_t)sublist_cap(rows);
  L.plist = take(kSubLists * cap * sizeof(int32_t));
  L.pcount = take(pcount_words(C, g) * kSubLists * kCtrStride * sizeof(uint32_t));
  L.objpart = take(R * (nt > G ? nt : G) * sizeof(double));  // per-group sweep partials or 64-column slices
  L.lcur = take(R * sizeof(double));
  L.lprev = take(R * sizeof(double));
  L.active = take(R);
  L.stopat = take(R * sizeof(int32_t));
  L.glist = take(G * kSubLists * cap * sizeof(int32_t));
  L.gcount = take(G * kSubLists * kCtrStride * sizeof(uint32_t));
  L.gpre = take(G * (kSubLists + 1) * sizeof(int32_t));
  L.gctl = take(sizeof(GramCtl));
  L.sctl = take(sizeof(SweepCtl));
  L.rowmap = take(R * sizeof(int32_t));
  L.counters = take(kSubLists * sizeof(Counters));
  L.hist = take(JARQ_MAX_RECORDED_SWEEPS * sizeof(SweepRecord));
  L.flags = take(sizeof(Flags));
  L.total = off;
  return L;
}

}  // namespace jarq

using namespace jarq;

namespace {

bool valid_params(const jarq_params* p) {
  if (p == nullptr) return false;
  if (p->rows < 1 || p->cols < 1) return false;
  if (p->group_size != 32 && p->group_size != 64 && p->group_size != 128) return false;
  if (p->cols % p->group_size != 0) return false;
  if (p->cols / p->group_size > 128) return false;   // G x G fp64 solve must fit in LDS
  if (p->bits < 1 || p->bits > 8) return false;
  if (p->sweeps < 0 || p->sweeps > 4096) return false;
  if (!(p->ridge_lambda >= 0.f) || !isfinite(p->ridge_lambda)) return false;
  if (!(p->ridge_rcond >= 0.f) || !isfinite(p->ridge_rcond)) return false;
  if (isnan(p->tau)) return false;
  if (p->ridge_accept != 0 && p->ridge_accept != 1) return false;
  if ((size_t)p->rows * (size_t)p->cols > ((size_t)1 << 40)) return false;
  return true;
}

bool aligned(const void* ptr, size_t a) { return ptr != nullptr && ((uintptr_t)ptr % a) == 0; }

jarq_status check_ws(const jarq_params* p, const void* ws, size_t bytes) {
  if (ws == nullptr || ((uintptr_t)ws % 256) != 0) return JARQ_EWORKSPACE;
  if (bytes < make_layout(p->rows, p->cols, p->group_size).total) return JARQ_EWORKSPACE;
  return JARQ_OK;
}

#define JQ_HIP(expr)                          \
  do {                                        \
    if ((expr) != hipSuccess) return JARQ_EHIP; \
  } while (0)

struct Ctx {
  int rows, cols, g, G, bits;
  char* ws;
  Layout lay;
  hipStream_t st;
  Counters* cnt() const { return (Counters*)(ws + lay.counters); }
  Flags* flags() const { return (Flags*)(ws + lay.flags); }
  SweepRecord* hist() const { return (SweepRecord*)(ws + lay.hist); }
  uint8_t* active() const { return (uint8_t*)(ws + lay.active); }
  int32_t* rowmap() const { return (int32_t*)(ws + lay.rowmap); }
  float* wh() const { return (float*)(ws + lay.wh); }
  float* gram() const { return (float*)(ws + lay.gram); }
  float* pbuf() const { return (float*)(ws + lay.p); }
  double* objpart() const { return (double*)(ws + lay.objpart); }
  GramCtl* gctl() const { return (GramCtl*)(ws + lay.gctl); }
  SweepCtl* sctl() const { return (SweepCtl*)(ws + lay.sctl); }
  uint32_t* gcount() const { return (uint32_t*)(ws + lay.gcount); }
  int nt() const { return (cols + kObjTile - 1) / kObjTile; }
  int panels() const { return pcount_words(cols, g); }
};

Ctx make_ctx(const jarq_params* p, void* ws, void* stream) {
  Ctx c;
  c.rows = p->rows;
  c.cols = p->cols;
  c.g = p->group_size;
  c.G = p->cols / p->group_size;
  c.bits = p->bits;
  c.ws = (char*)ws;
  c.lay = make_layout(c.rows, c.cols, c.g);
  c.st = (hipStream_t)stream;
  return c;
}

hipError_t enqueue_scale_step(const Ctx& c, const float* H, const uint8_t* codes, float* scales,
                              const int32_t* zeros, const uint8_t* active, float lam,
                              float rcond, int accept) {
  (void)H;
  hipError_t e = launch_gram(c.st, c.rows, c.cols, c.g, c.ws, c.lay, codes, zeros, c.gram(),
                             nullptr, nullptr, /*incremental=*/false);
  if (e != hipSuccess) return e;
  return launch_solve(c.st, c.rows, c.cols, c.g, c.gram(), c.wh(), codes, zeros,
                      (double*)(c.ws + c.lay.rhs), nullptr, scales, active, c.cnt(), c.flags(),
                      lam, rcond, accept, nullptr, nullptr);
}

struct NoHook {
  hipError_t operator()(int, int, int) const { return hipSuccess; }
};

// The Gauss-Seidel code update, panel by panel: each panel's groups are
// decoded in order by the Babai kernel, then their accepted changes are folded
// into the residual product of every later column.  `n` positions of the
// sweep at most (the current count in *n_dev when it is not null), position p
// holding layer row map_row(rowmap, p).  The per-panel row counters must be
// zero when the first Babai launch runs: zeroed here unless the caller's
// previous launch did (counts_zeroed).  With `lists` the Babai launches also
// append each row that accepted group i to the group's list (glist, gcount),
// whose counters the caller has zeroed.  hook(kind, panel, phase) runs before
// (phase 0) and after (phase 1) each launch: kind 0 Babai, 1 panel update.
template <typename Hook = NoHook>
hipError_t enqueue_babai(const Ctx& c, int n, const int32_t* rowmap, const int* n_dev,
                         uint8_t* codes, const float* scales, const int32_t* zeros,
                         const uint8_t* active, uint8_t* cand, uint8_t* decision,
                         bool counts_zeroed = false, bool lists = false, Hook hook = Hook()) {
  const int nb = panel_groups(c.g);
  if (!counts_zeroed) {
    hipError_t e0 = launch_zero_bytes(c.st, c.ws + c.lay.pcount,
                                      (size_t)c.panels() * kSubLists * kCtrStride * sizeof(uint32_t));
    if (e0 != hipSuccess) return e0;
  }
  for (int i0 = 0, q = 0; i0 < c.G; i0 += nb, ++q) {
    const int i1 = i0 + nb < c.G ? i0 + nb : c.G;
    hipError_t e = hook(0, q, 0);
    if (e == hipSuccess)
      e = launch_babai(c.st, n, c.cols, c.g, c.bits, i0, i1, c.pbuf(), c.ws, c.lay, codes,
                       scales, zeros, active, cand, decision, c.cnt(), rowmap, n_dev,
                       lists ? (int32_t*)(c.ws + c.lay.glist) : nullptr,
                       lists ? c.gcount() : nullptr, sublist_cap(c.rows));
    if (e == hipSuccess) e = hook(0, q, 1);
    if (e != hipSuccess) return e;
    if (i1 * c.g >= c.cols) break;  // no later columns to update
    e = hook(1, q, 0);
    if (e == hipSuccess)
      e = launch_panel_update(c.st, n, c.cols, c.g, i0 * c.g, i1 * c.g, c.ws, c.lay, scales,
                              c.pbuf(), rowmap);
    if (e == hipSuccess) e = hook(1, q, 1);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

jarq_status prepare_impl(const jarq_params* p, const float* W, const float* H, void* ws,
                         void* stream) {
  Ctx c = make_ctx(p, ws, stream);
  JQ_HIP(launch_zero_bytes(c.st, c.flags(), sizeof(Flags)));
  JQ_HIP(launch_zero_bytes(c.st, c.cnt(), kSubLists * sizeof(Counters)));
  JQ_HIP(launch_chol_groups(c.st, c.cols, c.g, H, c.ws, c.lay));
  JQ_HIP(launch_split_r(c.st, c.cols, c.g, c.ws, c.lay));
  JQ_HIP(launch_split_m(c.st, c.cols, c.g, H, c.ws, c.lay));
  JQ_HIP(launch_split_h(c.st, c.cols, H, c.ws, c.lay));
  JQ_HIP(launch_gemm_ah(c.st, c.rows, c.cols, c.g, false, W, nullptr, nullptr, nullptr, H, c.wh(),
                        nullptr));
  // T = W M^T and RW = W_i L_i, the constant parts of the residual product
  // and of the objective; W's two fp16 planes borrow P's memory
  _Float16* whi = (_Float16*)c.pbuf();
  _Float16* wlo = whi + (size_t)c.rows * c.cols;
  float* wrow = (float*)(c.ws + c.lay.wrow);
  JQ_HIP(launch_split_w(c.st, c.rows, c.cols, W, whi, wlo, wrow));
  JQ_HIP(launch_wm_product(c.st, c.rows, c.cols, c.ws, c.lay, whi, wlo, wrow));
  JQ_HIP(launch_rw_product(c.st, c.rows, c.cols, c.g, c.ws, c.lay, whi, wlo, wrow));
  Flags f{};
  JQ_HIP(hipMemcpyAsync(&f, c.flags(), sizeof(Flags), hipMemcpyDeviceToHost, c.st));
  JQ_HIP(hipStreamSynchronize(c.st));
  if (f.not_spd) return JARQ_ENOT_SPD;
  return JARQ_OK;
}

// Stage boundaries with a HIP event each (stages 0-3 are consecutive runs of
// kernels), and the code update's launches with a pair each (stage 4: the
// Babai kernels, stage 5: the panel updates, which alternate).
constexpr int kBoundaries = 5;
constexpr int kFirstLaunchStage = kBoundaries - 1;

// time_stages = false: no HIP events are created and stage_ms stays 0.
// host_alloc = false: nothing is allocated (the early-stopping check then
// reads the active count with a blocking copy).
jarq_status sweeps_impl(const jarq_params* p, const float* W, const float* H, uint8_t* codes,
                        float* scales, const int32_t* zeros, void* ws, void* stream,
                        jarq_stats* stats, bool time_stages = true, bool host_alloc = true) {
  (void)H;
  Ctx c = make_ctx(p, ws, stream);
  // Device-side input checks (codes in range, |zero point| <= 1024).
  JQ_HIP(launch_zero_bytes(c.st, c.flags(), sizeof(Flags)));
  JQ_HIP(launch_validate(c.st, c.rows, c.cols, c.g, c.bits, codes, zeros, c.flags()));
  Flags f{};
  JQ_HIP(hipMemcpyAsync(&f, c.flags(), sizeof(Flags), hipMemcpyDeviceToHost, c.st));
  JQ_HIP(hipStreamSynchronize(c.st));
  if (f.bad_codes || f.bad_zeros) return JARQ_EINVAL;

  // q - z as fp16, kept in step with the codes by the code update
  JQ_HIP(launch_codes_cz(c.st, c.rows, c.cols, c.g, codes, zeros, (_Float16*)(c.ws + c.lay.cz)));
  JQ_HIP(launch_fill_u8(c.st, c.active(), (size_t)c.rows, 1));
  JQ_HIP(launch_zero_bytes(c.st, c.ws + c.lay.stopat, (size_t)c.rows * sizeof(int32_t)));
  JQ_HIP(launch_zero_bytes(c.st, c.cnt(), kSubLists * sizeof(Counters)));
  JQ_HIP(launch_zero_bytes(c.st, c.ws + c.lay.lcur, (size_t)c.rows * sizeof(double)));
  JQ_HIP(launch_zero_bytes(c.st, c.ws + c.lay.lprev, (size_t)c.rows * sizeof(double)));
  JQ_HIP(launch_zero_bytes(c.st, c.hist(), JARQ_MAX_RECORDED_SWEEPS * sizeof(SweepRecord)));
  JQ_HIP(launch_zero_bytes(c.st, c.gctl(), sizeof(GramCtl)));
  JQ_HIP(launch_zero_bytes(c.st, c.sctl(), sizeof(SweepCtl)));
  JQ_HIP(launch_zero_bytes(c.st, c.gcount(), (size_t)c.G * kSubLists * kCtrStride * sizeof(uint32_t)));
  // every row active: rowmap = 0 .. rows - 1, sctl->n = rows
  JQ_HIP(launch_compact_rows(c.st, c.rows, c.active(), c.rowmap(), c.sctl()));

  // Active-set compaction (early stopping on): a sweep works on the rows still
  // active when it starts, in ascending order (rowmap), n of them (sctl->n).
  // Both stay on the device: every per-row kernel is sized for all rows and
  // reads n itself, so no sweep waits for the host.  Without early stopping
  // every row takes part in every sweep (no list).
  const bool stopping = p->tau >= 0.f;
  const int* n_dev = stopping ? &c.sctl()->n : nullptr;
  const int32_t* rmap = stopping ? c.rowmap() : nullptr;
  const int n = c.rows;

  const int K = p->sweeps;
  const int nrec = K < JARQ_MAX_RECORDED_SWEEPS ? K : JARQ_MAX_RECORDED_SWEEPS;
  const int npan = c.panels();
  const int per_sweep = kBoundaries + 4 * npan;  // boundaries + a pair per code-update launch
  std::vector<hipEvent_t> ev;  // empty unless stages are timed
  const uint32_t all_stages = (1u << JARQ_NUM_STAGES) - 1u;
  const uint32_t tmask = (stats == nullptr || !time_stages) ? 0u
                         : (stats->stage_mask & all_stages) ? (stats->stage_mask & all_stages)
                                                             : all_stages;
  // Boundary j is used when stage j - 1 or stage j (j < kBoundaries - 1) is timed.
  auto boundary_used = [&](int j) {
    return (j > 0 && ((tmask >> (j - 1)) & 1u)) || (j < kBoundaries - 1 && ((tmask >> j) & 1u));
  };
  if (stats != nullptr) {
    memset(stats, 0, sizeof(*stats));
    stats->stage_mask = tmask;
    if (tmask != 0u) {
      ev.resize((size_t)nrec * per_sweep);
      for (auto& e : ev) JQ_HIP(hipEventCreate(&e));
    }
  }
  auto mark = [&](int k, int j) -> hipError_t {
    if (tmask == 0u || k >= nrec || !boundary_used(j)) return hipSuccess;
    return hipEventRecord(ev[(size_t)k * per_sweep + j], c.st);
  };
  // boundary j's event, or null when it is not used
  auto boundary_event = [&](int k, int j) -> hipEvent_t {
    if (tmask == 0u || k >= nrec || !boundary_used(j)) return nullptr;
    return ev[(size_t)k * per_sweep + j];
  };
  // Early stopping: every fourth sweep the active count is copied behind that
  // sweep into pinned host memory; the host looks at it once the copy has
  // landed (an event query, no wait) and ends the run when no row is left.
  // The stream never drains for it; without pinned memory the copy blocks.
  SweepCtl* host_sc = nullptr;
  hipEvent_t sc_ev = nullptr;
  bool sc_pending = false;
  if (stopping && host_alloc) {
    if (hipHostMalloc((void**)&host_sc, sizeof(SweepCtl), hipHostMallocDefault) != hipSuccess)
      host_sc = nullptr;
    else if (hipEventCreateWithFlags(&sc_ev, hipEventDisableTiming) != hipSuccess) {
      (void)hipHostFree(host_sc);
      host_sc = nullptr;
      sc_ev = nullptr;
    }
  }
  jarq_status status = JARQ_OK;
  for (int k = 0; k < K; ++k) {
    // launches of the code update timed with a pair of events each
    auto hook = [&](int kind, int q, int phase) -> hipError_t {
      if (k >= nrec || !((tmask >> (kFirstLaunchStage + kind)) & 1u)) return hipSuccess;
      const size_t at = (size_t)k * per_sweep + kBoundaries + 2 * (kind * npan + q) + phase;
      return hipEventRecord(ev[at], c.st);
    };
    hipError_t e = mark(k, 0);
    if (e == hipSuccess)
      e = launch_gram(c.st, n, c.cols, c.g, c.ws, c.lay, codes, zeros, c.gram(), rmap, n_dev,
                      /*incremental=*/true);
    if (e == hipSuccess) e = mark(k, 1);
    if (e == hipSuccess)
      e = launch_solve(c.st, n, c.cols, c.g, c.gram(), c.wh(), codes, zeros,
                       (double*)(c.ws + c.lay.rhs), c.gctl(), scales, c.active(), c.cnt(),
                       c.flags(), p->ridge_lambda, p->ridge_rcond, p->ridge_accept, rmap, n_dev);
    // boundaries 2 and 3 are the residual product's own start and end times
    // (events attached to its dispatch: no marker in the stream around it)
    if (e == hipSuccess)
      e = launch_resid(c.st, n, c.cols, c.g, c.ws, c.lay, scales, c.pbuf(), rmap, n_dev,
                       boundary_event(k, 2), boundary_event(k, 3));
    if (e == hipSuccess)
      e = launch_group_objective(c.st, n, c.cols, c.g, c.ws, c.lay, scales, c.pbuf(), c.objpart(),
                                 rmap, n_dev);
    if (e == hipSuccess)
      e = launch_stop_check(c.st, n, c.G, c.objpart(), (double*)(c.ws + c.lay.lcur),
                            (double*)(c.ws + c.lay.lprev), c.active(),
                            (int32_t*)(c.ws + c.lay.stopat), k + 1, p->tau, rmap,
                            (uint32_t*)(c.ws + c.lay.pcount), npan * kSubLists, c.gcount(),
                            c.G * kSubLists, n_dev);
    if (e == hipSuccess) e = mark(k, 4);
    if (e == hipSuccess)
      e = enqueue_babai(c, n, rmap, n_dev, codes, scales, zeros, c.active(), nullptr, nullptr,
                        /*counts_zeroed=*/true, /*lists=*/true, hook);
    if (e == hipSuccess)
      e = launch_record_sweep(c.st, c.rows, (const double*)(c.ws + c.lay.lcur), c.active(),
                              c.cnt(),
                              c.hist() + (k < JARQ_MAX_RECORDED_SWEEPS ? k
                                                                        : JARQ_MAX_RECORDED_SWEEPS - 1),
                              c.sctl(), c.gctl(), c.gcount(), (int32_t*)(c.ws + c.lay.gpre),
                              c.G);
    // the rows still active after this sweep's stopping test, for the next one
    if (e == hipSuccess && stopping)
      e = launch_compact_rows(c.st, c.rows, c.active(), c.rowmap(), c.sctl());
    if (e != hipSuccess) {
      status = JARQ_EHIP;
      break;
    }
    if (stopping && (k + 1) % 4 == 0 && k + 1 < K) {
      // Every fourth sweep the host looks whether any row is left (a sweep
      // with no row left costs its launches only).
      if (host_sc != nullptr) {
        if (sc_pending) {
          const hipError_t q = hipEventQuery(sc_ev);
          if (q == hipSuccess) {
            sc_pending = false;
            if (host_sc->n == 0) break;
          } else if (q != hipErrorNotReady) {
            status = JARQ_EHIP;
            break;
          }
        }
        if (!sc_pending) {
          if (hipMemcpyAsync(host_sc, c.sctl(), sizeof(SweepCtl), hipMemcpyDeviceToHost, c.st) !=
                  hipSuccess ||
              hipEventRecord(sc_ev, c.st) != hipSuccess) {
            status = JARQ_EHIP;
            break;
          }
          sc_pending = true;
        }
      } else {
        SweepCtl sc{};
        if (hipMemcpyAsync(&sc, c.sctl(), sizeof(sc), hipMemcpyDeviceToHost, c.st) != hipSuccess ||
            hipStreamSynchronize(c.st) != hipSuccess) {
          status = JARQ_EHIP;
          break;
        }
        if (sc.n == 0) break;
      }
    }
  }
  if (hipStreamSynchronize(c.st) != hipSuccess) status = JARQ_EHIP;
  if (sc_ev != nullptr) (void)hipEventDestroy(sc_ev);
  if (host_sc != nullptr) (void)hipHostFree(host_sc);
  SweepCtl sc{};
  if (status == JARQ_OK) {
    if (hipMemcpy(&f, c.flags(), sizeof(Flags), hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(&sc, c.sctl(), sizeof(sc), hipMemcpyDeviceToHost) != hipSuccess)
      status = JARQ_EHIP;
    else if (f.solve_failed)
      status = JARQ_ESCALE_SOLVE;
  }
  if (stats != nullptr) {
    // sweeps that started with at least one active row
    const int run = sc.started;
    stats->sweeps_run = run;
    SweepRecord hist[JARQ_MAX_RECORDED_SWEEPS];
    if (hipMemcpy(hist, c.hist(), sizeof(hist), hipMemcpyDeviceToHost) == hipSuccess) {
      const int nk = run < nrec ? run : nrec;
      for (int k = 0; k < nk; ++k) {
        stats->objective_after_scales[k] = hist[k].objective_after_scales;
        stats->accepted_groups[k] = (int64_t)hist[k].accepted;
        stats->codes_changed[k] = (int64_t)hist[k].changed;
        stats->skipped_groups[k] = (int64_t)hist[k].skipped;
        stats->ridge_rows[k] = (int32_t)hist[k].ridge_rows;
        stats->rows_active[k] = (int32_t)hist[k].active_rows;
        stats->correction_blocks[k] = (int64_t)hist[k].corr_blocks;
        stats->gram_listed[k] = (int32_t)hist[k].gram_listed;
        const size_t b = (size_t)k * per_sweep;
        for (int j = 0; j < kBoundaries - 1; ++j) {
          float ms = 0.f;
          if ((tmask >> j) & 1u) hipEventElapsedTime(&ms, ev[b + j], ev[b + j + 1]);
          stats->stage_ms[k][j] = ms;
        }
        for (int kind = 0; kind < 2; ++kind) {
          float tot = 0.f;
          if ((tmask >> (kFirstLaunchStage + kind)) & 1u) {
            for (int q = 0; q < npan - kind; ++q) {
              float ms = 0.f;
              const size_t at = b + kBoundaries + 2 * (kind * npan + q);
              hipEventElapsedTime(&ms, ev[at], ev[at + 1]);
              tot += ms;
            }
          }
          stats->stage_ms[k][kFirstLaunchStage + kind] = tot;
        }
      }
      if (run > 0) {
        const int last = run - 1 < JARQ_MAX_RECORDED_SWEEPS ? run - 1 : JARQ_MAX_RECORDED_SWEEPS - 1;
        stats->rows_active_end = (int32_t)hist[last].active_rows;
      } else {
        stats->rows_active_end = c.rows;
      }
    }
    for (auto& e : ev) hipEventDestroy(e);
  }
  return status;
}

}  // namespace

// ---- workspace for callers that cannot allocate (jarq_refine_static) ----
// One array per GPU, created with the code object on each device and held
// until the process ends.  Host code never uses the array's name as an
// address: the device address comes from hipGetSymbolAddress, once per
// device, with that device current.
static __device__ __align__(256) unsigned char scratch[JARQ_STATIC_WORKSPACE_BYTES];

namespace {

constexpr int kMaxStaticDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxStaticDevices];

jarq_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxStaticDevices) return JARQ_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return JARQ_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return JARQ_OK;
}

}  // namespace

extern "C" {

size_t jarq_workspace_bytes(const jarq_params* p) {
  if (!valid_params(p)) return 0;
  return make_layout(p->rows, p->cols, p->group_size).total;
}

jarq_status jarq_prepare(const jarq_params* p, const float* W, const float* H, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16)) return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  return prepare_impl(p, W, H, workspace, stream);
}

jarq_status jarq_scale_step(const jarq_params* p, const float* H, const uint8_t* codes,
                            float* scales, const int32_t* zeros, void* workspace,
                            size_t workspace_bytes, void* stream) {
  if (!valid_params(p) || !aligned(H, 16) || !aligned(codes, 16) || !aligned(scales, 16) ||
      !aligned(zeros, 4))
    return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  Ctx c = make_ctx(p, workspace, stream);
  if (enqueue_scale_step(c, H, codes, scales, zeros, nullptr, p->ridge_lambda, p->ridge_rcond,
                         p->ridge_accept) !=
      hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_code_step(const jarq_params* p, const float* W, const float* H, uint8_t* codes,
                           const float* scales, const int32_t* zeros, void* workspace,
                           size_t workspace_bytes, void* stream, uint8_t* cand,
                           uint8_t* decision) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(codes, 16) ||
      !aligned(scales, 16) || !aligned(zeros, 4))
    return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  Ctx c = make_ctx(p, workspace, stream);
  (void)W;
  if (launch_codes_cz(c.st, c.rows, c.cols, c.g, codes, zeros, (_Float16*)(c.ws + c.lay.cz)) !=
          hipSuccess ||
      launch_resid(c.st, c.rows, c.cols, c.g, c.ws, c.lay, scales, c.pbuf(), nullptr, nullptr) !=
          hipSuccess)
    return JARQ_EHIP;
  if (enqueue_babai(c, c.rows, nullptr, nullptr, codes, scales, zeros, nullptr, cand, decision) !=
      hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_sweeps(const jarq_params* p, const float* W, const float* H, uint8_t* codes,
                        float* scales, const int32_t* zeros, void* workspace,
                        size_t workspace_bytes, void* stream, jarq_stats* stats) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(codes, 16) ||
      !aligned(scales, 16) || !aligned(zeros, 4))
    return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  return sweeps_impl(p, W, H, codes, scales, zeros, workspace, stream, stats);
}

jarq_status jarq_refine(const jarq_params* p, const float* W, const float* H, uint8_t* codes,
                        float* scales, const int32_t* zeros, void* workspace,
                        size_t workspace_bytes, void* stream, jarq_stats* stats) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(codes, 16) ||
      !aligned(scales, 16) || !aligned(zeros, 4))
    return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (stats != nullptr) {
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return JARQ_EHIP;
    hipEventRecord(e0, (hipStream_t)stream);
  }
  s = prepare_impl(p, W, H, workspace, stream);
  float prep_ms = 0.f;
  if (stats != nullptr) {
    hipEventRecord(e1, (hipStream_t)stream);
    hipEventSynchronize(e1);
    hipEventElapsedTime(&prep_ms, e0, e1);
    hipEventDestroy(e0);
    hipEventDestroy(e1);
  }
  if (s != JARQ_OK) return s;
  s = sweeps_impl(p, W, H, codes, scales, zeros, workspace, stream, stats);
  if (stats != nullptr) stats->prep_ms = prep_ms;
  return s;
}

jarq_status jarq_stop_sweeps(const jarq_params* p, const void* workspace, size_t workspace_bytes,
                             int32_t* stop_sweep, void* stream) {
  if (!valid_params(p) || !aligned(stop_sweep, 4)) return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  const Layout lay = make_layout(p->rows, p->cols, p->group_size);
  JQ_HIP(hipMemcpyAsync(stop_sweep, (const char*)workspace + lay.stopat,
                        (size_t)p->rows * sizeof(int32_t), hipMemcpyDeviceToDevice,
                        (hipStream_t)stream));
  return JARQ_OK;
}

jarq_status jarq_refine_static(const jarq_params* p, const float* W, const float* H,
                               uint8_t* codes, float* scales, const int32_t* zeros, void* stream,
                               jarq_stats* stats) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(codes, 16) ||
      !aligned(scales, 16) || !aligned(zeros, 4))
    return JARQ_EINVAL;
  if (make_layout(p->rows, p->cols, p->group_size).total > (size_t)JARQ_STATIC_WORKSPACE_BYTES)
    return JARQ_ESTATIC_LIMIT;
  void* ws = nullptr;
  jarq_status s = static_scratch(&ws);
  if (s != JARQ_OK) return s;
  s = prepare_impl(p, W, H, ws, stream);
  if (s != JARQ_OK) return s;
  return sweeps_impl(p, W, H, codes, scales, zeros, ws, stream, stats, /*time_stages=*/false,
                     /*host_alloc=*/false);
}

jarq_status jarq_objective(const jarq_params* p, const float* W, const float* H,
                           const uint8_t* codes, const float* scales, const int32_t* zeros,
                           void* workspace, size_t workspace_bytes, void* stream,
                           double* row_objective) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(codes, 16) ||
      !aligned(scales, 16) || !aligned(zeros, 4) || !aligned(row_objective, 8))
    return JARQ_EINVAL;
  jarq_status s = check_ws(p, workspace, workspace_bytes);
  if (s != JARQ_OK) return s;
  Ctx c = make_ctx(p, workspace, stream);
  if (launch_gemm_ah(c.st, c.rows, c.cols, c.g, true, W, codes, scales, zeros, H, nullptr,
                     c.objpart()) != hipSuccess)
    return JARQ_EHIP;
  if (launch_row_objective(c.st, c.rows, c.nt(), c.objpart(), row_objective) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_hessian_accumulate(const float* X, int64_t m, int32_t d, double alpha,
                                    double* Hacc, void* stream) {
  if (d < 1 || d > 32768 || d % 4 != 0 || m < 0 || m > INT32_MAX - 64 || !isfinite(alpha) ||
      !aligned(Hacc, 8))
    return JARQ_EINVAL;
  if (m == 0) return JARQ_OK;  // X may be NULL
  if (!aligned(X, 16)) return JARQ_EINVAL;
  if (launch_hessian_update((hipStream_t)stream, X, (int)m, d, alpha, Hacc) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_hessian_accumulate_bf16(const void* X, int64_t m, int32_t d, double alpha,
                                         double* Hacc, void* stream) {
  if (d < 1 || d > 32768 || d % 8 != 0 || m < 0 || m > INT32_MAX - 128 || !isfinite(alpha) ||
      !aligned(Hacc, 8))
    return JARQ_EINVAL;
  if (m == 0) return JARQ_OK;  // X may be NULL
  if (!aligned(X, 16)) return JARQ_EINVAL;
  if (launch_hessian_update_bf16((hipStream_t)stream, X, (int)m, d, alpha, Hacc) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_hessian_finalize(const double* Hacc, int32_t d, double damp, double nu2,
                                  float* H, void* stream) {
  if (d < 1 || d > 32768 || d % 4 != 0 || !(damp >= 0.0) || !isfinite(damp) || !(nu2 >= 0.0) ||
      !isfinite(nu2) || !aligned(Hacc, 8) || !aligned(H, 16))
    return JARQ_EINVAL;
  const uintptr_t h0 = (uintptr_t)H, h1 = h0 + (size_t)d * d * sizeof(float);
  const uintptr_t a0 = (uintptr_t)Hacc, a1 = a0 + (size_t)d * d * sizeof(double);
  if (h0 < a1 && a0 < h1) return JARQ_EINVAL;
  if (launch_hessian_finalize((hipStream_t)stream, Hacc, d, damp, nu2, H) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_rtn(const jarq_params* p, const float* W, uint8_t* codes, float* scales,
                     int32_t* zeros, void* stream) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(codes, 16) || !aligned(scales, 4) ||
      !aligned(zeros, 4))
    return JARQ_EINVAL;
  if (launch_rtn((hipStream_t)stream, W, p->rows, p->cols, p->group_size, p->bits, codes, scales,
                 zeros) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_cross_accumulate(const float* Xq, const float* X, int64_t m, int32_t d,
                                  double alpha, double* Dacc, void* stream) {
  if (d < 1 || d > 32768 || d % 4 != 0 || m < 0 || m > INT32_MAX - 64 || !isfinite(alpha) ||
      !aligned(Dacc, 8))
    return JARQ_EINVAL;
  if (m == 0) return JARQ_OK;  // Xq and X may be NULL
  if (!aligned(Xq, 16) || !aligned(X, 16)) return JARQ_EINVAL;
  if (launch_cross_update((hipStream_t)stream, Xq, X, (int)m, d, alpha, Dacc) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

size_t jarq_qep_workspace_bytes(const jarq_params* p) {
  if (!valid_params(p)) return 0;
  return qep_workspace_bytes(p->rows, p->cols);
}

jarq_status jarq_qep_correct(const jarq_params* p, const float* W, const float* H,
                             const double* D, double mu, float* Wcorr, void* workspace,
                             size_t workspace_bytes, void* stream) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(D, 8) ||
      !aligned(Wcorr, 16) || !(mu >= 0.0 && mu <= 1.0))
    return JARQ_EINVAL;
  if (workspace == nullptr || ((uintptr_t)workspace % 256) != 0 ||
      workspace_bytes < qep_workspace_bytes(p->rows, p->cols))
    return JARQ_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  int* flag = nullptr;
  if (launch_qep_correct(st, p->rows, p->cols, W, H, D, mu, Wcorr, (char*)workspace, &flag) !=
      hipSuccess)
    return JARQ_EHIP;
  int f = 0;
  JQ_HIP(hipMemcpyAsync(&f, flag, sizeof(int), hipMemcpyDeviceToHost, st));
  JQ_HIP(hipStreamSynchronize(st));
  return f ? JARQ_ENOT_SPD : JARQ_OK;
}

jarq_status jarq_canonicalize(const jarq_params* p, uint8_t* codes, float* scales,
                              int32_t* zeros, void* stream) {
  if (!valid_params(p) || !aligned(codes, 16) || !aligned(scales, 4) || !aligned(zeros, 4))
    return JARQ_EINVAL;
  if (launch_canonicalize((hipStream_t)stream, p->rows, p->cols, p->group_size, p->bits, codes,
                          scales, zeros) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_dequantize(const jarq_params* p, const uint8_t* codes, const float* scales,
                            const int32_t* zeros, const int32_t* perm, int32_t dtype, void* out,
                            void* stream) {
  if (!valid_params(p) || codes == nullptr || !aligned(scales, 4) || !aligned(zeros, 4) ||
      dtype < JARQ_F32 || dtype > JARQ_BF16 || !aligned(out, dtype == JARQ_F32 ? 4 : 2) ||
      (perm != nullptr && !aligned(perm, 4)))
    return JARQ_EINVAL;
  if (launch_dequantize((hipStream_t)stream, p->rows, p->cols, p->group_size, codes, scales,
                        zeros, perm, dtype, out) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_pack_codes(const jarq_params* p, const uint8_t* codes, uint32_t* packed,
                            void* stream) {
  if (!valid_params(p) || codes == nullptr || !aligned(packed, 4)) return JARQ_EINVAL;
  if (launch_pack((hipStream_t)stream, p->rows, p->cols, p->bits, codes, packed) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_unpack_codes(const jarq_params* p, const uint32_t* packed, uint8_t* codes,
                              void* stream) {
  if (!valid_params(p) || codes == nullptr || !aligned(packed, 4)) return JARQ_EINVAL;
  if (launch_unpack((hipStream_t)stream, p->rows, p->cols, p->bits, packed, codes) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_act_order(const float* H, int32_t d, int32_t* perm, void* stream) {
  if (d < 1 || d > 32768 || !aligned(H, 4) || !aligned(perm, 4)) return JARQ_EINVAL;
  if (launch_act_order((hipStream_t)stream, H, d, perm) != hipSuccess) return JARQ_EHIP;
  return JARQ_OK;
}

jarq_status jarq_permute(const jarq_params* p, const int32_t* perm, const float* W, const float* H,
                         float* Wp, float* Hp, void* stream) {
  if (!valid_params(p) || !aligned(perm, 4) || !aligned(W, 4) || !aligned(H, 4) ||
      !aligned(Wp, 4) || !aligned(Hp, 4))
    return JARQ_EINVAL;
  if (launch_permute((hipStream_t)stream, p->rows, p->cols, perm, W, H, Wp, Hp) != hipSuccess)
    return JARQ_EHIP;
  return JARQ_OK;
}

size_t jarq_gptq_workspace_bytes(const jarq_params* p) {
  if (!valid_params(p)) return 0;
  return gptq_workspace_bytes(p->rows, p->cols, p->group_size);
}

jarq_status jarq_gptq(const jarq_params* p, const float* W, const float* H, uint8_t* codes,
                      float* scales, int32_t* zeros, void* workspace, size_t workspace_bytes,
                      void* stream) {
  if (!valid_params(p) || !aligned(W, 16) || !aligned(H, 16) || !aligned(codes, 16) ||
      !aligned(scales, 4) || !aligned(zeros, 4))
    return JARQ_EINVAL;
  if (workspace == nullptr || ((uintptr_t)workspace % 256) != 0 ||
      workspace_bytes < gptq_workspace_bytes(p->rows, p->cols, p->group_size))
    return JARQ_EWORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  int* flag = nullptr;
  if (launch_gptq(st, p->rows, p->cols, p->group_size, p->bits, W, H, (char*)workspace, codes,
                  scales, zeros, &flag) != hipSuccess)
    return JARQ_EHIP;
  int f = 0;
  JQ_HIP(hipMemcpyAsync(&f, flag, sizeof(int), hipMemcpyDeviceToHost, st));
  JQ_HIP(hipStreamSynchronize(st));
  return f ? JARQ_ENOT_SPD : JARQ_OK;
}

const char* jarq_status_string(jarq_status s) {
  switch (s) {
    case JARQ_OK: return "ok";
    case JARQ_EINVAL: return "invalid argument";
    case JARQ_ENOT_SPD: return "a diagonal Hessian block is not positive definite";
    case JARQ_ESCALE_SOLVE: return "a scale solve failed after the ridge";
    case JARQ_EHIP: return "HIP runtime error";
    case JARQ_EWORKSPACE: return "workspace missing, too small or misaligned";
    case JARQ_ESTATIC_LIMIT:
      return "layer needs more workspace than the static scratch of jarq_refine_static";
    default: return "unknown status";
  }
}

int32_t jarq_abi_version(void) { return JARQ_ABI_VERSION; }

}  // extern "C"
