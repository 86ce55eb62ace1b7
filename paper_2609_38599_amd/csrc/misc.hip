// Small per-sweep kernels: row objectives, the early-stopping rule of App. E.2,
// fills (kernels rather than hipMemsetAsync so a captured graph replays them
// reliably), the per-sweep record, and the device-side input checks.
#include "jarq_internal.h"

namespace jarq {

__global__ void row_objective_kernel(int rows, int nt, const double* __restrict__ part,
                                     double* __restrict__ out) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  double s = 0.0;
  for (int t = 0; t < nt; ++t) s += part[(size_t)r * nt + t];
  out[r] = s;
}

hipError_t launch_row_objective(hipStream_t st, int rows, int nt, const double* objpart,
                                double* out) {
  hipLaunchKernelGGL(row_objective_kernel, dim3((rows + 255) / 256), dim3(256), 0, st, rows, nt,
                     objpart, out);
  return hipGetLastError();
}

// L_j^(k) = sum of the partials; at k >= 2 an active row stops (before its
// code update) when (L^(k-1) - L^(k)) / max(|L^(k-1)|, eps) <= tau or
// |L^(k-1) - L^(k)| <= tau (App. E.2, eq. (strict_stopping)).  The new scales
// are kept, and the iteration is recorded in stopat.
__global__ void stop_check_kernel(int n, int nt, const double* __restrict__ part,
                                  double* __restrict__ lcur, double* __restrict__ lprev,
                                  uint8_t* __restrict__ active, int32_t* __restrict__ stopat,
                                  int sweep, float tau,
                                  const int32_t* __restrict__ rowmap,
                                  uint32_t* __restrict__ zero_ctr, int nzero,
                                  uint32_t* __restrict__ zero_ctr2, int nzero2,
                                  const int* __restrict__ n_dev) {
  // counters the code update appends to start it at zero (its per-panel and
  // per-group row lists)
  if (blockIdx.x == 0) {
    for (int t = threadIdx.x; t < nzero; t += blockDim.x) zero_ctr[(size_t)t * kCtrStride] = 0u;
    for (int t = threadIdx.x; t < nzero2; t += blockDim.x) zero_ctr2[(size_t)t * kCtrStride] = 0u;
  }
  if (n_dev != nullptr) n = *n_dev;
  const int pos = blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= n) return;
  const int r = map_row(rowmap, pos);
  if (!active[r]) return;
  double s = 0.0;
  for (int t = 0; t < nt; ++t) s += part[(size_t)pos * nt + t];
  lcur[r] = s;
  if (tau >= 0.f && sweep >= 2) {
    const double prev = lprev[r];
    const double dec = prev - s;
    const double rel = dec / fmax(fabs(prev), (double)kFp32Eps);
    if (rel <= (double)tau || fabs(dec) <= (double)tau) {
      active[r] = 0;
      stopat[r] = sweep;
    }
  }
  lprev[r] = s;
}

hipError_t launch_stop_check(hipStream_t st, int n, int nt, const double* objpart,
                             double* lcur, double* lprev, uint8_t* active, int32_t* stopat,
                             int sweep, float tau, const int32_t* rowmap, uint32_t* zero_ctr,
                             int nzero, uint32_t* zero_ctr2, int nzero2, const int* n_dev) {
  if (n <= 0 || nzero < 0 || nzero2 < 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(stop_check_kernel, dim3((n + 255) / 256), dim3(256), 0, st, n, nt,
                     objpart, lcur, lprev, active, stopat, sweep, tau, rowmap, zero_ctr, nzero,
                     zero_ctr2, nzero2, n_dev);
  return hipGetLastError();
}

// Stream compaction of the active flags, one 1024-thread work-group: thread t
// counts its contiguous chunk of rows, an exclusive scan over the threads
// gives each chunk's first position, and the chunk is written in order.
__global__ __launch_bounds__(1024) void compact_rows_kernel(int rows,
                                                            const uint8_t* __restrict__ active,
                                                            int32_t* __restrict__ rowmap,
                                                            SweepCtl* __restrict__ sctl) {
  __shared__ int pre_s[1024];
  const int t = threadIdx.x;
  const int per = (rows + 1023) / 1024;
  const int b = min(t * per, rows), e = min(b + per, rows);
  int c = 0;
  for (int r = b; r < e; ++r) c += active[r] != 0;
  pre_s[t] = c;
  __syncthreads();
  for (int w = 1; w < 1024; w <<= 1) {  // inclusive scan (Hillis-Steele)
    const int v = t >= w ? pre_s[t - w] : 0;
    __syncthreads();
    pre_s[t] += v;
    __syncthreads();
  }
  int pos = pre_s[t] - c;
  for (int r = b; r < e; ++r)
    if (active[r] != 0) rowmap[pos++] = r;
  if (t == 1023) sctl->n = pre_s[1023];
}

hipError_t launch_compact_rows(hipStream_t st, int rows, const uint8_t* active, int32_t* rowmap,
                               SweepCtl* sctl) {
  hipLaunchKernelGGL(compact_rows_kernel, dim3(1), dim3(1024), 0, st, rows, active, rowmap, sctl);
  return hipGetLastError();
}

__global__ void fill_u8_kernel(uint8_t* __restrict__ p, size_t n, uint8_t v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

hipError_t launch_fill_u8(hipStream_t st, uint8_t* p, size_t n, uint8_t v) {
  if (n == 0) return hipSuccess;
  const size_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(fill_u8_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0,
                     st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_zero_bytes(hipStream_t st, void* p, size_t n) {
  return launch_fill_u8(st, (uint8_t*)p, n, 0);
}

// Sum of L over all rows (a stopped row keeps its last L, which is still its
// objective) in a fixed order, plus the counters; the counters are then reset.
// One 1024-thread work-group; each thread loads four rows before adding them
// (independent loads in flight), then a fixed-order tree over the threads.
constexpr int kRecordThreads = 1024;
__global__ __launch_bounds__(kRecordThreads) void record_sweep_kernel(
    int rows, const double* __restrict__ lcur, const uint8_t* __restrict__ active,
    Counters* __restrict__ cnt, SweepRecord* __restrict__ rec, SweepCtl* __restrict__ sctl,
    GramCtl* __restrict__ gctl, const uint32_t* __restrict__ gcount, int32_t* __restrict__ gpre,
    int G) {
  // prefix sums of the Gram row sub-lists, one group per thread (all loads
  // first)
  for (int x = threadIdx.x; x < G; x += kRecordThreads) {
    int c[kSubLists];
#pragma unroll
    for (int s = 0; s < kSubLists; ++s) c[s] = (int)gcount[((size_t)x * kSubLists + s) * kCtrStride];
    int acc = 0;
#pragma unroll
    for (int s = 0; s < kSubLists; ++s) {
      gpre[x * (kSubLists + 1) + s] = acc;
      acc += c[s];
    }
    gpre[x * (kSubLists + 1) + kSubLists] = acc;
  }
  // the counter copies: thread t < kSubLists reads copy t (then resets it)
  __shared__ Counters csum_s[kSubLists];
  if (threadIdx.x < kSubLists) {
    Counters* ct = cnt + threadIdx.x;
    Counters v{};
    v.accepted = ct->accepted;
    v.changed = ct->changed;
    v.skipped = ct->skipped;
    v.corr_blocks = ct->corr_blocks;
    v.ridge_rows = ct->ridge_rows;
    v.solve_failed = ct->solve_failed;
    csum_s[threadIdx.x] = v;
    ct->accepted = 0;
    ct->changed = 0;
    ct->skipped = 0;
    ct->corr_blocks = 0;
    ct->ridge_rows = 0;
    ct->solve_failed = 0;
    ct->active_rows = 0;
  }
  __shared__ double red[kRecordThreads];
  __shared__ unsigned int act[kRecordThreads];
  double s = 0.0;
  unsigned int a = 0;
  for (int r0 = threadIdx.x; r0 < rows; r0 += 4 * kRecordThreads) {
    double v[4];
    unsigned int b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = r0 + u * kRecordThreads;
      v[u] = r < rows ? lcur[r] : 0.0;
      b[u] = r < rows ? (active[r] ? 1u : 0u) : 0u;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      s += v[u];
      a += b[u];
    }
  }
  red[threadIdx.x] = s;
  act[threadIdx.x] = a;
  __syncthreads();
  for (int w = kRecordThreads / 2; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) {
      red[threadIdx.x] += red[threadIdx.x + w];
      act[threadIdx.x] += act[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    Counters sum{};
    for (int c = 0; c < kSubLists; ++c) {  // LDS, written before the tree's barriers
      sum.accepted += csum_s[c].accepted;
      sum.changed += csum_s[c].changed;
      sum.skipped += csum_s[c].skipped;
      sum.corr_blocks += csum_s[c].corr_blocks;
      sum.ridge_rows += csum_s[c].ridge_rows;
      sum.solve_failed += csum_s[c].solve_failed;
    }
    rec->objective_after_scales = red[0];
    rec->accepted = sum.accepted;
    rec->changed = sum.changed;
    rec->skipped = sum.skipped;
    rec->corr_blocks = sum.corr_blocks;
    rec->ridge_rows = sum.ridge_rows;
    rec->solve_failed = sum.solve_failed;
    rec->active_rows = act[0];
    const int started = sctl->n;
    rec->started_rows = (unsigned int)started;
    rec->gram_listed = (unsigned int)gctl->listed;
    if (started > 0) {
      sctl->started += 1;
      gctl->valid = 1;  // every row that took part has its matrix built
    }
  }
}

hipError_t launch_record_sweep(hipStream_t st, int rows, const double* lcur,
                               const uint8_t* active, Counters* cnt, SweepRecord* rec,
                               SweepCtl* sctl, GramCtl* gctl, const uint32_t* gcount,
                               int32_t* gpre, int G) {
  hipLaunchKernelGGL(record_sweep_kernel, dim3(1), dim3(kRecordThreads), 0, st, rows, lcur, active,
                     cnt, rec, sctl, gctl, gcount, gpre, G);
  return hipGetLastError();
}

__global__ void validate_kernel(int rows, int cols, int g, int qmax,
                                const uint8_t* __restrict__ codes,
                                const int32_t* __restrict__ zeros, Flags* __restrict__ flags) {
  const size_t n = (size_t)rows * cols;
  const int G = cols / g;
  int bad_q = 0, bad_z = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    bad_q += codes[i] > qmax;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < (size_t)rows * G;
       i += (size_t)gridDim.x * blockDim.x) {
    const int z = zeros[i];
    bad_z += (z > 1024 || z < -1024);  // q - z and 1024 + z stay exact in fp16
  }
  if (bad_q) atomicAdd(&flags->bad_codes, bad_q);
  if (bad_z) atomicAdd(&flags->bad_zeros, bad_z);
}

hipError_t launch_validate(hipStream_t st, int rows, int cols, int g, int bits,
                           const uint8_t* codes, const int32_t* zeros, Flags* flags) {
  hipLaunchKernelGGL(validate_kernel, dim3(1024), dim3(256), 0, st, rows, cols, g,
                     (1 << bits) - 1, codes, zeros, flags);
  return hipGetLastError();
}

}  // namespace jarq
