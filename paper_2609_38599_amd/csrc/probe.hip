// Calibration kernel for profiler counters of the local data share (LDS):
// a known number of bytes is written to and read from LDS, so that the LDS
// counters read for the kernels of the sweep can be scaled to bytes, and its
// rate shows what the LDS delivers to a streaming reader.
#include "jarq_internal.h"

namespace jarq {

namespace {
constexpr int kProbeThreads = 256;
constexpr int kProbeBytes = 32768;                        // LDS per work-group
constexpr int kProbeReads = kProbeBytes / (kProbeThreads * 16);  // 16-byte reads per thread per pass
}  // namespace

// Each work-group fills 32 KB of LDS (16 bytes per thread and store), then
// reads all of it `passes` times, thread t reading the 16-byte chunks t,
// t + 256, ...: a wavefront's 64 reads cover 1 KB of consecutive bytes (no
// bank conflict).  The reads are inline asm so that none is merged or hoisted
// out of the loop; their sum is written out so that none is dead.
__global__ __launch_bounds__(kProbeThreads) void lds_probe_kernel(int passes,
                                                                  float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) float buf[kProbeBytes / 4];
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < kProbeReads; ++i) {
    const int c = t + kProbeThreads * i;
    *(f32x4*)(buf + 4 * c) = f32x4{(float)c, 1.f, 2.f, 3.f};
  }
  __syncthreads();
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const uint32_t base = (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)buf;
  for (int p = 0; p < passes; ++p) {
    f32x4 v[kProbeReads];
#pragma unroll
    for (int i = 0; i < kProbeReads; ++i) {
      const uint32_t a = base + (uint32_t)((t + kProbeThreads * i) * 16);
      asm volatile("ds_read_b128 %0, %1" : "=v"(v[i]) : "v"(a));
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int i = 0; i < kProbeReads; ++i) acc += v[i];
  }
  out[(size_t)blockIdx.x * kProbeThreads + t] = acc[0] + acc[1] + acc[2] + acc[3];
}

}  // namespace jarq

using namespace jarq;

extern "C" {

int64_t jarq_lds_probe(int32_t workgroups, int32_t passes, float* out, void* stream) {
  if (workgroups < 1 || passes < 1 || out == nullptr || ((uintptr_t)out % 4) != 0) return -1;
  hipLaunchKernelGGL(lds_probe_kernel, dim3(workgroups), dim3(kProbeThreads), 0,
                     (hipStream_t)stream, passes, out);
  if (hipGetLastError() != hipSuccess) return -1;
  return (int64_t)workgroups * kProbeBytes * ((int64_t)passes + 1);
}

}  // extern "C"
