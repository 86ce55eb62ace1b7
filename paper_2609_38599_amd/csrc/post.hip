// After refinement: negative-scale canonicalization (App. E.3), dequantized
// weights in a floating-point dtype, packed b-bit codes, and the activation
// ordering a GPTQ host may use (refinement keeps its groups in the reordered
// coordinates and the weights return to the original ones on write-back,
// App. A.1 and App. E.2).
#include "jarq_internal.h"

namespace jarq {

namespace {
unsigned grid_of(long long n) {
  const long long b = (n + 255) / 256;
  return (unsigned)(b < 16384 ? b : 16384);
}
}  // namespace

// eq. (canonicalization): for s < 0, s' = -s, q' = qmax - q, z' = qmax - z,
// which represents the same weights.  One thread per group.
__global__ __launch_bounds__(256) void canonicalize_kernel(int rows, int cols, int g, int bits,
                                                           uint8_t* __restrict__ codes,
                                                           float* __restrict__ scales,
                                                           int32_t* __restrict__ zeros) {
  const int G = cols / g;
  const long long e = (long long)blockIdx.x * 256 + threadIdx.x;
  if (e >= (long long)rows * G) return;
  const float s = scales[e];
  if (!(s < 0.f)) return;
  const int qmax = (1 << bits) - 1;
  const long long row = e / G, grp = e % G;
  uint8_t* q = codes + row * cols + grp * g;
  for (int c = 0; c < g; c += 4) {
    uint32_t v = *(uint32_t*)(q + c);
    uint32_t out = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) out |= (uint32_t)(qmax - (int)((v >> (8 * i)) & 0xFF)) << (8 * i);
    *(uint32_t*)(q + c) = out;
  }
  scales[e] = -s;
  zeros[e] = qmax - zeros[e];
}

hipError_t launch_canonicalize(hipStream_t st, int rows, int cols, int g, int bits,
                               uint8_t* codes, float* scales, int32_t* zeros) {
  const long long n = (long long)rows * (cols / g);
  hipLaunchKernelGGL(canonicalize_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     rows, cols, g, bits, codes, scales, zeros);
  return hipGetLastError();
}

// Round-to-nearest-even fp32 -> bf16 bits (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
  const uint32_t r = u + 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(r >> 16);
}

// out[r][c] = s (q - z) in fp32, rounded once to the output dtype; with a
// permutation, position k of the refined layer is original column perm[k]
// (entries outside [0, cols) are skipped).
__global__ __launch_bounds__(256) void dequantize_kernel(int rows, int cols, int g,
                                                         const uint8_t* __restrict__ codes,
                                                         const float* __restrict__ scales,
                                                         const int32_t* __restrict__ zeros,
                                                         const int32_t* __restrict__ perm,
                                                         int dtype, void* __restrict__ out) {
  const long long n = (long long)rows * cols;
  const int G = cols / g;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256) {
    const long long r = e / cols;
    const int k = (int)(e % cols);
    const long long sg = r * G + k / g;
    const float v = scales[sg] * (float)((int)codes[e] - zeros[sg]);
    long long dst = e;
    if (perm != nullptr) {
      const int c = perm[k];
      if (c < 0 || c >= cols) continue;
      dst = r * cols + c;
    }
    if (dtype == 0)
      ((float*)out)[dst] = v;
    else if (dtype == 1)
      ((_Float16*)out)[dst] = (_Float16)v;
    else
      ((uint16_t*)out)[dst] = f32_to_bf16_bits(v);
  }
}

hipError_t launch_dequantize(hipStream_t st, int rows, int cols, int g, const uint8_t* codes,
                             const float* scales, const int32_t* zeros, const int32_t* perm,
                             int dtype, void* out) {
  const long long n = (long long)rows * cols;
  hipLaunchKernelGGL(dequantize_kernel, dim3(grid_of(n)), dim3(256), 0, st, rows, cols, g, codes,
                     scales, zeros, perm, dtype, out);
  return hipGetLastError();
}

// Row r's codes as one little-endian bit stream: code k occupies stream bits
// [k b, k b + b), stream bit t is bit t % 32 of word t / 32 of the row, rows
// start on a word boundary (wpr = ceil(cols b / 32) words per row).  One
// thread per word.
__global__ __launch_bounds__(256) void pack_kernel(int rows, int cols, int bits, int wpr,
                                                   const uint8_t* __restrict__ codes,
                                                   uint32_t* __restrict__ packed) {
  const long long n = (long long)rows * wpr;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256) {
    const long long r = e / wpr;
    const long long w = e % wpr;
    const long long t0 = 32 * w;                      // first stream bit of the word
    const int k0 = (int)(t0 / bits);
    const int k1 = (int)min((long long)cols - 1, (t0 + 31) / bits);
    uint32_t word = 0;
    for (int k = k0; k <= k1; ++k) {
      const long long shift = (long long)k * bits - t0;   // may be negative for k0
      const uint32_t q = codes[r * cols + k] & ((1u << bits) - 1u);
      if (shift >= 0)
        word |= q << shift;
      else
        word |= q >> (-shift);
    }
    packed[e] = word;
  }
}

__global__ __launch_bounds__(256) void unpack_kernel(int rows, int cols, int bits, int wpr,
                                                     const uint32_t* __restrict__ packed,
                                                     uint8_t* __restrict__ codes) {
  const long long n = (long long)rows * cols;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (long long)gridDim.x * 256) {
    const long long r = e / cols;
    const long long k = e % cols;
    const long long t = k * bits;
    const uint32_t* row = packed + r * wpr;
    const int w = (int)(t / 32), o = (int)(t % 32);
    uint64_t two = row[w];
    if (o + bits > 32) two |= (uint64_t)row[w + 1] << 32;
    codes[e] = (uint8_t)((two >> o) & ((1u << bits) - 1u));
  }
}

hipError_t launch_pack(hipStream_t st, int rows, int cols, int bits, const uint8_t* codes,
                       uint32_t* packed) {
  const int wpr = (int)(((long long)cols * bits + 31) / 32);
  hipLaunchKernelGGL(pack_kernel, dim3(grid_of((long long)rows * wpr)), dim3(256), 0, st, rows,
                     cols, bits, wpr, codes, packed);
  return hipGetLastError();
}

hipError_t launch_unpack(hipStream_t st, int rows, int cols, int bits, const uint32_t* packed,
                         uint8_t* codes) {
  const int wpr = (int)(((long long)cols * bits + 31) / 32);
  hipLaunchKernelGGL(unpack_kernel, dim3(grid_of((long long)rows * cols)), dim3(256), 0, st, rows,
                     cols, bits, wpr, packed, codes);
  return hipGetLastError();
}

// Activation ordering: channels by decreasing diag(H), ties by increasing
// index (a stable sort): rank(i) = #{j : h_j > h_i or (h_j == h_i and j < i)},
// perm[rank(i)] = i.  One thread per channel; diag staged through LDS.
__global__ __launch_bounds__(256) void act_order_kernel(const float* __restrict__ H, int d,
                                                        int32_t* __restrict__ perm) {
  __shared__ float hs[256];
  const int i = blockIdx.x * 256 + threadIdx.x;
  const float hi = i < d ? H[(long long)i * d + i] : 0.f;
  int rank = 0;
  for (int j0 = 0; j0 < d; j0 += 256) {
    __syncthreads();
    const int j = j0 + threadIdx.x;
    hs[threadIdx.x] = j < d ? H[(long long)j * d + j] : 0.f;
    __syncthreads();
    const int nj = min(256, d - j0);
    for (int t = 0; t < nj; ++t) {
      const float hj = hs[t];
      rank += (hj > hi || (hj == hi && j0 + t < i)) ? 1 : 0;
    }
  }
  if (i < d) perm[rank] = i;
}

hipError_t launch_act_order(hipStream_t st, const float* H, int d, int32_t* perm) {
  hipLaunchKernelGGL(act_order_kernel, dim3((d + 255) / 256), dim3(256), 0, st, H, d, perm);
  return hipGetLastError();
}

// Wp[r][k] = W[r][perm[k]], Hp[k][l] = H[perm[k]][perm[l]] (0 where an entry of
// perm is outside [0, d)).
__global__ __launch_bounds__(256) void permute_kernel(int rows, int d,
                                                      const int32_t* __restrict__ perm,
                                                      const float* __restrict__ W,
                                                      const float* __restrict__ H,
                                                      float* __restrict__ Wp,
                                                      float* __restrict__ Hp) {
  const long long nw = (long long)rows * d, nh = (long long)d * d;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < nw + nh;
       e += (long long)gridDim.x * 256) {
    if (e < nw) {
      const long long r = e / d;
      const int c = perm[e % d];
      Wp[e] = (c >= 0 && c < d) ? W[r * d + c] : 0.f;
    } else {
      const long long f = e - nw;
      const int a = perm[f / d], b = perm[f % d];
      Hp[f] = (a >= 0 && a < d && b >= 0 && b < d) ? H[(long long)a * d + b] : 0.f;
    }
  }
}

hipError_t launch_permute(hipStream_t st, int rows, int d, const int32_t* perm, const float* W,
                          const float* H, float* Wp, float* Hp) {
  const long long n = (long long)rows * d + (long long)d * d;
  hipLaunchKernelGGL(permute_kernel, dim3(grid_of(n)), dim3(256), 0, st, rows, d, perm, W, H, Wp,
                     Hp);
  return hipGetLastError();
}

}  // namespace jarq
