// The scalar policy around the attention path (Sec. 3.1 adaptive context management, Sec. 3.2
// denoising cache).  Only the latent dynamics D_t = MSE(z_{t-1}, z_{t-2}) touches the GPU: a
// streaming reduction over two latents, bound by HBM.  The rest (moving average, temporal
// window, pose-similarity gate, model-call schedule) is scalar host code.
//
// The reduction is deterministic: pass 1 runs a grid that depends only on n, each thread adds
// the squared differences of fixed 16-byte chunks (fp32 inside a chunk, fp64 across chunks),
// the workgroup reduces its threads in a fixed tree and writes one fp64 partial; pass 2 (one
// workgroup) adds the partials in a fixed order and divides by n.
#include <math.h>

#include "la_internal.h"

namespace la {
namespace {

constexpr int kMseThreads = 256;

// Squared differences of one 16-byte chunk: 4 fp32 or 8 bf16 values.
template <bool BF16>
__device__ inline float chunk_sq(u32x4 a, u32x4 b) {
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (BF16) {
      const float d0 = __uint_as_float(a[e] << 16) - __uint_as_float(b[e] << 16);
      const float d1 = __uint_as_float(a[e] & 0xffff0000u) - __uint_as_float(b[e] & 0xffff0000u);
      s = fmaf(d0, d0, s);
      s = fmaf(d1, d1, s);
    } else {
      const float d = __uint_as_float(a[e]) - __uint_as_float(b[e]);
      s = fmaf(d, d, s);
    }
  }
  return s;
}

__device__ inline float elem(const void* p, int64_t i, bool bf16) {
  if (bf16) return __uint_as_float((uint32_t)((const uint16_t*)p)[i] << 16);
  return ((const float*)p)[i];
}

// Fixed-order sum of one double per thread; thread 0 gets the total.
__device__ inline double block_sum(double x) {
  __shared__ double red[kMseThreads / 64];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = x;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < kMseThreads / 64; ++w) t += red[w];
  return t;
}

// Pass 1: chunk c (16 bytes) goes to thread (c mod G) of the grid, G = gridDim.x threads per
// block times blocks; each lane has UNROLL chunk loads in flight (non-temporal: both latents are
// read once).  The n % W trailing values (W values per chunk) are added by the first threads of
// workgroup 0.
template <bool BF16>
__global__ __launch_bounds__(kMseThreads) void mse_partial_kernel(const void* __restrict__ a,
                                                                  const void* __restrict__ b, int64_t n,
                                                                  double* __restrict__ partial) {
  constexpr int W = BF16 ? 8 : 4;
  constexpr int UNROLL = 4;
  const int64_t nchunk = n / W;
  const int64_t G = (int64_t)gridDim.x * kMseThreads;
  const int64_t g = (int64_t)blockIdx.x * kMseThreads + threadIdx.x;
  const u32x4* va = (const u32x4*)a;
  const u32x4* vb = (const u32x4*)b;
  double acc = 0.0;
  int64_t c = g;
  for (; c + (UNROLL - 1) * G < nchunk; c += UNROLL * G) {
    u32x4 x[UNROLL], y[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      x[u] = __builtin_nontemporal_load(va + c + u * G);
      y[u] = __builtin_nontemporal_load(vb + c + u * G);
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc += (double)chunk_sq<BF16>(x[u], y[u]);
  }
  for (; c < nchunk; c += G) acc += (double)chunk_sq<BF16>(va[c], vb[c]);
  if (blockIdx.x == 0 && threadIdx.x < n - nchunk * W) {
    const int64_t i = nchunk * W + threadIdx.x;
    const float d = elem(a, i, BF16) - elem(b, i, BF16);
    acc += (double)(d * d);
  }
  const double t = block_sum(acc);
  if (threadIdx.x == 0) partial[blockIdx.x] = t;
}

// Pass 2: partial p goes to thread p mod 256, in increasing p; then the fixed block tree.
__global__ __launch_bounds__(kMseThreads) void mse_final_kernel(const double* __restrict__ partial, int nb,
                                                                int64_t n, double* __restrict__ out) {
  double acc = 0.0;
  for (int p = threadIdx.x; p < nb; p += kMseThreads) acc += partial[p];
  const double t = block_sum(acc);
  if (threadIdx.x == 0) out[0] = t / (double)n;
}

}  // namespace

int mse_blocks(int64_t n, int bf16) {
  const int64_t nchunk = n / (bf16 ? 8 : 4);
  const int64_t want = (nchunk + 4 * kMseThreads - 1) / (4 * kMseThreads);
  return (int)(want < 1 ? 1 : (want > kMseMaxBlocks ? kMseMaxBlocks : want));
}

hipError_t launch_latent_mse(const void* a, const void* b, int64_t n, int bf16, double* out, void* ws,
                             hipStream_t st) {
  const int nb = mse_blocks(n, bf16);
  double* partial = (double*)ws;
  if (bf16)
    hipLaunchKernelGGL(mse_partial_kernel<true>, dim3(nb), dim3(kMseThreads), 0, st, a, b, n, partial);
  else
    hipLaunchKernelGGL(mse_partial_kernel<false>, dim3(nb), dim3(kMseThreads), 0, st, a, b, n, partial);
  hipLaunchKernelGGL(mse_final_kernel, dim3(1), dim3(kMseThreads), 0, st, partial, nb, n, out);
  return hipGetLastError();
}

}  // namespace la
