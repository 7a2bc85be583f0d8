// Block selection on gfx950 (Sec. 3.3: pooled proxies, block relevance scores, retained set).
//
// Three launches per call, all on the caller's stream:
//   pool_q        one workgroup per (head, query block): mean of the block's valid rows
//                 -> q_bar fp32 [BH, NQ, d] (workspace).  HBM-bound streaming read.
//   pool_k_score  one workgroup per (head, group of G historical key blocks): pools the G
//                 blocks into LDS (never written out) and immediately scores them against
//                 every q_bar of the head -> s fp32 [BH, NQ, M] (workspace).  The K read
//                 dominates the selection pass; it is a single coalesced streaming pass.
//   select_rows   one workgroup per (head, query block): softmax over the M scores, sort
//                 by (score desc, block asc), prefix scan of the sorted probabilities to
//                 the tau crossing (or a fixed count), merge with the forced blocks and
//                 emit the mask row, the count and the ascending block list.
#include <float.h>
#include <math.h>

#include "la_internal.h"

namespace la {
namespace {

constexpr int kThreads = 256;

__device__ inline void acc_bf16x8(float* a, u32x4 w) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    a[2 * e] += __uint_as_float(w[e] << 16);
    a[2 * e + 1] += __uint_as_float(w[e] & 0xffff0000u);
  }
}

// ---------------------------------------------------------------------------
// pooled queries

template <int D>
__global__ __launch_bounds__(kThreads) void pool_q_kernel(const uint16_t* __restrict__ q,
                                                          float* __restrict__ qbar, int Lq, int block,
                                                          int NQ) {
  constexpr int CH = D / 8;             // 16-byte chunks per row
  constexpr int RPP = kThreads / CH;    // rows one pass of the workgroup covers
  constexpr int MAXIT = 128 / RPP;      // passes for the largest block
  __shared__ float red[kThreads / 64][D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = blockIdx.x, bh = blockIdx.y;
  const int row0 = i * block;
  const int rows = min(block, Lq - row0);
  const int ch = tid % CH, rg = tid / CH;
  const uint16_t* base = q + ((size_t)bh * Lq + row0) * D + ch * 8;
  u32x4 w[MAXIT];
#pragma unroll
  for (int it = 0; it < MAXIT; ++it) {
    const int r = rg + it * RPP;
    if (r < rows) w[it] = *(const u32x4*)(base + (size_t)r * D);
    else w[it] = u32x4{0u, 0u, 0u, 0u};
  }
  float a[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int it = 0; it < MAXIT; ++it) acc_bf16x8(a, w[it]);
#pragma unroll
  for (int off = CH; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] += __shfl_xor(a[e], off);
  if (lane < CH)
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][lane * 8 + e] = a[e];
  __syncthreads();
  if (tid < D) {
    float s = 0.f;
#pragma unroll
    for (int wv = 0; wv < kThreads / 64; ++wv) s += red[wv][tid];
    qbar[((size_t)bh * NQ + i) * D + tid] = s / (float)rows;
  }
}

// ---------------------------------------------------------------------------
// pooled historical keys, scored against every pooled query of the head

template <int D, int G>
__global__ __launch_bounds__(kThreads) void pool_k_score_kernel(const uint16_t* __restrict__ k,
                                                                const float* __restrict__ qbar,
                                                                float* __restrict__ scores, int Lk,
                                                                int block, int NQ, int h0, int M,
                                                                float inv_sqrt_d) {
  constexpr int CH = D / 8;        // chunks per row
  constexpr int RG = 64 / CH;      // row groups inside one wave
  __shared__ float kbar[G][D];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = blockIdx.y;
  const int m0 = blockIdx.x * G;
  const int gcount = min(G, M - m0);
  const int ch = lane % CH, rg = lane / CH;
  const int iters = block / RG;    // multiple of 8 for block 64/128 and d 64/128
  const float inv_block = 1.0f / (float)block;
  for (int g = wave; g < gcount; g += kThreads / 64) {
    const int j = h0 + m0 + g;     // historical blocks are whole: no ragged rows
    const uint16_t* base = k + ((size_t)bh * Lk + (size_t)j * block) * D + ch * 8;
    float a[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int it0 = 0; it0 < iters; it0 += 8) {
      u32x4 w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) w[u] = *(const u32x4*)(base + (size_t)((it0 + u) * RG + rg) * D);
#pragma unroll
      for (int u = 0; u < 8; ++u) acc_bf16x8(a, w[u]);
    }
#pragma unroll
    for (int off = CH; off < 64; off <<= 1)
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] += __shfl_xor(a[e], off);
    if (lane < CH)
#pragma unroll
      for (int e = 0; e < 8; ++e) kbar[g][lane * 8 + e] = a[e] * inv_block;
  }
  __syncthreads();
  const int g = tid % G;
  if (g >= gcount) return;
  const f32x4* kr = (const f32x4*)kbar[g];
  for (int i = tid / G; i < NQ; i += kThreads / G) {
    const f32x4* qr = (const f32x4*)(qbar + ((size_t)bh * NQ + i) * D);
    float s = 0.f;
#pragma unroll 8
    for (int c = 0; c < D / 4; ++c) {
      const f32x4 x = qr[c], y = kr[c];
      s += x[0] * y[0];
      s += x[1] * y[1];
      s += x[2] * y[2];
      s += x[3] * y[3];
    }
    scores[((size_t)bh * NQ + i) * M + m0 + g] = s * inv_sqrt_d;
  }
}

// ---------------------------------------------------------------------------
// workgroup reductions / scans (256 threads, 4 waves)

__device__ inline float wave_max(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Exclusive scan of one int per thread across the workgroup; *total gets the sum.
__device__ inline int block_excl_scan(int x, int* sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int wv = 0; wv < kThreads / 64; ++wv) {
    if (wv < wave) base += sh[wv];
    tot += sh[wv];
  }
  __syncthreads();
  *total = tot;
  return base + incl - x;
}

__device__ inline float block_excl_scan_f(float x, float* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  float base = 0.f;
#pragma unroll
  for (int wv = 0; wv < kThreads / 64; ++wv)
    if (wv < wave) base += sh[wv];
  __syncthreads();
  return base + incl - x;
}

// Sort key: ascending key order = score descending, then candidate index ascending.
__device__ inline uint64_t sort_key(float s, int m) {
  if (s == 0.0f) s = 0.0f;                      // -0 and +0 compare equal
  uint32_t u = __float_as_uint(s);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);   // monotone in s
  return ((uint64_t)(~u) << 32) | (uint32_t)m;
}

// Writes the mask row (optional), the ascending kept list and its length from the
// per-block flags in LDS.
__device__ inline void emit_row(const uint8_t* flag, int NK, uint8_t* mask_row, int32_t* idx_row,
                                int32_t* count, int* sh_i) {
  const int tid = threadIdx.x;
  const int per = (NK + kThreads - 1) / kThreads;
  const int lo = min(tid * per, NK), hi = min(lo + per, NK);
  int cnt = 0;
  for (int j = lo; j < hi; ++j) cnt += flag[j];
  int total;
  int pos = block_excl_scan(cnt, sh_i, &total);
  for (int j = lo; j < hi; ++j)
    if (flag[j]) idx_row[pos++] = j;
  if (tid == 0) *count = total;
  if (mask_row)
    for (int j = tid; j < NK; j += kThreads) mask_row[j] = flag[j];
}

__global__ __launch_bounds__(kThreads) void select_rows_kernel(const float* __restrict__ scores, int NQ,
                                                               int NK, int M, int P, int h0, int h1,
                                                               float tau, int keep_fixed,
                                                               uint8_t* __restrict__ mask,
                                                               int32_t* __restrict__ counts,
                                                               int32_t* __restrict__ idx) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* keys = (uint64_t*)smem;                 // [P]
  float* prob = (float*)(keys + P);                 // [P], indexed by candidate
  uint8_t* flag = (uint8_t*)(prob + P);             // [NK]
  __shared__ float sh_f[kThreads / 64];
  __shared__ int sh_i[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = blockIdx.x, bh = blockIdx.y;
  const size_t row = (size_t)bh * NQ + i;
  const float* s = scores + row * (size_t)M;

  for (int j = tid; j < NK; j += kThreads) flag[j] = (j < h0 || j >= h1) ? 1 : 0;
  if (M > 0) {
    // softmax over the M candidates
    float mx = -FLT_MAX;
    for (int m = tid; m < M; m += kThreads) mx = fmaxf(mx, s[m]);
    mx = wave_max(mx);
    if (lane == 0) sh_f[wave] = mx;
    __syncthreads();
    mx = sh_f[0];
#pragma unroll
    for (int wv = 1; wv < kThreads / 64; ++wv) mx = fmaxf(mx, sh_f[wv]);
    __syncthreads();
    float sum = 0.f;
    for (int m = tid; m < M; m += kThreads) {
      const float e = expf(s[m] - mx);
      prob[m] = e;
      sum += e;
    }
    sum = wave_sum(sum);
    if (lane == 0) sh_f[wave] = sum;
    __syncthreads();
    sum = 0.f;
#pragma unroll
    for (int wv = 0; wv < kThreads / 64; ++wv) sum += sh_f[wv];
    for (int m = tid; m < P; m += kThreads) {
      if (m < M) {
        prob[m] = prob[m] / sum;
        keys[m] = sort_key(s[m], m);
      } else {
        keys[m] = ~(uint64_t)0;
      }
    }
    __syncthreads();
    // bitonic sort, ascending keys
    for (int kk = 2; kk <= P; kk <<= 1) {
      for (int jj = kk >> 1; jj > 0; jj >>= 1) {
        for (int t = tid; t < (P >> 1); t += kThreads) {
          const int a = (t / jj) * 2 * jj + (t % jj);
          const int b = a + jj;
          const uint64_t x = keys[a], y = keys[b];
          const bool up = (a & kk) == 0;
          if ((x > y) == up) {
            keys[a] = y;
            keys[b] = x;
          }
        }
        __syncthreads();
      }
    }
    int kstar;
    if (keep_fixed >= 0) {
      kstar = min(keep_fixed, M);
    } else if (tau >= 1.0f) {
      kstar = M;
    } else {
      // cumulative mass over ranks; first rank whose inclusive sum reaches tau
      const int per = (M + kThreads - 1) / kThreads;
      const int lo = min(tid * per, M), hi = min(lo + per, M);
      float local = 0.f;
      for (int r = lo; r < hi; ++r) local += prob[(uint32_t)keys[r]];
      float run = block_excl_scan_f(local, sh_f);
      int first = M;
      for (int r = lo; r < hi; ++r) {
        run += prob[(uint32_t)keys[r]];
        if (run >= tau) {
          first = r;
          break;
        }
      }
      // workgroup minimum
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) first = min(first, __shfl_xor(first, off));
      if (lane == 0) sh_i[wave] = first;
      __syncthreads();
      first = sh_i[0];
#pragma unroll
      for (int wv = 1; wv < kThreads / 64; ++wv) first = min(first, sh_i[wv]);
      __syncthreads();
      kstar = (first < M) ? first + 1 : M;
    }
    for (int r = tid; r < kstar; r += kThreads) flag[h0 + (int)(uint32_t)keys[r]] = 1;
  }
  __syncthreads();
  emit_row(flag, NK, mask ? mask + row * (size_t)NK : nullptr, idx + row * (size_t)NK, counts + row, sh_i);
}

__global__ __launch_bounds__(kThreads) void mask_to_list_kernel(const uint8_t* __restrict__ mask, int NQ,
                                                                int NK, int32_t* __restrict__ counts,
                                                                int32_t* __restrict__ idx) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint8_t* flag = (uint8_t*)smem;
  __shared__ int sh_i[kThreads / 64];
  const size_t row = (size_t)blockIdx.y * NQ + blockIdx.x;
  const uint8_t* mr = mask + row * (size_t)NK;
  for (int j = threadIdx.x; j < NK; j += kThreads) flag[j] = mr[j] ? 1 : 0;
  __syncthreads();
  emit_row(flag, NK, nullptr, idx + row * (size_t)NK, counts + row, sh_i);
}

int next_pow2(int x) {
  int p = 2;
  while (p < x) p <<= 1;
  return p;
}

}  // namespace

hipError_t launch_select(const Dims& dm, const void* q, const void* k, float tau, int keep_fixed,
                         uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, hipStream_t st) {
  float* qbar = (float*)ws;
  float* scores = (float*)((char*)ws + align256((size_t)dm.BH * dm.NQ * dm.d * sizeof(float)));
  const float inv_sqrt_d = 1.0f / sqrtf((float)dm.d);
  constexpr int G = 8;
  if (dm.M > 0) {
    dim3 gq(dm.NQ, dm.BH), gk(ceil_div(dm.M, G), dm.BH);
    if (dm.d == 128) {
      hipLaunchKernelGGL(pool_q_kernel<128>, gq, dim3(kThreads), 0, st, (const uint16_t*)q, qbar, dm.Lq,
                         dm.block, dm.NQ);
      hipLaunchKernelGGL((pool_k_score_kernel<128, G>), gk, dim3(kThreads), 0, st, (const uint16_t*)k, qbar,
                         scores, dm.Lk, dm.block, dm.NQ, dm.h0, dm.M, inv_sqrt_d);
    } else {
      hipLaunchKernelGGL(pool_q_kernel<64>, gq, dim3(kThreads), 0, st, (const uint16_t*)q, qbar, dm.Lq,
                         dm.block, dm.NQ);
      hipLaunchKernelGGL((pool_k_score_kernel<64, G>), gk, dim3(kThreads), 0, st, (const uint16_t*)k, qbar,
                         scores, dm.Lk, dm.block, dm.NQ, dm.h0, dm.M, inv_sqrt_d);
    }
  }
  const int P = dm.M > 0 ? next_pow2(dm.M) : 0;
  const size_t shmem = (size_t)P * (sizeof(uint64_t) + sizeof(float)) + (size_t)((dm.NK + 15) & ~15);
  hipLaunchKernelGGL(select_rows_kernel, dim3(dm.NQ, dm.BH), dim3(kThreads), shmem, st, scores, dm.NQ, dm.NK,
                     dm.M, P, dm.h0, dm.h1, tau, keep_fixed, mask, counts, idx);
  return hipGetLastError();
}

hipError_t launch_mask_to_list(const Dims& dm, const uint8_t* mask, int32_t* counts, int32_t* idx,
                               hipStream_t st) {
  const size_t shmem = (size_t)((dm.NK + 15) & ~15);
  hipLaunchKernelGGL(mask_to_list_kernel, dim3(dm.NQ, dm.BH), dim3(kThreads), shmem, st, mask, dm.NQ, dm.NK,
                     counts, idx);
  return hipGetLastError();
}

}  // namespace la
