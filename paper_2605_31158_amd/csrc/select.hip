// Block selection on gfx950 (Sec. 3.3: pooled proxies, block relevance scores, retained set).
//
// Three launches per call, all on the caller's stream:
//   pool_q        one wave per (head, query block): mean of the block's valid rows
//                 -> q_bar fp32 [BH, NQ, d] (workspace).  Streaming read, every load of a
//                 lane in flight at once.
//   pool_k_score  one workgroup per (head, group of G <= 32 historical key blocks): each wave pools
//                 whole blocks into LDS (never written out), then the workgroup scores the
//                 G pooled keys against every pooled query of the head with fp32 MFMA
//                 (v_mfma_f32_16x16x4_f32) -> s fp32 [BH, NQ, M] (workspace).  The K read is
//                 the dominant cost of selection; it is one coalesced streaming pass of
//                 non-temporal loads.
//   select_rows   one wave per (head, query block), no workgroup barriers: softmax over the
//                 M scores, then a radix select over the 32-bit order keys of the scores (4
//                 passes of 8 bits, per-wave LDS histogram) that finds the score at which the
//                 mass, accumulated from the highest score down, first reaches tau (or the
//                 count reaches the top-k size).  Masses are integer weights (2^48 exp(s - max),
//                 64-bit), so the sums are exact and independent of summation order, and the
//                 cutoff is taken from the weight left out, which stays accurate for tau near 1.
//                 Equal scores at the cutoff are taken in ascending block order.  The kept set is merged with the
//                 forced blocks and emitted, ascending, with lane ballots: mask row, count, list.
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

// Sums the `rows` valid rows of one block (rows x D bf16, row-major at `base`) with one wave.
// Lane l owns 16-byte chunk l % CH of rows l / CH + RG * r; every lane's loads are issued
// before any is consumed.  On return every lane holds the column sums of its chunk (8 floats).
// NT: non-temporal loads, for data read once per call (the historical keys, hundreds of MB):
// the stream then does not displace what the caches hold for the passes that follow.
template <int D, int BLOCK, bool NT = false>
__device__ inline void wave_block_sum(const uint16_t* __restrict__ base, int rows, float* a) {
  constexpr int CH = D / 8;           // chunks per row
  constexpr int RG = 64 / CH;         // row groups per wave
  constexpr int NL = BLOCK / RG;      // loads per lane
  constexpr int BATCH = NL > 16 ? 16 : NL;
  const int lane = threadIdx.x & 63;
  const int ch = lane % CH, rg = lane / CH;
#pragma unroll
  for (int e = 0; e < 8; ++e) a[e] = 0.f;
#pragma unroll
  for (int b0 = 0; b0 < NL; b0 += BATCH) {
    u32x4 w[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int r = rg + RG * (b0 + u);
      const u32x4* p = (const u32x4*)(base + (size_t)r * D + ch * 8);
      w[u] = r >= rows ? u32x4{0u, 0u, 0u, 0u} : NT ? __builtin_nontemporal_load(p) : *p;
    }
#pragma unroll
    for (int u = 0; u < BATCH; ++u) acc_bf16x8(a, w[u]);
  }
#pragma unroll
  for (int off = CH; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] += __shfl_xor(a[e], off);
}

// ---------------------------------------------------------------------------
// pooled blocks (the queries here; any [BH, L, D] tensor through launch_pool_blocks): one wave per
// block

template <int D, int BLOCK>
__global__ __launch_bounds__(kThreads) void pool_q_kernel(const uint16_t* __restrict__ q,
                                                          float* __restrict__ qbar, int Lq, int NQ) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = blockIdx.x * (kThreads / 64) + wave;
  const int bh = blockIdx.y;
  if (i >= NQ) return;
  const int row0 = i * BLOCK;
  const int rows = min(BLOCK, Lq - row0);
  float a[8];
  wave_block_sum<D, BLOCK>(q + ((size_t)bh * Lq + row0) * D, rows, a);
  constexpr int CH = D / 8;
  if (lane < CH) {
    const float inv = 1.0f / (float)rows;
    float* dst = qbar + ((size_t)bh * NQ + i) * D + lane * 8;
    *(f32x4*)dst = f32x4{a[0] * inv, a[1] * inv, a[2] * inv, a[3] * inv};
    *(f32x4*)(dst + 4) = f32x4{a[4] * inv, a[5] * inv, a[6] * inv, a[7] * inv};
  }
}

// ---------------------------------------------------------------------------
// pooled historical keys, scored against every pooled query of the head (fp32 MFMA)

constexpr int kPadF = 4;        // fp32 row padding in LDS (rows 16-B aligned, banks spread)
constexpr int kQChunk = 64;     // pooled-query rows staged in LDS at a time

__device__ inline f32x4 mfma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

constexpr int kScoreThreads = 512;   // 8 waves: one pooled block in flight per wave

// POOLED: the key means come in as kbar fp32 [BH, NK, D] (pooled by the caller) instead of
// being pooled here from k bf16 [BH, Lk, D].
template <int D, int BLOCK, int GB, bool POOLED>
__global__ __launch_bounds__(kScoreThreads) void pool_k_score_kernel(const void* __restrict__ kin,
                                                                const float* __restrict__ qbar,
                                                                float* __restrict__ scores, int Lk, int NK, int NQ,
                                                                int h0, int M, int G, float inv_sqrt_d) {
  constexpr int LD = D + kPadF;
  __shared__ __attribute__((aligned(16))) float kb[GB][LD];
  __shared__ __attribute__((aligned(16))) float qb[kQChunk][LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = blockIdx.y;
  const int m0 = blockIdx.x * G;               // G <= GB key blocks per workgroup
  const int gcount = min(G, M - m0);
  const int gpad = (gcount + 15) & ~15;          // rows of kb the MFMA tiles read
  constexpr int CH = D / 8;
  const float inv_block = 1.0f / (float)BLOCK;
  const uint16_t* __restrict__ k = (const uint16_t*)kin;
  const float* __restrict__ kbar = (const float*)kin;
  for (int g = wave; g < gpad; g += kScoreThreads / 64) {
    if (POOLED) {
      if (lane < D / 4) {
        f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f};
        if (g < gcount) x = *(const f32x4*)(kbar + ((size_t)bh * NK + h0 + m0 + g) * D + lane * 4);
        *(f32x4*)&kb[g][lane * 4] = x;
      }
    } else if (g < gcount) {
      const int j = h0 + m0 + g;   // historical blocks are whole: no ragged rows
      float a[8];
      wave_block_sum<D, BLOCK, true>(k + ((size_t)bh * Lk + (size_t)j * BLOCK) * D, BLOCK, a);
      if (lane < CH) {
        *(f32x4*)&kb[g][lane * 8] = f32x4{a[0] * inv_block, a[1] * inv_block, a[2] * inv_block, a[3] * inv_block};
        *(f32x4*)&kb[g][lane * 8 + 4] = f32x4{a[4] * inv_block, a[5] * inv_block, a[6] * inv_block, a[7] * inv_block};
      }
    } else if (lane < CH) {
      *(f32x4*)&kb[g][lane * 8] = f32x4{0.f, 0.f, 0.f, 0.f};
      *(f32x4*)&kb[g][lane * 8 + 4] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
  // S tile [query rows x GB] = q_bar (rows x D) . k_bar^T (D x GB), 16x16 MFMA tiles:
  // lane l supplies A[row l%16][k l/16] and B[k l/16][col l%16]; C rows 4(l/16)+i, col l%16.
  const int CT = gpad / 16;                       // column tiles
  const int NT = (kQChunk / 16) * CT;             // tiles per query chunk
  const int c16 = lane & 15, k4 = lane >> 4;
  for (int i0 = 0; i0 < NQ; i0 += kQChunk) {
    __syncthreads();                              // kb complete / previous chunk consumed
    const int nrows = min(kQChunk, NQ - i0);
    for (int e = tid; e < kQChunk * (D / 4); e += kScoreThreads) {
      const int r = e / (D / 4), c4 = e % (D / 4);
      f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
      if (r < nrows) v = *(const f32x4*)(qbar + ((size_t)bh * NQ + i0 + r) * D + c4 * 4);
      *(f32x4*)&qb[r][c4 * 4] = v;
    }
    __syncthreads();
    for (int t = wave; t < NT; t += kScoreThreads / 64) {
      const int rt = t / CT, ct = t % CT;
      if (16 * rt >= nrows) continue;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
      for (int kk = 0; kk < D; kk += 4)
        acc = mfma_f32(qb[16 * rt + c16][kk + k4], kb[16 * ct + c16][kk + k4], acc);
      const int col = 16 * ct + c16;
      if (col < gcount) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 16 * rt + 4 * k4 + i;
          if (r < nrows) scores[((size_t)bh * NQ + i0 + r) * M + m0 + col] = acc[i] * inv_sqrt_d;
        }
      }
    }
  }
}

// Order key: ascending key = score descending.  -0 and +0 map to the same key.
__device__ inline uint32_t order_key(float s) {
  if (s == 0.0f) s = 0.0f;
  uint32_t u = __float_as_uint(s);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);   // monotone increasing in s
  return ~u;
}

// ---------------------------------------------------------------------------
// wave-level helpers (one wave per query-block row: no workgroup barriers)

// Wave-wide reductions (every lane gets the result) and the inclusive scan, with DPP row
// operations and the row-pair / half-wave swaps: no LDS round trip.
template <typename Op>
__device__ inline uint32_t wave_allreduce(uint32_t x, Op op) {
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xb1, 0xf, 0xf, false));    // quad_perm 1,0,3,2
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4e, 0xf, 0xf, false));    // quad_perm 2,3,0,1
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x124, 0xf, 0xf, false));   // row_ror:4
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x128, 0xf, 0xf, false));   // row_ror:8
  const auto r16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);                 // rows 0<->1, 2<->3
  x = op((uint32_t)r16[0], (uint32_t)r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);                 // halves
  return op((uint32_t)r32[0], (uint32_t)r32[1]);
}
__device__ inline float wave_max(float x) {
  return __builtin_bit_cast(float, wave_allreduce(__builtin_bit_cast(uint32_t, x), [](uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b)));
  }));
}
__device__ inline uint64_t lanes_below(int lane) { return lane == 0 ? 0ull : (~0ull >> (64 - lane)); }

// All LDS operations this wave issued have completed before the next one starts.
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
}

// Emits the forced block range [lo, hi) at list position pos (mask bytes set to 1).
__device__ inline void emit_range(int lo, int hi, int pos, uint8_t* mask_row, int32_t* idx_row) {
  const int lane = threadIdx.x & 63;
  for (int j = lo + lane; j < hi; j += 64) {
    idx_row[pos + (j - lo)] = j;
    if (mask_row) mask_row[j] = 1;
  }
}

constexpr float kLog2e = 1.4426950408889634f;
// Weights of the tau rule: exp(s - max) in (0, 1] scaled by 2^48 and truncated, so a row of at most
// 4096 candidates sums below 2^60 and a candidate whose mass is above ~M 2^-48 keeps a weight.
constexpr float kWScale = 281474976710656.0f;   // 2^48

__device__ inline uint32_t wave_sum_u32(uint32_t x) {
  return wave_allreduce(x, [](uint32_t a, uint32_t b) { return a + b; });
}
__device__ inline uint32_t wave_min_u32(uint32_t x) {
  return wave_allreduce(x, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}
__device__ inline uint32_t wave_max_u32(uint32_t x) {
  return wave_allreduce(x, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}
__device__ inline uint64_t wave_sum_u64(uint64_t x) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) x += __shfl_xor(x, off);
  return x;
}
// inclusive prefix sum over the 64 lanes
__device__ inline uint64_t wave_incl_scan_u64(uint64_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}
__device__ inline uint64_t read_lane_u64(uint64_t x, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// One wave per (head, query block).  Lane l holds candidates m = l + 64 j, j < NPER.
// Each candidate carries an integer weight: floor(2^48 exp(s - max)) for the tau rule, 1 for the
// top-k rule.  The kept set is the shortest prefix in score order whose weight reaches a target
// T: for the tau rule T = W - floor((1 - tau) W) with W the row's total weight, i.e. the prefix
// reaches tau exactly when the weight it leaves out is at most (1 - tau) W.  Taking the cutoff
// from the dropped tail keeps it accurate for tau near 1, where the tail is tiny but each weight
// in it still has ~24 significant bits.  The sums are exact integers, so they do not depend on
// summation order (deterministic).
template <int NPER>
__global__ __launch_bounds__(kThreads) void select_rows_kernel(const float* __restrict__ scores, int NQ,
                                                               int NK, int M, int h0, int h1, float tau,
                                                               int keep_fixed, uint8_t* __restrict__ mask,
                                                               int32_t* __restrict__ counts,
                                                               int32_t* __restrict__ idx) {
  __shared__ unsigned long long hist_all[kThreads / 64][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = blockIdx.x * (kThreads / 64) + wave;
  const int bh = blockIdx.y;
  if (i >= NQ) return;
  unsigned long long* hist = hist_all[wave];
  const size_t row = (size_t)bh * NQ + i;
  const float* s = scores + row * (size_t)M;
  uint8_t* mask_row = mask ? mask + row * (size_t)NK : nullptr;
  int32_t* idx_row = idx + row * (size_t)NK;

  uint32_t uk[NPER];    // order keys
  uint64_t w[NPER];     // weights
  bool keep_all = keep_fixed < 0 ? tau >= 1.0f : keep_fixed >= M;
  uint64_t target = 0;
  {
    float sv[NPER];
#pragma unroll
    for (int j = 0; j < NPER; ++j) {
      const int m = lane + 64 * j;
      sv[j] = m < M ? s[m] : -FLT_MAX;
    }
    if (!keep_all) {
      if (keep_fixed >= 0) {
#pragma unroll
        for (int j = 0; j < NPER; ++j) w[j] = (lane + 64 * j < M) ? 1u : 0u;
        target = (uint64_t)keep_fixed;
      } else {
        // exp(s - max) = 2^((s - max) log2 e) <= 1, the top candidate's weight is 2^48
        float mx = -FLT_MAX;
#pragma unroll
        for (int j = 0; j < NPER; ++j) mx = fmaxf(mx, sv[j]);
        mx = wave_max(mx);
        uint64_t wl = 0;
#pragma unroll
        for (int j = 0; j < NPER; ++j) {
          const float e = (lane + 64 * j < M) ? __builtin_amdgcn_exp2f((sv[j] - mx) * kLog2e) : 0.f;
          w[j] = (uint64_t)(e * kWScale);
          wl += w[j];
        }
        const uint64_t total = wave_sum_u64(wl);
        // 1 - tau is exact in double; the product's rounding moves the limit by < 2^8 of the
        // total's 2^48-per-unit-mass scale
        const double drop = floor((1.0 - (double)tau) * (double)total);
        const uint64_t dmax = drop <= 0.0 ? 0ull : (drop >= (double)total ? total : (uint64_t)drop);
        target = total - dmax;
        if (target == 0) target = 1;     // any tau > 0 keeps at least the top candidate
      }
      uint64_t wl = 0;
#pragma unroll
      for (int j = 0; j < NPER; ++j) wl += w[j];
      if (wave_sum_u64(wl) < target) keep_all = true;   // the count never reaches the target
    }
#pragma unroll
    for (int j = 0; j < NPER; ++j) uk[j] = order_key(sv[j]);
  }
  // cutoff: smallest order key u* whose inclusive weight reaches the target (radix select,
  // passes of 8 bits over a per-wave 256-bin histogram; after the second pass, a crossing bin
  // whose candidates all share one key ends the search), then equal keys by block index
  uint32_t ustar = 0xffffffffu;
  int mstar = 0x7fffffff;
  const bool none = !keep_all && target == 0;
  if (!keep_all && !none) {
    uint32_t prefix = 0;
    uint64_t before = 0;
    bool found = false;
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
#pragma unroll
      for (int t = 0; t < 4; ++t) hist[4 * lane + t] = 0;
      wave_lds_sync();
#pragma unroll
      for (int j = 0; j < NPER; ++j) {
        const bool in = w[j] != 0 && (pass == 0 || (uk[j] >> (shift + 8)) == prefix);
        if (in) atomicAdd(&hist[(uk[j] >> shift) & 255u], (unsigned long long)w[j]);
      }
      wave_lds_sync();
      uint64_t b4[4];
      uint64_t loc = 0;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        loc += hist[4 * lane + t];
        b4[t] = loc;
      }
      const uint64_t excl = wave_incl_scan_u64(loc) - loc;
      int hit = -1;
#pragma unroll
      for (int t = 3; t >= 0; --t)
        if (before + excl + b4[t] >= target) hit = t;
      const unsigned long long bal = __ballot(hit >= 0);
      const int first = __ffsll(bal) - 1;              // lane holding the crossing bin
      const uint64_t below = before + excl + (hit > 0 ? b4[hit > 0 ? hit - 1 : 0] : 0);
      const int bin = 4 * lane + hit;
      prefix = (prefix << 8) | (uint32_t)__builtin_amdgcn_readlane(bin, first);
      before = read_lane_u64(below, first);
      if (pass == 1) {
        uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
        for (int j = 0; j < NPER; ++j) {
          if (w[j] != 0 && (uk[j] >> shift) == prefix) {
            kmin = min(kmin, uk[j]);
            kmax = max(kmax, uk[j]);
          }
        }
        kmin = wave_min_u32(kmin);
        if (kmin == wave_max_u32(kmax)) {
          ustar = kmin;
          found = true;
          break;
        }
      }
    }
    if (!found) ustar = prefix;
    int ntie = 0;
#pragma unroll
    for (int j = 0; j < NPER; ++j) ntie += (w[j] != 0 && uk[j] == ustar) ? 1 : 0;
    if (wave_sum_u32((uint32_t)ntie) > 1) {
      // equal scores at the cutoff: take them in ascending block order until the target
      uint64_t base = before;
#pragma unroll
      for (int j = 0; j < NPER; ++j) {
        const uint64_t wt = (w[j] != 0 && uk[j] == ustar) ? w[j] : 0;
        const uint64_t incl = wave_incl_scan_u64(wt);
        const bool cross = wt != 0 && base + incl >= target && base + incl - wt < target;
        const unsigned long long bal = __ballot(cross);
        if (bal) {
          mstar = 64 * j + __ffsll(bal) - 1;
          break;
        }
        base += read_lane_u64(incl, 63);
      }
    }
  }
  // emit: forced head, kept historical blocks (ascending), forced tail
  emit_range(0, h0, 0, mask_row, idx_row);
  int pos = h0;
#pragma unroll
  for (int j = 0; j < NPER; ++j) {
    const int m = lane + 64 * j;
    bool kept = false;
    if (m < M) {
      if (keep_all) kept = true;
      else if (!none) kept = w[j] != 0 && (uk[j] < ustar || (uk[j] == ustar && m <= mstar));
      if (mask_row) mask_row[h0 + m] = kept ? 1 : 0;
    }
    const unsigned long long bal = __ballot(kept);
    if (kept) idx_row[pos + __popcll(bal & lanes_below(lane))] = h0 + m;
    pos += __popcll(bal);
  }
  emit_range(h1, NK, pos, mask_row, idx_row);
  if (lane == 0) counts[row] = pos + (NK - h1);
}

// One wave per (head, query block): compacts a mask row into the ascending list.
__global__ __launch_bounds__(kThreads) void mask_to_list_kernel(const uint8_t* __restrict__ mask, int NQ,
                                                                int NK, int32_t* __restrict__ counts,
                                                                int32_t* __restrict__ idx) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i = blockIdx.x * (kThreads / 64) + wave;
  if (i >= NQ) return;
  const size_t row = (size_t)blockIdx.y * NQ + i;
  const uint8_t* mr = mask + row * (size_t)NK;
  int32_t* idx_row = idx + row * (size_t)NK;
  int pos = 0;
  for (int j0 = 0; j0 < NK; j0 += 64) {
    const int j = j0 + lane;
    const bool kept = j < NK && mr[j] != 0;
    const unsigned long long bal = __ballot(kept);
    if (kept) idx_row[pos + __popcll(bal & lanes_below(lane))] = j;
    pos += __popcll(bal);
  }
  if (lane == 0) counts[row] = pos;
}

// Scores of the pooled keys (pooled here from k, or given as kbar when POOLED) against qbar.
// Key blocks per workgroup when the keys are pooled here: the grid should fill the resident
// workgroup slots of the device
// (about three per CU, LDS-bound) in as few, as full rounds as possible: G = blocks / (rounds x
// slots), at most 32 (the LDS tile) and at least 8 (each workgroup stages the head's pooled
// queries once), so that no round runs on a fraction of the CUs.
inline int score_group(const Dims& dm) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    cus = 256;
  const int64_t slots = 3 * (int64_t)cus;
  const int64_t blocks = (int64_t)dm.BH * dm.M;
  const int64_t rounds = (blocks + 32 * slots - 1) / (32 * slots);
  const int64_t g = (blocks + rounds * slots - 1) / (rounds * slots);
  return (int)(g < 8 ? 8 : g > 32 ? 32 : g);
}

template <int D, int BLOCK, bool POOLED>
void launch_score(const Dims& dm, const void* kin, const float* qbar, float* scores, hipStream_t st) {
  const float inv_sqrt_d = 1.0f / sqrtf((float)dm.d);
  // pooled means in: the work is the scoring, so fewer, fuller workgroups (32 blocks when that
  // still gives one per CU, else 16)
  const int G = POOLED ? ((int64_t)ceil_div(dm.M, 32) * dm.BH >= 256 ? 32 : 16) : score_group(dm);
  hipLaunchKernelGGL((pool_k_score_kernel<D, BLOCK, 32, POOLED>), dim3(ceil_div(dm.M, G), dm.BH),
                     dim3(kScoreThreads), 0, st, kin, qbar, scores, dm.Lk, dm.NK, dm.NQ, dm.h0, dm.M, G, inv_sqrt_d);
}

template <int D, int BLOCK>
void launch_pools(const Dims& dm, const void* q, const void* k, float* qbar, float* scores, hipStream_t st) {
  hipLaunchKernelGGL((pool_q_kernel<D, BLOCK>), dim3(ceil_div(dm.NQ, kThreads / 64), dm.BH), dim3(kThreads), 0,
                     st, (const uint16_t*)q, qbar, dm.Lq, dm.NQ);
  launch_score<D, BLOCK, false>(dm, k, qbar, scores, st);
}

float* scores_ws(const Dims& dm, void* ws) {
  return (float*)((char*)ws + align256((size_t)dm.BH * dm.NQ * dm.d * sizeof(float)));
}

hipError_t launch_rows(const Dims& dm, const float* scores, float tau, int keep_fixed, uint8_t* mask,
                       int32_t* counts, int32_t* idx, hipStream_t st) {
  const dim3 grid(ceil_div(dm.NQ, kThreads / 64), dm.BH);
#define LA_SELECT(NPER)                                                                                      \
  hipLaunchKernelGGL(select_rows_kernel<NPER>, grid, dim3(kThreads), 0, st, scores, dm.NQ, dm.NK, dm.M, dm.h0, \
                     dm.h1, tau, keep_fixed, mask, counts, idx)
  // candidates per lane: the smallest instantiation that holds the row (every phase of the
  // kernel loops over all NPER slots of a lane)
  if (dm.M <= 64 * 4) LA_SELECT(4);
  else if (dm.M <= 64 * 8) LA_SELECT(8);
  else if (dm.M <= 64 * 12) LA_SELECT(12);
  else if (dm.M <= 64 * 16) LA_SELECT(16);
  else if (dm.M <= 64 * 20) LA_SELECT(20);
  else if (dm.M <= 64 * 25) LA_SELECT(25);
  else if (dm.M <= 64 * 32) LA_SELECT(32);
  else if (dm.M <= 64 * 48) LA_SELECT(48);
  else LA_SELECT(64);
#undef LA_SELECT
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const Dims& dm, const void* q, const void* k, float tau, int keep_fixed,
                         uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, hipStream_t st) {
  float* qbar = (float*)ws;
  float* scores = scores_ws(dm, ws);
  if (dm.M > 0) {
    if (dm.d == 128 && dm.block == 64) launch_pools<128, 64>(dm, q, k, qbar, scores, st);
    else if (dm.d == 128) launch_pools<128, 128>(dm, q, k, qbar, scores, st);
    else if (dm.block == 64) launch_pools<64, 64>(dm, q, k, qbar, scores, st);
    else launch_pools<64, 128>(dm, q, k, qbar, scores, st);
  }
  return launch_rows(dm, scores, tau, keep_fixed, mask, counts, idx, st);
}

hipError_t launch_select_pooled(const Dims& dm, const float* qbar, const float* kbar, float tau, int keep_fixed,
                                uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, hipStream_t st) {
  float* scores = scores_ws(dm, ws);
  if (dm.M > 0) {
    if (dm.d == 128) launch_score<128, 64, true>(dm, kbar, qbar, scores, st);
    else launch_score<64, 64, true>(dm, kbar, qbar, scores, st);
  }
  return launch_rows(dm, scores, tau, keep_fixed, mask, counts, idx, st);
}

hipError_t launch_pool_blocks(const Dims& dm, const void* x, int L, int NB, float* xbar, hipStream_t st) {
  const dim3 grid(ceil_div(NB, kThreads / 64), dm.BH);
  const uint16_t* xp = (const uint16_t*)x;
  if (dm.d == 128 && dm.block == 64) hipLaunchKernelGGL((pool_q_kernel<128, 64>), grid, dim3(kThreads), 0, st, xp, xbar, L, NB);
  else if (dm.d == 128) hipLaunchKernelGGL((pool_q_kernel<128, 128>), grid, dim3(kThreads), 0, st, xp, xbar, L, NB);
  else if (dm.block == 64) hipLaunchKernelGGL((pool_q_kernel<64, 64>), grid, dim3(kThreads), 0, st, xp, xbar, L, NB);
  else hipLaunchKernelGGL((pool_q_kernel<64, 128>), grid, dim3(kThreads), 0, st, xp, xbar, L, NB);
  return hipGetLastError();
}

hipError_t launch_mask_to_list(const Dims& dm, const uint8_t* mask, int32_t* counts, int32_t* idx,
                               hipStream_t st) {
  hipLaunchKernelGGL(mask_to_list_kernel, dim3(ceil_div(dm.NQ, kThreads / 64), dm.BH), dim3(kThreads), 0, st,
                     mask, dm.NQ, dm.NK, counts, idx);
  return hipGetLastError();
}

}  // namespace la
