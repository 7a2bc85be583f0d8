// Block-sparse attention forward on gfx950 (Sec. 3.3: attention over C_i = T u K^curr u S_i,
// one kept-block list per query block serving both K and V).
//
// Work decomposition
//   * A workgroup (4 waves) owns 128 consecutive query rows of one (batch, head): two query
//     blocks of 64 rows, or one of 128.  Each wave owns 32 rows, all inside one query block.
//   * The workgroup walks the union of its query blocks' kept lists in ascending block
//     order (a two-pointer merge over the sorted lists).  Every kept block is staged once in
//     LDS and consumed by the waves whose query block kept it; the other waves only help
//     load.  Forced (chunk) blocks are kept by every query block, so most tiles are shared.
//   * Key blocks are consumed in 64-key sub-tiles, staged by asynchronous direct-to-LDS
//     16-byte loads into a double buffer: sub-tile t+1 streams in while sub-tile t is
//     multiplied, with one workgroup barrier per sub-tile.
//   * Workgroup ids are remapped so that each XCD (each L2) works on consecutive (head,
//     row tile) units: the kept K/V blocks of a head stay hot in one XCD's L2.
//   * Few work units (small problems) split the key-block range across workgroups; the
//     partial (O, m, l) are merged by attn_combine (log-sum-exp merge).
//
// Per wave and 64-key sub-tile (d = 128):
//   S^T (64 keys x 32 queries) = K_tile (64 x d) . Q^T       32 x v_mfma_f32_16x16x32_bf16
//   online softmax over keys (fp32, base 2; the running max is only raised when a tile's
//   max exceeds it by more than 2^8, so most tiles skip the rescale of O)
//   O^T (d x 32) += V^T (d x 64) . P^T (64 x 32)              32 x v_mfma_f32_16x16x32_bf16
// S^T is computed transposed so that its accumulator layout (each lane holds 4 consecutive
// keys of one query column) is directly the B operand of the P.V product.  K and V tiles are
// row-major in LDS with a per-row XOR swizzle of the 16-byte chunks (conflict-free operand
// reads); the V^T operand is read with the LDS transpose load ds_read_b64_tr_b16.
#include <math.h>

#include "la_internal.h"

namespace la {
namespace {

constexpr int kThreads = 256;
constexpr int KT = 64;          // keys per sub-tile
constexpr int QW = 32;          // query rows per wave
constexpr int QR = 128;         // query rows per workgroup
constexpr int kEnd = 0x7fffffff;
constexpr float kRescaleSlack = 8.0f;   // log2 headroom before the running max is raised

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Per-row XOR swizzle of the 16-byte chunks of a tile row.  Chosen so that (a) the 16 rows
// one MFMA operand read touches map a fixed chunk to 16 distinct bank groups and (b) the
// transpose reads of V (8 rows x 2 adjacent chunks per half-wave) are conflict-free.
template <int D>
__device__ inline int swz(int r) {
  if constexpr (D == 128) return ((r & 7) << 1) | ((r >> 3) & 1);
  else return (((r >> 1) & 3) << 1) | ((r >> 3) & 1);
}

template <int D>
struct Tile {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int ROWB = D * 2;               // bytes per row
  static constexpr int RPI = 64 / CH;              // rows one wave-wide 1 KiB load covers
  static constexpr int NI = KT / (RPI * 4);        // loads per thread per matrix per sub-tile
  static constexpr int BYTES = KT * ROWB;          // one matrix sub-tile
};

// Issues the direct-to-LDS loads of one K and one V sub-tile (64 keys from key0; rows past
// Lk re-read row Lk-1, their logits are masked).  Lane l of a wave-wide load lands at
// dst + 16 l, so the swizzle is applied by choosing which global chunk each lane fetches.
template <int D>
__device__ inline void issue_tile(unsigned char* kdst, unsigned char* vdst, const uint16_t* __restrict__ kh,
                                  const uint16_t* __restrict__ vh, int key0, int Lk) {
  using T = Tile<D>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int n = 0; n < T::NI; ++n) {
    const int blk = 4 * n + wave;                  // which 1 KiB slab of the sub-tile
    const int r = T::RPI * blk + lane / T::CH;     // tile row of this lane's chunk
    const int p = lane % T::CH;                    // physical chunk slot in the row
    const int c = p ^ swz<D>(r);                   // logical chunk it holds
    int key = key0 + r;
    key = key < Lk ? key : Lk - 1;
    const size_t off = (size_t)key * D + c * 8;
    __builtin_amdgcn_global_load_lds((const void*)(kh + off), LDS_PTR(kdst + blk * 1024), 16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void*)(vh + off), LDS_PTR(vdst + blk * 1024), 16, 0, 0);
  }
}

struct Geom {
  int Lq, Lk, block, NQ, NK, F, chunk0;
};

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ idx, uint16_t* __restrict__ o,
    float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_m,
    float* __restrict__ part_l, Geom gm, int BH, int row_tiles, int splits, int units, float scale_log2) {
  using T = Tile<D>;
  constexpr int KS = D / 32;   // k-steps of Q.K^T
  constexpr int DT = D / 16;   // d tiles of P.V
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2][2][T::BYTES];   // [stage][K|V]

  // XCD-aware id: hardware places consecutive workgroup ids on consecutive XCDs (round
  // robin over 8); give each XCD a contiguous range of logical units.
  const int per_xcd = gridDim.x >> 3;
  const int hw = blockIdx.x;
  const int logical = (hw & 7) * per_xcd + (hw >> 3);
  if (logical >= units) return;
  const int sp = logical % splits;
  const int rt = (logical / splits) % row_tiles;
  const int bh = logical / (splits * row_tiles);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int row_base = rt * QR;
  const int r0w = row_base + wave * QW;                 // first query row of this wave
  const bool two = (gm.block == 64);
  const int qa = row_base / gm.block;
  const int qb = (two && qa + 1 < gm.NQ) ? qa + 1 : -1;
  const bool wave_b = two && wave >= 2;                 // waves 2, 3 own the second block
  const bool wave_rows = r0w < gm.Lq;

  const int32_t* la_ = idx + ((size_t)bh * gm.NQ + qa) * gm.NK;
  const int na = counts[(size_t)bh * gm.NQ + qa];
  const int32_t* lb_ = qb >= 0 ? idx + ((size_t)bh * gm.NQ + qb) * gm.NK : la_;
  const int nb = qb >= 0 ? counts[(size_t)bh * gm.NQ + qb] : 0;

  // split range of key blocks [jlo, jhi)
  const int jlo = (int)((int64_t)gm.NK * sp / splits);
  const int jhi = (int)((int64_t)gm.NK * (sp + 1) / splits);
  int pa = 0, pb = 0;
  if (splits > 1) {
    while (pa < na && la_[pa] < jlo) ++pa;
    while (pb < nb && lb_[pb] < jlo) ++pb;
  }
  int ja = pa < na ? la_[pa] : kEnd;
  int jb = pb < nb ? lb_[pb] : kEnd;

  const uint16_t* kh = k + (size_t)bh * gm.Lk * D;
  const uint16_t* vh = v + (size_t)bh * gm.Lk * D;

  // Q^T operand: lane holds Q[row r0w + 16 qt + c][32 ks + 8 g .. + 7]
  bf16x8 qreg[2][KS];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int row = r0w + 16 * qt + c;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 w = u32x4{0u, 0u, 0u, 0u};
      if (row < gm.Lq) w = *(const u32x4*)(q + ((size_t)bh * gm.Lq + row) * D + 32 * ks + 8 * g);
      qreg[qt][ks] = __builtin_bit_cast(bf16x8, w);
    }
  }
  // frame of each of this lane's two query rows (frame-causal mask)
  int qframe[2] = {0, 0};
  if (gm.F > 0) {
    qframe[0] = (r0w + c) / gm.F;
    qframe[1] = (r0w + 16 + c) / gm.F;
  }
  const int wave_first_frame = gm.F > 0 ? r0w / gm.F : 0;

  f32x4 oacc[DT][2];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt][0] = oacc[dt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY};
  float l_run[2] = {0.f, 0.f};

  const int nsub = gm.block / KT;
  // Merged walk over the two ascending lists: pop() yields the next kept block and which
  // of the two query blocks keep it; blocks at or past jhi end the walk.
  auto pop = [&](int& jj, bool& ua, bool& ub) {
    jj = min(ja, jb);
    if (jj >= jhi) {
      jj = kEnd;
      ua = ub = false;
      return;
    }
    ua = (ja == jj);
    ub = (jb == jj);
    if (ua) { ++pa; ja = pa < na ? la_[pa] : kEnd; }
    if (ub) { ++pb; jb = pb < nb ? lb_[pb] : kEnd; }
  };
  int cj, csub = 0;
  bool cA, cB;
  pop(cj, cA, cB);
  int stage = 0;
  if (cj != kEnd) issue_tile<D>(smem[0][0], smem[0][1], kh, vh, cj * gm.block, gm.Lk);
  while (cj != kEnd) {
    int nj = cj, nsb = csub + 1;
    bool nA = cA, nB = cB;
    if (nsb == nsub) {
      nsb = 0;
      pop(nj, nA, nB);
    }
    // this thread's loads of the current stage are done; the barrier makes every thread's
    // loads visible and guarantees the other stage is no longer being read
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (nj != kEnd)
      issue_tile<D>(smem[stage ^ 1][0], smem[stage ^ 1][1], kh, vh, nj * gm.block + nsb * KT, gm.Lk);
    const int key0 = cj * gm.block + csub * KT;
    const bool mine = (wave_b ? cB : cA) && wave_rows;
    const unsigned char* ks_base = smem[stage][0];
    const unsigned char* vs_base = smem[stage][1];
    if (mine) {
      // ---- S^T = K Q^T ----
      f32x4 sacc[4][2];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) sacc[kt][0] = sacc[kt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          const int r = 16 * kt + c;
          const int slot = (4 * ks + g) ^ swz<D>(r);
          const bf16x8 a = *(const bf16x8*)(ks_base + r * T::ROWB + slot * 16);
          sacc[kt][0] = mfma16(a, qreg[0][ks], sacc[kt][0]);
          sacc[kt][1] = mfma16(a, qreg[1][ks], sacc[kt][1]);
        }
      }
      // ---- masks: keys past Lk (ragged last block), frame-causal pairs in the chunk ----
      bool need_mask = key0 + KT > gm.Lk;
      if (gm.F > 0 && key0 + KT - 1 >= gm.chunk0)
        need_mask = need_mask || ((key0 + KT - 1 - gm.chunk0) / gm.F > wave_first_frame);
      if (need_mask) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = key0 + 16 * kt + 4 * g + i;
            const bool in_range = key < gm.Lk;
            const int kf = (gm.F > 0 && key >= gm.chunk0) ? (key - gm.chunk0) / gm.F : -1;
#pragma unroll
            for (int qt = 0; qt < 2; ++qt)
              if (!in_range || kf > qframe[qt]) sacc[kt][qt][i] = -INFINITY;
          }
      }
      // ---- online softmax (base 2, scaled logits, lazy rescale) ----
      float mt[2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, sacc[kt][qt][i]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        mt[qt] = mx * scale_log2;
      }
      const bool raise0 = mt[0] > m_run[0] + kRescaleSlack;
      const bool raise1 = mt[1] > m_run[1] + kRescaleSlack;
      if (__any(raise0 || raise1)) {
#pragma unroll
        for (int qt = 0; qt < 2; ++qt) {
          const bool raise = qt == 0 ? raise0 : raise1;
          const float m_new = raise ? mt[qt] : m_run[qt];
          const float alpha = raise ? __builtin_amdgcn_exp2f(m_run[qt] - m_new) : 1.0f;
          m_run[qt] = m_new;
          l_run[qt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) oacc[dt][qt] *= alpha;
        }
      }
      bf16x8 pb[2][2];
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const float m_use = (m_run[qt] == -INFINITY) ? 0.f : m_run[qt];
        float rs = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][qt][i], scale_log2, -m_use));
            sacc[kt][qt][i] = p;
            rs += p;
          }
        l_run[qt] += rs;
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2) {
          u32x4 w;
          w[0] = pack_bf16x2(sacc[2 * ks2][qt][0], sacc[2 * ks2][qt][1]);
          w[1] = pack_bf16x2(sacc[2 * ks2][qt][2], sacc[2 * ks2][qt][3]);
          w[2] = pack_bf16x2(sacc[2 * ks2 + 1][qt][0], sacc[2 * ks2 + 1][qt][1]);
          w[3] = pack_bf16x2(sacc[2 * ks2 + 1][qt][2], sacc[2 * ks2 + 1][qt][3]);
          pb[qt][ks2] = __builtin_bit_cast(bf16x8, w);
        }
      }
      // ---- O^T += V^T P^T : V^T operand by LDS transpose reads ----
      // lane (g, s = c) addresses key row 32 ks2 + 16 h + 4 g + s/4 at d = 16 dt + 4 (s%4);
      // the transpose hands it V[32 ks2 + 16 h + 4 g + j][16 dt + s], j = 0..3.
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          v4i16 half[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int r = 32 * ks2 + 16 * h + 4 * g + (c >> 2);
            const int chunk = 2 * dt + ((c & 3) >> 1);
            const int byte = r * T::ROWB + ((chunk ^ swz<D>(r)) << 4) + ((c & 1) << 3);
            half[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) v4i16*)(vs_base + byte));
          }
          const v4i16 lo = half[0], hi = half[1];
          typedef short v8i16 __attribute__((ext_vector_type(8)));
          const v8i16 a8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          const bf16x8 a = __builtin_bit_cast(bf16x8, a8);
          oacc[dt][0] = mfma16(a, pb[0][ks2], oacc[dt][0]);
          oacc[dt][1] = mfma16(a, pb[1][ks2], oacc[dt][1]);
        }
      }
    }
    cj = nj;
    csub = nsb;
    cA = nA;
    cB = nB;
    stage ^= 1;
  }

  // ---- epilogue ----
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    float l = l_run[qt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int qrow = r0w + 16 * qt + c;
    if (qrow >= gm.Lq) continue;
    if (splits == 1) {
      const float inv = l > 0.f ? 1.0f / l : 0.f;
      uint16_t* orow = o + ((size_t)bh * gm.Lq + qrow) * D + 4 * g;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        u32x2 w;
        w[0] = pack_bf16x2(oacc[dt][qt][0] * inv, oacc[dt][qt][1] * inv);
        w[1] = pack_bf16x2(oacc[dt][qt][2] * inv, oacc[dt][qt][3] * inv);
        *(u32x2*)(orow + 16 * dt) = w;
      }
      if (lse && g == 0)
        lse[(size_t)bh * gm.Lq + qrow] = l > 0.f ? (m_run[qt] + log2f(l)) * 0.69314718055994531f : -INFINITY;
    } else {
      const size_t prow = ((size_t)sp * BH + bh) * gm.Lq + qrow;
      float* po = part_o + prow * D + 4 * g;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) *(f32x4*)(po + 16 * dt) = oacc[dt][qt];
      if (g == 0) {
        part_m[prow] = m_run[qt];
        part_l[prow] = l;
      }
    }
  }
}

// Merges split partials: O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(const float* __restrict__ part_o,
                                                                const float* __restrict__ part_m,
                                                                const float* __restrict__ part_l,
                                                                uint16_t* __restrict__ o, float* __restrict__ lse,
                                                                int rows, int splits) {
  // one wave per query row, lanes over d
  const int wave = (blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wave >= rows) return;
  float m = -INFINITY;
  for (int s = 0; s < splits; ++s) m = fmaxf(m, part_m[(size_t)s * rows + wave]);
  const float m_use = (m == -INFINITY) ? 0.f : m;
  float l = 0.f;
  float acc[D / 64];
#pragma unroll
  for (int e = 0; e < D / 64; ++e) acc[e] = 0.f;
  for (int s = 0; s < splits; ++s) {
    const size_t pr = (size_t)s * rows + wave;
    const float w = exp2f(part_m[pr] - m_use);
    l += w * part_l[pr];
#pragma unroll
    for (int e = 0; e < D / 64; ++e) acc[e] += w * part_o[pr * D + lane + 64 * e];
  }
  const float inv = l > 0.f ? 1.0f / l : 0.f;
#pragma unroll
  for (int e = 0; e < D / 64; ++e) {
    const __bf16 b = (__bf16)(acc[e] * inv);
    o[(size_t)wave * D + lane + 64 * e] = __builtin_bit_cast(uint16_t, b);
  }
  if (lse && lane == 0) lse[wave] = l > 0.f ? (m + log2f(l)) * 0.69314718055994531f : -INFINITY;
}

}  // namespace

int attn_splits(const Dims& dm) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const int units = dm.BH * row_tiles;
  const int target = 512;      // two workgroups per CU on a 256-CU MI355X
  if (units >= target / 2) return 1;
  int s = ceil_div(target, units);
  s = s > 16 ? 16 : s;
  s = s > dm.NK ? dm.NK : s;
  return s < 1 ? 1 : s;
}

hipError_t launch_attn(const Dims& dm, const void* q, const void* k, const void* v, const int32_t* counts,
                       const int32_t* idx, float scale, void* o, float* lse, void* ws, int splits,
                       hipStream_t st) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const int units = dm.BH * row_tiles * splits;
  const int grid = ceil_div(units, 8) * 8;
  Geom gm{dm.Lq, dm.Lk, dm.block, dm.NQ, dm.NK, dm.frame_tokens, dm.chunk0};
  const float scale_log2 = scale * 1.4426950408889634f;
  float* part_o = nullptr;
  float* part_m = nullptr;
  float* part_l = nullptr;
  if (splits > 1) {
    const size_t rows = (size_t)splits * dm.BH * dm.Lq;
    part_o = (float*)ws;
    part_m = (float*)((char*)ws + align256(rows * dm.d * sizeof(float)));
    part_l = (float*)((char*)part_m + align256(rows * sizeof(float)));
  }
  if (dm.d == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(grid), dim3(kThreads), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, counts, idx, (uint16_t*)o, lse, part_o, part_m,
                       part_l, gm, dm.BH, row_tiles, splits, units, scale_log2);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(grid), dim3(kThreads), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, counts, idx, (uint16_t*)o, lse, part_o, part_m,
                       part_l, gm, dm.BH, row_tiles, splits, units, scale_log2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int rows = dm.BH * dm.Lq;
  const int cgrid = ceil_div(rows * 64, kThreads);
  if (dm.d == 128)
    hipLaunchKernelGGL(attn_combine_kernel<128>, dim3(cgrid), dim3(kThreads), 0, st, part_o, part_m, part_l,
                       (uint16_t*)o, lse, rows, splits);
  else
    hipLaunchKernelGGL(attn_combine_kernel<64>, dim3(cgrid), dim3(kThreads), 0, st, part_o, part_m, part_l,
                       (uint16_t*)o, lse, rows, splits);
  return hipGetLastError();
}

}  // namespace la
