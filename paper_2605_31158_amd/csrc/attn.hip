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
//   * Key blocks are consumed in 64-key sub-tiles, staged by asynchronous buffer-to-LDS
//     16-byte loads into a double buffer: sub-tile t+1 streams in while sub-tile t is
//     multiplied, with one workgroup barrier per sub-tile.  The buffer descriptor of a
//     sub-tile ends at Lk, so the ragged last block reads zeros past the end.
//   * Workgroup ids are remapped so that each XCD (each L2) works on consecutive (head,
//     row tile) units: the kept K/V blocks of a head stay hot in one XCD's L2.
//   * Few work units (small problems) split the key-block range across workgroups; the
//     partial (O, m, l) are merged by attn_combine (log-sum-exp merge).
//
// Per wave and 64-key sub-tile (d = 128):
//   S^T (64 keys x 32 queries) = K_tile (64 x d) . Q^T       16 x v_mfma_f32_32x32x16_bf16
//   online softmax over keys (fp32, base 2; the running max is only raised when a tile's
//   max exceeds it by more than 2^8, so most tiles skip the rescale of O)
//   O^T (d x 32) += V^T (d x 64) . P^T (64 x 32)              16 x v_mfma_f32_32x32x16_bf16
// S^T is computed transposed so that its accumulator layout (each lane holds 16 keys of one
// query column) is, 8 values at a time, directly the B operand of the P.V product.  K and V
// tiles are row-major in LDS with padded rows; every operand read is a lane base address
// plus a compile-time offset.  The V^T operand is read with the LDS transpose load
// ds_read_b64_tr_b16 (two per MFMA).
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
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
#define LDS_AS __attribute__((address_space(3)))

__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// LDS layout of one stage: a K tile and a V tile, each 64 key rows of D bf16, row-major with
// padded rows.  K rows are padded to D*2 + 16 bytes: the 32 key rows an MFMA operand read
// touches (16 per LDS cycle) start in distinct 16-byte bank groups.  V rows are padded to
// D*2 + 64 bytes: a transpose read touches 4 rows x 64 contiguous bytes per half-wave, which
// then cover all 64 banks exactly once.
template <int D>
struct Tile {
  static constexpr int KSTRIDE = D * 2 + 16;
  static constexpr int VSTRIDE = D * 2 + 64;
  static constexpr int KSLOTS = KSTRIDE / 16;          // 16-byte slots per K row
  static constexpr int VSLOTS = VSTRIDE / 16;
  static constexpr int KBYTES = KT * KSTRIDE;
  static constexpr int VBYTES = KT * VSTRIDE;
  static constexpr int KINST = KT * KSLOTS / 64;       // wave-wide 1 KiB loads per K tile
  static constexpr int VINST = KT * VSLOTS / 64;
  static constexpr int KPER = (KINST + 3) / 4;         // per wave (4 waves)
  static constexpr int VPER = (VINST + 3) / 4;
  static constexpr int STAGE = KBYTES + VBYTES;
};

// Global byte offset (inside a tile of 64 rows) that lane `lane` of load `n` fetches so that it
// lands at LDS slot 64 n + lane of a padded layout with `slots` slots per row; padding slots get
// an offset past any buffer (they read as zero).
template <int D>
__device__ inline uint32_t slot_offset(int n, int lane, int slots) {
  const int slot = 64 * n + lane;
  const int row = slot / slots, chunk = slot % slots;
  return chunk < D / 8 ? (uint32_t)(row * D * 2 + chunk * 16) : 0x7fffffffu;
}

// Issues this wave's buffer-to-LDS loads of one 64-key sub-tile (K and V) into `stage`.
// The buffer descriptors start at the sub-tile and end at Lk, so rows past Lk (and the
// padding slots, whose offsets lie past any buffer) read as zero.
template <int D>
__device__ inline void issue_tile(unsigned char* stage, const uint16_t* kh, const uint16_t* vh, int key0,
                                  int Lk, const uint32_t* koff, const uint32_t* voff, int wave) {
  using T = Tile<D>;
  // a sub-tile may start at or past Lk (second half of a ragged 128-key block): no valid rows
  const uint32_t nrec = key0 < Lk ? (uint32_t)(Lk - key0) * (uint32_t)(D * 2) : 0u;
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc((void*)(kh + (size_t)key0 * D), 0, nrec, 0x00020000);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc((void*)(vh + (size_t)key0 * D), 0, nrec, 0x00020000);
#pragma unroll
  for (int u = 0; u < T::KPER; ++u) {
    const int n = wave + 4 * u;
    if (T::KINST % 4 == 0 || n < T::KINST)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (LDS_AS void*)(stage + 1024 * n), 16, koff[u], 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < T::VPER; ++u) {
    const int n = wave + 4 * u;
    if (T::VINST % 4 == 0 || n < T::VINST)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (LDS_AS void*)(stage + T::KBYTES + 1024 * n), 16, voff[u], 0, 0, 0);
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
  constexpr int KS = D / 16;   // k-steps of Q.K^T (32x32x16)
  constexpr int DT = D / 32;   // d tiles of P.V
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * T::STAGE];

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
  const int c32 = lane & 31, h = lane >> 5;
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

  // lane-constant global offsets of this wave's tile loads
  uint32_t koff[T::KPER], voff[T::VPER];
#pragma unroll
  for (int u = 0; u < T::KPER; ++u) {
    const int n = wave + 4 * u;
    koff[u] = n < T::KINST ? slot_offset<D>(n, lane, T::KSLOTS) : 0x7fffffffu;
  }
#pragma unroll
  for (int u = 0; u < T::VPER; ++u) {
    const int n = wave + 4 * u;
    voff[u] = n < T::VINST ? slot_offset<D>(n, lane, T::VSLOTS) : 0x7fffffffu;
  }
  // Q^T operand (32x32x16 B): lane holds Q[row r0w + l%32][16 ks + 8 (l/32) .. + 7]
  bf16x8 qreg[KS];
  {
    const int row = r0w + c32;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 w = u32x4{0u, 0u, 0u, 0u};
      if (row < gm.Lq) w = *(const u32x4*)(q + ((size_t)bh * gm.Lq + row) * D + 16 * ks + 8 * h);
      qreg[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }
  const int qframe = gm.F > 0 ? (r0w + c32) / gm.F : 0;
  const int wave_first_frame = gm.F > 0 ? r0w / gm.F : 0;

  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;

  // LDS read bases (bytes within a stage): K operand row l%32, d offset 8 (l/32);
  // V^T transpose read, 16-lane group G = l/16, lane i = l%16: row 4 (l/32) + i/4 of the
  // 16-key step, d = 16 (G%2) + 4 (i%4).
  const int kbase = c32 * T::KSTRIDE + 16 * h;
  const int vbase = T::KBYTES + (4 * h + ((lane & 15) >> 2)) * T::VSTRIDE + 32 * ((lane >> 4) & 1) + 8 * (lane & 3);

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
  if (cj != kEnd) issue_tile<D>(smem, kh, vh, cj * gm.block, gm.Lk, koff, voff, wave);
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
      issue_tile<D>(smem + (stage ^ 1) * T::STAGE, kh, vh, nj * gm.block + nsb * KT, gm.Lk, koff, voff, wave);
    const int key0 = cj * gm.block + csub * KT;
    const bool mine = (wave_b ? cB : cA) && wave_rows;
    const unsigned char* sb = smem + stage * T::STAGE;
    if (mine) {
      // ---- S^T = K Q^T : two 32x32 tiles over keys 0..31, 32..63 ----
      f32x16 sacc[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) sacc[kt][i] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const bf16x8 a = *(const bf16x8*)(sb + kbase + kt * 32 * T::KSTRIDE + 32 * ks);
          sacc[kt] = mfma32(a, qreg[ks], sacc[kt]);
        }
      }
      // ---- masks: keys past Lk (ragged last block), frame-causal pairs in the chunk ----
      // lane holds keys key0 + 32 kt + 8 (i/4) + 4 (l/32) + i%4 of query r0w + l%32
      bool need_mask = key0 + KT > gm.Lk;
      if (gm.F > 0 && key0 + KT - 1 >= gm.chunk0)
        need_mask = need_mask || ((key0 + KT - 1 - gm.chunk0) / gm.F > wave_first_frame);
      if (need_mask) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = key0 + 32 * kt + 8 * (i >> 2) + 4 * h + (i & 3);
            bool ok = key < gm.Lk;
            if (gm.F > 0 && key >= gm.chunk0) ok = ok && ((key - gm.chunk0) / gm.F <= qframe);
            if (!ok) sacc[kt][i] = -INFINITY;
          }
      }
      // ---- online softmax (base 2, scaled logits, lazy rescale) ----
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kt][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mt = mx * scale_log2;
      const bool raise = mt > m_run + kRescaleSlack;
      if (__any(raise)) {
        const float m_new = raise ? mt : m_run;
        const float alpha = raise ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
      }
      const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
      float rs = 0.f;
      bf16x8 pb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          p[j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[s >> 1][8 * (s & 1) + j], scale_log2, -m_use));
          rs += p[j];
        }
        u32x4 w;
        w[0] = pack_bf16x2(p[0], p[1]);
        w[1] = pack_bf16x2(p[2], p[3]);
        w[2] = pack_bf16x2(p[4], p[5]);
        w[3] = pack_bf16x2(p[6], p[7]);
        pb[s] = __builtin_bit_cast(bf16x8, w);
      }
      l_run += rs;
      // ---- O^T += V^T P^T : V^T operand by LDS transpose reads ----
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const unsigned char* va = sb + vbase + (16 * s) * T::VSTRIDE + 64 * dt;
          const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(va));
          const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(va + 8 * T::VSTRIDE));
          const v8i16 a8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          oacc[dt] = mfma32(__builtin_bit_cast(bf16x8, a8), pb[s], oacc[dt]);
        }
      }
    }
    cj = nj;
    csub = nsb;
    cA = nA;
    cB = nB;
    stage ^= 1;
  }

  // ---- epilogue: lane holds O^T[32 dt + 8 (i/4) + 4 (l/32) + i%4][query r0w + l%32] ----
  float l = l_run + __shfl_xor(l_run, 32);
  const int qrow = r0w + c32;
  if (qrow < gm.Lq) {
    if (splits == 1) {
      const float inv = l > 0.f ? 1.0f / l : 0.f;
      uint16_t* orow = o + ((size_t)bh * gm.Lq + qrow) * D + 4 * h;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          u32x2 w;
          w[0] = pack_bf16x2(oacc[dt][4 * a4] * inv, oacc[dt][4 * a4 + 1] * inv);
          w[1] = pack_bf16x2(oacc[dt][4 * a4 + 2] * inv, oacc[dt][4 * a4 + 3] * inv);
          *(u32x2*)(orow + 32 * dt + 8 * a4) = w;
        }
      if (lse && h == 0)
        lse[(size_t)bh * gm.Lq + qrow] = l > 0.f ? (m_run + log2f(l)) * 0.69314718055994531f : -INFINITY;
    } else {
      const size_t prow = ((size_t)sp * BH + bh) * gm.Lq + qrow;
      float* po = part_o + prow * D + 4 * h;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4)
          *(f32x4*)(po + 32 * dt + 8 * a4) =
              f32x4{oacc[dt][4 * a4], oacc[dt][4 * a4 + 1], oacc[dt][4 * a4 + 2], oacc[dt][4 * a4 + 3]};
      if (h == 0) {
        part_m[prow] = m_run;
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
