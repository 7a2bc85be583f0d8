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
//   * Key blocks are consumed in 64-key sub-tiles staged by asynchronous buffer-to-LDS
//     16-byte loads into a double buffer: sub-tile t+1 streams in while sub-tile t is
//     multiplied, with one workgroup barrier per sub-tile.  The buffer descriptors end at Lk,
//     so the ragged last block reads zeros past the end.
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
constexpr float kRescaleSlack = 8.0f;   // log2 headroom before the running max is raised

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef float f32x2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
#define LDS_AS __attribute__((address_space(3)))

__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2v f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2v));
}

// LDS layout: K and V tiles of 64 key rows of D bf16, row-major with padded rows.  K rows are
// padded to D*2 + 16 bytes: the 32 key rows an MFMA operand read touches (16 per LDS cycle)
// start in distinct 16-byte bank groups.  V rows are padded to D*2 + 64 bytes: a transpose
// read touches 4 rows x 64 contiguous bytes per half-wave, which then cover all 64 banks once.
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

// Issues this wave's buffer-to-LDS loads of one 64-key tile of one matrix (NINST wave-wide
// loads over the workgroup, PER per wave) into `dst`.  The descriptor starts at the tile and
// ends at Lk: rows past Lk and padding slots read as zero.
template <int D, int NINST, int PER>
__device__ inline void issue_rows(unsigned char* dst, const uint16_t* base, int key0, int Lk, const uint32_t* off,
                                  int wave) {
  // a tile may start at or past Lk (second half of a ragged 128-key block): no valid rows
  const uint32_t nrec = key0 < Lk ? (uint32_t)(Lk - key0) * (uint32_t)(D * 2) : 0u;
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void*)(base + (size_t)key0 * D), 0, nrec, 0x00020000);
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int n = wave + 4 * u;
    if (NINST % 4 == 0 || n < NINST)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (LDS_AS void*)(dst + 1024 * n), 16, off[u], 0, 0, 0);
  }
}

struct Geom {
  int Lq, Lk, block, NQ, NK, F, chunk0;
};

// Per-wave constants of the tile loop.
struct WaveCtx {
  int key_lk;                // Lk
  int klimit;                // keys >= klimit are invisible to this lane's query row
  int klimit_wave;           // smallest klimit of the wave (tiles below it need no mask)
  int kbase, vbase;          // LDS read bases of this lane inside a K / V tile
  int h;                     // lane / 32
  float scale_log2;
};

// S^T = K Q^T for one 64-key tile: two 32x32 accumulators (keys 0..31, 32..63).
template <int D>
__device__ __forceinline__ void qk_tile(const unsigned char* __restrict__ kb, const bf16x8* qreg, f32x16* sacc,
                                        int kbase) {
  using T = Tile<D>;
  constexpr int KS = D / 16;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int i = 0; i < 16; ++i) sacc[kt][i] = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const bf16x8 a = *(const bf16x8*)(kb + kbase + kt * 32 * T::KSTRIDE + 32 * ks);
      sacc[kt] = mfma32(a, qreg[ks], sacc[kt]);
    }
  }
}

// Masks (ragged tail, frame-causal pairs), running max and the lazy rescale of O for one tile.
// Lane holds keys key0 + 32 kt + 8 (i/4) + 4 (l/32) + i%4 of its query row.
template <int D>
__device__ __forceinline__ void softmax_prep(f32x16* sacc, f32x16* oacc, float& m_run, float& l_run, int key0,
                                             const WaveCtx& w) {
  constexpr int DT = D / 32;
  if (key0 + KT > w.klimit_wave) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = key0 + 32 * kt + 8 * (i >> 2) + 4 * w.h + (i & 3);
        if (key >= w.klimit) sacc[kt][i] = -INFINITY;
      }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kt][i]);
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float mt = mx * w.scale_log2;
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
}

// P = 2^(S*scale - m) (row sums in fp32, P rounded to bf16 for the product), then
// O^T += V^T P^T with the V^T operand read by LDS transpose loads.
template <int D>
__device__ __forceinline__ void softmax_pv(const f32x16* sacc, const unsigned char* __restrict__ vb, f32x16* oacc,
                                           float m_run, float& l_run, const WaveCtx& w) {
  using T = Tile<D>;
  constexpr int DT = D / 32;
  const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
  float rs0 = 0.f, rs1 = 0.f;
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) {
    u32x4 pw;
#pragma unroll
    for (int j2 = 0; j2 < 4; ++j2) {
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[s4 >> 1][8 * (s4 & 1) + 2 * j2], w.scale_log2, -m_use));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[s4 >> 1][8 * (s4 & 1) + 2 * j2 + 1], w.scale_log2, -m_use));
      pw[j2] = pack_bf16x2(p0, p1);
      rs0 += p0;
      rs1 += p1;
    }
    const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const unsigned char* va = vb + w.vbase + (16 * s4) * T::VSTRIDE + 64 * dt;
      const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(va));
      const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(va + 8 * T::VSTRIDE));
      const v8i16 a8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      oacc[dt] = mfma32(__builtin_bit_cast(bf16x8, a8), pb, oacc[dt]);
    }
  }
  l_run += rs0 + rs1;
}

// ---------------------------------------------------------------------------
// Work plan.  A unit is 128 consecutive query rows of one (batch, head): two query blocks of
// 64 rows or one of 128 (list 0 = first block, list 1 = second).  Its tiles are the 64-key
// sub-tiles of the union of its kept lists, in ascending block order; entry = block << 4 |
// ownership bits (bit L: list L keeps the block).  A unit with no kept block still gets one
// (unowned) tile so that some workgroup writes its output.

constexpr int kPersist = 512;    // persistent workgroups: two per CU on a 256-CU MI355X

__device__ inline int block_excl_scan_i(int x, int* sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  __syncthreads();
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  int base = 0, tot = 0;
  for (int wv = 0; wv < (int)(blockDim.x >> 6); ++wv) {
    if (wv < wave) base += sh[wv];
    tot += sh[wv];
  }
  *total = tot;
  return base + incl - x;
}

__global__ __launch_bounds__(kThreads) void plan_union_kernel(const int32_t* __restrict__ counts,
                                                              const int32_t* __restrict__ idx, int NQ, int NK,
                                                              int block, int row_tiles, int32_t* __restrict__ ulist,
                                                              int32_t* __restrict__ ucount) {
  extern __shared__ __align__(16) uint32_t own[];     // 4 ownership bits per key block
  __shared__ int sh[kThreads / 64];
  const int u = blockIdx.x;
  const int bh = u / row_tiles, rt = u % row_tiles;
  const int tid = threadIdx.x;
  const int nwords = (NK + 7) >> 3;
  for (int i = tid; i < nwords; i += kThreads) own[i] = 0;
  __syncthreads();
  const int q0 = rt * QR / block;
  const int nlists = (block == 64 && q0 + 1 < NQ) ? 2 : 1;
  for (int L = 0; L < nlists; ++L) {
    const size_t row = (size_t)bh * NQ + q0 + L;
    const int n = min(max(counts[row], 0), NK);
    const int32_t* lst = idx + row * NK;
    for (int i = tid; i < n; i += kThreads) {
      const int j = lst[i];
      if ((unsigned)j < (unsigned)NK) atomicOr(&own[j >> 3], (1u << L) << ((j & 7) * 4));
    }
  }
  __syncthreads();
  const int per = (nwords + kThreads - 1) / kThreads;
  const int w0 = min(tid * per, nwords), w1 = min(w0 + per, nwords);
  int cnt = 0;
  for (int wi = w0; wi < w1; ++wi) {
    const uint32_t x = own[wi];
#pragma unroll
    for (int e = 0; e < 8; ++e) cnt += ((x >> (4 * e)) & 15u) ? 1 : 0;
  }
  int total;
  int pos = block_excl_scan_i(cnt, sh, &total);
  int32_t* out = ulist + (size_t)u * NK;
  for (int wi = w0; wi < w1; ++wi) {
    const uint32_t x = own[wi];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t bits = (x >> (4 * e)) & 15u;
      if (bits) out[pos++] = ((8 * wi + e) << 4) | (int)bits;
    }
  }
  if (tid == 0) ucount[u] = total;
}

// tstart[u] = tiles of units < u (each unit max(1, blocks * nsub) tiles); tstart[U] = total.
__global__ __launch_bounds__(1024) void plan_scan_kernel(const int32_t* __restrict__ ucount, int U, int nsub,
                                                         int64_t* __restrict__ tstart) {
  __shared__ int64_t sh[16];
  __shared__ int64_t carry;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int base = 0; base < U; base += 1024) {
    const int u = base + tid;
    const int64_t x = u < U ? (int64_t)max(1, ucount[u] * nsub) : 0;
    int64_t incl = x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int64_t y = ((int64_t)__shfl_up((int)(incl >> 32), off) << 32) | (uint32_t)__shfl_up((int)incl, off);
      if (lane >= off) incl += y;
    }
    if (lane == 63) sh[wave] = incl;
    __syncthreads();
    int64_t before = carry;
    for (int wv = 0; wv < wave; ++wv) before += sh[wv];
    if (u < U) tstart[u] = before + incl - x;
    __syncthreads();
    if (tid == 1023) carry = before + incl;
    __syncthreads();
  }
  if (tid == 0) tstart[U] = carry;
}

// Persistent workgroup lambda covers tiles [T lambda / P, T (lambda + 1) / P) of the global
// tile sequence.
__device__ inline int64_t range_begin(int64_t T, int lambda, int P) { return T * lambda / P; }

// One step of the double-buffered loop for tile i (staged in kcur, vcur); tile i+1 is issued
// into (knext, vnext) while i is multiplied.  The read and write buffers are distinct
// __shared__ arrays, so the compiler can see that reads never wait on the asynchronous writes.
struct TileRef {
  int key0;
  int bits;
  bool valid;
};

template <int D>
__device__ __forceinline__ void tile_step(const unsigned char* __restrict__ kcur, const unsigned char* __restrict__ vcur,
                                          unsigned char* __restrict__ knext, unsigned char* __restrict__ vnext,
                                          const TileRef& t0, const TileRef& t1, const uint16_t* kh,
                                          const uint16_t* vh, const uint32_t* koff, const uint32_t* voff, int wave,
                                          int my_list, bool wave_rows, const bf16x8* qreg, f32x16* oacc,
                                          float& m_run, float& l_run, const WaveCtx& w) {
  using T = Tile<D>;
  // this thread's loads of (kcur, vcur) are done; the barrier makes every thread's loads
  // visible and guarantees no wave still reads (knext, vnext), which held tile i-1
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (t1.valid) {
    issue_rows<D, T::KINST, T::KPER>(knext, kh, t1.key0, w.key_lk, koff, wave);
    issue_rows<D, T::VINST, T::VPER>(vnext, vh, t1.key0, w.key_lk, voff, wave);
  }
  if (((t0.bits >> my_list) & 1) && wave_rows) {
    f32x16 sacc[2];
    qk_tile<D>(kcur, qreg, sacc, w.kbase);
    softmax_prep<D>(sacc, oacc, m_run, l_run, t0.key0, w);
    softmax_pv<D>(sacc, vcur, oacc, m_run, l_run, w);
  }
}

__device__ inline TileRef tile_ref(const int32_t* __restrict__ ul, int64_t i, int64_t n, int nsub, int block,
                                   int nblocks) {
  TileRef t;
  t.valid = i < n;
  t.key0 = 0;
  t.bits = 0;
  if (t.valid && nblocks > 0) {
    const int e = ul[nsub == 2 ? (i >> 1) : i];
    t.key0 = (e >> 4) * block + (nsub == 2 ? (int)(i & 1) * KT : 0);
    t.bits = e & 15;
  }
  return t;
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const int32_t* __restrict__ ulist, const int32_t* __restrict__ ucount, const int64_t* __restrict__ tstart,
    uint16_t* __restrict__ o, float* __restrict__ lse, float* __restrict__ part_o, float* __restrict__ part_m,
    float* __restrict__ part_l, Geom gm, int BH, int row_tiles, int U, float scale_log2) {
  using T = Tile<D>;
  constexpr int KS = D / 16;   // k-steps of Q.K^T (32x32x16)
  constexpr int DT = D / 32;   // d tiles of P.V
  __shared__ __attribute__((aligned(1024))) unsigned char kbuf0[T::KBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char kbuf1[T::KBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char vbuf0[T::VBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char vbuf1[T::VBYTES];

  // XCD-aware range: hardware places consecutive workgroup ids on consecutive XCDs (round
  // robin over 8); the workgroups of one XCD get consecutive ranges, i.e. consecutive units
  // of the same heads, so each L2 keeps its heads' shared K/V.
  const int P = gridDim.x;
  const int lambda = (blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3);
  const int64_t Ttot = tstart[U];
  const int64_t t_begin = range_begin(Ttot, lambda, P), t_end = range_begin(Ttot, lambda + 1, P);
  if (t_begin >= t_end) return;
  // unit holding t_begin: largest u with tstart[u] <= t_begin
  int ulo = 0, uhi = U - 1;
  while (ulo < uhi) {
    const int mid = (ulo + uhi + 1) >> 1;
    if (tstart[mid] <= t_begin) ulo = mid;
    else uhi = mid - 1;
  }
  int u = ulo;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: keeps tile-issue math scalar
  const int c32 = lane & 31, h = lane >> 5;
  const int nsub = gm.block / KT;
  const int my_list = (gm.block == 64 && wave >= 2) ? 1 : 0;   // waves 2, 3 own the second block

  // lane-constant global offsets of this wave's tile loads
  uint32_t koff[T::KPER], voff[T::VPER];
#pragma unroll
  for (int uu = 0; uu < T::KPER; ++uu) {
    const int n = wave + 4 * uu;
    koff[uu] = n < T::KINST ? slot_offset<D>(n, lane, T::KSLOTS) : 0x7fffffffu;
  }
#pragma unroll
  for (int uu = 0; uu < T::VPER; ++uu) {
    const int n = wave + 4 * uu;
    voff[uu] = n < T::VINST ? slot_offset<D>(n, lane, T::VSLOTS) : 0x7fffffffu;
  }
  WaveCtx w;
  w.key_lk = gm.Lk;
  w.kbase = c32 * T::KSTRIDE + 16 * h;
  w.vbase = (4 * h + ((lane & 15) >> 2)) * T::VSTRIDE + 32 * ((lane >> 4) & 1) + 8 * (lane & 3);
  w.h = h;
  w.scale_log2 = scale_log2;

  int64_t t = t_begin;
  while (t < t_end) {
    const int64_t ts = tstart[u], te = tstart[u + 1];
    const int64_t a = t - ts, b = (te < t_end ? te : t_end) - ts;   // local tile range [a, b)
    const bool full = (a == 0) && (b == te - ts);
    const int bh = u / row_tiles, rt = u % row_tiles;
    const int row_base = rt * QR;
    const int r0w = row_base + wave * QW;               // first query row of this wave
    const bool wave_rows = r0w < gm.Lq;
    const int nblocks = ucount[u];
    const int32_t* ul = ulist + (size_t)u * gm.NK;
    const int64_t ntiles = (int64_t)nblocks * nsub;     // 0 for an empty unit (its dummy tile is unowned)
    const uint16_t* kh = k + (size_t)bh * gm.Lk * D;
    const uint16_t* vh = v + (size_t)bh * gm.Lk * D;

    // Q^T operand (32x32x16 B): lane holds Q[row r0w + l%32][16 ks + 8 (l/32) .. + 7]
    bf16x8 qreg[KS];
    {
      const int row = r0w + c32;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 qw = u32x4{0u, 0u, 0u, 0u};
        if (row < gm.Lq) qw = *(const u32x4*)(q + ((size_t)bh * gm.Lq + row) * D + 16 * ks + 8 * h);
        qreg[ks] = __builtin_bit_cast(bf16x8, qw);
      }
    }
    // Key n is visible to query row t when n < Lk and, with frames of F tokens inside the chunk,
    // when its chunk frame is not later than t's: n < chunk0 + (t / F + 1) F (context keys,
    // n < chunk0, always pass).  One limit per lane replaces per-key frame arithmetic.
    {
      const int64_t lim = gm.F > 0 ? (int64_t)gm.chunk0 + ((int64_t)(r0w + c32) / gm.F + 1) * gm.F : (int64_t)gm.Lk;
      const int64_t limw = gm.F > 0 ? (int64_t)gm.chunk0 + ((int64_t)r0w / gm.F + 1) * gm.F : (int64_t)gm.Lk;
      w.klimit = (int)(lim < gm.Lk ? lim : gm.Lk);
      w.klimit_wave = (int)(limw < gm.Lk ? limw : gm.Lk);
    }
    f32x16 oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.f;
    float m_run = -INFINITY;
    float l_run = 0.f;

    const int64_t bb = b < ntiles ? b : ntiles;         // real tiles of this piece (dummy tile: none)
    // previous unit's last tile may still be read from either buffer: sync before refilling
    __syncthreads();
    TileRef t0 = tile_ref(ul, a, bb, nsub, gm.block, nblocks);
    TileRef t1 = tile_ref(ul, a + 1, bb, nsub, gm.block, nblocks);
    if (t0.valid) {
      issue_rows<D, T::KINST, T::KPER>(kbuf0, kh, t0.key0, gm.Lk, koff, wave);
      issue_rows<D, T::VINST, T::VPER>(vbuf0, vh, t0.key0, gm.Lk, voff, wave);
    }
    int64_t i = a;
    while (t0.valid) {
      tile_step<D>(kbuf0, vbuf0, kbuf1, vbuf1, t0, t1, kh, vh, koff, voff, wave, my_list, wave_rows, qreg, oacc,
                   m_run, l_run, w);
      ++i;
      t0 = t1;
      t1 = tile_ref(ul, i + 1, bb, nsub, gm.block, nblocks);
      if (!t0.valid) break;
      tile_step<D>(kbuf1, vbuf1, kbuf0, vbuf0, t0, t1, kh, vh, koff, voff, wave, my_list, wave_rows, qreg, oacc,
                   m_run, l_run, w);
      ++i;
      t0 = t1;
      t1 = tile_ref(ul, i + 1, bb, nsub, gm.block, nblocks);
    }
    // no load is left in flight: the last step issued nothing (its next tile was invalid)

    // ---- output: lane holds O^T[32 dt + 8 (i/4) + 4 (l/32) + i%4][query r0w + l%32] ----
    const float l = l_run + __shfl_xor(l_run, 32);
    const int qrow = r0w + c32;
    if (qrow < gm.Lq) {
      if (full) {
        const float inv = l > 0.f ? 1.0f / l : 0.f;
        uint16_t* orow = o + ((size_t)bh * gm.Lq + qrow) * D + 4 * h;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int a4 = 0; a4 < 4; ++a4) {
            u32x2 ow;
            ow[0] = pack_bf16x2(oacc[dt][4 * a4] * inv, oacc[dt][4 * a4 + 1] * inv);
            ow[1] = pack_bf16x2(oacc[dt][4 * a4 + 2] * inv, oacc[dt][4 * a4 + 3] * inv);
            *(u32x2*)(orow + 32 * dt + 8 * a4) = ow;
          }
        if (lse && h == 0)
          lse[(size_t)bh * gm.Lq + qrow] = l > 0.f ? (m_run + log2f(l)) * 0.69314718055994531f : -INFINITY;
      } else {
        // a piece of a unit split across workgroups: the workgroup's first unit goes to slot
        // 2 lambda, its last (when it continues past the range) to slot 2 lambda + 1
        const int slot = 2 * lambda + (a > 0 ? 0 : 1);
        const size_t prow = (size_t)slot * QR + (qrow - row_base);
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
    t = ts + b;
    ++u;
  }
}

// Merges the pieces of units that were split across workgroups:
// O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s, over the pieces in workgroup order
// (deterministic).  Thread t owns 4 columns and QR * D / (4 * kThreads) rows of the unit, so
// the loads of all its rows are in flight together.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(const int64_t* __restrict__ tstart, int U, int P,
                                                                int row_tiles, int Lq,
                                                                const float* __restrict__ part_o,
                                                                const float* __restrict__ part_m,
                                                                const float* __restrict__ part_l,
                                                                uint16_t* __restrict__ o, float* __restrict__ lse) {
  constexpr int CG = D / 4;                 // 4-column groups per row
  constexpr int RSTEP = kThreads / CG;      // rows per pass
  constexpr int NI = QR / RSTEP;            // rows per thread
  const int u = blockIdx.x;
  const int64_t Ttot = tstart[U], ts = tstart[u], te = tstart[u + 1];
  // workgroup (range) holding tile t: largest lambda with T lambda / P <= t
  auto owner = [&](int64_t t) {
    int64_t lam = ((t + 1) * P + Ttot - 1) / Ttot - 1;
    return (int)(lam < P - 1 ? lam : P - 1);
  };
  const int la0 = owner(ts), la1 = owner(te - 1);
  if (la0 == la1) return;                               // not split: written directly
  const int bh = u / row_tiles, rt = u % row_tiles;
  const int cg = threadIdx.x % CG, r0 = threadIdx.x / CG;
  float m[NI], l[NI];
  f32x4 acc[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    m[i] = -INFINITY;
    l[i] = 0.f;
    acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // workgroups with an empty range (fewer tiles than workgroups) wrote no slot
  for (int lam = la0; lam <= la1; ++lam) {
    if (range_begin(Ttot, lam, P) == range_begin(Ttot, lam + 1, P)) continue;
    const int slot = lam == la0 ? 2 * lam + 1 : 2 * lam;
#pragma unroll
    for (int i = 0; i < NI; ++i) m[i] = fmaxf(m[i], part_m[(size_t)slot * QR + r0 + RSTEP * i]);
  }
  for (int lam = la0; lam <= la1; ++lam) {
    if (range_begin(Ttot, lam, P) == range_begin(Ttot, lam + 1, P)) continue;
    const int slot = lam == la0 ? 2 * lam + 1 : 2 * lam;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const size_t pr = (size_t)slot * QR + r0 + RSTEP * i;
      const float wgt = exp2f(part_m[pr] - (m[i] == -INFINITY ? 0.f : m[i]));
      l[i] += wgt * part_l[pr];
      const f32x4 po = *(const f32x4*)(part_o + pr * D + 4 * cg);
      acc[i] += wgt * po;
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int qrow = rt * QR + r0 + RSTEP * i;
    if (qrow < Lq) {
      const float inv = l[i] > 0.f ? 1.0f / l[i] : 0.f;
      u32x2 ow;
      ow[0] = pack_bf16x2(acc[i][0] * inv, acc[i][1] * inv);
      ow[1] = pack_bf16x2(acc[i][2] * inv, acc[i][3] * inv);
      *(u32x2*)(o + ((size_t)bh * Lq + qrow) * D + 4 * cg) = ow;
      if (lse && cg == 0)
        lse[(size_t)bh * Lq + qrow] = l[i] > 0.f ? (m[i] + log2f(l[i])) * 0.69314718055994531f : -INFINITY;
    }
  }
}

struct AttnWs {
  int32_t* ulist;
  int32_t* ucount;
  int64_t* tstart;
  float* part_o;
  float* part_m;
  float* part_l;
  size_t bytes;
};

AttnWs attn_ws_layout(const Dims& dm, void* base) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const size_t U = (size_t)dm.BH * row_tiles;
  const size_t slots = 2 * (size_t)kPersist;
  size_t off = 0;
  AttnWs w;
  char* b = (char*)base;
  w.ulist = (int32_t*)(b + off);
  off += align256(U * dm.NK * sizeof(int32_t));
  w.ucount = (int32_t*)(b + off);
  off += align256(U * sizeof(int32_t));
  w.tstart = (int64_t*)(b + off);
  off += align256((U + 1) * sizeof(int64_t));
  w.part_o = (float*)(b + off);
  off += align256(slots * QR * dm.d * sizeof(float));
  w.part_m = (float*)(b + off);
  off += align256(slots * QR * sizeof(float));
  w.part_l = (float*)(b + off);
  off += align256(slots * QR * sizeof(float));
  w.bytes = off;
  return w;
}

}  // namespace

size_t attn_ws_bytes(const Dims& dm) { return attn_ws_layout(dm, nullptr).bytes; }

hipError_t launch_attn(const Dims& dm, const void* q, const void* k, const void* v, const int32_t* counts,
                       const int32_t* idx, float scale, void* o, float* lse, void* ws, hipStream_t st) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const int U = dm.BH * row_tiles;
  const int nsub = dm.block / KT;
  AttnWs w = attn_ws_layout(dm, ws);
  Geom gm{dm.Lq, dm.Lk, dm.block, dm.NQ, dm.NK, dm.frame_tokens, dm.chunk0};
  const float scale_log2 = scale * 1.4426950408889634f;
  hipLaunchKernelGGL(plan_union_kernel, dim3(U), dim3(kThreads), (size_t)((dm.NK + 7) / 8) * sizeof(uint32_t), st,
                     counts, idx, dm.NQ, dm.NK, dm.block, row_tiles, w.ulist, w.ucount);
  hipLaunchKernelGGL(plan_scan_kernel, dim3(1), dim3(1024), 0, st, w.ucount, U, nsub, w.tstart);
  if (dm.d == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(kPersist), dim3(kThreads), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, w.ulist, w.ucount, w.tstart, (uint16_t*)o, lse,
                       w.part_o, w.part_m, w.part_l, gm, dm.BH, row_tiles, U, scale_log2);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(kPersist), dim3(kThreads), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, w.ulist, w.ucount, w.tstart, (uint16_t*)o, lse,
                       w.part_o, w.part_m, w.part_l, gm, dm.BH, row_tiles, U, scale_log2);
  if (dm.d == 128)
    hipLaunchKernelGGL(attn_combine_kernel<128>, dim3(U), dim3(kThreads), 0, st, w.tstart, U, kPersist, row_tiles,
                       dm.Lq, w.part_o, w.part_m, w.part_l, (uint16_t*)o, lse);
  else
    hipLaunchKernelGGL(attn_combine_kernel<64>, dim3(U), dim3(kThreads), 0, st, w.tstart, U, kPersist, row_tiles,
                       dm.Lq, w.part_o, w.part_m, w.part_l, (uint16_t*)o, lse);
  return hipGetLastError();
}

}  // namespace la
