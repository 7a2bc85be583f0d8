// Block-sparse attention forward on gfx950 (Sec. 3.3: attention over C_i = T u K^curr u S_i,
// one kept-block list per query block serving both K and V).
//
// Work decomposition
//   * A unit is 256 query rows of one (batch, head): four query blocks of 64 rows or two of 128.
//     Query blocks are grouped by the first historical key block they keep, so that blocks
//     which chose the same context share a unit.  Its tiles are the 64-key sub-tiles of the
//     union of its blocks' kept lists, in ascending key order, each tagged with which of the
//     unit's blocks kept it.
//   * A planner (two or three small kernels) computes the grouping, every unit's union list, the
//     schedule and one record per tile (first key, head, unit, ownership) in the tile sequence.
//     One persistent workgroup per CU runs, first, whole units handed out in rounds: in each
//     round the workgroups of one XCD start consecutive units of the same head together, so
//     they walk that head's shared chunk K/V in step and each K/V tile reaches the XCD's L2
//     about once per round; then an equal-work share of the remaining units (those past the
//     last full round and the longer ones), cut anywhere (stream-K).  A unit cut between two
//     shares leaves (O, m, l) partials that attn_combine merges with a log-sum-exp merge.  Heavy
//     query blocks therefore never bound the launch.
//
// The workgroup: 8 waves = two groups of four, one wave of each group per SIMD.  Each wave owns
// 32 query rows; the two waves of a SIMD own the two halves of the same query block, so both
// groups own the same tiles.  Per tile h the groups run two phases each, offset by one phase and
// separated by workgroup barriers:
//
//   phase    group 0                              group 1
//   A(h)     M(h): P.V of tile h-1, Q.K^T of h    V(h-1): softmax of tile h-1, then issues the
//                                                 loads of K(h+1) and V(h)
//   B(h)     V(h): softmax of tile h              M(h): P.V of tile h-1, Q.K^T of tile h, then
//                                                 waits for its loads
//
// so on every SIMD one wave feeds the matrix pipeline while the other does the softmax
// arithmetic.  K and V have two LDS stages each: K(h) in stage h & 1 is read in A(h) and B(h);
// V(h) in stage h & 1 is read in A(h+1) and B(h+1); the loads of K(h+1) and V(h), issued in
// A(h), overwrite the stages last read in B(h-1).  Only group 1 issues tile loads (asynchronous
// buffer-to-LDS, 16 bytes per lane); their buffer descriptors end at Lk, so the ragged last
// block reads zeros past the end.
//
// Per wave and 64-key tile (d = 128):
//   S^T (64 keys x 32 queries) = K_tile (64 x d) . Q^T       16 x v_mfma_f32_32x32x16_bf16
//   online softmax over keys (fp32, base 2; the running max is only raised when a tile's
//   max exceeds it by more than 2^8, so most tiles skip the rescale of O)
//   O^T (d x 32) += V^T (d x 64) . P^T (64 x 32)              16 x v_mfma_f32_32x32x16_bf16
// S^T is computed transposed so that its accumulator layout (each lane holds 16 keys of one
// query column) is, 8 values at a time, directly the B operand of the P.V product.  The V^T
// operand is read with the LDS transpose load ds_read_b64_tr_b16 (two per MFMA).
#include <math.h>

#include <type_traits>

#include "la_internal.h"

namespace la {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int KT = 64;          // keys per tile
constexpr int QW = 32;          // query rows per wave
constexpr int QR = 256;         // query rows per unit (workgroup)
constexpr int kMaxPersist = 256;        // persistent workgroups: one per CU, at most 256
// flags of a tile record (see TileRef)
constexpr int kFlFrom0 = 1 << 4, kFlToEnd = 1 << 5, kFlFirst = 1 << 6, kFlLast = 1 << 7, kFlValid = 1 << 8;
// Bits 16..22 of a tile record's flags: keys at the end of the tile that are padding (0..64).
constexpr int kFlPadShift = 16;

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

// Workgroup barrier that orders LDS accesses (waits for this wave's LDS operations).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup barrier for a wave with asynchronous tile loads in flight that it does not wait for
// here: the LDS release fence of lds_barrier would wait for them (they write LDS).  The empty
// asm statements keep the compiler from moving memory accesses across the barrier; every LDS
// read of the wave has been consumed by then.
__device__ __forceinline__ void barrier_keep_loads() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Waits until at most n of this wave's vector memory operations are outstanding (n < 16).
template <int n>
__device__ __forceinline__ void wait_vmem() {
  __builtin_amdgcn_s_waitcnt(0x0F70 | n);   // vmcnt(n), expcnt and lgkmcnt left at their maximum
}

// LDS layout: K and V tiles of 64 key rows of D bf16, row-major.  K rows are padded to D*2 + 16
// bytes: the 32 key rows an MFMA operand read touches (16 per LDS cycle) start in distinct
// 16-byte bank groups.  V rows are not padded; instead the 64-byte chunks of a row are permuted
// (chunk c of row r is stored at chunk c ^ vswz(r)): a transpose read touches 4 consecutive rows
// x 64 contiguous bytes per half-wave, and the permutation spreads those four pieces over all 64
// banks.  Every K operand read is a lane base plus a compile-time offset, every V read one of
// D/32 lane bases (base ^ 64 dt) plus a compile-time offset.  A tile is written by wave-wide
// 16-byte-per-lane loads (1 KiB each) of consecutive 16-byte slots; K padding slots read as zero.
template <int D>
struct Tile {
  static constexpr int KSTRIDE = D * 2 + 16;
  static constexpr int VSTRIDE = D * 2;
  static constexpr int KSLOTS = KSTRIDE / 16;          // 16-byte slots per K row
  static constexpr int VSLOTS = VSTRIDE / 16;
  static constexpr int KBYTES = KT * KSTRIDE;
  static constexpr int VBYTES = KT * VSTRIDE;
  static constexpr int KINST = KT * KSLOTS / 64;       // wave-wide loads per K tile: 4 KPER + 1
  static constexpr int VINST = KT * VSLOTS / 64;       // per V tile: 4 VPER
  static constexpr int KPER = KINST / 4;               // per loading wave (wave 0 loads one more)
  static constexpr int VPER = VINST / 4;
  static_assert(KINST % 4 == 1 && VINST % 4 == 0, "load split");
  // chunk permutation of V row r: rows 4i..4i+3 get four distinct chunks (D = 128: 4 chunks per
  // row) or, with 128-byte rows (D = 64), rows 4i, 4i+2 and 4i+1, 4i+3 get opposite chunks
  __device__ static constexpr int vswz(int r) { return D == 128 ? (r & 3) : ((r >> 1) & 1); }
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

// The same for the V layout: LDS slot 64 n + lane holds part w (16 bytes) of stored chunk pc of
// row r, i.e. logical chunk pc ^ vswz(r).
template <int D>
__device__ inline uint32_t vslot_offset(int n, int lane) {
  constexpr int SL = D / 8;
  const int slot = 64 * n + lane;
  const int row = slot / SL, sp = slot % SL;
  const int chunk = (sp >> 2) ^ Tile<D>::vswz(row);
  return (uint32_t)(row * D * 2 + chunk * 64 + (sp & 3) * 16);
}

// Loads of one tile of one matrix by one loading wave: a buffer descriptor that starts at the
// tile and ends at Lk (rows past Lk read as zero; an invalid tile reads nothing) and the LDS
// destination.  Load j fills LDS bytes [1024 (lw + 4 j), + 1024) of the tile.
struct TileLoad {
  __amdgpu_buffer_rsrc_t rsrc;
  unsigned char* dst;
};

template <int D>
__device__ inline TileLoad tile_load(unsigned char* dst, const uint16_t* base, int key0, int Lk, bool valid) {
  const uint32_t nrec = valid && key0 < Lk ? (uint32_t)(Lk - key0) * (uint32_t)(D * 2) : 0u;
  TileLoad t;
  t.rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(base + (size_t)(valid ? key0 : 0) * D), 0, nrec, 0x00020000);
  t.dst = dst;
  return t;
}

template <int NL>
struct LoadSet {
  TileLoad t;
  int lw;
  const uint32_t* off;      // off[j]: the lane's global offset for load j
  __device__ __forceinline__ void issue(int j) const { issue_at(lw + 4 * j, off[j]); }
  // load n of the tile with the lane offset o
  __device__ __forceinline__ void issue_at(int n, uint32_t o) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(t.rsrc, (LDS_AS void*)(t.dst + 1024 * n), 16, o, 0, 0, 0);
  }
};

struct Geom {
  int Lq, Lk, block, NQ, NK, F, chunk0;
  int BH, U;          // heads and units of the plan (bounds for the fields read from it)
};

// Per-wave constants of the tile loop (klimit, klimit_wave change with the unit).
struct WaveCtx {
  int key_lk;                // Lk
  int klimit;                // keys >= klimit are invisible to this lane's query row
  int klimit_wave;           // smallest klimit of the wave (tiles below it need no mask)
  int kbase, vbase;          // LDS read bases of this lane inside a K / V tile
  int h;                     // lane / 32
  float scale_log2;
};

// Scheduling-group masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSgMfma = 0x008;
constexpr int kSgDsRead = 0x100;

// S^T = K Q^T for one 64-key tile: two 32x32 accumulators (keys 0..31, 32..63).  The K operand
// reads run four MFMAs ahead of their use, so LDS latency overlaps the matrix pipeline.
template <int D>
__device__ __forceinline__ void qk_tile(const unsigned char* __restrict__ kb, const bf16x8* qreg, f32x16* sacc,
                                        int kbase) {
  using T = Tile<D>;
  constexpr int NS = 2 * (D / 16);       // MFMAs per tile: 2 key halves x D/16 k-steps
  constexpr int AHEAD = 4;
  bf16x8 ka[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i) ka[i] = *(const bf16x8*)(kb + kbase + (i & 1) * 32 * T::KSTRIDE + 32 * (i >> 1));
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int i = 0; i < 16; ++i) sacc[kt][i] = 0.f;
#pragma unroll
  for (int i = 0; i < NS; ++i) sacc[i & 1] = mfma32(ka[i], qreg[i >> 1], sacc[i & 1]);
  __builtin_amdgcn_sched_group_barrier(kSgDsRead, AHEAD, 0);
#pragma unroll
  for (int i = 0; i < NS - AHEAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kSgDsRead, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(kSgMfma, AHEAD, 0);
}

// O^T += V^T P^T for one 64-key tile (P in four bf16 B operands of 16 keys each).  The two
// transpose reads of each V^T operand run two MFMAs ahead of their use.  Column block dt of the
// lane's rows sits at vbase ^ (64 dt) (see Tile).
template <int D>
__device__ __forceinline__ void pv_tile(const unsigned char* __restrict__ vb, const bf16x8* pb, f32x16* oacc,
                                        int vbase) {
  using T = Tile<D>;
  constexpr int DT = D / 32;
  constexpr int NM = 4 * DT;             // MFMAs per tile
  constexpr int AHEAD = 2;
  bf16x8 va[NM];
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const int s4 = i / DT, dt = i % DT;
    const unsigned char* vp = vb + (vbase ^ (64 * dt)) + (16 * s4) * T::VSTRIDE;
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(vp));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(vp + 8 * T::VSTRIDE));
    const v8i16 a8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    va[i] = __builtin_bit_cast(bf16x8, a8);
  }
#pragma unroll
  for (int i = 0; i < NM; ++i) oacc[i % DT] = mfma32(va[i], pb[i / DT], oacc[i % DT]);
  __builtin_amdgcn_sched_group_barrier(kSgDsRead, 2 * AHEAD, 0);
#pragma unroll
  for (int i = 0; i < NM - AHEAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(kSgMfma, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kSgDsRead, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(kSgMfma, AHEAD, 0);
}

// Masks of one tile (ragged tail, frame-causal pairs, padding at the end of the tile): invisible
// keys get -inf.  Lane holds keys key0 + 32 kt + 8 (i/4) + 4 (l/32) + i%4 of its query row
// (column l%32); the two lanes l and l^32 together hold the row's 64 keys.
__device__ __forceinline__ void mask_tile(f32x16* sacc, int key0, int fl, const WaveCtx& w) {
  const int pad = (fl >> kFlPadShift) & 127;
  if (key0 + KT > w.klimit_wave || pad) {
    const int lim = min(w.klimit, key0 + KT - pad);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = key0 + 32 * kt + 8 * (i >> 2) + 4 * w.h + (i & 3);
        if (key >= lim) sacc[kt][i] = -INFINITY;
      }
  }
}

// P = 2^(S*scale - m) rounded to bf16 into the four B operands of the P.V product; returns the
// lane's sum of its 32 values (fp32, before rounding).
__device__ __forceinline__ float softmax_exp(const f32x16* sacc, bf16x8* pb, float m, float scale_log2) {
  const float m_use = (m == -INFINITY) ? 0.f : m;
  float rs0 = 0.f, rs1 = 0.f;
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) {
    u32x4 pw;
#pragma unroll
    for (int j2 = 0; j2 < 4; ++j2) {
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[s4 >> 1][8 * (s4 & 1) + 2 * j2], scale_log2, -m_use));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[s4 >> 1][8 * (s4 & 1) + 2 * j2 + 1], scale_log2, -m_use));
      pw[j2] = pack_bf16x2(p0, p1);
      rs0 += p0;
      rs1 += p1;
    }
    pb[s4] = __builtin_bit_cast(bf16x8, pw);
  }
  return rs0 + rs1;
}

// Softmax of one tile with a lazily raised running max (base 2).  P is first formed against the
// current max m_run, which is left alone while every lane's sum of its 32 values stays within
// 2^8 (so no value exceeds 2^8 and the O accumulators keep their range); otherwise, and on the
// first tile of a piece, the row max of the tile is taken, m_run raised to it, O and l rescaled,
// and P formed again.  Most tiles thus skip both the row max and the rescale.  A wave that does
// not own the tile (use false) runs the first pass on stale scores and drops the result.
template <int D>
__device__ __forceinline__ void softmax_tile(f32x16* sacc, bf16x8* pb, f32x16* oacc, float& m_run, float& l_run,
                                             float scale_log2, bool use) {
  constexpr int DT = D / 32;
  float rs = softmax_exp(sacc, pb, m_run, scale_log2);
  const bool redo = use && (m_run == -INFINITY || !(rs <= 256.f));
  if (__any(redo)) {
    if (use) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kt][i]);
      // lanes l and l^32: the swap gives every lane both halves' values
      const auto sw = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, mx),
                                                       __builtin_bit_cast(uint32_t, mx), false, false);
      mx = fmaxf(__builtin_bit_cast(float, (uint32_t)sw[0]), __builtin_bit_cast(float, (uint32_t)sw[1]));
      const float mt = mx * scale_log2;
      if (mt > m_run) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - mt);   // 0 while m_run is -inf
        m_run = mt;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[dt][i] *= alpha;
      }
    }
    rs = softmax_exp(sacc, pb, m_run, scale_log2);
  }
  l_run += use ? rs : 0.f;
}

// ---------------------------------------------------------------------------
// Work plan.  The query blocks of each (batch, head) bh are ordered by the first historical key
// block they keep and cut into groups of NL = 256 / block: unit u = (bh, g) holds query blocks
// qmap[u NL + L], L < NL (-1 past the last block).  Its tiles are the 64-key sub-tiles of the
// union of its lists in ascending block order, leaving out sub-tiles without a visible key (past
// Lk, or past the block's valid count); ulist[u NK (block / 64) + i] = block << 5 | sub-tile << 4
// | ownership bits (bit L: list L keeps the block), ucount[u] = sub-tiles.  The unit's tiles
// number max(1, ucount[u]): an empty unit gets one unowned tile, so that some workgroup writes
// its output.  The grouping only decides which rows share K/V tiles: any grouping gives the same
// result.

constexpr int kPlanThreads = 256;
constexpr int kMaxGroupNQ = 1024;   // heads with more query blocks keep the natural order

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

// 64-key sub-tiles of key block j that hold a visible key: the block's keys below Lk and, with
// kvalid, its first kvalid[j] keys (clamped to [0, block]); sub-tiles with none are left out of
// the plan (they would contribute nothing but masked MFMA work).
__device__ inline int block_subtiles(int j, int Lk, int block, const int32_t* __restrict__ kvalid) {
  int v = min(block, Lk - j * block);
  if (kvalid) v = min(v, min(max(kvalid[j], 0), block));
  return (v + KT - 1) / KT;
}

// One workgroup per unit: its query blocks (rank by (key, block index) inside the head) and the
// union of their lists with ownership bits, expanded into the sub-tiles that hold visible keys.
// The grouping key of a query block is the first entry of its list past the text blocks when
// that entry is historical (below h1), NK otherwise: the smallest kept historical block for an
// ascending list, as the selection writes them, and read in one or a few loads.  Any other
// list order only changes the grouping.
__global__ __launch_bounds__(kPlanThreads) void plan_union_kernel(const int32_t* __restrict__ counts,
                                                                  const int32_t* __restrict__ idx,
                                                                  const int32_t* __restrict__ kvalid, int NQ, int NK,
                                                                  int h0, int h1, int Lk, int block, int row_tiles,
                                                                  int32_t* __restrict__ qmap,
                                                                  int32_t* __restrict__ ulist,
                                                                  int32_t* __restrict__ ucount) {
  extern __shared__ __align__(16) uint32_t own[];     // 4 ownership bits per key block
  __shared__ int sh[kPlanThreads / 64];
  __shared__ int qsel[4];
  __shared__ int skey[kMaxGroupNQ];
  const int u = blockIdx.x;
  const int bh = u / row_tiles, g = u % row_tiles;
  const int tid = threadIdx.x;
  const int NL = QR / block;
  const int nsub = block / KT;
  const int nwords = (NK + 7) >> 3;
  for (int i = tid; i < nwords; i += kPlanThreads) own[i] = 0;
  if (tid < 4) qsel[tid] = -1;
  const bool grouped = NQ <= kMaxGroupNQ;
  if (grouped)
    for (int i = tid; i < NQ; i += kPlanThreads) {
      const size_t row = (size_t)bh * NQ + i;
      const int n = min(max(counts[row], 0), NK);
      const int32_t* lst = idx + row * NK;
      int key = NK;
      for (int a = 0; a < n; ++a) {
        const int j = lst[a];
        if (j >= h0) {
          key = j < h1 ? j : NK;
          break;
        }
      }
      skey[i] = key;
    }
  __syncthreads();
  if (grouped) {
    for (int i = tid; i < NQ; i += kPlanThreads) {
      const int ki = skey[i];
      int r = 0;
      for (int j = 0; j < NQ; ++j) {
        const int kj = skey[j];
        r += (kj < ki) || (kj == ki && j < i);
      }
      if (r >= g * NL && r < g * NL + NL) qsel[r - g * NL] = i;
    }
  } else if (tid < NL && g * NL + tid < NQ) {
    qsel[tid] = g * NL + tid;
  }
  __syncthreads();
  if (tid < NL) qmap[(size_t)u * NL + tid] = qsel[tid];
  for (int L = 0; L < NL; ++L) {
    const int qb = qsel[L];
    if (qb < 0) continue;
    const size_t row = (size_t)bh * NQ + qb;
    const int n = min(max(counts[row], 0), NK);
    const int32_t* lst = idx + row * NK;
    for (int i = tid; i < n; i += kPlanThreads) {
      const int j = lst[i];
      if ((unsigned)j < (unsigned)NK) atomicOr(&own[j >> 3], (1u << L) << ((j & 7) * 4));
    }
  }
  __syncthreads();
  const int per = (nwords + kPlanThreads - 1) / kPlanThreads;
  const int w0 = min(tid * per, nwords), w1 = min(w0 + per, nwords);
  int cnt = 0;
  for (int wi = w0; wi < w1; ++wi) {
    const uint32_t x = own[wi];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if ((x >> (4 * e)) & 15u) cnt += block_subtiles(8 * wi + e, Lk, block, kvalid);
  }
  int total;
  int pos = block_excl_scan_i(cnt, sh, &total);
  int32_t* out = ulist + (size_t)u * NK * nsub;
  for (int wi = w0; wi < w1; ++wi) {
    const uint32_t x = own[wi];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t bits = (x >> (4 * e)) & 15u;
      if (!bits) continue;
      const int j = 8 * wi + e;
      const int ns = block_subtiles(j, Lk, block, kvalid);
      for (int sub = 0; sub < ns; ++sub) out[pos++] = (j << 5) | (sub << 4) | (int)bits;
    }
  }
  if (tid == 0) ucount[u] = total;
}

// Where every unit's tiles go in the tile sequence, and which tiles each persistent workgroup
// takes.  Units are handed out in two parts:
//   * rounds of whole units: round r gives workgroup lambda = x PX + c (x its XCD, PX = P / 8
//     workgroups per XCD) the unit x R PX + r PX + c, for r < R, unless that unit is longer than
//     thr = T / (P R) tiles.  The workgroups of one XCD thus start consecutive units, i.e. query
//     blocks of the same head, at the same time and walk the head's shared chunk K/V in step,
//     so each K/V tile reaches that XCD's L2 about once per round instead of once per unit.  A
//     workgroup's round units sit one after another at dp_start[lambda] .. dp_start[lambda + 1];
//     by the length limit they add up to at most T / P tiles.
//   * the other units (those past R P and the longer ones), concatenated in unit order after
//     all round units, are shared by stream-K: workgroup lambda takes [sk_start[lambda],
//     sk_start[lambda + 1]), sized so that its round tiles plus this share come as close as
//     possible to T / P.  Units cut at these boundaries are merged afterwards.
// R = (U - P / 4) / P leaves at least P / 4 units to the second part (when U >= P / 4), which
// absorbs the differences in unit length.  tstart[u] = first tile of unit u; tstart[U] = T.
// Computed by one whole workgroup of kPlanThreads >= P threads (sh: its scan scratch); with
// `all` it writes tstart, dp_start and sk_start, and in any case the placing thread writes the
// first tile of unit `me` to *me_start (read after the workgroup's next barrier).
__device__ void schedule_units(const int32_t* __restrict__ ucount, int U, int P, int me, bool all,
                               int32_t* __restrict__ tstart, int32_t* __restrict__ dp_start,
                               int32_t* __restrict__ sk_start, int* sh, int* me_start) {
  const int tid = threadIdx.x;
  const int PX = P >> 3;
  const int R = U > P / 4 ? (U - P / 4) / P : 0;
  const int U1 = R * P;                       // units considered for the rounds
  auto tiles = [&](int u) { return max(1, ucount[u]); };
  auto round_unit = [&](int lambda, int r) { return (lambda / PX) * R * PX + r * PX + lambda % PX; };
  // each thread takes a contiguous run of units, so its loads are independent of each other
  const int C = (U + kPlanThreads - 1) / kPlanThreads;
  const int u_lo = min(U, tid * C), u_hi = min(U, u_lo + C);
  int part = 0;
  for (int u = u_lo; u < u_hi; ++u) part += tiles(u);
  int T;
  block_excl_scan_i(part, sh, &T);
  const int thr = R > 0 ? max(1, (int)((int64_t)T / ((int64_t)P * R))) : 0;
  auto in_rounds = [&](int u) { return u < U1 && tiles(u) <= thr; };
  // round tiles of workgroup tid
  int dp = 0;
  if (tid < P)
#pragma unroll 4
    for (int r = 0; r < R; ++r) {
      const int u = round_unit(tid, r);
      if (in_rounds(u)) dp += tiles(u);
    }
  int Tdp;
  const int dpa = block_excl_scan_i(dp, sh, &Tdp);
  if (tid < P) {
    if (all) dp_start[tid] = dpa;
    int pos = dpa;
    for (int r = 0; r < R; ++r) {
      const int u = round_unit(tid, r);
      if (in_rounds(u)) {
        if (all) tstart[u] = pos;
        if (u == me) *me_start = pos;
        pos += tiles(u);
      }
    }
  }
  if (all && tid == 0) dp_start[P] = Tdp;
  // units of the second part, in unit order after the round units
  int skp = 0;
  for (int u = u_lo; u < u_hi; ++u)
    if (!in_rounds(u)) skp += tiles(u);
  int Tsk_sum;
  int pos = Tdp + block_excl_scan_i(skp, sh, &Tsk_sum);
  for (int u = u_lo; u < u_hi; ++u)
    if (!in_rounds(u)) {
      if (all) tstart[u] = pos;
      if (u == me) *me_start = pos;
      pos += tiles(u);
    }
  if (!all) return;
  const int Tsk = T - Tdp;
  if (tid == 0) tstart[U] = T;
  // second-part shares: quota q = max(0, ceil(T / P) - round tiles), scaled to the Tsk tiles
  // (sum q >= P ceil(T / P) - Tdp >= Tsk, so no share exceeds its quota)
  const int q = tid < P ? max(0, (int)(((int64_t)T + P - 1) / P) - dp) : 0;
  int Q;
  const int qa = block_excl_scan_i(q, sh, &Q);
  if (tid < P) sk_start[tid] = Tdp + (Q > 0 ? (int)((int64_t)Tsk * qa / Q) : 0);
  if (tid == 0) sk_start[P] = T;
}

// The schedule (above) as a launch of its own: one workgroup writes tstart, dp_start, sk_start.
__global__ __launch_bounds__(kPlanThreads) void plan_sched_kernel(const int32_t* __restrict__ ucount, int U, int P,
                                                                  int32_t* __restrict__ tstart,
                                                                  int32_t* __restrict__ dp_start,
                                                                  int32_t* __restrict__ sk_start) {
  __shared__ int sh[kPlanThreads / 64];
  __shared__ int unused;
  schedule_units(ucount, U, P, -1, true, tstart, dp_start, sk_start, sh, &unused);
}

// Units up to which every workgroup of plan_tiles_kernel computes the schedule itself (each reads
// all U unit counts, U^2 reads in all) instead of a launch of plan_sched_kernel before it.
constexpr int kFoldSchedUnits = 1024;

// Expands unit u's union list into one record per 64-key tile at its place in the tile
// sequence.  With fold, every workgroup computes the schedule (above) for its own unit and
// workgroup 0 also writes tstart, dp_start and sk_start for the run and the merge; otherwise the
// place is read from tstart, written by plan_sched_kernel.  With kvalid (valid keys at the front
// of each key block), a tile's padding keys are counted into its flags.
__global__ __launch_bounds__(kPlanThreads) void plan_tiles_kernel(const int32_t* __restrict__ ulist,
                                                                  const int32_t* __restrict__ ucount,
                                                                  const int32_t* __restrict__ kvalid, int U,
                                                                  int P, bool fold, int32_t* __restrict__ tstart,
                                                                  int32_t* __restrict__ dp_start,
                                                                  int32_t* __restrict__ sk_start, int NK,
                                                                  int block, int row_tiles, int4* __restrict__ trec) {
  __shared__ int sh[kPlanThreads / 64];
  __shared__ int first_tile;
  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  if (fold) {
    if (tid == 0) first_tile = 0;
    schedule_units(ucount, U, P, u, u == 0, tstart, dp_start, sk_start, sh, &first_tile);
  } else if (tid == 0) {
    first_tile = tstart[u];
  }
  __syncthreads();
  const int nt = ucount[u], n = nt > 0 ? nt : 1;
  const int nsub = block / KT;
  const int bh = u / row_tiles;
  int4* out = trec + first_tile;
  const int32_t* ul = ulist + (size_t)u * NK * nsub;
  for (int a = tid; a < n; a += kPlanThreads) {
    int key0 = 0, bits = 0;
    if (nt > 0) {
      const int e = ul[a];
      const int j = e >> 5, sub = (e >> 4) & 1;
      key0 = j * block + sub * KT;
      bits = e & 15;
      if (kvalid) {
        const int kv = min(max(kvalid[j], 0), block) - sub * KT;
        bits |= (KT - min(max(kv, 0), KT)) << kFlPadShift;
      }
    }
    out[a] = int4{key0, bh, u, bits | (a == 0 ? kFlFrom0 : 0) | (a == n - 1 ? kFlToEnd : 0)};
  }
}

// The tiles of one workgroup: n1 round tiles from a1, then its stream-K share from a2; its tile
// t (0 <= t < N) is tile at(t) of the sequence.
struct WgTiles {
  int a1, n1, a2, N;
  int Lk, BH, U;          // bounds of a record's first key, head and unit
  __device__ int at(int t) const { return t < n1 ? a1 + t : a2 + (t - n1); }
};

// One tile of a workgroup's work (wave-uniform): record x = first key, y = (batch, head),
// z = unit, w = ownership bits (0..3) | from0 | to_end (the unit's first / last tile), plus
// first / last (the piece's, i.e. the unit's tiles inside this workgroup's round part or share)
// and valid.
struct TileRef {
  int key0, bh, unit, fl;
  __device__ bool valid() const { return fl & kFlValid; }
  __device__ bool owned(int list) const { return (fl >> list) & 1; }
};

__device__ inline TileRef make_tile(const int4& e, int t, const WgTiles& g) {
  TileRef r{0, 0, 0, 0};
  if (t < g.N) {
    // the fields are clamped into range, so that even a plan the workspace no longer holds
    // (overwritten by another call) reads and writes inside q, k, v, o and the workspace
    r.key0 = min(max(e.x, 0), g.Lk);
    r.bh = min(max(e.y, 0), g.BH - 1);
    r.unit = min(max(e.z, 0), g.U - 1);
    r.fl = e.w | kFlValid | ((e.w & kFlFrom0) || t == 0 || t == g.n1 ? kFlFirst : 0) |
           ((e.w & kFlToEnd) || t + 1 == g.N ? kFlLast : 0);
  }
  return r;
}

// The record of the workgroup's tile t, read through the constant address space: the records
// are written by an earlier kernel and never during this one, so the loads can go through the
// scalar cache (s_load).  t is clamped to the last tile (N > 0); make_tile ignores a record past
// the end.
typedef __attribute__((address_space(4))) const int cint32;
__device__ inline int4 load_tile(const int4* __restrict__ trec, int t, const WgTiles& g) {
  const cint32* r = (const cint32*)(trec + g.at(t < g.N ? t : g.N - 1));
  return int4{r[0], r[1], r[2], r[3]};
}

__device__ inline TileRef fetch_tile(const int4* __restrict__ trec, int t, const WgTiles& g) {
  return make_tile(load_tile(trec, t, g), t, g);
}

// State of one wave's running unit piece.
template <int D>
struct WaveState {
  f32x16 oacc[D / 32];
  f32x16 sacc[2];
  bf16x8 pb[4];
  bf16x8 qreg[D / 16];
  float m_run, l_run;
  bool rows;        // the wave's rows exist
  bool from0;       // the running piece starts at its unit's first tile
  int r0w;          // first query row of the wave in its (batch, head)
  int bh;
};

// Shared arguments of the phases.
struct KArgs {
  const uint16_t* q;
  uint16_t* o;
  float* lse;
  float* part_o;
  float* part_m;
  float* part_l;
  const int32_t* qmap;
  Geom gm;
  int lambda;
  int my_list;      // list of the unit (query block) the wave's rows belong to
  int r_sub;        // first row of the wave inside its query block
  int r_off;        // first row of the wave inside the unit: my_list * block + r_sub
  int c32, h;
};

// Starts a piece of the unit of tile t: zero O, reset the running max and sum, load the wave's
// Q rows.
template <int D>
__device__ __forceinline__ void start_piece(WaveState<D>& st, WaveCtx& w, const TileRef& t, const KArgs& ka) {
  constexpr int KS = D / 16, DT = D / 32;
  const Geom& gm = ka.gm;
  st.bh = t.bh;
  const int qb = ka.qmap[(size_t)t.unit * (QR / gm.block) + ka.my_list];
  st.r0w = qb >= 0 && qb < gm.NQ ? qb * gm.block + ka.r_sub : gm.Lq;
  st.rows = st.r0w < gm.Lq;
  st.from0 = t.fl & kFlFrom0;
  st.m_run = -INFINITY;
  st.l_run = 0.f;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) st.oacc[dt][i] = 0.f;
  // Q^T operand (32x32x16 B): lane holds Q[row r0w + l%32][16 ks + 8 (l/32) .. + 7]
  const int row = st.r0w + ka.c32;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    u32x4 qw = u32x4{0u, 0u, 0u, 0u};
    if (row < gm.Lq) qw = *(const u32x4*)(ka.q + ((size_t)st.bh * gm.Lq + row) * D + 16 * ks + 8 * ka.h);
    st.qreg[ks] = __builtin_bit_cast(bf16x8, qw);
  }
  // complete the Q loads here: left pending, they would make every later Q.K^T (reached also
  // without a piece start) wait for all vector memory traffic, the tile loads in flight included
  __builtin_amdgcn_s_waitcnt(0);
  // Key n is visible to query row t when n < Lk and, with frames of F tokens inside the chunk,
  // when its chunk frame is not later than t's: n < chunk0 + (t / F + 1) F (context keys,
  // n < chunk0, always pass).  One limit per lane replaces per-key frame arithmetic.
  const int64_t lim = gm.F > 0 ? (int64_t)gm.chunk0 + ((int64_t)row / gm.F + 1) * gm.F : (int64_t)gm.Lk;
  const int64_t limw = gm.F > 0 ? (int64_t)gm.chunk0 + ((int64_t)st.r0w / gm.F + 1) * gm.F : (int64_t)gm.Lk;
  w.klimit = (int)(lim < gm.Lk ? lim : gm.Lk);
  w.klimit_wave = (int)(limw < gm.Lk ? limw : gm.Lk);
}

// Ends a piece: the normalised bf16 output (and lse) when the piece is the whole unit, else the
// fp32 partial (O unnormalised, running max m, sum l) in slot 2 lambda (the first piece of the
// workgroup's stream-K share, which continues an earlier share) or 2 lambda + 1 (its last,
// continued by a later share).
// The stores are completed before returning (the tile-load waits count only tile loads).
template <int D>
__device__ __forceinline__ void end_piece(const WaveState<D>& st, bool to_end, const KArgs& ka) {
  constexpr int DT = D / 32;
  const Geom& gm = ka.gm;
  const int c32 = ka.c32, h = ka.h;
  // lane holds O^T[32 dt + 8 (i/4) + 4 (l/32) + i%4][query r0w + l%32]
  const float l = st.l_run + __shfl_xor(st.l_run, 32);
  const int qrow = st.r0w + c32;
  if (qrow >= gm.Lq) {
  } else if (st.from0 && to_end) {
    const float inv = l > 0.f ? 1.0f / l : 0.f;
    uint16_t* orow = ka.o + ((size_t)st.bh * gm.Lq + qrow) * D + 4 * h;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        u32x2 ow;
        ow[0] = pack_bf16x2(st.oacc[dt][4 * a4] * inv, st.oacc[dt][4 * a4 + 1] * inv);
        ow[1] = pack_bf16x2(st.oacc[dt][4 * a4 + 2] * inv, st.oacc[dt][4 * a4 + 3] * inv);
        *(u32x2*)(orow + 32 * dt + 8 * a4) = ow;
      }
    if (ka.lse && h == 0)
      ka.lse[(size_t)st.bh * gm.Lq + qrow] = l > 0.f ? (st.m_run + log2f(l)) * 0.69314718055994531f : -INFINITY;
  } else {
    const int slot = 2 * ka.lambda + (st.from0 ? 1 : 0);
    const size_t prow = (size_t)slot * QR + ka.r_off + c32;
    float* po = ka.part_o + prow * D + 4 * h;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4)
        *(f32x4*)(po + 32 * dt + 8 * a4) =
            f32x4{st.oacc[dt][4 * a4], st.oacc[dt][4 * a4 + 1], st.oacc[dt][4 * a4 + 2], st.oacc[dt][4 * a4 + 3]};
    if (h == 0) {
      ka.part_m[prow] = st.m_run;
      ka.part_l[prow] = l;
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
}

// M phase of tile `cur` (flags prev_fl of the previous tile): P.V of the previous tile, end of
// its piece, start of cur's piece, Q.K^T of cur.
template <int D>
__device__ __forceinline__ void m_phase(WaveState<D>& st, WaveCtx& w, int prev_fl, const TileRef& cur,
                                        const unsigned char* kcur, const unsigned char* vprev, const KArgs& ka) {
  if ((prev_fl & kFlValid) && ((prev_fl >> ka.my_list) & 1) && st.rows) pv_tile<D>(vprev, st.pb, st.oacc, w.vbase);
  if ((prev_fl & kFlValid) && (prev_fl & kFlLast)) end_piece<D>(st, prev_fl & kFlToEnd, ka);
  if (cur.valid() && (cur.fl & kFlFirst)) start_piece<D>(st, w, cur, ka);
  if (cur.valid() && cur.owned(ka.my_list) && st.rows) qk_tile<D>(kcur, st.qreg, st.sacc, w.kbase);
}

// V phase of tile `cur`: masks, softmax, P.
template <int D>
__device__ __forceinline__ void v_phase(WaveState<D>& st, const WaveCtx& w, const TileRef& cur, const KArgs& ka) {
  const bool use = cur.valid() && cur.owned(ka.my_list) && st.rows;
  if (use) mask_tile(st.sacc, cur.key0, cur.fl, w);
  softmax_tile<D>(st.sacc, st.pb, st.oacc, st.m_run, st.l_run, w.scale_log2, use);
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const int4* __restrict__ trec, const int32_t* __restrict__ dp_start, const int32_t* __restrict__ sk_start,
    const int32_t* __restrict__ qmap, uint16_t* __restrict__ o, float* __restrict__ lse, float* __restrict__ part_o,
    float* __restrict__ part_m, float* __restrict__ part_l, Geom gm, int Tcap, float scale_log2) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(1024))) unsigned char kb0[T::KBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char kb1[T::KBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char vb0[T::VBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char vb1[T::VBYTES];

  // XCD-aware numbering: hardware places consecutive workgroup ids on consecutive XCDs (round
  // robin over 8); lambda = x PX + c numbers the workgroups of XCD x consecutively, which is
  // the numbering the plan hands out its units in.  P is a multiple of 8.
  const int P = gridDim.x;
  const int lambda = (blockIdx.x & 7) * (P >> 3) + (blockIdx.x >> 3);
  // the workgroup's tiles, clamped into the record array (Tcap records)
  WgTiles g;
  g.a1 = min(max(dp_start[lambda], 0), Tcap);
  g.n1 = min(max(dp_start[lambda + 1] - g.a1, 0), Tcap - g.a1);
  g.a2 = min(max(sk_start[lambda], 0), Tcap);
  g.N = g.n1 + min(max(sk_start[lambda + 1] - g.a2, 0), Tcap - g.a2);
  g.Lk = gm.Lk;
  g.BH = gm.BH;
  g.U = gm.U;
  if (g.N <= 0) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: keeps tile-issue math scalar
  const bool g1 = wave >= 4;                                    // the lagging group
  const int lw = wave & 3;                                      // wave within its group
  const int c32 = lane & 31, h = lane >> 5;

  KArgs ka;
  ka.q = q;
  ka.o = o;
  ka.lse = lse;
  ka.part_o = part_o;
  ka.part_m = part_m;
  ka.part_l = part_l;
  ka.qmap = qmap;
  ka.gm = gm;
  ka.lambda = lambda;
  ka.c32 = c32;
  ka.h = h;
  // the two waves of SIMD s (s and s + 4) own the two 32-row halves of one 64-row query block,
  // or (128-row blocks) waves {0, 1, 4, 5} and {2, 3, 6, 7} own the two blocks
  if (gm.block == 64) {
    ka.my_list = wave & 3;
    ka.r_sub = (wave >> 2) * QW;
    ka.r_off = ka.my_list * 64 + ka.r_sub;
  } else {
    ka.my_list = (wave & 3) >> 1;
    ka.r_sub = ((wave & 1) * 2 + (wave >> 2)) * QW;
    ka.r_off = ka.my_list * 128 + ka.r_sub;
  }

  // lane-constant global offsets of this wave's tile loads (group 1 loads K and V: KPER + 1 and
  // VPER per wave, the last K load by wave 0 only)
  uint32_t koff[T::KPER + 1], voff[T::VPER];
#pragma unroll
  for (int j = 0; j <= T::KPER; ++j) koff[j] = slot_offset<D>(j < T::KPER ? lw + 4 * j : 4 * T::KPER, lane, T::KSLOTS);
#pragma unroll
  for (int j = 0; j < T::VPER; ++j) voff[j] = vslot_offset<D>(lw + 4 * j, lane);
  WaveCtx w;
  w.key_lk = gm.Lk;
  w.kbase = c32 * T::KSTRIDE + 16 * h;
  {
    const int vrow = 4 * h + ((lane & 15) >> 2);   // + multiples of 8 rows in the immediates
    w.vbase = vrow * T::VSTRIDE + 64 * T::vswz(vrow) + 32 * ((lane >> 4) & 1) + 8 * (lane & 3);
  }
  w.h = h;
  w.scale_log2 = scale_log2;
  w.klimit = gm.Lk;
  w.klimit_wave = gm.Lk;

  WaveState<D> st;
  st.m_run = -INFINITY;
  st.l_run = 0.f;
  st.rows = false;
  st.from0 = false;
  st.r0w = 0;
  st.bh = 0;

  const int N = g.N;
  int prev_fl = 0, prev_key0 = 0;      // the previous tile: flags and first key
  TileRef cur = fetch_tile(trec, 0, g);
  TileRef nxt = fetch_tile(trec, 1, g);

  // this (group 1) wave's loads of K(tile tk) into kdst and V(tile tv) into vdst
  auto issue_loads = [&](unsigned char* kdst, const TileRef& tk, unsigned char* vdst, const TileRef& tv) {
    const LoadSet<T::KPER> kl{tile_load<D>(kdst, k + (size_t)tk.bh * gm.Lk * D, tk.key0, gm.Lk, tk.valid()), lw, koff};
    const LoadSet<T::VPER> vl{tile_load<D>(vdst, v + (size_t)tv.bh * gm.Lk * D, tv.key0, gm.Lk, tv.valid()), lw, voff};
#pragma unroll
    for (int j = 0; j < T::KPER; ++j) kl.issue(j);
    if (lw == 0) kl.issue_at(4 * T::KPER, koff[T::KPER]);
#pragma unroll
    for (int j = 0; j < T::VPER; ++j) vl.issue(j);
  };
  // prologue: K of the first tile
  if (g1) {
    const LoadSet<T::KPER> a{tile_load<D>(kb0, k + (size_t)cur.bh * gm.Lk * D, cur.key0, gm.Lk, cur.valid()), lw,
                             koff};
#pragma unroll
    for (int j = 0; j < T::KPER; ++j) a.issue(j);
    if (lw == 0) a.issue_at(4 * T::KPER, koff[T::KPER]);
    __builtin_amdgcn_s_waitcnt(0);
  }
  lds_barrier();

  // Iteration h (phases A(h), B(h)); K(h) in kb[h & 1], V(h) in vb[h & 1].  Group 1 loads K(h+1)
  // and V(h) in A(h) and waits for them at the end of B(h).  The record of tile h + 2 is fetched
  // (scalar load) at the start of each V phase and decoded at its end, so that no scalar load is
  // outstanding during an M phase (it would force the LDS operand reads there to wait for all
  // LDS traffic).  Two iterations per trip, so that every buffer is a compile-time choice.
  auto run = [&](auto G1) {
    constexpr bool IS_G1 = decltype(G1)::value;
    TileRef nx2;
    auto iteration = [&](int hh, unsigned char* kc, unsigned char* kn, unsigned char* vc, unsigned char* vp) {
      if constexpr (!IS_G1) {
        m_phase<D>(st, w, prev_fl, cur, kc, vp, ka);
        lds_barrier();
        const int4 raw = load_tile(trec, hh + 2, g);
        v_phase<D>(st, w, cur, ka);
        nx2 = make_tile(raw, hh + 2, g);
        lds_barrier();
      } else {
        const int4 raw = load_tile(trec, hh + 2, g);
        v_phase<D>(st, w, TileRef{prev_key0, 0, 0, prev_fl}, ka);
        nx2 = make_tile(raw, hh + 2, g);
        issue_loads(kn, nxt, vc, cur);
        barrier_keep_loads();
        m_phase<D>(st, w, prev_fl, cur, kc, vp, ka);
        __builtin_amdgcn_s_waitcnt(0);
        lds_barrier();
      }
    };
    auto advance = [&]() {
      prev_fl = cur.fl;
      prev_key0 = cur.key0;
      cur = nxt;
      nxt = nx2;
    };
    for (int hh = 0;; hh += 2) {
      iteration(hh, kb0, kb1, vb0, vb1);
      advance();
      if (hh + 1 > N) break;
      iteration(hh + 1, kb1, kb0, vb1, vb0);
      advance();
      if (hh + 2 > N) break;
    }
  };
  if (g1) run(std::true_type{});
  else run(std::false_type{});
}

// Merges the pieces of units that were split across the stream-K shares of the workgroups:
// O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s, over the pieces in share order
// (deterministic).  Workgroup (lambda, c) handles rows [32 c, 32 c + 32) of the unit that starts
// inside workgroup lambda's share and continues past it, if there is one (each split unit has
// exactly one such share).  Units handed out in rounds are never split.
constexpr int kCombRows = 32;
constexpr int kCombThreads = 256;

template <int D>
__global__ __launch_bounds__(kCombThreads) void attn_combine_kernel(const int32_t* __restrict__ tstart,
                                                                    const int32_t* __restrict__ ucount,
                                                                    const int32_t* __restrict__ sk_start,
                                                                    const int4* __restrict__ trec,
                                                                    const int32_t* __restrict__ qmap, int P, int U,
                                                                    int Tcap, int row_tiles, int Lq, int block,
                                                                    const float* __restrict__ part_o,
                                                                    const float* __restrict__ part_m,
                                                                    const float* __restrict__ part_l,
                                                                    uint16_t* __restrict__ o,
                                                                    float* __restrict__ lse) {
  constexpr int CG = D / 4;                    // 4-column groups per row
  constexpr int RSTEP = kCombThreads / CG;     // rows per pass
  constexpr int NI = kCombRows / RSTEP;        // rows per thread
  constexpr int BATCH = 4;                     // pieces whose loads are in flight together
  const int lam0 = blockIdx.x;
  const int b = min(max(sk_start[lam0], 0), Tcap), e = min(max(sk_start[lam0 + 1], 0), Tcap);
  if (b >= e) return;
  // unit holding tile e - 1: its record names it (clamped, like every index read from the plan)
  const int u = min(max(trec[e - 1].z, 0), U - 1);
  const int ts = tstart[u], te = ts + max(1, ucount[u]);
  if (ts < b || te <= e) return;
  // The pieces of the unit, in share order: the last piece of this share (slot 2 lam0 + 1), then
  // the first piece (slot 2 lambda) of every later non-empty share that starts before the unit
  // ends.  Their slots are listed in LDS first, so that the loads of several pieces can be in
  // flight together.
  __shared__ int sh[kCombThreads / 64];
  __shared__ int pslot[kMaxPersist + 1];
  const int lam = lam0 + 1 + threadIdx.x;
  const int a = lam < P ? sk_start[lam] : 0, z = lam < P ? sk_start[lam + 1] : 0;
  const int take = lam < P && a < z && a < te;
  int np;
  const int pos = block_excl_scan_i(take, sh, &np);
  if (take) pslot[1 + pos] = 2 * lam;
  if (threadIdx.x == 0) pslot[0] = 2 * lam0 + 1;
  __syncthreads();
  np += 1;
  const int bh = u / row_tiles;
  const int cg = threadIdx.x % CG, r0 = blockIdx.y * kCombRows + threadIdx.x / CG;
  float m[NI], l[NI];
  f32x4 acc[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    m[i] = -INFINITY;
    l[i] = 0.f;
    acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // batches of pieces: all loads of a batch first, then one rescale of the running (m, l, O) to
  // the batch's max and the pieces added with weights 2^(m_s - m) (0 for an empty piece or a
  // slot past the last piece); no branches, so the loads of a batch overlap
  for (int pc0 = 0; pc0 < np; pc0 += BATCH) {
    float bm[BATCH][NI], bl[BATCH][NI];
    f32x4 bo[BATCH][NI];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const bool ok = pc0 + j < np;
      const size_t pr0 = (size_t)pslot[ok ? pc0 + j : 0] * QR + r0;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const size_t pr = pr0 + RSTEP * i;
        bm[j][i] = ok ? part_m[pr] : -INFINITY;
        bl[j][i] = ok ? part_l[pr] : 0.f;
        bo[j][i] = ok ? *(const f32x4*)(part_o + pr * D + 4 * cg) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      float mn = m[i];
#pragma unroll
      for (int j = 0; j < BATCH; ++j) mn = fmaxf(mn, bm[j][i]);
      const float mu = mn == -INFINITY ? 0.f : mn;
      const float a = exp2f(m[i] - mu);                // 0 while the running max is -inf
      l[i] *= a;
      acc[i] *= a;
#pragma unroll
      for (int j = 0; j < BATCH; ++j) {
        const float wgt = exp2f(bm[j][i] - mu);
        l[i] += wgt * bl[j][i];
        acc[i] += wgt * bo[j][i];
      }
      m[i] = mn;
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int r = r0 + RSTEP * i;                       // row inside the unit
    const int qb = qmap[(size_t)u * (QR / block) + r / block];
    const int qrow = qb * block + r % block;
    if (qb >= 0 && qb <= Lq / block && qrow < Lq) {
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
  int4* trec;
  int32_t* qmap;
  int32_t* ulist;
  int32_t* ucount;
  int32_t* tstart;
  int32_t* dp_start;
  int32_t* sk_start;
  float* part_o;
  float* part_m;
  float* part_l;
  size_t bytes;
};

// Records the workspace holds: at most max(1, NK (block / 64)) tiles per unit.
size_t attn_tile_capacity(const Dims& dm) {
  return (size_t)dm.BH * ceil_div(dm.Lq, QR) * (size_t)dm.NK * (dm.block / KT);
}

AttnWs attn_ws_layout(const Dims& dm, void* base) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const size_t U = (size_t)dm.BH * row_tiles;
  const size_t slots = 2 * (size_t)kMaxPersist;
  size_t off = 0;
  AttnWs w;
  char* b = (char*)base;
  // at most max(1, NK * nsub) tiles per unit
  w.trec = (int4*)(b + off);
  off += align256(U * (size_t)dm.NK * (dm.block / KT) * sizeof(int4));
  w.qmap = (int32_t*)(b + off);
  off += align256(U * (size_t)(QR / dm.block) * sizeof(int32_t));
  w.ulist = (int32_t*)(b + off);
  off += align256(U * (size_t)dm.NK * (dm.block / KT) * sizeof(int32_t));
  w.ucount = (int32_t*)(b + off);
  off += align256(U * sizeof(int32_t));
  w.tstart = (int32_t*)(b + off);
  off += align256((U + 1) * sizeof(int32_t));
  w.dp_start = (int32_t*)(b + off);
  off += align256((kMaxPersist + 1) * sizeof(int32_t));
  w.sk_start = (int32_t*)(b + off);
  off += align256((kMaxPersist + 1) * sizeof(int32_t));
  w.part_o = (float*)(b + off);
  off += align256(slots * QR * dm.d * sizeof(float));
  w.part_m = (float*)(b + off);
  off += align256(slots * QR * sizeof(float));
  w.part_l = (float*)(b + off);
  off += align256(slots * QR * sizeof(float));
  w.bytes = off;
  return w;
}

// Persistent workgroups: one per CU of the current device, a multiple of 8 (XCD round robin),
// at most kMaxPersist (the partial slots of the workspace are sized for that many).
int persistent_workgroups() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 8)
    cus = 8;
  const int p = cus < kMaxPersist ? cus : kMaxPersist;
  return p & ~7;
}

}  // namespace

size_t attn_ws_bytes(const Dims& dm) { return attn_ws_layout(dm, nullptr).bytes; }

hipError_t launch_attn_plan(const Dims& dm, const int32_t* counts, const int32_t* idx, const int32_t* kvalid,
                            void* ws, hipStream_t st) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const int U = dm.BH * row_tiles;
  AttnWs w = attn_ws_layout(dm, ws);
  hipLaunchKernelGGL(plan_union_kernel, dim3(U), dim3(kPlanThreads), (size_t)((dm.NK + 7) / 8) * sizeof(uint32_t),
                     st, counts, idx, kvalid, dm.NQ, dm.NK, dm.h0, dm.h1, dm.Lk, dm.block, row_tiles, w.qmap,
                     w.ulist, w.ucount);
  const int P = persistent_workgroups();
  const bool fold = U <= kFoldSchedUnits;
  if (!fold)
    hipLaunchKernelGGL(plan_sched_kernel, dim3(1), dim3(kPlanThreads), 0, st, w.ucount, U, P, w.tstart, w.dp_start,
                       w.sk_start);
  hipLaunchKernelGGL(plan_tiles_kernel, dim3(U), dim3(kPlanThreads), 0, st, w.ulist, w.ucount, kvalid, U, P, fold,
                     w.tstart, w.dp_start, w.sk_start, dm.NK, dm.block, row_tiles, w.trec);
  return hipGetLastError();
}

hipError_t launch_attn_run(const Dims& dm, const void* q, const void* k, const void* v, float scale, void* o,
                           float* lse, void* ws, hipStream_t st) {
  const int P = persistent_workgroups();
  AttnWs w = attn_ws_layout(dm, ws);
  const int Tcap = (int)attn_tile_capacity(dm);
  Geom gm{dm.Lq, dm.Lk, dm.block, dm.NQ, dm.NK, dm.frame_tokens, dm.chunk0, dm.BH, dm.BH * ceil_div(dm.Lq, QR)};
  const float scale_log2 = scale * 1.4426950408889634f;
  if (dm.d == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(P), dim3(kThreads), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, w.trec, w.dp_start, w.sk_start, w.qmap,
                       (uint16_t*)o, lse, w.part_o, w.part_m, w.part_l, gm, Tcap, scale_log2);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(P), dim3(kThreads), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k, (const uint16_t*)v, w.trec, w.dp_start, w.sk_start, w.qmap,
                       (uint16_t*)o, lse, w.part_o, w.part_m, w.part_l, gm, Tcap, scale_log2);
  return hipGetLastError();
}

hipError_t launch_attn_merge(const Dims& dm, void* o, float* lse, void* ws, hipStream_t st) {
  const int row_tiles = ceil_div(dm.Lq, QR);
  const int P = persistent_workgroups();
  AttnWs w = attn_ws_layout(dm, ws);
  const dim3 cgrid(P, QR / kCombRows);
  if (dm.d == 128)
    hipLaunchKernelGGL(attn_combine_kernel<128>, cgrid, dim3(kCombThreads), 0, st, w.tstart, w.ucount, w.sk_start, w.trec,
                       w.qmap, P, dm.BH * row_tiles, (int)attn_tile_capacity(dm), row_tiles, dm.Lq, dm.block,
                       w.part_o, w.part_m, w.part_l, (uint16_t*)o, lse);
  else
    hipLaunchKernelGGL(attn_combine_kernel<64>, cgrid, dim3(kCombThreads), 0, st, w.tstart, w.ucount, w.sk_start, w.trec,
                       w.qmap, P, dm.BH * row_tiles, (int)attn_tile_capacity(dm), row_tiles, dm.Lq, dm.block,
                       w.part_o, w.part_m, w.part_l, (uint16_t*)o, lse);
  return hipGetLastError();
}

hipError_t read_attn_schedule(const Dims& dm, const void* ws, int32_t* tstart, int32_t* ucount, int32_t* dp_start,
                              int32_t* sk_start, int* P, int* U, hipStream_t st) {
  const AttnWs w = attn_ws_layout(dm, const_cast<void*>(ws));
  *P = persistent_workgroups();
  *U = dm.BH * ceil_div(dm.Lq, QR);
  const struct {
    int32_t* dst;
    const int32_t* src;
    int n;
  } parts[4] = {{tstart, w.tstart, *U + 1}, {ucount, w.ucount, *U}, {dp_start, w.dp_start, *P + 1},
                {sk_start, w.sk_start, *P + 1}};
  for (const auto& c : parts) {
    if (!c.dst) continue;
    const hipError_t e = hipMemcpyAsync(c.dst, c.src, (size_t)c.n * sizeof(int32_t), hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace la
