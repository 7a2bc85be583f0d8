// 3-D block layout on gfx950 (Sec. 3.3: visual tokens in (B_t, B_h, B_w) blocks, and the fused
// Q-Prep / KV-Prep / Untile Scatter of its operator fusion).
//
// Every kernel here is a streaming copy bound by HBM: one workgroup per (block, head) moves the
// block's rows between the linear (AR) order and the block-major order, 16 bytes per lane, all of
// a lane's loads in flight before its first store.  A block's tokens are runs of bw consecutive
// tokens of one frame row (bw d 2 bytes each), so the linear-side accesses are whole runs and the
// block-major side is one contiguous span.
//   prep_kernel<NSRC = 1>  Q-Prep: chunk queries -> block-major Q, and the block means q_bar.
//   prep_kernel<NSRC = 2>  KV-Prep: K and V of one region (text, context or chunk) -> block-major
//                          K and V, and the block means k_bar of K.  One launch per region; the
//                          context region (read once per AR chunk, the bulk of the bytes) is read
//                          with non-temporal loads, so its stream does not displace the cached
//                          data of the passes that follow.
//   untile_kernel          block-major O (and lse) -> linear order, padding slots dropped.
// Means are sums of the bf16 values in fp32 over the block's valid tokens, then one multiply by
// 1 / count; padding slots load as zero and add nothing.
#include <type_traits>

#include "la_internal.h"

namespace la {
namespace {

constexpr int kTileThreads = 256;

// One run of consecutive tiled blocks cut from one stretch of the linear sequence: a run of T
// frames of Hs x Ws tokens in 3-D blocks, or (T == 0) n1d tokens in 1-D blocks of `block`.
struct Run {
  int blk0;    // first tiled block of the run (its row in the block-major buffer is blk0 block)
  int lin0;    // first linear token of the run
  int T;       // frames; 0 = 1-D blocks
  int n1d;     // tokens of a 1-D run
};

struct Grid3 {
  int Hs, Ws, bt, bh, bw;
  int nby, nbx;       // blocks per frame column / row
  int Lin;            // tokens per (b, h) in the linear buffer
  int Ltile;          // slots per (b, h) in the block-major buffer
  int NBbar;          // rows per (b, h) of the means buffer
};

// Where block n of a run lives in the linear sequence: first token, valid tokens and the extents
// (rows ey of ex tokens per frame) that map slot s to a token.
struct BlockMap {
  int base, valid, ey, ex;
  __device__ int token(int s, const Grid3& g) const {
    const int per_t = ey * ex;
    const int dt = s / per_t, r = s - dt * per_t;
    const int dy = r / ex, dx = r - dy * ex;
    return base + (dt * g.Hs + dy) * g.Ws + dx;
  }
};

template <int BLOCK>
__device__ inline BlockMap block_map(const Grid3& g, const Run& run, int n) {
  BlockMap m;
  if (run.T == 0) {
    m.base = run.lin0 + n * BLOCK;
    m.valid = min(BLOCK, run.n1d - n * BLOCK);
    m.ey = 1;
    m.ex = BLOCK;
    return m;
  }
  const int per_frame = g.nby * g.nbx;
  const int ct = n / per_frame, rem = n - ct * per_frame;
  const int cy = rem / g.nbx, cx = rem - cy * g.nbx;
  const int et = min(g.bt, run.T - ct * g.bt);
  m.ey = min(g.bh, g.Hs - cy * g.bh);
  m.ex = min(g.bw, g.Ws - cx * g.bw);
  m.valid = et * m.ey * m.ex;
  m.base = run.lin0 + ((ct * g.bt) * g.Hs + cy * g.bh) * g.Ws + cx * g.bw;
  return m;
}

__device__ inline void acc_bf16x8(float* a, u32x4 w) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    a[2 * e] += __uint_as_float(w[e] << 16);
    a[2 * e + 1] += __uint_as_float(w[e] & 0xffff0000u);
  }
}

// Token of every slot of block n (padding slots: the block's first token, a valid address whose
// load is then dropped), one slot per thread, into LDS.
template <int BLOCK>
__device__ inline void slot_tokens(const Grid3& g, const BlockMap& bm, int* tok) {
  for (int s = threadIdx.x; s < BLOCK; s += kTileThreads) tok[s] = bm.token(s < bm.valid ? s : 0, g);
  __syncthreads();
}

// Lane layout: chunk c = tid % CH (16 bytes of a row), slot tid / CH + RPP p for pass p.  The
// loads are unconditional (padding slots read the block's first token and are zeroed), so all
// NP (K: and NP V) loads of a lane are in flight before the first store.  NT: non-temporal loads.
template <int D, int BLOCK, int NSRC, bool NT = false>
__global__ __launch_bounds__(kTileThreads) void prep_kernel(const uint16_t* __restrict__ src0,
                                                            const uint16_t* __restrict__ src1,
                                                            uint16_t* __restrict__ dst0, uint16_t* __restrict__ dst1,
                                                            float* __restrict__ bar, Grid3 g, Run run) {
  constexpr int CH = D / 8;
  constexpr int RPP = kTileThreads / CH;
  constexpr int NP = BLOCK / RPP;
  __shared__ float red[kTileThreads / 64][D];
  __shared__ int tok[BLOCK];
  const int n = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, c = tid % CH, r0 = tid / CH;
  const BlockMap bm = block_map<BLOCK>(g, run, n);
  slot_tokens<BLOCK>(g, bm, tok);
  const uint16_t* s0 = src0 + (size_t)bh * g.Lin * D + c * 8;
  const uint16_t* s1 = NSRC == 2 ? src1 + (size_t)bh * g.Lin * D + c * 8 : nullptr;
  u32x4 a[NP], b[NSRC == 2 ? NP : 1];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int off = tok[r0 + RPP * p] * D;
    const u32x4* pa = (const u32x4*)(s0 + off);
    a[p] = NT ? __builtin_nontemporal_load(pa) : *pa;
    if constexpr (NSRC == 2) {
      const u32x4* pb = (const u32x4*)(s1 + off);
      b[p] = NT ? __builtin_nontemporal_load(pb) : *pb;
    }
  }
  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const bool ok = r0 + RPP * p < bm.valid;
    a[p] = ok ? a[p] : zero;
    if constexpr (NSRC == 2) b[p] = ok ? b[p] : zero;
  }
  uint16_t* d0 = dst0 + ((size_t)bh * g.Ltile + (size_t)(run.blk0 + n) * BLOCK) * D + c * 8;
  uint16_t* d1 = NSRC == 2 ? dst1 + ((size_t)bh * g.Ltile + (size_t)(run.blk0 + n) * BLOCK) * D + c * 8 : nullptr;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int off = (r0 + RPP * p) * D;
    *(u32x4*)(d0 + off) = a[p];
    if constexpr (NSRC == 2) *(u32x4*)(d1 + off) = b[p];
    acc_bf16x8(acc, a[p]);
  }
  if (!bar) return;
  // lanes of one wave with the same chunk: 64 / CH of them, CH apart
#pragma unroll
  for (int off = CH; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], off);
  const int lane = tid & 63, wave = tid >> 6;
  if (lane < CH) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][c * 8 + e] = acc[e];
  }
  __syncthreads();
  if (tid < D) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kTileThreads / 64; ++w) t += red[w][tid];
    bar[((size_t)bh * g.NBbar + run.blk0 + n) * D + tid] = t * (1.0f / (float)bm.valid);
  }
}

// Rows of padding slots are neither read nor written: their loads read the block's first row
// (a valid address) and their stores are skipped.
template <int D, int BLOCK>
__global__ __launch_bounds__(kTileThreads) void untile_kernel(const uint16_t* __restrict__ ot,
                                                              const float* __restrict__ lset,
                                                              uint16_t* __restrict__ o, float* __restrict__ lse,
                                                              Grid3 g, Run run) {
  constexpr int CH = D / 8;
  constexpr int RPP = kTileThreads / CH;
  constexpr int NP = BLOCK / RPP;
  __shared__ int tok[BLOCK];
  const int n = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, c = tid % CH, r0 = tid / CH;
  const BlockMap bm = block_map<BLOCK>(g, run, n);
  slot_tokens<BLOCK>(g, bm, tok);
  const size_t tile_row = (size_t)bh * g.Ltile + (size_t)(run.blk0 + n) * BLOCK;
  const uint16_t* src = ot + tile_row * D + c * 8;
  uint16_t* dst = o + (size_t)bh * g.Lin * D + c * 8;
  u32x4 a[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int s = r0 + RPP * p;
    a[p] = *(const u32x4*)(src + (s < bm.valid ? s : 0) * D);
  }
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int s = r0 + RPP * p;
    if (s < bm.valid) *(u32x4*)(dst + tok[s] * D) = a[p];
  }
  if (lse && lset) {
    for (int s = tid; s < bm.valid; s += kTileThreads) lse[(size_t)bh * g.Lin + tok[s]] = lset[tile_row + s];
  }
}

template <typename F>
bool dispatch(int d, int block, F f) {
  if (d == 128 && block == 128) return f(std::integral_constant<int, 128>(), std::integral_constant<int, 128>());
  if (d == 128 && block == 64) return f(std::integral_constant<int, 128>(), std::integral_constant<int, 64>());
  if (d == 64 && block == 128) return f(std::integral_constant<int, 64>(), std::integral_constant<int, 128>());
  if (d == 64 && block == 64) return f(std::integral_constant<int, 64>(), std::integral_constant<int, 64>());
  return false;
}

Grid3 grid3(const G3Dims& gd, int Lin, int Ltile, int NBbar) {
  return Grid3{gd.Hs, gd.Ws, gd.bt, gd.bh, gd.bw, gd.nby, gd.nbx, Lin, Ltile, NBbar};
}

}  // namespace

la_status make_g3dims(const la_grid3d* g, G3Dims* o) {
  if (!g) return LA_ERR_ARG;
  if (g->B < 1 || g->H < 1 || (g->d != 64 && g->d != 128)) return LA_ERR_SHAPE;
  if (g->block != 64 && g->block != 128) return LA_ERR_SHAPE;
  if (g->n_text < 0 || g->T_ctx < 0 || g->T_q < 1 || g->Hs < 1 || g->Ws < 1) return LA_ERR_SHAPE;
  if (g->bt < 1 || g->bh < 1 || g->bw < 1) return LA_ERR_SHAPE;
  if ((int64_t)g->bt * g->bh * g->bw > g->block) return LA_ERR_SHAPE;
  const int64_t F = (int64_t)g->Hs * g->Ws;
  const int64_t Lk_lin = g->n_text + ((int64_t)g->T_ctx + g->T_q) * F;
  if (Lk_lin * g->d >= (int64_t(1) << 31)) return LA_ERR_SHAPE;
  o->Hs = g->Hs; o->Ws = g->Ws; o->bt = g->bt; o->bh = g->bh; o->bw = g->bw;
  o->nby = ceil_div(g->Hs, g->bh);
  o->nbx = ceil_div(g->Ws, g->bw);
  const int64_t per_frame = (int64_t)o->nby * o->nbx;
  const int64_t NC = ((int64_t)g->T_ctx + g->bt - 1) / g->bt * per_frame;
  const int64_t NQ = ((int64_t)g->T_q + g->bt - 1) / g->bt * per_frame;
  const int64_t NT = (g->n_text + (int64_t)g->block - 1) / g->block;
  if (NT + NC + NQ > kMaxKeyBlocks) return LA_ERR_SHAPE;
  o->NT = (int)NT; o->NC = (int)NC; o->NQ = (int)NQ; o->NK = (int)(NT + NC + NQ);
  o->F = (int)F;
  o->Lq_lin = (int)(g->T_q * F);
  o->Lk_lin = (int)Lk_lin;
  o->shape = la_shape{g->B, g->H, o->NQ * g->block, o->NK * g->block, g->d, g->block, o->NT * g->block, 0};
  Dims dm;
  const la_status st = make_dims(&o->shape, &dm);
  if (st != LA_OK) return st;
  o->BH = dm.BH;
  o->n_text = g->n_text; o->T_ctx = g->T_ctx; o->T_q = g->T_q;
  o->d = g->d; o->block = g->block;
  return LA_OK;
}

hipError_t launch_prep_q(const G3Dims& gd, const void* q, void* q_tiled, float* qbar, hipStream_t st) {
  const Grid3 g = grid3(gd, gd.Lq_lin, gd.NQ * gd.block, gd.NQ);
  const Run run{0, 0, gd.T_q, 0};
  const dim3 grid(gd.NQ, gd.BH);
  const bool ok = dispatch(gd.d, gd.block, [&](auto D, auto BLOCK) {
    hipLaunchKernelGGL((prep_kernel<D(), BLOCK(), 1>), grid, dim3(kTileThreads), 0, st, (const uint16_t*)q,
                       nullptr, (uint16_t*)q_tiled, nullptr, qbar, g, run);
    return true;
  });
  return ok ? hipGetLastError() : hipErrorInvalidValue;
}

hipError_t launch_prep_kv(const G3Dims& gd, const void* k, const void* v, uint32_t parts, void* k_tiled,
                          void* v_tiled, float* kbar, hipStream_t st) {
  const Grid3 g = grid3(gd, gd.Lk_lin, gd.NK * gd.block, gd.NK);
  Run runs[3];
  int nblk[3], nr = 0;
  bool stream[3];
  if ((parts & LA_PART_TEXT) && gd.NT > 0) {
    runs[nr] = Run{0, 0, 0, gd.n_text};
    stream[nr] = false;
    nblk[nr++] = gd.NT;
  }
  if ((parts & LA_PART_CONTEXT) && gd.NC > 0) {
    runs[nr] = Run{gd.NT, gd.n_text, gd.T_ctx, 0};
    stream[nr] = true;
    nblk[nr++] = gd.NC;
  }
  if (parts & LA_PART_CHUNK) {
    runs[nr] = Run{gd.NT + gd.NC, gd.n_text + gd.T_ctx * gd.F, gd.T_q, 0};
    stream[nr] = false;
    nblk[nr++] = gd.NQ;
  }
  for (int i = 0; i < nr; ++i) {
    const dim3 grid(nblk[i], gd.BH);
    const Run run = runs[i];
    const bool ok = dispatch(gd.d, gd.block, [&](auto D, auto BLOCK) {
      if (stream[i])
        hipLaunchKernelGGL((prep_kernel<D(), BLOCK(), 2, true>), grid, dim3(kTileThreads), 0, st, (const uint16_t*)k,
                           (const uint16_t*)v, (uint16_t*)k_tiled, (uint16_t*)v_tiled, kbar, g, run);
      else
        hipLaunchKernelGGL((prep_kernel<D(), BLOCK(), 2>), grid, dim3(kTileThreads), 0, st, (const uint16_t*)k,
                           (const uint16_t*)v, (uint16_t*)k_tiled, (uint16_t*)v_tiled, kbar, g, run);
      return true;
    });
    if (!ok) return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_untile_o(const G3Dims& gd, const void* o_tiled, const float* lse_tiled, void* o, float* lse,
                           hipStream_t st) {
  const Grid3 g = grid3(gd, gd.Lq_lin, gd.NQ * gd.block, gd.NQ);
  const Run run{0, 0, gd.T_q, 0};
  const dim3 grid(gd.NQ, gd.BH);
  const bool ok = dispatch(gd.d, gd.block, [&](auto D, auto BLOCK) {
    hipLaunchKernelGGL((untile_kernel<D(), BLOCK()>), grid, dim3(kTileThreads), 0, st, (const uint16_t*)o_tiled,
                       lse_tiled, (uint16_t*)o, lse, g, run);
    return true;
  });
  return ok ? hipGetLastError() : hipErrorInvalidValue;
}

}  // namespace la
