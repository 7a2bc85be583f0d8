// Host side of the C ABI declared in include/la.h: argument validation, workspace
// sizing and kernel launches.  Nothing here allocates device memory.
#include <math.h>

#include <mutex>

#include "la_internal.h"

namespace la {

la_status make_dims(const la_shape* s, Dims* o) {
  if (!s) return LA_ERR_ARG;
  if (s->B < 1 || s->H < 1 || s->Lq < 1 || s->Lk < 1) return LA_ERR_SHAPE;
  if (s->d != 64 && s->d != 128) return LA_ERR_SHAPE;
  if (s->block != 64 && s->block != 128) return LA_ERR_SHAPE;
  if (s->n_text < 0 || s->frame_tokens < 0) return LA_ERR_SHAPE;
  if ((int64_t)s->Lq + s->n_text > (int64_t)s->Lk) return LA_ERR_SHAPE;
  // int32 element offsets inside one (b, h) slice and grid limits
  if ((int64_t)s->Lk * s->d >= (int64_t(1) << 31)) return LA_ERR_SHAPE;
  if ((int64_t)s->B * s->H >= 65536) return LA_ERR_SHAPE;
  o->B = s->B; o->H = s->H; o->Lq = s->Lq; o->Lk = s->Lk; o->d = s->d; o->block = s->block;
  o->n_text = s->n_text; o->frame_tokens = s->frame_tokens;
  o->BH = s->B * s->H;
  o->NQ = ceil_div(s->Lq, s->block);
  o->NK = ceil_div(s->Lk, s->block);
  if (o->NK > kMaxKeyBlocks) return LA_ERR_SHAPE;
  o->chunk0 = s->Lk - s->Lq;
  o->h0 = ceil_div(s->n_text, s->block);
  o->h1 = o->chunk0 / s->block;
  if (o->h1 < o->h0) o->h1 = o->h0;
  o->M = o->h1 - o->h0;
  if (o->M > kMaxCandidates) return LA_ERR_SHAPE;
  // the attention work plan numbers 64-key tiles with 32-bit indices: units of 256 query rows
  // times at most NK * block / 64 tiles each
  const int64_t units = (int64_t)o->BH * ceil_div(s->Lq, 256);
  if (units * o->NK * (s->block / 64) >= (int64_t(1) << 31)) return LA_ERR_SHAPE;
  return LA_OK;
}

size_t select_ws_bytes(const Dims& dm) {
  size_t qbar = (size_t)dm.BH * dm.NQ * dm.d * sizeof(float);
  size_t scores = (size_t)dm.BH * dm.NQ * (size_t)(dm.M > 0 ? dm.M : 1) * sizeof(float);
  return align256(qbar) + align256(scores);
}

}  // namespace la

using namespace la;

static bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

extern "C" {

size_t la_workspace_bytes(const la_shape* shape) {
  Dims dm;
  if (make_dims(shape, &dm) != LA_OK) return 0;
  size_t a = select_ws_bytes(dm);
  size_t b = attn_ws_bytes(dm);
  return a > b ? a : b;
}

static la_status select_common(const la_shape* shape, const void* q, const void* k, float tau,
                               int keep_fixed, uint8_t* mask, int32_t* counts, int32_t* idx,
                               void* ws, size_t ws_bytes, void* stream) {
  Dims dm;
  la_status st = make_dims(shape, &dm);
  if (st != LA_OK) return st;
  if (!q || !k || !counts || !idx) return LA_ERR_ARG;
  if (misaligned(q) || misaligned(k)) return LA_ERR_ARG;
  if (!ws || ws_bytes < select_ws_bytes(dm) || ((uintptr_t)ws & 255u)) return LA_ERR_WORKSPACE;
  hipError_t e = launch_select(dm, q, k, tau, keep_fixed, mask, counts, idx, ws, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_select_blocks(const la_shape* shape, const void* q, const void* k, float tau,
                           uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, size_t ws_bytes,
                           void* stream) {
  if (!(tau > 0.0f)) return LA_ERR_ARG;   // also rejects NaN
  return select_common(shape, q, k, tau, -1, mask, counts, idx, ws, ws_bytes, stream);
}

// Scratch of la_select_blocks_noalloc (pooled queries and scores of one call): a device array
// the code object carries, so the call needs no allocation.  Each device holds its own copy, at
// its own address, from module load until the process ends.  In host code `scratch` names a
// host-side stand-in; the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[LA_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up on the first call on that device (with
// it current) and kept.
la_status scratch_of_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LA_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LA_OK;
}
}  // namespace

la_status la_select_blocks_noalloc(const la_shape* shape, const void* q, const void* k, float tau,
                                   uint8_t* mask, int32_t* counts, int32_t* idx, void* stream) {
  if (!(tau > 0.0f)) return LA_ERR_ARG;
  Dims dm;
  la_status st = make_dims(shape, &dm);
  if (st != LA_OK) return st;
  if (!q || !k || !counts || !idx || misaligned(q) || misaligned(k)) return LA_ERR_ARG;
  if (select_ws_bytes(dm) > (size_t)LA_NOALLOC_SCRATCH_BYTES) return LA_ERR_WORKSPACE;
  void* ws = nullptr;
  st = scratch_of_current_device(&ws);
  if (st != LA_OK) return st;
  // every scratch byte the kernels read is written earlier in the same call: nothing to clear
  return select_common(shape, q, k, tau, -1, mask, counts, idx, ws, LA_NOALLOC_SCRATCH_BYTES, stream);
}

la_status la_select_blocks_topk(const la_shape* shape, const void* q, const void* k, int32_t keep_blocks,
                                uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, size_t ws_bytes,
                                void* stream) {
  if (keep_blocks < 0) return LA_ERR_ARG;
  return select_common(shape, q, k, 1.0f, keep_blocks, mask, counts, idx, ws, ws_bytes, stream);
}

static la_status select_pooled_common(const la_shape* shape, const float* qbar, const float* kbar, float tau,
                                      int keep_fixed, uint8_t* mask, int32_t* counts, int32_t* idx, void* ws,
                                      size_t ws_bytes, void* stream) {
  Dims dm;
  la_status st = make_dims(shape, &dm);
  if (st != LA_OK) return st;
  if (!qbar || !kbar || !counts || !idx) return LA_ERR_ARG;
  if (misaligned(qbar) || misaligned(kbar)) return LA_ERR_ARG;
  if (!ws || ws_bytes < select_ws_bytes(dm) || ((uintptr_t)ws & 255u)) return LA_ERR_WORKSPACE;
  hipError_t e = launch_select_pooled(dm, qbar, kbar, tau, keep_fixed, mask, counts, idx, ws, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_pool_blocks(const la_shape* shape, const void* x, int32_t which, float* xbar, void* stream) {
  Dims dm;
  la_status st = make_dims(shape, &dm);
  if (st != LA_OK) return st;
  if (which != LA_POOL_Q && which != LA_POOL_K) return LA_ERR_ARG;
  if (!x || !xbar || misaligned(x) || misaligned(xbar)) return LA_ERR_ARG;
  const int L = which == LA_POOL_Q ? dm.Lq : dm.Lk;
  const int NB = which == LA_POOL_Q ? dm.NQ : dm.NK;
  hipError_t e = launch_pool_blocks(dm, x, L, NB, xbar, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_select_pooled(const la_shape* shape, const float* qbar, const float* kbar, float tau, uint8_t* mask,
                           int32_t* counts, int32_t* idx, void* ws, size_t ws_bytes, void* stream) {
  if (!(tau > 0.0f)) return LA_ERR_ARG;
  return select_pooled_common(shape, qbar, kbar, tau, -1, mask, counts, idx, ws, ws_bytes, stream);
}

la_status la_select_pooled_topk(const la_shape* shape, const float* qbar, const float* kbar, int32_t keep_blocks,
                                uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, size_t ws_bytes,
                                void* stream) {
  if (keep_blocks < 0) return LA_ERR_ARG;
  return select_pooled_common(shape, qbar, kbar, 1.0f, keep_blocks, mask, counts, idx, ws, ws_bytes, stream);
}

static la_status attn_check(const la_shape* shape, Dims* dm, void* ws, size_t ws_bytes) {
  la_status st = make_dims(shape, dm);
  if (st != LA_OK) return st;
  if (!ws || ws_bytes < attn_ws_bytes(*dm) || ((uintptr_t)ws & 255u)) return LA_ERR_WORKSPACE;
  return LA_OK;
}

static la_status qkvo_check(const void* q, const void* k, const void* v, void* o, float scale) {
  if (!q || !k || !v || !o) return LA_ERR_ARG;
  if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(o)) return LA_ERR_ARG;
  if (isnan(scale) || isinf(scale)) return LA_ERR_ARG;
  return LA_OK;
}

static float effective_scale(float scale, const Dims& dm) {
  return scale > 0.0f ? scale : 1.0f / sqrtf((float)dm.d);
}

la_status la_sparse_attn_fwd_valid(const la_shape* shape, const void* q, const void* k, const void* v,
                                   const int32_t* counts, const int32_t* idx, const int32_t* kvalid, float scale,
                                   void* o, float* lse, void* ws, size_t ws_bytes, void* stream) {
  Dims dm;
  la_status st = attn_check(shape, &dm, ws, ws_bytes);
  if (st == LA_OK) st = qkvo_check(q, k, v, o, scale);
  if (st == LA_OK && (!counts || !idx)) st = LA_ERR_ARG;
  if (st != LA_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_attn_plan(dm, counts, idx, kvalid, ws, s);
  if (e == hipSuccess) e = launch_attn_run(dm, q, k, v, effective_scale(scale, dm), o, lse, ws, s);
  if (e == hipSuccess) e = launch_attn_merge(dm, o, lse, ws, s);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_sparse_attn_fwd(const la_shape* shape, const void* q, const void* k, const void* v,
                             const int32_t* counts, const int32_t* idx, float scale, void* o, float* lse,
                             void* ws, size_t ws_bytes, void* stream) {
  return la_sparse_attn_fwd_valid(shape, q, k, v, counts, idx, nullptr, scale, o, lse, ws, ws_bytes, stream);
}

la_status la_sparse_attn_plan_valid(const la_shape* shape, const int32_t* counts, const int32_t* idx,
                                    const int32_t* kvalid, void* ws, size_t ws_bytes, void* stream) {
  Dims dm;
  la_status st = attn_check(shape, &dm, ws, ws_bytes);
  if (st != LA_OK) return st;
  if (!counts || !idx) return LA_ERR_ARG;
  hipError_t e = launch_attn_plan(dm, counts, idx, kvalid, ws, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_sparse_attn_plan(const la_shape* shape, const int32_t* counts, const int32_t* idx, void* ws,
                              size_t ws_bytes, void* stream) {
  return la_sparse_attn_plan_valid(shape, counts, idx, nullptr, ws, ws_bytes, stream);
}

la_status la_sparse_attn_run(const la_shape* shape, const void* q, const void* k, const void* v, float scale,
                             void* o, float* lse, void* ws, size_t ws_bytes, void* stream) {
  Dims dm;
  la_status st = attn_check(shape, &dm, ws, ws_bytes);
  if (st == LA_OK) st = qkvo_check(q, k, v, o, scale);
  if (st != LA_OK) return st;
  hipError_t e = launch_attn_run(dm, q, k, v, effective_scale(scale, dm), o, lse, ws, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_sparse_attn_merge(const la_shape* shape, void* o, float* lse, void* ws, size_t ws_bytes,
                               void* stream) {
  Dims dm;
  la_status st = attn_check(shape, &dm, ws, ws_bytes);
  if (st != LA_OK) return st;
  if (!o || misaligned(o)) return LA_ERR_ARG;
  hipError_t e = launch_attn_merge(dm, o, lse, ws, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_sparse_attn_schedule(const la_shape* shape, const void* ws, size_t ws_bytes, int32_t* P,
                                  int32_t* U, int32_t* tstart, int32_t* ucount, int32_t* dp_start,
                                  int32_t* sk_start, void* stream) {
  Dims dm;
  la_status st = attn_check(shape, &dm, const_cast<void*>(ws), ws_bytes);
  if (st != LA_OK) return st;
  if (!P || !U) return LA_ERR_ARG;
  int p = 0, u = 0;
  hipError_t e = read_attn_schedule(dm, ws, tstart, ucount, dp_start, sk_start, &p, &u, (hipStream_t)stream);
  if (e != hipSuccess) return LA_ERR_HIP;
  *P = p;
  *U = u;
  return LA_OK;
}

la_status la_mask_to_list(const la_shape* shape, const uint8_t* mask, int32_t* counts, int32_t* idx,
                          void* stream) {
  Dims dm;
  la_status st = make_dims(shape, &dm);
  if (st != LA_OK) return st;
  if (!mask || !counts || !idx) return LA_ERR_ARG;
  hipError_t e = launch_mask_to_list(dm, mask, counts, idx, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_grid3d_shape(const la_grid3d* grid, la_shape* tiled) {
  if (!tiled) return LA_ERR_ARG;
  G3Dims gd;
  la_status st = make_g3dims(grid, &gd);
  if (st != LA_OK) return st;
  *tiled = gd.shape;
  return LA_OK;
}

la_status la_grid3d_valid(const la_grid3d* grid, int32_t* qvalid, int32_t* kvalid) {
  G3Dims gd;
  la_status st = make_g3dims(grid, &gd);
  if (st != LA_OK) return st;
  // tokens of 3-D block n of a run of T frames: the block's extents cut at the grid edges
  auto count3 = [&](int T, int n) {
    const int per_frame = gd.nby * gd.nbx;
    const int ct = n / per_frame, rem = n % per_frame;
    const int cy = rem / gd.nbx, cx = rem % gd.nbx;
    const int et = T - ct * gd.bt < gd.bt ? T - ct * gd.bt : gd.bt;
    const int ey = gd.Hs - cy * gd.bh < gd.bh ? gd.Hs - cy * gd.bh : gd.bh;
    const int ex = gd.Ws - cx * gd.bw < gd.bw ? gd.Ws - cx * gd.bw : gd.bw;
    return et * ey * ex;
  };
  if (qvalid)
    for (int n = 0; n < gd.NQ; ++n) qvalid[n] = count3(gd.T_q, n);
  if (kvalid) {
    for (int n = 0; n < gd.NT; ++n) kvalid[n] = gd.n_text - n * gd.block < gd.block ? gd.n_text - n * gd.block : gd.block;
    for (int n = 0; n < gd.NC; ++n) kvalid[gd.NT + n] = count3(gd.T_ctx, n);
    for (int n = 0; n < gd.NQ; ++n) kvalid[gd.NT + gd.NC + n] = count3(gd.T_q, n);
  }
  return LA_OK;
}

la_status la_prep_q_3d(const la_grid3d* grid, const void* q, void* q_tiled, float* qbar, void* stream) {
  G3Dims gd;
  la_status st = make_g3dims(grid, &gd);
  if (st != LA_OK) return st;
  if (!q || !q_tiled || misaligned(q) || misaligned(q_tiled) || misaligned(qbar)) return LA_ERR_ARG;
  hipError_t e = launch_prep_q(gd, q, q_tiled, qbar, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_prep_kv_3d(const la_grid3d* grid, const void* k, const void* v, uint32_t parts, void* k_tiled,
                        void* v_tiled, float* kbar, void* stream) {
  G3Dims gd;
  la_status st = make_g3dims(grid, &gd);
  if (st != LA_OK) return st;
  if (parts == 0 || (parts & ~(uint32_t)LA_PART_ALL)) return LA_ERR_ARG;
  if (!k || !v || !k_tiled || !v_tiled) return LA_ERR_ARG;
  if (misaligned(k) || misaligned(v) || misaligned(k_tiled) || misaligned(v_tiled) || misaligned(kbar))
    return LA_ERR_ARG;
  hipError_t e = launch_prep_kv(gd, k, v, parts, k_tiled, v_tiled, kbar, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_untile_o_3d(const la_grid3d* grid, const void* o_tiled, const float* lse_tiled, void* o, float* lse,
                         void* stream) {
  G3Dims gd;
  la_status st = make_g3dims(grid, &gd);
  if (st != LA_OK) return st;
  if (!o_tiled || !o || misaligned(o_tiled) || misaligned(o)) return LA_ERR_ARG;
  hipError_t e = launch_untile_o(gd, o_tiled, lse_tiled, o, lse, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_latent_mse(const void* z_a, const void* z_b, int64_t n, int32_t dtype, double* out, void* ws,
                        size_t ws_bytes, void* stream) {
  if (!z_a || !z_b || !out || n < 1) return LA_ERR_ARG;
  if (dtype != LA_DTYPE_F32 && dtype != LA_DTYPE_BF16) return LA_ERR_ARG;
  if (misaligned(z_a) || misaligned(z_b) || ((uintptr_t)out & 7u)) return LA_ERR_ARG;
  if (!ws || ws_bytes < LA_LATENT_MSE_WS_BYTES || ((uintptr_t)ws & 255u)) return LA_ERR_WORKSPACE;
  hipError_t e = launch_latent_mse(z_a, z_b, n, dtype == LA_DTYPE_BF16, out, ws, (hipStream_t)stream);
  return e == hipSuccess ? LA_OK : LA_ERR_HIP;
}

la_status la_dynamics_ema(double D_t, const double* D_bar_prev, double alpha, double* D_bar) {
  if (!D_bar || !(alpha > 0.0 && alpha <= 1.0) || !(D_t >= 0.0)) return LA_ERR_ARG;
  if (D_bar_prev && !(*D_bar_prev >= 0.0)) return LA_ERR_ARG;
  *D_bar = D_bar_prev ? alpha * D_t + (1.0 - alpha) * *D_bar_prev : D_t;
  return LA_OK;
}

la_status la_temporal_window(double D_bar, double kappa, int32_t L_m, int32_t* L_t) {
  if (!L_t || !(kappa > 0.0) || L_m < 1 || !(D_bar >= 0.0)) return LA_ERR_ARG;
  const double x = floor((double)L_m * kappa / (D_bar + kappa));
  *L_t = x < 1.0 ? 1 : (x > (double)L_m ? L_m : (int32_t)x);
  return LA_OK;
}

la_status la_pose_revisiting(const float* similarities, int32_t n, float tau_pose, int32_t* revisiting) {
  if (!revisiting || n < 0 || (n > 0 && !similarities) || isnan(tau_pose)) return LA_ERR_ARG;
  float mx = -INFINITY;
  for (int32_t j = 0; j < n; ++j) {
    if (isnan(similarities[j])) return LA_ERR_ARG;
    mx = similarities[j] > mx ? similarities[j] : mx;
  }
  *revisiting = (n > 0 && mx >= tau_pose) ? 1 : 0;
  return LA_OK;
}

la_status la_denoise_schedule(int32_t K, int32_t reuse, int32_t* source) {
  if (K < 1 || !source) return LA_ERR_ARG;
  for (int32_t i = 0; i < K; ++i) source[i] = (reuse && K > 2 && i > 0 && i < K - 1) ? 0 : i;
  return LA_OK;
}

const char* la_status_string(la_status s) {
  switch (s) {
    case LA_OK: return "ok";
    case LA_ERR_ARG: return "invalid argument";
    case LA_ERR_SHAPE: return "unsupported or inconsistent shape";
    case LA_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case LA_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

int32_t la_abi_version(void) { return 1; }

}  // extern "C"
