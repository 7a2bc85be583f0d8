// Internal declarations shared by the HIP translation units of libla (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "la.h"

namespace la {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr int kMaxCandidates = 4096;   // M limit of the selection sort (LDS-resident)
constexpr int kMaxKeyBlocks = 16384;   // NK limit (per-row flags live in LDS)

// Shape-derived quantities every entry point needs.
struct Dims {
  int B, H, Lq, Lk, d, block, n_text, frame_tokens;
  int BH, NQ, NK;
  int h0, h1, M;      // historical candidates are key blocks [h0, h1), M = h1 - h0
  int chunk0;         // first chunk key: Lk - Lq
};

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Validates the shape and fills Dims; LA_OK or LA_ERR_SHAPE.
la_status make_dims(const la_shape* s, Dims* out);

// Workspace layout of the selection pass: pooled queries then the score matrix.
size_t select_ws_bytes(const Dims& dm);
// Workspace of the attention pass: work plan (grouping, union lists, tile records, tile prefix
// sums) and the partial (O, m, l) slots of units split across persistent workgroups.
size_t attn_ws_bytes(const Dims& dm);

// Launchers (defined next to their kernels); they only enqueue.
hipError_t launch_select(const Dims& dm, const void* q, const void* k, float tau, int keep_fixed,
                         uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, hipStream_t st);
// Selection from pooled means given by the caller: qbar [BH, NQ, d], kbar [BH, NK, d].
hipError_t launch_select_pooled(const Dims& dm, const float* qbar, const float* kbar, float tau, int keep_fixed,
                                uint8_t* mask, int32_t* counts, int32_t* idx, void* ws, hipStream_t st);
// Block means of x [BH, L, d] in blocks of dm.block rows (ragged last block) into xbar [BH, NB, d].
hipError_t launch_pool_blocks(const Dims& dm, const void* x, int L, int NB, float* xbar, hipStream_t st);
hipError_t launch_mask_to_list(const Dims& dm, const uint8_t* mask, int32_t* counts, int32_t* idx,
                               hipStream_t st);
// The attention pass: work plan from the lists, the attention kernel over the plan, merge of
// the units split across workgroups.
// kvalid: valid keys at the front of each key block, or NULL (all valid).
hipError_t launch_attn_plan(const Dims& dm, const int32_t* counts, const int32_t* idx, const int32_t* kvalid,
                            void* ws, hipStream_t st);
hipError_t launch_attn_run(const Dims& dm, const void* q, const void* k, const void* v, float scale, void* o,
                           float* lse, void* ws, hipStream_t st);
hipError_t launch_attn_merge(const Dims& dm, void* o, float* lse, void* ws, hipStream_t st);
// Copies the schedule arrays of the plan in ws (any destination may be null) and reports the
// persistent workgroup count P and the unit count U they are sized by.
hipError_t read_attn_schedule(const Dims& dm, const void* ws, int32_t* tstart, int32_t* ucount, int32_t* dp_start,
                              int32_t* sk_start, int* P, int* U, hipStream_t st);

// The 3-D block layout of a la_grid3d: block counts, linear lengths and the tiled la_shape.
struct G3Dims {
  int Hs, Ws, bt, bh, bw, nby, nbx;
  int n_text, T_ctx, T_q, d, block, BH;
  int NT, NC, NQ, NK;   // text, context and chunk blocks; NK = NT + NC + NQ
  int F;                // tokens per frame
  int Lq_lin, Lk_lin;   // tokens of the linear query and key sequences
  la_shape shape;       // the tiled problem
};
// Validates the grid and fills G3Dims; LA_OK, LA_ERR_ARG or LA_ERR_SHAPE.
la_status make_g3dims(const la_grid3d* g, G3Dims* out);
hipError_t launch_prep_q(const G3Dims& gd, const void* q, void* q_tiled, float* qbar, hipStream_t st);
hipError_t launch_prep_kv(const G3Dims& gd, const void* k, const void* v, uint32_t parts, void* k_tiled,
                          void* v_tiled, float* kbar, hipStream_t st);
hipError_t launch_untile_o(const G3Dims& gd, const void* o_tiled, const float* lse_tiled, void* o, float* lse,
                           hipStream_t st);

// Latent dynamics (Sec. 3.1): mean squared difference of two latents of n values (fp32 or bf16)
// into out[0] (fp64), through at most kMseMaxBlocks fp64 partials in ws.
constexpr int kMseMaxBlocks = 1024;
int mse_blocks(int64_t n, int bf16);
hipError_t launch_latent_mse(const void* a, const void* b, int64_t n, int bf16, double* out, void* ws,
                             hipStream_t st);

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace la
