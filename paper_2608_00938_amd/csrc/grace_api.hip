// C ABI of the decode-attention library: argument validation on the host,
// dispatch to the gfx950 kernels, HIP error mapping.  Nothing here allocates
// or synchronises; the only state is the thread-local last HIP error and the
// per-GPU address of the allocation-free beam step's scratch array.
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "../../include/grace.h"
#include "kernels.hpp"

namespace {

thread_local int32_t g_last_hip_error = 0;

bool supported_d(int32_t d) { return d == 32 || d == 64 || d == 128; }

int32_t elem_bytes(int32_t dtype) { return dtype == GRACE_F32 ? 4 : 2; }

// Byte ranges [a, a+na) and [b, b+nb) overlap.
bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
  if (na <= 0 || nb <= 0) return false;
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

int32_t hip_status(hipError_t e) {
  if (e == hipSuccess) return GRACE_OK;
  g_last_hip_error = (int32_t)e;
  return GRACE_ERR_HIP;
}

// Common shape checks; sets rows and row bytes.
int32_t check_shape(int32_t B, int32_t M, int32_t H, int32_t d, int32_t dtype, int64_t& R,
                    int64_t& row_bytes) {
  if (dtype != GRACE_F32 && dtype != GRACE_BF16) return GRACE_ERR_UNSUPPORTED;
  if (!supported_d(d)) return GRACE_ERR_UNSUPPORTED;
  if (B < 0 || M < 0 || H < 1 || (int64_t)H * d >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  R = (int64_t)B * M;
  // each factor below 2^31 first, so that the product cannot overflow
  if (R >= ((int64_t)1 << 31) || R * H * d >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  row_bytes = (int64_t)H * d * elem_bytes(dtype);
  return GRACE_OK;
}

bool good_scale(float scale) { return isfinite(scale) && scale > 0.f; }

}  // namespace

extern "C" {

int32_t grace_abi_version(void) { return GRACE_ABI_VERSION; }

int32_t grace_debug_counts(uint32_t* counts) {
  if (!counts) return GRACE_ERR_NULL;
  for (int i = 0; i < GRACE_DEBUG_KINDS; ++i) counts[i] = 0;
#ifdef GRACE_DEBUG
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess) e = grace::debug_take_cross(counts);
  if (e == hipSuccess) e = grace::debug_take_self(counts);
  return hip_status(e);
#else
  return GRACE_ERR_UNSUPPORTED;
#endif
}

int32_t grace_last_hip_error(void) { return g_last_hip_error; }

const char* grace_status_string(int32_t status) {
  switch (status) {
    case GRACE_OK: return "ok";
    case GRACE_ERR_NULL: return "required pointer is NULL";
    case GRACE_ERR_SHAPE: return "size or index argument out of range";
    case GRACE_ERR_UNSUPPORTED: return "unsupported dtype or head dim";
    case GRACE_ERR_ALIAS: return "output overlaps an input";
    case GRACE_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t grace_cross_attn(const void* q, const void* enc_k, const void* enc_v,
                         const int32_t* enc_off, int32_t B, int32_t M, int32_t H, int32_t d,
                         int32_t sum_L, float scale, int32_t dtype, void* out, void* stream) {
  int64_t R, row_bytes;
  int32_t st = check_shape(B, M, H, d, dtype, R, row_bytes);
  if (st != GRACE_OK) return st;
  if (sum_L < 0 || (int64_t)sum_L * H * d >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (!good_scale(scale)) return GRACE_ERR_SHAPE;
  if (R == 0) return GRACE_OK;
  if (!q || !out || !enc_off || (sum_L > 0 && (!enc_k || !enc_v))) return GRACE_ERR_NULL;
  const int64_t qo_bytes = R * row_bytes, kv_bytes = (int64_t)sum_L * row_bytes;
  if (overlaps(out, qo_bytes, q, qo_bytes) || overlaps(out, qo_bytes, enc_k, kv_bytes) ||
      overlaps(out, qo_bytes, enc_v, kv_bytes) || overlaps(out, qo_bytes, enc_off, 4 * (B + 1)))
    return GRACE_ERR_ALIAS;
  return hip_status(grace::launch_cross_attn(q, enc_k, enc_v, enc_off, out, B, M, H, d, sum_L,
                                             scale, dtype == GRACE_BF16, (hipStream_t)stream));
}

int32_t grace_kv_append(void* k_pool, void* v_pool, const int32_t* table_prev,
                        int32_t* table_next, const int32_t* parents, const void* k_new,
                        const void* v_new, int32_t B, int32_t M, int32_t H, int32_t d,
                        int32_t T_max, int32_t step, int32_t dtype, int32_t* err_flag,
                        void* stream) {
  int64_t R, row_bytes;
  int32_t st = check_shape(B, M, H, d, dtype, R, row_bytes);
  if (st != GRACE_OK) return st;
  if (T_max < 1 || T_max > 8 || step < 0 || step >= T_max) return GRACE_ERR_SHAPE;
  if ((int64_t)T_max * R >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (R == 0) return GRACE_OK;
  if (!k_pool || !v_pool || !table_next || !k_new || !v_new) return GRACE_ERR_NULL;
  if (step > 0 && (!table_prev || !parents)) return GRACE_ERR_NULL;
  const int64_t slab = R * row_bytes, table_bytes = R * T_max * 4;
  char* k_slab = (char*)k_pool + step * slab;
  char* v_slab = (char*)v_pool + step * slab;
  if (step > 0 && overlaps(table_next, table_bytes, table_prev, table_bytes)) return GRACE_ERR_ALIAS;
  if (step > 0 && overlaps(table_next, table_bytes, parents, R * 4)) return GRACE_ERR_ALIAS;
  if (overlaps(k_slab, slab, v_slab, slab)) return GRACE_ERR_ALIAS;
  const bool copy_k = k_new != (const void*)k_slab;
  const bool copy_v = v_new != (const void*)v_slab;
  // A source that is not exactly its slab must not overlap any written slab.
  if (copy_k && (overlaps(k_new, slab, k_slab, slab) || overlaps(k_new, slab, v_slab, slab)))
    return GRACE_ERR_ALIAS;
  if (copy_v && (overlaps(v_new, slab, v_slab, slab) || overlaps(v_new, slab, k_slab, slab)))
    return GRACE_ERR_ALIAS;
  const int64_t pool_bytes = slab * T_max;
  if (overlaps(table_next, table_bytes, k_pool, pool_bytes) ||
      overlaps(table_next, table_bytes, v_pool, pool_bytes))
    return GRACE_ERR_ALIAS;
  return hip_status(grace::launch_kv_append(k_slab, v_slab, table_prev, table_next, parents,
                                            k_new, v_new, (int32_t)R, M, T_max, step,
                                            (int32_t)row_bytes, copy_k, copy_v, err_flag,
                                            (hipStream_t)stream));
}

int32_t grace_self_attn_step(const void* q, const void* k_pool, const void* v_pool,
                             const int32_t* table, int32_t B, int32_t M, int32_t H, int32_t d,
                             int32_t T_max, int32_t step, float scale, int32_t dtype, void* out,
                             void* stream) {
  int64_t R, row_bytes;
  int32_t st = check_shape(B, M, H, d, dtype, R, row_bytes);
  if (st != GRACE_OK) return st;
  if (T_max < 1 || T_max > 8 || step < 0 || step >= T_max) return GRACE_ERR_SHAPE;
  if ((int64_t)T_max * R >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (!good_scale(scale)) return GRACE_ERR_SHAPE;
  if (R == 0) return GRACE_OK;
  if (!q || !k_pool || !v_pool || !table || !out) return GRACE_ERR_NULL;
  const int64_t slab = R * row_bytes, pool_bytes = slab * T_max;
  if (overlaps(out, slab, q, slab) || overlaps(out, slab, k_pool, pool_bytes) ||
      overlaps(out, slab, v_pool, pool_bytes) || overlaps(out, slab, table, R * T_max * 4))
    return GRACE_ERR_ALIAS;
  return hip_status(grace::launch_self_attn_step(q, k_pool, v_pool, table, out, (int32_t)R, H, d,
                                                 T_max, step, scale, dtype == GRACE_BF16,
                                                 (hipStream_t)stream));
}

}  // extern "C"

namespace {

struct Range {
  const void* p;
  int64_t n;
};

// Shared by the fixed- and dynamic-width fused entry points: R = B*M_cur rows
// written this step, parents index B*M_prev previous rows, slab row stride R_s.
int32_t fused_impl(const void* q, const void* k_new, const void* v_new, void* k_pool,
                   void* v_pool, const int32_t* table_prev, int32_t* table_next,
                   const int32_t* parents, int32_t B, int32_t M_prev, int32_t M_cur, int32_t R_s,
                   int32_t H, int32_t d, int32_t T_max, int32_t step, float scale, int32_t dtype,
                   void* out, int32_t* err_flag, void* stream) {
  int64_t R, row_bytes;
  int32_t st = check_shape(B, M_cur, H, d, dtype, R, row_bytes);
  if (st != GRACE_OK) return st;
  if (T_max < 1 || T_max > 8 || step < 0 || step >= T_max) return GRACE_ERR_SHAPE;
  if (!good_scale(scale)) return GRACE_ERR_SHAPE;
  if (R == 0) return GRACE_OK;
  if (R_s < R || (int64_t)T_max * R_s >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if ((int64_t)R_s * H * d >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (step > 0 && (M_prev < 1 || (int64_t)B * M_prev > R_s)) return GRACE_ERR_SHAPE;
  if (!q || !k_new || !v_new || !k_pool || !v_pool || !table_next || !out) return GRACE_ERR_NULL;
  if (step > 0 && (!table_prev || !parents)) return GRACE_ERR_NULL;
  const int64_t rows_bytes = R * row_bytes, slab_bytes = (int64_t)R_s * row_bytes;
  char* k_slab = (char*)k_pool + step * slab_bytes;
  char* v_slab = (char*)v_pool + step * slab_bytes;
  const bool copy_k = k_new != (const void*)k_slab;
  const bool copy_v = v_new != (const void*)v_slab;
  const int64_t prev_table_bytes = step > 0 ? (int64_t)B * M_prev * T_max * 4 : 0;
  // Written ranges, then read ranges.  An uncopied slab is read (as k_new/v_new), not written.
  const Range writes[4] = {{out, rows_bytes},
                           {table_next, R * T_max * 4},
                           {copy_k ? k_slab : nullptr, copy_k ? rows_bytes : 0},
                           {copy_v ? v_slab : nullptr, copy_v ? rows_bytes : 0}};
  const Range reads[7] = {{q, rows_bytes},
                          {k_new, rows_bytes},
                          {v_new, rows_bytes},
                          {step > 0 ? table_prev : nullptr, prev_table_bytes},
                          {step > 0 ? parents : nullptr, step > 0 ? R * 4 : 0},
                          {k_pool, step * slab_bytes},
                          {v_pool, step * slab_bytes}};
  for (int i = 0; i < 4; ++i) {
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(writes[i].p, writes[i].n, writes[j].p, writes[j].n)) return GRACE_ERR_ALIAS;
    for (int j = 0; j < 7; ++j)
      if (overlaps(writes[i].p, writes[i].n, reads[j].p, reads[j].n)) return GRACE_ERR_ALIAS;
  }
  return hip_status(grace::launch_self_attn_fused(
      q, k_new, v_new, k_pool, v_pool, table_prev, table_next, parents, out, (int32_t)R, M_cur,
      M_prev, R_s, H, d, T_max, step, scale, dtype == GRACE_BF16, copy_k, copy_v, err_flag,
      (hipStream_t)stream));
}

}  // namespace

extern "C" {

int32_t grace_self_attn_step_fused(const void* q, const void* k_new, const void* v_new,
                                   void* k_pool, void* v_pool, const int32_t* table_prev,
                                   int32_t* table_next, const int32_t* parents, int32_t B,
                                   int32_t M, int32_t H, int32_t d, int32_t T_max, int32_t step,
                                   float scale, int32_t dtype, void* out, int32_t* err_flag,
                                   void* stream) {
  if (B < 0 || M < 0 || (int64_t)B * M >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  return fused_impl(q, k_new, v_new, k_pool, v_pool, table_prev, table_next, parents, B, M, M,
                    B * M, H, d, T_max, step, scale, dtype, out, err_flag, stream);
}

int32_t grace_self_attn_step_fused_dyn(const void* q, const void* k_new, const void* v_new,
                                       void* k_pool, void* v_pool, const int32_t* table_prev,
                                       int32_t* table_next, const int32_t* parents, int32_t B,
                                       int32_t M_prev, int32_t M_cur, int32_t R_s, int32_t H,
                                       int32_t d, int32_t T_max, int32_t step, float scale,
                                       int32_t dtype, void* out, int32_t* err_flag,
                                       void* stream) {
  return fused_impl(q, k_new, v_new, k_pool, v_pool, table_prev, table_next, parents, B, M_prev,
                    M_cur, R_s, H, d, T_max, step, scale, dtype, out, err_flag, stream);
}

int32_t grace_beam_scores(const void* logits, const float* prev_scores, const uint32_t* mask,
                          int32_t R, int32_t V, int32_t dtype, float* cand, float* row_max,
                          void* stream) {
  if (dtype != GRACE_F32 && dtype != GRACE_BF16) return GRACE_ERR_UNSUPPORTED;
  if (R < 0 || V < 1 || (int64_t)R * V >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (R == 0) return GRACE_OK;
  if (!logits || !prev_scores || !cand) return GRACE_ERR_NULL;
  const int64_t n = (int64_t)R * V;
  const int64_t mask_bytes = mask ? (int64_t)R * ((V + 31) / 32) * 4 : 0;
  const Range reads[3] = {{logits, n * elem_bytes(dtype)}, {prev_scores, R * 4}, {mask, mask_bytes}};
  for (const Range& r : reads) {
    if (overlaps(cand, n * 4, r.p, r.n)) return GRACE_ERR_ALIAS;
    if (row_max && overlaps(row_max, (int64_t)R * 4, r.p, r.n)) return GRACE_ERR_ALIAS;
  }
  if (row_max && overlaps(row_max, (int64_t)R * 4, cand, n * 4)) return GRACE_ERR_ALIAS;
  return hip_status(grace::launch_beam_scores(logits, prev_scores, mask, cand, row_max, R, V,
                                              dtype == GRACE_BF16, (hipStream_t)stream));
}

int32_t grace_beam_topk_max_k(void) { return grace::beam_topk_max_k(); }

int64_t grace_beam_topk_workspace_bytes(int32_t B, int32_t M, int32_t V) {
  if (B < 0 || M < 1 || V < 1 || (int64_t)M * V >= ((int64_t)1 << 31)) return -1;
  return (int64_t)grace::beam_topk_workspace_bytes(B, M, V);
}

int32_t grace_beam_topk(const float* cand, const float* row_max, int32_t B, int32_t M, int32_t V,
                        int32_t k, void* workspace, int64_t workspace_bytes, int32_t* parents,
                        int32_t* tokens, float* scores, void* stream) {
  if (B < 0 || M < 1 || V < 1 || (int64_t)M * V >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if ((int64_t)B * M * V >= ((int64_t)1 << 40)) return GRACE_ERR_SHAPE;
  if (k < 1 || k > grace::beam_topk_max_k() || (int64_t)k > (int64_t)M * V) return GRACE_ERR_SHAPE;
  if ((int64_t)B * k >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (B == 0) return GRACE_OK;
  if (!cand || !parents || !tokens || !scores || !workspace) return GRACE_ERR_NULL;
  const int64_t ws_need = (int64_t)grace::beam_topk_workspace_bytes(B, M, V);
  if (workspace_bytes < ws_need || ((uintptr_t)workspace & 7) != 0) return GRACE_ERR_SHAPE;
  const int64_t n = (int64_t)B * M * V * 4, outb = (int64_t)B * k * 4;
  const Range outs[4] = {{parents, outb}, {tokens, outb}, {scores, outb}, {workspace, ws_need}};
  for (int i = 0; i < 4; ++i) {
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return GRACE_ERR_ALIAS;
    if (overlaps(outs[i].p, outs[i].n, cand, n)) return GRACE_ERR_ALIAS;
    if (row_max && overlaps(outs[i].p, outs[i].n, row_max, (int64_t)B * M * 4)) return GRACE_ERR_ALIAS;
  }
  return hip_status(grace::launch_beam_topk(cand, row_max, B, M, V, k, workspace, parents, tokens,
                                            scores, (hipStream_t)stream));
}

int64_t grace_beam_step_workspace_bytes(int32_t B, int32_t M, int32_t V) {
  if (B < 0 || M < 1 || V < 1 || (int64_t)B * M * V >= ((int64_t)1 << 31)) return -1;
  return (int64_t)grace::beam_step_workspace_bytes(B, M, V);
}

}  // extern "C"

namespace {

// Sizes of a beam step (shared by the workspace and the allocation-free entry
// points); GRACE_OK, or the status to return, with B == 0 a no-op.
int32_t check_beam_step_sizes(int32_t B, int32_t M, int32_t V, int32_t k, int32_t dtype) {
  if (dtype != GRACE_F32 && dtype != GRACE_BF16) return GRACE_ERR_UNSUPPORTED;
  if (B < 0 || M < 1 || V < 1 || (int64_t)B * M * V >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (k < 1 || k > grace::beam_topk_max_k() || (int64_t)k > (int64_t)M * V) return GRACE_ERR_SHAPE;
  if ((int64_t)B * k >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  return GRACE_OK;
}

// Pointers and overlaps of a beam step whose workspace is [workspace, +ws_bytes).
int32_t check_beam_step_buffers(const void* logits, const float* prev_scores,
                                const uint32_t* mask, int32_t B, int32_t M, int32_t V, int32_t k,
                                int32_t dtype, const void* workspace, int64_t ws_bytes,
                                const int32_t* parents, const int32_t* tokens,
                                const float* scores) {
  if (!logits || !prev_scores || !parents || !tokens || !scores || !workspace) return GRACE_ERR_NULL;
  const int64_t R = (int64_t)B * M, outb = (int64_t)B * k * 4;
  const Range ins[3] = {{logits, R * V * elem_bytes(dtype)}, {prev_scores, R * 4},
                        {mask, mask ? R * ((V + 31) / 32) * 4 : 0}};
  const Range outs[4] = {{parents, outb}, {tokens, outb}, {scores, outb}, {workspace, ws_bytes}};
  for (int i = 0; i < 4; ++i) {
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return GRACE_ERR_ALIAS;
    for (const Range& r : ins)
      if (overlaps(outs[i].p, outs[i].n, r.p, r.n)) return GRACE_ERR_ALIAS;
  }
  return GRACE_OK;
}

// Workspace of grace_beam_step_noalloc: one copy of this array per GPU, kept
// until the process ends and shared by every call on that GPU.  Host code
// reaches it only through the device address scratch_address() looks up.
constexpr int64_t kNoAllocScratchBytes = GRACE_BEAM_STEP_NOALLOC_MAX_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current GPU's scratch array, looked up the first time
// a call runs on that GPU (with it current) and kept for later calls.
int32_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (dev < 0 || dev >= kMaxDevices) return GRACE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e);
    if (p == nullptr) return GRACE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GRACE_OK;
}

}  // namespace

extern "C" {

int32_t grace_beam_step(const void* logits, const float* prev_scores, const uint32_t* mask,
                        int32_t B, int32_t M, int32_t V, int32_t k, int32_t dtype,
                        void* workspace, int64_t workspace_bytes, int32_t* parents,
                        int32_t* tokens, float* scores, void* stream) {
  int32_t st = check_beam_step_sizes(B, M, V, k, dtype);
  if (st != GRACE_OK || B == 0) return st;
  if (!logits || !prev_scores || !parents || !tokens || !scores || !workspace) return GRACE_ERR_NULL;
  const int64_t ws_need = (int64_t)grace::beam_step_workspace_bytes(B, M, V);
  if (workspace_bytes < ws_need || ((uintptr_t)workspace & 7) != 0) return GRACE_ERR_SHAPE;
  st = check_beam_step_buffers(logits, prev_scores, mask, B, M, V, k, dtype, workspace, ws_need,
                               parents, tokens, scores);
  if (st != GRACE_OK) return st;
  return hip_status(grace::launch_beam_step(logits, prev_scores, mask, B, M, V, k,
                                            dtype == GRACE_BF16, workspace, parents, tokens,
                                            scores, (hipStream_t)stream));
}

int32_t grace_beam_step_noalloc(const void* logits, const float* prev_scores,
                                const uint32_t* mask, int32_t B, int32_t M, int32_t V, int32_t k,
                                int32_t dtype, int32_t* parents, int32_t* tokens, float* scores,
                                void* stream) {
  int32_t st = check_beam_step_sizes(B, M, V, k, dtype);
  if (st != GRACE_OK || B == 0) return st;
  const int64_t ws_need = (int64_t)grace::beam_step_workspace_bytes(B, M, V);
  if (ws_need > kNoAllocScratchBytes) return GRACE_ERR_SHAPE;
  if (!logits || !prev_scores || !parents || !tokens || !scores) return GRACE_ERR_NULL;
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != GRACE_OK) return st;
  st = check_beam_step_buffers(logits, prev_scores, mask, B, M, V, k, dtype, ws, ws_need, parents,
                               tokens, scores);
  if (st != GRACE_OK) return st;
  return hip_status(grace::launch_beam_step(logits, prev_scores, mask, B, M, V, k,
                                            dtype == GRACE_BF16, ws, parents, tokens, scores,
                                            (hipStream_t)stream));
}

}  // extern "C"

namespace {

int32_t check_gtm_index(const grace_gtm_index* x) {
  if (!x) return GRACE_ERR_NULL;
  if (x->vocab < 1 || x->vocab > 4096 || x->num_nodes < 1 || x->num_entries < 0)
    return GRACE_ERR_SHAPE;
  if (x->bitmask_words < 1 || x->bitmask_words > 8 || x->bloom_words < 1 || x->bloom_words > 4)
    return GRACE_ERR_UNSUPPORTED;
  if (x->bitmask_rows < 0 || x->bloom_rows < 0 || x->reserved != 0) return GRACE_ERR_SHAPE;
  if (!x->node_offsets || !x->child_nodes || !x->tokens || !x->bitmask_index || !x->bloom_index)
    return GRACE_ERR_NULL;
  if ((x->bitmask_rows > 0 && !x->bitmask_table) || (x->bloom_rows > 0 && !x->bloom_table))
    return GRACE_ERR_NULL;
  return GRACE_OK;
}

// Ranges of the index arrays (for alias checks against outputs).
void gtm_index_ranges(const grace_gtm_index* x, Range* r) {
  const int64_t E = x->num_entries;
  r[0] = {x->node_offsets, ((int64_t)x->num_nodes + 1) * 4};
  r[1] = {x->child_nodes, E * 4};
  r[2] = {x->tokens, E * 2};
  r[3] = {x->bitmask_index, E * 4};
  r[4] = {x->bloom_index, E * 4};
  r[5] = {x->bitmask_table, (int64_t)x->bitmask_rows * x->bitmask_words * 8};
  r[6] = {x->bloom_table, (int64_t)x->bloom_rows * x->bloom_words * 8};
}

}  // namespace

extern "C" {

int32_t grace_gtm_mask(const grace_gtm_index* index, const grace_gtm_user* user,
                       const int32_t* node_ids, int32_t B, int32_t M, uint32_t* mask,
                       int32_t* err_flag, void* stream) {
  int32_t st = check_gtm_index(index);
  if (st != GRACE_OK) return st;
  if (!user) return GRACE_ERR_NULL;
  if (user->max_locations < 0 || user->max_locations > 64 || user->reserved != 0)
    return GRACE_ERR_SHAPE;
  if (B < 0 || M < 0) return GRACE_ERR_SHAPE;
  const int64_t R = (int64_t)B * M, W = (index->vocab + 31) / 32;
  if (R >= ((int64_t)1 << 31) || R * W >= ((int64_t)1 << 31)) return GRACE_ERR_SHAPE;
  if (R == 0) return GRACE_OK;
  if (!node_ids || !mask || !user->bitmask || !user->num_locations) return GRACE_ERR_NULL;
  if (user->max_locations > 0 && !user->bloom) return GRACE_ERR_NULL;
  Range in[10];
  gtm_index_ranges(index, in);
  in[7] = {node_ids, R * 4};
  in[8] = {user->bitmask, (int64_t)B * index->bitmask_words * 8};
  in[9] = {user->bloom, (int64_t)B * user->max_locations * index->bloom_words * 8};
  for (const Range& r : in)
    if (overlaps(mask, R * W * 4, r.p, r.n)) return GRACE_ERR_ALIAS;
  if (overlaps(mask, R * W * 4, user->num_locations, (int64_t)B * 4)) return GRACE_ERR_ALIAS;
  return hip_status(grace::launch_gtm_mask(*index, *user, node_ids, (int32_t)R, M, mask, err_flag,
                                           (hipStream_t)stream));
}

int32_t grace_trie_advance(const grace_gtm_index* index, const int32_t* node_prev,
                           const int32_t* parents, const int32_t* tokens, int32_t B,
                           int32_t M_prev, int32_t k, int32_t* node_next, int32_t* err_flag,
                           void* stream) {
  int32_t st = check_gtm_index(index);
  if (st != GRACE_OK) return st;
  if (B < 0 || M_prev < 1 || k < 0 || (int64_t)B * k >= ((int64_t)1 << 31) ||
      (int64_t)B * M_prev >= ((int64_t)1 << 31))
    return GRACE_ERR_SHAPE;
  if ((int64_t)B * k == 0) return GRACE_OK;
  if (!node_prev || !parents || !tokens || !node_next) return GRACE_ERR_NULL;
  const int64_t n = (int64_t)B * k * 4;
  Range in[10];
  gtm_index_ranges(index, in);
  in[7] = {node_prev, (int64_t)B * M_prev * 4};
  in[8] = {parents, n};
  in[9] = {tokens, n};
  for (const Range& r : in)
    if (overlaps(node_next, n, r.p, r.n)) return GRACE_ERR_ALIAS;
  return hip_status(grace::launch_trie_advance(*index, node_prev, parents, tokens, B, M_prev, k,
                                               node_next, err_flag, (hipStream_t)stream));
}

}  // extern "C"
