// Internal launchers of the gfx950 kernels; the C ABI in grace_api.hip calls
// them after validating every argument.  Each returns the launch's HIP status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/grace.h"

namespace grace {

// Cross-attention, beam-as-query: grid over (request, head, beam tile).
hipError_t launch_cross_attn(const void* q, const void* enc_k, const void* enc_v,
                             const int32_t* enc_off, void* out, int32_t B, int32_t M, int32_t H,
                             int32_t d, int32_t sum_L, float scale, bool bf16, hipStream_t stream);

// Paged rearrangement + append.  k_slab/v_slab point at slab `step` of the pools.
hipError_t launch_kv_append(void* k_slab, void* v_slab, const int32_t* table_prev,
                            int32_t* table_next, const int32_t* parents, const void* k_new,
                            const void* v_new, int32_t R, int32_t M, int32_t T_max, int32_t step,
                            int32_t row_bytes, bool copy_k, bool copy_v, int32_t* err_flag,
                            hipStream_t stream);

// Paged self-attention over step+1 tokens.
hipError_t launch_self_attn_step(const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* table, void* out, int32_t R, int32_t H, int32_t d,
                                 int32_t T_max, int32_t step, float scale, bool bf16,
                                 hipStream_t stream);

// Fused append + attend: table update, slab write (unless aliased) and
// self-attention over step+1 tokens in one pass.  R = B*M rows this step,
// parents index B*M_prev previous rows, pool slabs have row stride R_s.
hipError_t launch_self_attn_fused(const void* q, const void* k_new, const void* v_new,
                                  void* k_pool, void* v_pool, const int32_t* table_prev,
                                  int32_t* table_next, const int32_t* parents, void* out, int32_t R,
                                  int32_t M, int32_t M_prev, int32_t R_s, int32_t H, int32_t d,
                                  int32_t T_max, int32_t step, float scale, bool bf16, bool copy_k,
                                  bool copy_v, int32_t* err_flag, hipStream_t stream);

// Beam candidate scores: prev[r] + log_softmax(logits[r]), -inf where filtered.
hipError_t launch_beam_scores(const void* logits, const float* prev, const uint32_t* mask,
                              float* cand, float* row_max, int32_t R, int32_t V, bool bf16,
                              hipStream_t stream);

// Per-request top-k over M*V candidates; k <= beam_topk_max_k(); workspace of
// beam_topk_workspace_bytes(B, M, V) bytes, 8-byte aligned.
hipError_t launch_beam_topk(const float* cand, const float* row_max, int32_t B, int32_t M,
                            int32_t V, int32_t k, void* workspace, int32_t* parents,
                            int32_t* tokens, float* scores, hipStream_t stream);
size_t beam_topk_workspace_bytes(int32_t B, int32_t M, int32_t V);
int32_t beam_topk_max_k();

// Score update and top-k in one: the same outputs as launch_beam_scores then
// launch_beam_topk, with the candidates recomputed from the logits instead of
// written out; workspace of beam_step_workspace_bytes(B, M, V) bytes.
hipError_t launch_beam_step(const void* logits, const float* prev, const uint32_t* mask,
                            int32_t B, int32_t M, int32_t V, int32_t k, bool bf16, void* workspace,
                            int32_t* parents, int32_t* tokens, float* scores, hipStream_t stream);
size_t beam_step_workspace_bytes(int32_t B, int32_t M, int32_t V);

// CD + GTM filter words of every beam row; next trie node of every new beam.
hipError_t launch_gtm_mask(const grace_gtm_index& index, const grace_gtm_user& user,
                           const int32_t* node_ids, int32_t R, int32_t M, uint32_t* mask,
                           int32_t* err_flag, hipStream_t stream);
hipError_t launch_trie_advance(const grace_gtm_index& index, const int32_t* node_prev,
                               const int32_t* parents, const int32_t* tokens, int32_t B,
                               int32_t M_prev, int32_t k, int32_t* node_next, int32_t* err_flag,
                               hipStream_t stream);

// Debug builds: add the device-check counters of the attention kernels' source
// files to acc[0 .. 7] and clear them (synchronous); release builds return
// hipErrorNotSupported.
hipError_t debug_take_cross(uint32_t* acc);
hipError_t debug_take_self(uint32_t* acc);

}  // namespace grace
