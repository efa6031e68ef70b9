// Paged self-attention over short Semantic-ID prefixes and the paged beam
// rearrangement that feeds it (GRACE, Sec. 3.3, Sec. 5.2, Sec. 5.3), for gfx950.
//
// Both kernels are HBM-bound gathers/copies: 16-byte vector loads and stores,
// every load of a row issued before any of its arithmetic, fp32 math, no LDS.
#include "common.hpp"
#include "kernels.hpp"

namespace grace {

// ---------------------------------------------------------------------------
// kv_append: new block-table rows from the parents' rows, fresh block for the
// current position, current token copied into its slab.
// ---------------------------------------------------------------------------

constexpr int kAppendThreads = 256;
constexpr int kAppendUnroll = 4;  // 16-byte chunks in flight per thread and tensor

__global__ void __launch_bounds__(kAppendThreads)
kv_append_kernel(u32x4* __restrict__ k_slab, u32x4* __restrict__ v_slab,
                 const int32_t* __restrict__ table_prev, int32_t* __restrict__ table_next,
                 const int32_t* __restrict__ parents, const u32x4* __restrict__ k_new,
                 const u32x4* __restrict__ v_new, int32_t R, int32_t M, int32_t T_max,
                 int32_t step, int32_t rows_per_block, int32_t chunks_per_row, int32_t copy_k,
                 int32_t copy_v, int32_t* __restrict__ err_flag) {
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int32_t nrows = (int32_t)min<int64_t>(rows_per_block, R - r0);
  if (nrows <= 0) return;

  // Table: nrows * (step+1) entries.
  const int32_t cols = step + 1;
  for (int32_t e = threadIdx.x; e < nrows * cols; e += kAppendThreads) {
    const int32_t i = (int32_t)r0 + e / cols;
    const int32_t j = e % cols;
    int32_t id;
    if (j == step) {
      id = step * R + i;
    } else {
      int32_t p = parents[i];
      if (p < 0 || p >= M) {
        if (err_flag) *err_flag = 1;
        p = p < 0 ? 0 : M - 1;
      }
      const int32_t src = (i / M) * M + p;
      id = table_prev[(int64_t)src * T_max + j];
    }
    table_next[(int64_t)i * T_max + j] = id;
  }

  // Slab copy: the rows are contiguous in both source and destination.
  const int64_t base = r0 * chunks_per_row;
  const int64_t n = (int64_t)nrows * chunks_per_row;
  for (int64_t c0 = threadIdx.x; c0 < n; c0 += (int64_t)kAppendThreads * kAppendUnroll) {
    u32x4 kb[kAppendUnroll], vb[kAppendUnroll];
#pragma unroll
    for (int u = 0; u < kAppendUnroll; ++u) {
      const int64_t c = c0 + (int64_t)u * kAppendThreads;
      if (c < n) {
        if (copy_k) kb[u] = k_new[base + c];
        if (copy_v) vb[u] = v_new[base + c];
      }
    }
#pragma unroll
    for (int u = 0; u < kAppendUnroll; ++u) {
      const int64_t c = c0 + (int64_t)u * kAppendThreads;
      if (c < n) {
        if (copy_k) k_slab[base + c] = kb[u];
        if (copy_v) v_slab[base + c] = vb[u];
      }
    }
  }
}

hipError_t launch_kv_append(void* k_slab, void* v_slab, const int32_t* table_prev,
                            int32_t* table_next, const int32_t* parents, const void* k_new,
                            const void* v_new, int32_t R, int32_t M, int32_t T_max, int32_t step,
                            int32_t row_bytes, bool copy_k, bool copy_v, int32_t* err_flag,
                            hipStream_t stream) {
  const int32_t chunks_per_row = row_bytes / 16;
  // About 32 KiB of each tensor per block.
  int32_t rows_per_block = (32 * 1024) / row_bytes;
  if (rows_per_block < 1) rows_per_block = 1;
  if (rows_per_block > 256) rows_per_block = 256;
  const int64_t blocks = ((int64_t)R + rows_per_block - 1) / rows_per_block;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks), dim3(kAppendThreads), 0, stream,
                     (u32x4*)k_slab, (u32x4*)v_slab, table_prev, table_next, parents,
                     (const u32x4*)k_new, (const u32x4*)v_new, R, M, T_max, step, rows_per_block,
                     chunks_per_row, (int32_t)copy_k, (int32_t)copy_v, err_flag);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// self_attn_step: one query per (row, head) over NT = step+1 paged tokens.
//
// The [R, H, d] arrays are walked as 16-byte chunks; a head is CH = d/VEC
// consecutive chunks and is owned by CH consecutive lanes (CH divides 64, so a
// head never straddles two waves).  Lane group sums give the scores, every
// lane of the group keeps all NT scores, and the softmax over NT <= 8 values
// runs in registers.  Each lane issues all of its q/K/V loads before any math.
// ---------------------------------------------------------------------------

constexpr int kSelfThreads = 256;

template <class T, int D, int NT, int U>
__global__ void __launch_bounds__(kSelfThreads)
self_attn_kernel(const u32x4* __restrict__ q, const u32x4* __restrict__ k_pool,
                 const u32x4* __restrict__ v_pool, const int32_t* __restrict__ table,
                 u32x4* __restrict__ out, int64_t total_chunks, int32_t chunks_per_row,
                 int32_t T_max, uint32_t nblocks, float c_scale) {
  constexpr int VEC = Chunk<T>::kElems;
  constexpr int CH = D / VEC;  // chunks (= lanes) per head
  const int64_t first = ((int64_t)blockIdx.x * kSelfThreads + threadIdx.x);
  const int64_t stride_u = (int64_t)gridDim.x * kSelfThreads;

  u32x4 qc[U], kc[U][NT], vc[U][NT];
  bool live[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t g = first + u * stride_u;
    live[u] = g < total_chunks;
    const int64_t gg = live[u] ? g : 0;
    const int64_t r = gg / chunks_per_row;
    const int32_t c = (int32_t)(gg - r * chunks_per_row);
    qc[u] = q[gg];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      uint32_t id = (uint32_t)table[r * T_max + j];
      id = id < nblocks ? id : nblocks - 1;
      const int64_t off = (int64_t)id * chunks_per_row + c;
      kc[u][j] = k_pool[off];
      vc[u][j] = v_pool[off];
    }
  }

#pragma unroll
  for (int u = 0; u < U; ++u) {
    float qf[VEC];
    Chunk<T>::unpack(qc[u], qf);
    float s[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      float kf[VEC];
      Chunk<T>::unpack(kc[u][j], kf);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc = __builtin_fmaf(qf[e], kf[e], acc);
      s[j] = group_sum<CH>(acc);
    }
    float mx = s[0];
#pragma unroll
    for (int j = 1; j < NT; ++j) mx = fmaxf(mx, s[j]);
    float p[NT], l = 0.f;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      p[j] = fast_exp2((s[j] - mx) * c_scale);
      l += p[j];
    }
    const float inv = 1.0f / l;
    float o[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = 0.f;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      float vf[VEC];
      Chunk<T>::unpack(vc[u][j], vf);
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[e] = __builtin_fmaf(p[j], vf[e], o[e]);
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] *= inv;
    if (live[u]) out[first + u * stride_u] = Chunk<T>::pack(o);
  }
}

template <class T, int D, int NT>
static hipError_t launch_self_nt(const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* table, void* out, int64_t total_chunks,
                                 int32_t chunks_per_row, int32_t T_max, uint32_t nblocks,
                                 float c_scale, hipStream_t stream) {
  // Two chunks per lane keep 2*(2*NT+1) 16-byte loads in flight per lane.
  constexpr int U = NT <= 4 ? 2 : 1;
  int64_t waves_needed = (total_chunks + 64 * U - 1) / (64 * U);
  int64_t blocks = (waves_needed + (kSelfThreads / 64) - 1) / (kSelfThreads / 64);
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL((self_attn_kernel<T, D, NT, U>), dim3((unsigned)blocks), dim3(kSelfThreads),
                     0, stream, (const u32x4*)q, (const u32x4*)k_pool, (const u32x4*)v_pool, table,
                     (u32x4*)out, total_chunks, chunks_per_row, T_max, nblocks, c_scale);
  return hipGetLastError();
}

template <class T, int D>
static hipError_t launch_self_d(const void* q, const void* k_pool, const void* v_pool,
                                const int32_t* table, void* out, int64_t total_chunks,
                                int32_t chunks_per_row, int32_t T_max, int32_t step,
                                uint32_t nblocks, float c_scale, hipStream_t stream) {
  switch (step + 1) {
#define GRACE_NT(n) \
  case n: return launch_self_nt<T, D, n>(q, k_pool, v_pool, table, out, total_chunks, \
                                         chunks_per_row, T_max, nblocks, c_scale, stream);
    GRACE_NT(1) GRACE_NT(2) GRACE_NT(3) GRACE_NT(4) GRACE_NT(5) GRACE_NT(6) GRACE_NT(7) GRACE_NT(8)
#undef GRACE_NT
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_self_attn_step(const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* table, void* out, int32_t R, int32_t H, int32_t d,
                                 int32_t T_max, int32_t step, float scale, bool bf16,
                                 hipStream_t stream) {
  const int32_t elem = bf16 ? 2 : 4;
  const int32_t chunks_per_row = H * d * elem / 16;
  const int64_t total_chunks = (int64_t)R * chunks_per_row;
  const uint32_t nblocks = (uint32_t)((int64_t)T_max * R);
  const float c = scale * kLog2e;
#define GRACE_SELF(TT, DD) \
  return launch_self_d<TT, DD>(q, k_pool, v_pool, table, out, total_chunks, chunks_per_row, \
                               T_max, step, nblocks, c, stream)
  if (bf16) {
    if (d == 32) GRACE_SELF(BF16, 32);
    if (d == 64) GRACE_SELF(BF16, 64);
    if (d == 128) GRACE_SELF(BF16, 128);
  } else {
    if (d == 32) GRACE_SELF(F32, 32);
    if (d == 64) GRACE_SELF(F32, 64);
    if (d == 128) GRACE_SELF(F32, 128);
  }
#undef GRACE_SELF
  return hipErrorInvalidValue;
}

}  // namespace grace
