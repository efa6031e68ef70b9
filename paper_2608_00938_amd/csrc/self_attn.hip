// Paged self-attention over short Semantic-ID prefixes and the paged beam
// rearrangement that feeds it (GRACE, Sec. 3.3, Sec. 5.2, Sec. 5.3), for gfx950.
//
// Both kernels are HBM-bound gathers/copies: 16-byte vector loads and stores,
// every load of a row issued before any of its arithmetic, fp32 math, no LDS.
#include "common.hpp"
#include "debug.hpp"
#include "kernels.hpp"

namespace grace {

GRACE_DEBUG_COUNTERS;

// ---------------------------------------------------------------------------
// kv_append: new block-table rows from the parents' rows, fresh block for the
// current position, current token copied into its slab.  One 16-byte chunk of
// the slab per lane (lane g: row g / chunks_per_row, column g % chunks_per_row);
// the lanes of a row also write its step+1 table entries.  The copy streams
// past the caches (nontemporal loads and stores): nothing reads it again soon.
// ---------------------------------------------------------------------------

constexpr int kAppendThreads = 256;

__global__ void __launch_bounds__(kAppendThreads)
kv_append_kernel(u32x4* __restrict__ k_slab, u32x4* __restrict__ v_slab,
                 const int32_t* __restrict__ table_prev, int32_t* __restrict__ table_next,
                 const int32_t* __restrict__ parents, const u32x4* __restrict__ k_new,
                 const u32x4* __restrict__ v_new, int64_t total_chunks, int32_t chunks_per_row,
                 int32_t R, int32_t M, int32_t T_max, int32_t step, int32_t copy_k,
                 int32_t copy_v, int32_t* __restrict__ err_flag) {
  const int64_t g = (int64_t)blockIdx.x * kAppendThreads + threadIdx.x;
  if (g >= total_chunks) return;
  u32x4 kb, vb;
  if (copy_k) kb = __builtin_nontemporal_load(&k_new[g]);
  if (copy_v) vb = __builtin_nontemporal_load(&v_new[g]);
  const int32_t r = (int32_t)(g / chunks_per_row);
  const int32_t c = (int32_t)(g - (int64_t)r * chunks_per_row);
  if (c <= step) {
    int64_t src = 0;
    if (step > 0) {
      int32_t p = parents[r];
      GRACE_DCHECK(0 <= p && p < M, kDbgParent);
      if (p < 0 || p >= M) {
        if (err_flag) *err_flag = 1;
        p = p < 0 ? 0 : M - 1;
      }
      src = (int64_t)(r / M) * M + p;
    }
    for (int32_t j = c; j <= step; j += chunks_per_row) {
      const int32_t id = j == step ? step * R + r : table_prev[src * T_max + j];
      table_next[(int64_t)r * T_max + j] = id;
    }
  }
  if (copy_k) __builtin_nontemporal_store(kb, &k_slab[g]);
  if (copy_v) __builtin_nontemporal_store(vb, &v_slab[g]);
}

hipError_t launch_kv_append(void* k_slab, void* v_slab, const int32_t* table_prev,
                            int32_t* table_next, const int32_t* parents, const void* k_new,
                            const void* v_new, int32_t R, int32_t M, int32_t T_max, int32_t step,
                            int32_t row_bytes, bool copy_k, bool copy_v, int32_t* err_flag,
                            hipStream_t stream) {
  const int32_t chunks_per_row = row_bytes / 16;
  const int64_t total = (int64_t)R * chunks_per_row;
  const int64_t blocks = (total + kAppendThreads - 1) / kAppendThreads;
  hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)blocks), dim3(kAppendThreads), 0, stream,
                     (u32x4*)k_slab, (u32x4*)v_slab, table_prev, table_next, parents,
                     (const u32x4*)k_new, (const u32x4*)v_new, total, chunks_per_row, R, M, T_max,
                     step, (int32_t)copy_k, (int32_t)copy_v, err_flag);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// self_attn_step: one query per (row, head) over NT = step+1 paged tokens.
//
// The [R, H, d] arrays are walked as 16-byte chunks; a head is CH = d/VEC
// consecutive chunks and is owned by CH consecutive lanes (CH divides 64, so a
// head never straddles two waves).  Lane group sums give the scores, every
// lane of the group keeps all NT scores, and the softmax over NT <= 8 values
// runs in registers.  One chunk per lane; each lane issues all of its q/K/V
// loads before any math.  Streams read or written once (q, the current token,
// the slab written, out) bypass the caches; ancestor blocks, which sibling
// beams share, are ordinary cached loads.
// When a row is a whole number of waves (H*d*elem a multiple of 1 KiB), the
// row index is wave-uniform and the table/parent reads become scalar loads.
// ---------------------------------------------------------------------------

constexpr int kSelfThreads = 256;

// Output chunk of one (row, head-slice): softmax over NT scores, weighted V.
template <class T, int D, int NT>
__device__ __forceinline__ u32x4 attend_chunk(const u32x4& qc, const u32x4* kc, const u32x4* vc,
                                              float c_scale) {
  constexpr int VEC = Chunk<T>::kElems;
  constexpr int CH = D / VEC;  // chunks (= lanes) per head
  float qf[VEC];
  Chunk<T>::unpack(qc, qf);
  float s[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    float kf[VEC];
    Chunk<T>::unpack(kc[j], kf);
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
    Chunk<T>::unpack(vc[j], vf);
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = __builtin_fmaf(p[j], vf[e], o[e]);
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) o[e] *= inv;
  return Chunk<T>::pack(o);
}

// Row of chunk g (g / chunks_per_row); computed once per wave, in scalar
// registers, when rows are whole waves.  Chunk and row indices fit 32 bits:
// the entry points bound R*H*d below 2^31.
template <bool UNIFORM>
__device__ __forceinline__ uint32_t row_of(uint32_t g, const FastDiv& per_row) {
  if constexpr (UNIFORM) return per_row.div(__builtin_amdgcn_readfirstlane(g));
  return per_row.div(g);
}

template <class T, int D, int NT, bool UNIFORM>
__global__ void __launch_bounds__(kSelfThreads)
self_attn_kernel(const u32x4* __restrict__ q, const u32x4* __restrict__ k_pool,
                 const u32x4* __restrict__ v_pool, const int32_t* __restrict__ table,
                 u32x4* __restrict__ out, uint32_t total_chunks, int32_t chunks_per_row,
                 FastDiv per_row, int32_t T_max, uint32_t nblocks, float c_scale) {
  const uint32_t g = xcd_remap(blockIdx.x, gridDim.x) * kSelfThreads + threadIdx.x;
  if (g >= total_chunks) return;   // wave-uniform when UNIFORM (rows are whole waves)
  const uint32_t r = row_of<UNIFORM>(g, per_row);
  const int32_t c = (int32_t)(g - r * (uint32_t)chunks_per_row);
  if constexpr (NT == 1) {
    // one token: its softmax weight is exactly 1, the output is its value
    uint32_t id = (uint32_t)table[(int64_t)r * T_max];
    GRACE_DCHECK(id < nblocks, kDbgBlockId);
    id = id < nblocks ? id : nblocks - 1;
    __builtin_nontemporal_store(v_pool[(int64_t)id * chunks_per_row + c], &out[g]);
    return;
  }
  u32x4 kc[NT], vc[NT];
  const u32x4 qc = __builtin_nontemporal_load(&q[g]);
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    uint32_t id = (uint32_t)table[(int64_t)r * T_max + j];
    GRACE_DCHECK(id < nblocks, kDbgBlockId);
    id = id < nblocks ? id : nblocks - 1;
    const int64_t off = (int64_t)id * chunks_per_row + c;
    kc[j] = k_pool[off];
    vc[j] = v_pool[off];
  }
  __builtin_nontemporal_store(attend_chunk<T, D, NT>(qc, kc, vc, c_scale), &out[g]);
}

// Fused append + attend (the paper's fused and paged self-attention): each row
// takes its parent's block ids for positions < step, writes them and its fresh
// block id to table_next, stores the current token's k/v into slab `step`, and
// attends over the ancestors' blocks plus the current token held in registers.
template <class T, int D, int NT, bool UNIFORM>
__global__ void __launch_bounds__(kSelfThreads)
self_attn_fused_kernel(const u32x4* __restrict__ q, const u32x4* __restrict__ k_new,
                       const u32x4* __restrict__ v_new, u32x4* __restrict__ k_pool,
                       u32x4* __restrict__ v_pool, const int32_t* __restrict__ table_prev,
                       int32_t* __restrict__ table_next, const int32_t* __restrict__ parents,
                       u32x4* __restrict__ out, uint32_t total_chunks, int32_t chunks_per_row,
                       FastDiv per_row, FastDiv per_request, int32_t R_s, int32_t M_prev,
                       int32_t T_max, uint32_t nblocks, float c_scale, int32_t copy_k,
                       int32_t copy_v, int32_t* __restrict__ err_flag) {
  constexpr int STEP = NT - 1;
  const uint32_t g = xcd_remap(blockIdx.x, gridDim.x) * kSelfThreads + threadIdx.x;
  if (g >= total_chunks) return;   // wave-uniform when UNIFORM (rows are whole waves)
  const uint32_t r = row_of<UNIFORM>(g, per_row);
  const int32_t c = (int32_t)(g - r * (uint32_t)chunks_per_row);

  u32x4 kc[NT], vc[NT];
  int32_t ids[NT > 1 ? NT - 1 : 1];
  if constexpr (STEP == 0) {
    // step 0: one token, whose softmax weight is exactly 1, so the output is
    // v_new; q is not needed, and k_new only for its copy into the slab
    vc[0] = __builtin_nontemporal_load(&v_new[g]);
    if (copy_k) __builtin_nontemporal_store(__builtin_nontemporal_load(&k_new[g]), &k_pool[g]);
    if (copy_v) __builtin_nontemporal_store(vc[0], &v_pool[g]);
    if (c == 0) table_next[(int64_t)r * T_max] = (int32_t)r;
    __builtin_nontemporal_store(vc[0], &out[g]);
    return;
  }
  const u32x4 qc = __builtin_nontemporal_load(&q[g]);
  kc[STEP] = __builtin_nontemporal_load(&k_new[g]);
  vc[STEP] = __builtin_nontemporal_load(&v_new[g]);
  if constexpr (STEP > 0) {
    int32_t p = parents[r];
    GRACE_DCHECK(0 <= p && p < M_prev, kDbgParent);
    if (p < 0 || p >= M_prev) {
      if (err_flag) *err_flag = 1;
      p = p < 0 ? 0 : M_prev - 1;
    }
    // the parent's row among B*M_prev (request r / M)
    const int64_t src = (int64_t)per_request.div(r) * M_prev + p;
#pragma unroll
    for (int j = 0; j < STEP; ++j) {
      uint32_t id = (uint32_t)table_prev[src * T_max + j];
      ids[j] = (int32_t)id;
      GRACE_DCHECK(id < nblocks, kDbgBlockId);
      id = id < nblocks ? id : nblocks - 1;
      const int64_t off = (int64_t)id * chunks_per_row + c;
      kc[j] = k_pool[off];
      vc[j] = v_pool[off];
    }
  }

  // Append: slab `step` (streamed past the caches) and the row's table entries.
  const int64_t slab = (int64_t)STEP * R_s * chunks_per_row;
  if (copy_k) __builtin_nontemporal_store(kc[STEP], &k_pool[slab + g]);
  if (copy_v) __builtin_nontemporal_store(vc[STEP], &v_pool[slab + g]);
  for (int32_t j = c; j <= STEP; j += chunks_per_row) {
    int32_t id = (int32_t)(STEP * R_s + r);
#pragma unroll
    for (int i = 0; i < STEP; ++i)
      if (j == i) id = ids[i];
    table_next[(int64_t)r * T_max + j] = id;
  }

  __builtin_nontemporal_store(attend_chunk<T, D, NT>(qc, kc, vc, c_scale), &out[g]);
}

struct SelfArgs {
  const void* q;
  const void* k_new;
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const int32_t* table_prev;  // fused: parents' rows; plain: the table to read
  int32_t* table_next;
  const int32_t* parents;
  void* out;
  uint32_t total_chunks;
  int32_t chunks_per_row, R, M, M_prev, T_max;
  uint32_t nblocks;
  float c_scale;
  int32_t copy_k, copy_v;
  int32_t* err_flag;
};

template <bool FUSED, class T, int D, int NT>
static hipError_t launch_self_nt(const SelfArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.total_chunks + kSelfThreads - 1) / kSelfThreads;
  const bool uniform = a.chunks_per_row % 64 == 0;
#define GRACE_GO(UNI)                                                                              \
  if constexpr (FUSED) {                                                                          \
    hipLaunchKernelGGL((self_attn_fused_kernel<T, D, NT, UNI>), dim3((unsigned)blocks),           \
                       dim3(kSelfThreads), 0, stream, (const u32x4*)a.q, (const u32x4*)a.k_new,   \
                       (const u32x4*)a.v_new, (u32x4*)a.k_pool, (u32x4*)a.v_pool, a.table_prev,   \
                       a.table_next, a.parents, (u32x4*)a.out, a.total_chunks, a.chunks_per_row,   \
                       FastDiv((uint32_t)a.chunks_per_row), FastDiv((uint32_t)a.M), a.R, a.M_prev, \
                       a.T_max, a.nblocks, a.c_scale, a.copy_k, a.copy_v, a.err_flag);             \
  } else {                                                                                        \
    hipLaunchKernelGGL((self_attn_kernel<T, D, NT, UNI>), dim3((unsigned)blocks),                 \
                       dim3(kSelfThreads), 0, stream, (const u32x4*)a.q, (const u32x4*)a.k_pool,  \
                       (const u32x4*)a.v_pool, a.table_prev, (u32x4*)a.out, a.total_chunks,        \
                       a.chunks_per_row, FastDiv((uint32_t)a.chunks_per_row), a.T_max, a.nblocks, \
                       a.c_scale);                                                                \
  }
  if (uniform) {
    GRACE_GO(true)
  } else {
    GRACE_GO(false)
  }
#undef GRACE_GO
  return hipGetLastError();
}

template <bool FUSED, class T, int D>
static hipError_t launch_self_d(const SelfArgs& a, int32_t step, hipStream_t stream) {
  switch (step + 1) {
#define GRACE_NT(n) \
  case n: return launch_self_nt<FUSED, T, D, n>(a, stream);
    GRACE_NT(1) GRACE_NT(2) GRACE_NT(3) GRACE_NT(4) GRACE_NT(5) GRACE_NT(6) GRACE_NT(7) GRACE_NT(8)
#undef GRACE_NT
    default: return hipErrorInvalidValue;
  }
}

template <bool FUSED>
static hipError_t launch_self_any(const SelfArgs& a, int32_t d, int32_t step, bool bf16,
                                  hipStream_t stream) {
#define GRACE_SELF(TT, DD) return launch_self_d<FUSED, TT, DD>(a, step, stream)
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

hipError_t debug_take_self(uint32_t* acc) {
#ifdef GRACE_DEBUG
  uint32_t tmp[kDbgKinds] = {};
  const uint32_t zero[kDbgKinds] = {};
  hipError_t e = hipMemcpyFromSymbol(tmp, HIP_SYMBOL(g_grace_debug), sizeof(tmp));
  if (e == hipSuccess) e = hipMemcpyToSymbol(HIP_SYMBOL(g_grace_debug), zero, sizeof(zero));
  for (int i = 0; i < kDbgKinds; ++i) acc[i] += tmp[i];
  return e;
#else
  (void)acc;
  return hipErrorNotSupported;
#endif
}

hipError_t launch_self_attn_step(const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* table, void* out, int32_t R, int32_t H, int32_t d,
                                 int32_t T_max, int32_t step, float scale, bool bf16,
                                 hipStream_t stream) {
  SelfArgs a = {};
  const int32_t elem = bf16 ? 2 : 4;
  a.q = q;
  a.k_pool = const_cast<void*>(k_pool);
  a.v_pool = const_cast<void*>(v_pool);
  a.table_prev = table;
  a.out = out;
  a.chunks_per_row = H * d * elem / 16;
  a.total_chunks = (uint32_t)((int64_t)R * a.chunks_per_row);   // below 2^29: R*H*d < 2^31
  a.R = R;
  a.T_max = T_max;
  a.nblocks = (uint32_t)((int64_t)T_max * R);
  a.c_scale = scale * kLog2e;
  return launch_self_any<false>(a, d, step, bf16, stream);
}

hipError_t launch_self_attn_fused(const void* q, const void* k_new, const void* v_new,
                                  void* k_pool, void* v_pool, const int32_t* table_prev,
                                  int32_t* table_next, const int32_t* parents, void* out, int32_t R,
                                  int32_t M, int32_t M_prev, int32_t R_s, int32_t H, int32_t d,
                                  int32_t T_max, int32_t step, float scale, bool bf16, bool copy_k,
                                  bool copy_v, int32_t* err_flag, hipStream_t stream) {
  SelfArgs a = {};
  const int32_t elem = bf16 ? 2 : 4;
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.table_prev = table_prev;
  a.table_next = table_next;
  a.parents = parents;
  a.out = out;
  a.chunks_per_row = H * d * elem / 16;
  a.total_chunks = (uint32_t)((int64_t)R * a.chunks_per_row);   // R = B*M rows written this step
  a.R = R_s;                                        // slab row stride of the pools
  a.M = M;
  a.M_prev = M_prev;
  a.T_max = T_max;
  a.nblocks = (uint32_t)((int64_t)T_max * R_s);
  a.c_scale = scale * kLog2e;
  a.copy_k = copy_k;
  a.copy_v = copy_v;
  a.err_flag = err_flag;
  return launch_self_any<true>(a, d, step, bf16, stream);
}

}  // namespace grace
