// Beam score update and per-request top-k (GRACE, Sec. 3.1, Sec. 3.3) for gfx950.
//
// scores: one wave per beam row.  The row's log-softmax over the vocabulary is
//   added to the beam's accumulated score; filtered tokens score -inf.  The
//   kernel also writes each row's best candidate score.
// top-k:  per request, slices of its M*V candidates spread over several
//   workgroups (maxima, histograms, gather), then one 1024-thread workgroup
//   for the boundary bin and one for the final ranking.
//   Candidates are totally ordered by an order-preserving 32-bit key of the
//   score (descending; -0 == +0; NaN below -inf), then by flat index m*V + v
//   (ascending), so the selection is unique.  Sampled path: a 4096-bin
//   histogram, over a sixteenth of the candidates, of the scores in the
//   64-unit window below the request's best score picks the bin above which
//   about 1.25 k candidates are expected; one pass gathers every candidate in
//   that bin and above and counts them, and the set is kept when it holds at
//   least k and fits the list.  Otherwise the full path: the same histogram
//   over every candidate finds the bin holding the k-th candidate, and only
//   candidates in that bin and above are gathered.  When the k-th candidate lies
//   outside the window or the gathered set would not fit, an exact radix
//   select on the key (four 8-bit digits) and an index-ordered collection of
//   the tied candidates take over.  Either way the k winners are sorted by
//   (key desc, index asc): ranked by a counting sort over the window bins and
//   a comparison inside each bin, or by a bitonic sort in LDS when a bin is crowded.
#include "common.hpp"
#include "kernels.hpp"

namespace grace {

// ---------------------------------------------------------------------------
// candidate scores
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

template <class T>
__device__ __forceinline__ float load_logit(const T* p);
template <>
__device__ __forceinline__ float load_logit<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_logit<uint16_t>(const uint16_t* p) {
  return __uint_as_float((uint32_t)*p << 16);
}

constexpr int kScoreThreads = 256;

// Generic row kernel (any V): lanes stride over the row.  CAND = false writes
// only the row's log-sum-exp (lse_out) and best score, for a top-k that
// recomputes each candidate from the logits.
template <class T, bool CAND = true>
__global__ void __launch_bounds__(kScoreThreads)
beam_scores_kernel(const T* __restrict__ logits, const float* __restrict__ prev,
                   const uint32_t* __restrict__ mask, float* __restrict__ cand,
                   float* __restrict__ row_max, float* __restrict__ lse_out, int32_t R, int32_t V) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * (kScoreThreads / 64) + (threadIdx.x >> 6);
  if (r >= R) return;   // whole waves
  const T* x = logits + r * V;
  float mx = -INFINITY;
  for (int v = lane; v < V; v += 64) mx = fmaxf(mx, load_logit(x + v));
  mx = wave_max(mx);
  float z = 0.f;
  for (int v = lane; v < V; v += 64) z += fast_exp2((load_logit(x + v) - mx) * kLog2e);
  z = wave_sum(z);
  const float lse = mx + logf(z);
  const float p = prev[r];
  const int32_t words = (V + 31) >> 5;
  float best = -INFINITY;
  float* out = cand + r * V;
  for (int v = lane; v < V; v += 64) {
    const bool ok = mask == nullptr || ((mask[r * words + (v >> 5)] >> (v & 31)) & 1u);
    const float s = ok ? p + (load_logit(x + v) - lse) : -INFINITY;
    if constexpr (CAND) out[v] = s;
    best = fmaxf(best, s);
  }
  best = wave_max(best);
  if (row_max != nullptr && lane == 0) row_max[r] = best;
  if (!CAND && lane == 0) lse_out[r] = lse;
}

// The row sums of exp take the hardware exp2 of a log2(e)-scaled argument
// (relative error about 1e-6 per term against 2^-24 for expf), which keeps
// the pass from being bound by the vector ALU.
// Row kernel for V a multiple of 8, V <= 512*NCH: each lane owns runs of 8
// consecutive tokens (one 16-byte bf16 load or two fp32 loads per run), the
// row stays in registers across the max, sum and output passes.
template <int NCH>
constexpr int score_rows_per_wave() { return NCH == 1 ? 4 : (NCH == 2 ? 2 : 1); }

template <class T, int NCH, bool CAND = true>
__global__ void __launch_bounds__(kScoreThreads)
beam_scores_vec_kernel(const T* __restrict__ logits, const float* __restrict__ prev,
                       const uint32_t* __restrict__ mask, float* __restrict__ cand,
                       float* __restrict__ row_max, float* __restrict__ lse_out, int32_t R,
                       int32_t V) {
  // RPW rows per wave, all their loads issued before the first reduction
  constexpr int RPW = score_rows_per_wave<NCH>();
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * (kScoreThreads / 64) + (threadIdx.x >> 6)) * RPW;
  const int32_t words = (V + 31) >> 5;
  float f[RPW][NCH][8];
  uint32_t bits[RPW][NCH];
  float p[RPW];
#pragma unroll
  for (int j = 0; j < RPW; ++j) {
    const int64_t r = r0 + j;
    if (r >= R) continue;   // whole waves
    const T* x = logits + r * V;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int v0 = c * 512 + 8 * lane;
      if (v0 < V) {
        if constexpr (sizeof(T) == 2) {
          Chunk<BF16>::unpack(*(const u32x4*)(x + v0), f[j][c]);
        } else {
          Chunk<F32>::unpack(*(const u32x4*)(x + v0), f[j][c]);
          Chunk<F32>::unpack(*(const u32x4*)(x + v0 + 4), f[j][c] + 4);
        }
        bits[j][c] = mask == nullptr ? 0xffu : (mask[r * words + (v0 >> 5)] >> (v0 & 31)) & 0xffu;
      }
    }
    p[j] = prev[r];
  }
#pragma unroll
  for (int j = 0; j < RPW; ++j) {
    const int64_t r = r0 + j;
    if (r >= R) continue;
    float mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      if (c * 512 + 8 * lane < V) {
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, f[j][c][e]);
      }
    mx = wave_max(mx);
    float z = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      if (c * 512 + 8 * lane < V) {
#pragma unroll
        for (int e = 0; e < 8; ++e) z += fast_exp2((f[j][c][e] - mx) * kLog2e);
      }
    z = wave_sum(z);
    const float lse = mx + logf(z);
    float best = -INFINITY;
    float* out = cand + r * V;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int v0 = c * 512 + 8 * lane;
      if (v0 >= V) continue;
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        o[e] = ((bits[j][c] >> e) & 1u) ? p[j] + (f[j][c][e] - lse) : -INFINITY;
        best = fmaxf(best, o[e]);
      }
      // streamed past the caches: the array is larger than L2 and MALL, and
      // the top-k reads it back with streaming loads as well
      if constexpr (CAND) {
        __builtin_nontemporal_store(Chunk<F32>::pack(o), (u32x4*)(out + v0));
        __builtin_nontemporal_store(Chunk<F32>::pack(o + 4), (u32x4*)(out + v0 + 4));
      }
    }
    best = wave_max(best);
    if (row_max != nullptr && lane == 0) row_max[r] = best;
    if (!CAND && lane == 0) lse_out[r] = lse;
  }
}

// ---------------------------------------------------------------------------
// top-k
// ---------------------------------------------------------------------------
constexpr int kTopkThreads = 1024;
constexpr int kHistBins = 4096;         // fast-path window bins
constexpr float kWindow = 64.0f;        // fast-path window below the best score
constexpr int kGatherCap = 8192;        // LDS entries for the exact sort

// Order-preserving key: larger key = better candidate.  -0 maps to +0's key,
// NaN to 0 (below -inf, whose key is 0x007fffff).
__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = __float_as_uint(x);
  if (x != x) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Sort key: key in the high word, inverted index in the low word, so that a
// descending sort puts better scores first and the lower index first on ties.
__device__ __forceinline__ uint64_t composite(uint32_t key, uint32_t idx) {
  return ((uint64_t)key << 32) | (uint64_t)(~idx);
}

__device__ __forceinline__ int window_bin(float x, float lo, float inv_w) {
  if (!(x >= lo)) return 0;   // below the window, -inf and NaN
  const float t = fminf((x - lo) * inv_w, (float)(kHistBins - 1));
  return (int)t;
}

// Add 1 to hist[bin] for every lane with pred set: one LDS atomic for the
// whole wave when all those lanes agree on the bin (crowded bins), else one
// per lane.  Called by the whole wave.
__device__ __forceinline__ void hist_add(uint32_t* hist, int bin, bool pred) {
  const uint64_t active = __ballot(pred);
  if (active == 0) return;
  const int lead = (int)__builtin_ctzll(active);
  const int b0 = __shfl(bin, lead);
  if (__ballot(pred && bin == b0) == active) {
    if ((int)(threadIdx.x & 63) == lead) atomicAdd(&hist[b0], (uint32_t)__popcll(active));
  } else if (pred) {
    atomicAdd(&hist[bin], 1u);
  }
}

// Append composites of the lanes with pred set to list at *count (wave-aggregated).
__device__ __forceinline__ void wave_append(uint64_t* list, uint32_t* count, bool pred,
                                            uint64_t value, uint32_t cap) {
  const uint64_t m = __ballot(pred);
  if (m == 0) return;
  const int lane = threadIdx.x & 63;
  const int lead = (int)__builtin_ctzll(m);
  uint32_t base = 0;
  if (lane == lead) base = atomicAdd(count, (uint32_t)__popcll(m));
  base = __shfl(base, lead);
  const uint32_t pos = base + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
  if (pred && pos < cap) list[pos] = value;
}

// Bitonic sort of list[0, n) descending; n a power of two <= capacity.
__device__ void bitonic_desc(uint64_t* list, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < (n >> 1); i += kTopkThreads) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = (lo & size) == 0;
        const uint64_t a = list[lo], b = list[hi];
        if ((a < b) == desc) {
          list[lo] = b;
          list[hi] = a;
        }
      }
      __syncthreads();
    }
  }
}

// Inclusive block scan of one uint32 per thread (1024 threads); returns the
// exclusive prefix; *total receives the sum.
__device__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* scratch, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t v = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(v, o);
    if (lane >= o) v += y;
  }
  if (lane == 63) scratch[wave] = v;
  __syncthreads();
  if (wave == 0) {
    uint32_t w = lane < kTopkThreads / 64 ? scratch[lane] : 0u;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const uint32_t y = __shfl_up(w, o);
      if (lane >= o) w += y;
    }
    if (lane < kTopkThreads / 64) scratch[16 + lane] = w;
  }
  __syncthreads();
  const uint32_t before = wave == 0 ? 0u : scratch[16 + wave - 1];
  *total = scratch[16 + kTopkThreads / 64 - 1];
  __syncthreads();
  return before + v - x;
}

// ---- multi-workgroup fast path: slices of a request over several workgroups ----
constexpr int kSliceThreads = 256;
constexpr int kMaxSlices = 64;
constexpr uint32_t kSliceTarget = 32768;   // candidates per slice (about)

__host__ __device__ inline int topk_slices(uint32_t N) {
  const uint32_t s = (N + kSliceTarget - 1) / kSliceTarget;
  return (int)(s < 1 ? 1 : (s > (uint32_t)kMaxSlices ? (uint32_t)kMaxSlices : s));
}

// Workspace of one call (per request b): slice maxima [S], slice histograms
// [S][kHistBins], info [kInfo] = {b*, count above b*, gathered count, fast
// flag, done flag, unused...}, gathered list [kGatherCap] of composites.
constexpr int kInfo = 8;
struct TopkWs {
  float* smax;
  uint32_t* hist;
  int32_t* info;
  uint64_t* list;
  int S;
  __host__ __device__ TopkWs(void* ws, int B, int S_) : S(S_) {
    char* p = (char*)ws;
    list = (uint64_t*)p;
    p += (size_t)B * kGatherCap * 8;
    hist = (uint32_t*)p;
    p += (size_t)B * S_ * kHistBins * 4;
    smax = (float*)p;
    p += (size_t)B * S_ * 4;
    info = (int32_t*)p;
  }
  __host__ __device__ static size_t bytes(int B, int S_) {
    return (size_t)B * kGatherCap * 8 + (size_t)B * S_ * kHistBins * 4 + (size_t)B * S_ * 4 +
           (size_t)B * kInfo * 4;
  }
};

// Where the top-k reads candidate scores: the array the score kernel wrote,
// or each score recomputed from the logits with the same operations and the
// row's stored log-sum-exp, so that both give the same bits.
struct CandArray {
  const float* cand;
  struct Row {   // one request's candidates
    const float* p;
    __device__ __forceinline__ float operator[](uint32_t i) const { return p[i]; }
    __device__ __forceinline__ float nt(uint32_t i) const { return __builtin_nontemporal_load(&p[i]); }
  };
  __device__ __forceinline__ Row request(int64_t b, uint32_t N) const {
    return Row{cand + b * (int64_t)N};
  }
};

template <class T>
struct CandFromLogits {
  const T* logits;
  const float* prev;
  const uint32_t* mask;   // NULL: every token allowed
  const float* lse;       // per row
  int32_t M, V;
  FastDiv per_row;        // request-local candidate index -> beam
  struct Row {
    const T* logits;
    const float* prev;
    const uint32_t* mask;
    const float* lse;
    int64_t r0;
    int32_t V;
    FastDiv per_row;
    __device__ __forceinline__ float operator[](uint32_t i) const {
      const uint32_t m = per_row.div(i), v = i - m * (uint32_t)V;
      const int64_t r = r0 + m;
      const int32_t words = (V + 31) >> 5;
      const bool ok = mask == nullptr || ((mask[r * words + (v >> 5)] >> (v & 31)) & 1u);
      return ok ? prev[r] + (load_logit(logits + r * V + v) - lse[r]) : -INFINITY;
    }
    __device__ __forceinline__ float nt(uint32_t i) const { return (*this)[i]; }
    // candidates i .. i+7 (i and V multiples of 8, so one row): one 16-byte
    // run of logits, as the score kernel's 8-token runs
    __device__ __forceinline__ void load8(uint32_t i, float (&x)[8]) const {
      const uint32_t m = per_row.div(i), v = i - m * (uint32_t)V;
      const int64_t r = r0 + m;
      const T* row = logits + r * V + v;
      float f[8];
      if constexpr (sizeof(T) == 2) {
        Chunk<BF16>::unpack(*(const u32x4*)row, f);
      } else {
        Chunk<F32>::unpack(*(const u32x4*)row, f);
        Chunk<F32>::unpack(*(const u32x4*)(row + 4), f + 4);
      }
      const int32_t words = (V + 31) >> 5;
      const uint32_t bits =
          mask == nullptr ? 0xffu : (mask[r * words + (v >> 5)] >> (v & 31)) & 0xffu;
      const float p = prev[r], l = lse[r];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = ((bits >> e) & 1u) ? p + (f[e] - l) : -INFINITY;
    }
  };
  __device__ __forceinline__ Row request(int64_t b, uint32_t) const {
    return Row{logits, prev, mask, lse, b * M, V, per_row};
  }
};

// Slice s of a request's N candidates; slices start on multiples of 8.
__device__ __forceinline__ void slice_range(uint32_t N, int S, int s, uint32_t& i0, uint32_t& i1) {
  const uint32_t per = ((N + S - 1) / S + 7u) & ~7u;
  i0 = min(N, (uint32_t)s * per);
  i1 = min(N, i0 + per);
}

__device__ float block_max_256(float x, float* scratch) {
  x = wave_max(x);
  if ((threadIdx.x & 63) == 0) scratch[threadIdx.x >> 6] = x;
  __syncthreads();
  x = fmaxf(fmaxf(scratch[0], scratch[1]), fmaxf(scratch[2], scratch[3]));
  __syncthreads();
  return x;
}

template <class Src>
__global__ void __launch_bounds__(kSliceThreads)
topk_slice_max_kernel(Src src, const float* __restrict__ row_max,
                      int32_t M, int32_t V, TopkWs ws) {
  __shared__ float scratch[4];
  const int s = blockIdx.x;
  const int64_t b = blockIdx.y;
  const uint32_t N = (uint32_t)M * (uint32_t)V;
  uint32_t i0, i1;
  slice_range(N, ws.S, s, i0, i1);
  float best = -INFINITY;
  if (row_max != nullptr) {
    if (i1 > i0)
      for (uint32_t m = i0 / V + threadIdx.x; m <= (i1 - 1) / V; m += kSliceThreads)
        best = fmaxf(best, row_max[b * M + m]);
  } else {
    const auto c = src.request(b, N);
    for (uint32_t i = i0 + threadIdx.x; i < i1; i += kSliceThreads) best = fmaxf(best, c[i]);
  }
  best = block_max_256(best, scratch);
  if (threadIdx.x == 0) ws.smax[b * ws.S + s] = best;
}

// The request's best score: the maximum of its slice maxima (S <= 64, one per
// lane), in every lane of the calling wave.
__device__ __forceinline__ float request_best(const TopkWs& ws, int64_t b) {
  const int lane = threadIdx.x & 63;
  return wave_max(lane < ws.S ? ws.smax[b * ws.S + lane] : -INFINITY);
}

// VEC8: eight consecutive candidates per thread through Src::Row::load8
// (V a multiple of 8).
template <class Src, bool VEC8>
__global__ void __launch_bounds__(kSliceThreads)
topk_slice_hist_kernel(Src src, int32_t M, int32_t V, TopkWs ws) {
  __shared__ uint32_t hist[kHistBins];
  const int s = blockIdx.x;
  const int64_t b = blockIdx.y;
  if (ws.info[b * kInfo + 4] != 0) return;   // the sampled path succeeded
  const uint32_t N = (uint32_t)M * (uint32_t)V;
  for (int i = threadIdx.x; i < kHistBins; i += kSliceThreads) hist[i] = 0u;
  __syncthreads();
  const float best = request_best(ws, b);
  if (best == best && best > -INFINITY && best < INFINITY) {
    const float lo = best - kWindow, inv_w = (float)kHistBins / kWindow;
    uint32_t i0, i1;
    slice_range(N, ws.S, s, i0, i1);
    const auto c = src.request(b, N);
    if constexpr (VEC8) {
      // four runs of eight in flight per thread
      constexpr uint32_t kBatch = 8 * kSliceThreads;
      for (uint32_t j0 = i0; j0 < i1; j0 += 4 * kBatch) {
        float x[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t i = j0 + u * kBatch + 8 * threadIdx.x;
          if (i < i1) {
            c.load8(i, x[u]);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[u][e] = -INFINITY;
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int bin = window_bin(x[u][e], lo, inv_w);
            if (bin > 0) atomicAdd(&hist[bin], 1u);
          }
      }
    } else
    // four candidates in flight per thread (streaming loads); one LDS atomic
    // per counted candidate
    for (uint32_t j0 = i0; j0 < i1; j0 += 4 * kSliceThreads) {
      float x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t i = j0 + u * kSliceThreads + threadIdx.x;
        x[u] = i < i1 ? c.nt(i) : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int bin = window_bin(x[u], lo, inv_w);
        if (bin > 0) atomicAdd(&hist[bin], 1u);
      }
    }
  }
  __syncthreads();
  uint32_t* out = ws.hist + (b * ws.S + s) * (int64_t)kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += kSliceThreads) out[i] = hist[i];
}

// The sample: of every group of 16 consecutive 128-byte chunks (512
// candidates) of a request's flat candidate array, the one chunk picked by a
// multiplicative hash of the group index (so that neither a row's token order
// nor the row length biases it).  A sixteenth of the candidates.
__device__ __forceinline__ uint32_t sample_chunk(uint32_t group) {
  return 16u * group + ((group * 0x9E3779B1u) >> 28);
}

// Histogram of the sampled candidates of kSampleGroup consecutive slices, in
// the same window and bins as the full slice histograms (written to the
// buffer of slice blockIdx.x; the sum then runs over the first
// sample_slices(S) buffers).
constexpr int kSampleGroup = 8;
__host__ __device__ inline int sample_slices(int S) { return (S + kSampleGroup - 1) / kSampleGroup; }

template <class Src, bool VEC8>
__global__ void __launch_bounds__(kSliceThreads)
topk_sample_hist_kernel(Src src, int32_t M, int32_t V, TopkWs ws) {
  __shared__ uint32_t hist[kHistBins];
  const int s = blockIdx.x;
  const int64_t b = blockIdx.y;
  const uint32_t N = (uint32_t)M * (uint32_t)V;
  for (int i = threadIdx.x; i < kHistBins; i += kSliceThreads) hist[i] = 0u;
  __syncthreads();
  const float best = request_best(ws, b);
  if (best == best && best > -INFINITY && best < INFINITY) {
    const float lo = best - kWindow, inv_w = (float)kHistBins / kWindow;
    uint32_t i0, i1, j0, j1;
    slice_range(N, ws.S, s * kSampleGroup, i0, j1);
    slice_range(N, ws.S, min(s * kSampleGroup + kSampleGroup, ws.S) - 1, j0, i1);
    const auto c = src.request(b, N);
    if constexpr (VEC8) {
      // four lanes per sampled chunk (runs of eight), four groups in flight
      constexpr int kSlots = kSliceThreads / 4;
      const int q = threadIdx.x >> 2, part = threadIdx.x & 3;
      const uint32_t g0 = i0 >> 9, g1 = (i1 + 511) >> 9;
      for (uint32_t gg = g0 + q; gg < g1; gg += 4 * kSlots) {
        float x[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t g = gg + u * kSlots;
          const uint32_t i = 32u * sample_chunk(g) + 8 * part;
          if (g < g1 && i >= i0 && i < i1) {
            c.load8(i, x[u]);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[u][e] = -INFINITY;
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int bin = window_bin(x[u][e], lo, inv_w);
            if (bin > 0) atomicAdd(&hist[bin], 1u);
          }
      }
    } else {
    // one sampled chunk per 32-lane half-wave and group, eight groups in flight
    const int half = threadIdx.x >> 5, l = threadIdx.x & 31;
    constexpr int kHalves = kSliceThreads / 32;
    const uint32_t g0 = i0 >> 9, g1 = (i1 + 511) >> 9;
    for (uint32_t gg = g0 + half; gg < g1; gg += 8 * kHalves) {
      float x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const uint32_t g = gg + u * kHalves;
        const uint32_t i = 32u * sample_chunk(g) + l;
        x[u] = g < g1 && i >= i0 && i < i1 ? c.nt(i) : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int bin = window_bin(x[u], lo, inv_w);
        if (bin > 0) atomicAdd(&hist[bin], 1u);
      }
    }
    }
  }
  __syncthreads();
  uint32_t* out = ws.hist + (b * ws.S + s) * (int64_t)kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += kSliceThreads) out[i] = hist[i];
}

// Sum of the first n_slices slice histograms of a request, bins [256 p,
// 256 p + 256) per workgroup, written over slice 0's histogram (each bin is
// read and written by one thread only).
constexpr int kReduceBins = 256;
__global__ void __launch_bounds__(kReduceBins)
topk_hist_reduce_kernel(TopkWs ws, int32_t n_slices, int32_t skip_if_done) {
  const int64_t b = blockIdx.y;
  if (skip_if_done && ws.info[b * kInfo + 4] != 0) return;
  const int bin = blockIdx.x * kReduceBins + threadIdx.x;
  uint32_t* h = ws.hist + b * ws.S * (int64_t)kHistBins + bin;
  // eight slices in flight per thread
  uint32_t part[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
  int j = 0;
  for (; j + 8 <= n_slices; j += 8)
#pragma unroll
    for (int u = 0; u < 8; ++u) part[u] += h[(int64_t)(j + u) * kHistBins];
  for (; j < n_slices; ++j) part[0] += h[(int64_t)j * kHistBins];
  h[0] = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
}

// SAMPLED: the histogram holds a sixteenth of the candidates.  The chosen bin
// is the highest whose sample count from the top reaches 1.25 k / 16, so that
// about 1.25 k candidates are expected at or above it; no fit check here, as
// the gather counts them exactly and topk_verify_kernel decides.
template <bool SAMPLED>
__global__ void __launch_bounds__(kTopkThreads)
topk_boundary_kernel(int32_t k_req, TopkWs ws) {
  __shared__ uint32_t scan[64];
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x;
  if (!SAMPLED && ws.info[b * kInfo + 4] != 0) return;   // the sampled path succeeded
  const int32_t k = SAMPLED ? (5 * k_req + 63) / 64 : k_req;
  __shared__ int32_t par[2];
  if (tid < 2) par[tid] = 0;
  // thread 0 owns the top 4 bins, in descending order
  const int t_rev = kTopkThreads - 1 - tid;
  uint32_t own[4] = {0u, 0u, 0u, 0u}, s4 = 0;
  const uint32_t* h = ws.hist + b * ws.S * (int64_t)kHistBins;   // the request's total
#pragma unroll
  for (int e = 0; e < 4; ++e) own[e] = h[4 * t_rev + 3 - e];
#pragma unroll
  for (int e = 0; e < 4; ++e) s4 += own[e];
  __syncthreads();
  uint32_t total;
  const uint32_t before = block_exclusive_scan(s4, scan, &total);
  if (before < (uint32_t)k && before + s4 >= (uint32_t)k) {
    uint32_t run = before;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (run < (uint32_t)k && run + own[e] >= (uint32_t)k) {
        par[0] = 4 * t_rev + 3 - e;
        par[1] = (int32_t)run;
        // fast only if everything in bins >= b* fits the gather list
        par[0] = (par[0] > 0 && (SAMPLED || run + own[e] <= (uint32_t)kGatherCap)) ? par[0] : 0;
      }
      run += own[e];
    }
  }
  __syncthreads();
  const float best = request_best(ws, b);   // whole waves
  if (tid == 0) {
    const bool finite = best == best && best > -INFINITY && best < INFINITY;
    const bool fast = finite && total >= (uint32_t)k && par[0] > 0;
    ws.info[b * kInfo + 0] = par[0];
    ws.info[b * kInfo + 1] = par[1];
    ws.info[b * kInfo + 2] = 0;          // gather counter
    ws.info[b * kInfo + 3] = fast ? 1 : 0;
    if (SAMPLED) ws.info[b * kInfo + 4] = 0;   // done flag of this call
  }
}

// After the gather at the sampled bin: the gathered set holds the k best
// exactly when at least k candidates lie at or above that bin; it is usable
// when it also fits the list.  Otherwise the full histogram path runs.
__global__ void __launch_bounds__(64)
topk_verify_kernel(int32_t B, int32_t k, TopkWs ws) {
  const int64_t b = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (b >= B) return;
  int32_t* info = ws.info + b * kInfo;
  const uint32_t n = (uint32_t)info[2];
  const bool ok = info[3] != 0 && n >= (uint32_t)k && n <= (uint32_t)kGatherCap;
  info[4] = ok ? 1 : 0;
}

// Gathered candidates are staged in LDS and flushed to the request's list
// with one global atomic per flush (same-address global atomics serialise).
constexpr int kStage = 2048;

template <class Src, bool VEC8>
__global__ void __launch_bounds__(kSliceThreads)
topk_gather_kernel(Src src, int32_t M, int32_t V, TopkWs ws) {
  constexpr int kCap = VEC8 ? 2 * kStage : kStage;
  __shared__ uint64_t stage[kCap];
  __shared__ uint32_t n_stage, base;
  const int s = blockIdx.x;
  const int64_t b = blockIdx.y;
  // whole workgroup: no fast path, or the sampled path already succeeded
  if (ws.info[b * kInfo + 3] == 0 || ws.info[b * kInfo + 4] != 0) return;
  const int bstar = ws.info[b * kInfo + 0];
  const uint32_t N = (uint32_t)M * (uint32_t)V;
  const float best = request_best(ws, b);
  const float lo = best - kWindow, inv_w = (float)kHistBins / kWindow;
  // every candidate in bin b* or above lies at or above the lower edge of bin
  // b* - 1 (a whole bin of slack against rounding): waves with no candidate
  // there skip the bin computation
  const float thr = lo + (float)(bstar - 1) * (kWindow / (float)kHistBins);
  uint32_t i0, i1;
  slice_range(N, ws.S, s, i0, i1);
  const auto c = src.request(b, N);
  uint32_t* count = (uint32_t*)&ws.info[b * kInfo + 2];
  uint64_t* list = ws.list + b * (int64_t)kGatherCap;
  if (threadIdx.x == 0) n_stage = 0;
  __syncthreads();
  auto flush = [&]() {
    __syncthreads();
    const uint32_t n = n_stage;
    if (n > 0) {
      if (threadIdx.x == 0) base = atomicAdd(count, n);
      __syncthreads();
      const uint32_t b0 = base;
      for (uint32_t j = threadIdx.x; j < n; j += kSliceThreads)
        if (b0 + j < (uint32_t)kGatherCap) list[b0 + j] = stage[j];
      __syncthreads();
      if (threadIdx.x == 0) n_stage = 0;
    }
    __syncthreads();
  };
  if constexpr (VEC8) {
    // runs of eight per thread, four batches in flight: each batch is staged
    // (at most kBatch entries, flushed before the stage can overflow) and the
    // batch four ahead is loaded in its registers
    constexpr uint32_t kBatch = 8 * kSliceThreads;
    float x[4][8];
    auto load_batch = [&](uint32_t j, float (&y)[8]) __attribute__((always_inline)) {
      const uint32_t i = j + 8 * threadIdx.x;
      if (i < i1) {
        c.load8(i, y);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = -INFINITY;
      }
    };
#pragma unroll
    for (int u = 0; u < 4; ++u) load_batch(i0 + u * kBatch, x[u]);
    for (uint32_t j0 = i0; j0 < i1; j0 += 4 * kBatch) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t i = j0 + u * kBatch + 8 * threadIdx.x;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (__ballot(x[u][e] >= thr) == 0) continue;   // whole wave
          const int bin = window_bin(x[u][e], lo, inv_w);
          wave_append(stage, &n_stage, i < i1 && bin >= bstar,
                      composite(order_key(x[u][e]), i + e), kCap);
        }
        __syncthreads();
        if (n_stage > (uint32_t)(kCap - kBatch)) flush();
        load_batch(j0 + (u + 4) * kBatch, x[u]);
      }
    }
  } else {
    for (uint32_t j0 = i0; j0 < i1; j0 += 4 * kSliceThreads) {
      float x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t i = j0 + u * kSliceThreads + threadIdx.x;
        x[u] = i < i1 ? c.nt(i) : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (__ballot(x[u] >= thr) == 0) continue;   // whole wave
        const uint32_t i = j0 + u * kSliceThreads + threadIdx.x;
        const int bin = window_bin(x[u], lo, inv_w);
        wave_append(stage, &n_stage, i < i1 && bin >= bstar, composite(order_key(x[u]), i), kCap);
      }
      // at most 4 * kSliceThreads more per iteration: flush before the stage can overflow
      __syncthreads();
      if (n_stage > (uint32_t)(kCap - 4 * kSliceThreads)) flush();
    }
  }
  flush();
}

struct TopkShared {
  uint32_t hist[256];
  uint64_t list[kGatherCap];
  uint32_t scan[64];
  int32_t ipar[4];
  // fast path: members per window bin (counted from the top bin down), then
  // the first position of each bin in the bin-ordered list
  uint32_t bin_count[kHistBins];
  uint32_t bin_start[kHistBins];
  uint32_t max_count;
};

// Bins at most this full are ranked by comparing a candidate with the other
// members of its bin; fuller bins take the bitonic sort.
constexpr uint32_t kRankBinCap = 512;

// The score a fast-path key came from (finite scores only; -0 is read back
// from the candidates because its key is +0's).
__device__ __forceinline__ float key_score(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
}

// Final selection: sort the gathered candidates (fast path), or an exact radix
// select over all the request's candidates (fallback), then emit k in order.
template <class Src>
__global__ void __launch_bounds__(kTopkThreads)
topk_final_kernel(Src src, int32_t M, int32_t V, int32_t k,
                  TopkWs ws, int32_t* __restrict__ parents, int32_t* __restrict__ tokens,
                  float* __restrict__ scores) {
  __shared__ TopkShared sh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t b = blockIdx.x;
  const uint32_t N = (uint32_t)M * (uint32_t)V;
  const auto c = src.request(b, N);
  if (tid < 4) sh.ipar[tid] = 0;

  uint32_t n_sel;
  if (ws.info[b * kInfo + 3] != 0) {
    n_sel = (uint32_t)ws.info[b * kInfo + 2];
    const uint64_t* list = ws.list + b * (int64_t)kGatherCap;
    // ---- rank by window bin: a counting sort over the bins, then each
    // candidate's place inside its bin from the bin's other members ----
    constexpr int kPer = kGatherCap / kTopkThreads;
    for (int i = tid; i < kHistBins; i += kTopkThreads) sh.bin_count[i] = 0u;
    if (tid == 0) sh.max_count = 0u;
    __syncthreads();
    const float best = request_best(ws, b);
    const float lo = best - kWindow, inv_w = (float)kHistBins / kWindow;
    uint64_t v[kPer];
    uint32_t rb[kPer], slot[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint32_t i = (uint32_t)(tid + j * kTopkThreads);
      if (i < n_sel) {
        v[j] = list[i];
        // the bin the gather saw: the key is the candidate's score, exactly
        rb[j] = (uint32_t)(kHistBins - 1 - window_bin(key_score((uint32_t)(v[j] >> 32)), lo, inv_w));
        slot[j] = atomicAdd(&sh.bin_count[rb[j]], 1u);
      }
    }
    __syncthreads();
    {
      uint32_t c4[4], s4 = 0, mx = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        c4[e] = sh.bin_count[4 * tid + e];
        s4 += c4[e];
        mx = max(mx, c4[e]);
      }
      if (mx > 0) atomicMax(&sh.max_count, mx);
      uint32_t total;
      uint32_t run = block_exclusive_scan(s4, sh.scan, &total);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sh.bin_start[4 * tid + e] = run;
        run += c4[e];
      }
    }
    __syncthreads();
    if (sh.max_count <= kRankBinCap) {
      // members of a bin that starts at or past k are not among the k best
#pragma unroll
      for (int j = 0; j < kPer; ++j)
        if ((uint32_t)(tid + j * kTopkThreads) < n_sel && sh.bin_start[rb[j]] < (uint32_t)k)
          sh.list[sh.bin_start[rb[j]] + slot[j]] = v[j];
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kPer; ++j) {
        if ((uint32_t)(tid + j * kTopkThreads) >= n_sel) continue;
        const uint32_t s0 = sh.bin_start[rb[j]], n = sh.bin_count[rb[j]];
        if (s0 >= (uint32_t)k) continue;
        uint32_t pos = s0;
        for (uint32_t e = 0; e < n; ++e) pos += sh.list[s0 + e] > v[j] ? 1u : 0u;
        if (pos < (uint32_t)k) {
          const uint32_t key = (uint32_t)(v[j] >> 32), idx = ~(uint32_t)(v[j] & 0xffffffffull);
          parents[b * k + pos] = (int32_t)(idx / (uint32_t)V);
          tokens[b * k + pos] = (int32_t)(idx % (uint32_t)V);
          scores[b * k + pos] = key == 0x80000000u ? c[idx] : key_score(key);
        }
      }
      return;
    }
    // a crowded bin: the bitonic sort below
    for (uint32_t i = tid; i < n_sel; i += kTopkThreads) sh.list[i] = list[i];
    __syncthreads();
  } else {
    // ---- exact radix select on the key, four 8-bit digits ----
    uint32_t prefix = 0, remaining = (uint32_t)k;
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      const uint32_t pmask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
      for (int i = tid; i < 256; i += kTopkThreads) sh.hist[i] = 0u;
      __syncthreads();
      for (uint32_t i0 = 0; i0 < N; i0 += kTopkThreads) {
        const uint32_t i = i0 + tid;
        const bool live = i < N;
        const uint32_t key = live ? order_key(c[i]) : 0u;
        hist_add(sh.hist, (int)((key >> shift) & 255u), live && (key & pmask) == prefix);
      }
      __syncthreads();
      if (wave == 0) {
        // digits from 255 down: 4 per lane, lane 0 owns 255..252
        uint32_t own[4], s4 = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          own[j] = sh.hist[255 - 4 * lane - j];
          s4 += own[j];
        }
        uint32_t inc = s4;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_up(inc, o);
          if (lane >= o) inc += y;
        }
        const uint32_t before = inc - s4;
        if (before < remaining && inc >= remaining) {
          uint32_t run = before;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (run < remaining && run + own[j] >= remaining) {
              sh.ipar[0] = 255 - 4 * lane - j;
              sh.ipar[1] = (int32_t)run;
            }
            run += own[j];
          }
        }
      }
      __syncthreads();
      prefix |= (uint32_t)sh.ipar[0] << shift;
      remaining -= (uint32_t)sh.ipar[1];
      __syncthreads();
    }
    // prefix is the k-th key T; `remaining` candidates equal to T are taken,
    // lowest index first, after the k - remaining candidates above T.
    const uint32_t T = prefix, need = remaining, gt_total = (uint32_t)k - remaining;
    uint32_t gt_base = 0, eq_base = 0;
    for (uint32_t i0 = 0; i0 < N && (gt_base < gt_total || eq_base < need);
         i0 += 4 * kTopkThreads) {
      uint32_t keys[4], ngt = 0, neq = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t i = i0 + 4 * tid + j;
        const bool in = i < N;
        keys[j] = in ? order_key(c[i]) : 0u;
        ngt += in && keys[j] > T;
        neq += in && keys[j] == T;
      }
      uint32_t total;
      const uint32_t pre = block_exclusive_scan((neq << 16) | ngt, sh.scan, &total);
      uint32_t pg = gt_base + (pre & 0xffffu), pe = eq_base + (pre >> 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t i = i0 + 4 * tid + j;
        if (i >= N) continue;
        if (keys[j] > T) {
          sh.list[pg++] = composite(keys[j], i);
        } else if (keys[j] == T) {
          if (pe < need) sh.list[gt_total + pe] = composite(keys[j], i);
          ++pe;
        }
      }
      gt_base += total & 0xffffu;
      eq_base += total >> 16;
    }
    __syncthreads();
    n_sel = (uint32_t)k;
  }

  // ---- sort the selected candidates, best first; emit the first k ----
  uint32_t n2 = 1;
  while (n2 < n_sel) n2 <<= 1;
  for (uint32_t i = n_sel + tid; i < n2; i += kTopkThreads) sh.list[i] = 0ull;
  __syncthreads();
  bitonic_desc(sh.list, (int)n2);
  for (int j = tid; j < k; j += kTopkThreads) {
    const uint32_t idx = ~(uint32_t)(sh.list[j] & 0xffffffffull);
    parents[b * k + j] = (int32_t)(idx / (uint32_t)V);
    tokens[b * k + j] = (int32_t)(idx % (uint32_t)V);
    scores[b * k + j] = c[idx];
  }
}

// The score kernels; with CAND = false they write lse_out instead of cand.
// Both modes pick the same kernel for a given V, so the log-sum-exp (and so
// every recomputed candidate) matches the written candidates bit for bit.
template <bool CAND>
static void launch_scores_mode(const void* logits, const float* prev, const uint32_t* mask,
                               float* cand, float* row_max, float* lse_out, int32_t R, int32_t V,
                               bool bf16, hipStream_t stream) {
  const int64_t blocks = ((int64_t)R + kScoreThreads / 64 - 1) / (kScoreThreads / 64);
  const dim3 grid((unsigned)blocks), block(kScoreThreads);
  constexpr int64_t kWaves = kScoreThreads / 64;
#define GRACE_SC(TT, NCH)                                                                       \
  hipLaunchKernelGGL((beam_scores_vec_kernel<TT, NCH, CAND>),                                   \
                     dim3((unsigned)(((int64_t)R + kWaves * score_rows_per_wave<NCH>() - 1) /    \
                                     (kWaves * score_rows_per_wave<NCH>()))),                    \
                     block, 0, stream, (const TT*)logits, prev, mask, cand, row_max, lse_out, R, V)
  // 16-byte runs need V a multiple of 8 and 16-byte aligned logits
  if (V % 8 == 0 && V <= 4096 && ((uintptr_t)logits & 15) == 0) {
    const int nch = (V + 511) / 512;
    if (bf16) {
      if (nch == 1) GRACE_SC(uint16_t, 1);
      else if (nch == 2) GRACE_SC(uint16_t, 2);
      else if (nch <= 4) GRACE_SC(uint16_t, 4);
      else GRACE_SC(uint16_t, 8);
    } else {
      if (nch == 1) GRACE_SC(float, 1);
      else if (nch == 2) GRACE_SC(float, 2);
      else if (nch <= 4) GRACE_SC(float, 4);
      else GRACE_SC(float, 8);
    }
  } else if (bf16) {
    hipLaunchKernelGGL((beam_scores_kernel<uint16_t, CAND>), grid, block, 0, stream,
                       (const uint16_t*)logits, prev, mask, cand, row_max, lse_out, R, V);
  } else {
    hipLaunchKernelGGL((beam_scores_kernel<float, CAND>), grid, block, 0, stream,
                       (const float*)logits, prev, mask, cand, row_max, lse_out, R, V);
  }
#undef GRACE_SC
}

hipError_t launch_beam_scores(const void* logits, const float* prev, const uint32_t* mask,
                              float* cand, float* row_max, int32_t R, int32_t V, bool bf16,
                              hipStream_t stream) {
  launch_scores_mode<true>(logits, prev, mask, cand, row_max, nullptr, R, V, bf16, stream);
  return hipGetLastError();
}

size_t beam_topk_workspace_bytes(int32_t B, int32_t M, int32_t V) {
  return TopkWs::bytes(B, topk_slices((uint32_t)M * (uint32_t)V));
}

template <class Src, bool VEC8>
static hipError_t launch_topk_src(Src src, const float* row_max, int32_t B, int32_t M, int32_t V,
                                  int32_t k, void* workspace, int32_t* parents, int32_t* tokens,
                                  float* scores, hipStream_t stream) {
  const int S = topk_slices((uint32_t)M * (uint32_t)V);
  const TopkWs ws(workspace, B, S);
  const dim3 slices((unsigned)S, (unsigned)B);
  hipLaunchKernelGGL(topk_slice_max_kernel<Src>, slices, dim3(kSliceThreads), 0, stream, src, row_max,
                     M, V, ws);
  // sampled path: a histogram of a sixteenth of the candidates picks a bin,
  // one full pass gathers everything at or above it, and the count decides
  hipLaunchKernelGGL((topk_sample_hist_kernel<Src, VEC8>), dim3((unsigned)sample_slices(S), (unsigned)B),
                     dim3(kSliceThreads), 0, stream, src, M, V, ws);
  hipLaunchKernelGGL(topk_hist_reduce_kernel, dim3(kHistBins / kReduceBins, (unsigned)B),
                     dim3(kReduceBins), 0, stream, ws, sample_slices(S), 0);
  hipLaunchKernelGGL(topk_boundary_kernel<true>, dim3((unsigned)B), dim3(kTopkThreads), 0, stream,
                     k, ws);
  hipLaunchKernelGGL((topk_gather_kernel<Src, VEC8>), slices, dim3(kSliceThreads), 0, stream, src,
                     M, V, ws);
  hipLaunchKernelGGL(topk_verify_kernel, dim3((unsigned)((B + 63) / 64)), dim3(64), 0, stream, B, k,
                     ws);
  // full path, for the requests whose sampled bin did not hold the k best
  hipLaunchKernelGGL((topk_slice_hist_kernel<Src, VEC8>), slices, dim3(kSliceThreads), 0, stream,
                     src, M, V, ws);
  hipLaunchKernelGGL(topk_hist_reduce_kernel, dim3(kHistBins / kReduceBins, (unsigned)B),
                     dim3(kReduceBins), 0, stream, ws, S, 1);
  hipLaunchKernelGGL(topk_boundary_kernel<false>, dim3((unsigned)B), dim3(kTopkThreads), 0, stream,
                     k, ws);
  hipLaunchKernelGGL((topk_gather_kernel<Src, VEC8>), slices, dim3(kSliceThreads), 0, stream, src,
                     M, V, ws);
  hipLaunchKernelGGL(topk_final_kernel<Src>, dim3((unsigned)B), dim3(kTopkThreads), 0, stream, src, M,
                     V, k, ws, parents, tokens, scores);
  return hipGetLastError();
}

hipError_t launch_beam_topk(const float* cand, const float* row_max, int32_t B, int32_t M,
                            int32_t V, int32_t k, void* workspace, int32_t* parents,
                            int32_t* tokens, float* scores, hipStream_t stream) {
  return launch_topk_src<CandArray, false>(CandArray{cand}, row_max, B, M, V, k, workspace, parents,
                                           tokens, scores, stream);
}

size_t beam_step_workspace_bytes(int32_t B, int32_t M, int32_t V) {
  return beam_topk_workspace_bytes(B, M, V) + (size_t)B * M * 8;
}

hipError_t launch_beam_step(const void* logits, const float* prev, const uint32_t* mask,
                            int32_t B, int32_t M, int32_t V, int32_t k, bool bf16, void* workspace,
                            int32_t* parents, int32_t* tokens, float* scores,
                            hipStream_t stream) {
  const int32_t R = B * M;
  // the top-k workspace, then the rows' log-sum-exp and best scores
  float* lse = (float*)((char*)workspace + beam_topk_workspace_bytes(B, M, V));
  float* row_max = lse + R;
  launch_scores_mode<false>(logits, prev, mask, nullptr, row_max, lse, R, V, bf16, stream);
  const FastDiv per_row((uint32_t)V);
#define GRACE_STEP(TT, VEC)                                                                      \
  return launch_topk_src<CandFromLogits<TT>, VEC>(                                               \
      CandFromLogits<TT>{(const TT*)logits, prev, mask, lse, M, V, per_row}, row_max, B, M, V, k, \
      workspace, parents, tokens, scores, stream)
  // runs of eight: V a multiple of 8 and 16-byte aligned logits
  const bool vec = V % 8 == 0 && ((uintptr_t)logits & 15) == 0;
  if (bf16) {
    if (vec) GRACE_STEP(uint16_t, true);
    GRACE_STEP(uint16_t, false);
  }
  if (vec) GRACE_STEP(float, true);
  GRACE_STEP(float, false);
#undef GRACE_STEP
}

int32_t beam_topk_max_k() { return kGatherCap / 2; }

}  // namespace grace
