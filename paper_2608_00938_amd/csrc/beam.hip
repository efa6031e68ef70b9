// Beam score update and per-request top-k (GRACE, Sec. 3.1, Sec. 3.3) for gfx950.
//
// scores: one wave per beam row.  The row's log-softmax over the vocabulary is
//   added to the beam's accumulated score; filtered tokens score -inf.  The
//   kernel also writes each row's best candidate score.
// top-k:  one 1024-thread workgroup per request over its M*V candidates.
//   Candidates are totally ordered by an order-preserving 32-bit key of the
//   score (descending; -0 == +0; NaN below -inf), then by flat index m*V + v
//   (ascending), so the selection is unique.  Fast path: a 4096-bin histogram
//   of the scores in the 64-unit window below the request's best score finds
//   the bin holding the k-th candidate; only candidates in that bin and above
//   are gathered into LDS and sorted exactly.  When the k-th candidate lies
//   outside the window or the gathered set would not fit, an exact radix
//   select on the key (four 8-bit digits) and an index-ordered collection of
//   the tied candidates take over.  Either way the k winners are sorted by
//   (key desc, index asc) with a bitonic sort in LDS.
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

template <class T>
__global__ void __launch_bounds__(kScoreThreads)
beam_scores_kernel(const T* __restrict__ logits, const float* __restrict__ prev,
                   const uint32_t* __restrict__ mask, float* __restrict__ cand,
                   float* __restrict__ row_max, int32_t R, int32_t V) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * (kScoreThreads / 64) + (threadIdx.x >> 6);
  if (r >= R) return;   // whole waves
  const T* x = logits + r * V;
  float mx = -INFINITY;
  for (int v = lane; v < V; v += 64) mx = fmaxf(mx, load_logit(x + v));
  mx = wave_max(mx);
  float z = 0.f;
  for (int v = lane; v < V; v += 64) z += expf(load_logit(x + v) - mx);
  z = wave_sum(z);
  const float lse = mx + logf(z);
  const float p = prev[r];
  const int32_t words = (V + 31) >> 5;
  float best = -INFINITY;
  float* out = cand + r * V;
  for (int v = lane; v < V; v += 64) {
    const bool ok = mask == nullptr || ((mask[r * words + (v >> 5)] >> (v & 31)) & 1u);
    const float s = ok ? p + (load_logit(x + v) - lse) : -INFINITY;
    out[v] = s;
    best = fmaxf(best, s);
  }
  best = wave_max(best);
  if (row_max != nullptr && lane == 0) row_max[r] = best;
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

struct TopkShared {
  uint32_t hist[kHistBins];
  uint64_t list[kGatherCap];
  uint32_t scan[64];
  uint32_t count[4];
  float fscratch[kTopkThreads / 64];
  int32_t ipar[4];
};

__global__ void __launch_bounds__(kTopkThreads)
beam_topk_kernel(const float* __restrict__ cand, const float* __restrict__ row_max, int32_t M,
                 int32_t V, int32_t k, int32_t* __restrict__ parents,
                 int32_t* __restrict__ tokens, float* __restrict__ scores) {
  __shared__ TopkShared sh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t b = blockIdx.x;
  const uint32_t N = (uint32_t)M * (uint32_t)V;
  const float* c = cand + b * (int64_t)N;

  // ---- best score of the request ----
  float best = -INFINITY;
  if (row_max != nullptr) {
    for (int32_t m = tid; m < M; m += kTopkThreads) best = fmaxf(best, row_max[b * M + m]);
  } else {
    for (uint32_t i = tid; i < N; i += kTopkThreads) best = fmaxf(best, c[i]);
  }
  best = wave_max(best);
  if (lane == 0) sh.fscratch[wave] = best;
  for (int i = tid; i < kHistBins; i += kTopkThreads) sh.hist[i] = 0u;
  if (tid < 4) {
    sh.count[tid] = 0u;
    sh.ipar[tid] = 0;
  }
  __syncthreads();
  best = -INFINITY;
#pragma unroll
  for (int w = 0; w < kTopkThreads / 64; ++w) best = fmaxf(best, sh.fscratch[w]);

  bool fast = best == best && best > -INFINITY && best < INFINITY;
  const float lo = best - kWindow;
  const float inv_w = (float)kHistBins / kWindow;

  // ---- fast path: window histogram (bin 0 is the catch-all, not counted) ----
  uint32_t c_gt = 0, bstar = 0;
  if (fast) {
    for (uint32_t i0 = 0; i0 < N; i0 += kTopkThreads) {
      const uint32_t i = i0 + tid;
      const bool live = i < N;
      const int bin = live ? window_bin(c[i], lo, inv_w) : 0;
      hist_add(sh.hist, bin, live && bin > 0);
    }
    __syncthreads();
    // suffix counts from the top bin: thread t owns bins [4t, 4t+4)
    const int t_rev = kTopkThreads - 1 - tid;   // thread 0 owns the top 4 bins
    uint32_t own[4], s4 = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      own[j] = sh.hist[4 * t_rev + 3 - j];   // descending bin order
      s4 += own[j];
    }
    uint32_t total;
    const uint32_t before = block_exclusive_scan(s4, sh.scan, &total);
    // find the bin where the running count from the top reaches k
    if (before < (uint32_t)k && before + s4 >= (uint32_t)k) {
      uint32_t run = before;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (run < (uint32_t)k && run + own[j] >= (uint32_t)k) {
          sh.ipar[0] = 4 * t_rev + 3 - j;
          sh.ipar[1] = (int32_t)run;
        }
        run += own[j];
      }
    }
    if (tid == 0 && total < (uint32_t)k) sh.ipar[0] = 0;   // k-th lies in the catch-all
    __syncthreads();
    bstar = (uint32_t)sh.ipar[0];
    c_gt = (uint32_t)sh.ipar[1];
    fast = bstar > 0 && c_gt + sh.hist[bstar] <= (uint32_t)kGatherCap;
  }

  uint32_t n_sel;
  if (fast) {
    // ---- gather every candidate in bin >= b* and sort exactly ----
    for (uint32_t i0 = 0; i0 < N; i0 += kTopkThreads) {
      const uint32_t i = i0 + tid;
      const bool live = i < N;
      const float x = live ? c[i] : -INFINITY;
      const int bin = live ? window_bin(x, lo, inv_w) : 0;
      wave_append(sh.list, &sh.count[0], live && bin >= (int)bstar, composite(order_key(x), i),
                  kGatherCap);
    }
    __syncthreads();
    n_sel = sh.count[0];
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
        // digits from 255 down: 4 per lane, lane 0 owns 252..255
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
        keys[j] = i < N ? order_key(c[i]) : 0u;
        const bool in = i < N;
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
        if (keys[j] > T) sh.list[pg++] = composite(keys[j], i);
        else if (keys[j] == T) {
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

  // ---- sort the gathered candidates, best first; emit the first k ----
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

hipError_t launch_beam_scores(const void* logits, const float* prev, const uint32_t* mask,
                              float* cand, float* row_max, int32_t R, int32_t V, bool bf16,
                              hipStream_t stream) {
  const int64_t blocks = ((int64_t)R + kScoreThreads / 64 - 1) / (kScoreThreads / 64);
  if (bf16)
    hipLaunchKernelGGL(beam_scores_kernel<uint16_t>, dim3((unsigned)blocks), dim3(kScoreThreads),
                       0, stream, (const uint16_t*)logits, prev, mask, cand, row_max, R, V);
  else
    hipLaunchKernelGGL(beam_scores_kernel<float>, dim3((unsigned)blocks), dim3(kScoreThreads), 0,
                       stream, (const float*)logits, prev, mask, cand, row_max, R, V);
  return hipGetLastError();
}

hipError_t launch_beam_topk(const float* cand, const float* row_max, int32_t B, int32_t M,
                            int32_t V, int32_t k, int32_t* parents, int32_t* tokens,
                            float* scores, hipStream_t stream) {
  hipLaunchKernelGGL(beam_topk_kernel, dim3((unsigned)B), dim3(kTopkThreads), 0, stream, cand,
                     row_max, M, V, k, parents, tokens, scores);
  return hipGetLastError();
}

int32_t beam_topk_max_k() { return kGatherCap / 2; }

}  // namespace grace
