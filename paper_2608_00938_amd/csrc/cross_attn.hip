// Beam-as-query cross-attention for gfx950 (GRACE, Sec. 5.1, App. B).
//
// The M beams of request b are the query rows of one contraction against that
// request's encoder K/V: O = softmax(scale * Q_b K_b^T) V_b per head.  A
// workgroup owns one (request, head, beam tile); K/V stream through LDS in
// token tiles that every beam of the tile reuses, so each encoder token is
// read from L2 once per beam tile, not once per beam.
//
// bf16 path (MFMA, cross_attn_bf16_kernel).  Each wave owns 64 beams (32 at
// head dim 128) and computes, per 32-key step,
//   S^T = K Q^T           v_mfma_f32_32x32x16_bf16; A = K rows from LDS, B = Q^T
//                         (the input bf16 values) held in registers;
//   P = exp2(c S^T)       VALU, c = scale*log2(e) applied to the fp32 scores,
//                         packed to bf16 in place;
//   O^T += V^T P^T        A = V^T read with ds_read_b64_tr_b16, B = P^T taken
//                         straight from the S^T registers;
//   l += 1^T P^T          the row sums of the applied bf16 weights, on the
//                         matrix core as well.
// The transposed orientation puts one beam per lane column in every product,
// so the probabilities never leave registers.  Q enters and O leaves through
// LDS as whole beam rows (direct-to-LDS loads, 16-byte row-major stores), so
// every global access instruction covers full rows instead of 16-byte pieces
// of 32 rows.
//
// fp32 path (VALU, cross_attn_f32_kernel).  d/32 lanes per beam, K/V tiles in
// LDS read as broadcasts, fp32 FMAs throughout.
#include <type_traits>

#include "common.hpp"
#include "debug.hpp"
#include "kernels.hpp"

namespace grace {

GRACE_DEBUG_COUNTERS;

__device__ __forceinline__ void request_span(const int32_t* off, int32_t b, int32_t sum_L,
                                             int32_t& o0, int32_t& L) {
  int32_t a = off[b], e = off[b + 1];
  if (threadIdx.x == 0) GRACE_DCHECK(0 <= a && a <= e && e <= sum_L, kDbgOffsets);
  a = a < 0 ? 0 : (a > sum_L ? sum_L : a);
  e = e < a ? a : (e > sum_L ? sum_L : e);
  o0 = a;
  L = e - a;
}

// ---------------------------------------------------------------------------
// fp32 VALU kernel.  G = d/32 consecutive lanes share a beam, each holding 32
// dims of its query and output accumulator (at most 64 live values per lane
// at any d); partial dot products meet in a DPP group sum.  K/V tiles sit in
// LDS and are read as broadcasts across the beams of the workgroup.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(64)
cross_attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                      const float* __restrict__ v, const int32_t* __restrict__ off,
                      float* __restrict__ out, int32_t M, int32_t H, int32_t sum_L,
                      int32_t n_mt, float c) {
  constexpr int TILE = 32;
  constexpr int G = D / 32;          // lanes per beam
  constexpr int kBeams = 64 / G;     // beams per workgroup
  __shared__ float ks[TILE][D];
  __shared__ float vs[TILE][D];
  const uint32_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int32_t mt = tile % n_mt;
  const int32_t bh = tile / n_mt;
  const int32_t h = bh % H, b = bh / H;
  const int part = threadIdx.x % G;  // dims part*32 .. part*32+31
  const int32_t m = mt * kBeams + threadIdx.x / G;
  int32_t o0, L;
  request_span(off, b, sum_L, o0, L);
  const int64_t E = (int64_t)H * D;
  const int64_t row = (int64_t)b * M + m;
  const int64_t col = (int64_t)h * D + part * 32;

  float qr[32], acc[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    qr[e] = m < M ? q[row * E + col + e] : 0.f;
    acc[e] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  for (int32_t t0 = 0; t0 < L; t0 += TILE) {
    const int32_t n = min(TILE, L - t0);
    __syncthreads();
    for (int i = threadIdx.x; i < TILE * D; i += 64) {
      const int key = i / D, cc = i % D;
      const int64_t src = (int64_t)(o0 + t0 + (key < n ? key : n - 1)) * E + h * D + cc;
      GRACE_DCHECK(o0 + t0 + (key < n ? key : n - 1) < sum_L, kDbgRow);
      ks[key][cc] = k[src];
      vs[key][cc] = v[src];
    }
    __syncthreads();
    float s[TILE];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < TILE; ++j) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < 32; ++e) a = __builtin_fmaf(qr[e], ks[j][part * 32 + e], a);
      a = group_sum<G>(a);
      s[j] = j < n ? a : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2((m_run - m_new) * c);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int e = 0; e < 32; ++e) acc[e] *= alpha;
#pragma unroll
    for (int j = 0; j < TILE; ++j) {
      const float p = fast_exp2((s[j] - m_new) * c);
      l_run += p;
#pragma unroll
      for (int e = 0; e < 32; ++e) acc[e] = __builtin_fmaf(p, vs[j][part * 32 + e], acc[e]);
    }
  }
  if (m < M) {
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
#pragma unroll
    for (int e = 0; e < 32; ++e) out[row * E + col + e] = acc[e] * inv;
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel: helpers
// ---------------------------------------------------------------------------
// XOR swizzle of the 16-byte chunk index within a token row of a tile in LDS:
// both the 16-row x one-chunk operand reads (K) and the transposed V reads
// (8 rows x 4 chunks) spread over all bank groups.
template <int D>
__device__ __forceinline__ int tile_swizzle(int row) {
  if constexpr (D == 32) return (row >> 2) & 3;
  if constexpr (D == 64) return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
  return ((row & 3) << 2) | ((row >> 2) & 3);
}

// One 16-byte direct global -> LDS load per lane (global_load_lds_dwordx4):
// lane reads base + byte_off and the wave's 64 chunks land contiguously at LDS
// byte address lds_wave_addr + 16 * lane (passed in m0).  base and lds_wave_addr must be
// wave-uniform (scalar registers).  Issued as inline asm so that the compiler
// neither waits for it before unrelated LDS reads nor drains it at every
// barrier: the kernel waits for these loads explicitly (wait_vmem_upto) right
// before the barrier that publishes the tile they fill.  NT marks data read
// once (the queries) as streaming, so that it does not displace the K/V tiles
// that the other beam tiles of the request still read.
template <bool NT = false>
__device__ __forceinline__ void load_to_lds(const void* base, uint32_t byte_off,
                                            uint32_t lds_wave_addr) {
  if constexpr (NT)
    asm volatile("global_load_lds_dwordx4 %0, %1 nt"
                 :
                 : "v"(byte_off), "s"(base), "{m0}"(lds_wave_addr)
                 : "memory");
  else
    asm volatile("global_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(byte_off), "s"(base), "{m0}"(lds_wave_addr)
                 : "memory");
}

// Workgroup barrier that orders LDS only: pending LDS operations complete,
// then s_barrier.  Outstanding global loads stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// max(a, b, c) as one v_max3_f32.  Written as asm: built from fmaxf the
// compiler first canonicalises every MFMA result (one extra v_max per value).
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// max over lanes l and l ^ 32 (v_permlane32_swap).
__device__ __forceinline__ float max_with_other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return max3(__uint_as_float(r[0]), __uint_as_float(r[1]), __uint_as_float(r[1]));
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel (head dims 32, 64 and 128).
//
// Work split.  A workgroup is four waves (one per SIMD) of 32*kMB beams each,
// and two workgroups share each CU, so every SIMD runs two independent waves.
// XCD-aware workgroup ordering (work_item) puts the beam tiles of one
// (request, head) on one XCD, whose L2 then serves that head's K/V to all of
// them, and gives every XCD the same share of each request.
//
// Software pipeline.  Each wave runs over 32-key steps so that its
// instruction stream always holds independent matrix and vector work:
//
//   step j:  exp2/pack of S(j)^T (VALU)                  -> P(j)
//            S(j+1)^T = K(j+1) Q^T (MFMA, accumulating)
//            O^T += V(j)^T P(j)^T and the row sums (MFMA, one chunk behind
//            the exp2/pack that produces its P; the last chunk is carried
//            into step j+1)
//
// in a fixed issue order: every 32x32x16 product is followed by the VALU work
// that fits under it (two multiply + exp2 pairs), so that one wave alone
// keeps both the matrix core and the VALU busy.  Q^T stays in registers as
// the input bf16 values; the softmax scale (times log2 e) multiplies the fp32
// scores just before exp2, so the only roundings ahead of the softmax are those
// of the inputs themselves.
//
// Stream.  K and V pass through two four-buffer LDS rings in tiles of kTileN
// keys, K one tile ahead of V: at the start of tile T the workgroup issues
// K(T+3) and V(T+2) (direct-to-LDS loads) and at its end waits for K(T+2) and
// V(T+1) and meets at one barrier, so tile T reads K(T), K(T+1) and V(T) while
// the buffers being filled were last read before the previous barrier.
//
// Softmax.  The fast pass takes no maximum: the scores go straight through
// exp2.  After the last step each wave checks that every beam's row sum lies
// in [2^-100, 2^64] and that its O is finite, and the waves vote.  If any beam
// fails, the whole workgroup redoes its tile with the safe pass (stepwise, not
// pipelined): an exponent shift per beam that starts at 0 and moves only when
// the first step's maximum lies outside [-64, 32] or a later step's maximum
// exceeds the shift by more than 32.  Then the shift becomes the running
// maximum, O and the row sums are rescaled, and every later score enters exp2
// as fma(S, c, -shift) in fp32.
// With the shift bounded this way exp2 never overflows (P <= 2^32) and the
// largest weight of a beam is at least 2^-64, so the safe pass gives the
// softmax of the definition for any input; the fast pass is kept only when its
// sums prove it neither overflowed nor lost precision to underflow.
//
// Row sums.  One v_mfma_f32_16x16x32_bf16 per 16-key chunk and beam block
// sums the applied bf16 weights: it reads the P^T fragment of the 32x32x16
// product as a 32-key x 16-column operand, in which column c holds beam c in
// its even 8-key groups and beam c+16 in its odd ones, so A rows with ones on
// the even (odd) groups give the sums of beam c (c+16).
// ---------------------------------------------------------------------------
template <int D>
struct Cfg {
  static constexpr int kWaves = 4;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kMB = D == 128 ? 1 : 2;         // 32-beam blocks per wave
  static constexpr int kBlockM = kWaves * kMB * 32;    // beams per workgroup
  static constexpr int kTileN = D == 128 ? 32 : 64;    // keys per LDS tile
  static constexpr int kSub = kTileN / 32;             // 32-key steps per tile
  static constexpr int kKS = D / 16;                   // 16-wide d steps of QK
  static constexpr int kDB = D / 32;                   // 32-wide d blocks of O
  static constexpr int kCPR = D / 8;                   // 16-byte chunks per token row
  static constexpr int kRowBytes = kCPR * 16;
  static constexpr int kSlots = kTileN * kCPR;
  static constexpr int kLoads = kSlots / kThreads;     // loads per thread per tile and tensor
  static constexpr int kTileBytes = kSlots * 16;
  static constexpr int kNBuf = 4;
  static constexpr int kLdsBytes = 2 * kNBuf * kTileBytes;
  static constexpr int kUnits = 2 * kMB;               // (16-key chunk, beam block) pairs per step
  static constexpr int kQKPerUnit = kKS * kMB / kUnits;
  static constexpr float kShiftHi = 32.0f;
  static constexpr float kShiftLo = -64.0f;
  static_assert(kSlots % kThreads == 0 && (kKS * kMB) % kUnits == 0, "even split");
  static_assert(kLoads * 2 <= 8, "wait_vmem_upto covers up to eight loads per tile");
  __device__ __forceinline__ static int slot(int key, int chunk) {
    return key * kCPR + (chunk ^ tile_swizzle<D>(key));
  }
  // Output staging layout: eight consecutive beam rows written at one chunk
  // index, and one row read whole, both fall on distinct 16-byte bank groups.
  __device__ __forceinline__ static int out_slot(int row, int chunk) {
    const int s = kCPR >= 8 ? (row & 7) : ((row >> 1) & (kCPR - 1));
    return row * kCPR + (chunk ^ s);
  }
};

// s_waitcnt vmcnt(n) for n in [0, 8].
__device__ __forceinline__ void wait_vmem_upto(int n) {
  switch (n) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(1)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(2)" ::: "memory"); break;
    case 3: asm volatile("s_waitcnt vmcnt(3)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
    case 5: asm volatile("s_waitcnt vmcnt(5)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(6)" ::: "memory"); break;
    case 7: asm volatile("s_waitcnt vmcnt(7)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
  }
}

// Work item of workgroup i: (beam tile mt, request b, head h).  Workgroup i
// runs on XCD x = i % 8.  When the head count is a multiple of 8, XCD x takes
// the heads h = x (mod 8) of every request, so each XCD gets the same mix of
// encoder lengths (the same work for ragged requests), and walks the requests
// starting at request x*B/8, so that at any time the XCDs read different
// requests' rows.  All beam tiles of one (request, head) run back to back on
// one XCD, whose L2 then serves that head's K/V to all of them.
__device__ __forceinline__ void work_item(uint32_t i, uint32_t n, int32_t n_mt, int32_t B,
                                          int32_t H, int32_t& mt, int32_t& b, int32_t& h) {
  constexpr uint32_t kXcds = 8;
  if (H % kXcds != 0) {
    const uint32_t tile = xcd_remap(i, n);
    mt = (int32_t)(tile % (uint32_t)n_mt);
    const uint32_t bh = tile / (uint32_t)n_mt;
    h = (int32_t)(bh % (uint32_t)H);
    b = (int32_t)(bh / (uint32_t)H);
    return;
  }
  const uint32_t x = i % kXcds, k = i / kXcds;
  const uint32_t hpx = (uint32_t)H / kXcds;            // heads per XCD and request
  const uint32_t p = k / (uint32_t)n_mt;                // (request, head) pair of this XCD
  mt = (int32_t)(k % (uint32_t)n_mt);
  const uint32_t shift = x * (((uint32_t)B + kXcds - 1) / kXcds);
  b = (int32_t)((p / hpx + shift) % (uint32_t)B);
  h = (int32_t)((p % hpx) * kXcds + x);
}

template <int D>
__global__ void __launch_bounds__(Cfg<D>::kThreads, 2)
cross_attn_bf16_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                            const uint16_t* __restrict__ v, const int32_t* __restrict__ off,
                            uint16_t* __restrict__ out, int32_t B, int32_t M, int32_t H,
                            int32_t sum_L, int32_t n_mt, float c) {
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(16))) char lds[C::kLdsBytes];
  char* const kbuf0 = lds;                              // K ring: 4 tiles
  char* const vbuf0 = lds + C::kNBuf * C::kTileBytes;   // V ring: 4 tiles

  int32_t mt, b, h;
  work_item(blockIdx.x, gridDim.x, n_mt, B, H, mt, b, h);
  if (threadIdx.x == 0)
    GRACE_DCHECK(0 <= b && b < B && 0 <= h && h < H && 0 <= mt && mt < n_mt, kDbgRow);
  int32_t o0, L;
  request_span(off, b, sum_L, o0, L);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int32_t E = H * D;   // 32-bit offsets: B*M*H*d and sum_L*H*d < 2^31 (checked by the API)
  const int32_t m_base = mt * C::kBlockM + wave * (C::kMB * 32);
  const bool active = m_base < M;
  const int32_t n = (L + C::kTileN - 1) / C::kTileN;   // LDS tiles
  const int32_t n_sub = (L + 31) / 32;                  // 32-key steps

  // Row-sum operands (16x16x32): lane = row (lane & 15), 8-key group lane >> 4.
  bf16x8 sum_a[C::kMB];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    const int row = lane & 15, odd = (lane >> 4) & 1;
    const uint32_t w = row == 2 * mb + odd ? 0x3f803f80u : 0u;
    sum_a[mb] = __builtin_bit_cast(bf16x8, u32x4{w, w, w, w});
  }

  // Direct-to-LDS tile loads (one tile of K or V per call).
  uint32_t dma_off[C::kLoads];
#pragma unroll
  for (int i = 0; i < C::kLoads; ++i) {
    const int sl = i * C::kThreads + threadIdx.x;
    const int key = sl / C::kCPR;
    const int chunk = (sl % C::kCPR) ^ tile_swizzle<D>(key);
    // modular uint32 arithmetic: offsets of rows past the request may wrap,
    // but every offset actually loaded (after clamping) is below 2^32
    dma_off[i] = ((uint32_t)key * (uint32_t)E + (uint32_t)(h * D + chunk * 8)) * 2u;
  }
  const uint32_t kb_addr = __builtin_amdgcn_readfirstlane(lds_addr(kbuf0) + wave * 64 * 16);
  const uint32_t vb_addr = kb_addr + C::kNBuf * C::kTileBytes;
  const uint16_t* const kreq = k + o0 * E;
  const uint16_t* const vreq = v + o0 * E;
  auto issue = [&](const uint16_t* req, uint32_t lds_base, int32_t t) __attribute__((always_inline)) {
    const int32_t t0 = t * C::kTileN;
    const uint16_t* base = req + t0 * E;
    const uint32_t dst = lds_base + (t & (C::kNBuf - 1)) * C::kTileBytes;
    if (t0 + C::kTileN <= L) {
#pragma unroll
      for (int i = 0; i < C::kLoads; ++i) {
        GRACE_DCHECK(o0 + t0 + (i * C::kThreads + (int)threadIdx.x) / C::kCPR < sum_L, kDbgRow);
        load_to_lds(base, dma_off[i], dst + i * C::kThreads * 16);
      }
    } else {
#pragma unroll
      for (int i = 0; i < C::kLoads; ++i) {
        const int key = (i * C::kThreads + (int)threadIdx.x) / C::kCPR;
        const int over = key - (L - 1 - t0);   // > 0: past the last token
        const uint32_t o = over > 0 ? dma_off[i] - (uint32_t)over * (uint32_t)E * 2u : dma_off[i];
        GRACE_DCHECK(o0 + t0 + (over > 0 ? key - over : key) < sum_L, kDbgRow);
        load_to_lds(base, o, dst + i * C::kThreads * 16);
      }
    }
  };
  // Loads of tile T's start (K(T+3), V(T+2)); returns how many this thread issued.
  auto prefetch = [&](int32_t T) __attribute__((always_inline)) -> int {
    int issued = 0;
    if (T + 3 < n) { issue(kreq, kb_addr, T + 3); issued += C::kLoads; }
    if (T + 2 < n) { issue(vreq, vb_addr, T + 2); issued += C::kLoads; }
    return issued;
  };
  // Tile T's end: K(T+2) and V(T+1) have landed (the loads of this tile's start
  // may still fly), then the barrier that publishes them.
  auto publish = [&](int issued) __attribute__((always_inline)) {
    wait_vmem_upto(issued);
    lds_barrier();
  };
  // The prologue's loads: K(0), K(1), V(0) with the queries, K(2), V(1)
  // once the queries are in registers.  Returns how many this thread issued.
  auto prologue_early = [&]() __attribute__((always_inline)) -> int {
    if (n > 0) issue(kreq, kb_addr, 0);
    if (n > 1) issue(kreq, kb_addr, 1);
    if (n > 0) issue(vreq, vb_addr, 0);
    return (n > 0 ? 2 : 0) * C::kLoads + (n > 1 ? C::kLoads : 0);
  };
  auto prologue_late = [&]() __attribute__((always_inline)) -> int {
    int late = 0;
    if (n > 2) { issue(kreq, kb_addr, 2); late += C::kLoads; }
    if (n > 1) { issue(vreq, vb_addr, 1); late += C::kLoads; }
    return late;
  };

  // Queries.  Each wave copies its beams' Q rows into a staging buffer of its
  // own (K buffer 2 or 3, V buffer 2 or 3: free until the loads that follow
  // the prologue barrier) in the tile layout, with direct-to-LDS loads whose
  // 64 lanes cover whole rows, then reads its Q^T fragments (B operand of
  // S^T = K Q^T) from there: lane holds 8 consecutive d of beam l32 of block
  // mb, for 16-wide d step ks.  Beams past M repeat beam M-1, whose results
  // are never stored.  The queries are issued first: they are needed first.
  char* const qbuf = wave < 2 ? kbuf0 + (2 + wave) * C::kTileBytes
                              : vbuf0 + wave * C::kTileBytes;
  if (active) {
    const uint16_t* const qbase = q + __builtin_amdgcn_readfirstlane((b * M + m_base) * E + h * D);
    const uint32_t q_lds = __builtin_amdgcn_readfirstlane(lds_addr(qbuf));
    const int last = M - 1 - m_base;
#pragma unroll
    for (int i = 0; i < C::kTileBytes / 1024; ++i) {
      const int sl = i * 64 + lane;
      const int row = sl / C::kCPR;
      const int chunk = (sl % C::kCPR) ^ tile_swizzle<D>(row);
      const int r = row < last ? row : last;
      GRACE_DCHECK(m_base + r < M, kDbgRow);
      load_to_lds<true>(qbase, (uint32_t)(r * E + chunk * 8) * 2u, q_lds + i * 1024);
    }
  }
  const int early = prologue_early();
  wait_vmem_upto(early);   // this wave's queries have landed
  bf16x8 qf[C::kMB][C::kKS];
  if (active) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks) {
        const u32x4 u = *(const u32x4*)(qbuf + C::slot(mb * 32 + l32, 2 * ks + hi) * 16);
        qf[mb][ks] = __builtin_bit_cast(bf16x8, u);
      }
  } else {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks) qf[mb][ks] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
  }
  wait_vmem_upto(0);   // K(0), K(1), V(0) have landed
  // publishes K(0), K(1), V(0); every staging buffer has been read
  lds_barrier();

  // LDS read offsets of this lane within a tile.  K (A of S^T): one per
  // 16-wide d step.  V^T (transposed reads): one per (8-row half, 32-wide d
  // block).  32-key steps add 32 rows, 16-key chunks 16 rows; row strides keep
  // the swizzle, so they and the buffer bases are immediates.
  uint32_t k_rd[C::kKS];
#pragma unroll
  for (int ks = 0; ks < C::kKS; ++ks) k_rd[ks] = lds_addr(kbuf0) + C::slot(l32, 2 * ks + hi) * 16;
  uint32_t v_rd[2][C::kDB];
  {
    const int g4 = lane >> 4, gi = lane & 15;
#pragma unroll
    for (int w = 0; w < 2; ++w)
#pragma unroll
      for (int db = 0; db < C::kDB; ++db) {
        const int dcol = db * 32 + 16 * (g4 & 1) + 4 * (gi & 3);
        const int row = 8 * w + 4 * (g4 >> 1) + (gi >> 2);
        v_rd[w][db] = lds_addr(vbuf0) + C::slot(row, dcol >> 3) * 16 + (dcol & 7) * 2;
      }
  }
  typedef __attribute__((address_space(3))) char lds_char;
  // K fragment of d step ks for the 32-key step `sub` of the tile in buffer `buf`.
  auto read_k = [&](int buf, int sub, int ks) __attribute__((always_inline)) -> bf16x8 {
    return __builtin_bit_cast(
        bf16x8, *(const __attribute__((address_space(3))) u32x4*)(
                    (lds_char*)(uintptr_t)k_rd[ks] + buf * C::kTileBytes + sub * 32 * C::kRowBytes));
  };
  // V^T fragments of 16-key chunk kc of the 32-key step `sub` of buffer `buf`.
  auto read_v = [&](int buf, int sub, int kc, bf16x8 (&vf)[C::kDB]) __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < C::kDB; ++db) {
      i16x4 part[2];
#pragma unroll
      for (int w = 0; w < 2; ++w)
        part[w] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4*)((lds_char*)(uintptr_t)v_rd[w][db] +
                                                         buf * C::kTileBytes +
                                                         (2 * sub + kc) * 16 * C::kRowBytes));
      typedef short i16x8 __attribute__((ext_vector_type(8)));
      const i16x8 both = __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
      vf[db] = __builtin_bit_cast(bf16x8, both);
    }
  };

  f32x16 o[C::kDB][C::kMB];
  f32x4 lsum = {0.f, 0.f, 0.f, 0.f};   // lanes 0-15: rows 2mb / 2mb+1 = beams c / c+16 of block mb
  float shift[C::kMB];   // safe pass: exponent shift of this lane's beam, exp2 units
  auto reset_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      shift[mb] = 0.f;
#pragma unroll
      for (int db = 0; db < C::kDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][mb][r] = 0.f;
    }
    lsum = f32x4{0.f, 0.f, 0.f, 0.f};
  };
  reset_acc();

  // O += V^T P^T and the row sums of P, one 16-key chunk of beam block mb.
  auto pv = [&](const bf16x8 (&vf)[C::kDB], const bf16x8& p, int mb) __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < C::kDB; ++db)
      o[db][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db], p, o[db][mb], 0, 0, 0);
    lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sum_a[mb], p, lsum, 0, 0, 0);
  };
  // exp2 of rows 8kc..8kc+7 of S^T block mb, packed to bf16 (a P^T fragment).
  auto exp_pack = [&](f32x16& s, int kc) __attribute__((always_inline)) -> bf16x8 {
    const int r0 = 8 * kc;
#pragma unroll
    for (int r = 0; r < 8; ++r) s[r0 + r] = fast_exp2(s[r0 + r]);
    const u32x4 u = {pack_bf16x2(s[r0 + 0], s[r0 + 1]), pack_bf16x2(s[r0 + 2], s[r0 + 3]),
                     pack_bf16x2(s[r0 + 4], s[r0 + 5]), pack_bf16x2(s[r0 + 6], s[r0 + 7])};
    return __builtin_bit_cast(bf16x8, u);
  };
  // Keys at or past L in step j get weight 0.
  auto mask_step = [&](f32x16 (&s)[C::kMB], int32_t j) __attribute__((always_inline)) {
    const int32_t k0 = j * 32;
    if (k0 + 32 > L) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (key >= L) {
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb) s[mb][r] = -INFINITY;
        }
      }
    }
  };
  const f32x16 zero16 = {};

  // ------------------------------ fast pass ------------------------------
  {
    // Two register sets, alternated by the parity of the step index (the tile
    // loop is unrolled over the ring, so parities are known at compile time):
    // scores of the current and the next step, and V^T fragments of a step's
    // two 16-key chunks, the second of which serves the chunk carried into the
    // next step.
    f32x16 s_set[2][C::kMB];
    bf16x8 v_set[2][2][C::kDB];
    bf16x8 pf[2][C::kMB];
    // The first step's carried chunk is an exact zero product.
#pragma unroll
    for (int db = 0; db < C::kDB; ++db)
      v_set[1][1][db] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb)
      pf[1][mb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});

    prologue_late();
    // Every scalar and LDS load issued so far is complete; saying so in a
    // form the compiler tracks (s_waitcnt with vmcnt and expcnt at their
    // maxima, lgkmcnt 0) lets it wait for exactly the LDS reads each product
    // needs in the loop below.  Otherwise a scalar load it still counts as
    // pending (it may return out of order) makes it wait for every
    // outstanding LDS read, the ones just issued included, once per step.
    __builtin_amdgcn_s_waitcnt(0xC07F);


    // Step j (parity P): K of step j+1 from buffer kbuf (32-key step ksub of
    // that tile), V of step j from buffer vbuf (step vsub).  The scores of
    // step j+1 past the last step are computed from stale LDS and never used.
    //
    // Unit u = (16-key chunk kc, beam block mb) issues, in this order: its QK
    // products, the PV products and row sum of the previous unit (unit 0: the
    // chunk carried from step j-1), each followed by a slice of its own VALU
    // work (8 exp2, then 4 packs), so that one wave keeps both the matrix
    // core and the VALU busy; fences keep the compiler from regrouping them.
    // LDS fragments are read one unit ahead of their products; with two steps
    // per tile, the first K fragments of step j+1 are read during step j (the
    // tile they come from was published one tile early).
    constexpr bool kCrossPrefetch = C::kSub == 2;
    bf16x8 kf_next[C::kQKPerUnit];   // first unit's K fragments of the next step
    auto unit_ks = [](int u, int qq) { return (u * C::kQKPerUnit + qq) / C::kMB; };
    auto read_unit_k = [&](int kbuf, int ksub, int u, bf16x8 (&kf)[C::kQKPerUnit])
                           __attribute__((always_inline)) {
#pragma unroll
      for (int qq = 0; qq < C::kQKPerUnit; ++qq)
        if (qq == 0 || unit_ks(u, qq) != unit_ks(u, qq - 1)) kf[qq] = read_k(kbuf, ksub, unit_ks(u, qq));
#pragma unroll
      for (int qq = 1; qq < C::kQKPerUnit; ++qq)
        if (unit_ks(u, qq) == unit_ks(u, qq - 1)) kf[qq] = kf[qq - 1];
    };
    auto step = [&](int32_t j, auto parity, int kbuf, int ksub, int vbuf, int vsub,
                    int kbuf_n, int ksub_n) __attribute__((always_inline)) {
      constexpr int P = decltype(parity)::value;
      f32x16(&s_cur)[C::kMB] = s_set[P];
      f32x16(&s_nxt)[C::kMB] = s_set[P ^ 1];
      bf16x8(&vf)[2][C::kDB] = v_set[P];
      const bf16x8(&vf_carry)[C::kDB] = v_set[P ^ 1][1];
      mask_step(s_cur, j);
      bf16x8 kf[2][C::kQKPerUnit];
      if constexpr (kCrossPrefetch) {
#pragma unroll
        for (int qq = 0; qq < C::kQKPerUnit; ++qq) kf[0][qq] = kf_next[qq];
      } else {
        read_unit_k(kbuf, ksub, 0, kf[0]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < C::kUnits; ++u) {
        const int kc = u / C::kMB, mb = u % C::kMB;
        // LDS reads for what comes next
        if (u == 0) read_v(vbuf, vsub, 0, vf[0]);
        if (u == (C::kMB > 1 ? C::kMB - 1 : 0)) read_v(vbuf, vsub, 1, vf[1]);
        if (u + 1 < C::kUnits)
          read_unit_k(kbuf, ksub, u + 1, kf[(u + 1) & 1]);
        else if constexpr (kCrossPrefetch)
          read_unit_k(kbuf_n, ksub_n, 0, kf_next);
        __builtin_amdgcn_sched_barrier(0);
        // this unit's VALU work, handed out in slices after each product
        f32x16& s = s_cur[mb];
        const int r0 = 8 * kc;
        u32x4 pw;
        int next_item = 0;
        constexpr int kM = C::kQKPerUnit + C::kDB;
        constexpr int kSlice = 8 / kM > 0 ? 8 / kM : 1;
        auto valu = [&](int count) __attribute__((always_inline)) {
#pragma unroll
          for (int c2 = 0; c2 < count; ++c2) {
            const int it = next_item + c2;
            if (it < 8) {
              s[r0 + it] = fast_exp2(s[r0 + it] * c);
            } else if (it < 12) {
              const int w = it - 8;
              pw[w] = pack_bf16x2(s[r0 + 2 * w], s[r0 + 2 * w + 1]);
            }
          }
          next_item += count;
        };
        // QK products of S(j+1)^T
#pragma unroll
        for (int qq = 0; qq < C::kQKPerUnit; ++qq) {
          const int qi = u * C::kQKPerUnit + qq;
          const int ks = qi / C::kMB, mq = qi % C::kMB;
          s_nxt[mq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[u & 1][qq], qf[mq][ks],
                                                              ks == 0 ? zero16 : s_nxt[mq], 0, 0, 0);
          valu(kSlice);
          __builtin_amdgcn_sched_barrier(0);
        }
        // PV of the previous chunk
        const bf16x8(&pvv)[C::kDB] = u == 0 ? vf_carry : vf[(u - 1) / C::kMB];
        const int pc = u == 0 ? 1 : (u - 1) / C::kMB;
        const int pm = u == 0 ? C::kMB - 1 : (u - 1) % C::kMB;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db) {
          o[db][pm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pvv[db], pf[pc][pm], o[db][pm], 0, 0, 0);
          valu(kSlice);
          __builtin_amdgcn_sched_barrier(0);
        }
        lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sum_a[pm], pf[pc][pm], lsum, 0, 0, 0);
        valu(12 - next_item);
        pf[kc][mb] = __builtin_bit_cast(bf16x8, pw);
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // S(0)^T, and the first K fragments of step 0 (they belong to step 1)
    if (active && n_sub > 0) {
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks) {
        const bf16x8 kf = read_k(0, 0, ks);
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb)
          s_set[0][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              kf, qf[mb][ks], ks == 0 ? zero16 : s_set[0][mb], 0, 0, 0);
      }
      if constexpr (kCrossPrefetch) read_unit_k(0, 1, 0, kf_next);
    }

    for (int32_t T0 = 0; T0 < n; T0 += C::kNBuf) {
#pragma unroll
      for (int i = 0; i < C::kNBuf; ++i) {
        const int32_t T = T0 + i;
        if (T < n) {
          const int issued = prefetch(T);
          if (active) {
#pragma unroll
            for (int s = 0; s < C::kSub; ++s) {
              const int32_t j = T * C::kSub + s;
              if (j < n_sub) {
                // K of step j+1 (this step's QK) and of step j+2 (prefetched)
                const int kb = s + 1 < C::kSub ? i : (i + 1) & (C::kNBuf - 1);
                const int kb2 = s + 2 < C::kSub ? i : (s + 2 < 2 * C::kSub ? (i + 1) & (C::kNBuf - 1)
                                                                           : (i + 2) & (C::kNBuf - 1));
                // T0 * kSub is even, so step j's parity is that of i * kSub + s
                if (((i * C::kSub + s) & 1) == 0)
                  step(j, std::integral_constant<int, 0>{}, kb, (s + 1) % C::kSub, i, s, kb2,
                       (s + 2) % C::kSub);
                else
                  step(j, std::integral_constant<int, 1>{}, kb, (s + 1) % C::kSub, i, s, kb2,
                       (s + 2) % C::kSub);
              }
            }
          }
          publish(issued);
        }
      }
    }
    // the last step's carried chunk
    if (active && n_sub > 0) {
      if ((n_sub - 1) & 1)
        pv(v_set[1][1], pf[1][C::kMB - 1], C::kMB - 1);
      else
        pv(v_set[0][1], pf[1][C::kMB - 1], C::kMB - 1);
    }
  }

  // Keep the fast pass only if every beam of the workgroup passes the check.
  bool rerun = false;
  {
    bool bad = false;
    if (active && n_sub > 0) {
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) {
        const float l = lsum[2 * mb], l2 = lsum[2 * mb + 1];   // lanes 0-15 hold the sums
        if ((lane & 15) == lane)
          bad |= !(l >= 0x1p-100f && l <= 0x1p64f) || !(l2 >= 0x1p-100f && l2 <= 0x1p64f);
        float chk = 0.f;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) chk = __builtin_fmaf(o[db][mb][r], 0.f, chk);
        bad |= chk != 0.f;   // inf * 0 and NaN * 0 are NaN
      }
    }
    // One vote word per wave in K buffer 3: every load has landed and no wave
    // reads LDS after the last tile's barrier, and the rerun's prologue fills
    // K buffers 0-2 and V buffers 0-1 only; K buffer 3 is next written at the
    // rerun's first tile, after its prologue barrier.
    int32_t* votes = (int32_t*)(kbuf0 + 3 * C::kTileBytes);
    const bool wave_bad = __any(bad);
    if (lane == 0) votes[wave] = wave_bad ? 1 : 0;
    lds_barrier();
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) rerun |= votes[w] != 0;
  }

  // ------------------------------ safe pass ------------------------------
  if (rerun) {
    reset_acc();
    prologue_early();
    const int late = prologue_late();
    wait_vmem_upto(late);
    lds_barrier();
    float alpha[C::kMB];
    for (int32_t T = 0; T < n; ++T) {
      const int issued = prefetch(T);
      const int buf = T & (C::kNBuf - 1);
      if (active) {
#pragma unroll 1
        for (int s = 0; s < C::kSub; ++s) {
          const int32_t j = T * C::kSub + s;
          if (j >= n_sub) break;
          // S(j)^T, then the exp2 arguments c*S - shift in fp32
          f32x16 sc[C::kMB];
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb) sc[mb] = zero16;
#pragma unroll
          for (int ks = 0; ks < C::kKS; ++ks) {
            const bf16x8 kf = read_k(buf, s, ks);
#pragma unroll
            for (int mb = 0; mb < C::kMB; ++mb)
              sc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[mb][ks], sc[mb], 0, 0, 0);
          }
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) sc[mb][r] = __builtin_fmaf(sc[mb][r], c, -shift[mb]);
          mask_step(sc, j);
          // each beam's maximum; move the shift of beams that need it
          float mx[C::kMB];
          bool any = false;
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb) {
            float m0 = max3(sc[mb][0], sc[mb][1], sc[mb][2]);
#pragma unroll
            for (int r = 3; r + 1 < 16; r += 2) m0 = max3(m0, sc[mb][r], sc[mb][r + 1]);
            m0 = max3(m0, sc[mb][15], sc[mb][15]);
            mx[mb] = max_with_other_half(m0);
            any |= j == 0 ? (mx[mb] > C::kShiftHi || mx[mb] < C::kShiftLo) : mx[mb] > C::kShiftHi;
          }
          if (__any(any)) {
#pragma unroll
            for (int mb = 0; mb < C::kMB; ++mb) {
              const bool need =
                  j == 0 ? (mx[mb] > C::kShiftHi || mx[mb] < C::kShiftLo) : mx[mb] > C::kShiftHi;
              const float ns = need ? shift[mb] + mx[mb] : shift[mb];
              const float delta = ns - shift[mb];
              alpha[mb] = fast_exp2(-delta);
              shift[mb] = ns;
#pragma unroll
              for (int r = 0; r < 16; ++r) sc[mb][r] -= delta;
              // O and the row sums hold only weights of the old shift
              const float alpha_hi = __shfl_xor(alpha[mb], 16);
              lsum[2 * mb] *= alpha[mb];
              lsum[2 * mb + 1] *= alpha_hi;
#pragma unroll
              for (int db = 0; db < C::kDB; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[db][mb][r] *= alpha[mb];
            }
          }
#pragma unroll
          for (int kc = 0; kc < 2; ++kc) {
            bf16x8 vfs[C::kDB];
            read_v(buf, s, kc, vfs);
#pragma unroll
            for (int mb = 0; mb < C::kMB; ++mb) pv(vfs, exp_pack(sc[mb], kc), mb);
          }
        }
      }
      publish(issued);
    }
  }

  // Output.  Each wave normalises its O^T, writes it to V buffer `wave` as
  // beam-major rows (out_slot layout), and stores whole rows from there: a
  // store instruction then writes 64 16-byte chunks that cover full rows
  // rather than 32 scattered 16-byte pieces.  The stores are streaming: O is
  // written once and no later access in the kernel reuses it.  Every wave is past the barrier
  // after its last LDS read (the vote's, or the safe pass's last tile), every
  // tile load has landed, and no wave touches another wave's buffer here.
  if (active) {
    char* const obuf = vbuf0 + wave * C::kTileBytes;
    // lane index opaque to the compiler, so that the addresses below are not
    // hoisted above the main loop (where they would only occupy registers)
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int l32e = ln & 31, hie = ln >> 5;
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      // beam l32's row sum: lane l32 & 15, row 2mb (l32 < 16) or 2mb+1
      const float s_lo = __shfl(lsum[2 * mb], l32e & 15);
      const float s_hi = __shfl(lsum[2 * mb + 1], l32e & 15);
      const float l_tot = l32e < 16 ? s_lo : s_hi;
      const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
#pragma unroll
      for (int db = 0; db < C::kDB; ++db)
#pragma unroll
        for (int gp = 0; gp < 2; ++gp) {
          // lane holds d = 32db + 16gp + {0..3} + 4hi (group 2gp) and + 8
          // (group 2gp+1); the swap with lane l ^ 32 leaves d 32db + 16gp +
          // 8hi + {0..7} in (a, b)
          uint32_t a[2], c2[2];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            a[e] = pack_bf16x2(o[db][mb][8 * gp + 2 * e] * inv, o[db][mb][8 * gp + 2 * e + 1] * inv);
            c2[e] = pack_bf16x2(o[db][mb][8 * gp + 4 + 2 * e] * inv,
                                o[db][mb][8 * gp + 4 + 2 * e + 1] * inv);
          }
          u32x4 chunk;
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const auto r = __builtin_amdgcn_permlane32_swap(a[e], c2[e], false, false);
            chunk[e] = r[0];
            chunk[2 + e] = r[1];
          }
          const int row = mb * 32 + l32e;
          *(u32x4*)(obuf + C::out_slot(row, 4 * db + 2 * gp + hie) * 16) = chunk;
        }
    }
    __builtin_amdgcn_wave_barrier();
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    constexpr int kRows = C::kMB * 32;
    constexpr int kRowsPerPass = 64 / C::kCPR;
#pragma unroll
    for (int i = 0; i < kRows / kRowsPerPass; ++i) {
      const int row = i * kRowsPerPass + ln / C::kCPR;
      const int ch = ln % C::kCPR;
      const u32x4 u = *(const u32x4*)(obuf + C::out_slot(row, ch) * 16);
      const int32_t m = m_base + row;
      GRACE_DCHECK(b * M + m < B * M || m >= M, kDbgRow);
      if (m < M) __builtin_nontemporal_store(u, (u32x4*)(out + (b * M + m) * E + h * D + ch * 8));
    }
  }
}

hipError_t debug_take_cross(uint32_t* acc) {
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

hipError_t launch_cross_attn(const void* q, const void* enc_k, const void* enc_v,
                             const int32_t* enc_off, void* out, int32_t B, int32_t M, int32_t H,
                             int32_t d, int32_t sum_L, float scale, bool bf16,
                             hipStream_t stream) {
  const float c = scale * kLog2e;
  if (bf16) {
#define GRACE_X(DD)                                                                           \
  {                                                                                           \
    const int32_t n_mt = (M + Cfg<DD>::kBlockM - 1) / Cfg<DD>::kBlockM;                    \
    const int64_t grid = (int64_t)B * H * n_mt;                                              \
    hipLaunchKernelGGL(cross_attn_bf16_kernel<DD>, dim3((unsigned)grid),                 \
                       dim3(Cfg<DD>::kThreads), 0, stream, (const uint16_t*)q,               \
                       (const uint16_t*)enc_k, (const uint16_t*)enc_v, enc_off, (uint16_t*)out, \
                       B, M, H, sum_L, n_mt, c);                                              \
    return hipGetLastError();                                                                 \
  }
    if (d == 32) GRACE_X(32)
    if (d == 64) GRACE_X(64)
    if (d == 128) GRACE_X(128)
#undef GRACE_X
  } else {
#define GRACE_X(DD)                                                                          \
  {                                                                                          \
    const int32_t n_mt = (M + 64 / (DD / 32) - 1) / (64 / (DD / 32));                       \
    const int64_t grid = (int64_t)B * H * n_mt;                                             \
    hipLaunchKernelGGL(cross_attn_f32_kernel<DD>, dim3((unsigned)grid), dim3(64), 0, stream, \
                       (const float*)q, (const float*)enc_k, (const float*)enc_v, enc_off,   \
                       (float*)out, M, H, sum_L, n_mt, c);                                   \
    return hipGetLastError();                                                                \
  }
    if (d == 32) GRACE_X(32)
    if (d == 64) GRACE_X(64)
    if (d == 128) GRACE_X(128)
#undef GRACE_X
  }
  return hipErrorInvalidValue;
}

}  // namespace grace
