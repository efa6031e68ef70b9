// Beam-as-query cross-attention for gfx950 (GRACE, Sec. 5.1, App. B).
//
// The M beams of request b are the query rows of one contraction against that
// request's encoder K/V.  A workgroup owns one (request, head, beam tile);
// K/V stream through LDS in token tiles that every beam of the tile reuses,
// so each encoder token is read from L2 once per beam tile, not once per beam.
//
// bf16 path (MFMA, cross_attn_bf16_dual_kernel).  Each wave owns 64 beams
// (32 at head dim 128) and, per tile, computes
//   S^T = K Q^T - shift   v_mfma_f32_32x32x16_bf16; A = K rows from LDS, B = Q^T
//                         (pre-multiplied by scale*log2(e)) held in registers,
//                         plus one rank-1 MFMA that subtracts the beam's shift,
//                         so S^T holds exp2 arguments directly;
//   P = exp2(S^T)         VALU, lazily re-shifted when a beam's running max
//                         grows by more than 8 (exp2 units);
//   O^T += V^T P^T        A = V^T read with ds_read_b64_tr_b16, B = P^T taken
//                         straight from the S^T registers as bf16;
//   l += 1^T P^T          the row sums of the applied bf16 weights, on the
//                         matrix core as well.
// The transposed orientation puts one beam per lane column in every product,
// so the probabilities never leave registers.
//
// fp32 path (VALU, cross_attn_f32_kernel).  One lane per beam, K/V tiles in LDS
// read as broadcasts, fp32 FMAs throughout.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace grace {

// ---------------------------------------------------------------------------
// XCD-aware tile order.  Consecutive workgroup ids go round-robin over the 8
// XCDs; remapping puts the beam tiles of one (request, head) on one XCD and
// close in time, so that XCD's L2 serves the request's K/V to all of them.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t xcd_remap(uint32_t i, uint32_t n) {
  constexpr uint32_t kXcds = 8;
  if (n % kXcds != 0) return i;
  return (i % kXcds) * (n / kXcds) + i / kXcds;
}

__device__ __forceinline__ void request_span(const int32_t* off, int32_t b, int32_t sum_L,
                                             int32_t& o0, int32_t& L) {
  int32_t a = off[b], e = off[b + 1];
  a = a < 0 ? 0 : (a > sum_L ? sum_L : a);
  e = e < a ? a : (e > sum_L ? sum_L : e);
  o0 = a;
  L = e - a;
}

// ---------------------------------------------------------------------------
// fp32 VALU kernel
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(64)
cross_attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k,
                      const float* __restrict__ v, const int32_t* __restrict__ off,
                      float* __restrict__ out, int32_t M, int32_t H, int32_t sum_L,
                      int32_t n_mt, float c) {
  constexpr int TILE = 32;
  __shared__ float ks[TILE][D];
  __shared__ float vs[TILE][D];
  const uint32_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int32_t mt = tile % n_mt;
  const int32_t bh = tile / n_mt;
  const int32_t h = bh % H, b = bh / H;
  const int32_t m = mt * 64 + threadIdx.x;
  int32_t o0, L;
  request_span(off, b, sum_L, o0, L);
  const int64_t E = (int64_t)H * D;
  const int64_t row = (int64_t)b * M + m;

  float qr[D], acc[D];
#pragma unroll
  for (int e = 0; e < D; ++e) {
    qr[e] = m < M ? q[row * E + h * D + e] : 0.f;
    acc[e] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  for (int32_t t0 = 0; t0 < L; t0 += TILE) {
    const int32_t n = min(TILE, L - t0);
    __syncthreads();
    for (int i = threadIdx.x; i < TILE * D; i += 64) {
      const int key = i / D, col = i % D;
      const int64_t src = (int64_t)(o0 + t0 + (key < n ? key : n - 1)) * E + h * D + col;
      ks[key][col] = k[src];
      vs[key][col] = v[src];
    }
    __syncthreads();
    float s[TILE];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < TILE; ++j) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < D; ++e) a = __builtin_fmaf(qr[e], ks[j][e], a);
      s[j] = j < n ? a : -INFINITY;
      mx = fmaxf(mx, s[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2((m_run - m_new) * c);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int e = 0; e < D; ++e) acc[e] *= alpha;
#pragma unroll
    for (int j = 0; j < TILE; ++j) {
      const float p = fast_exp2((s[j] - m_new) * c);
      l_run += p;
#pragma unroll
      for (int e = 0; e < D; ++e) acc[e] = __builtin_fmaf(p, vs[j][e], acc[e]);
    }
  }
  if (m < M) {
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) out[row * E + h * D + e] = acc[e] * inv;
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
// XOR swizzle of the 16-byte chunk index within a token (or beam) row of a
// tile in LDS: both the 16-row x one-chunk operand reads (K, Q) and the
// transposed V reads (8 rows x 4 chunks) spread over all bank groups.
template <int D>
__device__ __forceinline__ int tile_swizzle(int row) {
  if constexpr (D == 32) return (row >> 2) & 3;
  if constexpr (D == 64) return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
  return ((row & 3) << 2) | ((row >> 2) & 3);
}

// One 16-byte direct global -> LDS load per lane (global_load_lds_dwordx4):
// lane reads base + byte_off and the wave's 64 chunks land contiguously at LDS
// byte address lds_wave_addr + 16 * lane.  base and lds_wave_addr must be
// wave-uniform (scalar registers).  Issued as inline asm so that the compiler
// neither waits for it before unrelated LDS reads nor drains it at every
// barrier: the kernel waits for these loads explicitly (wait_vmem_keep) right
// before the barrier that publishes the tile they fill.
__device__ __forceinline__ void load_to_lds(const void* base, uint32_t byte_off,
                                            uint32_t lds_wave_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(byte_off), "s"(base), "s"(lds_wave_addr)
               : "memory", "m0");
}

// s_waitcnt vmcnt(0) issued as inline asm (the loads above are invisible to
// the compiler's wait tracking).
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// s_waitcnt vmcnt(n) for the n most recent loads still allowed in flight.
__device__ __forceinline__ void wait_vmem_keep(int n) {
  if (n >= 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if (n >= 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Workgroup barrier that orders LDS only: pending LDS operations complete,
// then s_barrier.  Outstanding global loads stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ __forceinline__ float round_to_bf16(float x) {
  return __uint_as_float((pack_bf16x2(x, 0.f) & 0xffffu) << 16);
}

// x rounded to the nearest value that is the sum of two bf16 numbers hi + lo
// with hi = bf16(x) (16 significant bits).
__device__ __forceinline__ float round_to_bf16x2(float x) {
  const float h = round_to_bf16(x);
  return h + round_to_bf16(x - h);
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
// bf16 MFMA kernel, two workgroups per CU (head dims 32, 64 and 128).
//
// A workgroup is four waves (one per SIMD) and two workgroups share each CU,
// so every SIMD runs two independent waves: while one is in its MFMA phase
// the other is usually in its softmax phase, and one workgroup's prologue
// (Q staging) and epilogue (O stores) overlap the other's tiles.
//
// Per tile t a wave runs its MFMA phase (O += V(t-1)^T P(t-1)^T and the row
// sums of P(t-1), then S(t)^T = K(t) Q^T [- shift]) and its softmax phase,
// then meets the other three waves at one barrier.  K and V each rotate
// through three LDS buffers: K(t+2) and V(t+1) are issued at the start of
// tile t and waited for at the end of tile t+1, two tiles after issue; the
// buffer each load overwrites was last read before the barrier that ended
// tile t-1.
//
// Exponent shift.  exp2 arguments are S^T minus a per-beam shift that starts
// at 0 and moves only when needed: when the first tile's maximum lies outside
// [-64, 32] or a later tile's maximum exceeds the shift by more than 32.  Then
// the shift becomes the running maximum (as a bf16 hi+lo pair, 16 significant
// bits), O and the row sums are rescaled, and from then on a rank-1 MFMA term
// subtracts it inside the S^T product.  With the shift bounded this way
// exp2 never overflows (P <= 2^32) and the largest weight of a beam is at
// least 2^-64, so the result is the softmax of the definition for any input;
// with the shift at 0 (scores within those bounds, the common case) the
// rank-1 term and every rescale are skipped.
//
// Row sums.  One v_mfma_f32_16x16x32_bf16 per 16-key chunk and beam block
// sums the applied bf16 weights: it reads the P^T fragment of the 32x32x16
// product as a 32-key x 16-column operand, in which column c holds beam c in
// its even 8-key groups and beam c+16 in its odd ones, so A rows with ones on
// the even (odd) groups give the sums of beam c (c+16).
// ---------------------------------------------------------------------------
template <int D>
struct Dual {
  static constexpr int kWaves = 4;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kMB = D == 128 ? 1 : 2;        // 32-beam blocks per wave
  static constexpr int kBlockM = kWaves * kMB * 32;   // beams per workgroup
  static constexpr int kBlockN = D == 128 ? 32 : 64;  // encoder tokens per tile
  static constexpr int kKB = kBlockN / 32;
  static constexpr int kKS = D / 16;
  static constexpr int kDB = D / 32;
  static constexpr int kKC = kBlockN / 16;
  static constexpr int kCPR = D / 8;
  static constexpr int kSlots = kBlockN * kCPR;
  static constexpr int kLoads = kSlots / kThreads;    // 16-byte loads per thread per tile and tensor
  static constexpr int kTileBytes = kSlots * 16;
  static constexpr int kNBuf = 3;
  static constexpr int kQChunks = kBlockM * kCPR / kThreads;
  static constexpr int kQBytes = kBlockM * D * 2;
  static constexpr int kLdsBytes = 2 * kNBuf * kTileBytes + kQBytes;
  static constexpr float kShiftHi = 32.0f;    // re-shift when a tile max exceeds the shift by this
  static constexpr float kShiftLo = -64.0f;   // ... or the first tile's max is below this
  static_assert(kSlots % kThreads == 0 && (kBlockM * kCPR) % kThreads == 0, "even split");
  __device__ __forceinline__ static int swz(int key) { return tile_swizzle<D>(key); }
  __device__ __forceinline__ static int slot(int key, int chunk) {
    return key * kCPR + (chunk ^ swz(key));
  }
};

template <int D>
__global__ void __launch_bounds__(Dual<D>::kThreads, 2)
cross_attn_bf16_dual_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                            const uint16_t* __restrict__ v, const int32_t* __restrict__ off,
                            uint16_t* __restrict__ out, int32_t M, int32_t H, int32_t sum_L,
                            int32_t n_mt, float c) {
  using C = Dual<D>;
  static_assert(C::kLoads * 2 <= 4, "wait_vmem_keep covers up to four loads per tile");
  __shared__ __attribute__((aligned(16))) char lds[C::kLdsBytes];
  char* const kbuf0 = lds;                                 // K tiles: 3 buffers
  char* const vbuf0 = lds + C::kNBuf * C::kTileBytes;      // V tiles: 3 buffers
  char* const qbuf = lds + 2 * C::kNBuf * C::kTileBytes;   // scaled Q of the beam tile

  const uint32_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int32_t mt = tile % n_mt;
  const int32_t bh = tile / n_mt;
  const int32_t h = bh % H, b = bh / H;
  int32_t o0, L;
  request_span(off, b, sum_L, o0, L);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int32_t E = H * D;   // 32-bit offsets: B*M*H*d and sum_L*H*d < 2^31 (checked by the API)
  const int32_t m_base = mt * C::kBlockM + wave * (C::kMB * 32);
  const bool active = m_base < M;

  // Row-sum operands (16x16x32): lane = row (lane & 15), 8-key group lane >> 4.
  bf16x8 sum_a[C::kMB];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    const int row = lane & 15, odd = (lane >> 4) & 1;
    const uint32_t w = row == 2 * mb + odd ? 0x3f803f80u : 0u;
    sum_a[mb] = __builtin_bit_cast(bf16x8, u32x4{w, w, w, w});
  }
  float shift[C::kMB];
  f32x16 o[C::kDB][C::kMB];
  f32x4 lsum = {0.f, 0.f, 0.f, 0.f};   // lanes 0-15: rows 2mb / 2mb+1 = beams c / c+16 of block mb
  bool biased = false;                 // some beam of the wave has a non-zero shift
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    shift[mb] = 0.f;
#pragma unroll
    for (int db = 0; db < C::kDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][mb][r] = 0.f;
  }
  f32x16 s[C::kKB][C::kMB];
  bf16x8 pf[C::kKC][C::kMB];

  const int32_t n = (L + C::kBlockN - 1) / C::kBlockN;

  // This lane's K/V slots of a tile: byte offsets from the tile's first token
  // row (the same for K and V); the last, partial tile clamps its tokens.
  uint32_t dma_off[C::kLoads];
#pragma unroll
  for (int i = 0; i < C::kLoads; ++i) {
    const int sl = i * C::kThreads + threadIdx.x;
    const int key = sl / C::kCPR;
    const int chunk = (sl % C::kCPR) ^ C::swz(key);
    // modular uint32 arithmetic: offsets of rows past the request may wrap,
    // but every offset actually loaded (after clamping) is below 2^32
    dma_off[i] = ((uint32_t)key * (uint32_t)E + (uint32_t)(h * D + chunk * 8)) * 2u;
  }
  const uint32_t kb_addr = __builtin_amdgcn_readfirstlane(lds_addr(kbuf0) + wave * 64 * 16);
  const uint32_t vb_addr = kb_addr + C::kNBuf * C::kTileBytes;
  const uint16_t* const kreq = k + o0 * E;
  const uint16_t* const vreq = v + o0 * E;
  auto issue = [&](const uint16_t* req, uint32_t lds_base, int32_t t) __attribute__((always_inline)) {
    const int32_t t0 = t * C::kBlockN;
    const uint16_t* base = req + t0 * E;
    const uint32_t dst = lds_base + (t % C::kNBuf) * C::kTileBytes;
    if (t0 + C::kBlockN <= L) {
#pragma unroll
      for (int i = 0; i < C::kLoads; ++i) load_to_lds(base, dma_off[i], dst + i * C::kThreads * 16);
    } else {
#pragma unroll
      for (int i = 0; i < C::kLoads; ++i) {
        const int key = (i * C::kThreads + (int)threadIdx.x) / C::kCPR;
        const int over = key - (L - 1 - t0);   // > 0: past the last token
        const uint32_t o = over > 0 ? dma_off[i] - (uint32_t)over * (uint32_t)E * 2u : dma_off[i];
        load_to_lds(base, o, dst + i * C::kThreads * 16);
      }
    }
  };

  // LDS read offsets of this lane within a tile.  K (A of S^T): one per
  // 16-wide d step; the 32-key blocks add kb * 32 rows.  V^T (transposed
  // reads): one per (8-row half, 32-wide d block); 16-key chunks add kc * 16
  // rows.  Row strides leave the swizzle unchanged, so they are immediates.
  uint32_t k_rd[C::kKS];
#pragma unroll
  for (int ks = 0; ks < C::kKS; ++ks) k_rd[ks] = C::slot(l32, 2 * ks + hi) * 16;
  uint32_t v_rd[2][C::kDB];
  {
    const int g4 = lane >> 4, gi = lane & 15;
#pragma unroll
    for (int w = 0; w < 2; ++w)
#pragma unroll
      for (int db = 0; db < C::kDB; ++db) {
        const int dcol = db * 32 + 16 * (g4 & 1) + 4 * (gi & 3);
        const int row = 8 * w + 4 * (g4 >> 1) + (gi >> 2);
        v_rd[w][db] = C::slot(row, dcol >> 3) * 16 + (dcol & 7) * 2;
      }
  }
  constexpr int kKeyRowBytes = C::kCPR * 16;

  // Prologue: the first K/V tiles go out before Q is staged, so their latency
  // overlaps the Q loads; one wait covers both.
  if (n > 0) issue(kreq, kb_addr, 0);
  if (n > 1) issue(kreq, kb_addr, 1);
  if (n > 0) issue(vreq, vb_addr, 0);
  // Stage Q (times c = scale*log2(e), re-rounded to bf16) in the K-tile slot
  // layout; beams past M repeat beam M-1, whose results are never stored.
#pragma unroll
  for (int i = 0; i < C::kQChunks; ++i) {
    const int sl = i * C::kThreads + threadIdx.x;
    const int beam = sl / C::kCPR;
    const int chunk = (sl % C::kCPR) ^ C::swz(beam);
    int32_t m = mt * C::kBlockM + beam;
    m = m < M ? m : M - 1;
    const u32x4 u = *(const u32x4*)(q + (b * M + m) * E + h * D + chunk * 8);
    float f[8];
    Chunk<BF16>::unpack(u, f);
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] *= c;
    *(u32x4*)(qbuf + sl * 16) = Chunk<BF16>::pack(f);
  }

  wait_vmem();                          // K(0), K(1), V(0) have landed
  lds_barrier();

  // Q^T fragments of this wave's beams.  At head dim 32 they stay in
  // registers for all tiles; at 64 and 128 they are re-read from LDS with the
  // K fragments of every tile (Q sits in the same slot layout, so the K read
  // offsets serve), which keeps the exp/PV phase within the register budget.
  constexpr bool kQInRegs = D == 32;
  const char* const qwave = qbuf + wave * (C::kMB * 32) * C::kCPR * 16;
  bf16x8 qf_res[kQInRegs ? C::kMB : 1][kQInRegs ? C::kKS : 1];
  if constexpr (kQInRegs) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks)
        qf_res[mb][ks] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)(qwave + k_rd[ks] + mb * 32 * C::kCPR * 16));
  }

  // S(t)^T = K(t) Q^T, starting from the shift term or from zero.
  auto qk = [&](const char* kbp, auto with_shift) __attribute__((always_inline)) {
    // K and Q fragments of one 16-wide d step, loaded one step ahead.
    auto load_ks = [&](int ks, bf16x8 (&kf)[C::kKB], bf16x8 (&qf)[C::kMB])
        __attribute__((always_inline)) {
#pragma unroll
      for (int kb = 0; kb < C::kKB; ++kb)
        kf[kb] = __builtin_bit_cast(bf16x8,
                                    *(const u32x4*)(kbp + k_rd[ks] + kb * 32 * kKeyRowBytes));
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) {
        if constexpr (kQInRegs)
          qf[mb] = qf_res[mb][ks];
        else
          qf[mb] = __builtin_bit_cast(
              bf16x8, *(const u32x4*)(qwave + k_rd[ks] + mb * 32 * kKeyRowBytes));
      }
    };
    bf16x8 kf[2][C::kKB], qf[2][C::kMB];
    load_ks(0, kf[0], qf[0]);
    const f32x16 zero = {};
#pragma unroll
    for (int ks = 0; ks < C::kKS; ++ks) {
      if (ks + 1 < C::kKS) load_ks(ks + 1, kf[(ks + 1) & 1], qf[(ks + 1) & 1]);
      const bf16x8(&k)[C::kKB] = kf[ks & 1];
      const bf16x8(&qq)[C::kMB] = qf[ks & 1];
#pragma unroll
      for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb) {
          if (ks > 0) {
            s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k[kb], qq[mb], s[kb][mb], 0, 0, 0);
          } else if constexpr (decltype(with_shift)::value) {
            // Rank-1 term S^T += 1 * (-shift): A has 1 in k-slots 0 and 1 of
            // lanes 0-31, B carries -shift of the lane's beam as a bf16 pair
            // (hi, lo) in those slots, so the MFMA adds exactly the 16-bit
            // shift (shift is a sum of two bf16 values).
            const float nhi = round_to_bf16(-shift[mb]);
            const uint32_t nb = pack_bf16x2(nhi, -shift[mb] - nhi);
            const bf16x8 one_a =
                __builtin_bit_cast(bf16x8, u32x4{hi == 0 ? 0x3f803f80u : 0u, 0u, 0u, 0u});
            const bf16x8 bias_b =
                __builtin_bit_cast(bf16x8, u32x4{hi == 0 ? nb : 0u, 0u, 0u, 0u});
            s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                k[kb], qq[mb],
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(one_a, bias_b, zero, 0, 0, 0), 0, 0, 0);
          } else {
            s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k[kb], qq[mb], zero, 0, 0, 0);
          }
        }
    }
  };

  // V(t)^T fragments (transposed LDS reads) of 16-key chunk kc.
  auto read_v = [&](int32_t t, int kc, bf16x8 (&vf)[C::kDB]) __attribute__((always_inline)) {
    const char* vb = vbuf0 + (t % C::kNBuf) * C::kTileBytes;
#pragma unroll
    for (int db = 0; db < C::kDB; ++db) {
      i16x4 part[2];
#pragma unroll
      for (int w = 0; w < 2; ++w)
        part[w] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4*)(
                (__attribute__((address_space(3))) char*)vb + v_rd[w][db] +
                kc * 16 * kKeyRowBytes));
      typedef short i16x8 __attribute__((ext_vector_type(8)));
      const i16x8 both = __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
      vf[db] = __builtin_bit_cast(bf16x8, both);
    }
  };
  // O += V^T P^T and the row sums of P for chunk kc, beam block mb.
  auto pv_chunk = [&](const bf16x8 (&vf)[C::kDB], int kc, int mb) __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < C::kDB; ++db)
      o[db][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db], pf[kc][mb], o[db][mb], 0, 0, 0);
    lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sum_a[mb], pf[kc][mb], lsum, 0, 0, 0);
  };
  // P = exp2(S^T) for chunk kc, beam block mb, as a bf16 fragment over pf.
  auto exp_chunk = [&](int kc, int mb) __attribute__((always_inline)) {
    const int kb = kc >> 1, r0 = 8 * (kc & 1);
#pragma unroll
    for (int r = 0; r < 8; ++r) s[kb][mb][r0 + r] = fast_exp2(s[kb][mb][r0 + r]);
    const u32x4 u = {pack_bf16x2(s[kb][mb][r0 + 0], s[kb][mb][r0 + 1]),
                     pack_bf16x2(s[kb][mb][r0 + 2], s[kb][mb][r0 + 3]),
                     pack_bf16x2(s[kb][mb][r0 + 4], s[kb][mb][r0 + 5]),
                     pack_bf16x2(s[kb][mb][r0 + 6], s[kb][mb][r0 + 7])};
    pf[kc][mb] = __builtin_bit_cast(bf16x8, u);
  };
  // All of tile t's P into O (V chunks read one ahead of their MFMAs).
  auto pv_tile = [&](int32_t t) __attribute__((always_inline)) {
    bf16x8 vf[2][C::kDB];
    read_v(t, 0, vf[0]);
#pragma unroll
    for (int kc = 0; kc < C::kKC; ++kc) {
      if (kc + 1 < C::kKC) read_v(t, kc + 1, vf[(kc + 1) & 1]);
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) pv_chunk(vf[kc & 1], kc, mb);
    }
  };
  // pv_tile(t - 1) fused with the exp/pack of tile t: chunk by chunk, the
  // MFMAs read P(t-1) from pf, then exp/pack writes P(t) into the same
  // registers; the scheduler interleaves each chunk's MFMAs with its VALU work.
  constexpr int kChunkMfma = C::kDB + 1;   // per (chunk, beam block)
  constexpr int kChunkValu = 8 + 4;        // 8 exp2 + 4 packs
  auto pv_exp_tile = [&](int32_t tv) __attribute__((always_inline)) {
    bf16x8 vf[2][C::kDB];
    read_v(tv, 0, vf[0]);
#pragma unroll
    for (int kc = 0; kc < C::kKC; ++kc) {
      if (kc + 1 < C::kKC) read_v(tv, kc + 1, vf[(kc + 1) & 1]);
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) {
        pv_chunk(vf[kc & 1], kc, mb);
        exp_chunk(kc, mb);
      }
    }
    // Pin P(t) here: without a use in this block the compiler sinks the
    // exp/pack work below the (rare) rescale branch, away from the MFMAs.
#pragma unroll
    for (int kc = 0; kc < C::kKC; ++kc)
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) asm volatile("" ::"v"(pf[kc][mb]));
    constexpr int kV = kChunkValu / kChunkMfma;
    constexpr int kVLast = kChunkValu - (kChunkMfma - 1) * kV;
#pragma unroll
    for (int g = 0; g < C::kKC * C::kMB; ++g) {
#pragma unroll
      for (int i = 0; i + 1 < kChunkMfma; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, kV, 0);   // then VALU
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, kVLast, 0);
    }
  };

  // Softmax bookkeeping of tile t on S(t)^T: mask the keys past L, take each
  // beam's maximum and, when a beam needs it (rare), move its shift.
  // Keys past L in the last, partial tile get weight 0.
  auto mask_tail = [&](int32_t t) __attribute__((always_inline)) {
    const int32_t t0 = t * C::kBlockN;
    if (t0 + C::kBlockN > L) {
#pragma unroll
      for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = t0 + kb * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
          if (key >= L) {
#pragma unroll
            for (int mb = 0; mb < C::kMB; ++mb) s[kb][mb][r] = -INFINITY;
          }
        }
    }
  };
  float alpha[C::kMB];
  auto softmax_shift = [&](int32_t t) __attribute__((always_inline)) -> bool {
    mask_tail(t);
    float mx[C::kMB];
    bool any = false;
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      // two independent max3 chains over the 16*kKB scores of the lane
      float m0 = max3(s[0][mb][0], s[0][mb][1], s[0][mb][2]);
      float m1 = max3(s[0][mb][3], s[0][mb][4], s[0][mb][5]);
#pragma unroll
      for (int i = 6; i + 3 < 16 * C::kKB; i += 4) {
        m0 = max3(m0, s[i >> 4][mb][i & 15], s[(i + 1) >> 4][mb][(i + 1) & 15]);
        m1 = max3(m1, s[(i + 2) >> 4][mb][(i + 2) & 15], s[(i + 3) >> 4][mb][(i + 3) & 15]);
      }
      // 16*kKB = 6 + 4j + 2: two scores left
      const float m = max3(max3(m0, m1, s[C::kKB - 1][mb][14]), s[C::kKB - 1][mb][15],
                           s[C::kKB - 1][mb][15]);
      mx[mb] = max_with_other_half(m);
      any |= t == 0 ? (mx[mb] > C::kShiftHi || mx[mb] < C::kShiftLo) : mx[mb] > C::kShiftHi;
    }
    if (__builtin_expect(__any(any), 0)) {
      // Move the shift of the beams that need it to their maximum.  O and the
      // row sums still lack P(t-1), which was weighted with the old shift:
      // they are rescaled by alpha once it is in (rescale_after).
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) {
        const bool need =
            t == 0 ? (mx[mb] > C::kShiftHi || mx[mb] < C::kShiftLo) : mx[mb] > C::kShiftHi;
        const float ns = need ? round_to_bf16x2(shift[mb] + mx[mb]) : shift[mb];
        const float delta = ns - shift[mb];
        alpha[mb] = fast_exp2(-delta);
        shift[mb] = ns;
#pragma unroll
        for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb][mb][r] -= delta;
      }
      biased = true;
      return true;
    }
    return false;
  };
  // O *= alpha and row sums *= alpha, per beam.
  auto rescale_after = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      // row sums: lanes 0-15 hold beam c (row 2mb) and beam c+16 (row 2mb+1)
      const float alpha_hi = __shfl_xor(alpha[mb], 16);
      lsum[2 * mb] *= alpha[mb];
      lsum[2 * mb + 1] *= alpha_hi;
#pragma unroll
      for (int db = 0; db < C::kDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][mb][r] *= alpha[mb];
    }
  };
  // Loads for tiles ahead of t, then (after this tile's work) the wait for
  // K(t+1) and V(t) and the barrier that publishes them.
  auto prefetch = [&](int32_t t) __attribute__((always_inline)) -> int {
    int issued = 0;
    if (t + 2 < n) { issue(kreq, kb_addr, t + 2); issued += C::kLoads; }
    if (t + 1 < n) { issue(vreq, vb_addr, t + 1); issued += C::kLoads; }
    return issued;
  };
  auto publish = [&](int issued) __attribute__((always_inline)) {
    wait_vmem_keep(issued);   // K(t+1) and V(t) have landed; K(t+2), V(t+1) may fly
    lds_barrier();
  };

  // One pass over the request's tokens.  Tile t: S(t)^T on the matrix core;
  // then the softmax of tile t on the VALU with the MFMAs of
  // O += V(t-1)^T P(t-1)^T interleaved into its exp/pack stream, so one wave
  // keeps both pipes busy.  Tile 0 has no P before it and the last P is
  // accumulated after the loop.
  //   fast pass (SAFE = false): the exponent shift stays 0 and no maximum is
  //     taken; the result is kept only if every beam's row sum lands in
  //     [2^-100, 2^64] and its outputs are finite (no overflow, no lost
  //     precision to underflow);
  //   safe pass (SAFE = true): the bookkeeping of the exponent shift described
  //     above, valid for any input.  Run by the whole workgroup when any of its
  //     beams failed the fast pass's check.
  auto run_pass = [&](auto safe) __attribute__((always_inline)) {
    constexpr bool SAFE = decltype(safe)::value;
    auto s_tile = [&](int32_t t) __attribute__((always_inline)) {
      const char* kbp = kbuf0 + (t % C::kNBuf) * C::kTileBytes;
      if (SAFE && biased)
        qk(kbp, std::true_type{});
      else
        qk(kbp, std::false_type{});
    };
    if (n > 0) {
      const int issued = prefetch(0);
      if (active) {
        s_tile(0);
        if constexpr (SAFE)
          softmax_shift(0);   // O and the row sums are still zero: no rescale
        else
          mask_tail(0);
#pragma unroll
        for (int kc = 0; kc < C::kKC; ++kc)
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb) exp_chunk(kc, mb);
      }
      publish(issued);
    }
    for (int32_t t = 1; t < n; ++t) {
      const int issued = prefetch(t);
      if (active) {
        s_tile(t);
        bool moved = false;
        if constexpr (SAFE)
          moved = softmax_shift(t);
        else
          mask_tail(t);
        pv_exp_tile(t - 1);
        if (SAFE && __builtin_expect(moved, 0)) rescale_after();
      }
      publish(issued);
    }
    if (active && n > 0) pv_tile(n - 1);
  };

  run_pass(std::false_type{});

  // Keep the fast pass only if every beam of the workgroup passes the check.
  {
    bool bad = false;
    if (active && n > 0) {
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
    // One vote word per wave in K buffer 2: no wave reads K after the last
    // tile's barrier, and the buffer is next written after the rerun's
    // prologue barrier (K(2)), by which time every wave has read the votes.
    // (An extra __shared__ word would push two workgroups past the CU's LDS.)
    int32_t* votes = (int32_t*)(kbuf0 + 2 * C::kTileBytes);
    const bool wave_bad = __any(bad);
    if (lane == 0) votes[wave] = wave_bad ? 1 : 0;
    lds_barrier();
    bool rerun = false;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) rerun |= votes[w] != 0;
    if (rerun) {
      // rare: the whole workgroup redoes the tokens with the exponent shift
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb) {
        shift[mb] = 0.f;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][mb][r] = 0.f;
      }
      lsum = f32x4{0.f, 0.f, 0.f, 0.f};
      biased = false;
      if (n > 0) issue(kreq, kb_addr, 0);
      if (n > 1) issue(kreq, kb_addr, 1);
      if (n > 0) issue(vreq, vb_addr, 0);
      wait_vmem();
      lds_barrier();
      run_pass(std::true_type{});
    }
  }

  if (active) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      // beam l32's row sum: lane l32 & 15, row 2mb (l32 < 16) or 2mb+1
      const float s_lo = __shfl(lsum[2 * mb], l32 & 15);
      const float s_hi = __shfl(lsum[2 * mb + 1], l32 & 15);
      const float l_tot = l32 < 16 ? s_lo : s_hi;
      const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
      const int32_t m = m_base + mb * 32 + l32;
      if (m < M) {
        uint16_t* dst = out + (b * M + m) * E + h * D + 4 * hi;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const u32x2 u = {pack_bf16x2(o[db][mb][4 * g + 0] * inv, o[db][mb][4 * g + 1] * inv),
                             pack_bf16x2(o[db][mb][4 * g + 2] * inv, o[db][mb][4 * g + 3] * inv)};
            *(u32x2*)(dst + db * 32 + 8 * g) = u;
          }
      }
    }
  }
}

hipError_t launch_cross_attn(const void* q, const void* enc_k, const void* enc_v,
                             const int32_t* enc_off, void* out, int32_t B, int32_t M, int32_t H,
                             int32_t d, int32_t sum_L, float scale, bool bf16,
                             hipStream_t stream) {
  const float c = scale * kLog2e;
  if (bf16) {
#define GRACE_X(DD)                                                                           \
  {                                                                                           \
    const int32_t n_mt = (M + Dual<DD>::kBlockM - 1) / Dual<DD>::kBlockM;                    \
    const int64_t grid = (int64_t)B * H * n_mt;                                              \
    hipLaunchKernelGGL(cross_attn_bf16_dual_kernel<DD>, dim3((unsigned)grid),                 \
                       dim3(Dual<DD>::kThreads), 0, stream, (const uint16_t*)q,               \
                       (const uint16_t*)enc_k, (const uint16_t*)enc_v, enc_off, (uint16_t*)out, \
                       M, H, sum_L, n_mt, c);                                                 \
    return hipGetLastError();                                                                 \
  }
    if (d == 32) GRACE_X(32)
    if (d == 64) GRACE_X(64)
    if (d == 128) GRACE_X(128)
#undef GRACE_X
  } else {
#define GRACE_X(DD)                                                                          \
  {                                                                                          \
    const int32_t n_mt = (M + 63) / 64;                                                      \
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
