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

// One 16-byte direct global -> LDS load per lane (global_load_lds_dwordx4);
// the wave's 64 chunks land contiguously at LDS byte address lds_wave_addr +
// 16 * lane.  Issued as inline asm so that the compiler neither waits for it
// before unrelated LDS reads nor drains it at every barrier: the kernel waits
// for these loads explicitly (wait_vmem) right before the barrier that
// publishes the tile they fill.  lds_wave_addr must be wave-uniform.
__device__ __forceinline__ void load_to_lds(const void* gsrc, uint32_t lds_wave_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gsrc), "s"(lds_wave_addr)
               : "memory", "m0");
}

// s_waitcnt vmcnt(0) issued as inline asm (the loads above are invisible to
// the compiler's wait tracking).
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

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

// ---------------------------------------------------------------------------
// bf16 MFMA kernel, two workgroups per CU (head dims 32, 64 and 128).
//
// A workgroup is four waves (one per SIMD) and two workgroups share each CU,
// so every SIMD runs two independent waves: while one is in its MFMA phase
// the other is usually in its softmax phase, and one workgroup's prologue
// (Q staging) and epilogue (O stores) overlap the other's tiles.
//
// Per tile t a wave runs its MFMA phase (O += V(t-1)^T P(t-1)^T, then
// S(t)^T = K(t) Q^T - shift) and its softmax phase, then meets the other three
// waves at one barrier.  K and V each rotate through three LDS buffers: K(t+2)
// and V(t+1) are issued (global_load_lds_dwordx4) at the start of tile t and
// waited for at the end of tile t+1, two tiles after issue; the buffer each
// load overwrites was last read before the barrier that ended tile t-1.
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
  static_assert(kSlots % kThreads == 0 && (kBlockM * kCPR) % kThreads == 0, "even split");
  __device__ __forceinline__ static int swz(int key) { return tile_swizzle<D>(key); }
  __device__ __forceinline__ static int slot(int key, int chunk) {
    return key * kCPR + (chunk ^ swz(key));
  }
};

// s_waitcnt vmcnt(n) for the n most recent loads still allowed in flight.
__device__ __forceinline__ void wait_vmem_keep(int n) {
  if (n >= 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if (n >= 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

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

  // Running shift of each beam, folded into S^T by a rank-1 MFMA term
  // S^T += 1 * (-shift): A has 1 in k-slots 0 and 1 of lanes 0-31, B carries
  // -shift of the lane's beam split into a bf16 pair (hi, lo) in those slots,
  // so the shift has 16 significant bits and is exactly what the MFMA adds.
  // Row sums: A = ones in rows 16*mb .. 16*mb+15 (all rows when one beam block),
  // B = P^T of beam block mb, so registers 8*mb .. 8*mb+7 of the lane owning
  // beam j accumulate beam j's sum.
  const bf16x8 one_a = __builtin_bit_cast(bf16x8, u32x4{hi == 0 ? 0x3f803f80u : 0u, 0u, 0u, 0u});
  bf16x8 ones_a[C::kMB];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    const uint32_t w = (C::kMB == 1 || (l32 >> 4) == mb) ? 0x3f803f80u : 0u;
    ones_a[mb] = __builtin_bit_cast(bf16x8, u32x4{w, w, w, w});
  }
  float shift[C::kMB];
  bf16x8 bias_b[C::kMB];
  f32x16 o[C::kDB][C::kMB];
  f32x16 lsum;
#pragma unroll
  for (int r = 0; r < 16; ++r) lsum[r] = 0.f;
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    shift[mb] = 0.f;
    bias_b[mb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
#pragma unroll
    for (int db = 0; db < C::kDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][mb][r] = 0.f;
  }
  f32x16 s[C::kKB][C::kMB];
  bf16x8 pf[C::kKC][C::kMB];

  const int32_t n = (L + C::kBlockN - 1) / C::kBlockN;
  auto src_of = [&](int i, int32_t t0) -> int32_t {
    const int sl = i * C::kThreads + threadIdx.x;
    const int key = sl / C::kCPR;
    const int chunk = (sl % C::kCPR) ^ C::swz(key);
    int32_t tok = t0 + key;
    tok = tok < L ? tok : L - 1;
    return (o0 + tok) * E + h * D + chunk * 8;
  };
  const uint32_t kb_addr = __builtin_amdgcn_readfirstlane(lds_addr(kbuf0) + wave * 64 * 16);
  const uint32_t vb_addr = kb_addr + C::kNBuf * C::kTileBytes;
  auto load_k = [&](int32_t t) {
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i)
      load_to_lds(k + src_of(i, t * C::kBlockN), kb_addr + (t % C::kNBuf) * C::kTileBytes + i * C::kThreads * 16);
  };
  auto load_v = [&](int32_t t) {
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i)
      load_to_lds(v + src_of(i, t * C::kBlockN), vb_addr + (t % C::kNBuf) * C::kTileBytes + i * C::kThreads * 16);
  };
  // Prologue: the first K/V tiles go out before Q is staged, so their latency
  // overlaps the Q loads; one wait covers both.
  if (n > 0) load_k(0);
  if (n > 1) load_k(1);
  if (n > 0) load_v(0);
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

  // Q^T fragments of this wave's beams, held in registers for all tiles.
  bf16x8 qf[C::kMB][C::kKS];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
    for (int ks = 0; ks < C::kKS; ++ks)
      qf[mb][ks] = __builtin_bit_cast(
          bf16x8, *(const u32x4*)(qbuf + C::slot(wave * (C::kMB * 32) + mb * 32 + l32, 2 * ks + hi) * 16));

  for (int32_t t = 0; t <= n; ++t) {
    int issued = 0;
    if (t + 2 < n) { load_k(t + 2); issued += C::kLoads; }
    if (t + 1 < n) { load_v(t + 1); issued += C::kLoads; }
    if (active) {
      // ---- MFMA phase: O += V(t-1)^T P(t-1)^T, then S(t)^T = K(t) Q^T - shift ----
      __builtin_amdgcn_s_setprio(1);
      if (t >= 1) {
        const char* vb = vbuf0 + ((t - 1) % C::kNBuf) * C::kTileBytes;
        const int g4 = lane >> 4, gi = lane & 15;
        bf16x8 vfr[C::kKC][C::kDB];
#pragma unroll
        for (int kc = 0; kc < C::kKC; ++kc)
#pragma unroll
          for (int db = 0; db < C::kDB; ++db) {
            const int dcol = db * 32 + 16 * (g4 & 1) + 4 * (gi & 3);
            i16x4 part[2];
#pragma unroll
            for (int w = 0; w < 2; ++w) {
              const int row = 16 * kc + 8 * w + 4 * (g4 >> 1) + (gi >> 2);
              const int byte = C::slot(row, dcol >> 3) * 16 + (dcol & 7) * 2;
              part[w] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                  (__attribute__((address_space(3))) i16x4*)(
                      (__attribute__((address_space(3))) char*)vb + byte));
            }
            typedef short i16x8 __attribute__((ext_vector_type(8)));
            const i16x8 both = __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
            vfr[kc][db] = __builtin_bit_cast(bf16x8, both);
          }
#pragma unroll
        for (int kc = 0; kc < C::kKC; ++kc) {
#pragma unroll
          for (int db = 0; db < C::kDB; ++db)
#pragma unroll
            for (int mb = 0; mb < C::kMB; ++mb)
              o[db][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[kc][db], pf[kc][mb], o[db][mb], 0, 0, 0);
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb)
            lsum = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ones_a[mb], pf[kc][mb], lsum, 0, 0, 0);
        }
      }
      if (t < n) {
        const char* kbp = kbuf0 + (t % C::kNBuf) * C::kTileBytes;
        bf16x8 kf[C::kKB][C::kKS];
#pragma unroll
        for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
          for (int ks = 0; ks < C::kKS; ++ks)
            kf[kb][ks] = __builtin_bit_cast(
                bf16x8, *(const u32x4*)(kbp + C::slot(kb * 32 + l32, 2 * ks + hi) * 16));
        const f32x16 zero = {};
#pragma unroll
        for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb)
            s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(one_a, bias_b[mb], zero, 0, 0, 0);
#pragma unroll
        for (int ks = 0; ks < C::kKS; ++ks)
#pragma unroll
          for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
            for (int mb = 0; mb < C::kMB; ++mb)
              s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kb][ks], qf[mb][ks], s[kb][mb], 0, 0, 0);
      }
      __builtin_amdgcn_s_setprio(0);

      if (t < n) {
        // ---- softmax phase of tile t: S^T holds exp2 arguments ----
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
        float mx[C::kMB];
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb) {
          float a[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) a[j] = fmaxf(s[0][mb][2 * j], s[0][mb][2 * j + 1]);
#pragma unroll
          for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
            for (int r = (kb == 0 ? 8 : 0); r < 16; r += 8)
#pragma unroll
              for (int j = 0; j < 4; ++j)
                a[j] = fmaxf(fmaxf(a[j], s[kb][mb][r + 2 * j]), s[kb][mb][r + 2 * j + 1]);
          mx[mb] = fmaxf(fmaxf(fmaxf(a[0], a[1]), a[2]), a[3]);
          mx[mb] = fmaxf(mx[mb], __shfl_xor(mx[mb], 32));
        }
        bool need[C::kMB];
        bool any = false;
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb) {
          need[mb] = t == 0 || mx[mb] > 8.0f;
          any |= need[mb];
        }
        if (__any(any)) {
#pragma unroll
          for (int mb = 0; mb < C::kMB; ++mb) {
            const float ns = need[mb] ? round_to_bf16x2(shift[mb] + mx[mb]) : shift[mb];
            const float delta = ns - shift[mb];
            const float alpha = t == 0 ? 1.0f : fast_exp2(-delta);
            shift[mb] = ns;
#pragma unroll
            for (int r = 0; r < (C::kMB == 1 ? 16 : 8); ++r) lsum[(C::kMB == 1 ? 0 : 8 * mb) + r] *= alpha;
#pragma unroll
            for (int db = 0; db < C::kDB; ++db)
#pragma unroll
              for (int r = 0; r < 16; ++r) o[db][mb][r] *= alpha;
#pragma unroll
            for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
              for (int r = 0; r < 16; ++r) s[kb][mb][r] -= delta;
            const float nhi = round_to_bf16(-ns);
            const uint32_t nb = pack_bf16x2(nhi, -ns - nhi);
            bias_b[mb] = __builtin_bit_cast(bf16x8, u32x4{hi == 0 ? nb : 0u, 0u, 0u, 0u});
          }
        }
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb) {
#pragma unroll
          for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kb][mb][r] = fast_exp2(s[kb][mb][r]);
#pragma unroll
          for (int kc = 0; kc < C::kKC; ++kc) {
            const int kb = kc >> 1, r0 = 8 * (kc & 1);
            const u32x4 u = {pack_bf16x2(s[kb][mb][r0 + 0], s[kb][mb][r0 + 1]),
                             pack_bf16x2(s[kb][mb][r0 + 2], s[kb][mb][r0 + 3]),
                             pack_bf16x2(s[kb][mb][r0 + 4], s[kb][mb][r0 + 5]),
                             pack_bf16x2(s[kb][mb][r0 + 6], s[kb][mb][r0 + 7])};
            pf[kc][mb] = __builtin_bit_cast(bf16x8, u);
          }
        }
      }
    }
    if (t < n) {
      wait_vmem_keep(issued);   // K(t+1) and V(t) have landed; K(t+2), V(t+1) may fly
      lds_barrier();
    }
  }

  if (active) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      const float l_tot = lsum[C::kMB == 1 ? 0 : 8 * mb];
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
