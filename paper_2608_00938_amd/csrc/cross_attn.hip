// Beam-as-query cross-attention for gfx950 (GRACE, Sec. 5.1, App. B).
//
// The M beams of request b are the query rows of one contraction against that
// request's encoder K/V.  A workgroup owns one (request, head, 256-beam tile);
// K/V stream through LDS in 64-token tiles that all 256 beams reuse, so each
// encoder token is read from L2 once per beam tile instead of once per beam.
//
// bf16 path (MFMA).  Each of the 4 waves owns 64 beams and computes, per tile,
//   S^T = K Q^T          (v_mfma_f32_32x32x16_bf16; A = K rows from LDS,
//                         B = Q^T held in registers for the whole kernel)
//   online softmax over the tile's keys in fp32 (exp2 with the scale folded)
//   O^T += V^T P^T       (A = V^T read from LDS with ds_read_b64_tr_b16,
//                         B = P^T taken straight from the S^T accumulators)
// Working in the transposed orientation puts one beam per lane column in both
// products, so the probabilities never leave registers.
//
// fp32 path (VALU).  One lane per beam, K/V tiles in LDS read as broadcasts,
// fp32 FMAs throughout; used for fp32 inputs, which only small shapes use.
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
template <int D>
struct CrossTile {
  static constexpr int kWaves = 4;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kMB = 2;                       // 32-beam blocks per wave
  static constexpr int kBlockM = kWaves * kMB * 32;   // beams per workgroup
  static constexpr int kBlockN = 64;                  // encoder tokens per tile
  static constexpr int kKB = kBlockN / 32;            // 32-key blocks of S^T
  static constexpr int kKS = D / 16;                  // k-steps of S^T = K Q^T
  static constexpr int kDB = D / 32;                  // 32-row blocks of O^T
  static constexpr int kKC = kBlockN / 16;            // k-chunks of O^T = V^T P^T
  static constexpr int kCPR = D / 8;                  // 16-byte chunks per token row
  static constexpr int kSlots = kBlockN * kCPR;       // 16-byte slots per tile and tensor
  static constexpr int kLoads = kSlots / kThreads;    // slots each thread stages
  static constexpr int kTileBytes = kSlots * 16;
  static constexpr int kOccupancy = D == 128 ? 1 : 2; // workgroups per CU (VGPR budget)
  static_assert(kSlots % kThreads == 0, "tile must split evenly over the workgroup");

  // XOR swizzle of the 16-byte chunk index within a token row, chosen so that
  // both the K operand reads (16 tokens x one chunk) and the transposed V reads
  // (8 tokens x 4 chunks) spread over all LDS bank groups.
  __device__ __forceinline__ static int swz(int key) {
    if constexpr (D == 32) return (key >> 2) & 3;
    if constexpr (D == 64) return (((key >> 1) & 1) << 2) | ((key >> 2) & 3);
    return ((key & 3) << 2) | ((key >> 2) & 3);
  }
  __device__ __forceinline__ static int slot(int key, int chunk) {
    return key * kCPR + (chunk ^ swz(key));
  }
};

template <int D>
__global__ void __launch_bounds__(CrossTile<D>::kThreads, CrossTile<D>::kOccupancy)
cross_attn_bf16_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                       const uint16_t* __restrict__ v, const int32_t* __restrict__ off,
                       uint16_t* __restrict__ out, int32_t M, int32_t H, int32_t sum_L,
                       int32_t n_mt, float c) {
  using C = CrossTile<D>;
  __shared__ __attribute__((aligned(16))) char lds[2 * C::kTileBytes];
  char* const k_lds = lds;
  char* const v_lds = lds + C::kTileBytes;

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
  const int64_t E = (int64_t)H * D;
  const int32_t m_base = mt * C::kBlockM + wave * (C::kMB * 32);

  // Q^T operand: lane holds beam (mb*32 + l32), head dims ks*16 + 8*hi .. +7.
  bf16x8 qf[C::kMB][C::kKS];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    const int32_t m = m_base + mb * 32 + l32;
    const uint16_t* src = q + ((int64_t)b * M + m) * E + h * D + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < C::kKS; ++ks) {
      u32x4 u = m < M ? *(const u32x4*)(src + ks * 16) : u32x4{0, 0, 0, 0};
      qf[mb][ks] = __builtin_bit_cast(bf16x8, u);
    }
  }

  f32x16 o[C::kDB][C::kMB];
#pragma unroll
  for (int db = 0; db < C::kDB; ++db)
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][mb][r] = 0.f;
  float m_run[C::kMB], l_run[C::kMB];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    m_run[mb] = -INFINITY;
    l_run[mb] = 0.f;
  }

  // Global -> register staging of one K/V tile, in LDS slot order.
  u32x4 kreg[C::kLoads], vreg[C::kLoads];
  const int32_t n_tiles = (L + C::kBlockN - 1) / C::kBlockN;
#define GRACE_LOAD_TILE(T0)                                                   \
  _Pragma("unroll") for (int i = 0; i < C::kLoads; ++i) {                     \
    const int s_ = i * C::kThreads + threadIdx.x;                             \
    const int key_ = s_ / C::kCPR;                                            \
    const int chunk_ = (s_ % C::kCPR) ^ C::swz(key_);                         \
    int32_t tok_ = (T0) + key_;                                               \
    tok_ = tok_ < L ? tok_ : L - 1;                                           \
    const int64_t src_ = (int64_t)(o0 + tok_) * E + h * D + chunk_ * 8;      \
    kreg[i] = *(const u32x4*)(k + src_);                                      \
    vreg[i] = *(const u32x4*)(v + src_);                                      \
  }
  if (n_tiles > 0) { GRACE_LOAD_TILE(0) }
  for (int32_t t = 0; t < n_tiles; ++t) {
    const int32_t t0 = t * C::kBlockN;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i) {
      const int s_ = i * C::kThreads + threadIdx.x;
      *(u32x4*)(k_lds + s_ * 16) = kreg[i];
      *(u32x4*)(v_lds + s_ * 16) = vreg[i];
    }
    __syncthreads();
    if (t + 1 < n_tiles) { GRACE_LOAD_TILE(t0 + C::kBlockN) }

    // S^T = K Q^T over the tile; all K fragments are read before the MFMAs.
    bf16x8 kf[C::kKB][C::kKS];
#pragma unroll
    for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks)
        kf[kb][ks] = __builtin_bit_cast(
            bf16x8, *(const u32x4*)(k_lds + C::slot(kb * 32 + l32, 2 * ks + hi) * 16));
    f32x16 s[C::kKB][C::kMB];
#pragma unroll
    for (int kb = 0; kb < C::kKB; ++kb) {
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][mb][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks)
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb)
          s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kb][ks], qf[mb][ks], s[kb][mb], 0, 0, 0);
    }
#undef GRACE_LOAD_TILE

    // Keys past the request's end (last tile only) drop out of the softmax.
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

    // Online softmax; each lane owns beam (mb*32 + l32) and half of the keys,
    // the partner lane (lane ^ 32) the other half.
    bf16x8 pf[C::kKC][C::kMB];
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][mb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      // Lazy rescale: keep the running shift unless some beam of the wave saw
      // its maximum grow by more than 2^8 in exp2 units (p stays <= 256).
      const bool grow = (mx - m_run[mb]) * c > 8.0f;
      if (__any(grow)) {
        const float m_new = fmaxf(m_run[mb], mx);
        const float alpha = fast_exp2((m_run[mb] - m_new) * c);
        m_run[mb] = m_new;
        l_run[mb] *= alpha;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][mb][r] *= alpha;
      }
      const float m_new = m_run[mb];
      const float mc = m_new * c;
      float lsum = 0.f;
#pragma unroll
      for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(__builtin_fmaf(s[kb][mb][r], c, -mc));
          s[kb][mb][r] = p;
          lsum += p;
        }
      l_run[mb] += lsum;
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

    // O^T += V^T P^T.  The A operand of chunk kc, row block db: lane holds head
    // dim db*32 + l32 and keys 16kc + 4hi + {0..3} and 16kc + 8 + 4hi + {0..3},
    // the same key order the P^T registers carry.
    const int grp = lane >> 4, gi = lane & 15;
#pragma unroll
    for (int kc = 0; kc < C::kKC; ++kc) {
#pragma unroll
      for (int db = 0; db < C::kDB; ++db) {
        const int dcol = db * 32 + 16 * (grp & 1) + 4 * (gi & 3);
        i16x4 part[2];
#pragma unroll
        for (int w = 0; w < 2; ++w) {
          const int row = 16 * kc + 8 * w + 4 * (grp >> 1) + (gi >> 2);
          const int byte = C::slot(row, dcol >> 3) * 16 + (dcol & 7) * 2;
          part[w] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) i16x4*)(
                  (__attribute__((address_space(3))) char*)v_lds + byte));
        }
        typedef short i16x8 __attribute__((ext_vector_type(8)));
        const i16x8 both = __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7);
        const bf16x8 a = __builtin_bit_cast(bf16x8, both);
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb)
          o[db][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kc][mb], o[db][mb], 0, 0, 0);
      }
    }
  }

  // Epilogue: combine the two key halves of each beam's denominator, scale and
  // store.  Lane holds head dims db*32 + 8*(r/4) + 4*hi + (r%4) of its beam.
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    const float l_tot = l_run[mb] + __shfl_xor(l_run[mb], 32);
    const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
    const int32_t m = m_base + mb * 32 + l32;
    if (m < M) {
      uint16_t* dst = out + ((int64_t)b * M + m) * E + h * D + 4 * hi;
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

// ---------------------------------------------------------------------------
// bf16 MFMA kernel, two-group ping-pong (head dims 64 and 128).
//
// Eight waves share the workgroup's K/V tiles; two waves run on each SIMD, one
// from group A (waves 0-3) and one from group B (waves 4-7).  Per 64-token tile
// a wave has an MFMA phase (O += V^T P^T for the previous tile, then S^T = K Q^T
// for this one) and a softmax phase (VALU: max, lazy rescale, exp2, row sums,
// bf16 packing).  Group B runs one half-period behind group A, and the two
// groups meet at a workgroup barrier after every half-period, so on each SIMD
// one wave keeps the matrix core busy while the other works the VALU.
//
// Half-period h: group A works phase h, group B phase h-1; phase 2t is the MFMA
// phase of tile t and phase 2t+1 its softmax.  K tiles live in two LDS buffers
// (tile t in buffer t%2, read in half-periods 2t and 2t+1), V tiles in two more
// (tile t read in 2t+2 and 2t+3).  Tiles go global -> LDS directly
// (global_load_lds_dwordx4, no staging registers): at the start of every even
// half-period 2u each wave issues its share of K(u+1) and V(u), whose buffers
// were last read in half-period 2u-1, and waits for them only at the end of
// half-period 2u+1, just before the barrier that hands them to all waves.
// ---------------------------------------------------------------------------
template <int D>
struct PingPong {
  static constexpr int kWaves = 8;
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
  static constexpr int kLoads = kSlots / kThreads;
  static constexpr int kTileBytes = kSlots * 16;
  static_assert(kSlots % kThreads == 0, "tile must split evenly over the workgroup");
  __device__ __forceinline__ static int swz(int key) { return CrossTile<D>::swz(key); }
  __device__ __forceinline__ static int slot(int key, int chunk) {
    return key * kCPR + (chunk ^ swz(key));
  }
};

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

template <int D>
__global__ void __launch_bounds__(PingPong<D>::kThreads, 1)
cross_attn_bf16_pp_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                          const uint16_t* __restrict__ v, const int32_t* __restrict__ off,
                          uint16_t* __restrict__ out, int32_t M, int32_t H, int32_t sum_L,
                          int32_t n_mt, float c) {
  using C = PingPong<D>;
  __shared__ __attribute__((aligned(16))) char lds[4 * C::kTileBytes];
  char* const kbuf0 = lds;                      // K tiles: buffers 0, 1
  char* const vbuf0 = lds + 2 * C::kTileBytes;  // V tiles: buffers 0, 1

  const uint32_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int32_t mt = tile % n_mt;
  const int32_t bh = tile / n_mt;
  const int32_t h = bh % H, b = bh / H;
  int32_t o0, L;
  request_span(off, b, sum_L, o0, L);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int group = wave >> 2;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  // 32-bit element offsets: the API guarantees B*M*H*d and sum_L*H*d < 2^31.
  const int32_t E = H * D;
  const int32_t m_base = mt * C::kBlockM + wave * (C::kMB * 32);
  const bool active = m_base < M;

  // Q^T operand, multiplied by c = scale*log2(e) and re-rounded to bf16, so the
  // MFMA produces exp2 arguments directly.
  bf16x8 qf[C::kMB][C::kKS];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    const int32_t m = m_base + mb * 32 + l32;
    const uint16_t* src = q + (b * M + m) * E + h * D + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < C::kKS; ++ks) {
      const u32x4 u = m < M ? *(const u32x4*)(src + ks * 16) : u32x4{0, 0, 0, 0};
      float f[8];
      Chunk<BF16>::unpack(u, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] *= c;
      qf[mb][ks] = __builtin_bit_cast(bf16x8, Chunk<BF16>::pack(f));
    }
  }

  // Running shift of each beam, folded into S^T by a rank-1 MFMA term
  // S^T += 1 * (-shift): A has 1 in k-slots 0 and 1 of lanes 0-31, B carries
  // -shift of the lane's beam split into a bf16 pair (hi, lo) in those slots,
  // so shifts carry 16 significant bits and are exactly what the MFMA adds.
  const bf16x8 one_a = __builtin_bit_cast(bf16x8, u32x4{hi == 0 ? 0x3f803f80u : 0u, 0u, 0u, 0u});
  float shift[C::kMB];
  bf16x8 bias_b[C::kMB];
  f32x16 o[C::kDB][C::kMB];
  float l_run[C::kMB];
#pragma unroll
  for (int mb = 0; mb < C::kMB; ++mb) {
    shift[mb] = 0.f;
    bias_b[mb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    l_run[mb] = 0.f;
#pragma unroll
    for (int db = 0; db < C::kDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][mb][r] = 0.f;
  }
  f32x16 s[C::kKB][C::kMB];
  bf16x8 pf[C::kKC][C::kMB];

  const int32_t n = (L + C::kBlockN - 1) / C::kBlockN;
  // Element offset of this thread's slot i of the tile starting at token t0.
  auto src_of = [&](int i, int32_t t0) -> int32_t {
    const int sl = i * C::kThreads + threadIdx.x;
    const int key = sl / C::kCPR;
    const int chunk = (sl % C::kCPR) ^ C::swz(key);
    int32_t tok = t0 + key;
    tok = tok < L ? tok : L - 1;
    return (o0 + tok) * E + h * D + chunk * 8;
  };
  // LDS byte address of this wave's 64 slots in K buffer 0 (wave-uniform).
  const uint32_t kb_addr = __builtin_amdgcn_readfirstlane(lds_addr(kbuf0) + wave * 64 * 16);
  const uint32_t vb_addr = kb_addr + 2 * C::kTileBytes;
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): Q fragments are in registers
  if (n > 0) {
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i) load_to_lds(k + src_of(i, 0), kb_addr + i * C::kThreads * 16);
  }
  wait_vmem();   // K(0) is in place
  lds_barrier();

  for (int32_t hp = 0; hp < 2 * n + 2; ++hp) {
    if ((hp & 1) == 0) {
      const int32_t u = hp >> 1;
      if (u + 1 < n) {
#pragma unroll
        for (int i = 0; i < C::kLoads; ++i)
          load_to_lds(k + src_of(i, (u + 1) * C::kBlockN),
                      kb_addr + ((u + 1) & 1) * C::kTileBytes + i * C::kThreads * 16);
      }
      if (u < n) {
#pragma unroll
        for (int i = 0; i < C::kLoads; ++i)
          load_to_lds(v + src_of(i, u * C::kBlockN), vb_addr + (u & 1) * C::kTileBytes + i * C::kThreads * 16);
      }
    }
    const int32_t ph = hp - group;
    if (active && ph >= 0) {
      const int32_t t = ph >> 1;
      if ((ph & 1) == 0) {
        // ---- MFMA phase: O += V(t-1)^T P(t-1)^T, then S(t)^T = K(t) Q^T - shift ----
        __builtin_amdgcn_s_setprio(1);
        if (t >= 1) {
          const char* vb = vbuf0 + ((t - 1) & 1) * C::kTileBytes;
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
          for (int kc = 0; kc < C::kKC; ++kc)
#pragma unroll
            for (int db = 0; db < C::kDB; ++db)
#pragma unroll
              for (int mb = 0; mb < C::kMB; ++mb)
                o[db][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[kc][db], pf[kc][mb], o[db][mb], 0, 0, 0);
        }
        if (t < n) {
          const char* kbp = kbuf0 + (t & 1) * C::kTileBytes;
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
      } else if (t < n) {
        // ---- softmax phase of tile t: S^T already holds exp2(arguments) ----
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
        // Tile maximum per beam: four v_max3 chains over the lane's keys, then
        // the partner lane's half.
        float mx[C::kMB];
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb) {
          float a[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) a[j] = fmaxf(s[0][mb][j], s[0][mb][j + 4]);
#pragma unroll
          for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
            for (int r = (kb == 0 ? 8 : 0); r < 16; r += 8)
#pragma unroll
              for (int j = 0; j < 4; ++j) a[j] = fmaxf(fmaxf(a[j], s[kb][mb][r + j]), s[kb][mb][r + j + 4]);
          mx[mb] = fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
          mx[mb] = fmaxf(mx[mb], __shfl_xor(mx[mb], 32));
        }
        // Lazy shift update: only when some beam of the wave exceeds its shift
        // by more than 8 in exp2 units (so p <= 256), and on the first tile.
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
            l_run[mb] *= alpha;
#pragma unroll
            for (int db = 0; db < C::kDB; ++db)
#pragma unroll
              for (int r = 0; r < 16; ++r) o[db][mb][r] *= alpha;
#pragma unroll
            for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
              for (int r = 0; r < 16; ++r) s[kb][mb][r] -= delta;
            const float nhi = round_to_bf16(-ns);
            const uint32_t nb = pack_bf16x2(nhi, -ns - nhi);   // exact: ns is a bf16 pair sum
            bias_b[mb] = __builtin_bit_cast(bf16x8, u32x4{hi == 0 ? nb : 0u, 0u, 0u, 0u});
          }
        }
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb) {
#pragma unroll
          for (int kb = 0; kb < C::kKB; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kb][mb][r] = fast_exp2(s[kb][mb][r]);
          float part[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) part[j] = s[0][mb][j] + s[0][mb][j + 8];
#pragma unroll
          for (int kb = 1; kb < C::kKB; ++kb)
#pragma unroll
            for (int j = 0; j < 8; ++j) part[j] += s[kb][mb][j] + s[kb][mb][j + 8];
          l_run[mb] += ((part[0] + part[1]) + (part[2] + part[3])) +
                       ((part[4] + part[5]) + (part[6] + part[7]));
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
    if (hp & 1) wait_vmem();   // this wave's share of K(u+1), V(u) has landed
    lds_barrier();
  }

  if (active) {
#pragma unroll
    for (int mb = 0; mb < C::kMB; ++mb) {
      const float l_tot = l_run[mb] + __shfl_xor(l_run[mb], 32);
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
    const int32_t n_mt = (M + CrossTile<DD>::kBlockM - 1) / CrossTile<DD>::kBlockM;          \
    const int64_t grid = (int64_t)B * H * n_mt;                                              \
    hipLaunchKernelGGL(cross_attn_bf16_kernel<DD>, dim3((unsigned)grid),                      \
                       dim3(CrossTile<DD>::kThreads), 0, stream, (const uint16_t*)q,          \
                       (const uint16_t*)enc_k, (const uint16_t*)enc_v, enc_off, (uint16_t*)out, \
                       M, H, sum_L, n_mt, c);                                                 \
    return hipGetLastError();                                                                 \
  }
    if (d == 32) GRACE_X(32)
#undef GRACE_X
#define GRACE_PP(DD)                                                                          \
  {                                                                                           \
    const int32_t n_mt = (M + PingPong<DD>::kBlockM - 1) / PingPong<DD>::kBlockM;            \
    const int64_t grid = (int64_t)B * H * n_mt;                                              \
    hipLaunchKernelGGL(cross_attn_bf16_pp_kernel<DD>, dim3((unsigned)grid),                   \
                       dim3(PingPong<DD>::kThreads), 0, stream, (const uint16_t*)q,           \
                       (const uint16_t*)enc_k, (const uint16_t*)enc_v, enc_off, (uint16_t*)out, \
                       M, H, sum_L, n_mt, c);                                                 \
    return hipGetLastError();                                                                 \
  }
    if (d == 64) GRACE_PP(64)
    if (d == 128) GRACE_PP(128)
#undef GRACE_PP
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
