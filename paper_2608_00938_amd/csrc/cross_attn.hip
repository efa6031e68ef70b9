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
      uint4 u = m < M ? *(const uint4*)(src + ks * 16) : make_uint4(0, 0, 0, 0);
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

  // Global -> register staging of one K/V tile (slot order = LDS order).
  uint4 kreg[C::kLoads], vreg[C::kLoads];
  auto load_tile = [&](int32_t t0) {
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i) {
      const int s = i * C::kThreads + threadIdx.x;
      const int key = s / C::kCPR;
      const int chunk = (s % C::kCPR) ^ C::swz(key);
      int32_t tok = t0 + key;
      tok = tok < L ? tok : L - 1;
      const int64_t src = (int64_t)(o0 + tok) * E + h * D + chunk * 8;
      kreg[i] = *(const uint4*)(k + src);
      vreg[i] = *(const uint4*)(v + src);
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < C::kLoads; ++i) {
      const int s = i * C::kThreads + threadIdx.x;
      *(uint4*)(k_lds + s * 16) = kreg[i];
      *(uint4*)(v_lds + s * 16) = vreg[i];
    }
  };

  const int32_t n_tiles = (L + C::kBlockN - 1) / C::kBlockN;
  if (n_tiles > 0) load_tile(0);
  for (int32_t t = 0; t < n_tiles; ++t) {
    const int32_t t0 = t * C::kBlockN;
    __syncthreads();
    store_tile();
    __syncthreads();
    if (t + 1 < n_tiles) load_tile(t0 + C::kBlockN);

    // S^T = K Q^T over the tile.
    f32x16 s[C::kKB][C::kMB];
#pragma unroll
    for (int kb = 0; kb < C::kKB; ++kb) {
#pragma unroll
      for (int mb = 0; mb < C::kMB; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][mb][r] = 0.f;
      const int key = kb * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < C::kKS; ++ks) {
        const uint4 u = *(const uint4*)(k_lds + C::slot(key, 2 * ks + hi) * 16);
        const bf16x8 a = __builtin_bit_cast(bf16x8, u);
#pragma unroll
        for (int mb = 0; mb < C::kMB; ++mb)
          s[kb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[mb][ks], s[kb][mb], 0, 0, 0);
      }
    }

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
      const float m_new = fmaxf(m_run[mb], mx);
      const float alpha = fast_exp2((m_run[mb] - m_new) * c);
      m_run[mb] = m_new;
      l_run[mb] *= alpha;
#pragma unroll
      for (int db = 0; db < C::kDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][mb][r] *= alpha;
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
        uint4 u;
        u.x = pack_bf16x2(s[kb][mb][r0 + 0], s[kb][mb][r0 + 1]);
        u.y = pack_bf16x2(s[kb][mb][r0 + 2], s[kb][mb][r0 + 3]);
        u.z = pack_bf16x2(s[kb][mb][r0 + 4], s[kb][mb][r0 + 5]);
        u.w = pack_bf16x2(s[kb][mb][r0 + 6], s[kb][mb][r0 + 7]);
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
          uint2 u;
          u.x = pack_bf16x2(o[db][mb][4 * g + 0] * inv, o[db][mb][4 * g + 1] * inv);
          u.y = pack_bf16x2(o[db][mb][4 * g + 2] * inv, o[db][mb][4 * g + 3] * inv);
          *(uint2*)(dst + db * 32 + 8 * g) = u;
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
