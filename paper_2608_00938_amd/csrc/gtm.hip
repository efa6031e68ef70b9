// Decode-time constraint filter (CD + GTM) and trie step (GRACE, Sec. 4, Sec. 5.4,
// App. A) for gfx950.
//
// gtm_mask: 16 lanes per beam row.  The lanes split the beam's child-entry
//   range (CSR), test the bitmask matcher first (stopping at the first word
//   that misses a user bit), then the Bloom matcher (stopping at the first
//   location it contains), and OR the surviving tokens into the row's filter
//   words in LDS, which they then store whole.  The request-side matchers are
//   shared by the beams of a request and stay in cache.
// trie_advance: one lane per new beam: binary search of its token among the
//   parent node's child tokens (ascending within a node's range).
#include "common.hpp"
#include "kernels.hpp"

namespace grace {

constexpr int kGtmThreads = 256;
constexpr int kGtmMaxWords = 128;   // vocab <= 4096
constexpr int kMaxBm = 8, kMaxBl = 4;

struct GtmDev {
  const int32_t* off;
  const int32_t* child;
  const int16_t* tok;
  const int32_t* bmi;
  const int32_t* bli;
  const uint64_t* bmt;
  const uint64_t* blt;
  int32_t nodes, entries, V, wbm, wbl, bm_rows, bl_rows;
};

struct UserDev {
  const uint64_t* bm;
  const uint64_t* bl;
  const int32_t* nloc;
  int32_t lmax;
};

// A beam row is handled by kLanesPerBeam consecutive lanes (four beams per
// wave): at the deeper trie levels a node has a handful of children, and more
// beams per wave keep more of the dependent lookups (node -> range -> entries
// -> matcher rows) in flight.
constexpr int kLanesPerBeam = 16;
constexpr int kBeamsPerBlock = kGtmThreads / kLanesPerBeam;

__global__ void __launch_bounds__(kGtmThreads)
gtm_mask_kernel(GtmDev ix, UserDev us, const int32_t* __restrict__ node_ids, int32_t R, int32_t M,
                uint32_t* __restrict__ mask, int32_t* __restrict__ err_flag) {
  __shared__ uint32_t words[kBeamsPerBlock][kGtmMaxWords];
  const int sub = threadIdx.x % kLanesPerBeam, slot = threadIdx.x / kLanesPerBeam;
  const int32_t r = (int32_t)blockIdx.x * kBeamsPerBlock + slot;
  const int W = (ix.V + 31) >> 5;
  for (int i = sub; i < W; i += kLanesPerBeam) words[slot][i] = 0u;
  __syncthreads();
  bool bad = false;
  if (r < R) {
    const int32_t node = node_ids[r];
    if (node >= 0 && node < ix.nodes) {
      const int32_t b = r / M;
      uint64_t u[kMaxBm];
#pragma unroll
      for (int j = 0; j < kMaxBm; ++j) u[j] = j < ix.wbm ? us.bm[(int64_t)b * ix.wbm + j] : 0ull;
      int32_t nloc = us.nloc[b];
      nloc = nloc < 0 ? 0 : (nloc > us.lmax ? us.lmax : nloc);
      const uint64_t* locs = us.bl + (int64_t)b * us.lmax * ix.wbl;
      int32_t e0 = ix.off[node], e1 = ix.off[node + 1];
      e0 = e0 < 0 ? 0 : (e0 > ix.entries ? ix.entries : e0);
      e1 = e1 < e0 ? e0 : (e1 > ix.entries ? ix.entries : e1);
      for (int32_t e = e0 + sub; e < e1; e += kLanesPerBeam) {
        const int32_t v = ix.tok[e], bi = ix.bmi[e], li = ix.bli[e];
        if (v < 0 || v >= ix.V || bi < 0 || bi >= ix.bm_rows || li < 0 || li >= ix.bl_rows) {
          bad = true;
          continue;
        }
        // bitmask: every user bit must be in the node matcher
        const uint64_t* m = ix.bmt + (int64_t)bi * ix.wbm;
        bool ok = true;
#pragma unroll
        for (int j = 0; j < kMaxBm; ++j) {
          if (j < ix.wbm && ok && (m[j] & u[j]) != u[j]) ok = false;
        }
        if (!ok) continue;
        // Bloom: some user location's filter must be contained in the matcher
        const uint64_t* g = ix.blt + (int64_t)li * ix.wbl;
        uint64_t gm[kMaxBl];
#pragma unroll
        for (int j = 0; j < kMaxBl; ++j) gm[j] = j < ix.wbl ? g[j] : ~0ull;
        bool found = false;
        for (int32_t q = 0; q < nloc && !found; ++q) {
          const uint64_t* l = locs + (int64_t)q * ix.wbl;
          bool in = true;
#pragma unroll
          for (int j = 0; j < kMaxBl; ++j) {
            if (j < ix.wbl && in) {
              const uint64_t x = l[j];
              in = (x & gm[j]) == x;
            }
          }
          found = in;
        }
        if (found) atomicOr(&words[slot][v >> 5], 1u << (v & 31));
      }
    } else if (node >= ix.nodes) {
      bad = true;   // negative ids are dead beams; ids past the trie are errors
    }
  }
  __syncthreads();
  if (r < R)
    for (int i = sub; i < W; i += kLanesPerBeam) mask[(int64_t)r * W + i] = words[slot][i];
  if (bad && err_flag) *err_flag = 1;
}

__global__ void __launch_bounds__(kGtmThreads)
trie_advance_kernel(GtmDev ix, const int32_t* __restrict__ node_prev,
                    const int32_t* __restrict__ parents, const int32_t* __restrict__ tokens,
                    int32_t n, int32_t M_prev, int32_t k, int32_t* __restrict__ node_next,
                    int32_t* __restrict__ err_flag) {
  const int32_t i = (int32_t)blockIdx.x * kGtmThreads + (int32_t)threadIdx.x;
  if (i >= n) return;
  const int32_t b = i / k, p = parents[i], v = tokens[i];
  int32_t out = -1;
  if (p < 0 || p >= M_prev) {
    if (err_flag) *err_flag = 1;
  } else {
    const int32_t node = node_prev[(int64_t)b * M_prev + p];
    if (node >= ix.nodes) {
      if (err_flag) *err_flag = 1;
    } else if (node >= 0) {
      int32_t lo = ix.off[node], end = ix.off[node + 1];
      lo = lo < 0 ? 0 : (lo > ix.entries ? ix.entries : lo);
      end = end < lo ? lo : (end > ix.entries ? ix.entries : end);
      int32_t hi = end;
      while (lo < hi) {   // first entry with token >= v
        const int32_t mid = (lo + hi) >> 1;
        if (ix.tok[mid] < v) lo = mid + 1;
        else hi = mid;
      }
      if (lo < end && ix.tok[lo] == v) out = ix.child[lo];
    }
  }
  node_next[i] = out;
}

static GtmDev to_dev(const grace_gtm_index& x) {
  return GtmDev{x.node_offsets, x.child_nodes, x.tokens, x.bitmask_index, x.bloom_index,
                x.bitmask_table, x.bloom_table, x.num_nodes, x.num_entries, x.vocab,
                x.bitmask_words, x.bloom_words, x.bitmask_rows, x.bloom_rows};
}

hipError_t launch_gtm_mask(const grace_gtm_index& index, const grace_gtm_user& user,
                           const int32_t* node_ids, int32_t R, int32_t M, uint32_t* mask,
                           int32_t* err_flag, hipStream_t stream) {
  const UserDev us{user.bitmask, user.bloom, user.num_locations, user.max_locations};
  const int64_t blocks = ((int64_t)R + kBeamsPerBlock - 1) / kBeamsPerBlock;
  hipLaunchKernelGGL(gtm_mask_kernel, dim3((unsigned)blocks), dim3(kGtmThreads), 0, stream,
                     to_dev(index), us, node_ids, R, M, mask, err_flag);
  return hipGetLastError();
}

hipError_t launch_trie_advance(const grace_gtm_index& index, const int32_t* node_prev,
                               const int32_t* parents, const int32_t* tokens, int32_t B,
                               int32_t M_prev, int32_t k, int32_t* node_next, int32_t* err_flag,
                               hipStream_t stream) {
  const int32_t n = B * k;
  hipLaunchKernelGGL(trie_advance_kernel, dim3((unsigned)((n + kGtmThreads - 1) / kGtmThreads)),
                     dim3(kGtmThreads), 0, stream, to_dev(index), node_prev, parents, tokens, n,
                     M_prev, k, node_next, err_flag);
  return hipGetLastError();
}

}  // namespace grace
