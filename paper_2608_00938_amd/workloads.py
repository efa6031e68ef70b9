"""Seeded synthetic inputs for one wide-beam decode step's attention.

This module holds shapes, random draws and parent-index distributions only: none
of the attention arithmetic lives here, so it can feed both the HIP path and the
CPU oracle without coupling them.

The production inputs of the paper (encoder outputs of its InterFormer-style
encoder, the beam-search parents chosen under constrained decoding) are not
public; these draws stand in for them with the paper's structure: request-major
beam rows (App. B), one encoder K/V per request shared by its beams (Sec. 3.2),
short Semantic-ID prefixes (at most ``steps`` tokens, Sec. 3.2) and parent
indices local to a request (Sec. 3.3, Sec. 5.3).

Value recipe: every Q/K/V tensor is N(0, 1) drawn in float32 by torch's
generator on the target device, multiplied by ``value_scale`` and rounded
(round-to-nearest-even) to the workload's dtype.  Each tensor has its own seed
derived from ``(seed, tensor tag, step)`` so any step regenerates on its own.
Parents: uniform on ``[0, M)`` or a finite Zipf law over ranks ``1..M``
(``P(k) ~ k**-s``) mapped to beams through a fresh random permutation per
(request, step).  Ragged encoder lengths: integer uniform on an inclusive range.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np
import torch

F32 = "f32"
BF16 = "bf16"
TORCH_DTYPES = {F32: torch.float32, BF16: torch.bfloat16}

_TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16}

# Tensor tags used in the per-tensor seed.
_TAG = {"enc_k": 1, "enc_v": 2, "q_cross": 3, "q_self": 4, "k_new": 5, "v_new": 6,
        "parents": 7, "lengths": 8, "perm": 9, "logits": 10, "prev_scores": 11, "mask": 12,
        "cand": 13, "dyn_parents": 14, "sids": 15, "ads": 16, "users": 17, "beam_nodes": 18}

# Beam step shapes of the paper's model (Sec. 3.2, Sec. 3.3): SID-token
# vocabulary and the dynamic per-step beam widths (M_1, ..., M_4).
VOCAB = 512
DYN_WIDTHS = (1, 512, 1024, 1024)


@dataclass(frozen=True)
class Workload:
    """Shape and distribution of one synthetic decode workload."""
    name: str
    dtype: str          # "f32" or "bf16": input, output and cache element type
    B: int              # requests
    M: int              # beams per request (fixed width at every step)
    H: int              # heads
    d: int              # head dim
    steps: int          # decode steps = Semantic-ID length; also the cache's T_max
    L: int = 0          # encoder length of every request (0 when ragged)
    L_lo: int = 0       # ragged encoder length range, inclusive
    L_hi: int = 0
    parents: str = "uniform"   # "uniform" or "zipf"
    zipf_s: float = 0.0
    value_scale: float = 1.0   # multiplier applied to the N(0,1) draws

    @property
    def R(self) -> int:
        return self.B * self.M

    @property
    def E(self) -> int:
        return self.H * self.d

    @property
    def ragged(self) -> bool:
        return self.L == 0

    @property
    def torch_dtype(self) -> torch.dtype:
        return _TORCH_DTYPE[self.dtype]

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == F32 else 2

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workload shapes the measurements and parity tests use, named by
# what they are.  Sizes: requests x beams, encoder length, heads x head dim.
WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", F32, B=1, M=16, H=2, d=32, steps=3, L=32,
                          parents="uniform", value_scale=1.0 / math.sqrt(32.0)),
    "bf16_b8_m256": Workload("bf16_b8_m256", BF16, B=8, M=256, H=8, d=64, steps=4, L=256,
                             parents="uniform"),
    "bf16_b32_m1024": Workload("bf16_b32_m1024", BF16, B=32, M=1024, H=8, d=64, steps=4,
                               L=512, parents="uniform"),
    "bf16_b64_m4096": Workload("bf16_b64_m4096", BF16, B=64, M=4096, H=16, d=64, steps=4,
                               L=1024, parents="zipf", zipf_s=1.1),
    "bf16_ragged_b128_m2048": Workload("bf16_ragged_b128_m2048", BF16, B=128, M=2048, H=8,
                                       d=128, steps=5, L_lo=64, L_hi=2048,
                                       parents="zipf", zipf_s=1.2),
}

# The paper's own microbenchmark shape (16 requests x 1024 beams, 128 encoder
# tokens, 16 heads x 128, prefixes of t+1 tokens for t = 0..3); measured beside
# the five workloads for comparison with the paper's GH200 timings.
PAPER_SHAPE = Workload("bf16_paper_b16_m1024", BF16, B=16, M=1024, H=16, d=128, steps=4, L=128,
                       parents="uniform")


def custom(name: str = "custom", **kw) -> Workload:
    """A workload of arbitrary shape (tests use it for edge cases)."""
    kw.setdefault("dtype", BF16)
    return Workload(name=name, **kw)


def _seed_int(seed: int, tag: str, step: int = 0, extra: int = 0) -> int:
    ss = np.random.SeedSequence([int(seed), _TAG[tag], int(step), int(extra)])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64(0x7FFF_FFFF_FFFF_FFFF))


def _rng(seed: int, tag: str, step: int = 0, extra: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(_seed_int(seed, tag, step, extra)))


def enc_lengths(wl: Workload, seed: int = 0) -> np.ndarray:
    """Encoder length of each request, int64 [B]."""
    if not wl.ragged:
        return np.full(wl.B, wl.L, dtype=np.int64)
    return _rng(seed, "lengths").integers(wl.L_lo, wl.L_hi + 1, size=wl.B).astype(np.int64)


def enc_offsets(wl: Workload, seed: int = 0) -> np.ndarray:
    """Packed offsets int32 [B+1] of the requests' encoder tokens."""
    off = np.zeros(wl.B + 1, dtype=np.int64)
    np.cumsum(enc_lengths(wl, seed), out=off[1:])
    assert off[-1] < 2**31
    return off.astype(np.int32)


def parents(wl: Workload, step: int, seed: int = 0) -> np.ndarray | None:
    """Request-local parent beam of every row at ``step``, int32 [B*M]; None at step 0."""
    if step == 0:
        return None
    rng = _rng(seed, "parents", step)
    if wl.parents == "uniform":
        return rng.integers(0, wl.M, size=wl.R).astype(np.int32)
    if wl.parents == "zipf":
        w = np.arange(1, wl.M + 1, dtype=np.float64) ** (-wl.zipf_s)
        ranks = rng.choice(wl.M, size=(wl.B, wl.M), p=w / w.sum())
        out = np.empty((wl.B, wl.M), dtype=np.int32)
        prng = _rng(seed, "perm", step)
        for b in range(wl.B):
            out[b] = prng.permutation(wl.M)[ranks[b]]
        return out.reshape(-1)
    raise ValueError(f"unknown parent distribution {wl.parents!r}")


def normal(shape, seed: int, tag: str, step: int, wl: Workload,
           device: str | torch.device = "cpu") -> torch.Tensor:
    """N(0,1) * value_scale draw of ``shape`` on ``device``, rounded to wl's dtype."""
    g = torch.Generator(device=device)
    g.manual_seed(_seed_int(seed, tag, step))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if wl.value_scale != 1.0:
        x.mul_(wl.value_scale)
    return x.to(wl.torch_dtype)


class DecodeInputs:
    """Lazily generated inputs of one workload on one device.

    ``enc_k``/``enc_v`` are packed ``[sum L, H, d]``; per step the cross- and
    self-attention queries and the new token's k/v are ``[B*M, H, d]``.
    """

    def __init__(self, wl: Workload, seed: int = 0, device: str | torch.device = "cpu"):
        self.wl, self.seed, self.device = wl, seed, torch.device(device)
        self.lengths = enc_lengths(wl, seed)
        self.offsets = enc_offsets(wl, seed)
        self.sum_L = int(self.offsets[-1])
        self._enc = None

    @property
    def enc_kv(self) -> tuple[torch.Tensor, torch.Tensor]:
        if self._enc is None:
            shp = (self.sum_L, self.wl.H, self.wl.d)
            self._enc = (normal(shp, self.seed, "enc_k", 0, self.wl, self.device),
                         normal(shp, self.seed, "enc_v", 0, self.wl, self.device))
        return self._enc

    def offsets_tensor(self) -> torch.Tensor:
        return torch.from_numpy(self.offsets).to(self.device)

    def step_tensor(self, tag: str, step: int) -> torch.Tensor:
        shp = (self.wl.R, self.wl.H, self.wl.d)
        return normal(shp, self.seed, tag, step, self.wl, self.device)

    def parents(self, step: int) -> np.ndarray | None:
        return parents(self.wl, step, self.seed)


# ---------------------------------------------------------------------------
# Beam-step inputs (score update and top-k).  Plain seeded draws: logits
# N(0, 3^2) (rounded to bf16 when asked), accumulated prefix log-probabilities
# -Gamma(step + 1, 3), and a filter that keeps each token with probability
# ``keep`` (packed 32 tokens per uint32 word, bit v % 32 of word v // 32).
# ---------------------------------------------------------------------------

def beam_logits(seed: int, step: int, R: int, V: int, dtype: str = BF16,
                device: str | torch.device = "cpu") -> torch.Tensor:
    x = torch.from_numpy(_rng(seed, "logits", step).standard_normal((R, V)).astype(np.float32) * 3)
    return x.to(TORCH_DTYPES[dtype]).to(device)


def beam_prev_scores(seed: int, step: int, R: int) -> np.ndarray:
    return (-_rng(seed, "prev_scores", step).gamma(step + 1.0, 3.0, size=R)).astype(np.float32)


def beam_mask(seed: int, step: int, R: int, V: int, keep: float = 0.6) -> np.ndarray:
    """uint32 [R, ceil(V/32)] filter words; bits past V are zero."""
    allowed = _rng(seed, "mask", step).random((R, V)) < keep
    words = (V + 31) // 32
    pad = np.zeros((R, words * 32), dtype=bool)
    pad[:, :V] = allowed
    w = pad.reshape(R, words, 32).astype(np.uint64) << np.arange(32, dtype=np.uint64)
    return w.sum(axis=2).astype(np.uint32)


def candidate_array(seed: int, B: int, M: int, V: int, kind: str = "normal") -> np.ndarray:
    """fp32 [B*M, V] candidate scores with a chosen structure (top-k test inputs).

    normal: -Gamma + N draws (distinct values); ties: values on a 0.25 grid;
    equal: every value equal; sparse: -inf except ~1% finite; wide: values
    spread over a range of ~4000; special: normal with NaN, +-0, +-inf mixed in.
    """
    rng = _rng(seed, "cand", 0, _KINDS.index(kind))
    shape = (B * M, V)
    if kind == "normal":
        x = -rng.gamma(3.0, 3.0, size=(B * M, 1)) + rng.standard_normal(shape) * 3
    elif kind == "ties":
        x = np.round((-rng.gamma(3.0, 3.0, size=(B * M, 1)) + rng.standard_normal(shape) * 3) * 4) / 4
    elif kind == "equal":
        x = np.full(shape, -7.5)
    elif kind == "sparse":
        x = np.where(rng.random(shape) < 0.01, rng.standard_normal(shape), -np.inf)
    elif kind == "wide":
        x = rng.uniform(-4000.0, 0.0, size=shape)
    elif kind == "special":
        x = rng.standard_normal(shape) * 3
        u = rng.random(shape)
        x = np.where(u < 0.02, np.nan, x)
        x = np.where((u >= 0.02) & (u < 0.05), 0.0, x)
        x = np.where((u >= 0.05) & (u < 0.08), -0.0, x)
        x = np.where((u >= 0.08) & (u < 0.10), -np.inf, x)
        x = np.where((u >= 0.10) & (u < 0.101), np.inf, x)
    else:
        raise ValueError(kind)
    return x.astype(np.float32)


_KINDS = ["normal", "ties", "equal", "sparse", "wide", "special"]


def dyn_parents(seed: int, step: int, B: int, M_prev: int, M_cur: int) -> np.ndarray:
    """Request-local parents int32 [B*M_cur], uniform in [0, M_prev)."""
    return _rng(seed, "dyn_parents", step).integers(0, M_prev, size=B * M_cur).astype(np.int32)


# ---------------------------------------------------------------------------
# Synthetic CD+GTM index (Sec. 4, App. A) and request attributes.  The paper's
# 30M-SID index and its targeting data are not public; this builds an index of
# the same form: a SID trie in CSR form whose child entries point to
# deduplicated bitmask (W_bm = 7 words) and Bloom (W_bl = 4 words) matcher rows,
# each node matcher the OR of the matchers of the ads below it.
#   SIDs: length 4 over |V| = 512; level l draws a Zipf(1.0) rank over C_l
#         choices (512, 128, 64, 32), mapped to a token by a per-prefix
#         bijection, so prefixes cluster as semantic IDs do.
#   Ads per SID: 1 + Geometric(0.7), capped at 11 (p50 1, p90 2 as in the
#         paper's index summary).
#   Bitmask: attributes of 200, 8, 4, 64 and 32 values (country, age, gender,
#         language, device) packed into 7 words; an ad allows every value of an
#         attribute with probability 0.5, else 1-5 random values.
#   Bloom: 256 bits, 3 hash bits per location id out of 10000; an ad targets
#         any location (all ones) with probability 0.4, else 1-8 locations.
#   Users: one value per attribute; 1-64 locations (most requests 1-8).
# ---------------------------------------------------------------------------
GTM_ATTRS = (200, 8, 4, 64, 32)
GTM_W_BM, GTM_W_BL, GTM_BLOOM_BITS, GTM_LOCS = 7, 4, 256, 10000


def _bloom_bits(loc: np.ndarray) -> np.ndarray:
    """Three bit positions in [0, 256) per location id (multiplicative hashing)."""
    loc = loc.astype(np.uint64)
    mults = np.array([0x9E3779B97F4A7C15, 0xC2B2AE3D27D4EB4F, 0x165667B19E3779F9], dtype=np.uint64)
    h = (loc[..., None] * mults) >> np.uint64(56)
    return h.astype(np.int64)


def _set_bits(words: np.ndarray, rows: np.ndarray, bits: np.ndarray):
    np.bitwise_or.at(words, (rows, bits // 64), np.left_shift(np.uint64(1), (bits % 64).astype(np.uint64)))


def gtm_index(seed: int, n_sids: int, V: int = 512, sid_len: int = 4) -> dict:
    rng = _rng(seed, "sids")
    choices = [V, 128, 64, 32][:sid_len]
    sids = np.empty((n_sids, sid_len), dtype=np.int64)
    key = np.zeros(n_sids, dtype=np.uint64)
    for l, C in enumerate(choices):
        w = 1.0 / np.arange(1, C + 1)
        rank = rng.choice(C, size=n_sids, p=w / w.sum()).astype(np.uint64)
        mult = (key * np.uint64(0x9E3779B97F4A7C15)) >> np.uint64(40)
        sids[:, l] = ((mult + rank * np.uint64(2 * (l + 1) + 1)) % np.uint64(V)).astype(np.int64)
        key = key * np.uint64(V + 1) + sids[:, l].astype(np.uint64) + np.uint64(1)
    sids = np.unique(sids, axis=0)
    n = sids.shape[0]
    # ads and their matchers
    arng = _rng(seed, "ads")
    n_ads = np.minimum(1 + arng.geometric(0.7, size=n) - 1, 11)
    ad_sid = np.repeat(np.arange(n), n_ads)
    A = ad_sid.shape[0]
    bm = np.zeros((A, GTM_W_BM), dtype=np.uint64)
    base = 0
    for size in GTM_ATTRS:
        any_all = arng.random(A) < 0.5
        rows = np.nonzero(any_all)[0]
        for v in range(size):
            _set_bits(bm, rows, np.full(rows.shape, base + v))
        rows = np.nonzero(~any_all)[0]
        cnt = arng.integers(1, 6, size=rows.shape[0])
        rr = np.repeat(rows, cnt)
        _set_bits(bm, rr, base + arng.integers(0, size, size=rr.shape[0]))
        base += size
    bl = np.zeros((A, GTM_W_BL), dtype=np.uint64)
    any_loc = arng.random(A) < 0.4
    bl[any_loc] = np.uint64(0xFFFFFFFFFFFFFFFF)
    rows = np.nonzero(~any_loc)[0]
    cnt = arng.integers(1, 9, size=rows.shape[0])
    rr = np.repeat(rows, cnt)
    bits = _bloom_bits(arng.integers(0, GTM_LOCS, size=rr.shape[0]))
    for j in range(3):
        _set_bits(bl, rr, bits[:, j])
    # trie levels: node ids in level order, root = 0
    level_ids, level_first = [], [1]
    inv_prev = np.zeros(n, dtype=np.int64)          # level-0 prefix id of every SID (the root)
    parent_of, token_of = [], []
    for l in range(sid_len):
        keys = np.concatenate([inv_prev[:, None], sids[:, l:l + 1]], axis=1)
        uniq, inv = np.unique(keys, axis=0, return_inverse=True)
        inv = inv.reshape(-1)
        first = level_first[-1]
        parent_of.append(uniq[:, 0] + (0 if l == 0 else level_first[-2]))
        token_of.append(uniq[:, 1])
        level_ids.append(first + inv)
        level_first.append(first + uniq.shape[0])
        inv_prev = inv
    num_nodes = level_first[-1]
    # node matchers: full SIDs OR their ads, then each level ORs its children
    node_bm = np.zeros((num_nodes, GTM_W_BM), dtype=np.uint64)
    node_bl = np.zeros((num_nodes, GTM_W_BL), dtype=np.uint64)
    leaf = level_ids[-1][ad_sid]
    np.bitwise_or.at(node_bm, leaf, bm)
    np.bitwise_or.at(node_bl, leaf, bl)
    for l in range(sid_len - 1, 0, -1):
        kids = np.arange(level_first[l], level_first[l + 1])
        np.bitwise_or.at(node_bm, parent_of[l], node_bm[kids])
        np.bitwise_or.at(node_bl, parent_of[l], node_bl[kids])
    # CSR child entries, ordered by (parent, token)
    child = np.arange(1, num_nodes)
    par = np.concatenate(parent_of)
    tok = np.concatenate(token_of)
    order = np.lexsort((tok, par))
    child, par, tok = child[order], par[order], tok[order]
    offsets = np.zeros(num_nodes + 1, dtype=np.int64)
    np.add.at(offsets, par + 1, 1)
    offsets = np.cumsum(offsets)
    bm_tab, bm_idx = np.unique(node_bm[child], axis=0, return_inverse=True)
    bl_tab, bl_idx = np.unique(node_bl[child], axis=0, return_inverse=True)
    return {"vocab": V, "sid_len": sid_len, "num_nodes": num_nodes, "level_first": level_first,
            "node_offsets": offsets.astype(np.int32), "child_nodes": child.astype(np.int32),
            "tokens": tok.astype(np.int16), "bitmask_index": bm_idx.reshape(-1).astype(np.int32),
            "bloom_index": bl_idx.reshape(-1).astype(np.int32),
            "bitmask_table": np.ascontiguousarray(bm_tab), "bloom_table": np.ascontiguousarray(bl_tab),
            "sids": sids, "ad_sid": ad_sid, "ad_bitmask": bm, "ad_bloom": bl}


def gtm_users(seed: int, B: int, L_max: int = 64) -> dict:
    rng = _rng(seed, "users")
    u = np.zeros((B, GTM_W_BM), dtype=np.uint64)
    base = 0
    for size in GTM_ATTRS:
        _set_bits(u, np.arange(B), base + rng.integers(0, size, size=B))
        base += size
    few = rng.integers(1, min(8, L_max) + 1, size=B)
    many = rng.integers(min(9, L_max), L_max + 1, size=B)
    n_loc = np.where(rng.random(B) < 0.9, few, many)
    bloom = np.zeros((B, L_max, GTM_W_BL), dtype=np.uint64)
    for b in range(B):
        bits = _bloom_bits(rng.integers(0, GTM_LOCS, size=int(n_loc[b])))
        for j in range(3):
            _set_bits(bloom[b], np.arange(int(n_loc[b])), bits[:, j])
    return {"bitmask": u, "bloom": bloom, "n_loc": n_loc.astype(np.int32), "L_max": L_max}


def gtm_beam_nodes(seed: int, index: dict, B: int, M: int, level: int) -> np.ndarray:
    """Node id of every beam (row b*M + m): a level-``level`` trie node (root at 0)."""
    lf = index["level_first"]
    if level == 0:
        return np.zeros(B * M, dtype=np.int32)
    lo, hi = lf[level - 1], lf[level]
    return _rng(seed, "beam_nodes", level).integers(lo, hi, size=B * M).astype(np.int32)
