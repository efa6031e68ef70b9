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

_TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16}

# Tensor tags used in the per-tensor seed.
_TAG = {"enc_k": 1, "enc_v": 2, "q_cross": 3, "q_self": 4, "k_new": 5, "v_new": 6,
        "parents": 7, "lengths": 8, "perm": 9}


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
