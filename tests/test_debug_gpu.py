"""The debug build (libgrace_debug.so, -DGRACE_DEBUG) on the GPU.

Clean runs: whole decodes (cross-attention, split and fused append + attend,
ragged requests, every head dim) through the debug build leave every
device-check counter at zero, and give the release build's outputs bit for bit
(the checks change no arithmetic).  Bad inputs that the kernels clamp (request
offsets out of order, block ids past the pool, parents out of range) are
counted by the debug build.  Every input here stays inside what the kernels'
own clamps handle.
"""
import math
import os
import sys

import numpy as np
import pytest
import torch

from paper_2608_00938_amd import grace as G
from paper_2608_00938_amd import workloads as W

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not os.path.exists(G._DEBUG_LIB_PATH),
                                 reason="debug build not present")]

KINDS = ("offsets", "parents", "block ids", "rows")


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _decode(wl, seed, dev, fused):
    inp = W.DecodeInputs(wl, seed, dev)
    ek, ev = inp.enc_kv
    off = inp.offsets_tensor()
    cache = G.KVCache(wl.B, wl.M, wl.H, wl.d, wl.steps, wl.torch_dtype, dev)
    outs = []
    for t in range(wl.steps):
        qc, qs = inp.step_tensor("q_cross", t), inp.step_tensor("q_self", t)
        kn, vn = inp.step_tensor("k_new", t), inp.step_tensor("v_new", t)
        par = inp.parents(t)
        par = None if par is None else torch.from_numpy(par).to(dev)
        xc = G.grace_cross_attn(qc, ek, ev, off, wl.M)
        if fused:
            xs = cache.append_attend(t, qs, kn, vn, par)
        else:
            cache.append(t, kn, vn, par)
            xs = cache.attend(t, qs)
        outs += [xc, xs, cache.table(t)[:, :t + 1].clone()]
    torch.cuda.synchronize()
    return outs


CASES = [
    ("bf16_b8_m256", None),
    ("ragged_d64", dict(dtype="bf16", B=3, M=300, H=8, d=64, steps=3, L_lo=1, L_hi=130)),
    ("ragged_d128", dict(dtype="bf16", B=2, M=513, H=2, d=128, steps=4, L_lo=63, L_hi=200,
                         parents="zipf", zipf_s=1.2)),
    ("ragged_d32", dict(dtype="bf16", B=5, M=70, H=3, d=32, steps=4, L_lo=1, L_hi=90)),
    ("f32_d128", dict(dtype="f32", B=2, M=40, H=2, d=128, steps=3, L_lo=5, L_hi=60)),
]


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_debug_build_clean_decode(gpu, monkeypatch, name, kw, fused):
    wl = W.WORKLOADS[name] if kw is None else W.custom(name=name, **kw)
    _log(f"[debug build] {wl.name} fused={fused}")
    release = _decode(wl, 3, gpu, fused)
    dbg = G.debug_library()
    G.grace_debug_counts(dbg)   # clear what earlier calls left
    monkeypatch.setattr(G, "_lib", dbg)
    checked = _decode(wl, 3, gpu, fused)
    counts = G.grace_debug_counts(dbg)
    _log(f"  counts {dict(zip(KINDS, counts))}")
    assert counts == [0] * G.GRACE_DEBUG_KINDS
    for i, (a, b) in enumerate(zip(release, checked)):
        assert torch.equal(a, b), i


def test_debug_build_counts_clamped_inputs(gpu, monkeypatch):
    dbg = G.debug_library()
    G.grace_debug_counts(dbg)
    monkeypatch.setattr(G, "_lib", dbg)
    B, M, H, d = 3, 64, 2, 64
    g = torch.Generator().manual_seed(5)
    q = torch.randn((B * M, H, d), generator=g).to(torch.bfloat16).to(gpu)
    kv = torch.randn((30, H, d), generator=g).to(torch.bfloat16).to(gpu)
    # request 1's offsets are out of order (20 > 10): clamped to an empty request
    off = torch.tensor([0, 20, 10, 30], dtype=torch.int32, device=gpu)
    G.grace_cross_attn(q, kv, kv, off, M)
    counts = G.grace_debug_counts(dbg)
    _log(f"[debug counts] offsets out of order: {counts}")
    assert counts[0] > 0 and counts[1:] == [0] * 7

    # a block id past the pool in one row's table: clamped to the last block
    wl = W.custom(dtype="bf16", B=2, M=16, H=2, d=64, steps=2, L=4)
    inp = W.DecodeInputs(wl, 9, gpu)
    cache = G.KVCache(wl.B, wl.M, wl.H, wl.d, wl.steps, wl.torch_dtype, gpu)
    cache.append(0, inp.step_tensor("k_new", 0), inp.step_tensor("v_new", 0))
    par = torch.from_numpy(inp.parents(1)).to(gpu)
    cache.append(1, inp.step_tensor("k_new", 1), inp.step_tensor("v_new", 1), par)
    G.grace_debug_counts(dbg)
    table = cache.table(1).clone()
    table[3, 0] = wl.steps * wl.R + 7
    G.grace_self_attn_step(inp.step_tensor("q_self", 1), cache.k_pool, cache.v_pool, table, wl.B,
                           wl.M, 1)
    counts = G.grace_debug_counts(dbg)
    _log(f"[debug counts] block id past the pool: {counts}")
    assert counts[2] > 0 and counts[0] == counts[1] == counts[3] == 0

    # a parent out of range in the fused step: clamped, err_flag set, counted
    bad = par.clone()
    bad[5] = wl.M + 3
    cache.append_attend(1, inp.step_tensor("q_self", 1), inp.step_tensor("k_new", 1),
                        inp.step_tensor("v_new", 1), bad)
    counts = G.grace_debug_counts(dbg)
    _log(f"[debug counts] parent out of range: {counts}")
    assert counts[1] > 0 and counts[3] == 0
    assert int(cache.err_flag.item()) == 1
