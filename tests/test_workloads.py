"""The seeded input generators: determinism, ranges and distribution shape."""
import numpy as np
import torch

from paper_2608_00938_amd import workloads as W


def test_named_workloads_shapes():
    w = W.WORKLOADS
    assert (w["tiny_fp32"].B, w["tiny_fp32"].M, w["tiny_fp32"].L, w["tiny_fp32"].H,
            w["tiny_fp32"].d, w["tiny_fp32"].steps, w["tiny_fp32"].dtype) == (1, 16, 32, 2, 32, 3, "f32")
    big = w["bf16_b64_m4096"]
    assert (big.B, big.M, big.L, big.H, big.d, big.steps, big.R, big.E) == (64, 4096, 1024, 16, 64, 4,
                                                                          262144, 1024)
    rag = w["bf16_ragged_b128_m2048"]
    assert rag.ragged and (rag.L_lo, rag.L_hi, rag.d, rag.steps) == (64, 2048, 128, 5)


def test_determinism_and_independence_of_step_draws():
    wl = W.WORKLOADS["bf16_b8_m256"].with_(B=2, M=8)
    a = W.DecodeInputs(wl, seed=3)
    b = W.DecodeInputs(wl, seed=3)
    assert torch.equal(a.step_tensor("q_self", 2), b.step_tensor("q_self", 2))
    # a step regenerates on its own, whatever was generated before it
    _ = b.step_tensor("k_new", 1)
    assert torch.equal(a.step_tensor("v_new", 3), b.step_tensor("v_new", 3))
    assert not torch.equal(a.step_tensor("q_self", 1), a.step_tensor("q_self", 2))
    assert not torch.equal(a.step_tensor("q_self", 1), W.DecodeInputs(wl, seed=4).step_tensor("q_self", 1))
    assert np.array_equal(a.parents(2), b.parents(2))
    assert a.parents(0) is None
    assert a.step_tensor("q_cross", 0).dtype == torch.bfloat16


def test_value_scale_of_tiny_workload():
    wl = W.WORKLOADS["tiny_fp32"]
    x = W.normal((4096, 64), 0, "enc_k", 0, wl).double()
    assert abs(x.std().item() - 1 / np.sqrt(32)) < 0.01
    assert x.dtype == torch.float64


def test_uniform_parents_range():
    wl = W.WORKLOADS["bf16_b32_m1024"]
    p = W.parents(wl, 1, seed=0)
    assert p.dtype == np.int32 and p.shape == (wl.R,)
    assert p.min() >= 0 and p.max() < wl.M
    # roughly uniform: every decile of beams is hit about equally
    h = np.bincount(p * 10 // wl.M, minlength=10) / p.size
    assert np.all(np.abs(h - 0.1) < 0.01)


def test_zipf_parents_concentration_and_permutation():
    wl = W.WORKLOADS["bf16_b64_m4096"].with_(B=4)
    p = W.parents(wl, 2, seed=0).reshape(wl.B, wl.M)
    assert p.min() >= 0 and p.max() < wl.M
    w = np.arange(1, wl.M + 1, dtype=np.float64) ** -1.1
    p1 = w[0] / w.sum()
    for b in range(wl.B):
        counts = np.bincount(p[b], minlength=wl.M)
        top = counts.max() / wl.M
        assert abs(top - p1) < 5 * np.sqrt(p1 / wl.M)   # the rank-1 beam's share
    # the most popular beam is a different one per request (a fresh permutation)
    tops = {int(np.bincount(p[b], minlength=wl.M).argmax()) for b in range(wl.B)}
    assert len(tops) > 1


def test_ragged_lengths_and_offsets():
    wl = W.WORKLOADS["bf16_ragged_b128_m2048"]
    L = W.enc_lengths(wl, seed=0)
    off = W.enc_offsets(wl, seed=0)
    assert L.min() >= 64 and L.max() <= 2048
    assert off[0] == 0 and np.all(np.diff(off) == L) and off.dtype == np.int32
    assert abs(L.mean() - 1056) < 120
