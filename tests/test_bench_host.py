"""Host-side checks of bench.py: the one-GPU refusal, the algorithmic byte and
flop counts the roofline fractions divide by, and the vector-ALU ceiling."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from oracle import grace_oracle as O  # noqa: E402
from paper_2608_00938_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr or "single MI355X" in p.stderr
    assert p.stdout.strip() == ""


def _tables(wl, parents_by_step):
    """Block tables of every step, built with the oracle's paged rearrangement."""
    tables, prev = [], None
    for t in range(wl.steps):
        prev = O.kv_append_table(prev, parents_by_step[t], wl.B, wl.M, t)
        tables.append(prev)
    return tables


@pytest.mark.parametrize("parents_kind", ["uniform", "zipf"])
def test_unique_ancestor_blocks_match_the_tables(parents_kind):
    """The distinct blocks that self-attention reads at position j of step t are
    the distinct entries of column j of that step's block table."""
    wl = W.custom("uniq", B=3, M=16, H=2, d=32, steps=4, L=8, parents=parents_kind,
                  zipf_s=1.1)
    par = [W.parents(wl, t, seed=5) for t in range(wl.steps)]
    tables = _tables(wl, par)
    for t in range(wl.steps):
        want = [int(np.unique(tables[t][:, j]).size) for j in range(t + 1)]
        assert bench.unique_ancestor_blocks(wl, par, t) == want


def test_algorithmic_counts_follow_the_definitions():
    wl = W.custom("alg", B=2, M=8, H=2, d=32, steps=3, L=16, parents="uniform")
    par = [W.parents(wl, t, seed=1) for t in range(wl.steps)]
    sum_L = wl.B * wl.L
    cross_flops, cross_bytes, append_b, self_b, self_logical, fused_b = bench.algorithmic(
        wl, sum_L, par)
    s, E, R = wl.elem_bytes, wl.E, wl.R
    # cross-attention: two multiply-adds per (beam, key, head, dim), Q/O once, K/V once
    assert cross_flops == sum(2 * 2 * wl.M * wl.L * wl.H * wl.d for _ in range(wl.B))
    assert cross_bytes == (2 * R + 2 * sum_L) * E * s
    tables = _tables(wl, par)
    for t in range(wl.steps):
        tab = R * 4 * (1 if t > 0 else 0) + R * t * 4 + R * (t + 1) * 4
        # append: k_new/v_new read, slab k/v written, parents and the tables
        assert append_b[t] == 4 * R * E * s + tab
        if t == 0:
            assert fused_b[t] == 5 * R * E * s + tab
            continue
        # fused: q, k_new, v_new read, slab k/v and out written, and every
        # distinct ancestor block (k and v) of positions j < t read once
        anc = sum(int(np.unique(tables[t][:, j]).size) for j in range(t))
        assert fused_b[t] == 6 * R * E * s + 2 * E * s * anc + tab
        # logical reads of the split attend: every row reads t+1 k and v blocks
        assert self_logical[t] == 2 * R * E * s + 2 * (t + 1) * R * E * s + R * (t + 1) * 4
        assert self_b[t] <= self_logical[t]


def test_vector_alu_ceiling():
    # 1 + 2 + 0.5 issue units of 4 cycles per 64 scores, 1024 SIMDs at 2.4 GHz
    cycles_per_64 = 4 * (1 + 2 + 0.5)
    assert bench.PEAK_SCORES_G == pytest.approx(1024 * 64 / cycles_per_64 * 2.4)
