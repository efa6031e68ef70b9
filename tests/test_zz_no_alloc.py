"""grace_beam_step_noalloc through the C ABI: the same parents, tokens and
scores, bit for bit, as grace_beam_step with a caller workspace, on two calls in
a row (the second smaller, so it runs over the first call's leftovers in the
scratch array), with the outputs given so that the call allocates nothing."""
import sys

import numpy as np
import pytest
import torch

from paper_2608_00938_amd import grace as G
from paper_2608_00938_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _case(dev, seed, B, M, V, k, dtype="bf16", keep=0.6):
    R = B * M
    logits = W.beam_logits(seed, 1, R, V, dtype, dev)
    prev = torch.from_numpy(W.beam_prev_scores(seed, 1, R)).to(dev)
    mask = torch.from_numpy(W.beam_mask(seed, 1, R, V, keep=keep).view(np.int32)).to(dev)
    return logits, prev, mask


def _outs(dev, B, k):
    return (torch.full((B, k), -7, dtype=torch.int32, device=dev),
            torch.full((B, k), -7, dtype=torch.int32, device=dev),
            torch.full((B, k), float("nan"), dtype=torch.float32, device=dev))


def test_noalloc_matches_workspace_entry_point_twice(gpu):
    # the first call fills most of the array (64 requests x 4096 beams x 512
    # tokens, the benchmark's beam step); the second is smaller
    shapes = [(64, 4096, 512, 4096, "bf16"), (3, 200, 100, 300, "f32")]
    for i, (B, M, V, k, dtype) in enumerate(shapes):
        _log(f"[noalloc] call {i}: B={B} M={M} V={V} k={k} {dtype}")
        logits, prev, mask = _case(gpu, 40 + i, B, M, V, k, dtype)
        want = G.grace_beam_step(logits, prev, B, M, k, mask=mask)
        p, t, s = _outs(gpu, B, k)
        torch.cuda.synchronize()
        G.grace_beam_step_noalloc(logits, prev, B, M, k, mask=mask, parents=p, tokens=t, scores=s)
        torch.cuda.synchronize()
        assert torch.equal(p, want[0]), "parents"
        assert torch.equal(t, want[1]), "tokens"
        assert torch.equal(s.view(torch.int32), want[2].view(torch.int32)), "scores (bitwise)"


def test_noalloc_rejects_oversized_step(gpu):
    """A step whose workspace exceeds the scratch array is refused before any
    launch (the C entry point on real device buffers, sizes too large)."""
    B, M, V, k = 128, 4096, 512, 16
    assert G.grace_beam_step_workspace_bytes(B, M, V) > G.BEAM_STEP_NOALLOC_MAX_BYTES
    buf = torch.zeros((1 << 20,), dtype=torch.int32, device=gpu)
    base = buf.data_ptr()
    st = G.library().grace_beam_step_noalloc(base, base + (1 << 18), None, B, M, V, k,
                                             G.GRACE_BF16, base + (1 << 19), base + (5 << 18),
                                             base + (6 << 18), torch.cuda.current_stream().cuda_stream)
    assert st == G.GRACE_ERR_SHAPE
    assert int(buf.abs().sum()) == 0
