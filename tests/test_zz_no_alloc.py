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


def test_noalloc_step_replays_in_a_graph(gpu):
    """The no-alloc step recorded in a HIP graph (the callers it is for): every
    replay, with other eager library work and host synchronisation in between,
    gives the workspace entry point's outputs bit for bit."""
    B, M, V, k = 4, 256, 512, 300
    logits, prev, mask = _case(gpu, 60, B, M, V, k)
    want = G.grace_beam_step(logits, prev, B, M, k, mask=mask)
    p, t, s = _outs(gpu, B, k)
    # one eager call first: the scratch array's address is looked up outside capture
    G.grace_beam_step_noalloc(logits, prev, B, M, k, mask=mask, parents=p, tokens=t, scores=s)
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    assert torch.equal(p, want[0]) and torch.equal(t, want[1])
    graph = G.capture(lambda: G.grace_beam_step_noalloc(logits, prev, B, M, k, mask=mask, parents=p,
                                                        tokens=t, scores=s), stream)
    other_logits, other_prev, _ = _case(gpu, 61, 2, 64, 100, 50, "f32")
    for rep in range(3):
        p.fill_(-7)
        t.fill_(-7)
        s.fill_(float("nan"))
        G.grace_beam_step_noalloc(other_logits, other_prev, 2, 64, 50)   # overwrites the scratch array
        torch.cuda.synchronize()
        graph.launch(stream)
        stream.synchronize()
        assert torch.equal(p, want[0]) and torch.equal(t, want[1]), rep
        assert torch.equal(s.view(torch.int32), want[2].view(torch.int32)), rep
        _log(f"  graph replay {rep}: identical")
    graph.destroy()
