"""Parity of the HIP path (through the C ABI) with the fp64 oracle on the GPU.

Every workload is compared element by element.  On the two largest (64 x 4096
beams and the ragged 128 x 2048), in exactly the launch configuration the
benchmark times, every self-attention output and block-table entry of every
step is checked, and every cross-attention output of the first and the last
step; the oracle then runs request by request in a pool of host threads, and
the steps in between are checked on sampled rows.  Tolerances: max abs error
<= 2e-2 for bf16 inputs (fp32 accumulation), <= 1e-5 for fp32.  Integer work
(block tables) and the pool copy are bit-exact.  Outputs start as NaN, so a
row the kernels never write cannot pass.
"""
import math
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2608_00938_amd import grace as G
from paper_2608_00938_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-5}


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


class Decode:
    """Runs the full decode of a workload on the GPU, one call per entry point per
    step; with ``fused`` the append and the self-attention are one fused call."""

    def __init__(self, wl, seed, device, fused=False):
        self.wl, self.seed, self.fused = wl, seed, fused
        self.inp = W.DecodeInputs(wl, seed, device)
        self.enc_k, self.enc_v = self.inp.enc_kv
        self.off = self.inp.offsets_tensor()
        self.scale = 1.0 / math.sqrt(wl.d)
        self.cache = G.KVCache(wl.B, wl.M, wl.H, wl.d, wl.steps, wl.torch_dtype, device)
        self.parents = [self.inp.parents(t) for t in range(wl.steps)]
        self.steps = []

    def run_step(self, t):
        wl, inp = self.wl, self.inp
        qc = inp.step_tensor("q_cross", t)
        qs = inp.step_tensor("q_self", t)
        kn = inp.step_tensor("k_new", t)
        vn = inp.step_tensor("v_new", t)
        par = None if self.parents[t] is None else torch.from_numpy(self.parents[t]).to(qc.device)
        nan = lambda: torch.full_like(qc, float("nan"))  # noqa: E731
        xc = G.grace_cross_attn(qc, self.enc_k, self.enc_v, self.off, wl.M, self.scale, out=nan())
        if self.fused:
            xs = self.cache.append_attend(t, qs, kn, vn, par, self.scale, out=nan())
        else:
            self.cache.append(t, kn, vn, par)
            xs = self.cache.attend(t, qs, self.scale, out=nan())
        rec = dict(qc=qc, qs=qs, kn=kn, vn=vn, xc=xc, xs=xs,
                   table=self.cache.table(t).clone())
        self.steps.append(rec)
        return rec


def _check_close(got, ref, dtype, what):
    err = float(np.max(np.abs(got - ref))) if got.size else 0.0
    _log(f"  {what}: max|err| = {err:.3e}  max|out| = {float(np.max(np.abs(ref))) if ref.size else 0:.3f}")
    assert np.all(np.isfinite(got)), what
    assert err <= TOL[dtype], f"{what}: {err} > {TOL[dtype]}"


def _full_check(dec):
    """Every output of every step against the oracle."""
    wl = dec.wl
    ek, ev = _np(dec.enc_k), _np(dec.enc_v)
    kp = np.zeros((wl.steps, wl.R, wl.H, wl.d))
    vp = np.zeros_like(kp)
    table = np.zeros((wl.R, wl.steps), dtype=np.int64)
    for t, rec in enumerate(dec.steps):
        ref = oracle.cross_attn(_np(rec["qc"]), ek, ev, dec.inp.offsets, wl.M, dec.scale)
        _check_close(_np(rec["xc"]), ref, wl.dtype, f"cross t={t}")
        kp, vp, tnew = oracle.kv_append(kp, vp, table, dec.parents[t], _np(rec["kn"]),
                                        _np(rec["vn"]), wl.B, wl.M, t)
        table = np.zeros((wl.R, wl.steps), dtype=np.int64)
        table[:, :t + 1] = tnew
        gpu_table = rec["table"].cpu().numpy()[:, :t + 1]
        assert np.array_equal(gpu_table, tnew), f"table t={t}"
        ref = oracle.self_attn_step(_np(rec["qs"]), kp, vp, table, t, dec.scale)
        _check_close(_np(rec["xs"]), ref, wl.dtype, f"self t={t}")
    # the pool holds every step's token bit-exactly
    for t, rec in enumerate(dec.steps):
        assert torch.equal(dec.cache.k_pool[t], rec["kn"]) and torch.equal(dec.cache.v_pool[t], rec["vn"])


def _sample_rows(wl, rng, n=48):
    R, M = wl.R, wl.M
    reqs = sorted({0, wl.B - 1, wl.B // 2, *rng.integers(0, wl.B, size=3).tolist()})
    rows = []
    for b in reqs:
        beams = {0, 1, 31, 32, 63, 64, 255, 256, M - 1, *rng.integers(0, M, size=n // len(reqs)).tolist()}
        rows += [b * M + m for m in sorted(x for x in beams if 0 <= x < M)]
    return np.array(sorted(set(rows)), dtype=np.int64)


def _sampled_check(dec, rng, cross_steps=None):
    """Sampled rows, each computed by the oracle from its request / ancestor
    chain (cross-attention only at ``cross_steps``, default every step)."""
    wl = dec.wl
    rows = _sample_rows(wl, rng)
    dev = dec.enc_k.device
    idx = torch.from_numpy(rows).to(dev)
    for t, rec in enumerate(dec.steps):
        if cross_steps is None or t in cross_steps:
            # cross-attention: one request at a time
            got = _np(rec["xc"].index_select(0, idx))
            ref = np.empty_like(got)
            for b in np.unique(rows // wl.M):
                sel = np.nonzero(rows // wl.M == b)[0]
                o0, o1 = int(dec.inp.offsets[b]), int(dec.inp.offsets[b + 1])
                ref[sel] = oracle.cross_attn_request(_np(rec["qc"].index_select(0, idx[sel])),
                                                     _np(dec.enc_k[o0:o1]), _np(dec.enc_v[o0:o1]),
                                                     dec.scale)
            _check_close(got, ref, wl.dtype, f"cross t={t} ({len(rows)} sampled rows)")
        # block table rows from the parents alone, bit-exact
        tab = oracle.table_rows(rows, t, dec.parents, wl.B, wl.M)
        gpu_tab = rec["table"].index_select(0, idx).cpu().numpy()[:, :t + 1]
        assert np.array_equal(gpu_tab, tab), f"table t={t}"
        # self-attention: gather each sampled row's prefix from the step inputs
        kpre = np.empty((len(rows), t + 1, wl.H, wl.d))
        vpre = np.empty_like(kpre)
        for j in range(t + 1):
            src = torch.from_numpy(tab[:, j] - j * wl.R).to(dev)
            kpre[:, j] = _np(dec.steps[j]["kn"].index_select(0, src))
            vpre[:, j] = _np(dec.steps[j]["vn"].index_select(0, src))
        ref = oracle.self_attn_rows(_np(rec["qs"].index_select(0, idx)), kpre, vpre, dec.scale)
        _check_close(_np(rec["xs"].index_select(0, idx)), ref, wl.dtype,
                     f"self t={t} ({len(rows)} sampled rows)")
        assert torch.equal(dec.cache.k_pool[t], rec["kn"]) and torch.equal(dec.cache.v_pool[t], rec["vn"])


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
@pytest.mark.parametrize("name", ["tiny_fp32", "bf16_b8_m256", "bf16_b32_m1024"])
def test_workload_full_parity(gpu, name, fused):
    wl = W.WORKLOADS[name]
    _log(f"[parity full] {name} seed=0 fused={fused}")
    dec = Decode(wl, 0, gpu, fused)
    for t in range(wl.steps):
        dec.run_step(t)
    torch.cuda.synchronize()
    _full_check(dec)


def _pool():
    """Host threads for the oracle (numpy releases the GIL in its matrix products
    and ufuncs), one BLAS thread each."""
    return ThreadPoolExecutor(max_workers=max(1, min(16, os.cpu_count() or 1)))


def _blas_single_thread():
    from threadpoolctl import threadpool_limits
    return threadpool_limits(limits=1)


def _cross_full_check(dec, t, chunk=1024):
    """Every cross-attention row of step t against the oracle, one (request,
    beam chunk) per oracle call."""
    wl = dec.wl
    qh = dec.steps[t]["qc"].float().cpu().numpy()
    got = dec.steps[t]["xc"].float().cpu().numpy()
    ek, ev = dec.enc_k.float().cpu().numpy(), dec.enc_v.float().cpu().numpy()
    off = dec.inp.offsets

    def one(b, m0):
        rows = slice(b * wl.M + m0, b * wl.M + min(wl.M, m0 + chunk))
        ref = oracle.cross_attn_request(qh[rows], ek[off[b]:off[b + 1]], ev[off[b]:off[b + 1]],
                                        dec.scale)
        g = got[rows].astype(np.float64)
        return (float(np.max(np.abs(g - ref))), bool(np.all(np.isfinite(g))),
                float(np.max(np.abs(ref))))

    with _blas_single_thread(), _pool() as ex:
        res = list(ex.map(lambda a: one(*a), [(b, m0) for b in range(wl.B)
                                              for m0 in range(0, wl.M, chunk)]))
    err = max(r[0] for r in res)
    _log(f"  cross t={t} all {wl.R} rows: max|err| = {err:.3e}  max|out| = "
         f"{max(r[2] for r in res):.3f}")
    assert all(r[1] for r in res), f"cross t={t}: non-finite output"
    assert err <= TOL[wl.dtype], f"cross t={t}: {err} > {TOL[wl.dtype]}"


def _self_full_check(dec, chunk=32768):
    """Every block-table entry (bit-exact) and every self-attention row of every
    step against the oracle: the table from the oracle's update rule over the
    whole batch, each row's prefix gathered from the step inputs through it."""
    wl = dec.wl
    dev = dec.enc_k.device
    table = None
    for t, rec in enumerate(dec.steps):
        table = oracle.kv_append_table(table, dec.parents[t], wl.B, wl.M, t)
        gpu_table = rec["table"].cpu().numpy()[:, :t + 1]
        assert np.array_equal(gpu_table, table), f"table t={t}"
        # each prefix position's rows, by slab: block id j*R + r is row r of step j
        src = [torch.from_numpy(np.ascontiguousarray(table[:, j] - j * wl.R)).to(dev)
               for j in range(t + 1)]
        jobs = []
        with _blas_single_thread(), _pool() as ex:
            for r0 in range(0, wl.R, chunk):
                sl = slice(r0, min(wl.R, r0 + chunk))
                q = rec["qs"][sl].float().cpu().numpy()
                kpre = np.stack([dec.steps[j]["kn"].index_select(0, src[j][sl]).float().cpu().numpy()
                                 for j in range(t + 1)], axis=1)
                vpre = np.stack([dec.steps[j]["vn"].index_select(0, src[j][sl]).float().cpu().numpy()
                                 for j in range(t + 1)], axis=1)
                g = rec["xs"][sl].float().cpu().numpy()

                def one(q=q, kpre=kpre, vpre=vpre, g=g):
                    ref = oracle.self_attn_rows(q, kpre, vpre, dec.scale)
                    g = g.astype(np.float64)
                    return (float(np.max(np.abs(g - ref))), bool(np.all(np.isfinite(g))),
                            float(np.max(np.abs(ref))))
                jobs.append(ex.submit(one))
            res = [j.result() for j in jobs]
        err = max(r[0] for r in res)
        _log(f"  self t={t} all {wl.R} rows: max|err| = {err:.3e}  max|out| = "
             f"{max(r[2] for r in res):.3f}")
        assert all(r[1] for r in res), f"self t={t}: non-finite output"
        assert err <= TOL[wl.dtype], f"self t={t}: {err} > {TOL[wl.dtype]}"
        assert torch.equal(dec.cache.k_pool[t], rec["kn"]) and torch.equal(dec.cache.v_pool[t], rec["vn"])


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
@pytest.mark.parametrize("name", ["bf16_b64_m4096", "bf16_ragged_b128_m2048"])
def test_large_workload_parity(gpu, name, fused):
    """Full size, the benchmark's launch configuration.  Self-attention and the
    tables: every row of every step.  Cross-attention (the same kernel on both
    self-attention paths): every row of step 0 on the split run and of the last
    step on the fused run; the other steps on sampled rows."""
    wl = W.WORKLOADS[name]
    _log(f"[parity large] {name} seed=0 fused={fused}")
    dec = Decode(wl, 0, gpu, fused)
    for t in range(wl.steps):
        dec.run_step(t)
    torch.cuda.synchronize()
    assert int(dec.cache.err_flag.item()) == 0
    _self_full_check(dec)
    t_full = wl.steps - 1 if fused else 0
    _cross_full_check(dec, t_full)
    _sampled_check(dec, np.random.default_rng(0), cross_steps=[t for t in range(wl.steps)
                                                               if t != t_full])
    assert torch.equal(dec.steps[0]["xs"], dec.steps[0]["vn"])


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
def test_paper_shape_sampled_parity(gpu, fused):
    """The paper's microbenchmark shape (16 x 1024 beams, 128 encoder tokens,
    16 heads x 128) that the benchmark times beside the paper's own figures."""
    wl = W.PAPER_SHAPE
    _log(f"[parity sampled] {wl.name} seed=0 fused={fused}")
    dec = Decode(wl, 0, gpu, fused)
    for t in range(wl.steps):
        dec.run_step(t)
    torch.cuda.synchronize()
    assert int(dec.cache.err_flag.item()) == 0
    _sampled_check(dec, np.random.default_rng(1))
    for rec in dec.steps:
        assert bool(torch.isfinite(rec["xc"]).all()) and bool(torch.isfinite(rec["xs"]).all())


EDGE = [
    # ragged tails: beams not a multiple of the 256-beam tile, keys not of the 64-token tile
    dict(dtype="bf16", B=3, M=300, H=3, d=64, steps=3, L_lo=1, L_hi=130),
    dict(dtype="bf16", B=2, M=17, H=1, d=32, steps=4, L_lo=60, L_hi=70),
    dict(dtype="bf16", B=2, M=513, H=2, d=128, steps=5, L_lo=63, L_hi=200),
    dict(dtype="f32", B=3, M=70, H=2, d=64, steps=3, L_lo=1, L_hi=100),
    dict(dtype="f32", B=1, M=5, H=3, d=128, steps=2, L=33),
    dict(dtype="f32", B=2, M=9, H=1, d=32, steps=8, L=1),
    dict(dtype="bf16", B=1, M=1, H=1, d=64, steps=8, L=1),
    dict(dtype="bf16", B=4, M=64, H=2, d=64, steps=4, L=64, parents="zipf", zipf_s=1.5),
    # head counts that are multiples of 8 take the XCD-interleaved work order;
    # request counts that are not multiples of 8 exercise its rotation
    dict(dtype="bf16", B=3, M=70, H=8, d=64, steps=2, L_lo=5, L_hi=150),
    dict(dtype="bf16", B=11, M=33, H=16, d=32, steps=2, L_lo=1, L_hi=90),
    dict(dtype="bf16", B=9, M=200, H=8, d=128, steps=2, L_lo=30, L_hi=260),
    # d = 64 with more than 256 beams: several 256-beam tiles per (request, head),
    # the last one partly past M, ragged tails, single-tile requests
    dict(dtype="bf16", B=3, M=700, H=8, d=64, steps=2, L_lo=1, L_hi=200),
    dict(dtype="bf16", B=2, M=1536, H=2, d=64, steps=2, L_lo=60, L_hi=400, parents="zipf", zipf_s=1.1),
]


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
@pytest.mark.parametrize("i", range(len(EDGE)))
def test_edge_shapes_full_parity(gpu, i, fused):
    kw = dict(EDGE[i])
    kw.setdefault("parents", "uniform")
    wl = W.custom(name=f"edge{i}", **kw)
    _log(f"[parity edge] {wl} fused={fused}")
    dec = Decode(wl, 1 + i, gpu, fused)
    for t in range(wl.steps):
        dec.run_step(t)
    torch.cuda.synchronize()
    _full_check(dec)


def _random_shape(i):
    """Seeded random small workload: any dtype, head dim, ragged or fixed encoder
    lengths (including tails shorter than a key tile), beam counts off the tile
    sizes, uniform or Zipf parents."""
    rng = np.random.default_rng(1000 + i)
    dtype = "f32" if i % 4 == 3 else "bf16"
    d = int(rng.choice([32, 64, 128]))
    kw = dict(dtype=dtype, B=int(rng.integers(1, 5)), M=int(rng.integers(1, 700)),
              H=int(rng.integers(1, 4)), d=d, steps=int(rng.integers(1, 9)))
    if rng.random() < 0.5:
        kw.update(L_lo=int(rng.integers(1, 40)), L_hi=int(rng.integers(40, 300)))
    else:
        kw.update(L=int(rng.integers(1, 300)))
    if rng.random() < 0.5:
        kw.update(parents="zipf", zipf_s=float(rng.uniform(0.8, 1.6)))
    else:
        kw.update(parents="uniform")
    return kw


@pytest.mark.parametrize("fused", [False, True], ids=["split", "fused"])
@pytest.mark.parametrize("i", range(10))
def test_random_shapes_full_parity(gpu, i, fused):
    kw = _random_shape(i)
    wl = W.custom(name=f"random{i}", **kw)
    _log(f"[parity random] {wl} fused={fused}")
    dec = Decode(wl, 50 + i, gpu, fused)
    for t in range(wl.steps):
        dec.run_step(t)
    torch.cuda.synchronize()
    _full_check(dec)


def test_first_step_is_v_new_bitwise(gpu):
    for dtype in ("bf16", "f32"):
        wl = W.custom(dtype=dtype, B=2, M=40, H=3, d=64, steps=2, L=8)
        dec = Decode(wl, 5, gpu)
        rec = dec.run_step(0)
        torch.cuda.synchronize()
        assert torch.equal(rec["xs"], rec["vn"]), dtype


def test_single_token_encoder_returns_v(gpu):
    """L_b = 1: every beam of the request reads that token's value."""
    for dtype in ("bf16", "f32"):
        wl = W.custom(dtype=dtype, B=3, M=100, H=2, d=128, steps=1, L=1)
        dec = Decode(wl, 6, gpu)
        rec = dec.run_step(0)
        torch.cuda.synchronize()
        want = dec.enc_v.repeat_interleave(wl.M, dim=0)
        assert torch.equal(rec["xc"], want), dtype


def test_empty_request_gives_zero_rows(gpu):
    wl = W.custom(dtype="bf16", B=3, M=20, H=2, d=64, steps=1, L=10)
    inp = W.DecodeInputs(wl, 0, gpu)
    ek, ev = inp.enc_kv
    off = torch.tensor([0, 10, 10, 20], dtype=torch.int32, device=gpu)   # request 1 is empty
    q = inp.step_tensor("q_cross", 0)
    out = G.grace_cross_attn(q, ek, ev, off, wl.M)
    torch.cuda.synchronize()
    assert bool((out[20:40] == 0).all())
    ref = oracle.cross_attn(_np(q), _np(ek), _np(ev), [0, 10, 10, 20], wl.M, 1 / 8)
    assert np.max(np.abs(_np(out) - ref)) <= TOL["bf16"]


def test_aliased_slab_append_matches_copy(gpu):
    """k_new/v_new written straight into the pool slab: the copy is skipped, results equal."""
    wl = W.custom(dtype="bf16", B=2, M=48, H=4, d=64, steps=3, L=16)
    a = Decode(wl, 7, gpu)
    for t in range(wl.steps):
        a.run_step(t)
    inp = a.inp
    cache = G.KVCache(wl.B, wl.M, wl.H, wl.d, wl.steps, wl.torch_dtype, gpu)
    for t in range(wl.steps):
        ks, vs = cache.slab(t)
        ks.copy_(inp.step_tensor("k_new", t))
        vs.copy_(inp.step_tensor("v_new", t))
        par = None if t == 0 else torch.from_numpy(a.parents[t]).to(gpu)
        cache.append(t, ks, vs, par)
        out = cache.attend(t, inp.step_tensor("q_self", t))
        torch.cuda.synchronize()
        assert torch.equal(out, a.steps[t]["xs"])
        assert torch.equal(cache.table(t)[:, :t + 1], a.steps[t]["table"][:, :t + 1])


def test_out_of_range_parent_sets_flag(gpu):
    wl = W.custom(dtype="bf16", B=2, M=8, H=1, d=32, steps=2, L=4)
    dec = Decode(wl, 8, gpu)
    dec.run_step(0)
    assert int(dec.cache.err_flag.item()) == 0
    dec.parents[1] = dec.parents[1].copy()
    dec.parents[1][3] = wl.M + 5
    dec.run_step(1)
    torch.cuda.synchronize()
    assert int(dec.cache.err_flag.item()) == 1
    # the bad row was clamped to the last beam of its request; the others are exact
    tab = dec.steps[1]["table"].cpu().numpy()
    assert tab[3, 0] == wl.M - 1


def test_deterministic_and_relabelling_invariant(gpu):
    wl = W.custom(dtype="bf16", B=2, M=96, H=2, d=64, steps=4, L=100, parents="zipf", zipf_s=1.2)
    a = Decode(wl, 9, gpu)
    b = Decode(wl, 9, gpu)
    for t in range(wl.steps):
        ra, rb = a.run_step(t), b.run_step(t)
        torch.cuda.synchronize()
        assert torch.equal(ra["xc"], rb["xc"]) and torch.equal(ra["xs"], rb["xs"])
    # permute physical blocks, remap the table: self-attention output is unchanged
    t = wl.steps - 1
    nblk = wl.steps * wl.R
    pi = torch.randperm(nblk, generator=torch.Generator().manual_seed(0)).to(gpu)
    kflat = a.cache.k_pool.reshape(nblk, wl.H, wl.d)
    vflat = a.cache.v_pool.reshape(nblk, wl.H, wl.d)
    kperm = torch.empty_like(kflat)
    vperm = torch.empty_like(vflat)
    kperm[pi] = kflat
    vperm[pi] = vflat
    table = a.steps[t]["table"].clone()
    table[:, :t + 1] = pi[table[:, :t + 1].long()].int()
    out = G.grace_self_attn_step(a.steps[t]["qs"], kperm.reshape(a.cache.k_pool.shape),
                                 vperm.reshape(a.cache.v_pool.shape), table, wl.B, wl.M, t)
    torch.cuda.synchronize()
    assert torch.equal(out, a.steps[t]["xs"])


def test_empty_batch_is_noop(gpu):
    q = torch.empty((0, 2, 64), dtype=torch.bfloat16, device=gpu)
    kv = torch.zeros((4, 2, 64), dtype=torch.bfloat16, device=gpu)
    off = torch.zeros(1, dtype=torch.int32, device=gpu)
    out = G.grace_cross_attn(q, kv, kv, off, 0)
    assert out.shape == (0, 2, 64)


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("bf16", 128), ("f32", 32), ("bf16", 32)])
def test_fused_equals_split_bitwise(gpu, dtype, d):
    """The fused pass reads the same bits and runs the same arithmetic as append
    followed by attend: outputs, tables and pools are identical."""
    wl = W.custom(dtype=dtype, B=3, M=37, H=5, d=d, steps=6, L=20, parents="zipf", zipf_s=1.3)
    a, b = Decode(wl, 11, gpu, fused=False), Decode(wl, 11, gpu, fused=True)
    for t in range(wl.steps):
        ra, rb = a.run_step(t), b.run_step(t)
        torch.cuda.synchronize()
        assert torch.equal(ra["xs"], rb["xs"]), f"out t={t}"
        assert torch.equal(ra["table"][:, :t + 1], rb["table"][:, :t + 1]), f"table t={t}"
    assert torch.equal(a.cache.k_pool, b.cache.k_pool) and torch.equal(a.cache.v_pool, b.cache.v_pool)


def test_fused_aliased_slab(gpu):
    """Fused call with k_new/v_new already in their slab: no copy, same results."""
    wl = W.custom(dtype="bf16", B=2, M=48, H=4, d=64, steps=3, L=16)
    a = Decode(wl, 7, gpu)
    for t in range(wl.steps):
        a.run_step(t)
    cache = G.KVCache(wl.B, wl.M, wl.H, wl.d, wl.steps, wl.torch_dtype, gpu)
    for t in range(wl.steps):
        ks, vs = cache.slab(t)
        ks.copy_(a.inp.step_tensor("k_new", t))
        vs.copy_(a.inp.step_tensor("v_new", t))
        par = None if t == 0 else torch.from_numpy(a.parents[t]).to(gpu)
        out = cache.append_attend(t, a.inp.step_tensor("q_self", t), ks, vs, par)
        torch.cuda.synchronize()
        assert torch.equal(out, a.steps[t]["xs"])
        assert torch.equal(cache.table(t)[:, :t + 1], a.steps[t]["table"][:, :t + 1])


def test_fused_out_of_range_parent_sets_flag(gpu):
    wl = W.custom(dtype="bf16", B=2, M=8, H=2, d=64, steps=2, L=4)   # rows of 256 B
    dec = Decode(wl, 8, gpu, fused=True)
    dec.run_step(0)
    torch.cuda.synchronize()
    assert int(dec.cache.err_flag.item()) == 0
    dec.parents[1] = dec.parents[1].copy()
    dec.parents[1][3] = -2
    dec.parents[1][12] = wl.M
    dec.run_step(1)
    torch.cuda.synchronize()
    assert int(dec.cache.err_flag.item()) == 1
    tab = dec.steps[1]["table"].cpu().numpy()
    assert tab[3, 0] == 0 and tab[12, 0] == 2 * wl.M - 1


def test_fused_wave_uniform_rows(gpu):
    """Rows of exactly 1 KiB and 2 KiB take the wave-uniform (scalar table read) path."""
    for H, d in ((8, 64), (8, 128)):
        wl = W.custom(dtype="bf16", B=2, M=33, H=H, d=d, steps=5, L=8, parents="zipf", zipf_s=1.1)
        dec = Decode(wl, 12, gpu, fused=True)
        for t in range(wl.steps):
            dec.run_step(t)
        torch.cuda.synchronize()
        _full_check(dec)


def _extreme_case(gpu, kind, B=3, M=96, H=2, d=64, L=200, seed=13):
    g = torch.Generator().manual_seed(seed)
    if kind == "huge":
        # each beam's query is 12x one of its request's keys: that key scores
        # ~138 in exp2 units, ~90 above the rest, so row sums are ~2^138
        k = torch.randn((B * L, H, d), generator=g)
        pick = torch.randint(0, L, (B * M,), generator=g) + (torch.arange(B * M) // M) * L
        q = 12 * k[pick]
    else:
        # keys anti-aligned with every query: all scores ~ -80 (log2 units ~ -115)
        u = torch.sign(torch.randn((B, 1, H, d), generator=g))
        q = (u + 0.05 * torch.randn((B, M, H, d), generator=g)).reshape(B * M, H, d)
        k = (-10 * u + 0.05 * torch.randn((B, L, H, d), generator=g)).reshape(B * L, H, d)
    v = torch.randn((B * L, H, d), generator=g)
    q, k, v = (x.to(torch.bfloat16) for x in (q, k, v))
    off = torch.arange(0, B * L + 1, L, dtype=torch.int32)
    return q, k, v, off


@pytest.mark.parametrize("kind,M", [("huge", 96), ("tiny", 96), ("huge", 520), ("tiny", 520)])
def test_cross_attn_extreme_scores_take_the_safe_pass(gpu, kind, M):
    """Scores whose exp2 sums leave [2^-100, 2^64] fail the fast pass's check;
    the workgroup's safe pass (exponent shift) still matches the fp64 oracle
    (M = 520: three 256-beam tiles, the last one mostly past M)."""
    q, k, v, off = _extreme_case(gpu, kind, M=M)
    M = q.shape[0] // (off.numel() - 1)
    _log(f"[cross extreme] {kind}")
    out = G.grace_cross_attn(q.to(gpu), k.to(gpu), v.to(gpu), off.to(gpu), M)
    torch.cuda.synchronize()
    ref = oracle.cross_attn(_np(q), _np(k), _np(v), off.numpy(), M, 1 / 8)
    _check_close(_np(out), ref, "bf16", f"cross {kind}")


def _wide_case(seed, B, M, H, d, L_lo, L_hi, std):
    """Q and K ~ N(0, std^2), V ~ N(0, 1), bf16, ragged encoder lengths."""
    g = torch.Generator().manual_seed(seed)
    lens = torch.randint(L_lo, L_hi + 1, (B,), generator=g)
    off = torch.cat([torch.zeros(1, dtype=torch.int64), lens.cumsum(0)]).to(torch.int32)
    n = int(off[-1])
    q = std * torch.randn((B * M, H, d), generator=g)
    k = std * torch.randn((n, H, d), generator=g)
    v = torch.randn((n, H, d), generator=g)
    return tuple(x.to(torch.bfloat16) for x in (q, k, v)) + (off,)


WIDE = [(d, std, 300) for d in (32, 64, 128) for std in (2.0, 3.0)] + \
    [(64, 4.0, 300), (128, 4.0, 300)] + [(64, std, 600) for std in (2.0, 3.0, 4.0)]


@pytest.mark.parametrize("d,std,M", WIDE, ids=[f"d{d}_std{s:g}_m{m}" for d, s, m in WIDE])
def test_cross_attn_wide_scores(gpu, d, std, M):
    """Un-normalised activations: with Q/K spread 2-4 the scores span tens of
    exp2 units, so any rounding of the scaled scores ahead of the softmax
    shows up in the weights.  Ragged lengths (tails shorter than a key tile)
    and a beam count off the tile; at spread 4 most rows also overflow the
    fast pass and take the safe one."""
    q, k, v, off = _wide_case(200 + d + int(10 * std) + M, B=3, M=M, H=2, d=d, L_lo=1, L_hi=300,
                              std=std)
    _log(f"[cross wide] d={d} std={std} M={M} L={np.diff(off.numpy()).tolist()}")
    out = G.grace_cross_attn(q.to(gpu), k.to(gpu), v.to(gpu), off.to(gpu), M)
    torch.cuda.synchronize()
    ref = oracle.cross_attn(_np(q), _np(k), _np(v), off.numpy(), M, 1 / math.sqrt(d))
    _check_close(_np(out), ref, "bf16", f"cross wide d={d} std={std}")


@pytest.mark.parametrize("d,M", [(32, 160), (64, 160), (128, 160), (64, 600)])
def test_cross_attn_near_tied_large_scores(gpu, d, M):
    """Scores of ~100-200 exp2 units (row sums far past 2^64: the safe pass)
    that are nearly tied: every query is ~12 u and every key is u plus a large
    component orthogonal to u (spread 8) plus a little noise along it, so the
    scores differ only by fractions of a unit while the keys themselves differ
    a lot.  A relative rounding of the scaled query of 2^-9 moves the scores by
    several tenths of a unit here; the weights must not move."""
    B, H, L = 2, 2, 200
    g = torch.Generator().manual_seed(300 + d + M)
    u = torch.sign(torch.randn((B, 1, H, d), generator=g))
    w = 8.0 * torch.randn((B, L, H, d), generator=g)
    w = w - (w * u).sum(-1, keepdim=True) / d * u
    q = (12 * u + 0.1 * torch.randn((B, M, H, d), generator=g)).reshape(B * M, H, d)
    k = (u + w + 0.05 * torch.randn((B, L, H, d), generator=g)).reshape(B * L, H, d)
    v = torch.randn((B * L, H, d), generator=g)
    q, k, v = (x.to(torch.bfloat16) for x in (q, k, v))
    off = torch.arange(0, B * L + 1, L, dtype=torch.int32)
    _log(f"[cross near-tie] d={d} M={M}")
    out = G.grace_cross_attn(q.to(gpu), k.to(gpu), v.to(gpu), off.to(gpu), M)
    torch.cuda.synchronize()
    ref, probs = oracle.cross_attn(_np(q), _np(k), _np(v), off.numpy(), M, 1 / math.sqrt(d),
                                   return_probs=True)
    # the case is what it claims: no key of a row holds most of the weight
    top = max(float(np.median(p.max(axis=-1))) for p in probs)
    _log(f"  median largest weight {top:.3f}")
    assert top < 0.2
    _check_close(_np(out), ref, "bf16", f"cross near-tie d={d}")


def test_decode_resumes_from_snapshot(gpu):
    """The pools and block tables are caller-owned, so a decode can be
    checkpointed: copying them after step 1 into a fresh cache and resuming
    there gives bit-identical outputs and tables for the remaining steps."""
    wl = W.custom(dtype="bf16", B=2, M=96, H=2, d=64, steps=5, L=40, parents="zipf", zipf_s=1.2)
    ref = Decode(wl, 15, gpu, fused=True)
    for t in range(wl.steps):
        ref.run_step(t)
    run = Decode(wl, 15, gpu, fused=True)
    for t in range(2):
        run.run_step(t)
    torch.cuda.synchronize()
    snap = [x.clone() for x in (run.cache.k_pool, run.cache.v_pool, *run.cache.tables)]
    resumed = Decode(wl, 15, gpu, fused=True)
    c = resumed.cache
    for dst, src in zip((c.k_pool, c.v_pool, *c.tables), snap):
        dst.copy_(src)
    resumed.steps = list(run.steps)
    for t in range(2, wl.steps):
        got = resumed.run_step(t)
        torch.cuda.synchronize()
        want = ref.steps[t]
        assert torch.equal(got["xs"], want["xs"]) and torch.equal(got["xc"], want["xc"]), t
        assert torch.equal(got["table"][:, :t + 1], want["table"][:, :t + 1]), t
    assert torch.equal(c.k_pool, ref.cache.k_pool) and torch.equal(c.v_pool, ref.cache.v_pool)
