"""The C ABI on the host: the library loads, exports every symbol the header
declares, and rejects bad arguments before any launch (no GPU needed: every
call here returns from the host-side checks)."""
import ctypes
import math
import os
import re

import pytest

from paper_2608_00938_amd import grace as G

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "grace.h")

lib_missing = not os.path.exists(G._LIB_PATH)
pytestmark = pytest.mark.skipif(lib_missing, reason="libgrace.so not built")

P = ctypes.c_void_p(0x10000)    # never dereferenced: every call below fails a host check
P2 = ctypes.c_void_p(0x20000)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(grace_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("grace_cross_attn", "grace_kv_append", "grace_self_attn_step",
              "grace_self_attn_step_fused", "grace_self_attn_step_fused_dyn",
              "grace_beam_scores", "grace_beam_topk", "grace_beam_topk_max_k",
              "grace_beam_topk_workspace_bytes", "grace_beam_step", "grace_beam_step_workspace_bytes",
              "grace_gtm_mask", "grace_trie_advance"):
        assert n in names


def test_debug_counts_in_the_release_build():
    """The release build has no device-check counters: zeros and UNSUPPORTED."""
    lib = G.library()
    buf = (ctypes.c_uint32 * 8)(*range(1, 9))
    assert lib.grace_debug_counts(buf) == G.GRACE_ERR_UNSUPPORTED
    assert list(buf) == [0] * 8
    assert lib.grace_debug_counts(None) == G.GRACE_ERR_NULL


def test_debug_build_exports_the_same_symbols():
    if not os.path.exists(G._DEBUG_LIB_PATH):
        pytest.skip("debug build not present")
    dbg = G.debug_library()
    for name in declared_functions():
        assert hasattr(dbg, name), name


def test_library_exports_every_declared_symbol():
    lib = G.library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert lib.grace_abi_version() == 1
    assert lib.grace_last_hip_error() == 0
    for st in range(6):
        assert lib.grace_status_string(st)


def cross(**kw):
    a = dict(q=P, k=P2, v=P2, off=P2, B=2, M=4, H=2, d=64, sum_L=8, scale=0.125, dtype=1, out=P,
             stream=None)
    a.update(kw)
    return G.library().grace_cross_attn(a["q"], a["k"], a["v"], a["off"], a["B"], a["M"], a["H"],
                                        a["d"], a["sum_L"], a["scale"], a["dtype"], a["out"],
                                        a["stream"])


def append(**kw):
    a = dict(kp=ctypes.c_void_p(0x100000), vp=ctypes.c_void_p(0x200000), tp=ctypes.c_void_p(0x300000),
             tn=ctypes.c_void_p(0x400000), par=ctypes.c_void_p(0x500000), kn=ctypes.c_void_p(0x600000),
             vn=ctypes.c_void_p(0x700000), B=2, M=4, H=2, d=64, T=4, step=1, dtype=1, err=None, stream=None)
    a.update(kw)
    return G.library().grace_kv_append(a["kp"], a["vp"], a["tp"], a["tn"], a["par"], a["kn"], a["vn"],
                                       a["B"], a["M"], a["H"], a["d"], a["T"], a["step"], a["dtype"],
                                       a["err"], a["stream"])


def selfattn(**kw):
    a = dict(q=ctypes.c_void_p(0x100000), kp=ctypes.c_void_p(0x200000), vp=ctypes.c_void_p(0x300000),
             tab=ctypes.c_void_p(0x400000), B=2, M=4, H=2, d=64, T=4, step=1, scale=0.125, dtype=1,
             out=ctypes.c_void_p(0x500000), stream=None)
    a.update(kw)
    return G.library().grace_self_attn_step(a["q"], a["kp"], a["vp"], a["tab"], a["B"], a["M"], a["H"],
                                            a["d"], a["T"], a["step"], a["scale"], a["dtype"], a["out"],
                                            a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(d=48), G.GRACE_ERR_UNSUPPORTED), (dict(d=256), G.GRACE_ERR_UNSUPPORTED),
    (dict(dtype=7), G.GRACE_ERR_UNSUPPORTED), (dict(H=0), G.GRACE_ERR_SHAPE),
    (dict(B=-1), G.GRACE_ERR_SHAPE), (dict(M=-3), G.GRACE_ERR_SHAPE),
    (dict(sum_L=-1), G.GRACE_ERR_SHAPE), (dict(scale=0.0), G.GRACE_ERR_SHAPE),
    (dict(scale=-1.0), G.GRACE_ERR_SHAPE), (dict(scale=math.nan), G.GRACE_ERR_SHAPE),
    (dict(scale=math.inf), G.GRACE_ERR_SHAPE), (dict(q=None), G.GRACE_ERR_NULL),
    (dict(out=None), G.GRACE_ERR_NULL), (dict(off=None), G.GRACE_ERR_NULL),
    (dict(k=None), G.GRACE_ERR_NULL), (dict(out=P2), G.GRACE_ERR_ALIAS),
    (dict(B=1 << 20, M=1 << 12, H=16), G.GRACE_ERR_SHAPE),
    # sizes whose products do not fit 64 bits are rejected without overflowing
    (dict(B=1 << 30, M=1 << 30, H=1 << 30), G.GRACE_ERR_SHAPE),
    (dict(B=0, H=1 << 30, sum_L=1 << 30), G.GRACE_ERR_SHAPE),
    (dict(B=0), G.GRACE_OK), (dict(M=0, q=None, out=None), G.GRACE_OK),
])
def test_cross_attn_rejects(kw, status):
    assert cross(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(T=0), G.GRACE_ERR_SHAPE), (dict(T=9), G.GRACE_ERR_SHAPE),
    (dict(step=4), G.GRACE_ERR_SHAPE), (dict(step=-1), G.GRACE_ERR_SHAPE),
    (dict(d=16), G.GRACE_ERR_UNSUPPORTED), (dict(dtype=2), G.GRACE_ERR_UNSUPPORTED),
    (dict(kp=None), G.GRACE_ERR_NULL), (dict(tn=None), G.GRACE_ERR_NULL),
    (dict(tp=None), G.GRACE_ERR_NULL), (dict(par=None), G.GRACE_ERR_NULL),
    (dict(tn=ctypes.c_void_p(0x300000)), G.GRACE_ERR_ALIAS),       # table_next == table_prev
    (dict(tn=ctypes.c_void_p(0x300010)), G.GRACE_ERR_ALIAS),       # partial overlap
    (dict(kn=ctypes.c_void_p(0x100000 + 8 * 256 + 64)), G.GRACE_ERR_ALIAS),  # inside slab 1
    (dict(B=0), G.GRACE_OK),
])
def test_kv_append_rejects(kw, status):
    assert append(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(T=9), G.GRACE_ERR_SHAPE), (dict(step=4), G.GRACE_ERR_SHAPE),
    (dict(scale=0.0), G.GRACE_ERR_SHAPE), (dict(d=100), G.GRACE_ERR_UNSUPPORTED),
    (dict(tab=None), G.GRACE_ERR_NULL),
    (dict(out=ctypes.c_void_p(0x100000)), G.GRACE_ERR_ALIAS),
    (dict(out=ctypes.c_void_p(0x200000 + 100)), G.GRACE_ERR_ALIAS),
    (dict(M=0), G.GRACE_OK),
])
def test_self_attn_rejects(kw, status):
    assert selfattn(**kw) == status


def fused(**kw):
    # Slab = B*M*H*d*2 = 2048 bytes; pools span 4 slabs.
    a = dict(q=ctypes.c_void_p(0x100000), kn=ctypes.c_void_p(0x200000), vn=ctypes.c_void_p(0x300000),
             kp=ctypes.c_void_p(0x400000), vp=ctypes.c_void_p(0x500000), tp=ctypes.c_void_p(0x600000),
             tn=ctypes.c_void_p(0x700000), par=ctypes.c_void_p(0x800000), B=2, M=4, H=2, d=64, T=4,
             step=1, scale=0.125, dtype=1, out=ctypes.c_void_p(0x900000), err=None, stream=None)
    a.update(kw)
    return G.library().grace_self_attn_step_fused(
        a["q"], a["kn"], a["vn"], a["kp"], a["vp"], a["tp"], a["tn"], a["par"], a["B"], a["M"],
        a["H"], a["d"], a["T"], a["step"], a["scale"], a["dtype"], a["out"], a["err"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(T=9), G.GRACE_ERR_SHAPE), (dict(step=4), G.GRACE_ERR_SHAPE),
    (dict(step=-1), G.GRACE_ERR_SHAPE), (dict(scale=math.nan), G.GRACE_ERR_SHAPE),
    (dict(d=16), G.GRACE_ERR_UNSUPPORTED), (dict(dtype=3), G.GRACE_ERR_UNSUPPORTED),
    (dict(q=None), G.GRACE_ERR_NULL), (dict(kn=None), G.GRACE_ERR_NULL),
    (dict(vp=None), G.GRACE_ERR_NULL), (dict(tn=None), G.GRACE_ERR_NULL),
    (dict(out=None), G.GRACE_ERR_NULL), (dict(tp=None), G.GRACE_ERR_NULL),
    (dict(par=None), G.GRACE_ERR_NULL),
    (dict(tn=ctypes.c_void_p(0x600000)), G.GRACE_ERR_ALIAS),            # table_next == table_prev
    (dict(tn=ctypes.c_void_p(0x800000 - 8)), G.GRACE_ERR_ALIAS),        # table_next over parents
    (dict(out=ctypes.c_void_p(0x100000 + 64)), G.GRACE_ERR_ALIAS),      # out over q
    (dict(out=ctypes.c_void_p(0x700000)), G.GRACE_ERR_ALIAS),           # out == table_next
    (dict(out=ctypes.c_void_p(0x400000 + 16)), G.GRACE_ERR_ALIAS),      # out over read slab 0
    (dict(q=ctypes.c_void_p(0x400000 + 2048 + 64)), G.GRACE_ERR_ALIAS),  # q inside written slab 1
    (dict(kn=ctypes.c_void_p(0x400000 + 2048 + 64)), G.GRACE_ERR_ALIAS),  # k_new inside slab 1
    (dict(kn=ctypes.c_void_p(0x500000 + 2048)), G.GRACE_ERR_ALIAS),     # k_new is v's slab 1
    (dict(tp=None, par=None, step=0, B=0), G.GRACE_OK),
    (dict(M=0), G.GRACE_OK),
])
def test_self_attn_fused_rejects(kw, status):
    assert fused(**kw) == status


def fused_dyn(**kw):
    # rows B*M_cur = 6 of 256 bytes; slab stride R_s rows
    a = dict(q=ctypes.c_void_p(0x100000), kn=ctypes.c_void_p(0x200000), vn=ctypes.c_void_p(0x300000),
             kp=ctypes.c_void_p(0x400000), vp=ctypes.c_void_p(0x500000), tp=ctypes.c_void_p(0x600000),
             tn=ctypes.c_void_p(0x700000), par=ctypes.c_void_p(0x800000), B=2, Mp=2, Mc=3, Rs=8, H=2,
             d=64, T=4, step=1, scale=0.125, dtype=1, out=ctypes.c_void_p(0x900000), err=None,
             stream=None)
    a.update(kw)
    return G.library().grace_self_attn_step_fused_dyn(
        a["q"], a["kn"], a["vn"], a["kp"], a["vp"], a["tp"], a["tn"], a["par"], a["B"], a["Mp"],
        a["Mc"], a["Rs"], a["H"], a["d"], a["T"], a["step"], a["scale"], a["dtype"], a["out"],
        a["err"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(Rs=5), G.GRACE_ERR_SHAPE),                       # R_s < B*M_cur
    (dict(Mp=0), G.GRACE_ERR_SHAPE), (dict(Mp=5), G.GRACE_ERR_SHAPE),   # B*M_prev > R_s
    (dict(Rs=1 << 29), G.GRACE_ERR_SHAPE),                 # T_max*R_s >= 2^31
    (dict(step=4), G.GRACE_ERR_SHAPE), (dict(d=48), G.GRACE_ERR_UNSUPPORTED),
    (dict(par=None), G.GRACE_ERR_NULL), (dict(q=None), G.GRACE_ERR_NULL),
    (dict(out=ctypes.c_void_p(0x400000 + 8)), G.GRACE_ERR_ALIAS),          # out over slab 0
    (dict(kn=ctypes.c_void_p(0x400000 + 8 * 256 + 16)), G.GRACE_ERR_ALIAS),  # inside slab 1
    (dict(tn=ctypes.c_void_p(0x600000 + 4)), G.GRACE_ERR_ALIAS),
    (dict(step=0, Mp=0, tp=None, par=None, B=0), G.GRACE_OK),
])
def test_self_attn_fused_dyn_rejects(kw, status):
    assert fused_dyn(**kw) == status


def beam_scores(**kw):
    a = dict(lg=ctypes.c_void_p(0x100000), prev=ctypes.c_void_p(0x200000), mask=None, R=4, V=40,
             dtype=1, cand=ctypes.c_void_p(0x300000), rmax=ctypes.c_void_p(0x400000), stream=None)
    a.update(kw)
    return G.library().grace_beam_scores(a["lg"], a["prev"], a["mask"], a["R"], a["V"], a["dtype"],
                                         a["cand"], a["rmax"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(V=0), G.GRACE_ERR_SHAPE), (dict(R=-1), G.GRACE_ERR_SHAPE),
    (dict(R=1 << 20, V=1 << 12), G.GRACE_ERR_SHAPE), (dict(dtype=2), G.GRACE_ERR_UNSUPPORTED),
    (dict(lg=None), G.GRACE_ERR_NULL), (dict(cand=None), G.GRACE_ERR_NULL),
    (dict(prev=None), G.GRACE_ERR_NULL),
    (dict(cand=ctypes.c_void_p(0x100000 + 64)), G.GRACE_ERR_ALIAS),      # over logits
    (dict(rmax=ctypes.c_void_p(0x300000 + 16)), G.GRACE_ERR_ALIAS),      # over cand
    (dict(mask=ctypes.c_void_p(0x300000 + 4)), G.GRACE_ERR_ALIAS),       # cand over mask
    (dict(R=0), G.GRACE_OK),
])
def test_beam_scores_rejects(kw, status):
    assert beam_scores(**kw) == status


def beam_topk(**kw):
    a = dict(cand=ctypes.c_void_p(0x100000), rmax=None, B=2, M=8, V=64, k=16,
             ws=ctypes.c_void_p(0x1000000), wsb=1 << 22,
             par=ctypes.c_void_p(0x200000), tok=ctypes.c_void_p(0x300000),
             sc=ctypes.c_void_p(0x400000), stream=None)
    a.update(kw)
    return G.library().grace_beam_topk(a["cand"], a["rmax"], a["B"], a["M"], a["V"], a["k"], a["ws"],
                                       a["wsb"], a["par"], a["tok"], a["sc"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), G.GRACE_ERR_SHAPE), (dict(k=8 * 64 + 1), G.GRACE_ERR_SHAPE),
    (dict(M=1 << 20, V=1 << 12, k=4), G.GRACE_ERR_SHAPE), (dict(M=0), G.GRACE_ERR_SHAPE),
    (dict(M=100, k=5000), G.GRACE_ERR_SHAPE),              # above grace_beam_topk_max_k
    (dict(B=(1 << 31) - 1, M=1 << 15, V=(1 << 16) - 1, k=4), G.GRACE_ERR_SHAPE),   # B*M*V >= 2^40
    (dict(cand=None), G.GRACE_ERR_NULL), (dict(tok=None), G.GRACE_ERR_NULL),
    (dict(par=ctypes.c_void_p(0x300000 + 8)), G.GRACE_ERR_ALIAS),
    (dict(sc=ctypes.c_void_p(0x100000 + 40)), G.GRACE_ERR_ALIAS),
    (dict(ws=None), G.GRACE_ERR_NULL), (dict(wsb=1024), G.GRACE_ERR_SHAPE),
    (dict(ws=ctypes.c_void_p(0x1000004)), G.GRACE_ERR_SHAPE),          # misaligned
    (dict(ws=ctypes.c_void_p(0x100000 + 64)), G.GRACE_ERR_ALIAS),      # over cand
    (dict(B=0), G.GRACE_OK),
])
def test_beam_topk_rejects(kw, status):
    assert beam_topk(**kw) == status


def beam_step(**kw):
    a = dict(logits=ctypes.c_void_p(0x100000), prev=ctypes.c_void_p(0x180000), mask=None, B=2, M=8,
             V=64, k=16, dtype=G.GRACE_BF16, ws=ctypes.c_void_p(0x1000000), wsb=1 << 22,
             par=ctypes.c_void_p(0x200000), tok=ctypes.c_void_p(0x300000),
             sc=ctypes.c_void_p(0x400000), stream=None)
    a.update(kw)
    return G.library().grace_beam_step(a["logits"], a["prev"], a["mask"], a["B"], a["M"], a["V"],
                                       a["k"], a["dtype"], a["ws"], a["wsb"], a["par"], a["tok"],
                                       a["sc"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), G.GRACE_ERR_UNSUPPORTED),
    (dict(k=0), G.GRACE_ERR_SHAPE), (dict(k=8 * 64 + 1), G.GRACE_ERR_SHAPE),
    (dict(B=1 << 10, M=1 << 12, V=1 << 10, k=4), G.GRACE_ERR_SHAPE),   # B*M*V >= 2^31
    (dict(M=0), G.GRACE_ERR_SHAPE), (dict(M=100, k=5000), G.GRACE_ERR_SHAPE),
    (dict(logits=None), G.GRACE_ERR_NULL), (dict(prev=None), G.GRACE_ERR_NULL),
    (dict(sc=None), G.GRACE_ERR_NULL), (dict(ws=None), G.GRACE_ERR_NULL),
    (dict(wsb=1024), G.GRACE_ERR_SHAPE), (dict(ws=ctypes.c_void_p(0x1000004)), G.GRACE_ERR_SHAPE),
    (dict(par=ctypes.c_void_p(0x300000 + 8)), G.GRACE_ERR_ALIAS),      # over tokens
    (dict(sc=ctypes.c_void_p(0x100000 + 40)), G.GRACE_ERR_ALIAS),      # over logits
    (dict(tok=ctypes.c_void_p(0x180000)), G.GRACE_ERR_ALIAS),          # over prev_scores
    (dict(mask=ctypes.c_void_p(0x200000 - 64)), G.GRACE_ERR_ALIAS),    # mask over parents
    (dict(ws=ctypes.c_void_p(0x100000 + 64)), G.GRACE_ERR_ALIAS),      # over logits
    (dict(B=0), G.GRACE_OK),
])
def test_beam_step_rejects(kw, status):
    assert beam_step(**kw) == status


def beam_step_noalloc(**kw):
    a = dict(logits=ctypes.c_void_p(0x100000), prev=ctypes.c_void_p(0x180000), mask=None, B=2, M=8,
             V=64, k=16, dtype=G.GRACE_BF16, par=ctypes.c_void_p(0x200000),
             tok=ctypes.c_void_p(0x300000), sc=ctypes.c_void_p(0x400000), stream=None)
    a.update(kw)
    return G.library().grace_beam_step_noalloc(a["logits"], a["prev"], a["mask"], a["B"], a["M"],
                                               a["V"], a["k"], a["dtype"], a["par"], a["tok"],
                                               a["sc"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), G.GRACE_ERR_UNSUPPORTED),
    (dict(k=0), G.GRACE_ERR_SHAPE), (dict(k=8 * 64 + 1), G.GRACE_ERR_SHAPE),
    (dict(B=1 << 10, M=1 << 12, V=1 << 10, k=4), G.GRACE_ERR_SHAPE),   # B*M*V >= 2^31
    (dict(B=128, M=4096, V=512, k=4096), G.GRACE_ERR_SHAPE),          # workspace > the scratch array
    (dict(M=0), G.GRACE_ERR_SHAPE),
    (dict(logits=None), G.GRACE_ERR_NULL), (dict(prev=None), G.GRACE_ERR_NULL),
    (dict(par=None), G.GRACE_ERR_NULL), (dict(sc=None), G.GRACE_ERR_NULL),
    (dict(B=0), G.GRACE_OK),
])
def test_beam_step_noalloc_rejects(kw, status):
    assert beam_step_noalloc(**kw) == status


def test_beam_step_noalloc_limit():
    """The header's limit is the binding's, and it holds the 64 x 4096 x 512 step."""
    text = open(HEADER).read()
    m = re.search(r"#define GRACE_BEAM_STEP_NOALLOC_MAX_BYTES \((\d+)ll << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == G.BEAM_STEP_NOALLOC_MAX_BYTES
    lib = G.library()
    assert lib.grace_beam_step_workspace_bytes(64, 4096, 512) <= G.BEAM_STEP_NOALLOC_MAX_BYTES
    assert lib.grace_beam_step_workspace_bytes(128, 4096, 512) > G.BEAM_STEP_NOALLOC_MAX_BYTES


def test_beam_step_workspace_bytes():
    lib = G.library()
    assert lib.grace_beam_step_workspace_bytes(2, 0, 64) == -1
    assert lib.grace_beam_step_workspace_bytes(1 << 10, 1 << 12, 1 << 10) == -1
    for B, M, V in ((1, 8, 64), (64, 4096, 512)):
        extra = lib.grace_beam_step_workspace_bytes(B, M, V) - lib.grace_beam_topk_workspace_bytes(B, M, V)
        assert extra == B * M * 8   # the rows' log-sum-exp and best score


def test_beam_topk_max_k_and_workspace():
    assert G.library().grace_beam_topk_max_k() == 4096
    lib = G.library()
    assert lib.grace_beam_topk_workspace_bytes(0, 1, 1) >= 0
    assert lib.grace_beam_topk_workspace_bytes(2, 0, 64) == -1
    small, big = lib.grace_beam_topk_workspace_bytes(1, 8, 64), lib.grace_beam_topk_workspace_bytes(64, 4096, 512)
    assert 0 < small < big < (128 << 20)


def _gtm_index(**kw):
    a = dict(vocab=512, num_nodes=10, num_entries=9, bitmask_words=7, bloom_words=4, bitmask_rows=5,
             bloom_rows=5, reserved=0, node_offsets=0x100000, child_nodes=0x200000, tokens=0x300000,
             bitmask_index=0x400000, bloom_index=0x500000, bitmask_table=0x600000,
             bloom_table=0x700000)
    a.update(kw)
    return G.GtmIndexC(*[a[f] for f, _ in G.GtmIndexC._fields_])


def _gtm_user(**kw):
    a = dict(max_locations=8, reserved=0, bitmask=0x800000, bloom=0x900000, num_locations=0xA00000)
    a.update(kw)
    return G.GtmUserC(*[a[f] for f, _ in G.GtmUserC._fields_])


@pytest.mark.parametrize("ix,us,extra,status", [
    (dict(vocab=0), {}, {}, G.GRACE_ERR_SHAPE), (dict(vocab=5000), {}, {}, G.GRACE_ERR_SHAPE),
    (dict(bitmask_words=9), {}, {}, G.GRACE_ERR_UNSUPPORTED),
    (dict(bloom_words=5), {}, {}, G.GRACE_ERR_UNSUPPORTED),
    (dict(reserved=1), {}, {}, G.GRACE_ERR_SHAPE), (dict(num_nodes=0), {}, {}, G.GRACE_ERR_SHAPE),
    (dict(tokens=0), {}, {}, G.GRACE_ERR_NULL), (dict(bloom_table=0), {}, {}, G.GRACE_ERR_NULL),
    ({}, dict(max_locations=65), {}, G.GRACE_ERR_SHAPE), ({}, dict(bitmask=0), {}, G.GRACE_ERR_NULL),
    ({}, {}, dict(mask=None), G.GRACE_ERR_NULL),
    ({}, {}, dict(mask=ctypes.c_void_p(0x300000 + 2)), G.GRACE_ERR_ALIAS),   # over tokens
    ({}, {}, dict(mask=ctypes.c_void_p(0xB00000 - 8)), G.GRACE_ERR_ALIAS),   # over node ids
    ({}, {}, dict(B=1 << 30, M=1 << 30), G.GRACE_ERR_SHAPE),
    ({}, {}, dict(B=0), G.GRACE_OK),
])
def test_gtm_mask_rejects(ix, us, extra, status):
    a = dict(nodes=ctypes.c_void_p(0xB00000), B=2, M=4, mask=ctypes.c_void_p(0xC00000))
    a.update(extra)
    idx, usr = _gtm_index(**ix), _gtm_user(**us)
    assert G.library().grace_gtm_mask(ctypes.byref(idx), ctypes.byref(usr), a["nodes"], a["B"], a["M"],
                                      a["mask"], None, None) == status


def test_gtm_mask_null_structs():
    lib = G.library()
    assert lib.grace_gtm_mask(None, ctypes.byref(_gtm_user()), P, 1, 1, P2, None, None) == G.GRACE_ERR_NULL
    assert lib.grace_gtm_mask(ctypes.byref(_gtm_index()), None, P, 1, 1, P2, None, None) == G.GRACE_ERR_NULL


@pytest.mark.parametrize("kw,status", [
    (dict(Mp=0), G.GRACE_ERR_SHAPE), (dict(k=-1), G.GRACE_ERR_SHAPE),
    (dict(par=None), G.GRACE_ERR_NULL),
    (dict(out=ctypes.c_void_p(0xD00000 + 4)), G.GRACE_ERR_ALIAS),     # over parents
    (dict(k=0), G.GRACE_OK),
])
def test_trie_advance_rejects(kw, status):
    a = dict(prev=ctypes.c_void_p(0xC00000), par=ctypes.c_void_p(0xD00000), tok=ctypes.c_void_p(0xE00000),
             B=2, Mp=4, k=3, out=ctypes.c_void_p(0xF00000))
    a.update(kw)
    idx = _gtm_index()
    assert G.library().grace_trie_advance(ctypes.byref(idx), a["prev"], a["par"], a["tok"], a["B"], a["Mp"],
                                          a["k"], a["out"], None, None) == status


def test_graph_api_rejects_null():
    lib = G.library()
    h = ctypes.c_void_p()
    assert lib.grace_graph_begin(None) == G.GRACE_ERR_NULL
    assert lib.grace_graph_end(None, ctypes.byref(h)) == G.GRACE_ERR_NULL
    assert lib.grace_graph_end(P, None) == G.GRACE_ERR_NULL
    assert lib.grace_graph_launch(None, None) == G.GRACE_ERR_NULL
    assert lib.grace_graph_destroy(None) == G.GRACE_OK


def test_binding_raises_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(G, "_lib", None)
    monkeypatch.setattr(G, "_LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        G.library()
