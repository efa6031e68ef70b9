"""Python binding of libgrace.so (argument marshalling only).

The entry points keep their C names and take torch tensors that already
live on the GPU; each call passes raw device pointers, sizes, the dtype code and
the current HIP stream to the library and turns a non-zero status into
:class:`GraceError`.  Every step of the computation runs in the library's HIP
kernels; there is no other code path, and a missing build raises on first use.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgrace.so")
_lib = None

GRACE_F32, GRACE_BF16 = 0, 1
GRACE_OK, GRACE_ERR_NULL, GRACE_ERR_SHAPE, GRACE_ERR_UNSUPPORTED, GRACE_ERR_ALIAS, GRACE_ERR_HIP = range(6)

_DTYPE_CODE = {torch.float32: GRACE_F32, torch.bfloat16: GRACE_BF16}

_c_int, _c_float, _c_void_p = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p


class GtmIndexC(ctypes.Structure):
    """Mirror of ``grace_gtm_index``."""
    _fields_ = [("vocab", ctypes.c_int32), ("num_nodes", ctypes.c_int32),
                ("num_entries", ctypes.c_int32), ("bitmask_words", ctypes.c_int32),
                ("bloom_words", ctypes.c_int32), ("bitmask_rows", ctypes.c_int32),
                ("bloom_rows", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("node_offsets", ctypes.c_void_p), ("child_nodes", ctypes.c_void_p),
                ("tokens", ctypes.c_void_p), ("bitmask_index", ctypes.c_void_p),
                ("bloom_index", ctypes.c_void_p), ("bitmask_table", ctypes.c_void_p),
                ("bloom_table", ctypes.c_void_p)]


class GtmUserC(ctypes.Structure):
    """Mirror of ``grace_gtm_user``."""
    _fields_ = [("max_locations", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("bitmask", ctypes.c_void_p), ("bloom", ctypes.c_void_p),
                ("num_locations", ctypes.c_void_p)]
_SIGNATURES = {
    "grace_cross_attn": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int,
                         _c_int, _c_int, _c_float, _c_int, _c_void_p, _c_void_p],
    "grace_kv_append": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                        _c_void_p, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int, _c_int,
                        _c_void_p, _c_void_p],
    "grace_self_attn_step": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int,
                             _c_int, _c_int, _c_int, _c_float, _c_int, _c_void_p, _c_void_p],
    "grace_self_attn_step_fused": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                   _c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int,
                                   _c_int, _c_int, _c_int, _c_float, _c_int, _c_void_p, _c_void_p,
                                   _c_void_p],
    "grace_self_attn_step_fused_dyn": [_c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                       _c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int,
                                       _c_int, _c_int, _c_int, _c_int, _c_int, _c_float, _c_int,
                                       _c_void_p, _c_void_p, _c_void_p],
    "grace_beam_scores": [_c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int, _c_void_p,
                          _c_void_p, _c_void_p],
    "grace_beam_topk_max_k": [],
    "grace_beam_topk_workspace_bytes": [_c_int, _c_int, _c_int],
    "grace_beam_topk": [_c_void_p, _c_void_p, _c_int, _c_int, _c_int, _c_int, _c_void_p,
                        ctypes.c_int64, _c_void_p, _c_void_p, _c_void_p, _c_void_p],
    "grace_beam_step_workspace_bytes": [_c_int, _c_int, _c_int],
    "grace_beam_step": [_c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int, _c_int, _c_int,
                        _c_void_p, ctypes.c_int64, _c_void_p, _c_void_p, _c_void_p, _c_void_p],
    "grace_beam_step_noalloc": [_c_void_p, _c_void_p, _c_void_p, _c_int, _c_int, _c_int, _c_int,
                                _c_int, _c_void_p, _c_void_p, _c_void_p, _c_void_p],
    "grace_gtm_mask": [ctypes.POINTER(GtmIndexC), ctypes.POINTER(GtmUserC), _c_void_p, _c_int,
                       _c_int, _c_void_p, _c_void_p, _c_void_p],
    "grace_trie_advance": [ctypes.POINTER(GtmIndexC), _c_void_p, _c_void_p, _c_void_p, _c_int,
                           _c_int, _c_int, _c_void_p, _c_void_p, _c_void_p],
    "grace_graph_begin": [_c_void_p],
    "grace_graph_end": [_c_void_p, ctypes.POINTER(_c_void_p)],
    "grace_graph_launch": [_c_void_p, _c_void_p],
    "grace_graph_destroy": [_c_void_p],
    "grace_graph_last_hip_error": [],
    "grace_debug_counts": [_c_void_p],
    "grace_status_string": [_c_int],
    "grace_last_hip_error": [],
    "grace_abi_version": [],
}


class GraceError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = library().grace_status_string(status).decode()
        if status == GRACE_ERR_HIP:
            msg += f" (hipError {library().grace_last_hip_error()})"
        super().__init__(f"{where}: {msg} [status {status}]")


_DEBUG_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgrace_debug.so")
_debug_lib = None
GRACE_DEBUG_KINDS = 8


def _load(path: str) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2608_00938_amd.build`")
    lib = ctypes.CDLL(path)
    for name, args in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = (ctypes.c_char_p if name == "grace_status_string" else
                      ctypes.c_int64 if name.endswith("_bytes") else _c_int)
    return lib


def library() -> ctypes.CDLL:
    """The loaded libgrace.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        _lib = _load(_LIB_PATH)
    return _lib


def debug_library() -> ctypes.CDLL:
    """libgrace_debug.so: the same entry points with the device-side index
    checks of the debug build (read with grace_debug_counts)."""
    global _debug_lib
    if _debug_lib is None:
        _debug_lib = _load(_DEBUG_LIB_PATH)
    return _debug_lib


def grace_debug_counts(lib=None) -> list:
    """Synchronise and read (and clear) the debug build's device-check counters:
    [offsets, parents, block ids, computed rows, 0, 0, 0, 0]."""
    lib = debug_library() if lib is None else lib
    buf = (ctypes.c_uint32 * GRACE_DEBUG_KINDS)()
    _check(lib.grace_debug_counts(buf), "grace_debug_counts")
    return list(buf)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(t: torch.Tensor):
    return torch.cuda.current_stream(t.device).cuda_stream


def _check(status: int, where: str):
    if status != GRACE_OK:
        raise GraceError(status, where)


def _dtype_code(t: torch.Tensor) -> int:
    try:
        return _DTYPE_CODE[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}") from None


def _contig(*ts):
    for t in ts:
        if t is not None and not t.is_contiguous():
            raise ValueError("tensors passed to libgrace must be contiguous")


def grace_cross_attn(q, enc_k, enc_v, enc_off, M: int, scale: float | None = None, out=None):
    """Beam-as-query cross-attention; q [B*M, H, d], enc_k/enc_v [sum_L, H, d],
    enc_off int32 [B+1] on the device.  Returns out [B*M, H, d]."""
    _contig(q, enc_k, enc_v, enc_off, out)
    R, H, d = q.shape
    B = enc_off.numel() - 1
    if M <= 0 and R == 0:
        M = 0
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if out is None:
        out = torch.empty_like(q)
    st = library().grace_cross_attn(_ptr(q), _ptr(enc_k), _ptr(enc_v), _ptr(enc_off), B, M, H, d,
                                    enc_k.shape[0], scale, _dtype_code(q), _ptr(out), _stream(q))
    _check(st, "grace_cross_attn")
    return out


def grace_kv_append(k_pool, v_pool, table_prev, table_next, parents, k_new, v_new, B: int,
                    M: int, step: int, err_flag=None):
    """Paged rearrangement + append at ``step``; pools [T_max, B*M, H, d], tables
    int32 [B*M, T_max], parents int32 [B*M] (None at step 0)."""
    _contig(k_pool, v_pool, table_prev, table_next, parents, k_new, v_new)
    T_max, R, H, d = k_pool.shape
    st = library().grace_kv_append(_ptr(k_pool), _ptr(v_pool), _ptr(table_prev), _ptr(table_next),
                                   _ptr(parents), _ptr(k_new), _ptr(v_new), B, M, H, d, T_max,
                                   step, _dtype_code(k_pool), _ptr(err_flag), _stream(k_pool))
    _check(st, "grace_kv_append")


def grace_self_attn_step(q, k_pool, v_pool, table, B: int, M: int, step: int,
                         scale: float | None = None, out=None):
    """Paged self-attention over step+1 tokens; returns out [B*M, H, d]."""
    _contig(q, k_pool, v_pool, table, out)
    T_max, R, H, d = k_pool.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if out is None:
        out = torch.empty_like(q)
    st = library().grace_self_attn_step(_ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(table), B, M,
                                        H, d, T_max, step, scale, _dtype_code(q), _ptr(out),
                                        _stream(q))
    _check(st, "grace_self_attn_step")
    return out


def grace_self_attn_step_fused(q, k_new, v_new, k_pool, v_pool, table_prev, table_next, parents,
                               B: int, M: int, step: int, scale: float | None = None, out=None,
                               err_flag=None):
    """Paged append and self-attention in one pass: writes table_next and slab
    ``step`` of the pools like :func:`grace_kv_append`, returns the attention of
    :func:`grace_self_attn_step` over table_next [B*M, H, d]."""
    _contig(q, k_new, v_new, k_pool, v_pool, table_prev, table_next, parents, out)
    T_max, R, H, d = k_pool.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if out is None:
        out = torch.empty_like(q)
    st = library().grace_self_attn_step_fused(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool), _ptr(table_prev),
        _ptr(table_next), _ptr(parents), B, M, H, d, T_max, step, scale, _dtype_code(q), _ptr(out),
        _ptr(err_flag), _stream(q))
    _check(st, "grace_self_attn_step_fused")
    return out


def grace_self_attn_step_fused_dyn(q, k_new, v_new, k_pool, v_pool, table_prev, table_next,
                                   parents, B: int, M_prev: int, M_cur: int, step: int,
                                   scale: float | None = None, out=None, err_flag=None):
    """Fused append + attend with per-step beam widths: q/k_new/v_new [B*M_cur, H, d];
    pools [T_max, R_s, H, d]; tables int32 [>= rows, T_max]; parents int32 [B*M_cur]
    in [0, M_prev).  Returns out [B*M_cur, H, d]."""
    _contig(q, k_new, v_new, k_pool, v_pool, table_prev, table_next, parents, out)
    T_max, R_s, H, d = k_pool.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if out is None:
        out = torch.empty_like(q)
    st = library().grace_self_attn_step_fused_dyn(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool), _ptr(table_prev),
        _ptr(table_next), _ptr(parents), B, M_prev, M_cur, R_s, H, d, T_max, step, scale,
        _dtype_code(q), _ptr(out), _ptr(err_flag), _stream(q))
    _check(st, "grace_self_attn_step_fused_dyn")
    return out


def grace_beam_scores(logits, prev_scores, mask=None, cand=None, row_max=None):
    """Candidate scores prev + log_softmax(logits), -inf where the packed mask
    (uint32 words as int32 [R, ceil(V/32)]) clears the bit.  logits [R, V]
    (fp32 or bf16); prev_scores fp32 [R].  Returns (cand fp32 [R, V], row_max fp32 [R])."""
    _contig(logits, prev_scores, mask, cand, row_max)
    R, V = logits.shape
    if cand is None:
        cand = torch.empty((R, V), dtype=torch.float32, device=logits.device)
    if row_max is None:
        row_max = torch.empty((R,), dtype=torch.float32, device=logits.device)
    st = library().grace_beam_scores(_ptr(logits), _ptr(prev_scores), _ptr(mask), R, V,
                                     _dtype_code(logits), _ptr(cand), _ptr(row_max),
                                     _stream(logits))
    _check(st, "grace_beam_scores")
    return cand, row_max


def grace_beam_topk_max_k() -> int:
    return library().grace_beam_topk_max_k()


def grace_beam_topk_workspace_bytes(B: int, M: int, V: int) -> int:
    return library().grace_beam_topk_workspace_bytes(B, M, V)


def grace_beam_topk(cand, B: int, M: int, k: int, row_max=None, parents=None, tokens=None,
                    scores=None, workspace=None):
    """Per-request top-k over cand [B*M, V] fp32.  Returns (parents, tokens, scores),
    each [B, k] (int32, int32, fp32), best first.  ``workspace``: a device uint8
    tensor of at least grace_beam_topk_workspace_bytes(B, M, V) bytes (allocated
    here when not given)."""
    _contig(cand, row_max, parents, tokens, scores, workspace)
    V = cand.shape[1]
    dev = cand.device
    need = grace_beam_topk_workspace_bytes(B, M, V)
    if workspace is None:
        workspace = torch.empty((max(need, 8),), dtype=torch.uint8, device=dev)
    if parents is None:
        parents = torch.empty((B, k), dtype=torch.int32, device=dev)
    if tokens is None:
        tokens = torch.empty((B, k), dtype=torch.int32, device=dev)
    if scores is None:
        scores = torch.empty((B, k), dtype=torch.float32, device=dev)
    st = library().grace_beam_topk(_ptr(cand), _ptr(row_max), B, M, V, k, _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _ptr(parents),
                                   _ptr(tokens), _ptr(scores), _stream(cand))
    _check(st, "grace_beam_topk")
    return parents, tokens, scores


def grace_beam_step_workspace_bytes(B: int, M: int, V: int) -> int:
    return library().grace_beam_step_workspace_bytes(B, M, V)


def grace_beam_step(logits, prev_scores, B: int, M: int, k: int, mask=None, parents=None,
                    tokens=None, scores=None, workspace=None):
    """Score update and per-request top-k in one call, without the candidate
    array: the same (parents, tokens, scores) as grace_beam_scores followed by
    grace_beam_topk.  logits [B*M, V] (fp32 or bf16), prev_scores fp32 [B*M],
    mask as for grace_beam_scores.  ``workspace``: a device uint8 tensor of at
    least grace_beam_step_workspace_bytes(B, M, V) bytes (allocated here when
    not given)."""
    _contig(logits, prev_scores, mask, parents, tokens, scores, workspace)
    V = logits.shape[1]
    dev = logits.device
    need = grace_beam_step_workspace_bytes(B, M, V)
    if workspace is None:
        workspace = torch.empty((max(need, 8),), dtype=torch.uint8, device=dev)
    if parents is None:
        parents = torch.empty((B, k), dtype=torch.int32, device=dev)
    if tokens is None:
        tokens = torch.empty((B, k), dtype=torch.int32, device=dev)
    if scores is None:
        scores = torch.empty((B, k), dtype=torch.float32, device=dev)
    st = library().grace_beam_step(_ptr(logits), _ptr(prev_scores), _ptr(mask), B, M, V, k,
                                   _dtype_code(logits), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _ptr(parents),
                                   _ptr(tokens), _ptr(scores), _stream(logits))
    _check(st, "grace_beam_step")
    return parents, tokens, scores


#: Largest workspace grace_beam_step_noalloc serves (GRACE_BEAM_STEP_NOALLOC_MAX_BYTES).
BEAM_STEP_NOALLOC_MAX_BYTES = 80 << 20


def grace_beam_step_noalloc(logits, prev_scores, B: int, M: int, k: int, mask=None, parents=None,
                            tokens=None, scores=None):
    """grace_beam_step without a workspace argument: the library's per-GPU
    scratch array serves as the workspace, so the call allocates no device
    memory when the outputs are given.  Calls that overlap in time on one GPU
    race on that array."""
    _contig(logits, prev_scores, mask, parents, tokens, scores)
    dev = logits.device
    if parents is None:
        parents = torch.empty((B, k), dtype=torch.int32, device=dev)
    if tokens is None:
        tokens = torch.empty((B, k), dtype=torch.int32, device=dev)
    if scores is None:
        scores = torch.empty((B, k), dtype=torch.float32, device=dev)
    st = library().grace_beam_step_noalloc(_ptr(logits), _ptr(prev_scores), _ptr(mask), B, M,
                                           logits.shape[1], k, _dtype_code(logits), _ptr(parents),
                                           _ptr(tokens), _ptr(scores), _stream(logits))
    _check(st, "grace_beam_step_noalloc")
    return parents, tokens, scores


def _dev(a, dtype, device):
    """numpy array -> contiguous device tensor (uint64 words travel as int64 bit patterns)."""
    import numpy as np
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(a).to(device=device, dtype=dtype)


class GtmIndex:
    """Device copy of a CD+GTM index (grace_gtm_index): CSR trie + matcher tables."""

    def __init__(self, ix: dict, device="cuda"):
        import numpy as np
        self.vocab = int(ix["vocab"])
        self.t = dict(
            node_offsets=_dev(ix["node_offsets"].astype(np.int32), torch.int32, device),
            child_nodes=_dev(ix["child_nodes"].astype(np.int32), torch.int32, device),
            tokens=_dev(ix["tokens"].astype(np.int16), torch.int16, device),
            bitmask_index=_dev(ix["bitmask_index"].astype(np.int32), torch.int32, device),
            bloom_index=_dev(ix["bloom_index"].astype(np.int32), torch.int32, device),
            bitmask_table=_dev(ix["bitmask_table"], torch.int64, device),
            bloom_table=_dev(ix["bloom_table"], torch.int64, device))
        bm, bl = ix["bitmask_table"], ix["bloom_table"]
        self.c = GtmIndexC(self.vocab, ix["node_offsets"].shape[0] - 1, ix["tokens"].shape[0],
                           bm.shape[1], bl.shape[1], bm.shape[0], bl.shape[0], 0,
                           *(_ptr(self.t[k]) for k in ("node_offsets", "child_nodes", "tokens",
                                                        "bitmask_index", "bloom_index",
                                                        "bitmask_table", "bloom_table")))


class GtmUsers:
    """Device copy of the requests' targeting attributes (grace_gtm_user)."""

    def __init__(self, us: dict, device="cuda"):
        self.t = dict(bitmask=_dev(us["bitmask"], torch.int64, device),
                      bloom=_dev(us["bloom"], torch.int64, device),
                      n_loc=_dev(us["n_loc"], torch.int32, device))
        self.c = GtmUserC(int(us["bloom"].shape[1]), 0, _ptr(self.t["bitmask"]),
                          _ptr(self.t["bloom"]), _ptr(self.t["n_loc"]))


def grace_gtm_mask(index: GtmIndex, users: GtmUsers, node_ids, B: int, M: int, mask=None,
                   err_flag=None):
    """Constraint filter words (int32 view of uint32) [B*M, ceil(V/32)] of the beams at node_ids."""
    _contig(node_ids, mask)
    W = (index.vocab + 31) // 32
    if mask is None:
        mask = torch.empty((B * M, W), dtype=torch.int32, device=node_ids.device)
    st = library().grace_gtm_mask(ctypes.byref(index.c), ctypes.byref(users.c), _ptr(node_ids), B, M,
                                  _ptr(mask), _ptr(err_flag), _stream(node_ids))
    _check(st, "grace_gtm_mask")
    return mask


def grace_trie_advance(index: GtmIndex, node_prev, parents, tokens, B: int, M_prev: int, k: int,
                       node_next=None, err_flag=None):
    """Trie node of every new beam [B*k] from its parent's node and its token."""
    _contig(node_prev, parents, tokens, node_next)
    if node_next is None:
        node_next = torch.empty((B * k,), dtype=torch.int32, device=node_prev.device)
    st = library().grace_trie_advance(ctypes.byref(index.c), _ptr(node_prev), _ptr(parents),
                                      _ptr(tokens), B, M_prev, k, _ptr(node_next), _ptr(err_flag),
                                      _stream(node_prev))
    _check(st, "grace_trie_advance")
    return node_next


class Graph:
    """An executable HIP graph recorded from library calls (grace_graph_*)."""

    def __init__(self, handle: int):
        self.handle = handle

    def launch(self, stream=None):
        st = torch.cuda.current_stream() if stream is None else stream
        _check(library().grace_graph_launch(self.handle, st.cuda_stream), "grace_graph_launch")

    def destroy(self):
        if self.handle:
            library().grace_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def capture(fn, stream) -> Graph:
    """Record the library calls ``fn()`` enqueues on ``stream`` (a torch.cuda.Stream
    other than the null stream) into a Graph; nothing runs until Graph.launch."""
    lib = library()
    with torch.cuda.stream(stream):
        _check(lib.grace_graph_begin(stream.cuda_stream), "grace_graph_begin")
        try:
            fn()
        finally:
            h = _c_void_p()
            st = lib.grace_graph_end(stream.cuda_stream, ctypes.byref(h))
    _check(st, "grace_graph_end")
    return Graph(h.value)


class KVCache:
    """Caller-side storage of the paged self-attention cache: the two pools and
    a pair of block tables used alternately (the update reads one, writes the
    other).  Allocation is torch's; all work is the library's."""

    def __init__(self, B: int, M: int, H: int, d: int, T_max: int, dtype: torch.dtype,
                 device="cuda"):
        """M is the beam width (the largest width when steps use dynamic widths)."""
        self.B, self.M, self.H, self.d, self.T_max = B, M, H, d, T_max
        R = B * M
        self.k_pool = torch.empty((T_max, R, H, d), dtype=dtype, device=device)
        self.v_pool = torch.empty((T_max, R, H, d), dtype=dtype, device=device)
        self.tables = [torch.zeros((R, T_max), dtype=torch.int32, device=device) for _ in range(2)]
        self.err_flag = torch.zeros(1, dtype=torch.int32, device=device)

    def table(self, step: int) -> torch.Tensor:
        """Block table valid after the append of ``step``."""
        return self.tables[step % 2]

    def slab(self, step: int):
        """Views of pool slab ``step``: writing k_new/v_new here makes the append copy-free."""
        return self.k_pool[step], self.v_pool[step]

    def append(self, step: int, k_new, v_new, parents=None):
        grace_kv_append(self.k_pool, self.v_pool, self.tables[(step + 1) % 2], self.tables[step % 2],
                        parents, k_new, v_new, self.B, self.M, step, self.err_flag)

    def attend(self, step: int, q, scale: float | None = None, out=None):
        return grace_self_attn_step(q, self.k_pool, self.v_pool, self.table(step), self.B, self.M,
                                    step, scale=scale, out=out)

    def append_attend_dyn(self, step: int, q, k_new, v_new, parents, M_prev: int, M_cur: int,
                          scale: float | None = None, out=None):
        """Fused append + attend at widths M_prev -> M_cur (<= M); slab rows stride B*M."""
        R = self.B * M_cur
        return grace_self_attn_step_fused_dyn(q, k_new, v_new, self.k_pool, self.v_pool,
                                              self.tables[(step + 1) % 2],
                                              self.tables[step % 2][:R], parents, self.B,
                                              M_prev, M_cur, step, scale=scale, out=out,
                                              err_flag=self.err_flag)

    def append_attend(self, step: int, q, k_new, v_new, parents=None, scale: float | None = None,
                      out=None):
        """:meth:`append` then :meth:`attend`, as one fused pass."""
        return grace_self_attn_step_fused(q, k_new, v_new, self.k_pool, self.v_pool,
                                          self.tables[(step + 1) % 2], self.tables[step % 2],
                                          parents, self.B, self.M, step, scale=scale, out=out,
                                          err_flag=self.err_flag)
