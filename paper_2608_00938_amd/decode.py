"""A fixed-length decode loop over the library's calls, capturable as one graph.

Per step t (beam width M_t per request) and decoder layer l:
cross-attention of the beams over the request's encoder K/V (Sec. 5.1), then
the fused paged append + self-attention (Sec. 5.2, Sec. 5.3) whose parents are
the previous step's top-k output.  After the layers, the constraint filter
(CD + GTM, Sec. 4, Sec. 5.4) of the beams' trie nodes, the beam score update (Sec. 3.1)
and top-k with k = M_{t+1} (Sec. 3.3) produce the next step's parents, prefix
scores and trie nodes on the device, so the whole loop runs without a host
round trip and is recorded as one graph (Sec. 5).

Inputs the model would compute (per-step queries, the current token's k/v and
the next-token logits, and the constraint filter's mask) are given as tensors;
this module only orchestrates: every buffer is allocated at construction and
``run`` only enqueues library calls.
"""
from __future__ import annotations

import math

import torch

from . import grace as G


class DecodeLoop:
    def __init__(self, B: int, widths, H: int, d: int, V: int, layers: int, enc_k, enc_v,
                 enc_off, step_inputs, logits, masks=None, k_final: int | None = None,
                 scale: float | None = None, gtm=None):
        """widths: beams per request at each step (M_0, ..., M_{T-1}).
        step_inputs[l][t]: dict(q_cross, q_self, k_new, v_new), each [B*M_t, H, d].
        logits[t]: [B*M_t, V]; masks[t]: packed filter words (int32 [B*M_t, ceil(V/32)]) or None.
        gtm: (GtmIndex, GtmUsers) to compute the filter of every step from the
        beams' trie nodes instead (masks is then ignored); beams start at the root.
        The top-k of step t keeps M_{t+1} beams; the last keeps k_final (default M_{T-1})."""
        self.B, self.widths, self.H, self.d, self.V, self.layers = B, tuple(widths), H, d, V, layers
        self.T = len(self.widths)
        self.enc_k, self.enc_v, self.enc_off = enc_k, enc_v, enc_off
        self.inputs, self.logits = step_inputs, logits
        self.masks = masks if masks is not None else [None] * self.T
        self.scale = 1.0 / math.sqrt(d) if scale is None else scale
        dev, dt = enc_k.device, enc_k.dtype
        Mmax = max(self.widths)
        self.caches = [G.KVCache(B, Mmax, H, d, self.T, dt, dev) for _ in range(layers)]
        self.k_out = [self.widths[t + 1] for t in range(self.T - 1)] + [k_final or self.widths[-1]]
        self.x_cross = [[torch.empty((B * M, H, d), dtype=dt, device=dev) for M in self.widths]
                        for _ in range(layers)]
        self.x_self = [[torch.empty((B * M, H, d), dtype=dt, device=dev) for M in self.widths]
                       for _ in range(layers)]
        self.prev0 = torch.zeros((B * self.widths[0],), dtype=torch.float32, device=dev)
        self.parents = [torch.empty((B, k), dtype=torch.int32, device=dev) for k in self.k_out]
        self.tokens = [torch.empty((B, k), dtype=torch.int32, device=dev) for k in self.k_out]
        self.scores = [torch.empty((B, k), dtype=torch.float32, device=dev) for k in self.k_out]
        ws = max(G.grace_beam_step_workspace_bytes(B, M, V) for M in self.widths)
        self.workspace = torch.empty((max(ws, 8),), dtype=torch.uint8, device=dev)
        self.gtm = gtm
        if gtm is not None:
            W = (V + 31) // 32
            self.masks = [torch.empty((B * M, W), dtype=torch.int32, device=dev) for M in self.widths]
            self.nodes = [torch.zeros((B * self.widths[0],), dtype=torch.int32, device=dev)] + \
                [torch.empty((B * k,), dtype=torch.int32, device=dev) for k in self.k_out]
            self.gtm_err = torch.zeros(1, dtype=torch.int32, device=dev)

    def run(self):
        """Enqueue the whole loop on the current stream."""
        B = self.B
        for t, M in enumerate(self.widths):
            M_prev = self.widths[t - 1] if t > 0 else 1
            par = self.parents[t - 1].view(-1) if t > 0 else None
            for l in range(self.layers):
                x = self.inputs[l][t]
                G.grace_cross_attn(x["q_cross"], self.enc_k, self.enc_v, self.enc_off, M,
                                   self.scale, out=self.x_cross[l][t])
                self.caches[l].append_attend_dyn(t, x["q_self"], x["k_new"], x["v_new"], par,
                                                 M_prev, M, self.scale, out=self.x_self[l][t])
            prev = self.prev0 if t == 0 else self.scores[t - 1].view(-1)
            if self.gtm is not None:
                index, users = self.gtm
                G.grace_gtm_mask(index, users, self.nodes[t], B, M, mask=self.masks[t],
                                 err_flag=self.gtm_err)
            # score update + top-k in one call: no [B*M, V] candidate array
            G.grace_beam_step(self.logits[t], prev, B, M, self.k_out[t], mask=self.masks[t],
                              parents=self.parents[t], tokens=self.tokens[t],
                              scores=self.scores[t], workspace=self.workspace)
            if self.gtm is not None:
                G.grace_trie_advance(self.gtm[0], self.nodes[t], self.parents[t].view(-1),
                                     self.tokens[t].view(-1), B, M, self.k_out[t],
                                     node_next=self.nodes[t + 1], err_flag=self.gtm_err)

    def capture(self, stream) -> "G.Graph":
        """Record run() on ``stream`` (not the null stream) as one graph."""
        return G.capture(self.run, stream)
