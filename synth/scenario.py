"""Device-resident scenarios: weights, drafter state and per-round inputs of a
workload, materialised on the GPU with the device generator and set up
through the library's own entry points (prefill by routing every row as
committed, or import of directly drawn committed K/V).  Used by the GPU tests
and by bench.py; it never touches the oracle.
"""
from __future__ import annotations

import numpy as np

from . import workloads as wl
from . import device as sdev


class Scenario:
    def __init__(self, w: wl.Workload, device: str = "cuda", build_context: bool = True):
        import torch
        import paper_2609_14717_amd as co
        self.w, self.device = w, device
        self.pt = wl.page_table(w)
        self.dims = co.make_dims(w.S, w.B, w.Dcat, w.d, w.L, w.Hq, w.Hkv, w.hd,
                                 w.max_pages_per_seq, self.pt.size, w.dtype, w.theta)
        self.st = co.alloc_state(self.dims, self.pt, device)
        self.rt = co.alloc_route(w.S, w.B, device)
        self.wf = sdev.materialise(w, wl.spec_wf(w), device)
        self.wkv = sdev.materialise(w, wl.spec_wkv(w), device)
        self.e = sdev.materialise(w, wl.spec_e(w), device)
        self.W = co.weights(self.wf, self.wkv, self.e)
        self.ws = torch.zeros(max(co.workspace_bytes(self.dims, co.CO_WS_ROUND), 256),
                              dtype=torch.uint8, device=device)
        self.ws_project = co.workspace_bytes(self.dims, co.CO_WS_PROJECT)
        self.ctx0 = wl.initial_ctx(w)
        self.torch = torch
        self.co = co
        if build_context:
            self.build_context()

    @property
    def tdtype(self):
        return self.torch.bfloat16 if self.w.dtype == "bf16" else self.torch.float32

    def build_context(self):
        """Fill the committed cache with the initial context of every sequence."""
        w, co, torch = self.w, self.co, self.torch
        if w.ctx_mode == "direct":
            for s in range(w.S):
                n = int(self.ctx0[s])
                k = sdev.materialise(w, wl.spec_kv_direct(w, "k", s, 0, n), self.device)
                v = sdev.materialise(w, wl.spec_kv_direct(w, "v", s, 0, n), self.device)
                co.carryover_import_kv(self.dims, s, 0, k, v, self.st)
                del k, v
            self.st["ctx_len"].copy_(torch.from_numpy(self.ctx0))
            return
        n = int(self.ctx0[0])
        assert np.all(self.ctx0 == n), "projected contexts have one length"
        if n == 0:
            return
        h = torch.empty((w.S, n, w.Dcat), dtype=self.tdtype, device=self.device)
        for s in range(w.S):
            st_, shape, strides, base, sigma = wl.spec_hctx(w, s, 0, n)
            sdev.fill(h[s], w.key(st_), shape, strides, base, sigma)
        self.prefill(h)

    def prefill(self, hidden):
        """Commit every row of hidden [S][n][Dcat] at positions ctx_len.. (no E)."""
        co, torch = self.co, self.torch
        S, n = hidden.shape[0], hidden.shape[1]
        d = self.dims
        pd = co.make_dims(S, n, d.feat_dim, d.model_dim, d.num_layers, d.num_q_heads,
                          d.num_kv_heads, d.head_dim, d.max_pages_per_seq, d.num_pages,
                          d.dtype, d.rope_theta)
        rt = co.alloc_route(S, n, self.device)
        ws = torch.empty(max(co.workspace_bytes(pd, co.CO_WS_PROJECT), 256), dtype=torch.uint8,
                         device=self.device)
        co.carryover_route(pd, None, None, co.CO_ROUTE_ACCEPT_ALL, self.st, rt)
        co.carryover_project_kv(pd, self.W, hidden, rt, self.st, ws)
        return rt

    def round_inputs(self, r: int):
        """(hidden, q, draft, target, m) of round r on the device; m on the host."""
        w, torch = self.w, self.torch
        m = wl.accepted_lengths(w, r)
        draft, target = wl.tokens_for(w, r, m)
        hidden = sdev.materialise(w, wl.spec_h(w, r), self.device)
        q = sdev.materialise(w, wl.spec_q(w, r), self.device)
        return (hidden, q, torch.from_numpy(draft).to(self.device),
                torch.from_numpy(target).to(self.device), m)

    def new_output(self):
        w, torch = self.w, self.torch
        out = torch.empty((w.L, w.S, w.B, w.Hq, w.hd), dtype=self.tdtype, device=self.device)
        lse = torch.empty((w.L, w.S, w.B, w.Hq), dtype=torch.float32, device=self.device)
        return out, lse
