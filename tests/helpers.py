"""Shared pieces of the parity tests: oracle-side construction of a workload's
state and rounds from the host generator, the comparison rules, and reading
the GPU's paged cache back by logical position."""
from __future__ import annotations

import numpy as np

import oracle
import synth
from synth import workloads as wl

TOL = {"bf16": 2e-2, "f32": 1e-4}


def host(w, spec, dtype=None):
    return synth.to_f64(wl.host_block(w, spec, dtype), dtype or w.dtype)


class OracleRun:
    """The oracle's view of a workload: weights, logical state, rounds."""

    def __init__(self, w, seqs=None, store=np.float64):
        self.w = w
        self.seqs = list(range(w.S)) if seqs is None else list(seqs)
        self.WF = host(w, wl.spec_wf(w))
        self.WKV = host(w, wl.spec_wkv(w))
        self.E = host(w, wl.spec_e(w))
        self.pt = wl.page_table(w)
        self.num_pages = self.pt.size
        self.st = oracle.State(w.S, w.L, w.Hkv, w.hd, store)
        self.ctx0 = wl.initial_ctx(w)
        self._carry = np.zeros(w.S, np.int32)
        for s in self.seqs:
            n = int(self.ctx0[s])
            if w.ctx_mode == "direct":
                k = host(w, wl.spec_kv_direct(w, "k", s, 0, n)).transpose(0, 2, 1, 3)
                v = host(w, wl.spec_kv_direct(w, "v", s, 0, n)).transpose(0, 2, 1, 3)
                self.st.set_committed(s, k, v)
            elif n:
                h = host(w, wl.spec_hctx(w, s, 0, n))
                k, v = oracle.project(h, self.E, np.zeros(n, bool), self.WF, self.WKV,
                                      np.arange(n), w.L, w.Hkv, w.hd, w.theta)
                self.st.commit_and_replace(s, k, v, k[:0], v[:0])

    def ctx_len(self):
        c = self.ctx0.copy()
        for s in self.seqs:
            c[s] = self.st.ck[s].shape[1]
        return c

    def carry_len(self):
        c = self._carry.copy()
        for s in self.seqs:
            c[s] = self.st.uk[s].shape[1]
        return c

    def round(self, r, mode="carry", attend=True, layers=None):
        w = self.w
        m = wl.accepted_lengths(w, r)
        draft, target = wl.tokens_for(w, r, m)
        rr = oracle.route(draft, target, self.ctx_len(), self.carry_len(), self.pt,
                          self.num_pages, mode)
        H = host(w, wl.spec_h(w, r))
        oracle.round_update(self.st, rr, H, self.E, self.WF, self.WKV, w.theta, mode,
                            seqs=self.seqs)
        if not attend:
            return rr, None, None
        Q = host(w, wl.spec_q(w, r))
        O, LSE = oracle.attend_state(self.st, Q, w.Hq, w.theta, seqs=self.seqs, layers=layers)
        return rr, O, LSE


def head_err(g, r):
    """max over head vectors of ||g - r||_inf / max(||r||_inf, 1e-30)."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    num = np.abs(g - r).max(axis=-1)
    den = np.maximum(np.abs(r).max(axis=-1), 1e-30)
    e = num / den
    return float(e.max()) if e.size else 0.0


def assert_heads_close(g, r, tol, what):
    assert np.all(np.isfinite(g)), f"{what}: non-finite GPU values"
    e = head_err(g, r)
    assert e <= tol, f"{what}: max head-vector rel err {e:.3e} > {tol}"
    return e


def to_np(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def gather_committed(st, pt, s, layer, t0, t1):
    """GPU committed K, V of sequence s, positions t0..t1-1: [n][Hkv][hd] each."""
    import torch
    pos = torch.arange(t0, t1, device=st["k_cache"].device)
    pages = st["page_table"][s][pos // 16].long()
    slots = (pos % 16).long()
    k = st["k_cache"][layer][pages, :, slots, :]                 # [n][Hkv][hd]
    v = st["v_cache"][layer][pages, :, :, slots]                 # [n][Hkv][hd]
    return to_np(k), to_np(v)


def gather_carry(st, s, layer, n):
    """GPU carry K, V of sequence s, rows 0..n-1: [n][Hkv][hd]."""
    import torch
    r = torch.arange(n, device=st["k_carry"].device)
    k = st["k_carry"][layer, s][r // 16, :, r % 16, :]
    v = st["v_carry"][layer, s][r // 16, :, :, r % 16]
    return to_np(k), to_np(v)
