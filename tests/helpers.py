"""Shared pieces of the parity tests: oracle-side construction of a workload's
state and rounds from the host generator, the comparison rules, and reading
the GPU's paged cache back by logical position."""
from __future__ import annotations

import numpy as np

import oracle
import synth
from synth import workloads as wl

TOL = {"bf16": 2e-2, "f32": 1e-4}


def host(w, spec, dtype=None, out=np.float64):
    """A described block, widened exactly to ``out`` (float64, or float32 for
    bf16/fp32 data that a float32 store keeps exactly)."""
    if out == np.float32:
        dt = dtype or w.dtype
        return wl.host_block(w, spec, "f32" if dt == "f32" else "bf16_f32")
    raw = wl.host_block(w, spec, dtype)
    return synth.to_f64(raw, dtype or w.dtype)


def seq_block(w, spec, axis, seqs):
    """A described block with only the rows ``seqs`` of axis ``axis`` drawn (others zero)."""
    st_, shape, strides, base, sigma = spec
    if len(seqs) == shape[axis]:
        return host(w, spec)
    out = np.zeros(shape, np.float64)
    sub = tuple(1 if i == axis else n for i, n in enumerate(shape))
    for s in seqs:
        blk = host(w, (st_, sub, strides, base + s * strides[axis], sigma))
        idx = [slice(None)] * len(shape)
        idx[axis] = slice(s, s + 1)
        out[tuple(idx)] = blk
    return out


def _rows_first(spec):
    """The same block described as [L][n][Hkv][hd] instead of [L][Hkv][n][hd]
    (every element keeps its logical index, so its value)."""
    st_, shape, strides, base, sigma = spec
    o = (0, 2, 1, 3)
    return st_, tuple(shape[i] for i in o), tuple(strides[i] for i in o), base, sigma


class OracleTrain:
    """The oracle's view of the training-shaped forward (Algorithm 2, second
    pass) for a sample of anchored blocks (virtual sequences)."""

    def __init__(self, w, sample):
        self.w = w
        S, A, B = w.S, w.anchors, w.B
        V = S * A
        self.sample = list(sample)
        self.WF = host(w, wl.spec_wf(w))
        self.WKV = host(w, wl.spec_wkv(w))
        self.E = host(w, wl.spec_e(w))
        self.a, self.u, self.a2 = wl.anchors(w)
        self.pt = wl.page_table(w)
        self.vpt = np.repeat(self.pt, A, axis=0)
        # the recorded responses, projected without E at positions 0..seq_len-1
        self.parent = {}
        for s in sorted({v // A for v in self.sample}):
            h = host(w, wl.spec_hctx(w, s, 0, w.seq_len))
            self.parent[s] = oracle.project(h, self.E, np.zeros(w.seq_len, bool), self.WF,
                                            self.WKV, np.arange(w.seq_len), w.L, w.Hkv, w.hd,
                                            w.theta)
        self.st = oracle.State(V, w.L, w.Hkv, w.hd)
        a2 = self.a2.ravel()
        for v in self.sample:
            k, vv = self.parent[v // A]
            n = int(a2[v])
            self.st.set_committed(v, k[:n].transpose(1, 0, 2, 3), vv[:n].transpose(1, 0, 2, 3))
        m = (B - self.u.ravel()).astype(np.int32)
        draft, target = wl.tokens_for(w, 0, m)
        self.rr = oracle.route(draft, target, self.a.ravel() + 1, np.zeros(V, np.int32), self.vpt,
                               self.pt.size, "carry_only")
        H = seq_block(w, wl.spec_h(w, 0, S=V), 0, self.sample)
        oracle.round_update(self.st, self.rr, H, self.E, self.WF, self.WKV, w.theta, "carry_only",
                            seqs=self.sample)
        Q = seq_block(w, wl.spec_q(w, 0, S=V), 1, self.sample)
        self.O, self.LSE = oracle.attend_state(self.st, Q, w.Hq, w.theta, seqs=self.sample)


class OracleRun:
    """The oracle's view of a workload: weights, logical state, rounds."""

    def __init__(self, w, seqs=None, store=np.float64, separate_projector=False, z_norm=False,
                 k_norm=False):
        self.w = w
        self.seqs = list(range(w.S)) if seqs is None else list(seqs)
        self.WF = host(w, wl.spec_wf(w))
        self.WFC = host(w, wl.spec_wfc(w)) if separate_projector else None
        self.ZN = (wl.znorm_gain_host(w, host(w, wl.spec_znorm(w), dtype="f32", out=np.float32))
                   .astype(np.float64) if z_norm else None)
        self.KN = (wl.knorm_gain_host(w, host(w, wl.spec_knorm(w), dtype="f32", out=np.float32))
                   .astype(np.float64) if k_norm else None)
        self.WKV = host(w, wl.spec_wkv(w))
        self.E = host(w, wl.spec_e(w))
        self.pt = wl.page_table(w)
        self.num_pages = self.pt.size
        self.st = oracle.State(w.S, w.L, w.Hkv, w.hd, store)
        self.ctx0 = wl.initial_ctx(w)
        # integer lengths of every sequence (the float state covers self.seqs only)
        self._ctx = self.ctx0.astype(np.int32).copy()
        self._carry = np.zeros(w.S, np.int32)
        for s in self.seqs:
            n = int(self.ctx0[s])
            if w.ctx_mode == "direct":
                wide = np.float32 if store == np.float32 else np.float64
                k = host(w, _rows_first(wl.spec_kv_direct(w, "k", s, 0, n)), out=wide)
                v = host(w, _rows_first(wl.spec_kv_direct(w, "v", s, 0, n)), out=wide)
                self.st.set_committed(s, k, v)
            elif n:
                h = host(w, wl.spec_hctx(w, s, 0, n))
                k, v = oracle.project(h, self.E, np.zeros(n, bool), self.WF, self.WKV,
                                      np.arange(n), w.L, w.Hkv, w.hd, w.theta,
                                      z_norm=self.ZN, k_norm=self.KN)
                self.st.commit_and_replace(s, k, v, k[:0], v[:0])

    def ctx_len(self):
        for s in self.seqs:
            assert self.st.ck[s].shape[1] == self._ctx[s]
        return self._ctx.copy()

    def carry_len(self):
        for s in self.seqs:
            assert self.st.uk[s].shape[1] == self._carry[s]
        return self._carry.copy()

    def seq_block(self, spec, axis):
        return seq_block(self.w, spec, axis, self.seqs)

    def round(self, r, mode="carry", attend=True, layers=None, m=None, bits=None):
        """One round; with ``bits`` the route takes the verifier's accept
        decisions [S][B] instead of the tokens."""
        w = self.w
        if bits is not None:
            rr = oracle.route(bits, None, self.ctx_len(), self.carry_len(), self.pt,
                              self.num_pages, mode, accept="bits")
        else:
            m = wl.accepted_lengths(w, r) if m is None else np.asarray(m, np.int32)
            draft, target = wl.tokens_for(w, r, m)
            rr = oracle.route(draft, target, self.ctx_len(), self.carry_len(), self.pt,
                              self.num_pages, mode)
        H = self.seq_block(wl.spec_h(w, r), 0)
        oracle.round_update(self.st, rr, H, self.E, self.WF, self.WKV, w.theta, mode,
                            seqs=self.seqs, WF_carry=self.WFC, z_norm=self.ZN,
                            k_norm=self.KN)
        self._ctx = np.asarray(rr["ctx_len"], np.int32).copy()
        self._carry = np.asarray(rr["carry_len"], np.int32).copy()
        if not attend:
            return rr, None, None
        Q = self.seq_block(wl.spec_q(w, r), 1)
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


def compare_round(sc, orc, rr, O, LSE, out, lse, rt, seqs, what):
    w = sc.w
    tol = TOL[w.dtype]
    # integer results: bit-exact
    np.testing.assert_array_equal(rt["accept_len"].cpu().numpy()[seqs], rr["accept_len"][seqs])
    np.testing.assert_array_equal(rt["row_pos"].cpu().numpy()[seqs], rr["row_pos"][seqs])
    np.testing.assert_array_equal(rt["row_dst"].cpu().numpy()[seqs], rr["row_dst"][seqs])
    np.testing.assert_array_equal(sc.st["ctx_len"].cpu().numpy()[seqs], rr["ctx_len"][seqs])
    np.testing.assert_array_equal(sc.st["carry_len"].cpu().numpy()[seqs], rr["carry_len"][seqs])
    # attention
    g = to_np(out)
    gl = lse.cpu().numpy().astype(np.float64)
    for s in seqs:
        assert_heads_close(g[:, s], O[:, s], tol, f"{what} O seq {s}")
        err = np.abs(gl[:, s] - LSE[:, s]).max()
        assert err <= tol, f"{what} LSE seq {s}: {err}"
    # rows written this round
    for s in seqs:
        m = int(rr["accept_len"][s])
        p0 = int(rr["ctx_len"][s]) - m
        for layer in range(w.L):
            if m:
                gk, gv = gather_committed(sc.st, sc.pt, s, layer, p0, p0 + m)
                assert_heads_close(gk, orc.st.ck[s][layer, p0:p0 + m], tol, f"{what} C_k s{s}")
                assert_heads_close(gv, orc.st.cv[s][layer, p0:p0 + m], tol, f"{what} C_v s{s}")
            u = int(rr["carry_len"][s])
            if u:
                gk, gv = gather_carry(sc.st, s, layer, u)
                assert_heads_close(gk, orc.st.uk[s][layer], tol, f"{what} U_k s{s}")
                assert_heads_close(gv, orc.st.uv[s][layer], tol, f"{what} U_v s{s}")
