"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types an oracle formula and compares it with itself: each
check is a closed form, an invariant stated by the paper, a textbook special
case, or a brute-force recomputation by a different route on tiny inputs.
The paper prints no worked example for this computation, so there is no
value from the paper itself to compare against.
"""
import math

import numpy as np
import pytest

import oracle
from synth import workloads as wl

RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------- RoPE

def test_rope_position_zero_is_identity():
    x = RNG.standard_normal((5, 64))
    np.testing.assert_array_equal(oracle.rope(x, 0, 1e4), x)


def test_rope_two_dims_is_plane_rotation():
    # hd = 2: one pair with inverse frequency theta^0 = 1 -> rotation by angle p
    for p in (1, 7, 123):
        y = oracle.rope(np.array([1.0, 0.0]), p, 1e4)
        np.testing.assert_allclose(y, [math.cos(p), math.sin(p)], rtol=0, atol=1e-15)
        y = oracle.rope(np.array([0.0, 1.0]), p, 1e4)
        np.testing.assert_allclose(y, [-math.sin(p), math.cos(p)], rtol=0, atol=1e-15)


def test_rope_pairing_and_frequencies():
    # hd = 4, theta = 100: pair (0, 2) turns at rate 1, pair (1, 3) at 100^(-2/4) = 0.1
    p = 3
    y = oracle.rope(np.array([1.0, 0, 0, 0]), p, 100.0)
    np.testing.assert_allclose(y, [math.cos(p), 0, math.sin(p), 0], atol=1e-15)
    y = oracle.rope(np.array([0, 1.0, 0, 0]), p, 100.0)
    np.testing.assert_allclose(y, [0, math.cos(0.1 * p), 0, math.sin(0.1 * p)], atol=1e-15)


def test_rope_norm_and_relative_position():
    q = RNG.standard_normal(128)
    k = RNG.standard_normal(128)
    for p, pp in ((5, 3), (3000, 17), (40000, 39999)):
        rq, rk = oracle.rope(q, p, 1e6), oracle.rope(k, pp, 1e6)
        assert abs(np.linalg.norm(rq) - np.linalg.norm(q)) < 1e-12
        # <R(q,p), R(k,p')> depends only on p - p'
        np.testing.assert_allclose(rq @ rk, oracle.rope(q, p - pp, 1e6) @ k, rtol=1e-10)


# ------------------------------------------------------------- attention

def test_attend_single_key_returns_its_value():
    q, k, v = RNG.standard_normal((3, 64)), RNG.standard_normal((1, 64)), RNG.standard_normal((1, 64))
    o, lse = oracle.attend(q, np.arange(3), k, v, 1e4)
    np.testing.assert_allclose(o, np.repeat(v, 3, axis=0), rtol=0, atol=1e-14)
    rq = oracle.rope(q, np.arange(3), 1e4)
    np.testing.assert_allclose(lse, rq @ k[0] / 8.0, rtol=1e-13)


def test_attend_zero_query_and_identical_keys_give_mean():
    v = RNG.standard_normal((9, 64))
    o, lse = oracle.attend(np.zeros((2, 64)), [0, 1], RNG.standard_normal((9, 64)), v, 1e4)
    np.testing.assert_allclose(o, np.repeat(v.mean(0, keepdims=True), 2, 0), atol=1e-14)
    np.testing.assert_allclose(lse, math.log(9), rtol=1e-14)
    k = np.repeat(RNG.standard_normal((1, 64)), 9, 0)
    o, _ = oracle.attend(RNG.standard_normal((2, 64)), [4, 5], k, v, 1e4)
    np.testing.assert_allclose(o, np.repeat(v.mean(0, keepdims=True), 2, 0), atol=1e-13)


def test_attend_two_keys_closed_form_scale():
    # q at position 0 (no rotation), keys e0*a and e0*b: logits a/sqrt(hd), b/sqrt(hd)
    hd = 16
    q = np.zeros((1, hd)); q[0, 0] = 1.0
    k = np.zeros((2, hd)); k[0, 0] = 3.0; k[1, 0] = -1.0
    # keys are stored rotated; position 0 keeps them as they are
    v = RNG.standard_normal((2, hd))
    o, lse = oracle.attend(q, [0], k, v, 1e4)
    a, b = 3.0 / 4.0, -1.0 / 4.0
    w0 = 1.0 / (1.0 + math.exp(b - a))
    np.testing.assert_allclose(o[0], w0 * v[0] + (1 - w0) * v[1], rtol=1e-14)
    np.testing.assert_allclose(lse[0], math.log(math.exp(a) + math.exp(b)), rtol=1e-14)


def test_attend_one_dominant_logit_selects_value():
    hd = 64
    q = np.zeros((1, hd)); q[0, 3] = 1.0
    k = RNG.standard_normal((20, hd)) * 0.01
    k[11, 3] = 2000.0
    v = RNG.standard_normal((20, hd))
    o, _ = oracle.attend(q, [0], k, v, 1e4)
    np.testing.assert_allclose(o[0], v[11], rtol=0, atol=1e-12)


def test_attend_empty_key_set():
    o, lse = oracle.attend(RNG.standard_normal((4, 64)), np.arange(4), np.zeros((0, 64)),
                           np.zeros((0, 64)), 1e4)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


def test_attend_shift_of_all_positions_and_key_order_invariance():
    hd, n = 64, 37
    q = RNG.standard_normal((4, hd))
    kraw = RNG.standard_normal((n, hd))
    v = RNG.standard_normal((n, hd))
    kpos = np.arange(n)
    o1, l1 = oracle.attend(q, 40 + np.arange(4), oracle.rope(kraw, kpos, 1e4), v, 1e4)
    d = 1234
    o2, l2 = oracle.attend(q, 40 + d + np.arange(4), oracle.rope(kraw, kpos + d, 1e4), v, 1e4)
    np.testing.assert_allclose(o1, o2, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(l1, l2, rtol=1e-10)
    perm = RNG.permutation(n)
    o3, l3 = oracle.attend(q, 40 + np.arange(4), oracle.rope(kraw, kpos, 1e4)[perm], v[perm], 1e4)
    np.testing.assert_allclose(o1, o3, rtol=1e-12, atol=1e-14)


def _merge(parts):
    """Closed-form merge of softmax partials (O_i, LSE_i) over disjoint key sets."""
    lses = np.array([p[1] for p in parts])
    M = lses.max(axis=0)
    M = np.where(np.isneginf(M), 0.0, M)
    w = np.exp(lses - M)
    O = sum(wi[:, None] * p[0] for wi, p in zip(w, parts))
    den = w.sum(axis=0)
    return O / den[:, None], M + np.log(den)


def test_concatenated_context_equals_two_segment_merge():
    """Attention over [C;U] equals the softmax merge of attention over C and over U,
    including arbitrary splits of C (with empty pieces)."""
    hd = 64
    q = RNG.standard_normal((32, hd))
    qpos = 500 + np.arange(32)
    C = oracle.rope(RNG.standard_normal((300, hd)), np.arange(300), 1e4)
    U = oracle.rope(RNG.standard_normal((9, hd)), 300 + np.arange(9), 1e4)
    VC, VU = RNG.standard_normal((300, hd)), RNG.standard_normal((9, hd))
    full = oracle.attend(q, qpos, np.concatenate([C, U]), np.concatenate([VC, VU]), 1e4)
    two = _merge([oracle.attend(q, qpos, C, VC, 1e4), oracle.attend(q, qpos, U, VU, 1e4)])
    np.testing.assert_allclose(two[0], full[0], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(two[1], full[1], rtol=1e-12)
    cuts = [0, 0, 17, 128, 128, 299, 300]
    parts = [oracle.attend(q, qpos, C[a:b], VC[a:b], 1e4) for a, b in zip(cuts[:-1], cuts[1:])]
    parts.append(oracle.attend(q, qpos, U, VU, 1e4))
    many = _merge(parts)
    np.testing.assert_allclose(many[0], full[0], rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------- projection

def _brute_project_row(h, e, add, WF, WKV, pos, L, Hkv, hd, theta):
    """One row by plain Python loops, slicing the weights per (layer, K|V, head)."""
    Dcat, d = len(h), WF.shape[0]
    x = [h[c] + (e[c] if add else 0.0) for c in range(Dcat)]
    z = [sum(WF[r][c] * x[c] for c in range(Dcat)) for r in range(d)]
    K = np.zeros((L, Hkv, hd)); V = np.zeros((L, Hkv, hd))
    for layer in range(L):
        for kind in range(2):
            for g in range(Hkv):
                base = ((layer * 2 + kind) * Hkv + g) * hd
                vec = [sum(WKV[base + t][r] * z[r] for r in range(d)) for t in range(hd)]
                if kind == 0:
                    half = hd // 2
                    out = [0.0] * hd
                    for i in range(half):
                        ang = pos * theta ** (-2.0 * i / hd)
                        out[i] = vec[i] * math.cos(ang) - vec[i + half] * math.sin(ang)
                        out[i + half] = vec[i + half] * math.cos(ang) + vec[i] * math.sin(ang)
                    K[layer, g] = out
                else:
                    V[layer, g] = vec
    return K, V


def test_project_matches_loop_brute_force():
    L, Hkv, hd, Dcat, d = 2, 2, 8, 12, 6
    M = 5
    H = RNG.standard_normal((M, Dcat)); E = RNG.standard_normal(Dcat)
    WF = RNG.standard_normal((d, Dcat)); WKV = RNG.standard_normal((2 * L * Hkv * hd, d))
    add = np.array([0, 0, 1, 1, 1], bool)
    pos = np.array([3, 4, 5, 6, 70])
    K, V = oracle.project(H, E, add, WF, WKV, pos, L, Hkv, hd, 1e4)
    for r in range(M):
        bk, bv = _brute_project_row(H[r], E, add[r], WF, WKV, pos[r], L, Hkv, hd, 1e4)
        np.testing.assert_allclose(K[r], bk, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(V[r], bv, rtol=1e-12, atol=1e-12)


def test_e_carry_placement_by_linearity():
    """(carry K/V of a row) - (committed-path K/V of the same row and position)
    = RoPE(W_K W_F E) and W_V W_F E; E = 0 makes them identical (Eq. 2)."""
    L, Hkv, hd, Dcat, d = 2, 2, 16, 48, 32
    H = RNG.standard_normal((4, Dcat)); E = RNG.standard_normal(Dcat)
    WF = RNG.standard_normal((d, Dcat)); WKV = RNG.standard_normal((2 * L * Hkv * hd, d))
    pos = np.array([10, 11, 12, 13])
    kc, vc = oracle.project(H, E, np.ones(4, bool), WF, WKV, pos, L, Hkv, hd, 1e4)
    k0, v0 = oracle.project(H, E, np.zeros(4, bool), WF, WKV, pos, L, Hkv, hd, 1e4)
    fe = WF @ E
    for layer in range(L):
        for g in range(Hkv):
            wk = WKV[((layer * 2 + 0) * Hkv + g) * hd:((layer * 2 + 0) * Hkv + g + 1) * hd]
            wv = WKV[((layer * 2 + 1) * Hkv + g) * hd:((layer * 2 + 1) * Hkv + g + 1) * hd]
            for r in range(4):
                np.testing.assert_allclose(kc[r, layer, g] - k0[r, layer, g],
                                           oracle.rope(wk @ fe, pos[r], 1e4), rtol=1e-9, atol=1e-9)
                np.testing.assert_allclose(vc[r, layer, g] - v0[r, layer, g], wv @ fe,
                                           rtol=1e-9, atol=1e-9)
    kz, vz = oracle.project(H, np.zeros(Dcat), np.ones(4, bool), WF, WKV, pos, L, Hkv, hd, 1e4)
    np.testing.assert_array_equal(kz, k0)
    np.testing.assert_array_equal(vz, v0)


# ------------------------------------------------------------------ route

def test_route_recovers_constructed_accept_lengths_exhaustively():
    """Tokens are built from a chosen m (draft == target on 0..m-1, differs at m);
    greedy verification must return exactly m, for every m in 0..B."""
    for B in (1, 4, 8, 16):
        w = wl.TINY.replace(B=B, S=B + 1)
        m = np.arange(B + 1, dtype=np.int32)
        draft, target = wl.tokens_for(w, 0, m)
        for s in range(B + 1):
            assert oracle.accept_len(draft[s], target[s]) == m[s]


def test_route_slots_and_lengths():
    S, B, P = 3, 8, 10
    pt = np.array([RNG.permutation(40)[:P] for _ in range(S)], np.int32)
    m = np.array([0, 5, 8], np.int32)
    w = wl.TINY.replace(B=B, S=S)
    draft, target = wl.tokens_for(w, 0, m)
    ctx = np.array([0, 37, 140], np.int32)
    r = oracle.route(draft, target, ctx, np.array([3, 3, 3]), pt, 40)
    np.testing.assert_array_equal(r["accept_len"], m)
    np.testing.assert_array_equal(r["ctx_len"], ctx + m)
    np.testing.assert_array_equal(r["carry_len"], B - m)
    # physical slot of logical position t: page_table[t // 16] * 16 + t % 16, as a dense map
    for s in range(S):
        phys = np.concatenate([np.arange(16) + 16 * pt[s][p] for p in range(P)])
        for j in range(B):
            if j < m[s]:
                assert r["row_dst"][s, j] == phys[ctx[s] + j]
            else:
                assert r["row_dst"][s, j] == -1 - (j - m[s])
    rb = oracle.route(draft, target, ctx, np.array([3, 3, 3]), pt, 40, mode="baseline")
    assert np.all(rb["carry_len"] == 0) and np.all(rb["row_dst"][1, 5:] == oracle.SKIP)
    ra = oracle.route(draft, target, ctx, np.array([3, 3, 3]), pt, 40, mode="accept_all")
    np.testing.assert_array_equal(ra["ctx_len"], ctx + B)


def test_route_errors_leave_sequence_unchanged():
    S, B, P = 3, 8, 4
    pt = np.tile(np.arange(P, dtype=np.int32), (S, 1))
    pt[2, 1] = 99                                    # out of the pool of 40 pages
    w = wl.TINY.replace(B=B, S=S)
    draft, target = wl.tokens_for(w, 0, np.array([8, 8, 8], np.int32))
    ctx = np.array([P * 16 - B + 1, -1, 10], np.int32)
    r = oracle.route(draft, target, ctx, np.array([2, 2, 2]), pt, 40)
    assert list(r["status"]) == [oracle.ERR_CAPACITY, oracle.ERR_LENGTH, oracle.ERR_PAGE_RANGE]
    np.testing.assert_array_equal(r["ctx_len"], ctx)
    np.testing.assert_array_equal(r["carry_len"], [2, 2, 2])
    assert np.all(r["row_dst"] == oracle.SKIP)


# ------------------------------------------------------------ whole rounds

def _tiny_setup(S=2, B=4, Dcat=12, d=8, L=2, Hq=4, Hkv=2, hd=8, seed=7):
    rng = np.random.default_rng(seed)
    return dict(S=S, B=B, Dcat=Dcat, d=d, L=L, Hq=Hq, Hkv=Hkv, hd=hd,
                WF=rng.standard_normal((d, Dcat)) * 0.3,
                WKV=rng.standard_normal((2 * L * Hkv * hd, d)) * 0.3,
                E=rng.standard_normal(Dcat), rng=rng)


def _run_incremental(t, ctx0_h, rounds, mode="carry", poison=False):
    """Drive the oracle through rounds; returns per-round (route, O, LSE)."""
    S, B, L, Hkv, hd, Hq = t["S"], t["B"], t["L"], t["Hkv"], t["hd"], t["Hq"]
    st = oracle.State(S, L, Hkv, hd)
    pt = np.tile(np.arange(64, dtype=np.int32), (S, 1))
    for s in range(S):
        n = len(ctx0_h[s])
        k, v = oracle.project(ctx0_h[s], t["E"], np.zeros(n, bool), t["WF"], t["WKV"],
                              np.arange(n), L, Hkv, hd, 1e4)
        st.commit_and_replace(s, k, v, k[:0], v[:0])
    outs = []
    for rnd in rounds:
        if poison:
            for s in range(S):
                st.uk[s][:] = np.nan
                st.uv[s][:] = np.nan
        r = oracle.route(rnd["draft"], rnd["target"], st.ctx_len(), st.carry_len(), pt, 64, mode)
        oracle.round_update(st, r, rnd["H"], t["E"], t["WF"], t["WKV"], 1e4, mode)
        O, LSE = oracle.attend_state(st, rnd["Q"], Hq, 1e4)
        outs.append((r, O, LSE, st.ctx_len(), st.carry_len()))
    return outs


def _make_rounds(t, n_rounds, ms):
    S, B, Dcat, L, Hq, hd = t["S"], t["B"], t["Dcat"], t["L"], t["Hq"], t["hd"]
    rng = t["rng"]
    out = []
    for r in range(n_rounds):
        m = np.array(ms[r], np.int32)
        target = rng.integers(0, 50, (S, B))
        draft = target.copy()
        for s in range(S):
            if m[s] < B:
                draft[s, m[s]] = (target[s, m[s]] + 1) % 50
        out.append(dict(draft=draft, target=target, m=m,
                        H=rng.standard_normal((S, B, Dcat)),
                        Q=rng.standard_normal((L, S, B, Hq, hd))))
    return out


def _brute_force_rounds(t, ctx0_h, rounds):
    """Full-history recomputation: every round, re-project every row ever
    committed from its stored state and position, plus the current carried rows,
    then attend with a dense mask over all rows ever seen and an unshifted exp."""
    S, B, L, Hkv, hd, Hq = t["S"], t["B"], t["L"], t["Hkv"], t["hd"], t["Hq"]
    G = Hq // Hkv
    hist = [[(ctx0_h[s][j], j, "acc", -1) for j in range(len(ctx0_h[s]))] for s in range(S)]
    res = []
    for ri, rnd in enumerate(rounds):
        for s in range(S):
            p0 = sum(1 for h in hist[s] if h[2] == "acc")
            m = 0
            while m < B and rnd["draft"][s][m] == rnd["target"][s][m]:
                m += 1
            for j in range(B):
                hist[s].append((rnd["H"][s][j], p0 + j, "acc" if j < m else "rej", ri))
        O = np.zeros((L, S, B, Hq, hd)); LSE = np.zeros((L, S, B, Hq))
        for s in range(S):
            rows = hist[s]
            ctx = sum(1 for h in rows if h[2] == "acc")
            # a row is visible iff committed, or rejected in *this* round
            vis = [h[2] == "acc" or h[3] == ri for h in rows]
            KV = [_brute_project_row(h[0], t["E"], h[2] == "rej", t["WF"], t["WKV"], h[1], L,
                                     Hkv, hd, 1e4) for h in rows]
            for layer in range(L):
                for i in range(B):
                    for h in range(Hq):
                        g = h // G
                        q = rnd["Q"][layer, s, i, h]
                        qp = ctx + i
                        half = hd // 2
                        rq = np.zeros(hd)
                        for a in range(half):
                            ang = qp * 1e4 ** (-2.0 * a / hd)
                            rq[a] = q[a] * math.cos(ang) - q[a + half] * math.sin(ang)
                            rq[a + half] = q[a + half] * math.cos(ang) + q[a] * math.sin(ang)
                        num = np.zeros(hd); den = 0.0
                        for kvr, ok in zip(KV, vis):
                            if not ok:
                                continue
                            wgt = math.exp(float(rq @ kvr[0][layer, g]) / math.sqrt(hd))
                            num += wgt * kvr[1][layer, g]
                            den += wgt
                        O[layer, s, i, h] = num / den
                        LSE[layer, s, i, h] = math.log(den)
        res.append((O, LSE))
    return res


def test_whole_rounds_match_full_history_brute_force():
    t = _tiny_setup()
    ctx0 = [t["rng"].standard_normal((n, t["Dcat"])) for n in (3, 6)]
    ms = [[1, 4], [0, 2], [4, 0], [2, 3], [4, 4], [3, 1]]
    rounds = _make_rounds(t, 6, ms)
    inc = _run_incremental(t, ctx0, rounds)
    bf = _brute_force_rounds(t, ctx0, rounds)
    for r, (a, b) in enumerate(zip(inc, bf)):
        np.testing.assert_array_equal(a[0]["accept_len"], ms[r])
        np.testing.assert_allclose(a[1], b[0], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(a[2], b[1], rtol=1e-12, atol=1e-12)


def test_lengths_over_a_chain():
    t = _tiny_setup(B=4)
    ctx0 = [t["rng"].standard_normal((n, t["Dcat"])) for n in (2, 5)]
    ms = t["rng"].integers(0, 5, (12, 2))
    outs = _run_incremental(t, ctx0, _make_rounds(t, 12, ms))
    for r, o in enumerate(outs):
        np.testing.assert_array_equal(o[3], np.array([2, 5]) + ms[: r + 1].sum(0))
        np.testing.assert_array_equal(o[4], 4 - ms[r])
        assert np.all(o[4] <= 4)


def test_zero_rejected_equals_baseline_exactly():
    t = _tiny_setup()
    ctx0 = [t["rng"].standard_normal((n, t["Dcat"])) for n in (3, 6)]
    rounds = _make_rounds(t, 4, [[4, 4]] * 4)
    a = _run_incremental(t, ctx0, rounds, "carry")
    b = _run_incremental(t, ctx0, rounds, "baseline")
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x[1], y[1])
        np.testing.assert_array_equal(x[2], y[2])
        assert np.all(x[4] == 0)


def test_carry_segment_is_replaced_never_read_stale():
    t = _tiny_setup()
    ctx0 = [t["rng"].standard_normal((n, t["Dcat"])) for n in (3, 6)]
    rounds = _make_rounds(t, 5, [[1, 2], [0, 4], [3, 1], [2, 2], [0, 0]])
    a = _run_incremental(t, ctx0, rounds, "carry", poison=False)
    b = _run_incremental(t, ctx0, rounds, "carry", poison=True)
    for x, y in zip(a, b):
        assert np.all(np.isfinite(y[1]))
        np.testing.assert_array_equal(x[1], y[1])


def test_baseline_differs_when_rows_are_rejected():
    t = _tiny_setup()
    ctx0 = [t["rng"].standard_normal((n, t["Dcat"])) for n in (3, 6)]
    rounds = _make_rounds(t, 2, [[1, 2], [0, 3]])
    a = _run_incremental(t, ctx0, rounds, "carry")
    b = _run_incremental(t, ctx0, rounds, "baseline")
    assert np.abs(a[0][1] - b[0][1]).max() > 1e-3


# ------------------------------------------------ stochastic verification (T = 1)

def test_accept_bits_give_the_run_before_the_first_rejection():
    """With accept decisions made by the verifier (rejection sampling at T = 1),
    m is the number of leading accepted positions, whatever follows the first
    rejection; bits built from a chosen m return exactly m, for every m."""
    for B in (1, 4, 8, 16):
        for m in range(B + 1):
            for _ in range(3):
                bits = RNG.integers(0, 2, B)
                bits[:m] = RNG.integers(1, 5, m)       # any nonzero value accepts
                if m < B:
                    bits[m] = 0
                assert oracle.accept_len_bits(bits) == m


def test_accept_bits_route_equals_token_route():
    """Greedy verification is the special case whose accept decision at each
    position is 'draft token equals target token': routing by those decisions
    gives exactly the token route (descriptors, lengths, status)."""
    w = wl.TINY.replace(B=8, S=9, rounds=2)
    pt = wl.page_table(w)
    ctx = wl.initial_ctx(w)
    m = np.arange(9, dtype=np.int32)
    draft, target = wl.tokens_for(w, 0, m)
    a = oracle.route(draft, target, ctx, np.zeros(9, np.int32), pt, pt.size)
    b = oracle.route((draft == target).astype(np.int32), None, ctx, np.zeros(9, np.int32), pt,
                     pt.size, accept="bits")
    for key in a:
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)
    np.testing.assert_array_equal(b["accept_len"], m)


# --------------------------------------------------- separate projector (Table 3(b))

def _proj_case():
    L, Hkv, hd, Dcat, d = 2, 2, 16, 48, 32
    H = RNG.standard_normal((5, Dcat))
    E = RNG.standard_normal(Dcat)
    WF = RNG.standard_normal((d, Dcat))
    WKV = RNG.standard_normal((2 * L * Hkv * hd, d))
    pos = np.arange(20, 25)
    flag = np.array([False, False, True, True, True])
    return L, Hkv, hd, H, E, WF, WKV, pos, flag


def test_separate_projector_with_f_itself_is_the_no_embedding_update():
    """A separate projector equal to F, with no embedding, projects carried
    rows exactly like committed ones."""
    L, Hkv, hd, H, E, WF, WKV, pos, flag = _proj_case()
    k1, v1 = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, WF_carry=WF)
    k0, v0 = oracle.project(H, E, np.zeros(5, bool), WF, WKV, pos, L, Hkv, hd, 1e4)
    np.testing.assert_allclose(k1, k0, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(v1, v0, rtol=1e-13, atol=1e-13)


def test_separate_projector_touches_only_carried_rows_and_is_linear():
    """Committed rows ignore the separate projector; carried rows ignore E and F
    and scale with the projector (everything after it is linear)."""
    L, Hkv, hd, H, E, WF, WKV, pos, flag = _proj_case()
    WC = RNG.standard_normal(WF.shape)
    ka, va = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, WF_carry=WC)
    kb, vb = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, WF_carry=3.0 * WC)
    kc, vc = oracle.project(H, 5.0 * E, flag, 2.0 * WF, WKV, pos, L, Hkv, hd, 1e4, WF_carry=WC)
    kd, vd = oracle.project(H, E, np.zeros(5, bool), WF, WKV, pos, L, Hkv, hd, 1e4)
    np.testing.assert_allclose(ka[~flag], kd[~flag], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(va[~flag], vd[~flag], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(kb[flag], 3.0 * ka[flag], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(vb[flag], 3.0 * va[flag], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(kc[flag], ka[flag], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(vc[flag], va[flag], rtol=1e-13, atol=1e-13)


# --------------------------------------------- attention mass on carried rows

def test_carry_mass_empty_and_full_segments():
    q = RNG.standard_normal((6, 16))
    k = RNG.standard_normal((9, 16))
    qpos = np.arange(30, 36)
    np.testing.assert_array_equal(oracle.carry_mass(q, qpos, k, k[:0], 1e4), np.zeros(6))
    np.testing.assert_allclose(oracle.carry_mass(q, qpos, k[:0], k, 1e4), np.ones(6), rtol=1e-15)
    np.testing.assert_array_equal(oracle.carry_mass(q, qpos, k[:0], k[:0], 1e4), np.zeros(6))


def test_carry_mass_of_identical_keys_is_the_carried_share():
    """Equal logits everywhere: every key gets 1/n of the weight."""
    q = RNG.standard_normal((4, 16))
    k = np.tile(RNG.standard_normal(16), (11, 1))
    mass = oracle.carry_mass(q, np.arange(4), k[:7], k[7:], 1e4)
    np.testing.assert_allclose(mass, np.full(4, 4 / 11), rtol=1e-14)


def test_carry_mass_equals_exp_of_segment_lse_difference():
    """Mass on U = exp(LSE over U alone - LSE over [C;U]), with both LSEs taken
    from the plain attention; the committed share is its complement."""
    q = RNG.standard_normal((5, 32))
    kc, ku = RNG.standard_normal((13, 32)), RNG.standard_normal((6, 32))
    v = RNG.standard_normal((19, 32))
    qpos = np.arange(100, 105)
    _, lse_all = oracle.attend(q, qpos, np.concatenate([kc, ku]), v, 1e4)
    _, lse_u = oracle.attend(q, qpos, ku, v[13:], 1e4)
    _, lse_c = oracle.attend(q, qpos, kc, v[:13], 1e4)
    mass = oracle.carry_mass(q, qpos, kc, ku, 1e4)
    np.testing.assert_allclose(mass, np.exp(lse_u - lse_all), rtol=1e-12)
    np.testing.assert_allclose(1.0 - mass, np.exp(lse_c - lse_all), rtol=1e-10)


def test_carry_mass_one_dominant_carried_logit():
    hd = 8
    q = np.zeros((1, hd))
    q[0, 0] = 1.0
    kc = np.zeros((5, hd))
    ku = np.zeros((2, hd))
    ku[1, 0] = 200.0                   # at position 0 the query is not rotated
    mass = oracle.carry_mass(q, np.array([0]), kc, ku, 1e4)
    assert 1.0 - mass[0] < 1e-15


# ------------------------------------------- normalisation of F's output (variant)

def test_z_norm_makes_the_update_scale_invariant():
    """With F's output RMS-normalised, scaling the target features (and E with
    them) by any c > 0 leaves every key and value unchanged (up to the epsilon),
    and the gain scales them linearly."""
    L, Hkv, hd, H, E, WF, WKV, pos, flag = _proj_case()
    g = RNG.uniform(0.5, 1.5, WF.shape[0])
    k1, v1 = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, z_norm=g)
    k2, v2 = oracle.project(7.0 * H, 7.0 * E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, z_norm=g)
    # the epsilon moves a row by eps / (2 mean(z^2)), about 1e-8 here
    np.testing.assert_allclose(k2, k1, rtol=1e-7, atol=1e-7)
    np.testing.assert_allclose(v2, v1, rtol=1e-7, atol=1e-7)
    k3, v3 = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, z_norm=2.0 * g)
    np.testing.assert_allclose(k3, 2.0 * k1, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v3, 2.0 * v1, rtol=1e-12, atol=1e-12)


def test_rms_norm_rows_have_unit_rms():
    z = RNG.standard_normal((6, 40)) * RNG.uniform(0.1, 10.0, (6, 1))
    y = oracle.rms_norm(z, np.ones(40))
    ms = np.mean(z * z, axis=1)
    np.testing.assert_allclose(np.mean(y * y, axis=1), ms / (ms + oracle.RMS_EPS), rtol=1e-12)


# --------------------------------------------------- block self-KV segment (variant)

def _self_case(ctx, B=4, L=1, Hkv=1, G=2, hd=16):
    st = oracle.State(1, L, Hkv, hd)
    if ctx:
        st.set_committed(0, RNG.standard_normal((L, ctx, Hkv, hd)),
                         RNG.standard_normal((L, ctx, Hkv, hd)))
    Q = RNG.standard_normal((L, 1, B, Hkv * G, hd))
    Ks = RNG.standard_normal((L, 1, B, Hkv, hd))
    Vs = RNG.standard_normal((L, 1, B, Hkv, hd))
    return st, Q, Ks, Vs


def test_self_segment_depends_on_relative_positions_only():
    """With no committed or carried keys, a query at ctx + i against self key j
    (rotated at ctx + j) sees only i - j: the output does not move with ctx."""
    st0, Q, Ks, Vs = _self_case(0)
    O0, L0 = oracle.attend_state_with_self(st0, Q, Ks, Vs, 2, 1e4)
    st1 = oracle.State(1, 1, 1, 16)
    st1.ctx_len = lambda: np.array([977], np.int32)       # shift every position by 977
    O1, L1 = oracle.attend_state_with_self(st1, Q, Ks, Vs, 2, 1e4)
    np.testing.assert_allclose(O1, O0, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(L1, L0, rtol=1e-9, atol=1e-11)


def test_self_segment_merges_with_the_context_by_the_lse_rule():
    """[C;U;S] in one softmax equals the log-sum-exp merge of the attention over
    [C;U] and the attention over S alone (Eq. 2's ctx, one more segment)."""
    st, Q, Ks, Vs = _self_case(37)
    O, LSE = oracle.attend_state_with_self(st, Q, Ks, Vs, 2, 1e4)
    Oc, Lc = oracle.attend_state(st, Q, 2, 1e4)
    empty = oracle.State(1, 1, 1, 16)
    empty.ctx_len = st.ctx_len                             # same query positions, no keys
    Os, Ls = oracle.attend_state_with_self(empty, Q, Ks, Vs, 2, 1e4)
    M = np.maximum(Lc, Ls)
    wc, ws = np.exp(Lc - M), np.exp(Ls - M)
    np.testing.assert_allclose(O, (wc[..., None] * Oc + ws[..., None] * Os) /
                               (wc + ws)[..., None], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(LSE, M + np.log(wc + ws), rtol=1e-12)


def test_self_segment_identical_keys_average_all_values():
    """All logits equal (zero keys in both segments): every query returns the
    mean of all committed and self values."""
    st, Q, Ks, Vs = _self_case(5)
    st.ck[0][:] = 0.0
    Ks[:] = 0.0
    O, _ = oracle.attend_state_with_self(st, Q, Ks, Vs, 2, 1e4)
    allv = np.concatenate([st.cv[0][0, :, 0], Vs[0, 0, :, 0]], axis=0)
    np.testing.assert_allclose(O[0, 0], np.broadcast_to(allv.mean(axis=0), O[0, 0].shape),
                               rtol=1e-12, atol=1e-12)


def test_k_norm_keys_have_the_gain_rms_and_values_are_untouched():
    """With unit gain every head's key has RMS sqrt(ms / (ms + eps)) after the
    rotation (which preserves norms); values do not change; scaling K's weights
    leaves the keys unchanged (up to the epsilon)."""
    L, Hkv, hd, H, E, WF, WKV, pos, flag = _proj_case()
    ones = np.ones((L, hd))
    k0, v0 = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4)
    k1, v1 = oracle.project(H, E, flag, WF, WKV, pos, L, Hkv, hd, 1e4, k_norm=ones)
    np.testing.assert_array_equal(v1, v0)
    ms = np.mean(k0 * k0, axis=-1)                      # rotation keeps the norm
    np.testing.assert_allclose(np.mean(k1 * k1, axis=-1), ms / (ms + oracle.RMS_EPS), rtol=1e-10)
    W2 = WKV.copy().reshape(L, 2, Hkv * hd, -1)
    W2[:, 0] *= 5.0                                     # keys only
    k2, v2 = oracle.project(H, E, flag, WF, W2.reshape(WKV.shape), pos, L, Hkv, hd, 1e4,
                            k_norm=ones)
    np.testing.assert_allclose(k2, k1, rtol=1e-7, atol=1e-7)
    np.testing.assert_array_equal(v2, v1)


def test_k_norm_gain_applies_before_the_rotation():
    """The gain multiplies the unrotated key: at position 0 (no rotation) the
    key is the normalised key times the gain, elementwise."""
    L, Hkv, hd, H, E, WF, WKV, pos, flag = _proj_case()
    g = RNG.uniform(0.5, 1.5, (L, hd))
    k1, _ = oracle.project(H, E, flag, WF, WKV, np.zeros(5), L, Hkv, hd, 1e4, k_norm=g)
    k0, _ = oracle.project(H, E, flag, WF, WKV, np.zeros(5), L, Hkv, hd, 1e4)
    r = np.sqrt(np.mean(k0 * k0, axis=-1, keepdims=True) + oracle.RMS_EPS)
    np.testing.assert_allclose(k1, k0 / r * g[None, :, None, :], rtol=1e-12, atol=1e-12)


# ------------------------------------------- backward of the second pass (Algorithm 2)

def _attn_case(nq=3, nk=5, hd=8):
    q = RNG.standard_normal((nq, hd))
    k = RNG.standard_normal((nk, hd))
    v = RNG.standard_normal((nk, hd))
    dO = RNG.standard_normal((nq, hd))
    qpos = np.array([7, 7, 9])[:nq]
    return q, qpos, k, v, dO


def _fd(f, x, h=1e-6):
    """Central finite differences of the scalar f at every element of x."""
    g = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        x0 = x[idx]
        x[idx] = x0 + h
        fp = f()
        x[idx] = x0 - h
        fm = f()
        x[idx] = x0
        g[idx] = (fp - fm) / (2 * h)
    return g


def test_attend_backward_matches_finite_differences():
    """Every element of dq, dk, dv against central differences of the forward
    oracle's sum(dO * O): a dropped term, a sign, a missing rotation or a
    transposed product fails it."""
    q, qpos, k, v, dO = _attn_case()
    theta = 100.0
    dq, dk, dv = oracle.attend_backward(q, qpos, k, v, dO, theta)
    loss = lambda: float(np.sum(dO * oracle.attend(q, qpos, k, v, theta)[0]))
    np.testing.assert_allclose(dq, _fd(loss, q), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dk, _fd(loss, k), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(dv, _fd(loss, v), rtol=1e-6, atol=1e-8)


def test_attend_backward_invariants():
    """Shifting every key by one vector leaves the softmax unchanged, so the
    keys' gradients sum to zero; the weights of a query sum to one, so the
    values' gradients sum to the sum of dO; no keys: zero gradients."""
    q, qpos, k, v, dO = _attn_case(nq=3, nk=7, hd=16)
    dq, dk, dv = oracle.attend_backward(q, qpos, k, v, dO, 1e4)
    np.testing.assert_allclose(dk.sum(axis=0), 0.0, atol=1e-12)
    np.testing.assert_allclose(dv.sum(axis=0), dO.sum(axis=0), rtol=1e-12, atol=1e-12)
    dq0, dk0, dv0 = oracle.attend_backward(q, qpos, k[:0], v[:0], dO, 1e4)
    assert not dq0.any() and dk0.shape == (0, 16) and dv0.shape == (0, 16)


def test_project_backward_matches_finite_differences():
    """Directional derivatives of sum(dK * K + dV * V) of the forward oracle
    along random directions of W_F, W_KV and E equal the inner products with
    the returned gradients."""
    L, Hkv, hd, H, E, WF, WKV, pos, flag = _proj_case()
    dK = RNG.standard_normal((5, L, Hkv, hd))
    dV = RNG.standard_normal((5, L, Hkv, hd))
    theta = 1e4
    dWF, dWKV, dE = oracle.project_backward(H, E, flag, WF, WKV, pos, L, Hkv, hd, theta, dK, dV)

    def loss(wf, wkv, e):
        k, v = oracle.project(H, e, flag, wf, wkv, pos, L, Hkv, hd, theta)
        return float(np.sum(dK * k) + np.sum(dV * v))

    h = 1e-6
    for name, grad in (("WF", dWF), ("WKV", dWKV), ("E", dE)):
        U = RNG.standard_normal(grad.shape)
        args_p = dict(wf=WF, wkv=WKV, e=E)
        args_m = dict(wf=WF, wkv=WKV, e=E)
        key = {"WF": "wf", "WKV": "wkv", "E": "e"}[name]
        args_p[key] = args_p[key] + h * U
        args_m[key] = args_m[key] - h * U
        fd = (loss(**args_p) - loss(**args_m)) / (2 * h)
        assert abs(fd - np.sum(grad * U)) <= 1e-6 * max(1.0, abs(fd)), name
    # rows without the embedding contribute nothing to dE
    _, _, dE0 = oracle.project_backward(H, E, np.zeros(5, bool), WF, WKV, pos, L, Hkv, hd,
                                        theta, dK, dV)
    assert not dE0.any()


# ------------------------------------ training-shaped second pass (Algorithm 2)
#
# Algorithm 2 steps 3-6: after the first pass from anchor a the verifier
# accepts m proposals; the anchor moves to a' = a + m + 1; the second pass
# reads the recorded prefix y_{<a'} (committed keys, projected without E at
# their own positions) plus the block's rejected rows Phi(H^rej + E_carry) at
# a' + r, and its queries sit at a' + i.  The oracle reaches this through
# route(mode="carry_only") and round_update(..., "carry_only"); these pins check
# that path against the algorithm's own statements and against a dense
# recomputation that shares none of the oracle's routing, state or attention.

def _tokens_with_lcp(m, B, rng, V=50):
    S = len(m)
    target = rng.integers(0, V, (S, B))
    draft = target.copy()
    for s in range(S):
        if m[s] < B:
            draft[s, m[s]] = (target[s, m[s]] + 1 + rng.integers(0, V - 1)) % V
    return draft.astype(np.int32), target.astype(np.int32)


def test_carry_only_route_follows_algorithm_2_shift():
    """For every accepted count m (all of 0..B): p0 = a + 1 (the window starts
    after the anchor), ctx_len = a + 1 + m = a', carry_len = B - m, no row is
    committed (rows j < m: SKIP), window row j >= m is carry row j - m at
    position a' + (j - m)."""
    rng = np.random.default_rng(21)
    B, P = 16, 8
    m = np.arange(B + 1, dtype=np.int32)
    S = len(m)
    a = rng.integers(0, P * 16 - B - 1, S).astype(np.int32)
    pt = np.array([rng.permutation(4 * P)[:P] for _ in range(S)], np.int32)
    draft, target = _tokens_with_lcp(m, B, rng)
    old_carry = rng.integers(0, B + 1, S).astype(np.int32)
    r = oracle.route(draft, target, a + 1, old_carry, pt, 4 * P, mode="carry_only")
    a2 = a + m + 1                                     # Algorithm 2 step 3
    np.testing.assert_array_equal(r["status"], 0)
    np.testing.assert_array_equal(r["accept_len"], m)
    np.testing.assert_array_equal(r["ctx_len"], a2)
    np.testing.assert_array_equal(r["carry_len"], B - m)
    for s in range(S):
        for j in range(B):
            assert r["row_pos"][s, j] == a[s] + 1 + j
            if j < m[s]:
                assert r["row_dst"][s, j] == oracle.SKIP
            else:
                rr = j - m[s]
                assert r["row_dst"][s, j] == -1 - rr
                assert r["row_pos"][s, j] == a2[s] + rr


def test_carry_only_update_keeps_committed_and_equals_carry_mode_carries():
    """carry_only leaves C exactly as it was and builds the same U as the
    ordinary carry update of the same rows (Eq. 2 with the same E and
    positions); only the committed rows differ, which carry_only never writes."""
    t = _tiny_setup(S=3, B=4)
    S, B, L, Hkv, hd = t["S"], t["B"], t["L"], t["Hkv"], t["hd"]
    rng = t["rng"]
    m = np.array([0, 2, 4], np.int32)
    draft, target = _tokens_with_lcp(m, B, rng)
    H = rng.standard_normal((S, B, t["Dcat"]))
    pt = np.tile(np.arange(8, dtype=np.int32), (S, 1))
    ctx0 = np.array([5, 9, 0], np.int32)
    ck = [rng.standard_normal((L, n, Hkv, hd)) for n in ctx0]
    cv = [rng.standard_normal((L, n, Hkv, hd)) for n in ctx0]
    sts = []
    for mode in ("carry_only", "carry"):
        st = oracle.State(S, L, Hkv, hd)
        for s in range(S):
            st.set_committed(s, ck[s], cv[s])
        before_k = [c.copy() for c in st.ck]
        before_v = [c.copy() for c in st.cv]
        r = oracle.route(draft, target, ctx0, np.zeros(S, np.int32), pt, 8, mode)
        oracle.round_update(st, r, H, t["E"], t["WF"], t["WKV"], 1e4, mode)
        sts.append((st, before_k, before_v, r))
    co_st, ck0, cv0, r_co = sts[0]
    ca_st, _, _, r_ca = sts[1]
    for s in range(S):
        np.testing.assert_array_equal(co_st.ck[s], ck0[s])
        np.testing.assert_array_equal(co_st.cv[s], cv0[s])
        np.testing.assert_array_equal(co_st.uk[s], ca_st.uk[s])
        np.testing.assert_array_equal(co_st.uv[s], ca_st.uv[s])
        assert ca_st.ck[s].shape[1] == ctx0[s] + m[s]
    np.testing.assert_array_equal(r_co["ctx_len"], r_ca["ctx_len"])
    np.testing.assert_array_equal(r_co["carry_len"], r_ca["carry_len"])


def _train_tiny(seed=31):
    """Two recorded responses of 24 positions, three anchors each, B = 4."""
    rng = np.random.default_rng(seed)
    n_resp, seq_len, A, B = 2, 24, 3, 4
    Dcat, d, L, Hq, Hkv, hd = 10, 6, 2, 4, 2, 8
    c = dict(n_resp=n_resp, seq_len=seq_len, A=A, B=B, Dcat=Dcat, d=d, L=L, Hq=Hq, Hkv=Hkv,
             hd=hd, theta=100.0)
    c["WF"] = rng.standard_normal((d, Dcat)) * 0.4
    c["WKV"] = rng.standard_normal((2 * L * Hkv * hd, d)) * 0.4
    c["E"] = rng.standard_normal(Dcat)
    c["Y"] = rng.standard_normal((n_resp, seq_len, Dcat))        # recorded target states
    c["a"] = np.array([np.sort(rng.choice(seq_len - B - 1, A, replace=False))
                       for _ in range(n_resp)], np.int32).ravel()
    c["u"] = np.array([0, 4, 2, 1, 3, 4], np.int32)              # rejected counts, incl. 0 and B
    c["H"] = rng.standard_normal((n_resp * A, B, Dcat))          # window states (first pass)
    c["Q"] = rng.standard_normal((L, n_resp * A, B, Hq, hd))
    return c


def _train_oracle(c, mode="carry_only", p0_shift=1):
    """The oracle's path through the training-shaped forward (as the GPU parity
    tests drive it)."""
    V, B, L, Hkv, hd = c["n_resp"] * c["A"], c["B"], c["L"], c["Hkv"], c["hd"]
    m = (B - c["u"]).astype(np.int32)
    a2 = c["a"] + m + 1
    st = oracle.State(V, L, Hkv, hd)
    for v in range(V):
        y = c["Y"][v // c["A"]]
        k, vv = oracle.project(y, c["E"], np.zeros(len(y), bool), c["WF"], c["WKV"],
                               np.arange(len(y)), L, Hkv, hd, c["theta"])
        n = int(a2[v])
        st.set_committed(v, k[:n].transpose(1, 0, 2, 3), vv[:n].transpose(1, 0, 2, 3))
    draft, target = _tokens_with_lcp(m, B, np.random.default_rng(5))
    pt = np.tile(np.arange(4, dtype=np.int32), (V, 1))
    r = oracle.route(draft, target, c["a"] + p0_shift, np.zeros(V, np.int32), pt, 4, mode)
    oracle.round_update(st, r, c["H"], c["E"], c["WF"], c["WKV"], c["theta"], mode)
    O, LSE = oracle.attend_state(st, c["Q"], c["Hq"], c["theta"])
    return r, O, LSE


def _train_brute(c):
    """Per block, from Algorithm 2 directly: committed = recorded rows t < a'
    projected by plain loops without E at position t; carried = window rows
    j >= m with E at position a + 1 + j; queries at a' + i; dense softmax with
    an unshifted exp, KV head = the query head's group."""
    V, B, L, Hq, Hkv, hd, th = (c["n_resp"] * c["A"], c["B"], c["L"], c["Hq"], c["Hkv"],
                                c["hd"], c["theta"])
    G = Hq // Hkv
    O = np.zeros((L, V, B, Hq, hd))
    LSE = np.zeros((L, V, B, Hq))
    for v in range(V):
        a, u = int(c["a"][v]), int(c["u"][v])
        m = B - u
        a2 = a + m + 1
        rows = [_brute_project_row(c["Y"][v // c["A"]][t], c["E"], False, c["WF"], c["WKV"], t,
                                   L, Hkv, hd, th) for t in range(a2)]
        rows += [_brute_project_row(c["H"][v][j], c["E"], True, c["WF"], c["WKV"], a + 1 + j,
                                    L, Hkv, hd, th) for j in range(m, B)]
        for layer in range(L):
            for i in range(B):
                for h in range(Hq):
                    g = h // G
                    q = oracle.rope(c["Q"][layer, v, i, h], a2 + i, th)
                    wts = np.array([math.exp(float(q @ kv[0][layer, g]) / math.sqrt(hd))
                                    for kv in rows])
                    vals = np.array([kv[1][layer, g] for kv in rows])
                    O[layer, v, i, h] = wts @ vals / wts.sum()
                    LSE[layer, v, i, h] = math.log(wts.sum())
    return O, LSE


def test_training_second_pass_matches_dense_brute_force():
    """The oracle's carry_only forward equals the dense per-block recomputation
    of Algorithm 2's second pass; two plausible mistakes (committing the
    accepted window rows too, or starting the window at the anchor instead of
    after it) are each caught by the same comparison."""
    c = _train_tiny()
    O_b, L_b = _train_brute(c)
    r, O, LSE = _train_oracle(c)
    np.testing.assert_array_equal(r["ctx_len"], c["a"] + (c["B"] - c["u"]) + 1)
    np.testing.assert_allclose(O, O_b, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(LSE, L_b, rtol=1e-12, atol=1e-12)
    # mutant 1: the accepted window rows are committed as well (duplicated keys)
    _, O1, _ = _train_oracle(c, mode="carry")
    assert np.abs(O1 - O_b).max() > 1e-3
    # mutant 2: the window starts at the anchor (p0 = a), so every carried row
    # and every query sits one position early
    _, O2, _ = _train_oracle(c, p0_shift=0)
    assert np.abs(O2 - O_b).max() > 1e-3


def test_carry_mass_state_matches_dense_per_head_recomputation():
    """carry_mass_state, for every (layer, sequence, block row, query head) of a
    state with three query heads per KV head, equals the share of the dense,
    unshifted softmax weights on the carried keys, with the KV head of query
    head h taken as h * Hkv // Hq; an interleaved head mapping is caught."""
    rng = np.random.default_rng(41)
    S, L, Hq, Hkv, hd, B = 2, 2, 6, 2, 8, 3
    st = oracle.State(S, L, Hkv, hd)
    for s, (n, u) in enumerate(((5, 2), (7, 3))):
        st.set_committed(s, rng.standard_normal((L, n, Hkv, hd)), rng.standard_normal((L, n, Hkv, hd)))
        st.uk[s] = rng.standard_normal((L, u, Hkv, hd))
        st.uv[s] = rng.standard_normal((L, u, Hkv, hd))
    Q = rng.standard_normal((L, S, B, Hq, hd))
    mass = oracle.carry_mass_state(st, Q, Hq, 1e4)

    def dense(kv_head_of):
        out = np.zeros((L, S, B, Hq))
        for s in range(S):
            n = st.ck[s].shape[1]
            for layer in range(L):
                for i in range(B):
                    for h in range(Hq):
                        g = kv_head_of(h)
                        q = oracle.rope(Q[layer, s, i, h], n + i, 1e4)
                        wc = [math.exp(float(q @ st.ck[s][layer, t, g]) / math.sqrt(hd))
                              for t in range(n)]
                        wu = [math.exp(float(q @ st.uk[s][layer, t, g]) / math.sqrt(hd))
                              for t in range(st.uk[s].shape[1])]
                        out[layer, s, i, h] = sum(wu) / (sum(wc) + sum(wu))
        return out

    np.testing.assert_allclose(mass, dense(lambda h: h * Hkv // Hq), rtol=1e-12, atol=1e-14)
    assert np.abs(dense(lambda h: h % Hkv) - mass).max() > 1e-3


# ------------------------------------- stochastic verification (T = 1), Appendix A
#
# The standard speculative-sampling rule: accept a proposal x ~ q with
# probability min(1, p(x)/q(x)); at the first rejection emit a token from the
# normalised residual max(0, p - q); after B acceptances a bonus from p.  Its
# defining property (the one Appendix A relies on) is that the emitted token
# is distributed exactly as p.  The pins check the oracle's discrete form of
# the rule against that property and against closed forms.

from fractions import Fraction  # noqa: E402

_GRID = (np.arange(1 << 24, dtype=np.uint64) << np.uint64(8)).astype(np.uint32)


def _softmax32(z):
    e = np.exp(z - z.max())
    return (e / e.sum()).astype(np.float32)


def _accepted_words(p_x, q_x):
    """Number of the 2^24 acceptance words for which the oracle accepts."""
    return int(np.count_nonzero(oracle.accept_test(_GRID, np.float32(p_x), np.float32(q_x))))


def _first_word_reaching(w, y):
    """Smallest 32-bit word whose draw is >= y (draws are non-decreasing in the word)."""
    lo, hi = 0, 1 << 32
    while lo < hi:
        mid = (lo + hi) // 2
        if oracle.sample_fixed(w, mid) >= y:
            hi = mid
        else:
            lo = mid + 1
    return lo


def _draw_probabilities(w):
    """Exact probability of every token under a uniform 32-bit word."""
    V = len(w)
    edges = [_first_word_reaching(w, y) for y in range(V)] + [1 << 32]
    return np.array([(edges[y + 1] - edges[y]) / 2.0 ** 32 for y in range(V)])


_VERIFY_CASES = [
    (np.array([0.7, 0.3], np.float32), np.array([0.4, 0.6], np.float32)),
    (np.array([0.2, 0.5, 0.3], np.float32), np.array([0.6, 0.1, 0.3], np.float32)),
    (np.array([0.0, 0.25, 0.75], np.float32), np.array([0.5, 0.5, 0.0], np.float32)),
]


def test_accept_share_is_min_one_p_over_q_on_small_vocabularies():
    """Over the whole grid of acceptance words, proposal x is accepted for
    exactly min(2^24, ceil(2^24 p(x) / q(x))) of them (u < p/q on a 24-bit
    grid), and the overall acceptance probability sum_x q(x) min(1, p/q) equals
    sum_x min(p(x), q(x)) to the grid's resolution."""
    for p, q in _VERIFY_CASES:
        tot = 0.0
        for x in range(len(p)):
            if q[x] == 0:
                continue
            n = _accepted_words(p[x], q[x])
            exact = Fraction(float(p[x])) / Fraction(float(q[x])) * (1 << 24)
            want = min(1 << 24, -(-exact.numerator // exact.denominator))   # ceil
            assert n == want, (p, q, x)
            tot += float(q[x]) * n / 2.0 ** 24
        assert abs(tot - float(np.minimum(p, q).sum())) <= len(p) * 2.0 ** -24


def test_emitted_token_is_distributed_as_the_target():
    """One proposal position: the token the verifier emits (the accepted
    proposal, else the residual draw) has the target's distribution p, to the
    grids' resolution; drawing the correction from max(0, q - p) instead, or
    from p itself, is caught."""
    for p, q in _VERIFY_CASES:
        V = len(p)
        acc = np.array([_accepted_words(p[x], q[x]) / 2.0 ** 24 if q[x] > 0 else 0.0
                        for x in range(V)])
        reject = float(np.sum(q.astype(np.float64) * (1.0 - acc)))

        def emitted(res_w):
            return q.astype(np.float64) * acc + reject * _draw_probabilities(res_w)

        got = emitted(oracle.fixed_weights(p, q))
        np.testing.assert_allclose(got, p.astype(np.float64), rtol=0, atol=4 * V * 2.0 ** -24)
        assert np.abs(emitted(oracle.fixed_weights(q, p)) - p).max() > 1e-2
        assert np.abs(emitted(oracle.fixed_weights(p)) - p).max() > 1e-2


def test_draws_are_monotone_cover_every_word_and_skip_zero_weights():
    rng = np.random.default_rng(61)
    p = _softmax32(rng.standard_normal(40) * 2)
    q = _softmax32(rng.standard_normal(40) * 2)
    w = oracle.fixed_weights(p, q)
    words = np.sort(rng.integers(0, 1 << 32, 2000, dtype=np.uint64))
    draws = [oracle.sample_fixed(w, int(u)) for u in words]
    assert all(b >= a for a, b in zip(draws, draws[1:]))
    probs = _draw_probabilities(w)
    assert abs(probs.sum() - 1.0) < 1e-12                 # every word yields a token
    assert np.all(probs[w == 0] == 0)                     # p <= q: never drawn
    np.testing.assert_allclose(probs, w / w.sum(), rtol=0, atol=2.0 ** -31)
    assert np.all(w[p.astype(np.float64) <= q.astype(np.float64)] == 0)
    assert oracle.sample_fixed(np.zeros(5, np.uint64), 123) == -1


def test_verify_p_equals_q_accepts_every_proposal():
    """Identical target and drafter distributions: every proposal is accepted
    whatever the words, and the bonus comes from p at the position after the
    block (the first and last tokens of p's support for the extreme words)."""
    rng = np.random.default_rng(62)
    B, V = 8, 50
    for _ in range(20):
        p = np.stack([_softmax32(rng.standard_normal(V) * 3) for _ in range(B + 1)])
        p[B, :3] = 0.0
        p[B, -2:] = 0.0
        draft = rng.integers(0, V, B)
        words = rng.integers(0, 1 << 32, B + 1, dtype=np.uint64).astype(np.uint32)
        m, nxt, st = oracle.verify_sample(draft, p, p[:B], words)
        assert (m, st) == (B, oracle.OK)
        assert p[B, nxt] > 0
        words[B] = 0
        assert oracle.verify_sample(draft, p, p[:B], words)[1] == 3
        words[B] = 0xFFFFFFFF
        assert oracle.verify_sample(draft, p, p[:B], words)[1] == V - 3


def test_verify_stops_at_the_first_rejection():
    """Acceptance words of 0 accept any proposal the target gives probability;
    a proposal the target gives none is always rejected; the correction is a
    token whose target probability exceeds the drafter's; positions after the
    first rejection do not matter; a token outside the vocabulary is an error."""
    rng = np.random.default_rng(63)
    B, V = 6, 30
    for m_want in range(B + 1):
        p = np.stack([_softmax32(rng.standard_normal(V) * 2) for _ in range(B + 1)])
        q = np.stack([_softmax32(rng.standard_normal(V) * 2) for _ in range(B)])
        draft = rng.integers(1, V, B)
        if m_want < B:
            p[m_want, draft[m_want]] = 0.0                 # rejected for every word
        words = np.zeros(B + 1, np.uint32)
        words[m_want + 1:] = rng.integers(0, 1 << 32, B - m_want, dtype=np.uint64)
        m, nxt, st = oracle.verify_sample(draft, p, q, words)
        assert (m, st) == (m_want, oracle.OK)
        if m < B:
            assert float(p[m, nxt]) > float(q[m, nxt])
        bits = np.array([bool(oracle.accept_test(words[j], p[j, draft[j]], q[j, draft[j]]))
                         for j in range(B)], np.int32)
        assert oracle.accept_len_bits(bits) == m
    bad = draft.copy()
    bad[2] = V
    assert oracle.verify_sample(bad, p, q, words) == (0, -1, oracle.ERR_TOKEN)
