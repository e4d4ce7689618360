"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Routing, acceptance lengths, descriptors and lengths must match bit for bit;
floating-point outputs (attention O and LSE, the committed rows written this
round, the carry rows) must match per head vector within 2e-2 (bf16) or 1e-4
(fp32) of max relative error.
"""
import numpy as np
import pytest

import oracle
from synth import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from helpers import (TOL, OracleRun, assert_heads_close, compare_round, gather_carry,  # noqa: E402
                     gather_committed, to_np)

SMALL_RAGGED = wl.RAGGED32.replace(name="small_ragged", S=3, L=2, ctx_lo=100, ctx_hi=2500,
                                   rounds=6, accept=("geom", 0.3), seed=0x5EED01)
SMALL_G4 = wl.Workload("small_g4_hd128", S=2, B=16, Dcat=512, d=256, L=2, Hq=8, Hkv=2, hd=128,
                       dtype="bf16", theta=1e6, ctx_lo=1500, ctx_hi=1500, ctx_mode="projected",
                       accept=("uniform",), rounds=4, seed=0x5EED02)
BATCH3_8B = wl.BATCH1_8B.replace(name="batch3_8b_short", S=3, ctx_lo=300, ctx_hi=300, rounds=4,
                                 seed=0x5EED04)
SMALL_F32 = wl.Workload("small_f32", S=2, B=8, Dcat=256, d=128, L=2, Hq=4, Hkv=1, hd=128,
                        dtype="f32", theta=1e4, ctx_lo=300, ctx_hi=300, ctx_mode="projected",
                        accept=("uniform",), rounds=4, seed=0x5EED03)


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from synth.scenario import Scenario
    return Scenario


def run_rounds(w, n_rounds, mode="carry", seqs=None, check_context=True, fold_e=True,
               extra_flags=0):
    import paper_2609_14717_amd as co
    Scenario = _gpu()
    print(f"[parity] workload={w.name} rounds={n_rounds} mode={mode} fold_e={fold_e} "
          f"flags={extra_flags}", flush=True)
    sc = Scenario(w, fold_e=fold_e)
    orc = OracleRun(w, seqs=seqs)
    seqs = orc.seqs
    if check_context and w.ctx_mode == "projected" and w.ctx_lo:
        n = int(sc.ctx0[0])
        for s in seqs[:2]:
            gk, gv = gather_committed(sc.st, sc.pt, s, 0, 0, n)
            assert_heads_close(gk, orc.st.ck[s][0], TOL[w.dtype], "prefill K")
            assert_heads_close(gv, orc.st.cv[s][0], TOL[w.dtype], "prefill V")
    flags = {"carry": 0, "baseline": co.CO_BASELINE_MODE}[mode] | extra_flags
    for r in range(n_rounds):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, flags,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r, mode)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, seqs, f"{w.name} r{r}")
    return sc, orc


@pytest.mark.parametrize("w", [SMALL_RAGGED, SMALL_G4, SMALL_F32, BATCH3_8B], ids=lambda w: w.name)
def test_small_chains(w):
    run_rounds(w, 4)


@pytest.mark.parametrize("w", [SMALL_RAGGED, SMALL_G4], ids=lambda w: w.name)
def test_small_chains_baseline_mode(w):
    run_rounds(w, 3, mode="baseline")


@pytest.mark.parametrize("w", [SMALL_RAGGED, SMALL_G4, BATCH3_8B], ids=lambda w: w.name)
def test_small_chains_e_in_kernel(w):
    """F(E) accumulated inside the projection instead of folded beforehand."""
    run_rounds(w, 3, fold_e=False)


# 256-row windows (16 sequences x 16) and a 3200-row prefill, small enough for
# the oracle, run through every large-tile GEMM variant, with F(E) folded
# beforehand and accumulated in the kernel.
WIDE64 = wl.Workload("wide_hd64", S=16, B=16, Dcat=1024, d=256, L=2, Hq=4, Hkv=2, hd=64,
                     dtype="bf16", theta=1e4, ctx_lo=200, ctx_hi=200, ctx_mode="projected",
                     accept=("geom", 0.3), rounds=3, seed=0x5EED06)
WIDE128 = wl.Workload("wide_hd128", S=16, B=16, Dcat=1536, d=512, L=1, Hq=8, Hkv=2, hd=128,
                      dtype="bf16", theta=1e6, ctx_lo=200, ctx_hi=200, ctx_mode="projected",
                      accept=("uniform",), rounds=3, seed=0x5EED07)


@pytest.mark.parametrize("fold", [True, False], ids=["folded", "in_kernel"])
@pytest.mark.parametrize("variant", range(7), ids=lambda v: f"v{v}")
@pytest.mark.parametrize("w", [WIDE64, WIDE128], ids=lambda w: w.name)
def test_wide_gemm_variants(w, variant, fold, tune):
    tune("gemm_wide_variant", variant)
    run_rounds(w, 2, fold_e=fold)


@pytest.mark.parametrize("w", [SMALL_G4, WIDE128, wl.RAGGED32], ids=lambda w: w.name)
def test_fold_e(w):
    """carryover_fold_e against F E in fp64 (fp32 accumulation of exact products)."""
    import paper_2609_14717_amd as co
    Scenario = _gpu()
    from helpers import host
    sc = Scenario(w, build_context=False)
    torch.cuda.synchronize()
    WF, E = host(w, wl.spec_wf(w)), host(w, wl.spec_e(w))
    ref = WF @ E
    mag = np.abs(WF) @ np.abs(E)
    got = sc.f_e.cpu().numpy().astype(np.float64)
    assert got.shape == ref.shape
    err = np.max(np.abs(got - ref) / mag)
    assert err <= 1e-5, err
    assert co.carryover_read_status(sc.st) == 0


def test_tiny_fp32_full():
    run_rounds(wl.TINY, 6)


def test_ragged_batch32_full():
    run_rounds(wl.RAGGED32, 3)


def test_batch1_8b_full():
    run_rounds(wl.BATCH1_8B, 2)


# Workgroup counts and round sizes forced far from the defaults, so that one
# workgroup walks many segments in several passes and rounds, wavefronts park
# and merge partial segments, and rounds hand a segment on to the next.
MANY_SEQS = wl.RAGGED32.replace(name="many_seqs", S=70, L=1, ctx_lo=1, ctx_hi=700, rounds=3,
                                accept=("geom", 0.25), seed=0x5EED05)
SLICINGS = [("1", "1"), ("1", "3"), ("3", "2"), ("7", "64"), ("1000", "")]


@pytest.mark.parametrize("w", [SMALL_RAGGED, SMALL_G4, MANY_SEQS], ids=lambda w: w.name)
@pytest.mark.parametrize("slicing", SLICINGS, ids=lambda s: f"wg{s[0]}_rt{s[1] or 'dflt'}")
def test_attention_slicings(w, slicing, tune):
    tune("attn_workgroups", slicing[0])
    if slicing[1]:
        tune("attn_round_tiles", slicing[1])
    run_rounds(w, 2)


def sampled_chain(w, rounds, samples, plan):
    """Chained serving rounds at full size in the launch configuration of a
    serving round.  Every round: routing, accepted lengths, descriptors and
    lengths of all sequences bit-exact; the committed rows written and the
    carry rows of the sequences in ``samples`` within tolerance.  ``plan(r)``
    lists the (sequences, layers) whose attention output is checked at round
    r (empty: none)."""
    import paper_2609_14717_amd as co
    Scenario = _gpu()
    tol = TOL[w.dtype]
    print(f"[parity] workload={w.name} rounds={rounds} samples={samples}", flush=True)
    sc = Scenario(w)
    orc = OracleRun(w, seqs=samples, store=np.float32)
    print(f"[parity] {w.name}: oracle state built", flush=True)
    n_out = 0
    for r in range(rounds):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, _, _ = orc.round(r, attend=False)
        for key in ("accept_len", "row_pos", "row_dst"):
            np.testing.assert_array_equal(sc.rt[key].cpu().numpy(), rr[key], err_msg=f"r{r} {key}")
        np.testing.assert_array_equal(sc.st["ctx_len"].cpu().numpy(), rr["ctx_len"])
        np.testing.assert_array_equal(sc.st["carry_len"].cpu().numpy(), rr["carry_len"])
        for s in samples:
            mm = int(rr["accept_len"][s])
            p0 = int(rr["ctx_len"][s]) - mm
            u = int(rr["carry_len"][s])
            for layer in range(w.L):
                if mm:
                    gk, gv = gather_committed(sc.st, sc.pt, s, layer, p0, p0 + mm)
                    assert_heads_close(gk, orc.st.ck[s][layer, p0:p0 + mm], tol,
                                       f"r{r} s{s} C_k l{layer}")
                    assert_heads_close(gv, orc.st.cv[s][layer, p0:p0 + mm], tol,
                                       f"r{r} s{s} C_v l{layer}")
                if u:
                    gk, gv = gather_carry(sc.st, s, layer, u)
                    assert_heads_close(gk, orc.st.uk[s][layer], tol, f"r{r} s{s} U_k l{layer}")
                    assert_heads_close(gv, orc.st.uv[s][layer], tol, f"r{r} s{s} U_v l{layer}")
        pieces = plan(r)
        if not pieces:
            continue
        g = to_np(out)
        gl = lse.cpu().numpy().astype(np.float64)
        Q = orc.seq_block(wl.spec_q(w, r), 1)
        for seqs, layers in pieces:
            O, LSE = oracle.attend_state(orc.st, Q, w.Hq, w.theta, seqs=seqs, layers=layers)
            for s in seqs:
                for layer in layers:
                    assert_heads_close(g[layer, s], O[layer, s], tol, f"r{r} s{s} O layer {layer}")
                    err = np.abs(gl[layer, s] - LSE[layer, s]).max()
                    assert err <= tol, f"r{r} s{s} LSE layer {layer}: {err}"
                    n_out += 1
        print(f"[parity] {w.name} round {r}: attention of "
              + "; ".join(f"seqs {list(s_)} layers {list(l_)}" for s_, l_ in pieces)
              + " checked", flush=True)
    print(f"[parity] {w.name}: {n_out} (sequence, layer) outputs checked", flush=True)


@pytest.mark.timeout(900)
def test_long_chain_5layer_full():
    """The 64-round, 5-layer chain at full size (16 sequences, contexts of
    16K-32K tokens, head_dim 128, 32/8 heads), every sequence tracked by the
    oracle: every round the routing, lengths and the committed and carry rows
    written of all 16 sequences in all 5 layers; the attention output of one
    (sequence, layer) every round (sequence r mod 16, layer r mod 5), of every
    sequence in layer 0 at rounds 0 and 31, and of every sequence in every
    layer at the last round."""
    w = wl.LONG_CHAIN
    R, S, L = w.rounds, w.S, w.L
    every = list(range(S))

    def plan(r):
        if r == R - 1:
            return [(every, list(range(L)))]
        if r in (0, R // 2 - 1):
            return [(every, [0])]
        return [([r % S], [r % L])]

    sampled_chain(w, R, every, plan)


def test_ragged_batch32_8b_full():
    """The batch-32 ragged round at the 8B widths (Dcat 20480 -> d 4096, 32/8
    heads of 128, contexts of 512-8192 tokens): four chained rounds, all 32
    sequences' rows and attention outputs against the oracle every round."""
    w = wl.RAGGED32_8B
    every = list(range(w.S))
    sampled_chain(w, 4, every, lambda r: [(every, [0])])


def test_train_fwd_sampled():
    """The training-shaped parallel forward at full size: 8 responses x 4096
    positions committed by prefill, 256 anchored blocks each (2048 virtual
    sequences sharing their response's pages), every block's rejected rows
    projected with E into its own carry segment, then block attention of all
    2048 blocks over their recorded prefix [0, a') plus their carry rows.
    Routing of all 2048 blocks bit-exact; the carry rows and the attention
    output of all 256 blocks of response 3 and of a sample of the others
    (first and last blocks, extreme anchors, full acceptance and full
    rejection); every prefilled row of response 3 and the first and last rows
    of the other sampled responses."""
    from helpers import OracleTrain
    Scenario = _gpu()
    from synth.scenario import TrainScenario
    import paper_2609_14717_amd as co
    w = wl.TRAIN_FWD
    tol = TOL[w.dtype]
    A = w.anchors
    a, u, a2 = wl.anchors(w)
    uf, a2f = u.ravel(), a2.ravel()
    sample = {0, A - 1, 7 * A, 8 * A - 1, int(np.argmin(a2f)), int(np.argmax(a2f))}
    for want in (0, w.B):                       # full acceptance, full rejection
        hit = np.flatnonzero(uf == want)
        if hit.size:
            sample.add(int(hit[0]))
    sample |= {int(x) for x in np.random.default_rng(5).choice(8 * A, 6, replace=False)}
    FULL = 3                                    # the response checked block by block
    sample |= set(range(FULL * A, (FULL + 1) * A))
    sample = sorted(sample)
    print(f"[parity] workload={w.name} sample={sample}", flush=True)
    sc = TrainScenario(w)
    out, lse = sc.forward()
    torch.cuda.synchronize()
    assert co.carryover_read_status(sc.vst) == 0 and co.carryover_read_status(sc.st) == 0
    orc = OracleTrain(w, sample)
    rr = orc.rr
    for key in ("accept_len", "row_pos", "row_dst"):
        np.testing.assert_array_equal(sc.vrt[key].cpu().numpy(), rr[key], err_msg=key)
    np.testing.assert_array_equal(sc.vst["ctx_len"].cpu().numpy(), rr["ctx_len"])
    np.testing.assert_array_equal(sc.vst["carry_len"].cpu().numpy(), rr["carry_len"])
    np.testing.assert_array_equal(rr["ctx_len"], a2f)
    g = to_np(out)
    gl = lse.cpu().numpy().astype(np.float64)
    for v in sample:
        nu = int(rr["carry_len"][v])
        for layer in range(w.L):
            if nu:
                gk, gv = gather_carry(sc.vst, v, layer, nu)
                assert_heads_close(gk, orc.st.uk[v][layer], tol, f"U_k v{v}")
                assert_heads_close(gv, orc.st.uv[v][layer], tol, f"U_v v{v}")
        assert_heads_close(g[:, v], orc.O[:, v], tol, f"O v{v}")
        err = np.abs(gl[:, v] - orc.LSE[:, v]).max()
        assert err <= tol, f"LSE v{v}: {err}"
    for s, (k, vv) in orc.parent.items():
        spans = [(0, w.seq_len)] if s == FULL else [(0, 40), (w.seq_len - 40, w.seq_len)]
        for layer in range(w.L):
            for t0, t1 in spans:
                gk, gv = gather_committed(sc.st, sc.pt, s, layer, t0, t1)
                assert_heads_close(gk, k[t0:t1, layer], tol, f"prefill K s{s}")
                assert_heads_close(gv, vv[t0:t1, layer], tol, f"prefill V s{s}")


# The grouped-prefix attention kernel on sequences with independent pages
# (every group streamed per wavefront), a partial last group (70 sequences),
# head_dim 128 with 32 query rows, and 64 query rows (served by the
# persistent kernel whatever the flag says).
SMALL_HD128_G2 = wl.Workload("small_hd128_g2", S=6, B=16, Dcat=512, d=256, L=2, Hq=4, Hkv=2,
                             hd=128, dtype="bf16", theta=1e6, ctx_lo=700, ctx_hi=700,
                             ctx_mode="projected", accept=("geom", 0.3), rounds=4, seed=0x5EED08)


@pytest.mark.parametrize("split", ["", "1", "3"], ids=lambda v: f"share{v or 'dflt'}")
@pytest.mark.parametrize("w", [SMALL_RAGGED, MANY_SEQS, SMALL_HD128_G2, SMALL_G4],
                         ids=lambda w: w.name)
def test_shared_prefix_flag_independent_pages(w, split, tune):
    import paper_2609_14717_amd as co
    if split:   # committed tiles per workgroup share: many shares, merged afterwards
        tune("attn_group_split_tiles", split)
    run_rounds(w, 2, extra_flags=co.CO_ATTN_SHARED_PREFIX)


# A small training-shaped forward checked for every block: 2 responses of 512
# positions, 10 anchored blocks each, so that groups of four blocks both share
# a response's pages and straddle two responses.
TRAIN_SMALL = wl.TRAIN_FWD.replace(name="train_small", S=2, seq_len=512, anchors=10,
                                   seed=0x5EED09)


def train_small_check(shared):
    from helpers import OracleTrain
    _gpu()
    from synth.scenario import TrainScenario
    import paper_2609_14717_amd as co
    w = TRAIN_SMALL
    tol = TOL[w.dtype]
    V = w.S * w.anchors
    print(f"[parity] workload={w.name} shared_prefix={shared}", flush=True)
    sc = TrainScenario(w)
    out, lse = sc.forward(shared_prefix=shared)
    torch.cuda.synchronize()
    assert co.carryover_read_status(sc.vst) == 0
    orc = OracleTrain(w, range(V))
    g = to_np(out)
    gl = lse.cpu().numpy().astype(np.float64)
    for v in range(V):
        assert_heads_close(g[:, v], orc.O[:, v], tol, f"O v{v}")
        err = np.abs(gl[:, v] - orc.LSE[:, v]).max()
        assert err <= tol, f"LSE v{v}: {err}"
        nu = int(orc.rr["carry_len"][v])
        if nu:
            gk, gv = gather_carry(sc.vst, v, 0, nu)
            assert_heads_close(gk, orc.st.uk[v][0], tol, f"U_k v{v}")
            assert_heads_close(gv, orc.st.uv[v][0], tol, f"U_v v{v}")
    for s, (k, vv) in orc.parent.items():
        gk, gv = gather_committed(sc.st, sc.pt, s, 0, 0, w.seq_len)
        assert_heads_close(gk, k[:, 0], tol, f"prefill K s{s}")
        assert_heads_close(gv, vv[:, 0], tol, f"prefill V s{s}")


@pytest.mark.parametrize("shared", [True, False], ids=["shared_prefix", "persistent"])
@pytest.mark.parametrize("split", ["", "3"], ids=lambda v: f"share{v or 'dflt'}")
def test_train_small_full(shared, split, tune):
    if split:
        tune("attn_group_split_tiles", split)
    train_small_check(shared)


# The fused small-width projection (both products in one kernel, Z in LDS),
# forced at small row counts: 80 rows (one partial 128-row block), the 512
# rows of the batch-32 round, and the committed and block calls of a small
# training-shaped forward.
FUSED_RAGGED = wl.RAGGED32.replace(name="fused_ragged", S=5, ctx_lo=100, ctx_hi=1500, rounds=3,
                                   seed=0x5EED0A)


@pytest.mark.parametrize("w", [FUSED_RAGGED, wl.RAGGED32], ids=lambda w: w.name)
def test_fused_projection(w, tune):
    tune("project_fused_min_rows", 1)
    run_rounds(w, 2)


def test_fused_projection_train_small(tune):
    tune("project_fused_min_rows", 1)
    train_small_check(True)


# Per-wavefront slices (head_dim 128, 64 query rows), forced on: full-size
# segments, pieces split over many slices (and several pieces per slice, with
# few workgroups), one-page contexts, carry-only windows and ragged lengths.
WAVE_RAGGED = wl.Workload("wave_ragged_hd128", S=6, B=16, Dcat=512, d=256, L=2, Hq=8, Hkv=2,
                          hd=128, dtype="bf16", theta=1e6, ctx_lo=1, ctx_hi=900,
                          ctx_mode="direct", accept=("geom", 0.3), rounds=4, seed=0x5EED0B)


@pytest.mark.parametrize("wgs", ["", "1", "3", "70"], ids=lambda v: f"wg{v or 'dflt'}")
@pytest.mark.parametrize("w", [SMALL_G4, BATCH3_8B, WAVE_RAGGED], ids=lambda w: w.name)
def test_wave_slices(w, wgs, tune):
    tune("attn_wave", 1)
    if wgs:
        tune("attn_workgroups", wgs)
    run_rounds(w, 3)


# The persistent path at the same shapes (no longer their default).
@pytest.mark.parametrize("w", [SMALL_G4, WAVE_RAGGED], ids=lambda w: w.name)
def test_persistent_hd128_64_rows(w, tune):
    tune("attn_wave", 0)
    run_rounds(w, 3)


# The same path at head_dim 64 (32 and 64 query rows, eight wavefronts per
# workgroup), forced on.  With 500 workgroups (4000 slices) most slices are
# empty and a segment's records span more than one merge batch; MANY_SEQS has
# enough segments for the merge's 16-dims-per-thread form.
@pytest.mark.parametrize("wgs", ["", "1", "5", "500"], ids=lambda v: f"wg{v or 'dflt'}")
@pytest.mark.parametrize("w", [SMALL_RAGGED, MANY_SEQS, WIDE64], ids=lambda w: w.name)
def test_wave_slices_hd64(w, wgs, tune):
    tune("attn_wave", 1)
    if wgs:
        tune("attn_workgroups", wgs)
    run_rounds(w, 3)
