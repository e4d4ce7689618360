"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Routing, acceptance lengths, descriptors and lengths must match bit for bit;
floating-point outputs (attention O and LSE, the committed rows written this
round, the carry rows) must match per head vector within 2e-2 (bf16) or 1e-4
(fp32) of max relative error.
"""
import numpy as np
import pytest

from synth import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from helpers import (TOL, OracleRun, assert_heads_close, gather_carry, gather_committed,  # noqa: E402
                     to_np)

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


def run_rounds(w, n_rounds, mode="carry", seqs=None, check_context=True):
    import paper_2609_14717_amd as co
    Scenario = _gpu()
    print(f"[parity] workload={w.name} rounds={n_rounds} mode={mode}", flush=True)
    sc = Scenario(w)
    orc = OracleRun(w, seqs=seqs)
    seqs = orc.seqs
    if check_context and w.ctx_mode == "projected" and w.ctx_lo:
        n = int(sc.ctx0[0])
        for s in seqs[:2]:
            gk, gv = gather_committed(sc.st, sc.pt, s, 0, 0, n)
            assert_heads_close(gk, orc.st.ck[s][0], TOL[w.dtype], "prefill K")
            assert_heads_close(gv, orc.st.cv[s][0], TOL[w.dtype], "prefill V")
    flags = {"carry": 0, "baseline": co.CO_BASELINE_MODE}[mode]
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
def test_attention_slicings(w, slicing, monkeypatch):
    monkeypatch.setenv("CO_ATTN_WORKGROUPS", slicing[0])
    if slicing[1]:
        monkeypatch.setenv("CO_ATTN_ROUND_TILES", slicing[1])
    run_rounds(w, 2)
