"""GPU parity of the variants next to the drafter step, through the C ABI,
against the fp64 oracle:

* routing by the verifier's accept decisions (stochastic verification, T = 1;
  Appendix A, "Why verification remains valid"), whatever follows the first
  rejection;
* the separate-projector update (Section 4, Table 3(b)): carried rows through a
  second fusion matrix, no E, on the small-tile, split-K, large-tile and fp32
  GEMM paths;
* the attention mass on the carried rows (Appendix "Attention to carried
  states"), from a finished attention call's LSE;
* the RMS normalisation of F's output before the K/V product, and of every key
  head before its rotation;
* the block's own rows as a third attention segment, merged into the
  attention over [C;U].
"""
import numpy as np
import pytest

import oracle
from synth import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from helpers import TOL, OracleRun, assert_heads_close, compare_round, host, to_np  # noqa: E402

EDGE = wl.RAGGED32.replace(name="var_edge", S=4, L=2, ctx_lo=40, ctx_hi=900, rounds=8,
                           accept=("geom", 0.25), seed=0x5EED20)
EDGE_F32 = EDGE.replace(name="var_edge_f32", dtype="f32", seed=0x5EED21)
HD128 = wl.Workload("var_hd128", S=3, B=16, Dcat=512, d=256, L=1, Hq=8, Hkv=2, hd=128,
                    dtype="bf16", theta=1e6, ctx_lo=60, ctx_hi=700, ctx_mode="direct",
                    accept=("geom", 0.3), rounds=6, seed=0x5EED22)
# 256 window rows: the large-tile GEMM; 3 x 16 rows of 20480 features: split-K
WIDE = wl.Workload("var_wide", S=16, B=16, Dcat=512, d=256, L=1, Hq=4, Hkv=2, hd=64,
                   dtype="bf16", theta=1e4, ctx_lo=30, ctx_hi=300, ctx_mode="direct",
                   accept=("geom", 0.25), rounds=4, seed=0x5EED23)
SPLIT = wl.BATCH1_8B.replace(name="var_split", S=3, ctx_lo=200, ctx_hi=200, rounds=4,
                             seed=0x5EED24)


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from synth.scenario import Scenario
    import paper_2609_14717_amd as co
    return Scenario, co


def accept_bits(w, r, m, seed):
    """Accept decisions that realise accepted prefixes m: non-zero before m,
    zero at m, arbitrary (seeded) after the first rejection."""
    rng = np.random.default_rng(seed + r)
    bits = rng.integers(0, 2, (len(m), w.B)).astype(np.int32)
    for s, mm in enumerate(m):
        bits[s, :mm] = rng.integers(1, 1000, mm)
        if mm < w.B:
            bits[s, mm] = 0
    return bits


@pytest.mark.parametrize("w", [EDGE, EDGE_F32], ids=lambda w: w.name)
def test_accept_bits_rounds(w):
    Scenario, co = _gpu()
    print(f"[variants] accept bits {w.name}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    for r in range(4):
        hidden, q, _, _, m = sc.round_inputs(r)
        if r == 1:
            m = np.array([0, w.B, 1, w.B - 1], np.int32)
        bits = accept_bits(w, r, m, 0x5EED25)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, torch.from_numpy(bits).cuda(), None, q, sc.st,
                           sc.rt, out, lse, co.CO_ROUTE_ACCEPT_BITS, sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r, bits=bits)
        np.testing.assert_array_equal(rr["accept_len"], m)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} bits r{r}")


@pytest.mark.parametrize("w", [EDGE, EDGE_F32, WIDE, SPLIT], ids=lambda w: w.name)
def test_separate_projector_rounds(w, tune):
    Scenario, co = _gpu()
    if w is WIDE:      # the large-tile kernel at any row count from 256
        tune("gemm_wide_variant", 3)
    print(f"[variants] separate projector {w.name}", flush=True)
    sc = Scenario(w, separate_projector=True)
    orc = OracleRun(w, separate_projector=True)
    for r in range(3):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} sep r{r}")


@pytest.mark.parametrize("w", [EDGE, EDGE_F32, HD128], ids=lambda w: w.name)
def test_carry_mass(w):
    Scenario, co = _gpu()
    print(f"[variants] carry mass {w.name}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    tol = TOL[w.dtype]
    B, S = w.B, w.S
    plans = [None, [B] * S, [0] * S, [0, B, 1, B - 1][:S] + [3] * max(0, S - 4), None]
    for r, m in enumerate(plans):
        hidden, q, draft, target, m = sc.round_inputs(r, m)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        mass = torch.full_like(lse, float("nan"))
        co.drafter_carry_mass(sc.dims, 0, w.L, q, sc.st, lse, mass)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        orc.round(r, m=m, attend=False)
        Q = orc.seq_block(wl.spec_q(w, r), 1)
        ref = oracle.carry_mass_state(orc.st, Q, w.Hq, w.theta, seqs=orc.seqs)
        got = mass.cpu().numpy().astype(np.float64)
        for s in orc.seqs:
            err = np.abs(got[:, s] - ref[:, s]).max()
            assert err <= tol, f"{w.name} r{r} mass seq {s}: {err}"
            if m[s] == B:                      # nothing carried: exactly zero
                assert np.all(got[:, s] == 0.0)
        print(f"[variants] {w.name} round {r}: mean carried mass {np.nanmean(ref):.4f}",
              flush=True)


@pytest.mark.parametrize("w", [EDGE, EDGE_F32, WIDE, SPLIT], ids=lambda w: w.name)
def test_z_norm_rounds(w, tune):
    """F's output RMS-normalised (gain) before the K/V product."""
    Scenario, co = _gpu()
    if w is WIDE:
        tune("gemm_wide_variant", 3)
    print(f"[variants] z norm {w.name}", flush=True)
    sc = Scenario(w, z_norm=True)
    orc = OracleRun(w, z_norm=True)
    for r in range(3):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} znorm r{r}")


def test_z_norm_fused_path(tune):
    """Where the fused projection would run (forced at 80 rows), the
    normalised update takes the two-product path and stays correct."""
    tune("project_fused_min_rows", 1)
    _z_norm_small()


def _z_norm_small():
    Scenario, co = _gpu()
    w = wl.RAGGED32.replace(name="var_znorm_fused", S=5, rounds=3, ctx_lo=100, ctx_hi=900,
                            seed=0x5EED26)
    sc, orc = Scenario(w, z_norm=True), OracleRun(w, z_norm=True)
    for r in range(2):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} r{r}")


@pytest.mark.parametrize("w", [EDGE, EDGE_F32, HD128, WIDE, SPLIT], ids=lambda w: w.name)
def test_k_norm_rounds(w, tune):
    """Every key head RMS-normalised (per-layer gain) before its rotation, on
    the small-tile (hd 64 and 128), large-tile, split-K and fp32 epilogues,
    also together with the normalisation of F's output."""
    Scenario, co = _gpu()
    if w is WIDE:
        tune("gemm_wide_variant", 3)
    zn = w is SPLIT
    print(f"[variants] k norm {w.name} (z norm {zn})", flush=True)
    sc = Scenario(w, k_norm=True, z_norm=zn)
    orc = OracleRun(w, k_norm=True, z_norm=zn)
    for r in range(3):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} knorm r{r}")


def test_k_norm_fused_path(tune):
    """Where the fused projection would run (forced at 80 rows), normalised
    keys take the two-product path and stay correct."""
    tune("project_fused_min_rows", 1)
    Scenario, co = _gpu()
    w = wl.RAGGED32.replace(name="var_knorm_fused", S=5, rounds=3, ctx_lo=100, ctx_hi=900,
                            seed=0x5EED27)
    sc, orc = Scenario(w, k_norm=True), OracleRun(w, k_norm=True)
    for r in range(2):
        hidden, q, draft, target, m = sc.round_inputs(r)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} r{r}")


@pytest.mark.parametrize("w", [EDGE, EDGE_F32, HD128], ids=lambda w: w.name)
def test_self_merge(w):
    """The block's own rows as a third segment: attention over [C;U;S]."""
    Scenario, co = _gpu()
    print(f"[variants] self segment {w.name}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    tol = TOL[w.dtype]
    B, S = w.B, w.S
    plans = [None, [B] * S, [0] * S, None]
    for r, m in enumerate(plans):
        hidden, q, draft, target, m = sc.round_inputs(r, m)
        out, lse = sc.new_output()
        co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0,
                           sc.ws)
        ks, vs = sc.self_kv(r)
        co.drafter_self_merge(sc.dims, 0, w.L, q, ks, vs, sc.st, out, lse)
        torch.cuda.synchronize()
        assert co.carryover_read_status(sc.st) == 0
        orc.round(r, m=m, attend=False)
        Q = orc.seq_block(wl.spec_q(w, r), 1)
        Ks = host(w, wl.spec_self(w, "k", r))
        Vs = host(w, wl.spec_self(w, "v", r))
        O, LSE = oracle.attend_state_with_self(orc.st, Q, Ks, Vs, w.Hq, w.theta, seqs=orc.seqs)
        g = to_np(out)
        gl = lse.cpu().numpy().astype(np.float64)
        for s in orc.seqs:
            assert_heads_close(g[:, s], O[:, s], tol, f"{w.name} r{r} O seq {s}")
            err = np.abs(gl[:, s] - LSE[:, s]).max()
            assert err <= tol, f"{w.name} r{r} LSE seq {s}: {err}"


# ------------------------------------------------ extras inside the one-pass merge

B8 = EDGE.replace(name="ext_b8", B=8, seed=0x5EED25)
B48 = wl.Workload("ext_b48", S=3, B=48, Dcat=256, d=128, L=1, Hq=2, Hkv=2, hd=64, dtype="bf16",
                  theta=1e4, ctx_lo=30, ctx_hi=900, ctx_mode="direct", accept=("geom", 0.1),
                  rounds=4, seed=0x5EED26)
EXTRAS = ["self", "mass", "both"]


def _ext_round(co, sc, orc, w, r, m, extra, tag, empty=(), no_committed=()):
    """One round, then drafter_block_attention_ext on the state it left with
    the round's queries; compared with the oracle's attention over [C;U;S]
    (or [C;U]) and its carried mass over [C;U].  Before the call, sequences in
    ``empty`` lose their committed and carry keys, those in ``no_committed``
    their committed keys."""
    hidden, q, draft, target, m = sc.round_inputs(r, m)
    out, lse = sc.new_output()
    co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, 0, sc.ws)
    orc.round(r, m=m, attend=False)
    for s in set(empty) | set(no_committed):
        sc.st["ctx_len"][s] = 0
        orc._ctx[s] = 0
        for st_ in (orc.st.ck, orc.st.cv):
            st_[s] = st_[s][:, :0]
    for s in empty:
        sc.st["carry_len"][s] = 0
        orc._carry[s] = 0
        for st_ in (orc.st.uk, orc.st.uv):
            st_[s] = st_[s][:, :0]
    with_self = extra in ("self", "both")
    with_mass = extra in ("mass", "both")
    ks, vs = sc.self_kv(r) if with_self else (None, None)
    out2 = torch.full_like(out, float("nan"))
    lse2 = torch.full_like(lse, float("nan"))
    mass = torch.full_like(lse, float("nan")) if with_mass else None
    co.drafter_block_attention_ext(sc.dims, 0, w.L, q, ks, vs, sc.st, out2, lse2, mass, 0, sc.ws)
    torch.cuda.synchronize()
    assert co.carryover_read_status(sc.st) == 0
    Q = orc.seq_block(wl.spec_q(w, r), 1)
    if with_self:
        Ks = host(w, wl.spec_self(w, "k", r))
        Vs = host(w, wl.spec_self(w, "v", r))
        O, LSE = oracle.attend_state_with_self(orc.st, Q, Ks, Vs, w.Hq, w.theta, seqs=orc.seqs)
    else:
        O, LSE = oracle.attend_state(orc.st, Q, w.Hq, w.theta, seqs=orc.seqs)
    tol = TOL[w.dtype]
    g = to_np(out2)
    gl = lse2.cpu().numpy().astype(np.float64)
    for s in orc.seqs:
        assert_heads_close(g[:, s], O[:, s], tol, f"{tag} O seq {s}")
        err = np.abs(gl[:, s] - LSE[:, s])
        assert np.all(np.isfinite(err) | (np.isinf(gl[:, s]) & np.isinf(LSE[:, s]))), \
            f"{tag} LSE seq {s}"
        assert np.nanmax(np.where(np.isinf(LSE[:, s]), 0.0, err)) <= tol, f"{tag} LSE seq {s}"
    if with_mass:
        ref = oracle.carry_mass_state(orc.st, Q, w.Hq, w.theta, seqs=orc.seqs)
        got = mass.cpu().numpy().astype(np.float64)
        for s in orc.seqs:
            err = np.abs(got[:, s] - ref[:, s]).max()
            assert err <= tol, f"{tag} mass seq {s}: {err}"
            if orc.st.uk[s].shape[1] == 0:     # nothing carried: exactly zero
                assert np.all(got[:, s] == 0.0), f"{tag} mass seq {s} not zero"
    return m


@pytest.mark.parametrize("extra", EXTRAS)
@pytest.mark.parametrize("w", [EDGE, EDGE_F32, HD128, B8, B48], ids=lambda w: w.name)
def test_attention_ext(w, extra):
    """The block's own rows and the carried mass inside the one-pass merge
    (bf16) or through the post-pass kernels (fp32): full and zero acceptance,
    a mix, head_dim 64 and 128, blocks of 8, 16 and 48 rows (two self tiles)."""
    Scenario, co = _gpu()
    print(f"[variants] ext {extra} {w.name}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    B, S = w.B, w.S
    for r, m in enumerate([None, [B] * S, [0] * S, None]):
        _ext_round(co, sc, orc, w, r, m, extra, f"{w.name} {extra} r{r}")


@pytest.mark.parametrize("wgs", ["1", "3", "70", "500"], ids=lambda v: f"wg{v}")
def test_attention_ext_slicings(wgs, tune):
    """Forced slicings of the persistent kernel with both extras: segments
    split across workgroups and wavefronts, self keys processed by whichever
    wavefront holds a segment's last tile."""
    Scenario, co = _gpu()
    tune("attn_workgroups", wgs)
    w = EDGE
    print(f"[variants] ext slicing wg={wgs}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    for r in range(3):
        _ext_round(co, sc, orc, w, r, None, "both", f"wg{wgs} r{r}")


def test_attention_ext_empty_context():
    """A sequence with no committed and no carry keys attends to its self keys
    alone (mass 0); another has carry keys only (mass 1 without self keys)."""
    Scenario, co = _gpu()
    w = EDGE
    sc, orc = Scenario(w), OracleRun(w)
    _ext_round(co, sc, orc, w, 0, [0, 3, w.B, 5], "both", "empty ctx", empty=(0,),
               no_committed=(1,))
    sc2, orc2 = Scenario(w), OracleRun(w)
    _ext_round(co, sc2, orc2, w, 0, [0, 3, w.B, 5], "mass", "carry only", no_committed=(1,))


# 64 block rows of one query head per KV head: 64 query rows at head_dim 128
# (the slices kernel's shape) and two self tiles
HD128_B64 = wl.Workload("ext_hd128_b64", S=3, B=64, Dcat=256, d=128, L=1, Hq=1, Hkv=1, hd=128,
                        dtype="bf16", theta=1e6, ctx_lo=30, ctx_hi=700, ctx_mode="direct",
                        accept=("geom", 0.1), rounds=4, seed=0x5EED27)


@pytest.mark.parametrize("wgs", ["", "1", "7"], ids=lambda v: f"wg{v or 'dflt'}")
@pytest.mark.parametrize("w", [EDGE, HD128, HD128_B64], ids=lambda w: w.name)
def test_attention_ext_wave_slices(w, wgs, tune):
    """Both extras on the per-wavefront slices kernel (head_dim 64 forced onto
    it, head_dim 128 there by default; 64 block rows: two self tiles staged
    through LDS), default and forced slice counts."""
    Scenario, co = _gpu()
    tune("attn_wave", 1)
    if wgs:
        tune("attn_workgroups", wgs)
    print(f"[variants] ext wave slices {w.name} wg={wgs or 'dflt'}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    for r, m in enumerate([None, [w.B] * w.S, [0] * w.S]):
        _ext_round(co, sc, orc, w, r, m, "both", f"wave {w.name} wg{wgs} r{r}",
                   empty=(1,) if r == 2 else ())
