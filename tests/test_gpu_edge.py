"""GPU edge cases of the drafter step, through the C ABI, against the fp64
oracle (or, where the paper fixes an identity, GPU against GPU bit for bit):
full and zero acceptance, zero carry = baseline, stale rows that must never be
read, empty key sets, capacity and page-range errors, pre-rotated queries,
layer subsets, the fused round against its three calls, every query-tile /
head-dim kernel variant, and an empty batch."""
import numpy as np
import pytest

from synth import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from helpers import TOL, OracleRun, assert_heads_close, compare_round, to_np  # noqa: E402

EDGE = wl.RAGGED32.replace(name="edge", S=4, L=2, ctx_lo=40, ctx_hi=900, rounds=8,
                           accept=("geom", 0.25), seed=0x5EED10)
# one drafter layer (K/V width 256): the shape of the batch-32 serving workload
EDGE1 = EDGE.replace(name="edge_l1", L=1, seed=0x5EED11)
# the fp32 path (chunked attention, split-K fp32 GEMM) on the same cases
EDGE_F32 = EDGE.replace(name="edge_f32", dtype="f32", seed=0x5EED12)
BOTH = pytest.mark.parametrize("w", [EDGE, EDGE1, EDGE_F32], ids=lambda w: w.name)


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from synth.scenario import Scenario
    import paper_2609_14717_amd as co
    return Scenario, co


def _round(co, sc, r, m=None, flags=0):
    hidden, q, draft, target, m = sc.round_inputs(r, m)
    out, lse = sc.new_output()
    co.carryover_round(sc.dims, sc.W, hidden, draft, target, q, sc.st, sc.rt, out, lse, flags,
                       sc.ws)
    torch.cuda.synchronize()
    return out, lse, q


@BOTH
def test_full_and_zero_acceptance(w):
    """m = B everywhere (carry segment empty), m = 0 everywhere (nothing
    committed, a full block carried), then a mix of both extremes."""
    Scenario, co = _gpu()
    B = w.B
    sc, orc = Scenario(w), OracleRun(w)
    for r, m in enumerate([[B] * 4, [0] * 4, [0, B, 1, B - 1], [B, 0, B, 0]]):
        out, lse, _ = _round(co, sc, r, m)
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r, m=m)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"edge m={m}")


@BOTH
def test_zero_carry_equals_baseline_bitexact(w):
    """With every proposal accepted, the carryover update equals the baseline
    update (Algorithm 1's two columns coincide): identical bits on the GPU."""
    Scenario, co = _gpu()
    a, b = Scenario(w), Scenario(w)
    for r in range(3):
        m = [w.B] * w.S
        oa, la, _ = _round(co, a, r, m, 0)
        ob, lb, _ = _round(co, b, r, m, co.CO_BASELINE_MODE)
        assert torch.equal(oa, ob) and torch.equal(la, lb)
        for key in ("k_cache", "v_cache", "ctx_len", "carry_len"):
            assert torch.equal(a.st[key], b.st[key]), key


def _poison(sc):
    """NaN into every carry row and every cache slot no sequence holds."""
    st = sc.st
    st["k_carry"].fill_(float("nan"))
    st["v_carry"].fill_(float("nan"))
    ctx = st["ctx_len"].cpu().numpy()
    pt = st["page_table"].cpu().numpy()
    live = np.zeros((st["k_cache"].shape[1], 16), bool)
    for s, n in enumerate(ctx):
        pos = np.arange(n)
        live[pt[s][pos // 16], pos % 16] = True
    dead = torch.from_numpy(~live).to(st["k_cache"].device)
    st["k_cache"].masked_fill_(dead[None, :, None, :, None], float("nan"))
    st["v_cache"].masked_fill_(dead[None, :, None, None, :], float("nan"))


@BOTH
def test_stale_rows_are_never_read(w):
    """Replace, never grow: the previous carry segment and every slot past a
    sequence's committed length may hold anything (NaN here); the next round's
    results are finite and identical to the unpoisoned run's."""
    Scenario, co = _gpu()
    a, b = Scenario(w), Scenario(w)
    orc = OracleRun(w)
    for r in range(4):
        if r >= 1:
            _poison(b)
        oa, la, _ = _round(co, a, r)
        ob, lb, _ = _round(co, b, r)
        rr, O, LSE = orc.round(r)
        assert torch.isfinite(ob.float()).all() and torch.equal(oa, ob) and torch.equal(la, lb)
        compare_round(a, orc, rr, O, LSE, oa, la, a.rt, orc.seqs, f"poison r{r}")


def test_empty_key_set_and_null_lse():
    """A sequence with no committed and no carried keys gets O = 0 and
    LSE = -inf; the others are unaffected; lse may be omitted."""
    Scenario, co = _gpu()
    w = EDGE
    sc, orc = Scenario(w), OracleRun(w)
    out, lse, q = _round(co, sc, 0)
    rr, O, LSE = orc.round(0)
    for s in (1, 3):                       # empty both segments of two sequences
        sc.st["ctx_len"][s] = 0
        sc.st["carry_len"][s] = 0
        empty = np.zeros((w.L, 0, w.Hkv, w.hd))
        orc.st.ck[s], orc.st.cv[s], orc.st.uk[s], orc.st.uv[s] = empty, empty, empty, empty
    O, LSE = oracle_attend(orc, q)
    out, lse = sc.new_output()
    co.drafter_block_attention(sc.dims, 0, w.L, q, sc.st, out, lse, 0, sc.ws)
    out2, _ = sc.new_output()
    co.drafter_block_attention(sc.dims, 0, w.L, q, sc.st, out2, None, 0, sc.ws)
    torch.cuda.synchronize()
    assert co.carryover_read_status(sc.st) == 0
    g, gl = to_np(out), lse.cpu().numpy()
    for s in range(w.S):
        if s in (1, 3):
            assert np.all(g[:, s] == 0) and np.all(np.isneginf(gl[:, s]))
        else:
            assert_heads_close(g[:, s], O[:, s], TOL[w.dtype], f"O s{s}")
            assert np.abs(gl[:, s] - LSE[:, s]).max() <= TOL[w.dtype]
    assert torch.equal(out, out2)


def oracle_attend(orc, q):
    import oracle
    Q = to_np(q)
    return oracle.attend_state(orc.st, Q, orc.w.Hq, orc.w.theta)


@BOTH
def test_capacity_error_leaves_sequence_unchanged(w):
    """A window that would pass the sequence's capacity is refused
    (CO_ERR_CAPACITY): that sequence keeps its lengths and stores nothing,
    the others proceed."""
    Scenario, co = _gpu()
    bad = 2
    sc = Scenario(w)
    orc = OracleRun(w, seqs=[0, 1, 3])
    cap = w.max_pages_per_seq * 16
    sc.st["ctx_len"][bad] = cap - w.B + 1
    orc._ctx[bad] = cap - w.B + 1
    out, lse, _ = _round(co, sc, 0)
    assert co.carryover_read_status(sc.st) == co.CO_ERR_CAPACITY
    rr, O, LSE = orc.round(0)
    assert rr["status"][bad] != 0 and rr["accept_len"][bad] == 0
    assert np.all(rr["row_dst"][bad] == -(2 ** 31))
    compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, [0, 1, 3], "capacity")
    for key in ("accept_len", "row_pos", "row_dst"):
        np.testing.assert_array_equal(sc.rt[key].cpu().numpy()[bad], rr[key][bad])
    assert int(sc.st["ctx_len"][bad]) == cap - w.B + 1 and int(sc.st["carry_len"][bad]) == 0


@BOTH
def test_page_range_error_leaves_sequence_unchanged(w):
    """A committed row whose page id is outside the pool is refused
    (CO_ERR_PAGE_RANGE): that sequence keeps its lengths, the others proceed."""
    Scenario, co = _gpu()
    bad = 3
    sc = Scenario(w)
    orc = OracleRun(w, seqs=[0, 1, 2])
    p0 = int(sc.ctx0[bad])
    page = (p0 + w.B - 1) // 16    # written by the window's last row; past the committed pages
    sc.st["page_table"][bad, page] = sc.dims.num_pages + 7
    orc.pt = orc.pt.copy()
    orc.pt[bad, page] = sc.dims.num_pages + 7
    m = [3, 5, 7, w.B]                            # the bad sequence commits its whole window
    out, lse, _ = _round(co, sc, 0, m)
    assert co.carryover_read_status(sc.st) == co.CO_ERR_PAGE_RANGE
    rr, O, LSE = orc.round(0, m=m)
    assert rr["status"][bad] != 0
    compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, [0, 1, 2], "page range")
    np.testing.assert_array_equal(sc.rt["row_dst"].cpu().numpy()[bad], rr["row_dst"][bad])
    assert int(sc.st["ctx_len"][bad]) == p0


def test_prerotated_queries():
    """CO_Q_PREROTATED: queries rotated by the caller (here with the oracle's
    rotation, then rounded to bf16) give the same attention."""
    import oracle
    Scenario, co = _gpu()
    w = EDGE
    sc, orc = Scenario(w), OracleRun(w)
    out, lse, q = _round(co, sc, 0)
    rr, O, LSE = orc.round(0)
    Q = to_np(q)
    ctx = rr["ctx_len"]
    qr = np.empty_like(Q)
    for s in range(w.S):
        pos = ctx[s] + np.arange(w.B)
        for layer in range(w.L):
            for h in range(w.Hq):
                qr[layer, s, :, h] = oracle.rope(Q[layer, s, :, h], pos, w.theta)
    qt = torch.from_numpy(qr).to(q.device).to(q.dtype).contiguous()
    out2, lse2 = sc.new_output()
    co.drafter_block_attention(sc.dims, 0, w.L, qt, sc.st, out2, lse2, co.CO_Q_PREROTATED, sc.ws)
    torch.cuda.synchronize()
    g = to_np(out2)
    for s in range(w.S):
        assert_heads_close(g[:, s], O[:, s], TOL[w.dtype], f"prerotated O s{s}")


def test_layer_subset():
    """Attention over layers [1, 2) only: q and out start at that layer."""
    Scenario, co = _gpu()
    w = EDGE
    sc, orc = Scenario(w), OracleRun(w)
    out, lse, q = _round(co, sc, 0)
    rr, O, LSE = orc.round(0)
    q1 = q[1:2].contiguous()
    out1 = torch.empty_like(q1)
    lse1 = torch.empty((1, w.S, w.B, w.Hq), dtype=torch.float32, device=q.device)
    co.drafter_block_attention(sc.dims, 1, 1, q1, sc.st, out1, lse1, 0, sc.ws)
    torch.cuda.synchronize()
    g = to_np(out1)
    for s in range(w.S):
        assert_heads_close(g[0, s], O[1, s], TOL[w.dtype], f"layer 1 O s{s}")
        assert np.abs(lse1[0, s].cpu().numpy() - LSE[1, s]).max() <= TOL[w.dtype]


@BOTH
def test_round_equals_its_three_calls_bitexact(w):
    """carryover_round == carryover_route + carryover_project_kv +
    drafter_block_attention on the same stream, bit for bit."""
    Scenario, co = _gpu()
    a, b = Scenario(w), Scenario(w)
    for r in range(3):
        oa, la, _ = _round(co, a, r)
        hidden, q, draft, target, _ = b.round_inputs(r)
        ob, lb = b.new_output()
        co.carryover_route(b.dims, draft, target, 0, b.st, b.rt)
        co.carryover_project_kv(b.dims, b.W, hidden, b.rt, b.st, b.ws, ws_bytes=b.ws_project)
        wsa = b.ws[b.ws_project:]
        co.drafter_block_attention(b.dims, 0, w.L, q, b.st, ob, lb, 0, wsa)
        torch.cuda.synchronize()
        assert torch.equal(oa, ob) and torch.equal(la, lb)
        for key in ("k_cache", "v_cache", "k_carry", "v_carry", "ctx_len", "carry_len"):
            assert torch.equal(a.st[key], b.st[key]), key


# one workload per bf16 attention instantiation: query tiles of 16 rows (B x G)
# by head_dim; the others (2 tiles at 64, 4 tiles at 128) run in the parity suite
SHAPES = [
    wl.Workload("nt1_hd64", S=3, B=16, Dcat=256, d=128, L=1, Hq=2, Hkv=2, hd=64, dtype="bf16",
                theta=1e4, ctx_lo=50, ctx_hi=1500, ctx_mode="direct", accept=("geom", 0.3),
                rounds=3, seed=0x5EED21),
    wl.Workload("nt3_hd64", S=3, B=16, Dcat=256, d=128, L=1, Hq=6, Hkv=2, hd=64, dtype="bf16",
                theta=1e4, ctx_lo=50, ctx_hi=1500, ctx_mode="direct", accept=("geom", 0.3),
                rounds=3, seed=0x5EED22),
    wl.Workload("nt4_hd64_b64", S=3, B=64, Dcat=256, d=128, L=1, Hq=2, Hkv=2, hd=64,
                dtype="bf16", theta=1e4, ctx_lo=50, ctx_hi=1500, ctx_mode="direct",
                accept=("geom", 0.1), rounds=3, seed=0x5EED23),
    wl.Workload("nt1_hd128", S=3, B=16, Dcat=256, d=128, L=1, Hq=2, Hkv=2, hd=128, dtype="bf16",
                theta=1e6, ctx_lo=50, ctx_hi=1500, ctx_mode="direct", accept=("geom", 0.3),
                rounds=3, seed=0x5EED24),
    wl.Workload("nt2_hd128", S=3, B=16, Dcat=256, d=128, L=1, Hq=4, Hkv=2, hd=128, dtype="bf16",
                theta=1e6, ctx_lo=50, ctx_hi=1500, ctx_mode="direct", accept=("geom", 0.3),
                rounds=3, seed=0x5EED25),
    wl.Workload("nt3_hd128_b48", S=3, B=48, Dcat=256, d=128, L=1, Hq=2, Hkv=2, hd=128,
                dtype="bf16", theta=1e6, ctx_lo=50, ctx_hi=1500, ctx_mode="direct",
                accept=("geom", 0.1), rounds=3, seed=0x5EED26),
    # 64 query rows at head_dim 128 (the wavefront-slices kernel) with two query
    # heads per KV head: rows of one position are lane pairs, not quads, so each
    # lane computes its own rotation angles
    wl.Workload("g2_hd128_b32", S=3, B=32, Dcat=256, d=128, L=1, Hq=4, Hkv=2, hd=128,
                dtype="bf16", theta=1e6, ctx_lo=50, ctx_hi=1500, ctx_mode="direct",
                accept=("geom", 0.2), rounds=3, seed=0x5EED2A),
]


@pytest.mark.parametrize("w", SHAPES, ids=lambda w: w.name)
def test_kernel_variants(w):
    Scenario, co = _gpu()
    print(f"[edge] workload={w.name}", flush=True)
    sc, orc = Scenario(w), OracleRun(w)
    for r in range(2):
        out, lse, _ = _round(co, sc, r)
        assert co.carryover_read_status(sc.st) == 0
        rr, O, LSE = orc.round(r)
        compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"{w.name} r{r}")


def test_empty_batch_is_a_no_op():
    """num_seqs = 0: every call succeeds and launches nothing."""
    _, co = _gpu()
    w = EDGE
    dims = co.make_dims(0, w.B, w.Dcat, w.d, w.L, w.Hq, w.Hkv, w.hd, 4, 8, w.dtype, w.theta)
    one = lambda dt=torch.int32: torch.zeros(64, dtype=dt, device="cuda")
    st = dict(ctx_len=one(), carry_len=one(), page_table=one(), k_cache=one(torch.bfloat16),
              v_cache=one(torch.bfloat16), k_carry=one(torch.bfloat16),
              v_carry=one(torch.bfloat16), status=one())
    rt = dict(accept_len=one(), row_pos=one(), row_dst=one())
    buf = one(torch.bfloat16)
    wsz = max(co.workspace_bytes(dims, co.CO_WS_ROUND), 256)
    ws = torch.zeros(wsz, dtype=torch.uint8, device="cuda")
    W = co.weights(buf, buf, buf)
    co.carryover_round(dims, W, buf, one(), one(), buf, st, rt, buf, one(torch.float32), 0, ws)
    co.drafter_block_attention(dims, 0, w.L, buf, st, buf, None, 0, ws)
    torch.cuda.synchronize()
    assert co.carryover_read_status(st) == 0
    assert torch.count_nonzero(buf) == 0


@pytest.mark.parametrize("which", ["f_e", "z_norm", "k_norm", "w_f_carry", "lse"])
def test_round_rejected_on_the_host_leaves_the_state_untouched(which):
    """A misaligned optional pointer of any step makes carryover_round return
    CO_ERR_INVALID_ARG before its first launch: lengths, route output and
    caches are exactly as before; the next valid round then runs as usual."""
    Scenario, co = _gpu()
    w = EDGE1
    sc, orc = Scenario(w), OracleRun(w)
    print(f"[edge] misaligned {which}", flush=True)
    before = {k: v.clone() for k, v in sc.st.items()}
    rt_before = {k: v.clone() for k, v in sc.rt.items()}
    hidden, q, draft, target, _ = sc.round_inputs(0)
    out, lse = sc.new_output()
    bad = sc.ws.data_ptr() + 2
    W = co.weights(sc.wf, sc.wkv, sc.e, bad if which == "f_e" else sc.f_e,
                   bad if which == "w_f_carry" else None, bad if which == "z_norm" else None,
                   bad if which == "k_norm" else None)
    with pytest.raises(co.CarryoverError) as ei:
        co.carryover_round(sc.dims, W, hidden, draft, target, q, sc.st, sc.rt, out,
                           bad if which == "lse" else lse, 0, sc.ws)
    assert ei.value.code == co.CO_ERR_INVALID_ARG
    torch.cuda.synchronize()
    for k, v in before.items():
        assert torch.equal(sc.st[k], v), k
    for k, v in rt_before.items():
        assert torch.equal(sc.rt[k], v), k
    out, lse, _ = _round(co, sc, 0)
    assert co.carryover_read_status(sc.st) == 0
    rr, O, LSE = orc.round(0)
    compare_round(sc, orc, rr, O, LSE, out, lse, sc.rt, orc.seqs, f"after rejected {which}")


# 64 chained rounds on contexts that grow across page boundaries, two layers,
# head_dim 64 and 128 (the two attention kernels of a serving round)
SPLIT = [EDGE.replace(name="split_hd64", S=5, rounds=64, accept=("geom", 0.3), seed=0x5EED40),
         wl.Workload("split_hd128", S=3, B=16, Dcat=512, d=256, L=2, Hq=8, Hkv=2, hd=128,
                     dtype="bf16", theta=1e6, ctx_lo=30, ctx_hi=700, ctx_mode="direct",
                     accept=("geom", 0.3), rounds=64, seed=0x5EED41)]


def _chain(co, sc, rounds, keep):
    """Rounds ``rounds`` of sc's chain; (out, lse) of each on the host in keep."""
    for r in rounds:
        out, lse, _ = _round(co, sc, r)
        assert co.carryover_read_status(sc.st) == 0
        keep[r] = (out.cpu(), lse.cpu())


def _live_rows(sc):
    """Every committed row [0, ctx_len) (gathered by logical position) and every
    carry row [0, carry_len) of every sequence and layer."""
    from helpers import gather_carry, gather_committed
    ctx = sc.st["ctx_len"].cpu().numpy()
    car = sc.st["carry_len"].cpu().numpy()
    rows = []
    for s in range(sc.w.S):
        for layer in range(sc.w.L):
            rows += gather_committed(sc.st, sc.pt, s, layer, 0, int(ctx[s]))
            rows += gather_carry(sc.st, s, layer, int(car[s]))
    return rows


@pytest.mark.parametrize("w", SPLIT, ids=lambda w: w.name)
def test_split_chain_equals_one_chain(w):
    """A chain of 64 rounds equals 32 rounds, a copy of the whole drafter state
    into freshly allocated buffers, and 32 more rounds on the copy: every
    round's output and LSE and every live committed and carry row bit for bit.
    Also the rewind the benchmark times from: after round 63, restoring only
    the lengths saved after round 31 and running rounds 32..63 again gives the
    same outputs bit for bit (rows beyond ctx_len are never read and the carry
    segment is replaced before it is read)."""
    Scenario, co = _gpu()
    R, H = w.rounds, w.rounds // 2
    print(f"[edge] split chain workload={w.name} rounds={R}", flush=True)
    a = Scenario(w)
    one = {}
    _chain(co, a, range(H), one)
    snap = (a.st["ctx_len"].clone(), a.st["carry_len"].clone())
    _chain(co, a, range(H, R), one)

    b = Scenario(w)
    two = {}
    _chain(co, b, range(H), two)
    fresh = co.alloc_state(b.dims, b.pt, "cuda")
    for k in fresh:
        fresh[k].copy_(b.st[k])
    b.st = fresh
    torch.cuda.synchronize()
    _chain(co, b, range(H, R), two)
    for r in range(R):
        assert torch.equal(one[r][0], two[r][0]) and torch.equal(one[r][1], two[r][1]), f"r{r}"
    for key in ("ctx_len", "carry_len"):
        assert torch.equal(a.st[key], b.st[key]), key
    for x, y in zip(_live_rows(a), _live_rows(b)):
        assert np.array_equal(x, y)

    a.st["ctx_len"].copy_(snap[0])
    a.st["carry_len"].copy_(snap[1])
    again = {}
    _chain(co, a, range(H, R), again)
    for r in range(H, R):
        assert torch.equal(one[r][0], again[r][0]) and torch.equal(one[r][1], again[r][1]), \
            f"rewound r{r}"
