"""GPU parity of stochastic verification (T = 1; Appendix A, "Why
verification remains valid"): accept decisions, accepted lengths and the
correction or bonus token of every sequence bit-exact against the oracle, and
the decisions routed by carryover_route / carryover_round under
CO_ROUTE_ACCEPT_BITS."""
import numpy as np
import pytest

import oracle
from synth import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(w, draft, p, q, words):
    import paper_2609_14717_amd as co
    S, B = draft.shape
    V = p.shape[-1]
    dims = co.make_dims(S, B, w.Dcat, w.d, w.L, w.Hq, w.Hkv, w.hd, 4, 4, w.dtype, w.theta)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    d_draft, d_p, d_q = dev(draft), dev(p), dev(q)
    d_words = dev(words.view(np.int32))
    bits = torch.full((S, B), -7, dtype=torch.int32, device="cuda")
    m = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    nxt = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    co.carryover_verify_sample(dims, V, d_draft, d_p, d_q, d_words, bits, m, nxt, status)
    torch.cuda.synchronize()
    return bits.cpu().numpy(), m.cpu().numpy(), nxt.cpu().numpy(), int(status.item())


def _check(w, draft, p, q, words, what):
    print(f"[verify] {what} S={draft.shape[0]} B={draft.shape[1]} V={p.shape[-1]}", flush=True)
    bits, m, nxt, status = _run(w, draft, p, q, words)
    want = [oracle.verify_sample(draft[s], p[s], q[s], words[s]) for s in range(len(draft))]
    np.testing.assert_array_equal(m, [x[0] for x in want], err_msg=f"{what}: accept_len")
    np.testing.assert_array_equal(nxt, [x[1] for x in want], err_msg=f"{what}: next token")
    B = draft.shape[1]
    np.testing.assert_array_equal(bits, (np.arange(B)[None, :] < m[:, None]).astype(np.int32))
    codes = {x[2] for x in want} - {oracle.OK}
    assert status == (codes.pop() if codes else 0)
    return m


@pytest.mark.parametrize("rnd", [0, 1, 2])
def test_verify_batch32_vocab1000(rnd):
    """The batch-32 serving round's shape (B = 16) over a 1000-token vocabulary."""
    _gpu()
    w = wl.RAGGED32
    _check(w, *wl.verify_inputs(w, rnd, 1000), f"batch32 round {rnd}")


@pytest.mark.parametrize("V", [1, 3, 1023, 1024, 1025, 4099, 32000])
def test_verify_ragged_vocabularies(V):
    """Vocabularies below, at and across the kernel's 1024-token steps."""
    _gpu()
    w = wl.RAGGED32.replace(B=7, seed=0x5EED21)
    _check(w, *wl.verify_inputs(w, 0, V, S=9), f"V={V}")


def test_verify_edge_cases():
    """p = q (every proposal accepted: bonus from p after the block); a
    proposal with zero probability under both (always rejected, and its
    residual is zero everywhere: the correction falls back to p); an empty
    bonus distribution (no token, -1); a window of 64 positions (two ballots)."""
    _gpu()
    w = wl.RAGGED32.replace(B=64, seed=0x5EED22)
    draft, p, q, words = wl.verify_inputs(w, 0, 300, S=6)
    q[0] = p[0, :64]                                      # p = q: all accepted
    q[1] = p[1, :64]
    x = draft[1, 5]
    p[1, 5, :] = 0.0
    p[1, 5, (x + 1) % 300] = 1.0
    q[1, 5] = p[1, 5]                                     # zero residual at the rejection
    p[1, 5, x] = q[1, 5, x] = 0.0
    q[2] = p[2, :64]
    p[2, 64] = 0.0                                        # no bonus distribution
    m = _check(w, draft, p, q, words, "edges")
    assert m[0] == 64 and m[1] == 5 and m[2] == 64


def test_verify_out_of_vocabulary_token_sets_status():
    _gpu()
    w = wl.RAGGED32.replace(B=5, seed=0x5EED23)
    draft, p, q, words = wl.verify_inputs(w, 0, 50, S=4)
    draft[2, 3] = 50
    m = _check(w, draft, p, q, words, "token range")
    assert m[2] == 0


def test_verified_decisions_drive_the_round():
    """The accept decisions written by the verification are the route's input
    under CO_ROUTE_ACCEPT_BITS: the round commits exactly the verified prefix."""
    _gpu()
    import paper_2609_14717_amd as co
    from synth.scenario import Scenario
    w = wl.RAGGED32.replace(name="verify_round", S=6, L=1, ctx_lo=100, ctx_hi=900, rounds=2,
                            seed=0x5EED24)
    sc = Scenario(w)
    draft, p, q, words = wl.verify_inputs(w, 0, 1000)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    bits = torch.zeros((w.S, w.B), dtype=torch.int32, device="cuda")
    m = torch.zeros(w.S, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(w.S, dtype=torch.int32, device="cuda")
    co.carryover_verify_sample(sc.dims, 1000, dev(draft), dev(p), dev(q), dev(words.view(np.int32)),
                               bits, m, nxt, sc.st["status"])
    ctx0 = sc.st["ctx_len"].clone()
    hidden, qq, _, _, _ = sc.round_inputs(0)
    out, lse = sc.new_output()
    co.carryover_round(sc.dims, sc.W, hidden, bits, None, qq, sc.st, sc.rt, out, lse,
                       co.CO_ROUTE_ACCEPT_BITS, sc.ws)
    torch.cuda.synchronize()
    assert co.carryover_read_status(sc.st) == 0
    want = np.array([oracle.verify_sample(draft[s], p[s], q[s], words[s])[0] for s in range(w.S)])
    np.testing.assert_array_equal(sc.rt["accept_len"].cpu().numpy(), want)
    np.testing.assert_array_equal((sc.st["ctx_len"] - ctx0).cpu().numpy(), want)
    np.testing.assert_array_equal(sc.st["carry_len"].cpu().numpy(), w.B - want)
