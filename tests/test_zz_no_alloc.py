"""carryover_round_noalloc (the round on the library's static device scratch,
for callers that cannot allocate) against carryover_round with a caller
workspace: the same inputs on two identical states give bit-identical
outputs, routes, lengths and caches.  Two workloads in a row, the second
smaller, so that the second call runs on the scratch the first one left."""
import numpy as np
import pytest

from synth import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

BIG = wl.RAGGED32                                   # the batch-32 serving round
SMALL = wl.RAGGED32.replace(name="noalloc_small", S=3, L=2, ctx_lo=60, ctx_hi=700, rounds=4,
                            seed=0x5EED31)


def _same(a, b, what):
    assert torch.equal(a, b), what


def _compare(w, rounds):
    import paper_2609_14717_amd as co
    from synth.scenario import Scenario
    print(f"[noalloc] workload={w.name} S={w.S} rounds={rounds}", flush=True)
    ref, new = Scenario(w), Scenario(w)
    for r in range(rounds):
        hidden, q, draft, target, _ = ref.round_inputs(r)
        out_a, lse_a = ref.new_output()
        out_b, lse_b = new.new_output()
        out_b.fill_(7)
        lse_b.fill_(7)
        co.carryover_round(ref.dims, ref.W, hidden, draft, target, q, ref.st, ref.rt, out_a,
                           lse_a, 0, ref.ws)
        co.carryover_round_noalloc(new.dims, new.W, hidden, draft, target, q, new.st, new.rt,
                                   out_b, lse_b, 0)
        torch.cuda.synchronize()
        assert co.carryover_read_status(ref.st) == 0 and co.carryover_read_status(new.st) == 0
        _same(out_a, out_b, f"r{r} out")
        _same(lse_a, lse_b, f"r{r} lse")
        for k in ref.rt:
            _same(ref.rt[k], new.rt[k], f"r{r} route {k}")
        for k in ref.st:
            _same(ref.st[k], new.st[k], f"r{r} state {k}")


def test_noalloc_round_matches_the_workspace_round():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _compare(BIG, 2)
    _compare(SMALL, 2)
