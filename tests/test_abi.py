"""Host-side checks of the C ABI: the library loads, exports every function
that include/carryover.h declares, and rejects bad arguments before it
enqueues anything (no compute call runs here)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2609_14717_amd as co

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "carryover.h")

pytestmark = pytest.mark.skipif(not os.path.exists(co.LIB_PATH), reason="library not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:co_status|size_t|const char\*)\s+(\w+)\s*\(", text,
                                 flags=re.M)))


def test_header_declares_the_four_calls_and_helpers():
    names = declared_functions()
    for n in ("carryover_route", "carryover_project_kv", "drafter_block_attention",
              "carryover_round"):
        assert n in names
    assert set(names) == set(co.EXPORTED)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", co.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for n in declared_functions():
        assert n in exported, n
        assert hasattr(co.lib(), n)


def _dims(**kw):
    base = dict(S=2, B=16, Dcat=768, d=256, L=1, Hq=4, Hkv=2, hd=64, max_pages_per_seq=8,
                num_pages=16, dtype="bf16", theta=1e4)
    base.update(kw)
    return co.make_dims(**base)


FAKE = 1 << 20      # an aligned, non-null address that is never dereferenced here


def _fake_state():
    return {k: FAKE for k in ("ctx_len", "carry_len", "page_table", "k_cache", "v_cache",
                              "k_carry", "v_carry", "status")}


def _fake_route():
    return {k: FAKE for k in ("accept_len", "row_pos", "row_dst")}


def _rc(fn):
    try:
        fn()
    except co.CarryoverError as e:
        return e.code
    return co.CO_OK


def test_status_strings():
    for code in range(10):
        assert co.status_string(code) != "unknown status"
    assert co.status_string(99) == "unknown status"


@pytest.mark.parametrize("kw,code", [
    (dict(hd=96), co.CO_ERR_UNSUPPORTED),
    (dict(Hq=6, Hkv=4), co.CO_ERR_UNSUPPORTED),
    (dict(Dcat=700), co.CO_ERR_UNSUPPORTED),
    (dict(B=0), co.CO_ERR_INVALID_ARG),
    (dict(theta=0.0), co.CO_ERR_INVALID_ARG),
])
def test_bad_dims_rejected_by_every_call(kw, code):
    d = _dims(**kw)
    st, rt = _fake_state(), _fake_route()
    W = co.weights(FAKE, FAKE, FAKE)
    assert _rc(lambda: co.carryover_route(d, FAKE, FAKE, 0, st, rt, stream=0)) == code
    assert _rc(lambda: co.carryover_project_kv(d, W, FAKE, rt, st, FAKE, stream=0,
                                               ws_bytes=1 << 30)) == code
    assert _rc(lambda: co.drafter_block_attention(d, 0, 1, FAKE, st, FAKE, None, 0, FAKE,
                                                  stream=0, ws_bytes=1 << 30)) == code
    assert _rc(lambda: co.drafter_carry_mass(d, 0, 1, FAKE, st, FAKE, FAKE, stream=0)) == code
    assert _rc(lambda: co.drafter_self_merge(d, 0, 1, FAKE, FAKE, FAKE, st, FAKE, FAKE,
                                             stream=0)) == code
    assert co.workspace_bytes(d) == 0


def test_page_size_must_be_16():
    d = _dims()
    d.page_size = 32
    assert _rc(lambda: co.carryover_route(d, FAKE, FAKE, 0, _fake_state(), _fake_route(),
                                          stream=0)) == co.CO_ERR_UNSUPPORTED


def test_attention_query_rows_limit():
    d = _dims(B=32, Hq=8, Hkv=2)          # 32 * 4 = 128 query rows per KV head
    assert _rc(lambda: co.drafter_block_attention(d, 0, 1, FAKE, _fake_state(), FAKE, None, 0,
                                                  FAKE, stream=0, ws_bytes=1 << 30)) \
        == co.CO_ERR_UNSUPPORTED


def test_null_and_misaligned_pointers():
    d = _dims()
    st = _fake_state()
    st["k_cache"] = 0
    W = co.weights(FAKE, FAKE, FAKE)
    assert _rc(lambda: co.carryover_project_kv(d, W, FAKE, _fake_route(), st, FAKE, stream=0,
                                               ws_bytes=1 << 30)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.carryover_route(d, None, FAKE, 0, _fake_state(), _fake_route(),
                                          stream=0)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.carryover_project_kv(d, W, FAKE + 2, _fake_route(), _fake_state(),
                                               FAKE, stream=0, ws_bytes=1 << 30)) \
        == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.drafter_block_attention(d, 0, 2, FAKE, _fake_state(), FAKE, None, 0,
                                                  FAKE, stream=0, ws_bytes=1 << 30)) \
        == co.CO_ERR_INVALID_ARG


def test_small_workspace_rejected():
    d = _dims()
    need_p = co.workspace_bytes(d, co.CO_WS_PROJECT)
    need_a = co.workspace_bytes(d, co.CO_WS_ATTENTION)
    assert need_p > 0 and need_a > 0
    assert co.workspace_bytes(d, co.CO_WS_ROUND) == need_p + need_a
    W = co.weights(FAKE, FAKE, FAKE)
    assert _rc(lambda: co.carryover_project_kv(d, W, FAKE, _fake_route(), _fake_state(), FAKE,
                                               stream=0, ws_bytes=need_p - 1)) \
        == co.CO_ERR_WORKSPACE
    assert _rc(lambda: co.drafter_block_attention(d, 0, 1, FAKE, _fake_state(), FAKE, None, 0,
                                                  FAKE, stream=0, ws_bytes=need_a - 1)) \
        == co.CO_ERR_WORKSPACE


def test_import_range_checked_on_host():
    d = _dims()
    lib = co.lib()
    s = co.state(_fake_state())
    for seq, pos0, n in ((2, 0, 1), (-1, 0, 1), (0, 120, 9), (0, -1, 1)):
        rc = lib.carryover_import_kv(ctypes.byref(d), seq, pos0, n, FAKE, FAKE, ctypes.byref(s),
                                     None)
        assert rc == co.CO_ERR_INVALID_ARG


def test_library_has_no_undefined_kernel_stubs():
    """Every kernel launched by the host code has its host-side stub (a kernel
    template whose host pass fails is otherwise dropped without a diagnostic)."""
    out = subprocess.run(["nm", "-D", "--undefined-only", co.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    assert "device_stub" not in out, out


def test_accept_bits_route_needs_no_target_tokens():
    """Under CO_ROUTE_ACCEPT_BITS the target tokens are unused (NULL accepted);
    the accept decisions themselves are still required."""
    d = _dims(S=0)
    assert _rc(lambda: co.carryover_route(d, FAKE, None, co.CO_ROUTE_ACCEPT_BITS, _fake_state(),
                                          _fake_route(), stream=0)) == co.CO_OK
    assert _rc(lambda: co.carryover_route(d, None, None, co.CO_ROUTE_ACCEPT_BITS, _fake_state(),
                                          _fake_route(), stream=0)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.carryover_route(d, FAKE, None, 0, _fake_state(), _fake_route(),
                                          stream=0)) == co.CO_ERR_INVALID_ARG


def test_carry_mass_arguments_checked_on_host():
    d = _dims()
    st = _fake_state()
    assert _rc(lambda: co.drafter_carry_mass(d, 0, 1, FAKE, st, None, FAKE, stream=0)) \
        == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.drafter_carry_mass(d, 0, 1, FAKE, st, FAKE, FAKE + 2, stream=0)) \
        == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.drafter_carry_mass(d, 1, 5, FAKE, st, FAKE, FAKE, stream=0)) \
        == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.drafter_carry_mass(_dims(B=80, Hq=2, Hkv=2), 0, 1, FAKE, st, FAKE,
                                             FAKE, stream=0)) == co.CO_ERR_UNSUPPORTED


def test_separate_projector_pointer_alignment_checked():
    d = _dims()
    W = co.weights(FAKE, FAKE, FAKE, None, FAKE + 2)
    assert _rc(lambda: co.carryover_project_kv(d, W, FAKE, _fake_route(), _fake_state(), FAKE,
                                               stream=0, ws_bytes=1 << 30)) \
        == co.CO_ERR_INVALID_ARG


def test_self_merge_arguments_checked_on_host():
    d = _dims()
    st = _fake_state()
    assert _rc(lambda: co.drafter_self_merge(d, 0, 1, FAKE, FAKE, FAKE, st, FAKE, None,
                                             stream=0)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.drafter_self_merge(d, 0, 1, FAKE, FAKE + 8, FAKE, st, FAKE, FAKE,
                                             stream=0)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: co.drafter_self_merge(d, 0, 2, FAKE, FAKE, FAKE, st, FAKE, FAKE,
                                             stream=0)) == co.CO_ERR_INVALID_ARG


def test_z_norm_pointer_alignment_checked():
    W = co.weights(FAKE, FAKE, FAKE, None, None, FAKE + 2)
    assert _rc(lambda: co.carryover_project_kv(_dims(), W, FAKE, _fake_route(), _fake_state(),
                                               FAKE, stream=0, ws_bytes=1 << 30)) \
        == co.CO_ERR_INVALID_ARG


def test_k_norm_pointer_alignment_checked():
    W = co.weights(FAKE, FAKE, FAKE, None, None, None, FAKE + 2)
    assert _rc(lambda: co.carryover_project_kv(_dims(), W, FAKE, _fake_route(), _fake_state(),
                                               FAKE, stream=0, ws_bytes=1 << 30)) \
        == co.CO_ERR_INVALID_ARG


def test_attention_backward_arguments_checked_on_host():
    st = _fake_state()

    def call(dims, group=1, dq=FAKE, wsb=1 << 30):
        return co.drafter_block_attention_backward(dims, 0, 1, FAKE, st, FAKE, FAKE, FAKE, group,
                                                   dq, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0,
                                                   ws_bytes=wsb)

    d = _dims()
    assert co.workspace_bytes(d, co.CO_WS_ATTENTION_BACKWARD) > 0
    assert _rc(lambda: call(d, group=0)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(d, dq=None)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(d, dq=FAKE + 4)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(d, wsb=16)) == co.CO_ERR_WORKSPACE
    assert _rc(lambda: call(_dims(dtype="f32"))) == co.CO_ERR_UNSUPPORTED
    assert _rc(lambda: call(_dims(hd=128))) == co.CO_ERR_UNSUPPORTED
    assert _rc(lambda: call(_dims(Hq=8))) == co.CO_ERR_UNSUPPORTED   # 64 query rows per KV head


def test_projection_backward_arguments_checked_on_host():
    def call(dims, W, dwf=FAKE, wsb=1 << 30):
        return co.carryover_project_kv_backward(dims, W, FAKE, _fake_route(), FAKE, FAKE, FAKE,
                                                FAKE, dwf, FAKE, FAKE, FAKE, stream=0,
                                                ws_bytes=wsb)

    d = _dims()
    W = co.weights(FAKE, FAKE, FAKE)
    assert co.workspace_bytes(d, co.CO_WS_PROJECT_BACKWARD) > 0
    assert _rc(lambda: call(d, W, dwf=None)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(d, W, wsb=16)) == co.CO_ERR_WORKSPACE
    assert _rc(lambda: call(_dims(dtype="f32"), W)) == co.CO_ERR_UNSUPPORTED
    for variant in (co.weights(FAKE, FAKE, FAKE, None, FAKE),
                    co.weights(FAKE, FAKE, FAKE, None, None, FAKE),
                    co.weights(FAKE, FAKE, FAKE, None, None, None, FAKE)):
        assert _rc(lambda: call(d, variant)) == co.CO_ERR_UNSUPPORTED


def _round(d, W, q=FAKE, lse=None, wsb=1 << 30, flags=0):
    return co.carryover_round(d, W, FAKE, FAKE, FAKE, q, _fake_state(), _fake_route(), FAKE, lse,
                              flags, FAKE, stream=0, ws_bytes=wsb)


@pytest.mark.parametrize("which", ["f_e", "w_f_carry", "z_norm", "k_norm", "lse", "q"])
def test_round_checks_every_step_before_its_first_launch(which):
    """A bad argument of any of the round's three steps is reported before the
    route is enqueued (no launch can run here: one would fail with
    CO_ERR_HIP, not CO_ERR_INVALID_ARG)."""
    d = _dims()
    bad = FAKE + 2
    W = co.weights(FAKE, FAKE, FAKE, bad if which == "f_e" else None,
                   bad if which == "w_f_carry" else None, bad if which == "z_norm" else None,
                   bad if which == "k_norm" else None)
    rc = _rc(lambda: _round(d, W, q=bad if which == "q" else FAKE,
                            lse=bad if which == "lse" else None))
    assert rc == co.CO_ERR_INVALID_ARG


def test_round_workspace_checked_before_its_first_launch():
    d = _dims()
    W = co.weights(FAKE, FAKE, FAKE)
    need = co.workspace_bytes(d, co.CO_WS_ROUND)
    assert _rc(lambda: _round(d, W, wsb=need - 1)) == co.CO_ERR_WORKSPACE
    assert _rc(lambda: _round(d, W, wsb=co.workspace_bytes(d, co.CO_WS_PROJECT) - 1)) \
        == co.CO_ERR_WORKSPACE


def test_verify_sample_arguments_checked_on_host():
    d = _dims()

    def call(vocab=1000, p=FAKE, words=FAKE, bits=FAKE, dims=d):
        return co.carryover_verify_sample(dims, vocab, FAKE, p, FAKE, words, bits, FAKE, FAKE,
                                          FAKE, stream=0)

    assert _rc(lambda: call(vocab=0)) == co.CO_ERR_UNSUPPORTED
    assert _rc(lambda: call(p=None)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(words=FAKE + 2)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(bits=None)) == co.CO_ERR_INVALID_ARG
    assert _rc(lambda: call(dims=_dims(B=0))) == co.CO_ERR_INVALID_ARG


def test_tuning_knobs():
    """Unknown knobs are refused; the attention workspace follows the
    workgroup override and returns to its size when it is cleared."""
    assert co.lib().carryover_set_tuning(len(co.TUNING), 1) == co.CO_ERR_INVALID_ARG
    assert co.lib().carryover_set_tuning(-1, 1) == co.CO_ERR_INVALID_ARG
    d = _dims()
    base = co.workspace_bytes(d, co.CO_WS_ATTENTION)
    try:
        co.set_tuning("attn_workgroups", 1000)
        assert co.workspace_bytes(d, co.CO_WS_ATTENTION) > base
    finally:
        co.reset_tuning()
    assert co.workspace_bytes(d, co.CO_WS_ATTENTION) == base


def test_noalloc_round_rejects_workloads_beyond_its_scratch():
    """carryover_round_noalloc refuses, on the host, dims whose round workspace
    exceeds its static scratch (here no device exists: any later step would
    fail with CO_ERR_HIP instead)."""
    from synth import workloads as wl
    w = wl.RAGGED32_8B.replace(S=96)
    d = co.make_dims(w.S, w.B, w.Dcat, w.d, w.L, w.Hq, w.Hkv, w.hd, w.max_pages_per_seq,
                     w.S * w.max_pages_per_seq, w.dtype, w.theta)
    assert co.workspace_bytes(d, co.CO_WS_ROUND) > co.NOALLOC_SCRATCH_BYTES
    assert _rc(lambda: co.carryover_round_noalloc(d, co.weights(FAKE, FAKE, FAKE), FAKE, FAKE,
                                                  FAKE, FAKE, _fake_state(), _fake_route(), FAKE,
                                                  None, 0, stream=0)) == co.CO_ERR_WORKSPACE
    small = _dims()
    assert co.workspace_bytes(small, co.CO_WS_ROUND) <= co.NOALLOC_SCRATCH_BYTES
    assert _rc(lambda: co.carryover_round_noalloc(small, co.weights(FAKE, FAKE, FAKE), FAKE, FAKE,
                                                  FAKE, FAKE, _fake_state(), _fake_route(), FAKE,
                                                  None, 0, stream=0)) == co.CO_ERR_HIP
