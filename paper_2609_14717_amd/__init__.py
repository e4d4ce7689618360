"""Python binding of libcarryover (the Carryover drafter step on MI355X).

Argument marshalling only: every step runs in the library's HIP kernels.
PyTorch supplies device memory and streams.  The entry points have the names
and meaning of the C ABI in ``include/carryover.h``; each takes torch tensors
(or raw device pointers) and an optional stream, and raises ``CarryoverError``
on a non-zero status.  There is no CPU fallback: importing works anywhere, but
every call needs the built library and a GPU.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcarryover.so")

CO_OK, CO_ERR_INVALID_ARG, CO_ERR_UNSUPPORTED, CO_ERR_WORKSPACE = 0, 1, 2, 3
CO_ERR_CAPACITY, CO_ERR_PAGE_RANGE, CO_ERR_HIP, CO_ERR_LENGTH, CO_ERR_GROUP = 4, 5, 6, 7, 8
CO_ERR_TOKEN = 9
CO_DTYPE_F32, CO_DTYPE_BF16 = 0, 1
CO_BASELINE_MODE, CO_ROUTE_ACCEPT_ALL, CO_ROUTE_CARRY_ONLY, CO_Q_PREROTATED = 1, 2, 4, 8
CO_ATTN_SHARED_PREFIX = 16
CO_ROUTE_ACCEPT_BITS = 32
CO_WS_PROJECT, CO_WS_ATTENTION, CO_WS_ROUND, CO_WS_ATTENTION_BACKWARD = 0, 1, 2, 3
CO_WS_PROJECT_BACKWARD = 4
# launch-shape overrides (carryover_set_tuning)
TUNING = {"gemm_wide_variant": 0, "gemm_no_wide": 1, "project_fused_min_rows": 2, "attn_wave": 3,
          "attn_workgroups": 4, "attn_round_tiles": 5, "attn_group_split_tiles": 6}
SKIP = -(2 ** 31)
PAGE = 16


class CarryoverError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} ({code})")


class co_dims(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("block", ctypes.c_int32),
                ("feat_dim", ctypes.c_int32), ("model_dim", ctypes.c_int32),
                ("num_layers", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("rope_theta", ctypes.c_float)]


class co_weights(ctypes.Structure):
    _fields_ = [("w_f", ctypes.c_void_p), ("w_kv", ctypes.c_void_p), ("e_carry", ctypes.c_void_p),
                ("f_e", ctypes.c_void_p), ("w_f_carry", ctypes.c_void_p),
                ("z_norm", ctypes.c_void_p),
                ("k_norm", ctypes.c_void_p)]


class co_state(ctypes.Structure):
    _fields_ = [("ctx_len", ctypes.c_void_p), ("carry_len", ctypes.c_void_p),
                ("page_table", ctypes.c_void_p), ("k_cache", ctypes.c_void_p),
                ("v_cache", ctypes.c_void_p), ("k_carry", ctypes.c_void_p),
                ("v_carry", ctypes.c_void_p), ("status", ctypes.c_void_p)]


class co_route(ctypes.Structure):
    _fields_ = [("accept_len", ctypes.c_void_p), ("row_pos", ctypes.c_void_p),
                ("row_dst", ctypes.c_void_p)]


_lib = None
_P = ctypes.POINTER
_v = ctypes.c_void_p


def lib():
    """The loaded shared library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_14717_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "carryover_route": [_P(co_dims), _v, _v, ctypes.c_uint32, _P(co_state), _P(co_route), _v],
            "carryover_project_kv": [_P(co_dims), _P(co_weights), _v, _P(co_route), _P(co_state),
                                     _v, ctypes.c_size_t, _v],
            "drafter_block_attention": [_P(co_dims), ctypes.c_int32, ctypes.c_int32, _v,
                                        _P(co_state), _v, _v, ctypes.c_uint32, _v, ctypes.c_size_t,
                                        _v],
            "drafter_block_attention_ext": [_P(co_dims), ctypes.c_int32, ctypes.c_int32, _v, _v,
                                            _v, _P(co_state), _v, _v, _v, ctypes.c_uint32, _v,
                                            ctypes.c_size_t, _v],
            "carryover_round": [_P(co_dims), _P(co_weights), _v, _v, _v, _v, _P(co_state),
                                _P(co_route), _v, _v, ctypes.c_uint32, _v, ctypes.c_size_t, _v],
            "carryover_fold_e": [_P(co_dims), _P(co_weights), _v, _v],
            "drafter_block_attention_backward": [_P(co_dims), ctypes.c_int32, ctypes.c_int32,
                                                 _v, _P(co_state), _v, _v, _v, ctypes.c_int32,
                                                 _v, _v, _v, _v, _v, ctypes.c_uint32, _v,
                                                 ctypes.c_size_t, _v],
            "carryover_project_kv_backward": [_P(co_dims), _P(co_weights), _v, _P(co_route),
                                              _v, _v, _v, _v, _v, _v, _v, _v, ctypes.c_size_t,
                                              _v],
            "drafter_carry_mass": [_P(co_dims), ctypes.c_int32, ctypes.c_int32, _v, _P(co_state),
                                   _v, _v, ctypes.c_uint32, _v],
            "drafter_self_merge": [_P(co_dims), ctypes.c_int32, ctypes.c_int32, _v, _v, _v,
                                   _P(co_state), _v, _v, ctypes.c_uint32, _v],
            "carryover_import_kv": [_P(co_dims), ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _v,
                                    _v, _P(co_state), _v],
            "carryover_verify_sample": [_P(co_dims), ctypes.c_int32, _v, _v, _v, _v, _v, _v, _v,
                                        _v, _v],
            "carryover_set_tuning": [ctypes.c_int32, ctypes.c_int64],
            "carryover_round_noalloc": [_P(co_dims), _P(co_weights), _v, _v, _v, _v,
                                        _P(co_state), _P(co_route), _v, _v, ctypes.c_uint32, _v],
            "carryover_workspace_bytes": [_P(co_dims), ctypes.c_int32],
            "carryover_read_status": [_P(co_state), _P(ctypes.c_int32), _v],
            "carryover_status_string": [ctypes.c_int32],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = ctypes.c_int32
        L.carryover_workspace_bytes.restype = ctypes.c_size_t
        L.carryover_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


EXPORTED = ("carryover_route", "carryover_project_kv", "drafter_block_attention",
            "drafter_block_attention_ext",
            "carryover_round", "carryover_fold_e", "drafter_carry_mass", "drafter_self_merge",
            "drafter_block_attention_backward", "carryover_project_kv_backward",
            "carryover_import_kv", "carryover_verify_sample", "carryover_set_tuning",
            "carryover_round_noalloc",
            "carryover_workspace_bytes", "carryover_read_status", "carryover_status_string")


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(rc, where):
    if rc != CO_OK:
        raise CarryoverError(rc, where)


def status_string(code: int) -> str:
    return lib().carryover_status_string(code).decode()


def make_dims(S, B, Dcat, d, L, Hq, Hkv, hd, max_pages_per_seq, num_pages, dtype, theta):
    return co_dims(S, B, Dcat, d, L, Hq, Hkv, hd, PAGE, max_pages_per_seq, num_pages,
                   CO_DTYPE_BF16 if dtype in ("bf16", CO_DTYPE_BF16) else CO_DTYPE_F32,
                   float(theta))


def weights(w_f, w_kv, e_carry, f_e=None, w_f_carry=None, z_norm=None, k_norm=None):
    """co_weights over device tensors; f_e (fp32 [model_dim], optional) from
    ``carryover_fold_e``; w_f_carry (optional) the separate carry projector;
    z_norm (fp32 [model_dim], optional) the RMS-norm gain of F's output;
    k_norm (fp32 [num_layers][head_dim], optional) the per-head key gain."""
    return co_weights(_ptr(w_f), _ptr(w_kv), _ptr(e_carry), _ptr(f_e), _ptr(w_f_carry),
                      _ptr(z_norm), _ptr(k_norm))


def state(t):
    """co_state over a dict of tensors (see ``alloc_state``)."""
    return co_state(_ptr(t["ctx_len"]), _ptr(t["carry_len"]), _ptr(t["page_table"]),
                    _ptr(t["k_cache"]), _ptr(t["v_cache"]), _ptr(t["k_carry"]),
                    _ptr(t["v_carry"]), _ptr(t["status"]))


def route(t):
    return co_route(_ptr(t["accept_len"]), _ptr(t["row_pos"]), _ptr(t["row_dst"]))


def workspace_bytes(dims, which=CO_WS_ROUND) -> int:
    return lib().carryover_workspace_bytes(ctypes.byref(dims), which)


def alloc_state(dims, page_table, device="cuda"):
    """Zero-initialised device buffers for one drafter state (layouts of carryover.h)."""
    import torch
    dt = torch.bfloat16 if dims.dtype == CO_DTYPE_BF16 else torch.float32
    L, Hkv, hd, S = dims.num_layers, dims.num_kv_heads, dims.head_dim, dims.num_seqs
    CP = -(-dims.block // PAGE)
    pt = torch.as_tensor(page_table, dtype=torch.int32).to(device).contiguous()
    assert tuple(pt.shape) == (S, dims.max_pages_per_seq)
    return dict(
        ctx_len=torch.zeros(S, dtype=torch.int32, device=device),
        carry_len=torch.zeros(S, dtype=torch.int32, device=device),
        page_table=pt,
        k_cache=torch.zeros((L, dims.num_pages, Hkv, PAGE, hd), dtype=dt, device=device),
        v_cache=torch.zeros((L, dims.num_pages, Hkv, hd, PAGE), dtype=dt, device=device),
        k_carry=torch.zeros((L, S, CP, Hkv, PAGE, hd), dtype=dt, device=device),
        v_carry=torch.zeros((L, S, CP, Hkv, hd, PAGE), dtype=dt, device=device),
        status=torch.zeros(1, dtype=torch.int32, device=device),
    )


def alloc_route(S, B, device="cuda"):
    import torch
    return dict(accept_len=torch.zeros(S, dtype=torch.int32, device=device),
                row_pos=torch.zeros((S, B), dtype=torch.int32, device=device),
                row_dst=torch.zeros((S, B), dtype=torch.int32, device=device))


# ---------------------------------------------------------------- entry points

def carryover_route(dims, draft_tok, target_tok, flags, st, rt, stream=None):
    s, r = state(st), route(rt)
    _check(lib().carryover_route(ctypes.byref(dims), _ptr(draft_tok), _ptr(target_tok), flags,
                                 ctypes.byref(s), ctypes.byref(r), _stream(stream)),
           "carryover_route")


def carryover_project_kv(dims, w, hidden, rt, st, ws, stream=None, ws_bytes=None):
    s, r = state(st), route(rt)
    nb = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().carryover_project_kv(ctypes.byref(dims), ctypes.byref(w), _ptr(hidden),
                                      ctypes.byref(r), ctypes.byref(s), _ptr(ws), nb,
                                      _stream(stream)), "carryover_project_kv")


def drafter_block_attention(dims, layer_begin, layer_count, q, st, out, lse, flags, ws,
                            stream=None, ws_bytes=None):
    s = state(st)
    nb = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().drafter_block_attention(ctypes.byref(dims), layer_begin, layer_count, _ptr(q),
                                         ctypes.byref(s), _ptr(out), _ptr(lse), flags, _ptr(ws),
                                         nb, _stream(stream)), "drafter_block_attention")


def drafter_block_attention_ext(dims, layer_begin, layer_count, q, k_self, v_self, st, out, lse,
                                mass, flags, ws, stream=None, ws_bytes=None):
    s = state(st)
    nb = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().drafter_block_attention_ext(ctypes.byref(dims), layer_begin, layer_count, _ptr(q),
                                             _ptr(k_self), _ptr(v_self), ctypes.byref(s),
                                             _ptr(out), _ptr(lse), _ptr(mass), flags, _ptr(ws), nb,
                                             _stream(stream)), "drafter_block_attention_ext")


def drafter_block_attention_backward(dims, layer_begin, layer_count, q, st, out, lse, d_out,
                                     seqs_per_group, d_q, d_k_cache, d_v_cache, d_k_carry,
                                     d_v_carry, ws, flags=0, stream=None, ws_bytes=None):
    s = state(st)
    nb = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().drafter_block_attention_backward(
        ctypes.byref(dims), layer_begin, layer_count, _ptr(q), ctypes.byref(s), _ptr(out),
        _ptr(lse), _ptr(d_out), seqs_per_group, _ptr(d_q), _ptr(d_k_cache), _ptr(d_v_cache),
        _ptr(d_k_carry), _ptr(d_v_carry), flags, _ptr(ws), nb, _stream(stream)),
        "drafter_block_attention_backward")


def carryover_project_kv_backward(dims, w, hidden, rt, d_k_cache, d_v_cache, d_k_carry,
                                  d_v_carry, d_w_f, d_w_kv, d_e_carry, ws, stream=None,
                                  ws_bytes=None):
    r = route(rt)
    nb = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().carryover_project_kv_backward(
        ctypes.byref(dims), ctypes.byref(w), _ptr(hidden), ctypes.byref(r), _ptr(d_k_cache),
        _ptr(d_v_cache), _ptr(d_k_carry), _ptr(d_v_carry), _ptr(d_w_f), _ptr(d_w_kv),
        _ptr(d_e_carry), _ptr(ws), nb, _stream(stream)), "carryover_project_kv_backward")


def drafter_carry_mass(dims, layer_begin, layer_count, q, st, lse, mass, flags=0, stream=None):
    s = state(st)
    _check(lib().drafter_carry_mass(ctypes.byref(dims), layer_begin, layer_count, _ptr(q),
                                    ctypes.byref(s), _ptr(lse), _ptr(mass), flags,
                                    _stream(stream)), "drafter_carry_mass")


def drafter_self_merge(dims, layer_begin, layer_count, q, k_self, v_self, st, out, lse, flags=0,
                       stream=None):
    s = state(st)
    _check(lib().drafter_self_merge(ctypes.byref(dims), layer_begin, layer_count, _ptr(q),
                                    _ptr(k_self), _ptr(v_self), ctypes.byref(s), _ptr(out),
                                    _ptr(lse), flags, _stream(stream)), "drafter_self_merge")


def carryover_round(dims, w, hidden, draft_tok, target_tok, q, st, rt, out, lse, flags, ws,
                    stream=None, ws_bytes=None):
    s, r = state(st), route(rt)
    nb = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().carryover_round(ctypes.byref(dims), ctypes.byref(w), _ptr(hidden),
                                 _ptr(draft_tok), _ptr(target_tok), _ptr(q), ctypes.byref(s),
                                 ctypes.byref(r), _ptr(out), _ptr(lse), flags, _ptr(ws), nb,
                                 _stream(stream)), "carryover_round")


NOALLOC_SCRATCH_BYTES = 128 << 20


def carryover_round_noalloc(dims, w, hidden, draft_tok, target_tok, q, st, rt, out, lse, flags,
                            stream=None):
    """carryover_round on the library's static per-device scratch (no workspace
    argument, no allocation); calls on one device must not overlap."""
    s, r = state(st), route(rt)
    _check(lib().carryover_round_noalloc(ctypes.byref(dims), ctypes.byref(w), _ptr(hidden),
                                         _ptr(draft_tok), _ptr(target_tok), _ptr(q),
                                         ctypes.byref(s), ctypes.byref(r), _ptr(out), _ptr(lse),
                                         flags, _stream(stream)), "carryover_round_noalloc")


def carryover_fold_e(dims, w, f_e, stream=None):
    """f_e[:] = F e_carry (fp32 [model_dim]), once per set of weights."""
    _check(lib().carryover_fold_e(ctypes.byref(dims), ctypes.byref(w), _ptr(f_e), _stream(stream)),
           "carryover_fold_e")


def carryover_import_kv(dims, seq, pos0, k_rows, v_rows, st, stream=None):
    s = state(st)
    n = k_rows.shape[2]
    _check(lib().carryover_import_kv(ctypes.byref(dims), seq, pos0, n, _ptr(k_rows),
                                     _ptr(v_rows), ctypes.byref(s), _stream(stream)),
           "carryover_import_kv")


def carryover_verify_sample(dims, vocab, draft_tok, p_target, q_draft, words, accept_bits,
                            accept_len, next_tok, status, stream=None):
    """T = 1 verification: accept decisions, accepted length and the correction
    or bonus token of every sequence (see include/carryover.h)."""
    _check(lib().carryover_verify_sample(ctypes.byref(dims), vocab, _ptr(draft_tok),
                                         _ptr(p_target), _ptr(q_draft), _ptr(words),
                                         _ptr(accept_bits), _ptr(accept_len), _ptr(next_tok),
                                         _ptr(status), _stream(stream)),
           "carryover_verify_sample")


def set_tuning(name, value):
    """Override a launch shape (``TUNING`` names it); -1 or None restores the default."""
    _check(lib().carryover_set_tuning(TUNING[name], -1 if value is None else int(value)),
           "carryover_set_tuning")


def reset_tuning():
    for name in TUNING:
        set_tuning(name, -1)


def carryover_read_status(st, stream=None) -> int:
    s = state(st)
    out = ctypes.c_int32(0)
    _check(lib().carryover_read_status(ctypes.byref(s), ctypes.byref(out), _stream(stream)),
           "carryover_read_status")
    return out.value
