"""Workload definitions and seeded host-side draws for the drafter step.

Every workload is synthetic.  The paper's evaluation suite, training prompts,
target models and trained drafters are not available, so seeded random
tensors with the paper's shapes stand in for them: block 16, five tapped
target layers, five drafter layers, concurrency up to 32, training length 4096
(Section 3 "Experimental setup"; Appendix B, Table 4).

Big tensors (weights, hidden states, queries, pre-existing committed K/V) are
described here by a named stream, a logical index layout and a standard
deviation; both the host generator (``synth.normal``) and the device generator
(``synth.device``) materialise them from that description.  Small integer
draws (accepted lengths, tokens, context lengths, page order, anchors) are
made on the host only and copied to the device.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import numpy as np

from . import stream_key, uniform_int, bernoulli, draw_u64

PAGE = 16
TCAP = 1 << 20          # logical position stride of per-sequence index layouts

# named sub-streams of a workload seed
ST_WF, ST_WKV, ST_E, ST_H, ST_TGT, ST_DRAFT, ST_M, ST_Q = 1, 2, 3, 4, 5, 6, 7, 8
ST_CTX0, ST_PAGES, ST_KDIR, ST_VDIR, ST_HCTX, ST_ANCHOR, ST_U = 9, 10, 11, 12, 13, 14, 15
ST_WFC = 16             # the separate carry projector (a variant next to the path)
ST_ZNORM, ST_KSELF, ST_VSELF = 17, 18, 19   # RMS-norm gain offsets; block self K/V
ST_KNORM = 20           # per-head key RMS-norm gain offsets
ST_DOUT = 21            # gradient of a loss with respect to the attention output
ST_VLOGIT, ST_VNOISE, ST_VDRAW, ST_VWORD = 22, 23, 24, 25   # T = 1 verification inputs


@dataclass(frozen=True)
class Workload:
    name: str
    S: int                 # sequences in the batch
    B: int                 # verified-window rows per sequence (= block queries)
    Dcat: int              # concatenated target feature width
    d: int                 # drafter width (output of the fusion projection F)
    L: int                 # drafter layers
    Hq: int
    Hkv: int
    hd: int
    dtype: str             # 'f32' or 'bf16'
    theta: float           # RoPE base
    ctx_lo: int            # initial committed length ~ U{ctx_lo..ctx_hi}
    ctx_hi: int
    ctx_mode: str          # 'projected': prefill from N(0,1) states; 'direct': K/V drawn directly
    accept: tuple          # ('uniform',) or ('geom', p)
    rounds: int            # rounds the state has capacity for
    seed: int
    vocab: int = 1000
    w_sigma: float = 0.02
    e_sigma: float = 0.02
    h_sigma: float = 1.0
    anchors: int = 0       # training-shaped forward: anchored blocks per sequence
    seq_len: int = 0       # training-shaped forward: recorded positions per sequence

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def n_kv(self) -> int:
        """Columns of the concatenated K/V weight: layers x (K, V) x heads x dim."""
        return 2 * self.L * self.Hkv * self.hd

    @property
    def sigma_z(self) -> float:
        """Std of an entry of F's output: w * sqrt(Dcat) * h."""
        return self.w_sigma * math.sqrt(self.Dcat) * self.h_sigma

    @property
    def sigma_kv(self) -> float:
        """Std of a projected key/value entry: w^2 * sqrt(Dcat * d) * h (RoPE keeps it)."""
        return self.w_sigma ** 2 * math.sqrt(self.Dcat * self.d) * self.h_sigma

    @property
    def sigma_q(self) -> float:
        """Query std chosen so that logits q.k / sqrt(hd) have unit std."""
        return 1.0 / self.sigma_kv

    @property
    def max_pages_per_seq(self) -> int:
        if self.seq_len:
            return -(-self.seq_len // PAGE)
        return -(-(self.ctx_hi + (self.rounds + 1) * self.B) // PAGE)

    @property
    def carry_pages(self) -> int:
        return -(-self.B // PAGE)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def key(self, stream: int) -> int:
        return stream_key(self.seed, stream)


def _seed(cfg: int) -> int:
    return 0xC0FFEE + 1000 * cfg


# The five workloads.  Widths "config-1" = Dcat 768 (3 x 256), d 256, 4/2 heads, hd 64.
TINY = Workload("tiny_fp32", S=1, B=8, Dcat=768, d=256, L=1, Hq=4, Hkv=2, hd=64, dtype="f32",
                theta=1e4, ctx_lo=128, ctx_hi=128, ctx_mode="projected", accept=("uniform",),
                rounds=8, seed=_seed(1))
BATCH1_8B = Workload("batch1_8b", S=1, B=16, Dcat=20480, d=4096, L=1, Hq=32, Hkv=8, hd=128,
                     dtype="bf16", theta=1e6, ctx_lo=2048, ctx_hi=2048, ctx_mode="projected",
                     accept=("uniform",), rounds=8, seed=_seed(2))
RAGGED32 = Workload("ragged_batch32", S=32, B=16, Dcat=768, d=256, L=1, Hq=4, Hkv=2, hd=64,
                    dtype="bf16", theta=1e4, ctx_lo=512, ctx_hi=8192, ctx_mode="direct",
                    accept=("geom", 0.25), rounds=1024, seed=_seed(3))
LONG_CHAIN = Workload("long_chain_5layer", S=16, B=16, Dcat=20480, d=4096, L=5, Hq=32, Hkv=8,
                      hd=128, dtype="bf16", theta=1e6, ctx_lo=16384, ctx_hi=32768,
                      ctx_mode="direct", accept=("geom", 0.3), rounds=64, seed=_seed(4))
# cfg3's batch, contexts and acceptance with cfg2's widths (and RoPE base):
# the large-width serving round, whose projection is a compute-bound GEMM.
RAGGED32_8B = Workload("ragged_batch32_8b", S=32, B=16, Dcat=20480, d=4096, L=1, Hq=32, Hkv=8,
                       hd=128, dtype="bf16", theta=1e6, ctx_lo=512, ctx_hi=8192,
                       ctx_mode="direct", accept=("geom", 0.25), rounds=256,
                       seed=_seed(3) + 500)
TRAIN_FWD = Workload("train_fwd", S=8, B=16, Dcat=768, d=256, L=1, Hq=4, Hkv=2, hd=64,
                     dtype="bf16", theta=1e4, ctx_lo=0, ctx_hi=0, ctx_mode="projected",
                     accept=("uniform",), rounds=0, seed=_seed(5), anchors=256, seq_len=4096)

WORKLOADS = {w.name: w for w in (TINY, BATCH1_8B, RAGGED32, RAGGED32_8B, LONG_CHAIN, TRAIN_FWD)}


# ----------------------------------------------------------------- host draws

def initial_ctx(w: Workload) -> np.ndarray:
    """Initial committed length of every sequence."""
    if w.ctx_lo == w.ctx_hi:
        return np.full(w.S, w.ctx_lo, dtype=np.int32)
    return uniform_int(w.key(ST_CTX0), np.arange(w.S), w.ctx_lo, w.ctx_hi).astype(np.int32)


def page_table(w: Workload, n_seqs: int | None = None) -> np.ndarray:
    """[S][max_pages_per_seq] table over a pool of S*max_pages pages in a seeded random order."""
    S = w.S if n_seqs is None else n_seqs
    P = w.max_pages_per_seq
    n = S * P
    perm = np.argsort(draw_u64(w.key(ST_PAGES), np.arange(n)), kind="stable")
    return perm.astype(np.int32).reshape(S, P)


def accepted_lengths(w: Workload, rnd: int, S: int | None = None) -> np.ndarray:
    """Accepted prefix length m in [0, B] of every sequence in round ``rnd``."""
    S = w.S if S is None else S
    B = w.B
    if w.accept[0] == "uniform":
        return uniform_int(w.key(ST_M), rnd * S + np.arange(S), 0, B).astype(np.int32)
    p = w.accept[1]
    idx = (rnd * S + np.arange(S))[:, None] * B + np.arange(B)[None, :]
    reject = bernoulli(w.key(ST_M), idx, p)             # each slot rejected w.p. p
    m = np.where(reject.any(axis=1), reject.argmax(axis=1), B)
    return m.astype(np.int32)


def tokens_for(w: Workload, rnd: int, m: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """(draft, target) int32 [S][B] whose longest common prefix is exactly m."""
    S, B, V = len(m), w.B, w.vocab
    idx = (rnd * S + np.arange(S))[:, None] * B + np.arange(B)[None, :]
    target = uniform_int(w.key(ST_TGT), idx, 0, V - 1)
    other = uniform_int(w.key(ST_DRAFT), idx, 0, V - 1)
    bump = uniform_int(w.key(ST_DRAFT), idx + (1 << 40), 1, V - 1)
    j = np.arange(B)[None, :]
    mm = m[:, None]
    draft = np.where(j < mm, target, np.where(j == mm, (target + bump) % V, other))
    return draft.astype(np.int32), target.astype(np.int32)


def anchors(w: Workload) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Training-shaped forward (Algorithm 2): initial anchors a [S][A], sorted
    and distinct in [0, seq_len - B - 1]; rejected counts u [S][A] ~ U{0..B};
    accepted m = B - u; shifted anchors a' = a + m + 1 (Algorithm 2 step 3).
    The verified window of anchor a starts at position a + 1, so its rejected
    rows sit at a' + r, r < u."""
    hi = w.seq_len - w.B                      # a in [0, hi - 1]
    a = np.empty((w.S, w.anchors), dtype=np.int32)
    for s in range(w.S):
        keys = draw_u64(w.key(ST_ANCHOR), s * TCAP + np.arange(hi))
        a[s] = np.sort(np.argsort(keys, kind="stable")[: w.anchors])
    u = uniform_int(w.key(ST_U), np.arange(w.S * w.anchors), 0, w.B).astype(np.int32)
    u = u.reshape(w.S, w.anchors)
    return a, u, a + (w.B - u) + 1


# ------------------------------------------------- logical layouts of big tensors
# Each returns (stream, shape, strides, base, sigma) describing a dense block.

def spec_wf(w):
    return ST_WF, (w.d, w.Dcat), (w.Dcat, 1), 0, w.w_sigma


def spec_wfc(w):
    """Separate projector for carried rows, shaped like F."""
    return ST_WFC, (w.d, w.Dcat), (w.Dcat, 1), 0, w.w_sigma


def spec_znorm(w):
    """Offsets of the RMS-norm gain of F's output, fp32: the gain is
    fp32(sigma_z) * (1 + offset), so that normalised rows keep the statistics
    of F's output (and K/V those of the projection)."""
    return ST_ZNORM, (w.d,), (1,), 0, 0.1


def znorm_gain_host(w, offsets):
    """The gain from its offsets, in fp32 as on the device."""
    return np.float32(w.sigma_z) * (np.float32(1.0) + np.asarray(offsets, np.float32))


def spec_knorm(w):
    """Offsets of the per-head key RMS-norm gain, fp32 [L][hd]: the gain is
    fp32(sigma_kv) * (1 + offset), so that normalised keys keep the statistics
    of projected keys."""
    return ST_KNORM, (w.L, w.hd), (w.hd, 1), 0, 0.1


def knorm_gain_host(w, offsets):
    """The key gain from its offsets, in fp32 as on the device."""
    return np.float32(w.sigma_kv) * (np.float32(1.0) + np.asarray(offsets, np.float32))


def spec_self(w, which, rnd, S=None):
    """Block self keys ('k', unrotated) or values ('v') of round ``rnd``:
    [L][S][B][Hkv][hd], with the statistics of projected K/V."""
    S = w.S if S is None else S
    st = ST_KSELF if which == "k" else ST_VSELF
    shape = (w.L, S, w.B, w.Hkv, w.hd)
    strides = (S * w.B * w.Hkv * w.hd, w.B * w.Hkv * w.hd, w.Hkv * w.hd, w.hd, 1)
    return st, shape, strides, rnd * w.L * S * w.B * w.Hkv * w.hd, w.sigma_kv


def spec_wkv(w):
    return ST_WKV, (w.n_kv, w.d), (w.d, 1), 0, w.w_sigma


def spec_e(w):
    return ST_E, (w.Dcat,), (1,), 0, w.e_sigma


def spec_h(w, rnd, S=None, B=None):
    """Verified-window states of round ``rnd``: [S][B][Dcat]."""
    S = w.S if S is None else S
    B = w.B if B is None else B
    base = rnd * S * B * w.Dcat
    return ST_H, (S, B, w.Dcat), (B * w.Dcat, w.Dcat, 1), base, w.h_sigma


def spec_hctx(w, s, t0, n):
    """States used to build committed context by prefill: [n][Dcat] of sequence s."""
    return ST_HCTX, (n, w.Dcat), (w.Dcat, 1), (s * TCAP + t0) * w.Dcat, w.h_sigma


def spec_q(w, rnd, S=None):
    """Un-rotated queries of round ``rnd``: [L][S][B][Hq][hd]."""
    S = w.S if S is None else S
    shape = (w.L, S, w.B, w.Hq, w.hd)
    strides = (S * w.B * w.Hq * w.hd, w.B * w.Hq * w.hd, w.Hq * w.hd, w.hd, 1)
    return ST_Q, shape, strides, rnd * w.L * S * w.B * w.Hq * w.hd, w.sigma_q


def spec_dout(w, S=None):
    """Output gradient dO of the attention (the backward's input): [L][S][B][Hq][hd],
    unit variance."""
    S = w.S if S is None else S
    shape = (w.L, S, w.B, w.Hq, w.hd)
    strides = (S * w.B * w.Hq * w.hd, w.B * w.Hq * w.hd, w.Hq * w.hd, w.hd, 1)
    return ST_DOUT, shape, strides, 0, 1.0


def spec_kv_direct(w, which, s, t0, n):
    """Directly drawn committed keys ('k') or values ('v') of sequence s at
    positions t0..t0+n-1: [L][Hkv][n][hd]."""
    st = ST_KDIR if which == "k" else ST_VDIR
    shape = (w.L, w.Hkv, n, w.hd)
    strides = (w.Hkv * TCAP * w.hd, TCAP * w.hd, w.hd, 1)
    return st, shape, strides, (s * w.L * w.Hkv * TCAP + t0) * w.hd, w.sigma_kv


def host_block(w: Workload, spec, dtype: str | None = None) -> np.ndarray:
    """Materialise a described block on the host (fp32 array or bf16 bits)."""
    from . import normal_block
    st, shape, strides, base, sigma = spec
    return normal_block(w.key(st), shape, strides, base, sigma, dtype or w.dtype)


# ------------------------------------------------ T = 1 verification inputs

def verify_inputs(w: Workload, rnd: int, vocab: int, S: int | None = None,
                  sigma_target: float = 2.0, sigma_gap: float = 1.0):
    """Inputs of stochastic verification for round ``rnd``: the target's
    distributions p [S][B+1][V] (softmax of logits ~ N(0, sigma_target^2)), the
    drafter's q [S][B][V] (softmax of the target logits plus N(0, sigma_gap^2)
    noise, so that the two disagree as a trained drafter and its target do),
    proposals x_j drawn from q_j [S][B], and the verifier's uniform words
    [S][B+1] (uint32).  p and q are fp32; their softmax is taken in fp64."""
    from . import normal_f32
    S = w.S if S is None else S
    B, V = w.B, vocab
    base = rnd * S * (B + 1) * V
    idx = base + np.arange(S * (B + 1) * V, dtype=np.int64)
    z = normal_f32(w.key(ST_VLOGIT), idx, sigma_target).astype(np.float64).reshape(S, B + 1, V)
    zq = z[:, :B] + normal_f32(w.key(ST_VNOISE), idx[: S * B * V], sigma_gap).astype(
        np.float64).reshape(S, B, V)

    def softmax(x):
        e = np.exp(x - x.max(axis=-1, keepdims=True))
        return e / e.sum(axis=-1, keepdims=True)

    p = softmax(z).astype(np.float32)
    q = softmax(zq).astype(np.float32)
    u = (draw_u64(w.key(ST_VDRAW), rnd * S * B + np.arange(S * B)) >> np.uint64(11)).astype(
        np.float64) * 2.0 ** -53
    cq = np.cumsum(q.astype(np.float64), axis=-1).reshape(S * B, V)
    draft = np.array([min(int(np.searchsorted(cq[i], u[i] * cq[i, -1], side="right")), V - 1)
                      for i in range(S * B)], np.int32).reshape(S, B)
    words = (draw_u64(w.key(ST_VWORD), rnd * S * (B + 1) + np.arange(S * (B + 1)))
             & np.uint64(0xFFFFFFFF)).astype(np.uint32).reshape(S, B + 1)
    return draft, p, q, words
