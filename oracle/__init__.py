"""fp64 CPU oracle of the Carryover drafter step.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path:
the two meet only in the seeded input generator (``synth``).

What it computes (paper: Section 2.1, Eqs. 1-2; Appendix A, Algorithm 1 and
the "Cache semantics" paragraph; Section 2 "Preliminaries"):

* greedy verification accepts the longest prefix m on which the draft agrees
  with the target's greedy tokens;
* the carryover update projects all B verified rows in one pass, with the
  carry embedding E added to the rejected rows m..B-1 *before* the fusion
  projection F; keys and values of layer l are K_l(F(x)) and V_l(F(x));
* keys are rotated once, at the row's absolute position, when projected;
* rows 0..m-1 are appended to the committed context C_l; rows m..B-1 replace
  the carryover segment U_l wholesale (U starts empty; full acceptance leaves
  it empty; it never holds more than B rows);
* the next draft's block queries (position ctx_len + i) attend to [C_l ; U_l]
  with a plain softmax; the baseline update (left column of Algorithm 1)
  projects only rows 0..m-1 and has no U.

Variants next to the path: stochastic verification (T = 1), where m is the run
of positions the verifier accepted by rejection sampling (Appendix A, "Why
verification remains valid"); the separate-projector update, where carried
rows go through a second fusion matrix instead of F + E (Section 4, Table
3(b)); the share of attention that falls on the carried rows (Appendix
"Attention to carried states"); the block's own rows as a third attention
segment [C ; U ; S]; and RMS normalisations of F's output before the K/V
projections and of every head's key before its rotation (the paper's
equations omit normalisation, Section 2.1); and the reverse mode of the
attention and of the projection, the training side of the second drafter pass
(Algorithm 2: gradients of W_F, W_KV, E_carry and of the queries, with the
target's states held constant).

Readings where the paper is silent (each one a stated choice of this oracle): no norm
and no bias in F, K_l, V_l; rotate-half RoPE with inverse frequency
theta^(-2i/hd); softmax scale 1/sqrt(hd); query head h reads KV head
h // (Hq/Hkv); window row j sits at position ctx_len_before + j; block queries
see every committed and carried key (no position mask).

All arithmetic is float64 on exact widenings of the stored inputs; nothing is
rounded in between.  Parity pins: see tests/test_oracle_*.py.  Every function
below is pinned by at least one of those tests.
"""
from __future__ import annotations

import math

import numpy as np

# status codes (mirrors of the library's data-dependent error codes)
OK, ERR_CAPACITY, ERR_PAGE_RANGE, ERR_LENGTH = 0, 4, 5, 7
SKIP = -(2 ** 31)
PAGE = 16


# ------------------------------------------------------------------ routing

def accept_len(draft: np.ndarray, target: np.ndarray) -> int:
    """Greedy verification: number of leading draft tokens equal to the
    target's greedy tokens (Section 2 "Preliminaries"; Section 2.2)."""
    m = 0
    while m < len(draft) and draft[m] == target[m]:
        m += 1
    return m


def accept_len_bits(bits: np.ndarray) -> int:
    """Stochastic verification (T = 1): the verifier decides acceptance of each
    proposal by rejection sampling (Appendix A, "Why verification remains
    valid"); the accepted prefix is the run of accepted positions before the
    first rejection.  bits[j] != 0 means position j was accepted."""
    m = 0
    while m < len(bits) and bits[m] != 0:
        m += 1
    return m


# Stochastic verification (T = 1) itself: the standard speculative-sampling
# rule that Appendix A ("Why verification remains valid") relies on.  A
# proposed token x drawn from the drafter's distribution q is accepted with
# probability min(1, p(x) / q(x)) under the target's distribution p; at the
# first rejection the verifier emits a correction drawn from the normalised
# residual max(0, p - q); when every proposal is accepted it emits a bonus
# token drawn from p at the position after the block.
#
# Both random draws are supplied as 32-bit words so that the oracle and the
# kernel make the same integer decisions:
#   * acceptance uses u = (word >> 8) * 2^-24, uniform on [0, 1) with 24 bits;
#     u * q(x) < p(x) is decided exactly (a 24-bit by 24-bit product is exact
#     in fp64): u < min(1, p / q) for u < 1, so a token the target gives no
#     probability is never accepted and p = q accepts every proposal;
#   * the correction or bonus is drawn by an inverse CDF over fixed-point
#     weights w(y) = floor(2^32 * d(y)), d(y) = p(y) - q(y) (an fp64
#     difference of the fp32 inputs) where positive, else 0 (d(y) = p(y) for a
#     bonus, and for a correction whose weights are all zero); with integer
#     sums, y is the smallest token whose running sum exceeds
#     t = floor(word * W / 2^32), W the total.  The weights approximate the
#     residual to 2^-32 per token.  No weight at all (not a distribution):
#     no token (-1).

ERR_TOKEN = 9            # a proposed token outside [0, vocab)


def accept_test(u_word, p_x, q_x):
    """Acceptance of one proposal: u * q(x) < p(x) with u = (u_word >> 8) * 2^-24.
    Vectorised (numpy broadcasting); p, q are fp32 values."""
    u = (np.asarray(u_word, np.uint64) >> np.uint64(8)).astype(np.float64) * 2.0 ** -24
    return u * np.asarray(q_x, np.float32).astype(np.float64) < \
        np.asarray(p_x, np.float32).astype(np.float64)


def fixed_weights(p_row, q_row=None):
    """Fixed-point sampling weights (uint64) of the residual max(0, p - q), or
    of p itself when q_row is None."""
    d = np.asarray(p_row, np.float32).astype(np.float64)
    if q_row is not None:
        d = d - np.asarray(q_row, np.float32).astype(np.float64)
    return np.floor(np.where(d > 0, d, 0.0) * 2.0 ** 32).astype(np.uint64)


def sample_fixed(w, u_word):
    """Inverse-CDF draw from fixed-point weights w (uint64): the smallest y
    with w[0] + ... + w[y] > floor(u_word * W / 2^32); -1 when W = 0."""
    cum = np.cumsum(np.asarray(w, np.uint64), dtype=np.uint64)
    W = int(cum[-1])
    if W == 0:
        return -1
    t = (int(u_word) * W) >> 32
    return int(np.searchsorted(cum, np.uint64(t), side="right"))


def verify_sample(draft, p, q, u_words):
    """T = 1 verification of one window.  draft [B] proposed tokens; p [B+1][V]
    target probabilities at the B proposal positions and the one after them;
    q [B][V] drafter probabilities; u_words [B+1] uint32 (acceptance word of
    each position, then the word of the correction or bonus draw).
    Returns (m, next_token, status): m = proposals accepted before the first
    rejection; next_token = the correction (m < B) or the bonus (m = B).  A
    proposed token outside [0, V) is an error: (0, -1, ERR_TOKEN)."""
    draft = np.asarray(draft)
    B, V = len(draft), np.asarray(p).shape[1]
    if np.any((draft < 0) | (draft >= V)):
        return 0, -1, ERR_TOKEN
    m = 0
    while m < B and bool(accept_test(u_words[m], p[m][draft[m]], q[m][draft[m]])):
        m += 1
    if m < B:
        w = fixed_weights(p[m], q[m])
        if not w.any():
            w = fixed_weights(p[m])
    else:
        w = fixed_weights(p[B])
    return m, sample_fixed(w, u_words[B]), OK


def route(draft, target, ctx_len, carry_len, page_table, num_pages, mode="carry",
          accept="tokens"):
    """Split every verified window by its accepted prefix (Eq. 1, Algorithm 1).

    mode: 'carry' (Carryover column), 'baseline' (Baseline column),
    'accept_all' (every row committed: building context by prefill),
    'carry_only' (rows 0..m-1 are already committed elsewhere and are skipped).
    accept: 'tokens' (greedy: draft vs target tokens) or 'bits' (``draft``
    holds the verifier's per-position accept decisions, ``target`` is unused).

    Returns a dict with accept_len [S], row_pos [S][B], row_dst [S][B]
    (>= 0: global committed slot page*16 + pos % 16; -1-r: carry row r;
    SKIP: not stored), new ctx_len [S], new carry_len [S] and a per-sequence
    status.  A sequence that fails a check keeps its lengths, stores no row
    and reports accept_len 0.
    """
    draft = np.asarray(draft)
    S, B = draft.shape
    out = dict(accept_len=np.zeros(S, np.int32), row_pos=np.zeros((S, B), np.int32),
               row_dst=np.full((S, B), SKIP, np.int32), ctx_len=np.array(ctx_len, np.int32).copy(),
               carry_len=np.array(carry_len, np.int32).copy(), status=np.zeros(S, np.int32),
               touched=np.ones(S, bool))
    cap = page_table.shape[1] * PAGE
    for s in range(S):
        p0 = int(ctx_len[s])
        if mode == "accept_all":
            m = B
        elif accept == "bits":
            m = accept_len_bits(draft[s])
        else:
            m = accept_len(draft[s], target[s])
        if p0 < 0:
            out["status"][s] = ERR_LENGTH
        elif p0 + B > cap:
            out["status"][s] = ERR_CAPACITY
        else:
            for j in range(m if mode in ("carry", "baseline", "accept_all") else 0):
                page = int(page_table[s][(p0 + j) // PAGE])
                if page < 0 or page >= num_pages:
                    out["status"][s] = ERR_PAGE_RANGE
                    break
        if out["status"][s] != OK:
            out["touched"][s] = False
            out["row_pos"][s] = p0 + np.arange(B) if p0 >= 0 else 0
            continue
        out["accept_len"][s] = m
        for j in range(B):
            pos = p0 + j
            out["row_pos"][s, j] = pos
            if j < m:
                if mode != "carry_only":
                    page = int(page_table[s][pos // PAGE])
                    out["row_dst"][s, j] = page * PAGE + pos % PAGE
            elif mode in ("carry", "carry_only"):
                out["row_dst"][s, j] = -1 - (j - m)
        out["ctx_len"][s] = p0 + m
        out["carry_len"][s] = (B - m) if mode in ("carry", "carry_only") else 0
    return out


# --------------------------------------------------------------- projection

def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of the last axis at absolute position(s) pos.

    Pairs (i, i + hd/2) are rotated by the angle pos * theta^(-2i/hd).
    ``pos`` broadcasts against x.shape[:-1].
    """
    x = np.asarray(x, dtype=np.float64)
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


RMS_EPS = 1e-6   # RMSNorm epsilon of the normalisation variant


def rms_norm(z, g):
    """Root-mean-square normalisation of each row of z, then an elementwise gain g."""
    z = np.asarray(z, np.float64)
    return z / np.sqrt(np.mean(z * z, axis=-1, keepdims=True) + RMS_EPS) * np.asarray(g, np.float64)


def project(H, E, add_e, WF, WKV, pos, L, Hkv, hd, theta, WF_carry=None, z_norm=None,
            k_norm=None):
    """Phi_l(H) of Eq. 1 for every layer, with E added to flagged rows before F
    (Eq. 2) and RoPE applied to the keys at each row's position.

    H [M][Dcat], E [Dcat], add_e [M] (bool), WF [d][Dcat], WKV [L*2*Hkv*hd][d]
    ordered (layer, K|V, head, dim), pos [M].
    WF_carry [d][Dcat]: the separate-projector variant (Section 4, "How should
    rejected states be distinguished?"; Table 3(b)): flagged rows are projected
    by this second fusion matrix instead of F, with no E.
    z_norm [d]: the normalisation variant: z = F(x) is RMS-normalised (gain
    z_norm) before the K/V projections (the equations omit normalisation,
    Section 2.1).
    k_norm [L][hd]: per-head key normalisation: every head's key is
    RMS-normalised (gain k_norm[l]) before it is rotated.
    Returns K, V as [M][L][Hkv][hd] float64.
    """
    H = np.asarray(H, np.float64)
    flag = np.asarray(add_e, bool)
    if WF_carry is None:
        x = H + flag[:, None].astype(np.float64) * np.asarray(E, np.float64)[None, :]
        z = x @ np.asarray(WF, np.float64).T                     # F
    else:
        z = np.where(flag[:, None], H @ np.asarray(WF_carry, np.float64).T,
                     H @ np.asarray(WF, np.float64).T)
    if z_norm is not None:
        z = rms_norm(z, z_norm)
    kv = (z @ np.asarray(WKV, np.float64).T).reshape(len(H), L, 2, Hkv, hd)
    k = kv[:, :, 0]
    if k_norm is not None:
        k = rms_norm(k, np.asarray(k_norm, np.float64)[None, :, None, :])
    k = rope(k, np.asarray(pos)[:, None, None], theta)
    return k, kv[:, :, 1].copy()


def project_backward(H, E, add_e, WF, WKV, pos, L, Hkv, hd, theta, dK, dV):
    """Reverse mode of ``project`` (the plain update: F with E on flagged rows,
    no separate projector, no normalisation) for the trained parameters W_F,
    W_KV and E_carry (Algorithm 2: the target's states H are constants).
    dK [M][L][Hkv][hd] is the gradient with respect to the rotated keys, dV
    with respect to the values.  The keys' gradient is rotated back at each
    row's position, the rows' K/V gradients form dJ [M][NKV] in W_KV's row
    order, and with x = H + flag E, z = F x: dW_KV = dJ^T z, dz = dJ W_KV,
    dW_F = dz^T x, dE = sum over flagged rows of F^T dz.
    Returns (dWF [d][Dcat], dWKV [NKV][d], dE [Dcat])."""
    H = np.asarray(H, np.float64)
    flag = np.asarray(add_e, bool)
    M = len(H)
    x = H + flag[:, None].astype(np.float64) * np.asarray(E, np.float64)[None, :]
    WF = np.asarray(WF, np.float64)
    WKV = np.asarray(WKV, np.float64)
    z = x @ WF.T
    dk = rope(np.asarray(dK, np.float64), -np.asarray(pos, np.float64)[:, None, None], theta)
    dJ = np.stack([dk, np.asarray(dV, np.float64)], axis=2).reshape(M, -1)
    dWKV = dJ.T @ z
    dz = dJ @ WKV
    dWF = dz.T @ x
    dE = (dz[flag] @ WF).sum(axis=0) if flag.any() else np.zeros(WF.shape[1])
    return dWF, dWKV, dE


# ---------------------------------------------------------------- attention

def attend(q, qpos, k, v, theta):
    """Softmax attention of unrotated queries q [nq][hd] at positions qpos over
    already-rotated keys k [nk][hd] and values v [nk][hd]; dense, two-pass.
    Returns (O [nq][hd], LSE [nq]); an empty key set gives O = 0, LSE = -inf."""
    q = rope(np.asarray(q, np.float64), np.asarray(qpos), theta)
    nq, hd = q.shape
    if len(k) == 0:
        return np.zeros((nq, hd)), np.full(nq, -np.inf)
    s = (q @ np.asarray(k, np.float64).T) / math.sqrt(hd)
    mx = s.max(axis=1, keepdims=True)
    w = np.exp(s - mx)
    den = w.sum(axis=1, keepdims=True)
    return (w @ np.asarray(v, np.float64)) / den, (mx + np.log(den))[:, 0]


def attend_backward(q, qpos, k, v, dO, theta):
    """Reverse mode of ``attend`` (the training side of the block attention,
    Algorithm 2: gradients of the second pass): given dO [nq][hd], the
    gradients of sum(dO * O) with respect to the unrotated queries q, the
    rotated keys k and the values v.  With P the softmax weights and
    D_i = sum_j P_ij (dO_i . v_j): dv = P^T dO; dS = P * (dO v^T - D); the
    rotated query's gradient dS k / sqrt(hd) is rotated back (the transpose of
    a rotation turns by the opposite angle); dk = dS^T (R q) / sqrt(hd).
    Returns (dq [nq][hd], dk [nk][hd], dv [nk][hd]); no keys: all zero."""
    q = np.asarray(q, np.float64)
    dO = np.asarray(dO, np.float64)
    nq, hd = q.shape
    k = np.asarray(k, np.float64).reshape(-1, hd)
    v = np.asarray(v, np.float64).reshape(-1, hd)
    if len(k) == 0:
        return np.zeros((nq, hd)), np.zeros((0, hd)), np.zeros((0, hd))
    qr = rope(q, np.asarray(qpos), theta)
    s = (qr @ k.T) / math.sqrt(hd)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    dv = p.T @ dO
    dp = dO @ v.T
    ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
    dqr = (ds @ k) / math.sqrt(hd)
    dk = (ds.T @ qr) / math.sqrt(hd)
    return rope(dqr, -np.asarray(qpos, np.float64), theta), dk, dv


def carry_mass(q, qpos, k_committed, k_carry, theta):
    """Share of each query's softmax attention that falls on the carried rows
    (the diagnostic of Appendix "Attention to carried states"): the weights of
    the attention over [C;U] summed over U.  q [nq][hd] unrotated at qpos; keys
    already rotated.  Zero when there are no keys at all."""
    q = rope(np.asarray(q, np.float64), np.asarray(qpos), theta)
    nq, hd = q.shape
    kc = np.asarray(k_committed, np.float64).reshape(-1, hd)
    ku = np.asarray(k_carry, np.float64).reshape(-1, hd)
    if len(kc) + len(ku) == 0:
        return np.zeros(nq)
    s = (q @ np.concatenate([kc, ku], axis=0).T) / math.sqrt(hd)
    w = np.exp(s - s.max(axis=1, keepdims=True))
    return w[:, len(kc):].sum(axis=1) / w.sum(axis=1)


# ------------------------------------------------------------ drafter state

class _RowStore:
    """Rows [L][n][Hkv][hd] of every sequence.  Appending writes into spare
    capacity instead of re-concatenating (a storage detail only: reading a
    sequence gives exactly the rows a concatenation would)."""

    def __init__(self, S, L, Hkv, hd, dtype):
        self._dtype = dtype
        self._buf = [np.zeros((L, 0, Hkv, hd), dtype) for _ in range(S)]
        self._n = [0] * S

    def __len__(self):
        return len(self._buf)

    def __getitem__(self, s):
        return self._buf[s][:, :self._n[s]]

    def __setitem__(self, s, rows):
        rows = np.asarray(rows)
        n = rows.shape[1]
        buf = np.empty(rows.shape[:1] + (n + n // 4 + 64,) + rows.shape[2:], self._dtype)
        buf[:, :n] = rows
        self._buf[s] = buf
        self._n[s] = n

    def __iter__(self):
        return (self[s] for s in range(len(self)))

    def append(self, s, rows):
        n, m = self._n[s], rows.shape[1]
        buf = self._buf[s]
        if n + m > buf.shape[1]:
            grown = np.empty(buf.shape[:1] + (n + m + (n + m) // 4 + 64,) + buf.shape[2:],
                             self._dtype)
            grown[:, :n] = buf[:, :n]
            self._buf[s] = buf = grown
        buf[:, n:n + m] = rows
        self._n[s] = n + m


class State:
    """Logical (unpaged) drafter KV of S sequences: committed C_l and carryover U_l."""

    def __init__(self, S, L, Hkv, hd, store=np.float64):
        self.S, self.L, self.Hkv, self.hd, self.store = S, L, Hkv, hd, store
        self.ck = _RowStore(S, L, Hkv, hd, store)
        self.cv = _RowStore(S, L, Hkv, hd, store)
        self.uk = _RowStore(S, L, Hkv, hd, store)
        self.uv = _RowStore(S, L, Hkv, hd, store)

    def ctx_len(self):
        return np.array([c.shape[1] for c in self.ck], np.int32)

    def carry_len(self):
        return np.array([u.shape[1] for u in self.uk], np.int32)

    def set_committed(self, s, k, v):
        """Install committed K/V [L][n][Hkv][hd] of sequence s (already rotated)."""
        self.ck[s] = np.asarray(k, self.store)
        self.cv[s] = np.asarray(v, self.store)

    def commit_and_replace(self, s, k_acc, v_acc, k_rej, v_rej):
        """C_l <- [C_l ; J_acc];  U_l <- J_rej (old U dropped).  Inputs [n][L][Hkv][hd]."""
        t = lambda a: np.asarray(a, self.store).transpose(1, 0, 2, 3)
        self.ck.append(s, t(k_acc))
        self.cv.append(s, t(v_acc))
        self.uk[s] = t(k_rej).copy()
        self.uv[s] = t(v_rej).copy()

    def context(self, s, layer, g):
        """ctx_l = [C_l ; U_l] for KV head g: (keys, values) [n][hd]."""
        k = np.concatenate([self.ck[s][layer, :, g], self.uk[s][layer, :, g]], axis=0)
        v = np.concatenate([self.cv[s][layer, :, g], self.uv[s][layer, :, g]], axis=0)
        return k.astype(np.float64), v.astype(np.float64)


def attend_state(state: State, Q, Hq, theta, seqs=None, layers=None):
    """Block attention of every (layer, sequence, query row, query head) over
    ctx = [C;U].  Q [L][S][B][Hq][hd] unrotated; query i sits at ctx_len + i.
    Returns O [L][S][B][Hq][hd], LSE [L][S][B][Hq] (NaN where not computed)."""
    L, S, B, _, hd = Q.shape
    G = Hq // state.Hkv
    O = np.full(Q.shape, np.nan)
    LSE = np.full(Q.shape[:-1], np.nan)
    ctx = state.ctx_len()
    for s in (range(S) if seqs is None else seqs):
        for layer in (range(L) if layers is None else layers):
            for g in range(state.Hkv):
                k, v = state.context(s, layer, g)
                heads = list(range(g * G, (g + 1) * G))
                q = Q[layer, s][:, heads].reshape(B * G, hd)
                qpos = np.repeat(ctx[s] + np.arange(B), G)
                o, lse = attend(q, qpos, k, v, theta)
                O[layer, s][:, heads] = o.reshape(B, G, hd)
                LSE[layer, s][:, heads] = lse.reshape(B, G)
    return O, LSE


def attend_state_with_self(state: State, Q, Kself, Vself, Hq, theta, seqs=None, layers=None):
    """Block attention over [C ; U ; S]: S is the block's own rows (the drafter's
    K/V of its B block positions, supplied by the caller), non-causal, with the
    keys rotated at the query positions ctx_len + i.  Kself, Vself
    [L][S][B][Hkv][hd] (keys unrotated).  Returns O, LSE like attend_state."""
    L, S, B, _, hd = Q.shape
    G = Hq // state.Hkv
    O = np.full(Q.shape, np.nan)
    LSE = np.full(Q.shape[:-1], np.nan)
    ctx = state.ctx_len()
    for s in (range(S) if seqs is None else seqs):
        pos = ctx[s] + np.arange(B)
        for layer in (range(L) if layers is None else layers):
            for g in range(state.Hkv):
                k, v = state.context(s, layer, g)
                ks = rope(np.asarray(Kself[layer, s, :, g], np.float64), pos, theta)
                k = np.concatenate([k, ks], axis=0)
                v = np.concatenate([v, np.asarray(Vself[layer, s, :, g], np.float64)], axis=0)
                heads = list(range(g * G, (g + 1) * G))
                q = Q[layer, s][:, heads].reshape(B * G, hd)
                o, lse = attend(q, np.repeat(pos, G), k, v, theta)
                O[layer, s][:, heads] = o.reshape(B, G, hd)
                LSE[layer, s][:, heads] = lse.reshape(B, G)
    return O, LSE


def carry_mass_state(state: State, Q, Hq, theta, seqs=None, layers=None):
    """carry_mass of every (layer, sequence, query row, query head) over the
    state's [C;U]; query i sits at ctx_len + i.  Returns [L][S][B][Hq] (NaN
    where not computed)."""
    L, S, B, _, hd = Q.shape
    G = Hq // state.Hkv
    out = np.full(Q.shape[:-1], np.nan)
    ctx = state.ctx_len()
    for s in (range(S) if seqs is None else seqs):
        for layer in (range(L) if layers is None else layers):
            for g in range(state.Hkv):
                heads = list(range(g * G, (g + 1) * G))
                q = Q[layer, s][:, heads].reshape(B * G, hd)
                qpos = np.repeat(ctx[s] + np.arange(B), G)
                mass = carry_mass(q, qpos, state.ck[s][layer, :, g], state.uk[s][layer, :, g],
                                  theta)
                out[layer, s][:, heads] = mass.reshape(B, G)
    return out


def round_update(state: State, r, H, E, WF, WKV, theta, mode="carry", seqs=None,
                 WF_carry=None, z_norm=None, k_norm=None):
    """Post-verification update of Algorithm 1 for the sequences in ``seqs``,
    given a route result ``r`` (see ``route``).  H [S][B][Dcat].  With
    ``WF_carry`` the carried rows use the separate projector (see project)."""
    S, B, _ = H.shape
    todo = []
    for s in (range(S) if seqs is None else seqs):
        if not r["touched"][s]:
            continue
        m = int(r["accept_len"][s])
        rows = np.arange(B) if mode in ("carry", "carry_only") else np.arange(m)
        todo.append((s, m, rows))
    if not todo:
        return
    # Eq. 1 acts on every row independently: the rows of all sequences go
    # through one call of ``project`` and are then split back per sequence.
    k_all, v_all = project(np.concatenate([H[s][rows] for s, _, rows in todo]), E,
                           np.concatenate([rows >= m for _, m, rows in todo]), WF, WKV,
                           np.concatenate([r["row_pos"][s][rows] for s, _, rows in todo]),
                           state.L, state.Hkv, state.hd, theta, WF_carry, z_norm, k_norm)
    at = 0
    for s, m, rows in todo:
        k, v = k_all[at:at + len(rows)], v_all[at:at + len(rows)]
        at += len(rows)
        if mode == "carry_only":
            k_acc, v_acc = k[:0], v[:0]
        else:
            k_acc, v_acc = k[:m], v[:m]
        if mode in ("carry", "carry_only"):
            k_rej, v_rej = k[m:], v[m:]
        else:
            k_rej, v_rej = k[:0], v[:0]
        state.commit_and_replace(s, k_acc, v_acc, k_rej, v_rej)
