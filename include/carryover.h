/*
 * carryover.h -- C ABI of the Carryover drafter step on MI355X (gfx950).
 *
 * One drafting round of a block-diffusion speculative drafter with Carryover
 * (paper: Section 2.1, Eqs. 1-2; Appendix A, Algorithm 1 and its "Cache
 * semantics" paragraph):
 *
 *   route      split each verified window of B rows by its accepted prefix m
 *              (greedy verification, Section 2 "Preliminaries");
 *   project    x = h (+ E_carry on rejected rows), z = F x, and for every
 *              drafter layer l: k = K_l z, v = V_l z; keys are rotated once at
 *              the row's absolute position; accepted rows are appended to the
 *              paged committed cache C_l, rejected rows replace the carryover
 *              segment U_l (at most B rows);
 *   attention  the next block's queries attend to ctx_l = [C_l ; U_l].
 *
 * Conventions shared by every call
 * --------------------------------
 * Ownership: every pointer is caller-owned device memory unless a comment says
 *   "host".  The library allocates nothing, frees nothing, keeps no pointer
 *   past the call and holds no global state besides per-device attributes
 *   and the launch-shape overrides of carryover_set_tuning.
 * Streams: every call only enqueues work on `stream` and returns; nothing
 *   synchronises except carryover_read_status.  Calls on distinct states are
 *   re-entrant.
 * Errors: problems visible on the host (null or misaligned pointer,
 *   unsupported shape or dtype, small workspace) return a non-zero co_status
 *   and enqueue nothing.  Problems that depend on device-resident data
 *   (capacity, page ids, negative lengths) are written to *state->status
 *   (first error wins); the offending sequence is left unchanged and the other
 *   sequences proceed.  The caller zeroes *status before first use.
 * Dtype: one element type per call for hidden states, weights, queries,
 *   caches and outputs (dims.dtype).  Accumulation, softmax and the optional
 *   LSE output are fp32.
 * Supported shapes: head_dim in {64, 128}; page_size == 16; num_q_heads a
 *   multiple of num_kv_heads with block * (num_q_heads / num_kv_heads) <= 64;
 *   feat_dim and model_dim multiples of 64; block >= 1.
 *
 * Memory layouts (row-major, innermost last; P = page_size = 16,
 * CP = ceil(block / 16), NKV = 2 * num_layers * num_kv_heads * head_dim):
 *   hidden      [num_seqs][block][feat_dim]         target features H, Eq. 1
 *   w_f         [model_dim][feat_dim]               fusion projection F
 *   w_kv        [NKV][model_dim], rows ordered (layer, K|V, kv head, dim)
 *   e_carry     [feat_dim]                          E_carry, Eq. 2
 *   q           [layers][num_seqs][block][num_q_heads][head_dim], un-rotated
 *   out         same shape as q
 *   lse         [layers][num_seqs][block][num_q_heads] fp32, natural log
 *   page_table  int32 [num_seqs][max_pages_per_seq]
 *   k_cache     [num_layers][num_pages][num_kv_heads][P][head_dim]
 *   v_cache     [num_layers][num_pages][num_kv_heads][head_dim][P]  (slot fastest)
 *   k_carry     [num_layers][num_seqs][CP][num_kv_heads][P][head_dim]
 *   v_carry     [num_layers][num_seqs][CP][num_kv_heads][head_dim][P]
 * Logical position t of sequence s lives in page page_table[s][t / 16], slot
 * t % 16.  Carry row r of sequence s lives in carry page r / 16, slot r % 16.
 */
#ifndef CARRYOVER_H
#define CARRYOVER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t;

typedef int32_t co_status;
enum {
  CO_OK = 0,
  CO_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, negative count        */
  CO_ERR_UNSUPPORTED = 2,   /* shape or dtype outside the supported set        */
  CO_ERR_WORKSPACE = 3,     /* workspace smaller than carryover_workspace_bytes */
  CO_ERR_CAPACITY = 4,      /* device: ctx_len + block > max_pages_per_seq * 16 */
  CO_ERR_PAGE_RANGE = 5,    /* device: page id outside [0, num_pages)          */
  CO_ERR_HIP = 6,           /* a HIP runtime call or launch failed             */
  CO_ERR_LENGTH = 7,        /* device: ctx_len outside [0, max_pages_per_seq * 16] or
                               carry_len outside [0, 16 * ceil(block / 16)]        */
  CO_ERR_GROUP = 8,         /* device: a sequence's committed page ids differ from its
                               group's first sequence (attention backward)          */
  CO_ERR_TOKEN = 9          /* device: a proposed token outside [0, vocab)
                               (carryover_verify_sample)                            */
};

enum { CO_DTYPE_F32 = 0, CO_DTYPE_BF16 = 1 };

/* flags */
#define CO_BASELINE_MODE    (1u << 0) /* Algorithm 1 left column: commit 0..m-1, no carry      */
#define CO_ROUTE_ACCEPT_ALL (1u << 1) /* m := block for every sequence (build context)         */
#define CO_ROUTE_CARRY_ONLY (1u << 2) /* rows 0..m-1 are already committed: store only carries */
#define CO_Q_PREROTATED     (1u << 3) /* queries already carry their rotary embedding          */
#define CO_ATTN_SHARED_PREFIX (1u << 4) /* bf16 attention: consecutive sequences are blocks of one
                                         recorded response whose committed keys are prefixes of
                                         the same pages (Algorithm 2); key tiles are read once
                                         per group of four (head_dim 64, or head_dim 128 with up
                                         to 32 query rows per KV head; other shapes ignore the
                                         flag).  Results do not depend on the flag.             */
#define CO_ROUTE_ACCEPT_BITS (1u << 5)  /* stochastic verification (T = 1): draft_tok holds the
                                         verifier's accept decision of every position (non-zero
                                         = accepted by its rejection sampling), target_tok is
                                         unused and may be NULL; m = the accepted positions
                                         before the first rejection                             */

typedef struct co_dims {
  int32_t num_seqs;           /* S: sequences in the batch                           */
  int32_t block;              /* B: verified-window rows = block queries per sequence */
  int32_t feat_dim;           /* width of a concatenated target feature row h        */
  int32_t model_dim;          /* d: width of F's output                              */
  int32_t num_layers;         /* L: drafter layers                                   */
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t page_size;          /* must be 16                                          */
  int32_t max_pages_per_seq;  /* columns of page_table                               */
  int32_t num_pages;          /* pages in the cache pool                             */
  int32_t dtype;              /* CO_DTYPE_F32 or CO_DTYPE_BF16                       */
  float rope_theta;           /* rotary base; inverse frequency theta^(-2i/head_dim) */
} co_dims;

typedef struct co_weights {
  const void* w_f;            /* F:  [model_dim][feat_dim]                 */
  const void* w_kv;           /* K_l, V_l of all layers: [NKV][model_dim]  */
  const void* e_carry;        /* E_carry: [feat_dim]                       */
  const float* f_e;           /* optional F e_carry, fp32 [model_dim], from carryover_fold_e;
                                 NULL: computed within every bf16 projection           */
  const void* w_f_carry;      /* optional separate projector for carried rows,
                                 [model_dim][feat_dim] (Section 4, "How should rejected
                                 states be distinguished?", Table 3(b)): when non-NULL,
                                 rows routed to the carry segment are projected by it
                                 instead of by F with E_carry (e_carry and f_e unused;
                                 costs a second F product)                            */
  const float* z_norm;        /* optional RMS-norm gain, fp32 [model_dim]: when non-NULL
                                 every row of z = F x is divided by its root mean square
                                 (epsilon 1e-6) and multiplied by z_norm before the K/V
                                 projections (normalisation variant; the equations omit
                                 normalisation, Section 2.1); model_dim <= 16384
                                 (CO_ERR_UNSUPPORTED otherwise)                       */
  const float* k_norm;        /* optional per-head key RMS-norm gain, fp32
                                 [num_layers][head_dim]: when non-NULL every key head of
                                 layer l is divided by its root mean square over head_dim
                                 (epsilon 1e-6) and multiplied by k_norm[l] before it is
                                 rotated; values are not normalised (normalisation
                                 variant, as z_norm).  Keys passed in by the caller
                                 (carryover_import_kv, drafter_self_merge) are taken as
                                 they are                                             */
} co_weights;

typedef struct co_state {
  int32_t* ctx_len;           /* [num_seqs] committed rows |C_l|           */
  int32_t* carry_len;         /* [num_seqs] carryover rows |U_l| <= block  */
  const int32_t* page_table;  /* [num_seqs][max_pages_per_seq]             */
  void* k_cache;
  void* v_cache;
  void* k_carry;
  void* v_carry;
  int32_t* status;            /* one int32: first data-dependent error     */
} co_state;

typedef struct co_route {
  int32_t* accept_len;        /* [num_seqs] m                                              */
  int32_t* row_pos;           /* [num_seqs][block] absolute position of window row j       */
  int32_t* row_dst;           /* [num_seqs][block] >= 0: global committed slot page*16+t%16;
                                 -1-r: carry row r; INT32_MIN: not stored                   */
} co_route;

/*
 * Route (Algorithm 1 "Given"; greedy verification, Section 2
 * "Preliminaries").  For every sequence s: m = length of the longest prefix on
 * which draft_tok[s][:] equals target_tok[s][:] (m = block with
 * CO_ROUTE_ACCEPT_ALL, where the token pointers may be NULL; with
 * CO_ROUTE_ACCEPT_BITS, the run of non-zero accept decisions in draft_tok at the
 * start of the window, Appendix A "Why verification remains valid");
 * p0 = ctx_len[s];
 * window row j sits at position p0 + j.  Rows j < m go to the committed slot of
 * position p0 + j (skipped under CO_ROUTE_CARRY_ONLY); rows j >= m become carry
 * row j - m (skipped under CO_BASELINE_MODE).  Then ctx_len[s] = p0 + m and
 * carry_len[s] = block - m (0 in baseline mode), which replaces the old
 * carryover segment.  Tokens: int32 [num_seqs][block], device.
 * Device errors: CO_ERR_LENGTH (p0 < 0), CO_ERR_CAPACITY
 * (p0 + block > max_pages_per_seq * 16), CO_ERR_PAGE_RANGE (a committed row's
 * page id outside [0, num_pages)); the sequence then keeps its lengths, stores
 * nothing (row_dst = INT32_MIN) and reports accept_len 0.
 */
co_status carryover_route(const co_dims* dims, const int32_t* draft_tok, const int32_t* target_tok,
                          uint32_t flags, co_state* state, const co_route* out, hipStream_t stream);

/*
 * Project (Eq. 1, Eq. 2; Algorithm 1 Carryover steps 1-6; "Cache semantics").
 * For every window row r = s * block + j described by `route`:
 * x = hidden[r] (+ e_carry when row_dst[r] names a carry row, Eq. 2), z = F x,
 * and for every layer l and KV head g: k = K_{l,g} z rotated at row_pos[r],
 * v = V_{l,g} z; the row is written to its committed slot or carry row in
 * every layer, or dropped when row_dst[r] == INT32_MIN.  F, K_l, V_l have no
 * bias and no normalisation.  `ws` must hold
 * carryover_workspace_bytes(dims, CO_WS_PROJECT) bytes (256-byte aligned).
 */
co_status carryover_project_kv(const co_dims* dims, const co_weights* w, const void* hidden,
                               const co_route* route, const co_state* state, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/*
 * Fold the carry embedding through F once per set of weights (Eq. 2 with F
 * linear, no bias): f_e[i] = sum_k w_f[i][k] * e_carry[k] for i < model_dim,
 * accumulated in fp32 from the stored values.  A bf16 projection then adds
 * f_e to F h of carry rows (F(h + E) = F h + F E) instead of recomputing F E
 * from e_carry; fp32 projections add e_carry to h and ignore f_e.  f_e:
 * caller-owned device memory, fp32 [model_dim], 16-byte aligned.
 */
co_status carryover_fold_e(const co_dims* dims, const co_weights* w, float* f_e,
                           hipStream_t stream);

/*
 * Block attention over ctx_l = [C_l ; U_l] (Eq. 2; Algorithm 1 step 7;
 * "Preliminaries": draft positions attend to KV built from target states).
 * For layers layer_begin .. layer_begin + layer_count - 1, every sequence s,
 * block query i and query head h: the query q[l'][s][i][h] (l' = l -
 * layer_begin) is rotated at position ctx_len[s] + i (unless
 * CO_Q_PREROTATED), scaled by 1/sqrt(head_dim) and attends, with no position
 * mask, to the ctx_len[s] committed keys of KV head h / (num_q_heads /
 * num_kv_heads) followed by its carry_len[s] carry keys.  out has q's layout;
 * lse (optional, may be NULL) receives the natural-log normaliser.  An empty
 * key set gives out = 0 and lse = -inf.  `ws` must hold
 * carryover_workspace_bytes(dims, CO_WS_ATTENTION) bytes (scratch; any
 * contents).  A workspace serves one call at a time.
 * Device errors: CO_ERR_LENGTH (ctx_len outside [0, max_pages_per_seq * 16]
 * or carry_len outside [0, 16 * ceil(block / 16)]): that sequence attends to
 * no key (out 0, lse -inf); CO_ERR_PAGE_RANGE (a page id of a committed key
 * outside [0, num_pages)): the keys of that page are left out.  The other
 * sequences proceed.
 */
co_status drafter_block_attention(const co_dims* dims, int32_t layer_begin, int32_t layer_count,
                                  const void* q, const co_state* state, void* out, float* lse,
                                  uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * drafter_block_attention with two extras computed in the same one-pass merge
 * (bf16: the keys stream once, every segment shares one online softmax):
 *   - the block's own rows as a third segment S (the drafter's keys and
 *     values of its B block positions, attended non-causally next to
 *     ctx = [C;U] of Eq. 2; "Preliminaries": draft positions attend within
 *     the block): out and lse are the attention over [C;U;S].  k_self, v_self:
 *     [layer_count][num_seqs][block][num_kv_heads][head_dim] in the call's
 *     dtype, 16-byte aligned, keys unrotated (rotated here at ctx_len + j for
 *     self row j, as the queries are).  Both NULL: no self segment.
 *   - carry_mass (optional, NULL: none), fp32 [layer_count][num_seqs][block]
 *     [num_q_heads]: the share of each query's softmax weight over [C;U] that
 *     falls on U (Appendix "Attention to carried states"; with S present its
 *     keys are left out of the share); 0 where [C;U] is empty.
 * Other arguments, workspace and errors as drafter_block_attention; with
 * neither extra the call is drafter_block_attention.  Supported: block <= 64
 * (CO_ERR_UNSUPPORTED otherwise).  bf16 computes both extras inside the
 * serving attention kernels (CO_ATTN_SHARED_PREFIX is then ignored); fp32
 * runs the attention, then drafter_carry_mass and drafter_self_merge on its
 * output, and needs lse (CO_ERR_INVALID_ARG when NULL).
 */
co_status drafter_block_attention_ext(const co_dims* dims, int32_t layer_begin,
                                      int32_t layer_count, const void* q, const void* k_self,
                                      const void* v_self, const co_state* state, void* out,
                                      float* lse, float* carry_mass, uint32_t flags, void* ws,
                                      size_t ws_bytes, hipStream_t stream);

/*
 * One full drafter round (Algorithm 1, Carryover column, or the Baseline
 * column with CO_BASELINE_MODE): route, project all layers, then attend with
 * every layer's queries q [num_layers][num_seqs][block][num_q_heads][head_dim].
 * `scratch` receives the route result.  All state stays on the device; there
 * is no host synchronisation.  `ws`: carryover_workspace_bytes(dims,
 * CO_WS_ROUND) bytes of scratch, 256-byte aligned.  flags: those of
 * carryover_route and drafter_block_attention.  Every host check of the three
 * steps (the weights' optional pointers included) is made before the first
 * launch, so a non-zero return leaves the state untouched.  Device errors:
 * those of the three steps.
 */
co_status carryover_round(const co_dims* dims, const co_weights* w, const void* hidden,
                          const int32_t* draft_tok, const int32_t* target_tok, const void* q,
                          co_state* state, const co_route* scratch, void* out, float* lse,
                          uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * carryover_round for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same round, with the same arguments except the workspace, which is the
 * library's own static device scratch of CO_NOALLOC_SCRATCH_BYTES (128 MiB)
 * per device, held from the device's first use until the process ends.  The
 * call allocates nothing.  Returns CO_ERR_WORKSPACE when
 * carryover_workspace_bytes(dims, CO_WS_ROUND) exceeds the scratch; other
 * errors as carryover_round.  Every call on a device shares that device's
 * scratch (which keeps the last call's contents, none of which a call reads
 * first): calls that overlap on one device -- on different streams or from
 * different threads -- race; serialise them.
 */
#define CO_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
co_status carryover_round_noalloc(const co_dims* dims, const co_weights* w, const void* hidden,
                                  const int32_t* draft_tok, const int32_t* target_tok,
                                  const void* q, co_state* state, const co_route* route_out,
                                  void* out, float* lse, uint32_t flags, hipStream_t stream);

/*
 * Stochastic verification (T = 1): the acceptance decision and the
 * correction or bonus token of the standard speculative-sampling rule that
 * Appendix A ("Why verification remains valid") relies on.  For every
 * sequence s, with the proposals x_j = draft_tok[s][j] (j < block), the
 * target's probabilities p_target [num_seqs][block + 1][vocab] (fp32; row
 * block is the position after the window) and the drafter's q_draft
 * [num_seqs][block][vocab] (fp32):
 *   proposal j is accepted iff u_j * q_j(x_j) < p_j(x_j), with
 *     u_j = (words[s][j] >> 8) * 2^-24 (decided exactly);
 *   m = the accepted proposals before the first rejection;
 *   accept_bits[s][j] = (j < m), int32 [num_seqs][block]: the accept decisions
 *     carryover_route and carryover_round take under CO_ROUTE_ACCEPT_BITS;
 *   accept_len[s] = m;
 *   next_tok[s] = the correction (m < block), drawn from max(0, p_m - q_m)
 *     normalised, or the bonus (m = block), drawn from p_block: with
 *     w(y) = floor(2^32 * d(y)), d(y) = p(y) - q(y) in fp64 where positive
 *     (p(y) for the bonus, and for a correction whose weights are all zero),
 *     the smallest y whose running sum of w exceeds
 *     floor(words[s][block] * W / 2^32), W the total; -1 if W = 0.
 * words: uint32 [num_seqs][block + 1] of uniform random bits.  Only num_seqs
 * and block of dims are used (the rest must still be valid).  status: one
 * int32 (e.g. a state's status word).  All pointers device, 4-byte aligned.
 * Device errors: CO_ERR_TOKEN (a proposal outside [0, vocab)); that sequence
 * gets m = 0, all bits 0 and next_tok -1.
 */
co_status carryover_verify_sample(const co_dims* dims, int32_t vocab, const int32_t* draft_tok,
                                  const float* p_target, const float* q_draft,
                                  const uint32_t* words, int32_t* accept_bits,
                                  int32_t* accept_len, int32_t* next_tok, int32_t* status,
                                  hipStream_t stream);

/*
 * Reverse mode of drafter_block_attention: the training side of the second
 * drafter pass (Algorithm 2, whose loss is differentiated through the second
 * draft's attention over ctx = [C;U], Eq. 2).  For the layers, q, state and
 * CO_Q_PREROTATED flag of a forward call whose output was `out` and whose LSE
 * (natural log, required) was `lse`, and the gradient d_out of a loss with
 * respect to out (q's layout, bf16):
 *   d_q [layer_count][num_seqs][block][num_q_heads][head_dim] fp32: the
 *     gradient with respect to q (un-rotated queries unless CO_Q_PREROTATED);
 *   d_k_cache, d_v_cache: fp32 arrays shaped like k_cache and v_cache; the
 *     entries of every committed key some block query sees are overwritten
 *     with the gradient with respect to the stored (rotated) key and the value,
 *     summed over every query that sees it; other entries are left unchanged;
 *   d_k_carry, d_v_carry: the same for the carry segment (shaped like k_carry,
 *     v_carry).
 * seqs_per_group: consecutive sequences g * n .. g * n + n - 1 read the same
 * committed page row (the blocks of one recorded response in training; they
 * may differ in ctx_len), and no page appears in two groups' rows; 1 when
 * sequences share no pages.  A sequence whose page ids differ from its group's
 * first sequence sets CO_ERR_GROUP.
 * Supported: bf16, head_dim 64, block * (num_q_heads / num_kv_heads) <= 32.
 * All pointers 16-byte aligned; `ws`: carryover_workspace_bytes(dims,
 * CO_WS_ATTENTION_BACKWARD) bytes of scratch, 256-byte aligned.  Device
 * errors: CO_ERR_LENGTH, CO_ERR_PAGE_RANGE (keys of a rejected page id get no
 * gradient), CO_ERR_GROUP.  Results are deterministic (no atomics).
 */
co_status drafter_block_attention_backward(
    const co_dims* dims, int32_t layer_begin, int32_t layer_count, const void* q,
    const co_state* state, const void* out, const float* lse, const void* d_out,
    int32_t seqs_per_group, float* d_q, float* d_k_cache, float* d_v_cache, float* d_k_carry,
    float* d_v_carry, uint32_t flags, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Reverse mode of carryover_project_kv for the trained parameters (Algorithm 2:
 * the second pass's loss reaches W_F, W_KV and E_carry through the K/V rows
 * of Eqs. 1-2; the target's states are constants).  For the dims, weights,
 * hidden rows and route of a forward carryover_project_kv call, and fp32
 * gradient arrays shaped like the caches (d_k_cache / d_v_cache like
 * k_cache / v_cache, d_k_carry / d_v_carry like k_carry / v_carry, e.g. from
 * drafter_block_attention_backward) holding the gradient of a loss with
 * respect to the stored (rotated) keys and the values: every row r with a
 * destination takes the gradient at that destination (committed slot or carry
 * row), its key gradient rotated back at row_pos[r]; rows that were not stored
 * contribute nothing.  With x_r = h_r (+ e_carry on carried rows) and
 * z_r = F x_r, the call ADDS
 *   d_w_f     fp32 [model_dim][feat_dim]:  sum_r (W_KV^T dJ_r) x_r^T,
 *   d_w_kv    fp32 [NKV][model_dim]:       sum_r dJ_r z_r^T,
 *   d_e_carry fp32 [feat_dim]:             sum over carried r of F^T W_KV^T dJ_r,
 * so that the two forward calls of a training step (committed rows, then the
 * blocks' carried rows) accumulate into the same arrays (zero them first).
 * Operands are rounded to bf16 for the products (fp32 sums); deterministic.
 * Supported: bf16; the plain update only (w_f_carry, z_norm and k_norm NULL,
 * else CO_ERR_UNSUPPORTED).  `ws`: carryover_workspace_bytes(dims,
 * CO_WS_PROJECT_BACKWARD) bytes, 256-byte aligned.
 */
co_status carryover_project_kv_backward(const co_dims* dims, const co_weights* w,
                                        const void* hidden, const co_route* route,
                                        const float* d_k_cache, const float* d_v_cache,
                                        const float* d_k_carry, const float* d_v_carry,
                                        float* d_w_f, float* d_w_kv, float* d_e_carry, void* ws,
                                        size_t ws_bytes, hipStream_t stream);

/*
 * Attention mass on the carried rows (the diagnostic of Appendix "Attention to
 * carried states"; for the carry segment U of ctx = [C;U], Eq. 2).  For every
 * (layer, sequence, block row i, query head h) of a drafter_block_attention
 * call made with the same dims, layers, q, state and CO_Q_PREROTATED flag:
 * mass = the sum over U of the softmax weights = exp(LSE_U - LSE), where LSE is
 * that call's LSE output (natural log) and LSE_U the log-sum-exp of the scaled
 * logits over the carry keys alone; 0 when U is empty or no key exists.
 * q as for drafter_block_attention; lse (input) and mass (output) fp32
 * [layer_count][num_seqs][block][num_q_heads].  flags: CO_Q_PREROTATED.
 * Enqueue after the attention call, before anything changes the state.
 * Supported shapes: those of drafter_block_attention with block <= 64.
 * Device errors: CO_ERR_LENGTH (a negative length, or carry_len > the carry
 * segment); that sequence's mass is then 0.
 */
co_status drafter_carry_mass(const co_dims* dims, int32_t layer_begin, int32_t layer_count,
                             const void* q, const co_state* state, const float* lse, float* mass,
                             uint32_t flags, hipStream_t stream);

/*
 * The block's own rows as a third attention segment S (the drafter's keys and
 * values of its B block positions, attended non-causally, next to
 * ctx = [C;U] of Eq. 2).  For every (layer, sequence, block row i, query head h)
 * of a drafter_block_attention call made with the same dims, layers, q, state
 * and CO_Q_PREROTATED flag, and with its lse output: the attention of the query
 * over the B self keys k_self (rotated here at positions ctx_len + j, j < B)
 * and values v_self is merged into out and lse in place by the log-sum-exp
 * rule, so that they hold the attention over [C;U;S] in one softmax.
 * k_self, v_self: [layer_count][num_seqs][block][num_kv_heads][head_dim] in
 * the call's dtype, keys unrotated.  out, lse: as written by the attention
 * call.  flags: CO_Q_PREROTATED.  Supported: the attention call's shapes with
 * block <= 64.  Device errors: CO_ERR_LENGTH (negative ctx_len); that
 * sequence is left as it was.
 */
co_status drafter_self_merge(const co_dims* dims, int32_t layer_begin, int32_t layer_count,
                             const void* q, const void* k_self, const void* v_self,
                             const co_state* state, void* out, float* lse, uint32_t flags,
                             hipStream_t stream);


/*
 * Write already-projected (keys already rotated) committed rows of one
 * sequence into the paged cache: k_rows, v_rows [num_layers][num_kv_heads]
 * [n_rows][head_dim] are stored at positions pos0 .. pos0 + n_rows - 1 of
 * sequence `seq`.  Lengths are not changed.  Host errors: seq or positions
 * outside the table (CO_ERR_INVALID_ARG); device: CO_ERR_PAGE_RANGE.
 */
co_status carryover_import_kv(const co_dims* dims, int32_t seq, int32_t pos0, int32_t n_rows,
                              const void* k_rows, const void* v_rows, const co_state* state,
                              hipStream_t stream);

enum { CO_WS_PROJECT = 0, CO_WS_ATTENTION = 1, CO_WS_ROUND = 2, CO_WS_ATTENTION_BACKWARD = 3,
       CO_WS_PROJECT_BACKWARD = 4 };

/* Workspace bytes a call needs for these dims (0 on unsupported dims). */
size_t carryover_workspace_bytes(const co_dims* dims, int32_t which);

/* Synchronise `stream` and copy *state->status to *host_out (host pointer). */
co_status carryover_read_status(const co_state* state, int32_t* host_out, hipStream_t stream);

/*
 * Launch-shape overrides, for tuning and for tests that force every kernel
 * variant.  Results never depend on them (beyond rounding order).  `value`
 * -1 restores the automatic choice.  Process-wide: set them while no call is
 * in flight.  Knobs:
 *   CO_TUNE_GEMM_WIDE_VARIANT       large-tile projection GEMM variant 0..6
 *   CO_TUNE_GEMM_NO_WIDE            1: never the large-tile projection GEMM
 *   CO_TUNE_PROJECT_FUSED_MIN_ROWS  rows from which the fused small-width
 *                                   projection runs (default 4096)
 *   CO_TUNE_ATTN_WAVE               0/1: bf16 attention by per-wavefront slices
 *   CO_TUNE_ATTN_WORKGROUPS         bf16 attention workgroups (or slices)
 *   CO_TUNE_ATTN_ROUND_TILES        tiles per wavefront per round, persistent
 *                                   attention kernel
 *   CO_TUNE_ATTN_GROUP_SPLIT_TILES  committed tiles per share, grouped-prefix
 *                                   attention
 * Returns CO_ERR_INVALID_ARG for an unknown knob.  Workspace sizes follow the
 * overrides in force when carryover_workspace_bytes is called.
 */
enum { CO_TUNE_GEMM_WIDE_VARIANT = 0, CO_TUNE_GEMM_NO_WIDE = 1, CO_TUNE_PROJECT_FUSED_MIN_ROWS = 2,
       CO_TUNE_ATTN_WAVE = 3, CO_TUNE_ATTN_WORKGROUPS = 4, CO_TUNE_ATTN_ROUND_TILES = 5,
       CO_TUNE_ATTN_GROUP_SPLIT_TILES = 6, CO_TUNE_COUNT = 7 };
co_status carryover_set_tuning(int32_t knob, int64_t value);

/* Static message for a status code. */
const char* carryover_status_string(co_status status);

#ifdef __cplusplus
}
#endif

#endif /* CARRYOVER_H */
