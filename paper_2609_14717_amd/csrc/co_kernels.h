// Launch interfaces of the gfx950 kernels (internal to libcarryover).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "co_device.h"

namespace co {

constexpr int kMaxHeadDim = 128;

struct RouteArgs {
  int S, B, max_pages, num_pages;
  uint32_t flags;
  const int32_t* draft;
  const int32_t* target;
  int32_t* ctx_len;
  int32_t* carry_len;
  const int32_t* page_table;
  int32_t* accept_len;
  int32_t* row_pos;
  int32_t* row_dst;
  int32_t* status;
};

// Where projected K/V rows go: the paged committed cache or the carry segment.
struct KvDest {
  int S, B, L, Hkv, hd, num_pages, CP;
  double rope_inv[kMaxHeadDim / 2];   // RoPE inverse frequencies theta^(-2i/hd)
  const int32_t* row_pos;
  const int32_t* row_dst;
  void* k_cache;
  void* v_cache;
  void* k_carry;
  void* v_carry;
  int32_t* status;
  const float* knorm;   // per-head key RMS-norm gain [L][hd], or null
};

struct ProjectArgs {
  int M, Dcat, d, dtype;
  const void* hidden;
  const void* wf;
  const void* wkv;
  const void* e;
  const float* fe;   // precomputed F(E) [d] (bf16 path), or null
  const void* wfc;   // separate carry projector [d][Dcat], or null
  const float* znorm;   // RMS-norm gain of F's output [d], or null
  KvDest dst;
  void* ws;
  // The round's route step, carried by the F product's launch (see
  // route_foldable), or null: the route has already been enqueued.
  const RouteArgs* route;
};

struct ProjectPlan {
  int f_tile, f_split;     // tile variant and K-splits of the F GEMM
  int kv_tile, kv_split;   // same for the K/V GEMM
  bool fused;              // both products in one kernel (small widths, many rows)
  size_t z_bytes, part_bytes, pe_bytes, total;
};

ProjectPlan plan_project(int M, int Dcat, int d, int n_kv, int hd, int dtype, int num_cus);

// Whether launch_project can run the route step inside its first launch: the
// F product then decides carried rows from the tokens itself, and the route's
// descriptors are complete before the K/V product reads them.
bool route_foldable(const ProjectArgs& a, const ProjectPlan& p);

constexpr int kNormMaxCols = 16384;   // widest F output the RMS normalisation takes

struct AttnArgs {
  int S, B, L, layer_begin, Hq, Hkv, hd, num_pages, max_pages, CP, dtype;
  uint32_t flags;
  double rope_inv[kMaxHeadDim / 2];   // RoPE inverse frequencies theta^(-2i/hd)
  const void* q;
  const int32_t* ctx_len;
  const int32_t* carry_len;
  const int32_t* page_table;
  const void* k_cache;
  const void* v_cache;
  const void* k_carry;
  const void* v_carry;
  void* out;
  float* lse;
  int32_t* status;
  float* ws;        // partial records of multi-chunk sequences
  // bf16 slice records: floats per query row after the hd output dims (m, l;
  // and with the extras below, the carry and self sums)
  int rec_sums;
  // extras of drafter_block_attention_ext (bf16 persistent kernel), or null:
  const void* k_self;   // the block's own keys [layers][S][B][Hkv][hd], unrotated
  const void* v_self;   // and values
  float* mass;          // share of the attention over [C;U] on U, [layers][S][B][Hq]
};

constexpr int kMaxAttnSeqs = 2048;   // sequences one bf16 attention launch can cover

struct AttnPlan {
  int chunk_pages, n_chunks;   // fp32 path
  int n_wg, hdr_floats;        // bf16 persistent path: workgroups, header floats
  int round_tiles;             // bf16 persistent path: tiles per wavefront per round
  int64_t park_off;            // bf16 persistent path: parked partials (workspace floats)
  bool wave;                   // bf16: per-wavefront slices (n_wg = slices, not workgroups)
  int nq_pad;
  bool ok;                     // false: shapes beyond what one launch can cover
  size_t bytes;
};

AttnPlan plan_attention(int S, int B, int L, int Hq, int Hkv, int hd, int max_pages, int num_pages,
                        int dtype, int num_cus);

// Reverse mode of the bf16 attention (head_dim 64, up to 32 query rows per KV
// head): `a` carries the forward's arguments with ws = the backward workspace.
struct BwdArgs {
  AttnArgs a;
  int layer_count, group;   // layers of the launch; sequences per shared page row
  const void* out;          // forward output O (bf16)
  const float* lse;         // forward LSE (natural log)
  const void* d_out;        // dO (bf16)
  float* d_q;               // [layers][S][B][Hq][hd]
  float* d_k_cache;         // like k_cache, fp32
  float* d_v_cache;         // like v_cache, fp32
  float* d_k_carry;         // like k_carry, fp32
  float* d_v_carry;         // like v_carry, fp32
};

size_t bwd_workspace_bytes(int S, int L, int Hkv, int hd, int num_pages, int CP);
hipError_t launch_attention_backward(const BwdArgs& b, hipStream_t stream);

// Plain fp32 product C (+)= A . B^T of bf16 operands with K contiguous; the
// K-split partials go to `part` (gemm_acc_ws_bytes).
size_t gemm_acc_ws_bytes(int M, int N, int K, int num_cus);
hipError_t launch_gemm_acc(const void* A, const void* B, int M, int N, int K, float* C,
                           bool accumulate, float* part, int num_cus, hipStream_t stream);

// Reverse mode of the K/V projection (bf16, plain update) for W_F, W_KV and
// E_carry: the rows' K/V gradients are gathered from fp32 gradient caches by
// the route's destinations.
struct ProjBwdArgs {
  int M, Dcat, d, L, Hkv, hd, S, B, num_pages, CP, num_cus;
  double rope_inv[kMaxHeadDim / 2];
  const void* hidden;
  const void* wf;
  const void* wkv;
  const void* e;
  const int32_t* row_dst;
  const int32_t* row_pos;
  const float *dk, *dv, *dkc, *dvc;   // gradient caches shaped like the caches
  float *dwf, *dwkv, *de;             // accumulated
  void* ws;
};

size_t proj_bwd_ws_bytes(int M, int Dcat, int d, int n_kv, int num_cus);
hipError_t launch_project_backward(const ProjBwdArgs& p, hipStream_t stream);

// Attention mass on the carried rows, from a finished attention call's LSE.
constexpr int kMaxCarryRows = 64;   // carry rows of one sequence (block <= 64)

struct MassArgs {
  int S, B, layer_begin, Hq, Hkv, hd, CP;
  uint32_t flags;
  double rope_inv[kMaxHeadDim / 2];   // RoPE inverse frequencies theta^(-2i/hd)
  const void* q;
  const int32_t* ctx_len;
  const int32_t* carry_len;
  const void* k_carry;
  const float* lse;
  float* mass;
  int32_t* status;
};

// The block's own rows as a third attention segment, merged into (O, LSE).
struct SelfArgs {
  int S, B, Hq, Hkv, hd;
  uint32_t flags;
  double rope_inv[kMaxHeadDim / 2];   // RoPE inverse frequencies theta^(-2i/hd)
  const void* q;
  const void* k_self;
  const void* v_self;
  const int32_t* ctx_len;
  void* out;
  float* lse;
  int32_t* status;
};

// Stochastic verification (T = 1): accept decisions and the correction or bonus.
struct VerifyArgs {
  int S, B, V;
  const int32_t* draft;    // [S][B]
  const float* p;          // [S][B + 1][V]
  const float* q;          // [S][B][V]
  const uint32_t* words;   // [S][B + 1]
  int32_t* accept_bits;    // [S][B]
  int32_t* accept_len;     // [S]
  int32_t* next_tok;       // [S]
  int32_t* status;
};

// Launch-shape override in force (-1: automatic); see carryover_set_tuning.
int64_t tuning(int knob);

hipError_t launch_route(const RouteArgs& a, hipStream_t stream);
hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream);
hipError_t launch_self_merge(const SelfArgs& a, int layer_count, int dtype, hipStream_t stream);
hipError_t launch_carry_mass(const MassArgs& a, int layer_count, int dtype, hipStream_t stream);
hipError_t launch_project(const ProjectArgs& a, const ProjectPlan& p, hipStream_t stream);
hipError_t launch_attention(const AttnArgs& a, const AttnPlan& p, int layer_count,
                            hipStream_t stream);
hipError_t launch_fold_e(const void* wf, const void* e, int d, int Dcat, int dtype, float* out,
                         hipStream_t stream);
hipError_t launch_import(const KvDest& d, int dtype, int seq, int pos0, int n, const void* k_rows,
                         const void* v_rows, const int32_t* page_table, int max_pages,
                         hipStream_t stream);

}  // namespace co
