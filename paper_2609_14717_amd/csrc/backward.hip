// Reverse mode of the block attention over ctx = [C ; U]: the training side of
// the second drafter pass (Algorithm 2 -- the loss of the second draft is
// differentiated through its attention and the K/V projection, with the
// target's states held constant; Eq. 2 gives the attended context).
//
// With S = (R q) k^T / sqrt(hd) per (layer, sequence, KV head), P the softmax
// weights, dO the output gradient and D_i = dO_i . O_i (= sum_j P_ij dO_i.v_j):
//   dV = P^T dO,   dS = P * (dO V^T - D),   dK = dS^T (R q) / sqrt(hd),
//   dq = R^T (dS K) / sqrt(hd).
// Committed keys may be shared by the blocks of one recorded response (the
// training layout: consecutive sequences of a group read the same page row),
// so their gradients are sums over the group's blocks.
//
// Four kernels; the products run on v_mfma_f32_32x32x16_bf16 (bf16 operands,
// fp32 sums):
//   prep   per (layer, KV head, sequence): the rotated, scaled queries (log2
//          units, as the forward forms them) and their transpose, dO packed
//          and transposed, and -LSE (log2 units) and -D, which the products
//          then take as their starting sums;
//   copy   every K page transposed ([hd][16]) and every V page in key-major
//          order ([16][hd]), so that all MFMA operands are 16-byte reads with
//          the contracted index contiguous;
//   attn   one launch with two kinds of workgroup (eight wavefronts each):
//          dkv    per (group, layer x KV head, run of eight 32-key committed
//                 tiles), one tile per wavefront: the tile's K and V stay in
//                 registers while the group's sequences stream by, each
//                 sequence's operands staged once per workgroup in LDS;
//                 S = Q K^T is formed with its query rows permuted (bits 2
//                 and 3 swapped) so that P and dS come out of the
//                 accumulators already in the operand layout of dV^T = dO^T P
//                 and dK^T = (R q)^T dS;
//          dq     per sixteen sequences of a group (two per wavefront) and
//                 layer x KV head: each committed tile of the group's page row
//                 staged once per workgroup in LDS; S^T = K Q^T (keys
//                 permuted the same way), dQ^T += K^T dS^T, then each
//                 sequence's carry tiles, and the rotation is undone;
//          both kinds of work shrink from the first keys of a response (seen
//          by all its blocks) to the last; in one grid the dq workgroups fill
//          the compute units the short dkv runs leave;
//   carry  carry keys belong to one sequence: their tiles take the dkv step
//          against that sequence alone.
// Keys masked in the forward (past ctx_len or carry_len, rejected page ids)
// get no gradient and contribute none.
#include <algorithm>

#include "co_kernels.h"

namespace co {

namespace {

constexpr float kLog2eB = 1.4426950408889634f;
constexpr float kLn2B = 0.6931471805599453f;
constexpr int kNqp = 32;   // query rows per (sequence, KV head): one 32-row MFMA tile
constexpr int kDkvTiles = 1;   // committed key tiles per dkv wavefront
constexpr int kDkvWaves = 8;   // wavefronts per dkv workgroup (consecutive tiles)
constexpr int kDqSeqs = 2;     // sequences per dq wavefront when groups share page rows
// One dkv ring slot (head_dim 64): the packed rotated queries and dO [32][64],
// their transposes [64][32], then -LSE (log2) and -D [32], bytes.
constexpr int kSlotQr = 0, kSlotDon = 4096, kSlotQrt = 8192, kSlotDot = 12288, kSlotL2 = 16384,
              kSlotDd = 16512, kSlotBytes = 16640;
// One dq ring slot: a committed tile's K rows and key-major V rows [32][64] and
// its K^T rows [64][32], bytes.
constexpr int kDqSlotK = 0, kDqSlotV = 4096, kDqSlotKt = 8192, kDqSlotBytes = 12288;
// Ring slots: a step's operands are staged two steps ahead.  (Deeper rings
// measured slower: the loops are bound by the LDS reads, not by the loads.)
constexpr int kDkvStages = 3, kDqStages = 3;
constexpr int kBwdSmem = kDkvStages * kSlotBytes > kDqStages * kDqSlotBytes
                             ? kDkvStages * kSlotBytes : kDqStages * kDqSlotBytes;
static_assert(kBwdSmem <= 160 * 1024, "one workgroup's LDS");
// XOR keys of the 16-byte chunks of a slot row.  LDS has 64 banks of 4 bytes:
// a 16-byte read serves sixteen lanes per pass, and the keys give those
// sixteen lanes sixteen different 16-byte bank groups.  Packed rows (128
// bytes, two per bank window) are read as rows perm23(l % 32), which for
// lanes 16i .. 16i + 15 are sixteen consecutive rows: bit 0 picks the half of
// the window, bits 1-3 the chunk key.  Transposed rows (64 bytes, four per
// window) are read as sixteen consecutive rows: bits 0-1 pick the quarter,
// bits 2-3 the chunk key.
__device__ __forceinline__ int swz_packed(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int swz_trans(int row) { return (row >> 2) & 3; }

// query (or key) index held by A-row / C-row rho when rows are permuted by
// swapping bits 2 and 3: then accumulator register r of lane l belongs to index
// 8 * (l / 32) + r for r < 8 and 16 + 8 * (l / 32) + r - 8 for r >= 8
__device__ __forceinline__ int perm23(int rho) {
  return (rho & ~12) | ((rho & 4) << 1) | ((rho & 8) >> 1);
}

// index of accumulator register r (permuted rows) for half h = lane / 32
__device__ __forceinline__ int acc_index(int r, int h) { return (r < 8 ? 0 : 16) + 8 * h + (r & 7); }

// Workspace pieces (bytes are 256-aligned by the host plan).
struct BwdWs {
  uint16_t *qr, *qrt, *don, *dot;   // [seg][S][32][hd] / [seg][S][hd][32]
  float *nlse2, *ndd;               // -LSE (log2 units), -D: [seg][S][32]
  uint16_t *kt, *vn;                // committed pages: [lc][num_pages][Hkv][hd][16] / [16][hd]
  uint16_t *ktc, *vnc;              // carry pages:     [lc][S][CP][Hkv][hd][16] / [16][hd]
};

__device__ __forceinline__ BwdWs bwd_ws(const BwdArgs& b) {
  const AttnArgs& a = b.a;
  const int64_t nseg = static_cast<int64_t>(b.layer_count) * a.Hkv;
  const int64_t qsz = nseg * a.S * kNqp * a.hd;
  const int64_t vsz = nseg * a.S * kNqp;
  const int64_t cpg = static_cast<int64_t>(b.layer_count) * a.num_pages * a.Hkv * kPage * a.hd;
  const int64_t cpc = static_cast<int64_t>(b.layer_count) * a.S * a.CP * a.Hkv * kPage * a.hd;
  auto up = [](int64_t bytes) { return (bytes + 255) / 256 * 256; };
  char* p = static_cast<char*>(static_cast<void*>(a.ws));
  BwdWs w;
  w.qr = reinterpret_cast<uint16_t*>(p); p += up(qsz * 2);
  w.qrt = reinterpret_cast<uint16_t*>(p); p += up(qsz * 2);
  w.don = reinterpret_cast<uint16_t*>(p); p += up(qsz * 2);
  w.dot = reinterpret_cast<uint16_t*>(p); p += up(qsz * 2);
  w.nlse2 = reinterpret_cast<float*>(p); p += up(vsz * 4);
  w.ndd = reinterpret_cast<float*>(p); p += up(vsz * 4);
  w.kt = reinterpret_cast<uint16_t*>(p); p += up(cpg * 2);
  w.vn = reinterpret_cast<uint16_t*>(p); p += up(cpg * 2);
  w.ktc = reinterpret_cast<uint16_t*>(p); p += up(cpc * 2);
  w.vnc = reinterpret_cast<uint16_t*>(p);
  return w;
}

__device__ __forceinline__ int64_t out_row_b(const AttnArgs& a, int layer_local, int s, int g,
                                             int n, int G) {
  const int i = n / G, hh = n % G;
  return ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq + g * G + hh;
}

// ------------------------------------------------------------------ prep
//
// grid (S, layer_count * Hkv), 256 threads: thread t takes query row t / 8 and
// the four rotation pairs (4p + e, 4p + e + hd/2), e < 4, p = t % 8 (hd 64).
template <int HD>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdArgs b) {
  static_assert(HD == 64, "pairs per thread");
  const AttnArgs& a = b.a;
  const BwdWs w = bwd_ws(b);
  const int s = blockIdx.x, seg = blockIdx.y;
  const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  const int t = threadIdx.x, qn = t >> 3, p = t & 7;
  const int64_t base = (static_cast<int64_t>(seg) * a.S + s) * kNqp;
  const int ctx = a.ctx_len[s];
  const bool live = qn < nq;
  const int64_t row = live ? out_row_b(a, layer_local, s, g, qn, G) * HD : 0;
  const uint16_t* Q = static_cast<const uint16_t*>(a.q);
  const uint16_t* O = static_cast<const uint16_t*>(b.out);
  const uint16_t* dO = static_cast<const uint16_t*>(b.d_out);
  const bool rotate = !(a.flags & CO_Q_PREROTATED);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2eB;
  float dsum = 0.f;
  u16x4 qlo, qhi, dlo, dhi;
  // the row's four pairs: 8-byte loads of each half
  const u16x4 z4 = {0, 0, 0, 0};
  const u16x4 xq = live ? *reinterpret_cast<const u16x4*>(Q + row + 4 * p) : z4;
  const u16x4 yq = live ? *reinterpret_cast<const u16x4*>(Q + row + 4 * p + HD / 2) : z4;
  const u16x4 xd = live ? *reinterpret_cast<const u16x4*>(dO + row + 4 * p) : z4;
  const u16x4 yd = live ? *reinterpret_cast<const u16x4*>(dO + row + 4 * p + HD / 2) : z4;
  const u16x4 xo = live ? *reinterpret_cast<const u16x4*>(O + row + 4 * p) : z4;
  const u16x4 yo = live ? *reinterpret_cast<const u16x4*>(O + row + 4 * p + HD / 2) : z4;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int i = 4 * p + e;
    float x = bf2f(xq[e]), y = bf2f(yq[e]);
    const float dx = bf2f(xd[e]), dy = bf2f(yd[e]);
    dsum = fmaf(dx, bf2f(xo[e]), fmaf(dy, bf2f(yo[e]), dsum));
    if (live && rotate) {
      float c, sn;
      rope_cos_sin_rev(ctx + qn / G, a.rope_inv[i] * kInv2Pi, &c, &sn);
      const float x2 = x * c - y * sn, y2 = y * c + x * sn;
      x = x2;
      y = y2;
    }
    qlo[e] = f2bf(x * qscale);
    qhi[e] = f2bf(y * qscale);
    dlo[e] = f2bf(dx);
    dhi[e] = f2bf(dy);
  }
  const int64_t qo = (base + qn) * HD;
  *reinterpret_cast<u16x4*>(w.qr + qo + 4 * p) = qlo;
  *reinterpret_cast<u16x4*>(w.qr + qo + 4 * p + HD / 2) = qhi;
  *reinterpret_cast<u16x4*>(w.don + qo + 4 * p) = dlo;
  *reinterpret_cast<u16x4*>(w.don + qo + 4 * p + HD / 2) = dhi;
  // the transposed copies ([hd][32] of this (seg, s)) go through LDS and leave
  // as one 16-byte store per thread each
  __shared__ __align__(16) uint16_t tq[HD][kNqp], td[HD][kNqp];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int i = 4 * p + e;
    tq[i][qn] = qlo[e];
    tq[i + HD / 2][qn] = qhi[e];
    td[i][qn] = dlo[e];
    td[i + HD / 2][qn] = dhi[e];
  }
  __syncthreads();
  {
    const int64_t to = base * HD;
    const int i = t >> 2, c = (t & 3) * 8;   // 256 threads x 8 elements = [64][32]
    *reinterpret_cast<u16x8*>(w.qrt + to + i * kNqp + c) = *reinterpret_cast<const u16x8*>(&tq[i][c]);
    *reinterpret_cast<u16x8*>(w.dot + to + i * kNqp + c) = *reinterpret_cast<const u16x8*>(&td[i][c]);
  }
  dsum += __shfl_xor(dsum, 1);
  dsum += __shfl_xor(dsum, 2);
  dsum += __shfl_xor(dsum, 4);
  if (p == 0) {
    // stored negated: the products below start their accumulators from them
    float l2 = INFINITY;   // padding rows: no weight anywhere
    if (live) {
      const float l = b.lse[out_row_b(a, layer_local, s, g, qn, G)];
      l2 = l * kLog2eB;    // -inf (no keys) stays -inf: such rows see no key either
    }
    w.nlse2[base + qn] = -l2;
    w.ndd[base + qn] = live ? -dsum : 0.f;
  }
}

// ------------------------------------------------------------------ copy
//
// Every K page of the launch's layers transposed to [hd][16] and every V page
// turned to [16][hd]; committed pages first, then carry pages.  One thread per
// 8 elements of a destination page.
template <int HD>
__global__ __launch_bounds__(256) void bwd_copy_kernel(BwdArgs b) {
  const AttnArgs& a = b.a;
  const BwdWs w = bwd_ws(b);
  constexpr int PE = kPage * HD;   // elements per page
  const int64_t n_com = static_cast<int64_t>(b.layer_count) * a.num_pages * a.Hkv;
  const int64_t n_car = static_cast<int64_t>(b.layer_count) * a.S * a.CP * a.Hkv;
  const int64_t item = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t pg = item / (PE / 8);
  const int c = static_cast<int>(item % (PE / 8)) * 8;
  if (pg >= n_com + n_car) return;
  const uint16_t *ks, *vs;
  uint16_t *kd, *vd;
  if (pg < n_com) {
    const int64_t lp = pg / (static_cast<int64_t>(a.num_pages) * a.Hkv);   // local layer
    const int64_t src = ((a.layer_begin + lp) * a.num_pages * a.Hkv + pg % (a.num_pages * a.Hkv)) * PE;
    ks = static_cast<const uint16_t*>(a.k_cache) + src;
    vs = static_cast<const uint16_t*>(a.v_cache) + src;
    kd = w.kt + pg * PE;
    vd = w.vn + pg * PE;
  } else {
    const int64_t pc = pg - n_com;
    const int64_t per = static_cast<int64_t>(a.S) * a.CP * a.Hkv;
    const int64_t src = ((a.layer_begin + pc / per) * per + pc % per) * PE;
    ks = static_cast<const uint16_t*>(a.k_carry) + src;
    vs = static_cast<const uint16_t*>(a.v_carry) + src;
    kd = w.ktc + pc * PE;
    vd = w.vnc + pc * PE;
  }
  // destination element c .. c+7: KT [dim][slot] = K [slot][dim]; VN [slot][dim] = V [dim][slot]
  u16x8 kv, vv;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int dim = (c + e) / kPage, slot = (c + e) % kPage;
    kv[e] = ks[slot * HD + dim];
    const int s2 = (c + e) / HD, d2 = (c + e) % HD;
    vv[e] = vs[d2 * kPage + s2];
  }
  *reinterpret_cast<u16x8*>(kd + c) = kv;
  *reinterpret_cast<u16x8*>(vd + c) = vv;
}

// ---------------------------------------------------- key-tile gradients
//
// One 32-key tile (two pages) against the 32 query rows of one sequence, keys
// in natural order as MFMA columns, query rows permuted.  kb/vb: the tile's
// K / V B-fragments (lane: key l % 32, dims 8 (l / 32) + 16 ks ..); valid
// keys: n0 in page 0, n1 in page 1.  Adds dV^T and (unscaled) dK^T.  NT tiles
// share each sequence's operands (more products per byte loaded).
template <int HD, int NT = 1>
struct KeyGrad {
  static constexpr int KS = HD / 16;   // k-steps over head dims
  static constexpr int MT = HD / 32;   // 32-row tiles of head dims
  f32x16 dkt[NT][MT], dvt[NT][MT];

  __device__ void zero() {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) dkt[t][m][r] = dvt[t][m][r] = 0.f;
  }

  // One sequence's operands of the step: its query rows (permuted) and dO
  // as A-fragments, their transposes, and -LSE / -D of the 16 query rows
  // this lane's accumulator registers hold (in accumulator order, so that
  // S - LSE and dP - D come out of the products with no further step).
  struct Block {
    u16x8 qa[KS], da[KS], qt[MT][2], dt[MT][2];
    f32x16 nl2, ndd;
    int n0[NT], n1[NT];   // valid keys of each tile's two pages for this sequence

    __device__ void load(const BwdWs& w, int64_t qbase, int lane) {
      const int r32 = lane & 31, h = lane >> 5;
      const int qp = perm23(r32);
      const uint16_t* qr = w.qr + (qbase + qp) * HD + 8 * h;
      const uint16_t* dn = w.don + (qbase + qp) * HD + 8 * h;
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        qa[k] = *reinterpret_cast<const u16x8*>(qr + 16 * k);
        da[k] = *reinterpret_cast<const u16x8*>(dn + 16 * k);
      }
      // transposed operands: lane dim = 32 m + l % 32, rows 16 j + 8 h ..
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int64_t off = qbase * HD + static_cast<int64_t>(32 * m + r32) * kNqp + 16 * j + 8 * h;
          qt[m][j] = *reinterpret_cast<const u16x8*>(w.qrt + off);
          dt[m][j] = *reinterpret_cast<const u16x8*>(w.dot + off);
        }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const f32x4 a0 = *reinterpret_cast<const f32x4*>(w.nlse2 + qbase + 16 * j + 8 * h);
        const f32x4 a1 = *reinterpret_cast<const f32x4*>(w.nlse2 + qbase + 16 * j + 8 * h + 4);
        const f32x4 b0 = *reinterpret_cast<const f32x4*>(w.ndd + qbase + 16 * j + 8 * h);
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(w.ndd + qbase + 16 * j + 8 * h + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          nl2[8 * j + e] = a0[e];
          nl2[8 * j + 4 + e] = a1[e];
          ndd[8 * j + e] = b0[e];
          ndd[8 * j + 4 + e] = b1[e];
        }
      }
    }
  };

  // The same operands from a staged copy in LDS (a dkv ring slot: rows with
  // their 16-byte chunks XOR-swizzled by swz_packed / swz_trans).
  __device__ static void load_lds(Block& q, const unsigned char* slot, int lane) {
    const int r32 = lane & 31, h = lane >> 5;
    const int qp = perm23(r32);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int o = (16 * j + 8 * h + 4 * c) * 4;
        const f32x4 a4 = *reinterpret_cast<const f32x4*>(slot + kSlotL2 + o);
        const f32x4 b4 = *reinterpret_cast<const f32x4*>(slot + kSlotDd + o);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          q.nl2[8 * j + 4 * c + e] = a4[e];
          q.ndd[8 * j + 4 * c + e] = b4[e];
        }
      }
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      const int off = qp * (2 * HD) + (((h + 2 * k) ^ swz_packed(qp)) << 4);
      q.qa[k] = *reinterpret_cast<const u16x8*>(slot + kSlotQr + off);
      q.da[k] = *reinterpret_cast<const u16x8*>(slot + kSlotDon + off);
    }
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = 32 * m + r32;
        const int off = row * (2 * kNqp) + (((2 * j + h) ^ swz_trans(row)) << 4);
        q.qt[m][j] = *reinterpret_cast<const u16x8*>(slot + kSlotQrt + off);
        q.dt[m][j] = *reinterpret_cast<const u16x8*>(slot + kSlotDot + off);
      }
  }

  __device__ void compute(const Block& q, const u16x8 (&kb)[NT][KS], const u16x8 (&vb)[NT][KS],
                          int lane) {
#pragma unroll
    for (int t = 0; t < NT; ++t) compute_tile(q, kb[t], vb[t], q.n0[t], q.n1[t], dkt[t], dvt[t], lane);
  }

  __device__ static void compute_tile(const Block& q, const u16x8 (&kb)[KS], const u16x8 (&vb)[KS],
                                      int n0, int n1, f32x16 (&dkt)[MT], f32x16 (&dvt)[MT],
                                      int lane) {
    const int r32 = lane & 31;
    // S - LSE and dP - D: the products start from -LSE and -D.  A key past
    // the sequence's length (this lane's column) starts from -inf instead, so
    // its P and dS are 0 (whatever its cache slot holds, it reaches only its
    // own column, which is not stored).
    f32x16 sc = q.nl2, dp = q.ndd;
    if (n0 < kPage || n1 < kPage) {
      const int key = r32;
      if (key < 16 ? key >= n0 : key - 16 >= n1) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] = -INFINITY;
      }
    }
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      sc = mfma32x32x16(q.qa[k], kb[k], sc);
      dp = mfma32x32x16(q.da[k], vb[k], dp);
    }
    u16x8 pb[2], sb[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float pv[8], sv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int r = 8 * j + e;
        const float pr = __builtin_amdgcn_exp2f(sc[r]);
        pv[e] = pr;
        sv[e] = pr * dp[r];
      }
      typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
      const u32x4v p4 = {cvt_pk_bf16(pv[0], pv[1]), cvt_pk_bf16(pv[2], pv[3]),
                         cvt_pk_bf16(pv[4], pv[5]), cvt_pk_bf16(pv[6], pv[7])};
      const u32x4v s4 = {cvt_pk_bf16(sv[0], sv[1]), cvt_pk_bf16(sv[2], sv[3]),
                         cvt_pk_bf16(sv[4], sv[5]), cvt_pk_bf16(sv[6], sv[7])};
      pb[j] = __builtin_bit_cast(u16x8, p4);
      sb[j] = __builtin_bit_cast(u16x8, s4);
    }
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        dvt[m] = mfma32x32x16(q.dt[m][j], pb[j], dvt[m]);
        dkt[m] = mfma32x32x16(q.qt[m][j], sb[j], dkt[m]);
      }
  }

  // dK (x ln 2: the queries were in log2 units) and dV of tile t's valid keys
  // into fp32 pages laid out like the caches: K [16][hd], V [hd][16].
  __device__ void store(int t, float* dk0, float* dk1, float* dv0, float* dv1, int n0, int n1,
                        int lane) const {
    const int key = lane & 31, h = lane >> 5;
    const bool p1 = key >= 16;
    const int slot = key & 15;
    if (slot >= (p1 ? n1 : n0)) return;
    float* dk = (p1 ? dk1 : dk0) + slot * HD;
    float* dv = (p1 ? dv1 : dv0) + slot;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int dim = 32 * m + 8 * (r >> 2) + 4 * h + (r & 3);
        dk[dim] = dkt[t][m][r] * kLn2B;
        dv[dim * kPage] = dvt[t][m][r];
      }
  }
};

// K / V B-fragments of a tile: lane key l % 32 (page l / 16 of the pair), dims
// 8 (l / 32) + 16 k; K from the cache layout [16][hd], V from the key-major copy.
template <int HD>
__device__ __forceinline__ void tile_frags(const uint16_t* k0, const uint16_t* k1,
                                           const uint16_t* v0, const uint16_t* v1, int lane,
                                           u16x8 (&kb)[HD / 16], u16x8 (&vb)[HD / 16]) {
  const int key = lane & 31, h = lane >> 5;
  const uint16_t* kr = (key < 16 ? k0 : k1) + (key & 15) * HD + 8 * h;
  const uint16_t* vr = (key < 16 ? v0 : v1) + (key & 15) * HD + 8 * h;
#pragma unroll
  for (int k = 0; k < HD / 16; ++k) {
    kb[k] = *reinterpret_cast<const u16x8*>(kr + 16 * k);
    vb[k] = *reinterpret_cast<const u16x8*>(vr + 16 * k);
  }
}

// Workgroups are dealt to the 8 XCDs round-robin.  Work items come in pairs
// (group, layer x KV head) whose items read the same data (the group's
// queries, or the keys of its page row); every pair is given to one XCD, its
// items on consecutive ids there, so that they share that XCD's L2.  Returns
// false for the padding ids of the launch (8 * ceil(n_pairs / 8) * per ids).
__device__ __forceinline__ bool xcd_item(int n_pairs, int per, int* pair, int* item) {
  const int i = blockIdx.x, xcd = i & 7, k = i >> 3;
  *pair = xcd + 8 * (k / per);
  *item = k % per;
  return *pair < n_pairs;
}

__device__ __forceinline__ bool len_ok(const AttnArgs& a, int ctx, int carry) {
  return ctx >= 0 && ctx <= a.max_pages * kPage && carry >= 0 && carry <= a.CP * kPage;
}

// ------------------------------------------------------------------- dkv
//
// One workgroup of kDkvWaves wavefronts per (group, layer x KV head, run of
// kDkvWaves consecutive committed key tiles), one tile per wavefront: the
// tile's K and V stay in registers while the group's sequences stream by.
// Each sequence's operands (16.3 KiB) are staged once per workgroup into an
// LDS ring slot by direct-to-LDS loads, two sequences ahead, and every
// wavefront reads its fragments from there.  The group's first sequence holds
// the page row; tiles no sequence of the group reaches are skipped.
template <int HD>
__device__ __forceinline__ void dkv_role(const BwdArgs& b, int pair, int unit, unsigned char* ring) {
  static_assert(HD == 64, "ring slot layout");
  static_assert(16 % kDkvWaves == 0, "the sixteen 1 KiB pieces of a slot split evenly");
  constexpr int NT = kDkvTiles, KS = HD / 16;
  const AttnArgs& a = b.a;
  const BwdWs w = bwd_ws(b);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int groups = (a.S + b.group - 1) / b.group;
  const int grp = pair % groups, seg = pair / groups;
  const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
  const int s0 = grp * b.group, s1 = min(a.S, s0 + b.group);
  const int kb0 = 32 * NT * kDkvWaves * unit;   // the workgroup's first key
  const int kbase = kb0 + 32 * NT * wave;       // this wavefront's first key
  int reach = 0;   // committed keys the group's sequences see
  for (int s = s0; s < s1; ++s) {
    const int ctx = a.ctx_len[s], carry = a.carry_len[s];
    if (len_ok(a, ctx, carry)) reach = max(reach, ctx);
  }
  if (kb0 >= reach) return;   // the whole workgroup, before any barrier
  const int32_t* pt = a.page_table + static_cast<int64_t>(s0) * a.max_pages;
  const int64_t pe = static_cast<int64_t>(kPage) * HD;
  const int64_t lay = static_cast<int64_t>(a.layer_begin + layer_local) * a.num_pages;
  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  // pages of this wavefront's tiles; pages no sequence reaches are not read
  int id[NT][2];
  bool bad[NT][2];
  u16x8 kb[NT][KS], vb[NT][KS];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int pg = kbase / kPage + 2 * t + p;
      const bool has = kbase + (2 * t + p) * kPage < reach;
      const int x = has ? pt[pg] : 0;
      bad[t][p] = has && (x < 0 || x >= a.num_pages);
      if (bad[t][p] && lane == 0) set_status(a.status, CO_ERR_PAGE_RANGE);
      id[t][p] = (has && !bad[t][p]) ? x : 0;
    }
    const int64_t c0 = ((lay + id[t][0]) * a.Hkv + g) * pe, c1 = ((lay + id[t][1]) * a.Hkv + g) * pe;
    const int64_t w0 = ((static_cast<int64_t>(layer_local) * a.num_pages + id[t][0]) * a.Hkv + g) * pe;
    const int64_t w1 = ((static_cast<int64_t>(layer_local) * a.num_pages + id[t][1]) * a.Hkv + g) * pe;
    tile_frags<HD>(kc + c0, kc + c1, w.vn + w0, w.vn + w1, lane, kb[t], vb[t]);
  }
  // valid keys of page p of tile t for a sequence (or the group) reaching n keys
  auto valid_keys = [&](int t, int p, int n) {
    return bad[t][p] ? 0 : max(0, min(kPage, n - kbase - (2 * t + p) * kPage));
  };
  KeyGrad<HD, NT> kg;
  kg.zero();
  // The group's sequences that see the workgroup's first key, walked from the
  // last one down (it sees the most keys, so every workgroup of the group
  // starts on the same sequence and the XCD's workgroups stage the same
  // operands at about the same time), 64 at a time as a lane mask.  Every
  // wavefront walks the same list, so all take the same barriers.
  const int none = s0 - 1;
  uint64_t mask = 0;
  int mbase = s1, mctx = 0;
  auto prev = [&](int x) {   // last sequence <= x that sees the workgroup, or none
    for (;;) {
      if (x < s0) return none;
      if (x < mbase) {
        const int top = x;
        mbase = max(s0, x - 63);
        const int y = mbase + lane;
        bool v = false;
        mctx = 0;
        if (y <= top) {
          const int ctx = a.ctx_len[y], carry = a.carry_len[y];
          v = len_ok(a, ctx, carry) && ctx > kb0;
          mctx = ctx;
        }
        mask = __ballot(v);
      }
      const int off = x - mbase;
      const uint64_t m = mask & (off == 63 ? ~0ull : ((1ull << (off + 1)) - 1));
      if (m) return mbase + 63 - static_cast<int>(__builtin_clzll(m));
      x = mbase - 1;
    }
  };
  // A sequence's operands into ring slot `slot` by direct-to-LDS loads: each
  // wavefront moves its 1 KiB pieces of the packed arrays (16-byte chunks of
  // a row XOR-swizzled by the row); wavefront 0 also moves -LSE and -D (16 lanes).
  auto stage_block = [&](int s, int slot) {
    const uint32_t base = lds_addr(ring) + slot * kSlotBytes;
    const int64_t qbase = (static_cast<int64_t>(seg) * a.S + s) * kNqp;
    // pieces P wave .. P wave + P - 1 (P = 16 / kDkvWaves): pieces 0-7 are the
    // packed arrays (rows of 128 bytes), 8-15 their transposes (rows of 64 bytes)
    constexpr int P = 16 / kDkvWaves;
#pragma unroll
    for (int x = 0; x < P; ++x) {
      const int piece = P * wave + x, arr = piece >> 2;
      const int off = (piece & 3) * 1024 + 16 * lane;
      const uint32_t dst = base + arr * 4096 + (piece & 3) * 1024;
      if (arr < 2) {
        const int row = off / (2 * HD), lg = ((off % (2 * HD)) >> 4) ^ swz_packed(row);
        lds_dma16_opaque((arr == 0 ? w.qr : w.don) + (qbase + row) * HD + lg * 8, dst);
      } else {
        const int row = off / (2 * kNqp), lg = ((off % (2 * kNqp)) >> 4) ^ swz_trans(row);
        lds_dma16_opaque((arr == 2 ? w.qrt : w.dot) + qbase * HD + row * kNqp + lg * 8, dst);
      }
    }
    if (wave == 0 && lane < 16) {
      const float* src = lane < 8 ? w.nlse2 + qbase + 4 * lane : w.ndd + qbase + 4 * (lane - 8);
      lds_dma16_opaque(src, base + kSlotL2);
    }
  };
  static_assert(kDkvStages == 3, "two sequences ahead");
  constexpr int P = 16 / kDkvWaves;   // loads per staged sequence; wavefront 0 has one more
  using Blk = typename KeyGrad<HD, NT>::Block;
  // the sequence in use, the next two, and their lengths (read from the walk's
  // window right after each step of it)
  int s = prev(s1 - 1);
  int sctx = s != none ? __builtin_amdgcn_readlane(mctx, s - mbase) : 0;
  int sn = s != none ? prev(s - 1) : none;
  int snctx = sn != none ? __builtin_amdgcn_readlane(mctx, sn - mbase) : 0;
  if (s != none) stage_block(s, 0);
  if (sn != none) stage_block(sn, 1);
  for (int slot = 0; s != none; slot = slot == kDkvStages - 1 ? 0 : slot + 1) {
    const int snn = sn != none ? prev(sn - 1) : none;
    const int snnctx = snn != none ? __builtin_amdgcn_readlane(mctx, snn - mbase) : 0;
    // this slot's loads are complete once at most the next sequence's remain
    // in flight (loads complete in order); then the barrier publishes them
    if (sn == none) wait_vm_lgkm_barrier<0>();
    else if (wave == 0) wait_vm_lgkm_barrier<P + 1>();
    else wait_vm_lgkm_barrier<P>();
    // every wavefront is past its reads of the slot staged two sequences ago
    if (snn != none) stage_block(snn, slot == 0 ? kDkvStages - 1 : slot - 1);
    Blk q;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      q.n0[t] = valid_keys(t, 0, sctx);
      q.n1[t] = valid_keys(t, 1, sctx);
    }
    if (q.n0[0] + q.n1[0] > 0) {   // the sequence reaches this wavefront's tile
      KeyGrad<HD, NT>::load_lds(q, ring + slot * kSlotBytes, lane);
      kg.compute(q, kb, vb, lane);
    }
    s = sn;
    sctx = snctx;
    sn = snn;
    snctx = snnctx;
  }
  // every key that some sequence of the group sees (keys past `reach` keep no gradient)
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int64_t o0 = ((lay + id[t][0]) * a.Hkv + g) * pe, o1 = ((lay + id[t][1]) * a.Hkv + g) * pe;
    kg.store(t, b.d_k_cache + o0, b.d_k_cache + o1, b.d_v_cache + o0, b.d_v_cache + o1,
             valid_keys(t, 0, reach), valid_keys(t, 1, reach), lane);
  }
}

// ----------------------------------------------------------- dkv, carry
//
// grid (S, layer_count * Hkv), one wavefront: the carry keys belong to one
// sequence, so their tiles take the dkv step against that sequence alone.
template <int HD>
__global__ __launch_bounds__(64, 2) void bwd_dkv_carry_kernel(BwdArgs b) {
  const AttnArgs& a = b.a;
  const BwdWs w = bwd_ws(b);
  const int lane = threadIdx.x;
  const int s = blockIdx.x, seg = blockIdx.y;
  const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
  const int ctx = a.ctx_len[s], carry = a.carry_len[s];
  if (!len_ok(a, ctx, carry) || carry == 0) return;
  const int64_t pe = static_cast<int64_t>(kPage) * HD;
  const int64_t lay = static_cast<int64_t>(a.layer_begin + layer_local);
  const int ncp = (carry + kPage - 1) / kPage;
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);
  const int64_t qbase = (static_cast<int64_t>(seg) * a.S + s) * kNqp;
  for (int cp0 = 0; cp0 < ncp; cp0 += 2) {
    const int cp1 = min(cp0 + 1, ncp - 1);
    const int n0 = min(kPage, carry - cp0 * kPage);
    const int n1 = cp0 + 1 < ncp ? min(kPage, carry - (cp0 + 1) * kPage) : 0;
    const int64_t r0 = ((lay * a.S + s) * a.CP + cp0) * a.Hkv + g;
    const int64_t r1 = ((lay * a.S + s) * a.CP + cp1) * a.Hkv + g;
    const int64_t q0 = ((static_cast<int64_t>(layer_local) * a.S + s) * a.CP + cp0) * a.Hkv + g;
    const int64_t q1 = ((static_cast<int64_t>(layer_local) * a.S + s) * a.CP + cp1) * a.Hkv + g;
    u16x8 kb[1][HD / 16], vb[1][HD / 16];
    tile_frags<HD>(kk + r0 * pe, kk + r1 * pe, w.vnc + q0 * pe, w.vnc + q1 * pe, lane, kb[0], vb[0]);
    KeyGrad<HD, 1> kg;
    kg.zero();
    typename KeyGrad<HD, 1>::Block q;
    q.load(w, qbase, lane);
    q.n0[0] = n0;
    q.n1[0] = n1;
    kg.compute(q, kb, vb, lane);
    kg.store(0, b.d_k_carry + r0 * pe, b.d_k_carry + r1 * pe, b.d_v_carry + r0 * pe,
             b.d_v_carry + r1 * pe, n0, n1, lane);
  }
}

// -------------------------------------------------------------------- dq
//
// One wavefront per NQ consecutive sequences of a group and layer x KV head:
// the committed tiles of the page row, then each sequence's carry tiles.
// Keys are the MFMA rows here (permuted), query rows the columns: lane l keeps
// query l % 32 of every sequence throughout.
//
// NQ = 2 (groups that share page rows): the workgroup's kDkvWaves wavefronts
// take 2 kDkvWaves consecutive sequences of one group, and every committed
// tile (K rows, the key-major V copy, the K^T copy: 12 KiB) is staged once
// per workgroup into an LDS ring slot by direct-to-LDS loads, two tiles ahead,
// for all of them.  NQ = 1 (one sequence per group): the wavefront loads its
// own tiles.
template <int HD, int NQ>
__device__ __forceinline__ void dq_role(const BwdArgs& b, int pair, int item, unsigned char* ring) {
  constexpr int KS = HD / 16, MT = HD / 32;
  constexpr bool kStaged = NQ > 1;
  static_assert(!kStaged || HD == 64, "ring slot layout");
  const AttnArgs& a = b.a;
  const BwdWs w = bwd_ws(b);
  const int lane = threadIdx.x & 63, r32 = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int groups = (a.S + b.group - 1) / b.group;
  const int grp = pair % groups, seg = pair / groups;
  const int gbeg = grp * b.group, gend = min(a.S, gbeg + b.group);
  const int sfirst = gbeg + NQ * item;   // item < 0: a staging-only wavefront
  if (!kStaged && sfirst >= gend) return;
  const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  const int64_t pe = static_cast<int64_t>(kPage) * HD;
  const int64_t lay = static_cast<int64_t>(a.layer_begin + layer_local);
  const int32_t* lead = a.page_table + static_cast<int64_t>(gbeg) * a.max_pages;
  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);

  // per sequence: lengths, this lane's query column (B-fragments of the
  // rotated queries and of dO), its LSE and D, and the dQ^T accumulators
  bool live[NQ];
  int ctx[NQ], carry[NQ], npc[NQ];
  u16x8 qb[NQ][KS], db[NQ][KS];
  float l2[NQ], dd[NQ];
  f32x16 dqt[NQ][MT];
  int npc_max = 0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int s = sfirst + q;
    live[q] = item >= 0 && s < gend;
    const int sc = live[q] ? s : gbeg;
    const int cr = a.ctx_len[sc], ur = a.carry_len[sc];
    const bool ok = live[q] && len_ok(a, cr, ur);
    if (live[q] && !ok && seg == 0 && lane == 0) set_status(a.status, CO_ERR_LENGTH);
    ctx[q] = ok ? cr : 0;
    carry[q] = ok ? ur : 0;
    npc[q] = (ctx[q] + kPage - 1) / kPage;
    npc_max = max(npc_max, npc[q]);
    const int64_t qbase = (static_cast<int64_t>(seg) * a.S + sc) * kNqp;
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      qb[q][k] = *reinterpret_cast<const u16x8*>(w.qr + (qbase + r32) * HD + 16 * k + 8 * h);
      db[q][k] = *reinterpret_cast<const u16x8*>(w.don + (qbase + r32) * HD + 16 * k + 8 * h);
    }
    l2[q] = -w.nlse2[qbase + r32];
    dd[q] = -w.ndd[qbase + r32];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) dqt[q][m][r] = 0.f;
    // a group's sequences read the group's page row: every page this sequence
    // sees must be the lead's (checked once, lane-parallel)
    if (b.group > 1 && live[q]) {
      const int32_t* own = a.page_table + static_cast<int64_t>(s) * a.max_pages;
      bool diff = false;
      for (int p = lane; p < npc[q]; p += 64) diff = diff || own[p] != lead[p];
      if (__ballot(diff) && lane == 0) set_status(a.status, CO_ERR_GROUP);
    }
  }

  const int kp = perm23(r32);   // the key this lane's A rows hold
  // One tile given its fragments: S^T and dP^T with the keys permuted (A rows
  // from K and the key-major V copy), then dQ^T += K^T dS^T for every
  // sequence q with keys in it.
  auto tile_math = [&](const u16x8 (&ka)[KS], const u16x8 (&va)[KS], const u16x8 (&kt)[MT][2],
                       const int (&n0)[NQ], const int (&n1)[NQ]) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      if (n0[q] + n1[q] == 0) continue;
      f32x16 sc, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[r] = dp[r] = 0.f;
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        sc = mfma32x32x16(ka[k], qb[q][k], sc);
        dp = mfma32x32x16(va[k], db[q][k], dp);
      }
      // dS = P (dP - D); keys past the length (rows here) give 0, whatever
      // their cache slots hold.  Most tiles are whole: no per-key test there.
      float sv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) sv[r] = __builtin_amdgcn_exp2f(sc[r] - l2[q]) * (dp[r] - dd[q]);
      if (n0[q] < kPage || n1[q] < kPage) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = acc_index(r, h);
          if (key < 16 ? key >= n0[q] : key - 16 >= n1[q]) sv[r] = 0.f;
        }
      }
      u16x8 sb[2];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
        const float* v = sv + 8 * jj;
        const u32x4v s4 = {cvt_pk_bf16(v[0], v[1]), cvt_pk_bf16(v[2], v[3]),
                           cvt_pk_bf16(v[4], v[5]), cvt_pk_bf16(v[6], v[7])};
        sb[jj] = __builtin_bit_cast(u16x8, s4);
      }
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) dqt[q][m] = mfma32x32x16(kt[m][jj], sb[jj], dqt[q][m]);
    }
  };
  // one tile from global memory (pages of K, the key-major V copy, the K^T copy)
  auto tile = [&](const uint16_t* k0, const uint16_t* k1, const uint16_t* v0, const uint16_t* v1,
                  const uint16_t* t0, const uint16_t* t1, const int (&n0)[NQ],
                  const int (&n1)[NQ]) {
    const uint16_t* kr = (kp < 16 ? k0 : k1) + (kp & 15) * HD + 8 * h;
    const uint16_t* vr = (kp < 16 ? v0 : v1) + (kp & 15) * HD + 8 * h;
    u16x8 ka[KS], va[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      ka[k] = *reinterpret_cast<const u16x8*>(kr + 16 * k);
      va[k] = *reinterpret_cast<const u16x8*>(vr + 16 * k);
    }
    // K^T A-fragments: lane dim 32 m + l % 32, keys 16 jj + 8 h .. (page jj)
    u16x8 kt[MT][2];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
        kt[m][jj] = *reinterpret_cast<const u16x8*>((jj ? t1 : t0) + (32 * m + r32) * kPage + 8 * h);
    tile_math(ka, va, kt, n0, n1);
  };
  // valid keys of the committed tile j's two pages for sequence q
  auto tile_keys = [&](int j, bool b0, bool b1, int (&n0)[NQ], int (&n1)[NQ]) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      n0[q] = (b0 || 2 * j >= npc[q]) ? 0 : min(kPage, ctx[q] - 2 * j * kPage);
      n1[q] = (b1 || 2 * j + 1 >= npc[q]) ? 0 : min(kPage, ctx[q] - (2 * j + 1) * kPage);
    }
  };

  if constexpr (kStaged) {
    // the workgroup's committed tiles: up to the longest of its sequences
    // (lanes 0-15 take the 16 sequences of the 8 wavefronts; every wavefront
    // computes the same count, so all take the same barriers)
    int wnpc = 0;
    {
      const int wq = lane / NQ, qq = lane % NQ;
      const int it = item + wave - wq;   // the item of wavefront wq (items run down with wave)
      const int s = gbeg + NQ * it + qq;
      if (lane < NQ * kDkvWaves && it >= 0 && s < gend) {
        const int cr = a.ctx_len[s], ur = a.carry_len[s];
        if (len_ok(a, cr, ur)) wnpc = (cr + kPage - 1) / kPage;
      }
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) wnpc = max(wnpc, __shfl_xor(wnpc, o));
      wnpc = __builtin_amdgcn_readfirstlane(wnpc);
    }
    const int nct = (wnpc + 1) / 2;
    // page ids of the lead row, 64 at a time as a lane vector; one copy for
    // the staging (two tiles ahead) and one for the tiles in use
    struct Ids {
      int v = 0, c = -1;
    } ahead, cur;
    auto page_id = [&](Ids& ids, int p) {   // uniform p; loads 64 ids when p leaves them
      if ((p >> 6) != ids.c) {
        ids.c = p >> 6;
        const int x = 64 * ids.c + lane;
        ids.v = x < a.max_pages ? lead[x] : 0;
      }
      return __builtin_amdgcn_readlane(ids.v, p & 63);
    };
    // tile j into ring slot `slot`: twelve 1 KiB pieces (K rows, V rows, K^T
    // rows), pieces wave and wave + 8 of this wavefront
    auto stage_tile = [&](int j, int slot) {
      const int p0 = 2 * j, p1 = min(2 * j + 1, wnpc - 1);
      int id0 = page_id(ahead, p0), id1 = page_id(ahead, p1);
      id0 = (id0 < 0 || id0 >= a.num_pages) ? 0 : id0;   // reported where the tile is used
      id1 = (id1 < 0 || id1 >= a.num_pages) ? 0 : id1;
      const uint32_t base = lds_addr(ring) + slot * kDqSlotBytes;
      const uint16_t* kpg[2] = {kc + ((lay * a.num_pages + id0) * a.Hkv + g) * pe,
                                kc + ((lay * a.num_pages + id1) * a.Hkv + g) * pe};
      const int64_t w0 = ((static_cast<int64_t>(layer_local) * a.num_pages + id0) * a.Hkv + g) * pe;
      const int64_t w1 = ((static_cast<int64_t>(layer_local) * a.num_pages + id1) * a.Hkv + g) * pe;
#pragma unroll
      for (int x = 0; x < (12 + kDkvWaves - 1) / kDkvWaves; ++x) {
        const int piece = wave + kDkvWaves * x;
        if (piece >= 12) break;
        const int arr = piece >> 2, off = (piece & 3) * 1024 + 16 * lane;
        const uint32_t dst = base + arr * 4096 + (piece & 3) * 1024;
        if (arr < 2) {   // key rows [32][64]: row r is slot r % 16 of page r / 16
          const int r = off / (2 * HD), c = ((off % (2 * HD)) >> 4) ^ swz_packed(r);
          const uint16_t* src = arr == 0 ? kpg[r >> 4] : w.vn + (r >> 4 ? w1 : w0);
          lds_dma16_opaque(src + (r & 15) * HD + c * 8, dst);
        } else {         // K^T rows [64][32]: dims, the two pages' 16 keys side by side
          const int d = off / (2 * kNqp), c = ((off % (2 * kNqp)) >> 4) ^ swz_trans(d);
          lds_dma16_opaque(w.kt + (c >> 1 ? w1 : w0) + d * kPage + (c & 1) * 8, dst);
        }
      }
    };
    static_assert(kDqStages == 3 && kDkvWaves == 8, "two tiles ahead; 2 or 1 pieces per wavefront");
    const bool two = wave < 12 - kDkvWaves;   // this wavefront stages two pieces per tile
    if (nct > 0) stage_tile(0, 0);
    if (nct > 1) stage_tile(1, 1);
    for (int j = 0, slot = 0; j < nct; ++j, slot = slot == kDqStages - 1 ? 0 : slot + 1) {
      // tile j's pieces are in once at most tile j + 1's remain in flight
      // (loads complete in order); then the barrier publishes them
      if (j + 1 >= nct) wait_vm_lgkm_barrier<0>();
      else if (two) wait_vm_lgkm_barrier<2>();
      else wait_vm_lgkm_barrier<1>();
      // every wavefront is past its reads of the slot of tile j - 1
      if (j + 2 < nct) stage_tile(j + 2, slot == 0 ? kDqStages - 1 : slot - 1);
      const int p0 = 2 * j, p1 = min(2 * j + 1, wnpc - 1);
      const int id0 = page_id(cur, p0), id1 = page_id(cur, p1);
      const bool b0 = id0 < 0 || id0 >= a.num_pages, b1 = id1 < 0 || id1 >= a.num_pages;
      if ((b0 || b1) && wave == 0 && lane == 0) set_status(a.status, CO_ERR_PAGE_RANGE);
      int n0[NQ], n1[NQ];
      tile_keys(j, b0, b1, n0, n1);
      int any = 0;
#pragma unroll
      for (int q = 0; q < NQ; ++q) any += n0[q] + n1[q];
      if (any > 0) {
        const unsigned char* sl = ring + slot * kDqSlotBytes;
        u16x8 ka[KS], va[KS], kt[MT][2];
#pragma unroll
        for (int k = 0; k < KS; ++k) {
          const int off = kp * (2 * HD) + (((2 * k + h) ^ swz_packed(kp)) << 4);
          ka[k] = *reinterpret_cast<const u16x8*>(sl + kDqSlotK + off);
          va[k] = *reinterpret_cast<const u16x8*>(sl + kDqSlotV + off);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) {
            const int d = 32 * m + r32;
            const int off = d * (2 * kNqp) + (((2 * jj + h) ^ swz_trans(d)) << 4);
            kt[m][jj] = *reinterpret_cast<const u16x8*>(sl + kDqSlotKt + off);
          }
        tile_math(ka, va, kt, n0, n1);
      }
    }
    if (item < 0) return;   // after the last barrier
  } else {
    // committed tiles of the sequence's own page row (the group's row)
    const int32_t* pt = a.page_table + static_cast<int64_t>(sfirst) * a.max_pages;
    const int nct_max = (npc_max + 1) / 2;
    for (int j = 0; j < nct_max; ++j) {
      const int p0 = 2 * j, p1 = min(2 * j + 1, npc_max - 1);
      int id0 = pt[p0], id1 = pt[p1];
      const bool b0 = id0 < 0 || id0 >= a.num_pages, b1 = id1 < 0 || id1 >= a.num_pages;
      if ((b0 || b1) && lane == 0) set_status(a.status, CO_ERR_PAGE_RANGE);
      int n0[NQ], n1[NQ];
      tile_keys(j, b0, b1, n0, n1);
      id0 = b0 ? 0 : id0;
      id1 = b1 ? 0 : id1;
      const int64_t c0 = ((lay * a.num_pages + id0) * a.Hkv + g) * pe;
      const int64_t c1 = ((lay * a.num_pages + id1) * a.Hkv + g) * pe;
      const int64_t w0 = ((static_cast<int64_t>(layer_local) * a.num_pages + id0) * a.Hkv + g) * pe;
      const int64_t w1 = ((static_cast<int64_t>(layer_local) * a.num_pages + id1) * a.Hkv + g) * pe;
      tile(kc + c0, kc + c1, w.vn + w0, w.vn + w1, w.kt + w0, w.kt + w1, n0, n1);
    }
  }
  // each sequence's carry tiles, against that sequence alone
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (!live[q]) continue;
    const int s = sfirst + q;
    const int ncp = (carry[q] + kPage - 1) / kPage;
    for (int cp0 = 0; cp0 < ncp; cp0 += 2) {
      const int cp1 = min(cp0 + 1, ncp - 1);
      const int64_t r0 = ((lay * a.S + s) * a.CP + cp0) * a.Hkv + g;
      const int64_t r1 = ((lay * a.S + s) * a.CP + cp1) * a.Hkv + g;
      const int64_t q0 = ((static_cast<int64_t>(layer_local) * a.S + s) * a.CP + cp0) * a.Hkv + g;
      const int64_t q1 = ((static_cast<int64_t>(layer_local) * a.S + s) * a.CP + cp1) * a.Hkv + g;
      int n0[NQ], n1[NQ];
#pragma unroll
      for (int x = 0; x < NQ; ++x) n0[x] = n1[x] = 0;
      n0[q] = min(kPage, carry[q] - cp0 * kPage);
      n1[q] = cp0 + 1 < ncp ? min(kPage, carry[q] - (cp0 + 1) * kPage) : 0;
      tile(kk + r0 * pe, kk + r1 * pe, w.vnc + q0 * pe, w.vnc + q1 * pe, w.ktc + q0 * pe,
           w.ktc + q1 * pe, n0, n1);
    }
  }
  // dq = R^T (dS K) / sqrt(hd): dims i and i + hd/2 sit in the same register of tiles m and m + MT/2
  const int qn = r32;
  if (qn >= nq) return;
  const float scale = rsqrtf(static_cast<float>(HD));
  const bool rotate = !(a.flags & CO_Q_PREROTATED);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (!live[q]) continue;
    const int pos = ctx[q] + qn / G;
    float* dq = b.d_q + out_row_b(a, layer_local, sfirst + q, g, qn, G) * HD;
#pragma unroll
    for (int m = 0; m < MT / 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = 32 * m + 8 * (r >> 2) + 4 * h + (r & 3);
        float x = dqt[q][m][r] * scale, y = dqt[q][m + MT / 2][r] * scale;
        if (rotate) {
          float c, sn;
          rope_cos_sin_rev(pos, a.rope_inv[i] * kInv2Pi, &c, &sn);
          const float x2 = x * c + y * sn, y2 = y * c - x * sn;
          x = x2;
          y = y2;
        }
        dq[i] = x;
        dq[i + HD / 2] = y;
      }
  }
}

// ------------------------------------------------------------- dkv + dq
//
// One launch for both kinds of workgroup.  Both kinds of work shrink with
// their rank r within a pair: dkv run r holds keys that fewer of the group's
// sequences see, dq workgroup r holds shorter sequences (it takes items
// items - 1 - (8 r + wave)).  Workgroups are dealt out by rank, the longest
// first: round r holds dkv run r and dq workgroup r of every pair, so the
// chip starts the longest work of both kinds at once and fills in with
// shorter work as units free up.  Workgroup i runs on XCD i % 8, and the
// pairs p with p % 8 == that XCD are the ones it takes, so all of a pair's
// workgroups share one XCD's L2.  Groups of one sequence (no shared rows):
// all dkv runs first, then one dq wavefront per pair.
template <int HD, int NQ>
__global__ __launch_bounds__(64 * kDkvWaves, kDkvWaves / 4) void bwd_attn_kernel(BwdArgs b, int n_dkv) {
  __shared__ __align__(16) unsigned char smem[kBwdSmem];   // the role's LDS ring
  const AttnArgs& a = b.a;
  const int groups = (a.S + b.group - 1) / b.group;
  const int n_pairs = groups * b.layer_count * a.Hkv;
  const int units = ((a.max_pages + 1) / 2 + kDkvTiles * kDkvWaves - 1) / (kDkvTiles * kDkvWaves);
  const int i = blockIdx.x, xcd = i & 7, wave = threadIdx.x >> 6;
  if (b.group == 1) {
    if (i < n_dkv) {
      const int k = i >> 3, pair = xcd + 8 * (k / units);
      if (pair < n_pairs) dkv_role<HD>(b, pair, k % units, smem);
    } else {   // eight pairs per workgroup
      const int pair = kDkvWaves * (i - n_dkv) + wave;
      if (pair < n_pairs) dq_role<HD, NQ>(b, pair, 0, smem);
    }
    return;
  }
  const int items = (b.group + NQ - 1) / NQ;             // dq wavefronts per pair
  const int per = (items + kDkvWaves - 1) / kDkvWaves;   // dq workgroups per pair
  const int ppx = (n_pairs + 7) / 8;                     // pairs per XCD
  const int k = i >> 3, r = k / (2 * ppx), rem = k % (2 * ppx);
  const int pair = xcd + 8 * (rem % ppx);
  if (pair >= n_pairs) return;
  if (rem < ppx) {
    if (r < units) dkv_role<HD>(b, pair, r, smem);
  } else if (r < per) {
    // all eight wavefronts take part (the staged tiles need every one of
    // them); item < 0 marks one with no sequence of its own
    dq_role<HD, NQ>(b, pair, items - 1 - (r * kDkvWaves + wave), smem);
  }
}

}  // namespace

size_t bwd_workspace_bytes(int S, int L, int Hkv, int hd, int num_pages, int CP) {
  const int64_t nseg = static_cast<int64_t>(L) * Hkv;
  auto up = [](int64_t bytes) { return (bytes + 255) / 256 * 256; };
  const int64_t qsz = nseg * S * kNqp * hd, vsz = nseg * S * kNqp;
  const int64_t cpg = static_cast<int64_t>(L) * num_pages * Hkv * kPage * hd;
  const int64_t cpc = static_cast<int64_t>(L) * S * CP * Hkv * kPage * hd;
  return static_cast<size_t>(4 * up(qsz * 2) + 2 * up(vsz * 4) + 2 * up(cpg * 2) + 2 * up(cpc * 2));
}

hipError_t launch_attention_backward(const BwdArgs& b, hipStream_t stream) {
  const AttnArgs& a = b.a;
  if (a.S == 0 || b.layer_count == 0) return hipSuccess;
  const int nseg = b.layer_count * a.Hkv;
  hipLaunchKernelGGL(bwd_prep_kernel<64>, dim3(a.S, nseg), dim3(256), 0, stream, b);
  const int64_t pages = static_cast<int64_t>(b.layer_count) * a.Hkv *
                        (static_cast<int64_t>(a.num_pages) + static_cast<int64_t>(a.S) * a.CP);
  const int64_t items = pages * (kPage * 64 / 8);
  hipLaunchKernelGGL(bwd_copy_kernel<64>, dim3(static_cast<unsigned>((items + 255) / 256)),
                     dim3(256), 0, stream, b);
  const int groups = (a.S + b.group - 1) / b.group;
  const int units = ((a.max_pages + 1) / 2 + kDkvTiles * kDkvWaves - 1) / (kDkvTiles * kDkvWaves);
  const int xpairs = (groups * nseg + 7) / 8 * 8;   // pairs per launch, padded to the 8 XCDs
  const int n_dkv = xpairs * units;
  hipLaunchKernelGGL(bwd_dkv_carry_kernel<64>, dim3(a.S, nseg), dim3(64), 0, stream, b);
  if (b.group > 1) {
    const int per = ((b.group + kDqSeqs - 1) / kDqSeqs + kDkvWaves - 1) / kDkvWaves;
    const int rounds = std::max(units, per);   // workgroups: 8 XCDs x 2 kinds x pairs per XCD
    hipLaunchKernelGGL((bwd_attn_kernel<64, kDqSeqs>), dim3(16 * (xpairs / 8) * rounds),
                       dim3(64 * kDkvWaves), 0, stream, b, n_dkv);
  } else {
    const int dq_wgs = (groups * nseg + kDkvWaves - 1) / kDkvWaves;
    hipLaunchKernelGGL((bwd_attn_kernel<64, 1>), dim3(n_dkv + dq_wgs), dim3(64 * kDkvWaves), 0,
                       stream, b, n_dkv);
  }
  return hipGetLastError();
}

}  // namespace co

// ============================================================================
// Reverse mode of the K/V projection (Eq. 1-2: x = h + E on carried rows,
// z = F x, k_l = R(pos) K_l z, v_l = V_l z) for the trained W_F, W_KV and
// E_carry, the target's states h held constant:
//   dJ_r = [R(pos_r)^T dk_r ; dv_r] for every layer and KV head (W_KV's row order),
//   dW_KV += sum_r dJ_r z_r^T,   dz_r = W_KV^T dJ_r,
//   dW_F  += sum_r dz_r h_r^T + u E^T,   dE += F^T u,   u = sum over carried r of dz_r.
// The products run on the projection's MFMA kernels with the summed index (the
// rows) contiguous in both operands, so the row-major inputs are transposed
// first; rows are padded with zeros to a multiple of 256.
namespace co {

namespace {

constexpr int kRowPad = 256;
constexpr int kDeParts = 4;   // dE = F^T u is summed over this many row ranges of F, then in order
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

struct PbWs {
  float *fe, *u, *upart, *dep, *t32, *part;
  uint16_t *ht, *dj, *djt, *ztb, *dztb, *wkvt;
  int Mp;
};

int64_t pb_up(int64_t b) { return (b + 255) / 256 * 256; }

PbWs pb_ws(void* ws, int M, int Dcat, int d, int n_kv) {
  PbWs w;
  w.Mp = (M + kRowPad - 1) / kRowPad * kRowPad;
  const int64_t Mp = w.Mp;
  char* p = static_cast<char*>(ws);
  w.fe = reinterpret_cast<float*>(p); p += pb_up(d * 4);
  w.u = reinterpret_cast<float*>(p); p += pb_up(d * 4);
  w.upart = reinterpret_cast<float*>(p); p += pb_up(d * (Mp / 2048 + 1) * 4);
  w.dep = reinterpret_cast<float*>(p); p += pb_up(static_cast<int64_t>(kDeParts) * Dcat * 4);
  w.t32 = reinterpret_cast<float*>(p); p += pb_up(d * Mp * 4);
  w.ht = reinterpret_cast<uint16_t*>(p); p += pb_up(Dcat * Mp * 2);
  w.dj = reinterpret_cast<uint16_t*>(p); p += pb_up(Mp * n_kv * 2);
  w.djt = reinterpret_cast<uint16_t*>(p); p += pb_up(Mp * n_kv * 2);
  w.ztb = reinterpret_cast<uint16_t*>(p); p += pb_up(d * Mp * 2);
  w.dztb = reinterpret_cast<uint16_t*>(p); p += pb_up(d * Mp * 2);
  w.wkvt = reinterpret_cast<uint16_t*>(p); p += pb_up(static_cast<int64_t>(d) * n_kv * 2);
  w.part = reinterpret_cast<float*>(p);
  return w;
}

// dst[c][r] = src[r][c] for r < R (zero for R <= r < Rp), c < C: 64 x 64 tiles
// through LDS, 16 bytes per global load and store.  C, Rp, src_ld and dst_ld
// are multiples of 64 (8 would do for the accesses; the tiles then stay whole)
// and both buffers 16-byte aligned.  Eight consecutive lanes cover one 128-byte
// row segment on both sides.
__global__ __launch_bounds__(256) void pb_transpose_kernel(const uint16_t* src, int R, int C,
                                                           int64_t src_ld, uint16_t* dst, int Rp,
                                                           int64_t dst_ld) {
  __shared__ __align__(16) uint16_t t[64][72];   // 144-byte rows keep 16-byte stores aligned
  const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int q = threadIdx.x + 256 * j, i = q >> 3, k = q & 7;
    const int r = r0 + i;
    u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
    if (r < R) v = *reinterpret_cast<const u16x8*>(src + r * src_ld + c0 + 8 * k);
    *reinterpret_cast<u16x8*>(&t[i][8 * k]) = v;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int q = threadIdx.x + 256 * j, c = q >> 3, k = q & 7;
    u16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = t[8 * k + e][c];
    *reinterpret_cast<u16x8*>(dst + (c0 + c) * dst_ld + r0 + 8 * k) = v;
  }
}

// dJ [Mp][NKV]: one thread per (row, layer, head, rotation pair), pairs fastest,
// so that a row's key gradients are read and its dJ columns written in
// contiguous runs (its value gradients, [hd][16] per page, come through L2
// for the rows of one page in turn).
__global__ __launch_bounds__(256) void pb_gather_kernel(ProjBwdArgs a, uint16_t* dj, int Mp) {
  const int half = a.hd / 2;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = static_cast<int64_t>(a.L) * a.Hkv * half * Mp;
  if (idx >= total) return;
  const int i = static_cast<int>(idx % half);
  const int64_t jp = idx / half;
  const int g = static_cast<int>(jp % a.Hkv);
  const int l = static_cast<int>((jp / a.Hkv) % a.L);
  const int r = static_cast<int>(jp / (static_cast<int64_t>(a.Hkv) * a.L));
  float klo = 0.f, khi = 0.f, vlo = 0.f, vhi = 0.f;
  const int32_t dst = r < a.M ? a.row_dst[r] : kSkip;
  const int64_t pe = static_cast<int64_t>(kPage) * a.hd;
  int64_t pg = -1;
  const float *kb = nullptr, *vb = nullptr;
  int slot = 0;
  if (dst >= 0) {
    const int page = dst / kPage;
    slot = dst % kPage;
    if (page < a.num_pages) {
      pg = (static_cast<int64_t>(l) * a.num_pages + page) * a.Hkv + g;
      kb = a.dk;
      vb = a.dv;
    }
  } else if (dst != kSkip) {
    const int c = -1 - dst, s = r / a.B;
    if (c < a.CP * kPage) {
      slot = c % kPage;
      pg = ((static_cast<int64_t>(l) * a.S + s) * a.CP + c / kPage) * a.Hkv + g;
      kb = a.dkc;
      vb = a.dvc;
    }
  }
  if (pg >= 0) {
    const float* kr = kb + pg * pe + slot * a.hd;
    const float* vr = vb + pg * pe + slot;
    const float k0 = kr[i], k1 = kr[i + half];
    vlo = vr[i * kPage];
    vhi = vr[(i + half) * kPage];
    float c, s;
    rope_cos_sin(a.row_pos[r], a.rope_inv[i], &c, &s);   // R^T: turn back by the row's angle
    klo = k0 * c + k1 * s;
    khi = k1 * c - k0 * s;
  }
  const int64_t jk = ((static_cast<int64_t>(l) * 2 + 0) * a.Hkv + g) * a.hd + i;
  const int64_t jv = ((static_cast<int64_t>(l) * 2 + 1) * a.Hkv + g) * a.hd + i;
  uint16_t* row = dj + static_cast<int64_t>(r) * (2 * a.L * a.Hkv * a.hd);
  row[jk] = f2bf(klo);
  row[jk + half] = f2bf(khi);
  row[jv] = f2bf(vlo);
  row[jv + half] = f2bf(vhi);
}

// Z^T (fp32 [d][M]) + F E on carried rows -> bf16 [d][Mp], padding rows zero:
// four rows per thread, with 16-byte loads where M is a multiple of 4.  Mp is a
// multiple of 4.
__global__ __launch_bounds__(256) void pb_zt_kernel(const float* t32, int d, int M, int Mp,
                                                    const int32_t* row_dst, const float* fe,
                                                    uint16_t* ztb) {
  const int64_t idx = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (idx >= static_cast<int64_t>(d) * Mp) return;
  const int r0 = static_cast<int>(idx % Mp), dd = static_cast<int>(idx / Mp);
  const float* src = t32 + static_cast<int64_t>(dd) * M + r0;
  f32x4 v = {0.f, 0.f, 0.f, 0.f};
  int32_t dst[4] = {kSkip, kSkip, kSkip, kSkip};
  if (r0 + 4 <= M && (M & 3) == 0) {
    v = *reinterpret_cast<const f32x4*>(src);
#pragma unroll
    for (int e = 0; e < 4; ++e) dst[e] = row_dst[r0 + e];
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (r0 + e < M) {
        v[e] = src[e];
        dst[e] = row_dst[r0 + e];
      }
  }
  const float f = fe[dd];
  u16x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = f2bf(v[e] + ((dst[e] < 0 && dst[e] != kSkip) ? f : 0.f));
  *reinterpret_cast<u16x4*>(ztb + idx) = o;
}

// dZ^T (fp32 [d][Mp]) -> bf16, and per (dd, chunk of 2048 rows) the sum over
// its carried rows (summed over chunks in pb_u_kernel): 8 rows per thread.
constexpr int kDzChunk = 2048;

__global__ __launch_bounds__(256) void pb_dz_kernel(const float* t32, int M, int Mp,
                                                    const int32_t* row_dst, uint16_t* dztb,
                                                    float* upart) {
  __shared__ float red[4];
  const int dd = blockIdx.x, ch = blockIdx.y;
  const int r0 = ch * kDzChunk + threadIdx.x * 8;
  float acc = 0.f;
  if (r0 < Mp) {
    const float* src = t32 + static_cast<int64_t>(dd) * Mp + r0;
    const f32x4 a = *reinterpret_cast<const f32x4*>(src);
    const f32x4 b = *reinterpret_cast<const f32x4*>(src + 4);
    u16x8 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = f2bf(a[e]);
      o[4 + e] = f2bf(b[e]);
    }
    *reinterpret_cast<u16x8*>(dztb + static_cast<int64_t>(dd) * Mp + r0) = o;
    int32_t x[8];
    // two 16-byte loads when the eight rows exist and the array is 16-byte
    // aligned (r0 is a multiple of 8)
    if (r0 + 8 <= M && (reinterpret_cast<uintptr_t>(row_dst) & 15) == 0) {
      const i32x4 x0 = *reinterpret_cast<const i32x4*>(row_dst + r0);
      const i32x4 x1 = *reinterpret_cast<const i32x4*>(row_dst + r0 + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = x0[e];
        x[4 + e] = x1[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = r0 + e < M ? row_dst[r0 + e] : kSkip;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (x[e] < 0 && x[e] != kSkip) acc += e < 4 ? a[e] : b[e - 4];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) upart[dd * gridDim.y + ch] = (red[0] + red[1]) + (red[2] + red[3]);
}

// u[dd] = sum of the chunk sums, in chunk order.
__global__ __launch_bounds__(256) void pb_u_kernel(const float* upart, int chunks, int d, float* u) {
  const int dd = blockIdx.x * 256 + threadIdx.x;
  if (dd >= d) return;
  float v = 0.f;
  for (int c = 0; c < chunks; ++c) v += upart[dd * chunks + c];
  u[dd] = v;
}

// dW_F[dd][c] += u[dd] E[c], one element per thread; threads c < Dcat also add
// the kDeParts partial sums of dE[c] (pb_de_kernel), in order.
__global__ __launch_bounds__(256) void pb_dwf_e_kernel(float* dwf, const float* u,
                                                       const uint16_t* e, int d, int Dcat,
                                                       float* de, const float* dep) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(d) * Dcat) return;
  dwf[i] += u[i / Dcat] * bf2f(e[i % Dcat]);
  if (i < Dcat) {
    float v = dep[i];
    for (int q = 1; q < kDeParts; ++q) v += dep[static_cast<int64_t>(q) * Dcat + i];
    de[i] += v;
  }
}

// Partial sums of dE[c] = sum_dd W_F[dd][c] u[dd]: workgroup (column block,
// part q) takes 64 columns and rows dd of part q; its four wavefronts take
// interleaved dd and are summed in a fixed order.
__global__ __launch_bounds__(256) void pb_de_kernel(float* dep, const float* u, const uint16_t* wf,
                                                    int d, int Dcat) {
  __shared__ float part[4][64];
  const int c = blockIdx.x * 64 + (threadIdx.x & 63), wv = threadIdx.x >> 6;
  const int per = (d + kDeParts - 1) / kDeParts, d0 = blockIdx.y * per, d1 = min(d, d0 + per);
  float acc = 0.f;
  if (c < Dcat)
    for (int dd = d0 + wv; dd < d1; dd += 4)
      acc = fmaf(bf2f(wf[static_cast<int64_t>(dd) * Dcat + c]), u[dd], acc);
  part[wv][threadIdx.x & 63] = acc;
  __syncthreads();
  if (wv == 0 && c < Dcat)
    dep[static_cast<int64_t>(blockIdx.y) * Dcat + c] =
        (part[0][threadIdx.x] + part[1][threadIdx.x]) + (part[2][threadIdx.x] + part[3][threadIdx.x]);
}

}  // namespace

size_t proj_bwd_ws_bytes(int M, int Dcat, int d, int n_kv, int num_cus) {
  const int64_t Mp = (M + kRowPad - 1) / kRowPad * kRowPad;
  size_t part = gemm_acc_ws_bytes(d, M, Dcat, num_cus);
  part = std::max(part, gemm_acc_ws_bytes(n_kv, d, static_cast<int>(Mp), num_cus));
  part = std::max(part, gemm_acc_ws_bytes(d, static_cast<int>(Mp), n_kv, num_cus));
  part = std::max(part, gemm_acc_ws_bytes(d, Dcat, static_cast<int>(Mp), num_cus));
  return static_cast<size_t>(2 * pb_up(d * 4) + pb_up(d * (Mp / 2048 + 1) * 4) +
                             pb_up(static_cast<int64_t>(kDeParts) * Dcat * 4) +
                             pb_up(d * Mp * 4) + pb_up(Dcat * Mp * 2) +
                             2 * pb_up(Mp * n_kv * 2) + 2 * pb_up(d * Mp * 2) +
                             pb_up(static_cast<int64_t>(d) * n_kv * 2)) + part;
}

hipError_t launch_project_backward(const ProjBwdArgs& a, hipStream_t stream) {
  if (a.M == 0) return hipSuccess;
  const int n_kv = 2 * a.L * a.Hkv * a.hd;
  // every transpose below has C, Rp and both leading dimensions multiples of 64
  // (Dcat and d are, Mp is a multiple of 256, NKV of 128)
  if (a.Dcat % 64 || a.d % 64 || n_kv % 64) return hipErrorInvalidValue;
  const PbWs w = pb_ws(a.ws, a.M, a.Dcat, a.d, n_kv);
  const int Mp = w.Mp;
  hipError_t err;
  if ((err = launch_fold_e(a.wf, a.e, a.d, a.Dcat, CO_DTYPE_BF16, w.fe, stream)) != hipSuccess)
    return err;
  auto transpose = [&](const void* src, int R, int C, int64_t src_ld, uint16_t* dst, int Rp,
                       int64_t dst_ld) {
    const dim3 grid(Rp / 64, C / 64);
    hipLaunchKernelGGL(pb_transpose_kernel, grid, dim3(256), 0, stream,
                       static_cast<const uint16_t*>(src), R, C, src_ld, dst, Rp, dst_ld);
  };
  transpose(a.hidden, a.M, a.Dcat, a.Dcat, w.ht, Mp, Mp);       // H^T [Dcat][Mp]
  transpose(a.wkv, n_kv, a.d, a.d, w.wkvt, n_kv, n_kv);          // W_KV^T [d][NKV]
  const int64_t items = static_cast<int64_t>(a.L) * a.Hkv * (a.hd / 2) * Mp;
  hipLaunchKernelGGL(pb_gather_kernel, dim3(static_cast<unsigned>((items + 255) / 256)), dim3(256),
                     0, stream, a, w.dj, Mp);
  transpose(w.dj, Mp, n_kv, n_kv, w.djt, Mp, Mp);                // dJ^T [NKV][Mp]
  // Z^T = F H^T (+ F E on carried rows)
  if ((err = launch_gemm_acc(a.wf, a.hidden, a.d, a.M, a.Dcat, w.t32, false, w.part, a.num_cus,
                             stream)) != hipSuccess)
    return err;
  const int64_t dm = static_cast<int64_t>(a.d) * Mp;
  hipLaunchKernelGGL(pb_zt_kernel, dim3(static_cast<unsigned>((dm / 4 + 255) / 256)), dim3(256), 0,
                     stream, w.t32, a.d, a.M, Mp, a.row_dst, w.fe, w.ztb);
  // dW_KV += dJ^T Z
  if ((err = launch_gemm_acc(w.djt, w.ztb, n_kv, a.d, Mp, a.dwkv, true, w.part, a.num_cus,
                             stream)) != hipSuccess)
    return err;
  // dZ^T = W_KV^T dJ^T
  if ((err = launch_gemm_acc(w.wkvt, w.dj, a.d, Mp, n_kv, w.t32, false, w.part, a.num_cus,
                             stream)) != hipSuccess)
    return err;
  const int chunks = (Mp + kDzChunk - 1) / kDzChunk;
  hipLaunchKernelGGL(pb_dz_kernel, dim3(a.d, chunks), dim3(256), 0, stream, w.t32, a.M, Mp,
                     a.row_dst, w.dztb, w.upart);
  hipLaunchKernelGGL(pb_u_kernel, dim3((a.d + 255) / 256), dim3(256), 0, stream, w.upart, chunks,
                     a.d, w.u);
  // dW_F += dZ^T H (+ u E^T), dE += F^T u
  if ((err = launch_gemm_acc(w.dztb, w.ht, a.d, a.Dcat, Mp, a.dwf, true, w.part, a.num_cus,
                             stream)) != hipSuccess)
    return err;
  const int64_t nf = static_cast<int64_t>(a.d) * a.Dcat;
  hipLaunchKernelGGL(pb_de_kernel, dim3((a.Dcat + 63) / 64, kDeParts), dim3(256), 0, stream, w.dep,
                     w.u, static_cast<const uint16_t*>(a.wf), a.d, a.Dcat);
  hipLaunchKernelGGL(pb_dwf_e_kernel, dim3(static_cast<unsigned>((nf + 255) / 256)), dim3(256), 0,
                     stream, a.dwf, w.u, static_cast<const uint16_t*>(a.e), a.d, a.Dcat, a.de, w.dep);
  return hipGetLastError();
}

}  // namespace co
