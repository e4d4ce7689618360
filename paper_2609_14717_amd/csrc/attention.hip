// Block-parallel drafter attention over ctx = [C ; U] (Eq. 2; Algorithm 1
// step 7; Section 2 "Preliminaries": every block query attends to K/V built
// from target states).  The committed segment C is read through the page
// table, the carryover segment U from the per-sequence carry pages; both are
// consumed by one online softmax, so the concatenation is never materialised.
//
// bf16 path (the serving path), a persistent load-balanced kernel:
//   * the keys of every (layer, KV head, sequence) -- ceil(ctx/16) committed
//     pages followed by ceil(carry/16) carry pages -- are cut into 32-key tiles,
//     and all tiles of all segments form one global sequence;
//   * one workgroup per CU takes an equal contiguous slice of that sequence
//     (no idle workgroups, no tail from ragged lengths), walking the segments
//     its slice touches; for each it rotates the B * (Hq/Hkv) queries of that KV
//     head into LDS once, then its wavefronts stream alternate tiles;
//   * keys and values go global -> LDS with direct-to-LDS 16-byte loads into a
//     ring private to each wavefront (NS tiles deep, exact vmcnt waits, no
//     workgroup barrier in the loop), K rows XOR-swizzled for conflict-free
//     fragment reads;
//   * S^T = K . Q^T per tile uses two 16-key MFMA M-tiles whose rows are keys
//     {8q+r} and {8q+4+r} (q = lane/16), so the softmax'ed scores a lane holds
//     are exactly the 8 keys it needs for O^T += V^T . P^T, with V pages stored
//     [head_dim][16 slots] -- no data movement between the two products;
//   * a segment finished inside one slice is normalised and written in place;
//     a segment split across slices leaves one unnormalised (O, max, sum)
//     record per slice and a small kernel combines them (log-sum-exp rule).
//     Combining inside the persistent kernel would need a device-scope release
//     per workgroup, which on this part writes back the L2 of the XCD.
// fp32 path: per-chunk workgroups with plain VALU arithmetic through LDS.
#include <stdlib.h>

#include "co_kernels.h"

namespace co {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxChunkPages = 256;   // page-id staging capacity (fp32 chunk / bf16 sub-chunk)

struct SeqInfo {
  int ctx, carry, npc, npt, nch;
  bool ok;
};

__device__ __forceinline__ SeqInfo seq_info(const AttnArgs& a, int s, int chunk_pages) {
  SeqInfo q;
  q.ctx = a.ctx_len[s];
  q.carry = a.carry_len[s];
  q.ok = q.ctx >= 0 && q.ctx <= a.max_pages * kPage && q.carry >= 0 && q.carry <= a.CP * kPage;
  q.npc = q.ok ? (q.ctx + kPage - 1) / kPage : 0;
  q.npt = q.ok ? q.npc + (q.carry + kPage - 1) / kPage : 0;
  q.nch = (q.npt + chunk_pages - 1) / chunk_pages;
  return q;
}

__device__ __forceinline__ float wave_max_across_groups(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}

__device__ __forceinline__ float wave_sum_across_groups(float v) {
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}

// Partial record of (layer, seq, kv head, chunk) on the fp32 path: O[nq_pad][hd],
// m[nq_pad], l[nq_pad] (m in log2 units of the scaled logits; O unnormalised).
__device__ __forceinline__ float* record_ptr(const AttnArgs& a, int layer_local, int s, int g,
                                             int c, int n_chunks, int nq_pad) {
  const int64_t rec = ((static_cast<int64_t>(layer_local) * a.S + s) * a.Hkv + g) * n_chunks + c;
  return a.ws + rec * nq_pad * (a.hd + 2);
}

__device__ __forceinline__ int64_t out_row(const AttnArgs& a, int layer_local, int s, int g, int n,
                                           int G) {
  const int i = n / G, hh = n % G;
  return ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq + g * G + hh;
}

// fp32 path: combine the chunk records of every (layer, sequence, KV head)
// whose key set spans more than one chunk, and write O (+ LSE).  The running
// maxima and sums of all chunks are staged in LDS with one round of independent
// loads and turned into per-(chunk, query) weights.
constexpr int kMaxMergeChunks = 64;
constexpr int kMaxMergeSlices = 4096;   // workgroups of one persistent launch

template <typename T>
__global__ __launch_bounds__(256) void attn_chunk_merge_kernel(AttnArgs a, int chunk_pages,
                                                         int n_chunks, int nq_pad) {
  __shared__ float w_lds[kMaxMergeChunks * 64];
  __shared__ float l_lds[kMaxMergeChunks * 64];
  const int s = blockIdx.x;
  const int layer_local = blockIdx.y / a.Hkv, g = blockIdx.y % a.Hkv;
  const SeqInfo si = seq_info(a, s, chunk_pages);
  if (si.nch <= 1) return;                 // finished by the chunk kernel
  const int hd = a.hd, G = a.Hq / a.Hkv, nq = a.B * G, q4 = hd / 4, nch = si.nch;
  const int tid = threadIdx.x;
  const float* base = record_ptr(a, layer_local, s, g, 0, n_chunks, nq_pad);
  const int64_t rec = static_cast<int64_t>(nq_pad) * (hd + 2);
  for (int idx = tid; idx < nch * nq_pad; idx += 256) {
    const int c = idx / nq_pad, n = idx % nq_pad;
    w_lds[idx] = base[c * rec + nq_pad * hd + n];
    l_lds[idx] = base[c * rec + nq_pad * hd + nq_pad + n];
  }
  __syncthreads();
  for (int n = tid; n < nq; n += 256) {
    float M = -INFINITY;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, w_lds[c * nq_pad + n]);
    float den = 0.f;
    for (int c = 0; c < nch; ++c) {
      const float m = w_lds[c * nq_pad + n];
      const float wgt = (m == -INFINITY) ? 0.f : exp2f(m - M);
      w_lds[c * nq_pad + n] = wgt;
      den += wgt * l_lds[c * nq_pad + n];
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    for (int c = 0; c < nch; ++c) w_lds[c * nq_pad + n] *= inv;
    if (a.lse && blockIdx.z == 0)
      a.lse[out_row(a, layer_local, s, g, n, G)] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
  }
  __syncthreads();
  T* out = static_cast<T*>(a.out);
  for (int idx = tid + blockIdx.z * 256; idx < nq * q4; idx += 256 * gridDim.z) {
    const int n = idx / q4, d = (idx % q4) * 4;
    const float* p = base + n * hd + d;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    int c = 0;
    for (; c + 4 <= nch; c += 4) {
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(p + (c + 0) * rec);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(p + (c + 1) * rec);
      const f32x4 v2 = *reinterpret_cast<const f32x4*>(p + (c + 2) * rec);
      const f32x4 v3 = *reinterpret_cast<const f32x4*>(p + (c + 3) * rec);
      acc += w_lds[(c + 0) * nq_pad + n] * v0;
      acc += w_lds[(c + 1) * nq_pad + n] * v1;
      acc += w_lds[(c + 2) * nq_pad + n] * v2;
      acc += w_lds[(c + 3) * nq_pad + n] * v3;
    }
    for (; c < nch; ++c) acc += w_lds[c * nq_pad + n] * *reinterpret_cast<const f32x4*>(p + c * rec);
    T* o = out + out_row(a, layer_local, s, g, n, G) * hd + d;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = to_elem<T>(acc[r]);
  }
}

// fp32 path: the same chunk partials, computed with plain VALU arithmetic through LDS,
// always combined through the workspace records.
template <int HD>
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnArgs a, int chunk_pages, int n_chunks,
                                                       int nq_pad) {
  constexpr int KT = 32;
  __shared__ float qs[64][HD + 1];
  __shared__ float os[64][HD + 1];
  __shared__ float ks[KT][HD + 1];
  __shared__ float vs[KT][HD + 1];
  __shared__ float sc[64][KT + 1];
  __shared__ float m_run[64], l_run[64], alpha_s[64];
  __shared__ int kvalid[KT];

  const int c = blockIdx.x, s = blockIdx.y;
  const int layer_local = blockIdx.z / a.Hkv, g = blockIdx.z % a.Hkv;
  const int layer = a.layer_begin + layer_local;
  const int tid = threadIdx.x;
  const SeqInfo si = seq_info(a, s, chunk_pages);
  if (!si.ok) {
    if (c == 0 && tid == 0) set_status(a.status, CO_ERR_LENGTH);
    return;
  }
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  if (si.npt == 0) {
    if (c != 0) return;
    float* out = static_cast<float*>(a.out);
    for (int idx = tid; idx < nq * HD; idx += 256)
      out[out_row(a, layer_local, s, g, idx / HD, G) * HD + idx % HD] = 0.f;
    if (a.lse)
      for (int n = tid; n < nq; n += 256) a.lse[out_row(a, layer_local, s, g, n, G)] = -INFINITY;
    return;
  }
  const int ctx = si.ctx, carry = si.carry, npc = si.npc;
  const int p_begin = c * chunk_pages;
  if (p_begin >= si.npt) return;
  const int p_end = min(p_begin + chunk_pages, si.npt);
  const float* Q = static_cast<const float*>(a.q);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;

  for (int idx = tid; idx < nq * (HD / 2); idx += 256) {
    const int n = idx / (HD / 2), p = idx % (HD / 2);
    const float* qrow = Q + out_row(a, layer_local, s, g, n, G) * HD;
    float lo = qrow[p], hi = qrow[p + HD / 2];
    if (!(a.flags & CO_Q_PREROTATED)) {
      float cs, sn;
      rope_cos_sin(ctx + n / G, rope_inv_freq(p, HD, a.log2_theta), &cs, &sn);
      const float l2 = lo * cs - hi * sn, h2 = hi * cs + lo * sn;
      lo = l2;
      hi = h2;
    }
    qs[n][p] = lo * qscale;
    qs[n][p + HD / 2] = hi * qscale;
  }
  for (int idx = tid; idx < 64 * HD; idx += 256) os[idx / HD][idx % HD] = 0.f;
  if (tid < 64) {
    m_run[tid] = -INFINITY;
    l_run[tid] = 0.f;
  }
  __syncthreads();

  const float* kc = static_cast<const float*>(a.k_cache);
  const float* vc = static_cast<const float*>(a.v_cache);
  const float* kk = static_cast<const float*>(a.k_carry);
  const float* vk = static_cast<const float*>(a.v_carry);
  for (int lp0 = p_begin; lp0 < p_end; lp0 += 2) {
    // stage 32 keys (two logical pages)
    for (int idx = tid; idx < KT * HD; idx += 256) {
      const int key = idx / HD, dd = idx % HD;
      const int lp = lp0 + (key >> 4), slot = key & 15;
      float kv = 0.f, vv = 0.f;
      int valid = 0;
      if (lp < p_end) {
        if (lp < npc) {
          const int phys = a.page_table[static_cast<int64_t>(s) * a.max_pages + lp];
          if (phys >= 0 && phys < a.num_pages) {
            valid = lp * kPage + slot < ctx;
            if (valid) {
              const int64_t off =
                  ((static_cast<int64_t>(layer) * a.num_pages + phys) * a.Hkv + g) * kPage * HD;
              kv = kc[off + slot * HD + dd];
              vv = vc[off + dd * kPage + slot];
            }
          } else if (dd == 0) {
            set_status(a.status, CO_ERR_PAGE_RANGE);
          }
        } else {
          const int cp = lp - npc;
          valid = cp * kPage + slot < carry;
          if (valid) {
            const int64_t off =
                (((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp) * a.Hkv + g) * kPage * HD;
            kv = kk[off + slot * HD + dd];
            vv = vk[off + dd * kPage + slot];
          }
        }
      }
      ks[key][dd] = kv;
      vs[key][dd] = vv;
      if (dd == 0) kvalid[key] = valid;
    }
    __syncthreads();
    for (int idx = tid; idx < nq * KT; idx += 256) {
      const int n = idx / KT, key = idx % KT;
      float dot = 0.f;
      for (int dd = 0; dd < HD; ++dd) dot += qs[n][dd] * ks[key][dd];
      sc[n][key] = kvalid[key] ? dot : -INFINITY;
    }
    __syncthreads();
    if (tid < nq) {
      float mx = -INFINITY;
      for (int key = 0; key < KT; ++key) mx = fmaxf(mx, sc[tid][key]);
      const float m_new = fmaxf(m_run[tid], mx);
      const float al = (m_new == -INFINITY) ? 1.f : exp2f(m_run[tid] - m_new);
      const float base = (m_new == -INFINITY) ? 0.f : m_new;
      float sum = 0.f;
      for (int key = 0; key < KT; ++key) {
        const float p = exp2f(sc[tid][key] - base);
        sc[tid][key] = p;
        sum += p;
      }
      l_run[tid] = l_run[tid] * al + sum;
      m_run[tid] = m_new;
      alpha_s[tid] = al;
    }
    __syncthreads();
    for (int idx = tid; idx < nq * HD; idx += 256) {
      const int n = idx / HD, dd = idx % HD;
      float v = os[n][dd] * alpha_s[n];
      for (int key = 0; key < KT; ++key) v += sc[n][key] * vs[key][dd];
      os[n][dd] = v;
    }
    __syncthreads();
  }
  if (si.nch == 1) {
    float* out = static_cast<float*>(a.out);
    for (int idx = tid; idx < nq * HD; idx += 256) {
      const int n = idx / HD;
      const float inv = l_run[n] > 0.f ? 1.f / l_run[n] : 0.f;
      out[out_row(a, layer_local, s, g, n, G) * HD + idx % HD] = os[n][idx % HD] * inv;
    }
    if (a.lse && tid < nq)
      a.lse[out_row(a, layer_local, s, g, tid, G)] =
          l_run[tid] > 0.f ? (m_run[tid] + log2f(l_run[tid])) * kLn2 : -INFINITY;
    return;
  }
  float* part = record_ptr(a, layer_local, s, g, c, n_chunks, nq_pad);
  for (int idx = tid; idx < nq * HD; idx += 256) part[idx] = os[idx / HD][idx % HD];
  if (tid < nq) {
    part[nq_pad * HD + tid] = m_run[tid];
    part[nq_pad * HD + nq_pad + tid] = l_run[tid];
  }
}

// ------------------------------------------------------- bf16 persistent path

// Tiles (32 keys = 2 logical pages) of sequence s; sequences with invalid
// lengths have none (the combine kernel reports them).
__device__ __forceinline__ int seq_tiles(const AttnArgs& a, int s) {
  const SeqInfo q = seq_info(a, s, 1);
  return (q.npt + 1) / 2;
}

// First tile of workgroup w's slice of T tiles split over n_wg workgroups.
__device__ __forceinline__ int64_t slice_begin(int64_t T, int w, int n_wg) {
  return T * w / n_wg;
}

// Workspace of the persistent path: a header with the tile prefix sums (S+1
// ints, written by workgroup 0) and the first global tile of every slice
// (n_wg+1 int64 from int offset slice_bounds_off(S), each written by its
// workgroup), both for the combine kernel; then one record per (slice,
// segment) pair: O[NQP][hd] unnormalised, m[NQP], l[NQP].
__host__ __device__ __forceinline__ int slice_bounds_off(int S) { return (S + 2) & ~1; }

__device__ __forceinline__ float* slot_ptr(const AttnArgs& a, int hdr_floats, int64_t slot,
                                           int nqp) {
  return a.ws + hdr_floats + slot * nqp * (a.hd + 2);
}

template <int HD, int NT, int NW, int NS>
__global__ __launch_bounds__(64 * NW) void attn_bf16_kernel(AttnArgs a, int layer_count, int n_wg,
                                                             int hdr_floats) {
  constexpr int KS = HD / 32;              // k-steps of S^T
  constexpr int MT = HD / 16;              // M-tiles of O^T
  constexpr int NQP = NT * 16;
  constexpr int NTHR = 64 * NW;
  constexpr int QLD = HD + 8;              // padded LDS row of rotated queries (bf16)
  constexpr int NRED = NW > 1 ? NW - 1 : 1;
  constexpr int ROWB = HD * 2;             // bytes of one key row
  constexpr int CPR = ROWB / 16;           // 16-byte chunks per key row
  constexpr int PAGE_BYTES = kPage * ROWB; // one page of K (or of V)
  constexpr int LPP = PAGE_BYTES / 1024;   // 1 KiB wave loads per page
  constexpr int TILE_BYTES = 4 * PAGE_BYTES;   // K page 0, K page 1, V page 0, V page 1
  constexpr int NL = 4 * LPP;              // direct-to-LDS loads per tile per wave
  constexpr int RING_BYTES = NW * NS * TILE_BYTES;
  constexpr int RED_BYTES = (NRED * NQP * (HD + 1) + 2 * NRED * NQP) * 4;
  constexpr int SMEM_BYTES = RING_BYTES > RED_BYTES ? RING_BYTES : RED_BYTES;
  constexpr int SUB_TILES = kMaxChunkPages / 2;
  static_assert(NL * (NS - 1) < 64, "vmcnt");
  // the ring, reused for the cross-wave merge once a segment is done
  __shared__ __align__(16) unsigned char smem[SMEM_BYTES];
  __shared__ __align__(16) uint16_t q_lds[NQP * QLD];
  __shared__ int pg_lds[kMaxChunkPages];
  __shared__ int tstart[kMaxAttnSeqs + 1];
  __shared__ double inv_lds[HD / 2];
  __shared__ int wave_tot[NW];
  float* red_o = reinterpret_cast<float*>(smem);                 // [NRED][NQP][HD + 1]
  float* red_m = red_o + NRED * NQP * (HD + 1);                  // [NRED][NQP]
  float* red_l = red_m + NRED * NQP;                             // [NRED][NQP]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = lane >> 4, col = lane & 15;
  const int S = a.S, G = a.Hq / a.Hkv, nq = a.B * G;

  // ---- tiles per sequence and their prefix sums (the same for every segment row)
  {
    const int per = (S + NTHR - 1) / NTHR, s0 = tid * per;
    int local = 0;
    for (int i = 0; i < per; ++i)
      if (s0 + i < S) local += seq_tiles(a, s0 + i);
    int v = local;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int u = __shfl_up(v, off);
      if (lane >= off) v += u;
    }
    if (lane == 63) wave_tot[wave] = v;
    if (tid < HD / 2) inv_lds[tid] = rope_inv_freq(tid, HD, a.log2_theta);
    __syncthreads();
    int run = v - local;
    for (int w = 0; w < wave; ++w) run += wave_tot[w];
    for (int i = 0; i < per; ++i)
      if (s0 + i < S) {
        tstart[s0 + i] = run;
        run += seq_tiles(a, s0 + i);
      }
    if (tid == NTHR - 1) tstart[S] = run;
    __syncthreads();
  }
  const int T1 = tstart[S];
  const int64_t T = static_cast<int64_t>(layer_count) * a.Hkv * T1;
  const int w = blockIdx.x;
  const int64_t r1 = slice_begin(T, w + 1, n_wg);
  {
    int* hdr = reinterpret_cast<int*>(a.ws);
    if (w == 0)
      for (int i = tid; i <= S; i += NTHR) hdr[i] = tstart[i];
    int64_t* bounds = reinterpret_cast<int64_t*>(hdr + slice_bounds_off(S));
    if (tid == 0) bounds[w + 1] = r1;
    if (tid == 0 && w == 0) bounds[0] = 0;
  }

  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* vc = static_cast<const uint16_t*>(a.v_cache);
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);
  const uint16_t* vk = static_cast<const uint16_t*>(a.v_carry);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;
  const uint16_t* Q = static_cast<const uint16_t*>(a.q);
  // key of S^T M-tile a / b at row rho = lane % 16: keys {8q + r} and {8q + 4 + r}
  const int key_a = 8 * (col >> 2) + (col & 3);
  const int key_b = key_a + 4;
  const int slot_base = (grp & 1) * 8;
  unsigned char* my_ring = smem + wave * NS * TILE_BYTES;
  // Per-lane source offsets (elements) of the direct-to-LDS loads of one page:
  // K rows land XOR-swizzled by (row mod CPR), V pages are copied as they are.
  int k_off[LPP], v_off[LPP];
#pragma unroll
  for (int q = 0; q < LPP; ++q) {
    const int byte = q * 1024 + lane * 16;
    const int r = byte / ROWB, pch = (byte % ROWB) / 16;
    k_off[q] = r * HD + (pch ^ (r & (CPR - 1))) * 8;
    v_off[q] = byte / 2;
  }
  // LDS byte offsets (within a tile) of this lane's K and V fragments
  uint32_t ka_off[KS], kb_off[KS], v_frag_off;
  {
    const int ra = key_a & 15, rb = key_b & 15;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int ch = ks * 4 + grp;
      ka_off[ks] = (key_a >> 4) * PAGE_BYTES + ra * ROWB + ((ch ^ (ra & (CPR - 1))) << 4);
      kb_off[ks] = (key_b >> 4) * PAGE_BYTES + rb * ROWB + ((ch ^ (rb & (CPR - 1))) << 4);
    }
    v_frag_off = (2 + (grp >> 1)) * PAGE_BYTES + col * 32 + slot_base * 2;
  }
  // Running maxima are kept as a lazily updated reference: p = 2^(s - ref) may
  // exceed 1 by up to 2^kRescale before the accumulators are rescaled, which
  // leaves the normalised result unchanged and skips most rescales.
  constexpr float kRescale = 8.f;

  for (int64_t cur = slice_begin(T, w, n_wg); cur < r1;) {
    // ---- locate the segment (layer, kv head, sequence) holding global tile cur
    const int seg = static_cast<int>(cur / T1);
    const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
    const int layer = a.layer_begin + layer_local;
    const int rr = static_cast<int>(cur % T1);
    int lo = 0, hi = S;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (tstart[mid] <= rr) lo = mid; else hi = mid;
    }
    const int s = lo;
    const int j0 = rr - tstart[s];
    const int nts = tstart[s + 1] - tstart[s];
    const int n = static_cast<int>(min(r1 - cur, static_cast<int64_t>(nts - j0)));
    const bool whole = j0 == 0 && n == nts;
    const SeqInfo si = seq_info(a, s, 1);
    const int64_t kv_layer = (static_cast<int64_t>(layer) * a.num_pages) * a.Hkv + g;
    const int64_t carry_base = ((static_cast<int64_t>(layer) * a.S + s) * a.CP) * a.Hkv + g;

    // ---- queries of this segment: rotate at ctx + i, fold 1/sqrt(hd)*log2(e), bf16 in LDS
    for (int idx = tid; idx < NQP * (HD / 2); idx += NTHR) {
      const int qn = idx / (HD / 2), p = idx % (HD / 2);
      float qlo = 0.f, qhi = 0.f;
      if (qn < nq) {
        const uint16_t* qrow = Q + out_row(a, layer_local, s, g, qn, G) * HD;
        qlo = bf2f(qrow[p]);
        qhi = bf2f(qrow[p + HD / 2]);
        if (!(a.flags & CO_Q_PREROTATED)) {
          float cs, sn;
          rope_cos_sin(si.ctx + qn / G, inv_lds[p], &cs, &sn);
          const float l2 = qlo * cs - qhi * sn, h2 = qhi * cs + qlo * sn;
          qlo = l2;
          qhi = h2;
        }
      }
      q_lds[qn * QLD + p] = f2bf(qlo * qscale);
      q_lds[qn * QLD + p + HD / 2] = f2bf(qhi * qscale);
    }

    f32x4 o[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) o[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run[NT], l_run[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      m_run[nt] = -INFINITY;
      l_run[nt] = 0.f;
    }
    u16x8 qf[NT][KS];

    for (int sub = 0; sub < n; sub += SUB_TILES) {
      const int sn_t = min(n - sub, SUB_TILES);            // tiles in this sub-chunk
      const int pbeg = 2 * (j0 + sub);                      // its first logical page
      const int pend = min(pbeg + 2 * sn_t, si.npt);
      __syncthreads();                                      // previous readers of pg_lds done
      for (int i = tid; i < pend - pbeg; i += NTHR) {
        const int lp = pbeg + i;
        int phys = -1;
        if (lp < si.npc) {
          phys = a.page_table[static_cast<int64_t>(s) * a.max_pages + lp];
          if (phys < 0 || phys >= a.num_pages) {
            set_status(a.status, CO_ERR_PAGE_RANGE);
            phys = -2;
          }
        }
        pg_lds[i] = phys;
      }
      __syncthreads();
      if (sub == 0) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            qf[nt][ks] =
                *reinterpret_cast<const u16x8*>(q_lds + (nt * 16 + col) * QLD + ks * 32 + grp * 8);
      }

      // Logical page lp -> K/V page addresses (wave-uniform) and valid slots.
      auto page = [&](int lp, const uint16_t*& kp, const uint16_t*& vp) -> int {
        kp = kk;
        vp = vk;
        if (lp >= pend) return 0;
        if (lp < si.npc) {
          const int phys = __builtin_amdgcn_readfirstlane(pg_lds[lp - pbeg]);
          if (phys < 0) return 0;
          const int64_t off = (kv_layer + static_cast<int64_t>(phys) * a.Hkv) * kPage * HD;
          kp = kc + off;
          vp = vc + off;
          return min(kPage, si.ctx - lp * kPage);
        }
        const int cp = lp - si.npc;
        const int64_t off = (carry_base + static_cast<int64_t>(cp) * a.Hkv) * kPage * HD;
        kp = kk + off;
        vp = vk + off;
        return min(kPage, si.carry - cp * kPage);
      };
      const int my_tiles = wave < sn_t ? (sn_t - 1 - wave) / NW + 1 : 0;
      auto issue = [&](int jj) {
        const int lp0 = pbeg + 2 * (wave + jj * NW);
        unsigned char* dst = my_ring + (jj % NS) * TILE_BYTES;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const uint16_t *kp, *vp;
          page(lp0 + half, kp, vp);
#pragma unroll
          for (int q = 0; q < LPP; ++q) {
            lds_dma16(kp + k_off[q], dst + half * PAGE_BYTES + q * 1024);
            lds_dma16(vp + v_off[q], dst + (2 + half) * PAGE_BYTES + q * 1024);
          }
        }
      };
#pragma unroll
      for (int jj = 0; jj < NS - 1; ++jj)
        if (jj < my_tiles) issue(jj);

      for (int jj = 0; jj < my_tiles; ++jj) {
        if (jj + NS - 1 < my_tiles) issue(jj + NS - 1);
        // valid slots of the tile's two pages (pages past the end have none)
        const int lp0 = pbeg + 2 * (wave + jj * NW);
        int n0 = 0, n1 = 0;
        if (lp0 < pend)
          n0 = lp0 < si.npc ? min(kPage, si.ctx - lp0 * kPage)
                            : min(kPage, si.carry - (lp0 - si.npc) * kPage);
        if (lp0 + 1 < pend)
          n1 = lp0 + 1 < si.npc ? min(kPage, si.ctx - (lp0 + 1) * kPage)
                                : min(kPage, si.carry - (lp0 + 1 - si.npc) * kPage);
        if (lp0 < si.npc && pg_lds[lp0 - pbeg] < 0) n0 = 0;
        if (lp0 + 1 < si.npc && lp0 + 1 < pend && pg_lds[lp0 + 1 - pbeg] < 0) n1 = 0;
        const bool partial = n0 < kPage || n1 < kPage;      // wave-uniform
        const int nv = (grp >> 1) ? n1 : n0;   // valid slots of the page holding my keys
        wait_stages_ahead<NL, NS>(min(NS - 1, my_tiles - 1 - jj));
        const unsigned char* tb = my_ring + (jj % NS) * TILE_BYTES;

        u16x8 ka[KS], kb[KS];
        {
          uint32_t aa[KS], ab[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            aa[ks] = lds_addr(tb + ka_off[ks]);
            ab[ks] = lds_addr(tb + kb_off[ks]);
          }
          if constexpr (KS == 2) {
            u16x8 v4[4];
            const uint32_t a4[4] = {aa[0], aa[1], ab[0], ab[1]};
            lds_read_group<4>(v4, a4);
            ka[0] = v4[0]; ka[1] = v4[1]; kb[0] = v4[2]; kb[1] = v4[3];
          } else {
            lds_read_group<KS>(ka, aa);
            lds_read_group<KS>(kb, ab);
          }
        }
        u16x8 va[MT];
        {
          const unsigned char* vb = tb + v_frag_off;
#pragma unroll
          for (int m4 = 0; m4 < MT; m4 += 4) {
            u16x8 v4[4];
            const uint32_t a4[4] = {lds_addr(vb + (m4 + 0) * 16 * 32), lds_addr(vb + (m4 + 1) * 16 * 32),
                                    lds_addr(vb + (m4 + 2) * 16 * 32), lds_addr(vb + (m4 + 3) * 16 * 32)};
            lds_read_group<4>(v4, a4);
#pragma unroll
            for (int i = 0; i < 4; ++i) va[m4 + i] = v4[i];
          }
          if (partial) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int e = 0; e < 8; ++e)
                if (slot_base + e >= nv) va[mt][e] = 0;   // invalid keys may hold anything
          }
        }

#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            sa = mfma16x16x32(ka[ks], qf[nt][ks], sa);
            sb = mfma16x16x32(kb[ks], qf[nt][ks], sb);
          }
          if (partial) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              sa[r] = (slot_base + r < nv) ? sa[r] : -INFINITY;
              sb[r] = (slot_base + 4 + r < nv) ? sb[r] : -INFINITY;
            }
          }
          float mx = fmaxf(fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3])),
                           fmaxf(fmaxf(sb[0], sb[1]), fmaxf(sb[2], sb[3])));
          mx = max_across_rows(mx);
          if (__any(mx > m_run[nt] + kRescale)) {
            // move the reference up (only where the tile exceeds it) and rescale
            const float m_new = mx > m_run[nt] + kRescale ? mx : m_run[nt];
            const float alpha = (m_new == m_run[nt]) ? 1.f : exp2f(m_run[nt] - m_new);
            l_run[nt] *= alpha;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) o[mt][nt] *= alpha;
            m_run[nt] = m_new;
          }
          const float base = (m_run[nt] == -INFINITY) ? 0.f : m_run[nt];
          float pa[4], pb[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {   // v_exp_f32: arguments are <= kRescale or -inf
            pa[r] = __builtin_amdgcn_exp2f(sa[r] - base);
            pb[r] = __builtin_amdgcn_exp2f(sb[r] - base);
          }
          l_run[nt] += (pa[0] + pa[1]) + (pa[2] + pa[3]) + (pb[0] + pb[1]) + (pb[2] + pb[3]);
          typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
          const u32x4v pk32 = {pack_bf16x2(pa[0], pa[1]), pack_bf16x2(pa[2], pa[3]),
                               pack_bf16x2(pb[0], pb[1]), pack_bf16x2(pb[2], pb[3])};
          const u16x8 pk = __builtin_bit_cast(u16x8, pk32);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) o[mt][nt] = mfma16x16x32(va[mt], pk, o[mt][nt]);
        }
      }
    }

#pragma unroll
    for (int nt = 0; nt < NT; ++nt) l_run[nt] = wave_sum_across_groups(l_run[nt]);

    // ---- merge the wavefronts through LDS (the drained ring) into wave 0
    __syncthreads();
    if constexpr (NW > 1) {
      if (wave > 0) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int qn = nt * 16 + col;
          if (grp == 0) {
            red_m[(wave - 1) * NQP + qn] = m_run[nt];
            red_l[(wave - 1) * NQP + qn] = l_run[nt];
          }
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              red_o[((wave - 1) * NQP + qn) * (HD + 1) + mt * 16 + grp * 4 + r] = o[mt][nt][r];
        }
      }
      __syncthreads();
      if (wave == 0) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int qn = nt * 16 + col;
          float M = m_run[nt];
#pragma unroll
          for (int wv = 1; wv < NW; ++wv) M = fmaxf(M, red_m[(wv - 1) * NQP + qn]);
          const float f0 = (m_run[nt] == -INFINITY) ? 0.f : exp2f(m_run[nt] - M);
          float lsum = l_run[nt] * f0;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) o[mt][nt] *= f0;
#pragma unroll
          for (int wv = 1; wv < NW; ++wv) {
            const float mw = red_m[(wv - 1) * NQP + qn];
            const float fw = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
            lsum += red_l[(wv - 1) * NQP + qn] * fw;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
              for (int r = 0; r < 4; ++r)
                o[mt][nt][r] += fw * red_o[((wv - 1) * NQP + qn) * (HD + 1) + mt * 16 + grp * 4 + r];
          }
          m_run[nt] = M;
          l_run[nt] = lsum;
        }
      }
    }

    if (wave == 0) {
      if (whole) {
        // the whole segment is in this slice: normalise and write O / LSE directly
        uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int qn = nt * 16 + col;
          if (qn >= nq) continue;
          const float inv = l_run[nt] > 0.f ? 1.f / l_run[nt] : 0.f;
          const int64_t row = out_row(a, layer_local, s, g, qn, G);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            u16x4 v;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = f2bf(o[mt][nt][r] * inv);
            *reinterpret_cast<u16x4*>(out + row * HD + mt * 16 + grp * 4) = v;
          }
          if (a.lse && grp == 0)
            a.lse[row] = l_run[nt] > 0.f ? (m_run[nt] + log2f(l_run[nt])) * kLn2 : -INFINITY;
        }
      } else {
        float* part = slot_ptr(a, hdr_floats, w + static_cast<int64_t>(seg) * S + s, NQP);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int qn = nt * 16 + col;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            *reinterpret_cast<f32x4*>(part + qn * HD + mt * 16 + grp * 4) = o[mt][nt];
          if (grp == 0) {
            part[NQP * HD + qn] = m_run[nt];
            part[NQP * HD + NQP + qn] = l_run[nt];
          }
        }
      }
    }
    __syncthreads();                                        // q_lds and smem are reused
    cur += n;
  }
}

// Combine the slice records of every (layer, KV head, sequence) split across
// slices, write O/LSE of segments without keys, and report invalid lengths.
// One thread per (query row, 4 output dims); record loads are issued in
// batches of kBatch so that their latencies overlap.
__global__ __launch_bounds__(256) void attn_bf16_combine_kernel(AttnArgs a, int layer_count,
                                                                int n_wg, int hdr_floats,
                                                                int nq_pad) {
  constexpr int kBatch = 8;
  const int s = blockIdx.x, seg = blockIdx.y;
  const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
  const int hd = a.hd, G = a.Hq / a.Hkv, nq = a.B * G, q4 = hd / 4;
  const int tid = threadIdx.x;
  const int* hdr = reinterpret_cast<const int*>(a.ws);
  const SeqInfo si = seq_info(a, s, 1);
  if (!si.ok && seg == 0 && tid == 0 && blockIdx.z == 0) set_status(a.status, CO_ERR_LENGTH);
  const int T1 = hdr[a.S];
  const int nts = hdr[s + 1] - hdr[s];
  uint16_t* out = static_cast<uint16_t*>(a.out);
  if (nts == 0) {                      // no keys: O = 0, LSE = -inf
    for (int idx = tid + blockIdx.z * 256; idx < nq * hd; idx += 256 * gridDim.z)
      out[out_row(a, layer_local, s, g, idx / hd, G) * hd + idx % hd] = 0;
    if (a.lse && blockIdx.z == 0)
      for (int qn = tid; qn < nq; qn += 256) a.lse[out_row(a, layer_local, s, g, qn, G)] = -INFINITY;
    return;
  }
  const int64_t A = static_cast<int64_t>(seg) * T1 + hdr[s];
  const int64_t* bounds = reinterpret_cast<const int64_t*>(hdr + slice_bounds_off(a.S));
  // slice w holds global tiles [bounds[w], bounds[w+1]); find the owners of the
  // segment's first and last tile (bounds is non-decreasing)
  auto owner = [&](int64_t x) {
    int lo = 0, hi = n_wg;                  // bounds[lo] <= x < bounds[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (bounds[mid] <= x) lo = mid; else hi = mid;
    }
    return lo;
  };
  const int w_lo = owner(A), w_hi = owner(A + nts - 1);
  if (w_lo == w_hi) return;            // finished in place
  const int nrec = w_hi - w_lo + 1;
  __shared__ float live_lds[kMaxMergeSlices];
  for (int i = tid; i < nrec; i += 256)   // an empty slice left no record
    live_lds[i] = bounds[w_lo + i] < bounds[w_lo + i + 1] ? 1.f : 0.f;
  __syncthreads();
  const int64_t rec = static_cast<int64_t>(nq_pad) * (hd + 2);
  // records of consecutive slices of one segment are consecutive slots
  const float* base = slot_ptr(a, hdr_floats, w_lo + static_cast<int64_t>(seg) * a.S + s, nq_pad);
  for (int idx = tid + blockIdx.z * 256; idx < nq * q4; idx += 256 * gridDim.z) {
    const int qn = idx / q4, d = (idx % q4) * 4;
    const float* pm = base + nq_pad * hd + qn;
    float M = -INFINITY;
    for (int r0 = 0; r0 < nrec; r0 += kBatch) {
      float mv[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) mv[i] = r0 + i < nrec ? pm[(r0 + i) * rec] : -INFINITY;
#pragma unroll
      for (int i = 0; i < kBatch; ++i)
        if (r0 + i < nrec && live_lds[r0 + i] != 0.f) M = fmaxf(M, mv[i]);
    }
    float den = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int r0 = 0; r0 < nrec; r0 += kBatch) {
      float mv[kBatch], lv[kBatch];
      f32x4 ov[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const bool in = r0 + i < nrec;
        mv[i] = in ? pm[(r0 + i) * rec] : -INFINITY;
        lv[i] = in ? pm[(r0 + i) * rec + nq_pad] : 0.f;
        ov[i] = in ? *reinterpret_cast<const f32x4*>(base + (r0 + i) * rec + qn * hd + d)
                   : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const bool live = r0 + i < nrec && live_lds[r0 + i] != 0.f;
        const float wgt = (!live || mv[i] == -INFINITY) ? 0.f : exp2f(mv[i] - M);
        den += wgt * lv[i];
        acc += wgt * ov[i];
      }
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const int64_t row = out_row(a, layer_local, s, g, qn, G);
    u16x4 v;
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = f2bf(acc[r] * inv);
    *reinterpret_cast<u16x4*>(out + row * hd + d) = v;
    if (a.lse && d == 0) a.lse[row] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
  }
}

}  // namespace

AttnPlan plan_attention(int S, int B, int L, int Hq, int Hkv, int hd, int max_pages, int dtype,
                        int num_cus) {
  AttnPlan p{};
  const int nq = B * (Hq / Hkv);
  p.nq_pad = (nq + 15) / 16 * 16;
  const int cp = (B + kPage - 1) / kPage;
  const int max_lp = max_pages + cp;
  p.ok = true;
  if (dtype == CO_DTYPE_BF16) {
    // persistent path: a fixed number of workgroups per CU, records for
    // (slice, segment) pairs
    p.variant = 1;
    if (const char* env = getenv("CO_ATTN_VARIANT")) p.variant = atoi(env) & 3;   // tuning
    p.n_wg = num_cus * (p.variant == 1 && hd == 64 ? 2 : 1);
    p.hdr_floats = (slice_bounds_off(S) + 2 * (p.n_wg + 1) + 63) / 64 * 64;
    p.ok = S <= kMaxAttnSeqs && p.n_wg <= kMaxMergeSlices;
    p.bytes = (static_cast<size_t>(p.hdr_floats) +
               (static_cast<size_t>(p.n_wg) + static_cast<size_t>(L) * Hkv * S) * p.nq_pad *
                   (hd + 2)) * 4;
  } else {
    // fp32 path: chunks of pages, one workgroup each
    p.chunk_pages = 32;
    while ((max_lp + p.chunk_pages - 1) / p.chunk_pages > kMaxMergeChunks) p.chunk_pages *= 2;
    p.ok = p.chunk_pages <= kMaxChunkPages;
    p.n_chunks = (max_lp + p.chunk_pages - 1) / p.chunk_pages;
    p.bytes = static_cast<size_t>(L) * S * Hkv * p.n_chunks * p.nq_pad * (hd + 2) * 4;
  }
  p.bytes = (p.bytes + 255) / 256 * 256;
  return p;
}

hipError_t launch_attention(const AttnArgs& a, const AttnPlan& p, int layer_count,
                            hipStream_t stream) {
  if (a.S == 0 || layer_count == 0) return hipSuccess;
  const int nt = p.nq_pad / 16;
  const int items = (a.B * (a.Hq / a.Hkv)) * (a.hd / 4);
  const dim3 mgrid(a.S, layer_count * a.Hkv, (items + 255) / 256);
  if (a.dtype == CO_DTYPE_BF16) {
    const dim3 grid(p.n_wg);
#define CO_ATTN_LAUNCH(HD, NT, NW, NS)                                                         \
  hipLaunchKernelGGL((attn_bf16_kernel<HD, NT, NW, NS>), grid, dim3(64 * NW), 0, stream, a,     \
                     layer_count, p.n_wg, p.hdr_floats)
    if (a.hd == 64 && nt == 2 && p.variant == 0) {
      CO_ATTN_LAUNCH(64, 2, 4, 4);
    } else if (a.hd == 64 && nt == 2 && p.variant == 2) {
      CO_ATTN_LAUNCH(64, 2, 8, 2);
    } else if (a.hd == 64) {
      switch (nt) {
        case 1: CO_ATTN_LAUNCH(64, 1, 4, 2); break;
        case 2: CO_ATTN_LAUNCH(64, 2, 4, 2); break;
        case 3: CO_ATTN_LAUNCH(64, 3, 4, 2); break;
        default: CO_ATTN_LAUNCH(64, 4, 4, 2); break;
      }
    } else {
      switch (nt) {
        case 1: CO_ATTN_LAUNCH(128, 1, 2, 3); break;
        case 2: CO_ATTN_LAUNCH(128, 2, 2, 3); break;
        case 3: CO_ATTN_LAUNCH(128, 3, 2, 3); break;
        default: CO_ATTN_LAUNCH(128, 4, 2, 3); break;
      }
    }
#undef CO_ATTN_LAUNCH
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(attn_bf16_combine_kernel, mgrid, dim3(256), 0, stream, a, layer_count,
                       p.n_wg, p.hdr_floats, p.nq_pad);
    return hipGetLastError();
  }
  const dim3 grid(p.n_chunks, a.S, layer_count * a.Hkv);
  if (a.hd == 64)
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  else
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.n_chunks <= 1) return err;
  hipLaunchKernelGGL(attn_chunk_merge_kernel<float>, mgrid, dim3(256), 0, stream, a, p.chunk_pages,
                     p.n_chunks, p.nq_pad);
  return hipGetLastError();
}

}  // namespace co
