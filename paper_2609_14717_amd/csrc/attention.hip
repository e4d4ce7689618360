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
#include <string.h>

#include <algorithm>

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
constexpr int kCombineWideSegs = 128;   // segments from which the merge takes 16 dims per thread
constexpr int kAttnWaves64 = 8, kAttnWaves128 = 4;             // wavefronts per workgroup
constexpr int kAttnRoundTiles64 = 64, kAttnRoundTiles128 = 128; // tiles per wavefront per round

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
      rope_cos_sin(ctx + n / G, a.rope_inv[p], &cs, &sn);
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
    // stage 32 keys (two logical pages): resolve both pages first, then issue
    // every element load of the tile before any is used
    const float* kp[2];
    const float* vp[2];
    int nvalid[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int lp = lp0 + q;
      kp[q] = vp[q] = nullptr;
      nvalid[q] = 0;
      if (lp >= p_end) continue;
      if (lp < npc) {
        const int phys = a.page_table[static_cast<int64_t>(s) * a.max_pages + lp];
        if (phys >= 0 && phys < a.num_pages) {
          const int64_t off =
              ((static_cast<int64_t>(layer) * a.num_pages + phys) * a.Hkv + g) * kPage * HD;
          kp[q] = kc + off;
          vp[q] = vc + off;
          nvalid[q] = min(kPage, ctx - lp * kPage);
        } else if (tid == 0) {
          set_status(a.status, CO_ERR_PAGE_RANGE);
        }
      } else {
        const int cp = lp - npc;
        const int64_t off =
            (((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp) * a.Hkv + g) * kPage * HD;
        kp[q] = kk + off;
        vp[q] = vk + off;
        nvalid[q] = min(kPage, carry - cp * kPage);
      }
    }
    constexpr int PER = KT * HD / 256;   // elements of the tile staged per thread
    float kr[PER], vr[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = tid + e * 256, key = idx / HD, dd = idx % HD;
      const int q = key >> 4, slot = key & 15;
      const bool ok = slot < nvalid[q];
      kr[e] = ok ? kp[q][slot * HD + dd] : 0.f;
      vr[e] = ok ? vp[q][dd * kPage + slot] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int idx = tid + e * 256, key = idx / HD, dd = idx % HD;
      ks[key][dd] = kr[e];
      vs[key][dd] = vr[e];
      if (dd == 0) kvalid[key] = (key & 15) < nvalid[key >> 4];
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
//
// The key tiles (32 keys = two logical pages) of all segments form one global
// order: segment (layer_local * Hkv + g) major, then sequence, then tile
// (committed pages first, then carry pages).  Global tile indices fit in int32
// (checked on the host).  Workgroup w owns the slice [T*w/n_wg, T*(w+1)/n_wg).
//
// Workspace of this path:
//   header (ints): tstart[S+1], the tiles before each sequence within a segment
//     (written by workgroup 0), then bounds[n_wg+1], the first tile of every
//     slice (each written by its workgroup);
//   records: one per (slice w, segment sigma = seg*S + s) pair, at slot
//     w + sigma -- injective over the pairs that occur because slices and
//     segments both follow the tile order: O[NQP][hd] unnormalised, m[NQP],
//     l[NQP] (m in log2 units of the scaled logits);
//   parked partials (large query tiles only): one record-shaped area per
//     wavefront, for a piece that another wavefront of the workgroup merges.

__device__ __forceinline__ float* slot_ptr(const AttnArgs& a, int hdr_floats, int64_t slot,
                                           int nqp) {
  return a.ws + hdr_floats + slot * nqp * (a.hd + a.rec_sums);
}

// The block's own rows (drafter_block_attention_ext) as 32-key tiles of a
// (layer, KV head, sequence): rows t0 .. t0 + 31 of k_self / v_self
// [layers][S][B][Hkv][HD] are loaded by the wavefront as lane jobs (keys: a row
// and the rotation pair of 16-byte chunks c, c + CPR/2; values: a row and a
// chunk), then written into a ring slot in the layout of a cached tile: keys
// rotated at ctx + row (as the queries are) with the slot's XOR swizzle,
// values transposed into the [HD][16] pages.  Rows past B are zero.
template <int HD>
struct SelfRows {
  static constexpr int ROWB = HD * 2, CPR = ROWB / 16, PAGE_BYTES = kPage * ROWB;
  static constexpr int KJ = (32 * CPR / 2) / 64, VJ = (32 * CPR) / 64;   // lane jobs
  u16x8 lo[KJ], hi[KJ], v8[VJ];

  __device__ void load(const AttnArgs& a, int s, int layer_local, int g, int t0, int lane) {
    const int64_t rs = static_cast<int64_t>(a.Hkv) * HD;   // row stride
    const int64_t base = ((static_cast<int64_t>(layer_local) * a.S + s) * a.B * a.Hkv + g) * HD;
    const uint16_t* ks = static_cast<const uint16_t*>(a.k_self) + base;
    const uint16_t* vs = static_cast<const uint16_t*>(a.v_self) + base;
#pragma unroll
    for (int i = 0; i < KJ; ++i) {
      const int jb = lane + 64 * i, row = t0 + jb / (CPR / 2), c = jb % (CPR / 2);
      lo[i] = hi[i] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
      if (row < a.B) {
        lo[i] = *reinterpret_cast<const u16x8*>(ks + row * rs + c * 8);
        hi[i] = *reinterpret_cast<const u16x8*>(ks + row * rs + c * 8 + HD / 2);
      }
    }
#pragma unroll
    for (int i = 0; i < VJ; ++i) {
      const int jb = lane + 64 * i, row = t0 + jb / CPR, c = jb % CPR;
      v8[i] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
      if (row < a.B) v8[i] = *reinterpret_cast<const u16x8*>(vs + row * rs + c * 8);
    }
  }

  // inv_rev: RoPE inverse frequencies in revolutions per position
  __device__ void store(unsigned char* slot, int t0, int ctx, int lane, const double* inv_rev) {
#pragma unroll
    for (int i = 0; i < KJ; ++i) {
      const int jb = lane + 64 * i, r = jb / (CPR / 2), c = jb % (CPR / 2);
      u16x8 x8 = lo[i], y8 = hi[i];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float cs, sn;
        rope_cos_sin_rev(ctx + t0 + r, inv_rev[c * 8 + e], &cs, &sn);
        const float x = bf2f(x8[e]), y = bf2f(y8[e]);
        x8[e] = f2bf(x * cs - y * sn);
        y8[e] = f2bf(y * cs + x * sn);
      }
      const int rp = r & 15;
      unsigned char* kpg = slot + (r >> 4) * PAGE_BYTES + rp * ROWB;
      *reinterpret_cast<u16x8*>(kpg + ((c ^ (rp & (CPR - 1))) << 4)) = x8;
      *reinterpret_cast<u16x8*>(kpg + (((c + CPR / 2) ^ (rp & (CPR - 1))) << 4)) = y8;
    }
#pragma unroll
    for (int i = 0; i < VJ; ++i) {
      const int jb = lane + 64 * i, r = jb / CPR, c = jb % CPR;
      uint16_t* vpg = reinterpret_cast<uint16_t*>(slot + (2 + (r >> 4)) * PAGE_BYTES);
#pragma unroll
      for (int e = 0; e < 8; ++e) vpg[(c * 8 + e) * kPage + (r & 15)] = v8[i][e];
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wavefront's own writes
  }
};

// The same rows staged through LDS instead of registers (for kernels with no
// registers to spare): raw rows land by direct-to-LDS loads in a free ring slot
// (keys [32][HD], then values [32][HD]; rows past B repeat row B - 1, their
// keys are masked by the caller), then are placed job by job into the slot of
// the tile layout.  The caller waits for the loads (vmcnt) between the two.
template <int HD>
__device__ void self_rows_raw(const AttnArgs& a, int s, int layer_local, int g, int t0, int lane,
                              uint32_t raw) {
  constexpr int ROWB = HD * 2, LOADS = 32 * ROWB / 1024;   // 1 KiB wavefront loads per half
  const int64_t rs = static_cast<int64_t>(a.Hkv) * HD;
  const int64_t base = ((static_cast<int64_t>(layer_local) * a.S + s) * a.B * a.Hkv + g) * HD;
  const uint16_t* ks = static_cast<const uint16_t*>(a.k_self) + base;
  const uint16_t* vs = static_cast<const uint16_t*>(a.v_self) + base;
#pragma unroll
  for (int q = 0; q < LOADS; ++q) {
    const int byte = q * 1024 + lane * 16, r = byte / ROWB, c = (byte % ROWB) / 16;
    const int64_t off = min(t0 + r, a.B - 1) * rs + c * 8;
    lds_dma16_opaque(ks + off, raw + q * 1024);
    lds_dma16_opaque(vs + off, raw + (LOADS + q) * 1024);
  }
}

template <int HD>
__device__ void self_rows_place(const unsigned char* raw, unsigned char* slot, int t0, int ctx,
                                int lane, const double* inv_rev) {
  constexpr int ROWB = HD * 2, CPR = ROWB / 16, PAGE_BYTES = kPage * ROWB;
  constexpr int KJ = (32 * CPR / 2) / 64, VJ = (32 * CPR) / 64;
  const unsigned char* rv = raw + 32 * ROWB;
#pragma unroll 2
  for (int i = 0; i < KJ; ++i) {
    const int jb = lane + 64 * i, r = jb / (CPR / 2), c = jb % (CPR / 2);
    u16x8 x8 = *reinterpret_cast<const u16x8*>(raw + r * ROWB + c * 16);
    u16x8 y8 = *reinterpret_cast<const u16x8*>(raw + r * ROWB + (c + CPR / 2) * 16);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float cs, sn;
      rope_cos_sin_rev(ctx + t0 + r, inv_rev[c * 8 + e], &cs, &sn);
      const float x = bf2f(x8[e]), y = bf2f(y8[e]);
      x8[e] = f2bf(x * cs - y * sn);
      y8[e] = f2bf(y * cs + x * sn);
    }
    const int rp = r & 15;
    unsigned char* kpg = slot + (r >> 4) * PAGE_BYTES + rp * ROWB;
    *reinterpret_cast<u16x8*>(kpg + ((c ^ (rp & (CPR - 1))) << 4)) = x8;
    *reinterpret_cast<u16x8*>(kpg + (((c + CPR / 2) ^ (rp & (CPR - 1))) << 4)) = y8;
  }
#pragma unroll 2
  for (int i = 0; i < VJ; ++i) {
    const int jb = lane + 64 * i, r = jb / CPR, c = jb % CPR;
    const u16x8 v8 = *reinterpret_cast<const u16x8*>(rv + r * ROWB + c * 16);
    uint16_t* vpg = reinterpret_cast<uint16_t*>(slot + (2 + (r >> 4)) * PAGE_BYTES);
#pragma unroll
    for (int e = 0; e < 8; ++e) vpg[(c * 8 + e) * kPage + (r & 15)] = v8[e];
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wavefront's own writes
}

// The part of one segment that lies in one slice (global tile indices).
struct Piece {
  int seg_begin, seg_end;   // the segment
  int begin, end;           // the piece
  int s, seg, ctx, carry;
};

template <int N>
__device__ __forceinline__ int pick_reg(const int (&v)[N], int i) {
  int r = v[0];
#pragma unroll
  for (int k = 1; k < N; ++k) r = (i == k) ? v[k] : r;
  return r;
}

template <int HD, int NT, int NW, int NS, int PQ, int RTM, bool EXT>
__global__ __launch_bounds__(64 * NW) void attn_bf16_kernel(AttnArgs a, int layer_count, int n_wg,
                                                             int hdr_floats, int round_tiles,
                                                             int64_t park_off) {
  constexpr int KS = HD / 32;              // k-steps of S^T
  constexpr int MT = HD / 16;              // M-tiles of O^T
  constexpr int NQP = NT * 16;
  constexpr int NTHR = 64 * NW;
  constexpr int QLD = HD + 8;              // padded LDS row of rotated queries (bf16)
  constexpr int QSZ = NQP * QLD;
  constexpr int ROWB = HD * 2;             // bytes of one key row
  constexpr int CPR = ROWB / 16;           // 16-byte chunks per key row
  constexpr int PAGE_BYTES = kPage * ROWB; // one page of K (or of V)
  constexpr int LPP = PAGE_BYTES / 1024;   // 1 KiB wave loads per page
  constexpr int TILE_BYTES = 4 * PAGE_BYTES;   // K page 0, K page 1, V page 0, V page 1
  constexpr int NL = 4 * LPP;              // direct-to-LDS loads per tile per wave
  constexpr int RING_BYTES = NW * NS * TILE_BYTES;
  constexpr int SLOT_LD = HD + 4;          // 16-byte aligned rows
  // per query row: m, l (and, with EXT, the sums over carry keys and self keys)
  constexpr int NSUM = EXT ? 4 : 2;
  constexpr int RECW = HD + NSUM;          // floats per query row of a record or parked partial
  constexpr int SLOT_FLOATS = NQP * SLOT_LD + NSUM * NQP;
  constexpr bool PARK_REGS = HD * NT <= 128;   // parked partial fits in 32 registers
  constexpr int RQ = RTM / 32;             // page-descriptor registers (64 pages each)
  constexpr int PMAX = 64;                 // pieces enumerated per pass
  constexpr int QV = (PQ * NQP * (HD / 8) + NTHR - 1) / NTHR;   // 4-pair query groups per thread
  constexpr int SPT = (kMaxAttnSeqs + NTHR - 1) / NTHR;         // sequences per thread (max)
  static_assert(NL * (NS - 1) < 64, "vmcnt");
  static_assert(!PARK_REGS || NW * SLOT_FLOATS * 4 <= RING_BYTES, "merge slots");
  static_assert((5 * kMaxAttnSeqs + 2) * 4 <= RING_BYTES, "set-up arrays");
  static_assert(RTM % 32 == 0 && PQ <= PMAX, "round shape");
  // the ring; the set-up arrays and the merge slots overlay it
  __shared__ __align__(16) unsigned char smem[RING_BYTES];
  __shared__ __align__(16) uint16_t q_lds[PQ * QSZ];
  __shared__ Piece pc[PMAX];
  __shared__ double inv_lds[HD / 2];
  __shared__ int scan_tot[2 * NW];
  __shared__ int next_rot, first_seq;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = lane >> 4, col = lane & 15;
  const int S = a.S, G = a.Hq / a.Hkv, nq = a.B * G;
  const int w = blockIdx.x;
  const int n_segs = layer_count * a.Hkv;
  int* tstart = reinterpret_cast<int*>(smem);   // [S+1]
  int* nstart = tstart + (S + 1);               // [S+1] non-empty sequences before s
  int* ne_seq = nstart + (S + 1);               // [S]   the k-th non-empty sequence
  int* ctx_s = ne_seq + S;                      // [S]
  int* carry_s = ctx_s + S;                     // [S]

  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* vc = static_cast<const uint16_t*>(a.v_cache);
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);
  const uint16_t* vk = static_cast<const uint16_t*>(a.v_carry);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;
  const uint16_t* Q = static_cast<const uint16_t*>(a.q);
  const bool rotate_q = !(a.flags & CO_Q_PREROTATED);
  if (tid < HD / 2)   // in revolutions per position
    inv_lds[tid] = a.rope_inv[tid] * kInv2Pi;
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
    const int ra_ = key_a & 15, rb_ = key_b & 15;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int ch = ks * 4 + grp;
      ka_off[ks] = (key_a >> 4) * PAGE_BYTES + ra_ * ROWB + ((ch ^ (ra_ & (CPR - 1))) << 4);
      kb_off[ks] = (key_b >> 4) * PAGE_BYTES + rb_ * ROWB + ((ch ^ (rb_ & (CPR - 1))) << 4);
    }
    v_frag_off = (2 + (grp >> 1)) * PAGE_BYTES + col * 32 + slot_base * 2;
  }
  // Running maxima are kept as a lazily updated reference: p = 2^(s - ref) may
  // exceed 1 by up to 2^kRescale before the accumulators are rescaled, which
  // leaves the normalised result unchanged and skips most rescales.
  constexpr float kRescale = 8.f;

  f32x4 o[MT][NT];
  float m_run[NT], l_run[NT];   // l_run: per-lane partial sums (reduce across groups to use)
  f32x4 o_pk[PARK_REGS ? MT : 1][PARK_REGS ? NT : 1];
  float m_pk[NT], l_pk[NT];
  // EXT: running sums over the carry keys (lu) and the block's own keys (ls),
  // on the same reference maximum as l_run
  float lu_run[NT], ls_run[NT], lu_pk[NT], ls_pk[NT];
  u16x8 qf[NT][KS];
  auto reset = [&]() {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) o[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      m_run[nt] = -INFINITY;
      l_run[nt] = 0.f;
      lu_run[nt] = 0.f;
      ls_run[nt] = 0.f;
    }
  };
  // queries of round piece slot j into the MFMA B fragments (after DMA has begun)
  auto load_q = [&](int j) {
    const uint16_t* qb = q_lds + j * QSZ;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      uint32_t ad[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        ad[ks] = lds_addr(reinterpret_cast<const unsigned char*>(qb + (nt * 16 + col) * QLD + ks * 32 + grp * 8));
      lds_read_group<KS>(qf[nt], ad);
    }
  };
  // a piece this wavefront merged completely: final output, or a slice record
  auto emit = [&](bool whole, int s, int seg, const float (&l_tot)[NT], const float (&lu_tot)[NT],
                  const float (&ls_tot)[NT]) {
    const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
    if (whole) {
      uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int qn = nt * 16 + col;
        if (qn >= nq) continue;
        const float inv = l_tot[nt] > 0.f ? 1.f / l_tot[nt] : 0.f;
        const int64_t row = out_row(a, layer_local, s, g, qn, G);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          u16x4 v;
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = f2bf(o[mt][nt][r] * inv);
          *reinterpret_cast<u16x4*>(out + row * HD + mt * 16 + grp * 4) = v;
        }
        if (a.lse && grp == 0)
          a.lse[row] = l_tot[nt] > 0.f ? (m_run[nt] + log2f(l_tot[nt])) * kLn2 : -INFINITY;
        if constexpr (EXT) {
          // share of the attention over [C;U] (the self keys left out) on U
          const float lcu = l_tot[nt] - ls_tot[nt];
          if (a.mass && grp == 0) a.mass[row] = lcu > 0.f ? lu_tot[nt] / lcu : 0.f;
        }
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
          part[NQP * HD + NQP + qn] = l_tot[nt];
          if constexpr (EXT) {
            part[NQP * HD + 2 * NQP + qn] = lu_tot[nt];
            part[NQP * HD + 3 * NQP + qn] = ls_tot[nt];
          }
        }
      }
    }
  };
  // fold a parked partial (O[NQP][ld], m[NQP], l[NQP]) into the accumulators
  auto absorb = [&](const float* p, int ld) {
    f32x4 po[MT][NT];
    float mo[NT], lo[NT], luo[NT], lso[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {   // one round trip for the whole partial
      const int qn = nt * 16 + col;
      mo[nt] = p[NQP * ld + qn];
      lo[nt] = p[NQP * ld + NQP + qn];
      if constexpr (EXT) {
        luo[nt] = p[NQP * ld + 2 * NQP + qn];
        lso[nt] = p[NQP * ld + 3 * NQP + qn];
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        po[mt][nt] = *reinterpret_cast<const f32x4*>(p + qn * ld + mt * 16 + grp * 4);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      // arguments are <= 0 or -inf: the hardware exp2 is exact enough and gives 0 at -inf
      const float M = fmaxf(m_run[nt], mo[nt]);
      const float f0 = (m_run[nt] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run[nt] - M);
      const float f1 = (mo[nt] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mo[nt] - M);
      // l_run stays a per-lane partial; the parked row total joins lane group 0
      l_run[nt] = l_run[nt] * f0 + (grp == 0 ? lo[nt] * f1 : 0.f);
      if constexpr (EXT) {
        lu_run[nt] = lu_run[nt] * f0 + (grp == 0 ? luo[nt] * f1 : 0.f);
        ls_run[nt] = ls_run[nt] * f0 + (grp == 0 ? lso[nt] * f1 : 0.f);
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) o[mt][nt] = o[mt][nt] * f0 + po[mt][nt] * f1;
      m_run[nt] = M;
    }
  };

  reset();
  bool carrying = false;   // this wavefront holds a piece continued from the previous round
  int rot = 0;             // wavefront that takes the first sub-slice of a round
  int r0 = 0, r1 = 0;
  for (int pass_begin = -1;;) {
    if (pass_begin >= r1) break;                        // after the last pass
    // ---- per-sequence tiles, their prefix sums and the non-empty sequences
    __syncthreads();                                    // smem is reused
    int T1, NE, seg0;
    {
      const int per = (S + NTHR - 1) / NTHR, s0 = tid * per;
      int nts[SPT], cx[SPT], cr[SPT];
      int tl = 0, nl = 0;
#pragma unroll
      for (int i = 0; i < SPT; ++i) {
        nts[i] = cx[i] = cr[i] = 0;
        if (i < per && s0 + i < S) {
          const SeqInfo q = seq_info(a, s0 + i, 1);
          nts[i] = (q.npt + 1) / 2;
          if (EXT && a.k_self && q.ok && nts[i] == 0) nts[i] = 1;   // its self keys follow the tile
          cx[i] = q.ctx;
          cr[i] = q.carry;
          tl += nts[i];
          nl += nts[i] > 0;
        }
      }
      int vt = tl, vn = nl;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int ut = __shfl_up(vt, off), un = __shfl_up(vn, off);
        if (lane >= off) {
          vt += ut;
          vn += un;
        }
      }
      if (lane == 63) {
        scan_tot[wave] = vt;
        scan_tot[NW + wave] = vn;
      }
      __syncthreads();
      int rt = vt - tl, rn = vn - nl;
      T1 = 0;
      NE = 0;
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        if (v < wave) {
          rt += scan_tot[v];
          rn += scan_tot[NW + v];
        }
        T1 += scan_tot[v];
        NE += scan_tot[NW + v];
      }
      const int T = n_segs * T1;
      if (pass_begin < 0) {
        const int64_t tw1 = static_cast<int64_t>(T) * (w + 1);
        if (tw1 <= 0xFFFFFFFFll) {   // 32-bit divisions
          r0 = static_cast<int>(static_cast<uint32_t>(tw1 - T) / static_cast<uint32_t>(n_wg));
          r1 = static_cast<int>(static_cast<uint32_t>(tw1) / static_cast<uint32_t>(n_wg));
        } else {
          r0 = static_cast<int>((tw1 - T) / n_wg);
          r1 = static_cast<int>(tw1 / n_wg);
        }
        int* hdr = reinterpret_cast<int*>(a.ws);
        if (tid == 0) {
          hdr[S + 1 + w + 1] = r1;
          if (w == 0) {
            hdr[S + 1] = 0;
            hdr[S] = T1;
          }
        }
        if (w == 0) {
          int x = rt;
#pragma unroll
          for (int i = 0; i < SPT; ++i)
            if (i < per && s0 + i < S) {
              hdr[s0 + i] = x;
              x += nts[i];
            }
        }
        pass_begin = r0;
        if (r0 >= r1) break;                            // an empty slice
      }
      seg0 = pass_begin / T1;
      const int rr = pass_begin - seg0 * T1;
#pragma unroll
      for (int i = 0; i < SPT; ++i)
        if (i < per && s0 + i < S) {
          tstart[s0 + i] = rt;
          nstart[s0 + i] = rn;
          ctx_s[s0 + i] = cx[i];
          carry_s[s0 + i] = cr[i];
          if (nts[i]) ne_seq[rn] = s0 + i;
          if (rt <= rr && rr < rt + nts[i]) first_seq = s0 + i;
          rt += nts[i];
          rn += nts[i] > 0;
        }
      if (tid == NTHR - 1) tstart[S] = rt;
      __syncthreads();
    }

    // ---- the next (up to PMAX) pieces of the slice, from pass_begin
    if (tid < PMAX) {
      const int gp = seg0 * NE + nstart[first_seq] + tid;   // global index of its segment
      Piece p;
      p.seg_begin = p.seg_end = p.begin = p.end = r1;
      p.s = p.seg = p.ctx = p.carry = 0;
      const int seg = gp / NE;
      if (seg < n_segs) {
        const int s = ne_seq[gp - seg * NE];
        p.seg_begin = seg * T1 + tstart[s];
        p.seg_end = seg * T1 + tstart[s + 1];
        p.begin = max(p.seg_begin, pass_begin);
        p.end = min(p.seg_end, r1);
        p.s = s;
        p.seg = seg;
        p.ctx = ctx_s[s];
        p.carry = carry_s[s];
        if (p.begin >= p.end) p.begin = p.end = r1;
      }
      pc[tid] = p;
    }
    __syncthreads();
    const int n_p = __popcll(__ballot(lane < PMAX && pc[lane].begin < pc[lane].end));
    const int pass_end = pc[n_p - 1].end;

    for (int ra = pass_begin, pa = 0; ra < pass_end;) {
      // ---- the round [ra, rb): pieces [pa, pb), at most PQ of them
      int rb = min(pass_end, ra + NW * round_tiles);
      if (pa + PQ < n_p) rb = min(rb, pc[pa + PQ].begin);
      int pb = pa + 1;
      while (pb < n_p && pc[pb].begin < rb) ++pb;
      const int nr = rb - ra;

      // this wavefront's sub-slice [sb, se) and the descriptors of its pages:
      // row >= 0 committed K/V row, -1-r carry row r, INT_MIN nothing to read
      const int k = (wave - rot + NW) % NW;
      const int sb = ra + static_cast<int>(static_cast<int64_t>(nr) * k / NW);
      const int se = ra + static_cast<int>(static_cast<int64_t>(nr) * (k + 1) / NW);
      int pg_row[RQ], pg_nv[RQ];
      int pt[RQ], pidx[RQ], lpv[RQ];
      {
#pragma unroll
        for (int q = 0; q < RQ; ++q) {   // page-table loads first
          const int jp = lane + 64 * q, t = sb + (jp >> 1);
          int i = pa;
          while (i + 1 < pb && pc[i].end <= t) ++i;
          pidx[q] = i;
          lpv[q] = 2 * (t - pc[i].seg_begin) + (jp & 1);
          const bool com = t < se && lpv[q] < (pc[i].ctx + kPage - 1) / kPage;
          pt[q] = a.page_table[com ? static_cast<int64_t>(pc[i].s) * a.max_pages + lpv[q] : 0];
        }
      }
      // stage the queries of the round's pieces, rotated at ctx + i and scaled
      {
        u16x4 qlo[QV], qhi[QV];
#pragma unroll
        for (int i = 0; i < QV; ++i) {   // loads first: one round trip for all
          const int idx = tid + i * NTHR;
          const int j = idx / (NQP * (HD / 8)), rem = idx % (NQP * (HD / 8));
          const int qn = rem / (HD / 8), p4 = (rem % (HD / 8)) * 4;
          int64_t off = 0;
          if (j < pb - pa && qn < nq) {
            const Piece& P = pc[pa + j];
            off = out_row(a, P.seg / a.Hkv, P.s, P.seg % a.Hkv, qn, G) * HD + p4;
          }
          qlo[i] = *reinterpret_cast<const u16x4*>(Q + off);
          qhi[i] = *reinterpret_cast<const u16x4*>(Q + off + HD / 2);
        }
#pragma unroll
        for (int i = 0; i < QV; ++i) {
          const int idx = tid + i * NTHR;
          const int j = idx / (NQP * (HD / 8)), rem = idx % (NQP * (HD / 8));
          const int qn = rem / (HD / 8), p4 = (rem % (HD / 8)) * 4;
          if (j >= pb - pa) continue;
          const bool live = qn < nq;
          const int pos = pc[pa + j].ctx + qn / G;
          u16x4 lo4, hi4;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float x = live ? bf2f(qlo[i][e]) : 0.f, y = live ? bf2f(qhi[i][e]) : 0.f;
            if (rotate_q) {
              float cs, sn;
              rope_cos_sin_rev(pos, inv_lds[p4 + e], &cs, &sn);
              const float x2 = x * cs - y * sn, y2 = y * cs + x * sn;
              x = x2;
              y = y2;
            }
            lo4[e] = f2bf(x * qscale);
            hi4[e] = f2bf(y * qscale);
          }
          uint16_t* dst = q_lds + j * QSZ + qn * QLD + p4;
          *reinterpret_cast<u16x4*>(dst) = lo4;
          *reinterpret_cast<u16x4*>(dst + HD / 2) = hi4;
        }
      }

      {
#pragma unroll
        for (int q = 0; q < RQ; ++q) {
          const int t = sb + ((lane + 64 * q) >> 1);
          const Piece& P = pc[pidx[q]];
          const int lp = lpv[q];
          const int npc = (P.ctx + kPage - 1) / kPage, npt = npc + (P.carry + kPage - 1) / kPage;
          const int layer = a.layer_begin + P.seg / a.Hkv, g = P.seg % a.Hkv;
          int row = INT_MIN, nv = 0;
          if (t < se && lp < npc) {
            const int phys = pt[q];
            if (phys >= 0 && phys < a.num_pages) {
              row = (layer * a.num_pages + phys) * a.Hkv + g;
              nv = min(kPage, P.ctx - lp * kPage);
            } else {
              set_status(a.status, CO_ERR_PAGE_RANGE);
            }
          } else if (t < se && lp < npt) {
            const int cp = lp - npc;
            row = -1 - (((layer * S + P.s) * a.CP + cp) * a.Hkv + g);
            nv = min(kPage, P.carry - cp * kPage);
          }
          pg_row[q] = row;
          pg_nv[q] = nv;
        }
      }
      // fields of the round's pieces, lane i for piece pa + i
      int f_beg = 0, f_end = 0, f_sbeg = 0, f_send = 0, f_s = 0, f_seg = 0;
      if (lane < pb - pa) {
        const Piece& P = pc[pa + lane];
        f_beg = P.begin;
        f_end = P.end;
        f_sbeg = P.seg_begin;
        f_send = P.seg_end;
        f_s = P.s;
        f_seg = P.seg;
      }

      // ---- stream the sub-slice
      const int ntw = se - sb;
      int pj = 0;                                       // current piece, relative to pa
      while (pj + 1 < pb - pa && __builtin_amdgcn_readlane(f_end, pj) <= sb) ++pj;
      int c_beg = __builtin_amdgcn_readlane(f_beg, pj), c_end = __builtin_amdgcn_readlane(f_end, pj);
      bool merger = carrying || sb == c_beg;
      bool holding = carrying;                          // accumulators hold a piece this wave merges
      bool parked = false;
      if (!carrying) reset();
      carrying = false;

      auto issue = [&](int jj) {
        unsigned char* dst = my_ring + (jj % NS) * TILE_BYTES;
        const int rv = pick_reg(pg_row, jj >> 5);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int row = __builtin_amdgcn_readlane(rv, (2 * jj + half) & 63);
          const uint16_t *kp = kk, *vp = vk;
          if (row >= 0) {
            kp = kc + static_cast<int64_t>(row) * (kPage * HD);
            vp = vc + static_cast<int64_t>(row) * (kPage * HD);
          } else if (row != INT_MIN) {
            kp = kk + static_cast<int64_t>(-1 - row) * (kPage * HD);
            vp = vk + static_cast<int64_t>(-1 - row) * (kPage * HD);
          }
#pragma unroll
          for (int q = 0; q < LPP; ++q) {
            lds_dma16(kp + k_off[q], dst + half * PAGE_BYTES + q * 1024);
            lds_dma16(vp + v_off[q], dst + (2 + half) * PAGE_BYTES + q * 1024);
          }
        }
      };
#pragma unroll
      for (int jj = 0; jj < NS - 1; ++jj)   // the first tiles load while the queries are staged
        if (jj < ntw) issue(jj);
      if (tid == 0) next_rot = -1;
      lds_barrier();                                    // queries staged
      if (ntw > 0) load_q(pj);

      // One 32-key tile from LDS (its two pages hold n0 and n1 valid keys):
      // S^T, the online softmax and O^T += V^T P^T.  kind: what this lane's
      // keys are (0 committed, 1 carry, 2 the block's own rows), for EXT sums.
      auto consume = [&](const unsigned char* tb, int n0, int n1, int kind) {
        const bool partial = n0 < kPage || n1 < kPage;      // wave-uniform
        const int nv = (grp >> 1) ? n1 : n0;   // valid slots of the page holding my keys
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
          f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            sa = mfma16x16x32(ka[ks], qf[nt][ks], sa);
            sb4 = mfma16x16x32(kb[ks], qf[nt][ks], sb4);
          }
          if (partial) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              sa[r] = (slot_base + r < nv) ? sa[r] : -INFINITY;
              sb4[r] = (slot_base + 4 + r < nv) ? sb4[r] : -INFINITY;
            }
          }
          float mx = fmaxf(fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3])),
                           fmaxf(fmaxf(sb4[0], sb4[1]), fmaxf(sb4[2], sb4[3])));
          mx = max_across_rows(mx);
          if (__any(mx > m_run[nt] + kRescale)) {
            // move the reference up (only where the tile exceeds it) and rescale
            const float m_new = mx > m_run[nt] + kRescale ? mx : m_run[nt];
            const float alpha = (m_new == m_run[nt]) ? 1.f : exp2f(m_run[nt] - m_new);
            l_run[nt] *= alpha;
            if constexpr (EXT) {
              lu_run[nt] *= alpha;
              ls_run[nt] *= alpha;
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) o[mt][nt] *= alpha;
            m_run[nt] = m_new;
          }
          const float base = (m_run[nt] == -INFINITY) ? 0.f : m_run[nt];
          float pa4[4], pb4[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {   // v_exp_f32: arguments are <= kRescale or -inf
            pa4[r] = __builtin_amdgcn_exp2f(sa[r] - base);
            pb4[r] = __builtin_amdgcn_exp2f(sb4[r] - base);
          }
          const float psum = (pa4[0] + pa4[1]) + (pa4[2] + pa4[3]) + (pb4[0] + pb4[1]) + (pb4[2] + pb4[3]);
          l_run[nt] += psum;
          if constexpr (EXT) {
            if (kind == 1) lu_run[nt] += psum;
            if (kind == 2) ls_run[nt] += psum;
          }
          typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
          const u32x4v pk32 = {pack_bf16x2(pa4[0], pa4[1]), pack_bf16x2(pa4[2], pa4[3]),
                               pack_bf16x2(pb4[0], pb4[1]), pack_bf16x2(pb4[2], pb4[3])};
          const u16x8 pk = __builtin_bit_cast(u16x8, pk32);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) o[mt][nt] = mfma16x16x32(va[mt], pk, o[mt][nt]);
        }

      };
      // EXT: this lane's keys in tile jj are carry keys (its page is a carry page)
      auto kind_of = [&](int jj) {
        if constexpr (EXT) {
          const int rv = pick_reg(pg_row, jj >> 5);
          const int row0 = __builtin_amdgcn_readlane(rv, (2 * jj) & 63);   // lane index uniform
          const int row1 = __builtin_amdgcn_readlane(rv, (2 * jj + 1) & 63);
          const int row = (grp >> 1) ? row1 : row0;
          return (row < 0 && row != INT_MIN) ? 1 : 0;
        } else {
          return 0;
        }
      };
      // EXT: the block's own rows of (layer, KV head, sequence) as 32-key
      // tiles in the ring slot just read, consumed like a cached tile
      // head_dim 64: the rows of the first segment that ends in this sub-slice
      // are loaded when the sub-slice starts, so that their round trip overlaps
      // the streaming of the tiles before that end
      constexpr bool PREF = EXT && HD == 64;
      SelfRows<HD> pre;
      int pre_end = -1;                                 // segment end the rows belong to
      auto self_tiles = [&](int s, int seg, int ctx, int seg_end, unsigned char* slot) {
        for (int t0 = 0; t0 < a.B; t0 += 32) {
          SelfRows<HD> rows;
          if (PREF && t0 == 0 && pre_end == seg_end)
            rows = pre;
          else
            rows.load(a, s, seg / a.Hkv, seg % a.Hkv, t0, lane);
          rows.store(slot, t0, ctx, lane, inv_lds);
          const int nb = a.B - t0;
          consume(slot, min(nb, kPage), max(0, min(nb - kPage, kPage)), 2);
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // read before the next rows land
        }
      };
      if constexpr (PREF) {
        if (a.k_self) {
          for (int i = pj; i < pb - pa; ++i) {           // wavefront-uniform
            if (__builtin_amdgcn_readlane(f_beg, i) >= se) break;
            const int send_i = __builtin_amdgcn_readlane(f_send, i);
            if (send_i <= se) {
              const int seg_i = __builtin_amdgcn_readlane(f_seg, i);
              pre.load(a, __builtin_amdgcn_readlane(f_s, i), seg_i / a.Hkv, seg_i % a.Hkv, 0, lane);
              pre_end = send_i;
              break;
            }
          }
        }
      }

      for (int j = 0; j < ntw; ++j) {
        if (j + NS - 1 < ntw) issue(j + NS - 1);
        const int t = sb + j;
        const int nvr = pick_reg(pg_nv, j >> 5);
        const int n0 = __builtin_amdgcn_readlane(nvr, (2 * j) & 63);
        const int n1 = __builtin_amdgcn_readlane(nvr, (2 * j + 1) & 63);
        wait_stages_ahead<NL, NS>(min(NS - 1, ntw - 1 - j));
        const unsigned char* tb = my_ring + (j % NS) * TILE_BYTES;
        if (t == c_beg && !carrying) holding = merger;

        consume(tb, n0, n1, kind_of(j));
        if constexpr (EXT) {
          // the segment's last tile: its self keys follow, in the slot just read
          if (a.k_self && t + 1 == __builtin_amdgcn_readlane(f_send, pj))
            self_tiles(__builtin_amdgcn_readlane(f_s, pj), __builtin_amdgcn_readlane(f_seg, pj),
                       pc[pa + pj].ctx, t + 1, my_ring + (j % NS) * TILE_BYTES);
        }
        // ---- the end of a piece, or of the sub-slice inside a piece
        if (t + 1 == c_end || j + 1 == ntw) {
          float l_tot[NT], lu_tot[NT], ls_tot[NT];
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            l_tot[nt] = wave_sum_across_groups(l_run[nt]);
            if constexpr (EXT) {
              lu_tot[nt] = wave_sum_across_groups(lu_run[nt]);
              ls_tot[nt] = wave_sum_across_groups(ls_run[nt]);
            }
          }
          const bool ends = t + 1 == c_end;
          if (merger && ends) {
            const int sbeg = __builtin_amdgcn_readlane(f_sbeg, pj);
            const int send = __builtin_amdgcn_readlane(f_send, pj);
            emit(c_beg == sbeg && c_end == send, __builtin_amdgcn_readlane(f_s, pj),
                 __builtin_amdgcn_readlane(f_seg, pj), l_tot, lu_tot, ls_tot);
            holding = false;
          } else if (!merger) {
            // the first piece of a sub-slice that began inside it: merged by the
            // wavefront that holds its beginning
            parked = true;
            if constexpr (PARK_REGS) {
#pragma unroll
              for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) o_pk[mt][nt] = o[mt][nt];
                m_pk[nt] = m_run[nt];
                l_pk[nt] = l_tot[nt];
                if constexpr (EXT) {
                  lu_pk[nt] = lu_tot[nt];
                  ls_pk[nt] = ls_tot[nt];
                }
              }
            } else {
              float* pp = a.ws + park_off + (static_cast<int64_t>(w) * NW + wave) * NQP * RECW;
#pragma unroll
              for (int nt = 0; nt < NT; ++nt) {
                const int qn = nt * 16 + col;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                  *reinterpret_cast<f32x4*>(pp + qn * HD + mt * 16 + grp * 4) = o[mt][nt];
                if (grp == 0) {
                  pp[NQP * HD + qn] = m_run[nt];
                  pp[NQP * HD + NQP + qn] = l_tot[nt];
                  if constexpr (EXT) {
                    pp[NQP * HD + 2 * NQP + qn] = lu_tot[nt];
                    pp[NQP * HD + 3 * NQP + qn] = ls_tot[nt];
                  }
                }
              }
            }
          } else {
            // merger whose piece goes on past the sub-slice: merged at the round's end
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              l_run[nt] = grp == 0 ? l_tot[nt] : 0.f;
              if constexpr (EXT) {
                lu_run[nt] = grp == 0 ? lu_tot[nt] : 0.f;
                ls_run[nt] = grp == 0 ? ls_tot[nt] : 0.f;
              }
            }
          }
          if (ends && j + 1 < ntw) {   // the next piece begins inside this sub-slice
            ++pj;
            c_beg = __builtin_amdgcn_readlane(f_beg, pj);
            c_end = __builtin_amdgcn_readlane(f_end, pj);
            merger = true;
            holding = true;
            reset();
            load_q(pj);
          }
        }
      }

      // ---- round end: merge the parked partials into the wavefront holding the piece
      __syncthreads();                                  // every ring is drained
      if constexpr (PARK_REGS) {
        if (parked) {
          float* sp = reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const int qn = nt * 16 + col;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              *reinterpret_cast<f32x4*>(sp + qn * SLOT_LD + mt * 16 + grp * 4) = o_pk[mt][nt];
            if (grp == 0) {
              sp[NQP * SLOT_LD + qn] = m_pk[nt];
              sp[NQP * SLOT_LD + NQP + qn] = l_pk[nt];
              if constexpr (EXT) {
                sp[NQP * SLOT_LD + 2 * NQP + qn] = lu_pk[nt];
                sp[NQP * SLOT_LD + 3 * NQP + qn] = ls_pk[nt];
              }
            }
          }
        }
      }
      __syncthreads();
      if (holding) {
        for (int k2 = k + 1; k2 < NW; ++k2) {
          const int sb2 = ra + static_cast<int>(static_cast<int64_t>(nr) * k2 / NW);
          const int se2 = ra + static_cast<int>(static_cast<int64_t>(nr) * (k2 + 1) / NW);
          if (sb2 >= c_end) break;
          if (sb2 == se2) continue;
          const int v2 = (k2 + rot) % NW;
          if constexpr (PARK_REGS)
            absorb(reinterpret_cast<const float*>(smem) + v2 * SLOT_FLOATS, SLOT_LD);
          else
            absorb(a.ws + park_off + (static_cast<int64_t>(w) * NW + v2) * NQP * RECW, HD);
        }
        if (c_end > rb) {
          if (lane == 0) next_rot = wave;               // goes on in the next round
        } else {
          float l_tot[NT], lu_tot[NT], ls_tot[NT];
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            l_tot[nt] = wave_sum_across_groups(l_run[nt]);
            if constexpr (EXT) {
              lu_tot[nt] = wave_sum_across_groups(lu_run[nt]);
              ls_tot[nt] = wave_sum_across_groups(ls_run[nt]);
            }
          }
          const int sbeg = __builtin_amdgcn_readlane(f_sbeg, pj);
          const int send = __builtin_amdgcn_readlane(f_send, pj);
          emit(c_beg == sbeg && c_end == send, __builtin_amdgcn_readlane(f_s, pj),
               __builtin_amdgcn_readlane(f_seg, pj), l_tot, lu_tot, ls_tot);
          holding = false;
        }
      }
      __syncthreads();                                  // slots consumed, next_rot visible
      const int nrot = next_rot;
      carrying = nrot >= 0 && wave == nrot;
      rot = nrot >= 0 ? nrot : 0;
      ra = rb;
      pa = (pc[pb - 1].end > rb) ? pb - 1 : pb;
    }
    pass_begin = pass_end;
  }
}

// Combine the slice records of every (layer, KV head, sequence) split across
// slices, write O/LSE of segments without keys, and report invalid lengths.
// One thread per (query row, DIMS output dims) merges the records: the row's
// maxima and sums and its DIMS partial dims of up to kBatch records are loaded
// at once, so a segment costs one round trip after the header loads.  Wide
// threads (16 dims) suit launches of many segments; with few segments, 4 dims
// per thread spread each segment over more workgroups.
template <int DIMS>
__global__ __launch_bounds__(256) void attn_bf16_combine_kernel(AttnArgs a, int layer_count,
                                                                int n_wg, int hdr_floats,
                                                                int nq_pad) {
  constexpr int kBatch = 8, kV = DIMS / 4;
  const int s = blockIdx.x, seg = blockIdx.y;
  const int layer_local = seg / a.Hkv, g = seg % a.Hkv;
  const int hd = a.hd, G = a.Hq / a.Hkv, nq = a.B * G, qd = hd / DIMS;
  const int tid = threadIdx.x;
  const int* hdr = reinterpret_cast<const int*>(a.ws);
  // slice w covers tiles [T w / n_wg, T (w + 1) / n_wg) of the T in the launch
  // (the launch records T after the slice starts)
  const int64_t T = hdr[a.S + 1 + n_wg];
  auto bnd = [&](int w) { return static_cast<int>(T * w / n_wg); };
  const SeqInfo si = seq_info(a, s, 1);
  if (!si.ok && seg == 0 && tid == 0 && blockIdx.z == 0) set_status(a.status, CO_ERR_LENGTH);
  const int T1 = hdr[a.S], ts = hdr[s];
  const int nts = hdr[s + 1] - ts;
  uint16_t* out = static_cast<uint16_t*>(a.out);
  if (nts == 0) {                      // no keys: O = 0, LSE = -inf
    for (int idx = tid + blockIdx.z * 256; idx < nq * hd; idx += 256 * gridDim.z)
      out[out_row(a, layer_local, s, g, idx / hd, G) * hd + idx % hd] = 0;
    if (a.lse && blockIdx.z == 0)
      for (int qn = tid; qn < nq; qn += 256) a.lse[out_row(a, layer_local, s, g, qn, G)] = -INFINITY;
    if (a.mass && blockIdx.z == 0)
      for (int qn = tid; qn < nq; qn += 256) a.mass[out_row(a, layer_local, s, g, qn, G)] = 0.f;
    return;
  }
  const int A = seg * T1 + ts;
  // owner of tile x: the last slice w with T w / n_wg <= x, i.e. the largest w
  // with T w < (x + 1) n_wg
  auto owner = [&](int x) {
    const int64_t w = ((static_cast<int64_t>(x) + 1) * n_wg + T - 1) / T - 1;
    return static_cast<int>(w < n_wg - 1 ? w : n_wg - 1);
  };
  // uniform over the workgroup: the record base below is a scalar pointer and
  // every load takes a 32-bit lane offset (fewer registers, more workgroups
  // resident per CU)
  const int w_lo = __builtin_amdgcn_readfirstlane(owner(A));
  const int w_hi = __builtin_amdgcn_readfirstlane(owner(A + nts - 1));
  if (w_lo == w_hi) return;            // finished in place
  const int nrec = w_hi - w_lo + 1;
  // with at least as many tiles as slices no slice is empty, so every slot in
  // [w_lo, w_hi] holds a record; otherwise an empty slice left none
  const bool all_full = T >= n_wg;
  const uint32_t rec = static_cast<uint32_t>(nq_pad) * (hd + a.rec_sums);
  const bool sums = a.rec_sums > 2;    // carry and self sums follow m and l
  // records of consecutive slices of one segment are consecutive slots
  const float* base = slot_ptr(a, hdr_floats, w_lo + static_cast<int64_t>(seg) * a.S + s, nq_pad);
  for (int idx = tid + blockIdx.z * 256; idx < nq * qd; idx += 256 * gridDim.z) {
    const int qn = idx / qd, d = (idx % qd) * DIMS;
    const uint32_t pm = static_cast<uint32_t>(nq_pad) * hd + qn;
    const uint32_t po = static_cast<uint32_t>(qn) * hd + d;
    float M = -INFINITY, den = 0.f, den_u = 0.f, den_s = 0.f;
    f32x4 acc[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int r0 = 0; r0 < nrec; r0 += kBatch) {   // usually one batch: one round trip
      float mv[kBatch], lv[kBatch], luv[kBatch], lsv[kBatch];
      f32x4 ov[kBatch][kV];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const bool in = r0 + i < nrec;
        const uint32_t ro = static_cast<uint32_t>(r0 + i) * rec;
        mv[i] = in ? base[ro + pm] : -INFINITY;
        lv[i] = in ? base[ro + pm + nq_pad] : 0.f;
        luv[i] = (in && sums) ? base[ro + pm + 2 * nq_pad] : 0.f;
        lsv[i] = (in && sums) ? base[ro + pm + 3 * nq_pad] : 0.f;
#pragma unroll
        for (int j = 0; j < kV; ++j)
          ov[i][j] = in ? *reinterpret_cast<const f32x4*>(base + (ro + po + 4 * j))
                        : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      float Mb = M;
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int w = w_lo + r0 + i;
        if (!(r0 + i < nrec && (all_full || bnd(w) < bnd(w + 1)))) mv[i] = -INFINITY;
        Mb = fmaxf(Mb, mv[i]);
      }
      const float f = (M == -INFINITY) ? 0.f : exp2f(M - Mb);
      den *= f;
      den_u *= f;
      den_s *= f;
#pragma unroll
      for (int j = 0; j < kV; ++j) acc[j] *= f;
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const float wgt = (mv[i] == -INFINITY) ? 0.f : exp2f(mv[i] - Mb);
        den += wgt * lv[i];
        den_u += wgt * luv[i];
        den_s += wgt * lsv[i];
#pragma unroll
        for (int j = 0; j < kV; ++j) acc[j] += wgt * ov[i][j];
      }
      M = Mb;
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const int64_t row = out_row(a, layer_local, s, g, qn, G);
#pragma unroll
    for (int j = 0; j < kV; ++j) {
      u16x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = f2bf(acc[j][r] * inv);
      *reinterpret_cast<u16x4*>(out + row * hd + d + 4 * j) = v;
    }
    if (a.lse && d == 0) a.lse[row] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
    if (a.mass && d == 0) {   // share of the attention over [C;U] (self keys left out) on U
      const float lcu = den - den_s;
      a.mass[row] = lcu > 0.f ? den_u / lcu : 0.f;
    }
  }
}

// ------------------------------------------------ bf16 32-key tile arithmetic
//
// Used by the grouped-prefix kernel below.  One wavefront
// owns NQT query tiles of 32 rows; the products use v_mfma_f32_32x32x16_bf16
// on 32 keys x 32 query rows.  S^T = K . Q^T takes K row rho from key pi(rho),
// pi swapping bits 2 and 3 of the key index; then lane l holds, for query
// l % 32, the keys 8*(l/32) .. +7 of both pages of the tile (registers 0-7:
// page 0, 8-15: page 1), which is exactly the B operand of O^T += V^T . P^T
// over those keys, and V pages stored [head_dim][16 slots] give the matching
// A operand with one 16-byte read.  The row maximum is a maximum over 16
// registers and one exchange between the two halves of the wavefront.  A
// tile in LDS is [K page 0][K page 1][V page 0][V page 1], K rows with their
// 16-byte chunks XOR-swizzled by the slot.
// EXT: two more running sums per query on the same reference, over the carry
// keys (lu) and the block's own keys (ls), for drafter_block_attention_ext.
template <int HD, int NQT, bool EXT = false>
struct Tile32 {
  static constexpr int KK = HD / 16, MO = HD / 32;
  static constexpr int ROWB = HD * 2, CPR = ROWB / 16;
  static constexpr int PAGE_BYTES = kPage * ROWB, LPP = PAGE_BYTES / 1024;
  static constexpr int TILE_BYTES = 4 * PAGE_BYTES;
  static constexpr int QLD = HD + 8;             // padded LDS row of staged queries (bf16)
  static constexpr float kRescale = 8.f;         // lazy rescale threshold (log2 units)

  f32x16 o[NQT][MO];
  float m_run[NQT], l_run[NQT];   // l_run: this half-wavefront's keys (summed at the end)
  float lu_run[NQT], ls_run[NQT];
  u16x8 qf[NQT][16 > KK ? KK : KK];
  uint32_t kf_off[KK], vf_off;
  int slot_base, half, r32;

  __device__ void setup(int lane) {
    half = lane >> 5;
    r32 = lane & 31;
    const int key = 16 * (r32 >> 4) + 8 * ((r32 >> 2) & 1) + 4 * ((r32 >> 3) & 1) + (r32 & 3);
    const int kslot = key & 15;
#pragma unroll
    for (int k = 0; k < KK; ++k) {
      const int ch = 2 * k + half;
      kf_off[k] = (key >> 4) * PAGE_BYTES + kslot * ROWB + ((ch ^ (kslot & (CPR - 1))) << 4);
    }
    vf_off = 2 * PAGE_BYTES + r32 * 32 + half * 16;
    slot_base = 8 * half;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
      for (int m = 0; m < MO; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[qt][m][r] = 0.f;
      m_run[qt] = -INFINITY;
      l_run[qt] = 0.f;
      lu_run[qt] = 0.f;
      ls_run[qt] = 0.f;
    }
  }

  // B fragments of the staged queries: rows qt * 32 + lane % 32 of `rows`
  __device__ void load_q(const uint16_t* rows) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int k = 0; k < KK; ++k)
        qf[qt][k] = *reinterpret_cast<const u16x8*>(rows + (qt * 32 + r32) * QLD + k * 16 + half * 8);
  }

  // one 32-key tile at tb: n0 / n1 valid keys in its two pages.  Scores are
  // formed relative to the running reference (accumulators start at -base),
  // then one rescale decision for the tile, the exponentials and the PV products.
  // kind0 / kind1 (EXT): the pages' keys are 0 committed, 1 carry, 2 the block's own.
  __device__ void step(const unsigned char* tb, int n0, int n1, int kind0 = 0, int kind1 = 0) {
    const bool partial = n0 < kPage || n1 < kPage;
    u16x8 kf[KK], vf[MO][2];
#pragma unroll
    for (int k = 0; k < KK; ++k) kf[k] = *reinterpret_cast<const u16x8*>(tb + kf_off[k]);
#pragma unroll
    for (int m = 0; m < MO; ++m)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        vf[m][j] = *reinterpret_cast<const u16x8*>(tb + vf_off + j * PAGE_BYTES + m * 32 * 32);
    f32x16 sc[NQT];
    float base[NQT];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      base[qt] = (m_run[qt] == -INFINITY) ? 0.f : m_run[qt];
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[qt][r] = -base[qt];
    }
#pragma unroll
    for (int k = 0; k < KK; ++k)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) sc[qt] = mfma32x32x16(kf[k], qf[qt][k], sc[qt]);
    if (partial) {
#pragma unroll
      for (int m = 0; m < MO; ++m)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (slot_base + e >= (j ? n1 : n0)) vf[m][j][e] = 0;   // invalid keys may hold anything
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (slot_base + (r & 7) >= ((r >> 3) ? n1 : n0)) sc[qt][r] = -INFINITY;
    }
    float mx[NQT];
    bool up = false;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      float v = fmaxf(fmaxf(fmaxf(sc[qt][0], sc[qt][1]), fmaxf(sc[qt][2], sc[qt][3])),
                      fmaxf(fmaxf(sc[qt][4], sc[qt][5]), fmaxf(sc[qt][6], sc[qt][7])));
      v = fmaxf(v, fmaxf(fmaxf(fmaxf(sc[qt][8], sc[qt][9]), fmaxf(sc[qt][10], sc[qt][11])),
                         fmaxf(fmaxf(sc[qt][12], sc[qt][13]), fmaxf(sc[qt][14], sc[qt][15]))));
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                       false, false);
      mx[qt] = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) + base[qt];
      up |= mx[qt] > m_run[qt] + kRescale;
    }
    if (__any(up)) {
      // move the reference up (only where the tile exceeds it) and rescale
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) {
        const float m_new = mx[qt] > m_run[qt] + kRescale ? mx[qt] : m_run[qt];
        const float alpha = (m_new == m_run[qt]) ? 1.f : exp2f(m_run[qt] - m_new);
        l_run[qt] *= alpha;
        if constexpr (EXT) {
          lu_run[qt] *= alpha;
          ls_run[qt] *= alpha;
        }
#pragma unroll
        for (int m = 0; m < MO; ++m) o[qt][m] *= alpha;
        m_run[qt] = m_new;
        const float shift = (m_new == -INFINITY) ? 0.f : m_new - base[qt];
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[qt][r] -= shift;
      }
    }
    u16x8 pk[NQT][2];
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r)   // v_exp_f32: arguments are <= kRescale or -inf
        p[r] = __builtin_amdgcn_exp2f(sc[qt][r]);
      const float p0 = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
      const float p1 = ((p[8] + p[9]) + (p[10] + p[11])) + ((p[12] + p[13]) + (p[14] + p[15]));
      l_run[qt] += p0 + p1;
      if constexpr (EXT) {   // registers 0-7 hold keys of page 0, 8-15 of page 1
        lu_run[qt] += (kind0 == 1 ? p0 : 0.f) + (kind1 == 1 ? p1 : 0.f);
        ls_run[qt] += (kind0 == 2 ? p0 : 0.f) + (kind1 == 2 ? p1 : 0.f);
      }
      typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const u32x4v w4 = {cvt_pk_bf16(p[8 * j + 0], p[8 * j + 1]), cvt_pk_bf16(p[8 * j + 2], p[8 * j + 3]),
                           cvt_pk_bf16(p[8 * j + 4], p[8 * j + 5]), cvt_pk_bf16(p[8 * j + 6], p[8 * j + 7])};
        pk[qt][j] = __builtin_bit_cast(u16x8, w4);
      }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int m = 0; m < MO; ++m)
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt) o[qt][m] = mfma32x32x16(vf[m][j], pk[qt][j], o[qt][m]);
  }

  // query tile qt: normalised output rows (bf16) and LSE; rows >= nq skipped
  __device__ void write_out(const AttnArgs& a, int layer_local, int s, int g, int qrow0, int nq) {
    uint16_t* out = static_cast<uint16_t*>(a.out);
    const int G = a.Hq / a.Hkv;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      const float l_tot = l_run[qt] + __shfl_xor(l_run[qt], 32);
      float lu = 0.f, ls = 0.f;
      if constexpr (EXT) {
        lu = lu_run[qt] + __shfl_xor(lu_run[qt], 32);
        ls = ls_run[qt] + __shfl_xor(ls_run[qt], 32);
      }
      const int qn = qrow0 + qt * 32 + r32;
      if (qn >= nq) continue;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      const int64_t row = out_row(a, layer_local, s, g, qn, G);
#pragma unroll
      for (int m = 0; m < MO; ++m)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          u16x4 v;
#pragma unroll
          for (int c = 0; c < 4; ++c) v[c] = f2bf(o[qt][m][4 * r4 + c] * inv);
          *reinterpret_cast<u16x4*>(out + row * HD + 32 * m + 8 * r4 + 4 * half) = v;
        }
      if (a.lse && half == 0)
        a.lse[row] = l_tot > 0.f ? (m_run[qt] + log2f(l_tot)) * kLn2 : -INFINITY;
      if constexpr (EXT) {   // share of the attention over [C;U] on U
        const float lcu = l_tot - ls;
        if (a.mass && half == 0) a.mass[row] = lcu > 0.f ? lu / lcu : 0.f;
      }
    }
  }

  // unnormalised record rows qrow0 .. of a share: O[nqp][HD], m[nqp], l[nqp]
  __device__ void write_record(float* rec, int nqp, int qrow0) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      const float l_tot = l_run[qt] + __shfl_xor(l_run[qt], 32);
      const int qn = qrow0 + qt * 32 + r32;
#pragma unroll
      for (int m = 0; m < MO; ++m)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4 v;
#pragma unroll
          for (int c = 0; c < 4; ++c) v[c] = o[qt][m][4 * r4 + c];
          *reinterpret_cast<f32x4*>(rec + qn * HD + 32 * m + 8 * r4 + 4 * half) = v;
        }
      float lu = 0.f, ls = 0.f;
      if constexpr (EXT) {
        lu = lu_run[qt] + __shfl_xor(lu_run[qt], 32);
        ls = ls_run[qt] + __shfl_xor(ls_run[qt], 32);
      }
      if (half == 0) {
        rec[nqp * HD + qn] = m_run[qt];
        rec[nqp * HD + nqp + qn] = l_tot;
        if constexpr (EXT) {
          rec[nqp * HD + 2 * nqp + qn] = lu;
          rec[nqp * HD + 3 * nqp + qn] = ls;
        }
      }
    }
  }
};

// Rotated (at position ctx + query / G), scaled (1/sqrt(hd), log2 units) bf16
// queries of rows qrow0 .. qrow0 + nrows - 1 of sequence s into LDS rows
// [nrows][HD + 8]; rows past the block are zero.  One wavefront.
template <int HD>
__device__ void stage_queries(const AttnArgs& a, uint16_t* rows, int nrows, int qrow0, bool live,
                              int s, int g, int layer_local, int ctx, const double* inv_rev,
                              int lane) {
  constexpr int QLD = HD + 8;
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  const uint16_t* Q = static_cast<const uint16_t*>(a.q);
  const bool rotate_q = !(a.flags & CO_Q_PREROTATED);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;
  for (int idx = lane; idx < nrows * (HD / 8); idx += 64) {
    const int r = idx / (HD / 8), p4 = (idx % (HD / 8)) * 4;
    const int qn = qrow0 + r;
    u16x4 lo4 = {0, 0, 0, 0}, hi4 = {0, 0, 0, 0};
    if (live && qn < nq) {
      const int64_t off = out_row(a, layer_local, s, g, qn, G) * HD + p4;
      const u16x4 ql = *reinterpret_cast<const u16x4*>(Q + off);
      const u16x4 qh = *reinterpret_cast<const u16x4*>(Q + off + HD / 2);
      const int pos = ctx + qn / G;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float x = bf2f(ql[e]), y = bf2f(qh[e]);
        if (rotate_q) {
          float cs, sn;
          rope_cos_sin_rev(pos, inv_rev[p4 + e], &cs, &sn);
          const float x2 = x * cs - y * sn, y2 = y * cs + x * sn;
          x = x2;
          y = y2;
        }
        lo4[e] = f2bf(x * qscale);
        hi4[e] = f2bf(y * qscale);
      }
    }
    *reinterpret_cast<u16x4*>(rows + r * QLD + p4) = lo4;
    *reinterpret_cast<u16x4*>(rows + r * QLD + p4 + HD / 2) = hi4;
  }
}

// Keys of page-pair t (pages 2t, 2t+1) below `limit`: the two page counts.
__device__ __forceinline__ int keys_in(int limit, int t, int h) {
  return min(kPage, max(0, limit - (2 * t + h) * kPage));
}

// Committed tiles per share of a grouped launch (CO_TUNE_ATTN_GROUP_SPLIT_TILES
// overrides it), and the number of shares that covers the longest sequence the
// page table allows.
constexpr int kGroupSplitTiles = 128;
int group_split_tiles() {
  const int64_t v = tuning(CO_TUNE_ATTN_GROUP_SPLIT_TILES);
  return v >= 1 && v <= 4096 ? static_cast<int>(v) : kGroupSplitTiles;
}
int group_splits(int max_pages) {
  const int tiles = (max_pages + 1) / 2, sp = group_split_tiles();
  return max(1, (tiles + sp - 1) / sp);
}

// Record of (layer, KV head, sequence, share) in the workspace.
__device__ __forceinline__ float* share_record(const AttnArgs& a, int layer_local, int g, int s,
                                               int n_splits, int split, int nqp, int hd) {
  return a.ws + ((((static_cast<int64_t>(layer_local) * a.Hkv + g) * a.S + s) * n_splits + split) *
                 (static_cast<int64_t>(nqp) * (hd + 2)));
}

// ------------------------------------------------ bf16 grouped-prefix path
//
// Blocks anchored in one recorded response (the training-shaped forward,
// Algorithm 2) are sequences whose committed keys are prefixes of the same
// pages.  Under CO_ATTN_SHARED_PREFIX a workgroup takes four consecutive
// sequences, one per wavefront, so that each key tile is read once for all of
// their block queries:
//   * the page ids of a chunk of pages are staged in LDS; the chunk is shared
//     when every wavefront's pages agree with those of the longest sequence
//     wherever its own keys reach;
//   * shared chunks stream through a 4-deep ring of 32-key tiles, each
//     wavefront loading one of a tile's four pages (K0, K1, V0, V1) with
//     direct-to-LDS loads and a barrier publishing the tile; a wavefront skips
//     tiles beyond its own length and masks the keys of its last one;
//   * chunks that are not shared are streamed by each wavefront on its own;
//   * the carry pages of each sequence come last; the result is normalised and
//     written in place, or, when the group's keys are split into shares, each
//     share leaves a record that the merge kernel combines.
// With head_dim 64 and 32 query rows a workgroup fits 168 VGPRs and about 35
// KiB of LDS, so three share a CU and hide each other's dependency latencies.
constexpr int kGroupSeqs = 4;       // sequences (wavefronts) per workgroup
constexpr int kGroupChunk = 128;    // pages whose ids are staged at a time

template <int HD, int NQT>
__global__ __launch_bounds__(256, HD == 64 ? (NQT == 1 ? 3 : 2) : 1)
void attn_group_kernel(AttnArgs a, int split_tiles, int n_splits) {
  using TT = Tile32<HD, NQT>;
  constexpr int NQP = NQT * 32, QLD = TT::QLD;
  constexpr int PAGE_BYTES = TT::PAGE_BYTES, LPP = TT::LPP, TILE_BYTES = TT::TILE_BYTES;
  constexpr int NS = 4;                          // ring tiles; one per wavefront when private
  static_assert(LPP * (NS - 1) < 64, "vmcnt");
  // the rotated queries are staged in the ring before the first tile lands
  constexpr int RING_BYTES = NS * TILE_BYTES;
  constexpr int Q_BYTES = kGroupSeqs * NQP * QLD * 2;
  __shared__ __align__(16) unsigned char ring[RING_BYTES > Q_BYTES ? RING_BYTES : Q_BYTES];
  uint16_t* q_lds = reinterpret_cast<uint16_t*>(ring);
  __shared__ int pid_lds[kGroupSeqs][kGroupChunk];
  __shared__ double inv_lds[HD / 2];
  __shared__ int npc_lds[kGroupSeqs];
  __shared__ int mismatch;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_groups = (a.S + kGroupSeqs - 1) / kGroupSeqs;
  // Workgroup ids are dealt to the 8 XCDs round-robin; renumbered, every XCD
  // takes a run of consecutive groups, whose shared pages then stay in its L2.
  int bx = blockIdx.x;
  if ((gridDim.x & 7) == 0) bx = (bx & 7) * (gridDim.x >> 3) + (bx >> 3);
  const int split = bx % n_splits;
  const int group = n_groups - 1 - bx / n_splits;   // later blocks reach furthest
  const int g = blockIdx.y, layer_local = blockIdx.z, layer = a.layer_begin + layer_local;
  const int s = group * kGroupSeqs + wave;
  const bool live = s < a.S;
  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* vc = static_cast<const uint16_t*>(a.v_cache);
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);
  const uint16_t* vk = static_cast<const uint16_t*>(a.v_carry);
  if (tid < HD / 2) inv_lds[tid] = a.rope_inv[tid] * kInv2Pi;

  // this wavefront's sequence
  int ctx = 0, carry = 0;
  if (live) {
    const SeqInfo si = seq_info(a, s, 1);
    if (si.ok) {
      ctx = si.ctx;
      carry = si.carry;
    } else if (lane == 0 && g == 0 && layer_local == 0) {
      set_status(a.status, CO_ERR_LENGTH);
    }
  }
  const int npc = (ctx + kPage - 1) / kPage;
  if (lane == 0) npc_lds[wave] = npc;
  if (tid == 0) mismatch = 0;
  __syncthreads();   // inv_lds, npc_lds

  int npc_max = 0, leader = 0;
#pragma unroll
  for (int v = 0; v < kGroupSeqs; ++v)
    if (npc_lds[v] > npc_max) {
      npc_max = npc_lds[v];
      leader = v;
    }
  // this workgroup's share of the group's committed tiles; the last share also
  // takes the carry keys.  Shares past the group's keys have nothing to do.
  const int t_all = (npc_max + 1) / 2;
  const int n_used = max(1, (t_all + split_tiles - 1) / split_tiles);
  if (split >= n_used) return;   // uniform, and no barrier follows for this workgroup
  const int t_beg = split * split_tiles, t_end = min(t_all, t_beg + split_tiles);
  const bool last_share = split == n_used - 1;

  stage_queries<HD>(a, q_lds + wave * NQP * QLD, NQP, 0, live, s, g, layer_local, ctx, inv_lds,
                    lane);
  __syncthreads();
  TT T;
  T.setup(lane);
  T.load_q(q_lds + wave * NQP * QLD);

  // per-lane source offsets (elements) of the loads of one page: K rows land
  // XOR-swizzled, V pages are copied as they are
  int k_off[LPP], v_off[LPP];
#pragma unroll
  for (int q = 0; q < LPP; ++q) {
    const int byte = q * 1024 + lane * 16;
    const int r = byte / TT::ROWB, pch = (byte % TT::ROWB) / 16;
    k_off[q] = r * HD + (pch ^ (r & (TT::CPR - 1))) * 8;
    v_off[q] = byte / 2;
  }
  const uint32_t ring_lds = lds_addr(ring);
  // page `phys` of this layer and KV head: base + phys * page_stride elements
  const int64_t page_stride = static_cast<int64_t>(a.Hkv) * kPage * HD;
  const int64_t head0 = (static_cast<int64_t>(layer) * a.num_pages * a.Hkv + g) * (kPage * HD);
  const uint16_t* kbase = kc + head0;
  const uint16_t* vbase = vc + head0;
  // one page (K or V) of a committed page id, or a harmless dummy (id < 0) -> LDS
  auto load_page = [&](bool is_v, int phys, uint32_t dst) {
    const uint16_t* src = is_v ? vk : kk;   // dummy: carry page 0 of layer 0
    if (phys >= 0) src = (is_v ? vbase : kbase) + phys * page_stride;
#pragma unroll
    for (int q = 0; q < LPP; ++q)
      lds_dma16_opaque(src + (is_v ? v_off[q] : k_off[q]), dst + q * 1024);
  };
  auto load_carry_page = [&](bool is_v, int cp, uint32_t dst) {
    const int64_t row = ((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp) * a.Hkv + g;
    const uint16_t* src = (is_v ? vk : kk) + row * (kPage * HD);
#pragma unroll
    for (int q = 0; q < LPP; ++q)
      lds_dma16_opaque(src + (is_v ? v_off[q] : k_off[q]), dst + q * 1024);
  };

  // ---- committed keys of this share, chunk by chunk
  const int p_end = min(npc_max, 2 * t_end);
  for (int c0 = 2 * t_beg; c0 < p_end; c0 += kGroupChunk) {
    const int cn = min(kGroupChunk, p_end - c0);
    __syncthreads();   // the previous chunk's tiles, page ids and flag are consumed
    if (tid == 0) mismatch = 0;
    for (int i = lane; i < cn; i += 64) {
      int id = -1;
      if (live && c0 + i < npc) {
        id = a.page_table[static_cast<int64_t>(s) * a.max_pages + c0 + i];
        if (id < 0 || id >= a.num_pages) {   // read as a dummy page, its keys masked
          set_status(a.status, CO_ERR_PAGE_RANGE);
          id = -1;
        }
      }
      pid_lds[wave][i] = id;
    }
    __syncthreads();
    bool bad = false;
    for (int i = lane; i < cn; i += 64)
      if (c0 + i < npc && pid_lds[wave][i] != pid_lds[leader][i]) bad = true;
    if (__any(bad) && lane == 0) mismatch = 1;
    __syncthreads();
    const int t0 = c0 / 2, t1 = min(t_end, (c0 + cn + 1) / 2);
    // the chunk's page ids of this wavefront and of the leader in registers,
    // lane i holding pages i and i + 64 (-1 past the chunk)
    const int my0 = lane < cn ? pid_lds[wave][lane] : -1;
    const int my1 = lane + 64 < cn ? pid_lds[wave][lane + 64] : -1;
    const int ld0 = lane < cn ? pid_lds[leader][lane] : -1;
    const int ld1 = lane + 64 < cn ? pid_lds[leader][lane + 64] : -1;
    auto pid_of = [&](int r0, int r1, int p) {   // p uniform, < kGroupChunk
      const int x0 = __builtin_amdgcn_readlane(r0, p & 63);
      const int x1 = __builtin_amdgcn_readlane(r1, p & 63);
      return p < 64 ? x0 : x1;
    };
    // keys of tile t in this wavefront: [32t, 32t + 32) clipped to ctx, and pages
    // whose id was rejected hold no valid keys
    auto keys = [&](int t, int h) {
      const int p = 2 * t + h - c0;
      if (p >= cn || pid_of(my0, my1, p) < 0) return 0;
      return keys_in(ctx, t, h);
    };
    if (!mismatch) {
      // shared: wavefront w loads page w of each tile (K0, K1, V0, V1) of the leader
      auto issue = [&](int t) {
        const int p = 2 * t + (wave & 1) - c0;
        const int phys = p < cn ? pid_of(ld0, ld1, p) : -1;
        load_page(wave >= 2, phys, ring_lds + (t % NS) * TILE_BYTES + wave * PAGE_BYTES);
      };
      for (int t = t0; t < min(t1, t0 + NS - 1); ++t) issue(t);
      for (int t = t0; t < t1; ++t) {
        const int ahead = min(NS - 2, t1 - 1 - t);
        if (ahead >= 2) wait_vm_lgkm_barrier<2 * LPP>();
        else if (ahead == 1) wait_vm_lgkm_barrier<LPP>();
        else wait_vm_lgkm_barrier<0>();
        if (t + NS - 1 < t1) issue(t + NS - 1);   // into the slot of tile t-1, read by all
        const int n0 = keys(t, 0), n1 = keys(t, 1);
        if (n0 + n1 > 0) T.step(ring + (t % NS) * TILE_BYTES, n0, n1);
      }
    } else {
      // pages differ between the sequences: each wavefront on its own, one slot each
      const int my_t1 = min(t1, (min(npc, c0 + cn) + 1) / 2);
      const uint32_t slot = ring_lds + wave * TILE_BYTES;
      for (int t = t0; t < my_t1; ++t) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the previous tile is consumed
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int p = 2 * t + h - c0;
          const int phys = p < cn ? pid_of(my0, my1, p) : -1;
          load_page(false, phys, slot + h * PAGE_BYTES);
          load_page(true, phys, slot + (2 + h) * PAGE_BYTES);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        const int n0 = keys(t, 0), n1 = keys(t, 1);
        if (n0 + n1 > 0) T.step(ring + wave * TILE_BYTES, n0, n1);
      }
    }
  }

  // ---- the carry segment of this sequence, two carry pages per tile
  __syncthreads();   // the ring is free
  if (last_share) {
    const uint32_t slot = ring_lds + wave * TILE_BYTES;
    const int ncp = (carry + kPage - 1) / kPage;
    for (int t = 0; 2 * t < ncp; ++t) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int cp = min(2 * t + h, ncp - 1);   // a missing second page repeats the first
        load_carry_page(false, cp, slot + h * PAGE_BYTES);
        load_carry_page(true, cp, slot + (2 + h) * PAGE_BYTES);
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      T.step(ring + wave * TILE_BYTES, keys_in(carry, t, 0), keys_in(carry, t, 1));
    }
  }

  // ---- normalise and write, or leave this share's record for the merge
  if (!live) return;
  if (n_used > 1)
    T.write_record(share_record(a, layer_local, g, s, n_splits, split, NQP, HD), NQP, 0);
  else
    T.write_out(a, layer_local, s, g, 0, a.B * (a.Hq / a.Hkv));
}

// Merge of the shares of a grouped launch (log-sum-exp rule), for sequences
// whose keys took more than one share: one thread per (query row, 4 dims).
// A share count follows from the longest committed length among the
// `group` consecutive sequences that shared a workgroup.
template <int HD>
__global__ __launch_bounds__(256) void attn_share_merge_kernel(AttnArgs a, int split_tiles,
                                                               int n_splits, int nqp, int group) {
  const int s = blockIdx.x, g = blockIdx.y, layer_local = blockIdx.z;
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  int npc_max = 0;
  const int g0 = s / group * group;
  for (int v = g0; v < min(g0 + group, a.S); ++v) {
    const SeqInfo si = seq_info(a, v, 1);
    if (si.ok) npc_max = max(npc_max, si.npc);
  }
  const int n_used = max(1, ((npc_max + 1) / 2 + split_tiles - 1) / split_tiles);
  if (n_used <= 1) return;   // written by the attention kernel
  const float* base = share_record(a, layer_local, g, s, n_splits, 0, nqp, HD);
  const int64_t rec = static_cast<int64_t>(nqp) * (HD + 2);
  uint16_t* out = static_cast<uint16_t*>(a.out);
  for (int idx = threadIdx.x; idx < nq * (HD / 4); idx += 256) {
    const int qn = idx / (HD / 4), d = (idx % (HD / 4)) * 4;
    float M = -INFINITY;
    for (int k = 0; k < n_used; ++k) M = fmaxf(M, base[k * rec + nqp * HD + qn]);
    float L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < n_used; ++k) {
      const float* r = base + k * rec;
      const float m = r[nqp * HD + qn];
      const float w = (m == -INFINITY) ? 0.f : exp2f(m - M);
      L += w * r[nqp * HD + nqp + qn];
      acc += w * *reinterpret_cast<const f32x4*>(r + qn * HD + d);
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int64_t row = out_row(a, layer_local, s, g, qn, G);
    u16x4 v;
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = f2bf(acc[c] * inv);
    *reinterpret_cast<u16x4*>(out + row * HD + d) = v;
    if (a.lse && d == 0) a.lse[row] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
  }
}

// ------------------------------------------ bf16 per-wavefront slices path
//
// For query tiles too large to stage more than one segment's queries in LDS
// next to the ring (head_dim 128, 64 query rows), every wavefront takes its
// own equal slice of the global tile order and walks it alone: no rounds, no
// barriers, no merging between wavefronts.  Per piece of a segment in the
// slice, the wavefront loads the queries straight into its MFMA fragments
// (rotated in registers: at head_dim 128 a lane holds both dims of each
// rotation pair), streams the piece's tiles through a private two-stage ring
// and then writes the normalised output (a whole segment) or a record for
// attn_bf16_combine_kernel (slices are wavefronts: record slot = slice + segment).
// Tiles of a sequence: its committed pages two by two, then its carry pages
// two by two.
constexpr int kWaveRing = 2;     // ring stages per wavefront
constexpr int kWaveMinTiles = 8; // tiles per slice below which fewer slices are launched

// wavefronts per workgroup: one per SIMD at head_dim 128 (registers), two at 64
constexpr int wave_waves(int hd) { return hd == 128 ? 4 : 8; }

template <int HD, int NQT, bool EXT>
__global__ __launch_bounds__(64 * wave_waves(HD), 1) void attn_wave_kernel(
    AttnArgs a, int layer_count, int n_slices, int hdr_floats) {
  // NQT tiles of 32 query rows, each its own Tile32 stepping over the same key
  // tile (one fragment set live at a time keeps the registers within budget)
  using TT = Tile32<HD, 1, EXT>;
  constexpr int NQP = NQT * 32, NW = wave_waves(HD), NS = kWaveRing, NTHR = 64 * NW;
  constexpr int PAGE_BYTES = TT::PAGE_BYTES, LPP = TT::LPP, TILE_BYTES = TT::TILE_BYTES;
  constexpr int KK = TT::KK;
  static_assert(4 * LPP * (NS - 1) < 64, "vmcnt");
  __shared__ __align__(16) unsigned char ring[NW * NS * TILE_BYTES];
  __shared__ int tstart[kMaxAttnSeqs + 1];
  __shared__ int ctx_l[kMaxAttnSeqs], carry_l[kMaxAttnSeqs];
  __shared__ int part[NTHR];
  __shared__ double inv_lds[HD / 2];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int S = a.S, G = a.Hq / a.Hkv, nq = a.B * G;
  if (tid < HD / 2) inv_lds[tid] = a.rope_inv[tid] * kInv2Pi;

  // ---- tiles per sequence and their prefix (the same in every workgroup)
  constexpr int SPT = (kMaxAttnSeqs + NTHR - 1) / NTHR;   // sequences per thread
  int nts[SPT];
  int sum = 0;
#pragma unroll
  for (int i = 0; i < SPT; ++i) {
    const int s = tid * SPT + i;
    nts[i] = 0;
    if (s < S) {
      const SeqInfo si = seq_info(a, s, 1);
      const int ctx = si.ok ? si.ctx : 0, carry = si.ok ? si.carry : 0;
      if (!si.ok && blockIdx.x == 0) set_status(a.status, CO_ERR_LENGTH);
      ctx_l[s] = ctx;
      carry_l[s] = carry;
      const int npc = (ctx + kPage - 1) / kPage, ncp = (carry + kPage - 1) / kPage;
      nts[i] = (npc + 1) / 2 + (ncp + 1) / 2;
      if (EXT && a.k_self && si.ok && nts[i] == 0) nts[i] = 1;   // its self keys follow the tile
    }
    sum += nts[i];
  }
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < NTHR; off <<= 1) {   // inclusive scan of the per-thread sums
    const int v = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  {
    int x = part[tid] - sum;
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
      const int s = tid * SPT + i;
      if (s < S) tstart[s] = x;
      x += nts[i];
    }
    if (tid == NTHR - 1) tstart[S] = part[NTHR - 1];
  }
  __syncthreads();
  const int T1 = tstart[S];
  const int n_segs = layer_count * a.Hkv;
  const int64_t t_all = static_cast<int64_t>(n_segs) * T1;
  const int w = blockIdx.x * NW + wave;
  const int t0 = static_cast<int>(t_all * w / n_slices);
  const int t1 = static_cast<int>(t_all * (w + 1) / n_slices);
  int* hdr = reinterpret_cast<int*>(a.ws);
  if (lane == 0) hdr[S + 1 + w] = t0;
  if (w == 0) {
    for (int s = lane; s <= S; s += 64) hdr[s] = tstart[s];
    if (lane == 0) hdr[S + 1 + n_slices] = static_cast<int>(t_all);
  }

  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* vc = static_cast<const uint16_t*>(a.v_cache);
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);
  const uint16_t* vk = static_cast<const uint16_t*>(a.v_carry);
  const uint16_t* Q = static_cast<const uint16_t*>(a.q);
  const bool rotate_q = !(a.flags & CO_Q_PREROTATED);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;
  // per-lane source offsets (elements) of the loads of one page: K rows land
  // XOR-swizzled, V pages are copied as they are
  int k_off[LPP], v_off[LPP];
#pragma unroll
  for (int q = 0; q < LPP; ++q) {
    const int byte = q * 1024 + lane * 16;
    const int r = byte / TT::ROWB, pch = (byte % TT::ROWB) / 16;
    k_off[q] = r * HD + (pch ^ (r & (TT::CPR - 1))) * 8;
    v_off[q] = byte / 2;
  }
  const uint32_t my_ring = lds_addr(ring) + wave * NS * TILE_BYTES;
  const int64_t page_stride = static_cast<int64_t>(a.Hkv) * kPage * HD;
  auto load_page = [&](const uint16_t* src, bool is_v, uint32_t dst) {
#pragma unroll
    for (int q = 0; q < LPP; ++q) lds_dma16_opaque(src + (is_v ? v_off[q] : k_off[q]), dst + q * 1024);
  };

  TT T[NQT];
  for (int t = t0; t < t1;) {
    // ---- the piece of one segment that starts at tile t
    const int seg = t / T1, local = t - seg * T1;
    int lo = 0, hi = S;   // the sequence: tstart[s] <= local < tstart[s + 1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (tstart[mid] <= local) lo = mid; else hi = mid;
    }
    const int s = lo;
    const int j0 = local - tstart[s];
    const int nts_s = tstart[s + 1] - tstart[s];
    const int pe = min(t1, seg * T1 + tstart[s + 1]);
    const int j1 = j0 + (pe - t);
    const int layer_local = seg / a.Hkv, g = seg % a.Hkv, layer = a.layer_begin + layer_local;
    const int ctx = ctx_l[s], carry = carry_l[s];
    const int npc = (ctx + kPage - 1) / kPage, nct = (npc + 1) / 2;
    const int ncp = (carry + kPage - 1) / kPage;

    // queries of the segment straight into the B fragments, rotated at ctx + i
    const bool quad = (G & 3) == 0;
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      T[qt].setup(lane);
      const int qn = qt * 32 + T[qt].r32;
      u16x8 raw[KK];
      const bool live = qn < nq;
      const int64_t base = live ? out_row(a, layer_local, s, g, qn, G) * HD : 0;
#pragma unroll
      for (int k = 0; k < KK; ++k)
        raw[k] = *reinterpret_cast<const u16x8*>(Q + base + k * 16 + T[qt].half * 8);
      const int pos = ctx + qn / G;
#pragma unroll
      for (int k = 0; k < KK / 2; ++k) {
        const int i0 = k * 16 + T[qt].half * 8;   // pair index of element 0 of this chunk
        // With G a multiple of 4 the four lanes of a quad hold rows of one
        // position and the same dims: each computes two of the chunk's eight
        // rotation angles and takes the rest from its neighbours.
        float c2[2] = {0.f, 0.f}, s2[2] = {0.f, 0.f};
        if (rotate_q && quad) {
#pragma unroll
          for (int u = 0; u < 2; ++u) rope_cos_sin_rev(pos, inv_lds[i0 + 2 * (lane & 3) + u], &c2[u], &s2[u]);
        }
        float xs[8], ys[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float x = live ? bf2f(raw[k][e]) : 0.f, y = live ? bf2f(raw[k + KK / 2][e]) : 0.f;
          if (rotate_q) {
            float cs, sn;
            if (quad) {
              cs = quad_bcast(c2[e & 1], e >> 1);
              sn = quad_bcast(s2[e & 1], e >> 1);
            } else {
              rope_cos_sin_rev(pos, inv_lds[i0 + e], &cs, &sn);
            }
            const float x2 = x * cs - y * sn, y2 = y * cs + x * sn;
            x = x2;
            y = y2;
          }
          xs[e] = x * qscale;
          ys[e] = y * qscale;
        }
        typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
        const u32x4v xp = {cvt_pk_bf16(xs[0], xs[1]), cvt_pk_bf16(xs[2], xs[3]),
                           cvt_pk_bf16(xs[4], xs[5]), cvt_pk_bf16(xs[6], xs[7])};
        const u32x4v yp = {cvt_pk_bf16(ys[0], ys[1]), cvt_pk_bf16(ys[2], ys[3]),
                           cvt_pk_bf16(ys[4], ys[5]), cvt_pk_bf16(ys[6], ys[7])};
        T[qt].qf[0][k] = __builtin_bit_cast(u16x8, xp);
        T[qt].qf[0][k + KK / 2] = __builtin_bit_cast(u16x8, yp);
      }
    }

    // tile j of the sequence: two committed pages, or two carry pages
    const int64_t head0 = (static_cast<int64_t>(layer) * a.num_pages * a.Hkv + g) * (kPage * HD);
    const int32_t* pt = a.page_table + static_cast<int64_t>(s) * a.max_pages;
    auto issue = [&](int j, int phys0, int phys1) {
      const uint32_t dst = my_ring + (j % NS) * TILE_BYTES;
      const uint16_t *k0, *k1, *v0, *v1;
      if (j < nct) {
        k0 = kc + head0 + phys0 * page_stride;
        v0 = vc + head0 + phys0 * page_stride;
        k1 = kc + head0 + phys1 * page_stride;
        v1 = vc + head0 + phys1 * page_stride;
      } else {
        // (clamped: a segment with self keys only has one empty tile)
        const int last = max(ncp - 1, 0);
        const int cp0 = min(2 * (j - nct), last), cp1 = min(cp0 + 1, last);
        const int64_t r0 = ((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp0) * a.Hkv + g;
        const int64_t r1 = ((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp1) * a.Hkv + g;
        k0 = kk + r0 * (kPage * HD);
        v0 = vk + r0 * (kPage * HD);
        k1 = kk + r1 * (kPage * HD);
        v1 = vk + r1 * (kPage * HD);
      }
      load_page(k0, false, dst);
      load_page(k1, false, dst + PAGE_BYTES);
      load_page(v0, true, dst + 2 * PAGE_BYTES);
      load_page(v1, true, dst + 3 * PAGE_BYTES);
    };
    auto keys = [&](int j, int h) {
      return j < nct ? keys_in(ctx, j, h) : keys_in(carry, j - nct, h);
    };
    // committed page ids of tiles [c0, c0 + 64): lane l holds pages 2(c0 + l), 2(c0 + l) + 1;
    // a rejected id reads page 0 with its keys masked
    int id0 = 0, id1 = 0, c0 = -(1 << 30), bad = 0;   // no window fetched yet
    auto fetch_ids = [&](int c) {
      c0 = c;
      const int jt = c + lane, p = 2 * jt;
      id0 = 0;
      id1 = 0;
      bad = 0;
      if (jt < nct) {
        const int x0 = pt[p];
        const int x1 = p + 1 < npc ? pt[p + 1] : x0;
        const bool b0 = x0 < 0 || x0 >= a.num_pages, b1 = x1 < 0 || x1 >= a.num_pages;
        if (b0 || b1) set_status(a.status, CO_ERR_PAGE_RANGE);
        id0 = b0 ? 0 : x0;
        id1 = b1 ? 0 : x1;
        bad = (b0 ? 1 : 0) | (b1 ? 2 : 0);
      }
    };
    auto tile_ids = [&](int j, int& p0, int& p1, int& b) {   // j uniform, committed
      if (j >= c0 + 64 || j < c0) fetch_ids(j);
      p0 = __builtin_amdgcn_readlane(id0, j - c0);
      p1 = __builtin_amdgcn_readlane(id1, j - c0);
      b = __builtin_amdgcn_readlane(bad, j - c0);
    };
    auto issue_tile = [&](int j, int& b) {
      int p0 = 0, p1 = 0;
      b = 0;
      if (j < nct) tile_ids(j, p0, p1, b);
      issue(j, p0, p1);
    };

    int bcur = 0, bnext = 0;
    issue_tile(j0, bcur);
    for (int j = j0; j < j1; ++j) {
      const bool more = j + 1 < j1;
      if (more) issue_tile(j + 1, bnext);   // into the slot of tile j - 1, consumed
      if (more) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(4 * LPP) : "memory");
      else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      const int n0 = (bcur & 1) ? 0 : keys(j, 0), n1 = (bcur & 2) ? 0 : keys(j, 1);
      if (n0 + n1 > 0) {
        const int kind = (EXT && j >= nct) ? 1 : 0;   // a tile is committed or carry
#pragma unroll
        for (int qt = 0; qt < NQT; ++qt)
          T[qt].step(ring + (wave * NS + j % NS) * TILE_BYTES, n0, n1, kind, kind);
      }
      bcur = bnext;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the ring's last tile is read
    if constexpr (EXT) {
      // the segment's end: its self keys, in the slot of its last tile
      if (a.k_self && j1 == nts_s) {
        // both ring slots are free: raw rows in one, the tile in the other
        unsigned char* slot = ring + (wave * NS + (j1 - 1) % NS) * TILE_BYTES;
        const unsigned char* raw = ring + (wave * NS + j1 % NS) * TILE_BYTES;
        static_assert(NS == 2 && 2 * 32 * HD * 2 <= TILE_BYTES, "self staging");
        for (int r0 = 0; r0 < a.B; r0 += 32) {
          self_rows_raw<HD>(a, s, layer_local, g, r0, lane, lds_addr(raw));
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          self_rows_place<HD>(raw, slot, r0, ctx, lane, inv_lds);
          const int nb = a.B - r0;
#pragma unroll
          for (int qt = 0; qt < NQT; ++qt)
            T[qt].step(slot, min(nb, kPage), max(0, min(nb - kPage, kPage)), 2, 2);
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // read before the next rows land
        }
      }
    }

    // ---- a whole segment: normalise and write; else a record for the combine
    float* rec = slot_ptr(a, hdr_floats, w + static_cast<int64_t>(seg) * S + s, NQP);
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      if (j0 == 0 && j1 == nts_s)
        T[qt].write_out(a, layer_local, s, g, qt * 32, nq);
      else
        T[qt].write_record(rec, NQP, qt * 32);
    }
    t = pe;
  }
}

}  // namespace

// Whether a launch takes the per-wavefront slices path where the shape allows
// it: by default at head_dim 128 with 64 query rows (measured faster at every
// such shape); CO_TUNE_ATTN_WAVE chooses.
static bool wave_slices_enabled(int hd) {
  const int64_t v = tuning(CO_TUNE_ATTN_WAVE);
  return v >= 0 ? v != 0 : hd == 128;
}

AttnPlan plan_attention(int S, int B, int L, int Hq, int Hkv, int hd, int max_pages, int num_pages,
                        int dtype, int num_cus) {
  AttnPlan p{};
  const int nq = B * (Hq / Hkv);
  p.nq_pad = (nq + 15) / 16 * 16;
  const int cp = (B + kPage - 1) / kPage;
  const int max_lp = max_pages + cp;
  p.ok = true;
  if (dtype == CO_DTYPE_BF16) {
    // persistent path: one workgroup on 7/8 of the CUs (as the per-wavefront
    // slices below: fewer concurrent page streams and records; measured faster
    // than one on every CU with 32 ragged contexts of 0.5-8K keys at head_dim
    // 64); a record per (slice, segment) pair and, for large query tiles, a
    // parking area per wavefront
    const int nw = hd == 64 ? kAttnWaves64 : kAttnWaves128;
    const int rtm = hd == 64 ? kAttnRoundTiles64 : kAttnRoundTiles128;
    p.n_wg = std::max(1, num_cus * 7 / 8);
    p.round_tiles = rtm;
    const int64_t wg_override = tuning(CO_TUNE_ATTN_WORKGROUPS);
    const bool wg_forced = wg_override >= 1 && wg_override <= kMaxMergeSlices;
    if (wg_forced) p.n_wg = static_cast<int>(wg_override);
    const int64_t rt_override = tuning(CO_TUNE_ATTN_ROUND_TILES);
    if (rt_override >= 1 && rt_override <= rtm) p.round_tiles = static_cast<int>(rt_override);
    p.hdr_floats = (S + 1 + p.n_wg + 1 + 63) / 64 * 64;
    const size_t rec = static_cast<size_t>(p.nq_pad) * (hd + 4);   // room for the extras' sums
    const size_t records = (static_cast<size_t>(p.n_wg) + static_cast<size_t>(L) * Hkv * S) * rec;
    const size_t park =
        hd * (p.nq_pad / 16) > 128 ? static_cast<size_t>(p.n_wg) * nw * rec : 0;
    p.park_off = static_cast<int64_t>(p.hdr_floats + records);
    p.bytes = (p.hdr_floats + records + park) * 4;
    // global tile indices, committed and carry K/V row indices are int32
    const int64_t tiles = static_cast<int64_t>(L) * Hkv * S * ((max_lp + 1) / 2);
    const int64_t rows_c = static_cast<int64_t>(L) * num_pages * Hkv;
    const int64_t rows_u = static_cast<int64_t>(L) * S * cp * Hkv;
    p.ok = S <= kMaxAttnSeqs && tiles < INT32_MAX && rows_c < INT32_MAX && rows_u < INT32_MAX;
    // per-wavefront slices for head_dim 128 with 64 query rows: the workspace
    // covers either path, so that the choice can change between calls
    // slices: one per wavefront of every CU, but no more than one per
    // kWaveMinTiles tiles the page table allows (few tiles in many slices would
    // only multiply the records to combine); the workgroup override sets it
    const int nw_h = wave_waves(hd);
    const int64_t cap_tiles = static_cast<int64_t>(L) * Hkv * S * ((max_pages + 1) / 2 + (cp + 1) / 2);
    int n_sl = p.n_wg * nw_h;
    if (!wg_forced) {
      // 7/8 of the CUs: measured faster than all of them at head_dim 128 (fewer
      // concurrent page streams, fewer records; 0.70 vs 0.69 of peak at the
      // 5-layer long chain)
      n_sl = std::max(1, num_cus * 7 / 8) * nw_h;
      const int64_t by_tiles = (cap_tiles / kWaveMinTiles + nw_h - 1) / nw_h * nw_h;
      n_sl = static_cast<int>(std::max<int64_t>(nw_h, std::min<int64_t>(n_sl, by_tiles)));
    }
    const bool wave_shape = (hd == 128 && p.nq_pad == 64) ||
                            (hd == 64 && (p.nq_pad == 32 || p.nq_pad == 64));
    if (wave_shape && n_sl <= kMaxMergeSlices) {
      const int hdr_w = (S + 1 + n_sl + 1 + 63) / 64 * 64;
      const size_t bytes_w =
          (hdr_w + (static_cast<size_t>(n_sl) + static_cast<size_t>(L) * Hkv * S) * rec) * 4;
      if (bytes_w > p.bytes) p.bytes = bytes_w;
      if (wave_slices_enabled(hd)) {
        p.wave = true;
        p.n_wg = n_sl;
        p.hdr_floats = hdr_w;
      }
    }
  } else {
    // fp32 path: chunks of pages, one workgroup each; short chunks, so that a
    // short context still spreads over many workgroups
    p.chunk_pages = 4;
    while ((max_lp + p.chunk_pages - 1) / p.chunk_pages > kMaxMergeChunks) p.chunk_pages *= 2;
    p.ok = p.chunk_pages <= kMaxChunkPages;
    p.n_chunks = (max_lp + p.chunk_pages - 1) / p.chunk_pages;
    p.bytes = static_cast<size_t>(L) * S * Hkv * p.n_chunks * p.nq_pad * (hd + 2) * 4;
  }
  if (dtype == CO_DTYPE_BF16) {
    // share records of the grouped-prefix path (CO_ATTN_SHARED_PREFIX), where it applies
    const int nq = B * (Hq / Hkv);
    if (hd == 64 || nq <= 32) {
      const size_t nqp = nq <= 32 ? 32 : 64;
      const size_t rec = static_cast<size_t>(L) * Hkv * S * group_splits(max_pages) * nqp * (hd + 2) * 4;
      if (rec > p.bytes) p.bytes = rec;
    }
  }
  p.bytes = (p.bytes + 255) / 256 * 256;
  return p;
}

hipError_t launch_attention(const AttnArgs& a, const AttnPlan& p, int layer_count,
                            hipStream_t stream) {
  if (a.S == 0 || layer_count == 0) return hipSuccess;
  const int nt = p.nq_pad / 16;
  // merge grid: one workgroup per 256 (query row, dims) items of a segment,
  // 16 dims per item with at least kCombineWideSegs segments, else 4
  const bool wide = static_cast<int64_t>(a.S) * layer_count * a.Hkv >= kCombineWideSegs;
  const int items = (a.B * (a.Hq / a.Hkv)) * (a.hd / (wide ? 16 : 4));
  const dim3 mgrid(a.S, layer_count * a.Hkv, (items + 255) / 256);
  const int items_f32 = (a.B * (a.Hq / a.Hkv)) * (a.hd / 4);
  const dim3 fgrid(a.S, layer_count * a.Hkv, (items_f32 + 255) / 256);
  // the extras (self segment, carry mass): the same kernels' EXT instantiations
  // (the grouped-prefix kernel has none: its launches take the other paths)
  const bool ext = a.k_self != nullptr || a.mass != nullptr;
  const int n_wg = p.n_wg, hdr_floats = p.hdr_floats;
  auto combine = [&]() {
    if (wide)
      hipLaunchKernelGGL(attn_bf16_combine_kernel<16>, mgrid, dim3(256), 0, stream, a, layer_count,
                         n_wg, hdr_floats, p.nq_pad);
    else
      hipLaunchKernelGGL(attn_bf16_combine_kernel<4>, mgrid, dim3(256), 0, stream, a, layer_count,
                         n_wg, hdr_floats, p.nq_pad);
  };
  // grouped kernel: any query count with head_dim 64, up to 32 rows with 128
  const int nq = a.B * (a.Hq / a.Hkv);
  const bool one = nq <= 32;
  if (a.dtype == CO_DTYPE_BF16 && !ext && (a.flags & CO_ATTN_SHARED_PREFIX) &&
      (a.hd == 64 || one)) {
    const int ns = group_splits(a.max_pages);
    const dim3 ggrid((a.S + kGroupSeqs - 1) / kGroupSeqs * ns, a.Hkv, layer_count);
    const int sp = group_split_tiles();
    if (a.hd == 64) {
      if (one) hipLaunchKernelGGL((attn_group_kernel<64, 1>), ggrid, dim3(256), 0, stream, a, sp, ns);
      else hipLaunchKernelGGL((attn_group_kernel<64, 2>), ggrid, dim3(256), 0, stream, a, sp, ns);
    } else {
      hipLaunchKernelGGL((attn_group_kernel<128, 1>), ggrid, dim3(256), 0, stream, a, sp, ns);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess || ns == 1) return err;
    const dim3 cgrid(a.S, a.Hkv, layer_count);
    const int nqp = one ? 32 : 64;
    if (a.hd == 64)
      hipLaunchKernelGGL(attn_share_merge_kernel<64>, cgrid, dim3(256), 0, stream, a, sp, ns, nqp, kGroupSeqs);
    else
      hipLaunchKernelGGL(attn_share_merge_kernel<128>, cgrid, dim3(256), 0, stream, a, sp, ns, nqp, kGroupSeqs);
    return hipGetLastError();
  }
  if (a.dtype == CO_DTYPE_BF16 && p.wave) {
    const int nw = wave_waves(a.hd);
    const dim3 wgrid(p.n_wg / nw), wblock(64 * nw);
#define CO_WAVE_LAUNCH(HD, NQT)                                                              \
  do {                                                                                       \
    if (ext)                                                                                 \
      hipLaunchKernelGGL((attn_wave_kernel<HD, NQT, true>), wgrid, wblock, 0, stream, a,     \
                         layer_count, p.n_wg, p.hdr_floats);                                 \
    else                                                                                     \
      hipLaunchKernelGGL((attn_wave_kernel<HD, NQT, false>), wgrid, wblock, 0, stream, a,    \
                         layer_count, p.n_wg, p.hdr_floats);                                 \
  } while (0)
    if (a.hd == 128)
      CO_WAVE_LAUNCH(128, 2);
    else if (p.nq_pad == 32)
      CO_WAVE_LAUNCH(64, 1);
    else
      CO_WAVE_LAUNCH(64, 2);
#undef CO_WAVE_LAUNCH
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    combine();
    return hipGetLastError();
  }
  if (a.dtype == CO_DTYPE_BF16) {
    const dim3 grid(n_wg);
// the extras run with half the wavefronts per workgroup and a deeper ring, so
// that their sums and the self rows fit in the registers (one wavefront per SIMD)
#define CO_ATTN_LAUNCH(HD, NT, NW, NS, PQ, RTM)                                                   \
  do {                                                                                            \
    if (ext)                                                                                      \
      hipLaunchKernelGGL((attn_bf16_kernel<HD, NT, NW / 2, NS * 2, PQ, RTM, true>), grid,         \
                         dim3(32 * NW), 0, stream, a, layer_count, n_wg, hdr_floats,              \
                         p.round_tiles, p.park_off);                                              \
    else                                                                                          \
      hipLaunchKernelGGL((attn_bf16_kernel<HD, NT, NW, NS, PQ, RTM, false>), grid, dim3(64 * NW), \
                         0, stream, a, layer_count, n_wg, hdr_floats, p.round_tiles, p.park_off);  \
  } while (0)
    if (a.hd == 64) {
      switch (nt) {
        case 1: CO_ATTN_LAUNCH(64, 1, kAttnWaves64, 2, 4, kAttnRoundTiles64); break;
        case 2: CO_ATTN_LAUNCH(64, 2, kAttnWaves64, 2, 4, kAttnRoundTiles64); break;
        case 3: CO_ATTN_LAUNCH(64, 3, kAttnWaves64, 2, 2, kAttnRoundTiles64); break;
        default: CO_ATTN_LAUNCH(64, 4, kAttnWaves64, 2, 2, kAttnRoundTiles64); break;
      }
    } else {
      switch (nt) {
        case 1: CO_ATTN_LAUNCH(128, 1, kAttnWaves128, 2, 4, kAttnRoundTiles128); break;
        case 2: CO_ATTN_LAUNCH(128, 2, kAttnWaves128, 2, 2, kAttnRoundTiles128); break;
        case 3: CO_ATTN_LAUNCH(128, 3, kAttnWaves128, 2, 1, kAttnRoundTiles128); break;
        default: CO_ATTN_LAUNCH(128, 4, kAttnWaves128, 2, 1, kAttnRoundTiles128); break;
      }
    }
#undef CO_ATTN_LAUNCH
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    combine();
    return hipGetLastError();
  }
  const dim3 grid(p.n_chunks, a.S, layer_count * a.Hkv);
  if (a.hd == 64)
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  else
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.n_chunks <= 1) return err;
  hipLaunchKernelGGL(attn_chunk_merge_kernel<float>, fgrid, dim3(256), 0, stream, a, p.chunk_pages,
                     p.n_chunks, p.nq_pad);
  return hipGetLastError();
}

}  // namespace co
