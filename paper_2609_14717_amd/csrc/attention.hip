// Block-parallel drafter attention over ctx = [C ; U] (Eq. 2; Algorithm 1
// step 7; Section 2 "Preliminaries": every block query attends to K/V built
// from target states).  The committed segment C is read through the page
// table, the carryover segment U from the per-sequence carry pages; both are
// consumed by one online softmax, so the concatenation is never materialised.
//
// Work split (flash-decoding style): the logical pages of a sequence --
// ceil(ctx/16) committed pages followed by ceil(carry/16) carry pages -- are
// cut into chunks of `chunk_pages`; one workgroup per (chunk, sequence,
// layer x KV head) computes all B * (Hq/Hkv) query rows of that KV head over
// its chunk.  A sequence that fits in one chunk is finished in place; otherwise
// each chunk leaves an unnormalised partial (O, running max, running sum) in
// the workspace and a second, light kernel combines the chunks of every such
// (layer, sequence, head) with the log-sum-exp rule.  (Combining inside the
// first kernel would need a device-scope release per workgroup, which on this
// part writes back the whole L2 of the XCD; the kernel boundary is cheaper.)
//
// bf16 path (gfx950 MFMA, wave64):
//   S^T = K . Q^T   per 32-key tile: two 16-key M-tiles whose rows are the
//                   keys {8q+r} and {8q+4+r} (q = lane/16, r < 4), so that the
//                   softmax'ed scores of lane group q are keys 8q..8q+7;
//   O^T += V^T . P^T with V pages stored [head_dim][16 slots]: every lane
//                   reads its 8 keys of one V row with one 16-byte load.
// Keys and values stream from HBM straight into registers, one tile ahead of
// the tile being computed; wavefronts of a workgroup take alternate tiles and
// are merged through LDS.  Queries are rotated once per workgroup into LDS.
#include "co_kernels.h"

namespace co {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaxChunkPages = 64;

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

// Partial record of (layer, seq, kv head, chunk): O[nq_pad][hd], m[nq_pad], l[nq_pad]
// (m in log2 units of the scaled logits; O unnormalised).
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

// Combine the chunk records of every (layer, sequence, KV head) whose key set
// spans more than one chunk, and write O (+ LSE).  One thread per (query row,
// 4 output dims); each thread issues all of its record loads at once.
template <typename T>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a, int chunk_pages,
                                                         int n_chunks, int nq_pad) {
  const int s = blockIdx.x;
  const int layer_local = blockIdx.y / a.Hkv, g = blockIdx.y % a.Hkv;
  const SeqInfo si = seq_info(a, s, chunk_pages);
  if (si.nch <= 1) return;                 // finished by the chunk kernel
  const int hd = a.hd, G = a.Hq / a.Hkv, nq = a.B * G, q4 = hd / 4;
  const float* base = record_ptr(a, layer_local, s, g, 0, n_chunks, nq_pad);
  const int64_t rec = static_cast<int64_t>(nq_pad) * (hd + 2);
  T* out = static_cast<T*>(a.out);
  for (int idx = threadIdx.x + blockIdx.z * 256; idx < nq * q4; idx += 256 * gridDim.z) {
    const int n = idx / q4, d = (idx % q4) * 4;
    float M = -INFINITY;
    for (int c = 0; c < si.nch; ++c) M = fmaxf(M, base[c * rec + nq_pad * hd + n]);
    float den = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < si.nch; ++c) {
      const float m = base[c * rec + nq_pad * hd + n];
      const float wgt = (m == -INFINITY) ? 0.f : exp2f(m - M);
      den += wgt * base[c * rec + nq_pad * hd + nq_pad + n];
      acc += wgt * *reinterpret_cast<const f32x4*>(base + c * rec + n * hd + d);
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    const int64_t row = out_row(a, layer_local, s, g, n, G);
    T* o = out + row * hd + d;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = to_elem<T>(acc[r] * inv);
    if (a.lse && d == 0) a.lse[row] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
  }
}

template <int HD>
struct Tile {
  u16x8 ka[HD / 32], kb[HD / 32], va[HD / 16];
  int nv;
};

template <int HD, int NT, int NW>
__global__ __launch_bounds__(64 * NW) void attn_bf16_kernel(AttnArgs a, int chunk_pages,
                                                             int n_chunks) {
  constexpr int KS = HD / 32;   // k-steps of S^T
  constexpr int MT = HD / 16;   // M-tiles of O^T
  constexpr int NQP = NT * 16;
  constexpr int NTHR = 64 * NW;
  constexpr int QLD = HD + 8;   // padded LDS row of rotated queries (bf16)
  constexpr int NRED = NW > 1 ? NW - 1 : 1;
  __shared__ __align__(16) uint16_t q_lds[NQP * QLD];
  __shared__ int pg_lds[kMaxChunkPages];
  __shared__ float red_o[NRED][NQP][HD + 1];
  __shared__ float red_m[NRED][NQP], red_l[NRED][NQP];

  const int c = blockIdx.x, s = blockIdx.y;
  const int layer_local = blockIdx.z / a.Hkv, g = blockIdx.z % a.Hkv;
  const int layer = a.layer_begin + layer_local;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = lane >> 4, col = lane & 15;

  const SeqInfo si = seq_info(a, s, chunk_pages);
  if (!si.ok) {
    if (c == 0 && tid == 0) set_status(a.status, CO_ERR_LENGTH);
    return;
  }
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  if (si.npt == 0) {            // no keys at all: O = 0, LSE = -inf
    if (c != 0) return;
    uint16_t* out = static_cast<uint16_t*>(a.out);
    for (int idx = tid; idx < nq * HD; idx += NTHR)
      out[out_row(a, layer_local, s, g, idx / HD, G) * HD + idx % HD] = 0;
    if (a.lse)
      for (int n = tid; n < nq; n += NTHR) a.lse[out_row(a, layer_local, s, g, n, G)] = -INFINITY;
    return;
  }
  const int p_begin = c * chunk_pages;
  if (p_begin >= si.npt) return;
  const int p_end = min(p_begin + chunk_pages, si.npt);
  const int n_tiles = (p_end - p_begin + 1) / 2;

  // ---- physical ids of this chunk's committed pages (-1: carry page, -2: bad id)
  for (int i = tid; i < p_end - p_begin; i += NTHR) {
    const int lp = p_begin + i;
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
  // ---- queries: rotate at ctx + i, fold 1/sqrt(hd) * log2(e), store bf16 in LDS
  {
    const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;
    const uint16_t* Q = static_cast<const uint16_t*>(a.q);
    for (int idx = tid; idx < NQP * (HD / 2); idx += NTHR) {
      const int n = idx / (HD / 2), p = idx % (HD / 2);
      float lo = 0.f, hi = 0.f;
      if (n < nq) {
        const uint16_t* qrow = Q + out_row(a, layer_local, s, g, n, G) * HD;
        lo = bf2f(qrow[p]);
        hi = bf2f(qrow[p + HD / 2]);
        if (!(a.flags & CO_Q_PREROTATED)) {
          float cs, sn;
          rope_cos_sin(si.ctx + n / G, rope_inv_freq(p, HD, a.log2_theta), &cs, &sn);
          const float l2 = lo * cs - hi * sn, h2 = hi * cs + lo * sn;
          lo = l2;
          hi = h2;
        }
      }
      q_lds[n * QLD + p] = f2bf(lo * qscale);
      q_lds[n * QLD + p + HD / 2] = f2bf(hi * qscale);
    }
  }
  __syncthreads();
  // Query fragments (B operand of S^T) stay in registers unless that would
  // crowd out the double-buffered K/V tiles; then they are re-read from LDS.
  constexpr bool kQInRegs = NT * KS <= 8;
  u16x8 qf[kQInRegs ? NT : 1][KS];
  if constexpr (kQInRegs) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[nt][ks] = *reinterpret_cast<const u16x8*>(q_lds + (nt * 16 + col) * QLD + ks * 32 + grp * 8);
  }
  auto qfrag = [&](int nt, int ks) -> u16x8 {
    if constexpr (kQInRegs) return qf[nt][ks];
    return *reinterpret_cast<const u16x8*>(q_lds + (nt * 16 + col) * QLD + ks * 32 + grp * 8);
  };

  // key of S^T M-tile a / b at row rho = lane % 16
  const int key_a = 8 * (col >> 2) + (col & 3);
  const int key_b = key_a + 4;
  const uint16_t* kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* vc = static_cast<const uint16_t*>(a.v_cache);
  const uint16_t* kk = static_cast<const uint16_t*>(a.k_carry);
  const uint16_t* vk = static_cast<const uint16_t*>(a.v_carry);

  auto page = [&](int lp, const uint16_t*& kp, const uint16_t*& vp, int& nvalid) {
    kp = kk;
    vp = vk;
    nvalid = 0;
    if (lp >= p_end) return;
    if (lp < si.npc) {
      const int phys = pg_lds[lp - p_begin];
      if (phys < 0) return;
      const int64_t off = ((static_cast<int64_t>(layer) * a.num_pages + phys) * a.Hkv + g) * kPage * HD;
      kp = kc + off;
      vp = vc + off;
      nvalid = min(kPage, si.ctx - lp * kPage);
    } else {
      const int cp = lp - si.npc;
      const int64_t off =
          (((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp) * a.Hkv + g) * kPage * HD;
      kp = kk + off;
      vp = vk + off;
      nvalid = min(kPage, si.carry - cp * kPage);
    }
  };
  auto load_tile = [&](int t, Tile<HD>& T) {
    const int lp0 = p_begin + 2 * t;
    const uint16_t *k0, *v0, *k1, *v1;
    int n0, n1;
    page(lp0, k0, v0, n0);
    page(lp0 + 1, k1, v1, n1);
    const uint16_t* pa = ((key_a >> 4) ? k1 : k0) + (key_a & 15) * HD + grp * 8;
    const uint16_t* pb = ((key_b >> 4) ? k1 : k0) + (key_b & 15) * HD + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      T.ka[ks] = *reinterpret_cast<const u16x8*>(pa + ks * 32);
      T.kb[ks] = *reinterpret_cast<const u16x8*>(pb + ks * 32);
    }
    // V (A operand of O^T): hd row 16*mt + col, keys 8*grp .. +7 (page grp/2)
    T.nv = (grp >> 1) ? n1 : n0;
    const uint16_t* pv = ((grp >> 1) ? v1 : v0) + col * kPage + (grp & 1) * 8;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) T.va[mt] = *reinterpret_cast<const u16x8*>(pv + mt * 16 * kPage);
  };

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

  auto compute_tile = [&](Tile<HD>& T) {
    const int slot_base = (grp & 1) * 8;
    // zero the values of invalid keys (their slots may hold anything)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (slot_base + e >= T.nv) T.va[mt][e] = 0;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u16x8 qv = qfrag(nt, ks);
        sa = mfma16x16x32(T.ka[ks], qv, sa);
        sb = mfma16x16x32(T.kb[ks], qv, sb);
      }
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sa[r] = (slot_base + r < T.nv) ? sa[r] : -INFINITY;
        sb[r] = (slot_base + 4 + r < T.nv) ? sb[r] : -INFINITY;
        mx = fmaxf(mx, fmaxf(sa[r], sb[r]));
      }
      mx = wave_max_across_groups(mx);
      const float m_new = fmaxf(m_run[nt], mx);
      const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m_run[nt] - m_new);
      const float base = (m_new == -INFINITY) ? 0.f : m_new;
      u16x8 pk;
      float psum = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float pa = exp2f(sa[r] - base), pb = exp2f(sb[r] - base);
        psum += pa + pb;
        pk[r] = f2bf(pa);
        pk[4 + r] = f2bf(pb);
      }
      l_run[nt] = l_run[nt] * alpha + psum;
      m_run[nt] = m_new;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        o[mt][nt] *= alpha;
        o[mt][nt] = mfma16x16x32(T.va[mt], pk, o[mt][nt]);
      }
    }
  };

  // tiles wave, wave + NW, ...; the next tile's loads are in flight during compute
  // (when the register file allows a second tile buffer)
  constexpr bool kPrefetch = MT * NT <= 16;
  if constexpr (!kPrefetch) {
    Tile<HD> t0;
    for (int t = wave; t < n_tiles; t += NW) {
      load_tile(t, t0);
      compute_tile(t0);
    }
  } else {
    Tile<HD> t0, t1;
    int t = wave;
    if (t < n_tiles) load_tile(t, t0);
    while (t < n_tiles) {
      if (t + NW < n_tiles) load_tile(t + NW, t1);
      compute_tile(t0);
      t += NW;
      if (t >= n_tiles) break;
      if (t + NW < n_tiles) load_tile(t + NW, t0);
      compute_tile(t1);
      t += NW;
    }
  }

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) l_run[nt] = wave_sum_across_groups(l_run[nt]);

  // ---- merge the wavefronts of this workgroup through LDS into wave 0
  if constexpr (NW > 1) {
    if (wave > 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int n = nt * 16 + col;
        if (grp == 0) {
          red_m[wave - 1][n] = m_run[nt];
          red_l[wave - 1][n] = l_run[nt];
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) red_o[wave - 1][n][mt * 16 + grp * 4 + r] = o[mt][nt][r];
      }
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int n = nt * 16 + col;
        float M = m_run[nt];
#pragma unroll
        for (int w = 1; w < NW; ++w) M = fmaxf(M, red_m[w - 1][n]);
        const float f0 = (m_run[nt] == -INFINITY) ? 0.f : exp2f(m_run[nt] - M);
        float lsum = l_run[nt] * f0;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) o[mt][nt] *= f0;
#pragma unroll
        for (int w = 1; w < NW; ++w) {
          const float mw = red_m[w - 1][n];
          const float fw = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
          lsum += red_l[w - 1][n] * fw;
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) o[mt][nt][r] += fw * red_o[w - 1][n][mt * 16 + grp * 4 + r];
        }
        m_run[nt] = M;
        l_run[nt] = lsum;
      }
    }
  }

  if (si.nch == 1) {
    // the whole key set is in this chunk: normalise and write O / LSE directly
    if (wave != 0) return;
    uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + col;
      if (n >= nq) continue;
      const float inv = l_run[nt] > 0.f ? 1.f / l_run[nt] : 0.f;
      const int64_t row = out_row(a, layer_local, s, g, n, G);
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
    return;
  }

  if (wave == 0) {
    float* part = record_ptr(a, layer_local, s, g, c, n_chunks, NQP);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + col;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        *reinterpret_cast<f32x4*>(part + n * HD + mt * 16 + grp * 4) = o[mt][nt];
      if (grp == 0) {
        part[NQP * HD + n] = m_run[nt];
        part[NQP * HD + NQP + n] = l_run[nt];
      }
    }
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

}  // namespace

AttnPlan plan_attention(int S, int B, int L, int Hq, int Hkv, int hd, int max_pages, int dtype) {
  (void)dtype;
  AttnPlan p{};
  const int nq = B * (Hq / Hkv);
  p.nq_pad = (nq + 15) / 16 * 16;
  const int cp = (B + kPage - 1) / kPage;
  const int max_lp = max_pages + cp;
  // Larger records (many query rows, wide heads) get longer chunks so that the
  // partial records stay a small fraction of the key/value bytes they summarise.
  p.chunk_pages = (hd == 64 && p.nq_pad <= 32) ? 32 : kMaxChunkPages;
  p.n_chunks = (max_lp + p.chunk_pages - 1) / p.chunk_pages;
  p.bytes = static_cast<size_t>(L) * S * Hkv * p.n_chunks * p.nq_pad * (hd + 2) * 4;
  p.bytes = (p.bytes + 255) / 256 * 256;
  return p;
}

hipError_t launch_attention(const AttnArgs& a_in, const AttnPlan& p, int layer_count,
                            hipStream_t stream) {
  if (a_in.S == 0 || layer_count == 0) return hipSuccess;
  const AttnArgs& a = a_in;
  const dim3 grid(p.n_chunks, a.S, layer_count * a.Hkv);
  const int nt = p.nq_pad / 16;
  if (a.dtype == CO_DTYPE_BF16) {
    if (a.hd == 64) {
      switch (nt) {
        case 1: hipLaunchKernelGGL((attn_bf16_kernel<64, 1, 4>), grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks); break;
        case 2: hipLaunchKernelGGL((attn_bf16_kernel<64, 2, 4>), grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks); break;
        case 3: hipLaunchKernelGGL((attn_bf16_kernel<64, 3, 4>), grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks); break;
        default: hipLaunchKernelGGL((attn_bf16_kernel<64, 4, 4>), grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks); break;
      }
    } else {
      switch (nt) {
        case 1: hipLaunchKernelGGL((attn_bf16_kernel<128, 1, 2>), grid, dim3(128), 0, stream, a, p.chunk_pages, p.n_chunks); break;
        case 2: hipLaunchKernelGGL((attn_bf16_kernel<128, 2, 2>), grid, dim3(128), 0, stream, a, p.chunk_pages, p.n_chunks); break;
        case 3: hipLaunchKernelGGL((attn_bf16_kernel<128, 3, 2>), grid, dim3(128), 0, stream, a, p.chunk_pages, p.n_chunks); break;
        default: hipLaunchKernelGGL((attn_bf16_kernel<128, 4, 2>), grid, dim3(128), 0, stream, a, p.chunk_pages, p.n_chunks); break;
      }
    }
  } else {
    if (a.hd == 64)
      hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
    else
      hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || p.n_chunks <= 1) return err;
  const int items = (a.B * (a.Hq / a.Hkv)) * (a.hd / 4);
  const dim3 mgrid(a.S, layer_count * a.Hkv, (items + 255) / 256);
  if (a.dtype == CO_DTYPE_BF16)
    hipLaunchKernelGGL(attn_merge_kernel<uint16_t>, mgrid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  else
    hipLaunchKernelGGL(attn_merge_kernel<float>, mgrid, dim3(256), 0, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  return hipGetLastError();
}

}  // namespace co
