// Block-parallel drafter attention over ctx = [C ; U] (Eq. 2; Algorithm 1
// step 7; Section 2 "Preliminaries": every block query attends to K/V built
// from target states).  The committed segment C is read through the page
// table, the carryover segment U from the per-sequence carry pages; both are
// consumed by one online softmax, so the concatenation is never materialised.
//
// Work split (flash-decoding style): the logical pages of a sequence --
// ceil(ctx/16) committed pages followed by ceil(carry/16) carry pages -- are
// cut into chunks of `chunk_pages`; one workgroup per (chunk, sequence,
// layer x KV head) computes an unnormalised partial (O, running max, running
// sum) for all B * (Hq/Hkv) query rows of that KV head, and a merge kernel
// combines the chunks with the usual log-sum-exp rule.
//
// bf16 path (gfx950 MFMA, wave64):
//   S^T = K . Q^T   per 32-key tile: two 16-key M-tiles whose rows are the
//                   keys {8q+r} and {8q+4+r} (q = lane/16, r < 4), so that the
//                   softmax'ed scores of lane group q are keys 8q..8q+7;
//   O^T += V^T . P^T with V pages stored [head_dim][16 slots]: every lane
//                   reads its 8 keys of one V row with one 16-byte load.
// Keys and values are read straight from HBM into registers (no reuse across
// wavefronts); wavefronts of a workgroup take alternate tiles of the chunk and
// are merged through LDS at the end.
#include "co_kernels.h"

namespace co {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct PageRef {
  const uint16_t* k;
  const uint16_t* v;
  int nvalid;
};

template <int HD>
__device__ __forceinline__ PageRef page_ref(const AttnArgs& a, int layer, int s, int g, int lp,
                                            int npc, int ctx, int carry, int p_end) {
  PageRef r;
  if (lp >= p_end) {
    r.k = static_cast<const uint16_t*>(a.k_carry);
    r.v = static_cast<const uint16_t*>(a.v_carry);
    r.nvalid = 0;
    return r;
  }
  if (lp < npc) {
    const int phys = a.page_table[static_cast<int64_t>(s) * a.max_pages + lp];
    if (phys < 0 || phys >= a.num_pages) {
      set_status(a.status, CO_ERR_PAGE_RANGE);
      r.k = static_cast<const uint16_t*>(a.k_carry);
      r.v = static_cast<const uint16_t*>(a.v_carry);
      r.nvalid = 0;
      return r;
    }
    const int64_t off = ((static_cast<int64_t>(layer) * a.num_pages + phys) * a.Hkv + g) * kPage * HD;
    r.k = static_cast<const uint16_t*>(a.k_cache) + off;
    r.v = static_cast<const uint16_t*>(a.v_cache) + off;
    r.nvalid = min(kPage, ctx - lp * kPage);
  } else {
    const int cp = lp - npc;
    const int64_t off =
        (((static_cast<int64_t>(layer) * a.S + s) * a.CP + cp) * a.Hkv + g) * kPage * HD;
    r.k = static_cast<const uint16_t*>(a.k_carry) + off;
    r.v = static_cast<const uint16_t*>(a.v_carry) + off;
    r.nvalid = min(kPage, carry - cp * kPage);
  }
  return r;
}

__device__ __forceinline__ float wave_max_across_groups(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}

__device__ __forceinline__ float wave_sum_across_groups(float v) {
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}

// Partial record of one (layer, seq, kv head, chunk): O[nq_pad][HD], m[nq_pad], l[nq_pad]
// (m in log2 units of the scaled logits; O unnormalised).
__device__ __forceinline__ float* partial_ptr(float* ws, int layer_local, int s, int g, int c,
                                              int S, int Hkv, int n_chunks, int nq_pad, int hd) {
  const int64_t rec = ((static_cast<int64_t>(layer_local) * S + s) * Hkv + g) * n_chunks + c;
  return ws + rec * nq_pad * (hd + 2);
}

template <int HD, int NT, int NW>
__global__ __launch_bounds__(64 * NW) void attn_bf16_kernel(AttnArgs a, int chunk_pages,
                                                             int n_chunks) {
  constexpr int KS = HD / 32;   // k-steps of S^T
  constexpr int MT = HD / 16;   // M-tiles of O^T
  constexpr int NQP = NT * 16;
  const int c = blockIdx.x, s = blockIdx.y;
  const int layer_local = blockIdx.z / a.Hkv, g = blockIdx.z % a.Hkv;
  const int layer = a.layer_begin + layer_local;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane >> 4, col = lane & 15;

  const int ctx = a.ctx_len[s], carry = a.carry_len[s];
  if (ctx < 0 || ctx > a.max_pages * kPage || carry < 0 || carry > a.CP * kPage) {
    if (c == 0 && threadIdx.x == 0) set_status(a.status, CO_ERR_LENGTH);
    return;
  }
  const int npc = (ctx + kPage - 1) / kPage;
  const int npt = npc + (carry + kPage - 1) / kPage;
  const int p_begin = c * chunk_pages;
  if (p_begin >= npt) return;
  const int p_end = min(p_begin + chunk_pages, npt);
  const int n_tiles = (p_end - p_begin + 1) / 2;

  const int G = a.Hq / a.Hkv, nq = a.B * G;

  // ---- queries: rotate at ctx + i, fold 1/sqrt(hd) * log2(e), keep as B fragments
  u16x8 qf[NT][KS];
  {
    const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;
    const double log2_theta = a.log2_theta;
    const uint16_t* Q = static_cast<const uint16_t*>(a.q);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + col;
      float x[KS][8];
      if (n < nq) {
        const int i = n / G, hh = n % G;
        const uint16_t* qrow =
            Q + ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq * HD +
            static_cast<int64_t>(g * G + hh) * HD;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const u16x8 v = *reinterpret_cast<const u16x8*>(qrow + ks * 32 + grp * 8);
#pragma unroll
          for (int e = 0; e < 8; ++e) x[ks][e] = bf2f(v[e]);
        }
        if (!(a.flags & CO_Q_PREROTATED)) {
          const int pos = ctx + i;
#pragma unroll
          for (int ks = 0; ks < KS / 2; ++ks)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              float cs, sn;
              rope_cos_sin(pos, rope_inv_freq(ks * 32 + grp * 8 + e, HD, log2_theta), &cs, &sn);
              const float lo = x[ks][e], hi = x[ks + KS / 2][e];
              x[ks][e] = lo * cs - hi * sn;
              x[ks + KS / 2][e] = hi * cs + lo * sn;
            }
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) x[ks][e] = 0.f;
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[nt][ks][e] = f2bf(x[ks][e] * qscale);
    }
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

  // key of S^T M-tile a / b at row rho = lane % 16
  const int key_a = 8 * (col >> 2) + (col & 3);
  const int key_b = key_a + 4;

  for (int t = wave; t < n_tiles; t += NW) {
    const int lp0 = p_begin + 2 * t;
    const PageRef p0 = page_ref<HD>(a, layer, s, g, lp0, npc, ctx, carry, p_end);
    const PageRef p1 = page_ref<HD>(a, layer, s, g, lp0 + 1, npc, ctx, carry, p_end);
    // K fragments (A operand of S^T); keys 16..31 of the tile live in the second page
    u16x8 ka[KS], kb[KS];
    {
      const uint16_t* pa = ((key_a >> 4) ? p1.k : p0.k) + (key_a & 15) * HD + grp * 8;
      const uint16_t* pb = ((key_b >> 4) ? p1.k : p0.k) + (key_b & 15) * HD + grp * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        ka[ks] = *reinterpret_cast<const u16x8*>(pa + ks * 32);
        kb[ks] = *reinterpret_cast<const u16x8*>(pb + ks * 32);
      }
    }
    // V fragments (A operand of O^T): hd row 16*mt + col, keys 8*grp .. +7
    u16x8 va[MT];
    const int vvalid = (grp >> 1) ? p1.nvalid : p0.nvalid;
    {
      const uint16_t* vbase = (grp >> 1) ? p1.v : p0.v;
      const int slot0 = (grp & 1) * 8;
      const uint16_t* pv = vbase + col * kPage + slot0;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        u16x8 v = *reinterpret_cast<const u16x8*>(pv + mt * 16 * kPage);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (slot0 + e >= vvalid) v[e] = 0;
        va[mt] = v;
      }
    }
    // validity of this lane's score rows: tile a row 4*grp+r is key 8*grp+r, tile b 8*grp+4+r
    const int slot_base = (grp & 1) * 8;
    const int nv = vvalid;

#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        sa = mfma16x16x32(ka[ks], qf[nt][ks], sa);
        sb = mfma16x16x32(kb[ks], qf[nt][ks], sb);
      }
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sa[r] = (slot_base + r < nv) ? sa[r] : -INFINITY;
        sb[r] = (slot_base + 4 + r < nv) ? sb[r] : -INFINITY;
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
        o[mt][nt] = mfma16x16x32(va[mt], pk, o[mt][nt]);
      }
    }
  }

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) l_run[nt] = wave_sum_across_groups(l_run[nt]);

  // ---- merge the wavefronts of this workgroup through LDS, then store the partial
  float* part = partial_ptr(a.ws, layer_local, s, g, c, a.S, a.Hkv, n_chunks, NQP, HD);
  if constexpr (NW > 1) {
    __shared__ float sm_o[NW - 1][NQP][HD + 1];
    __shared__ float sm_m[NW - 1][NQP];
    __shared__ float sm_l[NW - 1][NQP];
    if (wave > 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int n = nt * 16 + col;
        if (grp == 0) {
          sm_m[wave - 1][n] = m_run[nt];
          sm_l[wave - 1][n] = l_run[nt];
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) sm_o[wave - 1][n][mt * 16 + grp * 4 + r] = o[mt][nt][r];
      }
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + col;
      float M = m_run[nt];
#pragma unroll
      for (int w = 1; w < NW; ++w) M = fmaxf(M, sm_m[w - 1][n]);
      const float f0 = (m_run[nt] == -INFINITY) ? 0.f : exp2f(m_run[nt] - M);
      float lsum = l_run[nt] * f0;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) o[mt][nt] *= f0;
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        const float mw = sm_m[w - 1][n];
        const float fw = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
        lsum += sm_l[w - 1][n] * fw;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) o[mt][nt][r] += fw * sm_o[w - 1][n][mt * 16 + grp * 4 + r];
      }
      m_run[nt] = M;
      l_run[nt] = lsum;
    }
  }
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

// fp32 path: the same partials, computed with plain VALU arithmetic through LDS.
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
  const int ctx = a.ctx_len[s], carry = a.carry_len[s];
  if (ctx < 0 || ctx > a.max_pages * kPage || carry < 0 || carry > a.CP * kPage) {
    if (c == 0 && tid == 0) set_status(a.status, CO_ERR_LENGTH);
    return;
  }
  const int npc = (ctx + kPage - 1) / kPage;
  const int npt = npc + (carry + kPage - 1) / kPage;
  const int p_begin = c * chunk_pages;
  if (p_begin >= npt) return;
  const int p_end = min(p_begin + chunk_pages, npt);
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  const float* Q = static_cast<const float*>(a.q);
  const float qscale = rsqrtf(static_cast<float>(HD)) * kLog2e;

  for (int idx = tid; idx < nq * (HD / 2); idx += 256) {
    const int n = idx / (HD / 2), p = idx % (HD / 2);
    const int i = n / G, hh = n % G;
    const float* qrow = Q + ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq * HD +
                        static_cast<int64_t>(g * G + hh) * HD;
    float lo = qrow[p], hi = qrow[p + HD / 2];
    if (!(a.flags & CO_Q_PREROTATED)) {
      float cs, sn;
      rope_cos_sin(ctx + i, rope_inv_freq(p, HD, a.log2_theta), &cs, &sn);
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
  float* part = partial_ptr(a.ws, layer_local, s, g, c, a.S, a.Hkv, n_chunks, nq_pad, HD);
  for (int idx = tid; idx < nq * HD; idx += 256) part[idx] = os[idx / HD][idx % HD];
  if (tid < nq) {
    part[nq_pad * HD + tid] = m_run[tid];
    part[nq_pad * HD + nq_pad + tid] = l_run[tid];
  }
}

// Combine the chunk partials of one (sequence, layer, KV head) and write O (+ LSE).
template <typename T>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a, int chunk_pages,
                                                         int n_chunks, int nq_pad) {
  extern __shared__ float w_s[];          // [n_chunks][nq_pad] chunk weights
  __shared__ float inv_den[64];
  const int s = blockIdx.x;
  const int layer_local = blockIdx.y / a.Hkv, g = blockIdx.y % a.Hkv;
  const int tid = threadIdx.x;
  const int hd = a.hd, G = a.Hq / a.Hkv, nq = a.B * G;
  const int ctx = a.ctx_len[s], carry = a.carry_len[s];
  const bool ok = ctx >= 0 && ctx <= a.max_pages * kPage && carry >= 0 && carry <= a.CP * kPage;
  const int npt = ok ? (ctx + kPage - 1) / kPage + (carry + kPage - 1) / kPage : 0;
  const int nch = (npt + chunk_pages - 1) / chunk_pages;
  const float* base = partial_ptr(a.ws, layer_local, s, g, 0, a.S, a.Hkv, n_chunks, nq_pad, hd);
  const int64_t rec = static_cast<int64_t>(nq_pad) * (hd + 2);

  if (tid < nq) {
    float M = -INFINITY;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, base[c * rec + nq_pad * hd + tid]);
    float den = 0.f;
    for (int c = 0; c < nch; ++c) {
      const float m = base[c * rec + nq_pad * hd + tid];
      const float w = (m == -INFINITY) ? 0.f : exp2f(m - M);
      w_s[c * nq_pad + tid] = w;
      den += w * base[c * rec + nq_pad * hd + nq_pad + tid];
    }
    inv_den[tid] = den > 0.f ? 1.f / den : 0.f;
    if (a.lse) {
      const int i = tid / G, hh = tid % G;
      const int64_t oi = ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq + g * G + hh;
      a.lse[oi] = den > 0.f ? (M + log2f(den)) * kLn2 : -INFINITY;
    }
  }
  __syncthreads();
  T* out = static_cast<T*>(a.out);
  for (int idx = tid; idx < nq * hd; idx += 256) {
    const int n = idx / hd, dd = idx % hd;
    float acc = 0.f;
    for (int c = 0; c < nch; ++c) acc += w_s[c * nq_pad + n] * base[c * rec + n * hd + dd];
    const int i = n / G, hh = n % G;
    const int64_t oi =
        (((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq + g * G + hh) * hd + dd;
    out[oi] = to_elem<T>(acc * inv_den[n]);
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
  p.chunk_pages = 64;
  // keep the merge kernel's per-chunk weights within 32 KiB of LDS
  while (((max_lp + p.chunk_pages - 1) / p.chunk_pages) * p.nq_pad * 4 > 32768) p.chunk_pages *= 2;
  p.n_chunks = (max_lp + p.chunk_pages - 1) / p.chunk_pages;
  p.bytes = static_cast<size_t>(L) * S * Hkv * p.n_chunks * p.nq_pad * (hd + 2) * 4;
  p.bytes = (p.bytes + 255) / 256 * 256;
  return p;
}

hipError_t launch_attention(const AttnArgs& a, const AttnPlan& p, int layer_count,
                            hipStream_t stream) {
  if (a.S == 0 || layer_count == 0) return hipSuccess;
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
  if (err != hipSuccess) return err;
  const dim3 mgrid(a.S, layer_count * a.Hkv);
  const size_t lds = static_cast<size_t>(p.n_chunks) * p.nq_pad * 4;
  if (a.dtype == CO_DTYPE_BF16)
    hipLaunchKernelGGL(attn_merge_kernel<uint16_t>, mgrid, dim3(256), lds, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  else
    hipLaunchKernelGGL(attn_merge_kernel<float>, mgrid, dim3(256), lds, stream, a, p.chunk_pages, p.n_chunks, p.nq_pad);
  return hipGetLastError();
}

}  // namespace co
