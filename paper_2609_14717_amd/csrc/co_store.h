// K/V row stores shared by the projection kernels: rotate the key half of a
// head at the row's absolute position (RoPE applied once, when the row is
// projected: Appendix A, "Cache semantics") and scatter the row to its
// committed page slot or carry row.
#pragma once

#include "co_kernels.h"

namespace co {

// The table kv_store<T> expects for head pair i: radians (fp32) or revolutions
// (bf16) per position.
template <typename T>
__device__ __forceinline__ double rope_table(const KvDest& e, int i) {
  return sizeof(T) == 2 ? e.rope_inv[i] * kInv2Pi : e.rope_inv[i];
}

__device__ __forceinline__ bool is_carry_row(int32_t dst) { return dst < 0 && dst != kSkip; }

constexpr float kRmsEps = 1e-6f;   // epsilon of the RMS normalisation variants

// Per-head key normalisation (a variant; the equations omit normalisation,
// Section 2.1): the key half of head segment `seg` is divided by its root mean
// square over the hd dims and multiplied by the layer's gain, before it is
// rotated.  The segment's hd values are spread over `lanes` consecutive lanes
// (a power of two, aligned within the wavefront, all of them active and
// calling with the same seg), NP pairs (i0+p, i0+p+hd/2) per lane; the sum of
// squares is reduced across them.  Value segments, and calls without a gain,
// return unchanged.
template <int NP>
__device__ __forceinline__ void k_norm(const KvDest& e, int seg, int i0, int lanes, float* lo,
                                       float* hi) {
  if (e.knorm == nullptr || ((seg / e.Hkv) & 1) != 0) return;
  float ss = 0.f;
#pragma unroll
  for (int p = 0; p < NP; ++p) ss = fmaf(lo[p], lo[p], fmaf(hi[p], hi[p], ss));
  for (int off = lanes >> 1; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  const float r = rsqrtf(ss / static_cast<float>(e.hd) + kRmsEps);
  const float* g = e.knorm + (seg / (2 * e.Hkv)) * e.hd;
  const int half = e.hd / 2;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    lo[p] = lo[p] * r * g[i0 + p];
    hi[p] = hi[p] * r * g[i0 + p + half];
  }
}

// ------------------------------------------------------------- K/V stores

// Where a row of segment (layer, head g) lives: element offsets of its dim 0
// in the K page layout ([16][hd]) and of its token slot in the V page layout
// ([hd][16]), and which buffers.  ok is false for a skipped row and for a
// destination out of range (the status word then records it).
struct KvRow {
  int64_t kbase, vbase;
  bool carry, ok;
};

__device__ __forceinline__ KvRow kv_row(const KvDest& e, int row, int32_t dst, int layer, int g) {
  KvRow r{0, 0, false, false};
  if (dst == kSkip) return r;
  const int hd = e.hd;
  int64_t pg;
  int t;
  if (dst >= 0) {
    const int page = dst / kPage;
    t = dst % kPage;
    if (page >= e.num_pages) {
      set_status(e.status, CO_ERR_PAGE_RANGE);
      return r;
    }
    pg = (static_cast<int64_t>(layer) * e.num_pages + page) * e.Hkv + g;
  } else {
    const int c = -1 - dst;
    if (c >= e.CP * kPage) {
      set_status(e.status, CO_ERR_LENGTH);
      return r;
    }
    const int s = row / e.B, cp = c / kPage;
    t = c % kPage;
    pg = ((static_cast<int64_t>(layer) * e.S + s) * e.CP + cp) * e.Hkv + g;
    r.carry = true;
  }
  r.kbase = (pg * kPage + t) * hd;
  r.vbase = pg * hd * kPage + t;
  r.ok = true;
  return r;
}

// Store pairs (i0+p, i0+p+hd/2), p < NP, of head segment `seg` = (layer, K|V, head)
// of window row `row`.  lo/hi hold the unrotated fp32 values of those dims;
// inv_freq[i] = theta^(-2i/hd) in radians per position for fp32 stores, in
// revolutions per position (rope_table) for bf16 stores.
template <typename T, int NP>
__device__ inline void kv_store(const KvDest& e, int row, int32_t dst, int pos, int seg, int i0,
                         const float* lo, const float* hi, const double* inv_freq) {
  const int half = e.hd / 2;
  const int g = seg % e.Hkv;
  const int kind = (seg / e.Hkv) & 1;
  const int layer = seg / (2 * e.Hkv);
  const KvRow r = kv_row(e, row, dst, layer, g);
  if (!r.ok) return;
  if (kind == 0) {
    T* kptr = static_cast<T*>(r.carry ? e.k_carry : e.k_cache);
    if constexpr (sizeof(T) == 2 && NP == 4) {
      // the four dims of each half are contiguous (i0 is a multiple of 4 and
      // a row starts on a multiple of hd): one 8-byte store per half
      u16x4 k_lo, k_hi;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        float c, s;
        rope_cos_sin_rev(pos, inv_freq[i0 + p], &c, &s);
        k_lo[p] = f2bf(lo[p] * c - hi[p] * s);
        k_hi[p] = f2bf(hi[p] * c + lo[p] * s);
      }
      *reinterpret_cast<u16x4*>(kptr + r.kbase + i0) = k_lo;
      *reinterpret_cast<u16x4*>(kptr + r.kbase + i0 + half) = k_hi;
      return;
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      float c, s;
      if constexpr (sizeof(T) == 2)
        rope_cos_sin_rev(pos, inv_freq[i0 + p], &c, &s);
      else
        rope_cos_sin(pos, inv_freq[i0 + p], &c, &s);
      kptr[r.kbase + i0 + p] = to_elem<T>(lo[p] * c - hi[p] * s);
      kptr[r.kbase + i0 + p + half] = to_elem<T>(hi[p] * c + lo[p] * s);
    }
  } else {
    T* vptr = static_cast<T*>(r.carry ? e.v_carry : e.v_cache);
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      vptr[r.vbase + static_cast<int64_t>(i0 + p) * kPage] = to_elem<T>(lo[p]);
      vptr[r.vbase + static_cast<int64_t>(i0 + p + half) * kPage] = to_elem<T>(hi[p]);
    }
  }
}

}  // namespace co
