// Extra attention segments next to ctx = [C;U] (Eq. 2), computed from a
// finished attention call's O and LSE:
//   * the share of each block query's attention that falls on the carried rows
//     (the diagnostic of Appendix "Attention to carried states"): with LSE over
//     [C;U] and LSE_U over U alone, mass = exp(LSE_U - LSE);
//   * the block's own rows S as a third, non-causal segment: attention of the
//     queries over S alone, merged into (O, LSE) by the log-sum-exp rule, which
//     gives the attention over [C;U;S] in one softmax.
// Both segments hold at most `block` rows, so one workgroup per (sequence, KV
// head, layer) stages them in LDS in fp32.
#include "co_kernels.h"

namespace co {

namespace {

template <typename T, int HD>
__global__ __launch_bounds__(256) void carry_mass_kernel(MassArgs a) {
  constexpr int LD = HD + 4;                   // fp32 rows, 16-byte aligned
  constexpr int NQ = 64;                       // query rows per KV head (checked on the host)
  __shared__ __align__(16) float ks[kMaxCarryRows * LD];
  __shared__ __align__(16) float qs[NQ * LD];
  __shared__ float lg[NQ][kMaxCarryRows + 1];
  __shared__ double inv_lds[HD / 2];
  const int s = blockIdx.x, g = blockIdx.y, layer_local = blockIdx.z;
  const int layer = a.layer_begin + layer_local;
  const int tid = threadIdx.x;
  const int G = a.Hq / a.Hkv, nq = a.B * G;
  const int ctx = a.ctx_len[s];
  int carry = a.carry_len[s];
  if (ctx < 0 || carry < 0 || carry > a.CP * kPage) {
    if (tid == 0) set_status(a.status, CO_ERR_LENGTH);
    carry = 0;
  }
  auto row_of = [&](int n) {   // (layer, sequence, block row, query head) of query row n
    return ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + n / G) * a.Hq + g * G + n % G;
  };
  if (carry == 0) {            // nothing carried
    for (int n = tid; n < nq; n += 256) a.mass[row_of(n)] = 0.f;
    return;
  }
  // carry keys, fp32
  const T* kk = static_cast<const T*>(a.k_carry);
  for (int idx = tid; idx < carry * HD; idx += 256) {
    const int t = idx / HD, d = idx % HD;
    const int64_t off =
        ((((static_cast<int64_t>(layer) * a.S + s) * a.CP + t / kPage) * a.Hkv + g) * kPage +
         t % kPage) * HD + d;
    if constexpr (sizeof(T) == 2)
      ks[t * LD + d] = bf2f(kk[off]);
    else
      ks[t * LD + d] = kk[off];
  }
  if (tid < HD / 2)   // revolutions per position for bf16, radians for fp32
    inv_lds[tid] = sizeof(T) == 2 ? a.rope_inv[tid] * kInv2Pi : a.rope_inv[tid];
  __syncthreads();
  // queries rotated at ctx + i and scaled by 1/sqrt(hd), one pair per thread-step
  const T* Q = static_cast<const T*>(a.q);
  const float scale = rsqrtf(static_cast<float>(HD));
  for (int idx = tid; idx < nq * (HD / 2); idx += 256) {
    const int n = idx / (HD / 2), p = idx % (HD / 2);
    const int64_t base = row_of(n) * HD;
    float lo, hi;
    if constexpr (sizeof(T) == 2) {
      lo = bf2f(Q[base + p]);
      hi = bf2f(Q[base + p + HD / 2]);
    } else {
      lo = Q[base + p];
      hi = Q[base + p + HD / 2];
    }
    if (!(a.flags & CO_Q_PREROTATED)) {
      float c, sn;
      if constexpr (sizeof(T) == 2)
        rope_cos_sin_rev(ctx + n / G, inv_lds[p], &c, &sn);
      else
        rope_cos_sin(ctx + n / G, inv_lds[p], &c, &sn);
      const float l2 = lo * c - hi * sn, h2 = hi * c + lo * sn;
      lo = l2;
      hi = h2;
    }
    qs[n * LD + p] = lo * scale;
    qs[n * LD + p + HD / 2] = hi * scale;
  }
  __syncthreads();
  // logits of every (query row, carry key) pair
  for (int idx = tid; idx < nq * carry; idx += 256) {
    const int n = idx / carry, t = idx % carry;
    const f32x4* qv = reinterpret_cast<const f32x4*>(qs + n * LD);
    const f32x4* kv = reinterpret_cast<const f32x4*>(ks + t * LD);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int d = 0; d < HD / 4; ++d) acc += qv[d] * kv[d];
    lg[n][t] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  __syncthreads();
  // log-sum-exp over the carry keys, against the attention's LSE
  for (int n = tid; n < nq; n += 256) {
    float mx = -INFINITY;
    for (int t = 0; t < carry; ++t) mx = fmaxf(mx, lg[n][t]);
    float sum = 0.f;
    for (int t = 0; t < carry; ++t) sum += expf(lg[n][t] - mx);
    const int64_t row = row_of(n);
    const float lse = a.lse[row];
    a.mass[row] = lse == -INFINITY ? 0.f : expf(mx + logf(sum) - lse);
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void self_merge_kernel(SelfArgs a) {
  constexpr int LD = HD + 4;                   // fp32 rows, 16-byte aligned
  constexpr int NQ = 64;                       // query rows per KV head (checked on the host)
  constexpr int NB = kMaxCarryRows;            // block rows (checked on the host)
  __shared__ __align__(16) float ks[NB * LD];
  __shared__ __align__(16) float vs[NB * LD];
  __shared__ __align__(16) float qs[NQ * LD];
  __shared__ float lg[NQ][NB + 1];
  __shared__ float lse_s[NQ];
  __shared__ double inv_lds[HD / 2];
  const int s = blockIdx.x, g = blockIdx.y, layer_local = blockIdx.z;
  const int tid = threadIdx.x;
  const int B = a.B, G = a.Hq / a.Hkv, nq = B * G;
  const int ctx = a.ctx_len[s];
  if (ctx < 0) {
    if (tid == 0) set_status(a.status, CO_ERR_LENGTH);
    return;
  }
  if (tid < HD / 2)   // revolutions per position for bf16, radians for fp32
    inv_lds[tid] = sizeof(T) == 2 ? a.rope_inv[tid] * kInv2Pi : a.rope_inv[tid];
  __syncthreads();
  auto rot = [&](int pos, int p, float& lo, float& hi) {
    float c, sn;
    if constexpr (sizeof(T) == 2)
      rope_cos_sin_rev(pos, inv_lds[p], &c, &sn);
    else
      rope_cos_sin(pos, inv_lds[p], &c, &sn);
    const float l2 = lo * c - hi * sn, h2 = hi * c + lo * sn;
    lo = l2;
    hi = h2;
  };
  auto ld = [](const T* p, int64_t i) -> float {
    if constexpr (sizeof(T) == 2)
      return bf2f(p[i]);
    else
      return p[i];
  };
  // self keys rotated at their positions ctx + j, self values
  const T* Ks = static_cast<const T*>(a.k_self);
  const T* Vs = static_cast<const T*>(a.v_self);
  for (int idx = tid; idx < B * (HD / 2); idx += 256) {
    const int j = idx / (HD / 2), p = idx % (HD / 2);
    const int64_t base =
        (((static_cast<int64_t>(layer_local) * a.S + s) * B + j) * a.Hkv + g) * HD;
    float lo = ld(Ks, base + p), hi = ld(Ks, base + p + HD / 2);
    rot(ctx + j, p, lo, hi);
    ks[j * LD + p] = lo;
    ks[j * LD + p + HD / 2] = hi;
    vs[j * LD + p] = ld(Vs, base + p);
    vs[j * LD + p + HD / 2] = ld(Vs, base + p + HD / 2);
  }
  // queries rotated at ctx + i (unless pre-rotated) and scaled by 1/sqrt(hd)
  auto row_of = [&](int n) {
    return ((static_cast<int64_t>(layer_local) * a.S + s) * B + n / G) * a.Hq + g * G + n % G;
  };
  const T* Q = static_cast<const T*>(a.q);
  const float scale = rsqrtf(static_cast<float>(HD));
  for (int idx = tid; idx < nq * (HD / 2); idx += 256) {
    const int n = idx / (HD / 2), p = idx % (HD / 2);
    const int64_t base = row_of(n) * HD;
    float lo = ld(Q, base + p), hi = ld(Q, base + p + HD / 2);
    if (!(a.flags & CO_Q_PREROTATED)) rot(ctx + n / G, p, lo, hi);
    qs[n * LD + p] = lo * scale;
    qs[n * LD + p + HD / 2] = hi * scale;
  }
  __syncthreads();
  for (int idx = tid; idx < nq * B; idx += 256) {
    const int n = idx / B, j = idx % B;
    const f32x4* qv = reinterpret_cast<const f32x4*>(qs + n * LD);
    const f32x4* kv = reinterpret_cast<const f32x4*>(ks + j * LD);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int d = 0; d < HD / 4; ++d) acc += qv[d] * kv[d];
    lg[n][j] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  __syncthreads();
  // softmax over S: weights in place, LSE_S per query
  for (int n = tid; n < nq; n += 256) {
    float mx = -INFINITY;
    for (int j = 0; j < B; ++j) mx = fmaxf(mx, lg[n][j]);
    float sum = 0.f;
    for (int j = 0; j < B; ++j) {
      const float e = expf(lg[n][j] - mx);
      lg[n][j] = e;
      sum += e;
    }
    const float inv = 1.f / sum;
    for (int j = 0; j < B; ++j) lg[n][j] *= inv;
    lse_s[n] = mx + logf(sum);
  }
  __syncthreads();
  // O_S, then the merge with (O, LSE) over [C;U]
  T* out = static_cast<T*>(a.out);
  for (int idx = tid; idx < nq * HD; idx += 256) {
    const int n = idx / HD, d = idx % HD;
    float os = 0.f;
    for (int j = 0; j < B; ++j) os = fmaf(lg[n][j], vs[j * LD + d], os);
    const int64_t row = row_of(n);
    const float lc = a.lse[row], ls = lse_s[n];
    const float M = fmaxf(lc, ls);
    const float wc = expf(lc - M), ws = expf(ls - M);   // wc = 0 without context keys
    const float oc = ld(out, row * HD + d);
    out[row * HD + d] = to_elem<T>((wc * oc + ws * os) / (wc + ws));
  }
  __syncthreads();   // every thread has read the old LSE of its rows
  for (int n = tid; n < nq; n += 256) {
    const int64_t row = row_of(n);
    const float lc = a.lse[row], ls = lse_s[n];
    const float M = fmaxf(lc, ls);
    a.lse[row] = M + logf(expf(lc - M) + expf(ls - M));
  }
}

}  // namespace

hipError_t launch_self_merge(const SelfArgs& a, int layer_count, int dtype, hipStream_t stream) {
  if (a.S == 0 || layer_count == 0) return hipSuccess;
  const dim3 grid(a.S, a.Hkv, layer_count);
  if (dtype == CO_DTYPE_BF16) {
    if (a.hd == 64) hipLaunchKernelGGL((self_merge_kernel<uint16_t, 64>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((self_merge_kernel<uint16_t, 128>), grid, dim3(256), 0, stream, a);
  } else {
    if (a.hd == 64) hipLaunchKernelGGL((self_merge_kernel<float, 64>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((self_merge_kernel<float, 128>), grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_carry_mass(const MassArgs& a, int layer_count, int dtype, hipStream_t stream) {
  if (a.S == 0 || layer_count == 0) return hipSuccess;
  const dim3 grid(a.S, a.Hkv, layer_count);
  if (dtype == CO_DTYPE_BF16) {
    if (a.hd == 64) hipLaunchKernelGGL((carry_mass_kernel<uint16_t, 64>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((carry_mass_kernel<uint16_t, 128>), grid, dim3(256), 0, stream, a);
  } else {
    if (a.hd == 64) hipLaunchKernelGGL((carry_mass_kernel<float, 64>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((carry_mass_kernel<float, 128>), grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace co
