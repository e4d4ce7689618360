// Share of each block query's attention that falls on the carried rows (the
// diagnostic of Appendix "Attention to carried states"): with LSE the
// natural-log log-sum-exp over ctx = [C;U] that the attention call wrote, and
// LSE_U the same over the carry keys U alone, mass = exp(LSE_U - LSE).  The
// carry segment holds at most `block` rows, so one workgroup per (sequence,
// KV head, layer) stages them in LDS and each thread takes query rows.
#include "co_kernels.h"

namespace co {

namespace {

template <typename T, int HD>
__global__ __launch_bounds__(256) void carry_mass_kernel(MassArgs a) {
  __shared__ float ks[kMaxCarryRows][HD + 1];
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
  const T* kk = static_cast<const T*>(a.k_carry);
  for (int idx = tid; idx < carry * HD; idx += 256) {
    const int t = idx / HD, d = idx % HD;
    const int64_t off =
        ((((static_cast<int64_t>(layer) * a.S + s) * a.CP + t / kPage) * a.Hkv + g) * kPage +
         t % kPage) * HD + d;
    if constexpr (sizeof(T) == 2)
      ks[t][d] = bf2f(kk[off]);
    else
      ks[t][d] = kk[off];
  }
  if (tid < HD / 2)   // revolutions per position for bf16, radians for fp32
    inv_lds[tid] = sizeof(T) == 2 ? a.rope_inv[tid] * kInv2Pi : a.rope_inv[tid];
  __syncthreads();

  const T* Q = static_cast<const T*>(a.q);
  const float scale = rsqrtf(static_cast<float>(HD));
  for (int n = tid; n < nq; n += 256) {
    const int i = n / G, h = g * G + n % G;
    const int64_t row = ((static_cast<int64_t>(layer_local) * a.S + s) * a.B + i) * a.Hq + h;
    float q[HD];
#pragma unroll
    for (int d = 0; d < HD; ++d) {
      if constexpr (sizeof(T) == 2)
        q[d] = bf2f(Q[row * HD + d]);
      else
        q[d] = Q[row * HD + d];
    }
    if (!(a.flags & CO_Q_PREROTATED)) {
#pragma unroll
      for (int p = 0; p < HD / 2; ++p) {
        float c, sn;
        if constexpr (sizeof(T) == 2)
          rope_cos_sin_rev(ctx + i, inv_lds[p], &c, &sn);
        else
          rope_cos_sin(ctx + i, inv_lds[p], &c, &sn);
        const float lo = q[p], hi = q[p + HD / 2];
        q[p] = lo * c - hi * sn;
        q[p + HD / 2] = hi * c + lo * sn;
      }
    }
    // log-sum-exp of the scaled logits over the carry keys
    float mx = -INFINITY, sum = 0.f;
    for (int t = 0; t < carry; ++t) {
      float dot = 0.f;
#pragma unroll
      for (int d = 0; d < HD; ++d) dot = fmaf(q[d], ks[t][d], dot);
      const float lg = dot * scale;
      if (lg > mx) {
        sum = sum * expf(mx - lg) + 1.f;
        mx = lg;
      } else {
        sum += expf(lg - mx);
      }
    }
    const float lse = a.lse[row];
    a.mass[row] = (carry == 0 || lse == -INFINITY) ? 0.f : expf(mx + logf(sum) - lse);
  }
}

}  // namespace

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
