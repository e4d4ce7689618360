// Stochastic verification (T = 1): the acceptance decision and the correction
// or bonus draw of the standard speculative-sampling rule that Appendix A
// ("Why verification remains valid") relies on.  A proposal x ~ q at window
// position j is accepted with probability min(1, p_j(x) / q_j(x)); the first
// rejection at position m emits a token drawn from the normalised residual
// max(0, p_m - q_m); B acceptances emit a bonus drawn from p_B.
//
// Random draws arrive as 32-bit words, so the decisions are integer-exact:
//   * accept iff u * q(x) < p(x), u = (word >> 8) * 2^-24; the 24-bit by
//     24-bit product is exact in fp64, so this is the exact comparison;
//   * the draw uses fixed-point weights w(y) = floor(2^32 * d(y)) of the fp64
//     differences d(y) = p(y) - q(y) where positive (p(y) for a bonus, and for
//     a correction whose weights are all zero): y is the smallest token whose
//     running integer sum exceeds floor(word * W / 2^32), W the total weight.
//
// One workgroup per sequence.  The first wavefront takes the acceptance
// decisions with one ballot per 64 positions; then the workgroup streams the
// selected row of p (and q) twice: once for the total weight, once for the
// running sums, 1024 tokens per step with an exclusive scan across threads.
#include "co_kernels.h"

namespace co {

namespace {

constexpr int kVerifyThreads = 256;

__device__ __forceinline__ uint64_t fixed_weight(const float* p, const float* q, int64_t y) {
  double d = static_cast<double>(p[y]);
  if (q) d -= static_cast<double>(q[y]);
  return d > 0.0 ? static_cast<uint64_t>(d * 4294967296.0) : 0ull;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int off) {
  const uint32_t lo = __shfl_up(static_cast<uint32_t>(v), off);
  const uint32_t hi = __shfl_up(static_cast<uint32_t>(v >> 32), off);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Sum of the weights of a row over the workgroup (every thread gets it).
__device__ uint64_t row_total(const float* p, const float* q, int V, uint64_t* red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t s = 0;
  for (int64_t y = tid; y < V; y += kVerifyThreads) s += fixed_weight(p, q, y);
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += shfl_xor_u64(s, m);
  __syncthreads();   // red[] may still be read from a previous use
  if (lane == 0) red[wave] = s;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Smallest y with w(0) + ... + w(y) > t (t < the row's total weight).
__device__ int row_find(const float* p, const float* q, int V, uint64_t t, uint64_t* red,
                        int* found) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) *found = -1;
  uint64_t base = 0;
  for (int64_t c0 = 0; c0 < V; c0 += 4 * kVerifyThreads) {
    const int64_t y0 = c0 + 4 * tid;
    uint64_t w[4], own = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      w[k] = y0 + k < V ? fixed_weight(p, q, y0 + k) : 0ull;
      own += w[k];
    }
    uint64_t inc = own;   // inclusive scan within the wavefront
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint64_t o = shfl_up_u64(inc, off);
      if (lane >= off) inc += o;
    }
    __syncthreads();
    if (lane == 63) red[wave] = inc;
    __syncthreads();
    uint64_t before = base, total = 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (v < wave) before += red[v];
      total += red[v];
    }
    before += inc - own;   // exclusive prefix of this thread's first token
    if (before <= t && t < before + own) {
      uint64_t c = before;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        c += w[k];
        if (c > t) {
          *found = static_cast<int>(y0 + k);
          break;
        }
      }
    }
    base += total;
    if (base > t) break;   // uniform: every thread holds the same base
  }
  __syncthreads();
  return *found;
}

__global__ __launch_bounds__(kVerifyThreads) void verify_kernel(VerifyArgs a) {
  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int B = a.B, V = a.V;
  __shared__ uint64_t red[4];
  __shared__ int sh_m, sh_found;
  const int64_t prow0 = static_cast<int64_t>(s) * (B + 1);
  const int64_t qrow0 = static_cast<int64_t>(s) * B;
  if (tid < 64) {
    int m = B;
    bool bad = false;
    for (int j0 = 0; j0 < B; j0 += 64) {
      const int j = j0 + lane;
      bool rej = false;
      if (j < B) {
        const int x = a.draft[qrow0 + j];
        if (x < 0 || x >= V) {
          bad = true;
        } else {
          const double u = static_cast<double>(a.words[prow0 + j] >> 8) * 0x1p-24;
          const double pj = a.p[(prow0 + j) * V + x];
          const double qj = a.q[(qrow0 + j) * V + x];
          rej = !(u * qj < pj);
        }
      }
      const unsigned long long mask = __ballot(rej);
      if (mask && m == B) m = j0 + __ffsll(static_cast<long long>(mask)) - 1;
    }
    bad = __any(bad);
    if (lane == 0) sh_m = bad ? -1 : m;
  }
  __syncthreads();
  const int m = sh_m;
  int32_t* bits = a.accept_bits + qrow0;
  for (int j = tid; j < B; j += kVerifyThreads) bits[j] = j < m ? 1 : 0;
  if (m < 0) {
    if (tid == 0) {
      a.accept_len[s] = 0;
      a.next_tok[s] = -1;
      set_status(a.status, CO_ERR_TOKEN);
    }
    return;
  }
  const float* p = a.p + (prow0 + m) * V;
  const float* q = m < B ? a.q + (qrow0 + m) * V : nullptr;
  uint64_t W = row_total(p, q, V, red);
  if (W == 0 && q) {
    q = nullptr;
    W = row_total(p, q, V, red);
  }
  int next = -1;
  if (W) {
    const uint64_t u = a.words[prow0 + B];
    const uint64_t t = u * (W >> 32) + ((u * (W & 0xFFFFFFFFull)) >> 32);   // floor(u W / 2^32)
    next = row_find(p, q, V, t, red, &sh_found);
  }
  if (tid == 0) {
    a.accept_len[s] = m;
    a.next_tok[s] = next;
  }
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, hipStream_t stream) {
  if (a.S == 0) return hipSuccess;
  hipLaunchKernelGGL(verify_kernel, dim3(a.S), dim3(kVerifyThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace co
