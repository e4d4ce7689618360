// Route: split each verified window by its accepted prefix (Eq. 1;
// Algorithm 1 "Given" and steps 5-6; greedy verification, Section 2
// "Preliminaries").  One wavefront per sequence.
#include "co_kernels.h"

namespace co {

__global__ __launch_bounds__(64) void route_kernel(RouteArgs a) {
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  const int B = a.B;
  const int p0 = a.ctx_len[s];

  // m = first index where draft and target disagree (B if none), or, with
  // accept decisions, the first rejected position
  int m = B;
  if (!(a.flags & CO_ROUTE_ACCEPT_ALL)) {
    const bool bits = a.flags & CO_ROUTE_ACCEPT_BITS;
    const int32_t* dr = a.draft + static_cast<int64_t>(s) * B;
    const int32_t* tg = bits ? nullptr : a.target + static_cast<int64_t>(s) * B;
    for (int j0 = 0; j0 < B; j0 += 64) {
      const int j = j0 + lane;
      const bool diff = j < B && (bits ? dr[j] == 0 : dr[j] != tg[j]);
      const unsigned long long mask = __ballot(diff);
      if (mask) {
        m = j0 + __ffsll(static_cast<long long>(mask)) - 1;
        break;
      }
    }
  }

  const bool carry_only = a.flags & CO_ROUTE_CARRY_ONLY;
  const bool baseline = a.flags & CO_BASELINE_MODE;
  const int64_t cap = static_cast<int64_t>(a.max_pages) * kPage;
  const int32_t* pt = a.page_table + static_cast<int64_t>(s) * a.max_pages;

  int err = 0;
  if (p0 < 0) {
    err = CO_ERR_LENGTH;
  } else if (static_cast<int64_t>(p0) + B > cap) {
    err = CO_ERR_CAPACITY;
  } else if (!carry_only) {
    bool bad = false;
    for (int j = lane; j < m; j += 64) {
      const int page = pt[(p0 + j) / kPage];
      bad |= page < 0 || page >= a.num_pages;
    }
    if (__any(bad)) err = CO_ERR_PAGE_RANGE;
  }

  int32_t* pos_out = a.row_pos + static_cast<int64_t>(s) * B;
  int32_t* dst_out = a.row_dst + static_cast<int64_t>(s) * B;
  if (err) {
    for (int j = lane; j < B; j += 64) {
      pos_out[j] = p0 >= 0 ? p0 + j : 0;
      dst_out[j] = kSkip;
    }
    if (lane == 0) {
      a.accept_len[s] = 0;
      set_status(a.status, err);
    }
    return;
  }

  for (int j = lane; j < B; j += 64) {
    const int pos = p0 + j;
    int32_t dst = kSkip;
    if (j < m) {
      if (!carry_only) dst = pt[pos / kPage] * kPage + pos % kPage;
    } else if (!baseline) {
      dst = -1 - (j - m);
    }
    pos_out[j] = pos;
    dst_out[j] = dst;
  }
  if (lane == 0) {
    a.accept_len[s] = m;
    a.ctx_len[s] = p0 + m;
    a.carry_len[s] = baseline ? 0 : B - m;
  }
}

hipError_t launch_route(const RouteArgs& a, hipStream_t stream) {
  if (a.S == 0) return hipSuccess;
  hipLaunchKernelGGL(route_kernel, dim3(a.S), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace co
