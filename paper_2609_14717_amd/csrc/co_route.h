// One sequence's route step (Eq. 1; Algorithm 1 "Given" and steps 5-6;
// greedy verification, Section 2 "Preliminaries"), for one wavefront: the
// accepted prefix, the row descriptors and the new lengths.  Shared by the
// route kernel and by the F product's launch, which can carry it as extra
// workgroups (the F product itself does not read the descriptors then).
#pragma once

#include "co_kernels.h"
#include "co_store.h"

namespace co {

// m = first index where draft and target disagree (B if none), or, with
// accept decisions, the first rejected position; every lane returns m
__device__ __forceinline__ int route_accepted(const RouteArgs& a, int s, int lane) {
  const int B = a.B;
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
  return m;
}

// Whether row r (sequence r / B, window position r % B) becomes a carry row:
// a position at or after the first rejected one, outside baseline mode.  The
// same rule as route_sequence, read by one thread without the row descriptors
// (a sequence whose route step fails gets no rows at all, so its rows' F(E)
// term is never stored either way).
__device__ __forceinline__ bool route_row_carried(const RouteArgs& a, int r) {
  if (a.flags & (CO_ROUTE_ACCEPT_ALL | CO_BASELINE_MODE)) return false;
  const int s = r / a.B, j = r % a.B;
  const bool bits = a.flags & CO_ROUTE_ACCEPT_BITS;
  const int32_t* dr = a.draft + static_cast<int64_t>(s) * a.B;
  const int32_t* tg = bits ? nullptr : a.target + static_cast<int64_t>(s) * a.B;
  bool rejected = false;
  for (int i = 0; i <= j; ++i) rejected = rejected || (bits ? dr[i] == 0 : dr[i] != tg[i]);
  return rejected;
}

__device__ __forceinline__ void route_sequence(const RouteArgs& a, int s, int lane) {
  const int B = a.B;
  const int p0 = a.ctx_len[s];
  const int m = route_accepted(a, s, lane);

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

}  // namespace co
