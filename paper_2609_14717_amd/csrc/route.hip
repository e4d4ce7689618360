// Route: split each verified window by its accepted prefix (Eq. 1;
// Algorithm 1 "Given" and steps 5-6; greedy verification, Section 2
// "Preliminaries").  One wavefront per sequence.
#include "co_route.h"

namespace co {

__global__ __launch_bounds__(64) void route_kernel(RouteArgs a) {
  route_sequence(a, blockIdx.x, threadIdx.x);
}

hipError_t launch_route(const RouteArgs& a, hipStream_t stream) {
  if (a.S == 0) return hipSuccess;
  hipLaunchKernelGGL(route_kernel, dim3(a.S), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace co
