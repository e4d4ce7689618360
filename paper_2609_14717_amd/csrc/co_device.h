// Device helpers shared by the gfx950 kernels of the carryover drafter step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/carryover.h"

namespace co {

constexpr int kPage = 16;
constexpr int32_t kSkip = INT32_MIN;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

// fp32 -> bf16, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return static_cast<uint16_t>(b >> 16);
}

// Element conversions for the two storage types (fp32, bf16 bits).
template <typename T> __device__ __forceinline__ T to_elem(float v);
template <> __device__ __forceinline__ float to_elem<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t to_elem<uint16_t>(float v) { return f2bf(v); }

// Direct-to-LDS 16-byte load (global_load_lds_dwordx4): every lane supplies a
// global address; the 64 x 16 bytes land contiguously at lds_dst (uniform).  A
// plain function so that kernel templates do not instantiate the builtin in
// their host-side pass (where it would silently drop the kernel).
__device__ __forceinline__ void lds_dma16(const void* src, void* lds_dst) {
  __builtin_amdgcn_global_load_lds(src, lds_dst, 16, 0, 0);
}

// The same load issued as inline asm.  The compiler does not see it as a write
// to LDS, so it neither waits for it before LDS reads nor counts it in its own
// vmcnt waits (which therefore only ever wait longer than they need to); the
// caller orders it with the reads of its LDS slot through explicit vmcnt waits
// and barriers.  lds_dst must be wavefront-uniform.  M0 is reserved to the
// compiler (a clobber would be ignored), so the statement restores it.
__device__ __forceinline__ void lds_dma16_opaque(const void* src, uint32_t lds_dst) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(lds_dst)
      : "memory");
}

// s_waitcnt vmcnt(N) lgkmcnt(0), then a workgroup barrier, as one statement that
// no memory access is moved across.
template <int N>
__device__ __forceinline__ void wait_vm_lgkm_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

// Two fp32 values -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = static_cast<__bf16>(lo), b = static_cast<__bf16>(hi);
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, a)) |
         (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b)) << 16);
}

// The same pair conversion as one v_cvt_pk_bf16_f32 with both sources (the
// compiler otherwise converts one value at a time and merges the halves).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  uint32_t r;
  asm("v_cvt_pk_bf16_f32 %0, %1, %2" : "=v"(r) : "v"(lo), "v"(hi));
  return r;
}

// The value lane q of each group of four lanes holds, in all four (a DPP
// quad permutation: a full-rate move, no LDS round trip).  q is 0..3.
__device__ __forceinline__ float quad_bcast(float v, int q) {
  const int x = __float_as_int(v);
  switch (q) {
    case 0: return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x00, 0xF, 0xF, false));
    case 1: return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x55, 0xF, 0xF, false));
    case 2: return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xAA, 0xF, 0xF, false));
    default: return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xFF, 0xF, 0xF, false));
  }
}

// Max over the four 16-lane rows holding the same column (lanes l, l^16, l^32, l^48),
// with the gfx950 row-swap permutes instead of LDS permutes.
__device__ __forceinline__ float max_across_rows(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u16x8 v) { return __builtin_bit_cast(bf16x8, v); }

typedef float f32x16 __attribute__((ext_vector_type(16)));

// v_mfma_f32_32x32x16_bf16: acc[32x32] += A[32x16] * B[16x32].
// Lane l holds A row (l % 32), k = 8*(l/32) .. +7; B column (l % 32), same k;
// acc register r: column (l % 32), row 8*(r/4) + 4*(l/32) + (r % 4).
__device__ __forceinline__ f32x16 mfma32x32x16(u16x8 a, u16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_bf16: acc[16x16] += A[16x32] * B[32x16].
// Lane l holds A row (l % 16), k = 8*(l/16) .. +7; B column (l % 16), same k;
// acc column (l % 16), rows 4*(l/16) .. +3.
__device__ __forceinline__ f32x4 mfma16x16x32(u16x8 a, u16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// Rotary angle of pair index i at position pos: pos * theta^(-2i/hd).  The product
// and the reduction to [-pi, pi] are done in fp64 so that positions of 10^5 keep
// fp32 accuracy after the reduction; sin/cos are then taken in fp32.
__device__ __forceinline__ void rope_cos_sin(int pos, double inv_freq, float* c, float* s) {
  const double two_pi = 6.283185307179586476925286766559;
  double a = static_cast<double>(pos) * inv_freq;
  double k = rint(a * (1.0 / two_pi));
  float r = static_cast<float>(fma(-k, two_pi, a));
  sincosf(r, s, c);
}

// cos/sin of pos * inv_freq with the angle reduced to revolutions in fp64 and
// the hardware sine/cosine (which take revolutions; absolute error near 1e-6,
// far below bf16 rounding); used where results are stored as bf16.
__device__ __forceinline__ void rope_cos_sin_rev(int pos, double inv_freq_rev, float* c, float* s) {
  double r = static_cast<double>(pos) * inv_freq_rev;
  r -= rint(r);
  const float rf = static_cast<float>(r);
  *c = __builtin_amdgcn_cosf(rf);
  *s = __builtin_amdgcn_sinf(rf);
}

constexpr double kInv2Pi = 0.15915494309189533577;

__device__ __forceinline__ void set_status(int32_t* status, int32_t code) {
  if (status) atomicCAS(status, 0, code);
}

// s_waitcnt vmcnt(n) on gfx9: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14;
// expcnt (6:4) and lgkmcnt (11:8) left at "no wait".
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <int NL, int NSTAGE>
__device__ __forceinline__ void wait_stages_ahead(int ahead) {
  // at most NSTAGE-1 later stages may stay in flight
  if constexpr (NSTAGE >= 4) {
    if (ahead >= 3) { wait_vmcnt<3 * NL>(); return; }
  }
  if constexpr (NSTAGE >= 3) {
    if (ahead >= 2) { wait_vmcnt<2 * NL>(); return; }
  }
  if (ahead >= 1) { wait_vmcnt<NL>(); return; }
  wait_vmcnt<0>();
}

// Workgroup barrier that waits for this wavefront's LDS traffic only, leaving
// its direct-to-LDS global loads in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Groups of 16-byte LDS reads issued as inline asm, each group ending with its
// own lgkmcnt(0) so that the outputs are complete when the statement ends.
// The compiler cannot tell which ring slot an in-flight direct-to-LDS load
// targets and would otherwise wait for all of them (vmcnt(0)) before every LDS
// read; callers guarantee readiness of the slot they read with explicit vmcnt
// waits (and a barrier where other wavefronts filled the slot).
__device__ __forceinline__ uint32_t lds_addr(const unsigned char* p) {
  typedef __attribute__((address_space(3))) const unsigned char* lds_ptr;
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr)p));
}

template <int N>
__device__ __forceinline__ void lds_read_group(u16x8 (&v)[N], const uint32_t (&a)[N]);

template <>
__device__ __forceinline__ void lds_read_group<1>(u16x8 (&v)[1], const uint32_t (&a)[1]) {
  asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]) : "v"(a[0]) : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<2>(u16x8 (&v)[2], const uint32_t (&a)[2]) {
  asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]) : "v"(a[0]), "v"(a[1]) : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<4>(u16x8 (&v)[4], const uint32_t (&a)[4]) {
  asm volatile(
      "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\t"
      "ds_read_b128 %3, %7\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
      : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3])
      : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<3>(u16x8 (&v)[3], const uint32_t (&a)[3]) {
  asm volatile("ds_read_b128 %0, %3\n\tds_read_b128 %1, %4\n\tds_read_b128 %2, %5\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2])
               : "v"(a[0]), "v"(a[1]), "v"(a[2])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<5>(u16x8 (&v)[5], const uint32_t (&a)[5]) {
  asm volatile("ds_read_b128 %0, %5\n\tds_read_b128 %1, %6\n\tds_read_b128 %2, %7\n\tds_read_b128 %3, %8\n\tds_read_b128 %4, %9\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<6>(u16x8 (&v)[6], const uint32_t (&a)[6]) {
  asm volatile("ds_read_b128 %0, %6\n\tds_read_b128 %1, %7\n\tds_read_b128 %2, %8\n\tds_read_b128 %3, %9\n\tds_read_b128 %4, %10\n\tds_read_b128 %5, %11\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<7>(u16x8 (&v)[7], const uint32_t (&a)[7]) {
  asm volatile("ds_read_b128 %0, %7\n\tds_read_b128 %1, %8\n\tds_read_b128 %2, %9\n\tds_read_b128 %3, %10\n\tds_read_b128 %4, %11\n\tds_read_b128 %5, %12\n\tds_read_b128 %6, %13\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<8>(u16x8 (&v)[8], const uint32_t (&a)[8]) {
  asm volatile("ds_read_b128 %0, %8\n\tds_read_b128 %1, %9\n\tds_read_b128 %2, %10\n\tds_read_b128 %3, %11\n\tds_read_b128 %4, %12\n\tds_read_b128 %5, %13\n\tds_read_b128 %6, %14\n\tds_read_b128 %7, %15\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<9>(u16x8 (&v)[9], const uint32_t (&a)[9]) {
  asm volatile("ds_read_b128 %0, %9\n\tds_read_b128 %1, %10\n\tds_read_b128 %2, %11\n\tds_read_b128 %3, %12\n\tds_read_b128 %4, %13\n\tds_read_b128 %5, %14\n\tds_read_b128 %6, %15\n\tds_read_b128 %7, %16\n\tds_read_b128 %8, %17\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7]), "=&v"(v[8])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7]), "v"(a[8])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<10>(u16x8 (&v)[10], const uint32_t (&a)[10]) {
  asm volatile("ds_read_b128 %0, %10\n\tds_read_b128 %1, %11\n\tds_read_b128 %2, %12\n\tds_read_b128 %3, %13\n\tds_read_b128 %4, %14\n\tds_read_b128 %5, %15\n\tds_read_b128 %6, %16\n\tds_read_b128 %7, %17\n\tds_read_b128 %8, %18\n\tds_read_b128 %9, %19\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7]), "=&v"(v[8]), "=&v"(v[9])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7]), "v"(a[8]), "v"(a[9])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<11>(u16x8 (&v)[11], const uint32_t (&a)[11]) {
  asm volatile("ds_read_b128 %0, %11\n\tds_read_b128 %1, %12\n\tds_read_b128 %2, %13\n\tds_read_b128 %3, %14\n\tds_read_b128 %4, %15\n\tds_read_b128 %5, %16\n\tds_read_b128 %6, %17\n\tds_read_b128 %7, %18\n\tds_read_b128 %8, %19\n\tds_read_b128 %9, %20\n\tds_read_b128 %10, %21\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7]), "=&v"(v[8]), "=&v"(v[9]), "=&v"(v[10])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7]), "v"(a[8]), "v"(a[9]), "v"(a[10])
               : "memory");
}

template <>
__device__ __forceinline__ void lds_read_group<12>(u16x8 (&v)[12], const uint32_t (&a)[12]) {
  asm volatile("ds_read_b128 %0, %12\n\tds_read_b128 %1, %13\n\tds_read_b128 %2, %14\n\tds_read_b128 %3, %15\n\tds_read_b128 %4, %16\n\tds_read_b128 %5, %17\n\tds_read_b128 %6, %18\n\tds_read_b128 %7, %19\n\tds_read_b128 %8, %20\n\tds_read_b128 %9, %21\n\tds_read_b128 %10, %22\n\tds_read_b128 %11, %23\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7]), "=&v"(v[8]), "=&v"(v[9]), "=&v"(v[10]), "=&v"(v[11])
               : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7]), "v"(a[8]), "v"(a[9]), "v"(a[10]), "v"(a[11])
               : "memory");
}

}  // namespace co
