// Projection of verified window rows into drafter K/V (Eq. 1, Eq. 2;
// Algorithm 1 Carryover steps 1-6; "Cache semantics": keys rotated once at
// the row's absolute position).
//
//   F GEMM:   Z[M][d]   = (H + [carry row] E) . W_F^T        (E added before F)
//   K/V GEMM: J[M][NKV] = Z . W_KV^T, NKV = 2 * L * Hkv * hd (all layers at once)
//   epilogue: rotate the K half of every head at row_pos, round, and scatter
//             each row to its committed page slot or carry row (or drop it).
//
// bf16: LDS-staged, double-buffered MFMA (v_mfma_f32_16x16x32_bf16) GEMM,
// 256 threads = 4 wavefronts per 2-D tile, optional deterministic split-K
// through an fp32 workspace for skinny shapes (few rows, long K).
// fp32: a plain LDS-tiled VALU GEMM feeding the same epilogues.
#include "co_kernels.h"

namespace co {

namespace {

constexpr int kModePartial = 0, kModeZ = 1, kModeKV = 2;

struct GemmArgs {
  int M, N, K, k_per_split;
  const void* A;           // [M][K]
  const void* B;           // [N][K]
  const void* e;           // E added to carry rows of A (null: none)
  const int32_t* row_dst;  // carry rows: -1-r
  float* partial;          // [splits][M][N]
  void* z_out;             // [M][N]
  int mode;
  KvDest kv;
};

__device__ __forceinline__ bool is_carry_row(int32_t dst) { return dst < 0 && dst != kSkip; }

// ------------------------------------------------------------- K/V stores

// Store pairs (i0+p, i0+p+hd/2), p < NP, of head segment `seg` = (layer, K|V, head)
// of window row `row`.  lo/hi hold the unrotated fp32 values of those dims.
template <typename T, int NP>
__device__ void kv_store(const KvDest& e, int row, int seg, int i0, const float* lo,
                         const float* hi) {
  const int32_t dst = e.row_dst[row];
  if (dst == kSkip) return;
  const int hd = e.hd, half = hd / 2;
  const int g = seg % e.Hkv;
  const int kind = (seg / e.Hkv) & 1;
  const int layer = seg / (2 * e.Hkv);
  int64_t kbase, vbase;   // element offsets of dim 0 of this row in the K and V layouts
  T* kptr;
  T* vptr;
  if (dst >= 0) {
    const int page = dst / kPage, t = dst % kPage;
    if (page >= e.num_pages) {
      set_status(e.status, CO_ERR_PAGE_RANGE);
      return;
    }
    const int64_t pg = (static_cast<int64_t>(layer) * e.num_pages + page) * e.Hkv + g;
    kbase = (pg * kPage + t) * hd;
    vbase = pg * hd * kPage + t;
    kptr = static_cast<T*>(e.k_cache);
    vptr = static_cast<T*>(e.v_cache);
  } else {
    const int r = -1 - dst;
    if (r >= e.CP * kPage) {
      set_status(e.status, CO_ERR_LENGTH);
      return;
    }
    const int s = row / e.B;
    const int cp = r / kPage, t = r % kPage;
    const int64_t pg = ((static_cast<int64_t>(layer) * e.S + s) * e.CP + cp) * e.Hkv + g;
    kbase = (pg * kPage + t) * hd;
    vbase = pg * hd * kPage + t;
    kptr = static_cast<T*>(e.k_carry);
    vptr = static_cast<T*>(e.v_carry);
  }
  if (kind == 0) {
    const int pos = e.row_pos[row];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      float c, s;
      rope_cos_sin(pos, rope_inv_freq(i0 + p, hd, e.log2_theta), &c, &s);
      kptr[kbase + i0 + p] = to_elem<T>(lo[p] * c - hi[p] * s);
      kptr[kbase + i0 + p + half] = to_elem<T>(hi[p] * c + lo[p] * s);
    }
  } else {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      vptr[vbase + static_cast<int64_t>(i0 + p) * kPage] = to_elem<T>(lo[p]);
      vptr[vbase + static_cast<int64_t>(i0 + p + half) * kPage] = to_elem<T>(hi[p]);
    }
  }
}

// ------------------------------------------------------------ bf16 MFMA GEMM

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs g) {
  constexpr int BK = 64, LDK = BK + 8;
  constexpr int TM = BM / WM / 16, TN = BN / WN / 16;
  static_assert(WM * WN == 4 && TM >= 1 && TN >= 1, "tile");
  constexpr int kSmemU16 = 2 * (BM + BN) * LDK;
  __shared__ __align__(16) uint16_t smem[kSmemU16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);
  const int nk = (kend - kbeg) / BK;
  const uint16_t* A = static_cast<const uint16_t*>(g.A);
  const uint16_t* Bw = static_cast<const uint16_t*>(g.B);
  const uint16_t* E = static_cast<const uint16_t*>(g.e);

  constexpr int kAChunks = BM * BK / 8, kBChunks = BN * BK / 8;
  constexpr int kAPer = (kAChunks + 255) / 256, kBPer = (kBChunks + 255) / 256;
  u16x8 ra[kAPer], rb[kBPer];

  auto load_global = [&](int kt) {
    const int k0 = kbeg + kt * BK;
#pragma unroll
    for (int i = 0; i < kAPer; ++i) {
      const int c = tid + i * 256;
      u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
      if (c < kAChunks) {
        const int row = c / (BK / 8), kc = c % (BK / 8);
        const int gr = m0 + row;
        if (gr < g.M) {
          v = *reinterpret_cast<const u16x8*>(A + static_cast<int64_t>(gr) * g.K + k0 + kc * 8);
          if (E && is_carry_row(g.row_dst[gr])) {
            const u16x8 ev = *reinterpret_cast<const u16x8*>(E + k0 + kc * 8);
#pragma unroll
            for (int t = 0; t < 8; ++t) v[t] = f2bf(bf2f(v[t]) + bf2f(ev[t]));
          }
        }
      }
      ra[i] = v;
    }
#pragma unroll
    for (int i = 0; i < kBPer; ++i) {
      const int c = tid + i * 256;
      u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
      if (c < kBChunks) {
        const int row = c / (BK / 8), kc = c % (BK / 8);
        const int gn = n0 + row;
        if (gn < g.N)
          v = *reinterpret_cast<const u16x8*>(Bw + static_cast<int64_t>(gn) * g.K + k0 + kc * 8);
      }
      rb[i] = v;
    }
  };
  auto store_lds = [&](int buf) {
    uint16_t* sa = smem + buf * (BM + BN) * LDK;
    uint16_t* sb = sa + BM * LDK;
#pragma unroll
    for (int i = 0; i < kAPer; ++i) {
      const int c = tid + i * 256;
      if (c < kAChunks)
        *reinterpret_cast<u16x8*>(sa + (c / (BK / 8)) * LDK + (c % (BK / 8)) * 8) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < kBPer; ++i) {
      const int c = tid + i * 256;
      if (c < kBChunks)
        *reinterpret_cast<u16x8*>(sb + (c / (BK / 8)) * LDK + (c % (BK / 8)) * 8) = rb[i];
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    load_global(0);
    store_lds(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global(kt + 1);
    const uint16_t* sa = smem + buf * (BM + BN) * LDK;
    const uint16_t* sb = sa + BM * LDK;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      u16x8 af[TM], bfr[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = *reinterpret_cast<const u16x8*>(
            sa + ((wm * TM + a) * 16 + (lane & 15)) * LDK + ks * 32 + (lane >> 4) * 8);
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bfr[b] = *reinterpret_cast<const u16x8*>(
            sb + ((wn * TN + b) * 16 + (lane & 15)) * LDK + ks * 32 + (lane >> 4) * 8);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = mfma16x16x32(af[a], bfr[b], acc[a][b]);
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  if (g.mode == kModePartial) {
    float* out = g.partial + static_cast<int64_t>(blockIdx.z) * g.M * g.N;
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + (wm * TM + a) * 16 + (lane >> 4) * 4 + r;
          const int col = n0 + (wn * TN + b) * 16 + (lane & 15);
          if (row < g.M && col < g.N) out[static_cast<int64_t>(row) * g.N + col] = acc[a][b][r];
        }
    return;
  }

  // Stage the fp32 tile through LDS so the epilogue can work on whole rows.
  constexpr int LDC = BN + 4;
  static_assert(BM * LDC * 4 <= kSmemU16 * 2, "C tile must fit in the staging LDS");
  float* sc = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        sc[((wm * TM + a) * 16 + (lane >> 4) * 4 + r) * LDC + (wn * TN + b) * 16 + (lane & 15)] =
            acc[a][b][r];
  __syncthreads();

  if (g.mode == kModeZ) {
    uint16_t* z = static_cast<uint16_t*>(g.z_out);
    for (int c = tid; c < BM * BN / 8; c += 256) {
      const int row = c / (BN / 8), cc = c % (BN / 8);
      const int gr = m0 + row, gc = n0 + cc * 8;
      if (gr >= g.M || gc >= g.N) continue;
      u16x8 v;
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] = f2bf(sc[row * LDC + cc * 8 + t]);
      *reinterpret_cast<u16x8*>(z + static_cast<int64_t>(gr) * g.N + gc) = v;
    }
  } else {
    const int hd = g.kv.hd, q_per_seg = hd / 8;
    for (int c = tid; c < BM * BN / 8; c += 256) {
      const int row = c / (BN / 8), q = c % (BN / 8);
      const int seg_local = q / q_per_seg, i0 = (q % q_per_seg) * 4;
      const int gr = m0 + row, gc0 = n0 + seg_local * hd;
      if (gr >= g.M || gc0 >= g.N) continue;
      float lo[4], hi[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        lo[p] = sc[row * LDC + seg_local * hd + i0 + p];
        hi[p] = sc[row * LDC + seg_local * hd + hd / 2 + i0 + p];
      }
      kv_store<uint16_t, 4>(g.kv, gr, gc0 / hd, i0, lo, hi);
    }
  }
}

// ------------------------------------------------------------- fp32 GEMM

__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g) {
  constexpr int BM = 32, BN = 64, BK = 32;
  __shared__ float sa[BM][BK + 1];
  __shared__ float sb[BN][BK + 1];
  const int tid = threadIdx.x;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tr = tid / 16, tc = tid % 16;
  const float* A = static_cast<const float*>(g.A);
  const float* Bw = static_cast<const float*>(g.B);
  const float* E = static_cast<const float*>(g.e);
  float acc[2][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += BK) {
    for (int c = tid; c < BM * BK; c += 256) {
      const int r = c / BK, k = c % BK, gr = m0 + r;
      float v = 0.f;
      if (gr < g.M) {
        v = A[static_cast<int64_t>(gr) * g.K + k0 + k];
        if (E && is_carry_row(g.row_dst[gr])) v += E[k0 + k];
      }
      sa[r][k] = v;
    }
    for (int c = tid; c < BN * BK; c += 256) {
      const int r = c / BK, k = c % BK, gn = n0 + r;
      sb[r][k] = gn < g.N ? Bw[static_cast<int64_t>(gn) * g.K + k0 + k] : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int k = 0; k < BK; ++k) {
      const float a0 = sa[tr][k], a1 = sa[tr + 16][k];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float b = sb[tc + 16 * j][k];
        acc[0][j] += a0 * b;
        acc[1][j] += a1 * b;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = m0 + tr + 16 * i, col = n0 + tc + 16 * j;
      if (row < g.M && col < g.N) g.partial[static_cast<int64_t>(row) * g.N + col] = acc[i][j];
    }
}

// -------------------------------------------- epilogues over fp32 partials

template <typename T>
__global__ __launch_bounds__(256) void epi_z_kernel(const float* part, int splits, int M, int N,
                                                    T* z) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(M) * N) return;
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[static_cast<int64_t>(s) * M * N + i];
  z[i] = to_elem<T>(v);
}

template <typename T>
__global__ __launch_bounds__(256) void epi_kv_kernel(const float* part, int splits, int M, int N,
                                                     KvDest e) {
  const int half = e.hd / 2;
  const int64_t items = static_cast<int64_t>(M) * (N / 2);   // one pair per thread
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= items) return;
  const int row = static_cast<int>(i / (N / 2));
  const int rem = static_cast<int>(i % (N / 2));
  const int seg = rem / half, p = rem % half;
  const int64_t c_lo = static_cast<int64_t>(row) * N + seg * e.hd + p;
  float lo = 0.f, hi = 0.f;
  for (int s = 0; s < splits; ++s) {
    lo += part[static_cast<int64_t>(s) * M * N + c_lo];
    hi += part[static_cast<int64_t>(s) * M * N + c_lo + half];
  }
  kv_store<T, 1>(e, row, seg, p, &lo, &hi);
}

// Tile variants: 0 = 16x128 (1x4 waves), 1 = 64x128 (2x2), 2 = 128x128 (2x2).
constexpr int kTileBM[3] = {16, 64, 128};
constexpr int kTileBN = 128;

hipError_t launch_gemm_bf16(const GemmArgs& g, int tile, int splits, hipStream_t stream) {
  const dim3 grid((g.N + kTileBN - 1) / kTileBN, (g.M + kTileBM[tile] - 1) / kTileBM[tile],
                  splits);
  switch (tile) {
    case 0: hipLaunchKernelGGL((gemm_bf16_kernel<16, 128, 1, 4>), grid, dim3(256), 0, stream, g); break;
    case 1: hipLaunchKernelGGL((gemm_bf16_kernel<64, 128, 2, 2>), grid, dim3(256), 0, stream, g); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<128, 128, 2, 2>), grid, dim3(256), 0, stream, g); break;
  }
  return hipGetLastError();
}

int pick_tile(int M) { return M <= 16 ? 0 : (M <= 1024 ? 1 : 2); }

// Split K when the 2-D grid alone leaves most CUs idle and K is long enough.
int pick_split(int M, int N, int K, int tile, int num_cus) {
  const int tiles = ((N + kTileBN - 1) / kTileBN) * ((M + kTileBM[tile] - 1) / kTileBM[tile]);
  int split = 1;
  while (tiles * split * 2 <= 2 * num_cus && (K / (split * 2)) % 64 == 0 && K / (split * 2) >= 512)
    split *= 2;
  return split;
}

}  // namespace

ProjectPlan plan_project(int M, int Dcat, int d, int n_kv, int dtype, int num_cus) {
  ProjectPlan p{};
  const size_t es = dtype == CO_DTYPE_BF16 ? 2 : 4;
  if (dtype == CO_DTYPE_BF16) {
    p.f_tile = pick_tile(M);
    p.f_split = pick_split(M, d, Dcat, p.f_tile, num_cus);
    p.kv_tile = pick_tile(M);
    p.kv_split = pick_split(M, n_kv, d, p.kv_tile, num_cus);
  } else {
    p.f_tile = p.kv_tile = -1;
    p.f_split = p.kv_split = 1;
  }
  auto part = [&](int split, int N) -> size_t {
    return (dtype == CO_DTYPE_F32 || split > 1) ? static_cast<size_t>(split) * M * N * 4 : 0;
  };
  p.z_bytes = (static_cast<size_t>(M) * d * es + 255) / 256 * 256;
  const size_t pf = part(p.f_split, d), pk = part(p.kv_split, n_kv);
  p.part_bytes = ((pf > pk ? pf : pk) + 255) / 256 * 256;
  p.total = p.z_bytes + p.part_bytes;
  return p;
}

hipError_t launch_project(const ProjectArgs& a, const ProjectPlan& p, hipStream_t stream) {
  if (a.M == 0) return hipSuccess;
  const int n_kv = 2 * a.dst.L * a.dst.Hkv * a.dst.hd;
  char* ws = static_cast<char*>(a.ws);
  void* z = ws;
  float* part = reinterpret_cast<float*>(ws + p.z_bytes);
  hipError_t err;

  GemmArgs f{};
  f.M = a.M; f.N = a.d; f.K = a.Dcat;
  f.A = a.hidden; f.B = a.wf; f.e = a.e; f.row_dst = a.dst.row_dst;
  f.partial = part; f.z_out = z; f.kv = a.dst;
  GemmArgs kv{};
  kv.M = a.M; kv.N = n_kv; kv.K = a.d;
  kv.A = z; kv.B = a.wkv; kv.e = nullptr; kv.row_dst = a.dst.row_dst;
  kv.partial = part; kv.z_out = nullptr; kv.kv = a.dst;

  if (a.dtype == CO_DTYPE_F32) {
    f.k_per_split = f.K;
    kv.k_per_split = kv.K;
    f.mode = kv.mode = kModePartial;
    hipLaunchKernelGGL(gemm_f32_kernel, dim3((f.N + 63) / 64, (f.M + 31) / 32), dim3(256), 0,
                       stream, f);
    const int64_t nz = static_cast<int64_t>(a.M) * a.d;
    hipLaunchKernelGGL(epi_z_kernel<float>, dim3(static_cast<unsigned>((nz + 255) / 256)),
                       dim3(256), 0, stream, part, 1, a.M, a.d, static_cast<float*>(z));
    hipLaunchKernelGGL(gemm_f32_kernel, dim3((kv.N + 63) / 64, (kv.M + 31) / 32), dim3(256), 0,
                       stream, kv);
    const int64_t items = static_cast<int64_t>(a.M) * (n_kv / 2);
    hipLaunchKernelGGL(epi_kv_kernel<float>, dim3(static_cast<unsigned>((items + 255) / 256)),
                       dim3(256), 0, stream, part, 1, a.M, n_kv, a.dst);
    return hipGetLastError();
  }

  f.k_per_split = a.Dcat / p.f_split;
  f.mode = p.f_split > 1 ? kModePartial : kModeZ;
  if ((err = launch_gemm_bf16(f, p.f_tile, p.f_split, stream)) != hipSuccess) return err;
  if (p.f_split > 1) {
    const int64_t nz = static_cast<int64_t>(a.M) * a.d;
    hipLaunchKernelGGL(epi_z_kernel<uint16_t>, dim3(static_cast<unsigned>((nz + 255) / 256)),
                       dim3(256), 0, stream, part, p.f_split, a.M, a.d, static_cast<uint16_t*>(z));
  }
  kv.k_per_split = a.d / p.kv_split;
  kv.mode = p.kv_split > 1 ? kModePartial : kModeKV;
  if ((err = launch_gemm_bf16(kv, p.kv_tile, p.kv_split, stream)) != hipSuccess) return err;
  if (p.kv_split > 1) {
    const int64_t items = static_cast<int64_t>(a.M) * (n_kv / 2);
    hipLaunchKernelGGL(epi_kv_kernel<uint16_t>, dim3(static_cast<unsigned>((items + 255) / 256)),
                       dim3(256), 0, stream, part, p.kv_split, a.M, n_kv, a.dst);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------ cache import

template <typename T>
__global__ __launch_bounds__(256) void import_kernel(KvDest e, int seq, int pos0, int n,
                                                     const T* k_rows, const T* v_rows,
                                                     const int32_t* pt, int max_pages) {
  // element (layer, g, row, dim) of the [L][Hkv][n][hd] inputs
  const int64_t total = static_cast<int64_t>(e.L) * e.Hkv * n * e.hd;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= total) return;
  const int dim = static_cast<int>(i % e.hd);
  const int64_t r1 = i / e.hd;
  const int row = static_cast<int>(r1 % n);
  const int64_t lg = r1 / n;
  const int g = static_cast<int>(lg % e.Hkv), layer = static_cast<int>(lg / e.Hkv);
  const int pos = pos0 + row;
  const int page = pt[static_cast<int64_t>(seq) * max_pages + pos / kPage];
  if (page < 0 || page >= e.num_pages) {
    set_status(e.status, CO_ERR_PAGE_RANGE);
    return;
  }
  const int t = pos % kPage;
  const int64_t pg = (static_cast<int64_t>(layer) * e.num_pages + page) * e.Hkv + g;
  static_cast<T*>(e.k_cache)[(pg * kPage + t) * e.hd + dim] = k_rows[i];
  static_cast<T*>(e.v_cache)[(pg * e.hd + dim) * kPage + t] = v_rows[i];
}

hipError_t launch_import(const KvDest& d, int dtype, int seq, int pos0, int n, const void* k_rows,
                         const void* v_rows, const int32_t* page_table, int max_pages,
                         hipStream_t stream) {
  const int64_t total = static_cast<int64_t>(d.L) * d.Hkv * n * d.hd;
  if (total == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == CO_DTYPE_BF16)
    hipLaunchKernelGGL(import_kernel<uint16_t>, grid, dim3(256), 0, stream, d, seq, pos0, n,
                       static_cast<const uint16_t*>(k_rows), static_cast<const uint16_t*>(v_rows),
                       page_table, max_pages);
  else
    hipLaunchKernelGGL(import_kernel<float>, grid, dim3(256), 0, stream, d, seq, pos0, n,
                       static_cast<const float*>(k_rows), static_cast<const float*>(v_rows),
                       page_table, max_pages);
  return hipGetLastError();
}

}  // namespace co
