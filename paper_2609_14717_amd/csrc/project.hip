// Projection of verified window rows into drafter K/V (Eq. 1, Eq. 2;
// Algorithm 1 Carryover steps 1-6; "Cache semantics": keys rotated once at
// the row's absolute position).
//
//   F GEMM:   Z[M][d]   = H . W_F^T + [carry row] (E . W_F^T)  (F(H + E) by linearity)
//   K/V GEMM: J[M][NKV] = Z . W_KV^T, NKV = 2 * L * Hkv * hd (all layers at once)
//   epilogue: rotate the K half of every head at row_pos, round, and scatter
//             each row to its committed page slot or carry row (or drop it).
//
// bf16: MFMA (v_mfma_f32_16x16x32_bf16) GEMM, 256 threads = 4 wavefronts per
// 2-D tile.  Operands stream global -> LDS with direct-to-LDS 16-byte loads
// (global_load_lds_dwordx4) into an NSTAGE-deep ring of 128-wide K stages, so
// several stages are in flight without holding registers; each wavefront
// issues the same number of loads per stage and waits with an exact vmcnt.
// Rows are stored with their 16-byte chunks XOR-swizzled by (row mod 16) so
// that the 16 lanes reading one MFMA fragment hit distinct LDS banks.
// E_carry is staged with the operands; one extra MFMA tile whose rows all
// hold E accumulates F(E), added to carried rows in the epilogue.  Skinny
// shapes (few rows, long K) split K across workgroups deterministically
// through an fp32 workspace.
// fp32: a plain LDS-tiled VALU GEMM feeding the same epilogues.
#include "co_store.h"

namespace co {

namespace {

constexpr int kModePartial = 0, kModeZ = 1, kModeKV = 2;

struct GemmArgs {
  int M, N, K, k_per_split;
  const void* A;           // [M][K]
  const void* B;           // [N][K]
  const void* e;           // E: F(E) is added to carry rows (null: none)
  const int32_t* row_dst;  // carry rows: -1-r
  float* partial;          // [splits][M][N]
  float* partial_e;        // [splits][N]: F(E) per K-split (split-K with E only)
  void* z_out;             // [M][N]
  int mode;
  KvDest kv;
};

// Workgroup barrier for the staged ring.  Each wavefront has already waited
// (vmcnt) for its own direct-to-LDS loads of the stage it is about to read, and
// LDS reads are complete once their values feed the MFMAs, so no memory fence
// is needed -- a fence here would make every wavefront wait for all the later
// stages still in flight.  The empty asm keeps the compiler from moving LDS
// accesses across the barrier.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ------------------------------------------------------------ bf16 MFMA GEMM

template <int BM, int BN, int WM, int WN, int NSTAGE, bool HAS_E>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs g) {
  constexpr int BK = 128;                 // K elements per stage
  constexpr int ROWB = BK * 2;            // bytes per staged row
  constexpr int TM = BM / WM / 16, TN = BN / WN / 16;
  constexpr int ROWS = BM + BN;           // A rows, then B rows
  constexpr int LPW = ROWS / 16;          // 1 KiB loads (4 rows) per wave per stage
  constexpr int NL = LPW + (HAS_E ? 1 : 0);
  constexpr int E_OFF = ROWS * ROWB;
  constexpr int STAGE_BYTES = ROWS * ROWB + (HAS_E ? 4 * 1024 : 0);
  static_assert(WM * WN == 4 && TM >= 1 && TN >= 1 && ROWS % 16 == 0, "tile");
  static_assert(NL * (NSTAGE - 1) < 64, "vmcnt");
  constexpr int LDC = BN + 4;
  static_assert(BM * LDC * 4 <= NSTAGE * STAGE_BYTES, "C tile must fit in the ring");
  __shared__ __align__(16) unsigned char smem[NSTAGE * STAGE_BYTES];
  __shared__ double inv_tab[64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * g.k_per_split;
  const int klen = min(g.K - kbeg, g.k_per_split);
  const int nk = (klen + BK - 1) / BK;
  const int last_ks = (klen - (nk - 1) * BK) / 32;      // k-steps in the last stage
  const uint16_t* A = static_cast<const uint16_t*>(g.A);
  const uint16_t* Bw = static_cast<const uint16_t*>(g.B);
  const uint16_t* E = static_cast<const uint16_t*>(g.e);

  // row descriptors of the tile's rows (thread t: row t % BM), consumed only by
  // the epilogue; kept opaque until then so no wait lands before the main loop
  const bool need_rows = HAS_E || g.mode == kModeKV;
  int rd_dst = 0, rd_pos = 0;
  if (need_rows) {
    const int r = min(m0 + (tid % BM), g.M - 1);
    rd_dst = g.row_dst[r];
    if (g.mode == kModeKV) rd_pos = g.kv.row_pos[r];
  }

  auto issue = [&](int kt, int slot) {
    unsigned char* st = smem + slot * STAGE_BYTES;
    const int k0 = kbeg + kt * BK;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int i = wave * LPW + j;                    // 1 KiB block index (uniform)
      const int row = i * 4 + (lane >> 4);
      const int chunk = (lane & 15) ^ (row & 15);      // logical chunk landing at lane & 15
      const int kk = min(k0 + chunk * 8, g.K - 8);     // a short last stage reads in bounds
      const uint16_t* src;
      if (row < BM) {
        src = A + static_cast<int64_t>(min(m0 + row, g.M - 1)) * g.K + kk;
      } else {
        src = Bw + static_cast<int64_t>(min(n0 + row - BM, g.N - 1)) * g.K + kk;
      }
      lds_dma16(src, st + i * 1024);
    }
    if constexpr (HAS_E) {
      const int kk = min(k0 + (lane & 15) * 8, g.K - 8);
      lds_dma16(E + kk, st + E_OFF + wave * 1024);
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  // F(E) for this wavefront's columns: an extra M-tile whose rows all hold E
  // (F is linear, so F(h + E) = F(h) + F(E); added to carried rows at the end)
  f32x4 acc_e[HAS_E ? TN : 1];
#pragma unroll
  for (int b = 0; b < (HAS_E ? TN : 1); ++b) acc_e[b] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int st = 0; st < NSTAGE - 1; ++st)
    if (st < nk) issue(st, st);

  for (int kt = 0; kt < nk; ++kt) {
    if (kt + NSTAGE - 1 < nk) issue(kt + NSTAGE - 1, (kt + NSTAGE - 1) % NSTAGE);
    wait_stages_ahead<NL, NSTAGE>(min(NSTAGE - 1, nk - 1 - kt));
    stage_barrier();
    const unsigned char* st = smem + (kt % NSTAGE) * STAGE_BYTES;
    const int ksteps = kt == nk - 1 ? last_ks : BK / 32;
    // KG k-steps' fragments are read as one group of LDS reads with one wait
    constexpr int NR = TM + TN + (HAS_E ? 1 : 0);
    constexpr int KG = 4 * NR <= 12 ? 4 : (2 * NR <= 12 ? 2 : 1);
    auto kgroup = [&](int ks0) {
      u16x8 fr[KG * NR];
      uint32_t ad[KG * NR];
#pragma unroll
      for (int kk = 0; kk < KG; ++kk) {
        const int c = (ks0 + kk) * 4 + (lane >> 4);
#pragma unroll
        for (int a = 0; a < TM; ++a) {
          const int row = (wm * TM + a) * 16 + (lane & 15);
          ad[kk * NR + a] = lds_addr(st + row * ROWB + ((c ^ (row & 15)) << 4));
        }
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          const int row = BM + (wn * TN + b) * 16 + (lane & 15);
          ad[kk * NR + TM + b] = lds_addr(st + row * ROWB + ((c ^ (row & 15)) << 4));
        }
        if constexpr (HAS_E) ad[kk * NR + TM + TN] = lds_addr(st + E_OFF + (c << 4));
      }
      lds_read_group<KG * NR>(fr, ad);
#pragma unroll
      for (int kk = 0; kk < KG; ++kk) {
        const u16x8* f = fr + kk * NR;
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int b = 0; b < TN; ++b) acc[a][b] = mfma16x16x32(f[a], f[TM + b], acc[a][b]);
        if constexpr (HAS_E) {
#pragma unroll
          for (int b = 0; b < TN; ++b) acc_e[b] = mfma16x16x32(f[TM + TN], f[TM + b], acc_e[b]);
        }
      }
    };
    if (ksteps == BK / 32) {
#pragma unroll
      for (int ks = 0; ks < BK / 32; ks += KG) kgroup(ks);
    } else {
      // a short last stage: whole groups, then single k-steps
      for (int ks = 0; ks < ksteps; ks += KG) {
        if (ks + KG <= ksteps) {
          kgroup(ks);
        } else {
          for (int k1 = ks; k1 < ksteps; ++k1) {
            constexpr int NR1 = NR;
            u16x8 fr[NR1];
            uint32_t ad[NR1];
            const int c = k1 * 4 + (lane >> 4);
#pragma unroll
            for (int a = 0; a < TM; ++a) {
              const int row = (wm * TM + a) * 16 + (lane & 15);
              ad[a] = lds_addr(st + row * ROWB + ((c ^ (row & 15)) << 4));
            }
#pragma unroll
            for (int b = 0; b < TN; ++b) {
              const int row = BM + (wn * TN + b) * 16 + (lane & 15);
              ad[TM + b] = lds_addr(st + row * ROWB + ((c ^ (row & 15)) << 4));
            }
            if constexpr (HAS_E) ad[TM + TN] = lds_addr(st + E_OFF + (c << 4));
            lds_read_group<NR1>(fr, ad);
#pragma unroll
            for (int a = 0; a < TM; ++a)
#pragma unroll
              for (int b = 0; b < TN; ++b) acc[a][b] = mfma16x16x32(fr[a], fr[TM + b], acc[a][b]);
            if constexpr (HAS_E) {
#pragma unroll
              for (int b = 0; b < TN; ++b) acc_e[b] = mfma16x16x32(fr[TM + TN], fr[TM + b], acc_e[b]);
            }
          }
        }
      }
    }
    stage_barrier();
  }
  __syncthreads();

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
    if constexpr (HAS_E) {
      if (blockIdx.y == 0 && wm == 0 && lane < 16) {
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          const int col = n0 + (wn * TN + b) * 16 + lane;
          if (col < g.N) g.partial_e[static_cast<int64_t>(blockIdx.z) * g.N + col] = acc_e[b][0];
        }
      }
    }
    return;
  }

  // Stage the fp32 tile through LDS so the epilogue can work on whole rows.
  float* sc = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        sc[((wm * TM + a) * 16 + (lane >> 4) * 4 + r) * LDC + (wn * TN + b) * 16 + (lane & 15)] =
            acc[a][b][r];
  if (g.mode == kModeKV && tid < g.kv.hd / 2) inv_tab[tid] = g.kv.rope_inv[tid];
  __shared__ float fe_lds[HAS_E ? BN : 1];
  __shared__ int dst_lds[BM], pos_lds[BM];
  asm volatile("" : "+v"(rd_dst), "+v"(rd_pos));
  if (need_rows && tid < BM) {
    dst_lds[tid] = rd_dst;
    pos_lds[tid] = rd_pos;
  }
  if constexpr (HAS_E) {
    if (wm == 0 && lane < 16) {
#pragma unroll
      for (int b = 0; b < TN; ++b) fe_lds[(wn * TN + b) * 16 + lane] = acc_e[b][0];
    }
  }
  __syncthreads();

  if (g.mode == kModeZ) {
    uint16_t* z = static_cast<uint16_t*>(g.z_out);
    for (int c = tid; c < BM * BN / 8; c += 256) {
      const int row = c / (BN / 8), cc = c % (BN / 8);
      const int gr = m0 + row, gc = n0 + cc * 8;
      if (gr >= g.M || gc >= g.N) continue;
      u16x8 v;
      if constexpr (HAS_E) {
        const bool cy = is_carry_row(dst_lds[row]);
#pragma unroll
        for (int t = 0; t < 8; ++t)
          v[t] = f2bf(sc[row * LDC + cc * 8 + t] + (cy ? fe_lds[cc * 8 + t] : 0.f));
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t) v[t] = f2bf(sc[row * LDC + cc * 8 + t]);
      }
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
      kv_store<uint16_t, 4>(g.kv, gr, dst_lds[row], pos_lds[row], gc0 / hd, i0, lo, hi, inv_tab);
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
                                                    T* z, const float* part_e,
                                                    const int32_t* row_dst) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(M) * N) return;
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[static_cast<int64_t>(s) * M * N + i];
  if (part_e && is_carry_row(row_dst[i / N])) {
    const int col = static_cast<int>(i % N);
    for (int s = 0; s < splits; ++s) v += part_e[static_cast<int64_t>(s) * N + col];
  }
  z[i] = to_elem<T>(v);
}

template <typename T>
__global__ __launch_bounds__(256) void epi_kv_kernel(const float* part, int splits, int M, int N,
                                                     KvDest e) {
  __shared__ double inv_tab[64];
  const int half = e.hd / 2;
  if (threadIdx.x < half) inv_tab[threadIdx.x] = e.rope_inv[threadIdx.x];
  __syncthreads();
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
  kv_store<T, 1>(e, row, e.row_dst[row], e.row_pos[row], seg, p, &lo, &hi, inv_tab);
}

// Tile variants (BM x BN, waves WM x WN, ring depth):
//   0: 16 x 64, 1x4, 4 stages   skinny or few-row shapes, N tiles of 64
//   1: 16 x 128, 1x4, 3 stages  skinny shapes whose K/V heads are 128 wide
//   2: 64 x 128, 2x2, 2 stages  medium row counts
//   3: 128 x 128, 2x2, 2 stages many rows (prefill, training-shaped forward)
constexpr int kTileBM[4] = {16, 16, 64, 128};
constexpr int kTileBN[4] = {64, 128, 128, 128};

template <bool HAS_E>
hipError_t launch_gemm_bf16_t(const GemmArgs& g, int tile, int splits, hipStream_t stream) {
  const dim3 grid((g.N + kTileBN[tile] - 1) / kTileBN[tile],
                  (g.M + kTileBM[tile] - 1) / kTileBM[tile], splits);
  switch (tile) {
    case 0: hipLaunchKernelGGL((gemm_bf16_kernel<16, 64, 1, 4, 4, HAS_E>), grid, dim3(256), 0, stream, g); break;
    case 1: hipLaunchKernelGGL((gemm_bf16_kernel<16, 128, 1, 4, 3, HAS_E>), grid, dim3(256), 0, stream, g); break;
    case 2: hipLaunchKernelGGL((gemm_bf16_kernel<64, 128, 2, 2, 2, HAS_E>), grid, dim3(256), 0, stream, g); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<128, 128, 2, 2, 2, HAS_E>), grid, dim3(256), 0, stream, g); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& g, int tile, int splits, hipStream_t stream) {
  return g.e ? launch_gemm_bf16_t<true>(g, tile, splits, stream)
             : launch_gemm_bf16_t<false>(g, tile, splits, stream);
}

int tiles_of(int M, int N, int tile) {
  return ((N + kTileBN[tile] - 1) / kTileBN[tile]) * ((M + kTileBM[tile] - 1) / kTileBM[tile]);
}

// Split K when the 2-D grid alone leaves most CUs idle and K is long enough.
int pick_split(int M, int N, int K, int tile, int num_cus) {
  const int tiles = tiles_of(M, N, tile);
  int split = 1;
  while (tiles * split * 2 <= 2 * num_cus && (K / (split * 2)) % 128 == 0 &&
         K / (split * 2) >= 512)
    split *= 2;
  return split;
}

// Largest tile (fewest re-reads of the weights) whose grid, after splitting K,
// still gives at least half of the CUs work; otherwise the most parallel one.
// Tiles taller than the row count are skipped, and the 64-wide tile only holds
// whole heads when they are 64 wide.
void pick_gemm(int M, int N, int K, bool kv, int hd, int num_cus, int* tile, int* split) {
  const int narrow = (!kv || hd == 64) ? 0 : 1;
  int cand[3], nc = 0;
  if (M > 64) cand[nc++] = 3;
  if (M > 16) cand[nc++] = 2;
  cand[nc++] = narrow;
  int best = -1, best_wgs = -1, best_split = 1;
  for (int i = 0; i < nc; ++i) {
    const int t = cand[i];
    const int sp = pick_split(M, N, K, t, num_cus);
    const int wgs = tiles_of(M, N, t) * sp;
    if (wgs >= num_cus / 2) {
      *tile = t;
      *split = sp;
      return;
    }
    if (wgs > best_wgs) {
      best = t;
      best_wgs = wgs;
      best_split = sp;
    }
  }
  *tile = best;
  *split = best_split;
}

}  // namespace

ProjectPlan plan_project(int M, int Dcat, int d, int n_kv, int hd, int dtype, int num_cus) {
  ProjectPlan p{};
  const size_t es = dtype == CO_DTYPE_BF16 ? 2 : 4;
  if (dtype == CO_DTYPE_BF16) {
    pick_gemm(M, d, Dcat, false, hd, num_cus, &p.f_tile, &p.f_split);
    pick_gemm(M, n_kv, d, true, hd, num_cus, &p.kv_tile, &p.kv_split);
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
  p.pe_bytes = (static_cast<size_t>(p.f_split) * d * 4 + 255) / 256 * 256;
  p.total = p.z_bytes + p.part_bytes + p.pe_bytes;
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
  f.partial_e = reinterpret_cast<float*>(ws + p.z_bytes + p.part_bytes);
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
                       dim3(256), 0, stream, part, 1, a.M, a.d, static_cast<float*>(z),
                       static_cast<const float*>(nullptr), a.dst.row_dst);
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
                       dim3(256), 0, stream, part, p.f_split, a.M, a.d, static_cast<uint16_t*>(z),
                       static_cast<const float*>(a.e ? f.partial_e : nullptr), a.dst.row_dst);
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
