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
#include <stdlib.h>

#include <type_traits>

#include "co_route.h"
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
  const float* fe;         // precomputed F(E) [N], added to carry rows (e must be null)
  void* z_out;             // [M][N]
  int mode;
  int z_rows;              // Z mode: 0 every row, 1 rows that are not carry rows, 2 carry rows
  KvDest kv;
  // route_blocks > 0 (bf16 tile kernel, Z mode): the launch also carries the
  // round's route step, four sequences per extra workgroup row past the row
  // tiles, and carried rows are decided from the tokens instead of row_dst
  int route_blocks;
  RouteArgs route;
};

// Whether Z row `dst` is written under the row selection of a Z pass (the
// separate projector computes Z in two passes, one per kind of row).
__device__ __forceinline__ bool z_row_selected(int z_rows, int32_t dst) {
  return z_rows == 0 || (z_rows == 2) == is_carry_row(dst);
}

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
  const int row_tiles = (g.M + BM - 1) / BM;
  if (static_cast<int>(blockIdx.y) >= row_tiles) {   // the route step: one wavefront per sequence
    if (blockIdx.x == 0 && blockIdx.z == 0) {
      const int s = (blockIdx.y - row_tiles) * 4 + wave;
      if (s < g.route.S) route_sequence(g.route, s, lane);
    }
    return;
  }
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
  const bool carry_add = HAS_E || g.fe != nullptr;
  const bool need_rows = carry_add || g.mode == kModeKV || g.z_rows != 0;
  int rd_dst = 0, rd_pos = 0;
  if (need_rows) {
    const int r = min(m0 + (tid % BM), g.M - 1);
    if (g.route_blocks > 0)   // the route runs beside this product: decide from the tokens
      rd_dst = route_row_carried(g.route, r) ? -1 : 0;
    else
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
  if (g.mode == kModeKV && tid < g.kv.hd / 2) inv_tab[tid] = rope_table<uint16_t>(g.kv, tid);
  __shared__ float fe_lds[BN];
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
  } else {
    if (g.fe != nullptr && g.mode == kModeZ)
      for (int c = tid; c < BN; c += 256) fe_lds[c] = n0 + c < g.N ? g.fe[n0 + c] : 0.f;
  }
  __syncthreads();

  if (g.mode == kModeZ) {
    uint16_t* z = static_cast<uint16_t*>(g.z_out);
    for (int c = tid; c < BM * BN / 8; c += 256) {
      const int row = c / (BN / 8), cc = c % (BN / 8);
      const int gr = m0 + row, gc = n0 + cc * 8;
      if (gr >= g.M || gc >= g.N || !z_row_selected(g.z_rows, dst_lds[row])) continue;
      u16x8 v;
      if (carry_add) {
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
      // the hd/8 lanes of a head segment are consecutive and take the same branches
      k_norm<4>(g.kv, gc0 / hd, i0, q_per_seg, lo, hi);
      kv_store<uint16_t, 4>(g.kv, gr, dst_lds[row], pos_lds[row], gc0 / hd, i0, lo, hi, inv_tab);
    }
  }
}

// ------------------------------------------------- bf16 MFMA GEMM, large tiles
//
// For row counts in the hundreds and up.  2 x WGN wavefronts each own a
// (TMW*32) x (TNW*32) block of v_mfma_f32_32x32x16_bf16 tiles, so a workgroup
// tile is (64*TMW) x (32*TNW*WGN) and every fragment read from LDS feeds TMW or
// TNW MFMAs.  With WGN = 4 two wavefronts share each SIMD, so that one issues
// MFMAs while the other waits for its LDS reads or at the stage barrier.  K advances in BK-wide stages through an NS-deep LDS ring filled
// by direct-to-LDS loads issued as opaque inline asm: the compiler then
// schedules the LDS fragment reads freely around the MFMAs, while each
// wavefront waits for its own loads with an exact vmcnt and a barrier
// publishes a stage to the others.  A staged row holds BK bf16 (2*BK bytes);
// its 16-byte chunks are XOR-permuted so that the 16 lanes of one read phase
// (16 consecutive rows, one logical chunk) hit 16 distinct bank groups.
// Fragments are software-pipelined: k16 step h+1 is read while step h
// multiplies, and the next stage is published (and its slot refilled) during
// the stage's last step.  F(E) is accumulated on the VALU from the B fragments
// in registers (a lane holds 8 k values of one column), alternate k16 steps
// on the two wavefront rows; when F(E) is supplied precomputed (g.fe) the
// main loop carries no E at all.  Workgroup ids are renumbered so that each
// XCD (ids congruent mod 8) works on consecutive tiles, which share the same
// A panel and K range.
template <int TMW, int TNW, int BK, int NS, bool HAS_E, int WGN>
__global__ __launch_bounds__(128 * WGN, 1) void gemm_wide_kernel(GemmArgs g, int tiles_m, int tiles_n) {
  constexpr int NW = 2 * WGN, NT = 64 * NW;        // wavefronts, threads
  constexpr int ROWB = 2 * BK;                     // bytes per staged row
  constexpr int CPR = BK / 8;                      // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;                    // rows per 1 KiB load
  constexpr int RPL = 256 / ROWB;                  // rows per 256-byte bank line
  constexpr int H = BK / 16;                       // k16 steps per stage
  constexpr int BM = 64 * TMW, BN = 32 * TNW * WGN;
  constexpr int ROWS = BM + BN;
  constexpr int LPW = ROWS / RPI / NW;             // 1 KiB loads per wavefront per stage
  constexpr int NL = LPW + (HAS_E ? 1 : 0);
  constexpr int E_OFF = ROWS * ROWB;
  constexpr int STAGE = ROWS * ROWB + (HAS_E ? NW * 1024 : 0);
  constexpr int PASS = 64, LDC = BN + 4;           // epilogue: 64 fp32 rows at a time
  static_assert((BK == 32 || BK == 64) && ROWS % (NW * RPI) == 0 && NS >= 2, "tile");
  static_assert(WGN == 2 || WGN == 4, "wavefront columns");
  static_assert(NL * (NS - 1) < 64, "vmcnt");
  static_assert(PASS * LDC * 4 <= NS * STAGE, "C staging must fit in the ring");
  __shared__ __align__(16) unsigned char smem[NS * STAGE];
  __shared__ double inv_tab[64];
  __shared__ float fe_lds[2][BN];
  __shared__ int dst_lds[BM], pos_lds[BM];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  // Tile order: K-split major; within a split, groups of up to 4 row tiles
  // sweep the column tiles, so that consecutive indices form compact blocks
  // of tiles (4 x 8 for 32 indices) that share A and B panels.  Workgroup ids
  // are dealt to the 8 XCDs round-robin; renumbering them gives every XCD a
  // run of consecutive indices, whose shared panels then stay in its L2.
  const int total = gridDim.x;
  int t = blockIdx.x;
  if ((total & 7) == 0) t = (t & 7) * (total >> 3) + (t >> 3);
  const int per_split = tiles_m * tiles_n;
  const int sp = t / per_split, r = t % per_split;
  const int gm = min(4, tiles_m), grp = r / (gm * tiles_n);
  const int gsz = min(gm, tiles_m - grp * gm), rg = r % (gm * tiles_n);
  const int mt = grp * gm + rg % gsz, nt = rg / gsz;
  const int m0 = mt * BM, n0 = nt * BN;
  const int kbeg = sp * g.k_per_split;
  const int nk = min(g.K - kbeg, g.k_per_split) / BK;
  const uint16_t* A = static_cast<const uint16_t*>(g.A);
  const uint16_t* Bw = static_cast<const uint16_t*>(g.B);

  const bool carry_add = HAS_E || g.fe != nullptr;
  const bool need_rows = carry_add || g.mode == kModeKV || g.z_rows != 0;
  int rd_dst = 0, rd_pos = 0;
  if (need_rows) {
    const int r = min(m0 + (tid % BM), g.M - 1);
    rd_dst = g.row_dst[r];
    if (g.mode == kModeKV) rd_pos = g.kv.row_pos[r];
  }

  // this lane's source rows: load j of the wavefront fills rows RPI*(wave*LPW+j) ..
  const uint16_t* src[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int row = (wave * LPW + j) * RPI + lane / CPR;
    const int chunk = (lane % CPR) ^ ((row / RPL) % CPR);
    const uint16_t* base = row < BM ? A + static_cast<int64_t>(min(m0 + row, g.M - 1)) * g.K
                                    : Bw + static_cast<int64_t>(min(n0 + row - BM, g.N - 1)) * g.K;
    src[j] = base + kbeg + chunk * 8;
  }
  // E: every wavefront keeps its own copy of the stage's BK values (chunk c at c*16)
  const uint16_t* src_e =
      HAS_E ? static_cast<const uint16_t*>(g.e) + kbeg + (lane % CPR) * 8 : nullptr;
  const uint32_t ring = lds_addr(smem);

  auto issue = [&](int kt) {
    const uint32_t st = ring + (kt % NS) * STAGE;
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      lds_dma16_opaque(src[j] + kt * BK, st + (wave * LPW + j) * 1024);
    if constexpr (HAS_E) lds_dma16_opaque(src_e + kt * BK, st + E_OFF + wave * 1024);
  };

  f32x16 acc[TMW][TNW];
#pragma unroll
  for (int a = 0; a < TMW; ++a)
#pragma unroll
    for (int b = 0; b < TNW; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
  float fe[TNW];
#pragma unroll
  for (int b = 0; b < TNW; ++b) fe[b] = 0.f;

  // fragment offsets within a stage: row (lane % 32) of each 32-row tile; the
  // logical chunk of k16 step h is 2h + lane/32, stored permuted
  const int frow = (lane & 31) * ROWB;
  const int fswz = ((lane & 31) / RPL) % CPR;

  struct Frags {
    u16x8 a[TMW], b[TNW], e;
  };
  auto load = [&](int kt, int h, Frags& f) {
    const unsigned char* st = smem + (kt % NS) * STAGE;
    const int c = 2 * h + (lane >> 5);
    const int off = frow + ((c ^ fswz) << 4);
#pragma unroll
    for (int a = 0; a < TMW; ++a)
      f.a[a] = *reinterpret_cast<const u16x8*>(st + (wm * TMW + a) * 32 * ROWB + off);
#pragma unroll
    for (int b = 0; b < TNW; ++b)
      f.b[b] = *reinterpret_cast<const u16x8*>(st + (BM + (wn * TNW + b) * 32) * ROWB + off);
    if (HAS_E && (h & 1) == wm)
      f.e = *reinterpret_cast<const u16x8*>(st + E_OFF + wave * 1024 + c * 16);
  };
  // Marks fragments as read: the compiler places its LDS wait for them here (the
  // barrier that follows waits for all LDS reads anyway), so the MFMAs that
  // consume them do not also wait for the next stage's reads issued meanwhile.
  auto settle = [&](int h, Frags& f) {
#pragma unroll
    for (int a = 0; a < TMW; ++a) asm volatile("" : "+v"(f.a[a]));
#pragma unroll
    for (int b = 0; b < TNW; ++b) asm volatile("" : "+v"(f.b[b]));
    if (HAS_E && (h & 1) == wm) asm volatile("" : "+v"(f.e));
  };
  auto compute = [&](int h, const Frags& f) {
#pragma unroll
    for (int a = 0; a < TMW; ++a)
#pragma unroll
      for (int b = 0; b < TNW; ++b) acc[a][b] = mfma32x32x16(f.a[a], f.b[b], acc[a][b]);
    if (HAS_E && (h & 1) == wm) {
#pragma unroll
      for (int b = 0; b < TNW; ++b)
#pragma unroll
        for (int i = 0; i < 8; ++i) fe[b] = fmaf(bf2f(f.b[b][i]), bf2f(f.e[i]), fe[b]);
    }
  };
  // Wait until this wavefront's loads of the stage `ahead` stages before the
  // newest one issued have landed, then publish through the barrier.
  auto wait_stage = [&](int ahead) {
    if (NS >= 4 && ahead >= 3) wait_vm_lgkm_barrier<(NS >= 4 ? 3 * NL : 0)>();
    else if (NS >= 3 && ahead >= 2) wait_vm_lgkm_barrier<(NS >= 3 ? 2 * NL : 0)>();
    else if (ahead >= 1) wait_vm_lgkm_barrier<NL>();
    else wait_vm_lgkm_barrier<0>();
  };

  // Stage kt+1 is published by the barrier taken during the last k16 step of
  // stage kt; by then every wavefront holds all of stage kt in registers, so
  // its slot takes the loads of stage kt+NS.
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < nk) issue(s);
  Frags f0, f1;
  if (nk > 0) {
    wait_stage(min(NS - 1, nk - 1));
    load(0, 0, f0);
  }
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int h = 0; h < H; ++h) {
      Frags& cur = (h & 1) ? f1 : f0;
      Frags& nxt = (h & 1) ? f0 : f1;
      if (h + 1 < H) load(kt, h + 1, nxt);
      __builtin_amdgcn_sched_barrier(0);
      compute(h, cur);
      __builtin_amdgcn_sched_barrier(0);
      if (h + 2 == H) {
        settle(h + 1, nxt);
        if (kt + 1 < nk) {
          wait_stage(min(NS - 2, nk - 2 - kt));
          if (kt + NS < nk) issue(kt + NS);
          load(kt + 1, 0, cur);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // the ring is reused below: every wavefront must be done with its last stage
  wait_vm_lgkm_barrier<0>();

  if constexpr (HAS_E) {
    // the two k halves of each column sit in lanes l and l ^ 32
#pragma unroll
    for (int b = 0; b < TNW; ++b) fe[b] += __shfl_xor(fe[b], 32);
    if (lane < 32) {
#pragma unroll
      for (int b = 0; b < TNW; ++b) fe_lds[wm][(wn * TNW + b) * 32 + lane] = fe[b];
    }
  } else {
    if (g.fe != nullptr && g.mode == kModeZ)
      for (int c = tid; c < BN; c += NT) fe_lds[0][c] = n0 + c < g.N ? g.fe[n0 + c] : 0.f;
  }

  if (g.mode == kModePartial) {
    float* out = g.partial + static_cast<int64_t>(sp) * g.M * g.N;
#pragma unroll
    for (int a = 0; a < TMW; ++a)
#pragma unroll
      for (int b = 0; b < TNW; ++b) {
        const int col = n0 + (wn * TNW + b) * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + (wm * TMW + a) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < g.M && col < g.N) out[static_cast<int64_t>(row) * g.N + col] = acc[a][b][r];
        }
      }
    if constexpr (HAS_E) {
      __syncthreads();
      if (mt == 0)
        for (int c = tid; c < BN; c += NT)
          if (n0 + c < g.N)
            g.partial_e[static_cast<int64_t>(sp) * g.N + n0 + c] = fe_lds[0][c] + fe_lds[1][c];
    }
    return;
  }

  if (g.mode == kModeKV && tid < g.kv.hd / 2) inv_tab[tid] = rope_table<uint16_t>(g.kv, tid);
  asm volatile("" : "+v"(rd_dst), "+v"(rd_pos));
  if (need_rows && tid < BM) {
    dst_lds[tid] = rd_dst;
    pos_lds[tid] = rd_pos;
  }
  float* sc = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int p = 0; p < BM / PASS; ++p) {
    // the wavefronts holding rows p*64 .. +63 stage them as fp32
#pragma unroll
    for (int a = 0; a < TMW; ++a) {
      if ((wm * TMW + a) * 32 / PASS != p) continue;
#pragma unroll
      for (int b = 0; b < TNW; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = (wm * TMW + a) * 32 - p * PASS + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          sc[row * LDC + (wn * TNW + b) * 32 + (lane & 31)] = acc[a][b][r];
        }
    }
    __syncthreads();
    if (g.mode == kModeZ) {
      uint16_t* z = static_cast<uint16_t*>(g.z_out);
      for (int c = tid; c < PASS * BN / 8; c += NT) {
        const int rl = c / (BN / 8), cc = c % (BN / 8);
        const int row = p * PASS + rl;
        const int gr = m0 + row, gc = n0 + cc * 8;
        if (gr >= g.M || gc >= g.N || !z_row_selected(g.z_rows, dst_lds[row])) continue;
        u16x8 v;
        if (carry_add && is_carry_row(dst_lds[row])) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float f = HAS_E ? fe_lds[0][cc * 8 + q] + fe_lds[1][cc * 8 + q] : fe_lds[0][cc * 8 + q];
            v[q] = f2bf(sc[rl * LDC + cc * 8 + q] + f);
          }
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) v[q] = f2bf(sc[rl * LDC + cc * 8 + q]);
        }
        *reinterpret_cast<u16x8*>(z + static_cast<int64_t>(gr) * g.N + gc) = v;
      }
    } else {
      const int hd = g.kv.hd, q_per_seg = hd / 8;
      for (int c = tid; c < PASS * BN / 8; c += NT) {
        const int rl = c / (BN / 8), q = c % (BN / 8);
        const int row = p * PASS + rl;
        const int seg_local = q / q_per_seg, i0 = (q % q_per_seg) * 4;
        const int gr = m0 + row, gc0 = n0 + seg_local * hd;
        if (gr >= g.M || gc0 >= g.N) continue;
        float lo[4], hi[4];
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {
          lo[pp] = sc[rl * LDC + seg_local * hd + i0 + pp];
          hi[pp] = sc[rl * LDC + seg_local * hd + hd / 2 + i0 + pp];
        }
        k_norm<4>(g.kv, gc0 / hd, i0, q_per_seg, lo, hi);   // hd/8 consecutive lanes per segment
        kv_store<uint16_t, 4>(g.kv, gr, dst_lds[row], pos_lds[row], gc0 / hd, i0, lo, hi, inv_tab);
      }
    }
    __syncthreads();
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
  // K split blockIdx.z: k in [kb, ke), its partial product in slice blockIdx.z
  const int kb = blockIdx.z * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);
  float* out = g.partial + static_cast<int64_t>(blockIdx.z) * g.M * g.N;
  float acc[2][4] = {};
  for (int k0 = kb; k0 < ke; k0 += BK) {
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
      if (row < g.M && col < g.N) out[static_cast<int64_t>(row) * g.N + col] = acc[i][j];
    }
}

// ------------------------------------- fused projection, small widths
// At d = n_kv = 256 (one head_dim-64 segment per 64 K/V columns) and many
// rows, both products of a block of 128 rows run in one workgroup: Z = F(x)
// stays in LDS as bf16 and feeds the K/V product directly, whose rotation and
// scatter follow from registers.  Both products are computed transposed, with
// the weights as the MFMA A operand: a lane then holds four consecutive
// columns of one row, so Z rows are written to LDS 8 bytes at a time and the
// rotation pairs (i, i + 32) of a head lie in one lane.  Wavefront w owns
// columns 64w .. 64w + 63 of both products (one K/V segment).
constexpr int kFusedD = 256;                 // d and n_kv of the fused path
constexpr int kFusedBM = 128;                // rows per workgroup
constexpr int kFusedZLD = kFusedD * 2 + 16;  // bytes per Z row in LDS (padded against conflicts)

__global__ __launch_bounds__(256, 1) void proj_fused_kernel(ProjectArgs a) {
  // F stages are 64 deep (3 in the ring), K/V stages 32 deep (4 in the ring
  // behind the resident Z rows)
  constexpr int BM = kFusedBM, BK1 = 64, BK2 = 32, NS1 = 3, NS2 = 4;
  constexpr int ROWB1 = 2 * BK1, CPR1 = BK1 / 8, RPI1 = 64 / CPR1, RPL1 = 256 / ROWB1;
  constexpr int ROWB2 = 2 * BK2, CPR2 = BK2 / 8, RPI2 = 64 / CPR2, RPL2 = 256 / ROWB2;
  constexpr int TM = BM / 32, TN = 2;          // activation and weight tiles per wavefront
  constexpr int WR = kFusedD;                  // weight rows of a stage (both products)
  constexpr int LPW1 = (WR + BM) / RPI1 / 4;   // 1 KiB loads per wavefront, F stage
  constexpr int LPW2 = WR / RPI2 / 4;          // same, K/V stage
  constexpr int STAGE1 = (WR + BM) * ROWB1, STAGE2 = WR * ROWB2;
  constexpr int Z_BYTES = BM * kFusedZLD;
  constexpr int RING1 = NS1 * STAGE1, RING2 = Z_BYTES + NS2 * STAGE2;
  constexpr int LDS_BYTES = RING1 > RING2 ? RING1 : RING2;
  static_assert((WR + BM) % (4 * RPI1) == 0 && WR % (4 * RPI2) == 0, "tile");
  static_assert(LPW1 * (NS1 - 1) < 64 && LPW2 * NS2 < 64, "vmcnt");
  __shared__ __align__(16) unsigned char smem[LDS_BYTES];
  __shared__ double inv_tab[32];
  __shared__ __align__(16) float fe_lds[kFusedD];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m0 = blockIdx.x * BM;
  const int M = a.M, Dcat = a.Dcat;
  const uint16_t* X = static_cast<const uint16_t*>(a.hidden);
  const uint16_t* Wf = static_cast<const uint16_t*>(a.wf);
  const uint16_t* Wkv = static_cast<const uint16_t*>(a.wkv);

  // descriptors of this lane's rows (row m0 + 32 tm + lane % 32)
  int rdst[TM], rpos[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int r = min(m0 + 32 * tm + (lane & 31), M - 1);
    rdst[tm] = a.dst.row_dst[r];
    rpos[tm] = a.dst.row_pos[r];
  }
  // the rotation table through scalar loads (indexing the argument by lane
  // would make it a vector load, and the first wait on it would also wait for
  // the staged loads issued after it)
  if (tid == 0) {
#pragma unroll
    for (int i = 0; i < 32; ++i) inv_tab[i] = rope_table<uint16_t>(a.dst, i);
  }
  // F(E) of this thread's column, written to LDS once the F product is done
  // (the loads above are waited for there, when no staged load is in flight)
  float fe_mine = a.fe != nullptr ? a.fe[tid] : 0.f;

  // DMA sources: load j of this wavefront fills stage rows RPI*(wave*LPW+j) ..
  const uint16_t* src1[LPW1];
#pragma unroll
  for (int j = 0; j < LPW1; ++j) {
    const int row = (wave * LPW1 + j) * RPI1 + lane / CPR1;
    const int chunk = (lane % CPR1) ^ ((row / RPL1) % CPR1);
    const uint16_t* base = row < WR ? Wf + static_cast<int64_t>(row) * Dcat
                                    : X + static_cast<int64_t>(min(m0 + row - WR, M - 1)) * Dcat;
    src1[j] = base + chunk * 8;
  }
  const uint16_t* src2[LPW2];
#pragma unroll
  for (int j = 0; j < LPW2; ++j) {
    const int row = (wave * LPW2 + j) * RPI2 + lane / CPR2;
    const int chunk = (lane % CPR2) ^ ((row / RPL2) % CPR2);
    src2[j] = Wkv + static_cast<int64_t>(row) * kFusedD + chunk * 8;
  }
  const uint32_t lds0 = lds_addr(smem);
  // Every workgroup reads the same weights: the workgroups of one XCD (ids
  // congruent mod 8) start their K loops at different stages, so that they do
  // not all request the same weight lines from its L2 at the same time.
  const int nk1 = Dcat / BK1, nk2 = kFusedD / BK2;
  const int rot1 = (blockIdx.x >> 3) % nk1, rot2 = (blockIdx.x >> 3) % nk2;
  auto issue1 = [&](int kt) {
    const uint32_t st = lds0 + (kt % NS1) * STAGE1;
    const int ks = kt + rot1 < nk1 ? kt + rot1 : kt + rot1 - nk1;
#pragma unroll
    for (int j = 0; j < LPW1; ++j) lds_dma16_opaque(src1[j] + ks * BK1, st + (wave * LPW1 + j) * 1024);
  };
  auto issue2 = [&](int kt) {
    const uint32_t st = lds0 + Z_BYTES + (kt % NS2) * STAGE2;
    const int ks = kt + rot2 < nk2 ? kt + rot2 : kt + rot2 - nk2;
#pragma unroll
    for (int j = 0; j < LPW2; ++j) lds_dma16_opaque(src2[j] + ks * BK2, st + (wave * LPW2 + j) * 1024);
  };

  // fragment offsets within a stage: row lane % 32 of a 32-row tile, logical
  // 16-byte chunk 2h + lane / 32 of k16 step h, stored permuted
  const int frow1 = (lane & 31) * ROWB1, fswz1 = ((lane & 31) / RPL1) % CPR1;
  const int frow2 = (lane & 31) * ROWB2, fswz2 = ((lane & 31) / RPL2) % CPR2;
  struct Frags {
    u16x8 w[TN], x[TM];
  };
  auto load1 = [&](int kt, int h, Frags& f) {
    const unsigned char* st = smem + (kt % NS1) * STAGE1;
    const int off = frow1 + (((2 * h + (lane >> 5)) ^ fswz1) << 4);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
      f.w[tn] = *reinterpret_cast<const u16x8*>(st + (wave * 64 + tn * 32) * ROWB1 + off);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
      f.x[tm] = *reinterpret_cast<const u16x8*>(st + (WR + tm * 32) * ROWB1 + off);
  };
  // K/V stage: weights from the ring, Z (the B operand) from its resident rows
  auto load2 = [&](int kt, int h, Frags& f) {
    const unsigned char* st = smem + Z_BYTES + (kt % NS2) * STAGE2;
    const int off = frow2 + (((2 * h + (lane >> 5)) ^ fswz2) << 4);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
      f.w[tn] = *reinterpret_cast<const u16x8*>(st + (wave * 64 + tn * 32) * ROWB2 + off);
    const int ks = kt + rot2 < nk2 ? kt + rot2 : kt + rot2 - nk2;
    const int zoff = (lane & 31) * kFusedZLD + (ks * BK2 + h * 16 + 8 * (lane >> 5)) * 2;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
      f.x[tm] = *reinterpret_cast<const u16x8*>(smem + tm * 32 * kFusedZLD + zoff);
  };
  auto settle = [&](Frags& f) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) asm volatile("" : "+v"(f.w[tn]));
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) asm volatile("" : "+v"(f.x[tm]));
  };
  f32x16 acc[TN][TM];
  auto zero = [&]() {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[tn][tm][r] = 0.f;
  };
  auto compute = [&](const Frags& f) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) acc[tn][tm] = mfma32x32x16(f.w[tn], f.x[tm], acc[tn][tm]);
  };
  // stage kt+1 is published by the barrier taken in the last k16 step of stage
  // kt, after which stage kt's slot takes the loads of stage kt + NS
  auto run = [&](int nk, int NS, auto k16_steps, auto issue, auto load, auto wait_ahead) {
    constexpr int H = decltype(k16_steps)::value;   // k16 steps per stage
    Frags f0, f1;
    wait_ahead(min(NS - 1, nk - 1));
    load(0, 0, f0);
    for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
      for (int h = 0; h < H; ++h) {
        Frags& cur = (h & 1) ? f1 : f0;
        Frags& nxt = (h & 1) ? f0 : f1;
        if (h + 1 < H) load(kt, h + 1, nxt);
        __builtin_amdgcn_sched_barrier(0);
        compute(cur);
        __builtin_amdgcn_sched_barrier(0);
        if (h + 2 == H) {
          settle(nxt);
          if (kt + 1 < nk) {
            wait_ahead(min(NS - 2, nk - 2 - kt));
            if (kt + NS < nk) issue(kt + NS);
            load(kt + 1, 0, cur);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };
  // wait until the loads of the stage `ahead` stages before the newest one
  // issued have landed (ahead < ring depth), then publish through the barrier
  auto wait1 = [&](int ahead) {
    if (ahead >= 2) wait_vm_lgkm_barrier<2 * LPW1>();
    else if (ahead == 1) wait_vm_lgkm_barrier<LPW1>();
    else wait_vm_lgkm_barrier<0>();
  };
  auto wait2 = [&](int ahead) {
    if (ahead >= 3) wait_vm_lgkm_barrier<3 * LPW2>();
    else if (ahead == 2) wait_vm_lgkm_barrier<2 * LPW2>();
    else if (ahead == 1) wait_vm_lgkm_barrier<LPW2>();
    else wait_vm_lgkm_barrier<0>();
  };
  static_assert(NS1 <= 3 && NS2 <= 4, "wait1/wait2 cover these depths");

  // ---- Z^T = W_F x^T over Dcat
#pragma unroll
  for (int s = 0; s < NS1; ++s)
    if (s < nk1) issue1(s);
  zero();
  run(nk1, NS1, std::integral_constant<int, BK1 / 16>{}, issue1, load1, wait1);
  wait_vm_lgkm_barrier<0>();   // every wavefront is done with the F ring
  asm volatile("" : "+v"(fe_mine));
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) asm volatile("" : "+v"(rdst[tm]), "+v"(rpos[tm]));
  fe_lds[tid] = fe_mine;
  __syncthreads();

  // the K/V weights start streaming into the ring behind Z meanwhile
#pragma unroll
  for (int s = 0; s < NS2; ++s) issue2(s);

  // Z rows to LDS as bf16; carried rows get F(E) (added in fp32 before rounding)
#pragma unroll
  for (int tn = 0; tn < TN; ++tn)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = wave * 64 + tn * 32 + 8 * q + 4 * (lane >> 5);
      const f32x4 fe = *reinterpret_cast<const f32x4*>(fe_lds + n);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const bool carried = is_carry_row(rdst[tm]);
        u16x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = f2bf(acc[tn][tm][4 * q + j] + (carried ? fe[j] : 0.f));
        *reinterpret_cast<u16x4*>(smem + (tm * 32 + (lane & 31)) * kFusedZLD + n * 2) = v;
      }
    }

  // ---- K/V^T = W_KV Z^T over d
  zero();
  run(nk2, NS2, std::integral_constant<int, BK2 / 16>{}, issue2, load2, wait2);

  // ---- rotate keys at the row's position and store every row to its slot
  // (stores of a few bytes per lane: staging the rows in LDS for full-line
  // stores measured no faster, the write burst at the end of the kernel is
  // what this phase waits on)
  const int i_base = 4 * (lane >> 5);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int row = m0 + tm * 32 + (lane & 31);
    if (row >= M) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float lo[4], hi[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lo[j] = acc[0][tm][4 * q + j];
        hi[j] = acc[1][tm][4 * q + j];
      }
      kv_store<uint16_t, 4>(a.dst, row, rdst[tm], rpos[tm], wave, 8 * q + i_base, lo, hi, inv_tab);
    }
  }
}

// ------------------------------------------------- RMS norm of F's output
// The normalisation variant: every row of Z is divided by its root mean
// square (epsilon kRmsEps) and multiplied by the gain g before the K/V
// product.  One workgroup per row, fp32 arithmetic; every load of the row is
// issued before the first is used.  Rows of up to kNormMaxCols columns.

__device__ __forceinline__ float block_sum_256(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// In place, for a Z the GEMM wrote whole (no split partials).
template <typename T>
__global__ __launch_bounds__(256) void z_norm_kernel(T* z, int M, int d, const float* g) {
  constexpr int QMAX = kNormMaxCols / 1024;   // column quads per thread
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  T* zr = z + static_cast<int64_t>(row) * d;
  f32x4 v[QMAX];
  float ss = 0.f;
#pragma unroll
  for (int qi = 0; qi < QMAX; ++qi) {
    const int col = (tid + 256 * qi) * 4;
    v[qi] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (col < d) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (sizeof(T) == 2) v[qi][q] = bf2f(zr[col + q]); else v[qi][q] = zr[col + q];
      }
    }
  }
#pragma unroll
  for (int qi = 0; qi < QMAX; ++qi)
    ss += (v[qi][0] * v[qi][0] + v[qi][1] * v[qi][1]) + (v[qi][2] * v[qi][2] + v[qi][3] * v[qi][3]);
  const float r = rsqrtf(block_sum_256(ss, red) / static_cast<float>(d) + kRmsEps);
#pragma unroll
  for (int qi = 0; qi < QMAX; ++qi) {
    const int col = (tid + 256 * qi) * 4;
    if (col < d) {
#pragma unroll
      for (int q = 0; q < 4; ++q) zr[col + q] = to_elem<T>(v[qi][q] * r * g[col + q]);
    }
  }
}

// The epilogue of a split F product with the normalisation: the row's split
// partials are summed (plus F(E), or E's split partials, on carry rows), the
// row's sum of squares reduced over the workgroup, and the normalised row
// written once.  Rows not selected by z_rows (separate projector) are left.
template <typename T>
__global__ __launch_bounds__(256) void epi_z_norm_kernel(const float* part, int splits, int M,
                                                         int N, T* z, const float* part_e,
                                                         const float* fe, const int32_t* row_dst,
                                                         int z_rows, const float* g) {
  constexpr int QMAX = kNormMaxCols / 1024;
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  if (!z_row_selected(z_rows, row_dst[row])) return;   // uniform over the workgroup
  const bool carry = (part_e || fe) && is_carry_row(row_dst[row]);
  const int64_t MN = static_cast<int64_t>(M) * N;
  const float* pr = part + static_cast<int64_t>(row) * N;
  f32x4 v[QMAX];
  float ss = 0.f;
#pragma unroll
  for (int qi = 0; qi < QMAX; ++qi) {
    const int col = (tid + 256 * qi) * 4;
    v[qi] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (col < N) {
      for (int sp = 0; sp < splits; ++sp) v[qi] += *reinterpret_cast<const f32x4*>(pr + sp * MN + col);
      if (carry) {
        if (fe) {
          v[qi] += *reinterpret_cast<const f32x4*>(fe + col);
        } else {
          for (int sp = 0; sp < splits; ++sp)
            v[qi] += *reinterpret_cast<const f32x4*>(part_e + static_cast<int64_t>(sp) * N + col);
        }
      }
    }
    ss += (v[qi][0] * v[qi][0] + v[qi][1] * v[qi][1]) + (v[qi][2] * v[qi][2] + v[qi][3] * v[qi][3]);
  }
  const float r = rsqrtf(block_sum_256(ss, red) / static_cast<float>(N) + kRmsEps);
  T* zr = z + static_cast<int64_t>(row) * N;
#pragma unroll
  for (int qi = 0; qi < QMAX; ++qi) {
    const int col = (tid + 256 * qi) * 4;
    if (col < N) {
#pragma unroll
      for (int q = 0; q < 4; ++q) zr[col + q] = to_elem<T>(v[qi][q] * r * g[col + q]);
    }
  }
}

// -------------------------------------------- epilogues over fp32 partials

// Four consecutive columns per thread (N is a multiple of 64).
template <typename T>
__global__ __launch_bounds__(256) void epi_z_kernel(const float* part, int splits, int M, int N,
                                                    T* z, const float* part_e, const float* fe,
                                                    const int32_t* row_dst, int z_rows) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  const int64_t MN = static_cast<int64_t>(M) * N;
  if (i >= MN || !z_row_selected(z_rows, row_dst[i / N])) return;
  f32x4 v = *reinterpret_cast<const f32x4*>(part + i);
  for (int s = 1; s < splits; ++s) v += *reinterpret_cast<const f32x4*>(part + s * MN + i);
  if ((part_e || fe) && is_carry_row(row_dst[i / N])) {
    const int col = static_cast<int>(i % N);
    if (fe) {
      v += *reinterpret_cast<const f32x4*>(fe + col);
    } else {
      f32x4 e = *reinterpret_cast<const f32x4*>(part_e + col);
      for (int s = 1; s < splits; ++s) e += *reinterpret_cast<const f32x4*>(part_e + static_cast<int64_t>(s) * N + col);
      v += e;
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) z[i + q] = to_elem<T>(v[q]);
}

template <typename T>
__global__ __launch_bounds__(256) void epi_kv_kernel(const float* part, int splits, int M, int N,
                                                     KvDest e) {
  __shared__ double inv_tab[64];
  const int half = e.hd / 2;
  if (threadIdx.x < half) inv_tab[threadIdx.x] = rope_table<T>(e, threadIdx.x);
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
  k_norm<1>(e, seg, p, half, &lo, &hi);   // a segment's hd/2 pairs: consecutive, aligned lanes
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
                  (g.M + kTileBM[tile] - 1) / kTileBM[tile] + g.route_blocks, splits);
  switch (tile) {
    case 0: hipLaunchKernelGGL((gemm_bf16_kernel<16, 64, 1, 4, 4, HAS_E>), grid, dim3(256), 0, stream, g); break;
    case 1: hipLaunchKernelGGL((gemm_bf16_kernel<16, 128, 1, 4, 3, HAS_E>), grid, dim3(256), 0, stream, g); break;
    case 2: hipLaunchKernelGGL((gemm_bf16_kernel<64, 128, 2, 2, 2, HAS_E>), grid, dim3(256), 0, stream, g); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<128, 128, 2, 2, 2, HAS_E>), grid, dim3(256), 0, stream, g); break;
  }
  return hipGetLastError();
}

// Large-tile variants: eight wavefronts (2 x 4), each a block of 32 x 32
// tiles; stage depth BK, ring depth NS.  Two wavefronts per SIMD measured
// 3-11% faster than four wavefronts with twice the block at every projection
// shape (same tiles, same results bit for bit).
//   0: 256 x 256, BK 32 x 4   1: 256 x 128, BK 32 x 4   2: 128 x 256, BK 32 x 4
//   3: 256 x 256, BK 64 x 2   4: 256 x 128, BK 64 x 3   5: 128 x 256, BK 64 x 3
//   6: 128 x 128, BK 64 x 4 (enough workgroups for the K/V product without a K split)
constexpr int kWide = 4, kWideVariants = 7;
constexpr int kWideBM[kWideVariants] = {256, 256, 128, 256, 256, 128, 128};
constexpr int kWideBN[kWideVariants] = {256, 128, 256, 256, 128, 256, 128};

template <bool HAS_E>
hipError_t launch_gemm_wide_t(const GemmArgs& g, int variant, int splits, hipStream_t stream) {
  // in-kernel E keeps a copy of E per wavefront and stage, which fits the LDS
  // with four wavefronts (2 x 2, blocks twice as wide) but not with eight
  constexpr int W = HAS_E ? 2 : 4, X = 4 / W;
  const int tm = (g.M + kWideBM[variant] - 1) / kWideBM[variant];
  const int tn = (g.N + kWideBN[variant] - 1) / kWideBN[variant];
  const dim3 grid(tm * tn * splits), block(128 * W);
  switch (variant) {
    case 0: hipLaunchKernelGGL((gemm_wide_kernel<4, 2 * X, 32, 4, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
    case 1: hipLaunchKernelGGL((gemm_wide_kernel<4, X, 32, 4, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
    case 2: hipLaunchKernelGGL((gemm_wide_kernel<2, 2 * X, 32, 4, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
    case 3: hipLaunchKernelGGL((gemm_wide_kernel<4, 2 * X, 64, 2, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
    case 4: hipLaunchKernelGGL((gemm_wide_kernel<4, X, 64, 3, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
    case 5: hipLaunchKernelGGL((gemm_wide_kernel<2, 2 * X, 64, 3, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
    default: hipLaunchKernelGGL((gemm_wide_kernel<2, X, 64, 4, HAS_E, W>), grid, block, 0, stream, g, tm, tn); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& g, int tile, int splits, hipStream_t stream) {
  if (tile >= kWide)
    return g.e ? launch_gemm_wide_t<true>(g, tile - kWide, splits, stream)
               : launch_gemm_wide_t<false>(g, tile - kWide, splits, stream);
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
// Large-tile choice for shapes with hundreds of rows or more: the variant and
// K-split with the least estimated time, counting whole waves of workgroups at
// a per-CU MFMA rate (the 256 x 256 tile reads LDS least per flop) plus the
// fp32 partials that a split writes and reads back.  Returns false when no
// choice fills at least half of the CUs.  CO_TUNE_GEMM_WIDE_VARIANT = v restricts
// the choice to variant v at any size from 256 rows (tests and tuning).
// K elements per split: the stage depth of the tile variant divides it.
int split_len(int K, int split, int tile) {
  const int bk = tile >= kWide + 3 ? 64 : 32;
  return ((K + split - 1) / split + bk - 1) / bk * bk;
}

bool pick_wide(int M, int N, int K, bool kv, int num_cus, int* tile, int* split) {
  if (M < 256 || K % 64 != 0) return false;
  double best = 1e30;
  int bv = -1, bs = 1;
  const int64_t force = tuning(CO_TUNE_GEMM_WIDE_VARIANT);
  for (int v = 0; v < kWideVariants; ++v) {
    if (force >= 0 && force != v) continue;
    const int64_t tiles = static_cast<int64_t>((M + kWideBM[v] - 1) / kWideBM[v]) *
                          ((N + kWideBN[v] - 1) / kWideBN[v]);
    // relative main-loop rates measured on MI355X, each variant timed alone at
    // the projection shapes (the 64-deep stages and the square tile move the
    // fewest bytes per flop through LDS)
    constexpr double kEff[kWideVariants] = {0.98, 0.8, 0.8, 1.0, 0.86, 0.87, 0.86};
    const double eff = kEff[v];
    for (int s = 1; s <= 16; ++s) {
      const int kps = split_len(K, s, kWide + v);
      if (kps < 256 || (K + kps - 1) / kps != s) continue;
      const int64_t wgs = tiles * s;
      if (wgs < num_cus / 2 && force < 0) continue;
      const int64_t waves = (wgs + num_cus - 1) / num_cus;
      // main loop at the per-CU rate measured with operands streaming from HBM,
      // or the weights streamed from HBM once per row tile, whichever is longer
      const double t_mfma = static_cast<double>(waves) * kWideBM[v] * kWideBN[v] * kps * 2.0 /
                            (4.5e12 * eff);
      const double t_hbm = static_cast<double>((M + kWideBM[v] - 1) / kWideBM[v]) * N * K * 2.0 / 6.0e12;
      // split partials: their stores overlap the main loop; the epilogue kernel
      // reads them back (the K/V epilogue, with its rotation and page scatter,
      // measured at about half the rate of the Z epilogue)
      const double t_part = s > 1 ? static_cast<double>(s) * M * N * 4.0 / (kv ? 2.5e12 : 5.0e12) +
                                        (kv ? 4e-6 : 2e-6)
                                  : 0.0;
      const double t = (t_mfma > t_hbm ? t_mfma : t_hbm) + t_part;
      if (t < best) {
        best = t;
        bv = v;
        bs = s;
      }
    }
  }
  if (bv < 0) return false;
  *tile = kWide + bv;
  *split = bs;
  return true;
}

void pick_gemm(int M, int N, int K, bool kv, int hd, int num_cus, int* tile, int* split) {
  if (tuning(CO_TUNE_GEMM_NO_WIDE) <= 0 && pick_wide(M, N, K, kv, num_cus, tile, split)) return;
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

constexpr int kF32SplitK = 64;   // K per split of the fp32 GEMM

// Rows from which the fused small-width projection is used: below, the K-split
// two-product path spreads the weight reads over more workgroups.
static int fused_min_rows() {
  const int64_t v = tuning(CO_TUNE_PROJECT_FUSED_MIN_ROWS);
  if (v >= 1) return v < INT32_MAX ? static_cast<int>(v) : INT32_MAX;
  return 4096;
}

static int f32_splits(int K) {
  const int s = (K + kF32SplitK - 1) / kF32SplitK;
  return s < 1 ? 1 : (s > 32 ? 32 : s);
}

ProjectPlan plan_project(int M, int Dcat, int d, int n_kv, int hd, int dtype, int num_cus) {
  ProjectPlan p{};
  const size_t es = dtype == CO_DTYPE_BF16 ? 2 : 4;
  p.fused = dtype == CO_DTYPE_BF16 && d == kFusedD && n_kv == kFusedD && hd == 64 &&
            Dcat % 64 == 0 && M >= fused_min_rows();
  if (dtype == CO_DTYPE_BF16) {
    pick_gemm(M, d, Dcat, false, hd, num_cus, &p.f_tile, &p.f_split);
    pick_gemm(M, n_kv, d, true, hd, num_cus, &p.kv_tile, &p.kv_split);
  } else {
    // fp32: K split in pieces of two 32-deep steps, so that few dependent load
    // rounds lie on any workgroup's path (the shapes it serves are latency-bound)
    p.f_tile = p.kv_tile = -1;
    p.f_split = f32_splits(Dcat);
    p.kv_split = f32_splits(d);
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

bool route_foldable(const ProjectArgs& a, const ProjectPlan& p) {
  const bool sep = a.wfc != nullptr;
  const bool fused = !sep && a.znorm == nullptr && a.dst.knorm == nullptr && p.fused &&
                     (a.fe != nullptr || a.e == nullptr);
  return a.dtype == CO_DTYPE_BF16 && a.M > 0 && !sep && !fused && p.f_tile < kWide &&
         p.f_split == 1;
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
  f.A = a.hidden; f.B = a.wf; f.e = a.e; f.fe = nullptr; f.row_dst = a.dst.row_dst;
  f.partial = part; f.z_out = z; f.kv = a.dst;
  f.partial_e = reinterpret_cast<float*>(ws + p.z_bytes + p.part_bytes);
  GemmArgs kv{};
  kv.M = a.M; kv.N = n_kv; kv.K = a.d;
  kv.A = z; kv.B = a.wkv; kv.e = nullptr; kv.row_dst = a.dst.row_dst;
  kv.partial = part; kv.z_out = nullptr; kv.kv = a.dst;
  // Separate projector: Z in two passes, F for the rows that are not carry
  // rows, then the carry projector for the carry rows; no E either way.
  const bool sep = a.wfc != nullptr;
  const int passes = sep ? 2 : 1;
  if (sep) f.e = nullptr;

  if (a.dtype == CO_DTYPE_F32) {
    f.k_per_split = ((f.K + p.f_split - 1) / p.f_split + 31) / 32 * 32;
    kv.k_per_split = ((kv.K + p.kv_split - 1) / p.kv_split + 31) / 32 * 32;
    const int fs = (f.K + f.k_per_split - 1) / f.k_per_split;
    const int ks = (kv.K + kv.k_per_split - 1) / kv.k_per_split;
    f.mode = kv.mode = kModePartial;
    const int64_t nz = static_cast<int64_t>(a.M) * a.d / 4;
    for (int pass = 0; pass < passes; ++pass) {
      if (pass == 1) f.B = a.wfc;
      hipLaunchKernelGGL(gemm_f32_kernel, dim3((f.N + 63) / 64, (f.M + 31) / 32, fs), dim3(256),
                         0, stream, f);
      if (a.znorm != nullptr)
        hipLaunchKernelGGL(epi_z_norm_kernel<float>, dim3(a.M), dim3(256), 0, stream, part, fs,
                           a.M, a.d, static_cast<float*>(z), static_cast<const float*>(nullptr),
                           static_cast<const float*>(nullptr), a.dst.row_dst, sep ? pass + 1 : 0,
                           a.znorm);
      else
        hipLaunchKernelGGL(epi_z_kernel<float>, dim3(static_cast<unsigned>((nz + 255) / 256)),
                           dim3(256), 0, stream, part, fs, a.M, a.d, static_cast<float*>(z),
                           static_cast<const float*>(nullptr), static_cast<const float*>(nullptr),
                           a.dst.row_dst, sep ? pass + 1 : 0);
    }
    hipLaunchKernelGGL(gemm_f32_kernel, dim3((kv.N + 63) / 64, (kv.M + 31) / 32, ks), dim3(256),
                       0, stream, kv);
    const int64_t items = static_cast<int64_t>(a.M) * (n_kv / 2);
    hipLaunchKernelGGL(epi_kv_kernel<float>, dim3(static_cast<unsigned>((items + 255) / 256)),
                       dim3(256), 0, stream, part, ks, a.M, n_kv, a.dst);
    return hipGetLastError();
  }

  if (!sep && a.znorm == nullptr && a.dst.knorm == nullptr && p.fused &&
      (a.fe != nullptr || a.e == nullptr)) {
    hipLaunchKernelGGL(proj_fused_kernel, dim3((a.M + kFusedBM - 1) / kFusedBM), dim3(256), 0,
                       stream, a);
    return hipGetLastError();
  }
  if (a.fe != nullptr && !sep) {   // F(E) folded beforehand: the GEMM carries no E
    f.e = nullptr;
    f.fe = a.fe;
  }
  if (a.route != nullptr) {
    if (!route_foldable(a, p)) return hipErrorInvalidValue;   // the caller checks first
    f.route = *a.route;
    f.route_blocks = (a.route->S + 3) / 4;
  }
  f.k_per_split = split_len(a.Dcat, p.f_split, p.f_tile);
  f.mode = p.f_split > 1 ? kModePartial : kModeZ;
  for (int pass = 0; pass < passes; ++pass) {
    if (pass == 1) f.B = a.wfc;
    f.z_rows = sep ? pass + 1 : 0;
    if ((err = launch_gemm_bf16(f, p.f_tile, p.f_split, stream)) != hipSuccess) return err;
    if (p.f_split > 1 && a.znorm != nullptr) {   // normalised in the split epilogue
      hipLaunchKernelGGL(epi_z_norm_kernel<uint16_t>, dim3(a.M), dim3(256), 0, stream, part,
                         p.f_split, a.M, a.d, static_cast<uint16_t*>(z),
                         static_cast<const float*>(f.e ? f.partial_e : nullptr), f.fe,
                         a.dst.row_dst, f.z_rows, a.znorm);
    } else if (p.f_split > 1) {
      const int64_t nz = static_cast<int64_t>(a.M) * a.d / 4;
      hipLaunchKernelGGL(epi_z_kernel<uint16_t>, dim3(static_cast<unsigned>((nz + 255) / 256)),
                         dim3(256), 0, stream, part, p.f_split, a.M, a.d,
                         static_cast<uint16_t*>(z),
                         static_cast<const float*>(f.e ? f.partial_e : nullptr), f.fe,
                         a.dst.row_dst, f.z_rows);
    }
  }
  if (a.znorm != nullptr && p.f_split == 1)   // Z written whole by the GEMM: normalised in place
    hipLaunchKernelGGL(z_norm_kernel<uint16_t>, dim3(a.M), dim3(256), 0, stream,
                       static_cast<uint16_t*>(z), a.M, a.d, a.znorm);
  kv.k_per_split = split_len(a.d, p.kv_split, p.kv_tile);
  kv.mode = p.kv_split > 1 ? kModePartial : kModeKV;
  if ((err = launch_gemm_bf16(kv, p.kv_tile, p.kv_split, stream)) != hipSuccess) return err;
  if (p.kv_split > 1) {
    const int64_t items = static_cast<int64_t>(a.M) * (n_kv / 2);
    hipLaunchKernelGGL(epi_kv_kernel<uint16_t>, dim3(static_cast<unsigned>((items + 255) / 256)),
                       dim3(256), 0, stream, part, p.kv_split, a.M, n_kv, a.dst);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------- F(E) fold

// One wavefront per output: f_e[row] = sum_k wf[row][k] * e[k] in fp32, lanes
// striding over k in 8-element chunks, then a butterfly sum.
template <typename T>
__global__ __launch_bounds__(256) void fold_e_kernel(const T* wf, const T* e, int d, int Dcat,
                                                     float* out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= d) return;
  const T* w = wf + static_cast<int64_t>(row) * Dcat;
  float acc = 0.f;
  for (int k = lane * 8; k < Dcat; k += 512) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if constexpr (sizeof(T) == 2)
        acc = fmaf(bf2f(w[k + i]), bf2f(e[k + i]), acc);
      else
        acc = fmaf(w[k + i], e[k + i], acc);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) out[row] = acc;
}

hipError_t launch_fold_e(const void* wf, const void* e, int d, int Dcat, int dtype, float* out,
                         hipStream_t stream) {
  const dim3 grid((d + 3) / 4);
  if (dtype == CO_DTYPE_BF16)
    hipLaunchKernelGGL(fold_e_kernel<uint16_t>, grid, dim3(256), 0, stream,
                       static_cast<const uint16_t*>(wf), static_cast<const uint16_t*>(e), d, Dcat,
                       out);
  else
    hipLaunchKernelGGL(fold_e_kernel<float>, grid, dim3(256), 0, stream,
                       static_cast<const float*>(wf), static_cast<const float*>(e), d, Dcat, out);
  return hipGetLastError();
}

// ------------------------------------------------- plain products (backward)
//
// C[M][N] (fp32) = (accumulate ? C : 0) + A[M][K] . B[N][K]^T with bf16
// operands whose K is contiguous (K a multiple of 64), through the MFMA kernels
// above in K-split partial mode; the splits are summed in split order, so the
// result is deterministic.

namespace {

__global__ __launch_bounds__(256) void sum_splits_kernel(const float* part, int splits, int64_t n,
                                                         float* C, int accumulate) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  float v = accumulate ? C[i] : 0.f;
  int s = 0;
  for (; s + 8 <= splits; s += 8) {   // eight loads in flight, summed in split order
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = part[(s + k) * n + i];
#pragma unroll
    for (int k = 0; k < 8; ++k) v += x[k];
  }
  for (; s < splits; ++s) v += part[s * n + i];
  C[i] = v;
}

}  // namespace

size_t gemm_acc_ws_bytes(int M, int N, int K, int num_cus) {
  int tile, split;
  pick_gemm(M, N, K, false, 64, num_cus, &tile, &split);
  return (static_cast<size_t>(split) * M * N * 4 + 255) / 256 * 256;
}

hipError_t launch_gemm_acc(const void* A, const void* B, int M, int N, int K, float* C,
                           bool accumulate, float* part, int num_cus, hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  int tile, split;
  pick_gemm(M, N, K, false, 64, num_cus, &tile, &split);
  GemmArgs g{};
  g.M = M;
  g.N = N;
  g.K = K;
  g.A = A;
  g.B = B;
  g.mode = kModePartial;
  g.k_per_split = split_len(K, split, tile);
  const int splits = (K + g.k_per_split - 1) / g.k_per_split;
  // a single split that overwrites C writes it directly
  g.partial = (splits == 1 && !accumulate) ? C : part;
  hipError_t err = launch_gemm_bf16(g, tile, splits, stream);
  if (err != hipSuccess || g.partial == C) return err;
  const int64_t n = static_cast<int64_t>(M) * N;
  hipLaunchKernelGGL(sum_splits_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0,
                     stream, part, splits, n, C, accumulate ? 1 : 0);
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
