// Dual-path LoRA GEMM for gfx950 (MI355X): one pass over the frozen base
// weight W produces both the LoRA-off output x W^T and the LoRA-on output
// x W^T + s (x A^T) B^T (Sec. 3, "Dynamic LoRA" and "Stage 2: Hydra-PPO":
// the reference / reward roles are the same network with LoRA ignored).
//
// Structure (one 128 x 256 output tile per 256-thread workgroup):
//  * main loop over K in 64-wide slabs: the x slab [128 x 64], the W slab
//    [256 x 64] and the LoRA-down slab A [RP x 64] are staged through LDS
//    (double buffered, XOR-swizzled 16-byte chunks) and consumed by
//    v_mfma_f32_16x16x32_bf16; each of the 4 waves owns a 64 x 128 sub-tile;
//  * the rank-r product T = x A^T of the tile's 128 rows is accumulated in the
//    same loop from the x fragments already in registers (each wave owns 32
//    of the rows, so the work is balanced), and never leaves the chip;
//  * epilogue: the accumulators are the LoRA-off result.  s*T is split into
//    bf16 hi + lo parts and multiplied against [B; B] by MFMA, adding the
//    LoRA update to the same accumulators, which become the LoRA-on result.
//    With B = 0 or s = 0 the update adds exact zeros, so y_on == y_off.
//  * SCORE variant (CLM head, N = V): instead of storing logits, each row's
//    (max, sum exp) over the tile's 256 columns is reduced for both passes,
//    the sampled token's logit is picked up by the lane that holds it, and a
//    float4 partial per (row, column tile) is written for the combine kernel.
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

constexpr int BM = 128;        // tile rows (tokens)
constexpr int BN = 256;        // tile columns (outputs)
constexpr int BK = 64;         // K slab
constexpr int NT = 256;        // threads per workgroup (4 waves)
constexpr int WM = 64;         // wave tile rows
constexpr int WN = 128;        // wave tile columns
constexpr int TM = WM / 16;    // MFMA tiles per wave, rows
constexpr int TN = WN / 16;    // MFMA tiles per wave, columns
constexpr int CPR = BK / 8;    // 16-byte chunks per LDS row
constexpr int GROUP_M = 8;     // row tiles walked together (L2 reuse of W)

static_assert(kScoreTileN == BN, "score partials assume one partial per GEMM column tile");

// LDS chunk index of (row, 16-byte chunk c): chunks are XOR-swizzled by the
// row so that the 16 lanes reading one column of chunks hit distinct banks.
__device__ __forceinline__ int lds_idx(int row, int c) { return row * CPR + (c ^ (row & 7)); }

template <int RP>
struct Layout {
  static constexpr int XOFF = 0;
  static constexpr int WOFF = BM * CPR;
  static constexpr int AOFF = (BM + BN) * CPR;
  static constexpr int STAGE = (BM + BN + RP) * CPR;  // uint4 per stage
  // three stages when they fit in the 160 KB of LDS, else two
  static constexpr int NSTAGES = 3 * STAGE * 16 <= 160 * 1024 ? 3 : 2;
  static_assert(BM * 2 * RP * 2 <= STAGE * 16, "Ts must fit in one stage");
  static_assert(BN * RP * 2 + (2 * BM * 4 + BM) * 4 <= STAGE * 16, "Bs, red and tok must fit in one stage");
};

struct GemmArgs {
  LinearArgs lin;
  const int32_t* tokens;
  float4* part;
  float* zt;
  int ntm, ntn;
};

// Workgroup id -> (row tile, column tile).  Consecutive workgroup ids are
// dispatched to consecutive XCDs; when the tile count allows, each XCD gets a
// contiguous range of the logical order, and the logical order walks GROUP_M
// row tiles per column tile so that the tiles sharing a W slab run together.
__device__ __forceinline__ void tile_of(int bid, int ntm, int ntn, int& tm, int& tn) {
  const int total = ntm * ntn;
  int lid = bid;
  if ((total & 7) == 0) lid = (bid & 7) * (total >> 3) + (bid >> 3);
  const int per_group = GROUP_M * ntn;
  const int group = lid / per_group;
  const int first_m = group * GROUP_M;
  const int gsize = min(ntm - first_m, GROUP_M);
  const int in = lid - group * per_group;
  tm = first_m + in % gsize;
  tn = in / gsize;
}

template <int RP, bool SCORE>
__global__ __launch_bounds__(NT, 1) void lora_gemm_kernel(GemmArgs g) {
  using L = Layout<RP>;
  constexpr int NS = L::NSTAGES;
  // One array per pipeline stage, always addressed with compile-time stage
  // indices, so that the compiler's own waits for the LDS copies stay exact.
  __shared__ uint4 sm0[L::STAGE];
  __shared__ uint4 sm1[L::STAGE];
  __shared__ uint4 sm2[NS == 3 ? L::STAGE : 1];

  const LinearArgs& a = g.lin;
  const int M = a.M, N = a.N, K = a.K;
  const int t = threadIdx.x;
  const int lane = t & 63;
  // The wave index is made provably wave-uniform (an SGPR), so branches on it
  // are scalar branches: MFMAs must never sit under exec-masked divergence.
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wr = wave >> 1;  // wave row (0..1)
  const int wc = wave & 1;   // wave column (0..1)
  const int l16 = lane & 15;
  const int lg = lane >> 4;

  int tmi, tni;
  tile_of(blockIdx.x, g.ntm, g.ntn, tmi, tni);
  const int m0 = tmi * BM;
  const int n0 = tni * BN;

  // ---- global -> LDS copies.  One copy instruction moves 8 rows x 128 bytes
  // (64 lanes x 16 bytes) into 1 KB of LDS; lane i fills LDS chunk i of it,
  // so it fetches the global chunk that the swizzle maps there.  Buffer
  // resources cover exactly the tile's valid rows (rows past M, N or r read
  // as zeros); a chunk past K gets an out-of-range offset (zeros as well).
  const i32x4_t xr = make_rsrc_raw(a.x + (size_t)m0 * K, (uint32_t)min(BM, M - m0) * K * 2u);
  const i32x4_t wrs = make_rsrc_raw(a.W + (size_t)n0 * K, (uint32_t)min(BN, N - n0) * K * 2u);
  const i32x4_t arsrc = make_rsrc_raw(a.A, (uint32_t)min(a.r, RP) * K * 2u);
  const int row_bytes = K * 2;
  const int c = (lane & 7) ^ (lane >> 3);   // global chunk fetched by this lane
  const int rl = lane >> 3;                 // row within the 8-row copy
  constexpr int XI = BM / 8 / 4;            // copies per wave: x
  constexpr int WI = BN / 8 / 4;            //                  W
  constexpr int AI = RP / 8;                // copies in total: A
  constexpr int AIW = (AI + 3) / 4;         // most A copies one wave issues
  constexpr int DPW = XI + WI + AI / 4;     // fewest copies any wave issues per slab

  auto issue = [&](uint4* st, int kt) __attribute__((always_inline)) {
    const int k0 = kt * BK;
    const bool kv = k0 + c * 8 < K;
    const int kb = k0 * 2 + c * 16;
#pragma unroll
    for (int j = 0; j < XI; ++j) {
      const int ci = wave * XI + j;
      dma16(xr, st + L::XOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kb : kOutOfRange);
    }
#pragma unroll
    for (int j = 0; j < WI; ++j) {
      const int ci = wave * WI + j;
      dma16(wrs, st + L::WOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kb : kOutOfRange);
    }
#pragma unroll
    for (int j = 0; j < AIW; ++j) {
      const int ci = wave + 4 * j;
      if (ci < AI) dma16(arsrc, st + L::AOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kb : kOutOfRange);
    }
  };

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  constexpr int TJ = RP / 16;
  f32x4_t accT[2][TJ > 0 ? TJ : 1];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int j = 0; j < (TJ > 0 ? TJ : 1); ++j) accT[q][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const uint4* s) __attribute__((always_inline)) {
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      const int cc = kk * 4 + lg;
      uint4 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = s[L::XOFF + lds_idx(wr * WM + i * 16 + l16, cc)];
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = s[L::WOFF + lds_idx(wc * WN + j * 16 + l16, cc)];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(af[i], bfr[j], acc[i][j]);
      if constexpr (TJ > 0) {
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
          const uint4 alo = s[L::AOFF + lds_idx(j * 16 + l16, cc)];
          if (wc == 0) {
            accT[0][j] = mfma16(af[0], alo, accT[0][j]);
            accT[1][j] = mfma16(af[1], alo, accT[1][j]);
          } else {
            accT[0][j] = mfma16(af[2], alo, accT[0][j]);
            accT[1][j] = mfma16(af[3], alo, accT[1][j]);
          }
        }
      }
    }
  };

  // ---- pipeline: slab kt lives in stage kt % NS; slabs kt+1 .. kt+NS-2 are
  // in flight while slab kt is multiplied.  At the top of each step, the
  // wait leaves only the later slabs' copies outstanding, and the barrier
  // makes every wave's part of slab kt visible and retires the stage read in
  // the previous step, which is then refilled with slab kt + NS - 1.
  const int nkt = (K + BK - 1) / BK;
  auto step = [&](const uint4* cur, uint4* nxt, int kt) __attribute__((always_inline)) {
    if (kt + 1 < nkt) wait_vm_barrier<DPW * (NS - 2)>();
    else wait_vm_barrier<0>();
    if (kt + NS - 1 < nkt) issue(nxt, kt + NS - 1);
    compute(cur);
  };
  issue(sm0, 0);
  if constexpr (NS == 3) {
    if (nkt > 1) issue(sm1, 1);
    for (int kt = 0; kt < nkt; kt += 3) {
      step(sm0, sm2, kt);
      if (kt + 1 < nkt) step(sm1, sm0, kt + 1);
      if (kt + 2 < nkt) step(sm2, sm1, kt + 2);
    }
  } else {
    for (int kt = 0; kt < nkt; kt += 2) {
      step(sm0, sm1, kt);
      if (kt + 1 < nkt) step(sm1, sm0, kt + 1);
    }
  }
  wait_vm_barrier<0>();  // every wave is done with the stages before the epilogue reuses them

  // ---------------------------------------------------------------- epilogue
  // The stages are free again.  Layout:
  //   stage 0: Ts [BM][2 RP] bf16, s*T split into hi (columns 0..RP) and lo (RP..2RP)
  //   stage 1: Bs [BN][RP] bf16, the tile's rows of B zero padded to RP;
  //            SCORE only: red [2][BM][4] fp32 and tok [BM] int32 after it.
  uint16_t* Ts = reinterpret_cast<uint16_t*>(sm0);
  uint16_t* Bs = reinterpret_cast<uint16_t*>(sm1);
  float* red = reinterpret_cast<float*>(Bs + BN * RP);
  int* tok = reinterpret_cast<int*>(red + 2 * BM * 4);

  const bool want_on = SCORE || a.y_on != nullptr;
  if constexpr (TJ > 0) {
    if (want_on) {
      const float sc = a.s;
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = wr * WM + (wc * 2 + q) * 16 + lg * 4 + i;
            const int col = j * 16 + l16;
            const float v = sc * accT[q][j][i];
            const uint32_t hi = f32_to_bf16_rne(v);
            const uint32_t lo = f32_to_bf16_rne(v - bf16_to_f32(hi));
            Ts[row * 2 * RP + col] = (uint16_t)hi;
            Ts[row * 2 * RP + RP + col] = (uint16_t)lo;
          }
      for (int e = t; e < BN * RP; e += NT) {
        const int n = e / RP, j = e - (e / RP) * RP;
        const int gn = n0 + n;
        const bool ok = gn < N && j < a.r;
        const uint16_t v = a.B[ok ? (size_t)gn * a.r + j : 0];
        Bs[e] = ok ? v : (uint16_t)0;
      }
    }
  }
  if constexpr (SCORE) {
    for (int e = t; e < BM; e += NT) {
      const int row = m0 + e;
      const int v = g.tokens[row < M ? row : 0];
      tok[e] = row < M ? v : -1;
    }
  }
  __syncthreads();

  // s*T*B^T added by MFMA: A operand = [hi | lo] rows of Ts, B operand = [B; B].
  auto apply_lora = [&]() __attribute__((always_inline)) {
    if constexpr (TJ > 0) {
#pragma unroll
      for (int ks = 0; ks < (2 * RP) / 32; ++ks) {
        const int kofs = ks * 32 + lg * 8;   // k within [0, 2 RP)
        const int kb = kofs % RP;            // matching column of B
        uint4 tf[TM], bfr[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          tf[i] = *reinterpret_cast<const uint4*>(Ts + (wr * WM + i * 16 + l16) * 2 * RP + kofs);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[j] = *reinterpret_cast<const uint4*>(Bs + (wc * WN + j * 16 + l16) * RP + kb);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(tf[i], bfr[j], acc[i][j]);
      }
    }
  };

  if constexpr (!SCORE) {
    auto store = [&](float* y) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = n0 + wc * WN + j * 16 + l16;
          if (col >= N) continue;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = m0 + wr * WM + i * 16 + lg * 4 + e;
            if (row < M) y[(size_t)row * N + col] = acc[i][j][e];
          }
        }
    };
    if (a.y_off) store(a.y_off);
    if (a.y_on) {
      apply_lora();
      store(a.y_on);
    }
  } else {
    // Per-row (max, sum exp) over this wave's 128 columns, then over the two
    // waves sharing the rows.  Identical code for the off and on passes.
    auto row_stats = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rl = wr * WM + i * 16 + lg * 4 + e;
          const int tk = tok[rl];
          float mx = -INFINITY;
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int col = n0 + wc * WN + j * 16 + l16;
            if (col < N) mx = fmaxf(mx, acc[i][j][e]);
            // the lane holding the sampled token's column records its logit
            if (col == tk) g.zt[(size_t)(m0 + rl) * 2 + (slot >> 1)] = acc[i][j][e];
          }
          float sm = 0.f;
          if (mx != -INFINITY) {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              const int col = n0 + wc * WN + j * 16 + l16;
              if (col < N) sm += exp_e(acc[i][j][e] - mx);
            }
          }
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) {
            const float mo = __shfl_xor(mx, off);
            const float so = __shfl_xor(sm, off);
            lse_merge(mx, sm, mo, so);
          }
          if (l16 == 0) {
            red[(wc * BM + rl) * 4 + slot] = mx;
            red[(wc * BM + rl) * 4 + slot + 1] = sm;
          }
        }
    };
    row_stats(0);     // LoRA off
    apply_lora();
    row_stats(2);     // LoRA on
    __syncthreads();
    for (int e = t; e < BM; e += NT) {
      const int row = m0 + e;
      if (row >= M) continue;
      float mo = red[e * 4 + 0], so = red[e * 4 + 1];
      float mn = red[e * 4 + 2], sn = red[e * 4 + 3];
      lse_merge(mo, so, red[(BM + e) * 4 + 0], red[(BM + e) * 4 + 1]);
      lse_merge(mn, sn, red[(BM + e) * 4 + 2], red[(BM + e) * 4 + 3]);
      g.part[(size_t)row * g.ntn + tni] = make_float4(mo, so, mn, sn);
    }
  }
}

template <bool SCORE>
hipError_t launch(const GemmArgs& g, int rp, hipStream_t stream) {
  const dim3 grid(g.ntm * g.ntn), block(NT);
  switch (rp) {
    case 0: hipLaunchKernelGGL((lora_gemm_kernel<0, SCORE>), grid, block, 0, stream, g); break;
    case 16: hipLaunchKernelGGL((lora_gemm_kernel<16, SCORE>), grid, block, 0, stream, g); break;
    case 32: hipLaunchKernelGGL((lora_gemm_kernel<32, SCORE>), grid, block, 0, stream, g); break;
    case 64: hipLaunchKernelGGL((lora_gemm_kernel<64, SCORE>), grid, block, 0, stream, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int padded_rank(int r) { return r == 0 ? 0 : r <= 16 ? 16 : r <= 32 ? 32 : 64; }

}  // namespace

hipError_t launch_lora_gemm(const LinearArgs& a, hipStream_t stream) {
  GemmArgs g{};
  g.lin = a;
  g.ntm = (a.M + BM - 1) / BM;
  g.ntn = (a.N + BN - 1) / BN;
  const int rp = a.y_on ? padded_rank(a.r) : 0;
  return launch<false>(g, rp, stream);
}

hipError_t launch_score_gemm(const ScoreGemmArgs& s, hipStream_t stream) {
  GemmArgs g{};
  g.lin = s.lin;
  g.lin.y_off = nullptr;
  g.lin.y_on = nullptr;
  g.tokens = s.tokens;
  g.part = s.part;
  g.zt = s.zt;
  g.ntm = (s.lin.M + BM - 1) / BM;
  g.ntn = s.ntn;
  return launch<true>(g, padded_rank(s.lin.r), stream);
}

}  // namespace hydra
