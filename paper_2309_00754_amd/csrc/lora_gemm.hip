// Dual-path LoRA GEMM for gfx950 (MI355X): one pass over the frozen base
// weight W produces both the LoRA-off output x W^T and the LoRA-on output
// x W^T + s (x A^T) B^T (Sec. 3, "Dynamic LoRA" and "Stage 2: Hydra-PPO":
// the reference / reward roles are the same network with LoRA ignored).
//
// Structure (one 128 x 256 output tile per 256-thread workgroup, one
// workgroup per CU):
//  * the x slab [128 x 64], the W slab [256 x 64] and the LoRA-down slab
//    A [RP x 64] of each 64-wide K slab are copied straight from HBM/L2 into
//    LDS (buffer_load ... lds, no register staging) two slabs ahead, through
//    a three-stage ring of XOR-swizzled 16-byte chunks;
//  * each of the 4 waves owns a 64 x 128 sub-tile and runs
//    v_mfma_f32_32x32x16_bf16 with W as the A operand and x as the B operand,
//    so that every lane ends up holding four consecutive output columns of
//    one row (float4 stores in the epilogue); the LDS reads of the next
//    k-step and the copies of a later slab are slotted between the MFMAs;
//  * the rank-r product T = x A^T of the tile's 128 rows is accumulated in the
//    same loop (v_mfma_f32_16x16x32_bf16, 32 rows per wave, so the work is
//    balanced) and never leaves the chip;
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
constexpr int MT = WM / 32;    // 32-row x tiles per wave
constexpr int NTL = WN / 32;   // 32-row W tiles per wave
constexpr int CPR = BK / 8;    // 16-byte chunks per LDS row
constexpr int GROUP_M = 8;     // row tiles walked together (L2 reuse of W)

static_assert(kScoreTileN == BN, "score partials assume one partial per GEMM column tile");

// LDS chunk index of (row, 16-byte chunk c): chunks are XOR-swizzled by the
// row so that the lanes reading one column of chunks hit distinct banks.
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
  int vec4;  // outputs may be written with 16-byte stores (N % 4 == 0, 16-byte aligned)
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
  // indices.
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
  const int l32 = lane & 31;
  const int lh = lane >> 5;

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
  const int nkt = (K + BK - 1) / BK;

  // The epilogue's global inputs are fetched now, so that they have arrived
  // long before the main loop ends: the tile's rows of B (thread t holds row
  // n0 + t, zero padded to RP; rows past N read as zeros through the buffer
  // resource) and, for SCORE, the sampled token of row m0 + t.
  constexpr bool B_EARLY = RP > 0 && RP <= 32;
  uint32_t breg[B_EARLY ? RP : 1];
  const bool want_on = SCORE || a.y_on != nullptr;
  if constexpr (B_EARLY) {
    const __amdgpu_buffer_rsrc_t brs = make_rsrc(a.B + (size_t)n0 * a.r, (uint32_t)min(BN, N - n0) * a.r * 2u);
#pragma unroll
    for (int j = 0; j < RP; ++j) {
      const bool ok = want_on && j < a.r;
      const uint32_t v = __builtin_amdgcn_raw_buffer_load_b16(brs, ok ? (t * a.r + j) * 2 : kOutOfRange, 0, 0);
      breg[j] = ok ? v : 0u;
    }
  }
  int tok_early = -1;
  if constexpr (SCORE) {
    if (t < BM) {
      const int row = m0 + t;
      const int v = g.tokens[row < M ? row : 0];
      tok_early = row < M ? v : -1;
    }
  }

  f32x16_t acc[MT][NTL];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NTL; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  constexpr int TJ = RP / 16;
  constexpr int TJ1 = TJ > 0 ? TJ : 1;
  f32x4_t accT[2][TJ1];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int j = 0; j < TJ1; ++j) accT[q][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Register fragments of one 32-wide k-step: for each 16-wide half h, the W
  // rows (A operand) and x rows (B operand) of the 32x32x16 MFMAs; the x rows
  // of this wave's 32 T rows and the LoRA-down rows in the 16x16x32 layout.
  // Two sets alternate so that the next k-step's LDS reads overlap the
  // current k-step's MFMAs.
  struct Frag {
    uint4 w[2][NTL];
    uint4 x[2][MT];
    uint4 tx[2];
    uint4 a[TJ1];
  };
  Frag F0, F1;
  constexpr int NMAIN = 2 * MT * NTL;          // 32x32x16 MFMAs per k-step
  constexpr int NR = 2 * NTL + 2 * MT + (TJ > 0 ? 2 + TJ : 0);  // LDS reads per k-step
  constexpr int ND = XI + WI + AIW;           // copy instructions per wave per slab (at most)
  static_assert(ND <= NMAIN, "one copy slot per MFMA");

  auto read_one = [&](Frag& F, const uint4* s, int kk, int r) __attribute__((always_inline)) {
    if (r < 2 * NTL) {
      const int h = r / NTL, ni = r % NTL;
      F.w[h][ni] = s[L::WOFF + lds_idx(wc * WN + ni * 32 + l32, kk * 4 + 2 * h + lh)];
    } else if (r < 2 * NTL + 2 * MT) {
      const int h = (r - 2 * NTL) / MT, mi = (r - 2 * NTL) % MT;
      F.x[h][mi] = s[L::XOFF + lds_idx(wr * WM + mi * 32 + l32, kk * 4 + 2 * h + lh)];
    } else if (r < 2 * NTL + 2 * MT + 2) {
      const int q = r - 2 * NTL - 2 * MT;
      F.tx[q] = s[L::XOFF + lds_idx(wr * WM + (wc * 2 + q) * 16 + l16, kk * 4 + lg)];
    } else {
      const int j = r - 2 * NTL - 2 * MT - 2;
      F.a[j] = s[L::AOFF + lds_idx(j * 16 + l16, kk * 4 + lg)];
    }
  };
  auto dma_one = [&](uint4* st, int kofs, bool kv, int d) __attribute__((always_inline)) {
    if (d < XI) {
      const int ci = wave * XI + d;
      dma16(xr, st + L::XOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kofs : kOutOfRange);
    } else if (d < XI + WI) {
      const int ci = wave * WI + (d - XI);
      dma16(wrs, st + L::WOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kofs : kOutOfRange);
    } else {
      const int ci = wave + 4 * (d - XI - WI);
      if (ci < AI) dma16(arsrc, st + L::AOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kofs : kOutOfRange);
    }
  };
  auto issue_all = [&](uint4* st, int kt) __attribute__((always_inline)) {
    const int k0 = kt * BK;
#pragma unroll
    for (int d = 0; d < ND; ++d) dma_one(st, k0 * 2 + c * 16, k0 + c * 8 < K, d);
  };

  // Copy instructions [d0, d1) of a slab go out in one k-step, the rest in
  // the other, so that no k-step stalls on a burst of copies.
  constexpr int DA = (ND + 1) / 2;  // copies issued in k-step 0

  // One k-step: the NMAIN MFMAs of the wave tile on Fc (then the LoRA-down
  // MFMAs), with one LDS read that fills Fn and one copy of a later slab
  // slotted after each MFMA.  The scheduling barriers keep that order.
  auto kstep = [&](const Frag& Fc, Frag& Fn, const uint4* rs, int rkk, uint4* dst, int dkt, int d0, int d1)
      __attribute__((always_inline)) {
    const bool do_dma = d1 > d0;
    const int k0 = dkt * BK;
    const bool kv = dkt < nkt && k0 + c * 8 < K;
    const int kofs = k0 * 2 + c * 16;
#pragma unroll
    for (int m = 0; m < NMAIN; ++m) {
      const int h = m / (MT * NTL), mi = (m / NTL) % MT, ni = m % NTL;
      acc[mi][ni] = mfma32(Fc.w[h][ni], Fc.x[h][mi], acc[mi][ni]);
      if (m < NR) read_one(Fn, rs, rkk, m);
      if (do_dma && m >= d0 && m < d1) dma_one(dst, kofs, kv, m);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (TJ > 0) {
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        accT[0][j] = mfma16(Fc.tx[0], Fc.a[j], accT[0][j]);
        accT[1][j] = mfma16(Fc.tx[1], Fc.a[j], accT[1][j]);
      }
    }
#pragma unroll
    for (int r = NMAIN; r < NR; ++r) read_one(Fn, rs, rkk, r);
    __builtin_amdgcn_sched_barrier(0);
  };

  // ---- pipeline.  Slab kt lives in stage kt % NS.  Each iteration:
  //   k-step 0 of slab kt (MFMAs on F0) while F1 <- k-step 1 of slab kt and
  //     the first copies of slab kt + NS - 1 go into the stage freed one
  //     iteration ago;
  //   wait for slab kt + 1, barrier (stage kt is retired, kt + 1 visible);
  //   k-step 1 of slab kt (MFMAs on F1) while F0 <- k-step 0 of slab kt + 1
  //     and the remaining copies go out.
  // With NS = 3, at the barrier only the first part of slab kt + 2 (DAW per
  // wave at least) may still be in flight; with NS = 2 all copies of slab
  // kt + 1 go out in k-step 0 and are waited for at the barrier.  Past the
  // last slab the copies get out-of-range offsets (they write zeros into a
  // stage that is not read again) and the last iteration's reads fill
  // registers that are not used, so every iteration is the same straight-line
  // code.
  constexpr int DAW = NS == 3 ? (DA < XI + WI ? DA : XI + WI) : 0;
  auto iter = [&](const uint4* cur, uint4* dst, const uint4* nxt, int kt) __attribute__((always_inline)) {
    if constexpr (NS == 3) {
      kstep(F0, F1, cur, 1, dst, kt + 2, 0, DA);
      wait_vm_barrier<DAW>();
      kstep(F1, F0, nxt, 0, dst, kt + 2, DA, ND);
    } else {
      kstep(F0, F1, cur, 1, dst, kt + 1, 0, ND);
      wait_vm_barrier<0>();
      kstep(F1, F0, nxt, 0, nullptr, 0, 0, 0);
    }
  };
  issue_all(sm0, 0);
  if constexpr (NS == 3) {
    if (nkt > 1) {
      issue_all(sm1, 1);
      wait_vm_barrier<DPW>();
    } else {
      wait_vm_barrier<0>();
    }
  } else {
    wait_vm_barrier<0>();
  }
#pragma unroll
  for (int r = 0; r < NR; ++r) read_one(F0, sm0, 0, r);
  if constexpr (NS == 3) {
    for (int kt = 0; kt < nkt; kt += 3) {
      iter(sm0, sm2, sm1, kt);
      if (kt + 1 < nkt) iter(sm1, sm0, sm2, kt + 1);
      if (kt + 2 < nkt) iter(sm2, sm1, sm0, kt + 2);
    }
  } else {
    for (int kt = 0; kt < nkt; kt += 2) {
      iter(sm0, sm1, sm1, kt);
      if (kt + 1 < nkt) iter(sm1, sm0, sm0, kt + 1);
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

  if constexpr (TJ > 0) {
    if (want_on) {
      const float sc = a.s;
      // accT[q][j] holds T[wr*64 + (wc*2+q)*16 + 4 lg + e][16 j + l16]
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int row = wr * WM + (wc * 2 + q) * 16 + lg * 4 + e;
            const int col = j * 16 + l16;
            const float v = sc * accT[q][j][e];
            const uint32_t hi = f32_to_bf16_rne(v);
            const uint32_t lo = f32_to_bf16_rne(v - bf16_to_f32(hi));
            Ts[row * 2 * RP + col] = (uint16_t)hi;
            Ts[row * 2 * RP + RP + col] = (uint16_t)lo;
          }
      if constexpr (B_EARLY) {
        static_assert(BN == NT, "one B row per thread");
#pragma unroll
        for (int j = 0; j < RP; j += 2) *reinterpret_cast<uint32_t*>(Bs + t * RP + j) = breg[j] | (breg[j + 1] << 16);
      } else {
        // large ranks: all loads of the thread are issued before any store
        uint16_t v[RP];
#pragma unroll
        for (int i = 0; i < RP; ++i) {
          const int e = t + i * NT;
          const int n = e / RP, j = e % RP;
          const bool ok = n0 + n < N && j < a.r;
          const uint16_t u = a.B[ok ? (size_t)(n0 + n) * a.r + j : 0];
          v[i] = ok ? u : (uint16_t)0;
        }
#pragma unroll
        for (int i = 0; i < RP; ++i) Bs[t + i * NT] = v[i];
      }
    }
  }
  if constexpr (SCORE) {
    if (t < BM) tok[t] = tok_early;
  }
  __syncthreads();

  // s*T*B^T added by 32x32x16 MFMAs: A operand = rows of [B | B] (k < RP picks
  // B against the hi part, k >= RP against the lo part), B operand = rows of
  // Ts ([hi | lo] along k).
  auto apply_lora = [&]() __attribute__((always_inline)) {
    if constexpr (TJ > 0) {
#pragma unroll
      for (int ks = 0; ks < (2 * RP) / 16; ++ks) {
        const int kofs = ks * 16 + lh * 8;   // k within [0, 2 RP)
        const int kb = kofs % RP;            // matching column of B
        uint4 bfr[NTL], tf[MT];
#pragma unroll
        for (int ni = 0; ni < NTL; ++ni)
          bfr[ni] = *reinterpret_cast<const uint4*>(Bs + (wc * WN + ni * 32 + l32) * RP + kb);
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
          tf[mi] = *reinterpret_cast<const uint4*>(Ts + (wr * WM + mi * 32 + l32) * 2 * RP + kofs);
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
#pragma unroll
          for (int ni = 0; ni < NTL; ++ni) acc[mi][ni] = mfma32(bfr[ni], tf[mi], acc[mi][ni]);
      }
    }
  };

  // acc[mi][ni][4 i + e] holds y[wr*64 + mi*32 + l32][wc*128 + ni*32 + 8 i + 4 lh + e]
  if constexpr (!SCORE) {
    auto store = [&](float* y) __attribute__((always_inline)) {
#pragma unroll
      for (int mi = 0; mi < MT; ++mi) {
        const int row = m0 + wr * WM + mi * 32 + l32;
        if (row >= M) continue;
        float* yr = y + (size_t)row * N;
#pragma unroll
        for (int ni = 0; ni < NTL; ++ni)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int col = n0 + wc * WN + ni * 32 + 8 * i + 4 * lh;
            const f32x16_t& v = acc[mi][ni];
            if (g.vec4 && col + 3 < N) {
              *reinterpret_cast<float4*>(yr + col) = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (col + e < N) yr[col + e] = v[4 * i + e];
            }
          }
      }
    };
    if (a.y_off) store(a.y_off);
    if (a.y_on) {
      apply_lora();
      store(a.y_on);
    }
  } else {
    // Per-row (max, sum exp) over this wave's 128 columns (64 per lane, then
    // the lane pair l, l + 32), then over the two waves sharing the rows.
    // Identical code for the off and on passes.
    auto row_stats = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
      for (int mi = 0; mi < MT; ++mi) {
        const int rlc = wr * WM + mi * 32 + l32;
        const int tk = tok[rlc];
        float mx = -INFINITY;
#pragma unroll
        for (int ni = 0; ni < NTL; ++ni)
#pragma unroll
          for (int k = 0; k < 16; ++k) {
            const int col = n0 + wc * WN + ni * 32 + 8 * (k >> 2) + 4 * lh + (k & 3);
            if (col < N) mx = fmaxf(mx, acc[mi][ni][k]);
            // the lane holding the sampled token's column records its logit
            if (col == tk) g.zt[(size_t)(m0 + rlc) * 2 + (slot >> 1)] = acc[mi][ni][k];
          }
        float sm = 0.f;
        if (mx != -INFINITY) {
#pragma unroll
          for (int ni = 0; ni < NTL; ++ni)
#pragma unroll
            for (int k = 0; k < 16; ++k) {
              const int col = n0 + wc * WN + ni * 32 + 8 * (k >> 2) + 4 * lh + (k & 3);
              if (col < N) sm += exp_e(acc[mi][ni][k] - mx);
            }
        }
        const float mo = __shfl_xor(mx, 32);
        const float so = __shfl_xor(sm, 32);
        lse_merge(mx, sm, mo, so);
        if (lh == 0) {
          red[(wc * BM + rlc) * 4 + slot] = mx;
          red[(wc * BM + rlc) * 4 + slot + 1] = sm;
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

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

hipError_t launch_lora_gemm(const LinearArgs& a, hipStream_t stream) {
  GemmArgs g{};
  g.lin = a;
  g.ntm = (a.M + BM - 1) / BM;
  g.ntn = (a.N + BN - 1) / BN;
  g.vec4 = (a.N % 4 == 0) && (!a.y_off || aligned16(a.y_off)) && (!a.y_on || aligned16(a.y_on));
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
