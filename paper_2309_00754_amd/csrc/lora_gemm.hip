// Dual-path LoRA GEMM for gfx950 (MI355X): one pass over the frozen base
// weight W produces both the LoRA-off output x W^T and the LoRA-on output
// x W^T + s (x A^T) B^T (Sec. 3, "Dynamic LoRA" and "Stage 2: Hydra-PPO":
// the reference / reward roles are the same network with LoRA ignored).
//
// Structure (one 128 x 256 output tile per 512-thread workgroup, one
// workgroup per CU, two waves per SIMD):
//  * waves 4..7 are copy waves: they move the x slab [128 x 64], the W slab
//    [256 x 64] and the LoRA-down slab A [RP x 64] of each 64-wide K slab
//    straight from HBM/L2 into LDS (buffer_load ... lds, no register
//    staging), up to two slabs ahead, through a three-stage ring of
//    XOR-swizzled 16-byte chunks.  Vector-memory instructions issued by a
//    wave that also feeds the matrix cores stall its MFMA stream; with the
//    copies on their own waves the MFMA waves issue nothing but LDS reads
//    and MFMAs in the main loop;
//  * waves 0..3 each own a 64 x 128 sub-tile and run
//    v_mfma_f32_32x32x16_bf16 with W as the A operand and x as the B operand,
//    so that every lane ends up holding four consecutive output columns of
//    one row (float4 stores in the epilogue); the LDS reads of the next
//    16-wide k-step are slotted between the MFMAs of the current one;
//  * one workgroup barrier per slab hands the ring over: before it the copy
//    waves have waited for their copies of slab kt + 1 and the MFMA waves
//    have finished reading slab kt, after it the stage of slab kt is refilled
//    with slab kt + 3;
//  * the rank-r product T = x A^T of the tile's 128 rows is accumulated in the
//    same loop (v_mfma_f32_16x16x32_bf16, 32 rows per MFMA wave) and never
//    leaves the chip;
//  * epilogue: the accumulators are the LoRA-off result.  s*T is split into
//    bf16 hi + lo parts and multiplied against [B; B] by MFMA, adding the
//    LoRA update to the same accumulators, which become the LoRA-on result.
//    With B = 0 or s = 0 the update adds exact zeros, so y_on == y_off.  The
//    copy waves fetch the tile's rows of B at kernel start and stage them in
//    LDS for the epilogue.
#include <type_traits>

#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

constexpr int BM = 128;        // tile rows (tokens)
constexpr int BN = 256;        // tile columns (outputs)
constexpr int BK = 64;         // K slab
constexpr int NTM = 256;       // MFMA threads (waves 0..3)
constexpr int NT = 512;        // threads per workgroup (4 MFMA + 4 copy waves)
static_assert(BM == kGemmTileM && BN == kGemmTileN && NT == kGemmThreads, "launch shape known to the host checks");
constexpr int WM = 64;         // wave tile rows
constexpr int WN = 128;        // wave tile columns
constexpr int MT = WM / 32;    // 32-row x tiles per wave
constexpr int NTL = WN / 32;   // 32-row W tiles per wave
constexpr int CPR = BK / 8;    // 16-byte chunks per LDS row
constexpr int GROUP_M = 8;     // row tiles walked together (L2 reuse of W)

// LDS chunk index of (row, 16-byte chunk c): rows of 128 bytes, the chunk is
// XOR-ed with (row / 2) % 8, so that the 16 lanes of one read phase (16
// consecutive rows, one chunk: 8 even and 8 odd rows, each set covering the
// 8 chunk positions once) hit all 64 banks exactly once.
__device__ __forceinline__ int lds_idx(int row, int c) { return row * CPR + (c ^ ((row >> 1) & 7)); }

template <int RP>
struct Layout {
  static constexpr int XOFF = 0;
  static constexpr int WOFF = BM * CPR;
  static constexpr int AOFF = (BM + BN) * CPR;
  static constexpr int STAGE = (BM + BN + RP) * CPR;  // uint4 per stage
  // three stages when they fit in the 160 KB of LDS, else two
  static constexpr int NSTAGES = 3 * STAGE * 16 <= 160 * 1024 ? 3 : 2;
  static_assert(BM * 2 * RP * 2 <= STAGE * 16, "Ts must fit in one stage");
  static_assert(BN * RP * 2 <= STAGE * 16, "Bs must fit in one stage");
};

struct GemmArgs {
  LinearArgs lin;
  int ntm, ntn;
  int vec4;  // outputs may be written with 16-byte stores (N % 4 == 0, 16-byte aligned)
  // LoRA update from a pre-pass (TPRE kernels): ts [M x 2 RP] bf16 hi | lo parts
  // of s x A^T, bp [N x RP] bf16 B zero padded; nls extra slabs (0: no update)
  const uint16_t* ts;
  const uint16_t* bp;
  int nls;
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

// s_waitcnt with only the vector-memory counter (N outstanding at most).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0xF << 8) | (((N >> 4) & 3) << 14));
  asm volatile("" ::: "memory");
}

// LDS operations of this wave complete, then the workgroup barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt / expcnt untouched
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int V>
using IC = std::integral_constant<int, V>;

// RP: padded rank.  TPRE: the LoRA update comes from the pre-pass in the
// workspace and runs as g.nls extra slabs of the ring after the LoRA-off
// result has been stored; otherwise T is accumulated in the main loop and the
// update is applied in the epilogue.
template <int RP, bool TPRE>
__global__ __launch_bounds__(NT, 1) void lora_gemm_kernel(GemmArgs g) {
  constexpr int RA = TPRE ? 0 : RP;  // rows of A in every ring stage
  using L = Layout<RA>;
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
  const int wr = (wave >> 1) & 1;  // MFMA wave row (0..1)
  const int wc = wave & 1;         // MFMA wave column (0..1)
  const int l16 = lane & 15;
  const int lg = lane >> 4;
  const int l32 = lane & 31;
  const int lh = lane >> 5;

  int tmi, tni;
  tile_of(blockIdx.x, g.ntm, g.ntn, tmi, tni);
  const int m0 = tmi * BM;
  const int n0 = tni * BN;
  const int nkt = (K + BK - 1) / BK;
  const bool want_on = a.y_on != nullptr;

  constexpr int TJ = RA / 16;
  constexpr int TJ1 = TJ > 0 ? TJ : 1;
  constexpr int RP2 = RA > 0 ? RA / 2 : 1;
  const int nls = TPRE ? g.nls : 0;  // LoRA slabs after the nkt main slabs
  const int total = nkt + nls;

  // Epilogue layout (the stages are free again by then):
  //   stage 0: Ts [BM][2 RP] bf16, s*T split into hi (columns 0..RP) and lo (RP..2RP)
  //   stage 1: Bs [BN][RP] bf16, the tile's rows of B zero padded to RP.
  uint16_t* Ts = reinterpret_cast<uint16_t*>(sm0);
  uint16_t* Bs = reinterpret_cast<uint16_t*>(sm1);

  if (wave >= 4) {
    // ------------------------------------------------------------ copy waves
    const int cw = wave - 4;  // copy wave index (0..3), wave-uniform
    const int tl = t - NTM;   // copy thread index (0..255)
    // The tile's rows of B, fetched early and staged in LDS for the epilogue
    // (copy thread tl holds row n0 + tl, zero padded to RP, two bf16 per
    // register).
    uint32_t breg[RP2];

    if constexpr (RA > 0) {
      static_assert(BN == NT - NTM, "one B row per copy thread");
      const __amdgpu_buffer_rsrc_t brs = make_rsrc(a.B + (size_t)n0 * a.r, (uint32_t)min(BN, N - n0) * a.r * 2u);
      uint32_t v[RP];
#pragma unroll
      for (int j = 0; j < RP; ++j) {
        const bool ok = want_on && j < a.r;
        v[j] = __builtin_amdgcn_raw_buffer_load_b16(brs, ok ? (tl * a.r + j) * 2 : kOutOfRange, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < RP; j += 2) breg[j / 2] = (v[j] & 0xFFFFu) | (v[j + 1] << 16);
    }

    // One copy instruction moves 8 rows x 128 bytes (64 lanes x 16 bytes)
    // into 1 KB of LDS; lane i fills LDS chunk i of it, so it fetches the
    // global chunk that the swizzle maps there.  Buffer resources cover
    // exactly the tile's valid rows (rows past M, N or r read as zeros); a
    // chunk past K gets an out-of-range offset (zeros as well).  The copies
    // of a slab are dealt round-robin to the copy waves: x blocks 0..15, W
    // blocks 16..47, A blocks 48.., copy wave cw takes blocks cw, cw + 4, ...
    const i32x4_t xr = make_rsrc_raw(a.x + (size_t)m0 * K, (uint32_t)min(BM, M - m0) * K * 2u);
    const i32x4_t wrs = make_rsrc_raw(a.W + (size_t)n0 * K, (uint32_t)min(BN, N - n0) * K * 2u);
    const i32x4_t arsrc = make_rsrc_raw(RA > 0 ? a.A : nullptr, RA > 0 ? (uint32_t)min(a.r, RA) * K * 2u : 0u);
    const int row_bytes = K * 2;
    // Lane i fills LDS chunk i & 7 of row 8 ci + i / 8; every block ci this
    // wave copies has the parity of cw, so the global chunk it fetches is
    // (i & 7) ^ ((row / 2) % 8) = (i & 7) ^ (4 (cw & 1) + i / 16).
    const int c = (lane & 7) ^ (((cw & 1) << 2) | (lane >> 4));  // global chunk fetched by this lane
    const int rl = lane >> 3;                                    // row within the 8-row copy
    constexpr int XD = BM / 8, WD = BN / 8, AD = RA / 8;
    static_assert(XD % 4 == 0 && WD % 4 == 0, "x and W blocks split evenly over the copy waves");
    constexpr int XJ = XD / 4, WJ = WD / 4;
    constexpr int DMAX = XJ + WJ + (AD + 3) / 4;  // copies per slab of copy wave 0
    const int dn = XJ + WJ + (AD - cw + 3) / 4;   // copies per slab of this wave

    auto issue = [&](uint4* st, int kt) __attribute__((always_inline)) {
      const int k0 = kt * BK;
      const bool kv = k0 + c * 8 < K;
      const int kofs = k0 * 2 + c * 16;
#pragma unroll
      for (int j = 0; j < DMAX; ++j) {
        if (j < XJ) {
          const int ci = cw + 4 * j;
          dma16(xr, st + L::XOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kofs : kOutOfRange);
        } else if (j < XJ + WJ) {
          const int ci = cw + 4 * (j - XJ);
          dma16(wrs, st + L::WOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kofs : kOutOfRange);
        } else {
          const int ci = cw + 4 * (j - XJ - WJ);
          if (ci < AD) dma16(arsrc, st + L::AOFF + ci * 64, kv ? (ci * 8 + rl) * row_bytes + kofs : kOutOfRange);
        }
      }
    };
    // LoRA slab ls (TPRE): k in [64 ls, 64 ls + 64) of the 2 RP-long update; the
    // x-side rows are the tile's rows of ts ([hi | lo]), the W-side rows its
    // rows of bp, read at column k mod RP ([Bp | Bp]); k >= 2 RP reads zeros.
    // Same number of copies per wave as a main slab.
    const i32x4_t tsr = make_rsrc_raw(TPRE ? g.ts + (size_t)m0 * 2 * RP : nullptr,
                                      TPRE ? (uint32_t)min(BM, M - m0) * 2 * RP * 2u : 0u);
    const i32x4_t bpr = make_rsrc_raw(TPRE ? g.bp + (size_t)n0 * RP : nullptr,
                                      TPRE ? (uint32_t)min(BN, N - n0) * RP * 2u : 0u);
    auto issue_lora = [&](uint4* st, int ls) __attribute__((always_inline)) {
      const int kk = ls * BK + c * 8;
      const bool kv = kk < 2 * RP;
      const int kb = RP > 0 ? kk % (RP > 0 ? RP : 1) : 0;
#pragma unroll
      for (int j = 0; j < XJ + WJ; ++j) {
        if (j < XJ) {
          const int ci = cw + 4 * j;
          dma16(tsr, st + L::XOFF + ci * 64, kv ? (ci * 8 + rl) * (4 * RP) + kk * 2 : kOutOfRange);
        } else {
          const int ci = cw + 4 * (j - XJ);
          dma16(bpr, st + L::WOFF + ci * 64, kv ? (ci * 8 + rl) * (2 * RP) + kb * 2 : kOutOfRange);
        }
      }
    };
    auto issue_any = [&](uint4* st, int kt) __attribute__((always_inline)) {
      if (!TPRE || kt < nkt) issue(st, kt);
      else issue_lora(st, kt - nkt);
    };
    // Wait until only the copies of the `later` most recent slabs may still
    // be in flight.
    auto wait_slabs = [&](int later) __attribute__((always_inline)) {
      if (later <= 0) {
        wait_vm<0>();
      } else if (later == 1) {
        if (dn == DMAX) wait_vm<DMAX>(); else wait_vm<(DMAX > 0 ? DMAX - 1 : 0)>();
      } else {
        if (dn == DMAX) wait_vm<2 * DMAX>(); else wait_vm<(DMAX > 0 ? 2 * DMAX - 2 : 0)>();
      }
    };

    issue_any(sm0, 0);
    if (total > 1) issue_any(sm1, 1);
    if constexpr (NS == 3) {
      if (total > 2) issue_any(sm2, 2);
    }
    wait_slabs(min(NS - 1, total - 1));
    lds_barrier();  // slab 0 is in LDS
    // Before barrier kt: slab kt + 1 has landed.  After it: stage kt % NS is
    // no longer read and receives slab kt + NS.
    auto step_copy = [&](uint4* st, int kt) __attribute__((always_inline)) {
      wait_slabs(min(kt + NS - 1, total - 1) - (kt + 1));
      lds_barrier();
      if (kt + NS < total) issue_any(st, kt + NS);
    };
    if constexpr (NS == 3) {
      for (int kt = 0; kt < total; kt += 3) {
        step_copy(sm0, kt);
        if (kt + 1 < total) step_copy(sm1, kt + 1);
        if (kt + 2 < total) step_copy(sm2, kt + 2);
      }
    } else {
      for (int kt = 0; kt < total; kt += 2) {
        step_copy(sm0, kt);
        if (kt + 1 < total) step_copy(sm1, kt + 1);
      }
    }
    wait_vm<0>();
    lds_barrier();  // every wave is done with the stages
    if constexpr (TPRE) return;
    if constexpr (RA > 0) {
#pragma unroll
      for (int j = 0; j < RP; j += 2) *reinterpret_cast<uint32_t*>(Bs + tl * RP + j) = breg[j / 2];
    }
    __syncthreads();  // Ts and Bs staged
    return;
  }

  // -------------------------------------------------------------- MFMA waves
  f32x16_t acc[MT][NTL];
  f32x4_t accT[2][TJ1];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NTL; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int j = 0; j < TJ1; ++j) accT[q][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Register fragments of one 16-wide k-step (W rows as the A operand, x
  // rows as the B operand of the 32x32x16 MFMAs), double buffered so that
  // the next k-step's LDS reads overlap the current k-step's MFMAs, and the
  // T fragments of one 32-wide half slab (this wave's 32 x rows and the
  // LoRA-down rows, 16x16x32 layout), read in the even k-step and consumed
  // in the odd one.
  struct Frag {
    uint4 w[NTL];
    uint4 x[MT];
  };
  struct TFrag {
    uint4 tx[2];
    uint4 a[TJ1];
  };
  Frag F0, F1;
  TFrag TF;
  constexpr int NMAIN = MT * NTL;      // MFMAs per k-step
  constexpr int NRM = NTL + MT;        // main-fragment reads per k-step
  constexpr int NRT = TJ > 0 ? 2 + TJ : 0;  // T-fragment reads (even k-steps)

  // chunk (16 bytes = 8 k values) read by this lane in k-step s: lanes
  // 0..31 take k 16 s .. 16 s + 7, lanes 32..63 the next 8.
  auto read_main = [&](Frag& F, const uint4* s, int step, int r) __attribute__((always_inline)) {
    const int ch = 2 * step + lh;
    if (r < NTL) {
      F.w[r] = s[L::WOFF + lds_idx(wc * WN + r * 32 + l32, ch)];
    } else {
      const int mi = r - NTL;
      F.x[mi] = s[L::XOFF + lds_idx(wr * WM + mi * 32 + l32, ch)];
    }
  };
  auto read_t = [&](const uint4* s, int half, int r) __attribute__((always_inline)) {
    const int ch = 4 * half + lg;
    if (r < 2) {
      TF.tx[r] = s[L::XOFF + lds_idx(wr * WM + (wc * 2 + r) * 16 + l16, ch)];
    } else {
      TF.a[r - 2] = s[L::AOFF + lds_idx((r - 2) * 16 + l16, ch)];
    }
  };

  // k-step S of the current slab: MFMAs on Fc; reads of k-step S + 1 (of
  // `nxt` when S == 3) into Fn and, in even k-steps, of this half slab's T
  // fragments; in odd k-steps the T MFMAs of the half slab.
  auto kstep = [&](auto S, const Frag& Fc, Frag& Fn, const uint4* cur, const uint4* nxt)
      __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
    constexpr bool even = (s & 1) == 0;
    constexpr int NR = NRM + (even ? NRT : 0);
    const uint4* rs = s == 3 ? nxt : cur;
    constexpr int snext = (s + 1) & 3;
#pragma unroll
    for (int m = 0; m < NMAIN; ++m) {
      const int mi = m / NTL, ni = m % NTL;
      acc[mi][ni] = mfma32(Fc.w[ni], Fc.x[mi], acc[mi][ni]);
      if (m < NR) {
        if (m < NRM) read_main(Fn, rs, snext, m);
        else read_t(cur, s / 2, m - NRM);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int m = NMAIN; m < NR; ++m) {
      if (m < NRM) read_main(Fn, rs, snext, m);
      else read_t(cur, s / 2, m - NRM);
    }
    if constexpr (!even && TJ > 0) {
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        accT[0][j] = mfma16(TF.tx[0], TF.a[j], accT[0][j]);
        accT[1][j] = mfma16(TF.tx[1], TF.a[j], accT[1][j]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // Slab kt: k-steps 0..2 on `cur`; barrier (slab kt fully read, slab
  // kt + 1 landed); k-step 3, whose reads already take slab kt + 1 from
  // `nxt`.  Past the last slab those reads fill registers that are never
  // used, so every slab is the same straight-line code.
  auto slab = [&](const uint4* cur, const uint4* nxt) __attribute__((always_inline)) {
    kstep(IC<0>{}, F0, F1, cur, nxt);
    kstep(IC<1>{}, F1, F0, cur, nxt);
    kstep(IC<2>{}, F0, F1, cur, nxt);
    lds_barrier();
    kstep(IC<3>{}, F1, F0, cur, nxt);
  };

  // acc[mi][ni][4 i + e] holds y[wr*64 + mi*32 + l32][wc*128 + ni*32 + 8 i + 4 lh + e]
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
  lds_barrier();  // slab 0 is in LDS
#pragma unroll
  for (int r = 0; r < NRM; ++r) read_main(F0, sm0, 0, r);
  // TPRE: after the last main slab the accumulators are the LoRA-off result;
  // it is stored there, and the LoRA slabs (whose first fragments the last
  // main slab's k-step 3 has read) go on adding to the same accumulators.
  auto after = [&](int kt) __attribute__((always_inline)) {
    if constexpr (TPRE) {
      if (kt == nkt - 1 && a.y_off) store(a.y_off);
    }
  };
  if constexpr (NS == 3) {
    for (int kt = 0; kt < total; kt += 3) {
      slab(sm0, sm1);
      after(kt);
      if (kt + 1 < total) {
        slab(sm1, sm2);
        after(kt + 1);
      }
      if (kt + 2 < total) {
        slab(sm2, sm0);
        after(kt + 2);
      }
    }
  } else {
    for (int kt = 0; kt < total; kt += 2) {
      slab(sm0, sm1);
      after(kt);
      if (kt + 1 < total) {
        slab(sm1, sm0);
        after(kt + 1);
      }
    }
  }
  if constexpr (TPRE) {
    lds_barrier();  // every wave is done with the stages
    if (a.y_on) store(a.y_on);
    return;
  }
  lds_barrier();  // every wave is done with the stages before the epilogue reuses them

  // ---------------------------------------------------------------- epilogue
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
      }
    }
  __syncthreads();  // Ts and Bs staged

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

  if (a.y_off) store(a.y_off);
  if (a.y_on) {
    apply_lora();
    store(a.y_on);
  }
}

hipError_t launch(const GemmArgs& g, int rp, bool tpre, hipStream_t stream) {
  const dim3 grid(g.ntm * g.ntn), block(NT);
  if (tpre) {
    switch (rp) {
      case 16: hipLaunchKernelGGL((lora_gemm_kernel<16, true>), grid, block, 0, stream, g); break;
      case 32: hipLaunchKernelGGL((lora_gemm_kernel<32, true>), grid, block, 0, stream, g); break;
      case 64: hipLaunchKernelGGL((lora_gemm_kernel<64, true>), grid, block, 0, stream, g); break;
      case 128: hipLaunchKernelGGL((lora_gemm_kernel<128, true>), grid, block, 0, stream, g); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (rp) {
    case 0: hipLaunchKernelGGL((lora_gemm_kernel<0, false>), grid, block, 0, stream, g); break;
    case 16: hipLaunchKernelGGL((lora_gemm_kernel<16, false>), grid, block, 0, stream, g); break;
    case 32: hipLaunchKernelGGL((lora_gemm_kernel<32, false>), grid, block, 0, stream, g); break;
    case 64: hipLaunchKernelGGL((lora_gemm_kernel<64, false>), grid, block, 0, stream, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

hipError_t launch_lora_gemm(const LinearArgs& a, hipStream_t stream) {
  GemmArgs g{};
  g.lin = a;
  g.ntm = (a.M + BM - 1) / BM;
  g.ntn = (a.N + BN - 1) / BN;
  g.vec4 = (a.N % 4 == 0) && (!a.y_off || aligned16(a.y_off)) && (!a.y_on || aligned16(a.y_on));
  const int rp = a.y_on ? padded_rank(a.r) : 0;
  if (rp > 64) return hipErrorInvalidValue;  // needs the pre-pass workspace
  return launch(g, rp, false, stream);
}

hipError_t launch_lora_gemm_tpre(const LinearArgs& a, uint16_t* ts, uint16_t* bp, float* part, hipStream_t stream) {
  const int rp = a.y_on ? padded_rank(a.r) : 0;
  if (rp == 0) return launch_lora_gemm(a, stream);
  TpreArgs t{};
  t.x = a.x;
  t.A = a.A;
  t.B = a.B;
  t.s = a.s;
  t.M = a.M;
  t.N = a.N;
  t.K = a.K;
  t.r = a.r;
  t.ts = ts;
  t.bp = bp;
  t.part = part;
  const uint16_t* bp_used = nullptr;
  hipError_t e = launch_lora_tpre(t, rp, &bp_used, stream);
  if (e != hipSuccess) return e;
  GemmArgs g{};
  g.lin = a;
  g.ntm = (a.M + BM - 1) / BM;
  g.ntn = (a.N + BN - 1) / BN;
  g.vec4 = (a.N % 4 == 0) && (!a.y_off || aligned16(a.y_off)) && aligned16(a.y_on);
  g.ts = ts;
  g.bp = bp_used;
  g.nls = (2 * rp + BK - 1) / BK;
  return launch(g, rp, true, stream);
}

hipError_t launch_lora_gemm_slabs(const LinearArgs& a, const uint16_t* ts, const uint16_t* bp, int rp,
                                  hipStream_t stream) {
  GemmArgs g{};
  g.lin = a;
  g.ntm = (a.M + BM - 1) / BM;
  g.ntn = (a.N + BN - 1) / BN;
  g.vec4 = (a.N % 4 == 0) && (!a.y_off || aligned16(a.y_off)) && aligned16(a.y_on);
  g.ts = ts;
  g.bp = bp;
  g.nls = (2 * rp + BK - 1) / BK;
  return launch(g, rp, true, stream);
}

}  // namespace hydra
