// Fused CLM-head scoring GEMM for gfx950 (MI355X): the LoRA-off and LoRA-on
// logits z_off = h W^T and z_on = z_off + s (h A^T) B^T of the CLM head are
// reduced to per-row (max, sum exp) partials and the sampled token's logit
// without ever being written to memory (Sec. 3, the CLM head of pi^hydra;
// App. A, Alg. 1 / Alg. 2, reference and actor log-probabilities).
//
// The vocabulary dimension gives thousands of output tiles, so this GEMM uses
// the largest tile the register file allows, which moves the least data per
// MFMA through L2 and LDS (the matrix cores run power-limited, and data
// movement costs power):
//  * one 256 x 256 output tile per 256-thread workgroup (one wave per SIMD);
//    each wave owns a 128 x 128 sub-tile = 4 x 4 v_mfma_f32_32x32x16_bf16
//    tiles, 256 fp32 accumulators per lane (held in AGPRs);
//  * K slabs of 32 go through a four-stage LDS ring (32 KB per stage, rows of
//    64 bytes, 16-byte chunks XOR-swizzled by row / 4).  The copies
//    (buffer_load ... lds) are issued by the MFMA waves themselves, four per
//    16-wide k-step, three slabs ahead of use;
//  * one barrier per slab: before it every wave has read the slab's last
//    fragments and waited for its copies of the next slab, after it the freed
//    stage is refilled;
//  * the rank-r product T = h A^T is the same for every column tile of a row
//    block, so it is computed once by lora_t_kernel (bf16 hi + lo parts of
//    s*T in the workspace, with B zero padded to the padded rank RP next to
//    it) instead of in the main loop;
//  * the LoRA update s*T*B^T is then a GEMM with 2 RP more k values ([hi | lo]
//    against [B | B]); it runs as 2 RP / 32 more slabs through the same ring,
//    right after the per-row (max, sum exp) of the LoRA-off logits have been
//    taken from the accumulators, and the same statistics of the LoRA-on
//    logits follow.  The lane holding the sampled token's column records its
//    logit.  One float4 (max_off, sum_off, max_on, sum_on) per (row, column
//    tile) goes to the workspace for score_combine_kernel.
// With B = 0 or s = 0 the LoRA update adds exact zeros, so the on and off
// statistics (computed by the same code) are bit-identical and KL == 0.
//
// Two inputs (the actor pass and the LoRA-off pass each with their own final
// hidden states, App. A, Alg. 2): the grid holds twice the row tiles, the
// LoRA-off tile and the actor tile of each row block next to each other in
// the tile order (so both read a column block of W while it is in L2).  A
// LoRA-off tile takes only the LoRA-off statistics and runs no LoRA slabs;
// an actor tile runs the LoRA slabs over its own T and takes only the LoRA-on
// statistics.  Each writes its half of the (row, column tile) partial.
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

constexpr int BM = 256;        // tile rows (tokens)
constexpr int BN = 256;        // tile columns (vocabulary entries)
constexpr int BK = 32;         // K slab
constexpr int NT = 256;        // threads per workgroup (4 waves)
constexpr int WM = 128;        // wave tile rows
constexpr int WN = 128;        // wave tile columns
constexpr int MT = WM / 32;    // 32-row x tiles per wave
constexpr int NTL = WN / 32;   // 32-row W tiles per wave
constexpr int CPR = BK / 8;    // 16-byte chunks per LDS row
constexpr int NS = 4;          // ring stages
constexpr int STAGE = (BM + BN) * CPR;  // uint4 per stage (32 KB)
constexpr int XOFF = 0;
constexpr int WOFF = BM * CPR;
constexpr int GROUP_M = 8;     // row tiles walked together (L2 reuse of W)
constexpr int DPW = (BM + BN) / 16 / 4;  // copies per wave per slab (16 rows of 64 bytes each)

static_assert(kScoreTileN == BN, "one partial per GEMM column tile");
static_assert(kScoreTileM == BM && kScoreThreads == NT, "launch shape known to the host checks");
static_assert(DPW == 8, "the k-step schedule issues four copies per k-step");
static_assert(BM * 2 * 4 * 4 <= STAGE * 16, "the epilogue's row statistics fit in one stage");

// LDS chunk index of (row, 16-byte chunk c) in a stage: rows of 64 bytes, the
// chunk is XOR-ed with (row / 4) % 4 so that the 16 lanes of one read phase
// (16 consecutive rows, one chunk) cover all banks.
__device__ __forceinline__ int sidx(int row, int c) { return row * CPR + (c ^ ((row >> 2) & 3)); }

// Workgroup id -> (row tile, column tile): as in the dual GEMM, each XCD gets a
// contiguous range of the logical order when the tile count allows, and the
// logical order walks GROUP_M row tiles per column tile.
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

template <int N>
__device__ __forceinline__ void wait_vm_lds_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | (((N >> 4) & 3) << 14));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int V>
struct IC {
  static constexpr int value = V;
};

// RAGGED: the vocabulary is not a multiple of the column tile, so the last
// column tile masks the columns past N.
template <int RP, bool RAGGED, bool DUAL>
__global__ __launch_bounds__(NT, 1) void score_gemm_kernel(ScoreGemmArgs g) {
  __shared__ uint4 sm[NS][STAGE];

  const LinearArgs& a = g.lin;
  const int M = a.M, N = a.N, K = a.K;
  const int t = threadIdx.x;
  const int lane = t & 63;
  // wave-uniform (SGPR) wave index: MFMAs never sit under divergent control flow
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wr = wave >> 1;
  const int wc = wave & 1;
  const int l32 = lane & 31;
  const int lh = lane >> 5;

  constexpr bool dual = DUAL;
  int tmi, tni;
  tile_of(blockIdx.x, dual ? 2 * g.ntm : g.ntm, g.ntn, tmi, tni);
  // two inputs: row tile 2 i is the LoRA-off tile of row block i, 2 i + 1 its actor tile
  const bool is_act = dual && (tmi & 1) != 0;
  if (dual) tmi >>= 1;
  const bool do_off = !dual || !is_act;  // this tile takes the LoRA-off statistics
  const bool do_on = !dual || is_act;    // ... and / or the LoRA-on ones
  // (tile coordinates are made provably wave-uniform, so that everything
  // derived from them -- buffer descriptors, LDS bases -- lives in SGPRs)
  const int m0 = __builtin_amdgcn_readfirstlane(tmi * BM);
  const int n0 = __builtin_amdgcn_readfirstlane(tni * BN);
  const int nkt = (K + BK - 1) / BK;
  if (nkt < 1) __builtin_unreachable();  // K >= 8 is validated by the caller
  // The LoRA update s*T*B^T is a GEMM with 2 RP more k values: the rows of
  // [hi | lo] (s*T in bf16 hi and lo parts) against the rows of [Bp | Bp]
  // (B zero padded to RP).  Those run as LS more slabs of the same ring,
  // after the LoRA-off statistics have been taken from the accumulators.
  constexpr int LS = 2 * RP / BK;
  const int nsl = nkt + (do_on ? LS : 0);

  // the sampled tokens of this lane's four rows, fetched early
  int tk[MT];
#pragma unroll
  for (int mi = 0; mi < MT; ++mi) {
    const int row = m0 + wr * WM + mi * 32 + l32;
    tk[mi] = row < M ? g.tokens[row] : -1;
  }

  // ---- copies.  One copy instruction moves 16 rows x 64 bytes (64 lanes x
  // 16 bytes) into 1 KB of LDS; lane i fills LDS chunk i of it, so it fetches
  // the global chunk that the swizzle maps there.  Buffer resources cover
  // exactly the tile's valid rows (rows past M or N read as zeros); a chunk
  // past K gets an out-of-range offset (zeros as well), and so do all copies
  // of the slabs past the last one, which land in stages that are not read
  // again.  Wave w copies 16-row blocks w, w + 4, w + 8, w + 12 of the x side
  // (j < 4) and of the W side (j >= 4) of every slab.
  const i32x4_t xr = make_rsrc_raw((is_act ? g.x_act : a.x) + (size_t)m0 * K, (uint32_t)min(BM, M - m0) * K * 2u);
  const i32x4_t wrs = make_rsrc_raw(a.W + (size_t)n0 * K, (uint32_t)min(BN, N - n0) * K * 2u);
  const i32x4_t tsr = make_rsrc_raw(g.ts + (size_t)m0 * 2 * RP, (uint32_t)min(BM, M - m0) * 2 * RP * 2u);
  const i32x4_t bpr = make_rsrc_raw(g.bp + (size_t)n0 * RP, (uint32_t)min(BN, N - n0) * RP * 2u);
  const int row_bytes = K * 2;
  const int cg = (lane & 3) ^ ((lane >> 4) & 3);  // global chunk fetched by this lane
  const int rl = lane >> 2;                       // row within the 16-row copy
  // Copy j of slab kt.  MAIN: kt is known to be a slab of h and W (the
  // steady state); otherwise kt may also be a LoRA slab or past the end, and
  // source and offset are selected without branches.
  auto dma_one = [&](auto MAIN, uint4* st, int kt, int j) __attribute__((always_inline)) {
    const int ci = wave + 4 * (j & 3);
    const int row = ci * 16 + rl;
    uint4* dst = st + (j < 4 ? XOFF : WOFF) + ci * 64;
    const int k0 = kt * BK;
    const int off_main = k0 + cg * 8 < K ? row * row_bytes + k0 * 2 + cg * 16 : kOutOfRange;
    if constexpr (decltype(MAIN)::value) {
      dma16(j < 4 ? xr : wrs, dst, off_main);
    } else {
      const bool is_main = kt < nkt, is_lora = LS > 0 && kt >= nkt && kt < nsl;
      const int k = (kt - nkt) * BK + cg * 8;  // k within [0, 2 RP) in a LoRA slab
      const int off_lora = j < 4 ? (row * 2 * RP + k) * 2 : (row * RP + (k & (RP > 0 ? RP - 1 : 0))) * 2;
      const int off = is_main ? off_main : (is_lora ? off_lora : kOutOfRange);
      dma16(is_main ? (j < 4 ? xr : wrs) : (j < 4 ? tsr : bpr), dst, off);
    }
  };

  f32x16_t acc[MT][NTL];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NTL; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // Fragments of one 16-wide k-step: W rows (A operand) and h rows (B
  // operand), double buffered across k-steps.
  struct Frag {
    uint4 w[NTL];
    uint4 x[MT];
  };
  Frag F0, F1;
  auto read_one = [&](Frag& F, const uint4* st, int s, int r) __attribute__((always_inline)) {
    const int ch = 2 * s + lh;
    if (r < NTL)
      F.w[r] = st[WOFF + sidx(wc * WN + r * 32 + l32, ch)];
    else
      F.x[r - NTL] = st[XOFF + sidx(wr * WM + (r - NTL) * 32 + l32, ch)];
  };

  // k-step S of slab kt (stage `cur`): MFMAs on Fc, reads of the next k-step
  // into Fn (k-step 1 of this slab, or k-step 0 of slab kt + 1 from `nxt`),
  // and four copies: k-step 0 finishes slab kt + 3 (W side, into the stage
  // of slab kt - 1), k-step 1 starts slab kt + 4 (x side, into `cur`, free
  // after the barrier).
  auto kstep = [&](auto S, auto MAIN, const Frag& Fc, Frag& Fn, const uint4* rs, uint4* ddst, int dkt)
      __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
#pragma unroll
    for (int m = 0; m < MT * NTL; ++m) {
      const int mi = m / NTL, ni = m % NTL;
      acc[mi][ni] = mfma32(Fc.w[ni], Fc.x[mi], acc[mi][ni]);
      if (m < NTL + MT) read_one(Fn, rs, s ^ 1, m);
      if (m >= 8 && (m & 1) == 1) dma_one(MAIN, ddst, dkt, (s == 0 ? 4 : 0) + ((m - 9) >> 1));
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto slab = [&](auto MAIN, uint4* cur, uint4* nxt, uint4* prev, int kt) __attribute__((always_inline)) {
    kstep(IC<0>{}, MAIN, F0, F1, cur, prev, kt + 3);
    // slab kt + 1 must have landed: only the copies of slabs kt + 2 and kt + 3
    // (2 x DPW per wave) may still be in flight
    wait_vm_lds_barrier<2 * DPW>();
    kstep(IC<1>{}, MAIN, F1, F0, nxt, cur, kt + 4);
  };

  // prologue: slabs 0..2 and the x side of slab 3
#pragma unroll
  for (int j = 0; j < DPW; ++j) dma_one(IC<0>{}, sm[0], 0, j);
#pragma unroll
  for (int j = 0; j < DPW; ++j) dma_one(IC<0>{}, sm[1], 1, j);
#pragma unroll
  for (int j = 0; j < DPW; ++j) dma_one(IC<0>{}, sm[2], 2, j);
#pragma unroll
  for (int j = 0; j < 4; ++j) dma_one(IC<0>{}, sm[3], 3, j);
  wait_vm_lds_barrier<2 * DPW + 4>();
#pragma unroll
  for (int r = 0; r < NTL + MT; ++r) read_one(F0, sm[0], 0, r);
  // steady state: every copy issued by slabs kt .. kt + 3 (slabs up to kt + 7)
  // is a copy of h and W
  int kt = 0;
  for (; kt + 2 * NS <= nkt; kt += NS) {
    slab(IC<1>{}, sm[0], sm[1], sm[3], kt);
    slab(IC<1>{}, sm[1], sm[2], sm[0], kt + 1);
    slab(IC<1>{}, sm[2], sm[3], sm[1], kt + 2);
    slab(IC<1>{}, sm[3], sm[0], sm[2], kt + 3);
  }
  for (; kt < nkt; kt += NS) {
    slab(IC<0>{}, sm[0], sm[1], sm[3], kt);
    if (kt + 1 < nkt) slab(IC<0>{}, sm[1], sm[2], sm[0], kt + 1);
    if (kt + 2 < nkt) slab(IC<0>{}, sm[2], sm[3], sm[1], kt + 2);
    if (kt + 3 < nkt) slab(IC<0>{}, sm[3], sm[0], sm[2], kt + 3);
  }

  // ---------------------------------------------------------------- epilogue
  // acc[mi][ni][4 i + e] holds z[m0 + wr*128 + mi*32 + l32][n0 + wc*128 + ni*32 + 8 i + 4 lh + e].
  // Per row block mi: (max, sum exp) over this lane's 64 logits, merged with
  // the lane holding the row's other 64 (lane ^ 32).  For a ragged
  // vocabulary the logits of columns past N are taken as -inf (branch-free).
  // The lane holding the sampled token's column records its logit.
  const int wcol0 = n0 + wc * WN;
  auto row_stats = [&](int mi, int pass, float& mx, float& sm_) __attribute__((always_inline)) {
    float z[NTL * 16];
#pragma unroll
    for (int ni = 0; ni < NTL; ++ni)
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        // Read from the accumulator register here.  Left to itself the
        // compiler copies all 256 accumulators into VGPRs when the main loop
        // ends and, with the LoRA slabs still to come, spills a quarter of
        // them to scratch memory.
        float v;
        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(acc[mi][ni][k]));
        z[ni * 16 + k] = v;
      }
    if constexpr (RAGGED) {
      const int lim = N - wcol0 - 4 * lh;  // offsets at or past lim are past N
#pragma unroll
      for (int q = 0; q < NTL * 16; ++q)
        z[q] = (q >> 4) * 32 + 8 * ((q & 15) >> 2) + (q & 3) < lim ? z[q] : -INFINITY;
    }
    mx = -INFINITY;
#pragma unroll
    for (int q = 0; q < NTL * 16; ++q) mx = fmaxf(mx, z[q]);
    const int rel = tk[mi] - wcol0 - 4 * lh;  // column offset within this lane's half
    if (rel >= 0 && rel < WN && ((rel >> 2) & 1) == 0) {
      float v = 0.f;
#pragma unroll
      for (int q = 0; q < NTL * 16; ++q) v = ((q >> 4) * 32 + 8 * ((q & 15) >> 2) + (q & 3) == rel) ? z[q] : v;
      g.zt[(size_t)(m0 + wr * WM + mi * 32 + l32) * 2 + pass] = v;
    }
    sm_ = 0.f;
    if (mx != -INFINITY) {
      // e^(z - mx) = 2^(z log2 e - mx log2 e)
      const float mxs = mx * kLog2e;
#pragma unroll
      for (int q = 0; q < NTL * 16; ++q) sm_ += __builtin_amdgcn_exp2f(fmaf(z[q], kLog2e, -mxs));
    }
    const float mo = __shfl_xor(mx, 32);
    const float so = __shfl_xor(sm_, 32);
    lse_merge(mx, sm_, mo, so);
  };

  float st_off[MT][2], st_on[MT][2];
  if constexpr (DUAL) {
    // two inputs: an actor tile runs the LoRA slabs, then every tile takes
    // one kind of statistics through a single call site (so that the
    // accumulators are read in one place)
    if constexpr (LS > 0) {
      if (is_act) {
#pragma unroll
        for (int q = 0; q < LS; ++q) {
          const int kq = nkt + q;
          slab(IC<0>{}, sm[kq % NS], sm[(kq + 1) % NS], sm[(kq + NS - 1) % NS], kq);
        }
      }
    }
    const int pass = is_act ? 1 : 0;
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      __builtin_amdgcn_sched_barrier(0);
      row_stats(mi, pass, st_off[mi][0], st_off[mi][1]);
      st_on[mi][0] = st_off[mi][0];
      st_on[mi][1] = st_off[mi][1];
    }
  } else if (do_off) {
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      __builtin_amdgcn_sched_barrier(0);
      row_stats(mi, 0, st_off[mi][0], st_off[mi][1]);  // LoRA off
    }
  }
  if constexpr (DUAL) {
    // done above
  } else if constexpr (LS > 0) {
    // The LoRA slabs nkt .. nkt + LS - 1 (stage (nkt + q) % NS; the last main
    // slab already read the first k-step of slab nkt into F0).
#pragma unroll
    for (int q = 0; q < LS; ++q) {
      const int kq = nkt + q;
      slab(IC<0>{}, sm[kq % NS], sm[(kq + 1) % NS], sm[(kq + NS - 1) % NS], kq);
    }
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      __builtin_amdgcn_sched_barrier(0);
      row_stats(mi, 1, st_on[mi][0], st_on[mi][1]);  // LoRA on
    }
  } else {
    // no adapter: the LoRA-on logits are the LoRA-off logits
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      st_on[mi][0] = st_off[mi][0];
      st_on[mi][1] = st_off[mi][1];
      const int rel = tk[mi] - wcol0 - 4 * lh;
      if (rel >= 0 && rel < WN && ((rel >> 2) & 1) == 0) {
        const size_t zi = (size_t)(m0 + wr * WM + mi * 32 + l32) * 2;
        g.zt[zi + 1] = g.zt[zi];
      }
    }
  }
  wait_vm_lds_barrier<0>();  // every copy has landed and every wave is done with the ring

  // the two waves of a row block column pair merge their row statistics
  float* red = reinterpret_cast<float*>(sm[0]);  // [2][BM][4]
  if (lh == 0) {
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
      const int rloc = wr * WM + mi * 32 + l32;
      // (a tile of two inputs fills only its own half; the other half is never read)
      *reinterpret_cast<float4*>(red + (wc * BM + rloc) * 4) =
          make_float4(do_off ? st_off[mi][0] : 0.f, do_off ? st_off[mi][1] : 0.f, do_on ? st_on[mi][0] : 0.f,
                      do_on ? st_on[mi][1] : 0.f);
    }
  }
  __syncthreads();
  {
    const int row = m0 + t;
    if (t < BM && row < M) {
      const float4 p0 = *reinterpret_cast<const float4*>(red + t * 4);
      const float4 p1 = *reinterpret_cast<const float4*>(red + (BM + t) * 4);
      float mo = p0.x, so = p0.y, mn = p0.z, sn = p0.w;
      lse_merge(mo, so, p1.x, p1.y);
      lse_merge(mn, sn, p1.z, p1.w);
      float4* dst = g.part + (size_t)row * g.ntn + tni;
      if constexpr (!DUAL)
        *dst = make_float4(mo, so, mn, sn);
      else if (do_off)
        reinterpret_cast<float2*>(dst)[0] = make_float2(mo, so);
      else
        reinterpret_cast<float2*>(dst)[1] = make_float2(mn, sn);
    }
  }
}

// T = h A^T for 16 rows per workgroup; the 8 waves split K.  Writes the bf16
// hi and lo parts of s*T: ts[row][j] = hi, ts[row][RP + j] = lo (zero for
// j >= r), the x-side rows of the scoring GEMM's LoRA slabs.
template <int RP>
hipError_t launch_rp(const ScoreGemmArgs& s_in, hipStream_t stream) {
  ScoreGemmArgs s = s_in;
  const bool ragged = s.lin.N % BN != 0;
  if constexpr (RP > 0) {
    TpreArgs t{};
    t.x = s.x_act ? s.x_act : s.lin.x;
    t.A = s.lin.A;
    t.B = s.lin.B;
    t.s = s.lin.s;
    t.M = s.lin.M;
    t.N = s.lin.N;
    t.K = s.lin.K;
    t.r = s.lin.r;
    t.ts = s.ts;
    t.bp = s.bp_buf;
    t.part = s.tpart;
    const hipError_t e = launch_lora_tpre(t, RP, &s.bp, stream);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((s.x_act ? 2 : 1) * s.ntm * s.ntn);
  if (s.x_act) {
    if (ragged)
      hipLaunchKernelGGL((score_gemm_kernel<RP, true, true>), grid, dim3(NT), 0, stream, s);
    else
      hipLaunchKernelGGL((score_gemm_kernel<RP, false, true>), grid, dim3(NT), 0, stream, s);
  } else if (ragged) {
    hipLaunchKernelGGL((score_gemm_kernel<RP, true, false>), grid, dim3(NT), 0, stream, s);
  } else {
    hipLaunchKernelGGL((score_gemm_kernel<RP, false, false>), grid, dim3(NT), 0, stream, s);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_gemm(const ScoreGemmArgs& s_in, hipStream_t stream) {
  ScoreGemmArgs s = s_in;
  s.ntm = (s.lin.M + BM - 1) / BM;
  const int r = s.lin.r;
  switch (padded_rank(r)) {
    case 0: return launch_rp<0>(s, stream);
    case 16: return launch_rp<16>(s, stream);
    case 32: return launch_rp<32>(s, stream);
    case 64: return launch_rp<64>(s, stream);
    default: return launch_rp<128>(s, stream);
  }
}

}  // namespace hydra
