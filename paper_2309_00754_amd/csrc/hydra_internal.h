// Launchers shared between the C-ABI layer and the kernel translation units.
// Every launcher assumes its arguments were validated by hydra_api.cpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hydra {

struct LinearArgs {
  const uint16_t* x;  // [M x K] bf16
  const uint16_t* W;  // [N x K] bf16
  const uint16_t* A;  // [r x K] bf16
  const uint16_t* B;  // [N x r] bf16
  float s;
  int M, N, K, r;
  float* y_off;  // [M x N] or nullptr
  float* y_on;   // [M x N] or nullptr
};

// A group of G independent LoRA-switchable linears with the same M, N, K, r
// (e.g. the attention projections of one decode step), for one launch.
constexpr int kMaxGroup = 8;
struct GroupArgs {
  const uint16_t* x[kMaxGroup];
  const uint16_t* W[kMaxGroup];
  const uint16_t* A[kMaxGroup];
  const uint16_t* B[kMaxGroup];
  float* y_off[kMaxGroup];
  float* y_on[kMaxGroup];
  float s[kMaxGroup];
  int G, M, N, K, r;
};

// Base product y[m] = x[m] W^T for up to kStreamRows rows per W, G weights in
// one launch.  The rows of weight g come from segments seg0[g] ..
// seg0[g] + nseg[g] - 1, each a block of seg_rows consecutive input rows
// ([seg_rows x K] bf16 at x[s]) with its output rows ([seg_rows x N] fp32 at
// ya[s], and a second copy at yb[s]; either may be null): one segment per
// linear of a group, or one per input when several inputs share one W.
constexpr int kStreamRows = 8;
constexpr int kStreamSegs = 8;
struct StreamArgs {
  const uint16_t* W[kMaxGroup];
  const uint16_t* x[kStreamSegs];
  float* ya[kStreamSegs];
  float* yb[kStreamSegs];
  int seg0[kMaxGroup];
  int nseg[kMaxGroup];
  // segment (counted from seg0) of every row slot; kStreamSegs: no row
  // (32-bit entries: read with scalar loads)
  int seg_of[kMaxGroup][kStreamRows];
  int G, seg_rows, N, K;
};
// Fills seg_of from seg0 / nseg / seg_rows.
inline void stream_finish_args(StreamArgs& a) {
  for (int g = 0; g < a.G; ++g)
    for (int m = 0; m < kStreamRows; ++m) {
      const int sg = m / a.seg_rows;
      a.seg_of[g][m] = sg < a.nseg[g] ? sg : kStreamSegs;
    }
}

// Pre-pass of the LoRA update for the MFMA GEMMs: ts = bf16 hi and lo parts
// of s * x A^T ([M x 2 RP], hi in columns 0..RP, lo in RP..2 RP) and bp = B
// zero padded to RP columns ([N x RP]), RP = padded rank.
struct TpreArgs {
  const uint16_t* x;  // [M x K] bf16
  const uint16_t* A;  // [r x K] bf16
  const uint16_t* B;  // [N x r] bf16
  float s;
  int M, N, K, r;
  uint16_t* ts;       // [M x 2 RP] hi | lo of s T, or nullptr
  uint16_t* bp;       // used only when B itself cannot serve (r != RP or B not 16-byte aligned)
  float* part;        // [kTpreMaxChunks x M x RP] fp32 partial sums over K chunks
  uint16_t* tT;       // [2][RP][Mp] bf16 hi and lo planes of (s T)^T, rows M..Mp zero, or nullptr
  int Mp;             // leading dimension of tT (M rounded up to 32)
};
// K is split into at most kTpreMaxChunks chunks of at least 1024, so that
// the pre-pass spreads over many workgroups; the partial products are then
// added in chunk order (deterministic).
constexpr int kTpreMaxChunks = 8;
inline void tpre_chunks(int K, int& nkc, int& kch) {
  const int want = (K + 1023) / 1024;
  nkc = want < kTpreMaxChunks ? want : kTpreMaxChunks;
  kch = ((K + nkc - 1) / nkc + 31) / 32 * 32;  // a multiple of the 32-wide k-step
  nkc = (K + kch - 1) / kch;
}
// Launches the pre-pass; *bp_used is where the padded B rows are (a.bp, or
// a.B itself when it already has that layout).
hipError_t launch_lora_tpre(const TpreArgs& a, int rp, const uint16_t** bp_used, hipStream_t stream);
// Two pre-passes over the same M rows, neither with B to pad, in the same two
// launches.
hipError_t launch_lora_tpre2(const TpreArgs& a0, const TpreArgs& a1, int rp, hipStream_t stream);
// Up to kMaxGroup pre-passes over the same M rows in the same two launches;
// none may need its B padded (B null, or r == rp and B 16-byte aligned: the
// GEMM then reads B itself), else hipErrorInvalidValue.
hipError_t launch_lora_tpre_multi(const TpreArgs* as, int n, int rp, hipStream_t stream);
// Padded rank: the smallest of 16, 32, 64, 128 that holds r (0 for r == 0).
inline int padded_rank(int r) { return r == 0 ? 0 : r <= 16 ? 16 : r <= 32 ? 32 : r <= 64 ? 64 : 128; }

// Per (row, column tile) partial log-sum-exp state written by the fused
// CLM-head GEMM: (max_off, sumexp_off, max_on, sumexp_on).
struct ScoreGemmArgs {
  LinearArgs lin;          // N = V, y_off / y_on unused
  const int32_t* tokens;   // [M]
  float4* part;            // [M x ntn]
  float* zt;               // [M x 2]: (z_off[token], z_on[token])
  uint16_t* ts;            // [M x 2 RP] bf16: hi and lo parts of s * h A^T (RP = padded rank)
  const uint16_t* bp;      // [V x RP] bf16: B zero padded to RP columns (or B itself when r == RP)
  uint16_t* bp_buf;        // room for the padded copy
  float* tpart;            // LoRA pre-pass partial sums over K chunks
  int ntn;                 // number of column tiles
  int ntm;                 // number of row tiles (set by the launcher)
  // Two inputs (the actor pass and the LoRA-off pass have their own hidden
  // states): lin.x holds the LoRA-off rows, x_act the rows scored with the
  // head's LoRA; each row tile of either input is its own GEMM tile.
  const uint16_t* x_act;   // nullptr: one input (lin.x) for both passes
};

struct CombineArgs {
  const float4* part;      // [M x ntn]
  const float* zt;         // [M x 2]
  const int32_t* tokens;   // [M]
  int M, V, ntn;
  float* lp_on;
  float* lp_off;
  float* kl;
  float* lse_on;           // optional
  float* lse_off;          // optional
  int32_t* err;            // optional
  // reward head
  const uint16_t* h;       // [M x K]
  const uint16_t* w_rm;    // [K] or nullptr
  float* reward;           // [n_seq] or nullptr
  int n_seq, seq_len, K;
};

struct LogitsArgs {
  const float* on;
  const float* off;
  const int32_t* tokens;
  int M, V;
  float* lp_on;
  float* lp_off;
  float* kl;
  float* lse_on;
  float* lse_off;
  int32_t* err;
};

// Critic scalar head: values[m] = <h[m], w> (fp32 accumulation).
struct ValueHeadArgs {
  const uint16_t* h;  // [M x K] bf16
  const uint16_t* w;  // [K] bf16
  int M, K;
  float* values;      // [M]
};

// Per-token PPO reward and generalized advantage estimation over n_seq
// sequences of seq_len tokens (sequence-major).
struct GaeArgs {
  const float* kl;      // [M]
  const float* reward;  // [n_seq]
  const float* values;  // [M]
  int n_seq, seq_len, start;
  float beta, gamma, lam;
  float* rewards;       // [M] or nullptr
  float* advantages;    // [M]
  float* returns;       // [M]
};

// PPO update-stage losses over n_seq sequences of seq_len tokens.
struct PpoLossArgs {
  const float* lp_new;   // [M]
  const float* lp_old;   // [M]
  const float* adv;      // [M]
  const float* values;   // [M]
  const float* returns;  // [M]
  int n_seq, seq_len, start;
  float eps;
  float* losses;         // [3]: policy loss, value loss, clipped fraction
  float* d_lp;           // [M] or nullptr
  float* d_v;            // [M] or nullptr
};

// Backward of the LoRA-switchable linear with W frozen (see lora_backward.hip).
struct BackwardArgs {
  const uint16_t* x;   // [M x K]
  const uint16_t* Wt;  // [K x N], W transposed
  const uint16_t* A;   // [r x K]
  const uint16_t* B;   // [N x r]
  const uint16_t* dy;  // [M x N]
  float s;
  int M, N, K, r;
  float* dx;           // [M x K] or nullptr
  float* dA;           // [r x K] or nullptr
  float* dB;           // [N x r] or nullptr
};
// Workspace bytes of the backward, and the launcher (which assumes a
// workspace of at least that size, 16-byte aligned).
size_t backward_ws_bytes(int M, int N, int K, int rp);
hipError_t launch_lora_backward(const BackwardArgs& a, void* ws, hipStream_t stream);
// dst [Cp x Rp] bf16: dst[c][q] = src[q][c] for c < C, q < R (src [R x C]), else 0.
hipError_t launch_transpose_pad(const uint16_t* src, int R, int C, uint16_t* dst, int Rp, int Cp, hipStream_t stream);
// The GEMM of lora_gemm_kernel<RP, true> with its LoRA slabs already in memory
// (ts [M x 2 RP] hi | lo, bp [N x RP]).
hipError_t launch_lora_gemm_slabs(const LinearArgs& a, const uint16_t* ts, const uint16_t* bp, int rp,
                                  hipStream_t stream);

// Column-tile width of the fused scoring GEMM (number of vocabulary entries
// one workgroup reduces).
constexpr int kScoreTileN = 256;
// Launch shapes the host validation needs: a dispatch counts work-items in
// 32 bits, so (tiles x threads per workgroup) must stay below 2^32.
constexpr int kScoreTileM = 256;
constexpr int kScoreThreads = 256;
constexpr int kGemmTileM = 128;
constexpr int kGemmTileN = 256;
constexpr int kGemmThreads = 512;

hipError_t launch_lora_gemm(const LinearArgs& a, hipStream_t stream);
// The same with the LoRA update from the pre-pass: ts [M x 2 RP] and bp [N x RP]
// bf16 workspace (RP = padded rank of a.r, up to 128).
hipError_t launch_lora_gemm_tpre(const LinearArgs& a, uint16_t* ts, uint16_t* bp, float* part, hipStream_t stream);
hipError_t launch_lora_gemv_group(const GroupArgs& g, hipStream_t stream);
// y[m] = x[m] W^T for the rows of a StreamArgs (rows <= kStreamRows).
hipError_t launch_gemv_stream(const StreamArgs& a, hipStream_t stream);
// y_on += s (x A^T) B^T for the members of g with an adapter (M <= 8 rows).
hipError_t launch_lora_update(const GroupArgs& g, hipStream_t stream);
// The decode step of a group (M <= 8) in one launch.  ws (16-byte aligned,
// zero before its first use): kFusedCtlBytes of control words (the kernel
// keeps a call generation there), then kFusedTSlotBytes of tagged T slots
// (64-bit entries, [G][kStreamRows][padded rank]), then kFusedYBytes of
// tagged LoRA-off outputs (64-bit entries, [G][N][rows padded to 1, 2, 4 or
// 8]); both regions have a fixed size, and nothing else is ever written
// there, so that calls of any shape find only their own or older tags.
constexpr int kFusedBuckets = 32;
constexpr size_t kFusedCtlBytes = size_t(2 + kFusedBuckets) * 128;
constexpr size_t kFusedTSlotBytes = size_t(kMaxGroup) * kStreamRows * 128 * 8;
constexpr size_t kFusedYBytes = size_t(2) << 20;
constexpr size_t kFusedWsBytes = kFusedCtlBytes + kFusedTSlotBytes + kFusedYBytes;
hipError_t launch_gemv_fused(const GroupArgs& g, void* ws, hipStream_t stream);
hipError_t launch_score_gemm(const ScoreGemmArgs& a, hipStream_t stream);
hipError_t launch_value_head(const ValueHeadArgs& a, hipStream_t stream);
hipError_t launch_gae(const GaeArgs& a, hipStream_t stream);
hipError_t launch_ppo_loss(const PpoLossArgs& a, hipStream_t stream);
hipError_t launch_score_combine(const CombineArgs& a, hipStream_t stream);
hipError_t launch_score_logits(const LogitsArgs& a, hipStream_t stream);

}  // namespace hydra
