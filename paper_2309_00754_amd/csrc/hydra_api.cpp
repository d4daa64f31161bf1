// C ABI of libhydra: argument validation on the host, then kernel launches on
// the caller's stream.  Validation runs before any HIP call, so every argument
// error is reported without touching the device.
#include "../../include/hydra.h"

#include <hip/hip_runtime.h>

#include <mutex>

#include "hydra_internal.h"

namespace {

constexpr int64_t kMaxDim = (int64_t(1) << 31) - 1;
// Largest K: a 256-row slab of W must stay addressable with 32-bit byte offsets.
constexpr int64_t kMaxK = int64_t(1) << 21;
constexpr int kDecodeMaxRows = 16;
// Largest row count (tokens) of the linear, scoring and backward calls and
// largest output width (N, V).  A dispatch counts its work-items in 32 bits;
// with these limits every launch fits, the MFMA tile grids being checked on
// top (grid_ok).
constexpr int64_t kMaxRows = int64_t(1) << 20;
constexpr int64_t kMaxCols = int64_t(1) << 21;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
bool dim_ok(int64_t v) { return v >= 1 && v <= kMaxDim; }
bool grid_ok(int64_t blocks, int64_t threads) { return blocks >= 1 && blocks * threads < (int64_t(1) << 32); }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// M rows, N outputs, K inputs of one LoRA-switchable linear (and of the GEMM
// of the backward): K a multiple of 8 up to 2^21, the limits above, and the
// dual GEMM's tile grid within one dispatch.
bool linear_shape_ok(int64_t M, int64_t N, int64_t K) {
  return M >= 1 && M <= kMaxRows && N >= 1 && N <= kMaxCols && K >= 1 && K <= kMaxK && K % 8 == 0 &&
         grid_ok(cdiv(M, hydra::kGemmTileM) * cdiv(N, hydra::kGemmTileN), hydra::kGemmThreads);
}

hydra_status from_hip(hipError_t e) { return e == hipSuccess ? HYDRA_OK : HYDRA_ERR_HIP; }

// Column tiles of the fused scoring GEMM and the workspace they need.
int64_t score_tiles(int64_t V) { return (V + hydra::kScoreTileN - 1) / hydra::kScoreTileN; }
size_t score_part_bytes(int64_t M, int64_t V) { return size_t(M) * size_t(score_tiles(V)) * sizeof(float4); }
// Workspace of hydra_score: per (row, column tile) partials, then per row the
// gathered token logits (2 fp32), then (16-byte aligned) per row the bf16 hi
// and lo parts of s * h A^T (room for 2 x 128 bf16), then per vocabulary row
// B zero padded to the padded rank (room for 128 bf16), then (16-byte
// aligned) the LoRA pre-pass's partial sums over K chunks (room for 8 chunks
// x 128 fp32 per row).
size_t score_zt_offset(int64_t M, int64_t V) { return score_part_bytes(M, V); }
size_t score_ts_offset(int64_t M, int64_t V) {
  return (score_zt_offset(M, V) + size_t(M) * 2 * sizeof(float) + 15) & ~size_t(15);
}
size_t score_bp_offset(int64_t M, int64_t V) { return score_ts_offset(M, V) + size_t(M) * 2 * HYDRA_MAX_RANK * 2; }
size_t score_part_offset(int64_t M, int64_t V) {
  return (score_bp_offset(M, V) + size_t(V) * HYDRA_MAX_RANK * 2 + 15) & ~size_t(15);
}
size_t score_ws_bytes(int64_t M, int64_t V) {
  return score_part_offset(M, V) + size_t(hydra::kTpreMaxChunks) * size_t(M) * HYDRA_MAX_RANK * 4;
}

// Workspace of the GEMM's LoRA pre-pass: ts [M][2 RP] bf16, then (16-byte
// aligned) bp [N][RP] bf16, then (16-byte aligned) the partial sums over K
// chunks [8][M][RP] fp32.
size_t linear_bp_offset(int64_t M, int rp) { return (size_t(M) * 2 * rp * 2 + 15) & ~size_t(15); }
size_t linear_part_offset(int64_t M, int64_t N, int rp) {
  return (linear_bp_offset(M, rp) + size_t(N) * rp * 2 + 15) & ~size_t(15);
}
size_t linear_ws_bytes(int64_t M, int64_t N, int rp) {
  return rp == 0 ? 0 : linear_part_offset(M, N, rp) + size_t(hydra::kTpreMaxChunks) * size_t(M) * rp * 4;
}

}  // namespace

extern "C" {

hydra_status hydra_lora_linear(const uint16_t* x, const uint16_t* W, const uint16_t* A, const uint16_t* B, float s,
                               int64_t M, int64_t N, int64_t K, int64_t r, float* y_off, float* y_on,
                               void* stream) {
  return hydra_lora_linear_group(1, &x, &W, &A, &B, &s, M, N, K, r, &y_off, &y_on, stream);
}

}  // extern "C"

namespace {

// Argument checks of a group call (host only); fills g and any_on.
hydra_status group_check(int64_t G, const uint16_t* const* x, const uint16_t* const* W, const uint16_t* const* A,
                         const uint16_t* const* B, const float* s, int64_t M, int64_t N, int64_t K, int64_t r,
                         float* const* y_off, float* const* y_on, hydra::GroupArgs& g, bool& any_on) {
  if (G < 1 || G > HYDRA_MAX_GROUP) return HYDRA_ERR_SHAPE;
  if (!x || !W || !s) return HYDRA_ERR_NULL;
  if (!y_off && !y_on) return HYDRA_ERR_NULL;
  if (!linear_shape_ok(M, N, K)) return HYDRA_ERR_SHAPE;
  if (r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  g = hydra::GroupArgs{};
  g.G = int(G);
  g.M = int(M);
  g.N = int(N);
  g.K = int(K);
  g.r = int(r);
  any_on = false;
  for (int64_t i = 0; i < G; ++i) {
    float* yo = y_off ? y_off[i] : nullptr;
    float* yn = y_on ? y_on[i] : nullptr;
    if (!x[i] || !W[i]) return HYDRA_ERR_NULL;
    if (!yo && !yn) return HYDRA_ERR_NULL;
    if (yo && yo == yn) return HYDRA_ERR_SHAPE;
    const bool lora = yn && r > 0;
    const uint16_t* Ai = A ? A[i] : nullptr;
    const uint16_t* Bi = B ? B[i] : nullptr;
    if (lora && (!Ai || !Bi)) return HYDRA_ERR_NULL;
    if (!aligned(x[i], 16) || !aligned(W[i], 16)) return HYDRA_ERR_ALIGN;
    if (lora && (!aligned(Ai, 16) || !aligned(Bi, 2))) return HYDRA_ERR_ALIGN;
    if ((yo && !aligned(yo, 4)) || (yn && !aligned(yn, 4))) return HYDRA_ERR_ALIGN;
    g.x[i] = x[i];
    g.W[i] = W[i];
    g.A[i] = lora ? Ai : nullptr;
    g.B[i] = lora ? Bi : nullptr;
    g.y_off[i] = yo;
    g.y_on[i] = yn;
    g.s[i] = s[i];
    any_on = any_on || lora;
  }
  return HYDRA_OK;
}

// M > 16, padded rank <= 64: one dual GEMM per member.
hydra_status group_gemm(const hydra::GroupArgs& g, hipStream_t st) {
  for (int i = 0; i < g.G; ++i) {
    hydra::LinearArgs a{};
    a.x = g.x[i];
    a.W = g.W[i];
    a.A = g.A[i];
    a.B = g.B[i];
    a.s = g.s[i];
    a.M = g.M;
    a.N = g.N;
    a.K = g.K;
    a.r = g.A[i] ? g.r : 0;
    a.y_off = g.y_off[i];
    a.y_on = g.y_on[i];
    const hipError_t e = hydra::launch_lora_gemm(a, st);
    if (e != hipSuccess) return HYDRA_ERR_HIP;
  }
  return HYDRA_OK;
}

}  // namespace

extern "C" {

hydra_status hydra_lora_linear_group(int64_t G, const uint16_t* const* x, const uint16_t* const* W,
                                     const uint16_t* const* A, const uint16_t* const* B, const float* s, int64_t M,
                                     int64_t N, int64_t K, int64_t r, float* const* y_off, float* const* y_on,
                                     void* stream) {
  hydra::GroupArgs g{};
  bool any_on = false;
  const hydra_status chk = group_check(G, x, W, A, B, s, M, N, K, r, y_off, y_on, g, any_on);
  if (chk != HYDRA_OK) return chk;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (M <= kDecodeMaxRows) {
    // y_on of a member without an adapter equals its y_off: the kernel's
    // update adds s * 0 there, because that member's A and B read as zeros.
    if (!any_on) g.r = 0;
    return from_hip(hydra::launch_lora_gemv_group(g, st));
  }
  if (any_on && hydra::padded_rank(g.r) > 64) return HYDRA_ERR_WORKSPACE;  // see hydra_lora_linear_ws
  return group_gemm(g, st);
}

}  // extern "C"

namespace {
// Workspace of hydra_lora_linear_group_ws: the control words and the tagged
// T slots of the single-launch decode (a fixed size, whatever the shape),
// then above 16 rows at padded rank 128 one pre-pass workspace of
// hydra_lora_linear_ws per member, so the T slots are never overwritten and
// the members' pre-passes can run in the same launches.
size_t group_ws_bytes(int64_t G, int64_t M, int64_t N, int rp) {
  return hydra::kFusedWsBytes + (M > kDecodeMaxRows && rp > 64 ? size_t(G) * linear_ws_bytes(M, N, rp) : 0);
}
}  // namespace

extern "C" {

hydra_status hydra_lora_linear_group_workspace_bytes(int64_t G, int64_t M, int64_t N, int64_t r, size_t* bytes) {
  if (!bytes) return HYDRA_ERR_NULL;
  if (G < 1 || G > HYDRA_MAX_GROUP || M < 1 || M > kMaxRows || N < 1 || N > kMaxCols || r < 0 ||
      r > HYDRA_MAX_RANK)
    return HYDRA_ERR_SHAPE;
  *bytes = group_ws_bytes(G, M, N, hydra::padded_rank(int(r)));
  return HYDRA_OK;
}

hydra_status hydra_lora_linear_group_ws(int64_t G, const uint16_t* const* x, const uint16_t* const* W,
                                        const uint16_t* const* A, const uint16_t* const* B, const float* s,
                                        int64_t M, int64_t N, int64_t K, int64_t r, float* const* y_off,
                                        float* const* y_on, void* workspace, size_t workspace_bytes,
                                        void* stream) {
  hydra::GroupArgs g{};
  bool any_on = false;
  const hydra_status chk = group_check(G, x, W, A, B, s, M, N, K, r, y_off, y_on, g, any_on);
  if (chk != HYDRA_OK) return chk;
  const int rp = any_on ? hydra::padded_rank(int(r)) : 0;
  if (!workspace) return HYDRA_ERR_NULL;
  if (workspace_bytes < group_ws_bytes(G, M, N, hydra::padded_rank(int(r))))
    return HYDRA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (!any_on) g.r = 0;
  if (M <= hydra::kStreamRows) return from_hip(hydra::launch_gemv_fused(g, workspace, st));
  if (M <= kDecodeMaxRows) {
    if (rp <= 64) return from_hip(hydra::launch_lora_gemv_group(g, st));
    // rank 128 above 8 rows: the two row halves in turn
    hydra::GroupArgs lo = g, hi = g;
    lo.M = hydra::kStreamRows;
    hi.M = g.M - hydra::kStreamRows;
    for (int i = 0; i < g.G; ++i) {
      hi.x[i] = g.x[i] + size_t(hydra::kStreamRows) * g.K;
      hi.y_off[i] = g.y_off[i] ? g.y_off[i] + size_t(hydra::kStreamRows) * g.N : nullptr;
      hi.y_on[i] = g.y_on[i] ? g.y_on[i] + size_t(hydra::kStreamRows) * g.N : nullptr;
    }
    const hipError_t e = hydra::launch_gemv_fused(lo, workspace, st);
    return from_hip(e != hipSuccess ? e : hydra::launch_gemv_fused(hi, workspace, st));
  }
  if (rp <= 64) return group_gemm(g, st);
  // rank 128 above 16 rows: each member through the pre-pass GEMM over a workspace body of its own.  When the GEMM
  // reads every member's B as it is (rows of exactly the padded rank, 16-byte aligned), the members' pre-passes
  // run together, in one pair of launches, before the GEMMs; otherwise each member in turn, padding its B.
  const size_t body_bytes = linear_ws_bytes(M, N, rp);
  uint8_t* const body0 = static_cast<uint8_t*>(workspace) + hydra::kFusedWsBytes;
  hydra::LinearArgs la[hydra::kMaxGroup];
  hydra::TpreArgs ta[hydra::kMaxGroup];
  int nj = 0;
  bool together = true;
  for (int i = 0; i < g.G; ++i) {
    hydra::LinearArgs& a = la[i];
    a = hydra::LinearArgs{};
    a.x = g.x[i];
    a.W = g.W[i];
    a.A = g.A[i];
    a.B = g.B[i];
    a.s = g.s[i];
    a.M = g.M;
    a.N = g.N;
    a.K = g.K;
    a.r = g.A[i] ? g.r : 0;
    a.y_off = g.y_off[i];
    a.y_on = g.y_on[i];
    if (a.r > 0 && a.y_on) {
      uint8_t* body = body0 + size_t(i) * body_bytes;
      hydra::TpreArgs& t = ta[nj++];
      t = hydra::TpreArgs{};
      t.x = a.x;
      t.A = a.A;
      t.B = a.B;
      t.s = a.s;
      t.M = a.M;
      t.N = a.N;
      t.K = a.K;
      t.r = a.r;
      t.ts = reinterpret_cast<uint16_t*>(body);
      t.bp = reinterpret_cast<uint16_t*>(body + linear_bp_offset(M, rp));
      t.part = reinterpret_cast<float*>(body + linear_part_offset(M, N, rp));
      together = together && a.r == rp && aligned(a.B, 16);
    }
  }
  if (together && nj > 1) {
    if (hydra::launch_lora_tpre_multi(ta, nj, rp, st) != hipSuccess) return HYDRA_ERR_HIP;
    int j = 0;
    for (int i = 0; i < g.G; ++i) {
      const hydra::LinearArgs& a = la[i];
      const hipError_t e = a.r > 0 && a.y_on ? hydra::launch_lora_gemm_slabs(a, ta[j++].ts, a.B, rp, st)
                                             : hydra::launch_lora_gemm(a, st);
      if (e != hipSuccess) return HYDRA_ERR_HIP;
    }
    return HYDRA_OK;
  }
  for (int i = 0; i < g.G; ++i) {
    uint8_t* body = body0 + size_t(i) * body_bytes;
    const hipError_t e = hydra::launch_lora_gemm_tpre(
        la[i], reinterpret_cast<uint16_t*>(body), reinterpret_cast<uint16_t*>(body + linear_bp_offset(M, rp)),
        reinterpret_cast<float*>(body + linear_part_offset(M, N, rp)), st);
    if (e != hipSuccess) return HYDRA_ERR_HIP;
  }
  return HYDRA_OK;
}

hydra_status hydra_lora_linear_workspace_bytes(int64_t M, int64_t N, int64_t r, size_t* bytes) {
  if (!bytes) return HYDRA_ERR_NULL;
  if (M < 1 || M > kMaxRows || N < 1 || N > kMaxCols || r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  *bytes = linear_ws_bytes(M, N, hydra::padded_rank(int(r)));
  return HYDRA_OK;
}

hydra_status hydra_lora_linear_ws(const uint16_t* x, const uint16_t* W, const uint16_t* A, const uint16_t* B,
                                  float s, int64_t M, int64_t N, int64_t K, int64_t r, float* y_off, float* y_on,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  if (!x || !W) return HYDRA_ERR_NULL;
  if (!y_off && !y_on) return HYDRA_ERR_NULL;
  if (!linear_shape_ok(M, N, K)) return HYDRA_ERR_SHAPE;
  if (r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  const bool lora = y_on && r > 0;
  if (lora && (!A || !B)) return HYDRA_ERR_NULL;
  if (y_off && y_off == y_on) return HYDRA_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(W, 16)) return HYDRA_ERR_ALIGN;
  if (lora && (!aligned(A, 16) || !aligned(B, 2))) return HYDRA_ERR_ALIGN;
  if ((y_off && !aligned(y_off, 4)) || (y_on && !aligned(y_on, 4))) return HYDRA_ERR_ALIGN;
  if (M <= kDecodeMaxRows || !lora)  // no GEMM update: the workspace is not used
    return hydra_lora_linear_group(1, &x, &W, &A, &B, &s, M, N, K, lora ? r : 0, &y_off, &y_on, stream);
  const int rp = hydra::padded_rank(int(r));
  const size_t need = linear_ws_bytes(M, N, rp);
  if (!workspace) return HYDRA_ERR_NULL;
  if (workspace_bytes < need) return HYDRA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  hydra::LinearArgs a{};
  a.x = x;
  a.W = W;
  a.A = A;
  a.B = B;
  a.s = s;
  a.M = int(M);
  a.N = int(N);
  a.K = int(K);
  a.r = int(r);
  a.y_off = y_off;
  a.y_on = y_on;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  return from_hip(hydra::launch_lora_gemm_tpre(a, reinterpret_cast<uint16_t*>(ws),
                                               reinterpret_cast<uint16_t*>(ws + linear_bp_offset(M, rp)),
                                               reinterpret_cast<float*>(ws + linear_part_offset(M, N, rp)),
                                               reinterpret_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {
// Argument checks of the multi-input linear (host only; the rank limit of the
// plain call is checked by the caller).
hydra_status multi_check(const uint16_t* x_off, const uint16_t* W, int64_t n_on, const uint16_t* const* x_on,
                         const uint16_t* const* A, const uint16_t* const* B, const float* s, int64_t M, int64_t N,
                         int64_t K, int64_t r, float* y_off, float* const* y_on) {
  if (!W) return HYDRA_ERR_NULL;
  if (n_on < 0 || n_on > HYDRA_MAX_ADAPTERS) return HYDRA_ERR_SHAPE;
  if ((x_off == nullptr) != (y_off == nullptr)) return HYDRA_ERR_NULL;
  if (!x_off && n_on == 0) return HYDRA_ERR_NULL;
  if (n_on > 0 && (!x_on || !y_on || !s || (r > 0 && (!A || !B)))) return HYDRA_ERR_NULL;
  if (!linear_shape_ok(M, N, K)) return HYDRA_ERR_SHAPE;
  if (r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  if (!aligned(W, 16) || (x_off && !aligned(x_off, 16)) || (y_off && !aligned(y_off, 4))) return HYDRA_ERR_ALIGN;
  for (int64_t a = 0; a < n_on; ++a) {
    if (!x_on[a] || !y_on[a] || (r > 0 && (!A[a] || !B[a]))) return HYDRA_ERR_NULL;
    if (!aligned(x_on[a], 16) || !aligned(y_on[a], 4)) return HYDRA_ERR_ALIGN;
    if (r > 0 && (!aligned(A[a], 16) || !aligned(B[a], 2))) return HYDRA_ERR_ALIGN;
    if (y_on[a] == y_off) return HYDRA_ERR_SHAPE;
    for (int64_t b = 0; b < a; ++b)
      if (y_on[b] == y_on[a]) return HYDRA_ERR_SHAPE;
  }
  return HYDRA_OK;
}
}  // namespace

extern "C" {

hydra_status hydra_lora_linear_multi(const uint16_t* x_off, const uint16_t* W, int64_t n_on,
                                     const uint16_t* const* x_on, const uint16_t* const* A,
                                     const uint16_t* const* B, const float* s, int64_t M, int64_t N, int64_t K,
                                     int64_t r, float* y_off, float* const* y_on, void* stream) {
  const hydra_status chk = multi_check(x_off, W, n_on, x_on, A, B, s, M, N, K, r, y_off, y_on);
  if (chk != HYDRA_OK) return chk;
  // Above the decode sizes the adapters run on the dual GEMM, which holds
  // ranks up to 64 (hydra_lora_linear_ws serves rank 128 there): rejected
  // here, before the LoRA-off output is launched.
  if (M > kDecodeMaxRows && n_on > 0 && r > 0 && hydra::padded_rank(int(r)) > 64) return HYDRA_ERR_WORKSPACE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (M > hydra::kStreamRows) {
    // One launch per input (the MFMA kernels are bound by arithmetic, not by reads of W).
    if (x_off) {
      const hydra_status e = hydra_lora_linear(x_off, W, nullptr, nullptr, 0.f, M, N, K, 0, y_off, nullptr, stream);
      if (e != HYDRA_OK) return e;
    }
    for (int64_t a = 0; a < n_on; ++a) {
      const hydra_status e = hydra_lora_linear(x_on[a], W, r > 0 ? A[a] : nullptr, r > 0 ? B[a] : nullptr, s[a], M,
                                               N, K, r, nullptr, y_on[a], stream);
      if (e != HYDRA_OK) return e;
    }
    return HYDRA_OK;
  }
  // Decode shape: the inputs' rows are stacked, up to kStreamRows rows per
  // pass, and every pass reads W once for all of its rows; then the LoRA
  // update of each y_on.
  const int n_in = (x_off ? 1 : 0) + int(n_on);
  hydra::StreamArgs sa{};
  auto fresh = [&]() {
    sa = hydra::StreamArgs{};
    sa.G = 1;
    sa.seg_rows = int(M);
    sa.N = int(N);
    sa.K = int(K);
    sa.W[0] = W;
  };
  fresh();
  for (int i = 0; i < n_in; ++i) {
    const bool off = x_off && i == 0;
    if ((sa.nseg[0] + 1) * M > hydra::kStreamRows) {
      if (hydra::launch_gemv_stream(sa, st) != hipSuccess) return HYDRA_ERR_HIP;
      fresh();
    }
    const int sg = sa.nseg[0]++;
    sa.x[sg] = off ? x_off : x_on[i - (x_off ? 1 : 0)];
    sa.ya[sg] = off ? y_off : y_on[i - (x_off ? 1 : 0)];
  }
  if (hydra::launch_gemv_stream(sa, st) != hipSuccess) return HYDRA_ERR_HIP;
  if (r == 0 || n_on == 0) return HYDRA_OK;
  hydra::GroupArgs g{};
  g.G = int(n_on);
  g.M = int(M);
  g.N = int(N);
  g.K = int(K);
  g.r = int(r);
  for (int64_t a = 0; a < n_on; ++a) {
    g.x[a] = x_on[a];
    g.A[a] = A[a];
    g.B[a] = B[a];
    g.y_on[a] = y_on[a];
    g.s[a] = s[a];
  }
  return from_hip(hydra::launch_lora_update(g, st));
}

hydra_status hydra_lora_linear_multi_workspace_bytes(int64_t M, int64_t N, int64_t r, size_t* bytes) {
  return hydra_lora_linear_workspace_bytes(M, N, r, bytes);
}

hydra_status hydra_lora_linear_multi_ws(const uint16_t* x_off, const uint16_t* W, int64_t n_on,
                                        const uint16_t* const* x_on, const uint16_t* const* A,
                                        const uint16_t* const* B, const float* s, int64_t M, int64_t N, int64_t K,
                                        int64_t r, float* y_off, float* const* y_on, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  const hydra_status chk = multi_check(x_off, W, n_on, x_on, A, B, s, M, N, K, r, y_off, y_on);
  if (chk != HYDRA_OK) return chk;
  if (!workspace) return HYDRA_ERR_NULL;
  const int rp = hydra::padded_rank(int(r));
  const bool pre = M > kDecodeMaxRows && n_on > 0 && rp > 64;  // the adapters take the pre-pass GEMM
  if (pre && workspace_bytes < linear_ws_bytes(M, N, rp)) return HYDRA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  if (!pre) return hydra_lora_linear_multi(x_off, W, n_on, x_on, A, B, s, M, N, K, r, y_off, y_on, stream);
  // one GEMM per input: the LoRA-off input on the dual GEMM without adapter,
  // each adapter's input through the pre-pass GEMM, sharing the workspace
  if (x_off) {
    const hydra_status e = hydra_lora_linear(x_off, W, nullptr, nullptr, 0.f, M, N, K, 0, y_off, nullptr, stream);
    if (e != HYDRA_OK) return e;
  }
  for (int64_t a = 0; a < n_on; ++a) {
    const hydra_status e = hydra_lora_linear_ws(x_on[a], W, A[a], B[a], s[a], M, N, K, r, nullptr, y_on[a], workspace,
                                                workspace_bytes, stream);
    if (e != HYDRA_OK) return e;
  }
  return HYDRA_OK;
}

hydra_status hydra_score_workspace_bytes(int64_t M, int64_t V, size_t* bytes) {
  if (!bytes) return HYDRA_ERR_NULL;
  if (M < 1 || M > kMaxRows || V < 1 || V > kMaxCols) return HYDRA_ERR_SHAPE;
  *bytes = score_ws_bytes(M, V);
  return HYDRA_OK;
}

}  // extern "C"

namespace {

// Argument checks of the fused scoring pass, except the workspace (host only).
hydra_status score_check(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B,
                         const int32_t* tokens, const uint16_t* w_rm, int64_t n_seq, int64_t seq_len, int64_t K,
                         int64_t V, int64_t r, float* lp_on, float* lp_off, float* kl, float* reward,
                         float* lse_on, float* lse_off, int32_t* err_flag) {
  if (!h || !W_lm || !tokens || !lp_on || !lp_off || !kl) return HYDRA_ERR_NULL;
  if (!dim_ok(n_seq) || !dim_ok(seq_len) || !dim_ok(K) || !dim_ok(V) || (K % 8) != 0 || K > kMaxK)
    return HYDRA_ERR_SHAPE;
  if (n_seq > kMaxDim / seq_len) return HYDRA_ERR_SHAPE;
  const int64_t M = n_seq * seq_len;
  if (M > kMaxRows || V > kMaxCols) return HYDRA_ERR_SHAPE;
  if (!grid_ok(cdiv(M, hydra::kScoreTileM) * cdiv(V, hydra::kScoreTileN), hydra::kScoreThreads))
    return HYDRA_ERR_SHAPE;
  if (r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  if (r > 0 && (!A || !B)) return HYDRA_ERR_NULL;
  if (!aligned(h, 16) || !aligned(W_lm, 16)) return HYDRA_ERR_ALIGN;
  if (r > 0 && (!aligned(A, 16) || !aligned(B, 2))) return HYDRA_ERR_ALIGN;
  if (!aligned(tokens, 4) || !aligned(lp_on, 4) || !aligned(lp_off, 4) || !aligned(kl, 4)) return HYDRA_ERR_ALIGN;
  if ((reward && !aligned(reward, 4)) || (lse_on && !aligned(lse_on, 4)) || (lse_off && !aligned(lse_off, 4)) ||
      (err_flag && !aligned(err_flag, 4)) || (w_rm && !aligned(w_rm, 2)))
    return HYDRA_ERR_ALIGN;
  return HYDRA_OK;
}

// The fused scoring pass's launches over a checked workspace of at least
// score_ws_bytes(M, V) bytes, 16-byte aligned.
hydra_status score_launch(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B, float s,
                          const int32_t* tokens, const uint16_t* w_rm, int64_t n_seq, int64_t seq_len, int64_t K,
                          int64_t V, int64_t r, float* lp_on, float* lp_off, float* kl, float* reward,
                          float* lse_on, float* lse_off, void* workspace, int32_t* err_flag, hipStream_t st,
                          const uint16_t* h_act = nullptr) {
  const int64_t M = n_seq * seq_len;
  float4* part = reinterpret_cast<float4*>(workspace);
  float* zt = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + score_zt_offset(M, V));
  uint16_t* ts = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(workspace) + score_ts_offset(M, V));
  uint16_t* bp = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(workspace) + score_bp_offset(M, V));

  hydra::ScoreGemmArgs g{};
  g.lin.x = h;
  g.lin.W = W_lm;
  g.lin.A = r > 0 ? A : nullptr;
  g.lin.B = r > 0 ? B : nullptr;
  g.lin.s = s;
  g.lin.M = int(M);
  g.lin.N = int(V);
  g.lin.K = int(K);
  g.lin.r = int(r);
  g.tokens = tokens;
  g.part = part;
  g.zt = zt;
  g.ts = ts;
  g.bp = bp;
  g.bp_buf = bp;
  g.tpart = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + score_part_offset(M, V));
  g.ntn = int(score_tiles(V));
  g.x_act = h_act;
  hipError_t e = hydra::launch_score_gemm(g, st);
  if (e != hipSuccess) return HYDRA_ERR_HIP;

  hydra::CombineArgs c{};
  c.part = part;
  c.zt = zt;
  c.tokens = tokens;
  c.M = int(M);
  c.V = int(V);
  c.ntn = g.ntn;
  c.lp_on = lp_on;
  c.lp_off = lp_off;
  c.kl = kl;
  c.lse_on = lse_on;
  c.lse_off = lse_off;
  c.err = err_flag;
  c.h = h;
  c.w_rm = w_rm;
  c.reward = reward;
  c.n_seq = int(n_seq);
  c.seq_len = int(seq_len);
  c.K = int(K);
  return from_hip(hydra::launch_score_combine(c, st));
}

// Device scratch of hydra_score_noalloc: a file-scope device array, one copy
// on every GPU the library runs on, held until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is used.
__device__ __align__(256) uint8_t scratch[HYDRA_SCORE_NOALLOC_MAX_BYTES];

constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// Device address of `scratch` on the device of `stream` (the current device for
// the null stream).
hipError_t scratch_address(hipStream_t stream, void** out) {
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  int dev = cur;
  if (stream != nullptr) {
    hipDevice_t d = 0;
    e = hipStreamGetDevice(stream, &d);
    if (e != hipSuccess) return e;
    dev = int(d);
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(g_scratch_once[dev], [dev, cur]() {
    hipError_t err = hipSuccess;
    if (dev != cur) err = hipSetDevice(dev);
    void* p = nullptr;
    if (err == hipSuccess) err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t back = hipSetDevice(cur);
      if (err == hipSuccess) err = back;
    }
    g_scratch_ptr[dev] = err == hipSuccess ? p : nullptr;
    g_scratch_err[dev] = err;
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  *out = g_scratch_ptr[dev];
  return *out != nullptr ? hipSuccess : hipErrorInvalidSymbol;
}

}  // namespace

extern "C" {

hydra_status hydra_score(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B, float s,
                         const int32_t* tokens, const uint16_t* w_rm, int64_t n_seq, int64_t seq_len, int64_t K,
                         int64_t V, int64_t r, float* lp_on, float* lp_off, float* kl, float* reward,
                         float* lse_on, float* lse_off, void* workspace, size_t workspace_bytes, int32_t* err_flag,
                         void* stream) {
  const hydra_status chk = score_check(h, W_lm, A, B, tokens, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl,
                                       reward, lse_on, lse_off, err_flag);
  if (chk != HYDRA_OK) return chk;
  if (!workspace) return HYDRA_ERR_WORKSPACE;
  if (workspace_bytes < score_ws_bytes(n_seq * seq_len, V)) return HYDRA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  return score_launch(h, W_lm, A, B, s, tokens, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl, reward, lse_on,
                      lse_off, workspace, err_flag, reinterpret_cast<hipStream_t>(stream));
}

hydra_status hydra_score_two_input(const uint16_t* h_act, const uint16_t* h_off, const uint16_t* W_lm,
                                   const uint16_t* A, const uint16_t* B, float s, const int32_t* tokens,
                                   const uint16_t* w_rm, int64_t n_seq, int64_t seq_len, int64_t K, int64_t V,
                                   int64_t r, float* lp_on, float* lp_off, float* kl, float* reward, float* lse_on,
                                   float* lse_off, void* workspace, size_t workspace_bytes, int32_t* err_flag,
                                   void* stream) {
  if (!h_act) return HYDRA_ERR_NULL;
  const hydra_status chk = score_check(h_off, W_lm, A, B, tokens, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl,
                                       reward, lse_on, lse_off, err_flag);
  if (chk != HYDRA_OK) return chk;
  const int64_t M = n_seq * seq_len;
  // twice the row tiles of the one-input pass
  if (!grid_ok(2 * cdiv(M, hydra::kScoreTileM) * cdiv(V, hydra::kScoreTileN), hydra::kScoreThreads))
    return HYDRA_ERR_SHAPE;
  if (!aligned(h_act, 16)) return HYDRA_ERR_ALIGN;
  if (!workspace) return HYDRA_ERR_WORKSPACE;
  if (workspace_bytes < score_ws_bytes(M, V)) return HYDRA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  return score_launch(h_off, W_lm, A, B, s, tokens, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl, reward, lse_on,
                      lse_off, workspace, err_flag, reinterpret_cast<hipStream_t>(stream), h_act);
}

hydra_status hydra_score_noalloc(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B,
                                 float s, const int32_t* tokens, const uint16_t* w_rm, int64_t n_seq,
                                 int64_t seq_len, int64_t K, int64_t V, int64_t r, float* lp_on, float* lp_off,
                                 float* kl, float* reward, float* lse_on, float* lse_off, int32_t* err_flag,
                                 void* stream) {
  const hydra_status chk = score_check(h, W_lm, A, B, tokens, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl,
                                       reward, lse_on, lse_off, err_flag);
  if (chk != HYDRA_OK) return chk;
  if (score_ws_bytes(n_seq * seq_len, V) > size_t(HYDRA_SCORE_NOALLOC_MAX_BYTES)) return HYDRA_ERR_WORKSPACE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  void* ws = nullptr;
  if (scratch_address(st, &ws) != hipSuccess) return HYDRA_ERR_HIP;
  return score_launch(h, W_lm, A, B, s, tokens, w_rm, n_seq, seq_len, K, V, r, lp_on, lp_off, kl, reward, lse_on,
                      lse_off, ws, err_flag, st);
}

hydra_status hydra_value_head(const uint16_t* h, const uint16_t* w_v, int64_t M, int64_t K, float* values,
                              void* stream) {
  if (!h || !w_v || !values) return HYDRA_ERR_NULL;
  if (M < 1 || M > kMaxRows || !dim_ok(K) || (K % 8) != 0 || K > kMaxK) return HYDRA_ERR_SHAPE;
  if (!aligned(h, 16) || !aligned(w_v, 16) || !aligned(values, 4)) return HYDRA_ERR_ALIGN;
  hydra::ValueHeadArgs a{};
  a.h = h;
  a.w = w_v;
  a.M = int(M);
  a.K = int(K);
  a.values = values;
  return from_hip(hydra::launch_value_head(a, reinterpret_cast<hipStream_t>(stream)));
}

hydra_status hydra_ppo_loss(const float* lp_new, const float* lp_old, const float* advantages, const float* values,
                            const float* returns, int64_t n_seq, int64_t seq_len, int64_t start, float eps,
                            float* losses, float* d_lp, float* d_v, void* stream) {
  if (!lp_new || !lp_old || !advantages || !values || !returns || !losses) return HYDRA_ERR_NULL;
  if (!dim_ok(n_seq) || !dim_ok(seq_len) || n_seq > kMaxRows / seq_len) return HYDRA_ERR_SHAPE;  // M <= 2^20
  if (start < 0 || start >= seq_len) return HYDRA_ERR_SHAPE;
  if (!(eps >= 0.f && eps < 1.f)) return HYDRA_ERR_SHAPE;
  const void* ins[5] = {lp_new, lp_old, advantages, values, returns};
  const void* outs[3] = {losses, d_lp, d_v};
  for (const void* o : outs) {
    if (!o) continue;
    for (const void* i : ins)
      if (o == i) return HYDRA_ERR_SHAPE;
  }
  if (losses == d_lp || losses == d_v || (d_lp && d_lp == d_v)) return HYDRA_ERR_SHAPE;
  for (const void* p : ins)
    if (!aligned(p, 4)) return HYDRA_ERR_ALIGN;
  for (const void* p : outs)
    if (p && !aligned(p, 4)) return HYDRA_ERR_ALIGN;
  hydra::PpoLossArgs a{};
  a.lp_new = lp_new;
  a.lp_old = lp_old;
  a.adv = advantages;
  a.values = values;
  a.returns = returns;
  a.n_seq = int(n_seq);
  a.seq_len = int(seq_len);
  a.start = int(start);
  a.eps = eps;
  a.losses = losses;
  a.d_lp = d_lp;
  a.d_v = d_v;
  return from_hip(hydra::launch_ppo_loss(a, reinterpret_cast<hipStream_t>(stream)));
}

hydra_status hydra_transpose_bf16(const uint16_t* src, int64_t R, int64_t C, uint16_t* dst, void* stream) {
  if (!src || !dst) return HYDRA_ERR_NULL;
  if (R < 1 || C < 1 || R > kMaxK || C > kMaxK || !grid_ok(cdiv(R, 64) * cdiv(C, 64), 256)) return HYDRA_ERR_SHAPE;
  if (static_cast<const void*>(src) == static_cast<const void*>(dst)) return HYDRA_ERR_SHAPE;
  if (!aligned(src, 2) || !aligned(dst, 2)) return HYDRA_ERR_ALIGN;
  return from_hip(hydra::launch_transpose_pad(src, int(R), int(C), dst, int(R), int(C),
                                              reinterpret_cast<hipStream_t>(stream)));
}

namespace {
// Sizes the backward accepts: N and K both serve as a GEMM's inner dimension
// (multiples of 8, at most 2^21), M as for the forward, and the dx GEMM's
// tile grid ([M x K] output) within one dispatch.
bool backward_shape_ok(int64_t M, int64_t N, int64_t K, int64_t r) {
  return linear_shape_ok(M, K, N) && K % 8 == 0 && r >= 0 && r <= HYDRA_MAX_RANK;
}
}  // namespace

hydra_status hydra_lora_linear_backward_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t r, size_t* bytes) {
  if (!bytes) return HYDRA_ERR_NULL;
  if (!backward_shape_ok(M, N, K, r)) return HYDRA_ERR_SHAPE;
  *bytes = hydra::backward_ws_bytes(int(M), int(N), int(K), hydra::padded_rank(int(r)));
  return HYDRA_OK;
}

hydra_status hydra_lora_linear_backward(const uint16_t* x, const uint16_t* Wt, const uint16_t* A, const uint16_t* B,
                                        float s, const uint16_t* dy, int64_t M, int64_t N, int64_t K, int64_t r,
                                        float* dx, float* dA, float* dB, void* workspace, size_t workspace_bytes,
                                        void* stream) {
  if (!backward_shape_ok(M, N, K, r)) return HYDRA_ERR_SHAPE;
  if (r == 0) dA = dB = nullptr;  // empty
  if (!dx && !dA && !dB) return HYDRA_ERR_NULL;
  if (!dy || (dx && !Wt) || (r > 0 && (!A || !B)) || ((dA || dB) && !x)) return HYDRA_ERR_NULL;
  if ((dx && (dx == dA || dx == dB)) || (dA && dA == dB)) return HYDRA_ERR_SHAPE;
  if (!aligned(dy, 16) || (x && !aligned(x, 16)) || (dx && !aligned(Wt, 16))) return HYDRA_ERR_ALIGN;
  if (r > 0 && (!aligned(A, 16) || !aligned(B, 2))) return HYDRA_ERR_ALIGN;
  if ((dx && !aligned(dx, 4)) || (dA && !aligned(dA, 4)) || (dB && !aligned(dB, 4))) return HYDRA_ERR_ALIGN;
  const size_t need = hydra::backward_ws_bytes(int(M), int(N), int(K), hydra::padded_rank(int(r)));
  if (need > 0) {
    if (!workspace) return HYDRA_ERR_NULL;
    if (workspace_bytes < need) return HYDRA_ERR_WORKSPACE;
    if (!aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  }
  hydra::BackwardArgs a{};
  a.x = x;
  a.Wt = Wt;
  a.A = A;
  a.B = B;
  a.dy = dy;
  a.s = s;
  a.M = int(M);
  a.N = int(N);
  a.K = int(K);
  a.r = int(r);
  a.dx = dx;
  a.dA = dA;
  a.dB = dB;
  return from_hip(hydra::launch_lora_backward(a, workspace, reinterpret_cast<hipStream_t>(stream)));
}

hydra_status hydra_ppo_advantages(const float* kl, const float* reward, const float* values, int64_t n_seq,
                                  int64_t seq_len, int64_t start, float beta, float gamma, float lam, float* rewards,
                                  float* advantages, float* returns, void* stream) {
  if (!kl || !reward || !values || !advantages || !returns) return HYDRA_ERR_NULL;
  if (!dim_ok(n_seq) || !dim_ok(seq_len) || n_seq > kMaxRows / seq_len) return HYDRA_ERR_SHAPE;  // M <= 2^20
  if (start < 0 || start >= seq_len) return HYDRA_ERR_SHAPE;
  // outputs are written while inputs are still read: no output may be an input
  const void* ins[3] = {kl, reward, values};
  const void* outs[3] = {rewards, advantages, returns};
  for (const void* o : outs) {
    if (!o) continue;
    for (const void* i : ins)
      if (o == i) return HYDRA_ERR_SHAPE;
  }
  if (advantages == returns || (rewards && (rewards == advantages || rewards == returns))) return HYDRA_ERR_SHAPE;
  if (!aligned(kl, 4) || !aligned(reward, 4) || !aligned(values, 4) || !aligned(advantages, 4) ||
      !aligned(returns, 4) || (rewards && !aligned(rewards, 4)))
    return HYDRA_ERR_ALIGN;
  hydra::GaeArgs a{};
  a.kl = kl;
  a.reward = reward;
  a.values = values;
  a.n_seq = int(n_seq);
  a.seq_len = int(seq_len);
  a.start = int(start);
  a.beta = beta;
  a.gamma = gamma;
  a.lam = lam;
  a.rewards = rewards;
  a.advantages = advantages;
  a.returns = returns;
  return from_hip(hydra::launch_gae(a, reinterpret_cast<hipStream_t>(stream)));
}

hydra_status hydra_score_logits(const float* logits_on, const float* logits_off, const int32_t* tokens, int64_t M,
                                int64_t V, float* lp_on, float* lp_off, float* kl, float* lse_on, float* lse_off,
                                int32_t* err_flag, void* stream) {
  if (!logits_on || !logits_off || !tokens || !lp_on || !lp_off || !kl) return HYDRA_ERR_NULL;
  if (M < 1 || M > kMaxRows || V < 1 || V > kMaxCols) return HYDRA_ERR_SHAPE;
  if (!aligned(logits_on, 16) || !aligned(logits_off, 16)) return HYDRA_ERR_ALIGN;
  if (!aligned(tokens, 4) || !aligned(lp_on, 4) || !aligned(lp_off, 4) || !aligned(kl, 4)) return HYDRA_ERR_ALIGN;
  if ((lse_on && !aligned(lse_on, 4)) || (lse_off && !aligned(lse_off, 4)) || (err_flag && !aligned(err_flag, 4)))
    return HYDRA_ERR_ALIGN;
  hydra::LogitsArgs o{};
  o.on = logits_on;
  o.off = logits_off;
  o.tokens = tokens;
  o.M = int(M);
  o.V = int(V);
  o.lp_on = lp_on;
  o.lp_off = lp_off;
  o.kl = kl;
  o.lse_on = lse_on;
  o.lse_off = lse_off;
  o.err = err_flag;
  return from_hip(hydra::launch_score_logits(o, reinterpret_cast<hipStream_t>(stream)));
}

const char* hydra_status_string(hydra_status status) {
  switch (status) {
    case HYDRA_OK: return "HYDRA_OK";
    case HYDRA_ERR_NULL: return "HYDRA_ERR_NULL: a required pointer is NULL";
    case HYDRA_ERR_SHAPE: return "HYDRA_ERR_SHAPE: a size is out of range or inconsistent";
    case HYDRA_ERR_ALIGN: return "HYDRA_ERR_ALIGN: a pointer is not aligned as required";
    case HYDRA_ERR_UNSUPPORTED: return "HYDRA_ERR_UNSUPPORTED: valid request that the library does not handle";
    case HYDRA_ERR_WORKSPACE: return "HYDRA_ERR_WORKSPACE: workspace missing or too small";
    case HYDRA_ERR_HIP: return "HYDRA_ERR_HIP: the HIP runtime reported a launch error";
  }
  return "unknown hydra_status";
}

int hydra_abi_version(void) { return 1; }

}  // extern "C"
