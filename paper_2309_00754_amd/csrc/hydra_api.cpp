// C ABI of libhydra: argument validation on the host, then kernel launches on
// the caller's stream.  Validation runs before any HIP call, so every argument
// error is reported without touching the device.
#include "../../include/hydra.h"

#include <hip/hip_runtime.h>

#include "hydra_internal.h"

namespace {

constexpr int64_t kMaxDim = (int64_t(1) << 31) - 1;
// Largest K: a 256-row slab of W must stay addressable with 32-bit byte offsets.
constexpr int64_t kMaxK = int64_t(1) << 21;
constexpr int kDecodeMaxRows = 16;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
bool dim_ok(int64_t v) { return v >= 1 && v <= kMaxDim; }

hydra_status from_hip(hipError_t e) { return e == hipSuccess ? HYDRA_OK : HYDRA_ERR_HIP; }

// Column tiles of the fused scoring GEMM and the workspace they need.
int64_t score_tiles(int64_t V) { return (V + hydra::kScoreTileN - 1) / hydra::kScoreTileN; }
size_t score_part_bytes(int64_t M, int64_t V) { return size_t(M) * size_t(score_tiles(V)) * sizeof(float4); }
size_t score_ws_bytes(int64_t M, int64_t V) { return score_part_bytes(M, V) + size_t(M) * 2 * sizeof(float); }

}  // namespace

extern "C" {

hydra_status hydra_lora_linear(const uint16_t* x, const uint16_t* W, const uint16_t* A, const uint16_t* B, float s,
                               int64_t M, int64_t N, int64_t K, int64_t r, float* y_off, float* y_on,
                               void* stream) {
  if (!x || !W) return HYDRA_ERR_NULL;
  if (!y_off && !y_on) return HYDRA_ERR_NULL;
  if (!dim_ok(M) || !dim_ok(N) || !dim_ok(K) || (K % 8) != 0 || K > kMaxK) return HYDRA_ERR_SHAPE;
  if (r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  if (y_off && y_off == y_on) return HYDRA_ERR_SHAPE;
  const bool lora = y_on && r > 0;
  if (lora && (!A || !B)) return HYDRA_ERR_NULL;
  if (!aligned(x, 16) || !aligned(W, 16)) return HYDRA_ERR_ALIGN;
  if (lora && (!aligned(A, 16) || !aligned(B, 2))) return HYDRA_ERR_ALIGN;
  if ((y_off && !aligned(y_off, 4)) || (y_on && !aligned(y_on, 4))) return HYDRA_ERR_ALIGN;

  hydra::LinearArgs a{};
  a.x = x;
  a.W = W;
  a.A = lora ? A : nullptr;
  a.B = lora ? B : nullptr;
  a.s = s;
  a.M = int(M);
  a.N = int(N);
  a.K = int(K);
  a.r = lora ? int(r) : 0;
  a.y_off = y_off;
  a.y_on = y_on;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (M <= kDecodeMaxRows) return from_hip(hydra::launch_lora_gemv(a, st));
  return from_hip(hydra::launch_lora_gemm(a, st));
}

hydra_status hydra_score_workspace_bytes(int64_t M, int64_t V, size_t* bytes) {
  if (!bytes) return HYDRA_ERR_NULL;
  if (!dim_ok(M) || !dim_ok(V)) return HYDRA_ERR_SHAPE;
  *bytes = score_ws_bytes(M, V);
  return HYDRA_OK;
}

hydra_status hydra_score(const uint16_t* h, const uint16_t* W_lm, const uint16_t* A, const uint16_t* B, float s,
                         const int32_t* tokens, const uint16_t* w_rm, int64_t n_seq, int64_t seq_len, int64_t K,
                         int64_t V, int64_t r, float* lp_on, float* lp_off, float* kl, float* reward,
                         float* lse_on, float* lse_off, void* workspace, size_t workspace_bytes, int32_t* err_flag,
                         void* stream) {
  if (!h || !W_lm || !tokens || !lp_on || !lp_off || !kl) return HYDRA_ERR_NULL;
  if (!dim_ok(n_seq) || !dim_ok(seq_len) || !dim_ok(K) || !dim_ok(V) || (K % 8) != 0 || K > kMaxK)
    return HYDRA_ERR_SHAPE;
  if (n_seq > kMaxDim / seq_len) return HYDRA_ERR_SHAPE;
  const int64_t M = n_seq * seq_len;
  if (r < 0 || r > HYDRA_MAX_RANK) return HYDRA_ERR_SHAPE;
  if (r > 0 && (!A || !B)) return HYDRA_ERR_NULL;
  if (!workspace) return HYDRA_ERR_WORKSPACE;
  if (workspace_bytes < score_ws_bytes(M, V)) return HYDRA_ERR_WORKSPACE;
  if (!aligned(h, 16) || !aligned(W_lm, 16) || !aligned(workspace, 16)) return HYDRA_ERR_ALIGN;
  if (r > 0 && (!aligned(A, 16) || !aligned(B, 2))) return HYDRA_ERR_ALIGN;
  if (!aligned(tokens, 4) || !aligned(lp_on, 4) || !aligned(lp_off, 4) || !aligned(kl, 4)) return HYDRA_ERR_ALIGN;
  if ((reward && !aligned(reward, 4)) || (lse_on && !aligned(lse_on, 4)) || (lse_off && !aligned(lse_off, 4)) ||
      (err_flag && !aligned(err_flag, 4)) || (w_rm && !aligned(w_rm, 2)))
    return HYDRA_ERR_ALIGN;

  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  float4* part = reinterpret_cast<float4*>(workspace);
  float* zt = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + score_part_bytes(M, V));

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
  g.ntn = int(score_tiles(V));
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

hydra_status hydra_score_logits(const float* logits_on, const float* logits_off, const int32_t* tokens, int64_t M,
                                int64_t V, float* lp_on, float* lp_off, float* kl, float* lse_on, float* lse_off,
                                int32_t* err_flag, void* stream) {
  if (!logits_on || !logits_off || !tokens || !lp_on || !lp_off || !kl) return HYDRA_ERR_NULL;
  if (!dim_ok(M) || !dim_ok(V)) return HYDRA_ERR_SHAPE;
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
    case HYDRA_ERR_UNSUPPORTED: return "HYDRA_ERR_UNSUPPORTED: request not handled by this build";
    case HYDRA_ERR_WORKSPACE: return "HYDRA_ERR_WORKSPACE: workspace missing or too small";
    case HYDRA_ERR_HIP: return "HYDRA_ERR_HIP: the HIP runtime reported a launch error";
  }
  return "unknown hydra_status";
}

int hydra_abi_version(void) { return 1; }

}  // extern "C"
