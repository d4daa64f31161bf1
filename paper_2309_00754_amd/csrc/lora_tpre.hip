// Pre-pass of the LoRA update of the MFMA GEMMs (the dual-output linear with
// a workspace, and the fused CLM-head scoring GEMM).  T = x A^T is the same
// for every column tile of a row block, so it is computed once here instead
// of inside every tile (at rank 128 against 256-column tiles the in-tile
// product would add half of the base MFMA work):
//  * lora_t_part_kernel: one workgroup per 16 rows and K chunk (K split into
//    up to 8 chunks of at least 1024, so that many workgroups share the
//    work), 8 waves taking 32-wide k-steps in turn
//    (v_mfma_f32_16x16x32_bf16, fp32 accumulation), their partial tiles
//    summed in LDS in wave order and written to the workspace;
//  * lora_t_finish_kernel: the chunk partials added in chunk order, s * T
//    split into a bf16 hi part and a bf16 lo part (the rounding error of hi),
//    so that the GEMM's bf16 MFMAs add s T B^T to within ~2^-16 relative;
//    extra workgroups pad B to the padded rank when B's own rows cannot be
//    read as they are (r not 16, 32, 64 or 128, or B not 16-byte aligned).
// Both GEMMs then add s T B^T as 2 RP more k values of their main loop:
// rows of [hi | lo] against rows of [Bp | Bp].
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

constexpr int T_WAVES = 8;
constexpr int T_UNROLL = 4;

// Partial T over K chunk blockIdx.y for 16 rows: the 8 waves take the chunk's
// 32-wide k-steps in turn, T_UNROLL at a time (all their loads in flight
// before the first MFMA); their partial tiles are summed in LDS in wave order.
template <int RP>
__global__ __launch_bounds__(T_WAVES * 64) void lora_t_part_kernel(TpreArgs a, int kch) {
  constexpr int TJ = RP / 16;
  __shared__ f32x4_t red[T_WAVES][TJ][64];
  const int M = a.M, K = a.K;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int l16 = lane & 15;
  const int lg = lane >> 4;
  const int m0 = blockIdx.x * 16;
  const int kc = blockIdx.y;
  const __amdgpu_buffer_rsrc_t hrs = make_rsrc(a.x + (size_t)m0 * K, (uint32_t)min(16, M - m0) * K * 2u);
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(a.A, (uint32_t)min(a.r, RP) * K * 2u);
  f32x4_t acc[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int ks0 = kc * (kch / 32);
  const int ks1 = min((K + 31) / 32, ks0 + kch / 32);
  for (int k0 = ks0 + wave; k0 < ks1; k0 += T_WAVES * T_UNROLL) {
    uint4 hf[T_UNROLL], af[T_UNROLL][TJ];
#pragma unroll
    for (int u = 0; u < T_UNROLL; ++u) {
      const int k = (k0 + u * T_WAVES) * 32 + lg * 8;
      const bool kv = k0 + u * T_WAVES < ks1 && k < K;
      hf[u] = buf_load16(hrs, kv ? (l16 * K + k) * 2 : kOutOfRange);
#pragma unroll
      for (int j = 0; j < TJ; ++j) af[u][j] = buf_load16(ars, kv ? ((j * 16 + l16) * K + k) * 2 : kOutOfRange);
    }
#pragma unroll
    for (int u = 0; u < T_UNROLL; ++u)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[j] = mfma16(hf[u], af[u][j], acc[j]);
  }
  // acc[j] lane l holds T[m0 + 4 (l / 16) + i][16 j + l % 16]
#pragma unroll
  for (int j = 0; j < TJ; ++j) red[wave][j][lane] = acc[j];
  __syncthreads();
  for (int e = t; e < 16 * RP; e += T_WAVES * 64) {
    const int rl = e / RP, j = e % RP;
    const int row = m0 + rl;
    if (row >= M) continue;
    const int src = (rl >> 2) * 16 + (j & 15);
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < T_WAVES; ++w) v += red[w][j >> 4][src][rl & 3];
    a.part[((size_t)kc * M + row) * RP + j] = v;
  }
}

// s * T from the chunk partials (added in chunk order), split into bf16 hi and
// lo parts (and / or kept in fp32); the workgroups past the rows write B zero
// padded to RP when the GEMM cannot read B itself.
template <int RP>
__global__ __launch_bounds__(256) void lora_t_finish_kernel(TpreArgs a, int nkc, int tblocks) {
  if ((int)blockIdx.x < tblocks) {
    const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= (size_t)a.M * RP) return;
    const size_t row = e / RP, j = e % RP;
    float v = 0.f;
    for (int c = 0; c < nkc; ++c) v += a.part[((size_t)c * a.M + row) * RP + j];
    v *= a.s;
    if (a.t32) a.t32[e] = v;
    if (a.ts) {
      const uint32_t hi = f32_to_bf16_rne(v);
      const uint32_t lo = f32_to_bf16_rne(v - bf16_to_f32(hi));
      a.ts[row * 2 * RP + j] = (uint16_t)hi;
      a.ts[row * 2 * RP + RP + j] = (uint16_t)lo;
    }
    return;
  }
  const size_t total = (size_t)a.N * RP;
  const size_t nb = gridDim.x - tblocks;
  for (size_t e = (blockIdx.x - tblocks) * 256 + threadIdx.x; e < total; e += nb * 256) {
    const int n = (int)(e / RP), j = (int)(e % RP);
    a.bp[e] = j < a.r ? a.B[(size_t)n * a.r + j] : (uint16_t)0;
  }
}

template <int RP>
hipError_t launch_rp(const TpreArgs& a, const uint16_t** bp_used, hipStream_t stream) {
  int nkc, kch;
  tpre_chunks(a.K, nkc, kch);
  hipLaunchKernelGGL((lora_t_part_kernel<RP>), dim3((a.M + 15) / 16, nkc), dim3(T_WAVES * 64), 0, stream, a, kch);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // B serves as its own padded copy when its rows already are RP bf16, 16-byte
  // aligned; no B at all (a.B null): nothing to pad
  const bool direct = a.B == nullptr || (a.r == RP && (reinterpret_cast<uintptr_t>(a.B) & 15) == 0);
  if (bp_used) *bp_used = a.B == nullptr ? nullptr : direct ? a.B : a.bp;
  const int tblocks = (int)(((size_t)a.M * RP + 255) / 256);
  const size_t total = (size_t)a.N * RP;
  const int bblocks = direct ? 0 : (int)((total + 255) / 256 < 2048 ? (total + 255) / 256 : 2048);
  hipLaunchKernelGGL((lora_t_finish_kernel<RP>), dim3(tblocks + bblocks), dim3(256), 0, stream, a, nkc, tblocks);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lora_tpre(const TpreArgs& a, int rp, const uint16_t** bp_used, hipStream_t stream) {
  switch (rp) {
    case 16: return launch_rp<16>(a, bp_used, stream);
    case 32: return launch_rp<32>(a, bp_used, stream);
    case 64: return launch_rp<64>(a, bp_used, stream);
    case 128: return launch_rp<128>(a, bp_used, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hydra
