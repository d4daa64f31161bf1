// Decode-shaped (M <= 16) LoRA-switchable linear for gfx950.
//
// At decode time (App. A, Alg. 1 / Alg. 2: "generate ... for T steps") each
// linear sees one new token per sequence, so the work is a stream over W at
// HBM rate with almost no arithmetic intensity.  Design:
//  * one workgroup per 16 output columns; its WAVES waves split K.  Each lane
//    loads 16 contiguous bytes of one W row straight from global memory into
//    the B operand of v_mfma_f32_16x16x32_bf16 (W is output-major, so a row
//    of W is a column of W^T); the x rows (<= 16) fill the A operand.  No LDS
//    staging on the hot path; UNROLL k-steps of loads are issued before their
//    MFMAs so that each CU keeps many W bytes in flight;
//  * the LoRA-down rows A (<= 64) are consumed the same way, giving
//    T = x A^T in fp32 next to the base product (A is small and shared by all
//    workgroups, so it is served from L2);
//  * partial sums of the waves are combined in LDS in a fixed order; then
//    y_off = x W^T and y_on = y_off + s * sum_j T[m][j] B[n][j] in fp32.
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

constexpr int NB = 16;  // output columns per workgroup

template <int RP, int WAVES, int UNROLL>
__global__ __launch_bounds__(WAVES * 64) void lora_gemv_kernel(LinearArgs a) {
  constexpr int TJ = RP / 16;
  constexpr int NACC = 1 + TJ;
  __shared__ f32x4_t red[WAVES][NACC][64];
  __shared__ float Ts[16][RP > 0 ? RP : 1];

  const int M = a.M, N = a.N, K = a.K;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15;
  const int lg = lane >> 4;
  const int n0 = blockIdx.x * NB;

  const int ksteps = (K + 31) / 32;
  const int per_wave = (ksteps + WAVES - 1) / WAVES;
  const int ks0 = wave * per_wave;
  const int ks1 = min(ksteps, ks0 + per_wave);

  // Buffer resources cover exactly the valid rows of x (M), of this
  // workgroup's W slab (<= 16 rows) and of A (r): other rows read as zeros,
  // as does a k chunk past K (out-of-range offset).
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(a.x, (uint32_t)M * K * 2u);
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(a.W + (size_t)n0 * K, (uint32_t)min(NB, N - n0) * K * 2u);
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(a.A, (uint32_t)min(a.r, RP) * K * 2u);
  const int row_off = l16 * K * 2 + lg * 16;

  f32x4_t acc[NACC];
#pragma unroll
  for (int j = 0; j < NACC; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int ks = ks0; ks < ks1; ks += UNROLL) {
    uint4 xf[UNROLL], wf[UNROLL], af[UNROLL][TJ > 0 ? TJ : 1];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const bool kv = (ks + u) < ks1 && (ks + u) * 32 + lg * 8 < K;
      const int off = kv ? row_off + (ks + u) * 64 : kOutOfRange;
      wf[u] = buf_load16(wrs, off);
      xf[u] = buf_load16(xrs, off);
#pragma unroll
      for (int j = 0; j < TJ; ++j) af[u][j] = buf_load16(ars, kv ? off + j * 16 * K * 2 : kOutOfRange);
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      acc[0] = mfma16(xf[u], wf[u], acc[0]);
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[1 + j] = mfma16(xf[u], af[u][j], acc[1 + j]);
    }
  }

#pragma unroll
  for (int j = 0; j < NACC; ++j) red[wave][j][lane] = acc[j];
  __syncthreads();

  // Wave 0 sums the per-wave partials in wave order.  Its lane holds
  // D[m = 4 lg + e][n0 + l16] of the base product and T[m = 4 lg + e][16 j + l16]
  // of the LoRA-down product.
  f32x4_t sum[NACC];
  if (wave == 0) {
#pragma unroll
    for (int j = 0; j < NACC; ++j) {
      sum[j] = red[0][j][lane];
      for (int w = 1; w < WAVES; ++w) sum[j] += red[w][j][lane];
    }
    if constexpr (TJ > 0) {
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) Ts[lg * 4 + e][j * 16 + l16] = sum[1 + j][e];
    }
  }
  __syncthreads();
  if (wave != 0) return;

  const int n = n0 + l16;
  if (n >= N) return;
  float bn[RP > 0 ? RP : 1];
#pragma unroll
  for (int j = 0; j < RP; ++j) {
    const bool ok = j < a.r;
    const uint16_t v = a.B[ok ? (size_t)n * a.r + j : 0];
    bn[j] = ok ? bf16_to_f32(v) : 0.f;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int m = lg * 4 + e;
    if (m >= M) continue;
    const float yo = sum[0][e];
    if (a.y_off) a.y_off[(size_t)m * N + n] = yo;
    if (a.y_on) {
      float d = 0.f;
#pragma unroll
      for (int j = 0; j < RP; ++j) d = fmaf(Ts[m][j], bn[j], d);
      a.y_on[(size_t)m * N + n] = yo + a.s * d;
    }
  }
}

template <int RP>
hipError_t launch_rp(const LinearArgs& a, hipStream_t stream) {
  constexpr int WAVES = 16, UNROLL = 8;
  const dim3 grid((a.N + NB - 1) / NB), block(WAVES * 64);
  hipLaunchKernelGGL((lora_gemv_kernel<RP, WAVES, UNROLL>), grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lora_gemv(const LinearArgs& a, hipStream_t stream) {
  const int r = a.y_on ? a.r : 0;
  if (r == 0) return launch_rp<0>(a, stream);
  if (r <= 16) return launch_rp<16>(a, stream);
  if (r <= 32) return launch_rp<32>(a, stream);
  return launch_rp<64>(a, stream);
}

}  // namespace hydra
