// Decode-shaped (M <= 16) LoRA-switchable linear for gfx950, for one or a
// group of linears in a single launch.
//
// At decode time (App. A, Alg. 1 / Alg. 2: "generate ... for T steps") each
// linear sees one new token per sequence, so the work is a stream over W at
// HBM rate with almost no arithmetic intensity.  Design:
//  * grid = (column blocks of NB outputs) x (linears of the group); the
//    WAVES waves of a workgroup split K.  Each lane loads 16 contiguous bytes
//    of a W row straight from global memory into the B operand of
//    v_mfma_f32_16x16x32_bf16 (W is output-major, so a row of W is a column
//    of W^T); the x rows (<= 16) fill the A operand.  No LDS on the hot path;
//    UNROLL k-steps of loads are issued before their MFMAs;
//  * the LoRA-down rows A (<= 64) are consumed the same way, giving
//    T = x A^T in fp32 next to the base product; every workgroup reads A (it
//    is small and L2-resident), so the widest column block that still fills
//    the chip (NB = 64, 32 or 16) is used to amortise it over more of W;
//  * the tile's rows of B are fetched into LDS at kernel start; the waves'
//    partial sums are combined in LDS in a fixed order (wave w sums
//    accumulator w), then one thread per output forms
//    y_off = x W^T and y_on = y_off + s * sum_j T[m][j] B[n][j] in fp32.
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

template <int RP, int NB, int WAVES, int UNROLL>
__global__ __launch_bounds__(WAVES * 64) void lora_gemv_kernel(GroupArgs ga) {
  constexpr int CT = NB / 16;        // 16-column MFMA tiles per workgroup
  constexpr int TJ = RP / 16;        // 16-column tiles of T
  constexpr int NACC = CT + TJ;
  static_assert(NACC <= WAVES, "one wave per accumulator in the reduction");
  __shared__ f32x4_t red[WAVES][NACC][64];
  __shared__ f32x4_t fin[NACC][64];
  __shared__ uint16_t Bs[NB][RP > 0 ? RP : 1];

  const int gi = blockIdx.y;
  const uint16_t* __restrict__ X = ga.x[gi];
  const uint16_t* __restrict__ Wt = ga.W[gi];
  const uint16_t* __restrict__ At = ga.A[gi];
  const uint16_t* __restrict__ Bt = ga.B[gi];
  float* __restrict__ y_off = ga.y_off[gi];
  float* __restrict__ y_on = ga.y_on[gi];
  const float s = ga.s[gi];
  const int M = ga.M, N = ga.N, K = ga.K, r = ga.r;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int l16 = lane & 15;
  const int lg = lane >> 4;
  const int n0 = blockIdx.x * NB;

  // A member of the group without y_on has no adapter (A, B may be NULL):
  // its A and B descriptors cover zero bytes, so every read of them is a zero.
  const bool has_lora = y_on != nullptr && At != nullptr && Bt != nullptr;

  // B rows of this column block, zero padded to RP (read once, early).
  if constexpr (RP > 0) {
    const __amdgpu_buffer_rsrc_t brs =
        make_rsrc(has_lora ? Bt + (size_t)n0 * r : nullptr, has_lora ? (uint32_t)min(NB, N - n0) * r * 2u : 0u);
    for (int e = t; e < NB * RP; e += WAVES * 64) {
      const int n = e / RP, j = e % RP;
      const bool ok = j < r;
      const uint32_t v = __builtin_amdgcn_raw_buffer_load_b16(brs, ok ? (n * r + j) * 2 : kOutOfRange, 0, 0);
      Bs[n][j] = ok ? (uint16_t)v : (uint16_t)0;
    }
  }

  const int ksteps = (K + 31) / 32;
  const int per_wave = (ksteps + WAVES - 1) / WAVES;
  const int ks0 = wave * per_wave;
  const int ks1 = min(ksteps, ks0 + per_wave);

  // Buffer resources cover exactly the valid rows of x (M), of this
  // workgroup's W rows and of A (r): other rows read as zeros, as does a k
  // chunk past K (out-of-range offset).
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(X, (uint32_t)M * K * 2u);
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(Wt + (size_t)n0 * K, (uint32_t)min(NB, N - n0) * K * 2u);
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(has_lora ? At : nullptr, has_lora ? (uint32_t)min(r, RP) * K * 2u : 0u);
  const int row_off = l16 * K * 2 + lg * 16;
  const int tile_off = 16 * K * 2;

  f32x4_t acc[NACC];
#pragma unroll
  for (int j = 0; j < NACC; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int ks = ks0; ks < ks1; ks += UNROLL) {
    uint4 xf[UNROLL], wf[UNROLL][CT], af[UNROLL][TJ > 0 ? TJ : 1];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const bool kv = (ks + u) < ks1 && (ks + u) * 32 + lg * 8 < K;
      const int off = kv ? row_off + (ks + u) * 64 : kOutOfRange;
#pragma unroll
      for (int c = 0; c < CT; ++c) wf[u][c] = buf_load16(wrs, kv ? off + c * tile_off : kOutOfRange);
      xf[u] = buf_load16(xrs, off);
#pragma unroll
      for (int j = 0; j < TJ; ++j) af[u][j] = buf_load16(ars, kv ? off + j * tile_off : kOutOfRange);
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
#pragma unroll
      for (int c = 0; c < CT; ++c) acc[c] = mfma16(xf[u], wf[u][c], acc[c]);
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[CT + j] = mfma16(xf[u], af[u][j], acc[CT + j]);
    }
  }

#pragma unroll
  for (int j = 0; j < NACC; ++j) red[wave][j][lane] = acc[j];
  __syncthreads();
  // Wave w sums accumulator w over the waves, in wave order.
  if (wave < NACC) {
    f32x4_t sum = red[0][wave][lane];
    for (int w = 1; w < WAVES; ++w) sum += red[w][wave][lane];
    fin[wave][lane] = sum;
  }
  __syncthreads();

  // fin[c][lane] holds D[m = 4 (lane / 16) + e][col 16 c + lane % 16] of the
  // base product (c < CT) or of T (c >= CT).  One thread per output (m, n).
  if (t >= M * NB) return;
  const int m = t / NB, nl = t % NB;
  const int n = n0 + nl;
  if (n >= N) return;
  const int src_lane = (m >> 2) * 16;
  const float yo = fin[nl >> 4][src_lane + (nl & 15)][m & 3];
  if (y_off) y_off[(size_t)m * N + n] = yo;
  if (y_on) {
    float d = 0.f;
    if constexpr (RP > 0) {
#pragma unroll
      for (int j = 0; j < RP; ++j)
        d = fmaf(fin[CT + (j >> 4)][src_lane + (j & 15)][m & 3], bf16_to_f32(Bs[nl][j]), d);
    }
    y_on[(size_t)m * N + n] = yo + s * d;
  }
}

template <int RP, int NB>
hipError_t launch_cfg(const GroupArgs& g, hipStream_t stream) {
  // 16 waves split K; every wave keeps 8 k-steps of W in flight (4 at NB = 64).
  constexpr int WAVES = 16, UNROLL = NB >= 64 ? 4 : 8;
  const dim3 grid((g.N + NB - 1) / NB, g.G), block(WAVES * 64);
  hipLaunchKernelGGL((lora_gemv_kernel<RP, NB, WAVES, UNROLL>), grid, block, 0, stream, g);
  return hipGetLastError();
}

template <int NB>
hipError_t launch_nb(const GroupArgs& g, int rp, hipStream_t stream) {
  switch (rp) {
    case 0: return launch_cfg<0, NB>(g, stream);
    case 16: return launch_cfg<16, NB>(g, stream);
    case 32: return launch_cfg<32, NB>(g, stream);
    default: return launch_cfg<64, NB>(g, stream);
  }
}

}  // namespace

hipError_t launch_lora_gemv_group(const GroupArgs& g, hipStream_t stream) {
  bool any_on = false;
  for (int i = 0; i < g.G; ++i) any_on = any_on || g.y_on[i] != nullptr;
  const int r = any_on ? g.r : 0;
  const int rp = r == 0 ? 0 : r <= 16 ? 16 : r <= 32 ? 32 : 64;
  // The widest column block that still gives at least one workgroup per CU:
  // wider blocks amortise the per-workgroup reads of A over more of W.
  const long wg64 = (long)((g.N + 63) / 64) * g.G;
  const long wg32 = (long)((g.N + 31) / 32) * g.G;
  if (wg64 >= 256) return launch_nb<64>(g, rp, stream);
  if (wg32 >= 256) return launch_nb<32>(g, rp, stream);
  return launch_nb<16>(g, rp, stream);
}

}  // namespace hydra
