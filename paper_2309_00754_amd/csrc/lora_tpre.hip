// Pre-pass of the LoRA update of the MFMA GEMMs (the dual-output linear with
// a workspace, and the fused CLM-head scoring GEMM).  T = x A^T is the same
// for every column tile of a row block, so it is computed once here instead
// of inside every tile (at rank 128 against 256-column tiles the in-tile
// product would add half of the base MFMA work):
//  * lora_t_part_kernel (padded ranks 16, 32): one workgroup per 16 rows and
//    K chunk (K split into up to 8 chunks of at least 1024, so that many
//    workgroups share the work), 8 waves taking 32-wide k-steps in turn
//    (v_mfma_f32_16x16x32_bf16, fp32 accumulation), their partial tiles
//    summed in LDS in wave order and written to the workspace;
//  * lora_t_part_wide_kernel (padded ranks 64, 128): one workgroup per 128
//    rows and K chunk, each wave 32 rows x RP on v_mfma_f32_32x32x16_bf16,
//    A staged in LDS per 256-wide sub-chunk, so that A is read once per 128
//    rows;
//  * lora_t_finish_kernel: the chunk partials added in chunk order, s * T
//    split into a bf16 hi part and a bf16 lo part (the rounding error of hi),
//    so that the GEMM's bf16 MFMAs add s T B^T to within ~2^-16 relative;
//    extra workgroups pad B to the padded rank when B's own rows cannot be
//    read as they are (r not 16, 32, 64 or 128, or B not 16-byte aligned).
// Both GEMMs then add s T B^T as 2 RP more k values of their main loop:
// rows of [hi | lo] against rows of [Bp | Bp].  Both kernels can also run two
// such pre-passes over the same rows in one launch (the backward's s dy B and
// s x A^T).
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

constexpr int T_WAVES = 8;
constexpr int T_UNROLL = 4;

// Partial T over K chunk kc for the 16 rows of blockIdx.x: the 8 waves take
// the chunk's 32-wide k-steps in turn, T_UNROLL at a time (all their loads in
// flight before the first MFMA); their partial tiles are summed in LDS in
// wave order.
template <int RP>
__device__ __forceinline__ void t_part(const TpreArgs& a, int kch, int kc) {
  constexpr int TJ = RP / 16;
  __shared__ f32x4_t red[T_WAVES][TJ][64];
  const int M = a.M, K = a.K;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int l16 = lane & 15;
  const int lg = lane >> 4;
  const int m0 = blockIdx.x * 16;
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

// Up to kMaxGroup pre-passes over the same number of rows in one launch
// (the backward runs s dy B and s x A^T together, a group of linears one
// per member): job j has K chunks ybeg[j] .. ybeg[j + 1] - 1 of blockIdx.y
// and finish blocks bbeg[j] .. bbeg[j + 1] - 1.
struct TpreJobs {
  TpreArgs a[kMaxGroup];
  int kch[kMaxGroup];
  int nkc[kMaxGroup];
  int ybeg[kMaxGroup + 1];
  int bbeg[kMaxGroup + 1];
  int n;
};
// The job that owns item v of a prefix table (wave-uniform).
__device__ __forceinline__ int job_of(const int* beg, int n, int v) {
  int j = 0;
  for (int i = 1; i < n; ++i) j = v >= beg[i] ? i : j;
  return __builtin_amdgcn_readfirstlane(j);
}

template <int RP>
__global__ __launch_bounds__(T_WAVES * 64) void lora_t_part_kernel(TpreJobs jobs) {
  const int y = blockIdx.y;
  const int j = job_of(jobs.ybeg, jobs.n, y);
  t_part<RP>(jobs.a[j], jobs.kch[j], y - jobs.ybeg[j]);
}

// Wide ranks (RP = 64, 128): a workgroup of W_WAVES waves owns W_WAVES x 32
// rows and one K chunk; each wave accumulates its 32 rows x RP columns of T
// with v_mfma_f32_32x32x16_bf16 (A rows as the A operand, x rows as the B
// operand).  The chunk goes in sub-chunks of W_SUB k: the workgroup stages
// the sub-chunk of A ([RP x W_SUB], rows padded by 16 bytes so that the
// 32-row fragment reads hit every bank once) in LDS, so A is read once per
// W_WAVES x 32 rows (the 16-row form above reads it once per 16 rows: 8x
// the x traffic at RP = 128).  Each wave holds the x slice and A pieces of
// two sub-chunks in registers: the next one's loads are in flight while the
// current one is staged and multiplied.
constexpr int kWideFrom = 64;  // padded ranks from which the wide form runs
constexpr int W_WAVES = 4;
constexpr int W_ROWS = W_WAVES * 32;
constexpr int W_SUB = 128;
constexpr int W_LDA = W_SUB + 8;  // LDS row stride of the A sub-chunk (bf16)

// K chunks of the wide form: at most kTpreMaxChunks, each at least 256 wide
// (a multiple of the 16-wide k-step), so that small M still spreads over
// many workgroups.
inline void tpre_wide_chunks(int K, int& nkc, int& kch) {
  const int want = (K + 255) / 256;
  nkc = want < kTpreMaxChunks ? want : kTpreMaxChunks;
  kch = ((K + nkc - 1) / nkc + 15) / 16 * 16;
  nkc = (K + kch - 1) / kch;
}

template <int RP>
__device__ __forceinline__ void t_part_wide(const TpreArgs& a, int kch, int kc) {
  constexpr int RA = RP < 32 ? 32 : RP;            // rows of A staged (rows RP.. read as zeros)
  constexpr int TJ = RA / 32;
  constexpr int XS = W_SUB / 16;                   // 16-wide k-steps per sub-chunk
  constexpr int AV = RA * (W_SUB / 8) / (W_WAVES * 64);  // 16-byte pieces of A per thread per sub-chunk
  static_assert(AV * W_WAVES * 64 == RA * (W_SUB / 8), "the A sub-chunk splits evenly over the threads");
  __shared__ uint16_t as[RA][W_LDA];
  const int M = a.M, K = a.K;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int l32 = lane & 31, lh = lane >> 5;
  // (made provably wave-uniform: the descriptor built from them must live in
  // SGPRs, or every load becomes a loop over the lanes' descriptors)
  const int m0 = __builtin_amdgcn_readfirstlane(blockIdx.x * W_ROWS + wave * 32);
  const int rows = __builtin_amdgcn_readfirstlane(max(0, min(32, M - m0)));
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(a.x + (size_t)min(m0, M) * K, (uint32_t)rows * K * 2u);
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(a.A, (uint32_t)min(a.r, RP) * K * 2u);
  f32x16_t acc[TJ];
#pragma unroll
  for (int j = 0; j < TJ; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
  const int k_begin = kc * kch;
  const int k_end = min(K, k_begin + kch);
  // x slice and A pieces of the sub-chunk at kb into registers
  auto load = [&](int kb, uint4 (&xf)[XS], uint4 (&av)[AV]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < XS; ++u) {
      const int k = kb + u * 16 + lh * 8;
      xf[u] = buf_load16(xrs, k < k_end ? (l32 * K + k) * 2 : kOutOfRange);
    }
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int c = t + i * W_WAVES * 64;
      const int row = c / (W_SUB / 8), k = kb + (c % (W_SUB / 8)) * 8;
      av[i] = buf_load16(ars, k < k_end ? (row * K + k) * 2 : kOutOfRange);
    }
  };
  // A pieces into LDS (after every wave is done with the previous sub-chunk), then the MFMAs
  auto stage_and_multiply = [&](const uint4 (&xf)[XS], const uint4 (&av)[AV]) __attribute__((always_inline)) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int c = t + i * W_WAVES * 64;
      *reinterpret_cast<uint4*>(&as[c / (W_SUB / 8)][(c % (W_SUB / 8)) * 8]) = av[i];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < XS; ++u)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        acc[j] = mfma32(*reinterpret_cast<const uint4*>(&as[j * 32 + l32][u * 16 + lh * 8]), xf[u], acc[j]);
  };
  // two register sets: the next sub-chunk's loads are in flight while the current one is staged and multiplied
  uint4 xf0[XS], av0[AV], xf1[XS], av1[AV];
  if (k_begin < k_end) load(k_begin, xf0, av0);
  for (int kb = k_begin; kb < k_end; kb += 2 * W_SUB) {
    const int kb1 = kb + W_SUB;
    if (kb1 < k_end) load(kb1, xf1, av1);
    stage_and_multiply(xf0, av0);
    if (kb1 >= k_end) break;
    if (kb1 + W_SUB < k_end) load(kb1 + W_SUB, xf0, av0);
    stage_and_multiply(xf1, av1);
  }
  // acc[j] element 4 i + e holds T[m0 + l32][32 j + 8 i + 4 lh + e]
  const int row = m0 + l32;
  if (row >= M) return;
  float* out = a.part + ((size_t)kc * M + row) * RP;
#pragma unroll
  for (int j = 0; j < TJ; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (32 * j + 8 * i < RP)
        *reinterpret_cast<float4*>(out + 32 * j + 8 * i + 4 * lh) =
            make_float4(acc[j][4 * i], acc[j][4 * i + 1], acc[j][4 * i + 2], acc[j][4 * i + 3]);
}

template <int RP>
__global__ __launch_bounds__(W_WAVES * 64) void lora_t_part_wide_kernel(TpreJobs jobs) {
  const int y = blockIdx.y;
  const int j = job_of(jobs.ybeg, jobs.n, y);
  t_part_wide<RP>(jobs.a[j], jobs.kch[j], y - jobs.ybeg[j]);
}

// s * T of element e = row * RP + j from the chunk partials (added in chunk
// order), split into bf16 hi and lo parts, written row-major (ts) and / or
// transposed (tT, whose rows M..Mp are written as zeros).
template <int RP>
__device__ __forceinline__ void t_finish(const TpreArgs& a, int nkc, size_t e) {
  const int rows = a.tT ? a.Mp : a.M;
  if (e >= (size_t)rows * RP) return;
  const size_t row = e / RP, j = e % RP;
  uint32_t hi = 0, lo = 0;
  if (row < (size_t)a.M) {
    // all chunk loads in flight (nkc <= kTpreMaxChunks), then added in chunk order
    float p[kTpreMaxChunks];
#pragma unroll
    for (int c = 0; c < kTpreMaxChunks; ++c) p[c] = c < nkc ? a.part[((size_t)c * a.M + row) * RP + j] : 0.f;
    float v = 0.f;
#pragma unroll
    for (int c = 0; c < kTpreMaxChunks; ++c)
      if (c < nkc) v += p[c];
    v *= a.s;
    hi = f32_to_bf16_rne(v);
    lo = f32_to_bf16_rne(v - bf16_to_f32(hi));
    if (a.ts) {
      a.ts[row * 2 * RP + j] = (uint16_t)hi;
      a.ts[row * 2 * RP + RP + j] = (uint16_t)lo;
    }
  }
  if (a.tT) {
    a.tT[j * a.Mp + row] = (uint16_t)hi;
    a.tT[(RP + j) * a.Mp + row] = (uint16_t)lo;
  }
}

// Workgroups [bbeg[j], bbeg[j + 1]) finish job j; those past the last job's
// write job 0's B zero padded to RP when the GEMM cannot read B itself (a
// single job only).
template <int RP>
__global__ __launch_bounds__(256) void lora_t_finish_kernel(TpreJobs jobs) {
  const int b = blockIdx.x;
  const int nb_fin = jobs.bbeg[jobs.n];
  if (b < nb_fin) {
    const int j = job_of(jobs.bbeg, jobs.n, b);
    t_finish<RP>(jobs.a[j], jobs.nkc[j], (size_t)(b - jobs.bbeg[j]) * 256 + threadIdx.x);
    return;
  }
  const TpreArgs& a0 = jobs.a[0];
  const size_t total = (size_t)a0.N * RP;
  const size_t nb = gridDim.x - nb_fin;
  for (size_t e = (size_t)(b - nb_fin) * 256 + threadIdx.x; e < total; e += nb * 256) {
    const int n = (int)(e / RP), j = (int)(e % RP);
    a0.bp[e] = j < a0.r ? a0.B[(size_t)n * a0.r + j] : (uint16_t)0;
  }
}

template <int RP>
hipError_t launch_rp(const TpreArgs* as, int n, const uint16_t** bp_used, hipStream_t stream) {
  constexpr bool wide = RP >= kWideFrom;
  TpreJobs jobs{};
  jobs.n = n;
  jobs.ybeg[0] = 0;
  jobs.bbeg[0] = 0;
  for (int j = 0; j < n; ++j) {
    jobs.a[j] = as[j];
    (wide ? tpre_wide_chunks : tpre_chunks)(as[j].K, jobs.nkc[j], jobs.kch[j]);
    jobs.ybeg[j + 1] = jobs.ybeg[j] + jobs.nkc[j];
    jobs.bbeg[j + 1] = jobs.bbeg[j] + (int)(((size_t)(as[j].tT ? as[j].Mp : as[j].M) * RP + 255) / 256);
  }
  const int M = as[0].M;  // (every job has the same rows)
  if constexpr (wide)
    hipLaunchKernelGGL((lora_t_part_wide_kernel<RP>), dim3((M + W_ROWS - 1) / W_ROWS, jobs.ybeg[n]),
                       dim3(W_WAVES * 64), 0, stream, jobs);
  else
    hipLaunchKernelGGL((lora_t_part_kernel<RP>), dim3((M + 15) / 16, jobs.ybeg[n]), dim3(T_WAVES * 64), 0, stream,
                       jobs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // B serves as its own padded copy when its rows already are RP bf16, 16-byte
  // aligned; no B at all (B null): nothing to pad.  Only a single job pads.
  const TpreArgs& a0 = as[0];
  const bool direct = n > 1 || a0.B == nullptr || (a0.r == RP && (reinterpret_cast<uintptr_t>(a0.B) & 15) == 0);
  if (bp_used) *bp_used = a0.B == nullptr ? nullptr : direct ? a0.B : a0.bp;
  const size_t total = (size_t)a0.N * RP;
  const int bblocks = direct ? 0 : (int)((total + 255) / 256 < 2048 ? (total + 255) / 256 : 2048);
  hipLaunchKernelGGL((lora_t_finish_kernel<RP>), dim3(jobs.bbeg[n] + bblocks), dim3(256), 0, stream, jobs);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_lora_tpre(const TpreArgs& a, int rp, const uint16_t** bp_used, hipStream_t stream) {
  switch (rp) {
    case 16: return launch_rp<16>(&a, 1, bp_used, stream);
    case 32: return launch_rp<32>(&a, 1, bp_used, stream);
    case 64: return launch_rp<64>(&a, 1, bp_used, stream);
    case 128: return launch_rp<128>(&a, 1, bp_used, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_lora_tpre_multi(const TpreArgs* as, int n, int rp, hipStream_t stream) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  for (int j = 0; j < n; ++j) {
    if (as[j].M != as[0].M) return hipErrorInvalidValue;
    // no job may need its B padded: B absent, or rows of exactly rp bf16, 16-byte aligned
    if (as[j].B && (as[j].r != rp || (reinterpret_cast<uintptr_t>(as[j].B) & 15) != 0)) return hipErrorInvalidValue;
  }
  switch (rp) {
    case 16: return launch_rp<16>(as, n, nullptr, stream);
    case 32: return launch_rp<32>(as, n, nullptr, stream);
    case 64: return launch_rp<64>(as, n, nullptr, stream);
    case 128: return launch_rp<128>(as, n, nullptr, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_lora_tpre2(const TpreArgs& a0, const TpreArgs& a1, int rp, hipStream_t stream) {
  if (a0.B || a1.B) return hipErrorInvalidValue;
  const TpreArgs as[2] = {a0, a1};
  return launch_lora_tpre_multi(as, 2, rp, stream);
}

}  // namespace hydra
