// Decode-shaped (M <= 16) LoRA-switchable linear for gfx950, for one or a
// group of linears in a single launch.
//
// At decode time (App. A, Alg. 1 / Alg. 2: "generate ... for T steps") each
// linear sees one new token per sequence, so the work is a stream over W at
// HBM rate with almost no arithmetic intensity.  Two kernels:
//  * M <= 8 (lora_gemv_dot_kernel): grid = (blocks of NB rows of W) x
//    (linears of the group), 8 waves per workgroup, each wave owning NB / 8
//    rows of W over all of K.  A wave reads a W row as whole 1 KB lines (lane
//    l takes 8 consecutive k values of every 512-wide chunk), the matching 16
//    bytes of each x row, and accumulates with v_dot2c_f32_bf16 in fp32.  The
//    loads of the next chunk are issued before the current chunk is used.
//    The rank-r LoRA-down rows A are streamed the same way (AR rows per
//    wave), giving T = x A^T next to the base product.  At the end each
//    wave's per-lane partial sums are reduced across the 64 lanes by a
//    halving exchange (32 values in 32 shuffles), and one thread per output
//    forms y_off and y_on = y_off + s * sum_j T[m][j] B[n][j];
//  * 8 < M <= 16 (lora_gemv_mfma_kernel): x rows fill the A operand of
//    v_mfma_f32_16x16x32_bf16, the W rows its B operand; the waves split K
//    and their partial tiles are combined in LDS in a fixed order.
// Both reduce in a fixed order (results are deterministic and the same for a
// linear called alone or inside a group).
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

template <int RP, int NB, int WAVES, int UNROLL>
__global__ __launch_bounds__(WAVES * 64) void lora_gemv_mfma_kernel(GroupArgs ga) {
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

// ---------------------------------------------------------------- M <= 8
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;

// acc + <w, x> over 8 bf16 pairs, fp32 accumulation (v_dot2c_f32_bf16)
__device__ __forceinline__ float dot8(const uint4& w, const uint4& x, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.x), __builtin_bit_cast(bf16x2_t, x.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.y), __builtin_bit_cast(bf16x2_t, x.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.z), __builtin_bit_cast(bf16x2_t, x.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w.w), __builtin_bit_cast(bf16x2_t, x.w), acc, false);
  return acc;
}

// Sum V per-lane values over the 64 lanes of the wave.  Each exchange step
// (lane distance o = 32, 16, ...) hands half of the remaining values to the
// partner lane and adds the other half; once one value is left the
// remaining distances are summed in full.  Afterwards v[0] holds the total of
// value index sum_s bit(lane, o_s) * V / 2^(s+1) (lanes that differ only in
// the low bits used by the full sums hold the same total).
template <int V>
__device__ __forceinline__ void wave_reduce_scatter(float (&v)[V], int lane) {
  static_assert(V >= 1 && V <= 64 && (V & (V - 1)) == 0, "power of two, at most 64 values");
  int o = 32;
#pragma unroll
  for (int cnt = V; cnt > 1; cnt >>= 1, o >>= 1) {
    const bool up = (lane & o) != 0;
#pragma unroll
    for (int q = 0; q < cnt / 2; ++q) {
      const float send = up ? v[q] : v[q + cnt / 2];
      const float keep = up ? v[q + cnt / 2] : v[q];
      v[q] = keep + __shfl_xor(send, o);
    }
  }
  for (; o >= 1; o >>= 1) v[0] += __shfl_xor(v[0], o);
}

// value index held by `lane` after wave_reduce_scatter<V>
template <int V>
__device__ __forceinline__ int reduced_index(int lane) {
  int idx = 0, o = 32;
#pragma unroll
  for (int half = V / 2; half >= 1; half >>= 1, o >>= 1) idx += (lane & o) ? half : 0;
  return idx;
}
// lanes that write a reduced value: one per index (the low lane bits that
// were summed in full are zero)
template <int V>
__device__ __forceinline__ bool reduced_writer(int lane) {
  const int low = 64 / V - 1;  // bits summed in full
  return (lane & low) == 0;
}

constexpr int DW = 8;     // waves per workgroup
constexpr int DKC = 512;  // k values per chunk (64 lanes x 8)

// MB >= M x rows, RPW rows of W and AR rows of A per wave.
template <int MB, int RPW, int AR>
__global__ __launch_bounds__(DW * 64) void lora_gemv_dot_kernel(GroupArgs ga) {
  constexpr int NB = RPW * DW;  // W rows per workgroup
  constexpr int RP = AR * DW;   // padded rank
  constexpr int VY = RPW * MB;  // partial sums per lane: base product
  constexpr int VT = AR * MB;   //                       T
  static_assert(VY <= 64 && VT <= 64, "at most 64 partial sums per lane");
  __shared__ float ysh[NB][MB];
  __shared__ float tsh[RP > 0 ? RP : 1][MB];
  __shared__ uint16_t bsh[NB][RP > 0 ? RP : 1];

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
  const int n0 = blockIdx.x * NB;

  // A member of the group without y_on has no adapter (A, B may be NULL):
  // its A and B descriptors cover zero bytes, so every read of them is a zero.
  const bool has_lora = y_on != nullptr && At != nullptr && Bt != nullptr;

  // Rows of B of this block, zero padded to RP: loaded now into registers
  // (thread t holds elements t, t + 512, ... of the NB x RP block) and
  // written to LDS only after the main loop, so that nothing waits for them.
  constexpr int BPT = RP > 0 ? (NB * RP + DW * 64 - 1) / (DW * 64) : 1;
  uint32_t bv[BPT];
  if constexpr (RP > 0) {
    const __amdgpu_buffer_rsrc_t brs =
        make_rsrc(has_lora ? Bt + (size_t)n0 * r : nullptr, has_lora ? (uint32_t)min(NB, N - n0) * r * 2u : 0u);
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      const int e = t + q * DW * 64;
      const int n = e / RP, j = e % RP;
      bv[q] = __builtin_amdgcn_raw_buffer_load_b16(brs, (e < NB * RP && j < r) ? (n * r + j) * 2 : kOutOfRange, 0, 0);
    }
  }

  // Buffer resources cover exactly the valid rows of x (M), of this block's
  // rows of W and of A (r): other rows read as zeros, as does a chunk past K.
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(X, (uint32_t)M * K * 2u);
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(Wt + (size_t)n0 * K, (uint32_t)min(NB, N - n0) * K * 2u);
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(has_lora ? At : nullptr, has_lora ? (uint32_t)min(r, RP) * K * 2u : 0u);
  const int nch = (K + DKC - 1) / DKC;

  struct Ld {
    uint4 x[MB];
    uint4 w[RPW];
    uint4 a[AR > 0 ? AR : 1];
  };
  float acc[VY], acct[VT > 0 ? VT : 1];
#pragma unroll
  for (int q = 0; q < VY; ++q) acc[q] = 0.f;
#pragma unroll
  for (int q = 0; q < (VT > 0 ? VT : 1); ++q) acct[q] = 0.f;

  // Each workgroup walks the chunks starting at its own offset (wrapping
  // around): all workgroups read the same x rows and LoRA-down rows, and
  // this keeps them from all asking for the same lines at the same moment.
  // The order depends only on the column block, so a linear gives the same
  // bits alone or inside a group.
  const int c0 = blockIdx.x % nch;
  auto load = [&](Ld& L, int cc) __attribute__((always_inline)) {
    const int c = cc < nch ? (cc + c0 >= nch ? cc + c0 - nch : cc + c0) : nch;
    const int k = c * DKC + lane * 8;
    const bool kv = c < nch && k < K;
#pragma unroll
    for (int m = 0; m < MB; ++m) L.x[m] = buf_load16(xrs, kv ? (m * K + k) * 2 : kOutOfRange);
#pragma unroll
    for (int i = 0; i < RPW; ++i) L.w[i] = buf_load16(wrs, kv ? ((wave * RPW + i) * K + k) * 2 : kOutOfRange);
#pragma unroll
    for (int j = 0; j < AR; ++j) L.a[j] = buf_load16(ars, kv ? ((wave * AR + j) * K + k) * 2 : kOutOfRange);
  };
  auto use = [&](const Ld& L) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < RPW; ++i)
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[i * MB + m] = dot8(L.w[i], L.x[m], acc[i * MB + m]);
#pragma unroll
    for (int j = 0; j < AR; ++j)
#pragma unroll
      for (int m = 0; m < MB; ++m) acct[j * MB + m] = dot8(L.a[j], L.x[m], acct[j * MB + m]);
  };
  // Two chunks in flight when both load sets fit in the register budget.
  constexpr bool DOUBLE = MB + RPW + AR <= 16;
  if constexpr (DOUBLE) {
    Ld L0, L1;
    load(L0, 0);
    load(L1, 1);
    // (scheduling barriers keep each refill right after the use of its
    // buffer, so that one chunk is always in flight while the other is used)
    for (int c = 0; c < nch; c += 2) {
      use(L0);
      __builtin_amdgcn_sched_barrier(0);
      load(L0, c + 2);
      __builtin_amdgcn_sched_barrier(0);
      use(L1);  // zeros past the last chunk
      __builtin_amdgcn_sched_barrier(0);
      load(L1, c + 3);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    Ld L0;
    for (int c = 0; c < nch; ++c) {
      load(L0, c);
      use(L0);
    }
  }

  if constexpr (RP > 0) {
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      const int e = t + q * DW * 64;
      if (e < NB * RP) bsh[e / RP][e % RP] = (uint16_t)bv[q];
    }
  }
  // partial sums of the wave -> totals over the 64 lanes -> LDS
  wave_reduce_scatter<VY>(acc, lane);
  if (reduced_writer<VY>(lane)) {
    const int q = reduced_index<VY>(lane);
    ysh[wave * RPW + q / MB][q % MB] = acc[0];
  }
  if constexpr (VT > 0) {
    wave_reduce_scatter<VT>(acct, lane);
    if (reduced_writer<VT>(lane)) {
      const int q = reduced_index<VT>(lane);
      tsh[wave * AR + q / MB][q % MB] = acct[0];
    }
  }
  __syncthreads();

  // one thread per output (m, n): y_off = x W^T, y_on = y_off + s * T B^T
  for (int e = t; e < M * NB; e += DW * 64) {
    const int m = e / NB, nl = e % NB;
    const int n = n0 + nl;
    if (n >= N) continue;
    const float yo = ysh[nl][m];
    if (y_off) y_off[(size_t)m * N + n] = yo;
    if (y_on) {
      float d = 0.f;
      if constexpr (RP > 0) {
#pragma unroll
        for (int j = 0; j < RP; ++j) d = fmaf(tsh[j][m], bf16_to_f32(bsh[nl][j]), d);
      }
      y_on[(size_t)m * N + n] = yo + s * d;
    }
  }
}

template <int MB, int RPW>
hipError_t launch_dot_mb(const GroupArgs& g, int rp, hipStream_t stream) {
  const dim3 grid((g.N + RPW * DW - 1) / (RPW * DW), g.G), block(DW * 64);
  switch (rp) {
    case 0: hipLaunchKernelGGL((lora_gemv_dot_kernel<MB, RPW, 0>), grid, block, 0, stream, g); break;
    case 16: hipLaunchKernelGGL((lora_gemv_dot_kernel<MB, RPW, 2>), grid, block, 0, stream, g); break;
    case 32: hipLaunchKernelGGL((lora_gemv_dot_kernel<MB, RPW, 4>), grid, block, 0, stream, g); break;
    default: hipLaunchKernelGGL((lora_gemv_dot_kernel<MB, RPW, 8>), grid, block, 0, stream, g); break;
  }
  return hipGetLastError();
}

template <int RP, int NB>
hipError_t launch_cfg(const GroupArgs& g, hipStream_t stream) {
  // 16 waves split K; every wave keeps 8 k-steps of W in flight (4 at NB = 64).
  constexpr int WAVES = 16, UNROLL = NB >= 64 ? 4 : 8;
  const dim3 grid((g.N + NB - 1) / NB, g.G), block(WAVES * 64);
  hipLaunchKernelGGL((lora_gemv_mfma_kernel<RP, NB, WAVES, UNROLL>), grid, block, 0, stream, g);
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
  if (g.M <= 4) return launch_dot_mb<4, 8>(g, rp, stream);
  if (g.M <= 8) return launch_dot_mb<8, 4>(g, rp, stream);
  // The widest column block that still gives at least one workgroup per CU:
  // wider blocks amortise the per-workgroup reads of A over more of W.
  const long wg64 = (long)((g.N + 63) / 64) * g.G;
  const long wg32 = (long)((g.N + 31) / 32) * g.G;
  if (wg64 >= 256) return launch_nb<64>(g, rp, stream);
  if (wg32 >= 256) return launch_nb<32>(g, rp, stream);
  return launch_nb<16>(g, rp, stream);
}

}  // namespace hydra
