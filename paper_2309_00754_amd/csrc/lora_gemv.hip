// Decode-shaped (M <= 16) LoRA-switchable linear for gfx950, for one or a
// group of linears in a single call.
//
// At decode time (App. A, Alg. 1 / Alg. 2, the token-by-token generation step) each
// linear sees one new token per sequence, so the work is a stream over W at
// HBM rate with almost no arithmetic intensity.
//  * M <= 8: two kernels.  gemv_stream_kernel computes the base product x W^T
//    with one wave per row of W (16 rows per workgroup): the many small work
//    units let the hardware dispatcher balance the HBM stream across the
//    chip, which a static split of the rows over persistent workgroups does
//    not (per-wave bandwidth varies by a factor of two).  A wave reads its
//    row as whole 1 KB lines (lane l takes 8 consecutive k of every 512-wide
//    chunk), the workgroup's x rows come from LDS, the dot products run on
//    v_dot2c_f32_bf16 in fp32, and the 64 lanes are summed by a halving
//    exchange.  It writes y_off and the base part of y_on.  Then, for the
//    members with an adapter, lora_update_kernel adds s * (x A^T) B^T to y_on:
//    forming T = x A^T once per workgroup of 256 columns instead of once per
//    16 rows keeps the reads of A off the stream.
//  * 8 < M <= 16 (lora_gemv_mfma_kernel): x rows fill the A operand of
//    v_mfma_f32_16x16x32_bf16, the W rows its B operand; the waves split K
//    and their partial tiles are combined in LDS in a fixed order.
// Every reduction runs in a fixed order (results are deterministic and the
// same for a linear called alone or inside a group).
#include "../../include/hydra.h"
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

  // B rows of this column block, zero padded to RP: requested first, held in
  // registers, and written to LDS only after the main loop, so that their
  // latency overlaps the loads of W instead of preceding them.
  constexpr int BPT = RP > 0 ? (NB * RP + WAVES * 64 - 1) / (WAVES * 64) : 1;  // B values per thread
  uint32_t bv[BPT];
  if constexpr (RP > 0) {
    const __amdgpu_buffer_rsrc_t brs =
        make_rsrc(has_lora ? Bt + (size_t)n0 * r : nullptr, has_lora ? (uint32_t)min(NB, N - n0) * r * 2u : 0u);
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int e = t + i * WAVES * 64;
      const int n = e / RP, j = e % RP;
      const bool ok = e < NB * RP && j < r;
      bv[i] = __builtin_amdgcn_raw_buffer_load_b16(brs, ok ? (n * r + j) * 2 : kOutOfRange, 0, 0);
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

  if constexpr (RP > 0) {
#pragma unroll
    for (int i = 0; i < BPT; ++i) {
      const int e = t + i * WAVES * 64;
      if (e < NB * RP) Bs[e / RP][e % RP] = (uint16_t)bv[i];  // (zero past r: out-of-range reads)
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
      // (the empty asm keeps the two values in registers: without it the
      // compiler turns the lane-dependent choice into a dynamically indexed
      // read of the whole array, a long chain of selects)
      float lo = v[q], hi = v[q + cnt / 2];
      asm volatile("" : "+v"(lo), "+v"(hi));
      const float send = up ? lo : hi;
      const float keep = up ? hi : lo;
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
// a lane that holds reduced index v after wave_reduce_scatter<V>: the index
// bits are the lane bits o = 32, 16, ... (v's most significant bit first)
template <int V>
__device__ __forceinline__ int reduced_lane(int v) {
  int lane = 0, o = 32;
#pragma unroll
  for (int half = V / 2; half >= 1; half >>= 1, o >>= 1) lane |= (v & half) ? o : 0;
  return lane;
}
// lanes that write a reduced value: one per index (the low lane bits that
// were summed in full are zero)
template <int V>
__device__ __forceinline__ bool reduced_writer(int lane) {
  const int low = 64 / V - 1;  // bits summed in full
  return (lane & low) == 0;
}

constexpr int DKC = 512;  // k values per chunk (64 lanes x 8)

// x rows staged in LDS per K segment: MB rows x SEG chunks of 512 k (32 KB).
template <int MB>
struct XSeg {
  static constexpr int SEG = MB <= 4 ? 8 : 4;  // chunks per segment
  static constexpr int ELEMS = MB * SEG * 64;   // uint4 per segment
};

// Stage x[m][c0 * 512 ... (c0 + SEG) * 512) for m < MB in LDS: element
// (m, u, lane) holds the 8 k values that lane `lane` of any wave uses in chunk
// c0 + u.  Rows past M and k past K read as zeros.
template <int MB, int NT, int SEG = XSeg<MB>::SEG>
__device__ __forceinline__ void stage_x(uint4* xsh, __amdgpu_buffer_rsrc_t xrs, int c0, int nch, int K, int t) {
  static_assert(SEG <= XSeg<MB>::SEG, "a segment fits the staging buffer");
  for (int e = t; e < MB * SEG * 64; e += NT) {
    const int m = e / (SEG * 64), u = (e / 64) % SEG, l = e % 64;
    const int c = c0 + u, k = c * DKC + l * 8;
    xsh[e] = buf_load16(xrs, (c < nch && k < K) ? (m * K + k) * 2 : kOutOfRange);
  }
}

// The same from the segments of a StreamArgs weight (row m: segment
// seg0 + m / seg_rows, row m % seg_rows of it; rows past the weight's
// segments read as zeros).  Every wave stages whole 64-element runs of one
// row (the runs are 64-aligned and the stride is a multiple of 64), so the row
// index, and with it the segment pointer, is wave-uniform: scalar loads of
// the kernel arguments, then a buffer load per lane.
template <int MB, int NT>
__device__ __forceinline__ void stage_x_segs(uint4* xsh, const StreamArgs& sa, int gi, int c0, int nch, int t) {
  constexpr int SEG = XSeg<MB>::SEG;
  constexpr int ELEMS = XSeg<MB>::ELEMS;
  constexpr int PER = (ELEMS + NT - 1) / NT;  // elements per thread
  static_assert(NT % 64 == 0, "whole waves");
  const int K = sa.K;
  uint4 v[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {  // every load in flight before the first LDS write
    const int e = t + q * NT;
    const int m = __builtin_amdgcn_readfirstlane(e / (SEG * 64));
    const int u = (e / 64) % SEG, l = e % 64;
    const int c = c0 + u, k = c * DKC + l * 8;
    const int sg = m < kStreamRows ? sa.seg_of[gi][m] : kStreamSegs;
    const bool have = sg < kStreamSegs;
    const uint16_t* row = have ? sa.x[sa.seg0[gi] + sg] + (size_t)(m - sg * sa.seg_rows) * K : nullptr;
    const __amdgpu_buffer_rsrc_t rrs = make_rsrc(row, have ? (uint32_t)K * 2u : 0u);
    v[q] = buf_load16(rrs, (e < ELEMS && c < nch && k < K) ? k * 2 : kOutOfRange);
  }
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = t + q * NT;
    if (e < ELEMS) xsh[e] = v[q];
  }
}

constexpr int SW = 16;  // waves (= rows of W) per workgroup of the base kernel

// Base product of one weight of the launch: y[m][n] = <x[m], W[n]> for the
// rows of the row table, one wave per row n of W.  Small work units let the
// hardware dispatcher balance the HBM stream across the chip; the x rows are
// shared by the workgroup's 16 rows of W through LDS.  Each output row is
// written to its first (ya) and second (yb) destination when present: for a
// single linear these are y_off and the base part of y_on (the LoRA update of
// y_on, when there is one, is added by lora_update_kernel afterwards); for
// several inputs sharing W they are the inputs' own outputs.
template <int MB>
__global__ __launch_bounds__(SW * 64) void gemv_stream_kernel(StreamArgs sa) {
  constexpr int SEG = XSeg<MB>::SEG;
  __shared__ uint4 xsh[XSeg<MB>::ELEMS];
  const int gi = blockIdx.y;
  const uint16_t* __restrict__ Wt = sa.W[gi];
  const int N = sa.N, K = sa.K;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n = blockIdx.x * SW + wave;
  const bool row_ok = n < N;
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(Wt + (size_t)min(n, N - 1) * K, row_ok ? (uint32_t)K * 2u : 0u);
  const int nch = (K + DKC - 1) / DKC;

  auto load_seg = [&](uint4 (&b)[SEG], int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < SEG; ++u) {
      const int c = c0 + u, k = c * DKC + lane * 8;
      b[u] = buf_load16(wrs, (c < nch && k < K) ? k * 2 : kOutOfRange);
    }
  };
  float acc[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m] = 0.f;
  // (a second segment buffer would take the kernel past 64 VGPRs, i.e. below
  // two 16-wave workgroups per CU; segments after the first are rare: K > 4096)
  for (int c0 = 0; c0 < nch; c0 += SEG) {
    uint4 wb[SEG];
    load_seg(wb, c0);
    if (c0 > 0) __syncthreads();  // every wave is done with the previous x segment
    stage_x_segs<MB, SW * 64>(xsh, sa, gi, c0, nch, t);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < SEG; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[m] = dot8(wb[u], xsh[(m * SEG + u) * 64 + lane], acc[m]);
  }
  wave_reduce_scatter<MB>(acc, lane);
  // the output row pointers are read as wave-uniform values (scalar loads of
  // the kernel arguments) and chosen per lane afterwards
  const int m = reduced_index<MB>(lane);
  float* ya = nullptr;
  float* yb = nullptr;
#pragma unroll
  for (int q = 0; q < MB; ++q) {
    const int sg = sa.seg_of[gi][q];
    if (sg < kStreamSegs) {  // wave-uniform
      const size_t mr = (size_t)(q - sg * sa.seg_rows);
      float* pa = sa.ya[sa.seg0[gi] + sg];
      float* pb = sa.yb[sa.seg0[gi] + sg];
      pa = pa ? pa + mr * N : nullptr;
      pb = pb ? pb + mr * N : nullptr;
      ya = m == q ? pa : ya;
      yb = m == q ? pb : yb;
    }
  }
  if (row_ok && reduced_writer<MB>(lane)) {
    if (ya) ya[n] = acc[0];
    if (yb) yb[n] = acc[0];
  }
}

constexpr int UW = 16;   // waves per workgroup of the LoRA update
// columns of y_on per workgroup (fewer at rank 128, for the registers and LDS
// that hold the block of B)
constexpr int update_cols(int rp) { return rp <= 64 ? 256 : 128; }
// rows of A per wave in the T pass: 8, or 4 with 8 rows of x up to rank 64
// (8 x 8 partial sums per lane would spill)
constexpr int upd_urw(int mb, int rp) { return mb >= 8 && rp <= 64 ? 4 : 8; }

// y_on += s * T B^T with T = x A^T, for the members of the group that have an
// adapter.  Every workgroup forms T itself: the 16 waves split A into RP / 8
// row groups of 8 rows and the K chunks into 128 / RP chunk groups; a wave
// requests its rows of A and its pieces of x for one chunk at a time (both
// L2 hits once the first workgroup has touched them), reduces its partial
// sums across its lanes, and the partials of the chunk groups are added in a
// fixed order.  The rows of B and the current values of y_on are requested
// first, so that their latency overlaps the T pass.  The block of B is held in
// LDS row by row ([column][j]) at padded ranks up to 32, and transposed with
// padded rows ([j][column]) from rank 64 on: there the lanes of a wave, which
// hold consecutive columns, would otherwise read LDS addresses 2 * RP bytes
// apart, all in one bank at RP = 128.  From rank 64 on the T pass also stages
// the pieces of x in LDS once per workgroup: with one or two chunk groups the
// 16 waves would otherwise each request all of x, as many bytes as their rows
// of A.
template <int MB, int RP>
__global__ __launch_bounds__(UW * 64) void lora_update_kernel(GroupArgs ga) {
  constexpr int NT = UW * 64;
  constexpr int UNB = update_cols(RP);
  constexpr int URW = upd_urw(MB, RP);
  constexpr int GR = RP / URW;                     // row groups
  constexpr int GC = UW / GR;                      // chunk groups
  constexpr int VT = URW * MB;                     // partial sums of T per lane
  constexpr int BPT = UNB * RP / NT;               // bf16 of B per thread
  constexpr int OPT = (UNB * MB + NT - 1) / NT;    // outputs per thread
  static_assert(GR * GC == UW && VT <= 64 && BPT >= 1, "shape");
  __shared__ float part[UW][VT];      // per-wave partial T, index j_local * MB + m
  __shared__ float4 tsh[MB][RP / 4];  // T[m][j]
  constexpr bool BT = RP >= 64;                    // B block transposed in LDS
  constexpr int BLD = BT ? UNB + 2 : RP;           // u16 per LDS row of the block
  __shared__ uint16_t bsh[BT ? RP : UNB][BLD];
  // from rank 64 on, x is staged in LDS per round of GC chunks ([chunk][m][lane])
  constexpr bool XS = RP >= 64;
  constexpr int XE = XS ? GC * MB * 64 : 1;        // 16-byte pieces of x per round
  constexpr int XPT = (XE + NT - 1) / NT;
  static_assert(!XS || BT, "the staged T pass writes the B block in the transposed layout");
  __shared__ uint4 xsh[XE];
  const int gi = blockIdx.y;
  const uint16_t* __restrict__ X = ga.x[gi];
  const uint16_t* __restrict__ At = ga.A[gi];
  const uint16_t* __restrict__ Bt = ga.B[gi];
  float* __restrict__ y_on = ga.y_on[gi];
  if (y_on == nullptr || At == nullptr || Bt == nullptr) return;  // member without an adapter
  const float s = ga.s[gi];
  const int M = ga.M, N = ga.N, K = ga.K, r = ga.r;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int n0 = blockIdx.x * UNB;
  const int nb = min(UNB, N - n0);

  // B block [nb x r], zero padded to RP: requested now into registers,
  // written to LDS after the T pass.
  const __amdgpu_buffer_rsrc_t brs = make_rsrc(Bt + (size_t)n0 * r, (uint32_t)nb * r * 2u);
  uint32_t bv[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) {
    const int e = t + q * NT, nl = e / RP, j = e % RP;
    bv[q] = __builtin_amdgcn_raw_buffer_load_b16(brs, j < r ? (nl * r + j) * 2 : kOutOfRange, 0, 0);
  }
  float yv[OPT];
#pragma unroll
  for (int q = 0; q < OPT; ++q) {
    const int e = t + q * NT, m = e / UNB, nl = e % UNB;
    yv[q] = (e < UNB * MB && m < M && nl < nb) ? y_on[(size_t)m * N + n0 + nl] : 0.f;
  }

  // T pass: wave = (row group, chunk group); rows of A beyond r read as zeros
  const int rg = wave / GC, cg = wave % GC;
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(X, (uint32_t)M * K * 2u);
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(At, (uint32_t)r * K * 2u);
  const int nch = (K + DKC - 1) / DKC;
  float acc[VT];
#pragma unroll
  for (int q = 0; q < VT; ++q) acc[q] = 0.f;
  if constexpr (XS) {
    // Rounds of GC chunks: the workgroup stages the round's x pieces in LDS
    // once (instead of every row group requesting them) while each wave's
    // rows of A are in flight.  A wave whose chunk lies past K adds zeros.
    const int nround = (nch + GC - 1) / GC;
    for (int rd = 0; rd < nround; ++rd) {
      const int c = rd * GC + cg;
      const int k = c * DKC + lane * 8;
      const bool kv = c < nch && k < K;
      uint4 av[URW];
#pragma unroll
      for (int j = 0; j < URW; ++j) av[j] = buf_load16(ars, kv ? ((rg * URW + j) * K + k) * 2 : kOutOfRange);
      uint4 xs[XPT];
#pragma unroll
      for (int q = 0; q < XPT; ++q) {
        const int e = t + q * NT, ch = e / (MB * 64), m = (e / 64) % MB;
        const int cc = rd * GC + ch, kk = cc * DKC + (e % 64) * 8;
        xs[q] = buf_load16(xrs, (e < XE && cc < nch && kk < K) ? (m * K + kk) * 2 : kOutOfRange);
      }
      if (rd == 0) {
        // the block of B goes to LDS now (its loads were issued first, so only
        // they are waited for), which frees its registers for the T pass
#pragma unroll
        for (int q = 0; q < BPT; ++q) {
          const int e = t + q * NT;
          bsh[e % RP][e / RP] = (uint16_t)bv[q];
        }
      }
      if (rd > 0) __syncthreads();  // every wave is done with the previous round's x
#pragma unroll
      for (int q = 0; q < XPT; ++q)
        if (t + q * NT < XE) xsh[t + q * NT] = xs[q];
      __syncthreads();
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        const uint4 xv = xsh[(cg * MB + m) * 64 + lane];
#pragma unroll
        for (int j = 0; j < URW; ++j) acc[j * MB + m] = dot8(av[j], xv, acc[j * MB + m]);
        __builtin_amdgcn_sched_barrier(0);  // one row of x in registers at a time
      }
    }
  } else {
    for (int c = cg; c < nch; c += GC) {
      const int k = c * DKC + lane * 8;
      const bool kv = k < K;
      uint4 av[URW], xv[MB];
#pragma unroll
      for (int j = 0; j < URW; ++j) av[j] = buf_load16(ars, kv ? ((rg * URW + j) * K + k) * 2 : kOutOfRange);
#pragma unroll
      for (int m = 0; m < MB; ++m) xv[m] = buf_load16(xrs, kv ? (m * K + k) * 2 : kOutOfRange);
      __builtin_amdgcn_sched_barrier(0);  // all of the chunk's loads in flight before the first use
#pragma unroll
      for (int j = 0; j < URW; ++j)
#pragma unroll
        for (int m = 0; m < MB; ++m) acc[j * MB + m] = dot8(av[j], xv[m], acc[j * MB + m]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  wave_reduce_scatter<VT>(acc, lane);
  if (reduced_writer<VT>(lane)) part[wave][reduced_index<VT>(lane)] = acc[0];
  if constexpr (!XS) {
#pragma unroll
    for (int q = 0; q < BPT; ++q) {
      const int e = t + q * NT;
      if constexpr (BT)
        bsh[e % RP][e / RP] = (uint16_t)bv[q];
      else
        bsh[e / RP][e % RP] = (uint16_t)bv[q];
    }
  }
  __syncthreads();
  // T[m][j] = sum over the chunk groups, in chunk-group order
  if (t < RP * MB) {
    const int j = t / MB, m = t % MB;
    const int g = j / URW, q = (j % URW) * MB + m;
    float v = part[g * GC][q];
    for (int c2 = 1; c2 < GC; ++c2) v += part[g * GC + c2][q];
    reinterpret_cast<float*>(&tsh[m][0])[j] = v;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < OPT; ++q) {
    const int e = t + q * NT, m = e / UNB, nl = e % UNB;
    if (e < UNB * MB && m < M && nl < nb) {
      auto b_at = [&](int j) __attribute__((always_inline)) {
        if constexpr (BT)
          return bf16_to_f32(bsh[j][nl]);
        else
          return bf16_to_f32(bsh[nl][j]);
      };
      float d = 0.f;
#pragma unroll
      for (int j4 = 0; j4 < RP / 4; ++j4) {
        const float4 tv = tsh[m][j4];
        d = fmaf(tv.x, b_at(4 * j4 + 0), d);
        d = fmaf(tv.y, b_at(4 * j4 + 1), d);
        d = fmaf(tv.z, b_at(4 * j4 + 2), d);
        d = fmaf(tv.w, b_at(4 * j4 + 3), d);
      }
      y_on[(size_t)m * N + n0 + nl] = yv[q] + s * d;
    }
  }
}

template <int MB>
hipError_t launch_update_mb(const GroupArgs& g, int rp, hipStream_t stream) {
  const int cols = update_cols(rp);
  const dim3 grid((g.N + cols - 1) / cols, g.G), block(UW * 64);
  switch (rp) {
    case 16: hipLaunchKernelGGL((lora_update_kernel<MB, 16>), grid, block, 0, stream, g); break;
    case 32: hipLaunchKernelGGL((lora_update_kernel<MB, 32>), grid, block, 0, stream, g); break;
    case 64: hipLaunchKernelGGL((lora_update_kernel<MB, 64>), grid, block, 0, stream, g); break;
    default: hipLaunchKernelGGL((lora_update_kernel<MB, 128>), grid, block, 0, stream, g); break;
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
    default: return launch_cfg<64, NB>(g, stream);  // (rank 128 is split into row halves above)
  }
}


// ---------------------------------------------------------------- decode in one launch
// The decode step of a group (M <= 8 rows per member) in a single launch,
// with a small caller workspace.  The first workgroups of the grid form T =
// x A^T of every member with an adapter (one wave per row of A, the same
// routine as a row of W) and publish it in the workspace; the other
// workgroups stream the rows of W, write y_off, and add s T B^T to their own
// rows to write y_on.
//
// Publishing without a flush or a second round trip: every T value is stored
// together with a 32-bit tag in one 64-bit device-coherent store, and a
// reader accepts T only when every tag it loaded equals the tag of the
// current call.  The tag of a call is derived from a generation word in the
// workspace: each workgroup reads it with the same returning atomic that
// reports the read (the atomic adds one to a count in the low half of a
// 64-bit word whose high half is the generation), and one extra workgroup at
// the end of the grid, the keeper, waits until every count is complete and
// then advances the generation and clears the counts.  Every workgroup of a
// call therefore sees the same generation, every T value carrying the next
// tag was computed by this call, and values left by earlier calls carry
// older tags.  The keeper starts after every other workgroup has started
// (the hardware dispatches in grid order), so its wait is short and runs
// beside the W stream instead of after it.
//
// A W workgroup loads its member's T right at its start next to its rows of
// W (one entry per thread); if T was not complete yet (only the first
// workgroups, which run next to the T workgroups), it loads it again after
// its dot products, in a bounded loop, and past the bound forms T itself
// through the same routine (same bits).  If the keeper's own bounded wait
// runs out, it sets the poison bit of the generation word instead of leaving
// a generation that a late reader could share with the next call: from then
// on every W workgroup forms T itself (same bits, slower) until the caller
// zeroes the workspace again.  The caller's bound word, when set, bounds
// both waits.
struct FusedArgs {
  GroupArgs ga;
  uint32_t* ctl;   // control words (layout below)
  uint64_t* tsl;   // tagged T [G][kStreamRows][RP]: (tag << 32) | value bits
  int nT;          // T workgroups per member (RP / 8)
  int nWB;         // W workgroups per member (ceil(N / 16))
  int total;       // T and W workgroups; workgroup `total` is the keeper
  int nbk;         // count buckets in use
};
// Control words.  Line 0 holds the caller's wait bound (word kCtlBound);
// line 1 is spare; line 2 + q (q < kFusedBuckets) holds the 64-bit word of
// bucket q: low half the count of workgroups b with b % nbk == q that have
// read the generation in this call, high half a copy of the generation word
// (every line holds the same copy: the reads spread over the lines).
constexpr int kCtlLine = 32;  // 32-bit words per 128-byte line
constexpr int kCtlBound = kMaxGroup;
constexpr int kCtlBucket0 = 2 * kCtlLine;
static_assert(kFusedCtlBytes == HYDRA_GROUP_WS_CONTROL_BYTES && kCtlBound == HYDRA_GROUP_WS_BOUND_WORD,
              "control area as documented in hydra.h");
static_assert(kFusedCtlBytes == size_t(kCtlBucket0 / kCtlLine + kFusedBuckets) * 128, "bucket lines");
static_assert(kFusedTSlotBytes == HYDRA_GROUP_WS_T_BYTES, "T region as documented in hydra.h");
static_assert(kFusedYBytes == HYDRA_GROUP_WS_Y_BYTES, "y_off region as documented in hydra.h");
constexpr uint32_t kPoison = 1u << 31;
constexpr uint32_t kGenMask = kPoison - 1;
constexpr uint32_t kDefaultWaitBound = 1u << 18;  // s_sleep(1) rounds (~10 ms)
constexpr uint32_t kFinalWaitBound = 1u << 24;    // s_sleep(1) rounds (~1 s)

__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_dev(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t* bucket_word(uint32_t* ctl, int q) {
  return reinterpret_cast<uint64_t*>(ctl + kCtlBucket0 + q * kCtlLine);
}
// The tag that T values of a call with generation word w carry.
__device__ __forceinline__ uint32_t tag_of(uint32_t w) { return (w + 1u) & kGenMask; }

// T rows j0 .. j0 + 7 of one member: T[m][j] = <x[m], A[j]> for rows j < r
// (zero otherwise).  Thread t < 8 MB (wave 0) gets the value of row
// j0 + t / MB, m = t % MB.  Wave w takes row j0 + w / 2 and the chunks c with
// c % 2 == w % 2 of every x segment, so a block of eight rows costs each wave
// half a row; the two partial sums of a row are added in chunk-class order
// through LDS.  (Blocks of 8 rather than 4 rows halve the T workgroups, which
// hold resident slots without streaming W: 16.5 against 16.9 us for the four
// 2048 x 2048 projections at 6 rows and rank 128.)  Every wave of the
// workgroup must call this; it ends with a workgroup barrier.
constexpr int kTRows = 8;   // rows of A per T block
constexpr int kTSplit = SW / kTRows;
template <int MB>
__device__ __forceinline__ float t_rows_dot(const uint16_t* A, int r, int j0, const uint16_t* X, int M, int K,
                                            uint4* xsh, float (*tpart)[MB], int t, int lane, int wave) {
  constexpr int SEG = XSeg<MB>::SEG;
  static_assert(SEG % kTSplit == 0, "every wave takes whole chunks of each segment");
  static_assert(kTRows * MB <= 64, "the stores stay in wave 0");
  const int j = j0 + wave / kTSplit;
  const int cls = wave % kTSplit;
  const bool ok = j < r;
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(ok ? A + (size_t)j * K : nullptr, ok ? (uint32_t)K * 2u : 0u);
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(X, (uint32_t)M * K * 2u);
  const int nch = (K + DKC - 1) / DKC;
  float acc[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m] = 0.f;
  for (int c0 = 0; c0 < nch; c0 += SEG) {
    uint4 ab[SEG / kTSplit];
#pragma unroll
    for (int u = 0; u < SEG / kTSplit; ++u) {
      const int c = c0 + u * kTSplit + cls, k = c * DKC + lane * 8;
      ab[u] = buf_load16(ars, (c < nch && k < K) ? k * 2 : kOutOfRange);
    }
    __syncthreads();  // every wave is done with the previous contents of xsh
    stage_x<MB, SW * 64>(xsh, xrs, c0, nch, K, t);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < SEG / kTSplit; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[m] = dot8(ab[u], xsh[(m * SEG + u * kTSplit + cls) * 64 + lane], acc[m]);
  }
  wave_reduce_scatter<MB>(acc, lane);
  if (reduced_writer<MB>(lane)) tpart[wave][reduced_index<MB>(lane)] = acc[0];
  __syncthreads();
  float v = 0.f;
  if (t < kTRows * MB) {
    const int q = t / MB, m = t % MB;
    v = tpart[q * kTSplit][m];
#pragma unroll
    for (int c = 1; c < kTSplit; ++c) v += tpart[q * kTSplit + c][m];
  }
  __syncthreads();
  return v;
}

// The keeper (wave 0 of the last workgroup): lane q < nbk watches bucket q,
// one load per poll for all buckets, until every workgroup of the call has
// read the generation (bounded); then it writes the next generation, with
// the poison bit if the bound ran out, and zero counts to every line.
__device__ __forceinline__ void keeper(const FusedArgs& fa, int wave, int lane) {
  if (wave != 0) return;
  const int q = lane;
  const bool mine = q < fa.nbk;
  const uint32_t want = mine ? (uint32_t)((fa.total - q + fa.nbk - 1) / fa.nbk) : 0u;
  uint32_t bound = ld_dev(&fa.ctl[kCtlBound]);
  if (bound == 0u) bound = kFinalWaitBound;
  uint64_t w = ld_dev(bucket_word(fa.ctl, mine ? q : 0));
  uint32_t it = 0;
  bool done;
  while (!(done = __builtin_amdgcn_ballot_w64(mine && (uint32_t)w < want) == 0ull) && ++it < bound) {
    __builtin_amdgcn_s_sleep(1);
    w = ld_dev(bucket_word(fa.ctl, mine ? q : 0));
  }
  // every copy of the generation word is the same; past the bound the
  // poison bit is set and stays set
  const uint32_t gw = __builtin_amdgcn_readfirstlane((uint32_t)(w >> 32));
  const uint32_t next = tag_of(gw) | (gw & kPoison) | (done ? 0u : kPoison);
  if (q < kFusedBuckets) st_dev(bucket_word(fa.ctl, q), (uint64_t)next << 32);
}

// A T workgroup: rows jb * 8 .. jb * 8 + 7 of T of one member, each value
// published with the call's tag in one 64-bit device-coherent store.  Thread
// 0 holds the generation word its atomic returned.
template <int MB, int RP>
__device__ __forceinline__ void publish_t(const FusedArgs& fa, int bid, uint64_t gword, uint4* xsh, int t, int lane,
                                          int wave) {
  constexpr int TS = RP > 0 ? RP : 1;
  const GroupArgs& ga = fa.ga;
  const int gi = bid / fa.nT, jb = bid - (bid / fa.nT) * fa.nT;
  const bool on = ga.y_on[gi] != nullptr && ga.A[gi] != nullptr && ga.B[gi] != nullptr;
  if (!on) return;
  __shared__ float tpart[SW][MB];
  const float v = t_rows_dot<MB>(ga.A[gi], ga.r, jb * kTRows, ga.x[gi], ga.M, ga.K, xsh, tpart, t, lane, wave);
  if (wave == 0) {
    // (the whole wave is active here, lane 0 holds the atomic's value)
    const uint64_t tag = tag_of(__builtin_amdgcn_readfirstlane((uint32_t)(gword >> 32)));
    const int q = t / MB, m = t % MB;
    if (t < kTRows * MB && m < ga.M)
      st_dev(&fa.tsl[(gi * kStreamRows + m) * TS + jb * kTRows + q], (tag << 32) | __float_as_uint(v));
  }
}

template <int MB, int RP>
__global__ __launch_bounds__(SW * 64, 8) void gemv_fused_kernel(FusedArgs fa) {
  constexpr int TS = RP > 0 ? RP : 1;
  __shared__ uint4 xsh[XSeg<MB>::ELEMS];
  const GroupArgs& ga = fa.ga;
  const int M = ga.M, N = ga.N, K = ga.K, r = ga.r;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int bid = blockIdx.x;
  const int nTall = ga.G * fa.nT;
  if (RP > 0 && bid == fa.total) {
    keeper(fa, wave, lane);
    return;
  }
  // Read the generation word and report the read (one returning atomic; its
  // value is waited for only where it is used).
  uint64_t gword = 0;
  if (RP > 0 && wave == 0 && lane == 0)
    gword = __hip_atomic_fetch_add(bucket_word(fa.ctl, bid % fa.nbk), uint64_t(1), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
  float acc[MB];
  if (bid < nTall) {
    publish_t<MB, RP>(fa, bid, gword, xsh, t, lane, wave);
    return;
  }
  // ---------------------------------------------- rows of W
  // Every thread requests one entry of its member's T (tagged; MB x RP <=
  // 1024 entries, one per thread) and its row of B next to its first half
  // segment of W; after the first x stage (which waits for all of them) each
  // checks its tag and puts the value in LDS.  Up to 4 rows of x, the rows
  // of W stream in segments of half the staging width (4 KB per wave), so
  // that a thread whose entry was not published yet requests it again just
  // before the last segment's loads, behind half of this workgroup's loads
  // instead of all of them; the shallower queue also serves the rows of W
  // faster.  At 8 rows the segments stay whole (2 KB per wave already).
  constexpr int SEG = MB <= 4 ? XSeg<MB>::SEG / 2 : XSeg<MB>::SEG;
  constexpr int RPL = (TS + 63) / 64;  // j values per lane
  static_assert(MB * TS <= SW * 64, "one T entry per thread");
  __shared__ float tsh[MB][TS];
  __shared__ uint32_t gw_sh, okw[SW];
  const int idx = bid - nTall;
  const int gi = idx / fa.nWB, nb = idx - (idx / fa.nWB) * fa.nWB;
  const int n = nb * 16 + wave;
  const bool row_ok = n < N;
  float* const yo = ga.y_off[gi];
  float* const yn = ga.y_on[gi];
  const bool on = RP > 0 && yn != nullptr && ga.A[gi] != nullptr && ga.B[gi] != nullptr;
  const __amdgpu_buffer_rsrc_t wrs =
      make_rsrc(row_ok ? ga.W[gi] + (size_t)n * K : nullptr, row_ok ? (uint32_t)K * 2u : 0u);
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(ga.x[gi], (uint32_t)M * K * 2u);
  const int nch = (K + DKC - 1) / DKC;
  // this thread's T entry: row t / TS, j = t % TS (the slots of a member are
  // [kStreamRows][TS], so the entry is slot t)
  const bool tent = on && t < MB * TS && t / TS < M;
  const uint64_t* const tslot = fa.tsl + (size_t)gi * kStreamRows * TS + t;
  // tag check of this thread's entry, value into LDS, one flag per wave;
  // returns whether this entry is good
  auto take_t = [&](uint64_t raw) __attribute__((always_inline)) -> bool {
    const bool good = !tent || (uint32_t)(raw >> 32) == tag_of(gw_sh);
    if (tent) tsh[t / TS][t % TS] = __uint_as_float((uint32_t)raw);
    const uint64_t bad = __builtin_amdgcn_ballot_w64(!good);
    if (lane == 0) okw[wave] = bad == 0ull ? 1u : 0u;
    return good;
  };
  // every wave's flag (after a barrier); wave-uniform
  auto all_ok = [&]() __attribute__((always_inline)) -> bool {
    uint32_t v = (gw_sh & kPoison) == 0u ? 1u : 0u;
#pragma unroll
    for (int w = 0; w < SW; ++w) v &= okw[w];
    return v != 0u;
  };
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m] = 0.f;
  float bv[RPL];
#pragma unroll
  for (int q = 0; q < RPL; ++q) bv[q] = 0.f;
  uint64_t traw = 0;
  if (tent) traw = ld_dev(tslot);
  bool stale = false;  // this thread's entry failed its last check
  for (int c0 = 0; c0 < nch; c0 += SEG) {
    const bool again = c0 > 0 && c0 + SEG >= nch && stale;  // the last segment: request the entry again
    if (again) traw = ld_dev(tslot);
    uint4 wb[SEG];
#pragma unroll
    for (int u = 0; u < SEG; ++u) {
      const int c = c0 + u, k = c * DKC + lane * 8;
      wb[u] = buf_load16(wrs, (c < nch && k < K) ? k * 2 : kOutOfRange);
    }
    if (c0 == 0 && on) {
      const __amdgpu_buffer_rsrc_t brs =
          make_rsrc(row_ok ? ga.B[gi] + (size_t)n * r : nullptr, row_ok ? (uint32_t)r * 2u : 0u);
#pragma unroll
      for (int q = 0; q < RPL; ++q) {
        const int jj = q * 64 + lane;
        bv[q] = bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(brs, jj < r ? jj * 2 : kOutOfRange, 0, 0));
      }
    }
    if (c0 > 0) __syncthreads();  // every wave is done with the previous x segment
    stage_x<MB, SW * 64, SEG>(xsh, xrs, c0, nch, K, t);
    if (c0 == 0 && on && t == 0) gw_sh = (uint32_t)(gword >> 32);
    __syncthreads();
    if (on && (c0 == 0 || __builtin_amdgcn_ballot_w64(again) != 0ull)) stale = !take_t(traw);
#pragma unroll
    for (int u = 0; u < SEG; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[m] = dot8(wb[u], xsh[(m * SEG + u) * 64 + lane], acc[m]);
  }
  wave_reduce_scatter<MB>(acc, lane);
  const int m = reduced_index<MB>(lane);
  const bool writer = reduced_writer<MB>(lane) && m < M && row_ok;
  if (writer && yo) yo[(size_t)m * N + n] = acc[0];
  if (on) {
    __syncthreads();  // every wave's flag and T entry are in LDS
    if (!all_ok()) {
      // T was not complete when this workgroup requested it: load it again
      // (bounded; the decision is taken by the whole workgroup), or form it here
      bool ready = false;
      if ((gw_sh & kPoison) == 0u) {
        uint32_t bound = ld_dev(&fa.ctl[kCtlBound]);
        if (bound == 0u) bound = kDefaultWaitBound;
        for (uint32_t it = 0; it < bound; ++it) {
          if (it > 0) __builtin_amdgcn_s_sleep(1);
          __syncthreads();  // every wave has read the previous flags
          take_t(tent ? ld_dev(tslot) : uint64_t(0));
          __syncthreads();
          if ((ready = all_ok())) break;
        }
      }
      if (!ready) {
        // T formed here, block by block as the T workgroups do
        __shared__ float tpart2[SW][MB];
        __syncthreads();  // every wave is done with the flags and tsh
        for (int q = t; q < MB * TS; q += SW * 64) tsh[q / TS][q % TS] = 0.f;
        for (int jb = 0; jb < fa.nT; ++jb) {
          const float v = t_rows_dot<MB>(ga.A[gi], r, jb * kTRows, ga.x[gi], M, K, xsh, tpart2, t, lane, wave);
          const int q = t / MB, mm = t % MB;
          if (t < kTRows * MB && mm < M) tsh[mm][jb * kTRows + q] = v;
        }
        __syncthreads();
      }
    }
    // d[m] = sum_j T[m][j] B[n][j]: lane l holds j = l, l + 64
    float part[MB];
#pragma unroll
    for (int mm = 0; mm < MB; ++mm) {
      part[mm] = 0.f;
#pragma unroll
      for (int q = 0; q < RPL; ++q) {
        const int jj = q * 64 + lane;
        part[mm] = fmaf(jj < TS && mm < M ? tsh[mm][jj] : 0.f, bv[q], part[mm]);
      }
    }
    wave_reduce_scatter<MB>(part, lane);
    if (writer) yn[(size_t)m * N + n] = acc[0] + ga.s[gi] * part[0];
  } else if (writer && yn) {
    yn[(size_t)m * N + n] = acc[0];
  }
}

// ---------------------------------------------------------------- decode in one launch, small ranks
// At padded rank 16 and up to 4 rows of x the rows of A are few (16 per
// member: 64 KB at K = 2048, read from L2 after the first workgroup of each
// XCD) and their registers fit beside those of W (at rank 32, or 8 rows, the
// kernel would spill; those run the published-T kernel below), so every
// workgroup forms T = x A^T itself: wave w streams its row of W and row w of
// A against the same staged x, in the same segments, so the
// A requests ride with the W requests and no workgroup waits for another.
// T is reduced by the same butterfly as the rows of W (the same bits in every
// workgroup) and shared through LDS.  Each segment issues its x loads first,
// then the rows of W and A (the first also the row of B), all unconditional
// (out-of-range offsets where there is nothing to load), so that the
// compiler's waits count exactly the requests issued after the one they wait
// for: waiting for x never waits for W, and the dot products wait for each
// chunk as it arrives.
template <int MB, int RP>
__global__ __launch_bounds__(SW * 64, 8) void gemv_selft_kernel(GroupArgs ga) {
  static_assert((RP == 0 || RP == 16) && MB <= 4, "rank 0 or 16, up to 4 rows");
  constexpr int AR = RP / 16;                            // rows of A per wave
  constexpr int TS = RP > 0 ? RP : 1;
  constexpr int SEG = MB <= 4 ? XSeg<MB>::SEG / 2 : XSeg<MB>::SEG;
  constexpr int XE = MB * SEG * 64;                      // staged x elements per segment
  constexpr int XPER = (XE + SW * 64 - 1) / (SW * 64);   // ... per thread
  __shared__ uint4 xsh[XSeg<MB>::ELEMS];
  __shared__ float tsh[MB][TS];
  const int M = ga.M, N = ga.N, K = ga.K, r = ga.r;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int nWB = (N + SW - 1) / SW;
  const int gi = blockIdx.x / nWB, nb = blockIdx.x - (blockIdx.x / nWB) * nWB;
  const int n = nb * 16 + wave;
  const bool row_ok = n < N;
  float* const yo = ga.y_off[gi];
  float* const yn = ga.y_on[gi];
  const bool on = RP > 0 && yn != nullptr && ga.A[gi] != nullptr && ga.B[gi] != nullptr;
  const __amdgpu_buffer_rsrc_t wrs =
      make_rsrc(row_ok ? ga.W[gi] + (size_t)n * K : nullptr, row_ok ? (uint32_t)K * 2u : 0u);
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(ga.x[gi], (uint32_t)M * K * 2u);
  const __amdgpu_buffer_rsrc_t brs =
      make_rsrc(on && row_ok ? ga.B[gi] + (size_t)n * r : nullptr, on && row_ok ? (uint32_t)r * 2u : 0u);
  __amdgpu_buffer_rsrc_t ars[AR > 0 ? AR : 1];
#pragma unroll
  for (int q = 0; q < AR; ++q) {
    const int j = wave + 16 * q;
    const bool ok = on && j < r;
    ars[q] = make_rsrc(ok ? ga.A[gi] + (size_t)j * K : nullptr, ok ? (uint32_t)K * 2u : 0u);
  }
  const int nch = (K + DKC - 1) / DKC;
  float acc[MB], tacc[AR > 0 ? AR : 1][MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    acc[m] = 0.f;
#pragma unroll
    for (int q = 0; q < AR; ++q) tacc[q][m] = 0.f;
  }
  uint32_t braw = 0u;  // this lane's entry of the row of B (j = lane), converted in the epilogue
  for (int c0 = 0; c0 < nch; c0 += SEG) {
    uint4 xv[XPER];
#pragma unroll
    for (int q = 0; q < XPER; ++q) {
      const int e = t + q * SW * 64;
      const int m = e / (SEG * 64), u = (e / 64) % SEG, l = e % 64;
      const int c = c0 + u, k = c * DKC + l * 8;
      xv[q] = buf_load16(xrs, (e < XE && c < nch && k < K) ? (m * K + k) * 2 : kOutOfRange);
    }
    asm volatile("" ::: "memory");
    uint4 wb[SEG], ab[AR > 0 ? AR : 1][SEG];
#pragma unroll
    for (int u = 0; u < SEG; ++u) {
      const int c = c0 + u, k = c * DKC + lane * 8;
      const int off = (c < nch && k < K) ? k * 2 : kOutOfRange;
      wb[u] = buf_load16(wrs, off);
#pragma unroll
      for (int q = 0; q < AR; ++q) ab[q][u] = buf_load16(ars[q], off);
    }
    if constexpr (RP > 0) {
      // (every segment issues it; past the first its offset is out of range)
      const uint32_t bnew = __builtin_amdgcn_raw_buffer_load_b16(brs, c0 == 0 && lane < r ? lane * 2 : kOutOfRange, 0, 0);
      braw |= bnew;  // zero except in the first segment
    }
    asm volatile("" ::: "memory");
    if (c0 > 0) __syncthreads();  // every wave is done with the previous x segment
#pragma unroll
    for (int q = 0; q < XPER; ++q) {
      const int e = t + q * SW * 64;
      if (e < XE) xsh[e] = xv[q];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < SEG; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        const uint4 xm = xsh[(m * SEG + u) * 64 + lane];
        acc[m] = dot8(wb[u], xm, acc[m]);
#pragma unroll
        for (int q = 0; q < AR; ++q) tacc[q][m] = dot8(ab[q][u], xm, tacc[q][m]);
      }
  }
  wave_reduce_scatter<MB>(acc, lane);
  const int m = reduced_index<MB>(lane);
  const bool writer = reduced_writer<MB>(lane) && m < M && row_ok;
  if (writer && yo) yo[(size_t)m * N + n] = acc[0];
  if constexpr (RP > 0) {
    if (on) {
#pragma unroll
      for (int q = 0; q < AR; ++q) {
        wave_reduce_scatter<MB>(tacc[q], lane);
        if (reduced_writer<MB>(lane)) tsh[m][wave + 16 * q] = tacc[q][0];  // T[m][j] (zero for j >= r)
      }
      __syncthreads();
      // d[m] = sum_j T[m][j] B[n][j]: lane l holds j = l
      float part[MB];
#pragma unroll
      for (int mm = 0; mm < MB; ++mm) part[mm] = lane < RP && mm < M ? tsh[mm][lane] * bf16_to_f32(braw) : 0.f;
      wave_reduce_scatter<MB>(part, lane);
      if (writer) yn[(size_t)m * N + n] = acc[0] + ga.s[gi] * part[0];
      return;
    }
  }
  if (writer && yn) yn[(size_t)m * N + n] = acc[0];
}

// ---------------------------------------------------------------- decode in one launch, LoRA at the tail
// The same three kinds of workgroup as gemv_fused_kernel, plus a fourth, but
// no workgroup that streams W ever waits:
//  * T workgroups (first in the grid) publish tagged T as there;
//  * W workgroups stream their 16 rows of W exactly as gemv_selft_kernel does
//    at rank 0 and write y_off; for a member with an adapter they also
//    publish each value of y_off, tagged like T, in the workspace, and leave
//    y_on alone;
//  * update workgroups (after all W workgroups in the grid, so they start as
//    the stream ends) each take 128 rows of one member (64 from rank 64 on,
//    or with 8 rows of x): they load the rows of
//    B and the published T, form d = s T B^T, wait (bounded) for the tagged
//    y_off of their rows and write y_on = y_off + d.  Every y_off they wait
//    for comes from a workgroup the hardware dispatched earlier.
//  * the keeper, as there.
// An update workgroup that finds a value missing past its bound (or a
// poisoned generation) computes T, or its rows' y_off, itself, through the
// same routines as the T and W workgroups, so the bits are the same.
struct SplitArgs {
  FusedArgs f;
  uint64_t* ysl;  // tagged y_off [G][N][MB]: (tag << 32) | value bits
  int nUB;        // update workgroups per member
};
// threads per row of an update workgroup (each takes RP / that many j) and
// rows per update workgroup
constexpr int upd_tpr(int mb, int rp) { return rp >= 64 || mb == 8 ? 16 : 8; }
constexpr int upd_rows(int mb, int rp) { return SW * 64 / upd_tpr(mb, rp); }

// Base products <x[m], W[n]> of the 16 rows n = nb * 16 + wave of member gi,
// one wave per row, streamed as in gemv_selft_kernel at rank 0: each segment
// issues its x loads first, then the row of W, all unconditional (out-of-range
// offsets where there is nothing to load), so that waiting for x never waits
// for W.  Returns this lane's sum after the reduce-scatter (row n, m =
// reduced_index<MB>(lane)).  Every wave of the workgroup must call it (it has
// workgroup barriers).  With gw_dst set, thread 0 stores the high half of
// its gword there before the first barrier, for the whole workgroup to read.
template <int MB>
__device__ __forceinline__ float stream_rows(const GroupArgs& ga, int gi, int nb, uint4* xsh, int t, int lane,
                                             int wave, uint32_t* gw_dst, uint64_t gword) {
  constexpr int SEG = MB <= 4 ? XSeg<MB>::SEG / 2 : XSeg<MB>::SEG;
  constexpr int XE = MB * SEG * 64;                      // staged x elements per segment
  constexpr int XPER = (XE + SW * 64 - 1) / (SW * 64);   // ... per thread
  const int M = ga.M, N = ga.N, K = ga.K;
  const int n = nb * 16 + wave;
  const bool row_ok = n < N;
  const __amdgpu_buffer_rsrc_t wrs =
      make_rsrc(row_ok ? ga.W[gi] + (size_t)n * K : nullptr, row_ok ? (uint32_t)K * 2u : 0u);
  const __amdgpu_buffer_rsrc_t xrs = make_rsrc(ga.x[gi], (uint32_t)M * K * 2u);
  const int nch = (K + DKC - 1) / DKC;
  float acc[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m] = 0.f;
#pragma unroll 1
  for (int c0 = 0; c0 < nch; c0 += SEG) {
    uint4 xv[XPER];
#pragma unroll
    for (int q = 0; q < XPER; ++q) {
      const int e = t + q * SW * 64;
      const int m = e / (SEG * 64), u = (e / 64) % SEG, l = e % 64;
      const int c = c0 + u, k = c * DKC + l * 8;
      xv[q] = buf_load16(xrs, (e < XE && c < nch && k < K) ? (m * K + k) * 2 : kOutOfRange);
    }
    asm volatile("" ::: "memory");
    uint4 wb[SEG];
#pragma unroll
    for (int u = 0; u < SEG; ++u) {
      const int c = c0 + u, k = c * DKC + lane * 8;
      wb[u] = buf_load16(wrs, (c < nch && k < K) ? k * 2 : kOutOfRange);
    }
    asm volatile("" ::: "memory");
    if (c0 > 0) __syncthreads();  // every wave is done with the previous x segment
#pragma unroll
    for (int q = 0; q < XPER; ++q) {
      const int e = t + q * SW * 64;
      if (e < XE) xsh[e] = xv[q];
    }
    if (gw_dst && t == 0) *gw_dst = (uint32_t)(gword >> 32);  // (the same value in every segment)
    __syncthreads();
#pragma unroll
    for (int u = 0; u < SEG; ++u)
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[m] = dot8(wb[u], xsh[(m * SEG + u) * 64 + lane], acc[m]);
  }
  wave_reduce_scatter<MB>(acc, lane);
  return acc[0];
}

template <int MB, int RP>
__global__ __launch_bounds__(SW * 64, 8) void gemv_split_kernel(SplitArgs sa) {
  static_assert(RP > 0 && RP <= 64, "the split form carries a LoRA update up to rank 64");
  constexpr int TS = RP;
  const FusedArgs& fa = sa.f;
  __shared__ uint4 xsh[XSeg<MB>::ELEMS];
  __shared__ uint32_t gw_sh;
  const GroupArgs& ga = fa.ga;
  const int M = ga.M, N = ga.N, K = ga.K, r = ga.r;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int bid = blockIdx.x;
  const int nTall = ga.G * fa.nT;
  const int nWall = ga.G * fa.nWB;
  if (bid == fa.total) {
    keeper(fa, wave, lane);
    return;
  }
  // the generation, read and reported by one returning atomic
  uint64_t gword = 0;
  if (wave == 0 && lane == 0)
    gword = __hip_atomic_fetch_add(bucket_word(fa.ctl, bid % fa.nbk), uint64_t(1), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
  if (bid < nTall) {
    publish_t<MB, RP>(fa, bid, gword, xsh, t, lane, wave);
    return;
  }
  if (bid < nTall + nWall) {
    // ---------------------------------------------- rows of W
    const int idx = bid - nTall;
    const int gi = idx / fa.nWB, nb = idx - (idx / fa.nWB) * fa.nWB;
    float* const yo = ga.y_off[gi];
    float* const yn = ga.y_on[gi];
    const bool on = yn != nullptr && ga.A[gi] != nullptr && ga.B[gi] != nullptr;
    const float v = stream_rows<MB>(ga, gi, nb, xsh, t, lane, wave, on ? &gw_sh : nullptr, gword);
    const int n = nb * 16 + wave;
    const int m = reduced_index<MB>(lane);
    const bool writer = reduced_writer<MB>(lane) && m < M && n < N;
    if (writer && yo) yo[(size_t)m * N + n] = v;
    if (on) {
      // (gw_sh was written before the stream's first barrier)
      if (writer && (gw_sh & kPoison) == 0u)
        st_dev(&sa.ysl[((size_t)gi * N + n) * MB + m], ((uint64_t)tag_of(gw_sh) << 32) | __float_as_uint(v));
    } else if (writer && yn) {
      yn[(size_t)m * N + n] = v;
    }
    return;
  }
  // ---------------------------------------------- LoRA update of y_on
  __shared__ float tsh[MB][TS];
  __shared__ uint32_t okw[SW];
  const int uidx = bid - nTall - nWall;
  const int gi = uidx / sa.nUB, ub = uidx - (uidx / sa.nUB) * sa.nUB;
  float* const yn = ga.y_on[gi];
  if (yn == nullptr || ga.A[gi] == nullptr || ga.B[gi] == nullptr) return;  // member without an adapter
  constexpr int TPR = upd_tpr(MB, RP);
  constexpr int UR = upd_rows(MB, RP);
  constexpr int JPT = RP / TPR;  // j values per thread
  static_assert(JPT * TPR == RP && TPR >= MB, "whole j ranges; thread q of a row writes m = q");
  const int nl = t / TPR, q = t % TPR;
  const int n = ub * UR + nl;
  const bool row_ok = n < N;
  // this thread's piece of the row of B (j = q JPT .. q JPT + JPT - 1, zero past r), requested first; one
  // descriptor for the member's whole B (a per-row descriptor would not be wave-uniform)
  const __amdgpu_buffer_rsrc_t brs = make_rsrc(ga.B[gi], (uint32_t)N * r * 2u);
  uint32_t braw[JPT];
#pragma unroll
  for (int i = 0; i < JPT; ++i) {
    const int j = q * JPT + i;
    braw[i] = __builtin_amdgcn_raw_buffer_load_b16(brs, row_ok && j < r ? (n * r + j) * 2 : kOutOfRange, 0, 0);
  }
  // this thread's entry of T (one per thread: row t / TS, j = t % TS)
  const bool tent = t < MB * TS && t / TS < M;
  const uint64_t* const tslot = fa.tsl + (size_t)gi * kStreamRows * TS + t;
  uint64_t traw = tent ? ld_dev(tslot) : 0ull;
  // this thread's tagged y_off (thread q of a row takes m = q)
  const bool yent = row_ok && q < MB && q < M;
  const uint64_t* const yslot = sa.ysl + ((size_t)gi * N + n) * MB + q;
  uint64_t yraw = yent ? ld_dev(yslot) : 0ull;
  if (t == 0) gw_sh = (uint32_t)(gword >> 32);
  __syncthreads();
  const uint32_t gw = gw_sh;
  const bool poisoned = (gw & kPoison) != 0u;
  const uint32_t tag = tag_of(gw);
  uint32_t bound = ld_dev(&fa.ctl[kCtlBound]);
  if (bound == 0u) bound = kDefaultWaitBound;
  // T into LDS: every entry tagged with this call's tag, else (bounded) again, else formed here
  auto take_t = [&](uint64_t raw) __attribute__((always_inline)) -> bool {
    const bool good = !tent || (uint32_t)(raw >> 32) == tag;
    if (tent) tsh[t / TS][t % TS] = __uint_as_float((uint32_t)raw);
    const uint64_t bad = __builtin_amdgcn_ballot_w64(!good);
    if (lane == 0) okw[wave] = bad == 0ull ? 1u : 0u;
    return good;
  };
  auto all_ok = [&]() __attribute__((always_inline)) -> bool {
    uint32_t v = 1u;
#pragma unroll
    for (int w = 0; w < SW; ++w) v &= okw[w];
    return v != 0u;
  };
  bool ready = false;
  if (!poisoned) {
    take_t(traw);
    __syncthreads();
    ready = all_ok();
    for (uint32_t it = 0; !ready && it < bound; ++it) {
      __builtin_amdgcn_s_sleep(1);
      __syncthreads();  // every wave has read the previous flags
      take_t(tent ? ld_dev(tslot) : 0ull);
      __syncthreads();
      ready = all_ok();
    }
  }
  if (!ready) {
    __shared__ float tpart[SW][MB];
    __syncthreads();  // every wave is done with the flags and tsh
    for (int e = t; e < MB * TS; e += SW * 64) tsh[e / TS][e % TS] = 0.f;
    for (int jb = 0; jb < fa.nT; ++jb) {
      const float v = t_rows_dot<MB>(ga.A[gi], r, jb * kTRows, ga.x[gi], M, K, xsh, tpart, t, lane, wave);
      const int qq = t / MB, mm = t % MB;
      if (t < kTRows * MB && mm < M) tsh[mm][jb * kTRows + qq] = v;
    }
  }
  __syncthreads();  // T complete in LDS
  // d[m] over this thread's j range, then summed over the row's TPR threads (butterfly: every thread of the row
  // ends with the same bits)
  float d[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) {
    d[m] = 0.f;
#pragma unroll
    for (int i = 0; i < JPT; ++i) {
      const int j = q * JPT + i;
      d[m] = fmaf(j < TS && m < M ? tsh[m][j] : 0.f, bf16_to_f32(braw[i]), d[m]);
    }
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1)
#pragma unroll
    for (int m = 0; m < MB; ++m) d[m] += __shfl_xor(d[m], o);
  float dq = 0.f;
#pragma unroll
  for (int m = 0; m < MB; ++m) dq = q == m ? d[m] : dq;
  // the row's y_off, published by its W workgroup (bounded wait), else formed here
  bool ygood = !yent || (!poisoned && (uint32_t)(yraw >> 32) == tag);
  if (!poisoned)
    for (uint32_t it = 0; !ygood && it < bound; ++it) {
      __builtin_amdgcn_s_sleep(1);
      yraw = ld_dev(yslot);
      ygood = (uint32_t)(yraw >> 32) == tag;
    }
  const uint64_t badw = __builtin_amdgcn_ballot_w64(!ygood);
  if (lane == 0) okw[wave] = badw == 0ull ? 1u : 0u;
  __syncthreads();
  const float s = ga.s[gi];
  if (all_ok()) {
    if (yent) yn[(size_t)q * N + n] = __uint_as_float((uint32_t)yraw) + s * dq;
    return;
  }
  // some y_off did not arrive: this workgroup streams its own rows (16 per pass, the W workgroups' routine and
  // bits) and writes every row's y_on from them
  __shared__ float ysh[UR][MB];
  __syncthreads();  // every wave is done with the flags
  for (int p = 0; p < UR / 16; ++p) {
    const int nb = (ub * UR) / 16 + p;
    const float v = stream_rows<MB>(ga, gi, nb, xsh, t, lane, wave, nullptr, 0ull);
    const int m = reduced_index<MB>(lane);
    if (reduced_writer<MB>(lane)) ysh[p * 16 + wave][m] = v;
  }
  __syncthreads();
  if (row_ok && q < MB && q < M) yn[(size_t)q * N + n] = ysh[nl][q] + s * dq;
}

template <int MB>
hipError_t launch_split_mb(const SplitArgs& sa, int rp, hipStream_t stream) {
  const dim3 grid(sa.f.total + 1), block(SW * 64);
  switch (rp) {
    case 16: hipLaunchKernelGGL((gemv_split_kernel<MB, 16>), grid, block, 0, stream, sa); break;
    case 32: hipLaunchKernelGGL((gemv_split_kernel<MB, 32>), grid, block, 0, stream, sa); break;
    case 64: hipLaunchKernelGGL((gemv_split_kernel<MB, 64>), grid, block, 0, stream, sa); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int MB>
hipError_t launch_selft_mb(const GroupArgs& g, int rp, hipStream_t stream) {
  const dim3 grid(g.G * ((g.N + SW - 1) / SW)), block(SW * 64);
  if (rp == 16)
    hipLaunchKernelGGL((gemv_selft_kernel<MB, 16>), grid, block, 0, stream, g);
  else
    hipLaunchKernelGGL((gemv_selft_kernel<MB, 0>), grid, block, 0, stream, g);
  return hipGetLastError();
}

template <int MB>
hipError_t launch_fused_mb(const FusedArgs& fa, int rp, hipStream_t stream) {
  // the keeper runs only where there is T to publish
  const dim3 grid(fa.total + (rp > 0 ? 1 : 0)), block(SW * 64);
  switch (rp) {
    case 0: hipLaunchKernelGGL((gemv_fused_kernel<MB, 0>), grid, block, 0, stream, fa); break;
    case 16: hipLaunchKernelGGL((gemv_fused_kernel<MB, 16>), grid, block, 0, stream, fa); break;
    case 32: hipLaunchKernelGGL((gemv_fused_kernel<MB, 32>), grid, block, 0, stream, fa); break;
    case 64: hipLaunchKernelGGL((gemv_fused_kernel<MB, 64>), grid, block, 0, stream, fa); break;
    default: hipLaunchKernelGGL((gemv_fused_kernel<MB, 128>), grid, block, 0, stream, fa); break;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemv_stream(const StreamArgs& a_in, hipStream_t stream) {
  StreamArgs a = a_in;
  stream_finish_args(a);
  const dim3 grid((a.N + SW - 1) / SW, a.G), block(SW * 64);
  int rows = 0;
  for (int i = 0; i < a.G; ++i) rows = a.nseg[i] * a.seg_rows > rows ? a.nseg[i] * a.seg_rows : rows;
  if (rows <= 1) hipLaunchKernelGGL((gemv_stream_kernel<1>), grid, block, 0, stream, a);
  else if (rows <= 2) hipLaunchKernelGGL((gemv_stream_kernel<2>), grid, block, 0, stream, a);
  else if (rows <= 4) hipLaunchKernelGGL((gemv_stream_kernel<4>), grid, block, 0, stream, a);
  else hipLaunchKernelGGL((gemv_stream_kernel<8>), grid, block, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gemv_fused(const GroupArgs& g, void* ws, hipStream_t stream) {
  bool any_on = false;
  for (int i = 0; i < g.G; ++i) any_on = any_on || (g.y_on[i] && g.A[i] && g.B[i]);
  const int rp = any_on ? padded_rank(g.r) : 0;
  // Up to 4 rows: rank 0 takes the plain stream of gemv_selft_kernel (26.0
  // against 26.4 us for the four Llama-7B projections), and rank 16 with
  // K <= 2048 forms T in every workgroup (12.4 against 13.1 us for four
  // 2048 x 2048 projections); the workspace is not used.  At K = 4096 the rows
  // of A, as many bytes per workgroup as its rows of W, slow the stream more
  // than the hand-off of published T costs (34.4 against 30.6 us).
  if (g.M <= 4 && (rp == 0 || (rp == 16 && g.K <= 2048))) {
    if (g.M <= 1) return launch_selft_mb<1>(g, rp, stream);
    if (g.M <= 2) return launch_selft_mb<2>(g, rp, stream);
    return launch_selft_mb<4>(g, rp, stream);
  }
  FusedArgs fa{};
  fa.ga = g;
  fa.ctl = static_cast<uint32_t*>(ws);
  fa.tsl = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + kFusedCtlBytes);
  fa.nT = rp / kTRows;
  fa.nWB = (g.N + SW - 1) / SW;
  const int mb = g.M <= 1 ? 1 : g.M <= 2 ? 2 : g.M <= 4 ? 4 : 8;
  // Up to rank 64 the LoRA update runs at the tail of the grid and no
  // workgroup that streams W waits: four Llama-7B projections (M = 4, K = N =
  // 4096, r = 16) take 29.2-30.0 against 30.6-32.1 us, four 2048 x 2048 at M
  // = 6 take 13.7-14.3 against 15.7-16.1 us.  At rank 128 the tail takes
  // longer than the hand-off it saves (M = 4: 31.1 against 30.1 us; M = 8:
  // 47.2 against 38.7 us), so rank 128 keeps gemv_fused_kernel.
  if (rp > 0 && rp <= 64 && (size_t)g.G * g.N * mb * 8 <= kFusedYBytes) {
    SplitArgs sa{};
    sa.f = fa;
    sa.ysl = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + kFusedCtlBytes + kFusedTSlotBytes);
    const int ur = upd_rows(mb, rp);
    sa.nUB = (g.N + ur - 1) / ur;
    sa.f.total = g.G * (fa.nT + fa.nWB + sa.nUB);
    sa.f.nbk = sa.f.total < kFusedBuckets ? sa.f.total : kFusedBuckets;
    if (mb == 1) return launch_split_mb<1>(sa, rp, stream);
    if (mb == 2) return launch_split_mb<2>(sa, rp, stream);
    if (mb == 4) return launch_split_mb<4>(sa, rp, stream);
    return launch_split_mb<8>(sa, rp, stream);
  }
  fa.total = g.G * (fa.nT + fa.nWB);
  fa.nbk = fa.total < kFusedBuckets ? fa.total : kFusedBuckets;
  if (g.M <= 1) return launch_fused_mb<1>(fa, rp, stream);
  if (g.M <= 2) return launch_fused_mb<2>(fa, rp, stream);
  if (g.M <= 4) return launch_fused_mb<4>(fa, rp, stream);
  return launch_fused_mb<8>(fa, rp, stream);
}

hipError_t launch_lora_update(const GroupArgs& g, hipStream_t stream) {
  const int rp = padded_rank(g.r);
  if (rp == 0) return hipSuccess;
  if (g.M <= 1) return launch_update_mb<1>(g, rp, stream);
  if (g.M <= 2) return launch_update_mb<2>(g, rp, stream);
  if (g.M <= 4) return launch_update_mb<4>(g, rp, stream);
  return launch_update_mb<8>(g, rp, stream);
}

hipError_t launch_lora_gemv_group(const GroupArgs& g, hipStream_t stream) {
  bool any_on = false;
  for (int i = 0; i < g.G; ++i) any_on = any_on || g.y_on[i] != nullptr;
  const int r = any_on ? g.r : 0;
  const int rp = padded_rank(r);
  if (g.M > kStreamRows && rp > 64) {
    // rank 128 above 8 rows: the MFMA kernel's per-workgroup T does not fit;
    // the rows go through the stream and update kernels in two halves
    GroupArgs lo = g, hi = g;
    lo.M = kStreamRows;
    hi.M = g.M - kStreamRows;
    for (int i = 0; i < g.G; ++i) {
      hi.x[i] = g.x[i] + (size_t)kStreamRows * g.K;
      hi.y_off[i] = g.y_off[i] ? g.y_off[i] + (size_t)kStreamRows * g.N : nullptr;
      hi.y_on[i] = g.y_on[i] ? g.y_on[i] + (size_t)kStreamRows * g.N : nullptr;
    }
    const hipError_t e = launch_lora_gemv_group(lo, stream);
    return e != hipSuccess ? e : launch_lora_gemv_group(hi, stream);
  }
  if (g.M <= kStreamRows) {
    // base product of every member into y_off and y_on, then the LoRA update of y_on
    StreamArgs sa{};
    sa.G = g.G;
    sa.seg_rows = g.M;
    sa.N = g.N;
    sa.K = g.K;
    for (int i = 0; i < g.G; ++i) {
      sa.W[i] = g.W[i];
      sa.seg0[i] = i;
      sa.nseg[i] = 1;
      sa.x[i] = g.x[i];
      sa.ya[i] = g.y_off[i];
      sa.yb[i] = g.y_on[i];
    }
    hipError_t e = launch_gemv_stream(sa, stream);
    if (e != hipSuccess || rp == 0) return e;
    return launch_lora_update(g, stream);
  }
  // The widest column block that still gives at least one workgroup per CU:
  // wider blocks amortise the per-workgroup reads of A over more of W.
  const long wg64 = (long)((g.N + 63) / 64) * g.G;
  const long wg32 = (long)((g.N + 31) / 32) * g.G;
  if (wg64 >= 256) return launch_nb<64>(g, rp, stream);
  if (wg32 >= 256) return launch_nb<32>(g, rp, stream);
  return launch_nb<16>(g, rp, stream);
}

}  // namespace hydra
