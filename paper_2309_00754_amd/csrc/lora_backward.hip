// Backward of the LoRA-switchable linear with the base weight frozen (the
// update stage of Hydra-PPO trains only the active adapter, Sec. 3 and
// App. A, Alg. 2).  With y = x W^T + s (x A^T) B^T, T = x A^T and U = dy B:
//   dx = dy W + s U A,   dA = s U^T x,   dB = s dy^T T.
// Steps, all on one stream:
//  1. B^T and A^T, zero padded to the padded rank RP (transpose_pad_kernel,
//     both in one launch);
//  2. the LoRA pre-pass of the forward GEMM (lora_tpre.hip) twice, in one
//     pair of launches: s U from dy against the rows of B^T, s T from x
//     against A, each as bf16 hi and lo parts (row-major for step 3,
//     transposed for step 4);
//  3. dx by the forward's MFMA GEMM run on (dy, W^T), its LoRA slabs being
//     [hi | lo](s U) against rows of A^T: one pass over W^T, as in the forward;
//  4. dA and dB as sums of outer products over the rows m:
//     out[j][c] = sum_m P[m][j] Q[m][c] with (P, Q) = (s U, x) and (s T, dy),
//     on MFMAs (lora_outer_part_kernel: per row chunk partials, laid out like
//     the output), then the chunks added in chunk order
//     (lora_outer_finish_kernel, one thread per output element); dA and dB
//     share each of the two launches.  Every sum has a fixed order: the results
//     are the same from run to run.
#include <algorithm>

#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

// ------------------------------------------------------------ transpose_pad
constexpr int TP = 64;  // tile edge

struct TransposeJob {
  const uint16_t* src;  // [R x C]
  uint16_t* dst;        // [Cp x Rp]
  int R, C, Rp, Cp;
  int gx;               // tiles along Cp
};

// dst[c][q] = src[q][c] inside src's [R x C], zero outside, for the 64 x 64
// tile b of the job (tile b % gx along dst's rows, b / gx along its columns).
__device__ __forceinline__ void transpose_tile(const TransposeJob& j, int b) {
  __shared__ uint16_t tile[TP][TP + 2];
  const int c0 = (b % j.gx) * TP, q0 = (b / j.gx) * TP;
  const int lx = threadIdx.x & 63, ly = threadIdx.x >> 6;
  uint16_t v[TP / 4];
#pragma unroll
  for (int i = 0; i < TP / 4; ++i) {
    const int q = q0 + ly + 4 * i, c = c0 + lx;
    v[i] = (q < j.R && c < j.C) ? j.src[(size_t)q * j.C + c] : (uint16_t)0;
  }
#pragma unroll
  for (int i = 0; i < TP / 4; ++i) tile[ly + 4 * i][lx] = v[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < TP / 4; ++i) {
    const int c = c0 + ly + 4 * i, q = q0 + lx;
    if (c < j.Cp && q < j.Rp) j.dst[(size_t)c * j.Rp + q] = tile[lx][ly + 4 * i];
  }
}

// Up to two transposes in one launch: workgroups [0, n0) take job j0's tiles,
// the rest j1's.
__global__ __launch_bounds__(256) void transpose_pad_kernel(TransposeJob j0, int n0, TransposeJob j1) {
  const int b = blockIdx.x;
  if (b < n0)
    transpose_tile(j0, b);
  else
    transpose_tile(j1, b - n0);
}

TransposeJob transpose_job(const uint16_t* src, int R, int C, uint16_t* dst, int Rp, int Cp, int& tiles) {
  TransposeJob j{src, dst, R, C, Rp, Cp, (Cp + TP - 1) / TP};
  tiles = j.gx * ((Rp + TP - 1) / TP);
  return j;
}

// ---------------------------------------------------------- outer products
constexpr int O_WAVES = 4;
constexpr int O_COLS = 256;        // columns per workgroup: 64 per wave, four 16-column MFMA tiles
constexpr int O_KS = 32;           // rows per k-step (the k of one 16x16x32 MFMA)
constexpr int O_LD = O_COLS + 4;   // LDS row stride in bf16 (130 dwords; see outer_part)
constexpr int O_TARGET_WG = 256;   // workgroups the chunking aims for (both products together: twice that)
constexpr int O_MIN_ROWS = 128;    // fewest rows per chunk

struct OuterArgs {
  const uint16_t* PT;  // [2][RP][Mp] bf16: hi and lo planes of P^T (P = s U or s T)
  const uint16_t* Q;   // [M x C] bf16
  float* part;         // [nch x RP x C] (jc) or [nch x C x RP] fp32
  float* out;          // [r x C] (jc) or [C x r] fp32
  int M, Mp, C, RP, r;
  int mch, nch;        // rows per chunk (multiple of O_KS), chunks
  int jc;              // partials and output j-major
  int tiles;           // column tiles of O_COLS
};

// Partial out[j][c] = sum_m P[m][j] Q[m][c] over the rows of one chunk, for
// every j and the 256 columns of one tile (b = tile + tiles * chunk), on
// v_mfma_f32_16x16x32_bf16: A operand = 16 j x 32 m of P^T (its hi plane,
// then its lo plane: ~16 significant bits of P), B operand = 32 m x 16
// columns of Q.  The MFMA wants eight consecutive m per lane, but m is Q's
// row index, so each 32-row slab of Q goes through LDS (row-major, double
// buffered, one barrier per slab) and every lane gathers its column's eight
// values with 16-bit reads.  With a row stride of 130 dwords the four row
// groups of one read land in disjoint bank windows.  Each wave owns 64
// columns and all RP j, so one slab in LDS serves every 16-wide j group.
template <int RP>
__device__ __forceinline__ void outer_part(const OuterArgs& a, int b) {
  constexpr int JG = RP / 16;
  __shared__ uint16_t qs[2][O_KS][O_LD];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int l16 = lane & 15, lg = lane >> 4;
  const int tile = b % a.tiles;
  const int ch = b / a.tiles;
  const int c0 = tile * O_COLS;
  const int m_begin = ch * a.mch;
  const int m_end = min(a.M, m_begin + a.mch);
  const int nks = (m_end - m_begin + O_KS - 1) / O_KS;
  // slab copies: thread t moves 16 bytes (8 columns) of rows t / 32 + 8 u
  const int lr = t >> 5, lc = (t & 31) * 8;
  uint4 qv[4];
  auto load = [&](int ks) __attribute__((always_inline)) {
    const int m0 = m_begin + ks * O_KS;
    const int rows = min(O_KS, m_end - m0);
    const __amdgpu_buffer_rsrc_t qrs = make_rsrc(a.Q + (size_t)m0 * a.C, (uint32_t)rows * a.C * 2u);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int row = lr + 8 * u;
      qv[u] = buf_load16(qrs, (row < rows && c0 + lc < a.C) ? (row * a.C + c0 + lc) * 2 : kOutOfRange);
    }
  };
  auto store = [&](int st) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint2* d = reinterpret_cast<uint2*>(&qs[st][lr + 8 * u][lc]);
      d[0] = uint2{qv[u].x, qv[u].y};
      d[1] = uint2{qv[u].z, qv[u].w};
    }
  };
  f32x4_t acc[JG][4];
#pragma unroll
  for (int g = 0; g < JG; ++g)
#pragma unroll
    for (int s = 0; s < 4; ++s) acc[g][s] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // A operands of slab ks (rows 16 g + l16 of the hi and lo planes, m0 + 8 lg .. + 7; Mp is a multiple of 32).
  // Up to padded rank 32 they are requested a slab ahead, so that their latency overlaps the previous slab's
  // MFMAs; at higher ranks the second set of registers would cost occupancy, and they are requested in the slab.
  constexpr bool PF = JG <= 2;
  uint4 ap[JG][2], an[PF ? JG : 1][2];
  auto load_p = [&](int ks, uint4 (&d)[JG][2]) __attribute__((always_inline)) {
    const int m0 = m_begin + ks * O_KS;
#pragma unroll
    for (int g = 0; g < JG; ++g) {
      const uint16_t* p = a.PT + (size_t)(g * 16 + l16) * a.Mp + m0 + 8 * lg;
      d[g][0] = *reinterpret_cast<const uint4*>(p);
      d[g][1] = *reinterpret_cast<const uint4*>(p + (size_t)a.RP * a.Mp);
    }
  };
  if constexpr (PF) load_p(0, ap);
  load(0);
  store(0);
  if (nks > 1) load(1);
  __syncthreads();
  for (int ks = 0; ks < nks; ++ks) {
    const int st = ks & 1;
    if constexpr (PF) {
      if (ks + 1 < nks) load_p(ks + 1, an);
    } else {
      load_p(ks, ap);
    }
    // B operands: column wave * 64 + 16 s + l16, rows 8 lg .. 8 lg + 7 of the slab
    uint4 bq[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint16_t* q = &qs[st][8 * lg][wave * 64 + s * 16 + l16];
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (uint32_t)q[(2 * i) * O_LD] | ((uint32_t)q[(2 * i + 1) * O_LD] << 16);
      bq[s] = uint4{w[0], w[1], w[2], w[3]};
    }
#pragma unroll
    for (int g = 0; g < JG; ++g)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        acc[g][s] = mfma16(ap[g][0], bq[s], acc[g][s]);
        acc[g][s] = mfma16(ap[g][1], bq[s], acc[g][s]);
      }
    if (ks + 1 < nks) {
      store(st ^ 1);  // stage st ^ 1 was last read before the previous barrier
      if (ks + 2 < nks) load(ks + 2);
      if constexpr (PF) {
#pragma unroll
        for (int g = 0; g < JG; ++g) {
          ap[g][0] = an[g][0];
          ap[g][1] = an[g][1];
        }
      }
    }
    __syncthreads();
  }

  // acc[g][s] lane l holds out[16 g + 4 lg + e][c0 + 64 wave + 16 s + l16]; partials laid out like the output
  const size_t zc = (size_t)ch * a.RP * a.C;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int c = c0 + wave * 64 + s * 16 + l16;
    if (c >= a.C) continue;
#pragma unroll
    for (int g = 0; g < JG; ++g) {
      const int j = g * 16 + 4 * lg;
      if (a.jc) {
#pragma unroll
        for (int e = 0; e < 4; ++e) a.part[zc + (size_t)(j + e) * a.C + c] = acc[g][s][e];
      } else {
        *reinterpret_cast<f32x4_t*>(a.part + zc + (size_t)c * a.RP + j) = acc[g][s];
      }
    }
  }
}

// dA's and dB's partials in one launch: workgroups [0, n0) for o0, the rest o1.
template <int RP>
__global__ __launch_bounds__(O_WAVES * 64) void lora_outer_part_kernel(OuterArgs o0, int n0, OuterArgs o1) {
  const int b = blockIdx.x;
  if (b < n0)
    outer_part<RP>(o0, b);
  else
    outer_part<RP>(o1, b - n0);
}

constexpr int F_UNROLL = 8;

// out[e] = sum over chunks, in chunk order, of the partials of output element
// e; the loads of F_UNROLL chunks in flight before they are added.
__device__ __forceinline__ void outer_finish(const OuterArgs& a, size_t e) {
  if (e >= (size_t)a.r * a.C) return;
  const size_t src = a.jc ? e : e / a.r * a.RP + e % a.r;  // partial layout [RP x C] or [C x RP]
  const size_t stride = (size_t)a.RP * a.C;
  float v = 0.f;
  int ch = 0;
  for (; ch + F_UNROLL <= a.nch; ch += F_UNROLL) {
    float t[F_UNROLL];
#pragma unroll
    for (int u = 0; u < F_UNROLL; ++u) t[u] = a.part[src + (size_t)(ch + u) * stride];
#pragma unroll
    for (int u = 0; u < F_UNROLL; ++u) v += t[u];
  }
  for (; ch < a.nch; ++ch) v += a.part[src + (size_t)ch * stride];
  a.out[e] = v;
}

// One thread per output element; workgroups [0, n0) for o0, the rest o1.
__global__ __launch_bounds__(256) void lora_outer_finish_kernel(OuterArgs o0, int n0, OuterArgs o1) {
  const int b = blockIdx.x;
  if (b < n0)
    outer_finish(o0, (size_t)b * 256 + threadIdx.x);
  else
    outer_finish(o1, (size_t)(b - n0) * 256 + threadIdx.x);
}

// Rows per chunk and number of chunks of the outer products over M rows and
// C columns: enough chunks for about O_TARGET_WG workgroups, each chunk a
// multiple of O_KS rows and at least O_MIN_ROWS.
void outer_chunks(int M, int C, int& mch, int& nch) {
  const int64_t tiles = (C + O_COLS - 1) / O_COLS;
  const int64_t want = std::max<int64_t>(1, (O_TARGET_WG + tiles - 1) / tiles);
  int64_t rows = (M + want - 1) / want;
  rows = std::max<int64_t>(O_MIN_ROWS, (rows + O_KS - 1) / O_KS * O_KS);
  mch = (int)rows;
  nch = (int)((M + rows - 1) / rows);
}

int padded_rows(int M) { return (M + O_KS - 1) / O_KS * O_KS; }

OuterArgs outer_job(const uint16_t* PT, const uint16_t* Q, int M, int C, int rp, int r, float* part, float* out,
                    bool jc, int& parts, int& finishes) {
  OuterArgs o{PT, Q, part, out, M, padded_rows(M), C, rp, r, 0, 0, jc ? 1 : 0, (C + O_COLS - 1) / O_COLS};
  outer_chunks(M, C, o.mch, o.nch);
  parts = o.tiles * o.nch;
  finishes = (int)(((size_t)r * C + 255) / 256);
  return o;
}

template <int RP>
void launch_outer_rp(const OuterArgs& o0, int p0, const OuterArgs& o1, int p1, hipStream_t stream) {
  hipLaunchKernelGGL((lora_outer_part_kernel<RP>), dim3(p0 + p1), dim3(O_WAVES * 64), 0, stream, o0, p0, o1);
}

hipError_t launch_outer(const OuterArgs& o0, int p0, int f0, const OuterArgs& o1, int p1, int f1, int rp,
                        hipStream_t stream) {
  switch (rp) {
    case 16: launch_outer_rp<16>(o0, p0, o1, p1, stream); break;
    case 32: launch_outer_rp<32>(o0, p0, o1, p1, stream); break;
    case 64: launch_outer_rp<64>(o0, p0, o1, p1, stream); break;
    case 128: launch_outer_rp<128>(o0, p0, o1, p1, stream); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lora_outer_finish_kernel, dim3(f0 + f1), dim3(256), 0, stream, o0, f0, o1);
  return hipGetLastError();
}

// ------------------------------------------------------- workspace layout
size_t up256(size_t v) { return (v + 255) / 256 * 256; }

struct BwdLayout {
  size_t bt, at, tsu, uT, tT, tpart, tpart2, opa, opb, total;
};

BwdLayout layout(int M, int N, int K, int rp) {
  BwdLayout l{};
  size_t o = 0;
  l.bt = o;    o += up256((size_t)rp * N * 2);                      // B^T [RP x N] bf16
  l.at = o;    o += up256((size_t)K * rp * 2);                      // A^T [K x RP] bf16
  l.tsu = o;   o += up256((size_t)M * 2 * rp * 2);                  // hi | lo of s U [M x 2 RP] bf16
  const size_t Mp = (size_t)padded_rows(M);
  l.uT = o;    o += up256(2 * (size_t)rp * Mp * 2);                 // hi | lo planes of (s U)^T [2][RP][Mp] bf16
  l.tT = o;    o += up256(2 * (size_t)rp * Mp * 2);                 // hi | lo planes of (s T)^T [2][RP][Mp] bf16
  l.tpart = o; o += up256((size_t)kTpreMaxChunks * M * rp * 4);     // pre-pass partials (s U)
  l.tpart2 = o; o += up256((size_t)kTpreMaxChunks * M * rp * 4);    // pre-pass partials (s T)
  int mch, nch_a, nch_b;
  outer_chunks(M, K, mch, nch_a);
  outer_chunks(M, N, mch, nch_b);
  const size_t oa = (size_t)nch_a * rp * K, ob = (size_t)nch_b * rp * N;
  l.opa = o;   o += up256(oa * 4);                                  // dA's outer-product partials
  l.opb = o;   o += up256(ob * 4);                                  // dB's outer-product partials
  l.total = o;
  return l;
}

}  // namespace

hipError_t launch_transpose_pad(const uint16_t* src, int R, int C, uint16_t* dst, int Rp, int Cp,
                                hipStream_t stream) {
  int n;
  const TransposeJob j = transpose_job(src, R, C, dst, Rp, Cp, n);
  hipLaunchKernelGGL(transpose_pad_kernel, dim3(n), dim3(256), 0, stream, j, n, j);
  return hipGetLastError();
}

size_t backward_ws_bytes(int M, int N, int K, int rp) { return rp == 0 ? 0 : layout(M, N, K, rp).total; }

hipError_t launch_lora_backward(const BackwardArgs& a, void* ws, hipStream_t stream) {
  const int rp = padded_rank(a.r);
  hipError_t e;
  if (rp == 0) {  // no adapter: dx = dy W only
    if (!a.dx) return hipSuccess;
    LinearArgs g{};
    g.x = a.dy;
    g.W = a.Wt;
    g.M = a.M;
    g.N = a.K;
    g.K = a.N;
    g.y_off = a.dx;
    return launch_lora_gemm(g, stream);
  }
  const BwdLayout l = layout(a.M, a.N, a.K, rp);
  uint8_t* w = static_cast<uint8_t*>(ws);
  uint16_t* bt = reinterpret_cast<uint16_t*>(w + l.bt);
  uint16_t* at = reinterpret_cast<uint16_t*>(w + l.at);
  const bool want_u = a.dx || a.dA;  // s U = s dy B
  const bool want_t = a.dB != nullptr;  // s T = s x A^T

  // 1. B^T [RP x N] (for s U) and A^T [K x RP] (the dx GEMM's LoRA rows), one launch
  {
    int n0 = 0, n1 = 0;
    TransposeJob j0{}, j1{};
    if (want_u) j0 = transpose_job(a.B, a.N, a.r, bt, a.N, rp, n0);
    if (a.dx) j1 = transpose_job(a.A, a.r, a.K, at, rp, a.K, n1);
    if (n0 + n1 > 0) {
      hipLaunchKernelGGL(transpose_pad_kernel, dim3(n0 + n1), dim3(256), 0, stream, j0, n0, j1);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  // 2. the pre-passes: s U from dy against the rows of B^T (hi | lo for dx, fp32 for dA), s T from x (fp32)
  TpreArgs u{}, tt{};
  u.x = a.dy;
  u.A = bt;
  u.s = a.s;
  u.M = a.M;
  u.K = a.N;
  u.r = a.r;
  u.ts = a.dx ? reinterpret_cast<uint16_t*>(w + l.tsu) : nullptr;
  u.part = reinterpret_cast<float*>(w + l.tpart);
  u.tT = a.dA ? reinterpret_cast<uint16_t*>(w + l.uT) : nullptr;
  u.Mp = padded_rows(a.M);
  tt.x = a.x;
  tt.A = a.A;
  tt.s = a.s;
  tt.M = a.M;
  tt.K = a.K;
  tt.r = a.r;
  tt.part = reinterpret_cast<float*>(w + l.tpart2);
  tt.tT = reinterpret_cast<uint16_t*>(w + l.tT);
  tt.Mp = padded_rows(a.M);
  if (want_u && want_t)
    e = launch_lora_tpre2(u, tt, rp, stream);
  else
    e = launch_lora_tpre(want_u ? u : tt, rp, nullptr, stream);
  if (e != hipSuccess) return e;
  // 3. dx = dy W + s U A: the GEMM over W^T with slabs ([hi | lo](s U), A^T)
  if (a.dx) {
    LinearArgs g{};
    g.x = a.dy;
    g.W = a.Wt;
    g.s = a.s;
    g.M = a.M;
    g.N = a.K;
    g.K = a.N;
    g.r = a.r;
    g.y_on = a.dx;
    if ((e = launch_lora_gemm_slabs(g, u.ts, at, rp, stream)) != hipSuccess) return e;
  }
  // 4. dA[j][k] = sum_m sU[m][j] x[m][k] and dB[n][j] = sum_m dy[m][n] sT[m][j]: partials, then the finish
  int p0 = 0, f0 = 0, p1 = 0, f1 = 0;
  OuterArgs o0{}, o1{};
  if (a.dA)
    o0 = outer_job(u.tT, a.x, a.M, a.K, rp, a.r, reinterpret_cast<float*>(w + l.opa), a.dA, true, p0, f0);
  if (a.dB)
    o1 = outer_job(tt.tT, a.dy, a.M, a.N, rp, a.r, reinterpret_cast<float*>(w + l.opb), a.dB, false, p1, f1);
  if (p0 + p1 > 0)
    if ((e = launch_outer(o0, p0, f0, o1, p1, f1, rp, stream)) != hipSuccess) return e;
  return hipSuccess;
}

}  // namespace hydra
