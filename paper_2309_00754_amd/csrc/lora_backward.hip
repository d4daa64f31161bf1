// Backward of the LoRA-switchable linear with the base weight frozen (the
// update stage of Hydra-PPO trains only the active adapter, Sec. 3 and
// App. A, Alg. 2).  With y = x W^T + s (x A^T) B^T, T = x A^T and U = dy B:
//   dx = dy W + s U A,   dA = s U^T x,   dB = s dy^T T.
// Steps, all on one stream:
//  1. B^T and A^T, zero padded to the padded rank RP (transpose_pad_kernel);
//  2. the LoRA pre-pass of the forward GEMM (lora_tpre.hip) twice: s U from
//     dy against the rows of B^T (hi | lo bf16 parts for step 3, fp32 for
//     step 4), s T from x against A (fp32);
//  3. dx by the forward's MFMA GEMM run on (dy, W^T), its LoRA slabs being
//     [hi | lo](s U) against rows of A^T: one pass over W^T, as in the forward;
//  4. dA and dB as sums of outer products over the rows m:
//     out[j][c] = sum_m P[m][j] Q[m][c] with (P, Q) = (s U, x) and (s T, dy),
//     vector fp32 FMAs (lora_outer_part_kernel: per row chunk partials), then
//     the chunks added in chunk order and written in the output's layout
//     (lora_outer_finish_kernel).  Every sum has a fixed order: the results
//     are the same from run to run.
#include <algorithm>

#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

// ------------------------------------------------------------ transpose_pad
constexpr int TP = 64;  // tile edge

// dst [Cp x Rp]: dst[c][q] = src[q][c] inside src's [R x C], zero outside.
__global__ __launch_bounds__(256) void transpose_pad_kernel(const uint16_t* __restrict__ src, int R, int C,
                                                            uint16_t* __restrict__ dst, int Rp, int Cp) {
  __shared__ uint16_t tile[TP][TP + 2];
  const int c0 = blockIdx.x * TP, q0 = blockIdx.y * TP;
  const int lx = threadIdx.x & 63, ly = threadIdx.x >> 6;
#pragma unroll 4
  for (int i = ly; i < TP; i += 4) {
    const int q = q0 + i, c = c0 + lx;
    tile[i][lx] = (q < R && c < C) ? src[(size_t)q * C + c] : (uint16_t)0;
  }
  __syncthreads();
#pragma unroll 4
  for (int i = ly; i < TP; i += 4) {
    const int c = c0 + i, q = q0 + lx;
    if (c < Cp && q < Rp) dst[(size_t)c * Rp + q] = tile[lx][i];
  }
}

// ---------------------------------------------------------- outer products
constexpr int O_WAVES = 4;
constexpr int O_JT = 16;          // j values per workgroup
constexpr int O_COLS = 256;       // columns per workgroup, 4 per lane
constexpr int O_UNROLL = 4;       // rows per wave with loads in flight together
constexpr int O_WIN = 256;        // rows of P staged in LDS at a time
constexpr int O_TARGET_WG = 1024;  // workgroups the chunking aims for

struct OuterArgs {
  const float* P;      // [M x RP] fp32
  const uint16_t* Q;   // [M x C] bf16
  float* part;         // [nch x RP x C] fp32
  int M, C, RP, mch;   // mch: rows per chunk (multiple of 16)
};

__device__ __forceinline__ uint2 buf_load8(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, 0));
}

// Partial out[j][c] over the rows of chunk blockIdx.z for j in the 16-wide
// group blockIdx.y and 256 columns of tile blockIdx.x.  The 4 waves take the
// rows in turn (row i of a window goes to wave i % 4), each lane 4 columns x
// 16 j in registers; the wave sums are added in wave order at the end.
__global__ __launch_bounds__(O_WAVES * 64) void lora_outer_part_kernel(OuterArgs a) {
  __shared__ float ps[O_WIN][O_JT];
  __shared__ f32x4_t red[O_WAVES - 1][O_JT / 2][64];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int jg = blockIdx.y;
  const int c = blockIdx.x * O_COLS + lane * 4;
  const int m_begin = blockIdx.z * a.mch;
  const int m_end = min(a.M, m_begin + a.mch);
  float acc[O_JT][4];
#pragma unroll
  for (int j = 0; j < O_JT; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[j][e] = 0.f;

  for (int w0 = m_begin; w0 < m_end; w0 += O_WIN) {
    const int rows = min(O_WIN, m_end - w0);
    __syncthreads();  // the previous window's P is no longer read
    for (int e = t; e < rows * O_JT; e += O_WAVES * 64) {
      const int rl = e / O_JT, jj = e % O_JT;
      ps[rl][jj] = a.P[(size_t)(w0 + rl) * a.RP + jg * O_JT + jj];
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t qrs = make_rsrc(a.Q + (size_t)w0 * a.C, (uint32_t)rows * a.C * 2u);
    for (int r0 = wave; r0 < rows; r0 += O_WAVES * O_UNROLL) {
      uint2 q[O_UNROLL];
#pragma unroll
      for (int u = 0; u < O_UNROLL; ++u) {
        const int rl = r0 + u * O_WAVES;
        q[u] = buf_load8(qrs, (rl < rows && c < a.C) ? (rl * a.C + c) * 2 : kOutOfRange);
      }
#pragma unroll
      for (int u = 0; u < O_UNROLL; ++u) {
        const int rl = r0 + u * O_WAVES;  // wave-uniform
        if (rl >= rows) break;
        const float qf[4] = {bf16_to_f32(q[u].x & 0xFFFFu), bf16_to_f32(q[u].x >> 16),
                             bf16_to_f32(q[u].y & 0xFFFFu), bf16_to_f32(q[u].y >> 16)};
        const f32x4_t* pr = reinterpret_cast<const f32x4_t*>(&ps[rl][0]);
#pragma unroll
        for (int j4 = 0; j4 < O_JT / 4; ++j4) {
          const f32x4_t p = pr[j4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[j4 * 4 + 0][e] += p[0] * qf[e];
            acc[j4 * 4 + 1][e] += p[1] * qf[e];
            acc[j4 * 4 + 2][e] += p[2] * qf[e];
            acc[j4 * 4 + 3][e] += p[3] * qf[e];
          }
        }
      }
    }
  }

  // wave sums added in wave order, half of the j values at a time
  float* out = a.part + ((size_t)blockIdx.z * a.RP + jg * O_JT) * a.C + c;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    __syncthreads();
    if (wave > 0) {
#pragma unroll
      for (int j = 0; j < O_JT / 2; ++j)
        red[wave - 1][j][lane] = f32x4_t{acc[h * 8 + j][0], acc[h * 8 + j][1], acc[h * 8 + j][2], acc[h * 8 + j][3]};
    }
    __syncthreads();
    if (wave == 0 && c < a.C) {
#pragma unroll
      for (int j = 0; j < O_JT / 2; ++j) {
        f32x4_t v{acc[h * 8 + j][0], acc[h * 8 + j][1], acc[h * 8 + j][2], acc[h * 8 + j][3]};
#pragma unroll
        for (int w = 0; w < O_WAVES - 1; ++w) v += red[w][j][lane];
        *reinterpret_cast<f32x4_t*>(out + (size_t)(h * 8 + j) * a.C) = v;
      }
    }
  }
}

constexpr int F_COLS = 64;

// out = sum over chunks (in chunk order) of the partials, for j < r: layout
// [r x C] (jc != 0) or [C x r]; one workgroup per 64 columns and 16 j values,
// staged through LDS for the [C x r] layout so that both layouts are written
// row by row.
__global__ __launch_bounds__(256) void lora_outer_finish_kernel(const float* __restrict__ part, int nch, int RP,
                                                                int C, int r, float* __restrict__ out, int jc) {
  __shared__ float tile[O_JT][F_COLS + 1];
  const int c0 = blockIdx.x * F_COLS, j0 = blockIdx.y * O_JT;
  const int t = threadIdx.x;
  const int cc = t & 63;
  const int c = c0 + cc;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  for (int ch = 0; ch < nch; ++ch) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = j0 + (t >> 6) + 4 * i;
      if (c < C && j < r) v[i] += part[((size_t)ch * RP + j) * C + c];
    }
  }
  if (jc) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = j0 + (t >> 6) + 4 * i;
      if (c < C && j < r) out[(size_t)j * C + c] = v[i];
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) tile[(t >> 6) + 4 * i][cc] = v[i];
  __syncthreads();
  const int nj = min(O_JT, r - j0);
  const int ncol = min(F_COLS, C - c0);
  for (int e = t; e < ncol * nj; e += 256) {
    const int ci = e / nj, jj = e % nj;
    out[(size_t)(c0 + ci) * r + j0 + jj] = tile[jj][ci];
  }
}

// Rows per chunk and number of chunks of the outer products over M rows and
// C columns at padded rank RP: enough chunks for about O_TARGET_WG
// workgroups, each chunk a multiple of 16 rows.
void outer_chunks(int M, int C, int rp, int& mch, int& nch) {
  const int64_t tiles = (int64_t)((C + O_COLS - 1) / O_COLS) * (rp / O_JT);
  const int64_t want = std::max<int64_t>(1, (O_TARGET_WG + tiles - 1) / tiles);
  int64_t rows = (M + want - 1) / want;
  rows = std::max<int64_t>(16, (rows + 15) / 16 * 16);
  mch = (int)rows;
  nch = (int)((M + rows - 1) / rows);
}

hipError_t launch_outer(const float* P, const uint16_t* Q, int M, int C, int rp, int r, float* part, float* out,
                        bool jc, hipStream_t stream) {
  OuterArgs o{P, Q, part, M, C, rp, 0};
  int nch;
  outer_chunks(M, C, rp, o.mch, nch);
  hipLaunchKernelGGL(lora_outer_part_kernel, dim3((C + O_COLS - 1) / O_COLS, rp / O_JT, nch), dim3(O_WAVES * 64), 0,
                     stream, o);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lora_outer_finish_kernel, dim3((C + F_COLS - 1) / F_COLS, (r + O_JT - 1) / O_JT), dim3(256), 0,
                     stream, (const float*)part, nch, rp, C, r, out, jc ? 1 : 0);
  return hipGetLastError();
}

// ------------------------------------------------------- workspace layout
size_t up256(size_t v) { return (v + 255) / 256 * 256; }

struct BwdLayout {
  size_t bt, at, tsu, u32, t32, tpart, opart, total;
};

BwdLayout layout(int M, int N, int K, int rp) {
  BwdLayout l{};
  size_t o = 0;
  l.bt = o;    o += up256((size_t)rp * N * 2);                      // B^T [RP x N] bf16
  l.at = o;    o += up256((size_t)K * rp * 2);                      // A^T [K x RP] bf16
  l.tsu = o;   o += up256((size_t)M * 2 * rp * 2);                  // hi | lo of s U [M x 2 RP] bf16
  l.u32 = o;   o += up256((size_t)M * rp * 4);                      // s U [M x RP] fp32
  l.t32 = o;   o += up256((size_t)M * rp * 4);                      // s T [M x RP] fp32
  l.tpart = o; o += up256((size_t)kTpreMaxChunks * M * rp * 4);     // pre-pass partials
  int mch, nch_a, nch_b;
  outer_chunks(M, K, rp, mch, nch_a);
  outer_chunks(M, N, rp, mch, nch_b);
  const size_t oa = (size_t)nch_a * rp * K, ob = (size_t)nch_b * rp * N;
  l.opart = o; o += up256((oa > ob ? oa : ob) * 4);                 // outer-product partials
  l.total = o;
  return l;
}

}  // namespace

hipError_t launch_transpose_pad(const uint16_t* src, int R, int C, uint16_t* dst, int Rp, int Cp,
                                hipStream_t stream) {
  hipLaunchKernelGGL(transpose_pad_kernel, dim3((Cp + TP - 1) / TP, (Rp + TP - 1) / TP), dim3(256), 0, stream, src,
                     R, C, dst, Rp, Cp);
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
  uint16_t* tsu = reinterpret_cast<uint16_t*>(w + l.tsu);
  float* u32 = reinterpret_cast<float*>(w + l.u32);
  float* t32 = reinterpret_cast<float*>(w + l.t32);
  float* tpart = reinterpret_cast<float*>(w + l.tpart);
  float* opart = reinterpret_cast<float*>(w + l.opart);

  if (a.dx || a.dA) {  // s U = s dy B, from dy against the rows of B^T
    if ((e = launch_transpose_pad(a.B, a.N, a.r, bt, a.N, rp, stream)) != hipSuccess) return e;
    TpreArgs u{};
    u.x = a.dy;
    u.A = bt;
    u.s = a.s;
    u.M = a.M;
    u.N = 0;
    u.K = a.N;
    u.r = a.r;
    u.ts = a.dx ? tsu : nullptr;
    u.part = tpart;
    u.t32 = a.dA ? u32 : nullptr;
    if ((e = launch_lora_tpre(u, rp, nullptr, stream)) != hipSuccess) return e;
  }
  if (a.dx) {  // dx = dy W + s U A: the GEMM over W^T with slabs (s U, A^T)
    if ((e = launch_transpose_pad(a.A, a.r, a.K, at, rp, a.K, stream)) != hipSuccess) return e;
    LinearArgs g{};
    g.x = a.dy;
    g.W = a.Wt;
    g.s = a.s;
    g.M = a.M;
    g.N = a.K;
    g.K = a.N;
    g.r = a.r;
    g.y_on = a.dx;
    if ((e = launch_lora_gemm_slabs(g, tsu, at, rp, stream)) != hipSuccess) return e;
  }
  if (a.dA)  // dA[j][k] = sum_m sU[m][j] x[m][k]
    if ((e = launch_outer(u32, a.x, a.M, a.K, rp, a.r, opart, a.dA, true, stream)) != hipSuccess) return e;
  if (a.dB) {  // dB[n][j] = sum_m dy[m][n] sT[m][j]
    TpreArgs tt{};
    tt.x = a.x;
    tt.A = a.A;
    tt.s = a.s;
    tt.M = a.M;
    tt.N = 0;
    tt.K = a.K;
    tt.r = a.r;
    tt.part = tpart;
    tt.t32 = t32;
    if ((e = launch_lora_tpre(tt, rp, nullptr, stream)) != hipSuccess) return e;
    if ((e = launch_outer(t32, a.dy, a.M, a.N, rp, a.r, opart, a.dB, false, stream)) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace hydra
