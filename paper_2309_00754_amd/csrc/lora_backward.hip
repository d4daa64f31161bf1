// Backward of the LoRA-switchable linear with the base weight frozen (the
// update stage of Hydra-PPO trains only the active adapter, Sec. 3 and
// App. A, Alg. 2).  With y = x W^T + s (x A^T) B^T, T = x A^T and U = dy B:
//   dx = dy W + s U A,   dA = s U^T x,   dB = s dy^T T.
// Steps, all on one stream:
//  1. B^T and A^T, zero padded to the padded rank RP (transpose_pad_kernel,
//     both in one launch);
//  2. the LoRA pre-pass of the forward GEMM (lora_tpre.hip) twice, in one
//     pair of launches: s U from dy against the rows of B^T (hi | lo bf16
//     parts for step 3, fp32 for step 4), s T from x against A (fp32);
//  3. dx by the forward's MFMA GEMM run on (dy, W^T), its LoRA slabs being
//     [hi | lo](s U) against rows of A^T: one pass over W^T, as in the forward;
//  4. dA and dB as sums of outer products over the rows m:
//     out[j][c] = sum_m P[m][j] Q[m][c] with (P, Q) = (s U, x) and (s T, dy),
//     vector fp32 FMAs (lora_outer_part_kernel: per row chunk partials, laid
//     out like the output), then the chunks added in chunk order
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
constexpr int O_JT = 16;          // j values per workgroup
constexpr int O_COLS = 256;       // columns per workgroup, 4 per lane
constexpr int O_UNROLL = 16;      // rows per wave with loads in flight together
constexpr int O_WIN = 256;        // rows of P staged in LDS at a time
constexpr int O_TARGET_WG = 512;  // workgroups the chunking aims for
constexpr int O_MIN_ROWS = 64;    // fewest rows per chunk

struct OuterArgs {
  const float* P;      // [M x RP] fp32
  const uint16_t* Q;   // [M x C] bf16
  float* part;         // [nch x RP x C] (jc) or [nch x C x RP] fp32
  float* out;          // [r x C] (jc) or [C x r] fp32
  int M, C, RP, r;
  int mch, nch;        // rows per chunk (multiple of 16), chunks
  int jc;              // partials and output j-major
  int tiles;           // column tiles of O_COLS
};

__device__ __forceinline__ uint2 buf_load8(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, 0));
}

// Partial out[j][c] over the rows of one chunk, for one 16-wide group of j and
// the 256 columns of one tile (b = tile + tiles * (jg + RP / 16 * chunk)).  The
// 4 waves take the rows in turn (row i of a window goes to wave i % 4), each
// lane 4 columns x 16 j in registers; the wave sums are added in wave order
// at the end.
__device__ __forceinline__ void outer_part(const OuterArgs& a, int b) {
  __shared__ float ps[O_WIN][O_JT];
  __shared__ f32x4_t red[O_WAVES - 1][O_JT / 2][64];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int tile = b % a.tiles;
  const int rest = b / a.tiles;
  const int jg = rest % (a.RP / O_JT);
  const int ch = rest / (a.RP / O_JT);
  const int c = tile * O_COLS + lane * 4;
  const int m_begin = ch * a.mch;
  const int m_end = min(a.M, m_begin + a.mch);
  float acc[O_JT][4];
#pragma unroll
  for (int j = 0; j < O_JT; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[j][e] = 0.f;

  for (int w0 = m_begin; w0 < m_end; w0 += O_WIN) {
    const int rows = min(O_WIN, m_end - w0);
    const __amdgpu_buffer_rsrc_t qrs = make_rsrc(a.Q + (size_t)w0 * a.C, (uint32_t)rows * a.C * 2u);
    uint2 q[O_UNROLL];
    auto load = [&](int r0) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < O_UNROLL; ++u) {
        const int rl = r0 + u * O_WAVES;
        q[u] = buf_load8(qrs, (rl < rows && c < a.C) ? (rl * a.C + c) * 2 : kOutOfRange);
      }
    };
    load(wave);  // the window's first rows of Q in flight while P is staged
    __syncthreads();  // the previous window's P is no longer read
    for (int e = t; e < rows * O_JT; e += O_WAVES * 64) {
      const int rl = e / O_JT, jj = e % O_JT;
      ps[rl][jj] = a.P[(size_t)(w0 + rl) * a.RP + jg * O_JT + jj];
    }
    __syncthreads();
    for (int r0 = wave; r0 < rows; r0 += O_WAVES * O_UNROLL) {
      if (r0 != wave) load(r0);
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

  // wave sums added in wave order, half of the j values at a time; the
  // partials are laid out like the output (j-major or column-major), so that
  // the finish reads them in the order it writes
  const size_t zc = (size_t)ch * a.RP * a.C;
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
      f32x4_t v[O_JT / 2];
#pragma unroll
      for (int j = 0; j < O_JT / 2; ++j) {
        v[j] = f32x4_t{acc[h * 8 + j][0], acc[h * 8 + j][1], acc[h * 8 + j][2], acc[h * 8 + j][3]};
#pragma unroll
        for (int w = 0; w < O_WAVES - 1; ++w) v[j] += red[w][j][lane];
      }
      const int j0 = jg * O_JT + h * 8;
      if (a.jc) {
#pragma unroll
        for (int j = 0; j < O_JT / 2; ++j)
          *reinterpret_cast<f32x4_t*>(a.part + zc + (size_t)(j0 + j) * a.C + c) = v[j];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float* o = a.part + zc + (size_t)(c + e) * a.RP + j0;
          *reinterpret_cast<f32x4_t*>(o) = f32x4_t{v[0][e], v[1][e], v[2][e], v[3][e]};
          *reinterpret_cast<f32x4_t*>(o + 4) = f32x4_t{v[4][e], v[5][e], v[6][e], v[7][e]};
        }
      }
    }
  }
}

// dA's and dB's partials in one launch: workgroups [0, n0) for o0, the rest o1.
__global__ __launch_bounds__(O_WAVES * 64) void lora_outer_part_kernel(OuterArgs o0, int n0, OuterArgs o1) {
  const int b = blockIdx.x;
  if (b < n0)
    outer_part(o0, b);
  else
    outer_part(o1, b - n0);
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
// C columns at padded rank RP: enough chunks for about O_TARGET_WG
// workgroups, each chunk a multiple of 16 rows and at least O_MIN_ROWS.
void outer_chunks(int M, int C, int rp, int& mch, int& nch) {
  const int64_t tiles = (int64_t)((C + O_COLS - 1) / O_COLS) * (rp / O_JT);
  const int64_t want = std::max<int64_t>(1, (O_TARGET_WG + tiles - 1) / tiles);
  int64_t rows = (M + want - 1) / want;
  rows = std::max<int64_t>(O_MIN_ROWS, (rows + 15) / 16 * 16);
  mch = (int)rows;
  nch = (int)((M + rows - 1) / rows);
}

OuterArgs outer_job(const float* P, const uint16_t* Q, int M, int C, int rp, int r, float* part, float* out, bool jc,
                    int& parts, int& finishes) {
  OuterArgs o{P, Q, part, out, M, C, rp, r, 0, 0, jc ? 1 : 0, (C + O_COLS - 1) / O_COLS};
  outer_chunks(M, C, rp, o.mch, o.nch);
  parts = o.tiles * (rp / O_JT) * o.nch;
  finishes = (int)(((size_t)r * C + 255) / 256);
  return o;
}

// ------------------------------------------------------- workspace layout
size_t up256(size_t v) { return (v + 255) / 256 * 256; }

struct BwdLayout {
  size_t bt, at, tsu, u32, t32, tpart, tpart2, opa, opb, total;
};

BwdLayout layout(int M, int N, int K, int rp) {
  BwdLayout l{};
  size_t o = 0;
  l.bt = o;    o += up256((size_t)rp * N * 2);                      // B^T [RP x N] bf16
  l.at = o;    o += up256((size_t)K * rp * 2);                      // A^T [K x RP] bf16
  l.tsu = o;   o += up256((size_t)M * 2 * rp * 2);                  // hi | lo of s U [M x 2 RP] bf16
  l.u32 = o;   o += up256((size_t)M * rp * 4);                      // s U [M x RP] fp32
  l.t32 = o;   o += up256((size_t)M * rp * 4);                      // s T [M x RP] fp32
  l.tpart = o; o += up256((size_t)kTpreMaxChunks * M * rp * 4);     // pre-pass partials (s U)
  l.tpart2 = o; o += up256((size_t)kTpreMaxChunks * M * rp * 4);    // pre-pass partials (s T)
  int mch, nch_a, nch_b;
  outer_chunks(M, K, rp, mch, nch_a);
  outer_chunks(M, N, rp, mch, nch_b);
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
  u.t32 = a.dA ? reinterpret_cast<float*>(w + l.u32) : nullptr;
  tt.x = a.x;
  tt.A = a.A;
  tt.s = a.s;
  tt.M = a.M;
  tt.K = a.K;
  tt.r = a.r;
  tt.part = reinterpret_cast<float*>(w + l.tpart2);
  tt.t32 = reinterpret_cast<float*>(w + l.t32);
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
    o0 = outer_job(u.t32, a.x, a.M, a.K, rp, a.r, reinterpret_cast<float*>(w + l.opa), a.dA, true, p0, f0);
  if (a.dB)
    o1 = outer_job(tt.t32, a.dy, a.M, a.N, rp, a.r, reinterpret_cast<float*>(w + l.opb), a.dB, false, p1, f1);
  if (p0 + p1 > 0) {
    hipLaunchKernelGGL(lora_outer_part_kernel, dim3(p0 + p1), dim3(O_WAVES * 64), 0, stream, o0, p0, o1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(lora_outer_finish_kernel, dim3(f0 + f1), dim3(256), 0, stream, o0, f0, o1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace hydra
