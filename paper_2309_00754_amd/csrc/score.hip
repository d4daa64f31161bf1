// Scoring kernels for gfx950: sampled-token log-probabilities under the
// LoRA-on (actor) and LoRA-off (reference) passes, their difference as the
// per-token KL estimate, and the scalar reward head (Sec. 3, the two heads of
// pi^hydra; App. A, Alg. 1 / Alg. 2, the step that scores the generated
// sequences with LoRA off for the reward and the reference log-probabilities;
// the KL weight beta of App. B is applied by the caller).
//
//  * score_logits_vec_kernel (V % 4 == 0) / score_logits_kernel (other V):
//    one workgroup per token row streams both fp32 logit rows once, keeping
//    a per-thread running (max, sum exp) and reducing it across the
//    workgroup in a fixed tree.
//  * score_combine_kernel: one wave per token row merges the per-column-tile
//    partials written by the fused CLM-head GEMM (row maximum, then the sum
//    of the partial sums rescaled to it, each by a fixed butterfly), then
//    forms lse, lp and KL; extra workgroups compute the reward head's dot
//    products.
// The LoRA-on and LoRA-off statistics always go through the same code, so
// equal logit rows give bit-identical results and KL == 0 exactly.
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

__device__ __forceinline__ void wave_merge(float& m, float& s) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float mo = __shfl_xor(m, off);
    const float so = __shfl_xor(s, off);
    lse_merge(m, s, mo, so);
  }
}

__device__ __forceinline__ void finish_row(int row, int tk, int V, float z_on, float z_off, float m_on, float s_on,
                                           float m_off, float s_off, const LogitsArgs& o) {
  const float lse_on = m_on + log_e(s_on);
  const float lse_off = m_off + log_e(s_off);
  const bool ok = tk >= 0 && tk < V;
  const float lp_on = ok ? z_on - lse_on : __builtin_nanf("");
  const float lp_off = ok ? z_off - lse_off : __builtin_nanf("");
  o.lp_on[row] = lp_on;
  o.lp_off[row] = lp_off;
  o.kl[row] = lp_on - lp_off;
  if (o.lse_on) o.lse_on[row] = lse_on;
  if (o.lse_off) o.lse_off[row] = lse_off;
  if (!ok && o.err) atomicOr(o.err, 1);
}

// Running (max, sum exp) update with a batch of values whose maximum is bm.
__device__ __forceinline__ void absorb_max(float& m, float& s, float bm) {
  const float mn = fmaxf(m, bm);
  if (mn != m) {
    s = (m == -INFINITY) ? 0.f : s * exp_e(m - mn);
    m = mn;
  }
}

// General V (any alignment of the row length): scalar loads.
template <int THREADS, int U>
__global__ __launch_bounds__(THREADS) void score_logits_kernel(LogitsArgs o) {
  constexpr int NW = THREADS / 64;
  __shared__ float red[4][NW];
  const int row = blockIdx.x;
  const int t = threadIdx.x;
  const int V = o.V;
  const float* zon = o.on + (size_t)row * V;
  const float* zoff = o.off + (size_t)row * V;

  // The sampled token's two logits are fetched first, so that their latency
  // overlaps the streaming pass instead of following the reduction.
  int tk = 0;
  float z_on = 0.f, z_off = 0.f;
  if (t == 0) {
    tk = o.tokens[row];
    if (tk >= 0 && tk < V) {
      z_on = zon[tk];
      z_off = zoff[tk];
    }
  }

  float m_on = -INFINITY, s_on = 0.f, m_off = -INFINITY, s_off = 0.f;
  for (int base = t; base < V; base += THREADS * U) {
    float a[U], b[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * THREADS;
      a[u] = i < V ? zon[i] : -INFINITY;
      b[u] = i < V ? zoff[i] : -INFINITY;
    }
    float bm_on = -INFINITY, bm_off = -INFINITY;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      bm_on = fmaxf(bm_on, a[u]);
      bm_off = fmaxf(bm_off, b[u]);
    }
    absorb_max(m_on, s_on, bm_on);
    absorb_max(m_off, s_off, bm_off);
    if (m_on != -INFINITY) {
#pragma unroll
      for (int u = 0; u < U; ++u) s_on += exp_e(a[u] - m_on);
    }
    if (m_off != -INFINITY) {
#pragma unroll
      for (int u = 0; u < U; ++u) s_off += exp_e(b[u] - m_off);
    }
  }

  wave_merge(m_on, s_on);
  wave_merge(m_off, s_off);
  const int lane = t & 63, w = t >> 6;
  if (lane == 0) {
    red[0][w] = m_on;
    red[1][w] = s_on;
    red[2][w] = m_off;
    red[3][w] = s_off;
  }
  __syncthreads();
  if (t == 0) {
    float mo = red[0][0], so = red[1][0], mf = red[2][0], sf = red[3][0];
    for (int i = 1; i < NW; ++i) {
      lse_merge(mo, so, red[0][i], red[1][i]);
      lse_merge(mf, sf, red[2][i], red[3][i]);
    }
    finish_row(row, tk, V, z_on, z_off, mo, so, mf, sf, o);
  }
}

// The same for V % 4 == 0, streaming both rows as 16-byte buffer loads (zero
// past the row; the block's last batch masks those to -inf).  Running state
// per thread in base 2: m2 = max z * log2 e and s = sum 2^(z log2 e - m2),
// one FMA and one exp2 per logit.  The block combines by a max first (wave
// butterfly, then LDS), one rescale per thread, then sums (wave butterfly,
// then LDS in wave order).
template <int THREADS, int U>
__global__ __launch_bounds__(THREADS) void score_logits_vec_kernel(LogitsArgs o) {
  constexpr int NW = THREADS / 64;
  constexpr int STEP = THREADS * U;  // float4 per batch
  __shared__ float rmax[2][NW];
  __shared__ float rsum[2][NW];
  const int row = blockIdx.x, t = threadIdx.x, V = o.V;
  const float* zon = o.on + (size_t)row * V;
  const float* zoff = o.off + (size_t)row * V;
  // the sampled token's two logits first: their latency overlaps the stream
  int tk = 0;
  float z_on = 0.f, z_off = 0.f;
  if (t == 0) {
    tk = o.tokens[row];
    if (tk >= 0 && tk < V) {
      z_on = zon[tk];
      z_off = zoff[tk];
    }
  }
  const int nv4 = V >> 2;
  const __amdgpu_buffer_rsrc_t ron = make_rsrc(zon, (uint32_t)nv4 * 16u);
  const __amdgpu_buffer_rsrc_t roff = make_rsrc(zoff, (uint32_t)nv4 * 16u);
  float m_on = -INFINITY, s_on = 0.f, m_off = -INFINITY, s_off = 0.f;
  auto absorb = [&](float& m, float& sum, const float4 (&a)[U]) __attribute__((always_inline)) {
    float bm = a[0].x;
#pragma unroll
    for (int u = 0; u < U; ++u) bm = fmaxf(fmaxf(bm, a[u].x), fmaxf(fmaxf(a[u].y, a[u].z), a[u].w));
    const float mn = fmaxf(m, bm * kLog2e);
    sum = (m == -INFINITY) ? 0.f : sum * __builtin_amdgcn_exp2f(m - mn);
    m = mn;
    if (mn == -INFINITY) return;  // nothing but -inf so far
    float acc = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u)
      acc += (__builtin_amdgcn_exp2f(fmaf(a[u].x, kLog2e, -mn)) + __builtin_amdgcn_exp2f(fmaf(a[u].y, kLog2e, -mn))) +
             (__builtin_amdgcn_exp2f(fmaf(a[u].z, kLog2e, -mn)) + __builtin_amdgcn_exp2f(fmaf(a[u].w, kLog2e, -mn)));
    sum += acc;
  };
  const int nb = (nv4 + STEP - 1) / STEP;  // batches (block-uniform)
  for (int b = 0; b < nb; ++b) {
    float4 a[U], c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = t + b * STEP + u * THREADS;
      const int off = i < nv4 ? i * 16 : kOutOfRange;
      a[u] = __builtin_bit_cast(float4, buf_load16(ron, off));
      c[u] = __builtin_bit_cast(float4, buf_load16(roff, off));
    }
    if (b == nb - 1) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (t + b * STEP + u * THREADS >= nv4) {
          a[u] = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
          c[u] = a[u];
        }
    }
    absorb(m_on, s_on, a);
    absorb(m_off, s_off, c);
  }
  float wm_on = m_on, wm_off = m_off;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    wm_on = fmaxf(wm_on, __shfl_xor(wm_on, off));
    wm_off = fmaxf(wm_off, __shfl_xor(wm_off, off));
  }
  const int lane = t & 63, w = t >> 6;
  if (lane == 0) {
    rmax[0][w] = wm_on;
    rmax[1][w] = wm_off;
  }
  __syncthreads();
  float bm_on = rmax[0][0], bm_off = rmax[1][0];
#pragma unroll
  for (int i = 1; i < NW; ++i) {
    bm_on = fmaxf(bm_on, rmax[0][i]);
    bm_off = fmaxf(bm_off, rmax[1][i]);
  }
  float v_on = (m_on == -INFINITY) ? 0.f : s_on * __builtin_amdgcn_exp2f(m_on - bm_on);
  float v_off = (m_off == -INFINITY) ? 0.f : s_off * __builtin_amdgcn_exp2f(m_off - bm_off);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    v_on += __shfl_xor(v_on, off);
    v_off += __shfl_xor(v_off, off);
  }
  if (lane == 0) {
    rsum[0][w] = v_on;
    rsum[1][w] = v_off;
  }
  __syncthreads();
  if (t == 0) {
    float so = rsum[0][0], sf = rsum[1][0];
    for (int i = 1; i < NW; ++i) {
      so += rsum[0][i];
      sf += rsum[1][i];
    }
    // natural-log maxima for finish_row: lse = m + ln(s)
    finish_row(row, tk, V, z_on, z_off, bm_on / kLog2e, so, bm_off / kLog2e, sf, o);
  }
}

// One wave per token row; the workgroups past the rows compute the reward head.
constexpr int CB_THREADS = 256;
constexpr int CB_ROWS = CB_THREADS / 64;

__global__ __launch_bounds__(CB_THREADS) void score_combine_kernel(CombineArgs c) {
  const int t = threadIdx.x;
  const int nrow_blocks = (c.M + CB_ROWS - 1) / CB_ROWS;
  if ((int)blockIdx.x < nrow_blocks) {
    // (the wave index made provably wave-uniform: the row's buffer descriptor
    // then lives in SGPRs, with no per-lane loop around its loads)
    const int row = blockIdx.x * CB_ROWS + __builtin_amdgcn_readfirstlane(t >> 6);
    if (row >= c.M) return;
    const int lane = t & 63;
    // token and gathered logits first: their latency overlaps the merge
    const int tk = c.tokens[row];
    const bool ok = tk >= 0 && tk < c.V;
    float z_off = 0.f, z_on = 0.f;
    if (lane == 0 && ok) {
      z_off = c.zt[(size_t)row * 2 + 0];
      z_on = c.zt[(size_t)row * 2 + 1];
    }
    // Two passes over the row's partials (the second from cache): the row
    // maximum of each kind by a max butterfly, then sum_i s_i e^(m_i - max)
    // by an add butterfly, one exponential per partial.
    // Lane l takes partials l, l + 64, ..., four per round: the round's loads
    // are issued together (past the row they read as zeros and are masked by
    // selects, no branches).
    const int ntn = c.ntn;
    const __amdgpu_buffer_rsrc_t pr = make_rsrc(c.part + (size_t)row * ntn, (uint32_t)ntn * 16u);
    constexpr int RJ = 4;
    float mo = -INFINITY, mn = -INFINITY;
    for (int j0 = lane; j0 < ntn; j0 += 64 * RJ) {
      float4 q[RJ];
#pragma unroll
      for (int u = 0; u < RJ; ++u) {
        const int j = j0 + 64 * u;
        q[u] = __builtin_bit_cast(float4, buf_load16(pr, j < ntn ? j * 16 : kOutOfRange));
      }
#pragma unroll
      for (int u = 0; u < RJ; ++u) {
        const bool v = j0 + 64 * u < ntn;
        mo = fmaxf(mo, v ? q[u].x : -INFINITY);
        mn = fmaxf(mn, v ? q[u].z : -INFINITY);
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      mo = fmaxf(mo, __shfl_xor(mo, off));
      mn = fmaxf(mn, __shfl_xor(mn, off));
    }
    // (a partial with no columns has s = 0; an all-empty row keeps max = -inf and sum 0)
    const bool live_o = mo != -INFINITY, live_n = mn != -INFINITY;
    float so = 0.f, sn = 0.f;
    for (int j0 = lane; j0 < ntn; j0 += 64 * RJ) {
      float4 q[RJ];
#pragma unroll
      for (int u = 0; u < RJ; ++u) {
        const int j = j0 + 64 * u;
        q[u] = __builtin_bit_cast(float4, buf_load16(pr, j < ntn ? j * 16 : kOutOfRange));
      }
#pragma unroll
      for (int u = 0; u < RJ; ++u) {
        const bool v = j0 + 64 * u < ntn;
        const float eo = __fmul_rn(q[u].y, exp_e(q[u].x - mo));
        const float en = __fmul_rn(q[u].w, exp_e(q[u].z - mn));
        so = (v && live_o) ? __fadd_rn(so, eo) : so;
        sn = (v && live_n) ? __fadd_rn(sn, en) : sn;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      so = __fadd_rn(so, __shfl_xor(so, off));
      sn = __fadd_rn(sn, __shfl_xor(sn, off));
    }
    if (lane == 0) {
      LogitsArgs o{};
      o.lp_on = c.lp_on;
      o.lp_off = c.lp_off;
      o.kl = c.kl;
      o.lse_on = c.lse_on;
      o.lse_off = c.lse_off;
      o.err = c.err;
      finish_row(row, tk, c.V, z_on, z_off, mn, sn, mo, so, o);
    }
    return;
  }
  // reward head: one workgroup per sequence, fixed-order fp32 dot product.
  // Thread t takes the 8-element groups t, t + 256, ... of the row (K is a
  // multiple of 8), four groups per round with every load of a round issued
  // before its multiply-adds (16-byte loads of h; of w_rm too when it is
  // 16-byte aligned, else 2-byte ones); groups past the row read as zeros.
  const int b = blockIdx.x - nrow_blocks;
  if (b >= c.n_seq || c.w_rm == nullptr || c.reward == nullptr) return;
  __shared__ float part[CB_THREADS];
  const uint16_t* hr = c.h + ((size_t)b * c.seq_len + c.seq_len - 1) * c.K;
  const __amdgpu_buffer_rsrc_t hs = make_rsrc(hr, (uint32_t)c.K * 2u);
  const __amdgpu_buffer_rsrc_t ws = make_rsrc(c.w_rm, (uint32_t)c.K * 2u);
  const bool wvec = (reinterpret_cast<uintptr_t>(c.w_rm) & 15) == 0;
  const int ng = c.K / 8;
  constexpr int RG = 4;  // groups per round
  float acc = 0.f;
  auto fma8 = [&](const uint4& h8, const uint4& w8) __attribute__((always_inline)) {
    const uint32_t hw[4] = {h8.x, h8.y, h8.z, h8.w};
    const uint32_t ww[4] = {w8.x, w8.y, w8.z, w8.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc = fmaf(bf16_to_f32(hw[e] & 0xFFFFu), bf16_to_f32(ww[e] & 0xFFFFu), acc);
      acc = fmaf(bf16_to_f32(hw[e] >> 16), bf16_to_f32(ww[e] >> 16), acc);
    }
  };
  if (wvec) {
    for (int g0 = t; g0 < ng; g0 += RG * CB_THREADS) {
      uint4 hv[RG], wv[RG];
#pragma unroll
      for (int u = 0; u < RG; ++u) {
        const int gi = g0 + u * CB_THREADS;
        const int off = gi < ng ? gi * 16 : kOutOfRange;
        hv[u] = buf_load16(hs, off);
        wv[u] = buf_load16(ws, off);
      }
#pragma unroll
      for (int u = 0; u < RG; ++u) fma8(hv[u], wv[u]);
    }
  } else {
    for (int g0 = t; g0 < ng; g0 += RG * CB_THREADS) {
      uint4 hv[RG];
      uint32_t w16[RG][8];
#pragma unroll
      for (int u = 0; u < RG; ++u) {
        const int gi = g0 + u * CB_THREADS;
        hv[u] = buf_load16(hs, gi < ng ? gi * 16 : kOutOfRange);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          w16[u][e] = __builtin_amdgcn_raw_buffer_load_b16(ws, gi < ng ? gi * 16 + 2 * e : kOutOfRange, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < RG; ++u)
        fma8(hv[u], make_uint4(w16[u][0] | (w16[u][1] << 16), w16[u][2] | (w16[u][3] << 16),
                               w16[u][4] | (w16[u][5] << 16), w16[u][6] | (w16[u][7] << 16)));
    }
  }
  part[t] = acc;
  __syncthreads();
  for (int w = CB_THREADS / 2; w > 0; w >>= 1) {
    if (t < w) part[t] += part[t + w];
    __syncthreads();
  }
  if (t == 0) c.reward[b] = part[0];
}

}  // namespace

hipError_t launch_score_logits(const LogitsArgs& o, hipStream_t stream) {
  constexpr int THREADS = 512, U = 4;
  const dim3 grid(o.M), block(THREADS);
  if ((o.V & 3) == 0 && (reinterpret_cast<uintptr_t>(o.on) & 15) == 0 && (reinterpret_cast<uintptr_t>(o.off) & 15) == 0)
    hipLaunchKernelGGL((score_logits_vec_kernel<THREADS, U>), grid, block, 0, stream, o);
  else
    hipLaunchKernelGGL((score_logits_kernel<THREADS, U>), grid, block, 0, stream, o);
  return hipGetLastError();
}

hipError_t launch_score_combine(const CombineArgs& c, hipStream_t stream) {
  const int nrow_blocks = (c.M + CB_ROWS - 1) / CB_ROWS;
  const int nrew = (c.w_rm && c.reward) ? c.n_seq : 0;
  const dim3 grid(nrow_blocks + nrew), block(CB_THREADS);
  hipLaunchKernelGGL(score_combine_kernel, grid, block, 0, stream, c);
  return hipGetLastError();
}

}  // namespace hydra
