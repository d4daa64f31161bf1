// Scoring kernels for gfx950: sampled-token log-probabilities under the
// LoRA-on (actor) and LoRA-off (reference) passes, their difference as the
// per-token KL estimate, and the scalar reward head (Sec. 3, the two heads of
// pi^hydra; App. A, Alg. 1 / Alg. 2, "compute reward and reference log
// probabilities"; the KL weight beta of App. B is applied by the caller).
//
//  * score_logits_kernel: one workgroup per token row streams both fp32
//    logit rows once (float4 loads), keeping a per-thread running
//    (max, sum exp) and reducing it across the workgroup in a fixed tree.
//  * score_combine_kernel: one wave per token row merges the per-column-tile
//    partials written by the fused CLM-head GEMM in tile order, then forms
//    lse, lp and KL; extra workgroups compute the reward head's dot products.
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

template <int THREADS, int U, bool VEC>
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
  if constexpr (VEC) {
    const int nv4 = V >> 2;
    const float4* pon = reinterpret_cast<const float4*>(zon);
    const float4* poff = reinterpret_cast<const float4*>(zoff);
    for (int base = t; base < nv4; base += THREADS * U) {
      float4 a[U], b[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = base + u * THREADS;
        const bool v = i < nv4;
        a[u] = v ? pon[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        b[u] = v ? poff[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      }
      float bm_on = -INFINITY, bm_off = -INFINITY;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        bm_on = fmaxf(bm_on, fmaxf(fmaxf(a[u].x, a[u].y), fmaxf(a[u].z, a[u].w)));
        bm_off = fmaxf(bm_off, fmaxf(fmaxf(b[u].x, b[u].y), fmaxf(b[u].z, b[u].w)));
      }
      absorb_max(m_on, s_on, bm_on);
      absorb_max(m_off, s_off, bm_off);
      if (m_on != -INFINITY) {
#pragma unroll
        for (int u = 0; u < U; ++u)
          s_on += (exp_e(a[u].x - m_on) + exp_e(a[u].y - m_on)) + (exp_e(a[u].z - m_on) + exp_e(a[u].w - m_on));
      }
      if (m_off != -INFINITY) {
#pragma unroll
        for (int u = 0; u < U; ++u)
          s_off += (exp_e(b[u].x - m_off) + exp_e(b[u].y - m_off)) + (exp_e(b[u].z - m_off) + exp_e(b[u].w - m_off));
      }
    }
  } else {
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

// One wave per token row; the workgroups past the rows compute the reward head.
constexpr int CB_THREADS = 256;
constexpr int CB_ROWS = CB_THREADS / 64;

__global__ __launch_bounds__(CB_THREADS) void score_combine_kernel(CombineArgs c) {
  const int t = threadIdx.x;
  const int nrow_blocks = (c.M + CB_ROWS - 1) / CB_ROWS;
  if ((int)blockIdx.x < nrow_blocks) {
    const int row = blockIdx.x * CB_ROWS + (t >> 6);
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
    const float4* p = c.part + (size_t)row * c.ntn;
    float mo = -INFINITY, so = 0.f, mn = -INFINITY, sn = 0.f;
    for (int j = lane; j < c.ntn; j += 64) {
      const float4 q = p[j];
      lse_merge(mo, so, q.x, q.y);
      lse_merge(mn, sn, q.z, q.w);
    }
    wave_merge(mn, sn);
    wave_merge(mo, so);
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
  // reward head: one workgroup per sequence, fixed-order fp32 dot product
  const int b = blockIdx.x - nrow_blocks;
  if (b >= c.n_seq || c.w_rm == nullptr || c.reward == nullptr) return;
  __shared__ float part[CB_THREADS];
  const uint16_t* hr = c.h + ((size_t)b * c.seq_len + c.seq_len - 1) * c.K;
  float acc = 0.f;
  for (int k = t; k < c.K; k += CB_THREADS) acc = fmaf(bf16_to_f32(hr[k]), bf16_to_f32(c.w_rm[k]), acc);
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
  if ((o.V & 3) == 0)
    hipLaunchKernelGGL((score_logits_kernel<THREADS, U, true>), grid, block, 0, stream, o);
  else
    hipLaunchKernelGGL((score_logits_kernel<THREADS, U, false>), grid, block, 0, stream, o);
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
