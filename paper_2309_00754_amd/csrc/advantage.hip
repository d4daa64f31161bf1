// PPO advantage step for gfx950: the critic's per-token values from its
// scalar head, the per-token PPO reward, and generalized advantage estimation
// (Sec. 2, "Stage 3: PPO": GAE builds the advantage estimates from the reward
// using V; App. A, Alg. 2: critic values on the generated sequence, then the
// advantages from the reward and reference log-probabilities; App. B: KL
// weight beta, GAE gamma and lambda).
//
//  * value_head_kernel: V[m] = <h[m], w_v>.  Each wave takes two rows, which
//    share every chunk of w_v it loads; lane l takes 8 consecutive k of every
//    512-wide chunk (whole 1 KB lines), a batch of 8 chunks is requested
//    before the first is used, and the dot products run on v_dot2c_f32_bf16
//    with fp32 accumulation; the lanes are summed by a fixed butterfly.
//  * gae_kernel: one wave per sequence.  r_t = -beta KL_t on response tokens
//    (t >= start), plus the sequence reward on its last token; delta_t = r_t +
//    gamma V_{t+1} - V_t (V_T = 0); A_t = delta_t + gamma lambda A_{t+1}
//    (A_T = 0); returns A_t + V_t; positions before start are written as 0.
//    The recursion is a linear one, evaluated as a reverse scan: lane j owns
//    a contiguous chunk of positions, folds it into (F_j, B_j) = ((gamma
//    lambda)^len, the chunk's advantage at its first position with a zero
//    advantage after it), a Kogge-Stone suffix scan over the lanes combines
//    (F, B) pairs, and each lane then runs its chunk backwards from the
//    advantage that follows it.  Chunks of up to 16 positions keep their
//    residuals in registers (all their loads issued up front); longer ones
//    are recomputed in the second pass.  Fixed order throughout:
//    deterministic.
//  * ppo_loss_kernel: the update stage's losses (Sec. 2, "Stage 3: PPO"): the
//    clipped surrogate on the ratio rho = exp(lp_new - lp_old) and the
//    critic's squared-error loss on the returns, means over the response
//    tokens, with their per-token gradients.  One workgroup: thread t takes
//    tokens t, t + 1024, ..., and the partial sums meet in a fixed tree.
#include "hydra_device.h"
#include "hydra_internal.h"

namespace hydra {
namespace {

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;

__device__ __forceinline__ float dot8(const uint4& a, const uint4& b, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.x), __builtin_bit_cast(bf16x2_t, b.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.y), __builtin_bit_cast(bf16x2_t, b.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.z), __builtin_bit_cast(bf16x2_t, b.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.w), __builtin_bit_cast(bf16x2_t, b.w), acc, false);
  return acc;
}

constexpr int VH_WAVES = 4;  // waves per workgroup
constexpr int VH_ROWS = 2;   // rows per wave (sharing each w_v chunk)
constexpr int VH_BATCH = 8;  // 512-wide chunks requested before use

__global__ __launch_bounds__(VH_WAVES * 64) void value_head_kernel(ValueHeadArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int row0 = (blockIdx.x * VH_WAVES + wave) * VH_ROWS;
  if (row0 >= a.M) return;  // wave-uniform
  const int K = a.K;
  const int nrows = min(VH_ROWS, a.M - row0);
  // rows past M read as zeros through the descriptor
  const __amdgpu_buffer_rsrc_t hrs = make_rsrc(a.h + (size_t)row0 * K, (uint32_t)nrows * K * 2u);
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(a.w, (uint32_t)K * 2u);
  const int nch = (K + 511) / 512;
  float acc[VH_ROWS];
#pragma unroll
  for (int i = 0; i < VH_ROWS; ++i) acc[i] = 0.f;
  for (int c0 = 0; c0 < nch; c0 += VH_BATCH) {
    uint4 hv[VH_BATCH][VH_ROWS], wv[VH_BATCH];
#pragma unroll
    for (int u = 0; u < VH_BATCH; ++u) {
      const int k = (c0 + u) * 512 + lane * 8;
      const bool kv = c0 + u < nch && k < K;
      wv[u] = buf_load16(wrs, kv ? k * 2 : kOutOfRange);
#pragma unroll
      for (int i = 0; i < VH_ROWS; ++i) hv[u][i] = buf_load16(hrs, kv ? (i * K + k) * 2 : kOutOfRange);
    }
#pragma unroll
    for (int u = 0; u < VH_BATCH; ++u)
#pragma unroll
      for (int i = 0; i < VH_ROWS; ++i) acc[i] = dot8(hv[u][i], wv[u], acc[i]);
  }
#pragma unroll
  for (int i = 0; i < VH_ROWS; ++i) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc[i] += __shfl_xor(acc[i], o);
  }
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < VH_ROWS; ++i)
      if (i < nrows) a.values[row0 + i] = acc[i];
  }
}

constexpr int GAE_REG = 16;  // chunk length held in registers

__global__ __launch_bounds__(64) void gae_kernel(GaeArgs a) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int T = a.seq_len;
  const int C = (T + 63) / 64;  // positions per lane
  const int t0 = lane * C;
  const int t1 = min(T, t0 + C);
  const size_t base = (size_t)b * T;
  const float c = a.gamma * a.lam;
  const float rew = a.reward[b];

  auto reward_at = [&](int t, float kl) __attribute__((always_inline)) {
    float r = t >= a.start ? -a.beta * kl : 0.f;
    if (t == T - 1) r += rew;
    return r;
  };
  auto delta_at = [&](int t) __attribute__((always_inline)) {
    const float v1 = t + 1 < T ? a.values[base + t + 1] : 0.f;
    return fmaf(a.gamma, v1, reward_at(t, a.kl[base + t])) - a.values[base + t];
  };

  // this lane's chunk folded with a zero advantage after it
  float F = 1.f, Bv = 0.f;
  float dl[GAE_REG], vl[GAE_REG], rl[GAE_REG];
  const bool in_regs = C <= GAE_REG;
  if (in_regs) {
    float kv[GAE_REG], vv[GAE_REG + 1];
#pragma unroll
    for (int i = 0; i < GAE_REG; ++i) {
      const int t = t0 + i;
      kv[i] = t < t1 ? a.kl[base + t] : 0.f;
      vv[i] = t < t1 ? a.values[base + t] : 0.f;
    }
    vv[GAE_REG] = 0.f;
#pragma unroll
    for (int i = 0; i < GAE_REG; ++i) {
      const int t = t0 + i;
      const float v1 = i + 1 < C ? vv[i + 1] : (t1 < T ? a.values[base + t1] : 0.f);
      rl[i] = reward_at(t, kv[i]);
      vl[i] = vv[i];
      dl[i] = fmaf(a.gamma, v1, rl[i]) - vv[i];
    }
#pragma unroll
    for (int i = GAE_REG - 1; i >= 0; --i) {
      if (t0 + i < t1) {
        Bv = fmaf(c, Bv, dl[i]);
        F *= c;
      }
    }
  } else {
    for (int t = t1 - 1; t >= t0; --t) {
      Bv = fmaf(c, Bv, delta_at(t));
      F *= c;
    }
  }
  // suffix scan over lanes: (F, B)_j <- (F_j F_{j+o}, B_j + F_j B_{j+o})
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float Fo = __shfl_down(F, o);
    const float Bo = __shfl_down(Bv, o);
    if (lane + o < 64) {
      Bv = fmaf(F, Bo, Bv);
      F *= Fo;
    }
  }
  // advantage right after this lane's chunk = the suffix result of lane + 1
  float A = __shfl_down(Bv, 1);
  if (lane == 63) A = 0.f;
  if (in_regs) {
#pragma unroll
    for (int i = GAE_REG - 1; i >= 0; --i) {
      const int t = t0 + i;
      if (t < t1) {
        A = fmaf(c, A, dl[i]);
        const bool resp = t >= a.start;
        a.advantages[base + t] = resp ? A : 0.f;
        a.returns[base + t] = resp ? A + vl[i] : 0.f;
        if (a.rewards) a.rewards[base + t] = rl[i];
      }
    }
  } else {
    for (int t = t1 - 1; t >= t0; --t) {
      A = fmaf(c, A, delta_at(t));
      const bool resp = t >= a.start;
      a.advantages[base + t] = resp ? A : 0.f;
      a.returns[base + t] = resp ? A + a.values[base + t] : 0.f;
      if (a.rewards) a.rewards[base + t] = reward_at(t, a.kl[base + t]);
    }
  }
}

constexpr int PL_THREADS = 1024;

__global__ __launch_bounds__(PL_THREADS) void ppo_loss_kernel(PpoLossArgs a) {
  __shared__ float red[3][PL_THREADS / 64];
  const int t = threadIdx.x;
  const int T = a.seq_len;
  const int M = a.n_seq * T;
  const float inv_n = 1.f / ((float)a.n_seq * (float)(T - a.start));
  const float lo_b = 1.f - a.eps, hi_b = 1.f + a.eps;
  float pg = 0.f, vl = 0.f, cf = 0.f;
  for (int m = t; m < M; m += PL_THREADS) {
    float dl = 0.f, dv = 0.f;
    if (m % T >= a.start) {
      const float rho = exp_e(a.lp_new[m] - a.lp_old[m]);
      const float A = a.adv[m];
      const float un = rho * A;
      const float cl = fminf(fmaxf(rho, lo_b), hi_b) * A;
      if (un <= cl) {
        pg += un;
        dl = -un * inv_n;
      } else {
        pg += cl;
        cf += 1.f;
      }
      const float d = a.values[m] - a.returns[m];
      vl = fmaf(0.5f * d, d, vl);
      dv = d * inv_n;
    }
    if (a.d_lp) a.d_lp[m] = dl;
    if (a.d_v) a.d_v[m] = dv;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    pg += __shfl_xor(pg, o);
    vl += __shfl_xor(vl, o);
    cf += __shfl_xor(cf, o);
  }
  const int lane = t & 63, w = t >> 6;
  if (lane == 0) {
    red[0][w] = pg;
    red[1][w] = vl;
    red[2][w] = cf;
  }
  __syncthreads();
  if (t == 0) {
    float sp = 0.f, sv = 0.f, sc = 0.f;
    for (int i = 0; i < PL_THREADS / 64; ++i) {
      sp += red[0][i];
      sv += red[1][i];
      sc += red[2][i];
    }
    a.losses[0] = -sp * inv_n;
    a.losses[1] = sv * inv_n;
    a.losses[2] = sc * inv_n;
  }
}

}  // namespace

hipError_t launch_value_head(const ValueHeadArgs& a, hipStream_t stream) {
  const int rows_per_wg = VH_WAVES * VH_ROWS;
  hipLaunchKernelGGL(value_head_kernel, dim3((a.M + rows_per_wg - 1) / rows_per_wg), dim3(VH_WAVES * 64), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_ppo_loss(const PpoLossArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(ppo_loss_kernel, dim3(1), dim3(PL_THREADS), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gae(const GaeArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(gae_kernel, dim3(a.n_seq), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace hydra
