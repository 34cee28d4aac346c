// Offline optimisation of the exit policy's Q-network on the device
// (gfx950), Section 3.2 with the training hyperparameters of Section 4.1:
// noisy-layer initialisation, replay-ring writes (the decisions of a policy
// step with their Section 3.1.3 rewards, or caller transitions), one learning
// update in one block (n-step TD target from the target network, mean square
// error, gradient, Adam), and the acting weights of the exit policy.
//
// The networks are tiny (3 -> H -> 2, H <= 128) and a mini-batch is a few
// dozen transitions, so an update is a single block whose every sum runs in
// a fixed order: the same inputs give the same bits.
#include "kernels.h"

namespace lede {

namespace {

// f(x) = sgn(x) sqrt(|x|) of factorised noisy layers
__device__ __forceinline__ float noise_f(float x) { return copysignf(sqrtf(fabsf(x)), x); }

// Noise of parameter p of a set, from the f-values of one draw laid out as
// f(eps_in1) [3], f(eps_out1) [H], f(eps_in2) [H], f(eps_out2) [2].
__device__ __forceinline__ float noise_of(const float* nf, int H, int p) {
  const float *fi1 = nf, *fo1 = nf + 3, *fi2 = nf + 3 + H, *fo2 = nf + 3 + 2 * H;
  if (p < 3 * H) return fo1[p / 3] * fi1[p % 3];
  p -= 3 * H;
  if (p < H) return fo1[p];
  p -= H;
  if (p < 2 * H) return fo2[p / H] * fi2[p % H];
  return fo2[p - 2 * H];
}

}  // namespace

// mu ~ U(-1/sqrt(p), 1/sqrt(p)) from the caller's uniforms and sigma =
// sigma0 / sqrt(p), p the fan-in (3 for layer 1, H for layer 2); the target
// network starts equal; Adam moments start at zero.
__global__ void k_dqn_init(DqnInitArgs a) {
  const int H = a.H, P = dqn_params(H);
  const float r3 = sqrtf(3.f), rh = sqrtf((float)H);
  for (int p = blockIdx.x * blockDim.x + threadIdx.x; p < P; p += gridDim.x * blockDim.x) {
    const float fan = p < 4 * H ? r3 : rh;
    const float mu = (2.f * a.u[p] - 1.f) / fan, sg = a.sigma0 / fan;
    a.theta[p] = mu;
    a.theta[P + p] = sg;
    a.target[p] = mu;
    a.target[P + p] = sg;
    a.m[p] = 0.f;
    a.m[P + p] = 0.f;
    a.v[p] = 0.f;
    a.v[P + p] = 0.f;
  }
}

// One learning update (one block of DQN_THREADS).
__global__ __launch_bounds__(DQN_THREADS) void k_dqn_update(DqnUpdateArgs a) {
  constexpr int PMAX = 6 * DQN_MAX_HIDDEN + 2, NMAX = 2 * DQN_MAX_HIDDEN + 5;
  __shared__ float w_on[PMAX], w_tg[PMAX], grad[PMAX];
  __shared__ float nf_on[NMAX], nf_tg[NMAX];
  __shared__ float pre[DQN_MAX_BH], pre_t[DQN_MAX_BH];   // pre_t later holds the hidden deltas
  __shared__ float sx[DQN_MAX_BATCH][3], sn[DQN_MAX_BATCH][3];
  __shared__ float ret[DQN_MAX_BATCH], dq[DQN_MAX_BATCH], d2[DQN_MAX_BATCH];
  __shared__ int act[DQN_MAX_BATCH], boot[DQN_MAX_BATCH];
  const int tid = threadIdx.x, NT = DQN_THREADS;
  const int H = a.H, B = a.B, P = dqn_params(H), NC = dqn_noise(H);
  // parameter p = tid + NT i of a set: its mean and scale, their Adam
  // moments and the target's, all requested up front (one round trip)
  constexpr int PI = (6 * DQN_MAX_HIDDEN + 2 + DQN_THREADS - 1) / DQN_THREADS;
  float th_mu[PI], th_sg[PI], m_mu[PI], m_sg[PI], v_mu[PI], v_sg[PI], tg_mu[PI], tg_sg[PI];
#pragma unroll
  for (int i = 0; i < PI; ++i) {
    const int p = tid + NT * i;
    if (p < P) {
      th_mu[i] = a.theta[p];
      th_sg[i] = a.theta[P + p];
      tg_mu[i] = a.target[p];
      tg_sg[i] = a.target[P + p];
      m_mu[i] = a.m[p];
      m_sg[i] = a.m[P + p];
      v_mu[i] = a.v[p];
      v_sg[i] = a.v[P + p];
    }
  }

  // noise of both networks, then their weights for this draw
  for (int i = tid; i < NC; i += NT) {
    nf_on[i] = noise_f(a.noise[i]);
    nf_tg[i] = noise_f(a.noise[NC + i]);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < PI; ++i) {
    const int p = tid + NT * i;
    if (p < P) {
      w_on[p] = th_mu[i] + th_sg[i] * noise_of(nf_on, H, p);
      w_tg[p] = tg_mu[i] + tg_sg[i] * noise_of(nf_tg, H, p);
    }
  }
  // sampled transitions: position floor(m * n_valid / 2^24) of the stored
  // ones (oldest first), the discounted sum of up to n rewards (stopping
  // after a terminal one) and the state n transitions later
  for (int b = tid; b < B; b += NT) {
    const float x = fminf(fmaxf(a.u[b] * 16777216.f, 0.f), 16777215.f);
    const uint64_t mq = (uint64_t)(uint32_t)x;
    const int j = (int)((mq * (uint64_t)a.n_valid) >> 24);
    const float* s0 = a.ring + (size_t)((a.oldest + j) % a.capacity) * DQN_SLOT;
    sx[b][0] = s0[0];
    sx[b][1] = s0[1];
    sx[b][2] = s0[2];
    act[b] = s0[3] > 0.5f ? 1 : 0;
    // every reward and terminal flag of the window is requested before the
    // first is used (one round trip), then folded in order
    float2 rd[DQN_MAX_N];
#pragma unroll
    for (int k = 0; k < DQN_MAX_N; ++k)
      if (k < a.n) rd[k] = *(const float2*)(a.ring + (size_t)((a.oldest + j + k) % a.capacity) * DQN_SLOT + 4);
    float R = 0.f, gk = 1.f;
    int bt = 1;
#pragma unroll
    for (int k = 0; k < DQN_MAX_N; ++k) {
      if (k < a.n && bt) {
        R += gk * rd[k].x;
        gk *= a.gamma;
        if (rd[k].y != 0.f) bt = 0;
      }
    }
    ret[b] = R;
    boot[b] = bt;
    const float* s1 = a.ring + (size_t)((a.oldest + j + a.n) % a.capacity) * DQN_SLOT;
    sn[b][0] = bt ? s1[0] : 0.f;
    sn[b][1] = bt ? s1[1] : 0.f;
    sn[b][2] = bt ? s1[2] : 0.f;
  }
  __syncthreads();
  // hidden pre-activations W1 s + b1 (online on s_t, target on s_{t+n})
  for (int e = tid; e < B * H; e += NT) {
    const int b = e / H, h = e % H;
    pre[e] = w_on[3 * h] * sx[b][0] + w_on[3 * h + 1] * sx[b][1] + w_on[3 * h + 2] * sx[b][2] + w_on[3 * H + h];
    pre_t[e] = w_tg[3 * h] * sn[b][0] + w_tg[3 * h + 1] * sn[b][1] + w_tg[3 * h + 2] * sn[b][2] + w_tg[3 * H + h];
  }
  __syncthreads();
  // Q-values, targets y = R + gamma^n max_a' Qbar(s_{t+n}, a') and TD errors
  for (int b = tid; b < B; b += NT) {
    float o0 = 0.f, o1 = 0.f, t0 = 0.f, t1 = 0.f;
    for (int h = 0; h < H; ++h) {
      const float r = fmaxf(pre[b * H + h], 0.f), rt = fmaxf(pre_t[b * H + h], 0.f);
      o0 += w_on[4 * H + h] * r;
      o1 += w_on[5 * H + h] * r;
      t0 += w_tg[4 * H + h] * rt;
      t1 += w_tg[5 * H + h] * rt;
    }
    const float q = act[b] ? o1 + w_on[6 * H + 1] : o0 + w_on[6 * H];
    float y = ret[b];
    if (boot[b]) y += a.gamma_n * fmaxf(t0 + w_tg[6 * H], t1 + w_tg[6 * H + 1]);
    const float d = q - y;
    d2[b] = d * d;
    dq[b] = 2.f * d / (float)B;
  }
  __syncthreads();
  // loss; output-layer gradients; hidden deltas dq W2[a] [pre > 0]
  if (tid == 0) {
    float L = 0.f;
    for (int b = 0; b < B; ++b) L += d2[b];
    a.loss_out[0] = L / (float)B;
  }
  for (int e = tid; e < 2 * H + 2; e += NT) {
    float g = 0.f;
    if (e < 2 * H) {
      const int ac = e / H, h = e % H;
      for (int b = 0; b < B; ++b)
        if (act[b] == ac) g += dq[b] * fmaxf(pre[b * H + h], 0.f);
      grad[4 * H + e] = g;
    } else {
      const int ac = e - 2 * H;
      for (int b = 0; b < B; ++b)
        if (act[b] == ac) g += dq[b];
      grad[6 * H + ac] = g;
    }
  }
  for (int e = tid; e < B * H; e += NT) {
    const int b = e / H, h = e % H;
    pre_t[e] = pre[e] > 0.f ? dq[b] * w_on[4 * H + act[b] * H + h] : 0.f;
  }
  __syncthreads();
  // first-layer gradients
  for (int e = tid; e < 4 * H; e += NT) {
    float g = 0.f;
    if (e < 3 * H) {
      const int h = e / 3, i = e % 3;
      for (int b = 0; b < B; ++b) g += pre_t[b * H + h] * sx[b][i];
    } else {
      const int h = e - 3 * H;
      for (int b = 0; b < B; ++b) g += pre_t[b * H + h];
    }
    grad[e] = g;
  }
  __syncthreads();
  // Adam: d/dmu = g, d/dsigma = g * noise
  auto adam = [&](float g, float& th, float& m, float& v, size_t q) {
    m = a.beta1 * m + (1.f - a.beta1) * g;
    v = a.beta2 * v + (1.f - a.beta2) * g * g;
    a.m[q] = m;
    a.v[q] = v;
    const float mh = m / a.bc1, vh = v / a.bc2;
    th -= a.lr * (mh / (sqrtf(vh) + a.eps));
    a.theta[q] = th;
  };
#pragma unroll
  for (int i = 0; i < PI; ++i) {
    const int p = tid + NT * i;
    if (p < P) {
      const float g = grad[p];
      adam(g, th_mu[i], m_mu[i], v_mu[i], p);
      adam(g * noise_of(nf_on, H, p), th_sg[i], m_sg[i], v_sg[i], (size_t)P + p);
    }
  }
}

// The decisions of one exit-policy step as transitions: the stored action is
// the executed one (the last candidate layer exits by force); an exit scores
// its draft (draft 1 at a candidate layer, draft j at the pass that keeps it)
// as accepted when j <= accepted; a continue gets the continue penalty.
__global__ void k_dqn_record(DqnRecordArgs a) {
  const int i = threadIdx.x;
  if (i < a.n_dec && i >= a.n_dec - a.capacity) {
    const float* d = a.log + i * POLICY_LOG;
    const int kind = (int)d[0], where = (int)d[1];
    int exec = d[7] > 0.5f ? 1 : 0;
    if (kind == 0 && where == a.l_star) exec = 1;
    const int draft = kind == 0 ? 1 : where;
    const float r = exec == 0 ? a.r_continue : (draft <= a.accepted ? a.r_accept : a.r_reject);
    float* slot = a.ring + (size_t)(((int64_t)a.head + i) % a.capacity) * DQN_SLOT;
    slot[0] = d[2];
    slot[1] = d[3];
    slot[2] = d[4];
    slot[3] = (float)exec;
    slot[4] = r;
    slot[5] = (a.end_episode && i == a.n_dec - 1) ? 1.f : 0.f;
    slot[6] = 0.f;
    slot[7] = 0.f;
  }
  if (i == 0 && a.end_episode && a.n_dec == 0 && a.prev_newest >= 0)
    a.ring[(size_t)a.prev_newest * DQN_SLOT + 5] = 1.f;
}

// Caller transitions [n][6] appended to the ring (only the last `capacity`
// of them land when n exceeds it).
__global__ void k_dqn_push(DqnPushArgs a) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < a.n; i += gridDim.x * blockDim.x) {
    if (i < a.n - a.capacity) continue;
    const float* t = a.src + (size_t)i * 6;
    float* slot = a.ring + (size_t)(((int64_t)a.head + i) % a.capacity) * DQN_SLOT;
    for (int f = 0; f < 6; ++f) slot[f] = t[f];
    slot[6] = 0.f;
    slot[7] = 0.f;
  }
}

__global__ void k_dqn_copy(const float* src, float* dst, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) dst[i] = src[i];
}

// Weights of the acting network (one noise draw, or the means) written into
// the exit policy's W1, b1, W2, b2.
__global__ __launch_bounds__(DQN_THREADS) void k_dqn_act(DqnActArgs a) {
  __shared__ float nf[2 * DQN_MAX_HIDDEN + 5];
  const int H = a.H, P = dqn_params(H), NC = dqn_noise(H);
  for (int i = threadIdx.x; i < NC; i += DQN_THREADS) nf[i] = a.noise ? noise_f(a.noise[i]) : 0.f;
  __syncthreads();
  for (int p = threadIdx.x; p < P; p += DQN_THREADS) {
    const float w = a.noise ? a.theta[p] + a.theta[P + p] * noise_of(nf, H, p) : a.theta[p];
    if (p < 3 * H) a.w1[p] = w;
    else if (p < 4 * H) a.b1[p - 3 * H] = w;
    else if (p < 6 * H) a.w2[p - 4 * H] = w;
    else a.b2[p - 6 * H] = w;
  }
}

hipError_t launch_dqn_init(const DqnInitArgs& a, hipStream_t s) {
  const int P = dqn_params(a.H);
  hipLaunchKernelGGL(k_dqn_init, dim3((P + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_dqn_update(const DqnUpdateArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_dqn_update, dim3(1), dim3(DQN_THREADS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_dqn_record(const DqnRecordArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_dqn_record, dim3(1), dim3(128), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_dqn_push(const DqnPushArgs& a, hipStream_t s) {
  const int g = std::min(1024, (a.n + 255) / 256);
  hipLaunchKernelGGL(k_dqn_push, dim3(g), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_dqn_copy(const float* src, float* dst, int n, hipStream_t s) {
  hipLaunchKernelGGL(k_dqn_copy, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_dqn_act(const DqnActArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_dqn_act, dim3(1), dim3(DQN_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace lede
