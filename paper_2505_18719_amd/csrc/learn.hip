// Learning-phase kernels of VLA-RL (Alg. 1 after the rollout loop, Eq. 2):
// generalised advantage estimation over a window of steps, the PPO-clip
// surrogate with its gradient w.r.t. the token log-probabilities, and the
// gradient of those log-probabilities w.r.t. the action logits.
#include <hip/hip_runtime.h>

#include "common.h"
#include "kernels.h"

namespace vla {
namespace {

constexpr int kGaeChunks = 16;  // waves per workgroup; each takes one slice of the time axis

// One workgroup per 64 environments, wave w the time slice [t0_w, t1_w).
// The recursion A_t = delta_t + k_t A_{t+1} (k_t = gamma lam (1 - d_{t+1}))
// is affine in A_{t+1}, so a slice maps the advantage after it to the one at
// its start as A_{t0} = P + Q A_{t1}.  Pass 1 composes each slice's map, the
// slice maps are chained backwards from A_M = 0 in LDS, and pass 2 replays
// each slice from its true incoming advantage, writing A_t and A_t + V_t.
// Every wave reads rows t of 64 consecutive environments (coalesced).
__global__ __launch_bounds__(64 * kGaeChunks) void gae_kernel(GaeArgs a) {
  __shared__ float P[kGaeChunks][64], Q[kGaeChunks][64], Ain[kGaeChunks][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + lane;
  const int N = a.n_env, M = a.n_steps;
  const int L = (M + kGaeChunks - 1) / kGaeChunks;
  const int t0 = min(M, w * L), t1 = min(M, t0 + L);
  const bool live = n < N;
  const float gl = a.gamma * a.lam;
  float p = 0.f, q = 1.f;
  if (live) {
    float vn = a.values[(size_t)t1 * N + n];
    for (int t = t1 - 1; t >= t0; --t) {
      const float c = a.dones[(size_t)(t + 1) * N + n] ? 0.f : 1.f;
      const float v = a.values[(size_t)t * N + n];
      const float delta = a.rewards[(size_t)t * N + n] + a.gamma * c * vn - v;
      p = delta + gl * c * p;
      q = gl * c * q;
      vn = v;
    }
  }
  P[w][lane] = p;
  Q[w][lane] = q;
  __syncthreads();
  if (w == 0) {
    float nxt = 0.f;  // A_M
    for (int c = kGaeChunks - 1; c >= 0; --c) {
      Ain[c][lane] = nxt;
      nxt = P[c][lane] + Q[c][lane] * nxt;
    }
  }
  __syncthreads();
  if (!live) return;
  float adv = Ain[w][lane];
  float vn = a.values[(size_t)t1 * N + n];
  for (int t = t1 - 1; t >= t0; --t) {
    const float c = a.dones[(size_t)(t + 1) * N + n] ? 0.f : 1.f;
    const float v = a.values[(size_t)t * N + n];
    const float delta = a.rewards[(size_t)t * N + n] + a.gamma * c * vn - v;
    adv = delta + gl * c * adv;
    a.advantages[(size_t)t * N + n] = adv;
    if (a.returns) a.returns[(size_t)t * N + n] = adv + v;
    vn = v;
  }
}

// PPO-clip over n actions in one workgroup: thread i takes actions i, i + 1024,
// ... in order, the partial sums are combined by fixed wave and LDS trees, so
// the loss is the same bits on every run.
constexpr int kPpoThreads = 1024;
__global__ __launch_bounds__(kPpoThreads) void ppo_clip_kernel(PpoArgs a) {
  __shared__ float red[2][kPpoThreads / 64];
  const int tid = threadIdx.x;
  float s_surr = 0.f, s_clip = 0.f;
  for (int t = tid; t < a.n; t += kPpoThreads) {
    const float* ln = a.logp_new + (size_t)t * a.n_tokens;
    const float* lo = a.logp_old + (size_t)t * a.n_tokens;
    float sn = 0.f, so = 0.f;
    for (int i = 0; i < a.n_tokens; ++i) {
      sn += ln[i];
      so += lo[i];
    }
    const float rho = expf(sn - so);
    const float A = a.advantages[t];
    const float rc = fminf(fmaxf(rho, 1.f - a.eps), 1.f + a.eps);
    const bool clipped = (A > 0.f && rho > 1.f + a.eps) || (A < 0.f && rho < 1.f - a.eps);
    s_surr += fminf(rho * A, rc * A);
    s_clip += clipped ? 1.f : 0.f;
    const float g = clipped ? 0.f : -rho * A / (float)a.n;
    float* dl = a.dlogp + (size_t)t * a.n_tokens;
    for (int i = 0; i < a.n_tokens; ++i) dl[i] = g;
  }
  s_surr = wave_sum(s_surr);
  s_clip = wave_sum(s_clip);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = s_surr;
    red[1][tid >> 6] = s_clip;
  }
  __syncthreads();
  if (tid < 64) {
    float u = tid < kPpoThreads / 64 ? red[0][tid] : 0.f;
    float c = tid < kPpoThreads / 64 ? red[1][tid] : 0.f;
    u = wave_sum(u);
    c = wave_sum(c);
    if (tid == 0) {
      a.stats[0] = -u / (float)a.n;
      a.stats[1] = c / (float)a.n;
    }
  }
}

// d log softmax(z / T)[k] / dz_j = (1[j = k] - p_j) / T, scaled by the
// arriving gradient; one wave per row, bins j = lane + 64 u.
__global__ __launch_bounds__(256) void logprob_backward_kernel(LogprobBwdArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows) return;
  const float* z = a.logits + (size_t)row * a.bins;
  float zt[4];
  float m = -INFINITY;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int j = lane + 64 * u;
    zt[u] = j < a.bins ? z[j] / a.temperature : -INFINITY;
    m = fmaxf(m, zt[u]);
  }
  m = wave_max(m);
  float e[4], se = 0.f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    e[u] = lane + 64 * u < a.bins ? expf(zt[u] - m) : 0.f;
    se += e[u];
  }
  se = wave_sum(se);
  const int k = a.tokens[row] - a.action_begin;
  const float g = (k >= 0 && k < a.bins) ? a.dlogp[row] / a.temperature : __builtin_nanf("");
  const float inv = 1.f / se;
  float* dz = a.dlogits + (size_t)row * a.bins;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int j = lane + 64 * u;
    if (j < a.bins) dz[j] = g * ((j == k ? 1.f : 0.f) - e[u] * inv);
  }
}

}  // namespace

hipError_t launch_gae(const GaeArgs& a, hipStream_t s) {
  if (a.n_env <= 0 || a.n_steps <= 0) return hipSuccess;
  hipLaunchKernelGGL(gae_kernel, dim3((a.n_env + 63) / 64), dim3(64 * kGaeChunks), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ppo_clip(const PpoArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ppo_clip_kernel, dim3(1), dim3(kPpoThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_logprob_backward(const LogprobBwdArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.bins <= 0 || a.bins > 256) return hipErrorInvalidValue;
  hipLaunchKernelGGL(logprob_backward_kernel, dim3((a.rows + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace vla
