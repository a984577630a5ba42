"""CPU oracle of the learning-phase arithmetic of VLA-RL (TEST INFRASTRUCTURE ONLY).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  It shares no code with the HIP library and the library
never calls it.

What it computes (arXiv 2505.18719, Alg. 1 after the rollout loop, and
Sec. 3.3 "Learning Phase"), in float64 numpy:
  * generalised advantage estimates over a window of M steps of N parallel
    environments, bootstrapped with the value of the observation after the
    window (Alg. 1 passes V_M to GAE), with episode boundaries given by the
    terminal indicators d_t of Alg. 1;
  * the clipped surrogate objective of Eq. 2, where the policy ratio of an
    action is exp of the difference of the action log-probabilities, each the
    sum of its token log-probabilities (Eq. 1), and its gradient with respect
    to every token log-probability;
  * the gradient of a token log-probability log softmax(z / T)[k] over the
    action bins with respect to the action logits z, which carries the
    surrogate's gradient back into the teacher-forced pass.

Readings where the paper is silent: d_t flags that o_t is the first
observation of a new episode, so the transition from step t to step t+1
continues an episode exactly when d_{t+1} = 0 (d_0 enters no transition of
the window); the objective of Eq. 2 is averaged over the actions of the batch
and the loss a minimiser uses is its negative; gamma, lambda and epsilon are
arguments (the paper gives no values).
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


def gae(rewards, values, dones, gamma: float, lam: float) -> Tuple[np.ndarray, np.ndarray]:
    """Advantages and returns of Alg. 1's GAE step.

    rewards [M, N]; values [M + 1, N] (row M is the bootstrap V_M); dones
    [M + 1, N] (d_t of Alg. 1; row 0 is not used).  With c_t = 1 - d_{t+1}:
        delta_t = r_t + gamma c_t V_{t+1} - V_t
        A_t     = delta_t + gamma lam c_t A_{t+1},   taken backwards from t = M-1 with A_M = 0
    and the return R_t = A_t + V_t (the value model's regression target).
    """
    r = np.asarray(rewards, dtype=np.float64)
    v = np.asarray(values, dtype=np.float64)
    d = np.asarray(dones, dtype=np.float64)
    M = r.shape[0]
    assert v.shape[0] == M + 1 and d.shape[0] == M + 1
    adv = np.zeros_like(r)
    nxt = np.zeros(r.shape[1:])
    for t in range(M - 1, -1, -1):
        cont = 1.0 - d[t + 1]
        delta = r[t] + gamma * cont * v[t + 1] - v[t]
        nxt = delta + gamma * lam * cont * nxt
        adv[t] = nxt
    return adv, adv + v[:M]


def ppo_clip(logp_new, logp_old, advantages, eps: float):
    """Clipped surrogate of Eq. 2 over n actions of n_tok tokens each.

    logp_new, logp_old [n, n_tok] token log-probabilities; advantages [n].
    The action log-probability is the token sum (Eq. 1), the ratio
    rho = exp(sum logp_new - sum logp_old), and the objective
        J = mean_t min(rho_t A_t, clip(rho_t, 1 - eps, 1 + eps) A_t).
    Returns (loss = -J, clipped fraction, dloss/dlogp_new [n, n_tok]).  The
    clipped term is the minimum exactly when A_t > 0 and rho_t > 1 + eps or
    A_t < 0 and rho_t < 1 - eps; there the loss does not depend on logp_new,
    otherwise d(-J)/dlogp_new[t, i] = -rho_t A_t / n for every token i.
    """
    ln = np.asarray(logp_new, dtype=np.float64)
    lo = np.asarray(logp_old, dtype=np.float64)
    a = np.asarray(advantages, dtype=np.float64)
    n = ln.shape[0]
    rho = np.exp(ln.sum(axis=1) - lo.sum(axis=1))
    surr = np.minimum(rho * a, np.clip(rho, 1.0 - eps, 1.0 + eps) * a)
    clipped = ((a > 0) & (rho > 1.0 + eps)) | ((a < 0) & (rho < 1.0 - eps))
    g = np.where(clipped, 0.0, -rho * a / n)
    return -surr.mean(), clipped.mean(), np.repeat(g[:, None], ln.shape[1], axis=1)


def logprob_grad(logits, tokens, action_begin: int, temperature: float, dlogp) -> np.ndarray:
    """dlogits [rows, bins] = dlogp * d log softmax(z / T)[k] / dz.

    logits [rows, bins] (raw, before temperature); tokens [rows] vocabulary
    ids, bin k = token - action_begin; dlogp [rows] the gradient arriving at
    each token log-probability.  With p = softmax(z / T):
        d log p_k / d z_j = (1[j = k] - p_j) / T.
    """
    z = np.asarray(logits, dtype=np.float64)
    k = np.asarray(tokens, dtype=np.int64) - action_begin
    s = z / temperature
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    onehot = np.zeros_like(p)
    onehot[np.arange(z.shape[0]), k] = 1.0
    return np.asarray(dlogp, dtype=np.float64)[:, None] * (onehot - p) / temperature
