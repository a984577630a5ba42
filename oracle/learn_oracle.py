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
    surrogate's gradient back into the teacher-forced pass;
  * the backward of that pass: the gradients of the PPO-clip loss with
    respect to the LoRA factors A, B of every adapted projection (the policy
    is trained through LoRA adapters merged as W0 + s B A, Sec. 3.3), by the
    chain rule through the head, the final RMSNorm and every decoder block.

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


# ----------------------------------------------------------------------------
# backward of the teacher-forced pass: gradients of the PPO-clip loss with
# respect to the LoRA factors (Sec. 3.3: the policy is trained through LoRA
# adapters; the Learning Phase minimises -J of Eq. 2)
# ----------------------------------------------------------------------------
from . import vla_oracle as vo  # noqa: E402

PROJ = ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")


def merged_layers(w, adapters, scale: float, mode: str = "ideal"):
    """Per-layer float64 weights W0 + s B A (rounded to bf16 in "bf16" mode,
    the weights a rollout after the merge runs on); norms unchanged."""
    out = []
    for li, lw0 in enumerate(w["layers"]):
        lw = {k: vo.to_f64(t) for k, t in lw0.items()}
        for k, (a, b) in (adapters[li] if adapters is not None else {}).items():
            m = lw[k] + scale * (vo.to_f64(b) @ vo.to_f64(a))
            lw[k] = vo.bf16_round(m) if mode == "bf16" else m
        out.append(lw)
    return out


def _layer_forward(cfg, lw, x, rnd):
    """One decoder block on a whole sequence, keeping what the backward reads."""
    L, d = x.shape
    H, hd = cfg.n_heads, cfg.head_dim
    pos = np.arange(L)
    c = {"x": x}
    c["u1"] = u1 = rnd(vo.rms_norm(x, lw["attn_norm"], cfg.rms_eps))
    q = rnd(vo.apply_rope((u1 @ lw["wq"].T).reshape(L, H, hd), pos, cfg.rope_base))
    k = rnd(vo.apply_rope((u1 @ lw["wk"].T).reshape(L, H, hd), pos, cfg.rope_base))
    v = rnd((u1 @ lw["wv"].T).reshape(L, H, hd))
    o, p = vo.causal_attention(q, k, v, pos, pos, return_probs=True)
    c.update(q=q, k=k, v=v, p=p)
    c["o"] = o = rnd(o.reshape(L, d))
    c["xm"] = xm = x + o @ lw["wo"].T
    c["u2"] = u2 = rnd(vo.rms_norm(xm, lw["mlp_norm"], cfg.rms_eps))
    c["g"], c["up"] = u2 @ lw["wgate"].T, u2 @ lw["wup"].T
    c["h"] = h = rnd(vo.silu(c["g"]) * c["up"])
    return xm + h @ lw["wdown"].T, c


def rms_norm_backward(x, gain, eps: float, dy):
    """dx of y = x r gain, r = (mean(x^2) + eps)^(-1/2), over the last axis."""
    d = x.shape[-1]
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    gd = dy * gain
    return r * gd - x * r ** 3 * np.sum(x * gd, axis=-1, keepdims=True) / d


def rope_backward(dy, pos, base: float):
    """Gradient through the rotary embedding: the transposed (inverse) rotation
    of each (i, i + hd/2) pair."""
    return vo.apply_rope(dy, -np.asarray(pos, dtype=np.float64), base)


def _layer_backward(cfg, lw, c, dout, dw):
    """Backward of one block: returns dx and adds dL/dW of every projection to dw."""
    x, L = c["x"], c["x"].shape[0]
    H, hd = cfg.n_heads, cfg.head_dim
    pos = np.arange(L)
    # MLP
    dh = dout @ lw["wdown"]
    dw["wdown"] += dout.T @ c["h"]
    g, up = c["g"], c["up"]
    sg = 1.0 / (1.0 + np.exp(-g))
    dg = dh * up * sg * (1.0 + g * (1.0 - sg))   # d silu(g) / dg = s (1 + g (1 - s))
    dup = dh * g * sg
    du2 = dg @ lw["wgate"] + dup @ lw["wup"]
    dw["wgate"] += dg.T @ c["u2"]
    dw["wup"] += dup.T @ c["u2"]
    dxm = dout + rms_norm_backward(c["xm"], lw["mlp_norm"], cfg.rms_eps, du2)
    # attention
    do = dxm @ lw["wo"]
    dw["wo"] += dxm.T @ c["o"]
    doh = np.transpose(do.reshape(L, H, hd), (1, 0, 2))
    qh, kh, vh = (np.transpose(c[n], (1, 0, 2)) for n in ("q", "k", "v"))
    p = c["p"]                                        # [H, L, L]
    scale = 1.0 / np.sqrt(hd)
    dv = np.matmul(np.transpose(p, (0, 2, 1)), doh)   # P^T dO
    dp = np.matmul(doh, np.transpose(vh, (0, 2, 1)))  # dO V^T
    ds = p * (dp - np.sum(dp * p, axis=-1, keepdims=True))
    dq = np.matmul(ds, kh) * scale
    dk = np.matmul(np.transpose(ds, (0, 2, 1)), qh) * scale
    dq = rope_backward(np.transpose(dq, (1, 0, 2)), pos, cfg.rope_base).reshape(L, -1)
    dk = rope_backward(np.transpose(dk, (1, 0, 2)), pos, cfg.rope_base).reshape(L, -1)
    dv = np.transpose(dv, (1, 0, 2)).reshape(L, -1)
    u1 = c["u1"]
    du1 = dq @ lw["wq"] + dk @ lw["wk"] + dv @ lw["wv"]
    dw["wq"] += dq.T @ u1
    dw["wk"] += dk.T @ u1
    dw["wv"] += dv.T @ u1
    return dxm + rms_norm_backward(x, lw["attn_norm"], cfg.rms_eps, du1)


def ppo_lora_grads(cfg, w, adapters, scale: float, vis, prompt_ids, prompt_lens, actions, logp_old,
                   advantages, eps: float, temperature: float, mode: str = "ideal"):
    """Loss -J of Eq. 2 over a minibatch of stored actions and its gradients
    with respect to every LoRA factor, through the teacher-forced pass.

    The policy's weights are W = W0 + s B A (Sec. 3.3); the action
    log-probabilities are the sums of the teacher-forced token log-probabilities
    (Eq. 1) over [visual ; prompt ; stored actions] (as vla_token_logprobs
    scores them), and the loss is ppo_clip's.  "ideal": float64 throughout;
    "bf16": the forward rounds where the rollout path stores bf16 (the
    backward is the exact chain rule through those values, a rounding treated
    as the identity).  Returns {"loss", "clip_frac", "logp", "grads"}, grads[l]
    = {projection: (dA, dB)} for the adapted projections of layer l.
    """
    rnd = vo._rounder(mode)
    layers = merged_layers(w, adapters, scale, mode)
    W = vo.as_weights(w, cfg)
    prompts = vo._split_prompts(np.asarray(prompt_ids), np.asarray(prompt_lens))
    a0, na, B = cfg.action_begin, cfg.n_actions, len(prompts)
    acts = np.asarray(actions, dtype=np.int64).reshape(B, na)
    # forward of every sequence, keeping the caches
    runs = []
    logp = np.zeros((B, na))
    for b in range(B):
        x = np.concatenate([vo.prefix_embeddings(cfg, W, vis[b], prompts[b]), W.embed_rows(acts[b])])
        L = x.shape[0] - na
        caches = []
        for lw in layers:
            x, c = _layer_forward(cfg, lw, x, rnd)
            caches.append(c)
        hrows = x[L - 1:L - 1 + na]
        z = vo.action_logits(cfg, W, hrows, rnd)
        for i in range(na):
            logp[b, i] = vo.token_stats(z[i], int(acts[b, i]) - a0, temperature)[0]
        runs.append((L, x, caches, z))
    loss, frac, dlogp = ppo_clip(logp, logp_old, advantages, eps)
    dws = [{k: np.zeros_like(lw[k]) for k in PROJ} for lw in layers]
    for b, (L, xL, caches, z) in enumerate(runs):
        dz = logprob_grad(z, acts[b], a0, temperature, dlogp[b])
        du = dz @ W.lm_action
        dx = np.zeros_like(xL)
        dx[L - 1:L - 1 + na] = rms_norm_backward(xL[L - 1:L - 1 + na], W.final_norm, cfg.rms_eps, du)
        for li in range(len(layers) - 1, -1, -1):
            dx = _layer_backward(cfg, layers[li], caches[li], dx, dws[li])
    grads = []
    for li in range(len(layers)):
        gl = {}
        for k, (a, bm) in (adapters[li] if adapters is not None else {}).items():
            a, bm = vo.to_f64(a), vo.to_f64(bm)
            gl[k] = (scale * bm.T @ dws[li][k], scale * dws[li][k] @ a.T)
        grads.append(gl)
    return {"loss": loss, "clip_frac": frac, "logp": logp, "grads": grads}
