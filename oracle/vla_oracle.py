"""CPU oracle for batched VLA rollout inference (TEST INFRASTRUCTURE ONLY).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this module.  It shares no code with the HIP library and the library
never calls it.

What it computes (VLA-RL, arXiv 2505.18719):
  * the policy pi_theta(v_out | o_t, v_in) of Sec. 3.3: an OpenVLA-style
    Llama-2 decoder (Sec. 3.1) run over [visual tokens ; prompt tokens],
    followed by auto-regressive generation of |A| = 7 action tokens, each a
    discrete bin of one action dimension (Sec. 3.1, Eq. 1);
  * per-token log-probabilities whose sum is the action log-probability of
    Eq. 1 (Alg. 1, rollout phase), and the entropy of each token distribution
    (the rollout entropy monitored in Sec. 4.2);
  * the teacher-forced recompute of those log-probabilities for stored
    actions, i.e. the numerator of the PPO ratio of Eq. 2;
  * the weights the rollout runs on: the original checkpoint with the updated
    LoRA adapters merged in, rounded to bf16 (Sec. 3.3, Rollout Phase);
  * the post-processing f of Alg. 1 / Sec. 3.3 that turns the action tokens
    into a continuous robot action (each token a bin of one action dimension);
  * the value estimate V(o_t, v_in) of Alg. 1 by a value model of the policy's
    own architecture (the "homogeneous value model" of Fig. 2): the decoder
    over the same prefix, then a linear value head on the final-normed hidden
    state of the last prefix row.

The decoder block is the standard Llama-2 one: pre-RMSNorm, rotary position
embedding (half-split pairing), causal softmax attention, SwiGLU MLP and
residual adds; no biases; untied embedding and LM head.  Sampling is
restricted to the action bins (the last ``action_bins`` vocabulary ids) at
temperature T (Sec. 4.3 trains at T = 1.5) by Gumbel-max with supplied noise.

Arithmetic is plain numpy in float64; matmul is the only library primitive.
Two precision modes:
  * ``"ideal"``: float64 throughout on the exact bf16 weights and inputs;
  * ``"bf16"``: the same, but a value is rounded to bf16 (round to nearest
    even, via float32) at each point where the bf16 GPU path stores it in
    bf16 -- the RMSNorm outputs that feed a matmul, q and k after RoPE, v, the
    attention output, and the SwiGLU product.  The paper runs its rollout in
    bfloat16 (Sec. 3.5 "Infrastructure"); these are the rounding points of that
    contract.  Everything else (residual stream, scores, probabilities) stays
    float64.

The sampling decision argmax(z/T + g) is taken in float32, the precision the
kernel takes it in; log-probabilities and entropy are float64.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

MODES = ("ideal", "bf16")


# ----------------------------------------------------------------------------
# scalar helpers
# ----------------------------------------------------------------------------
def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (nearest even) through float32; returns float64."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(f)
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32).astype(np.float64)
    out[nan] = np.nan
    return out


def _rounder(mode: str):
    if mode not in MODES:
        raise ValueError(f"mode must be one of {MODES}")
    return bf16_round if mode == "bf16" else (lambda a: a)


def to_f64(t) -> np.ndarray:
    """bf16/fp32 torch tensor or numpy array -> float64 numpy array (exact)."""
    if isinstance(t, torch.Tensor):
        return t.detach().to("cpu", torch.float64).numpy()
    return np.asarray(t, dtype=np.float64)


# ----------------------------------------------------------------------------
# decoder pieces (Llama-2 block)
# ----------------------------------------------------------------------------
def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_angles(pos: np.ndarray, head_dim: int, base: float) -> np.ndarray:
    """angle[p, i] = pos_p * base^(-2i/head_dim), i < head_dim/2."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / head_dim)
    return np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]


def apply_rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate each (x_i, x_{i+hd/2}) pair of every head by angle(pos, i).

    x: [L, H, hd]; pos: [L].
    """
    hd = x.shape[-1]
    half = hd // 2
    ang = rope_angles(pos, hd, base)[:, None, :]          # [L, 1, half]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
                     k_pos: np.ndarray, return_probs: bool = False):
    """softmax(q k^T / sqrt(hd) masked to k_pos <= q_pos) v, per head.

    q: [Lq, H, hd]; k, v: [Lk, H, hd].  Returns [Lq, H, hd] (and probs [H, Lq, Lk]).
    """
    hd = q.shape[-1]
    qh = np.transpose(q, (1, 0, 2))                      # [H, Lq, hd]
    kh = np.transpose(k, (1, 0, 2))
    vh = np.transpose(v, (1, 0, 2))
    s = np.matmul(qh, np.transpose(kh, (0, 2, 1))) / np.sqrt(hd)   # [H, Lq, Lk]
    allowed = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    s = np.where(allowed[None], s, -np.inf)
    s = s - np.max(s, axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / np.sum(p, axis=-1, keepdims=True)
    o = np.transpose(np.matmul(p, vh), (1, 0, 2))        # [Lq, H, hd]
    return (o, p) if return_probs else o


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class Weights:
    """float64 views of a bf16 weight set, converted on first use and cached."""

    def __init__(self, w: Dict[str, object], cfg, cache_layers: bool = True):
        self.cfg = cfg
        self._w = w
        self._cache_layers = cache_layers
        self._layers: Dict[int, Dict[str, np.ndarray]] = {}
        a0, a1 = cfg.action_begin, cfg.action_begin + cfg.action_bins
        self.lm_action = to_f64(w["lm_head"][a0:a1])      # [A, d]
        self.final_norm = to_f64(w["final_norm"])
        self._embed = w["embed"]

    def embed_rows(self, ids: Sequence[int]) -> np.ndarray:
        idx = torch.as_tensor(np.asarray(ids, dtype=np.int64))
        return to_f64(self._embed[idx])

    def layer(self, i: int) -> Dict[str, np.ndarray]:
        if i in self._layers:
            return self._layers[i]
        lw = {k: to_f64(t) for k, t in self._w["layers"][i].items()}
        if self._cache_layers:
            self._layers[i] = lw
        return lw


def as_weights(w, cfg, cache_layers: bool = True) -> Weights:
    return w if isinstance(w, Weights) else Weights(w, cfg, cache_layers)


def decoder_layer(cfg, lw: Dict[str, np.ndarray], x: np.ndarray, pos: np.ndarray,
                  cache: Optional[Dict[str, np.ndarray]], rnd) -> np.ndarray:
    """One pre-norm Llama block on rows x [L, d] at positions pos.

    ``cache`` holds this layer's rotated keys and values of earlier positions
    ({"k": [S, H, hd], "v": [S, H, hd], "pos": [S]}); the new rows are appended
    to it.  Attention sees the cached rows followed by the new ones.
    """
    L, d = x.shape
    H, hd = cfg.n_heads, cfg.head_dim
    u = rnd(rms_norm(x, lw["attn_norm"], cfg.rms_eps))
    q = (u @ lw["wq"].T).reshape(L, H, hd)
    k = (u @ lw["wk"].T).reshape(L, H, hd)
    v = (u @ lw["wv"].T).reshape(L, H, hd)
    q = rnd(apply_rope(q, pos, cfg.rope_base))
    k = rnd(apply_rope(k, pos, cfg.rope_base))
    v = rnd(v)
    if cache is not None:
        if "k" in cache:
            cache["k"] = np.concatenate([cache["k"], k], axis=0)
            cache["v"] = np.concatenate([cache["v"], v], axis=0)
            cache["pos"] = np.concatenate([cache["pos"], pos])
        else:
            cache["k"], cache["v"], cache["pos"] = k, v, np.asarray(pos)
        kk, vv, kp = cache["k"], cache["v"], cache["pos"]
    else:
        kk, vv, kp = k, v, pos
    o = rnd(causal_attention(q, kk, vv, pos, kp).reshape(L, d))
    x = x + o @ lw["wo"].T
    u = rnd(rms_norm(x, lw["mlp_norm"], cfg.rms_eps))
    h = rnd(silu(u @ lw["wgate"].T) * (u @ lw["wup"].T))
    return x + h @ lw["wdown"].T


def action_logits(cfg, W: Weights, h_rows: np.ndarray, rnd) -> np.ndarray:
    """Final RMSNorm of hidden rows, then the LM head restricted to the action
    bins: logits over the last ``action_bins`` vocabulary ids only."""
    u = rnd(rms_norm(h_rows, W.final_norm, cfg.rms_eps))
    return u @ W.lm_action.T


def sample_bin(z: np.ndarray, g: np.ndarray, temperature: float):
    """Gumbel-max over the action bins at temperature T.

    The sampled bin is argmax_j (z_j / T + g_j), decided in float32 with the
    lowest index winning an exact tie; it is a draw from softmax(z / T).
    Returns (bin, log p(bin), entropy of softmax(z/T), top-2 margin of z/T + g).
    """
    z = np.asarray(z, dtype=np.float64)
    s32 = z.astype(np.float32) / np.float32(temperature) + np.asarray(g, dtype=np.float32)
    k = int(np.argmax(s32))
    zt = z / temperature
    m = np.max(zt)
    lse = m + np.log(np.sum(np.exp(zt - m)))
    logp_all = zt - lse
    ent = float(-np.sum(np.exp(logp_all) * logp_all))
    s64 = zt + np.asarray(g, dtype=np.float64)
    top2 = np.partition(s64, -2)[-2:]
    return k, float(logp_all[k]), ent, float(top2[1] - top2[0])


def token_stats(z: np.ndarray, bin_index: int, temperature: float):
    """log p and entropy of softmax(z / T) at a given bin."""
    zt = np.asarray(z, dtype=np.float64) / temperature
    m = np.max(zt)
    lse = m + np.log(np.sum(np.exp(zt - m)))
    logp_all = zt - lse
    return float(logp_all[bin_index]), float(-np.sum(np.exp(logp_all) * logp_all))


# ----------------------------------------------------------------------------
# per-environment drivers
# ----------------------------------------------------------------------------
def prefix_embeddings(cfg, W: Weights, vis_b, prompt_b: np.ndarray) -> np.ndarray:
    """x^0 = [visual embeddings ; embedding rows of the prompt ids]."""
    return np.concatenate([to_f64(vis_b), W.embed_rows(prompt_b)], axis=0)


def forward_rows(cfg, W: Weights, x0: np.ndarray, mode: str = "bf16") -> np.ndarray:
    """Full causal forward of one sequence with no KV cache: final hidden rows."""
    rnd = _rounder(mode)
    pos = np.arange(x0.shape[0])
    x = x0
    for li in range(cfg.n_layers):
        x = decoder_layer(cfg, W.layer(li), x, pos, None, rnd)
    return x


def rollout_env(cfg, W: Weights, vis_b, prompt_b, gumbel_b: np.ndarray, temperature: float,
                mode: str = "bf16", feed_tokens: Optional[Sequence[int]] = None) -> Dict[str, np.ndarray]:
    """Prefill one environment's prefix, then generate |A| action tokens with a
    KV cache.  Token i comes from the logits at position L-1+i; tokens 0..5 are
    fed back, the last is not (nothing consumes it).

    ``feed_tokens`` (vocabulary ids) replaces the oracle's own samples as the
    tokens fed back, so that logits can be compared along another sampler's
    trajectory; the oracle's own choice is still reported in ``tokens``.
    """
    rnd = _rounder(mode)
    n_act, a0 = cfg.n_actions, cfg.action_begin
    x0 = prefix_embeddings(cfg, W, vis_b, prompt_b)
    L = x0.shape[0]
    caches: List[Dict[str, np.ndarray]] = [dict() for _ in range(cfg.n_layers)]
    x = x0
    pos = np.arange(L)
    for li in range(cfg.n_layers):
        x = decoder_layer(cfg, W.layer(li), x, pos, caches[li], rnd)
    h_last = x[-1:]
    out = {k: np.zeros(n_act, dtype=t) for k, t in
           (("tokens", np.int32), ("logp", np.float64), ("entropy", np.float64), ("margin", np.float64))}
    out["logits"] = np.zeros((n_act, cfg.action_bins), dtype=np.float64)
    for i in range(n_act):
        z = action_logits(cfg, W, h_last, rnd)[0]
        k, _, _, margin = sample_bin(z, gumbel_b[i], temperature)
        fed = k + a0 if feed_tokens is None else int(feed_tokens[i])
        lp, ent = token_stats(z, fed - a0, temperature)
        out["tokens"][i], out["margin"][i] = k + a0, margin
        out["logp"][i], out["entropy"][i], out["logits"][i] = lp, ent, z
        if i + 1 == n_act:
            break
        x = W.embed_rows([fed])
        p = np.array([L + i])
        for li in range(cfg.n_layers):
            x = decoder_layer(cfg, W.layer(li), x, p, caches[li], rnd)
        h_last = x
    return out


def teacher_forced_env(cfg, W: Weights, vis_b, prompt_b, actions_b: Sequence[int],
                       temperature: float, mode: str = "bf16") -> Dict[str, np.ndarray]:
    """Full forward over [visual ; prompt ; the |A| given action tokens] with no
    cache; token i is scored by the logits at row L-1+i (the numerator of the
    PPO ratio, Eq. 2)."""
    rnd = _rounder(mode)
    a0 = cfg.action_begin
    x0 = np.concatenate([prefix_embeddings(cfg, W, vis_b, prompt_b), W.embed_rows(actions_b)])
    L = x0.shape[0] - len(actions_b)
    h = forward_rows(cfg, W, x0, mode)
    z = action_logits(cfg, W, h[L - 1:L - 1 + cfg.n_actions], rnd)
    logp = np.zeros(cfg.n_actions)
    ent = np.zeros(cfg.n_actions)
    for i in range(cfg.n_actions):
        logp[i], ent[i] = token_stats(z[i], int(actions_b[i]) - a0, temperature)
    return {"logp": logp, "entropy": ent, "logits": z}


# ----------------------------------------------------------------------------
# batched front ends (environments are independent)
# ----------------------------------------------------------------------------
def _split_prompts(prompt_ids: np.ndarray, prompt_lens: np.ndarray) -> List[np.ndarray]:
    offs = np.concatenate([[0], np.cumsum(np.asarray(prompt_lens, dtype=np.int64))])
    return [np.asarray(prompt_ids[offs[b]:offs[b + 1]]) for b in range(len(prompt_lens))]


def rollout(cfg, w, vis, prompt_ids, prompt_lens, gumbel, temperature: float,
            mode: str = "bf16", envs: Optional[Sequence[int]] = None,
            feed_tokens: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
    """Batched rollout of Alg. 1's policy step over the selected environments.

    ``feed_tokens``, if given, is indexed by environment id ([B, 7] for the
    whole batch).  Returns tokens int32 [n, 7], logp / entropy / margin
    [n, 7], logits [n, 7, A] and ``logp_sum`` [n] (the action log-probability
    of Eq. 1) for the n selected environments.
    """
    W = as_weights(w, cfg)
    prompts = _split_prompts(prompt_ids, prompt_lens)
    envs = list(range(len(prompts))) if envs is None else list(envs)
    res = [rollout_env(cfg, W, vis[b], prompts[b], np.asarray(gumbel[b]), temperature, mode,
                       None if feed_tokens is None else feed_tokens[b]) for b in envs]
    out = {k: np.stack([r[k] for r in res]) for k in res[0]}
    out["logp_sum"] = out["logp"].sum(axis=1)
    return out


def teacher_forced(cfg, w, vis, prompt_ids, prompt_lens, actions, temperature: float,
                   mode: str = "bf16", envs: Optional[Sequence[int]] = None) -> Dict[str, np.ndarray]:
    """Teacher-forced log-probs / entropies of given action tokens [B, 7]."""
    W = as_weights(w, cfg)
    prompts = _split_prompts(prompt_ids, prompt_lens)
    envs = list(range(len(prompts))) if envs is None else list(envs)
    res = [teacher_forced_env(cfg, W, vis[b], prompts[b], actions[b], temperature, mode) for b in envs]
    out = {k: np.stack([r[k] for r in res]) for k in res[0]}
    out["logp_sum"] = out["logp"].sum(axis=1)
    return out


def prefill_logits(cfg, w, vis, prompt_ids, prompt_lens, mode: str = "bf16",
                   envs: Optional[Sequence[int]] = None) -> np.ndarray:
    """Action-bin logits at the last prefix row of each selected environment."""
    W = as_weights(w, cfg)
    rnd = _rounder(mode)
    prompts = _split_prompts(prompt_ids, prompt_lens)
    envs = list(range(len(prompts))) if envs is None else list(envs)
    rows = [forward_rows(cfg, W, prefix_embeddings(cfg, W, vis[b], prompts[b]), mode)[-1:] for b in envs]
    return action_logits(cfg, W, np.concatenate(rows), rnd)


def values(cfg, w, vis, prompt_ids, prompt_lens, value_head, mode: str = "bf16",
           envs: Optional[Sequence[int]] = None) -> np.ndarray:
    """Value estimates V(o_t, v_in) of Alg. 1 (one per selected environment)
    by a value model with the decoder architecture of the policy and weights
    ``w``: the final RMSNorm of the hidden state at the last prefix row (bf16
    at the head's input in bf16 mode, as for the action head) dotted with the
    value head [d]."""
    W = as_weights(w, cfg)
    rnd = _rounder(mode)
    prompts = _split_prompts(prompt_ids, prompt_lens)
    envs = list(range(len(prompts))) if envs is None else list(envs)
    rows = [forward_rows(cfg, W, prefix_embeddings(cfg, W, vis[b], prompts[b]), mode)[-1:] for b in envs]
    u = rnd(rms_norm(np.concatenate(rows), W.final_norm, cfg.rms_eps))
    return u @ to_f64(value_head)


# ----------------------------------------------------------------------------
# LoRA merge (Sec. 3.3, Rollout Phase: the updated LoRA weights are merged with
# the original checkpoint before the rollout)
# ----------------------------------------------------------------------------
def lora_merge(w0, lora_a, lora_b, scale: float) -> np.ndarray:
    """Merged weight of one linear layer, W = W0 + scale * B A (LoRA: a rank-r
    update B [out, r] A [r, in] of W0 [out, in], scale = alpha / r), computed in
    float64 from the original weights and rounded to bf16 (nearest even,
    through float32 -- the precision the kernel rounds from).  Returns float64."""
    return bf16_round(to_f64(w0) + float(scale) * (to_f64(lora_b) @ to_f64(lora_a)))


def merge_weights(w: Dict[str, object], adapters: List[Dict[str, tuple]], scale: float,
                  layers: Optional[Sequence[int]] = None) -> Dict[str, object]:
    """A copy of the weight set ``w`` (bf16 torch tensors) with ``adapters[i]``
    (per projection key: (A, B)) merged into layer ``layers[i]`` (all layers in
    order by default)."""
    layers = list(range(len(adapters))) if layers is None else list(layers)
    out = {k: v for k, v in w.items() if k != "layers"}
    out["layers"] = [dict(lw) for lw in w["layers"]]
    for li, ad in zip(layers, adapters):
        for k, (a, b) in ad.items():
            m = lora_merge(w["layers"][li][k], a, b, scale)
            out["layers"][li][k] = torch.from_numpy(m).to(torch.bfloat16)
    return out


def extract_actions(tokens, action_begin: int, bins: int, lo, hi) -> np.ndarray:
    """Continuous actions a = f(v_out) of Alg. 1: token i of an environment's
    action sequence is a bin of action dimension i (Sec. 3.3), bin
    k = token - action_begin of `bins` uniform bins over [lo_i, hi_i] (the
    per-dimension range the policy's actions were discretised over), and the
    action value is that bin's centre lo_i + (k + 1/2) (hi_i - lo_i) / bins.
    tokens [n, n_dims]; lo, hi [n_dims]; tokens outside the bins give NaN."""
    k = np.asarray(tokens, dtype=np.int64) - action_begin
    lo = np.asarray(lo, dtype=np.float64)
    hi = np.asarray(hi, dtype=np.float64)
    a = lo + (k + 0.5) * (hi - lo) / bins
    return np.where((k >= 0) & (k < bins), a, np.nan)
