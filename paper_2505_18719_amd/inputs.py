"""Seeded synthetic workloads for batched VLA rollout inference.

This module only *draws* inputs; it holds none of the decoder's arithmetic.
Both the HIP path and the CPU oracle consume exactly the bytes produced here.

Workloads stand in for what VLA-RL's rollout phase feeds its policy
(Alg. 1; Sec. 3.3 "Rollout Phase"): projected visual patch embeddings of the
current observation followed by instruction-prompt token ids, through an
OpenVLA-style Llama-2 decoder (Sec. 3.1).  The LIBERO observations, the
tokenizer and the trained checkpoint are not used: weights are random
N(0, 0.02) in bf16, visual embeddings N(0, 1) in bf16, prompt ids uniform in
[1, 31000), and the Gumbel noise used for sampling is supplied explicitly.

Seeding: every stream is derived from ``numpy.random.SeedSequence([seed,
stream, index...])`` so that each tensor can be regenerated independently.
Large normal tensors are drawn with ``torch.Generator`` on the requested
device; a weight set is therefore a function of (seed, device type): tests
always draw on one device and copy the bytes to the other.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np
import torch

# Stream ids of SeedSequence([seed, stream, ...]).
_S_WEIGHT, _S_VIS, _S_PROMPT_LEN, _S_PROMPT_ID, _S_GUMBEL, _S_ACTIONS, _S_GAIN, _S_LORA, _S_LEARN = range(9)


@dataclasses.dataclass(frozen=True)
class VlaConfig:
    """Decoder and rollout sizes (Llama-2-style decoder, OpenVLA action tokens)."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    vocab: int = 32064
    action_bins: int = 256          # the last 256 vocabulary ids are the action bins
    n_actions: int = 7              # |A| = 7 degrees of freedom (Eq. 1)
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    n_visual: int = 256             # projected visual patch tokens per observation
    batch: int = 4
    prompt_min: int = 16            # prompt length drawn uniformly in [prompt_min, prompt_max]
    prompt_max: int = 16
    page_size: int = 16
    prompt_id_hi: int = 31000       # prompt ids are uniform in [1, min(prompt_id_hi, action_begin))

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def action_begin(self) -> int:
        return self.vocab - self.action_bins

    @property
    def max_seq(self) -> int:
        return self.n_visual + self.prompt_max + self.n_actions

    def replace(self, **kw) -> "VlaConfig":
        return dataclasses.replace(self, **kw)


# The five workloads: tiny and mid decoders, and the OpenVLA-7B (Llama-2-7B)
# shape at batch 8, 64 (ragged prompts) and 128 (PPO-update minibatch).
TINY = VlaConfig("tiny_b4", n_layers=2, d_model=256, n_heads=4, d_ffn=688,
                 batch=4, prompt_min=16, prompt_max=16)
MID = VlaConfig("mid_b16", n_layers=8, d_model=1024, n_heads=16, d_ffn=2752,
                batch=16, prompt_min=32, prompt_max=32)
L7B_B8 = VlaConfig("openvla7b_b8", n_layers=32, d_model=4096, n_heads=32, d_ffn=11008,
                   batch=8, prompt_min=32, prompt_max=32)
L7B_B64 = VlaConfig("openvla7b_b64_ragged", n_layers=32, d_model=4096, n_heads=32,
                    d_ffn=11008, batch=64, prompt_min=16, prompt_max=48)
L7B_B128 = VlaConfig("openvla7b_b128_ppo", n_layers=32, d_model=4096, n_heads=32,
                     d_ffn=11008, batch=128, prompt_min=32, prompt_max=32)

PRESETS = {c.name: c for c in (TINY, MID, L7B_B8, L7B_B64, L7B_B128)}

LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wgate", "wup", "wdown")


def _seed(*key: int) -> int:
    return int(np.random.SeedSequence(list(key)).generate_state(1, np.uint64)[0] & ((1 << 63) - 1))


def _normal(shape, std: float, key, device) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(*key))
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(torch.bfloat16)


def layer_shapes(cfg: VlaConfig) -> Dict[str, tuple]:
    d, f = cfg.d_model, cfg.d_ffn
    return {"attn_norm": (d,), "wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
            "mlp_norm": (d,), "wgate": (f, d), "wup": (f, d), "wdown": (d, f)}


def make_weights(cfg: VlaConfig, seed: int = 0, device="cpu", std: float = 0.02,
                 gain_jitter: bool = False) -> Dict[str, object]:
    """Random-init decoder weights, bf16, row-major ``[out_features, in_features]``.

    Linear weights ~ N(0, std).  RMSNorm gains are 1, or 1 + N(0, 0.02) when
    ``gain_jitter`` is set (exercises the gain multiply).  Embedding and LM head
    are untied; there are no biases.
    """
    d, v = cfg.d_model, cfg.vocab
    dev = torch.device(device)

    def gain(key):
        if not gain_jitter:
            return torch.ones(d, dtype=torch.bfloat16, device=dev)
        return (1.0 + _normal((d,), 0.02, (seed, _S_GAIN) + key, dev).float()).to(torch.bfloat16)

    w: Dict[str, object] = {
        "embed": _normal((v, d), std, (seed, _S_WEIGHT, 0), dev),
        "lm_head": _normal((v, d), std, (seed, _S_WEIGHT, 1), dev),
        "final_norm": gain((2**20,)),
        "layers": [],
    }
    for li in range(cfg.n_layers):
        lw = {}
        for j, (k, shp) in enumerate(layer_shapes(cfg).items()):
            if k.endswith("norm"):
                lw[k] = gain((li, j))
            else:
                lw[k] = _normal(shp, std, (seed, _S_WEIGHT, 100 + li, j), dev)
        w["layers"].append(lw)
    return w


# Linear layers a LoRA adapter attaches to, with the weight-dict key of each.
LORA_PROJECTIONS = ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")


def make_lora(cfg: VlaConfig, rank: int, seed: int = 0, device="cpu", std: float = 0.02,
              layers=None) -> List[Dict[str, tuple]]:
    """Seeded LoRA adapters for every projection of the given layers (all by
    default): per layer ``{key: (A [rank, in_features], B [out_features, rank])}``,
    bf16, entries ~ N(0, std) (a trained adapter has both factors non-zero)."""
    layers = range(cfg.n_layers) if layers is None else layers
    shapes = layer_shapes(cfg)
    out = []
    for li in layers:
        ad = {}
        for j, k in enumerate(LORA_PROJECTIONS):
            n_out, n_in = shapes[k]
            ad[k] = (_normal((rank, n_in), std, (seed, _S_LORA, li, j, 0), torch.device(device)),
                     _normal((n_out, rank), std, (seed, _S_LORA, li, j, 1), torch.device(device)))
        out.append(ad)
    return out


def weights_to(w: Dict[str, object], device) -> Dict[str, object]:
    out = {k: (t.to(device) if isinstance(t, torch.Tensor) else t) for k, t in w.items() if k != "layers"}
    out["layers"] = [{k: t.to(device) for k, t in lw.items()} for lw in w["layers"]]
    return out


@dataclasses.dataclass
class RolloutInputs:
    vis: torch.Tensor            # bf16 [B, n_visual, d]
    prompt_lens: np.ndarray      # int32 [B]
    prompt_ids: np.ndarray       # int32 [sum(prompt_lens)], packed env by env
    gumbel: np.ndarray           # fp32 [B, n_actions, action_bins]

    @property
    def batch(self) -> int:
        return int(self.prompt_lens.shape[0])

    @property
    def prefix_lens(self) -> np.ndarray:
        return self.prompt_lens.astype(np.int64) + self.vis.shape[1]

    def env_prompt(self, b: int) -> np.ndarray:
        off = int(self.prompt_lens[:b].sum())
        return self.prompt_ids[off:off + int(self.prompt_lens[b])]


def gumbel_noise(cfg: VlaConfig, batch: int, seed: int = 0, step: int = 0) -> np.ndarray:
    """Standard Gumbel noise g = -log(-log u), u = (k + 1/2) / 2^24, k uniform
    in [0, 2^24); evaluated in fp64 and rounded once to fp32."""
    rng = np.random.default_rng([seed, _S_GUMBEL, step])
    k = rng.integers(0, 1 << 24, size=(batch, cfg.n_actions, cfg.action_bins), dtype=np.int64)
    u = (k.astype(np.float64) + 0.5) / float(1 << 24)
    return (-np.log(-np.log(u))).astype(np.float32)


def make_inputs(cfg: VlaConfig, batch: Optional[int] = None, seed: int = 0, step: int = 0,
                device="cpu", prompt_lens: Optional[List[int]] = None) -> RolloutInputs:
    """One environment step's observations for ``batch`` environments."""
    b = cfg.batch if batch is None else batch
    if prompt_lens is None:
        rng = np.random.default_rng([seed, _S_PROMPT_LEN, step])
        lens = rng.integers(cfg.prompt_min, cfg.prompt_max + 1, size=b).astype(np.int32)
    else:
        lens = np.asarray(prompt_lens, dtype=np.int32)
        assert lens.shape == (b,)
    rng = np.random.default_rng([seed, _S_PROMPT_ID, step])
    ids = rng.integers(1, min(cfg.prompt_id_hi, cfg.action_begin), size=int(lens.sum())).astype(np.int32)
    vis = _normal((b, cfg.n_visual, cfg.d_model), 1.0, (seed, _S_VIS, step), torch.device(device))
    return RolloutInputs(vis=vis, prompt_lens=lens, prompt_ids=ids,
                         gumbel=gumbel_noise(cfg, b, seed, step))


def stored_actions(cfg: VlaConfig, batch: int, seed: int = 0, step: int = 0) -> np.ndarray:
    """Uniformly drawn action tokens (vocabulary ids in the action range),
    standing in for the tokens a PPO minibatch stored during rollout."""
    rng = np.random.default_rng([seed, _S_ACTIONS, step])
    bins = rng.integers(0, cfg.action_bins, size=(batch, cfg.n_actions))
    return (bins + cfg.action_begin).astype(np.int32)


def rollout_window(n_env: int, n_steps: int, seed: int = 0, p_done: float = 0.01):
    """A synthetic window of Alg. 1's rollout buffer, time-major: rewards
    [M, N] fp32 (a sparse success reward of 1 with probability p_done plus a
    dense N(0, 0.1) process reward), values [M + 1, N] fp32 ~ U(0, 1) and
    episode-start flags dones [M + 1, N] uint8 with P(1) = p_done."""
    rng = np.random.default_rng([seed, _S_LEARN, n_env, n_steps])
    dones = (rng.random((n_steps + 1, n_env)) < p_done).astype(np.uint8)
    rewards = (rng.random((n_steps, n_env)) < p_done) + rng.normal(scale=0.1, size=(n_steps, n_env))
    values = rng.random((n_steps + 1, n_env))
    return rewards.astype(np.float32), values.astype(np.float32), dones


def ppo_minibatch(n: int, n_tokens: int = 7, seed: int = 0, spread: float = 0.1):
    """Token log-probabilities of n stored actions under the old policy
    (negative, -Exp(mean 4), about the range of a 256-bin token at T = 1.5),
    the same under an updated policy shifted by N(0, spread) per token, and
    N(0, 1) advantages; all fp32 numpy."""
    rng = np.random.default_rng([seed, _S_LEARN + 1, n, n_tokens])
    old = -rng.exponential(scale=4.0, size=(n, n_tokens))
    new = old + rng.normal(scale=spread, size=old.shape)
    adv = rng.normal(size=n)
    return old.astype(np.float32), new.astype(np.float32), adv.astype(np.float32)
