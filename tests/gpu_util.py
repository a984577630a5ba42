"""Shared helpers of the GPU parity tests (inputs on the device, oracle on the
host, comparisons with the tolerances of the rollout contract)."""
import sys

import numpy as np
import torch

import oracle
from paper_2505_18719_amd import inputs

LOGIT_TOL = 3e-2      # max |logit difference|, bf16 weights with fp32 accumulation
LOGP_TOL = 1e-2       # max |log-prob difference|
TIE_EPS = 1e-3        # near-tie scale of the Gumbel-max scores


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class Setup:
    """Weights drawn on the GPU, copied once to the host for the oracle."""

    def __init__(self, cfg, seed=0, gain_jitter=False, max_batch=None, max_seq=None):
        from paper_2505_18719_amd.vla import VlaModel
        self.cfg = cfg
        self.w = inputs.make_weights(cfg, seed=seed, device="cuda", gain_jitter=gain_jitter)
        self.wc = inputs.weights_to(self.w, "cpu")
        self.model = VlaModel(cfg, self.w, max_batch=max_batch, max_seq=max_seq)
        self.W = oracle.as_weights(self.wc, cfg)

    def inputs(self, batch=None, seed=0, step=0, prompt_lens=None):
        inp = inputs.make_inputs(self.cfg, batch=batch, seed=seed, step=step, device="cuda",
                                 prompt_lens=prompt_lens)
        dev = {"vis": inp.vis, "ids": torch.from_numpy(inp.prompt_ids).cuda(),
               "gumbel": torch.from_numpy(inp.gumbel).cuda()}
        return inp, dev


def compare_rollout(cfg, W, inp, gpu, T, envs=None, mode="bf16", label=""):
    """Oracle fed with the GPU's own tokens; returns the error statistics.

    Tokens are checked three ways: (1) sampling is exact -- each GPU token is
    the oracle sampler's Gumbel-max choice on the GPU's own logits and the
    supplied noise (no exclusion); (2) the stated criterion -- against the
    oracle's logits, tokens are bit-exact except where the oracle's top-2
    score margin (of z/T + g) is below TIE_EPS; (3) the margin that the
    measured logit difference cannot bridge, max(TIE_EPS, 2 * max|dz| / T).
    The counts of (2) and (3) are returned separately: ``strict`` counts the
    mismatches at margins >= TIE_EPS, ``mismatches`` the sampler mismatches
    plus those at margins >= the bridge margin.
    """
    envs = list(range(inp.batch)) if envs is None else list(envs)
    toks = gpu["tokens"].cpu().numpy()
    ref = oracle.rollout(cfg, W, inp.vis.cpu(), inp.prompt_ids, inp.prompt_lens, inp.gumbel, T, mode=mode,
                         envs=envs, feed_tokens=toks)
    lg = gpu["logits"].cpu().numpy()[envs]
    lp = gpu["logp"].cpu().numpy()[envs]
    en = gpu["entropy"].cpu().numpy()[envs]
    dl = np.abs(lg - ref["logits"]).max()
    dp = np.abs(lp - ref["logp"]).max()
    de = np.abs(en - ref["entropy"]).max()
    a0 = cfg.action_begin
    samp_bad = 0
    for ei, b in enumerate(envs):
        for i in range(cfg.n_actions):
            k = oracle.sample_bin(lg[ei, i].astype(np.float64), inp.gumbel[b, i], T)[0]
            samp_bad += int(toks[b, i] != a0 + k)
    thr = max(TIE_EPS, 2.0 * dl / T)
    margin = ref["margin"]
    diff = toks[envs] != ref["tokens"]
    tie = margin < TIE_EPS
    band = (margin >= TIE_EPS) & (margin < thr)
    clear = margin >= thr
    mism = int((diff & clear).sum())
    strict = int((diff & ~tie).sum())
    bad_margins = ", ".join(f"{m:.2e}" for m in np.sort(margin[diff]))
    log(f"[{label}] mode={mode} envs={len(envs)} max|dlogit|={dl:.3e} max|dlogp|={dp:.3e} "
        f"max|dH|={de:.3e} sampler mismatches={samp_bad}; tokens {diff.size}: margin < {TIE_EPS:.0e}: "
        f"{int(tie.sum())} ({int((diff & tie).sum())} differ), in [{TIE_EPS:.0e}, {thr:.1e}): {int(band.sum())} "
        f"({int((diff & band).sum())} differ), beyond: {int(clear.sum())} ({mism} differ); "
        f"margins of differing tokens: [{bad_margins}]")
    return dict(dlogit=dl, dlogp=dp, dent=de, mismatches=mism + samp_bad, strict=strict + samp_bad,
                near=int((diff & ~clear).sum()), band=int(band.sum()), ref=ref)
