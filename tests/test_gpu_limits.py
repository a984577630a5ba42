"""The size limits of the library on the GPU: a batch above the decode GEMM's
128 rows (the layer stack runs per chunk of environments) together with
sequences at the 320-row maximum and empty prompts, checked against the CPU
oracle on sampled environments, the teacher-forced pass included, and an
environment in the second chunk decoded alone."""
import numpy as np
import pytest
import torch

from gpu_util import LOGIT_TOL, LOGP_TOL, Setup, compare_rollout, log
from paper_2505_18719_amd import inputs

pytestmark = pytest.mark.gpu

LIMITS = inputs.TINY.replace(name="tiny_limits_b200", batch=200, prompt_min=0, prompt_max=57)


@pytest.fixture(scope="module")
def lim():
    assert LIMITS.max_seq == 320
    return Setup(LIMITS, seed=21)


def _inputs(S):
    lens = np.random.default_rng(21).integers(0, 58, size=LIMITS.batch).astype(np.int32)
    lens[[0, 130, 199]] = [57, 57, 0]  # full-length sequences in both chunks, an empty prompt
    return S.inputs(seed=21, prompt_lens=lens)


def test_batch_above_128_at_max_seq_matches_oracle(lim):
    S = lim
    inp, dev = _inputs(S)
    T = 1.5
    S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
    out = S.model.decode_actions(dev["gumbel"], T)
    torch.cuda.synchronize()
    envs = [0, 1, 127, 128, 130, 199]
    st = compare_rollout(S.cfg, S.W, inp, out, T, envs=envs, label="b200 max_seq 320")
    assert st["dlogit"] <= LOGIT_TOL and st["dlogp"] <= LOGP_TOL and st["mismatches"] == 0 and st["strict"] == 0
    # teacher-forced over the full sequences (320 rows for environments 0 and 130)
    tf = S.model.token_logprobs(dev["vis"], dev["ids"], inp.prompt_lens, out["tokens"].clone(), T)
    torch.cuda.synchronize()
    dd = np.abs(tf["logp"].cpu().numpy()[envs] - st["ref"]["logp"]).max()
    log(f"[b200 teacher-forced] max|dlogp| vs oracle={dd:.3e}")
    assert dd <= LOGP_TOL


def test_environment_in_the_second_chunk_alone_is_bit_identical(lim):
    S = lim
    inp, dev = _inputs(S)
    S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
    full = {k: v.clone() for k, v in S.model.decode_actions(dev["gumbel"], 1.5).items()}
    for b in (130, 199):
        off = int(inp.prompt_lens[:b].sum())
        ids1 = dev["ids"][off:off + int(inp.prompt_lens[b])].contiguous()
        S.model.prefill(dev["vis"][b:b + 1].contiguous(), ids1, inp.prompt_lens[b:b + 1])
        one = S.model.decode_actions(dev["gumbel"][b:b + 1].contiguous(), 1.5)
        torch.cuda.synchronize()
        for k in full:
            assert torch.equal(one[k][0], full[k][b]), (b, k)


def test_max_batch_512_rollout_matches_oracle():
    """The largest batch a handle accepts (512: four decode chunks), sequences up to 320 rows."""
    cfg = LIMITS.replace(name="tiny_limits_b512", batch=512)
    S = Setup(cfg, seed=22)
    inp, dev = S.inputs(seed=22)
    S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
    out = S.model.decode_actions(dev["gumbel"], 1.5)
    torch.cuda.synchronize()
    envs = [0, 255, 384, 511, int(np.argmax(inp.prompt_lens))]
    st = compare_rollout(cfg, S.W, inp, out, 1.5, envs=envs, label="b512")
    S.model.close()
    assert st["dlogit"] <= LOGIT_TOL and st["dlogp"] <= LOGP_TOL and st["mismatches"] == 0 and st["strict"] == 0
