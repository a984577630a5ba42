"""Parity at the OpenVLA-7B shape, in the launch configurations the benchmark
times: the GPU runs the whole batch, the oracle recomputes sampled
environments one by one (environments are independent, so a subset is exact
for those rows).  The oracle's float64 copy of the 7B weights takes ~52 GB of
host memory."""
import time

import numpy as np
import pytest
import torch

import oracle
from gpu_util import LOGIT_TOL, LOGP_TOL, compare_rollout, log
from paper_2505_18719_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def big():
    from paper_2505_18719_amd.vla import VlaModel
    t0 = time.time()
    cfg = inputs.L7B_B128
    w = inputs.make_weights(cfg, seed=0, device="cuda")
    model = VlaModel(inputs.L7B_B64, w, max_batch=128, max_seq=inputs.L7B_B64.max_seq)
    wc = inputs.weights_to(w, "cpu")
    W = oracle.as_weights(wc, cfg)
    log(f"[7b] weights ready in {time.time() - t0:.1f}s")
    yield model, W
    model.close()


def _gpu_rollout(model, cfg, seed, T):
    inp = inputs.make_inputs(cfg, seed=seed, device="cuda")
    ids = torch.from_numpy(inp.prompt_ids).cuda()
    z0 = model.prefill(inp.vis, ids, inp.prompt_lens)
    out = model.decode_actions(torch.from_numpy(inp.gumbel).cuda(), T)
    torch.cuda.synchronize()
    return inp, ids, z0, out


def test_7b_b64_ragged_rollout_sampled_envs(big):
    model, W = big
    cfg = inputs.L7B_B64
    inp, _, z0, out = _gpu_rollout(model, cfg, 0, 1.5)
    toks = out["tokens"].cpu().numpy()
    assert ((toks >= cfg.action_begin) & (toks < cfg.vocab)).all()
    assert torch.isfinite(out["logp"]).all() and (out["logp"] <= 0).all()
    envs = [int(np.argmin(inp.prefix_lens)), int(np.argmax(inp.prefix_lens))]
    t0 = time.time()
    st = compare_rollout(cfg, W, inp, out, 1.5, envs=envs, label="7b b64 ragged")
    log(f"[7b] oracle on {len(envs)} envs (prefix {inp.prefix_lens[envs].tolist()}) in {time.time() - t0:.1f}s")
    assert st["dlogit"] <= LOGIT_TOL and st["dlogp"] <= LOGP_TOL and st["mismatches"] == 0


def test_7b_b8_rollout(big):
    model, W = big
    cfg = inputs.L7B_B8
    inp, _, z0, out = _gpu_rollout(model, cfg, 1, 1.0)
    st = compare_rollout(cfg, W, inp, out, 1.0, envs=[5], label="7b b8")
    assert st["dlogit"] <= LOGIT_TOL and st["dlogp"] <= LOGP_TOL and st["mismatches"] == 0


def test_7b_b128_teacher_forced_sampled_envs(big):
    model, W = big
    cfg = inputs.L7B_B128
    inp = inputs.make_inputs(cfg, seed=2, device="cuda")
    acts = inputs.stored_actions(cfg, cfg.batch, seed=2)
    tf = model.token_logprobs(inp.vis, torch.from_numpy(inp.prompt_ids).cuda(), inp.prompt_lens,
                              torch.from_numpy(acts).cuda(), 1.5)
    torch.cuda.synchronize()
    assert torch.isfinite(tf["logp"]).all()
    envs = [0, 127]
    ref = oracle.teacher_forced(cfg, W, inp.vis.cpu(), inp.prompt_ids, inp.prompt_lens, acts, 1.5, envs=envs)
    dl = np.abs(tf["logits"].cpu().numpy()[envs] - ref["logits"]).max()
    dp = np.abs(tf["logp"].cpu().numpy()[envs] - ref["logp"]).max()
    de = np.abs(tf["entropy"].cpu().numpy()[envs] - ref["entropy"]).max()
    log(f"[7b b128 teacher-forced] max|dlogit|={dl:.3e} max|dlogp|={dp:.3e} max|dH|={de:.3e}")
    assert dl <= LOGIT_TOL and dp <= LOGP_TOL and de <= LOGP_TOL
