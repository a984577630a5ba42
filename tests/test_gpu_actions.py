"""Parity of the action extraction f of Alg. 1 (tokens -> continuous robot
action, one uniform-bin dimension per token) with the CPU oracle, on random
tokens and on the tokens of a rollout of the tiny decoder."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import Setup, log
from paper_2505_18719_amd import inputs, vla

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def _ranges(n_dims, seed):
    rng = np.random.default_rng(seed)
    lo = rng.uniform(-1.5, 0.2, size=n_dims).astype(np.float32)
    hi = (lo + rng.uniform(0.05, 2.5, size=n_dims)).astype(np.float32)
    return lo, hi


def _check(tok, begin, bins, lo, hi):
    got = vla.extract_actions(torch.from_numpy(tok).cuda(), begin, bins, torch.from_numpy(lo).cuda(),
                              torch.from_numpy(hi).cuda()).cpu().numpy()
    ref = oracle.extract_actions(tok, begin, bins, lo, hi)
    bad = np.isnan(ref)
    assert np.array_equal(np.isnan(got), bad)
    # fp32: the width, the scaling and the add each round once
    tol = 4 * U32 * (np.abs(lo) + np.abs(hi) + np.abs(ref))
    err = np.abs(got - ref)
    assert np.all(err[~bad] <= np.broadcast_to(tol, ref.shape)[~bad])
    return got, err


@pytest.mark.parametrize("n,n_dims,bins", [(64, 7, 256), (1000, 7, 256), (3, 5, 1), (1, 16, 100)])
def test_extract_actions_matches_oracle(n, n_dims, bins):
    begin = 31808
    rng = np.random.default_rng(n + n_dims)
    tok = (begin + rng.integers(0, bins, size=(n, n_dims))).astype(np.int32)
    tok.flat[::11] = begin + bins - 1  # the top bin
    lo, hi = _ranges(n_dims, n)
    _, err = _check(tok, begin, bins, lo, hi)
    log(f"[extract n={n} dims={n_dims} bins={bins}] max|da|={err.max():.3e}")


def test_extract_actions_out_of_range_tokens_are_nan():
    begin, bins = 500, 256
    tok = np.array([[begin - 1, begin, begin + 255, begin + 256]], dtype=np.int32)
    lo, hi = _ranges(4, 1)
    got, _ = _check(tok, begin, bins, lo, hi)
    assert np.isnan(got[0, 0]) and np.isnan(got[0, 3]) and not np.isnan(got[0, 1:3]).any()


def test_extract_actions_of_a_rollout():
    S = Setup(inputs.TINY, seed=13)
    inp, dev = S.inputs(seed=13)
    S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
    out = S.model.decode_actions(dev["gumbel"], 1.5)
    torch.cuda.synchronize()
    lo, hi = _ranges(S.cfg.n_actions, 13)
    _check(out["tokens"].cpu().numpy(), S.cfg.action_begin, S.cfg.action_bins, lo, hi)
    S.model.close()
