"""The persistent decode layer kernel (one cooperative launch per decoder
layer and decode step, grid barriers between its phases) against the
per-kernel decode path: the same inputs give the same bits, at tiny, mid and
7B width, with one and with several 128-row decode chunks, and no barrier
wait times out."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, log
from paper_2505_18719_amd import inputs

pytestmark = pytest.mark.gpu

FLAG_SYNC_TIMEOUT = 4


def _both_paths(S, inp, dev, T):
    outs = []
    for path in (0, 1):
        S.model.debug_decode_path(path)
        S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
        out = S.model.decode_actions(dev["gumbel"], T)
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in out.items()})
        assert S.model.read_flags() & FLAG_SYNC_TIMEOUT == 0
    S.model.debug_decode_path(0)
    return outs


@pytest.mark.parametrize("name", ["tiny_ragged", "mid", "7b_width_2l_b64", "tiny_b200"])
def test_persistent_decode_matches_the_per_kernel_path_bitwise(name):
    if name == "tiny_ragged":
        cfg, T, lens = inputs.TINY.replace(name=name, batch=5, prompt_min=0, prompt_max=40), 1.5, [0, 40, 7, 33, 16]
    elif name == "mid":
        cfg, T, lens = inputs.MID, 1.0, None
    elif name == "7b_width_2l_b64":
        cfg, T, lens = inputs.L7B_B64.replace(n_layers=2), 1.5, None
    else:
        cfg, T, lens = inputs.TINY.replace(name=name, batch=200, prompt_min=0, prompt_max=57), 1.5, None
    S = Setup(cfg, seed=11)
    inp, dev = S.inputs(seed=11, prompt_lens=lens)
    log(f"[decode paths {name}] batch {inp.batch}")
    ref, got = _both_paths(S, inp, dev, T)
    for k in ref:
        same = torch.equal(ref[k], got[k])
        if not same:
            d = (ref[k].double() - got[k].double()).abs().max().item()
            log(f"[decode paths {name}] {k} differs, max |d| {d:.3e}")
        assert same, k
    log(f"[decode paths {name}] tokens, log-probs, entropies, logits: identical bits")
    S.model.close()


def test_persistent_decode_repeats_bit_exactly():
    S = Setup(inputs.L7B_B64.replace(n_layers=2), seed=12)
    S.model.debug_decode_path(1)
    inp, dev = S.inputs(seed=12)
    outs = []
    for _ in range(3):
        S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
        out = S.model.decode_actions(dev["gumbel"], 1.5)
        torch.cuda.synchronize()
        outs.append({k: v.clone() for k, v in out.items()})
    for o in outs[1:]:
        for k in o:
            assert torch.equal(o[k], outs[0][k]), k
    assert S.model.read_flags() == 0
    S.model.close()
