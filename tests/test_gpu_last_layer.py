"""The last decoder layer computes its attention output, O projection and MLP
only for the rows read afterwards; every other row of that layer would only
have fed the KV cache.  Each row's arithmetic does not depend on which rows
run with it, so the results must be the same bits as computing every row
(the debug layer limit set to the full depth computes every row)."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, log
from paper_2505_18719_amd import inputs

pytestmark = pytest.mark.gpu


def _all_passes(S, inp, dev, T=1.5):
    out = {"prefill": S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens).clone()}
    dec = S.model.decode_actions(dev["gumbel"], T)
    out.update({f"decode_{k}": v.clone() for k, v in dec.items()})
    tf = S.model.token_logprobs(dev["vis"], dev["ids"], inp.prompt_lens, dec["tokens"].clone(), T)
    out.update({f"tf_{k}": v.clone() for k, v in tf.items()})
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    head = (torch.randn(S.cfg.d_model, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    out["value"] = S.model.value(dev["vis"], dev["ids"], inp.prompt_lens, head).clone()
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("cfg", [
    inputs.TINY.replace(name="tiny_ragged_ll", batch=6, prompt_min=0, prompt_max=40),
    inputs.MID,
    inputs.L7B_B64.replace(n_layers=2),
], ids=["tiny_ragged", "mid", "7b_width_2l_b64"])
def test_pruned_last_layer_is_bit_identical_to_every_row(cfg):
    S = Setup(cfg, seed=31, gain_jitter=cfg.d_model < 4096)
    inp, dev = S.inputs(seed=31)
    pruned = _all_passes(S, inp, dev)
    S.model.debug_layer_limit(cfg.n_layers)  # every row of the last layer
    full = _all_passes(S, inp, dev)
    S.model.debug_layer_limit(0)
    again = _all_passes(S, inp, dev)
    S.model.close()
    for k in pruned:
        assert torch.equal(pruned[k], full[k]), k
        assert torch.equal(pruned[k], again[k]), k
    log(f"[{cfg.name}] pruned last layer == every row, bitwise, over {len(pruned)} outputs")
