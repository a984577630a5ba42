"""Parity of the backward of the teacher-forced pass (the PPO update's
gradient, Eq. 2 and Sec. 3.3 Learning Phase) with the CPU oracle: the loss,
the teacher-forced log-probs and the gradients of every LoRA factor of every
adapted projection, through the head, the final RMSNorm and every decoder
block (SwiGLU, RMSNorm, causal attention with rotary embedding)."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, log
from oracle import learn_oracle as lo
from paper_2505_18719_amd import inputs, vla

pytestmark = pytest.mark.gpu

PROJ = ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")


def _case(cfg, seed, rank=8, std=0.05, scale=0.5, layers_adapted=None, keys=PROJ):
    S = Setup(cfg, seed=seed)
    L = cfg.n_layers
    full = inputs.make_lora(cfg, rank, seed=seed, device="cuda", std=std)
    layers_adapted = range(L) if layers_adapted is None else layers_adapted
    ad = [{k: full[li][k] for k in keys} if li in layers_adapted else {} for li in range(L)]
    for li, layer in enumerate(ad):
        for k, (a, b) in layer.items():
            rp = (rank + 7) // 8 * 8  # the merge takes ranks in multiples of 8: zero rows of A, columns of B
            ap = torch.zeros(rp, a.shape[1], dtype=a.dtype, device=a.device)
            bp = torch.zeros(b.shape[0], rp, dtype=b.dtype, device=b.device)
            ap[:rank], bp[:, :rank] = a, b
            S.model.lora_merge(li, k, S.w["layers"][li][k], ap, bp.contiguous(), scale)
    inp, dev = S.inputs(seed=seed)
    B, T, eps = inp.batch, 1.5, 0.2
    acts = torch.from_numpy(inputs.stored_actions(cfg, B, seed=seed)).cuda()
    tf = S.model.token_logprobs(dev["vis"], dev["ids"], inp.prompt_lens, acts, T)
    rng = np.random.default_rng(seed)
    old = tf["logp"].cpu().numpy() + rng.normal(scale=0.03, size=(B, cfg.n_actions))
    adv = inputs.ppo_minibatch(B, seed=seed)[2]
    old[0] += -0.3 if adv[0] > 0 else 0.3  # action 0 clipped
    logp_old = torch.from_numpy(old.astype(np.float32)).cuda()
    advt = torch.from_numpy(adv).cuda()
    stats, lp_new, grads = S.model.ppo_lora_grads(dev["vis"], dev["ids"], inp.prompt_lens, acts, logp_old, advt,
                                                  eps, T, ad, scale)
    torch.cuda.synchronize()
    adc = [{k: (a.cpu(), b.cpu()) for k, (a, b) in layer.items()} for layer in ad]
    args = (cfg, S.wc, adc, scale, inp.vis.cpu(), inp.prompt_ids, inp.prompt_lens, acts.cpu().numpy(),
            logp_old.cpu().numpy(), adv, eps, T)
    ref = lo.ppo_lora_grads(*args, mode="bf16")
    ideal = lo.ppo_lora_grads(*args, mode="ideal")
    # how far the bf16 contract alone moves the oracle: the scale of any bf16 implementation's error
    ref["gap_logp"] = float(np.abs(ref["logp"] - ideal["logp"]).max())
    ref["gap_grad"] = max(np.linalg.norm(ref["grads"][li][k][f] - ideal["grads"][li][k][f])
                          / np.linalg.norm(ideal["grads"][li][k][f])
                          for li in range(cfg.n_layers) for k in ref["grads"][li] for f in (0, 1))
    S.model.close()
    return stats.cpu().numpy(), lp_new.cpu().numpy(), grads, ref


def _errors(grads, ref):
    out = {}
    for li, layer in enumerate(grads):
        for k, (ga, gb) in layer.items():
            for f, g in enumerate((ga, gb)):
                r = ref["grads"][li][k][f]
                g = g.cpu().double().numpy()
                out[(li, k, "AB"[f])] = (np.linalg.norm(g - r) / np.linalg.norm(r), np.abs(g - r).max() / np.abs(r).max())
    return out


# Gradient tolerance: the backward rounds its GEMM operands (activations and
# gradients) to bf16 and accumulates in fp32, against the oracle's exact chain
# rule through the same bf16-rounded forward; each layer the gradient crosses
# adds about one bf16 unit (2^-8) of relative error, so the bar on a tensor's
# relative error is (n_layers + 1) 2^-8 of its norm (1.5 times that for its
# largest entry), or twice the distance between the oracle's own bf16 and fp64
# gradients where that is larger (the wide 7B-width sums).  The log-probs use
# the stated 1e-2, or twice the oracle's bf16-vs-fp64 gap where larger, as the
# forward tests at full width do.
def _grad_tol(n_layers, gap):
    unit = (n_layers + 1) * 2.0 ** -8
    return max(unit, 2 * gap), 1.5 * max(unit, 2 * gap)


def _check(label, stats, lp, grads, ref, adv, n_layers):
    dlp = np.abs(lp - ref["logp"]).max()
    # the loss moves with the teacher-forced log-probs: rho changes by at most
    # n_actions * max|dlogp| in its exponent
    na = lp.shape[1]
    bound = np.mean(np.abs(adv)) * 1.3 * (np.expm1(na * dlp) + 1e-6) + 1e-6
    log(f"[{label}] loss gpu {stats[0]:.6f} oracle {ref['loss']:.6f} (bound {bound:.1e}); clipped {stats[1]:.3f} "
        f"vs {ref['clip_frac']:.3f}; max|dlogp| {dlp:.2e}")
    errs = _errors(grads, ref)
    worst_n = max(v[0] for v in errs.values())
    worst_m = max(v[1] for v in errs.values())
    log(f"[{label}] {len(errs)} gradient tensors: worst relative-norm error {worst_n:.3e}, relative-max {worst_m:.3e}")
    log(f"[{label}] oracle bf16-vs-fp64 gap: log-probs {ref['gap_logp']:.2e}, gradients {ref['gap_grad']:.2e}")
    assert dlp <= max(1e-2, 2 * ref["gap_logp"])
    n = len(adv)
    assert round(float(stats[1]) * n) == round(ref["clip_frac"] * n)  # the same actions clipped
    assert abs(stats[0] - ref["loss"]) <= bound
    tol_n, tol_m = _grad_tol(n_layers, ref["gap_grad"])
    assert worst_n <= tol_n and worst_m <= tol_m


def test_tiny_lora_gradients_match_oracle():
    """Both layers, all seven projections, rank 8, ragged prompts (empty ones included)."""
    cfg = inputs.TINY.replace(name="tiny_bwd", batch=4, prompt_min=0, prompt_max=16)
    stats, lp, grads, ref = _case(cfg, seed=41)
    _check("tiny bwd", stats, lp, grads, ref, inputs.ppo_minibatch(cfg.batch, seed=41)[2], cfg.n_layers)


def test_partial_adapters_and_odd_rank():
    """Adapters on the last layer's q, v and down projections only, rank 5: the
    other projections get no gradient buffers and the backward still runs
    through every layer."""
    cfg = inputs.TINY.replace(name="tiny_bwd_partial", batch=3, prompt_min=4, prompt_max=12)
    stats, lp, grads, ref = _case(cfg, seed=43, rank=5, layers_adapted=[cfg.n_layers - 1], keys=("wq", "wv", "wdown"))
    assert all(not g for g in grads[:-1]) and set(grads[-1]) == {"wq", "wv", "wdown"}
    _check("tiny bwd partial", stats, lp, grads, ref, inputs.ppo_minibatch(cfg.batch, seed=43)[2], cfg.n_layers)


def test_mid_lora_gradients_match_oracle():
    """Mid decoder (8 layers, d 1024, 16 heads): the gradient through eight layers."""
    cfg = inputs.MID.replace(batch=2)
    stats, lp, grads, ref = _case(cfg, seed=44, std=0.02)
    _check("mid bwd", stats, lp, grads, ref, inputs.ppo_minibatch(cfg.batch, seed=44)[2], cfg.n_layers)


def test_7b_width_two_layers_lora_gradients_match_oracle():
    """OpenVLA-7B width (d 4096, 32 heads of 128, FFN 11008), two layers, two
    environments: the head_dim-128 attention backward and the full-size GEMMs."""
    cfg = inputs.L7B_B8.replace(n_layers=2, batch=2)
    stats, lp, grads, ref = _case(cfg, seed=45, std=0.01)
    _check("7b-width 2L bwd", stats, lp, grads, ref, inputs.ppo_minibatch(cfg.batch, seed=45)[2], cfg.n_layers)


@pytest.mark.parametrize("rank", [48, 64])
def test_large_ranks_split_the_stacked_groups(rank):
    """Ranks 48 and 64 (16-row-aligned slots of 48 and 64 rows): at most two factors
    fit the 128-row operand of the low-rank products, so q, k, v run as two
    batches (q, k, then v) and gate, up fill all 128 rows."""
    cfg = inputs.TINY.replace(name=f"tiny_bwd_r{rank}", batch=3, prompt_min=2, prompt_max=14)
    stats, lp, grads, ref = _case(cfg, seed=47 + rank, rank=rank, std=0.03)
    _check(f"tiny bwd rank {rank}", stats, lp, grads, ref, inputs.ppo_minibatch(cfg.batch, seed=47 + rank)[2],
           cfg.n_layers)


def test_7b_width_longest_sequences():
    """Two environments of exactly 320 rows (256 visual + 57 prompt + 7 actions),
    the longest sequence the attention kernels hold: all ten 32-row chunks of the
    attention backward's LDS tiles in use, at head_dim 128, one layer."""
    cfg = inputs.L7B_B8.replace(name="openvla7b_full_len", n_layers=1, batch=2, prompt_min=57, prompt_max=57)
    assert cfg.max_seq == 320
    stats, lp, grads, ref = _case(cfg, seed=46, std=0.01)
    _check("7b-width 320-row bwd", stats, lp, grads, ref, inputs.ppo_minibatch(cfg.batch, seed=46)[2], cfg.n_layers)


@pytest.mark.parametrize("cfg", [inputs.TINY.replace(name="tiny_modes", batch=3, prompt_min=0, prompt_max=16),
                                 inputs.L7B_B8.replace(n_layers=2, batch=2)], ids=["tiny", "7b-width-2L"])
def test_keep_and_recompute_modes_give_the_same_bits(cfg):
    """The training forward that keeps every layer's activations and the one
    that keeps only the layer inputs (the backward recomputing the rest) run
    the same arithmetic: loss, log-probs and every gradient agree bit for bit."""
    S = Setup(cfg, seed=5)
    ad = inputs.make_lora(cfg, 8, seed=5, device="cuda", std=0.05)
    for li, layer in enumerate(ad):
        for k, (a, b) in layer.items():
            S.model.lora_merge(li, k, S.w["layers"][li][k], a, b, 0.5)
    inp, dev = S.inputs(seed=5)
    B, T = inp.batch, 1.5
    acts = torch.from_numpy(inputs.stored_actions(cfg, B, seed=5)).cuda()
    old = S.model.token_logprobs(dev["vis"], dev["ids"], inp.prompt_lens, acts, T)["logp"].contiguous()
    old = (old + 0.05).contiguous()
    adv = torch.from_numpy(inputs.ppo_minibatch(B, seed=5)[2]).cuda()
    out = {}
    for mode in (vla.TRAIN_KEEP, vla.TRAIN_RECOMPUTE):
        log(f"[modes {cfg.name}] training mode {mode}")
        st, lp, gr = S.model.ppo_lora_grads(dev["vis"], dev["ids"], inp.prompt_lens, acts, old, adv, 0.2, T, ad, 0.5,
                                           mode=mode)
        torch.cuda.synchronize()
        out[mode] = (st.cpu(), lp.cpu(), [{k: (ga.cpu(), gb.cpu()) for k, (ga, gb) in layer.items()} for layer in gr])
    S.model.close()
    (s0, l0, g0), (s1, l1, g1) = out[vla.TRAIN_KEEP], out[vla.TRAIN_RECOMPUTE]
    assert torch.equal(s0, s1) and torch.equal(l0, l1)
    n = 0
    for a, b in zip(g0, g1):
        for k in a:
            assert torch.equal(a[k][0], b[k][0]) and torch.equal(a[k][1], b[k][1]), k
            n += 2
    assert n == 14 * cfg.n_layers


def test_training_workspace_sizes_select_the_mode():
    """A workspace of the keep size runs the keep mode, one of the recompute size
    the recompute mode, observed through the profiled launches (the recompute
    re-runs each layer's QKV, O and gate/up GEMMs and its attention before the
    layer's backward), with the same bits; one byte less than the recompute
    size is refused with VLA_EWORKSPACE before any device work."""
    import ctypes
    cfg = inputs.TINY.replace(name="tiny_ws", batch=2, prompt_min=4, prompt_max=8)
    S = Setup(cfg, seed=9)
    ad = inputs.make_lora(cfg, 8, seed=9, device="cuda")
    for li, layer in enumerate(ad):
        for k, (a, b) in layer.items():
            S.model.lora_merge(li, k, S.w["layers"][li][k], a, b, 0.5)
    inp, dev = S.inputs(seed=9)
    acts = torch.from_numpy(inputs.stored_actions(cfg, inp.batch, seed=9)).cuda()
    old = S.model.token_logprobs(dev["vis"], dev["ids"], inp.prompt_lens, acts, 1.0)["logp"].contiguous()
    adv = torch.from_numpy(inputs.ppo_minibatch(inp.batch, seed=9)[2]).cuda()
    lib = vla.load_library()
    sizes = {}
    for mode in (vla.TRAIN_RECOMPUTE, vla.TRAIN_KEEP):
        n = ctypes.c_size_t()
        assert lib.vla_train_workspace_size(ctypes.byref(S.model.c_cfg), mode, ctypes.byref(n)) == 0
        sizes[mode] = n.value
    assert sizes[vla.TRAIN_KEEP] > sizes[vla.TRAIN_RECOMPUTE]
    runs = {}
    for mode in (vla.TRAIN_KEEP, vla.TRAIN_RECOMPUTE):
        S.model.profile_begin(("prefill_gemm", "prefill_attn"))
        st, lp, gr = S.model.ppo_lora_grads(dev["vis"], dev["ids"], inp.prompt_lens, acts, old, adv, 0.2, 1.0, ad,
                                            0.5, mode=mode)
        prof = S.model.profile_end()
        torch.cuda.synchronize()
        assert S.model._train_ws.numel() == sizes[mode]
        runs[mode] = (prof, st.cpu(), lp.cpu(), [{k: (a.cpu(), b.cpu()) for k, (a, b) in l.items()} for l in gr])
        log(f"[workspace modes] mode {mode}: {prof['prefill_gemm']['launches']} prefill GEMM and "
            f"{prof['prefill_attn']['launches']} attention launches")
    keep, rec = runs[vla.TRAIN_KEEP], runs[vla.TRAIN_RECOMPUTE]
    L = cfg.n_layers
    assert rec[0]["prefill_gemm"]["launches"] == keep[0]["prefill_gemm"]["launches"] + 3 * L
    assert rec[0]["prefill_attn"]["launches"] == keep[0]["prefill_attn"]["launches"] + L
    assert np.isfinite(rec[1].numpy()).all()
    assert torch.equal(keep[1], rec[1]) and torch.equal(keep[2], rec[2])
    for a, b in zip(keep[3], rec[3]):
        for k in a:
            assert torch.equal(a[k][0], b[k][0]) and torch.equal(a[k][1], b[k][1]), k
    # one byte short of the recompute size: refused on the host
    S.model._train_ws_mode = None
    S.model._train_ws = None
    small = torch.empty(sizes[vla.TRAIN_RECOMPUTE] - 1, dtype=torch.uint8, device="cuda")
    S.model._train_ws, S.model._train_ws_mode = small, "short"
    with pytest.raises(vla.VlaError) as err:
        S.model.ppo_lora_grads(dev["vis"], dev["ids"], inp.prompt_lens, acts, old, adv, 0.2, 1.0, ad, 0.5,
                               mode="short")
    assert err.value.code == -3
    S.model.close()
