"""Pins of the CPU oracle against facts that do not come from the oracle itself:
library routines (torch's bf16 cast, RMSNorm, scaled-dot-product attention,
HuggingFace's Llama decoder), closed forms, invariants of the mathematics and
brute force on tiny inputs.  Every function of the oracle is reached by at
least one pin whose failure a plausible slip (dropped term, wrong sign or
index, transposed operand) would trigger.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import vla_oracle as vo
from paper_2505_18719_amd.inputs import TINY, gumbel_noise, make_inputs, make_weights

# A very small decoder for brute-force and library pins: 2 layers, d 64,
# 4 heads of 16, FFN 96, vocabulary 600 of which the last 256 are action bins.
PIN = TINY.replace(name="pin", d_model=64, n_heads=4, d_ffn=96, vocab=600, n_visual=8,
                   batch=3, prompt_min=3, prompt_max=6)


@pytest.fixture(scope="module")
def pin_setup():
    w = make_weights(PIN, seed=3, gain_jitter=True)
    inp = make_inputs(PIN, seed=5)
    return w, inp


# ---------------------------------------------------------------- bf16 rounding
def test_bf16_round_matches_torch_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(size=4000) * 10.0 ** rng.integers(-8, 8, 4000),
                        [0.0, -0.0, 1.0, 65504.0, 3.0e38]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(vo.bf16_round(x), ref)


def test_bf16_round_ties_to_even():
    # bf16 keeps 7 explicit mantissa bits: the spacing above 1 is 2^-7.
    assert vo.bf16_round(np.array([1 + 2.0 ** -8]))[0] == 1.0
    assert vo.bf16_round(np.array([1 + 3 * 2.0 ** -8]))[0] == 1 + 2.0 ** -6
    assert vo.bf16_round(np.array([1 + 2.0 ** -8 + 2.0 ** -20]))[0] == 1 + 2.0 ** -7


# ---------------------------------------------------------------- RMSNorm
def test_rms_norm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(1)
    x = rng.normal(size=(5, 64)) * 3
    y = vo.rms_norm(x, np.ones(64), 1e-6)
    ms = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), np.sqrt(ms / (ms + 1e-6)), rtol=1e-12)
    np.testing.assert_allclose(vo.rms_norm(7.5 * x, np.ones(64), 0.0), vo.rms_norm(x, np.ones(64), 0.0),
                               rtol=1e-12)


def test_rms_norm_matches_torch_library():
    rng = np.random.default_rng(2)
    x, g = rng.normal(size=(7, 96)), 1 + 0.1 * rng.normal(size=96)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6)
    np.testing.assert_allclose(vo.rms_norm(x, g, 1e-6), ref.numpy(), rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- RoPE
def test_rope_preserves_norm_and_position_zero_is_identity():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(9, 3, 32))
    pos = np.arange(9) * 37
    y = vo.apply_rope(x, pos, 1e4)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    np.testing.assert_allclose(vo.apply_rope(x, np.zeros(9), 1e4), x, rtol=0, atol=0)


def test_rope_equals_complex_rotation():
    # Pair (x_i, x_{i+hd/2}) as the complex number x_i + i*x_{i+hd/2}, rotated
    # by exp(i * pos * base^(-2i/hd)).
    rng = np.random.default_rng(4)
    hd, pos = 16, np.array([0, 1, 5, 300])
    x = rng.normal(size=(4, 2, hd))
    c = x[..., : hd // 2] + 1j * x[..., hd // 2:]
    freq = np.array([10000.0 ** (-2 * i / hd) for i in range(hd // 2)])
    rot = c * np.exp(1j * pos[:, None, None] * freq[None, None, :])
    ref = np.concatenate([rot.real, rot.imag], axis=-1)
    np.testing.assert_allclose(vo.apply_rope(x, pos, 1e4), ref, rtol=1e-12, atol=1e-12)
    # First pair at position 1 is rotated by exactly one radian.
    e = np.zeros((1, 1, hd)); e[0, 0, 0] = 1.0
    y = vo.apply_rope(e, np.array([1]), 1e4)
    assert y[0, 0, 0] == pytest.approx(math.cos(1.0)) and y[0, 0, hd // 2] == pytest.approx(math.sin(1.0))


def test_rope_scores_depend_only_on_relative_position():
    rng = np.random.default_rng(5)
    q, k = rng.normal(size=(1, 1, 32)), rng.normal(size=(1, 1, 32))
    def score(m, n):
        return float(np.sum(vo.apply_rope(q, np.array([m]), 1e4) * vo.apply_rope(k, np.array([n]), 1e4)))
    for m, n, s in [(7, 3, 100), (40, 40, 11), (2, 250, 17)]:
        assert score(m, n) == pytest.approx(score(m + s, n + s), rel=1e-10, abs=1e-10)
    assert abs(score(10, 3) - score(3, 10)) > 1e-6   # but not symmetric in (m, n)


# ---------------------------------------------------------------- attention
def test_attention_matches_torch_sdpa_and_rows_sum_to_one():
    rng = np.random.default_rng(6)
    L, H, hd = 11, 3, 16
    q, k, v = (rng.normal(size=(L, H, hd)) for _ in range(3))
    o, p = vo.causal_attention(q, k, v, np.arange(L), np.arange(L), return_probs=True)
    t = lambda a: torch.from_numpy(np.transpose(a, (1, 0, 2)))[None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=True)
    np.testing.assert_allclose(o, np.transpose(ref[0].numpy(), (1, 0, 2)), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=0, atol=1e-14)
    assert np.all(p[:, np.arange(L)[:, None] < np.arange(L)[None, :]] == 0)
    np.testing.assert_allclose(o[0], v[0], rtol=1e-14)          # first query sees only key 0


def test_attention_with_cached_keys_equals_slice_of_full():
    rng = np.random.default_rng(7)
    L, H, hd = 9, 2, 8
    q, k, v = (rng.normal(size=(L, H, hd)) for _ in range(3))
    full = vo.causal_attention(q, k, v, np.arange(L), np.arange(L))
    tail = vo.causal_attention(q[6:], k, v, np.arange(6, L), np.arange(L))
    np.testing.assert_allclose(tail, full[6:], rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------- whole decoder vs a library
def _hf_model(cfg, w):
    transformers = pytest.importorskip("transformers")
    hc = transformers.LlamaConfig(
        vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.d_ffn,
        num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
        num_key_value_heads=cfg.n_heads, rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_base,
        max_position_embeddings=512, attention_bias=False, mlp_bias=False, tie_word_embeddings=False)
    hc._attn_implementation = "eager"
    m = transformers.LlamaForCausalLM(hc).double().eval()
    sd = {"model.embed_tokens.weight": w["embed"], "lm_head.weight": w["lm_head"],
          "model.norm.weight": w["final_norm"]}
    names = {"attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm",
             "wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "wgate": "mlp.gate_proj", "wup": "mlp.up_proj",
             "wdown": "mlp.down_proj"}
    for i, lw in enumerate(w["layers"]):
        for k, n in names.items():
            sd[f"model.layers.{i}.{n}.weight"] = lw[k]
    m.load_state_dict({k: v.double() for k, v in sd.items()}, strict=True)
    inv = m.model.rotary_emb.inv_freq.double()
    ref = torch.tensor([cfg.rope_base ** (-2 * i / cfg.head_dim) for i in range(cfg.head_dim // 2)],
                       dtype=torch.float64)
    torch.testing.assert_close(inv, ref, rtol=1e-6, atol=0)   # library uses the same RoPE frequencies
    return m


def test_decoder_matches_huggingface_llama(pin_setup):
    """The composed decoder equals transformers' LlamaForCausalLM on the same
    weights (its RMSNorm and RoPE run in fp32, hence the 1e-5 tolerance)."""
    w, inp = pin_setup
    m = _hf_model(PIN, w)
    got = oracle.prefill_logits(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, mode="ideal")
    a0 = PIN.action_begin
    for b in range(inp.batch):
        x0 = oracle.prefix_embeddings(PIN, vo.as_weights(w, PIN), inp.vis[b], inp.env_prompt(b))
        with torch.no_grad():
            ref = m(inputs_embeds=torch.from_numpy(x0)[None]).logits[0, -1, a0:].numpy()
        np.testing.assert_allclose(got[b], ref, rtol=0, atol=2e-5 * np.abs(ref).max())


def test_prompt_ids_equal_their_embedding_rows(pin_setup):
    w, inp = pin_setup
    W = vo.as_weights(w, PIN)
    ids = inp.env_prompt(0)
    vis_as_tokens = torch.cat([inp.vis[0], w["embed"][torch.as_tensor(ids[:2].astype(np.int64))]])
    a = oracle.forward_rows(PIN, W, oracle.prefix_embeddings(PIN, W, vis_as_tokens, ids[2:]))
    b = oracle.forward_rows(PIN, W, oracle.prefix_embeddings(PIN, W, inp.vis[0], ids))
    np.testing.assert_array_equal(a, b)


def test_zero_blocks_reduce_to_action_head_gemv():
    cfg = PIN.replace(batch=2)
    w = make_weights(cfg, seed=9)
    for lw in w["layers"]:
        lw["wo"].zero_(); lw["wdown"].zero_()
    inp = make_inputs(cfg, seed=9)
    z = oracle.prefill_logits(cfg, w, inp.vis, inp.prompt_ids, inp.prompt_lens, mode="ideal")
    for b in range(2):
        x_last = inp.vis[b, -1].double().numpy() if inp.prompt_lens[b] == 0 else \
            w["embed"][int(inp.env_prompt(b)[-1])].double().numpy()
        u = x_last / np.sqrt(np.mean(x_last ** 2) + cfg.rms_eps)
        ref = w["lm_head"][cfg.action_begin:].double().numpy() @ u
        np.testing.assert_allclose(z[b], ref, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- KV cache and batching
@pytest.mark.parametrize("mode", ["ideal", "bf16"])
def test_kv_cached_decode_equals_full_forward(pin_setup, mode):
    w, inp = pin_setup
    r = oracle.rollout(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, inp.gumbel, 1.5, mode=mode)
    tf = oracle.teacher_forced(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, r["tokens"], 1.5, mode=mode)
    np.testing.assert_allclose(r["logits"], tf["logits"], rtol=0, atol=1e-11)
    # PPO ratio of Eq. 2 is exactly 1 at theta = theta_old.
    np.testing.assert_allclose(np.exp(tf["logp_sum"] - r["logp_sum"]), 1.0, rtol=0, atol=1e-11)
    np.testing.assert_allclose(tf["entropy"], r["entropy"], rtol=0, atol=1e-11)


def test_environment_alone_equals_environment_in_ragged_batch(pin_setup):
    w, inp = pin_setup
    full = oracle.rollout(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, inp.gumbel, 1.0)
    b = 1
    one = oracle.rollout(PIN, w, inp.vis[b:b + 1], inp.env_prompt(b), inp.prompt_lens[b:b + 1],
                         inp.gumbel[b:b + 1], 1.0)
    np.testing.assert_array_equal(one["tokens"][0], full["tokens"][b])
    np.testing.assert_array_equal(one["logits"][0], full["logits"][b])


def test_contract_rounding_is_small_but_present(pin_setup):
    w, inp = pin_setup
    a = oracle.prefill_logits(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, mode="ideal")
    b = oracle.prefill_logits(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, mode="bf16")
    d = np.abs(a - b).max()
    assert 1e-6 < d < 3e-2


# ---------------------------------------------------------------- sampler and Eq. 1
def test_sampler_closed_forms():
    A = 256
    z = np.zeros(A)
    k, lp, ent, _ = vo.sample_bin(z, np.zeros(A), 1.5)
    assert k == 0                                   # exact tie -> lowest index
    assert lp == pytest.approx(-math.log(A), abs=1e-12) and ent == pytest.approx(math.log(A), abs=1e-12)
    rng = np.random.default_rng(8)
    z = rng.normal(size=A)
    assert vo.sample_bin(z, np.zeros(A), 1.0)[0] == int(np.argmax(z))     # g = 0 -> argmax
    g = np.zeros(A); g[17] = 100.0
    assert vo.sample_bin(z, g, 1.5)[0] == 17
    lps = np.array([vo.token_stats(z, j, 1.5)[0] for j in range(A)])
    assert np.exp(lps).sum() == pytest.approx(1.0, abs=1e-12)
    # log-probabilities are those of softmax(z / T): ratios follow exp((z_i - z_j)/T)
    assert lps[3] - lps[9] == pytest.approx((z[3] - z[9]) / 1.5, abs=1e-12)
    # entropy falls as temperature falls and tends to 0 for T -> 0
    assert vo.token_stats(z, 0, 0.5)[1] < vo.token_stats(z, 0, 1.5)[1]
    assert vo.token_stats(z, 0, 1e-3)[1] < 1e-6


def test_sampler_margin_is_the_top2_gap_of_the_scores():
    """The margin that decides which tokens are near-ties (Eq. 1 sampling at
    temperature T, Sec. 4.3): the gap between the two largest scores
    z_j / T + g_j, in float64.  Hand cases chosen so that dropping g, dropping
    T or taking the gap in float32 gives another value."""
    z = np.array([3.0, 1.5, 0.0, -2.0])
    g = np.array([0.0, 1.2, 0.5, 0.0])
    # scores z/T + g at T = 1.5: [2.0, 2.2, 0.5, -4/3] -> bin 1, gap 0.2
    # (without g: [2, 1, 0, -4/3], gap 1; without T: [3, 2.7, 0.5, -2], gap 0.3)
    k, _, _, margin = vo.sample_bin(z, g, 1.5)
    assert k == 1 and margin == pytest.approx(0.2, abs=1e-15)
    # a gap of 3e-9 at scores near 0.1 is below float32's spacing there (7.5e-9):
    # a float32 margin would be 0 or 7.5e-9
    z = np.array([0.1, 0.1 + 3e-9, -1.0])
    margin = vo.sample_bin(z, np.zeros(3), 1.0)[3]
    assert margin == pytest.approx(3e-9, abs=1e-16)
    # at an exact tie of the scores the margin is 0 and the lowest bin wins
    k, _, _, margin = vo.sample_bin(np.array([0.5, 1.0, 0.0]), np.array([0.5, 0.0, 0.2]), 1.0)
    assert k == 0 and margin == 0.0


def test_gumbel_max_frequencies_follow_softmax():
    """Chi-square test: Gumbel-max with the generator's noise draws bins with
    probability softmax(z / T)."""
    scipy_stats = pytest.importorskip("scipy.stats")
    A, T, n = 256, 1.5, 14000 * 7
    rng = np.random.default_rng(10)
    z = rng.normal(size=A) * 1.3
    g = gumbel_noise(PIN, 14000, seed=11).reshape(n, A)
    counts = np.bincount([vo.sample_bin(z, g[i], T)[0] for i in range(n)], minlength=A)
    p = np.exp(z / T - np.max(z / T)); p /= p.sum()
    exp = n * p
    keep = exp >= 5
    obs, ex = counts[keep], exp[keep]
    if not keep.all():                                  # pool the rare bins into one cell
        obs, ex = np.append(obs, counts[~keep].sum()), np.append(ex, exp[~keep].sum())
    assert scipy_stats.chisquare(obs, ex).pvalue > 1e-4


def test_eq1_joint_distribution_normalises_by_enumeration():
    """With 2 action bins and 7 tokens, the exp of Eq. 1's sum of token
    log-probs over all 2^7 action sequences must add to 1: the token
    log-probs are proper auto-regressive conditionals."""
    cfg = PIN.replace(action_bins=2, batch=1)
    w = make_weights(cfg, seed=12)
    inp = make_inputs(cfg, seed=12)
    W = vo.as_weights(w, cfg)
    total = 0.0
    for code in range(2 ** cfg.n_actions):
        acts = [cfg.action_begin + ((code >> i) & 1) for i in range(cfg.n_actions)]
        r = vo.teacher_forced_env(cfg, W, inp.vis[0], inp.env_prompt(0), acts, 1.5, "ideal")
        total += math.exp(r["logp"].sum())
    assert total == pytest.approx(1.0, abs=1e-12)


def test_rollout_outputs_are_action_tokens_and_consistent(pin_setup):
    w, inp = pin_setup
    r = oracle.rollout(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, inp.gumbel, 1.5)
    assert r["tokens"].shape == (inp.batch, PIN.n_actions)
    assert np.all((r["tokens"] >= PIN.action_begin) & (r["tokens"] < PIN.vocab))
    np.testing.assert_allclose(r["logp_sum"], r["logp"].sum(1), rtol=1e-14)
    assert np.all(r["logp"] < 0) and np.all(r["entropy"] > 0) and np.all(r["margin"] >= 0)
    # each token is the Gumbel-max choice of the logits at its step
    for b in range(inp.batch):
        for i in range(PIN.n_actions):
            s = r["logits"][b, i] / 1.5 + inp.gumbel[b, i]
            assert r["tokens"][b, i] - PIN.action_begin == int(np.argmax(s))


# ---------------------------------------------------------------------------
# LoRA merge (Sec. 3.3, Rollout Phase)
# ---------------------------------------------------------------------------
def _bf16(x):
    return torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)


def test_lora_merge_zero_update_returns_the_checkpoint_exactly():
    g = torch.Generator().manual_seed(21)
    w0 = (torch.randn(48, 80, generator=g) * 0.02).to(torch.bfloat16)
    a = (torch.randn(8, 80, generator=g) * 0.02).to(torch.bfloat16)
    b = torch.zeros(48, 8, dtype=torch.bfloat16)
    m = oracle.lora_merge(w0, a, b, 0.5)
    assert np.array_equal(m, w0.double().numpy())


def test_lora_merge_exact_rank_one_case():
    """Rank 1 with values whose products and sums are exact in bf16:
    W0 = 1/2 everywhere, B = [0, 1/8, 1/4, ...] (column), A = [1, 2, 4, ...]
    (row), scale 2 -> W[i, j] = 1/2 + 2 * (i/8) * 2^j."""
    rows, cols = 6, 5
    w0 = _bf16(np.full((rows, cols), 0.5))
    b = _bf16(np.arange(rows)[:, None] / 8.0)
    a = _bf16(2.0 ** np.arange(cols)[None, :])
    expect = 0.5 + 2.0 * (np.arange(rows)[:, None] / 8.0) * (2.0 ** np.arange(cols)[None, :])
    assert np.array_equal(oracle.lora_merge(w0, a, b, 2.0), expect)


def test_lora_merge_rounds_to_nearest_even():
    """1 + 2^-8 lies halfway between the bf16 neighbours 1 and 1 + 2^-7: the
    even one (1) wins; 1 + 3 * 2^-8 rounds up to the even 1 + 2^-6."""
    w0 = _bf16([[1.0, 1.0]])
    a = _bf16([[1.0, 3.0]])
    b = _bf16([[2.0 ** -8]])
    assert np.array_equal(oracle.lora_merge(w0, a, b, 1.0), [[1.0, 1.0 + 2.0 ** -6]])


def test_lora_merge_matches_the_unmerged_lora_forward():
    """The merged layer applied to inputs equals the LoRA forward pass
    x W0^T + scale (x A^T) B^T up to the bf16 rounding of the merged weights
    (relative error <= 2^-9 per element): catches a transposed product, a wrong
    scale or sign, or factors used in the wrong order."""
    g = torch.Generator().manual_seed(22)
    out_f, in_f, r, scale = 96, 160, 16, 0.75
    w0 = (torch.randn(out_f, in_f, generator=g) * 0.02).to(torch.bfloat16)
    a = (torch.randn(r, in_f, generator=g) * 0.05).to(torch.bfloat16)
    b = (torch.randn(out_f, r, generator=g) * 0.05).to(torch.bfloat16)
    x = torch.randn(7, in_f, generator=g, dtype=torch.float64)
    merged = torch.from_numpy(oracle.lora_merge(w0, a, b, scale))
    lora = torch.nn.functional.linear(x, w0.double()) + scale * torch.nn.functional.linear(
        torch.nn.functional.linear(x, a.double()), b.double())
    got = torch.nn.functional.linear(x, merged)
    exact_w = w0.double() + scale * (b.double() @ a.double())
    bound = 2.0 ** -9 * (x.abs() @ exact_w.abs().t()) + 1e-12
    assert bool(((got - lora).abs() <= bound).all())
    # and the update is really there: dropping it is far outside the bound
    assert bool(((torch.nn.functional.linear(x, w0.double()) - lora).abs() > bound).any())


def test_merge_weights_touches_only_the_adapted_projections():
    from paper_2505_18719_amd.inputs import make_lora
    w = make_weights(PIN, seed=23)
    ad = make_lora(PIN, 4, seed=23, layers=[1])
    m = oracle.merge_weights(w, ad, 0.5, layers=[1])
    for li, lw in enumerate(w["layers"]):
        for k, t in lw.items():
            same = torch.equal(m["layers"][li][k], t)
            assert same == (li != 1 or k.endswith("norm")), (li, k)
    assert torch.equal(m["embed"], w["embed"]) and torch.equal(m["lm_head"], w["lm_head"])


# ---------------------------------------------------------------------------
# Value model (Alg. 1: V_t <- V(o_t, v_in); a value model of the policy's own
# architecture, Fig. 2)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("mode", ["ideal", "bf16"])
def test_value_with_an_action_row_as_head_is_that_action_logit(pin_setup, mode):
    """The value head and the action head read the same final-normed hidden
    state of the last prefix row: with row k of the LM head's action rows as
    the value head, the value is exactly the prefill's action logit k."""
    w, inp = pin_setup
    z = oracle.prefill_logits(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, mode=mode)
    for k in (0, 3, PIN.action_bins - 1):
        v = oracle.values(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens,
                          w["lm_head"][PIN.action_begin + k], mode=mode)
        np.testing.assert_allclose(v, z[:, k], rtol=0, atol=1e-13)


def test_value_zero_blocks_reduce_to_a_dot_product():
    """With W_o = W_down = 0 every layer is the identity: the value is the
    head dotted with the RMS-normalised last prefix embedding."""
    cfg = PIN.replace(batch=2)
    w = make_weights(cfg, seed=19)
    for lw in w["layers"]:
        lw["wo"].zero_(); lw["wdown"].zero_()
    inp = make_inputs(cfg, seed=19)
    head = torch.linspace(-1, 1, cfg.d_model).to(torch.bfloat16)
    v = oracle.values(cfg, w, inp.vis, inp.prompt_ids, inp.prompt_lens, head, mode="ideal")
    for b in range(2):
        x_last = inp.vis[b, -1].double().numpy() if inp.prompt_lens[b] == 0 else \
            w["embed"][int(inp.env_prompt(b)[-1])].double().numpy()
        u = x_last / np.sqrt(np.mean(x_last ** 2) + cfg.rms_eps)
        assert v[b] == pytest.approx(float(head.double().numpy() @ u), rel=1e-12, abs=1e-12)


def test_value_is_linear_in_the_head(pin_setup):
    w, inp = pin_setup
    g = torch.Generator().manual_seed(31)
    h1 = (torch.randn(PIN.d_model, generator=g) * 0.02).to(torch.bfloat16)
    h2 = (torch.randn(PIN.d_model, generator=g) * 0.02).to(torch.bfloat16)
    v1 = oracle.values(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, h1, mode="ideal")
    v2 = oracle.values(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, h2, mode="ideal")
    v12 = oracle.values(PIN, w, inp.vis, inp.prompt_ids, inp.prompt_lens, h1.double() + h2.double(), mode="ideal")
    np.testing.assert_allclose(v12, v1 + v2, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------------------
# learning phase: GAE (Alg. 1), PPO-clip (Eq. 2 with Eq. 1), log-prob gradient
# ---------------------------------------------------------------------------
from oracle import learn_oracle as lo  # noqa: E402


def test_gae_worked_example_by_hand():
    """M = 3, one environment, gamma = lambda = 1/2; d_2 = 1 ends the episode
    between steps 1 and 2.  By hand: delta = (0.625, -0.25, 3),
    A = (0.5625, -0.25, 3), returns A + V = (1.0625, 0, 4)."""
    r = np.array([[1.0], [0.0], [2.0]])
    v = np.array([[0.5], [0.25], [1.0], [4.0]])
    d = np.array([[0], [0], [1], [0]], dtype=np.uint8)
    adv, ret = lo.gae(r, v, d, 0.5, 0.5)
    assert np.array_equal(adv[:, 0], [0.5625, -0.25, 3.0])
    assert np.array_equal(ret[:, 0], [1.0625, 0.0, 4.0])


def _gae_inputs(M, N, seed, p_done=0.1):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=(M, N)), rng.normal(size=(M + 1, N)),
            (rng.random((M + 1, N)) < p_done).astype(np.uint8))


def test_gae_equals_the_explicit_discounted_sum_of_td_residuals():
    """GAE's definition: A_t = sum_l (gamma lambda)^l delta_{t+l}, the sum cut
    at the first episode end after t, by brute force over every (t, l)."""
    M, N, g, lam = 23, 5, 0.97, 0.9
    r, v, d = _gae_inputs(M, N, 1, p_done=0.15)
    adv, _ = lo.gae(r, v, d, g, lam)
    for n in range(N):
        for t in range(M):
            total, w = 0.0, 1.0
            for s in range(t, M):
                nonterminal = 1.0 - d[s + 1, n]
                delta = r[s, n] + g * v[s + 1, n] * nonterminal - v[s, n]
                total += w * delta
                if nonterminal == 0.0:
                    break
                w *= g * lam
            assert abs(adv[t, n] - total) <= 1e-12 * max(1.0, abs(total)), (t, n)


def test_gae_lambda_one_is_the_bootstrapped_discounted_return():
    """lambda = 1, no episode end: A_t + V_t = sum_{s >= t} gamma^(s-t) r_s + gamma^(M-t) V_M."""
    M, N, g = 17, 3, 0.9
    r, v, _ = _gae_inputs(M, N, 2)
    d = np.zeros((M + 1, N), dtype=np.uint8)
    _, ret = lo.gae(r, v, d, g, 1.0)
    for t in range(M):
        want = sum(g ** (s - t) * r[s] for s in range(t, M)) + g ** (M - t) * v[M]
        assert np.allclose(ret[t], want, rtol=1e-12, atol=1e-12)


def test_gae_special_cases():
    M, N, g = 9, 4, 0.95
    r, v, d = _gae_inputs(M, N, 3, p_done=0.3)
    adv0, _ = lo.gae(r, v, d, g, 0.0)          # lambda = 0: one-step TD residual
    cont = 1.0 - d[1:].astype(np.float64)
    assert np.allclose(adv0, r + g * cont * v[1:] - v[:M], rtol=0, atol=1e-14)
    advg, _ = lo.gae(r, v, d, 0.0, 0.7)        # gamma = 0: r_t - V_t
    assert np.allclose(advg, r - v[:M], rtol=0, atol=1e-14)
    ones = np.ones((M + 1, N), dtype=np.uint8)  # every step ends an episode
    adv1, _ = lo.gae(r, v, ones, g, 0.9)
    assert np.allclose(adv1, r - v[:M], rtol=0, atol=1e-14)


def test_ppo_clip_hand_cases():
    """eps = 0.2, one token per action (n = 4):
    rho 1.5, A +1 -> clipped term 1.2, no gradient;
    rho 0.9, A -2 -> -1.8, d loss / d logp = -rho A / n = 0.45;
    rho 0.5, A -1 -> clipped term -0.8, no gradient;
    rho 2.0, A -1 -> -2.0 (the unclipped term is the smaller), gradient 0.5.
    J = (1.2 - 1.8 - 0.8 - 2.0) / 4 = -0.85."""
    rho = np.array([1.5, 0.9, 0.5, 2.0])
    a = np.array([1.0, -2.0, -1.0, -1.0])
    loss, frac, g = lo.ppo_clip(np.log(rho)[:, None], np.zeros((4, 1)), a, 0.2)
    assert abs(loss - 0.85) < 1e-12 and frac == 0.5
    assert np.allclose(g[:, 0], [0.0, 0.45, 0.0, 0.5], rtol=0, atol=1e-12)


def test_ppo_ratio_one_at_the_old_policy():
    """theta = theta_old: rho = 1, nothing is clipped, J = mean A and the
    gradient of every token is -A / n (Eq. 2's ratio is 1 at the old policy)."""
    rng = np.random.default_rng(4)
    lp = -rng.random((50, 7)) * 8
    a = rng.normal(size=50)
    loss, frac, g = lo.ppo_clip(lp, lp, a, 0.2)
    assert abs(loss + a.mean()) < 1e-14 and frac == 0.0
    assert np.allclose(g, np.repeat(-a[:, None] / 50, 7, axis=1), rtol=0, atol=1e-15)


def test_ppo_gradient_matches_finite_differences():
    rng = np.random.default_rng(5)
    n, k, eps = 12, 7, 0.2
    lo_ = -rng.random((n, k)) * 6
    ln = lo_ + rng.normal(scale=0.15, size=(n, k))
    a = rng.normal(size=n)
    rho = np.exp(ln.sum(1) - lo_.sum(1))
    assert np.all(np.minimum(abs(rho - 1.2), abs(rho - 0.8)) > 1e-3)  # away from the kinks
    _, _, g = lo.ppo_clip(ln, lo_, a, eps)
    h = 1e-6
    for t in range(n):
        for i in (0, k - 1):
            up, dn = ln.copy(), ln.copy()
            up[t, i] += h
            dn[t, i] -= h
            fd = (lo.ppo_clip(up, lo_, a, eps)[0] - lo.ppo_clip(dn, lo_, a, eps)[0]) / (2 * h)
            assert abs(fd - g[t, i]) < 1e-8, (t, i)
    assert 0 < (g == 0).all(axis=1).sum() < n  # both branches were exercised


def test_logprob_grad_matches_finite_differences_of_the_token_logprob():
    """Against finite differences of the rollout oracle's own log-prob
    (token_stats), which shares no code with logprob_grad."""
    rng = np.random.default_rng(6)
    bins, T, begin = 256, 1.5, 1000
    z = rng.normal(scale=1.5, size=(3, bins))
    tok = begin + np.array([0, 77, 255])
    dl = np.array([0.7, -1.3, 2.0])
    dz = lo.logprob_grad(z, tok, begin, T, dl)
    h = 1e-6
    for r in range(3):
        for j in (0, 5, int(tok[r] - begin), 255):
            up, dn = z[r].copy(), z[r].copy()
            up[j] += h
            dn[j] -= h
            fd = (vo.token_stats(up, int(tok[r] - begin), T)[0] - vo.token_stats(dn, int(tok[r] - begin), T)[0]) / (2 * h)
            assert abs(dl[r] * fd - dz[r, j]) < 1e-8, (r, j)
    assert np.allclose(dz.sum(axis=1), 0.0, atol=1e-14)  # softmax rows sum to one


def test_logprob_grad_uniform_logits_closed_form():
    bins, T = 256, 1.5
    dz = lo.logprob_grad(np.full((1, bins), 0.3), [42], 0, T, [2.0])
    want = np.full(bins, -2.0 / (T * bins))
    want[42] += 2.0 / T
    assert np.allclose(dz[0], want, rtol=0, atol=1e-15)


# ---------------------------------------------------------------------------
# action extraction f (Alg. 1): action tokens -> continuous action
# ---------------------------------------------------------------------------
def test_extract_actions_hand_values():
    """4 bins over [-1, 1] have centres -0.75, -0.25, 0.25, 0.75; over [0, 2]
    the centres shift by 1; a token outside the bins gives NaN."""
    a = oracle.extract_actions([[10, 13, 11], [12, 9, 14]], 10, 4, [-1, 0, -1], [1, 2, 1])
    assert np.array_equal(a[0], [-0.75, 1.75, -0.25])
    assert a[1, 0] == 0.25 and np.isnan(a[1, 1]) and np.isnan(a[1, 2])


def test_extract_actions_inverts_an_independent_discretiser():
    """Discretise random continuous actions into 256 uniform bins per
    dimension (floor of the scaled offset); the extracted action is the
    centre of the bin the value fell in, so within half a bin width of it."""
    rng = np.random.default_rng(7)
    lo = rng.uniform(-2, 0, size=7)
    hi = lo + rng.uniform(0.1, 3, size=7)
    x = lo + rng.random((500, 7)) * (hi - lo)
    w = (hi - lo) / 256
    k = np.minimum(np.floor((x - lo) / w), 255).astype(np.int64)
    a = oracle.extract_actions(k + 31808, 31808, 256, lo, hi)
    assert np.all(np.abs(a - x) <= w / 2 + 1e-12)
    assert np.all((a > lo + k * w) & (a < lo + (k + 1) * w))
    centres = oracle.extract_actions(np.arange(256)[:, None] + np.zeros((1, 7), int), 0, 256, lo, hi)
    assert np.all(np.diff(centres, axis=0) > 0)
    assert np.allclose(centres.mean(axis=0), (lo + hi) / 2, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# backward of the teacher-forced pass: LoRA gradients of the PPO-clip loss
# ---------------------------------------------------------------------------
from paper_2505_18719_amd.inputs import VlaConfig, make_lora  # noqa: E402

BWD_CFG = VlaConfig("bwd_pin", n_layers=2, d_model=32, n_heads=2, d_ffn=48, vocab=80, action_bins=16,
                    n_actions=3, n_visual=4, batch=3, prompt_min=0, prompt_max=5)


def _bwd_setup(seed=0):
    cfg = BWD_CFG
    w = make_weights(cfg, seed=seed, device="cpu")
    inp = make_inputs(cfg, seed=seed, prompt_lens=[2, 5, 0])
    ad = make_lora(cfg, 4, seed=seed, device="cpu", std=0.2)
    rng = np.random.default_rng(seed)
    acts = cfg.action_begin + rng.integers(0, cfg.action_bins, size=(cfg.batch, cfg.n_actions))
    adv = rng.normal(size=cfg.batch)
    return cfg, w, inp, ad, acts, adv


def _fd_loss(cfg, w, inp, ad, s, acts, logp_old, adv, eps, T):
    """The loss from the forward oracle on fp64-merged weights (no backward code)."""
    w2 = dict(w)
    w2["layers"] = [{k: torch.from_numpy(v) for k, v in lw.items()} for lw in lo.merged_layers(w, ad, s)]
    logp = oracle.teacher_forced(cfg, w2, inp.vis, inp.prompt_ids, inp.prompt_lens, acts, T, mode="ideal")["logp"]
    return lo.ppo_clip(logp, logp_old, adv, eps)[0]


def test_lora_grads_match_central_differences_of_the_forward_oracle():
    """Every projection of both layers, both factors: the analytic gradient of
    -J (Eq. 2 through the teacher-forced pass) against central differences of
    the loss computed by the forward oracle alone; one action clipped."""
    cfg, w, inp, ad, acts, adv = _bwd_setup()
    s, eps, T = 0.5, 0.2, 1.5
    ad = [{k: (lo.vo.to_f64(a), lo.vo.to_f64(b)) for k, (a, b) in layer.items()} for layer in ad]
    base = lo.ppo_lora_grads(cfg, w, ad, s, inp.vis, inp.prompt_ids, inp.prompt_lens, acts,
                             np.zeros((cfg.batch, cfg.n_actions)), adv, eps, T)
    rng = np.random.default_rng(1)
    logp_old = base["logp"] + rng.normal(scale=0.02, size=base["logp"].shape)
    logp_old[0] -= 0.2 if adv[0] > 0 else -0.2     # action 0 beyond the clip edge on its side
    res = lo.ppo_lora_grads(cfg, w, ad, s, inp.vis, inp.prompt_ids, inp.prompt_lens, acts, logp_old, adv, eps, T)
    assert res["clip_frac"] == 1.0 / cfg.batch
    assert abs(res["loss"] - _fd_loss(cfg, w, inp, ad, s, acts, logp_old, adv, eps, T)) < 1e-12
    h, worst = 1e-5, 0.0
    for li in range(cfg.n_layers):
        for k in lo.PROJ:
            for f in (0, 1):  # A, then B
                g = res["grads"][li][k][f]
                scale_g = max(np.abs(g).max(), 1e-12)
                for idx in [tuple(rng.integers(0, n) for n in g.shape) for _ in range(2)]:
                    pert = [{kk: (a.copy(), b.copy()) for kk, (a, b) in layer.items()} for layer in ad]
                    pert[li][k][f][idx] += h
                    up = _fd_loss(cfg, w, inp, pert, s, acts, logp_old, adv, eps, T)
                    pert[li][k][f][idx] -= 2 * h
                    dn = _fd_loss(cfg, w, inp, pert, s, acts, logp_old, adv, eps, T)
                    fd = (up - dn) / (2 * h)
                    worst = max(worst, abs(fd - g[idx]) / scale_g)
                    assert abs(fd - g[idx]) <= 1e-6 * scale_g + 1e-10, (li, k, f, idx, fd, g[idx])
    assert worst < 1e-6


def test_lora_grads_ratio_one_is_the_policy_gradient():
    """At theta = theta_old (logp_old = logp_new) nothing is clipped and the
    gradient is -(1/n) sum_b A_b grad log pi(a_b): with one unit advantage on
    one action and zeros elsewhere it is -(1/n) times that action's
    log-probability gradient, which is linear in the advantages."""
    cfg, w, inp, ad, acts, adv = _bwd_setup(seed=2)
    s, eps, T = 0.5, 0.2, 1.5
    zero = np.zeros((cfg.batch, cfg.n_actions))
    lp = lo.ppo_lora_grads(cfg, w, ad, s, inp.vis, inp.prompt_ids, inp.prompt_lens, acts, zero, adv, eps, T)["logp"]
    full = lo.ppo_lora_grads(cfg, w, ad, s, inp.vis, inp.prompt_ids, inp.prompt_lens, acts, lp, adv, eps, T)
    assert full["clip_frac"] == 0.0 and abs(full["loss"] + adv.mean()) < 1e-12
    parts = []
    for b in range(cfg.batch):
        e = np.zeros(cfg.batch)
        e[b] = adv[b]
        parts.append(lo.ppo_lora_grads(cfg, w, ad, s, inp.vis, inp.prompt_ids, inp.prompt_lens, acts, lp, e, eps,
                                       T)["grads"])
    for li in range(cfg.n_layers):
        for k in lo.PROJ:
            for f in (0, 1):
                tot = sum(p[li][k][f] for p in parts)
                assert np.allclose(full["grads"][li][k][f], tot, rtol=1e-10, atol=1e-14)
