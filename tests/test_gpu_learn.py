"""Parity of the learning-phase kernels (vla_learn.h) with the CPU oracle:
GAE over a rollout window (Alg. 1), the PPO-clip objective of Eq. 2 with its
token gradient, and the gradient of the token log-probabilities w.r.t. the
action logits, also chained onto a teacher-forced pass of the decoder."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, log
from oracle import learn_oracle as lo
from paper_2505_18719_amd import inputs, vla

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24  # unit roundoff of fp32


def _gae_bound(r, v, d, gamma, lam, adv_ref):
    """Per-element bound on |A_gpu - A_exact|: each step's rounding (a few
    units of the magnitudes it touches) is carried back with weight
    (gamma lam)^l, plus the rounding of chaining the 16 slice maps."""
    M = r.shape[0]
    cont = 1.0 - d[1:].astype(np.float64)
    mag = np.abs(r) + np.abs(v[:M]) + np.abs(v[1:]) + np.abs(adv_ref)
    S = np.zeros_like(mag)
    nxt = np.zeros(mag.shape[1])
    for t in range(M - 1, -1, -1):
        nxt = mag[t] + gamma * lam * cont[t] * nxt
        S[t] = nxt
    return 8 * U32 * S + 4 * U32 * (M / 16 + 2) * np.abs(adv_ref).max()


def _run_gae(N, M, gamma, lam, seed=0, p_done=0.01, returns=True):
    r, v, d = inputs.rollout_window(N, M, seed=seed, p_done=p_done)
    dev = [torch.from_numpy(x).cuda() for x in (r, v, d)]
    adv, ret = vla.gae(*dev, gamma, lam)
    torch.cuda.synchronize()
    a_ref, ret_ref = lo.gae(r, v, d, gamma, lam)
    return r, v, d, adv.cpu().numpy(), ret.cpu().numpy(), a_ref, ret_ref


@pytest.mark.parametrize("N,M,p_done", [(64, 512, 0.01), (70, 37, 0.2), (3, 1, 0.0), (130, 5, 0.3),
                                        (4096, 128, 0.02)])
def test_gae_matches_oracle(N, M, p_done):
    gamma, lam = 0.99, 0.95
    r, v, d, adv, ret, a_ref, ret_ref = _run_gae(N, M, gamma, lam, seed=N + M, p_done=p_done)
    bound = _gae_bound(r, v, d, gamma, lam, a_ref)
    err = np.abs(adv - a_ref)
    log(f"[gae N={N} M={M}] max|dA|={err.max():.3e} (worst err/bound {np.max(err / bound):.3f})")
    assert np.all(err <= bound)
    assert np.all(np.abs(ret - ret_ref) <= bound + 2 * U32 * np.abs(ret_ref))


def test_gae_every_step_terminal_is_exact():
    """d_{t+1} = 1 everywhere: A_t = r_t - V_t, one fp32 rounding of the exact difference."""
    N, M = 64, 40
    r, v, _ = inputs.rollout_window(N, M, seed=1)
    d = np.ones((M + 1, N), dtype=np.uint8)
    adv, _ = vla.gae(torch.from_numpy(r).cuda(), torch.from_numpy(v).cuda(), torch.from_numpy(d).cuda(), 0.99, 0.95)
    want = (r.astype(np.float64) - v[:M]).astype(np.float32)
    assert np.array_equal(adv.cpu().numpy(), want)


def test_gae_special_parameters_and_null_returns():
    N, M = 65, 50
    r, v, d = inputs.rollout_window(N, M, seed=2, p_done=0.1)
    dev = [torch.from_numpy(x).cuda() for x in (r, v, d)]
    for gamma, lam in ((0.9, 0.0), (0.0, 0.7), (1.0, 1.0)):
        adv = torch.empty(M, N, device="cuda")
        lib = vla.load_library()
        vla._check(lib.vla_gae(N, M, vla._ptr(dev[0]), vla._ptr(dev[1]), vla._ptr(dev[2]), gamma, lam,
                               vla._ptr(adv), None, vla._stream(adv.device)))
        torch.cuda.synchronize()
        a_ref, _ = lo.gae(r, v, d, gamma, lam)
        assert np.all(np.abs(adv.cpu().numpy() - a_ref) <= _gae_bound(r, v, d, gamma, lam, a_ref)), (gamma, lam)


def _ppo_check(n, k, eps, seed, spread=0.1, adv_zero_frac=0.0):
    old, new, adv = inputs.ppo_minibatch(n, k, seed=seed, spread=spread)
    if adv_zero_frac:
        adv[: int(n * adv_zero_frac)] = 0.0
    dev = [torch.from_numpy(x).cuda() for x in (new, old, adv)]
    stats, g = vla.ppo_clip(*dev, eps)
    stats2, g2 = vla.ppo_clip(*dev, eps)
    torch.cuda.synchronize()
    assert torch.equal(stats, stats2) and torch.equal(g, g2)  # fixed reduction order
    loss_ref, frac_ref, g_ref = lo.ppo_clip(new, old, adv, eps)
    # the kernel sums k fp32 log-probs per side: the ratio's relative error
    abs_sum = np.abs(new.astype(np.float64)).sum(1) + np.abs(old.astype(np.float64)).sum(1)
    drho = (k + 2) * U32 * abs_sum + 4 * U32
    rho = np.exp(new.astype(np.float64).sum(1) - old.astype(np.float64).sum(1))
    margin = np.minimum(np.abs(rho - (1 + eps)), np.abs(rho - (1 - eps))) / rho
    sure = margin > 4 * drho
    gg, ga = g.cpu().numpy(), stats.cpu().numpy()
    # unambiguous actions: the oracle's gradient within the ratio's error
    tol = (drho[:, None] + 4 * U32) * np.abs(rho * adv)[:, None] / n
    assert np.all(np.abs(gg - g_ref)[sure] <= tol[sure])
    # near a clipping edge either branch is correct
    for t in np.where(~sure)[0]:
        assert np.all(gg[t] == 0) or np.allclose(gg[t], -rho[t] * adv[t] / n, rtol=10 * drho[t], atol=0)
    assert np.all(gg == gg[:, :1])  # every token of an action gets the same gradient (Eq. 1)
    surr_mag = np.abs(rho * adv).mean()
    assert abs(ga[0] - loss_ref) <= (np.max(drho) + (n / 1024 + 16) * U32) * surr_mag * 2 + 1e-12
    assert abs(ga[1] - frac_ref) <= (~sure).sum() / n + 1e-7
    log(f"[ppo n={n} k={k}] loss {ga[0]:.6f} vs {loss_ref:.6f}, clipped {ga[1]:.4f}, ambiguous {(~sure).sum()}")
    return ga, gg


@pytest.mark.parametrize("n,k,spread", [(128, 7, 0.1), (5000, 7, 0.05), (1, 1, 0.3), (1031, 16, 0.05)])
def test_ppo_clip_matches_oracle(n, k, spread):
    _ppo_check(n, k, 0.2, seed=n + k, spread=spread, adv_zero_frac=0.01)


def test_ppo_ratio_one_at_the_old_policy():
    """logp_new == logp_old: rho = 1 exactly, nothing clipped, loss = -mean A
    and every token's gradient is -A / n (one fp32 rounding)."""
    n, k = 300, 7
    old, _, adv = inputs.ppo_minibatch(n, k, seed=9)
    o, a = torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda()
    stats, g = vla.ppo_clip(o, o.clone(), a, 0.2)
    torch.cuda.synchronize()
    s = stats.cpu().numpy()
    assert s[1] == 0.0
    assert abs(s[0] + adv.astype(np.float64).mean()) <= 20 * U32 * np.abs(adv).mean()
    want = (-adv.astype(np.float64) / n).astype(np.float32)
    assert np.array_equal(g.cpu().numpy(), np.repeat(want[:, None], k, axis=1))


def _bwd_check(rows, bins, T, seed, bad_row=None):
    rng = np.random.default_rng(seed)
    begin = 31808 if bins == 256 else 1000
    z = rng.normal(scale=1.5, size=(rows, bins)).astype(np.float32)
    tok = (begin + rng.integers(0, bins, size=rows)).astype(np.int32)
    if bad_row is not None:
        tok[bad_row] = begin - 1
    dl = rng.normal(size=rows).astype(np.float32)
    dz = vla.logprob_backward(torch.from_numpy(z).cuda(), torch.from_numpy(tok).cuda(), begin, T,
                              torch.from_numpy(dl).cuda())
    torch.cuda.synchronize()
    got = dz.cpu().numpy()
    ok = np.ones(rows, bool)
    if bad_row is not None:
        assert np.all(np.isnan(got[bad_row]))
        ok[bad_row] = False
        tok[bad_row] = begin
    ref = lo.logprob_grad(z, tok, begin, T, dl)
    # p_j carries the rounding of z / T and of exp (a few units each, relative to p_j)
    tol = 32 * U32 * (np.abs(dl)[:, None] / T + np.abs(ref))
    err = np.abs(got - ref)
    assert np.all(err[ok] <= tol[ok]), float(np.max(err[ok] / tol[ok]))
    log(f"[logprob bwd rows={rows} bins={bins}] max|d dz|={err[ok].max():.3e}")


@pytest.mark.parametrize("rows,bins", [(896, 256), (5, 100), (1, 1), (3, 255)])
def test_logprob_backward_matches_oracle(rows, bins):
    _bwd_check(rows, bins, 1.5, seed=rows + bins)


def test_logprob_backward_out_of_range_token_gives_a_nan_row():
    _bwd_check(9, 256, 1.0, seed=3, bad_row=4)


def test_ppo_chain_on_a_teacher_forced_pass():
    """Rollout (old log-probs), teacher-forced pass of the same tokens under
    the same weights (new log-probs and logits), PPO-clip, then the logits
    gradient -- each step against the oracle fed the GPU's own inputs; the
    ratio is 1 up to the two passes' rounding (Eq. 2 at theta = theta_old)."""
    S = Setup(inputs.TINY, seed=11)
    cfg, T = S.cfg, 1.5
    inp, dev = S.inputs(seed=11)
    B = inp.batch
    S.model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
    out = S.model.decode_actions(dev["gumbel"], T)
    tf = S.model.token_logprobs(dev["vis"], dev["ids"], inp.prompt_lens, out["tokens"], T)
    torch.cuda.synchronize()
    adv = torch.from_numpy(inputs.ppo_minibatch(B, seed=11)[2]).cuda()
    stats, g = vla.ppo_clip(tf["logp"].contiguous(), out["logp"].contiguous(), adv, 0.2)
    dz = vla.logprob_backward(tf["logits"].reshape(B * cfg.n_actions, cfg.action_bins).contiguous(),
                              out["tokens"].reshape(-1).contiguous(), cfg.action_begin, T,
                              g.reshape(-1).contiguous())
    torch.cuda.synchronize()
    ln, lo_, a = tf["logp"].cpu().numpy(), out["logp"].cpu().numpy(), adv.cpu().numpy()
    assert np.max(np.abs(ln - lo_)) < 1e-2  # same weights: the ratio is ~1
    loss_ref, frac_ref, g_ref = lo.ppo_clip(ln, lo_, a, 0.2)
    assert frac_ref == 0.0 and stats[1].item() == 0.0
    # ratio error of the kernel's fp32 sums of 7 log-probs per side
    drho = 9 * U32 * (np.abs(ln).sum(1) + np.abs(lo_).sum(1)).max() + 4 * U32
    assert abs(stats[0].item() - loss_ref) <= 2 * drho * np.abs(a).mean() + 1e-7
    assert np.allclose(g.cpu().numpy(), g_ref, rtol=2 * drho, atol=0)
    gg = g.cpu().numpy().astype(np.float64).reshape(-1)
    ref = lo.logprob_grad(tf["logits"].reshape(B * cfg.n_actions, -1).cpu().numpy(),
                          out["tokens"].reshape(-1).cpu().numpy(), cfg.action_begin, T, gg)
    err = np.abs(dz.cpu().numpy() - ref)
    log(f"[ppo chain tiny] loss {stats[0].item():.6f} vs {loss_ref:.6f}; max|d dz|={err.max():.3e}")
    assert np.all(err <= 32 * U32 * (np.abs(gg)[:, None] / T + np.abs(ref)))
    S.model.close()
