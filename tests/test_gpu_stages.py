"""Stage-by-stage parity of one decoder layer: every bf16 rounding point of
the rollout's precision contract (Sec. 3.5: the rollout runs in bf16) is read
back from the GPU and compared with the oracle's arithmetic applied to the
GPU's own input of that stage.

For each stage the test reports the fraction of bf16 values that differ from
the oracle's rounding ("flips"; an fp32 accumulation lands within a few fp32
units of the exact value, so it rounds the other way only when the exact
value lies that close to a bf16 rounding boundary) and checks every element
against a bound derived from fp32 arithmetic: one bf16 unit at the value plus
the fp32 accumulation error of the stage.  Stages (one layer, Llama block):
  u1 = bf16(RMSNorm(x))            attention norm
  q, k = bf16(RoPE(u1 W^T)), v = bf16(u1 Wv^T)
  o  = bf16(softmax(q k^T / sqrt(hd)) v)   (from the GPU's q, k, v)
  xm = x + o Wo^T                  fp32 residual
  u2 = bf16(RMSNorm(xm))           MLP norm
  h  = bf16(silu(u2 Wg^T) * (u2 Wu^T))
  x' = xm + h Wd^T
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import Setup, log
from oracle import vla_oracle as vo
from paper_2505_18719_amd import inputs

pytestmark = pytest.mark.gpu

EPS32 = 2.0 ** -24
MAX_FLIP_RATE = 0.02


def _unfrag(buf, R, K):
    """Rows 0..R-1 of a frag-layout bf16 matrix with K columns (vla_debug.h)."""
    KB = K // 32 + 1
    r = np.arange(R)[:, None]
    k = np.arange(K)[None, :]
    idx = ((((r >> 4) * KB + (k >> 5)) << 6) + (r & 15) + (((k & 31) >> 3) << 4)) * 8 + (k & 7)
    raw = buf.view(torch.int16).cpu().numpy()[idx]
    return torch.from_numpy(raw).view(torch.bfloat16).double().numpy()


def _bf16_ulp(x):
    """Spacing of bf16 values at |x| (8 significant bits)."""
    a = np.maximum(np.abs(x), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def _check_bf16(label, got, exp_exact, err_abs):
    """got: GPU bf16 values; exp_exact: the oracle's unrounded values; err_abs:
    per-element bound of the fp32 arithmetic's distance from them."""
    exp = vo.bf16_round(exp_exact)
    flips = float(np.mean(got != exp))
    bound = _bf16_ulp(exp) + err_abs
    excess = float(np.max(np.abs(got - exp) - bound))
    log(f"  {label}: {got.size} values, flips {flips:.4%}, max|d| {np.abs(got - exp).max():.3e}, "
        f"max(|d| - bound) {excess:.2e}")
    assert excess <= 0.0, label
    assert flips <= MAX_FLIP_RATE, label
    return flips


def _check_f32(label, got, exp, err_abs):
    d = np.abs(got - exp)
    excess = float(np.max(d - err_abs))
    log(f"  {label}: max|d| {d.max():.3e} (bound {err_abs.max():.2e}), max(|d| - bound) {excess:.2e}")
    assert excess <= 0.0, label


def _kv(pool, b, n, B, H, hd, max_pages, transposed):
    """Keys / values 0..n-1 of environment b from a page pool (env b's page p is physical page p*B + b)."""
    P = pool.reshape(-1, H, *((hd, 16) if transposed else (16, hd)))
    out = np.empty((n, H, hd))
    for t in range(n):
        pg = P[(t // 16) * B + b]
        out[t] = pg[:, :, t % 16] if transposed else pg[:, t % 16, :]
    return out


def _read(model, which, layer, n, dtype):
    buf = torch.empty(n, dtype=dtype, device="cuda")
    model.debug_read(which, layer, buf)
    torch.cuda.synchronize()
    return buf


def _layer_stages(S, inp, dev, layer):
    cfg, model, W = S.cfg, S.model, S.W
    d, H, hd, F = cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ffn
    Fp = (F + 255) // 256 * 256
    B = inp.batch
    L = inp.prefix_lens.astype(int)
    M = int(L.sum())
    row0 = np.concatenate([[0], np.cumsum(L)])
    max_seq = cfg.max_seq
    max_pages = (max_seq + 15) // 16
    lw = W.layer(layer)
    eps = cfg.rms_eps
    frag_n = ((M + 15) // 16) * (d // 32 + 1) * 512

    def run(stop):
        model.debug_layer_limit(layer + 1)
        model.debug_stop(stop)
        model.prefill(dev["vis"], dev["ids"], inp.prompt_lens)
        torch.cuda.synchronize()

    try:
        run(1)
        x = _read(model, 0, 0, M * d, torch.float32).cpu().double().numpy().reshape(M, d)
        u1 = _unfrag(_read(model, 4, 0, frag_n, torch.bfloat16), M, d)
        run(2)
        q = _read(model, 1, 0, M * d, torch.bfloat16).cpu().double().numpy().reshape(M, d)
        n_pool = B * max_pages * H * 16 * hd
        kp = _read(model, 2, layer, n_pool, torch.bfloat16).cpu().double().numpy()
        vp = _read(model, 3, layer, n_pool, torch.bfloat16).cpu().double().numpy()
        o = _unfrag(_read(model, 4, 0, frag_n, torch.bfloat16), M, d)
        run(3)
        xm = _read(model, 0, 0, M * d, torch.float32).cpu().double().numpy().reshape(M, d)
        u2 = _unfrag(_read(model, 4, 0, frag_n, torch.bfloat16), M, d)
        run(0)
        x1 = _read(model, 0, 0, M * d, torch.float32).cpu().double().numpy().reshape(M, d)
        h_n = ((M + 15) // 16) * (Fp // 32 + 1) * 512
        h = _unfrag(_read(model, 9, 0, h_n, torch.bfloat16), M, Fp)[:, :F]
    finally:
        model.debug_stop(0)
        model.debug_layer_limit(0)

    flips = {}
    log(f"[stages {cfg.name} layer {layer}] rows {M}")
    # attention norm: fp32 sum of squares and scaling, a few fp32 units
    ref = vo.rms_norm(x, lw["attn_norm"], eps)
    flips["u1"] = _check_bf16("u1 = bf16(RMSNorm(x))", u1, ref, 8 * EPS32 * np.abs(ref))
    # q, k after RoPE and v, from the GPU's u1 (fp32 accumulation over d, then the rotation)
    pos = np.concatenate([np.arange(l) for l in L])
    acc = np.abs(u1) @ np.abs(np.concatenate([lw["wq"], lw["wk"], lw["wv"]])).T * d * EPS32
    qe = (u1 @ lw["wq"].T).reshape(M, H, hd)
    ke = (u1 @ lw["wk"].T).reshape(M, H, hd)
    ve = u1 @ lw["wv"].T
    # the rotation mixes a pair: each output's error is at most the sum of the pair's errors
    # plus the rotation's own rounding (a few fp32 units of the pair's magnitude)
    def rot_err(e, val):
        e = e.reshape(M, H, hd)
        val = np.abs(val)
        half = hd // 2
        pe = e[..., :half] + e[..., half:] + 4 * EPS32 * (val[..., :half] + val[..., half:])
        return np.concatenate([pe, pe], axis=-1).reshape(M, d)
    qr = vo.apply_rope(qe, pos, cfg.rope_base).reshape(M, d)
    kr = vo.apply_rope(ke, pos, cfg.rope_base)
    flips["q"] = _check_bf16("q = bf16(RoPE(u1 Wq^T))", q, qr, rot_err(acc[:, :d], qe))
    kg = np.concatenate([_kv(kp, b, L[b], B, H, hd, max_pages, False) for b in range(B)])
    vg = np.concatenate([_kv(vp, b, L[b], B, H, hd, max_pages, True) for b in range(B)])
    flips["k"] = _check_bf16("k = bf16(RoPE(u1 Wk^T)) (KV pages)", kg.reshape(M, d), kr.reshape(M, d),
                             rot_err(acc[:, d:2 * d], ke))
    flips["v"] = _check_bf16("v = bf16(u1 Wv^T) (KV pages)", vg.reshape(M, d), ve, acc[:, 2 * d:])
    # attention from the GPU's q, k, v: scores over bf16 inputs in fp32, P split into two bf16
    # halves (~16 significant bits) for the P V product
    oe = np.empty((M, d))
    oerr = np.empty((M, d))
    for b in range(B):
        rs = slice(row0[b], row0[b + 1])
        qb = q[rs].reshape(L[b], H, hd)
        kb, vb = kg[rs], vg[rs]
        ob, p = vo.causal_attention(qb, kb, vb, np.arange(L[b]), np.arange(L[b]), return_probs=True)
        oe[rs] = ob.reshape(L[b], d)
        # |dP| <= 2^-16 P (hi+lo split) + the score error (hd fp32 units of sum |q||k|) through exp
        sc_err = np.einsum("lhd,thd->hlt", np.abs(qb), np.abs(kb)) * hd * EPS32 / np.sqrt(hd)
        dp = p * (2.0 ** -16 + 2 * sc_err + 8 * EPS32)
        oerr[rs] = np.transpose(np.matmul(dp, np.transpose(np.abs(vb), (1, 0, 2))), (1, 0, 2)).reshape(L[b], d) * 2
    flips["o"] = _check_bf16("o = bf16(attention(q, k, v))", o, oe, oerr)
    # O projection and the residual add (fp32)
    xme = x + o @ lw["wo"].T
    _check_f32("xm = x + o Wo^T", xm, xme, (np.abs(o) @ np.abs(lw["wo"]).T) * d * EPS32 + 2 * EPS32 * np.abs(xme))
    ref = vo.rms_norm(xm, lw["mlp_norm"], eps)
    flips["u2"] = _check_bf16("u2 = bf16(RMSNorm(xm))", u2, ref, 8 * EPS32 * np.abs(ref))
    # SwiGLU from the GPU's u2
    ge, ue = u2 @ lw["wgate"].T, u2 @ lw["wup"].T
    dg = (np.abs(u2) @ np.abs(lw["wgate"]).T) * d * EPS32
    du = (np.abs(u2) @ np.abs(lw["wup"]).T) * d * EPS32
    sg = vo.silu(ge)
    he = sg * ue
    herr = 1.1 * dg * np.abs(ue) + np.abs(sg) * du + 8 * EPS32 * np.abs(he)
    flips["h"] = _check_bf16("h = bf16(silu(u2 Wg^T) (u2 Wu^T))", h, he, herr)
    x1e = xm + h @ lw["wdown"].T
    _check_f32("x' = xm + h Wd^T", x1, x1e, (np.abs(h) @ np.abs(lw["wdown"]).T) * F * EPS32 + 2 * EPS32 * np.abs(x1e))
    return flips


TINY_RAGGED = inputs.TINY.replace(name="tiny_ragged", batch=5, prompt_min=0, prompt_max=40)


@pytest.mark.parametrize("layer", [0, 1])
def test_tiny_layer_stages(layer):
    S = Setup(TINY_RAGGED, seed=1, gain_jitter=True)
    inp, dev = S.inputs(seed=3, prompt_lens=[0, 40, 7, 33, 16])
    _layer_stages(S, inp, dev, layer)
    S.model.close()


@pytest.mark.parametrize("layer", [0, 7])
def test_mid_layer_stages(layer):
    S = Setup(inputs.MID, seed=0)
    inp, dev = S.inputs(seed=0, batch=3)
    _layer_stages(S, inp, dev, layer)
    S.model.close()
