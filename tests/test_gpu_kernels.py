"""Kernel-level parity on the GPU: the prefill MFMA GEMM, the decode split-K
GEMM and the Gumbel-max sampler against float64 / oracle references."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import log

pytestmark = pytest.mark.gpu


def _rand_bf16(shape, seed, scale=1.0):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return (torch.randn(shape, generator=g, device="cuda") * scale).to(torch.bfloat16)


def _check_matmul(C, A, W, label):
    a, w = A.double().cpu(), W.double().cpu()
    ref = a @ w.T
    bound = A.shape[1] * 1.2e-7 * (a.abs() @ w.abs().T) + 1e-30
    err = (C.double().cpu() - ref).abs()
    log(f"[{label}] M,N,K={tuple(A.shape[:1]) + tuple(W.shape)} max|err|={err.max().item():.3e} "
        f"max err/bound={(err / bound).max().item():.3f}")
    assert bool((err <= bound).all())


# (M, N, K): tiny, ragged M and N with more tiles than CUs per workgroup round
# or fewer, several rounds per workgroup, long K
@pytest.mark.parametrize("M,N,K", [(1, 64, 128), (300, 384, 384), (513, 1408, 768), (256, 256, 4096),
                                   (1000, 3072, 1024), (4100, 16448, 256)])
def test_prefill_gemm_matches_float64(M, N, K):
    from paper_2505_18719_amd import vla
    A, W = _rand_bf16((M, K), 1), _rand_bf16((N, K), 2, 0.02)
    C = vla.debug_gemm(A, W)
    torch.cuda.synchronize()
    _check_matmul(C, A, W, "gemm")


def test_prefill_gemm_rows_independent_of_tiling():
    """A row's result is bit-identical however many rows are multiplied with it
    (one workgroup round at M = 256, forty tile rows and a partial last round
    at M = 10240): the batch-composition invariance of the prefill GEMM."""
    from paper_2505_18719_amd import vla
    A, W = _rand_bf16((10240, 512), 11), _rand_bf16((2048, 512), 12, 0.02)
    C_small = vla.debug_gemm(A[:256].contiguous(), W)
    C_big = vla.debug_gemm(A, W)
    torch.cuda.synchronize()
    assert torch.equal(C_small, C_big[:256])
    _check_matmul(C_big[-300:], A[-300:], W, "gemm-last-round")


def test_prefill_gemm_7b_shape_sampled_rows():
    """QKV projection at the 7B batch-64 prefill shape (M = 18432 packed rows)."""
    from paper_2505_18719_amd import vla
    M, N, K = 18432, 12288, 4096
    A, W = _rand_bf16((M, K), 3), _rand_bf16((N, K), 4, 0.02)
    C = vla.debug_gemm(A, W)
    torch.cuda.synchronize()
    rows = torch.tensor([0, 1, 255, 256, 4097, 9000, M - 2, M - 1], device="cuda")
    _check_matmul(C[rows], A[rows], W, "gemm-7b-sampled")


# (N, K, workgroups): whole tiles only, stream-K only, whole tiles plus a
# stream-K remainder, a single unit, and the 7B shapes on 256 workgroups
@pytest.mark.parametrize("M", [1, 7, 16, 33, 64, 128])
@pytest.mark.parametrize("N,K,wg", [(256, 4096, 256), (1024, 768, 3), (768, 256, 5), (64, 256, 1),
                                    (4096, 11008, 256), (12288, 4096, 256), (22016, 4096, 256), (4096, 4096, 256)])
def test_decode_skinny_gemm_matches_float64(M, N, K, wg):
    from paper_2505_18719_amd import vla
    A, W = _rand_bf16((M, K), 5 + M), _rand_bf16((N, K), 6, 0.02)
    C = vla.debug_skinny(A, W, wg)
    torch.cuda.synchronize()
    _check_matmul(C, A, W, f"skinny wg={wg}")


@pytest.mark.parametrize("N,K", [(22016, 4096), (4096, 11008), (12288, 4096)])
def test_decode_skinny_gemm_is_deterministic(N, K):
    from paper_2505_18719_amd import vla
    A, W = _rand_bf16((64, K), 11), _rand_bf16((N, K), 12, 0.02)
    C1 = vla.debug_skinny(A, W, 256)
    C2 = vla.debug_skinny(A, W, 256)
    torch.cuda.synchronize()
    assert torch.equal(C1, C2)


@pytest.mark.parametrize("T", [1.0, 1.5])
def test_sampler_matches_oracle(T):
    from paper_2505_18719_amd import vla
    from paper_2505_18719_amd.inputs import TINY, gumbel_noise
    B, A, na, a0 = 64, 256, 7, 31808
    rng = np.random.default_rng(7)
    z = (rng.normal(size=(B, A)) * 1.3).astype(np.float32)
    z[3] = 0.5                      # exact tie across all bins ...
    g = gumbel_noise(TINY, B, seed=9)
    g[3, 2] = 0.25                  # ... and in the noise: lowest index wins
    out = vla.debug_sample(torch.from_numpy(z).cuda(), torch.from_numpy(g).cuda(), 2, T, a0)
    torch.cuda.synchronize()
    tok = out["tokens"][:, 2].cpu().numpy()
    lp = out["logp"][:, 2].cpu().numpy()
    en = out["entropy"][:, 2].cpu().numpy()
    for b in range(B):
        k, lpr, enr, _ = oracle.sample_bin(z[b].astype(np.float64), g[b, 2], T)
        assert tok[b] == a0 + k, b
        assert abs(lp[b] - lpr) < 1e-5 and abs(en[b] - enr) < 1e-5
    assert tok[3] == a0
    assert torch.equal(out["logits"][:, 2].cpu(), torch.from_numpy(z))
    assert torch.equal(out["next"].cpu(), out["tokens"][:, 2].cpu())
    assert bool((out["tokens"][:, [0, 1, 3, 4, 5, 6]] == -1).all())   # other steps untouched
