"""The decode projection without a scratch argument (vla_debug_skinny_noalloc,
for callers that cannot allocate: its split-K partials live in a fixed device
array) against the entry point that takes the caller's scratch
(vla_debug_skinny): the same bits on two calls in a row, the second with a
smaller input, and sizes beyond the fixed array refused on the host."""
import ctypes

import pytest
import torch

from paper_2505_18719_amd import vla

pytestmark = pytest.mark.gpu

VLA_ESHAPE, VLA_EUNSUPPORTED = -2, -7


def _operands(M, N, K, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    A = torch.randn(M, K, generator=g, device="cuda").to(torch.bfloat16)
    W = (torch.randn(N, K, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    return vla.debug_pack_frag(A), vla.debug_pack_frag(W)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def test_noalloc_gives_the_bits_of_the_scratch_entry_point_on_two_calls():
    lib = vla.load_library()
    # the decode's QKV shape at batch 64, then a smaller call on the same fixed array
    for (M, N, K, wg, seed) in ((64, 12288, 4096, 256, 1), (16, 4096, 1024, 200, 2)):
        Af, Wf = _operands(M, N, K, seed)
        scratch = torch.empty(16 * M * N, dtype=torch.float32, device="cuda")
        ref = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        got = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        print(f"[no-alloc] M {M} N {N} K {K} workgroups {wg}", flush=True)
        assert lib.vla_debug_skinny(Af.data_ptr(), Wf.data_ptr(), M, N, K, wg, scratch.data_ptr(), ref.data_ptr(),
                                    _stream()) == 0
        rc = lib.vla_debug_skinny_noalloc(Af.data_ptr(), Wf.data_ptr(), M, N, K, wg, got.data_ptr(), _stream())
        assert rc == 0, lib.vla_last_error()
        torch.cuda.synchronize()
        assert torch.isfinite(ref).all()
        assert torch.equal(got, ref)


def test_noalloc_refuses_sizes_beyond_its_fixed_scratch():
    lib = vla.load_library()
    # 128 x 131072 partial sums (one slot at least) exceed the 2^23-float array: refused before any launch
    M, N, K = 128, 131072, 256
    Af, Wf = _operands(M, N, K, 3)
    C = torch.empty(M, N, dtype=torch.float32, device="cuda")
    rc = lib.vla_debug_skinny_noalloc(Af.data_ptr(), Wf.data_ptr(), M, N, K, 256, C.data_ptr(), _stream())
    assert rc == VLA_ESHAPE and b"2^23" in lib.vla_last_error()
    # more rows than the decode GEMM takes
    rc = lib.vla_debug_skinny_noalloc(Af.data_ptr(), Wf.data_ptr(), 129, 64, 256, 256, C.data_ptr(), _stream())
    assert rc == VLA_EUNSUPPORTED
