"""Host-side checks of the C-ABI library (no GPU needed): it loads, exports
every function its headers declare, and validates configurations and
arguments before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2505_18719_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def vla():
    from paper_2505_18719_amd import vla as binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2505_18719_amd import build
        build.build(verbose=False)
    binding.load_library()
    return binding


def _declared_functions():
    names = set()
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            txt = open(os.path.join(ROOT, "include", f)).read()
            names |= set(re.findall(r"^(?:int|void|const char\*|size_t)\s+(vla_\w+)\(", txt, re.M))
    return sorted(names)


@pytest.mark.parametrize("header", ["vla.h", "vla_learn.h", "vla_debug.h"])
@pytest.mark.parametrize("lang", ["c", "c++"])
def test_each_header_compiles_on_its_own(header, lang, tmp_path):
    """A C-ABI header includes what it uses: it compiles alone, as C99 and as
    C++, with warnings as errors (only the host compiler is needed)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc" if lang == "c" else "g++")
    if cc is None:
        pytest.skip("no host compiler")
    src = tmp_path / ("h.c" if lang == "c" else "h.cpp")
    src.write_text(f'#include "{header}"\nint main(void) {{ return 0; }}\n')
    std = ["-std=c99", "-pedantic"] if lang == "c" else ["-std=c++17"]
    r = subprocess.run([cc, *std, "-Wall", "-Wextra", "-Werror", "-fsyntax-only", "-I", os.path.join(ROOT, "include"),
                        str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_headers_declare_the_rollout_entry_points():
    names = _declared_functions()
    for n in ("vla_prefill", "vla_decode_actions", "vla_token_logprobs", "vla_create", "vla_workspace_size",
              "vla_destroy", "vla_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(vla):
    lib = vla.load_library()
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_workspace_size_and_config_validation(vla):
    lib = vla.load_library()
    n = ctypes.c_size_t()
    c = vla.make_config(inputs.L7B_B64, max_batch=64)
    assert lib.vla_workspace_size(ctypes.byref(c), ctypes.byref(n)) == 0
    # repacked weights (~13.2 GB incl. embedding) + KV pool for 64 x 320 tokens (~10.7 GB) + activations
    assert 20e9 < n.value < 40e9
    bad = [dict(head_dim_override=96), dict(max_seq=400), dict(action_bins=300), dict(max_batch=0),
           dict(n_actions=0), dict(page_size=8)]
    for b in bad:
        c = vla.make_config(inputs.TINY)
        for k, v in b.items():
            setattr(c, "head_dim" if k == "head_dim_override" else k, v)
        rc = lib.vla_workspace_size(ctypes.byref(c), ctypes.byref(n))
        assert rc in (-1, -7), (b, rc)
        assert lib.vla_last_error().decode()
    assert lib.vla_workspace_size(None, ctypes.byref(n)) == -1


def test_create_rejects_null_arguments_before_device_work(vla):
    lib = vla.load_library()
    c = vla.make_config(inputs.TINY)
    h = ctypes.c_void_p()
    assert lib.vla_create(ctypes.byref(c), None, None, 0, None, ctypes.byref(h)) == -1
    assert "NULL" in lib.vla_last_error().decode()
    assert lib.vla_prefill(None, 1, None, None, None, None, None) == -1
    assert lib.vla_decode_actions(None, 1, None, 1.0, None, None, None, None, None) == -1
    lib.vla_destroy(None)


def test_lora_merge_validates_arguments_before_the_device(vla):
    """Null handle, unknown projection, bad rank or scale are rejected by the
    host code (no model or device memory is touched)."""
    lib = vla.load_library()
    p = ctypes.c_void_p(16)  # never dereferenced: validation fails first
    assert lib.vla_lora_merge(None, 0, 0, p, p, p, 8, 1.0, None) == -1
    assert b"model is NULL" in lib.vla_last_error()
    arr = (ctypes.c_void_p * 7)(*([p] * 7))
    assert lib.vla_lora_merge_layer(None, 0, arr, arr, arr, 8, 1.0, None) == -1
    assert b"model is NULL" in lib.vla_last_error()


def test_learning_entry_points_validate_on_the_host(vla):
    """vla_learn.h: bad sizes, parameters and null buffers are rejected, and
    empty windows are no-ops, all before any device work."""
    lib = vla.load_library()
    p = ctypes.c_void_p(16)  # never dereferenced: validation fails first
    assert lib.vla_gae(4, 8, p, p, p, 1.5, 0.9, p, p, None) == -1
    assert b"gamma" in lib.vla_last_error()
    assert lib.vla_gae(4, 8, p, p, p, 0.99, float("nan"), p, p, None) == -1
    assert lib.vla_gae(-1, 8, p, p, p, 0.99, 0.9, p, p, None) == -1
    assert lib.vla_gae(0, 8, None, None, None, 0.99, 0.9, None, None, None) == 0
    assert lib.vla_gae(4, 0, None, None, None, 0.99, 0.9, None, None, None) == 0
    assert lib.vla_gae(4, 8, p, None, p, 0.99, 0.9, p, None, None) == -1
    assert lib.vla_ppo_clip(0, 7, p, p, p, 0.2, p, p, None) == -1
    assert lib.vla_ppo_clip(4, 17, p, p, p, 0.2, p, p, None) == -1
    assert lib.vla_ppo_clip(4, 7, p, p, p, -0.1, p, p, None) == -1
    assert lib.vla_ppo_clip(4, 7, p, p, p, float("inf"), p, p, None) == -1
    assert lib.vla_ppo_clip(4, 7, p, p, None, 0.2, p, p, None) == -1
    assert lib.vla_logprob_backward(4, 257, 0, p, p, 1.0, p, p, None) == -7
    assert lib.vla_logprob_backward(4, 256, 0, p, p, 0.0, p, p, None) == -1
    assert lib.vla_logprob_backward(0, 256, 0, None, None, 1.5, None, None, None) == 0
    assert lib.vla_logprob_backward(4, 256, 0, p, None, 1.5, p, p, None) == -1


def test_extract_actions_validates_on_the_host(vla):
    lib = vla.load_library()
    p = ctypes.c_void_p(16)  # never dereferenced: validation fails first
    assert lib.vla_extract_actions(4, 0, p, 0, 256, p, p, p, None) == -1
    assert lib.vla_extract_actions(4, 7, p, 0, 300, p, p, p, None) == -7
    assert lib.vla_extract_actions(4, 7, p, 0, 256, None, p, p, None) == -1
    assert lib.vla_extract_actions(0, 7, None, 0, 256, None, None, None, None) == 0


def test_lora_gradient_entry_validates_on_the_host(vla):
    """vla_ppo_lora_grads rejects a NULL model, bad batch, rank, parameters and a
    missing workspace before any device work."""
    lib = vla.load_library()
    p = ctypes.c_void_p(16)  # never dereferenced: validation fails first
    lora = vla._Lora(8, 0.5, None, None, None, None)
    assert lib.vla_ppo_lora_grads(None, 1, p, p, p, p, p, p, 0.2, 1.5, ctypes.byref(lora), p, 1, p, None, None) == -1
    assert b"model is NULL" in lib.vla_last_error()
    n = ctypes.c_size_t()
    c = vla.make_config(inputs.TINY)
    assert lib.vla_train_workspace_size(ctypes.byref(c), 0, ctypes.byref(n)) == 0 and n.value > 0
    n_keep = ctypes.c_size_t()
    assert lib.vla_train_workspace_size(ctypes.byref(c), 1, ctypes.byref(n_keep)) == 0 and n_keep.value > n.value
    assert lib.vla_train_workspace_size(ctypes.byref(c), 2, ctypes.byref(n)) == -1
    assert lib.vla_train_workspace_size(None, 0, ctypes.byref(n)) == -1
