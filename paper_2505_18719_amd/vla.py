"""ctypes binding of ``libvla.so`` (argument marshalling only).

Every step of the rollout path runs in the HIP library; this module only
passes device pointers of torch tensors, the current HIP stream and host
arrays through the C ABI of ``include/vla.h``.  Importing it fails loudly if
the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvla.so")

VLA_OK = 0
STATUS = {-1: "VLA_EINVAL", -2: "VLA_ESHAPE", -3: "VLA_EWORKSPACE", -4: "VLA_EHIP", -6: "VLA_ESTATE",
          -7: "VLA_EUNSUPPORTED"}
FLAG_BAD_PROMPT_ID = 1
FLAG_BAD_ACTION = 2

EXPORTS = ("vla_workspace_size", "vla_create", "vla_prefill", "vla_decode_actions", "vla_token_logprobs",
           "vla_value", "vla_lora_merge", "vla_lora_merge_layer", "vla_read_device_flags", "vla_profile_begin", "vla_profile_end", "vla_destroy",
           "vla_last_error", "vla_extract_actions", "vla_gae", "vla_ppo_clip", "vla_logprob_backward",
           "vla_train_workspace_size", "vla_ppo_lora_grads")
# projections a LoRA adapter merges into (VLA_PROJ_* order), by weight-dict key
PROJECTIONS = ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")
PROF_CATEGORIES = ("prefill_gemm", "prefill_attn", "decode_gemm", "decode_attn", "decode_layer")
# training modes of vla_ppo_lora_grads (VLA_TRAIN_*): recompute each layer's forward, or keep it
TRAIN_RECOMPUTE, TRAIN_KEEP = 0, 1
DEBUG_EXPORTS = ("vla_debug_gemm", "vla_debug_skinny", "vla_debug_pack_frag", "vla_debug_sample", "vla_debug_read",
                 "vla_debug_set_layer_limit", "vla_debug_set_stop", "vla_debug_skinny_noalloc",
                 "vla_debug_set_decode_path", "vla_debug_trace_decode_layer")


class VlaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class _Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "d_model", "n_heads", "head_dim", "d_ffn", "vocab",
                                              "action_bins", "action_begin", "n_actions", "n_visual")] + \
               [("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float)] + \
               [(n, ctypes.c_int32) for n in ("max_batch", "max_seq", "page_size")]


_PP = ctypes.POINTER(ctypes.c_void_p)


class _Weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p), ("final_norm", ctypes.c_void_p)] + \
               [(n, _PP) for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wgate", "wup", "wdown")]


class _Lora(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("scale", ctypes.c_float), ("a", _PP), ("b", _PP), ("grad_a", _PP),
                ("grad_b", _PP)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it is missing: there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(path)
    i32, vp, f32 = ctypes.c_int32, ctypes.c_void_p, ctypes.c_float
    lib.vla_workspace_size.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(ctypes.c_size_t)]
    lib.vla_create.argtypes = [ctypes.POINTER(_Config), ctypes.POINTER(_Weights), vp, ctypes.c_size_t, vp,
                               ctypes.POINTER(vp)]
    lib.vla_prefill.argtypes = [vp, i32, vp, vp, vp, vp, vp]
    lib.vla_decode_actions.argtypes = [vp, i32, vp, f32, vp, vp, vp, vp, vp]
    lib.vla_token_logprobs.argtypes = [vp, i32, vp, vp, vp, vp, f32, vp, vp, vp, vp]
    lib.vla_lora_merge.argtypes = [vp, i32, i32, vp, vp, vp, i32, f32, vp]
    lib.vla_lora_merge_layer.argtypes = [vp, i32, vp, vp, vp, i32, f32, vp]
    lib.vla_value.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp]
    lib.vla_read_device_flags.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_uint32)]
    lib.vla_extract_actions.argtypes = [i32, i32, vp, i32, i32, vp, vp, vp, vp]
    lib.vla_train_workspace_size.argtypes = [ctypes.POINTER(_Config), i32, ctypes.POINTER(ctypes.c_size_t)]
    lib.vla_ppo_lora_grads.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, f32, f32, ctypes.POINTER(_Lora), vp,
                                       ctypes.c_size_t, vp, vp, vp]
    lib.vla_gae.argtypes = [i32, i32, vp, vp, vp, f32, f32, vp, vp, vp]
    lib.vla_ppo_clip.argtypes = [i32, i32, vp, vp, vp, f32, vp, vp, vp]
    lib.vla_logprob_backward.argtypes = [i32, i32, i32, vp, vp, f32, vp, vp, vp]
    lib.vla_profile_begin.argtypes = [vp, ctypes.c_uint32]
    lib.vla_profile_end.argtypes = [vp, vp, vp, vp]
    lib.vla_destroy.argtypes = [vp]
    lib.vla_destroy.restype = None
    lib.vla_last_error.restype = ctypes.c_char_p
    lib.vla_debug_gemm.argtypes = [vp, vp, i32, i32, i32, vp, vp]
    lib.vla_debug_skinny.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp]
    lib.vla_debug_skinny_noalloc.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp]
    lib.vla_debug_pack_frag.argtypes = [vp, i32, i32, i32, vp, vp]
    lib.vla_debug_sample.argtypes = [vp, i32, i32, i32, i32, i32, vp, f32, vp, vp, vp, vp, vp, vp]
    lib.vla_debug_read.argtypes = [vp, i32, i32, vp, ctypes.c_size_t, vp]
    lib.vla_debug_set_layer_limit.argtypes = [vp, i32]
    lib.vla_debug_set_stop.argtypes = [vp, i32]
    lib.vla_debug_set_decode_path.argtypes = [vp, i32]
    lib.vla_debug_trace_decode_layer.argtypes = [vp, i32, vp]
    for name in EXPORTS + DEBUG_EXPORTS:
        if name not in ("vla_destroy", "vla_last_error"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(code: int) -> None:
    if code != VLA_OK:
        raise VlaError(code, _lib.vla_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def make_config(cfg, max_batch: Optional[int] = None, max_seq: Optional[int] = None) -> _Config:
    return _Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ffn, cfg.vocab, cfg.action_bins,
                   cfg.action_begin, cfg.n_actions, cfg.n_visual, cfg.rope_base, cfg.rms_eps,
                   cfg.batch if max_batch is None else max_batch, cfg.max_seq if max_seq is None else max_seq,
                   cfg.page_size)


def workspace_bytes(cfg, max_batch: Optional[int] = None, max_seq: Optional[int] = None) -> int:
    lib = load_library()
    c = make_config(cfg, max_batch, max_seq)
    n = ctypes.c_size_t()
    _check(lib.vla_workspace_size(ctypes.byref(c), ctypes.byref(n)))
    return n.value


class VlaModel:
    """A model handle over a caller-owned workspace (a torch uint8 tensor)."""

    def __init__(self, cfg, weights: Dict[str, object], max_batch: Optional[int] = None,
                 max_seq: Optional[int] = None, device="cuda"):
        self.lib = load_library()
        self.cfg = cfg
        self.device = torch.device(device)
        self.c_cfg = make_config(cfg, max_batch, max_seq)
        n = ctypes.c_size_t()
        _check(self.lib.vla_workspace_size(ctypes.byref(self.c_cfg), ctypes.byref(n)))
        self.workspace = torch.empty(n.value, dtype=torch.uint8, device=self.device)
        L = cfg.n_layers
        arrays = {}
        for k in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wgate", "wup", "wdown"):
            arr = (ctypes.c_void_p * L)(*[_ptr(weights["layers"][i][k]).value for i in range(L)])
            arrays[k] = arr
        self._keep = arrays
        w = _Weights(_ptr(weights["embed"]), _ptr(weights["lm_head"]), _ptr(weights["final_norm"]),
                     *[ctypes.cast(arrays[k], _PP) for k in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                                              "wgate", "wup", "wdown")])
        h = ctypes.c_void_p()
        _check(self.lib.vla_create(ctypes.byref(self.c_cfg), ctypes.byref(w), _ptr(self.workspace),
                                   ctypes.c_size_t(n.value), _stream(self.device), ctypes.byref(h)))
        self.handle = h

    # --------------------------------------------------------------- rollout
    def prefill(self, vis: torch.Tensor, prompt_ids: torch.Tensor, prompt_lens: np.ndarray,
                out: Optional[torch.Tensor] = None) -> torch.Tensor:
        lens = np.ascontiguousarray(prompt_lens, dtype=np.int32)
        B = int(lens.shape[0])
        if out is None:
            out = torch.empty(B, self.cfg.action_bins, dtype=torch.float32, device=self.device)
        _check(self.lib.vla_prefill(self.handle, B, _ptr(vis), _ptr(prompt_ids),
                                    lens.ctypes.data_as(ctypes.c_void_p), _ptr(out), _stream(self.device)))
        self._last_batch = B
        return out

    def decode_actions(self, gumbel: torch.Tensor, temperature: float, batch: Optional[int] = None,
                       with_logits: bool = True, out: Optional[Dict[str, torch.Tensor]] = None
                       ) -> Dict[str, torch.Tensor]:
        B = self._last_batch if batch is None else batch
        na, A = self.cfg.n_actions, self.cfg.action_bins
        if out is None:
            out = {"tokens": torch.empty(B, na, dtype=torch.int32, device=self.device),
                   "logp": torch.empty(B, na, dtype=torch.float32, device=self.device),
                   "entropy": torch.empty(B, na, dtype=torch.float32, device=self.device)}
            if with_logits:
                out["logits"] = torch.empty(B, na, A, dtype=torch.float32, device=self.device)
        _check(self.lib.vla_decode_actions(self.handle, B, _ptr(gumbel), float(temperature), _ptr(out["tokens"]),
                                           _ptr(out["logp"]), _ptr(out.get("entropy")), _ptr(out.get("logits")),
                                           _stream(self.device)))
        return out

    def token_logprobs(self, vis: torch.Tensor, prompt_ids: torch.Tensor, prompt_lens: np.ndarray,
                       actions: torch.Tensor, temperature: float, with_logits: bool = True
                       ) -> Dict[str, torch.Tensor]:
        lens = np.ascontiguousarray(prompt_lens, dtype=np.int32)
        B = int(lens.shape[0])
        na, A = self.cfg.n_actions, self.cfg.action_bins
        out = {"logp": torch.empty(B, na, dtype=torch.float32, device=self.device),
               "entropy": torch.empty(B, na, dtype=torch.float32, device=self.device)}
        if with_logits:
            out["logits"] = torch.empty(B, na, A, dtype=torch.float32, device=self.device)
        _check(self.lib.vla_token_logprobs(self.handle, B, _ptr(vis), _ptr(prompt_ids),
                                           lens.ctypes.data_as(ctypes.c_void_p), _ptr(actions), float(temperature),
                                           _ptr(out["logp"]), _ptr(out["entropy"]), _ptr(out.get("logits")),
                                           _stream(self.device)))
        return out

    def value(self, vis: torch.Tensor, prompt_ids: torch.Tensor, prompt_lens: np.ndarray,
              value_head: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Value estimates [batch] of the decoder held by this handle with the given head."""
        lens = np.ascontiguousarray(prompt_lens, dtype=np.int32)
        B = int(lens.shape[0])
        assert value_head.dtype == torch.bfloat16 and value_head.is_contiguous() and value_head.is_cuda
        if out is None:
            out = torch.empty(B, dtype=torch.float32, device=self.device)
        _check(self.lib.vla_value(self.handle, B, _ptr(vis), _ptr(prompt_ids), lens.ctypes.data_as(ctypes.c_void_p),
                                  _ptr(value_head), _ptr(out), _stream(self.device)))
        return out

    def lora_merge(self, layer: int, projection: str, w0: torch.Tensor, lora_a: torch.Tensor,
                   lora_b: torch.Tensor, scale: float) -> None:
        """W = bf16(w0 + scale * lora_b @ lora_a) for one projection ('wq' ..
        'wdown') of one layer; w0 is the original checkpoint weight."""
        rank = int(lora_a.shape[0])
        for t in (w0, lora_a, lora_b):
            assert t.dtype == torch.bfloat16 and t.is_contiguous() and t.is_cuda
        _check(self.lib.vla_lora_merge(self.handle, layer, PROJECTIONS.index(projection), _ptr(w0), _ptr(lora_a),
                                       _ptr(lora_b), rank, float(scale), _stream(self.device)))

    def lora_merge_layer(self, layer: int, w0: Dict[str, torch.Tensor], adapters: Dict[str, tuple],
                         scale: float) -> None:
        """lora_merge of every projection of `layer` that `adapters` ({key: (lora_a, lora_b)}, one shared
        rank) holds, in one launch; w0 holds the original checkpoint weights by key."""
        n = len(PROJECTIONS)
        ws, As, Bs = (ctypes.c_void_p * n)(), (ctypes.c_void_p * n)(), (ctypes.c_void_p * n)()
        ranks = set()
        for i, key in enumerate(PROJECTIONS):
            if key not in adapters:
                continue
            a, b = adapters[key]
            for t in (w0[key], a, b):
                assert t.dtype == torch.bfloat16 and t.is_contiguous() and t.is_cuda
            ws[i], As[i], Bs[i] = _ptr(w0[key]), _ptr(a), _ptr(b)
            ranks.add(int(a.shape[0]))
        assert len(ranks) <= 1, "the adapters of one call share their rank"
        rank = ranks.pop() if ranks else 8
        _check(self.lib.vla_lora_merge_layer(self.handle, layer, ws, As, Bs, rank, float(scale), _stream(self.device)))

    def ppo_lora_grads(self, vis: torch.Tensor, prompt_ids: torch.Tensor, prompt_lens: np.ndarray,
                       actions: torch.Tensor, logp_old: torch.Tensor, advantages: torch.Tensor, eps: float,
                       temperature: float, adapters, scale: float, mode: int = TRAIN_KEEP):
        """Gradients of the PPO-clip loss w.r.t. the LoRA factors (vla_ppo_lora_grads).
        adapters: per layer {projection key: (A [r, in], B [out, r])} bf16 device tensors
        (layers or keys absent: not adapted).  mode: TRAIN_KEEP (the forward keeps every
        layer's activations) or TRAIN_RECOMPUTE (the workspace for it, the backward
        recomputes them).  Returns (stats [loss, clipped fraction], logp_new [batch,
        n_actions], grads: per layer {key: (dA, dB)})."""
        lens = np.ascontiguousarray(prompt_lens, dtype=np.int32)
        B = int(lens.shape[0])
        L = self.cfg.n_layers
        if getattr(self, "_train_ws_mode", None) != mode:
            self._train_ws = None
            n = ctypes.c_size_t()
            _check(self.lib.vla_train_workspace_size(ctypes.byref(self.c_cfg), int(mode), ctypes.byref(n)))
            self._train_ws = torch.empty(n.value, dtype=torch.uint8, device=self.device)
            self._train_ws_mode = mode
        ranks = {int(a.shape[0]) for ad in adapters for a, _ in ad.values()}
        assert len(ranks) == 1, "one rank for every adapter"
        rank = ranks.pop()
        arr = [[None] * (L * 7) for _ in range(4)]
        grads = [dict() for _ in range(L)]
        for li, ad in enumerate(adapters):
            for key, (a, b) in ad.items():
                p = PROJECTIONS.index(key)
                for t in (a, b):
                    assert t.dtype == torch.bfloat16 and t.is_contiguous() and t.is_cuda
                ga = torch.empty(a.shape, dtype=torch.float32, device=self.device)
                gb = torch.empty(b.shape, dtype=torch.float32, device=self.device)
                grads[li][key] = (ga, gb)
                for j, t in enumerate((a, b, ga, gb)):
                    arr[j][li * 7 + p] = t.data_ptr()
        ptrs = [(ctypes.c_void_p * (L * 7))(*arr[j]) for j in range(4)]
        lora = _Lora(rank, float(scale), *[ctypes.cast(p, _PP) for p in ptrs])
        stats = torch.empty(2, dtype=torch.float32, device=self.device)
        logp_new = torch.empty(B, self.cfg.n_actions, dtype=torch.float32, device=self.device)
        for t, name in ((logp_old, "logp_old"), (advantages, "advantages")):
            if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous fp32 device tensor")
        _check(self.lib.vla_ppo_lora_grads(self.handle, B, _ptr(vis), _ptr(prompt_ids),
                                           lens.ctypes.data_as(ctypes.c_void_p), _ptr(actions), _ptr(logp_old),
                                           _ptr(advantages), float(eps), float(temperature), ctypes.byref(lora),
                                           _ptr(self._train_ws), self._train_ws.numel(), _ptr(stats), _ptr(logp_new),
                                           _stream(self.device)))
        return stats, logp_new, grads

    def read_flags(self) -> int:
        v = ctypes.c_uint32()
        _check(self.lib.vla_read_device_flags(self.handle, _stream(self.device), ctypes.byref(v)))
        return v.value

    def profile_begin(self, categories=PROF_CATEGORIES) -> None:
        mask = 0
        for c in categories:
            mask |= 1 << PROF_CATEGORIES.index(c)
        _check(self.lib.vla_profile_begin(self.handle, mask))

    def profile_end(self) -> Dict[str, dict]:
        """Per category: summed kernel ms, summed algorithmic work (flops or
        bytes) and launch count of the launches recorded since profile_begin."""
        n = len(PROF_CATEGORIES)
        ms, work = (ctypes.c_double * n)(), (ctypes.c_double * n)()
        cnt = (ctypes.c_int64 * n)()
        _check(self.lib.vla_profile_end(self.handle, ms, work, cnt))
        return {c: {"ms": ms[i], "work": work[i], "launches": int(cnt[i])} for i, c in enumerate(PROF_CATEGORIES)}

    def debug_read(self, which: int, layer: int, out: torch.Tensor) -> torch.Tensor:
        _check(self.lib.vla_debug_read(self.handle, which, layer, _ptr(out), out.numel() * out.element_size(),
                                       _stream(self.device)))
        return out

    def debug_layer_limit(self, n_layers: int) -> None:
        _check(self.lib.vla_debug_set_layer_limit(self.handle, n_layers))

    def debug_decode_path(self, persistent: int) -> None:
        """0: one kernel per projection and consumer (default); 1: decode steps on the persistent layer
        kernel where the device allows (vla_debug.h)."""
        _check(self.lib.vla_debug_set_decode_path(self.handle, persistent))

    def debug_trace_decode_layer(self, layer: int, stamps: Optional[torch.Tensor]) -> None:
        _check(self.lib.vla_debug_trace_decode_layer(self.handle, layer, _ptr(stamps)))

    def debug_stop(self, stage: int) -> None:
        """Stop point inside the last layer of a layer-limited pass (vla_debug.h)."""
        _check(self.lib.vla_debug_set_stop(self.handle, stage))

    def close(self) -> None:
        if getattr(self, "handle", None):
            torch.cuda.current_stream(self.device).synchronize()
            self.lib.vla_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------------------ test hooks
def debug_pack_frag(X: torch.Tensor) -> torch.Tensor:
    """Row-major bf16 [R, K] -> frag layout (flat, ceil(R/16) * (K/32 + 1) * 512 elements; pad rows and
    the spare block of each 16-row block zero)."""
    lib = load_library()
    R, K = X.shape
    out = torch.zeros(((R + 15) // 16) * (K // 32 + 1) * 512, dtype=torch.bfloat16, device=X.device)
    _check(lib.vla_debug_pack_frag(_ptr(X), R, K, X.stride(0), _ptr(out), _stream(X.device)))
    return out


def debug_gemm(A: torch.Tensor, W: torch.Tensor) -> torch.Tensor:
    lib = load_library()
    M, K = A.shape
    N = W.shape[0]
    Af, Wf = debug_pack_frag(A), debug_pack_frag(W)
    C = torch.empty(M, N, dtype=torch.float32, device=A.device)
    _check(lib.vla_debug_gemm(_ptr(Af), _ptr(Wf), M, N, K, _ptr(C), _stream(A.device)))
    return C


def debug_skinny(A: torch.Tensor, W: torch.Tensor, workgroups: int = 256) -> torch.Tensor:
    lib = load_library()
    M, K = A.shape
    N = W.shape[0]
    Af, Wf = debug_pack_frag(A), debug_pack_frag(W)
    scratch = torch.empty(16 * M * N, dtype=torch.float32, device=A.device)
    C = torch.empty(M, N, dtype=torch.float32, device=A.device)
    _check(lib.vla_debug_skinny(_ptr(Af), _ptr(Wf), M, N, K, workgroups, _ptr(scratch), _ptr(C), _stream(A.device)))
    return C


def debug_sample(z: torch.Tensor, gumbel: torch.Tensor, step: int, temperature: float, action_begin: int):
    lib = load_library()
    B, A = z.shape
    na = gumbel.shape[1]
    dev = z.device
    tokens = torch.full((B, na), -1, dtype=torch.int32, device=dev)
    nxt = torch.empty(B, dtype=torch.int32, device=dev)
    logp = torch.full((B, na), float("nan"), dtype=torch.float32, device=dev)
    ent = torch.full((B, na), float("nan"), dtype=torch.float32, device=dev)
    logits = torch.zeros(B, na, A, dtype=torch.float32, device=dev)
    _check(lib.vla_debug_sample(_ptr(z), B, A, na, step, action_begin, _ptr(gumbel), float(temperature),
                                _ptr(tokens), _ptr(nxt), _ptr(logp), _ptr(ent), _ptr(logits), _stream(dev)))
    return {"tokens": tokens, "next": nxt, "logp": logp, "entropy": ent, "logits": logits}


def extract_actions(tokens: torch.Tensor, action_begin: int, bins: int, range_lo: torch.Tensor,
                    range_hi: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Continuous actions [n, n_dims] from action tokens (vla_extract_actions)."""
    lib = load_library()
    n, k = tokens.shape
    if tokens.dtype != torch.int32 or not tokens.is_cuda or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous int32 device tensor")
    for t in (range_lo, range_hi):
        if t.dtype != torch.float32 or not t.is_cuda or t.numel() != k:
            raise ValueError("ranges must be fp32 device tensors of n_dims entries")
    if out is None:
        out = torch.empty(n, k, dtype=torch.float32, device=tokens.device)
    _check(lib.vla_extract_actions(n, k, _ptr(tokens), int(action_begin), int(bins), _ptr(range_lo),
                                   _ptr(range_hi), _ptr(out), _stream(tokens.device)))
    return out


# ---------------------------------------------------------------- learning phase (vla_learn.h)
def _dev(t: torch.Tensor, dtype, name: str) -> torch.Tensor:
    if t.dtype != dtype or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} device tensor")
    return t


def gae(rewards: torch.Tensor, values: torch.Tensor, dones: torch.Tensor, gamma: float, lam: float,
        advantages: Optional[torch.Tensor] = None, returns: Optional[torch.Tensor] = None):
    """Advantages and returns [M, N] of Alg. 1's GAE step; rewards [M, N],
    values [M + 1, N] fp32, dones [M + 1, N] uint8 (vla_gae)."""
    lib = load_library()
    M, N = rewards.shape
    _dev(rewards, torch.float32, "rewards")
    _dev(values, torch.float32, "values")
    _dev(dones, torch.uint8, "dones")
    if tuple(values.shape) != (M + 1, N) or tuple(dones.shape) != (M + 1, N):
        raise ValueError("values and dones must be [M + 1, N]")
    if advantages is None:
        advantages = torch.empty(M, N, dtype=torch.float32, device=rewards.device)
    if returns is None:
        returns = torch.empty(M, N, dtype=torch.float32, device=rewards.device)
    _check(lib.vla_gae(N, M, _ptr(rewards), _ptr(values), _ptr(dones), float(gamma), float(lam), _ptr(advantages),
                       _ptr(returns), _stream(rewards.device)))
    return advantages, returns


def ppo_clip(logp_new: torch.Tensor, logp_old: torch.Tensor, advantages: torch.Tensor, eps: float,
             dlogp: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None):
    """(stats [loss, clipped fraction], dloss/dlogp_new [n, n_tokens]) of Eq. 2 (vla_ppo_clip)."""
    lib = load_library()
    n, k = logp_new.shape
    for t, name in ((logp_new, "logp_new"), (logp_old, "logp_old"), (advantages, "advantages")):
        _dev(t, torch.float32, name)
    if tuple(logp_old.shape) != (n, k) or tuple(advantages.shape) != (n,):
        raise ValueError("logp_old must be [n, n_tokens] and advantages [n]")
    if dlogp is None:
        dlogp = torch.empty(n, k, dtype=torch.float32, device=logp_new.device)
    if stats is None:
        stats = torch.empty(2, dtype=torch.float32, device=logp_new.device)
    _check(lib.vla_ppo_clip(n, k, _ptr(logp_new), _ptr(logp_old), _ptr(advantages), float(eps), _ptr(stats),
                            _ptr(dlogp), _stream(logp_new.device)))
    return stats, dlogp


def logprob_backward(logits: torch.Tensor, tokens: torch.Tensor, action_begin: int, temperature: float,
                     dlogp: torch.Tensor, dlogits: Optional[torch.Tensor] = None) -> torch.Tensor:
    """dlogits [rows, bins] of the token log-probabilities (vla_logprob_backward)."""
    lib = load_library()
    rows, bins = logits.shape
    _dev(logits, torch.float32, "logits")
    _dev(tokens, torch.int32, "tokens")
    _dev(dlogp, torch.float32, "dlogp")
    if tokens.numel() != rows or dlogp.numel() != rows:
        raise ValueError("tokens and dlogp need one entry per row")
    if dlogits is None:
        dlogits = torch.empty(rows, bins, dtype=torch.float32, device=logits.device)
    _check(lib.vla_logprob_backward(rows, bins, int(action_begin), _ptr(logits), _ptr(tokens), float(temperature),
                                    _ptr(dlogp), _ptr(dlogits), _stream(logits.device)))
    return dlogits
