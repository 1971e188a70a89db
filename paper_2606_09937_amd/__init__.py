"""Python binding of librksc, the MI355X (gfx950) RKSC library.

The functions named like the C ABI (rksc_verify_forward, rksc_prefill,
rksc_decode_step, rksc_asks_gate, ...) only marshal torch device tensors into
pointers and call the library; every step runs in the library's HIP kernels
(the block table and the KV probe are the library's host C++). torch is used
for device memory and streams only. If librksc.so is not built, every call
raises: there is no fallback path.

Convenience wrappers (verify_forward, prefill, Decoder, prefix_extend,
asks_similarity, asks_gate, cgee_gate, BlockTable, KVProbe) allocate outputs
and workspaces with torch and call the C ABI.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = [
    "RkscError", "load_library", "library_path",
    "rksc_abi_version", "rksc_verify_workspace_size", "rksc_verify_forward", "rksc_verify_window",
    "rksc_asks_similarity", "rksc_status_string", "rksc_last_error",
    "rksc_test_gemm", "rksc_test_gemm_kind", "rksc_test_gemm_live", "rksc_test_gemm_plan", "rksc_test_gate_up_swiglu", "rksc_test_attention",
    "verify_forward", "asks_similarity", "prefill", "rksc_prefill", "rksc_prefill_workspace_size", "model_config",
    "BranchCache", "Decoder", "rksc_decode_workspace_size", "rksc_decode_suffix", "rksc_decode_step",
    "rksc_cgee_gate", "cgee_gate", "RKSC_ABI_VERSION", "BlockTable", "KVProbe",
    "rksc_prefix_extend", "rksc_prefix_extend_workspace_size", "prefix_extend", "rksc_asks_gate", "asks_gate",
    "rksc_gate_up_tiled_bytes", "rksc_tile_gate_up", "tile_gate_up",
    "RKSC_OK", "RKSC_ERR_INVALID_ARGUMENT", "RKSC_ERR_UNSUPPORTED",
    "RKSC_ERR_WORKSPACE_TOO_SMALL", "RKSC_ERR_HIP", "RKSC_F32", "RKSC_BF16", "RKSC_MAX_BRANCHES",
    "RKSC_MAX_PREFIX_SEGMENTS", "PrefixCache", "PrefixKV",
]

RKSC_OK = 0
RKSC_ERR_INVALID_ARGUMENT = -1
RKSC_ERR_UNSUPPORTED = -2
RKSC_ERR_WORKSPACE_TOO_SMALL = -3
RKSC_ERR_HIP = -4
RKSC_F32 = 0
RKSC_BF16 = 1
RKSC_MAX_BRANCHES = 64
RKSC_MAX_PREFIX_SEGMENTS = 8
RKSC_ABI_VERSION = 8

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_PKG_DIR, "librksc.so")


class RkscError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"rksc status {status}: {message}")
        self.status = status


class ModelConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
        ("dtype", ctypes.c_int32),
    ]


class LayerWeights(ctypes.Structure):
    _fields_ = [
        ("attn_norm", ctypes.c_void_p), ("w_qkv", ctypes.c_void_p), ("w_o", ctypes.c_void_p),
        ("ffn_norm", ctypes.c_void_p), ("w_gate_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p),
        ("w_gate_up_tiled", ctypes.c_void_p),
    ]


class Weights(ctypes.Structure):
    _fields_ = [
        ("cfg", ModelConfig), ("embed", ctypes.c_void_p), ("layers", ctypes.POINTER(LayerWeights)),
        ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
    ]


class PrefixKV(ctypes.Structure):
    pass


PrefixKV._fields_ = [("n_prefix", ctypes.c_int32), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                     ("parent", ctypes.POINTER(PrefixKV))]


class PrefixCache:
    """A shared prefix made of caches in position order (tree sharing, Sec. 2.2): segments
    [(k, v), ...], each [L, Hkv, n_i, hd] in the model dtype, the root's first. Pass it as
    `prefix_k` (with prefix_v None) wherever a prefix cache is taken; the library reads the
    segments in place as one prefix of n_prefix = sum n_i entries."""

    def __init__(self, segments):
        self.segments = [(k, v) for k, v in segments]

    @property
    def n_prefix(self) -> int:
        return sum(int(k.shape[2]) for k, _ in self.segments)

    def extend(self, k, v) -> "PrefixCache":
        """The prefix of a search-tree node's children: these segments, then the node's own cache."""
        return PrefixCache(self.segments + [(k, v)])


class BranchKVStruct(ctypes.Structure):
    _fields_ = [("capacity", ctypes.c_int32), ("length", ctypes.c_int32), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p)]


_lib = None


def load_library():
    """Load librksc.so from the package directory (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2606_09937_amd.build` "
            "(the verify pass has no non-HIP implementation)")
    lib = ctypes.CDLL(path)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    lib.rksc_abi_version.restype = i32
    lib.rksc_abi_version.argtypes = []
    lib.rksc_gate_up_tiled_bytes.restype = sz
    lib.rksc_gate_up_tiled_bytes.argtypes = [ctypes.POINTER(ModelConfig)]
    lib.rksc_tile_gate_up.restype = i32
    lib.rksc_tile_gate_up.argtypes = [ctypes.POINTER(ModelConfig), vp, vp, sz, vp]
    lib.rksc_verify_workspace_size.restype = sz
    lib.rksc_verify_workspace_size.argtypes = [ctypes.POINTER(ModelConfig), i32, i32, i32]
    lib.rksc_verify_forward.restype = i32
    lib.rksc_verify_forward.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV), vp, i32, i32, f32, i32,
                                        vp, vp, vp, vp, sz, vp]
    lib.rksc_verify_forward_noalloc.restype = i32
    lib.rksc_verify_forward_noalloc.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV), vp, i32, i32,
                                                f32, i32, vp, vp, vp, vp]
    lib.rksc_test_verify_precision.restype = i32
    lib.rksc_test_verify_precision.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV), vp, i32, i32, f32,
                                               i32, vp, vp, vp, vp, sz, vp, ctypes.c_uint32]
    lib.rksc_verify_window.restype = i32
    lib.rksc_verify_window.argtypes = [ctypes.POINTER(ModelConfig), i32, i32, i32]
    lib.rksc_verify_forward_window.restype = i32
    lib.rksc_verify_forward_window.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV), vp, i32, i32, f32,
                                               i32, vp, vp, vp, vp, sz, vp, i32]
    lib.rksc_prefill_workspace_size.restype = sz
    lib.rksc_prefill_workspace_size.argtypes = [ctypes.POINTER(ModelConfig), i32]
    lib.rksc_prefill.restype = i32
    lib.rksc_prefill.argtypes = [ctypes.POINTER(Weights), vp, i32, vp, vp, vp, vp, sz, vp]
    lib.rksc_decode_workspace_size.restype = sz
    lib.rksc_decode_workspace_size.argtypes = [ctypes.POINTER(ModelConfig), i32, i32, i32]
    lib.rksc_decode_suffix.restype = i32
    lib.rksc_decode_suffix.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV),
                                       ctypes.POINTER(BranchKVStruct), vp, i32, i32, vp, vp, vp, vp, sz, vp]
    lib.rksc_decode_step.restype = i32
    lib.rksc_decode_step.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV),
                                     ctypes.POINTER(BranchKVStruct), vp, i32, vp, vp, vp, vp, sz, vp]
    lib.rksc_prefix_extend_workspace_size.restype = sz
    lib.rksc_prefix_extend_workspace_size.argtypes = [ctypes.POINTER(ModelConfig), i32, i32]
    lib.rksc_prefix_extend.restype = i32
    lib.rksc_prefix_extend.argtypes = [ctypes.POINTER(Weights), ctypes.POINTER(PrefixKV), vp, i32, vp, vp, vp, vp,
                                       sz, vp]
    lib.rksc_asks_gate.restype = i32
    lib.rksc_asks_gate.argtypes = [vp, vp, i32, i32, i32, f32, f32, vp, vp, vp]
    lib.rksc_cgee_gate.restype = i32
    lib.rksc_cgee_gate.argtypes = [vp, i32, i32, f32, f32, vp, vp, vp, vp, vp]
    i64 = ctypes.c_int64
    lib.rksc_block_table_create.restype = vp
    lib.rksc_block_table_create.argtypes = [i32]
    lib.rksc_block_table_destroy.restype = None
    lib.rksc_block_table_destroy.argtypes = [vp]
    lib.rksc_block_table_insert.restype = i32
    lib.rksc_block_table_insert.argtypes = [vp, i64, f32, i32]
    lib.rksc_block_table_set_score.restype = i32
    lib.rksc_block_table_set_score.argtypes = [vp, i64, f32]
    lib.rksc_block_table_remove.restype = i32
    lib.rksc_block_table_remove.argtypes = [vp, i64]
    lib.rksc_block_table_evict.restype = i32
    lib.rksc_block_table_evict.argtypes = [vp, ctypes.POINTER(i64), i32, ctypes.POINTER(i32)]
    lib.rksc_block_table_size.restype = i32
    lib.rksc_block_table_size.argtypes = [vp]
    lib.rksc_block_table_evicted_total.restype = i64
    lib.rksc_block_table_evicted_total.argtypes = [vp]
    lib.rksc_kv_probe_create.restype = vp
    lib.rksc_kv_probe_create.argtypes = [i32]
    lib.rksc_kv_probe_destroy.restype = None
    lib.rksc_kv_probe_destroy.argtypes = [vp]
    lib.rksc_kv_probe_workspace_size.restype = sz
    lib.rksc_kv_probe_workspace_size.argtypes = [ctypes.POINTER(ModelConfig), i32, i32, i32]
    lib.rksc_kv_probe_decide.restype = i32
    lib.rksc_kv_probe_decide.argtypes = [vp, ctypes.POINTER(Weights), vp, i32, vp, i32, i32, vp, sz, vp,
                                         ctypes.POINTER(i32), ctypes.POINTER(f32), ctypes.POINTER(i32)]
    lib.rksc_kv_probe_lookup.restype = i32
    lib.rksc_kv_probe_lookup.argtypes = [vp, i32, ctypes.POINTER(i32), ctypes.POINTER(f32)]
    lib.rksc_asks_similarity.restype = i32
    lib.rksc_asks_similarity.argtypes = [vp, i32, i32, i32, f32, vp, vp]
    lib.rksc_status_string.restype = ctypes.c_char_p
    lib.rksc_status_string.argtypes = [i32]
    lib.rksc_last_error.restype = ctypes.c_char_p
    lib.rksc_last_error.argtypes = []
    lib.rksc_test_gemm.restype = i32
    lib.rksc_test_gemm.argtypes = [i32, vp, vp, vp, vp, i32, i32, i32, i32, ctypes.POINTER(i32), vp]
    lib.rksc_test_gemm_kind.restype = i32
    lib.rksc_test_gemm_kind.argtypes = [i32, vp, vp, vp, vp, i32, i32, i32, i32, i32, ctypes.POINTER(i32), vp]
    lib.rksc_test_gemm_live.restype = i32
    lib.rksc_test_gemm_live.argtypes = [i32, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp,
                                        ctypes.POINTER(i32), vp]
    lib.rksc_test_gate_up_swiglu.restype = i32
    lib.rksc_test_gate_up_swiglu.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, vp]
    lib.rksc_test_gemm_plan.restype = i32
    lib.rksc_test_gemm_plan.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(i32)]
    lib.rksc_test_attention.restype = i32
    lib.rksc_test_attention_scratch_size.restype = sz
    lib.rksc_test_attention_scratch_size.argtypes = [i32, i32, i32, i32, i32, i32, i32]
    lib.rksc_test_attention.argtypes = [i32, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, sz, vp]
    _lib = lib
    return lib


def _check(status: int):
    if status != RKSC_OK:
        lib = load_library()
        raise RkscError(status, lib.rksc_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to librksc must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


class _Args:
    """Argument checks before pointers are handed to the library: every tensor's
    dtype and shape (None entries match any size) first, then, in done(), that
    all of them live on a GPU. Raises ValueError naming the argument."""

    def __init__(self):
        self._seen = []

    def __call__(self, t, name: str, dtype=None, shape=None, ndim: Optional[int] = None):
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name} must be a torch tensor (got {type(t).__name__})")
        if dtype is not None and t.dtype != dtype:
            raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
        if ndim is not None and t.dim() != ndim:
            raise ValueError(f"{name} must have {ndim} dimensions (got shape {tuple(t.shape)})")
        if shape is not None:
            if t.dim() != len(shape) or any(w is not None and int(g) != int(w) for g, w in zip(t.shape, shape)):
                want = "[" + ", ".join("*" if w is None else str(w) for w in shape) + "]"
                raise ValueError(f"{name} must have shape {want} (got {list(t.shape)})")
        self._seen.append((name, t))
        return t

    def done(self):
        for name, t in self._seen:
            if not t.is_cuda:
                raise ValueError(f"{name} must be a GPU tensor (got device {t.device})")


def _model_dtype(shape):
    return torch.bfloat16 if shape.dtype == "bf16" else torch.float32


def _check_weights(need, weights, need_lm_head: bool = True):
    """Every weight tensor of the decoder: model dtype (fp32 gains), torch Linear shapes."""
    shape = weights.shape
    dt = _model_dtype(shape)
    d, F, V = shape.d_model, shape.d_ff, shape.vocab
    H, Hkv, hd = shape.n_heads, shape.n_kv_heads, shape.head_dim
    need(weights.embed, "embed", dt, (V, d))
    need(weights.final_norm, "final_norm", torch.float32, (d,))
    if need_lm_head or weights.lm_head is not None:
        need(weights.lm_head, "lm_head", dt, (V, d))
    for i, lw in enumerate(weights.layers):
        need(lw["attn_norm"], f"layer {i} attn_norm", torch.float32, (d,))
        need(lw["ffn_norm"], f"layer {i} ffn_norm", torch.float32, (d,))
        need(lw["w_qkv"], f"layer {i} w_qkv", dt, ((H + 2 * Hkv) * hd, d))
        need(lw["w_o"], f"layer {i} w_o", dt, (d, H * hd))
        need(lw["w_gate_up"], f"layer {i} w_gate_up", dt, (2 * F, d))
        need(lw["w_down"], f"layer {i} w_down", dt, (d, F))
        if lw.get("w_gate_up_tiled") is not None:
            need(lw["w_gate_up_tiled"], f"layer {i} w_gate_up_tiled", dt, (2 * F, d))


def _check_prefix(need, weights, prefix_k, prefix_v, name="prefix"):
    """The shared prefix: a cache [L, Hkv, n, hd] in the model dtype (k and v), a PrefixCache of such
    segments (in prefix_k, prefix_v None), or nothing (both None). Returns the total n."""
    if prefix_k is None and prefix_v is None:
        return 0
    if isinstance(prefix_k, PrefixCache):
        if prefix_v is not None:
            raise ValueError(f"{name}: pass a PrefixCache as {name}_k with {name}_v None")
        if len(prefix_k.segments) > RKSC_MAX_PREFIX_SEGMENTS:
            raise ValueError(f"{name}: at most {RKSC_MAX_PREFIX_SEGMENTS} segments")
        return sum(_check_prefix(need, weights, k, v, f"{name} segment {i}")
                   for i, (k, v) in enumerate(prefix_k.segments))
    shape = weights.shape
    dims = (len(weights.layers), shape.n_kv_heads, None, shape.head_dim)
    need(prefix_k, f"{name}_k", _model_dtype(shape), dims)
    n = int(prefix_k.shape[2])
    need(prefix_v, f"{name}_v", _model_dtype(shape), dims[:2] + (n, dims[3]))
    return n


def _prefix_len(prefix_k) -> int:
    """Entries of a prefix: a cache tensor, a PrefixCache or None."""
    if prefix_k is None:
        return 0
    if isinstance(prefix_k, PrefixCache):
        return prefix_k.n_prefix
    return int(prefix_k.shape[2])


def _prefix_struct(prefix_k, prefix_v):
    """rksc_prefix_kv of the prefix (a chain for a PrefixCache); returns (struct, objects to keep)."""
    if not isinstance(prefix_k, PrefixCache):
        kv = PrefixKV(_prefix_len(prefix_k), _ptr(prefix_k), _ptr(prefix_v))
        return kv, [kv]
    keep, prev = [], None
    for k, v in prefix_k.segments:
        kv = PrefixKV(int(k.shape[2]), _ptr(k), _ptr(v))
        if prev is not None:
            kv.parent = ctypes.pointer(prev)
        keep.append(kv)
        prev = kv
    if prev is None:
        prev = PrefixKV(0, None, None)
        keep.append(prev)
    return prev, keep


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def model_config(shape) -> ModelConfig:
    """C config from any object with the decoder shape attributes (e.g. workloads.ModelShape)."""
    return ModelConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                       shape.d_ff, shape.vocab, float(shape.rms_eps), float(shape.rope_base),
                       RKSC_BF16 if shape.dtype == "bf16" else RKSC_F32)


def rksc_abi_version() -> int:
    return int(load_library().rksc_abi_version())


def rksc_status_string(status: int) -> str:
    return load_library().rksc_status_string(status).decode()


def rksc_last_error() -> str:
    return load_library().rksc_last_error().decode()


def rksc_verify_workspace_size(shape, n_branches: int, branch_len: int, n_prefix: int) -> int:
    cfg = model_config(shape)
    n = int(load_library().rksc_verify_workspace_size(ctypes.byref(cfg), n_branches, branch_len, n_prefix))
    if n == 0:
        raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())
    return n


def _weights_struct(weights):
    shape = weights.shape
    layers = (LayerWeights * len(weights.layers))()
    for i, lw in enumerate(weights.layers):
        layers[i] = LayerWeights(_ptr(lw["attn_norm"]), _ptr(lw["w_qkv"]), _ptr(lw["w_o"]), _ptr(lw["ffn_norm"]),
                                 _ptr(lw["w_gate_up"]), _ptr(lw["w_down"]), _ptr(lw.get("w_gate_up_tiled")))
    cfg = model_config(shape)
    cfg.n_layers = len(weights.layers)
    w = Weights(cfg, _ptr(weights.embed), layers, _ptr(weights.final_norm), _ptr(weights.lm_head))
    return w, layers


def rksc_verify_window(shape, n_branches: int, branch_len: int, n_prefix: int) -> int:
    """The exit window rksc_verify_forward takes for this pass (a cost model of the schedule)."""
    cfg = model_config(shape)
    w = int(load_library().rksc_verify_window(ctypes.byref(cfg), int(n_branches), int(branch_len), int(n_prefix)))
    if w == 0:
        raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())
    return w


def rksc_verify_forward(weights, prefix_k, prefix_v, branch_tokens, tau: float, patience: int,
                        entropy: torch.Tensor, exit_layer: torch.Tensor, hidden_last: Optional[torch.Tensor],
                        workspace: torch.Tensor, stream=None, window: Optional[int] = None) -> None:
    """Marshal torch device tensors into rksc_verify_forward (asynchronous on `stream`);
    with `window`, into rksc_verify_forward_window.

    weights: object with .shape (decoder shape), .embed, .layers (dicts of tensors), .final_norm, .lm_head.
    prefix_k/prefix_v: [L, Hkv, n, hd] device tensors. branch_tokens: [B, s] int32 device.
    """
    need = _Args()
    _check_weights(need, weights)
    n = _check_prefix(need, weights, prefix_k, prefix_v)
    need(branch_tokens, "branch_tokens", torch.int32, ndim=2)
    B, s = branch_tokens.shape
    L, d = len(weights.layers), weights.shape.d_model
    need(entropy, "entropy", torch.float32, (L, B))
    need(exit_layer, "exit_layer", torch.int32, (B,))
    if hidden_last is not None:
        need(hidden_last, "hidden_last", torch.float32, (L, B, d))
    need(workspace, "workspace", torch.uint8, ndim=1)
    need.done()
    lib = load_library()
    w, layers_keepalive = _weights_struct(weights)
    kv, kv_keep = _prefix_struct(prefix_k, prefix_v)
    args = (ctypes.byref(w), ctypes.byref(kv), _ptr(branch_tokens), int(B), int(s), float(tau), int(patience),
            _ptr(entropy), _ptr(exit_layer), _ptr(hidden_last), _ptr(workspace),
            int(workspace.numel() * workspace.element_size()), _stream(stream))
    if window is None:
        st = lib.rksc_verify_forward(*args)
    else:
        st = lib.rksc_verify_forward_window(*args, int(window))
    del layers_keepalive
    _check(st)


RKSC_NOALLOC_SCRATCH_BYTES = 128 << 20


def rksc_verify_forward_noalloc(weights, prefix_k, prefix_v, branch_tokens, tau: float, patience: int,
                                entropy: torch.Tensor, exit_layer: torch.Tensor,
                                hidden_last: Optional[torch.Tensor], stream=None) -> None:
    """Marshal torch device tensors into rksc_verify_forward_noalloc (the verify pass on the
    library's own device array of RKSC_NOALLOC_SCRATCH_BYTES; no workspace argument)."""
    need = _Args()
    _check_weights(need, weights)
    n = _check_prefix(need, weights, prefix_k, prefix_v)
    need(branch_tokens, "branch_tokens", torch.int32, ndim=2)
    B, s = branch_tokens.shape
    L, d = len(weights.layers), weights.shape.d_model
    need(entropy, "entropy", torch.float32, (L, B))
    need(exit_layer, "exit_layer", torch.int32, (B,))
    if hidden_last is not None:
        need(hidden_last, "hidden_last", torch.float32, (L, B, d))
    need.done()
    lib = load_library()
    w, layers_keepalive = _weights_struct(weights)
    kv, kv_keep = _prefix_struct(prefix_k, prefix_v)
    st = lib.rksc_verify_forward_noalloc(ctypes.byref(w), ctypes.byref(kv), _ptr(branch_tokens), int(B), int(s),
                                         float(tau), int(patience), _ptr(entropy), _ptr(exit_layer),
                                         _ptr(hidden_last), _stream(stream))
    del layers_keepalive
    _check(st)


# Operand sites of the precision ablation (rksc_test_verify_precision).
RKSC_DROP = {"qkv": 0x01, "o": 0x02, "gate_up": 0x04, "down": 0x08, "q": 0x10, "own_kv": 0x20, "p": 0x40,
             "lm_head": 0x80}


def rksc_test_verify_precision(weights, prefix_k, prefix_v, branch_tokens, tau: float, patience: int,
                               drop_mask: int, stream=None):
    """The verify pass with the chosen operand sites at bf16 precision (RKSC_DROP bits); returns
    (entropy [L, B], exit_layer [B], hidden_last [L, B, d]) device tensors."""
    need = _Args()
    _check_weights(need, weights)
    n = _check_prefix(need, weights, prefix_k, prefix_v)
    need(branch_tokens, "branch_tokens", torch.int32, ndim=2)
    need.done()
    B, s = branch_tokens.shape
    L, d, dev = len(weights.layers), weights.shape.d_model, branch_tokens.device
    ws = torch.empty(rksc_verify_workspace_size(weights.shape, B, s, n), dtype=torch.uint8, device=dev)
    ent = torch.empty((L, B), dtype=torch.float32, device=dev)
    ex = torch.empty((B,), dtype=torch.int32, device=dev)
    hid = torch.empty((L, B, d), dtype=torch.float32, device=dev)
    w, keep = _weights_struct(weights)
    kv, kv_keep = _prefix_struct(prefix_k, prefix_v)
    _check(load_library().rksc_test_verify_precision(ctypes.byref(w), ctypes.byref(kv), _ptr(branch_tokens), int(B),
                                                     int(s), float(tau), int(patience), _ptr(ent), _ptr(ex),
                                                     _ptr(hid), _ptr(ws), ws.numel(), _stream(stream),
                                                     int(drop_mask)))
    del keep
    return ent, ex, hid


def rksc_prefill_workspace_size(shape, n_prefix: int) -> int:
    cfg = model_config(shape)
    n = int(load_library().rksc_prefill_workspace_size(ctypes.byref(cfg), n_prefix))
    if n == 0:
        raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())
    return n


def rksc_prefill(weights, tokens: torch.Tensor, k_out: torch.Tensor, v_out: torch.Tensor, h_root: torch.Tensor,
                 workspace: torch.Tensor, stream=None) -> None:
    """Marshal torch device tensors into rksc_prefill (asynchronous on `stream`).

    tokens [n] int32 device; k_out/v_out [L, Hkv, n, hd] of the model dtype; h_root [L, d] fp32.
    """
    need = _Args()
    _check_weights(need, weights, need_lm_head=False)
    need(tokens, "tokens", torch.int32, ndim=1)
    n, L = int(tokens.numel()), len(weights.layers)
    shape = weights.shape
    dims = (L, shape.n_kv_heads, n, shape.head_dim)
    need(k_out, "k_out", _model_dtype(shape), dims)
    need(v_out, "v_out", _model_dtype(shape), dims)
    need(h_root, "h_root", torch.float32, (L, shape.d_model))
    need(workspace, "workspace", torch.uint8, ndim=1)
    need.done()
    lib = load_library()
    w, layers_keepalive = _weights_struct(weights)
    st = lib.rksc_prefill(ctypes.byref(w), _ptr(tokens), int(tokens.numel()), _ptr(k_out), _ptr(v_out),
                          _ptr(h_root), _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                          _stream(stream))
    del layers_keepalive
    _check(st)


def rksc_asks_similarity(hidden: torch.Tensor, alpha: float, S: torch.Tensor, stream=None) -> None:
    """Marshal hidden [L, B, d] fp32 and S [B, B] fp32 device tensors into rksc_asks_similarity."""
    need = _Args()
    need(hidden, "hidden", torch.float32, ndim=3)
    L, B, d = hidden.shape
    need(S, "S", torch.float32, (B, B))
    need.done()
    _check(load_library().rksc_asks_similarity(_ptr(hidden), int(L), int(B), int(d), float(alpha), _ptr(S),
                                               _stream(stream)))


def rksc_test_gemm_plan(M: int, N: int, K: int, bf16: bool = True, splits: int = 0, kind: int = -1) -> dict:
    """The GEMM plan of rksc_test_gemm for this shape (host only, nothing is launched)."""
    plan = (ctypes.c_int32 * 5)()
    _check(load_library().rksc_test_gemm_plan(RKSC_BF16 if bf16 else RKSC_F32, M, N, K, splits, kind, plan))
    return dict(zip(("kind", "bm", "bn", "splits", "k_per_split"), list(plan)))


def rksc_test_gemm(A, W: torch.Tensor, splits: int = 0, stream=None, kind: int = -1):
    """Kernel-level GEMM: returns the fp32 split partials [splits_used, M, N].

    bf16 W: A is the pair (A_hi, A_lo) of bf16 [M, K] planes; fp32 W: A is an fp32 [M, K] tensor.
    kind: -1 the library's choice, 0 the 128-row-tile kernel, 1 the 256 x 256-tile kernel, 2 the
    weight-streaming kernel for at most 32 rows (kinds 1 and 2 bf16 only).
    """
    if W.dtype == torch.bfloat16:
        a_hi, a_lo = A
        dt = RKSC_BF16
    else:
        a_hi, a_lo = A, None
        dt = RKSC_F32
    need = _Args()
    need(a_hi, "A", W.dtype, ndim=2)
    M, K = a_hi.shape
    if a_lo is not None:
        need(a_lo, "A_lo", torch.bfloat16, (M, K))
    need(W, "W", None, (None, K))
    need.done()
    N = W.shape[0]
    P = torch.empty((8, M, N), dtype=torch.float32, device=a_hi.device)
    used = ctypes.c_int32(0)
    _check(load_library().rksc_test_gemm_kind(dt, _ptr(a_hi), _ptr(a_lo), _ptr(W), _ptr(P), M, N, K, splits,
                                              kind, ctypes.byref(used), _stream(stream)))
    return P[: used.value]


def rksc_test_gemm_live(A, W: torch.Tensor, live_count: int, branch_len: int, P: torch.Tensor, splits: int = 0,
                        kind: int = -1, stream=None) -> int:
    """rksc_test_gemm_kind with only live_count * branch_len of the M rows live (a control block
    as after branch exits). P [8, M, N] fp32 is written in the live rows only; returns the
    number of splits used."""
    if W.dtype == torch.bfloat16:
        a_hi, a_lo = A
        dt = RKSC_BF16
    else:
        a_hi, a_lo = A, None
        dt = RKSC_F32
    need = _Args()
    need(a_hi, "A", W.dtype, ndim=2)
    M, K = a_hi.shape
    if a_lo is not None:
        need(a_lo, "A_lo", torch.bfloat16, (M, K))
    need(W, "W", None, (None, K))
    N = W.shape[0]
    need(P, "P", torch.float32, (8, M, N))
    need.done()
    ctrl = torch.empty(4096, dtype=torch.uint8, device=a_hi.device)
    used = ctypes.c_int32(0)
    _check(load_library().rksc_test_gemm_live(dt, _ptr(a_hi), _ptr(a_lo), _ptr(W), _ptr(P), M, N, K, splits, kind,
                                              int(live_count), int(branch_len), _ptr(ctrl), ctypes.byref(used),
                                              _stream(stream)))
    return used.value


def rksc_test_gate_up_swiglu(A, W: torch.Tensor, fused: bool, stream=None) -> torch.Tensor:
    """The gate|up projection and its SwiGLU through the library's kernels: A = (hi, lo) bf16 planes
    [M, K], W [2F, K] bf16. Returns a = silu(gate) * up [M, F] as fp32 (hi + lo of the output planes)."""
    a_hi, a_lo = A
    need = _Args()
    need(a_hi, "A", torch.bfloat16, ndim=2)
    M, K = a_hi.shape
    need(a_lo, "A_lo", torch.bfloat16, (M, K))
    need(W, "W", torch.bfloat16, (None, K))
    need.done()
    F = int(W.shape[0]) // 2
    out = torch.empty((2, M, F), dtype=torch.bfloat16, device=a_hi.device)
    P = torch.empty((8, M, 2 * F), dtype=torch.float32, device=a_hi.device)
    _check(load_library().rksc_test_gate_up_swiglu(_ptr(a_hi), _ptr(a_lo), _ptr(W), _ptr(out), _ptr(P), M, F, K,
                                                   1 if fused else 0, _stream(stream)))
    return out[0].float() + out[1].float()


def rksc_test_attention(q, prefix_k, prefix_v, k_own, v_own, dtype, stream=None):
    """Kernel-level shared-prefix attention: q [B*s, H, hd], own [B, Hkv, s, hd] fp32; prefix [Hkv, n, hd]
    of `dtype` (torch.bfloat16 or torch.float32). Returns o [B*s, H*hd] as fp32 (bf16 hi/lo planes are
    recombined here for the bf16 path)."""
    need = _Args()
    need(q, "q", torch.float32, ndim=3)
    Ms, H, hd = q.shape
    need(k_own, "k_own", torch.float32, ndim=4)
    B, Hkv, s, _ = k_own.shape
    need(k_own, "k_own", torch.float32, (B, Hkv, s, hd))
    need(v_own, "v_own", torch.float32, (B, Hkv, s, hd))
    n = 0
    if prefix_k is not None:
        need(prefix_k, "prefix_k", dtype, (Hkv, None, hd))
        n = int(prefix_k.shape[1])
        need(prefix_v, "prefix_v", dtype, (Hkv, n, hd))
    need.done()
    dt = RKSC_BF16 if dtype == torch.bfloat16 else RKSC_F32
    o = torch.empty((Ms, H * hd), dtype=torch.float32, device=q.device)
    lib = load_library()
    nbytes = int(lib.rksc_test_attention_scratch_size(dt, B, n, s, H, Hkv, hd))
    scratch = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    _check(lib.rksc_test_attention(dt, _ptr(q), _ptr(prefix_k), _ptr(prefix_v), _ptr(k_own), _ptr(v_own), _ptr(o),
                                   B, n, s, H, Hkv, hd, _ptr(scratch), nbytes, _stream(stream)))
    if dt == RKSC_BF16:
        planes = o.view(torch.bfloat16).view(2, Ms, H * hd)
        return planes[0].float() + planes[1].float()
    return o


def verify_forward(weights, prefix_k, prefix_v, branch_tokens, tau: float, patience: int,
                   return_hidden: bool = False, workspace: Optional[torch.Tensor] = None, stream=None,
                   window: Optional[int] = None):
    """Allocate outputs (and the workspace unless given) and run the verify pass.

    Returns (entropy [L, B] fp32, exit_layer [B] int32[, hidden_last [L, B, d] fp32]) on the device.
    """
    shape = weights.shape
    B, s = branch_tokens.shape
    dev = branch_tokens.device
    L = len(weights.layers)
    if workspace is None:
        n_prefix = _prefix_len(prefix_k)
        workspace = torch.empty(rksc_verify_workspace_size(shape, B, s, n_prefix), dtype=torch.uint8, device=dev)
    entropy = torch.empty((L, B), dtype=torch.float32, device=dev)
    exit_layer = torch.empty((B,), dtype=torch.int32, device=dev)
    hidden = torch.empty((L, B, shape.d_model), dtype=torch.float32, device=dev) if return_hidden else None
    rksc_verify_forward(weights, prefix_k, prefix_v, branch_tokens, tau, patience, entropy, exit_layer, hidden,
                        workspace, stream, window)
    return (entropy, exit_layer, hidden) if return_hidden else (entropy, exit_layer)


def prefill(weights, tokens: torch.Tensor, workspace: Optional[torch.Tensor] = None, stream=None):
    """Allocate the cache and root rows (and the workspace unless given) and run the root forward.

    Returns (k [L, Hkv, n, hd], v [L, Hkv, n, hd] of the model dtype, h_root [L, d] fp32 unit rows).
    """
    shape = weights.shape
    n = int(tokens.numel())
    dev = tokens.device
    L = len(weights.layers)
    dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    if workspace is None:
        workspace = torch.empty(rksc_prefill_workspace_size(shape, n), dtype=torch.uint8, device=dev)
    k = torch.empty((L, shape.n_kv_heads, n, shape.head_dim), dtype=dtype, device=dev)
    v = torch.empty_like(k)
    h_root = torch.empty((L, shape.d_model), dtype=torch.float32, device=dev)
    rksc_prefill(weights, tokens.contiguous(), k, v, h_root, workspace, stream)
    return k, v, h_root


def rksc_gate_up_tiled_bytes(shape) -> int:
    """Bytes of one layer's tiled gate|up copy; 0 if the model has no tiled layout."""
    return int(load_library().rksc_gate_up_tiled_bytes(ctypes.byref(model_config(shape))))


def rksc_tile_gate_up(shape, w_gate_up: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """Marshal one layer's gate|up weight [2F, d] and an output tensor of the same shape and dtype
    (device) into rksc_tile_gate_up."""
    need = _Args()
    dt = _model_dtype(shape)
    need(w_gate_up, "w_gate_up", dt, (2 * shape.d_ff, shape.d_model))
    need(out, "out", dt, (2 * shape.d_ff, shape.d_model))
    need.done()
    _check(load_library().rksc_tile_gate_up(ctypes.byref(model_config(shape)), _ptr(w_gate_up), _ptr(out),
                                            int(out.numel() * out.element_size()), _stream(stream)))


def tile_gate_up(weights, stream=None) -> bool:
    """Give every layer of `weights` its tiled gate|up copy (layer dict key "w_gate_up_tiled"), which
    the library then streams instead of w_gate_up where the 128-row projection tiles run; the outputs
    do not change. Returns False (and changes nothing) for a model without a tiled layout."""
    if rksc_gate_up_tiled_bytes(weights.shape) == 0:
        return False
    for lw in weights.layers:
        out = torch.empty_like(lw["w_gate_up"])
        rksc_tile_gate_up(weights.shape, lw["w_gate_up"], out, stream)
        lw["w_gate_up_tiled"] = out
    return True


def asks_similarity(hidden: torch.Tensor, alpha: float, stream=None) -> torch.Tensor:
    L, B, d = hidden.shape
    S = torch.empty((B, B), dtype=torch.float32, device=hidden.device)
    rksc_asks_similarity(hidden, alpha, S, stream)
    return S


class BranchCache:
    """A branch set's own K/V cache ([L, B, Hkv, capacity, hd] device tensors of the
    model dtype) and the rksc_branch_kv struct whose `length` the decode calls advance."""

    def __init__(self, shape, n_layers: int, n_branches: int, capacity: int, device):
        dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        dims = (n_layers, n_branches, shape.n_kv_heads, capacity, shape.head_dim)
        self.k = torch.zeros(dims, dtype=dtype, device=device)
        self.v = torch.zeros(dims, dtype=dtype, device=device)
        self.n_branches = n_branches
        self.struct = BranchKVStruct(int(capacity), 0, _ptr(self.k), _ptr(self.v))

    @property
    def length(self) -> int:
        return int(self.struct.length)

    @property
    def capacity(self) -> int:
        return int(self.struct.capacity)


def rksc_decode_workspace_size(shape, n_branches: int, suffix_len: int, n_prefix: int) -> int:
    cfg = model_config(shape)
    n = int(load_library().rksc_decode_workspace_size(ctypes.byref(cfg), n_branches, suffix_len, n_prefix))
    if n == 0:
        raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())
    return n


def _check_decode_outputs(need, weights, cache, B, next_token, p_top, conf, workspace):
    shape = weights.shape
    dims = (len(weights.layers), B, shape.n_kv_heads, cache.capacity, shape.head_dim)
    need(cache.k, "branch cache k", _model_dtype(shape), dims)
    need(cache.v, "branch cache v", _model_dtype(shape), dims)
    need(next_token, "next_token", torch.int32, (B,))
    need(p_top, "p_top", torch.float32, (B,))
    need(conf, "conf", torch.float32, (B,))
    need(workspace, "workspace", torch.uint8, ndim=1)
    need.done()


def rksc_decode_suffix(weights, prefix_k, prefix_v, cache: BranchCache, suffix_tokens: torch.Tensor,
                       next_token: torch.Tensor, p_top: torch.Tensor, conf: torch.Tensor, workspace: torch.Tensor,
                       stream=None) -> None:
    """Marshal torch device tensors into rksc_decode_suffix (asynchronous on `stream`)."""
    need = _Args()
    _check_weights(need, weights)
    n = _check_prefix(need, weights, prefix_k, prefix_v)
    need(suffix_tokens, "suffix_tokens", torch.int32, ndim=2)
    B, s = suffix_tokens.shape
    _check_decode_outputs(need, weights, cache, B, next_token, p_top, conf, workspace)
    lib = load_library()
    w, layers_keepalive = _weights_struct(weights)
    kv, kv_keep = _prefix_struct(prefix_k, prefix_v)
    st = lib.rksc_decode_suffix(ctypes.byref(w), ctypes.byref(kv), ctypes.byref(cache.struct), _ptr(suffix_tokens),
                                int(B), int(s), _ptr(next_token), _ptr(p_top), _ptr(conf), _ptr(workspace),
                                int(workspace.numel() * workspace.element_size()), _stream(stream))
    del layers_keepalive
    _check(st)


def rksc_decode_step(weights, prefix_k, prefix_v, cache: BranchCache, tokens: torch.Tensor,
                     next_token: torch.Tensor, p_top: torch.Tensor, conf: torch.Tensor, workspace: torch.Tensor,
                     stream=None) -> None:
    """Marshal torch device tensors into rksc_decode_step (asynchronous on `stream`)."""
    need = _Args()
    _check_weights(need, weights)
    n = _check_prefix(need, weights, prefix_k, prefix_v)
    need(tokens, "tokens", torch.int32, ndim=1)
    _check_decode_outputs(need, weights, cache, int(tokens.numel()), next_token, p_top, conf, workspace)
    lib = load_library()
    w, layers_keepalive = _weights_struct(weights)
    kv, kv_keep = _prefix_struct(prefix_k, prefix_v)
    st = lib.rksc_decode_step(ctypes.byref(w), ctypes.byref(kv), ctypes.byref(cache.struct), _ptr(tokens),
                              int(tokens.numel()), _ptr(next_token), _ptr(p_top), _ptr(conf), _ptr(workspace),
                              int(workspace.numel() * workspace.element_size()), _stream(stream))
    del layers_keepalive
    _check(st)


def rksc_cgee_gate(conf: torch.Tensor, n_steps: int, tau_conf: float, r_gap: float, p_mean: Optional[torch.Tensor],
                   fired: torch.Tensor, winner: torch.Tensor, stats: Optional[torch.Tensor], stream=None) -> None:
    """Marshal torch device tensors into rksc_cgee_gate (asynchronous on `stream`)."""
    need = _Args()
    need(conf, "conf", torch.float32, ndim=1)
    B = int(conf.numel())
    if p_mean is not None:
        need(p_mean, "p_mean", torch.float32, (B,))
    need(fired, "fired", torch.int32, (1,))
    need(winner, "winner", torch.int32, (1,))
    if stats is not None:
        need(stats, "stats", torch.float32, (3,))
    need.done()
    st = load_library().rksc_cgee_gate(_ptr(conf), int(conf.numel()), int(n_steps), float(tau_conf), float(r_gap),
                                       _ptr(p_mean), _ptr(fired), _ptr(winner), _ptr(stats), _stream(stream))
    _check(st)


def cgee_gate(conf: torch.Tensor, n_steps: int, tau_conf: float = 0.70, r_gap: float = 0.06, stream=None):
    """Eq. cgee_gate on the device: returns (fired [1] int32, winner [1] int32, p_mean [B], stats [3]) tensors."""
    dev = conf.device
    fired = torch.empty((1,), dtype=torch.int32, device=dev)
    winner = torch.empty((1,), dtype=torch.int32, device=dev)
    p_mean = torch.empty_like(conf)
    stats = torch.empty((3,), dtype=torch.float32, device=dev)
    rksc_cgee_gate(conf, n_steps, tau_conf, r_gap, p_mean, fired, winner, stats, stream)
    return fired, winner, p_mean, stats


class Decoder:
    """The stepwise batched decode loop over a shared prefix cache: allocates the
    branch cache, the workspace and the running confidence once, then
    `suffix(tokens [B, s])` and `step(tokens [B])` run rksc_decode_suffix /
    rksc_decode_step; `n_steps` counts the tokens generated (the t of Eq. gen_conf)."""

    def __init__(self, weights, prefix_k, prefix_v, n_branches: int, suffix_len: int, capacity: int, device):
        shape = weights.shape
        self.weights, self.prefix_k, self.prefix_v = weights, prefix_k, prefix_v
        n = _prefix_len(prefix_k)
        self.cache = BranchCache(shape, len(weights.layers), n_branches, capacity, device)
        self.workspace = torch.empty(rksc_decode_workspace_size(shape, n_branches, suffix_len, n),
                                     dtype=torch.uint8, device=device)
        self.next_token = torch.empty((n_branches,), dtype=torch.int32, device=device)
        self.p_top = torch.empty((n_branches,), dtype=torch.float32, device=device)
        self.conf = torch.zeros((n_branches,), dtype=torch.float32, device=device)
        self.n_steps = 0

    def suffix(self, suffix_tokens: torch.Tensor, stream=None):
        rksc_decode_suffix(self.weights, self.prefix_k, self.prefix_v, self.cache, suffix_tokens.contiguous(),
                           self.next_token, self.p_top, self.conf, self.workspace, stream)
        self.n_steps = 1
        return self.next_token, self.p_top

    def step(self, tokens: Optional[torch.Tensor] = None, stream=None):
        """One decode step; tokens defaults to the previous step's next_token (greedy)."""
        tok = self.next_token if tokens is None else tokens.contiguous()
        rksc_decode_step(self.weights, self.prefix_k, self.prefix_v, self.cache, tok, self.next_token,
                         self.p_top, self.conf, self.workspace, stream)
        self.n_steps += 1
        return self.next_token, self.p_top

    def gate(self, tau_conf: float = 0.70, r_gap: float = 0.06, stream=None):
        return cgee_gate(self.conf, self.n_steps, tau_conf, r_gap, stream)


class BlockTable:
    """The RSBCM block table (rksc_block_table_*): host-side, no GPU needed."""

    def __init__(self, capacity: int):
        lib = load_library()
        self._lib = lib
        self.capacity = int(capacity)
        self._t = lib.rksc_block_table_create(int(capacity))
        if not self._t:
            raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())

    def __del__(self):
        if getattr(self, "_t", None):
            self._lib.rksc_block_table_destroy(self._t)
            self._t = None

    def insert(self, block_id: int, score: float, depth: int) -> None:
        _check(self._lib.rksc_block_table_insert(self._t, int(block_id), float(score), int(depth)))

    def set_score(self, block_id: int, score: float) -> None:
        _check(self._lib.rksc_block_table_set_score(self._t, int(block_id), float(score)))

    def remove(self, block_id: int) -> None:
        _check(self._lib.rksc_block_table_remove(self._t, int(block_id)))

    def evict(self) -> list:
        """Alg. RsbcmEvict: the evicted ids, in eviction order."""
        need = max(0, len(self) - self.capacity)
        buf = (ctypes.c_int64 * max(1, need))()
        n = ctypes.c_int32(0)
        _check(self._lib.rksc_block_table_evict(self._t, buf, max(1, need), ctypes.byref(n)))
        return [int(buf[i]) for i in range(n.value)]

    def __len__(self) -> int:
        return int(self._lib.rksc_block_table_size(self._t))

    @property
    def evicted_total(self) -> int:
        return int(self._lib.rksc_block_table_evicted_total(self._t))


class KVProbe:
    """The KV probe (rksc_kv_probe_*): per 64-token prefix bucket, times the three paths once
    and keeps the verdict."""

    def __init__(self, reps: int = 3):
        lib = load_library()
        self._lib = lib
        self._p = lib.rksc_kv_probe_create(int(reps))
        if not self._p:
            raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())

    def __del__(self):
        if getattr(self, "_p", None):
            self._lib.rksc_kv_probe_destroy(self._p)
            self._p = None

    @staticmethod
    def workspace_size(shape, n_prefix: int, n_branches: int, suffix_len: int) -> int:
        cfg = model_config(shape)
        n = int(load_library().rksc_kv_probe_workspace_size(ctypes.byref(cfg), n_prefix, n_branches, suffix_len))
        if n == 0:
            raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())
        return n

    def decide(self, weights, prefix_tokens: torch.Tensor, suffix_tokens: torch.Tensor,
               workspace: Optional[torch.Tensor] = None, stream=None):
        """Returns (share: bool, times_ms [full, prefix, suffix], probed: bool)."""
        need = _Args()
        _check_weights(need, weights)
        need(prefix_tokens, "prefix_tokens", torch.int32, ndim=1)
        need(suffix_tokens, "suffix_tokens", torch.int32, ndim=2)
        B, s = suffix_tokens.shape
        n = int(prefix_tokens.numel())
        if workspace is None:
            workspace = torch.empty(self.workspace_size(weights.shape, n, B, s), dtype=torch.uint8,
                                    device=prefix_tokens.device)
        need(workspace, "workspace", torch.uint8, ndim=1)
        need.done()
        w, keep = _weights_struct(weights)
        share = ctypes.c_int32(0)
        probed = ctypes.c_int32(0)
        times = (ctypes.c_float * 3)()
        st = self._lib.rksc_kv_probe_decide(self._p, ctypes.byref(w), _ptr(prefix_tokens), n, _ptr(suffix_tokens),
                                            int(B), int(s), _ptr(workspace),
                                            int(workspace.numel() * workspace.element_size()), _stream(stream),
                                            ctypes.byref(share), times, ctypes.byref(probed))
        del keep
        _check(st)
        return bool(share.value), [float(t) for t in times], bool(probed.value)

    def lookup(self, n_prefix: int):
        """The stored verdict of n_prefix's bucket: None if never probed, else (share, times_ms)."""
        share = ctypes.c_int32(0)
        times = (ctypes.c_float * 3)()
        _check(self._lib.rksc_kv_probe_lookup(self._p, int(n_prefix), ctypes.byref(share), times))
        return None if share.value < 0 else (bool(share.value), [float(t) for t in times])


def rksc_prefix_extend_workspace_size(shape, n_parent: int, n_new: int) -> int:
    cfg = model_config(shape)
    n = int(load_library().rksc_prefix_extend_workspace_size(ctypes.byref(cfg), n_parent, n_new))
    if n == 0:
        raise RkscError(RKSC_ERR_INVALID_ARGUMENT, rksc_last_error())
    return n


def rksc_prefix_extend(weights, parent_k, parent_v, tokens: torch.Tensor, k_out: torch.Tensor, v_out: torch.Tensor,
                       h_node: Optional[torch.Tensor], workspace: torch.Tensor, stream=None) -> None:
    """Marshal torch device tensors into rksc_prefix_extend (asynchronous on `stream`)."""
    need = _Args()
    _check_weights(need, weights, need_lm_head=False)
    n = _check_prefix(need, weights, parent_k, parent_v, "parent")
    need(tokens, "tokens", torch.int32, ndim=1)
    shape, L = weights.shape, len(weights.layers)
    dims = (L, shape.n_kv_heads, int(tokens.numel()), shape.head_dim)
    need(k_out, "k_out", _model_dtype(shape), dims)
    need(v_out, "v_out", _model_dtype(shape), dims)
    if h_node is not None:
        need(h_node, "h_node", torch.float32, (L, shape.d_model))
    need(workspace, "workspace", torch.uint8, ndim=1)
    need.done()
    lib = load_library()
    w, keep = _weights_struct(weights)
    kv, kv_keep = _prefix_struct(parent_k, parent_v)
    st = lib.rksc_prefix_extend(ctypes.byref(w), ctypes.byref(kv), _ptr(tokens), int(tokens.numel()), _ptr(k_out),
                                _ptr(v_out), _ptr(h_node), _ptr(workspace),
                                int(workspace.numel() * workspace.element_size()), _stream(stream))
    del keep
    _check(st)


def prefix_extend(weights, parent_k, parent_v, tokens: torch.Tensor, stream=None):
    """A tree node's cache on top of its parent's prefix (a cache, or a PrefixCache in parent_k):
    returns (k [L, Hkv, m, hd], v, h_node [L, d] unit rows), the node's own m entries. The node's
    children read PrefixCache(parent segments).extend(k, v) as their prefix."""
    shape = weights.shape
    n = _prefix_len(parent_k)
    m = int(tokens.numel())
    dev = tokens.device
    L = len(weights.layers)
    dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    ws = torch.empty(rksc_prefix_extend_workspace_size(shape, n, m), dtype=torch.uint8, device=dev)
    k = torch.empty((L, shape.n_kv_heads, m, shape.head_dim), dtype=dtype, device=dev)
    v = torch.empty_like(k)
    h = torch.empty((L, shape.d_model), dtype=torch.float32, device=dev)
    rksc_prefix_extend(weights, parent_k, parent_v, tokens.contiguous(), k, v, h, ws, stream)
    return k, v, h


def rksc_asks_gate(hidden: torch.Tensor, h_root: torch.Tensor, alpha: float, tau: float, sigma: torch.Tensor,
                   shared: torch.Tensor, stream=None) -> None:
    """Marshal torch device tensors into rksc_asks_gate (asynchronous on `stream`)."""
    need = _Args()
    need(hidden, "hidden", torch.float32, ndim=3)
    L, B, d = hidden.shape
    need(h_root, "h_root", torch.float32, (L, d))
    need(sigma, "sigma", torch.float32, (B,))
    need(shared, "shared", torch.int32, (B,))
    need.done()
    _check(load_library().rksc_asks_gate(_ptr(hidden), _ptr(h_root), L, B, d, float(alpha), float(tau), _ptr(sigma),
                                         _ptr(shared), _stream(stream)))


def asks_gate(hidden: torch.Tensor, h_root: torch.Tensor, alpha: float = 1.5, tau: float = 0.82, stream=None):
    """Alg. AsksGate on the device: returns (sigma [B] fp32, shared [B] int32)."""
    L, B, d = hidden.shape
    sigma = torch.empty((B,), dtype=torch.float32, device=hidden.device)
    shared = torch.empty((B,), dtype=torch.int32, device=hidden.device)
    rksc_asks_gate(hidden.contiguous(), h_root.contiguous(), alpha, tau, sigma, shared, stream)
    return sigma, shared
