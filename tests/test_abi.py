"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments before touching the device. CPU only: no call here reaches a launch."""
import ctypes
import dataclasses
import math
import os
import re

import pytest

import paper_2606_09937_amd as rk
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails before any launch


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(rksc_\w+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rk.library_path()):
        pytest.fail("librksc.so is not built (run __graft_entry__.build())")
    return rk.load_library()


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert "rksc_verify_forward" in names and "rksc_asks_similarity" in names
    for name in names:
        assert hasattr(lib, name), f"{name} declared in include/ but not exported"
    assert rk.rksc_abi_version() == 8


def test_status_strings(lib):
    assert rk.rksc_status_string(0) == "ok"
    assert rk.rksc_status_string(-3) == "workspace too small"
    assert rk.rksc_status_string(-4) == "HIP error"


def _shape(**kw):
    return workloads.get("tiny").model.__class__(**{**workloads.get("tiny").model.__dict__, **kw})


@pytest.mark.parametrize("kw,needle", [
    (dict(head_dim=96), "head_dim"),
    (dict(n_heads=6, n_kv_heads=4), "n_heads"),
    (dict(d_ff=690), "d_ff"),
    (dict(d_model=250), "d_model"),
    (dict(vocab=0), "vocab"),
    (dict(n_layers=0), "n_layers"),
])
def test_workspace_size_rejects_bad_shapes(lib, kw, needle):
    with pytest.raises(rk.RkscError) as e:
        rk.rksc_verify_workspace_size(_shape(**kw), 4, 16, 64)
    assert needle in str(e.value)


@pytest.mark.parametrize("B,s", [(0, 16), (65, 16), (4, 0)])
def test_workspace_size_rejects_bad_batch(lib, B, s):
    with pytest.raises(rk.RkscError):
        rk.rksc_verify_workspace_size(workloads.get("tiny").model, B, s, 64)


def test_workspace_size_grows_with_batch(lib):
    shape = workloads.get("tiny").model
    a = rk.rksc_verify_workspace_size(shape, 1, 16, 64)
    b = rk.rksc_verify_workspace_size(shape, 4, 16, 64)
    c = rk.rksc_verify_workspace_size(shape, 4, 64, 64)
    assert 0 < a < b < c
    with pytest.raises(rk.RkscError):
        rk.rksc_verify_workspace_size(shape, 4, 16, -1)


def _call(lib, shape, B=4, s=16, tau=0.05, patience=1, ws_bytes=None, ws_ptr=0x10000, null=None, n_prefix=8):
    cfg = rk.model_config(shape)
    layers = (rk.LayerWeights * shape.n_layers)()
    for i in range(shape.n_layers):
        layers[i] = rk.LayerWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    if null == "layer":
        layers[shape.n_layers - 1] = rk.LayerWeights(FAKE, FAKE, None, FAKE, FAKE, FAKE)
    w = rk.Weights(cfg, FAKE, layers, FAKE, None if null == "lm_head" else FAKE)
    kv = rk.PrefixKV(n_prefix, None if null == "prefix" else FAKE, FAKE)
    need = lib.rksc_verify_workspace_size(ctypes.byref(cfg), B, s, n_prefix) if 1 <= B <= 64 and s >= 1 else 0
    size = need if ws_bytes is None else ws_bytes
    args = [ctypes.byref(w), ctypes.byref(kv), None if null == "tokens" else FAKE, B, s, tau, patience,
            None if null == "entropy" else FAKE, None if null == "exit" else FAKE, None,
            ctypes.c_void_p(ws_ptr), size, None]
    if null == "weights":
        args[0] = None
    return lib.rksc_verify_forward(*args)


@pytest.mark.parametrize("null", ["weights", "tokens", "entropy", "exit", "lm_head", "layer", "prefix"])
def test_verify_rejects_null_pointers(lib, null):
    assert _call(lib, workloads.get("tiny").model, null=null) == rk.RKSC_ERR_INVALID_ARGUMENT
    assert rk.rksc_last_error() != ""


@pytest.mark.parametrize("tau,patience", [(float("nan"), 1), (-0.1, 1), (0.1, 0), (0.1, -3)])
def test_verify_rejects_bad_rule(lib, tau, patience):
    assert _call(lib, workloads.get("tiny").model, tau=tau, patience=patience) == rk.RKSC_ERR_INVALID_ARGUMENT


def test_verify_rejects_small_or_misaligned_workspace(lib):
    shape = workloads.get("tiny").model
    cfg = rk.model_config(shape)
    need = lib.rksc_verify_workspace_size(ctypes.byref(cfg), 4, 16, 8)
    assert _call(lib, shape, ws_bytes=need - 1) == rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert str(need) in rk.rksc_last_error()
    assert _call(lib, shape, ws_ptr=0x10010) == rk.RKSC_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("B,s,code", [(0, 16, rk.RKSC_ERR_INVALID_ARGUMENT), (65, 16, rk.RKSC_ERR_INVALID_ARGUMENT),
                                      (4, 0, rk.RKSC_ERR_INVALID_ARGUMENT)])
def test_verify_rejects_bad_batch(lib, B, s, code):
    assert _call(lib, workloads.get("tiny").model, B=B, s=s, ws_bytes=1 << 30) == code


def test_verify_rejects_unsupported_head_dim(lib):
    shape = _shape(head_dim=32)
    assert _call(lib, shape, ws_bytes=1 << 30) == rk.RKSC_ERR_UNSUPPORTED
    assert "head_dim" in rk.rksc_last_error()


def test_asks_rejects_bad_arguments(lib):
    assert lib.rksc_asks_similarity(None, 2, 2, 8, 0.5, FAKE, None) == rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_asks_similarity(FAKE, 0, 2, 8, 0.5, FAKE, None) == rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_asks_similarity(FAKE, 2, 2, 8, math.inf, FAKE, None) == rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_asks_similarity(FAKE, 2, 2, 8, math.nan, FAKE, None) == rk.RKSC_ERR_INVALID_ARGUMENT


def test_testing_entry_points_reject_bad_shapes(lib):
    used = ctypes.c_int32(0)
    assert lib.rksc_test_gemm(1, FAKE, FAKE, FAKE, FAKE, 4, 4, 12, 0, ctypes.byref(used), None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_test_gemm(1, FAKE, None, FAKE, FAKE, 4, 4, 16, 0, ctypes.byref(used), None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_test_gemm_kind(1, FAKE, FAKE, FAKE, FAKE, 4, 4, 16, 0, 3, ctypes.byref(used), None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_test_gemm_kind(1, FAKE, FAKE, FAKE, FAKE, 33, 4, 16, 0, 2, ctypes.byref(used), None) == \
        rk.RKSC_ERR_UNSUPPORTED
    assert lib.rksc_test_gemm_kind(1, FAKE, FAKE, FAKE, FAKE, 17, 4, 16400, 0, 2, ctypes.byref(used), None) == \
        rk.RKSC_ERR_UNSUPPORTED
    assert lib.rksc_test_gemm_kind(1, FAKE, FAKE, FAKE, FAKE, 4, 6, 16, 0, 2, ctypes.byref(used), None) == \
        rk.RKSC_ERR_UNSUPPORTED
    assert lib.rksc_test_gemm_kind(0, FAKE, None, FAKE, FAKE, 4, 4, 16, 0, 2, ctypes.byref(used), None) == \
        rk.RKSC_ERR_UNSUPPORTED
    assert lib.rksc_test_gemm_kind(0, FAKE, None, FAKE, FAKE, 4, 4, 16, 0, 1, ctypes.byref(used), None) == \
        rk.RKSC_ERR_UNSUPPORTED
    assert lib.rksc_test_attention(1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 4, 4, 4, 2, 32, FAKE, 1 << 20, None) == \
        rk.RKSC_ERR_UNSUPPORTED


def test_prefill_rejects_bad_arguments(lib):
    shape = workloads.get("tiny").model
    cfg = rk.model_config(shape)
    assert lib.rksc_prefill_workspace_size(ctypes.byref(cfg), 0) == 0
    assert lib.rksc_prefill_workspace_size(ctypes.byref(cfg), 64) > 0
    layers = (rk.LayerWeights * shape.n_layers)()
    for i in range(shape.n_layers):
        layers[i] = rk.LayerWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    w = rk.Weights(cfg, FAKE, layers, FAKE, FAKE)
    ws = lib.rksc_prefill_workspace_size(ctypes.byref(cfg), 64)
    ok_ws = ctypes.c_void_p(0x100000)   # 256-byte aligned, never touched
    assert lib.rksc_prefill(ctypes.byref(w), None, 64, FAKE, FAKE, FAKE, ok_ws, ws, None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_prefill(ctypes.byref(w), FAKE, 0, FAKE, FAKE, FAKE, ok_ws, ws, None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_prefill(ctypes.byref(w), FAKE, 64, FAKE, FAKE, None, ok_ws, ws, None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_prefill(ctypes.byref(w), FAKE, 64, FAKE, FAKE, FAKE, ok_ws, ws - 1, None) == \
        rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert lib.rksc_prefill(ctypes.byref(w), FAKE, 64, FAKE, FAKE, FAKE, ctypes.c_void_p(0x100010), ws, None) == \
        rk.RKSC_ERR_INVALID_ARGUMENT


def _fake_weights(shape):
    cfg = rk.model_config(shape)
    layers = (rk.LayerWeights * shape.n_layers)()
    for i in range(shape.n_layers):
        layers[i] = rk.LayerWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    return rk.Weights(cfg, FAKE, layers, FAKE, FAKE), layers, cfg


def test_decode_rejects_bad_arguments(lib):
    shape = workloads.get("tiny").model
    w, _keep, cfg = _fake_weights(shape)
    assert lib.rksc_decode_workspace_size(ctypes.byref(cfg), 4, 16, -1) == 0
    assert lib.rksc_decode_workspace_size(ctypes.byref(cfg), 0, 16, 8) == 0
    assert lib.rksc_decode_workspace_size(ctypes.byref(cfg), 4, 0, 8) == 0
    ws = lib.rksc_decode_workspace_size(ctypes.byref(cfg), 4, 16, 8)
    assert ws >= lib.rksc_verify_workspace_size(ctypes.byref(cfg), 4, 16, 8)
    assert ws >= lib.rksc_verify_workspace_size(ctypes.byref(cfg), 4, 1, 8)
    ok_ws = ctypes.c_void_p(0x100000)
    kv = rk.PrefixKV(8, FAKE, FAKE)
    I = rk.RKSC_ERR_INVALID_ARGUMENT

    def suffix(bkv, s=16, B=4, tokens=FAKE, outs=(FAKE, FAKE, FAKE), wsb=ws, wsp=ok_ws, kvp=kv):
        return lib.rksc_decode_suffix(ctypes.byref(w), ctypes.byref(kvp) if kvp else None,
                                      ctypes.byref(bkv) if bkv else None, tokens, B, s, *outs, wsp, wsb, None)

    def step(bkv, B=4, wsb=ws):
        return lib.rksc_decode_step(ctypes.byref(w), ctypes.byref(kv), ctypes.byref(bkv), FAKE, B, FAKE, FAKE, FAKE,
                                    ok_ws, wsb, None)

    good = rk.BranchKVStruct(32, 0, FAKE, FAKE)
    assert suffix(None) == I
    assert suffix(good, kvp=None) == I
    assert suffix(rk.BranchKVStruct(32, 0, None, FAKE)) == I
    assert suffix(good, tokens=None) == I
    assert suffix(good, outs=(FAKE, None, FAKE)) == I
    assert suffix(good, outs=(FAKE, FAKE, None)) == I
    assert suffix(good, s=0) == I
    assert suffix(good, B=0) == I and suffix(good, B=65) == I
    assert suffix(rk.BranchKVStruct(15, 0, FAKE, FAKE)) == I              # capacity < s
    assert suffix(rk.BranchKVStruct(32, 3, FAKE, FAKE)) == I              # suffix needs an empty cache
    assert suffix(good, wsb=ws - 1) == rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert suffix(good, wsp=ctypes.c_void_p(0x100040)) == I
    assert suffix(good, kvp=rk.PrefixKV(-1, FAKE, FAKE)) == I
    assert suffix(good, kvp=rk.PrefixKV(8, None, FAKE)) == I
    full = rk.BranchKVStruct(32, 32, FAKE, FAKE)
    assert step(full) == I                                                 # no free entry
    assert full.length == 32
    assert step(rk.BranchKVStruct(32, -1, FAKE, FAKE)) == I
    assert step(rk.BranchKVStruct(32, 5, FAKE, FAKE), wsb=16) == rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert "workspace" in rk.rksc_last_error()


def test_cgee_gate_rejects_bad_arguments(lib):
    I = rk.RKSC_ERR_INVALID_ARGUMENT
    assert lib.rksc_cgee_gate(None, 4, 3, 0.7, 0.06, None, FAKE, FAKE, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 4, 3, 0.7, 0.06, None, None, FAKE, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 4, 3, 0.7, 0.06, None, FAKE, None, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 0, 3, 0.7, 0.06, None, FAKE, FAKE, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 65, 3, 0.7, 0.06, None, FAKE, FAKE, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 4, 0, 0.7, 0.06, None, FAKE, FAKE, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 4, 3, math.nan, 0.06, None, FAKE, FAKE, None, None) == I
    assert lib.rksc_cgee_gate(FAKE, 4, 3, 0.7, math.nan, None, FAKE, FAKE, None, None) == I


def test_prefix_extend_and_asks_gate_reject_bad_arguments(lib):
    shape = workloads.get("tiny").model
    w, _keep, cfg = _fake_weights(shape)
    assert lib.rksc_prefix_extend_workspace_size(ctypes.byref(cfg), -1, 4) == 0
    assert lib.rksc_prefix_extend_workspace_size(ctypes.byref(cfg), 8, 0) == 0
    ws = lib.rksc_prefix_extend_workspace_size(ctypes.byref(cfg), 8, 4)
    assert ws > 0
    ok_ws = ctypes.c_void_p(0x100000)
    I = rk.RKSC_ERR_INVALID_ARGUMENT
    par = rk.PrefixKV(8, ctypes.c_void_p(0x2000000), ctypes.c_void_p(0x3000000))

    def ext(parent=par, tokens=FAKE, m=4, k=ctypes.c_void_p(0x5000000), v=ctypes.c_void_p(0x6000000), wsp=ok_ws,
            wsb=ws):
        return lib.rksc_prefix_extend(ctypes.byref(w), ctypes.byref(parent) if parent else None, tokens, m, k, v,
                                      None, wsp, wsb, None)

    assert ext(parent=None) == I
    assert ext(tokens=None) == I
    assert ext(m=0) == I
    assert ext(k=None) == I
    assert ext(wsp=None) == I
    assert ext(wsp=ctypes.c_void_p(0x100010)) == I
    assert ext(wsb=ws - 1) == rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert ext(parent=rk.PrefixKV(8, None, FAKE)) == I
    assert ext(parent=rk.PrefixKV(-1, FAKE, FAKE)) == I
    # the child cache may not overlap the parent's
    assert ext(k=ctypes.c_void_p(0x2000000 + 64)) == I
    assert "overlap" in rk.rksc_last_error()
    G = lib.rksc_asks_gate
    assert G(None, FAKE, 2, 4, 8, 1.5, 0.8, FAKE, FAKE, None) == I
    assert G(FAKE, FAKE, 2, 4, 8, 1.5, 0.8, FAKE, None, None) == I
    assert G(FAKE, FAKE, 0, 4, 8, 1.5, 0.8, FAKE, FAKE, None) == I
    assert G(FAKE, FAKE, 2, 4, 8, math.inf, 0.8, FAKE, FAKE, None) == I
    assert G(FAKE, FAKE, 2, 4, 8, 1.5, math.nan, FAKE, FAKE, None) == I


def test_asks_gate_rejects_unsupported_shapes(lib):
    U = rk.RKSC_ERR_UNSUPPORTED
    assert lib.rksc_asks_gate(FAKE, FAKE, 257, 4, 8, 1.5, 0.8, FAKE, FAKE, None) == U
    assert lib.rksc_asks_gate(FAKE, FAKE, 2, 4, 10, 1.5, 0.8, FAKE, FAKE, None) == U


# ---- the Python binding checks dtype, shape and device before it hands a pointer to the library

def _bf16_tiny():
    import dataclasses
    return dataclasses.replace(workloads.get("tiny").model, dtype="bf16")


def _meta(shape, dtype):
    import torch
    return torch.empty(shape, dtype=dtype, device="meta")


def test_marshal_rejects_wrong_dtype_shape_and_host_tensors(lib):
    import torch
    shape = _bf16_tiny()
    mw = workloads.make_model(shape, seed=1)          # host tensors: rejected before any call
    L, d, Hkv, hd = shape.n_layers, shape.d_model, shape.n_kv_heads, shape.head_dim
    pk = _meta((L, Hkv, 8, hd), torch.bfloat16)
    tok = _meta((2, 4), torch.int32)
    ent, ex, ws = _meta((L, 2), torch.float32), _meta((2,), torch.int32), _meta((1 << 20,), torch.uint8)

    def verify(**kw):
        a = dict(weights=mw, prefix_k=pk, prefix_v=pk, branch_tokens=tok, tau=0.1, patience=1, entropy=ent,
                 exit_layer=ex, hidden_last=None, workspace=ws)
        a.update(kw)
        with pytest.raises(ValueError) as e:
            rk.rksc_verify_forward(**a)
        return str(e.value)

    assert "GPU" in verify()                                                  # host weights
    mw_meta = workloads.ModelWeights(shape, _meta(mw.embed.shape, torch.bfloat16),
                                     [{k: _meta(v.shape, v.dtype) for k, v in lw.items()} for lw in mw.layers],
                                     _meta((d,), torch.float32), _meta(mw.lm_head.shape, torch.bfloat16))
    assert "embed" in verify(weights=workloads.ModelWeights(shape, mw_meta.embed.float(), mw_meta.layers,
                                                            mw_meta.final_norm, mw_meta.lm_head))
    assert "prefix_k" in verify(weights=mw_meta, prefix_k=_meta((L, Hkv, 8, hd), torch.float32))
    assert "prefix_k" in verify(weights=mw_meta, prefix_k=_meta((L, Hkv + 1, 8, hd), torch.bfloat16))
    assert "prefix_v" in verify(weights=mw_meta, prefix_v=_meta((L, Hkv, 9, hd), torch.bfloat16))
    assert "branch_tokens" in verify(weights=mw_meta, branch_tokens=_meta((2, 4), torch.int64))
    assert "entropy" in verify(weights=mw_meta, entropy=_meta((L, 3), torch.float32))
    assert "hidden_last" in verify(weights=mw_meta, hidden_last=_meta((L, 2, d), torch.bfloat16))
    assert "GPU" in verify(weights=mw_meta)                                   # meta is not a GPU either
    bad = [dict(lw) for lw in mw_meta.layers]
    bad[1]["w_down"] = _meta((d, shape.d_ff + 8), torch.bfloat16)
    assert "layer 1 w_down" in verify(weights=workloads.ModelWeights(shape, mw_meta.embed, bad, mw_meta.final_norm,
                                                                     mw_meta.lm_head))

    with pytest.raises(ValueError, match="hidden must be torch.float32"):
        rk.rksc_asks_similarity(_meta((2, 3, 8), torch.bfloat16), 0.5, _meta((3, 3), torch.float32))
    with pytest.raises(ValueError, match="S must have shape"):
        rk.rksc_asks_similarity(_meta((2, 3, 8), torch.float32), 0.5, _meta((2, 2), torch.float32))
    with pytest.raises(ValueError, match="GPU"):
        rk.rksc_asks_similarity(torch.zeros((2, 3, 8)), 0.5, torch.zeros((3, 3)))
    with pytest.raises(ValueError, match="tokens must be torch.int32"):
        rk.rksc_prefill(mw_meta, _meta((8,), torch.int64), pk, pk, _meta((L, d), torch.float32), ws)
    with pytest.raises(ValueError, match="h_root"):
        rk.rksc_asks_gate(_meta((L, 2, d), torch.float32), _meta((L + 1, d), torch.float32), 1.5, 0.8,
                          _meta((2,), torch.float32), _meta((2,), torch.int32))
    with pytest.raises(ValueError, match="fired"):
        rk.rksc_cgee_gate(_meta((4,), torch.float32), 3, 0.7, 0.06, None, _meta((1,), torch.int64),
                          _meta((1,), torch.int32), None)


def test_noalloc_refuses_oversized_pass_before_any_hip_call(lib):
    """rksc_verify_forward_noalloc checks the pass's workspace against its fixed array on the host
    first: a larger pass is refused with RKSC_ERR_WORKSPACE_TOO_SMALL (no device is touched)."""
    wl = workloads.get("7b_tot")
    w, _keep, cfg = _fake_weights(wl.model)
    kv = rk.PrefixKV(wl.prefix_len, FAKE, FAKE)
    need = lib.rksc_verify_workspace_size(ctypes.byref(cfg), wl.n_branches, wl.branch_len, wl.prefix_len)
    assert need > rk.RKSC_NOALLOC_SCRATCH_BYTES
    st = lib.rksc_verify_forward_noalloc(ctypes.byref(w), ctypes.byref(kv), FAKE, wl.n_branches, wl.branch_len,
                                         0.02, 2, FAKE, FAKE, None, None)
    assert st == rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert str(need) in rk.rksc_last_error() and "allocation-free" in rk.rksc_last_error()
    assert lib.rksc_verify_forward_noalloc(None, ctypes.byref(kv), FAKE, 1, 1, 0.02, 2, FAKE, FAKE, None,
                                           None) == rk.RKSC_ERR_INVALID_ARGUMENT
    bad = workloads.get("tiny").model
    w2, _k2, _ = _fake_weights(dataclasses.replace(bad, head_dim=32))
    assert lib.rksc_verify_forward_noalloc(ctypes.byref(w2), ctypes.byref(rk.PrefixKV(8, FAKE, FAKE)), FAKE, 4, 16,
                                           0.02, 2, FAKE, FAKE, None, None) == rk.RKSC_ERR_UNSUPPORTED
    # the header's limit is the binding's
    text = open(os.path.join(ROOT, "include", "rksc.h")).read()
    assert "#define RKSC_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)" in text
    assert rk.RKSC_NOALLOC_SCRATCH_BYTES == 128 << 20


def test_exit_window_cost_model(lib):
    """The exit window of the default schedule (host only): a power of two with window * B <= 64, the
    value the cost model gives at each workload, and no window at all for an invalid shape."""
    expect = {"7b_single": 8, "7b_tot": 2, "7b_large_vocab": 4, "10b_long": 2, "10b_decode": 2,
              "7b_paper_verify": 4, "tiny": 1, "tiny_deep": 1}
    for name, w in expect.items():
        wl = workloads.get(name)
        got = rk.rksc_verify_window(wl.model, wl.n_branches, wl.branch_len, wl.prefix_len)
        assert got == w, (name, got)
    shape = workloads.get("7b_single").model
    for B in (1, 2, 5, 8, 9, 16, 17, 32, 33, 64):
        for s, n in ((1, 0), (16, 64), (128, 1024), (256, 16384)):
            w = rk.rksc_verify_window(shape, B, s, n)
            assert w in (1, 2, 4, 8) and w * B <= 64
    # more work per layer never asks for a larger window (the probe is a smaller share)
    ws = [rk.rksc_verify_window(shape, 1, s, 1024) for s in (1, 16, 128, 1024, 4096)]
    assert ws == sorted(ws, reverse=True)
    with pytest.raises(rk.RkscError):
        rk.rksc_verify_window(shape, 0, 16, 64)
    with pytest.raises(rk.RkscError):
        rk.rksc_verify_window(_shape(head_dim=32), 4, 16, 64)


def test_prefix_chain_limits_before_any_launch(lib):
    """A prefix chain longer than RKSC_MAX_PREFIX_SEGMENTS caches, or a cycle, is refused during
    validation; so is a tree node whose children's chain would be too long."""
    shape = workloads.get("tiny").model
    w, _keep, cfg = _fake_weights(shape)
    ws = lib.rksc_verify_workspace_size(ctypes.byref(cfg), 4, 16, 9 * 8)
    ok_ws = ctypes.c_void_p(0x100000)
    segs = []
    for i in range(rk.RKSC_MAX_PREFIX_SEGMENTS + 1):
        seg = rk.PrefixKV(8, ctypes.c_void_p(0x1000000 * (i + 1)), ctypes.c_void_p(0x1000000 * (i + 1) + 0x800000))
        if segs:
            seg.parent = ctypes.pointer(segs[-1])
        segs.append(seg)

    def verify(kv):
        return lib.rksc_verify_forward(ctypes.byref(w), ctypes.byref(kv), FAKE, 4, 16, 0.1, 1, FAKE, FAKE, None,
                                       ok_ws, ws, None)

    assert verify(segs[-1]) == rk.RKSC_ERR_UNSUPPORTED and "chain" in rk.rksc_last_error()
    cyc = rk.PrefixKV(8, FAKE, FAKE)
    cyc.parent = ctypes.pointer(cyc)
    assert verify(cyc) == rk.RKSC_ERR_UNSUPPORTED
    bad = rk.PrefixKV(8, FAKE, FAKE)
    bad.parent = ctypes.pointer(rk.PrefixKV(4, None, FAKE))
    assert verify(bad) == rk.RKSC_ERR_INVALID_ARGUMENT
    ext_ws = lib.rksc_prefix_extend_workspace_size(ctypes.byref(cfg), 8 * 8, 4)
    full = segs[rk.RKSC_MAX_PREFIX_SEGMENTS - 1]     # a chain of exactly the maximum
    st = lib.rksc_prefix_extend(ctypes.byref(w), ctypes.byref(full), FAKE, 4, ctypes.c_void_p(0x70000000),
                                ctypes.c_void_p(0x78000000), None, ok_ws, ext_ws, None)
    assert st == rk.RKSC_ERR_UNSUPPORTED and "children" in rk.rksc_last_error()


def test_tile_gate_up_rejects_bad_arguments(lib):
    """rksc_tile_gate_up and rksc_gate_up_tiled_bytes validate on the host: an fp32 or untileable
    model, NULL, short, misaligned or overlapping buffers are refused before any launch."""
    shape = dataclasses.replace(_bf16_tiny(), d_ff=768)     # 2 d_ff = 6 x 256
    cfg = rk.model_config(shape)
    need = lib.rksc_gate_up_tiled_bytes(ctypes.byref(cfg))
    assert need == 2 * shape.d_ff * shape.d_model * 2
    I, U = rk.RKSC_ERR_INVALID_ARGUMENT, rk.RKSC_ERR_UNSUPPORTED
    src, dst = ctypes.c_void_p(0x10000000), ctypes.c_void_p(0x20000000)
    T = lib.rksc_tile_gate_up
    assert T(ctypes.byref(cfg), None, dst, need, None) == I
    assert T(ctypes.byref(cfg), src, None, need, None) == I
    assert T(ctypes.byref(cfg), src, dst, need - 1, None) == I and str(need) in rk.rksc_last_error()
    assert T(ctypes.byref(cfg), ctypes.c_void_p(0x10000008), dst, need, None) == I
    assert T(ctypes.byref(cfg), src, ctypes.c_void_p(0x10000000 + need - 64), need, None) == I
    assert "overlap" in rk.rksc_last_error()
    for bad in (workloads.get("tiny").model, dataclasses.replace(shape, dtype="f32"), _bf16_tiny()):
        c2 = rk.model_config(bad)
        assert (2 * bad.d_ff) % 256 or bad.dtype != "bf16"
        assert lib.rksc_gate_up_tiled_bytes(ctypes.byref(c2)) == 0
        assert T(ctypes.byref(c2), src, dst, 1 << 30, None) == U
    assert lib.rksc_gate_up_tiled_bytes(ctypes.byref(rk.model_config(_shape(head_dim=96)))) == 0


def test_verify_rejects_misplaced_tiled_weight(lib):
    """A layer's w_gate_up_tiled is read only where the layout exists: set on an fp32 model it is
    refused as unsupported, and a misaligned pointer as invalid, before any launch."""
    shape = workloads.get("tiny").model
    assert shape.dtype != "bf16"
    w, layers, cfg = _fake_weights(shape)
    layers[1].w_gate_up_tiled = FAKE
    ws = lib.rksc_verify_workspace_size(ctypes.byref(cfg), 4, 16, 8)
    kv = rk.PrefixKV(8, FAKE, FAKE)
    ok_ws = ctypes.c_void_p(0x100000)
    st = lib.rksc_verify_forward(ctypes.byref(w), ctypes.byref(kv), FAKE, 4, 16, 0.1, 1, FAKE, FAKE, None, ok_ws,
                                 ws, None)
    assert st == rk.RKSC_ERR_UNSUPPORTED and "layer 1" in rk.rksc_last_error()
    pw = lib.rksc_prefill_workspace_size(ctypes.byref(cfg), 8)
    assert lib.rksc_prefill(ctypes.byref(w), FAKE, 8, FAKE, FAKE, FAKE, ok_ws, pw, None) == rk.RKSC_ERR_UNSUPPORTED
    w2, layers2, cfg2 = _fake_weights(dataclasses.replace(_bf16_tiny(), d_ff=768))
    layers2[0].w_gate_up_tiled = ctypes.c_void_p(0x1008)
    ws2 = lib.rksc_verify_workspace_size(ctypes.byref(cfg2), 4, 16, 8)
    st = lib.rksc_verify_forward(ctypes.byref(w2), ctypes.byref(kv), FAKE, 4, 16, 0.1, 1, FAKE, FAKE, None,
                                 ok_ws, ws2, None)
    assert st == rk.RKSC_ERR_INVALID_ARGUMENT and "aligned" in rk.rksc_last_error()
    layers2[0].w_gate_up_tiled = None
    w3, layers3, cfg3 = _fake_weights(_bf16_tiny())                # 2 d_ff = 1376: no tiled layout
    layers3[1].w_gate_up_tiled = FAKE
    ws3 = lib.rksc_verify_workspace_size(ctypes.byref(cfg3), 4, 16, 8)
    st = lib.rksc_verify_forward(ctypes.byref(w3), ctypes.byref(kv), FAKE, 4, 16, 0.1, 1, FAKE, FAKE, None,
                                 ok_ws, ws3, None)
    assert st == rk.RKSC_ERR_UNSUPPORTED
