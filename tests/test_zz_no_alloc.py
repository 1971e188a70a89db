"""The allocation-free verify entry point (rksc_verify_forward_noalloc, for callers
that cannot allocate device memory) against rksc_verify_forward with a caller
workspace: the same kernels on the same inputs, so the outputs must be bitwise
identical; checked on consecutive calls (the second with a smaller input, on the
array the first call left behind), at the 7B headline shape, and against the
float64 oracle on a small shape."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import compare_verify, host_view, log, oracle_cfg, to_np

pytestmark = pytest.mark.gpu
DEV = "cuda"

GQA = workloads.ModelShape(n_layers=4, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=1376, vocab=5000,
                           dtype="bf16", lm_head_scale=6.0)


def _inputs(shape, B, n, s, seed, n_layers=None):
    mw = workloads.make_model(shape, seed=seed, device=DEV, n_layers=n_layers)
    kv = workloads.make_prefix_kv(shape, n, seed=seed, device=DEV, n_layers=n_layers)
    toks = workloads.make_tokens(B * s, shape.vocab, seed=seed, device=DEV).reshape(B, s).contiguous()
    return mw, kv, toks


def _both(mw, kv, toks, tau, patience):
    L, (B, _) = len(mw.layers), toks.shape
    d = mw.shape.d_model
    ent = torch.empty((L, B), dtype=torch.float32, device=DEV)
    ex = torch.empty((B,), dtype=torch.int32, device=DEV)
    hid = torch.empty((L, B, d), dtype=torch.float32, device=DEV)
    rk.rksc_verify_forward_noalloc(mw, kv.k, kv.v, toks, tau, patience, ent, ex, hid)
    torch.cuda.synchronize()
    got = (to_np(ent), to_np(ex), to_np(hid))
    ref = rk.verify_forward(mw, kv.k, kv.v, toks, tau, patience, return_hidden=True)
    torch.cuda.synchronize()
    return got, tuple(to_np(t) for t in ref)


def _same(got, ref, label):
    for a, b, name in zip(got, ref, ("entropy", "exit_layer", "hidden_last")):
        np.testing.assert_array_equal(a, b, err_msg=f"{label}: {name} differs from rksc_verify_forward")


def test_noalloc_consecutive_calls_match_workspace_entry_point():
    mw, kv, toks = _inputs(GQA, 5, 100, 40, seed=61)
    for tau, pat in ((0.3, 1), (0.0, 1)):
        log(f"[noalloc] B=5 s=40 tau={tau}")
        got, ref = _both(mw, kv, toks, tau, pat)
        _same(got, ref, f"B=5 s=40 tau={tau}")
        # the second call, smaller, on the array the first one filled
        small = toks[:3, :9].contiguous()
        log(f"[noalloc] B=3 s=9 tau={tau}")
        got_s, ref_s = _both(mw, kv, small, tau, pat)
        _same(got_s, ref_s, f"B=3 s=9 tau={tau}")
        hv = host_view(mw)
        _, ex_o, _, ent_o, hid_o = oracle.verify_forward(hv, oracle_cfg(GQA, GQA.n_layers), kv.k.cpu(), kv.v.cpu(),
                                                         small.cpu().numpy(), tau, pat)
        stats = compare_verify(got_s[0], got_s[1], got_s[2], ent_o, hid_o, ex_o, tau, label="noalloc small")
        log(f"[noalloc] small vs oracle {stats}")


def test_noalloc_headline_shape():
    """The 7B single-branch verify (32 layers, 1024-token prefix, 128 tokens) fits the array."""
    wl = workloads.get("7b_single")
    assert rk.rksc_verify_workspace_size(wl.model, 1, 128, 1024) <= rk.RKSC_NOALLOC_SCRATCH_BYTES
    mw, kv, toks = _inputs(wl.model, wl.n_branches, wl.prefix_len, wl.branch_len, seed=42)
    for tau in (wl.tau, 0.2):
        log(f"[noalloc] 7b_single tau={tau}")
        got, ref = _both(mw, kv, toks, tau, wl.patience)
        _same(got, ref, f"7b_single tau={tau}")
    # with the pre-tiled gate|up copy (the bench's setting) the outputs are the same bits
    mt = workloads.ModelWeights(mw.shape, mw.embed, [dict(lw) for lw in mw.layers], mw.final_norm, mw.lm_head)
    assert rk.tile_gate_up(mt)
    log("[noalloc] 7b_single with the tiled gate|up copy")
    got_t, ref_t = _both(mt, kv, toks, 0.2, wl.patience)
    _same(got_t, ref_t, "7b_single tiled")
    _same(got_t, ref, "7b_single tiled against untiled")
    del mt
    # then a smaller call again, after the large one
    small = dataclasses.replace(wl.model, n_layers=3)
    mw3, kv3, toks3 = _inputs(small, 2, 64, 16, seed=9, n_layers=3)
    got, ref = _both(mw3, kv3, toks3, 0.1, 1)
    _same(got, ref, "3-layer 7B width after the headline call")


def test_noalloc_refuses_a_pass_larger_than_the_array():
    wl = workloads.get("7b_tot")
    need = rk.rksc_verify_workspace_size(wl.model, wl.n_branches, wl.branch_len, wl.prefix_len)
    assert need > rk.RKSC_NOALLOC_SCRATCH_BYTES
    shape = dataclasses.replace(wl.model, n_layers=1)
    mw, kv, _ = _inputs(shape, 1, 16, 1, seed=3, n_layers=1)
    toks = torch.zeros((wl.n_branches, wl.branch_len), dtype=torch.int32, device=DEV)
    ent = torch.full((1, wl.n_branches), 7.0, device=DEV)
    ex = torch.full((wl.n_branches,), -5, dtype=torch.int32, device=DEV)
    kv_big = workloads.PrefixKV(torch.zeros((1, shape.n_kv_heads, wl.prefix_len, shape.head_dim),
                                            dtype=torch.bfloat16, device=DEV),
                                torch.zeros((1, shape.n_kv_heads, wl.prefix_len, shape.head_dim),
                                            dtype=torch.bfloat16, device=DEV))
    with pytest.raises(rk.RkscError) as e:
        rk.rksc_verify_forward_noalloc(mw, kv_big.k, kv_big.v, toks, 0.02, 2, ent, ex, None)
    assert e.value.status == rk.RKSC_ERR_WORKSPACE_TOO_SMALL and "allocation-free" in str(e.value)
    torch.cuda.synchronize()
    assert (ent == 7.0).all() and (ex == -5).all(), "a refused call wrote its outputs"
