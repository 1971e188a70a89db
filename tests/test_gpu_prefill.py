"""Parity of the HIP root forward (rksc_prefill through the C ABI) with the float64
oracle's prefill (Eq. prefix_fwd), and of the verify pass run on the GPU-built
prefix cache with the oracle's verify pass on the oracle-built cache.

Bars: cache rows (one key or value vector of one layer, KV head and token) and
unit root rows within 2e-2 norm-relative (the hidden-state bar; bf16 storage of
the cache adds 2^-9); the end-to-end verify to the verify bars; sigma_b against
the root (Eq. asks_sim) within 1e-3.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import HIDDEN_RTOL, SIM_ATOL, compare_verify, host_view, log, oracle_cfg, to_np

pytestmark = pytest.mark.gpu
DEV = "cuda"

GQA_BF16 = workloads.ModelShape(n_layers=3, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=1376,
                                vocab=5000, dtype="bf16", lm_head_scale=6.0)


def _row_rel(a, ref):
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.linalg.norm(a - ref, axis=-1)
    den = np.maximum(np.linalg.norm(ref, axis=-1), 1e-30)
    return num / den


def _prefill_parity(shape, n, seed, label, n_layers=None):
    mw = workloads.make_model(shape, seed=seed, device=DEV, n_layers=n_layers)
    L = len(mw.layers)
    toks = workloads.make_tokens(n, shape.vocab, seed=seed, name="prefix", device=DEV)
    log(f"[{label}] gpu prefill n={n}")
    k, v, h_root = rk.prefill(mw, toks)
    torch.cuda.synchronize()
    log(f"[{label}] oracle prefill")
    pk, pv, hr = oracle.prefill(host_view(mw), oracle_cfg(shape, L), toks.cpu().numpy())
    rk_k, rk_v = to_np(k.float()), to_np(v.float())
    ek, ev = _row_rel(rk_k, pk), _row_rel(rk_v, pv)
    eh = _row_rel(to_np(h_root), oracle.unit_rows(hr))
    log(f"[{label}] max rel err K {ek.max():.2e} V {ev.max():.2e} h_root {eh.max():.2e}")
    assert ek.max() <= HIDDEN_RTOL and ev.max() <= HIDDEN_RTOL and eh.max() <= HIDDEN_RTOL
    np.testing.assert_allclose(np.linalg.norm(to_np(h_root), axis=-1), 1.0, atol=1e-5)
    return mw, toks, (k, v, h_root), (pk, pv, hr)


@pytest.mark.parametrize("name", ["tiny", "tiny_deep"])
def test_prefill_fp32(name):
    wl = workloads.get(name)
    _prefill_parity(wl.model, wl.prefix_len, 21, f"prefill {name}")


@pytest.mark.parametrize("shape,n", [
    (dataclasses.replace(workloads.get("tiny_deep").model, dtype="bf16"), 64),
    (GQA_BF16, 100), (GQA_BF16, 129), (GQA_BF16, 1),
], ids=["tiny_deep_bf16_64", "gqa_bf16_100", "gqa_bf16_129", "gqa_bf16_1"])
def test_prefill_bf16(shape, n):
    _prefill_parity(shape, n, 22, f"prefill {shape.d_model}x{shape.n_layers} n={n}")


def test_prefill_then_verify_and_root_similarity():
    """The GPU cache feeds the GPU verify; the oracle cache feeds the oracle verify (end to end),
    and sigma_b of every branch against the root rows matches the oracle's."""
    wl = workloads.get("tiny_deep")
    shape = dataclasses.replace(wl.model, dtype="bf16")
    mw, _, (k, v, h_root), (pk, pv, hr) = _prefill_parity(shape, wl.prefix_len, 23, "prefill+verify")
    B, s = wl.n_branches, wl.branch_len
    toks = workloads.make_tokens(B * s, shape.vocab, seed=23, device=DEV).reshape(B, s).contiguous()
    # The cache is stored in the model's storage type: the oracle's verify reads its own cache rounded
    # the same way (bf16, round to nearest even), so the comparison isolates the two passes' arithmetic.
    pk_b = torch.from_numpy(pk).to(torch.bfloat16).float().numpy()
    pv_b = torch.from_numpy(pv).to(torch.bfloat16).float().numpy()
    for tau, pat in ((0.3, 1), (0.0, 1)):
        ent, ex, hid = rk.verify_forward(mw, k, v, toks, tau, pat, return_hidden=True)
        torch.cuda.synchronize()
        ent, ex, hid = to_np(ent), to_np(ex), to_np(hid)
        L = len(mw.layers)
        _, ex_ref, _, ent_ref, hid_ref = oracle.verify_forward(host_view(mw), oracle_cfg(shape, L), pk_b, pv_b,
                                                               toks.cpu().numpy(), tau, pat)
        stats = compare_verify(ent, ex, hid, ent_ref, hid_ref, ex_ref, tau, label=f"prefill->verify tau={tau}")
        log(f"[prefill->verify tau={tau}] exits gpu={ex.tolist()} oracle={ex_ref.tolist()} {stats}")
    # sigma_b (Eq. asks_sim, Alg. AsksGate): the root's unit rows appended as one more branch.
    hb = torch.from_numpy(np.nan_to_num(hid).astype(np.float32)).to(DEV)
    both = torch.cat([hb, h_root[:, None, :]], dim=1).contiguous()
    S = to_np(rk.asks_similarity(both, wl.alpha))
    sig_ref = oracle.root_similarity(hid_ref, oracle.unit_rows(hr), wl.alpha)
    err = np.abs(S[:B, B] - sig_ref).max()
    log(f"[sigma_b] gpu {S[:B, B].round(5).tolist()} oracle {sig_ref.round(5).tolist()} max err {err:.2e}")
    assert err <= SIM_ATOL
    assert abs(S[B, B] - 1.0) <= SIM_ATOL


def test_prefill_7b_shape_two_layers():
    """Full 7B width and the 1024-token prefix of the single-branch verify workload, first two layers."""
    wl = workloads.get("7b_single")
    _prefill_parity(wl.model, wl.prefix_len, 42, "prefill 7b", n_layers=2)
