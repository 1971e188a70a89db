"""Parity of the HIP batched decode (rksc_decode_suffix and rksc_decode_step through
the C ABI) and of the CGEE gate (rksc_cgee_gate) with the float64 oracle.

Inputs are teacher-forced: the suffix and every decode step's tokens are seeded
draws fed to both sides (never the GPU's own argmax). The prefix cache is the
oracle's prefill rounded to the model's storage type, and the oracle's decode
steps read its own branch cache rounded the same way, as the GPU stores it.

Bars:
  - branch cache rows (one key or value vector of one layer, branch, KV head and
    entry) within HIDDEN_RTOL norm-relative;
  - p_top (the step's max softmax probability, Eq. gen_conf) within P_ATOL: with
    logits off by at most d, p_top moves by at most about 2 d p_top, and the
    hi/lo-split activations keep d near 1e-3 for logits of size ~10;
  - next_token: the oracle's logit at the GPU's token within Z_ATOL of the
    oracle's maximum (the argmax is unique only up to near-ties);
  - conf within t * P_ATOL of the oracle's running sum;
  - the gate exactly, on the GPU's own fp32 confidences (cases away from the
    thresholds: the GPU decides in fp32, the oracle in fp64).
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import HIDDEN_RTOL, host_view, log, oracle_cfg, to_np

pytestmark = pytest.mark.gpu
DEV = "cuda"
P_ATOL = 5e-3
Z_ATOL = 5e-2

GQA_BF16 = workloads.ModelShape(n_layers=3, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=1376,
                                vocab=5000, dtype="bf16", lm_head_scale=6.0)


def _row_rel(a, ref):
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return np.linalg.norm(a - ref, axis=-1) / np.maximum(np.linalg.norm(ref, axis=-1), 1e-30)


def _storage(x, dtype):
    """The oracle's cache as the GPU stores it (bf16: round to nearest even)."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16).double().numpy()
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def _check_step(label, z_ref, tok, p_top, sample):
    tok_ref, p_ref = oracle.top1(z_ref)
    for j, b in enumerate(sample):
        t = int(tok[b])
        assert 0 <= t < z_ref.shape[1], f"{label} branch {b}: token {t} out of range"
        gap = z_ref[j].max() - z_ref[j, t]
        assert gap <= Z_ATOL, f"{label} branch {b}: gpu token {t} logit {gap:.3e} below the max ({tok_ref[j]})"
        assert abs(p_top[b] - p_ref[j]) <= P_ATOL, f"{label} branch {b}: p_top {p_top[b]} vs {p_ref[j]}"
    return p_ref


def _decode_parity(shape, n, B, s, steps, seed, label, n_layers=None, sample=None, synthetic_prefix=False):
    """Suffix + `steps` teacher-forced steps on the GPU (all B branches); the oracle checks the
    branches in `sample` (default all) at every step, and their branch cache at the end."""
    mw = workloads.make_model(shape, seed=seed, device=DEV, n_layers=n_layers)
    L = len(mw.layers)
    host, cfg = host_view(mw), oracle_cfg(shape, L)
    sample = list(range(B)) if sample is None else sample
    if n == 0:
        pk = pv = None
        k = v = None
    elif synthetic_prefix:
        kv = workloads.make_prefix_kv(shape, n, seed=seed, n_layers=L)
        pk, pv = kv.k.double().numpy(), kv.v.double().numpy()
        k, v = kv.k.to(DEV), kv.v.to(DEV)
    else:
        prefix = workloads.make_tokens(n, shape.vocab, seed=seed, name="prefix").numpy()
        log(f"[{label}] oracle prefill n={n}")
        pk, pv, _ = oracle.prefill(host, cfg, prefix)
        pk, pv = _storage(pk, shape.dtype), _storage(pv, shape.dtype)
        tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        k = torch.from_numpy(pk).to(tdt).to(DEV).contiguous()
        v = torch.from_numpy(pv).to(tdt).to(DEV).contiguous()
    suffix = workloads.make_tokens(B * s, shape.vocab, seed=seed, name="suffix").reshape(B, s)
    gen = workloads.make_tokens(max(steps, 1) * B, shape.vocab, seed=seed, name="decode").reshape(-1, B)

    dec = rk.Decoder(mw, k, v, B, s, capacity=s + steps, device=DEV)
    log(f"[{label}] gpu suffix B={B} s={s} n={n} L={L}")
    tok, pt = dec.suffix(suffix.to(DEV))
    torch.cuda.synchronize()
    gpu_tok, gpu_p = [to_np(tok).copy()], [to_np(pt).copy()]
    for j in range(steps):
        log(f"[{label}] gpu step {j + 1} (cache length {dec.cache.length})")
        tok, pt = dec.step(gen[j].to(DEV).contiguous())
        torch.cuda.synchronize()
        gpu_tok.append(to_np(tok).copy())
        gpu_p.append(to_np(pt).copy())
    conf = to_np(dec.conf)
    assert dec.cache.length == s + steps and dec.n_steps == steps + 1

    log(f"[{label}] oracle suffix + {steps} steps on branches {sample}")
    sub = np.asarray(sample)
    ck, cv, z = oracle.decode_suffix(host, cfg, pk, pv, suffix.numpy()[sub])
    p_refs = [_check_step(f"{label} suffix", z, gpu_tok[0], gpu_p[0], sample)]
    for j in range(steps):
        k1, v1, z = oracle.decode_step(host, cfg, pk, pv, _storage(ck, shape.dtype), _storage(cv, shape.dtype),
                                       gen[j].numpy()[sub])
        ck, cv = np.concatenate([ck, k1], axis=3), np.concatenate([cv, v1], axis=3)
        p_refs.append(_check_step(f"{label} step {j + 1}", z, gpu_tok[j + 1], gpu_p[j + 1], sample))
    p_refs = np.stack(p_refs)                                     # [t, len(sample)]
    perr = max(float(np.abs(np.stack(gpu_p)[:, sub] - p_refs).max()), 0.0)
    cerr = float(np.abs(conf[sub] - p_refs.sum(axis=0)).max())
    assert cerr <= (steps + 1) * P_ATOL, f"{label}: conf err {cerr}"
    gk = to_np(dec.cache.k.float())[:, sub, :, : s + steps]
    gv = to_np(dec.cache.v.float())[:, sub, :, : s + steps]
    ek, ev = _row_rel(gk, ck).max(), _row_rel(gv, cv).max()
    log(f"[{label}] max p_top err {perr:.2e} conf err {cerr:.2e} cache K {ek:.2e} V {ev:.2e}")
    assert ek <= HIDDEN_RTOL and ev <= HIDDEN_RTOL
    return dec, p_refs


@pytest.mark.parametrize("name", ["tiny", "tiny_deep"])
def test_decode_fp32(name):
    wl = workloads.get(name)
    _decode_parity(wl.model, wl.prefix_len, wl.n_branches, wl.branch_len, 3, 31, f"decode {name}")


@pytest.mark.parametrize("shape,n,B,s,steps", [
    (dataclasses.replace(workloads.get("tiny_deep").model, dtype="bf16"), 64, 4, 16, 3),
    (GQA_BF16, 100, 5, 62, 4),     # the own keys cross a block of 64 during the steps
    (GQA_BF16, 129, 1, 1, 2),      # one branch, one-token suffix
    (GQA_BF16, 0, 3, 5, 2),        # no prefix: own keys only
    (GQA_BF16, 700, 6, 9, 2),      # several split-KV chunks of the prefix
    (GQA_BF16, 300, 20, 4, 2),     # more than 16 branches: the 128-row projections instead of the weight stream
], ids=["tiny_deep_bf16", "gqa_cross64", "gqa_single", "gqa_noprefix", "gqa_chunks", "gqa_b20"])
def test_decode_bf16(shape, n, B, s, steps):
    _decode_parity(shape, n, B, s, steps, 32, f"decode {shape.d_model}x{shape.n_layers} n={n} B={B} s={s}")


def test_decode_7b_shape_two_layers():
    """Full 7B width, B = 8 branches over a 1024-token prefix, two layers; the oracle samples two branches."""
    wl = workloads.get("7b_single")
    _decode_parity(wl.model, wl.prefix_len, 8, 8, 1, 42, "decode 7b", n_layers=2, sample=[0, 5],
                   synthetic_prefix=True)


def test_decode_loop_and_gate_end_to_end():
    """The GPU's running confidence feeds the GPU gate; the oracle gate runs on the oracle's own
    confidences (Eq. gen_conf). Decisions must agree unless the oracle's inputs are within the
    p_top bar of a threshold or of a tie."""
    shape = dataclasses.replace(workloads.get("tiny").model, dtype="bf16")
    dec, p_refs = _decode_parity(shape, 64, 4, 8, 5, 33, "decode+gate")
    conf = to_np(dec.conf)
    p_ref = oracle.gen_confidence(p_refs)
    srt = np.sort(p_ref)
    for tau, rg in ((0.70, 0.06), (0.72, 0.10), (0.0, 0.0), (1.01, 0.0), (srt[-1] - 0.05, 0.0)):
        fired, winner, p_mean, stats = dec.gate(tau, rg)
        torch.cuda.synchronize()
        pm = to_np(p_mean)
        np.testing.assert_allclose(pm, conf / dec.n_steps, rtol=1e-6)
        assert np.abs(pm - p_ref).max() <= P_ATOL
        ref = oracle.cgee_gate(p_ref, tau, rg)
        st = to_np(stats)
        log(f"[gate tau={tau:.3f} r={rg}] gpu fired={int(to_np(fired)[0])} winner={int(to_np(winner)[0])} "
            f"stats={st.round(4).tolist()} oracle {ref}")
        if srt[-1] - srt[-2] > 2 * P_ATOL:
            assert int(to_np(winner)[0]) == ref["winner"]
        if abs(ref["max"] - tau) > P_ATOL and abs(ref["gap"] - rg) > 4 * P_ATOL / max(ref["max"], 1e-3):
            assert bool(to_np(fired)[0]) == ref["fired"]
        np.testing.assert_allclose(st[:2], [ref["max"], ref["second"]], atol=P_ATOL)


def _gate_gpu(conf, n_steps, tau, rg):
    c = torch.tensor(np.asarray(conf, dtype=np.float32), device=DEV)
    fired, winner, p_mean, stats = rk.cgee_gate(c, n_steps, tau, rg)
    torch.cuda.synchronize()
    return bool(to_np(fired)[0]), int(to_np(winner)[0]), to_np(p_mean), to_np(stats)


def test_gate_paper_examples_on_gpu():
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "cgee_gate_examples.json")) as f:
        g = json.load(f)
    rng = np.random.default_rng(3)
    for ex in g["examples"]:
        p = np.concatenate([[ex["max"], ex["second"]], rng.uniform(0, ex["second"], g["n_branches"] - 2)])
        p = p[rng.permutation(len(p))]
        t = 32
        fired, winner, pm, st = _gate_gpu(p * t, t, g["tau_conf"], g["r_gap"])
        assert fired == ex["fires"], ex["name"]
        assert winner == int(np.argmax(p))
        assert round(float(st[2]), 2) == ex["printed_gap_ratio"]


def test_gate_random_ties_nan_single():
    """Seeded confidences; the oracle takes p = conf / t from the same fp32 conf values in fp64."""
    rng = np.random.default_rng(4)
    for B in (1, 2, 3, 8, 33, 64):
        for trial in range(6):
            p = rng.uniform(0.2, 1.0, B)
            if B > 1 and trial % 3 == 1:
                p[rng.integers(0, B)] = p.max()
            if B > 2 and trial % 3 == 2:
                p[rng.integers(0, B)] = np.nan
            t = int(rng.integers(1, 129))
            tau, rg = float(rng.uniform(0.3, 0.95)), float(rng.uniform(0.0, 0.4))
            conf = (p * t).astype(np.float32)
            fired, winner, pm, st = _gate_gpu(conf, t, tau, rg)
            p_in = conf.astype(np.float64) / t
            np.testing.assert_allclose(pm, p_in, rtol=1e-7)
            ref = oracle.cgee_gate(p_in, tau, rg)
            assert winner == ref["winner"], (B, trial)
            if abs(ref["max"] - tau) > 1e-5 and abs(ref["gap"] - rg) > 1e-5:
                assert fired == ref["fired"], (B, trial, ref)
            np.testing.assert_allclose(st, [ref["max"], ref["second"], ref["gap"]], rtol=1e-5, atol=1e-7)
    fired, winner, _, st = _gate_gpu([np.nan, np.nan], 4, 0.0, 0.0)
    assert not fired and winner == -1 and np.isnan(st[0])
