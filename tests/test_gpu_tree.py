"""Parity of tree sharing (rksc_prefix_extend) and of the ASKS gate
(rksc_asks_gate) with the float64 oracle, and the two execution paths the gate
selects (Sec. 2.2): a shared branch runs over the root cache, a branch below tau
over its own recomputed cache.

Bars: new cache rows and unit node rows within HIDDEN_RTOL norm-relative (the
node's cache holds only its own rows); verify outputs to the verify bars of
gpu_util; sigma within SIM_ATOL, and the shared flags equal unless the oracle's
sigma is within SIM_ATOL of tau (the device decides in fp32, the oracle in
fp64)."""
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
    return np.linalg.norm(a - ref, axis=-1) / np.maximum(np.linalg.norm(ref, axis=-1), 1e-30)


def _bf(x, dtype):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16).double().numpy()
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def _tdt(dtype):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


@pytest.mark.parametrize("shape,n,m", [
    (dataclasses.replace(workloads.get("tiny_deep").model, dtype="bf16"), 64, 20),
    (workloads.get("tiny").model, 64, 7),
    (GQA_BF16, 100, 33),
    (GQA_BF16, 0, 9),
], ids=["tiny_deep_bf16", "tiny_f32", "gqa_bf16", "gqa_empty_parent"])
def test_prefix_extend_matches_oracle(shape, n, m):
    mw = workloads.make_model(shape, seed=61, device=DEV)
    host, cfg = host_view(mw), oracle_cfg(shape, len(mw.layers))
    root = workloads.make_tokens(max(n, 1), shape.vocab, seed=61, name="prefix").numpy()[:n]
    node = workloads.make_tokens(m, shape.vocab, seed=61, name="node")
    if n:
        pk, pv, _ = oracle.prefill(host, cfg, root)
        pk, pv = _bf(pk, shape.dtype), _bf(pv, shape.dtype)
        gk = torch.from_numpy(pk).to(_tdt(shape.dtype)).to(DEV).contiguous()
        gv = torch.from_numpy(pv).to(_tdt(shape.dtype)).to(DEV).contiguous()
    else:
        pk = pv = gk = gv = None
    log(f"[extend n={n} m={m}] gpu")
    k, v, h = rk.prefix_extend(mw, gk, gv, node.to(DEV))
    torch.cuda.synchronize()
    ck, cv, ch = oracle.prefix_extend(host, cfg, pk, pv, node.numpy())
    # the node's cache holds its own m entries only; the parent is read in place, never copied
    assert k.shape[2] == m and v.shape[2] == m
    ek = _row_rel(to_np(k.float()), ck[:, :, n:]).max()
    ev = _row_rel(to_np(v.float()), cv[:, :, n:]).max()
    eh = _row_rel(to_np(h), oracle.unit_rows(ch)).max()
    log(f"[extend n={n} m={m}] new rows K {ek:.2e} V {ev:.2e} h_node {eh:.2e}")
    assert ek <= HIDDEN_RTOL and ev <= HIDDEN_RTOL and eh <= HIDDEN_RTOL


def test_tree_of_thought_sharing_end_to_end():
    """Root -> two depth-1 nodes (each computed once) -> a depth-2 node under each -> two leaves
    per node, verified over the chain root, node (, node) read in place: every leaf matches the
    oracle's verify over the concatenated cache of its path."""
    wl = workloads.get("tiny_deep")
    shape = dataclasses.replace(wl.model, dtype="bf16")
    mw = workloads.make_model(shape, seed=62, device=DEV)
    L = len(mw.layers)
    host, cfg = host_view(mw), oracle_cfg(shape, L)
    root = workloads.make_tokens(64, shape.vocab, seed=62, name="prefix", device=DEV)
    rk_k, rk_v, _ = rk.prefill(mw, root)
    ok_k, ok_v, _ = oracle.prefill(host, cfg, root.cpu().numpy())
    ok_k, ok_v = _bf(ok_k, "bf16"), _bf(ok_v, "bf16")
    root_cache = rk.PrefixCache([(rk_k, rk_v)])
    for node_id in range(2):
        node = workloads.make_tokens(12, shape.vocab, seed=62 + node_id, name="node", device=DEV)
        nk, nv, _ = rk.prefix_extend(mw, root_cache, None, node)
        onk, onv, _ = oracle.prefix_extend(host, cfg, ok_k, ok_v, node.cpu().numpy())
        onk, onv = _bf(onk, "bf16"), _bf(onv, "bf16")            # [root; node] entries
        path1 = root_cache.extend(nk, nv)
        # one level further: a 7-token node under this one, read over the chain root, node1
        node2 = workloads.make_tokens(7, shape.vocab, seed=80 + node_id, name="node", device=DEV)
        n2k, n2v, _ = rk.prefix_extend(mw, path1, None, node2)
        o2k, o2v, _ = oracle.prefix_extend(host, cfg, onk, onv, node2.cpu().numpy())
        o2k, o2v = _bf(o2k, "bf16"), _bf(o2v, "bf16")            # [root; node1; node2]
        path2 = path1.extend(n2k, n2v)
        leaves = workloads.make_tokens(2 * 8, shape.vocab, seed=70 + node_id, device=DEV).reshape(2, 8).contiguous()
        for depth, path, (rk_, rv_) in ((1, path1, (onk, onv)), (2, path2, (o2k, o2v))):
            for tau in (0.3, 0.0):
                ent, ex, hid = rk.verify_forward(mw, path, None, leaves, tau, 1, return_hidden=True)
                torch.cuda.synchronize()
                _, ex_ref, _, ent_ref, hid_ref = oracle.verify_forward(host, cfg, rk_, rv_, leaves.cpu().numpy(), tau,
                                                                       1)
                stats = compare_verify(to_np(ent), to_np(ex), to_np(hid), ent_ref, hid_ref, ex_ref, tau,
                                       label=f"node {node_id} depth {depth} tau={tau}")
                log(f"[tree node {node_id} depth {depth} tau={tau}] exits {to_np(ex).tolist()} "
                    f"oracle {ex_ref.tolist()} {stats}")


def test_asks_gated_execution_end_to_end():
    """Branches with their own phrasings of the prompt: each phrasing's root rows (its own prefill)
    go through the device gate against the root's; a shared branch verifies its suffix over the
    root cache, the others over their own phrasing's cache. Identical phrasings share."""
    wl = workloads.get("tiny_deep")
    shape = dataclasses.replace(wl.model, dtype="bf16")
    mw = workloads.make_model(shape, seed=63, device=DEV)
    L = len(mw.layers)
    host, cfg = host_view(mw), oracle_cfg(shape, L)
    n, B, s = 48, 4, 8
    root = workloads.make_tokens(n, shape.vocab, seed=63, name="prefix", device=DEV)
    other = workloads.make_tokens(2 * n, shape.vocab, seed=63, name="phrasing", device=DEV).reshape(2, n)
    phr = [root, other[0].contiguous(), root, other[1].contiguous()]
    rk_k, rk_v, rk_h = rk.prefill(mw, root)
    own = [rk.prefill(mw, p) for p in phr]
    hidden = torch.stack([o[2] for o in own], dim=1).contiguous()          # [L, B, d]
    for tau in (0.82, 0.5, -1.0):
        sigma, shared = rk.asks_gate(hidden, rk_h, wl.alpha, tau)
        torch.cuda.synchronize()
        o_h = [oracle.unit_rows(oracle.prefill(host, cfg, p.cpu().numpy())[2]) for p in phr]
        o_sigma, o_shared = oracle.asks_gate(np.stack(o_h, axis=1), o_h[0], wl.alpha, tau)
        sg, sh = to_np(sigma), to_np(shared)
        log(f"[asks tau={tau}] sigma gpu {sg.round(4).tolist()} oracle {o_sigma.round(4).tolist()} "
            f"shared {sh.tolist()}")
        assert np.abs(sg - o_sigma).max() <= SIM_ATOL
        for b in range(B):
            if abs(o_sigma[b] - tau) > SIM_ATOL:
                assert bool(sh[b]) == bool(o_shared[b])
        assert sh[0] == 1 and sh[2] == 1                                   # identical phrasings
    # Execute the oracle's choice at tau = 0.82 (checked above to be the device's away from tau) on
    # both sides, and compare every branch with the oracle's path.
    o_h = [oracle.unit_rows(oracle.prefill(host, cfg, p.cpu().numpy())[2]) for p in phr]
    sh = oracle.asks_gate(np.stack(o_h, axis=1), o_h[0], wl.alpha, 0.82)[1]
    sfx = workloads.make_tokens(B * s, shape.vocab, seed=64, device=DEV).reshape(B, s).contiguous()
    for b in range(B):
        k, v = (rk_k, rk_v) if sh[b] else own[b][:2]
        toks = sfx[b:b + 1].contiguous()
        ent, ex, hid = rk.verify_forward(mw, k, v, toks, 0.0, 1, return_hidden=True)
        torch.cuda.synchronize()
        src = root if sh[b] else phr[b]
        ok_k, ok_v, _ = oracle.prefill(host, cfg, src.cpu().numpy())
        _, ex_ref, _, ent_ref, hid_ref = oracle.verify_forward(host, cfg, _bf(ok_k, "bf16"), _bf(ok_v, "bf16"),
                                                               toks.cpu().numpy(), 0.0, 1)
        compare_verify(to_np(ent), to_np(ex), to_np(hid), ent_ref, hid_ref, ex_ref, 0.0,
                       label=f"asks branch {b} shared={int(sh[b])}")
