"""Precision budget of the verify pass (reading of Eq. entropy's 1e-2-nat bar): the
library carries fp32 operands as bf16 hi + lo pairs at every MFMA site. This
ablation drops the lo part at one site at a time (rksc_test_verify_precision) on
the 7B headline shape at full depth and on the large-vocab shape with 8 branches,
measures the largest entropy and hidden-row errors against the float64 oracle,
and prints the table. The library's own scheme (drop_mask 0) must meet the bars."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import ENTROPY_ATOL, HIDDEN_RTOL, host_view, log, oracle_cfg, to_np

pytestmark = pytest.mark.gpu
DEV = "cuda"

SITES = [("none", 0)] + [(k, v) for k, v in rk.RKSC_DROP.items()] + [
    ("attention (q, own_kv, p)", rk.RKSC_DROP["q"] | rk.RKSC_DROP["own_kv"] | rk.RKSC_DROP["p"]),
    ("qkv+o", rk.RKSC_DROP["qkv"] | rk.RKSC_DROP["o"]),
    ("qkv+o+attention", rk.RKSC_DROP["qkv"] | rk.RKSC_DROP["o"] | rk.RKSC_DROP["q"] | rk.RKSC_DROP["own_kv"]
     | rk.RKSC_DROP["p"]),
    ("gate_up+down", rk.RKSC_DROP["gate_up"] | rk.RKSC_DROP["down"]),
    ("all", 0xFF),
]


def _table(name, n_layers, branches):
    wl = workloads.get(name)
    shape = wl.model
    mw = workloads.make_model(shape, seed=42, device=DEV, n_layers=n_layers)
    kv = workloads.make_prefix_kv(shape, wl.prefix_len, seed=42, device=DEV, n_layers=n_layers)
    toks = workloads.make_tokens(wl.n_branches * wl.branch_len, shape.vocab, seed=42,
                                 device=DEV).reshape(wl.n_branches, wl.branch_len).contiguous()
    L = n_layers
    log(f"[precision {name}] oracle on branches {branches}")
    _, _, _, ent_ref, hid_ref = oracle.verify_forward(host_view(mw), oracle_cfg(shape, L), kv.k.cpu(), kv.v.cpu(),
                                                      toks.cpu().numpy()[branches], 0.0, 1)
    rows = []
    for site, mask in SITES:
        ent, ex, hid = rk.rksc_test_verify_precision(mw, kv.k, kv.v, toks, 0.0, 1, mask)
        torch.cuda.synchronize()
        ent, hid = to_np(ent)[:, branches], to_np(hid)[:, branches]
        e_err = np.abs(ent - ent_ref)
        h_rel = np.linalg.norm(hid - hid_ref, axis=-1) / np.linalg.norm(hid_ref, axis=-1)
        d_err = np.abs(np.diff(ent, axis=0) - np.diff(ent_ref, axis=0))
        rows.append((site, mask, float(e_err.max()), float(np.median(e_err)), float(d_err.max()), float(h_rel.max())))
    log(f"[precision {name}] L={L} branches={branches}: site dropped | max |dH| nats | median |dH| | "
        f"max delta err | max hidden rel")
    for site, mask, emax, emed, dmax, hmax in rows:
        ok = "ok" if emax <= ENTROPY_ATOL and hmax <= HIDDEN_RTOL else "FAILS"
        log(f"[precision {name}] {site:26s} 0x{mask:02x} | {emax:.2e} | {emed:.2e} | {dmax:.2e} | {hmax:.2e} | {ok}")
    base = rows[0]
    assert base[2] <= ENTROPY_ATOL and base[5] <= HIDDEN_RTOL
    return rows


def test_precision_sites_7b_single():
    wl = workloads.get("7b_single")
    _table("7b_single", wl.model.n_layers, [0])


def test_precision_sites_paper_verify():
    _table("7b_paper_verify", 28, [0, 5])
