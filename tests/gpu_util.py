"""Shared helpers of the GPU parity tests: device-resident inputs, a host view of
them for the oracle, and the parity criteria of the verify pass."""
from __future__ import annotations

import dataclasses
import math
import sys

import numpy as np
import torch

import workloads

ENTROPY_ATOL = 1e-2      # nats
HIDDEN_RTOL = 2e-2       # per (layer, branch) row, norm-relative
SIM_ATOL = 1e-3
NEAR_TAU = 1e-2          # an exit flip is excused if some oracle delta is this close to tau


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


class HostLayers:
    """Lazy host copies of device layer weights (bf16 stays bf16; the oracle widens exactly). A tiled
    gate|up copy is a device storage layout only and is left out."""

    def __init__(self, layers):
        self._layers = layers

    def __len__(self):
        return len(self._layers)

    def __getitem__(self, i):
        return {k: v.detach().cpu() for k, v in self._layers[i].items() if k != "w_gate_up_tiled"}


@dataclasses.dataclass
class HostModel:
    embed: torch.Tensor
    layers: HostLayers
    final_norm: torch.Tensor
    lm_head: torch.Tensor


def host_view(mw: workloads.ModelWeights) -> HostModel:
    return HostModel(mw.embed.detach().cpu(), HostLayers(mw.layers), mw.final_norm.detach().cpu(),
                     mw.lm_head.detach().cpu())


def oracle_cfg(shape, n_layers):
    return dataclasses.replace(shape, n_layers=n_layers)


def near_threshold(ent_ref_full: np.ndarray, tau: float, upto: int) -> bool:
    """True if some oracle delta |H_l - H_{l-1}|, 2 <= l <= upto, is within NEAR_TAU of tau."""
    for l in range(2, min(upto, len(ent_ref_full)) + 1):
        if abs(abs(ent_ref_full[l - 1] - ent_ref_full[l - 2]) - tau) <= NEAR_TAU:
            return True
    return False


def compare_verify(ent_gpu, ex_gpu, hid_gpu, ent_ref_full, hid_ref_full, ex_ref, tau, branches=None,
                   label=""):
    """Check GPU outputs against the oracle's full-depth values.

    ent_gpu [L, B], ex_gpu [B], hid_gpu [L, B, d] or None (numpy, GPU side);
    ent_ref_full [L, Bo], hid_ref_full [L, Bo, d], ex_ref [Bo] from the oracle, where
    branches[j] is the GPU branch index of oracle column j (default: all, in order).
    Returns a dict of statistics; raises AssertionError on a violation.
    """
    L = ent_gpu.shape[0]
    if branches is None:
        branches = list(range(ent_gpu.shape[1]))
    stats = {"max_entropy_err": 0.0, "max_hidden_rel": 0.0, "exit_match": 0, "near_threshold": 0}
    for j, b in enumerate(branches):
        eg, er = int(ex_gpu[b]), int(ex_ref[j])
        assert 1 <= eg <= L, f"{label} branch {b}: exit layer {eg} out of range"
        # NaN exactly after the GPU's own exit.
        assert not np.isnan(ent_gpu[:eg, b]).any(), f"{label} branch {b}: NaN entropy before exit"
        assert np.isnan(ent_gpu[eg:, b]).all(), f"{label} branch {b}: entropy not NaN after exit"
        if hid_gpu is not None:
            assert not np.isnan(hid_gpu[:eg, b]).any(), f"{label} branch {b}: NaN hidden before exit"
            assert np.isnan(hid_gpu[eg:, b]).all(), f"{label} branch {b}: hidden not NaN after exit"
        if eg == er:
            stats["exit_match"] += 1
        else:
            assert near_threshold(ent_ref_full[:, j], tau, max(eg, er)), (
                f"{label} branch {b}: exit {eg} (gpu) vs {er} (oracle), no oracle delta within "
                f"{NEAR_TAU} of tau={tau}; oracle H={ent_ref_full[:, j]}, gpu H={ent_gpu[:, b]}")
            stats["near_threshold"] += 1
        upto = min(eg, er)
        err = np.abs(ent_gpu[:upto, b] - ent_ref_full[:upto, j])
        stats["max_entropy_err"] = max(stats["max_entropy_err"], float(err.max()))
        assert err.max() <= ENTROPY_ATOL, (
            f"{label} branch {b}: entropy error {err.max():.3e} > {ENTROPY_ATOL} "
            f"(layer {int(err.argmax()) + 1}); gpu {ent_gpu[:upto, b]} oracle {ent_ref_full[:upto, j]}")
        if hid_gpu is not None:
            for l in range(upto):
                ref = hid_ref_full[l, j]
                rel = float(np.linalg.norm(hid_gpu[l, b] - ref) / np.linalg.norm(ref))
                stats["max_hidden_rel"] = max(stats["max_hidden_rel"], rel)
                assert rel <= HIDDEN_RTOL, f"{label} branch {b} layer {l + 1}: hidden rel error {rel:.3e}"
    return stats


def to_np(t):
    return t.detach().float().cpu().numpy() if t.dtype != torch.int32 else t.detach().cpu().numpy()


def entropy_of_uniform(V):
    return math.log(V)
