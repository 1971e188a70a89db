"""The host runtime of librksc on the CPU: the RSBCM block table (Alg. RsbcmEvict)
against the oracle's eviction, bit-exact on ids and order, over seeded random
operation sequences; and the argument checks of the block table and the KV
probe (which validate before any GPU call)."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2606_09937_amd as rk
import workloads

FAKE = ctypes.c_void_p(0x1000)   # never dereferenced


class OracleTable:
    """The oracle's view of a block table: insertion-ordered (id, score, depth) entries."""

    def __init__(self, cap):
        self.cap, self.rows = cap, []

    def insert(self, i, score, depth):
        self.rows.append((i, float(np.float32(score)), depth))

    def set_score(self, i, score):
        self.rows = [(j, float(np.float32(score)) if j == i else s, d) for j, s, d in self.rows]

    def remove(self, i):
        self.rows = [r for r in self.rows if r[0] != i]

    def evict(self):
        self.rows, ev = oracle.rsbcm_evict(self.rows, self.cap)
        return ev


def test_block_table_stress_test_count():
    """App. RSBCM validation through the library: capacity 4, 8 branch blocks per solve,
    20 solves -> 4 evictions each, 80 in total."""
    rng = np.random.default_rng(20)
    total = 0
    for problem in range(20):
        t, o = rk.BlockTable(4), OracleTable(4)
        for b in range(8):
            sc, dp = float(rng.uniform(0, 1)), int(rng.integers(0, 4))
            t.insert(1000 * problem + b, sc, dp)
            o.insert(1000 * problem + b, sc, dp)
        ev = t.evict()
        assert ev == o.evict() and len(ev) == 4 and len(t) == 4 and t.evicted_total == 4
        total += len(ev)
    assert total == 80


@pytest.mark.parametrize("seed", range(8))
def test_block_table_matches_oracle_random_ops(seed):
    rng = np.random.default_rng(100 + seed)
    cap = int(rng.integers(0, 12))
    t, o = rk.BlockTable(cap), OracleTable(cap)
    next_id, live = 0, []
    evicted_total = 0
    for _ in range(400):
        op = rng.uniform()
        if op < 0.5 or not live:
            # scores from a small set make equal omegas (ties) common
            sc = float(rng.choice([0.5, 0.25, 1.0, float(rng.uniform(-0.5, 1.5))]))
            dp = int(rng.integers(0, 4))
            t.insert(next_id, sc, dp)
            o.insert(next_id, sc, dp)
            live.append(next_id)
            next_id += 1
        elif op < 0.65:
            i = int(rng.choice(live))
            sc = float(rng.uniform(0, 1))
            t.set_score(i, sc)
            o.set_score(i, sc)
        elif op < 0.75:
            i = int(rng.choice(live))
            t.remove(i)
            o.remove(i)
            live.remove(i)
        else:
            ev = t.evict()
            assert ev == o.evict()
            evicted_total += len(ev)
            live = [i for i in live if i not in ev]
            assert len(t) == len(o.rows) <= cap
        assert len(t) == len(o.rows)
    assert t.evicted_total == evicted_total


def test_block_table_rejects_bad_arguments():
    lib = rk.load_library()
    assert lib.rksc_block_table_create(-1) is None
    t = rk.BlockTable(2)
    t.insert(7, 0.5, 1)
    with pytest.raises(rk.RkscError):
        t.insert(7, 0.4, 0)                    # duplicate id
    with pytest.raises(rk.RkscError):
        t.insert(8, float("nan"), 0)
    with pytest.raises(rk.RkscError):
        t.insert(8, 0.5, -1)
    with pytest.raises(rk.RkscError):
        t.set_score(99, 0.5)
    with pytest.raises(rk.RkscError):
        t.remove(99)
    t.insert(8, 0.1, 0)
    t.insert(9, 0.2, 0)
    n = ctypes.c_int32(-1)
    buf = (ctypes.c_int64 * 1)()
    # one block must go but the output array holds none: nothing is evicted
    assert lib.rksc_block_table_evict(t._t, buf, 0, ctypes.byref(n)) == rk.RKSC_ERR_INVALID_ARGUMENT
    assert len(t) == 3
    assert lib.rksc_block_table_evict(None, buf, 1, ctypes.byref(n)) == rk.RKSC_ERR_INVALID_ARGUMENT
    assert t.evict() == [8] and len(t) == 2
    assert lib.rksc_block_table_size(None) == -1


def test_kv_probe_rejects_bad_arguments_before_any_launch():
    lib = rk.load_library()
    assert lib.rksc_kv_probe_create(0) is None
    shape = workloads.get("tiny").model
    cfg = rk.model_config(shape)
    assert lib.rksc_kv_probe_workspace_size(ctypes.byref(cfg), 0, 4, 8) == 0
    assert lib.rksc_kv_probe_workspace_size(ctypes.byref(cfg), 64, 0, 8) == 0
    ws = lib.rksc_kv_probe_workspace_size(ctypes.byref(cfg), 64, 4, 8)
    assert ws >= lib.rksc_decode_workspace_size(ctypes.byref(cfg), 4, 72, 0)
    p = rk.KVProbe(3)
    assert p.lookup(64) is None
    share = ctypes.c_int32(0)
    layers = (rk.LayerWeights * shape.n_layers)()
    for i in range(shape.n_layers):
        layers[i] = rk.LayerWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    w = rk.Weights(cfg, FAKE, layers, FAKE, FAKE)
    I = rk.RKSC_ERR_INVALID_ARGUMENT
    call = lambda **k: lib.rksc_kv_probe_decide(  # noqa: E731
        k.get("p", p._p), ctypes.byref(w), k.get("pt", FAKE), k.get("n", 64), FAKE, 4, 8,
        k.get("wsp", ctypes.c_void_p(0x100000)), k.get("wsb", ws), None, k.get("share", ctypes.byref(share)),
        None, None)
    assert call(p=None) == I
    assert call(share=None) == I
    assert call(n=0) == I
    assert call(pt=None) == I
    assert call(wsp=None) == I
    assert call(wsp=ctypes.c_void_p(0x100080)) == I
    assert call(wsb=ws - 1) == rk.RKSC_ERR_WORKSPACE_TOO_SMALL
    assert p.lookup(64) is None                # nothing was stored
