"""The pre-tiled gate|up weight (rksc_tile_gate_up; rksc_layer_weights.w_gate_up_tiled).

The copy is a pure storage layout: its bytes are the stated block permutation of
w_gate_up, and every call that reads it returns outputs bitwise identical to the
same call without it (that plain path is the one the oracle parity tests pin).
One verify case on the tiled weights is also checked against the oracle."""
import numpy as np
import pytest
import torch

import paper_2606_09937_amd as rk
import workloads
from gpu_util import compare_verify, host_view, log, oracle_cfg, to_np

import oracle

pytestmark = pytest.mark.gpu
DEV = "cuda"

# 2 d_ff = 44 x 256: the 128-row gate|up plans take 256-column tiles from 64 to 256 rows.
MID = workloads.ModelShape(n_layers=2, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128, d_ff=5632,
                           vocab=6000, dtype="bf16", lm_head_scale=6.0)


def _tiled_copy(mw):
    """The same weights with every layer's tiled gate|up copy added (the plain model is untouched)."""
    mt = workloads.ModelWeights(mw.shape, mw.embed, [dict(lw) for lw in mw.layers], mw.final_norm, mw.lm_head)
    assert rk.tile_gate_up(mt)
    torch.cuda.synchronize()
    return mt


def _uses_tiles(shape, M):
    """Whether the gate|up projection of M rows runs the kernel that reads the tiled copy."""
    p = rk.rksc_test_gemm_plan(M, 2 * shape.d_ff, shape.d_model)
    return p["kind"] == 0 and p["bn"] == 256 and p["k_per_split"] % 64 == 0


def _bits(t):
    return to_np(t.contiguous().view(torch.int16) if t.dtype == torch.bfloat16 else t)


@pytest.mark.parametrize("name", ["mid", "7b"])
def test_tiled_layout_is_the_block_permutation(name):
    shape = MID if name == "mid" else workloads.get("7b_single").model
    mw = workloads.make_model(shape, seed=5, device=DEV, n_layers=1)
    w = mw.layers[0]["w_gate_up"]
    F2, d = w.shape
    assert rk.rksc_gate_up_tiled_bytes(shape) == w.numel() * 2
    out = torch.full_like(w, float("nan"))
    rk.rksc_tile_gate_up(shape, w, out)
    torch.cuda.synchronize()
    want = w.view(F2 // 256, 256, d // 64, 64).permute(0, 2, 1, 3).contiguous().view(F2, d)
    assert torch.equal(out.view(torch.int16), want.view(torch.int16))


def test_fp32_and_untileable_models_have_no_tiled_copy():
    tiny = workloads.get("tiny").model
    mw = workloads.make_model(tiny, seed=5, device=DEV)
    assert rk.rksc_gate_up_tiled_bytes(tiny) == 0
    assert not rk.tile_gate_up(mw) and "w_gate_up_tiled" not in mw.layers[0]
    # set by hand on a model without the layout, it is refused before any launch
    mw.layers[1]["w_gate_up_tiled"] = mw.layers[1]["w_gate_up"].clone()
    kv = workloads.make_prefix_kv(tiny, 8, seed=5, device=DEV)
    toks = workloads.make_tokens(16, tiny.vocab, seed=5, device=DEV).reshape(1, 16)
    with pytest.raises(rk.RkscError, match="w_gate_up_tiled"):
        rk.verify_forward(mw, kv.k, kv.v, toks, 0.1, 1)


@pytest.mark.parametrize("case,B,s,n,tiles", [
    ("mid_64rows", 4, 16, 200, True),
    ("mid_128rows", 1, 128, 300, True),
    ("mid_256rows", 2, 128, 100, True),
    ("mid_1024rows", 8, 128, 64, False),
    ("7b_128rows_2layers", 1, 128, 1024, True),
    ("28l_128rows_2layers", 1, 128, 512, True),    # d = 3584, 2F = 148 x 256
])
def test_verify_with_tiled_copy_is_bitwise_identical(case, B, s, n, tiles):
    if case.startswith("7b"):
        shape, L = workloads.get("7b_single").model, 2
    elif case.startswith("28l"):
        shape, L = workloads.get("7b_paper_verify").model, 2
    else:
        shape, L = MID, None
    assert _uses_tiles(shape, B * s) == tiles
    mw = workloads.make_model(shape, seed=23, device=DEV, n_layers=L)
    kv = workloads.make_prefix_kv(shape, n, seed=23, device=DEV, n_layers=L)
    toks = workloads.make_tokens(B * s, shape.vocab, seed=23, device=DEV).reshape(B, s).contiguous()
    mt = _tiled_copy(mw)
    for tau, patience in ((0.0, 1), (10.0, 1)):     # no exit; every branch out at layer 2
        log(f"[{case}] tau={tau}")
        a = rk.verify_forward(mw, kv.k, kv.v, toks, tau, patience, return_hidden=True)
        b = rk.verify_forward(mt, kv.k, kv.v, toks, tau, patience, return_hidden=True)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            np.testing.assert_array_equal(_bits(x), _bits(y))


def test_verify_with_tiled_copy_matches_oracle():
    B, s, n = 1, 128, 160
    mw = _tiled_copy(workloads.make_model(MID, seed=31, device=DEV))
    kv = workloads.make_prefix_kv(MID, n, seed=31, device=DEV)
    toks = workloads.make_tokens(B * s, MID.vocab, seed=31, device=DEV).reshape(B, s).contiguous()
    tau, patience = 0.05, 1
    ent, ex, hid = (to_np(t) for t in rk.verify_forward(mw, kv.k, kv.v, toks, tau, patience, return_hidden=True))
    log("[mid tiled] oracle")
    _, ex_ref, _, ent_ref, hid_ref = oracle.verify_forward(host_view(mw), oracle_cfg(MID, MID.n_layers),
                                                           kv.k.cpu(), kv.v.cpu(), toks.cpu().numpy(), tau,
                                                           patience)
    stats = compare_verify(ent, ex, hid, ent_ref, hid_ref, ex_ref, tau, label="mid tiled")
    log(f"[mid tiled] {stats}")


def test_prefill_extend_and_decode_with_tiled_copy_are_bitwise_identical():
    """Root forward (200 rows), tree-node extension (64 rows) and a decode suffix of 4 x 16 rows with
    two one-token steps (4 rows: the weight-streaming plan, which ignores the copy)."""
    mw = workloads.make_model(MID, seed=41, device=DEV)
    mt = _tiled_copy(mw)
    root = workloads.make_tokens(200, MID.vocab, seed=41, name="root", device=DEV)
    node = workloads.make_tokens(64, MID.vocab, seed=41, name="node", device=DEV)
    suffix = workloads.make_tokens(64, MID.vocab, seed=41, name="suffix", device=DEV).reshape(4, 16).contiguous()
    gen = workloads.make_tokens(8, MID.vocab, seed=41, name="decode", device=DEV).reshape(2, 4)
    assert _uses_tiles(MID, 200) and _uses_tiles(MID, 64)
    outs = []
    for m in (mw, mt):
        k, v, h = rk.prefill(m, root)
        ek, ev, eh = rk.prefix_extend(m, k, v, node)
        dec = rk.Decoder(m, k, v, 4, 16, capacity=18, device=DEV)
        got = [k, v, h, ek, ev, eh, *(t.clone() for t in dec.suffix(suffix))]
        for j in range(2):
            got += [t.clone() for t in dec.step(gen[j].contiguous())]
        got += [dec.conf, dec.cache.k, dec.cache.v]
        torch.cuda.synchronize()
        outs.append([_bits(t) for t in got])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)
