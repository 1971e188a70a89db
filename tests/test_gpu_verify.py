"""Parity of the HIP verify pass (rksc_verify_forward through the C ABI) with the
float64 oracle, on the same seeded inputs.

Bars: exit_layer identical except where an oracle entropy delta lies within
1e-2 nats of tau; entropy within 1e-2 nats; hidden rows within 2e-2 relative;
outputs NaN exactly after each branch's exit.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import compare_verify, host_view, log, oracle_cfg, to_np

pytestmark = pytest.mark.gpu
DEV = "cuda"

# Small bf16 decoders with ragged tails everywhere: d_ff and vocab not multiples
# of the tiles, G = 4 and G = 7 grouped-query attention, odd branch counts.
GQA_BF16 = workloads.ModelShape(n_layers=4, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=1376,
                                vocab=5000, dtype="bf16", lm_head_scale=6.0)
G7_BF16 = workloads.ModelShape(n_layers=3, d_model=448, n_heads=7, n_kv_heads=1, head_dim=64, d_ff=1200,
                               vocab=3001, dtype="bf16", lm_head_scale=6.0)


def _inputs(shape, B, n, s, seed, device=DEV, n_layers=None):
    mw = workloads.make_model(shape, seed=seed, device=device, n_layers=n_layers)
    kv = workloads.make_prefix_kv(shape, n, seed=seed, device=device, n_layers=n_layers)
    toks = workloads.make_tokens(B * s, shape.vocab, seed=seed, device=device).reshape(B, s).contiguous()
    return mw, kv, toks


def _run_gpu(mw, kv, toks, tau, patience):
    ent, ex, hid = rk.verify_forward(mw, kv.k, kv.v, toks, tau, patience, return_hidden=True)
    torch.cuda.synchronize()
    return to_np(ent), to_np(ex), to_np(hid)


def _run_oracle(mw, kv, toks, tau, patience, branches=None):
    shape = mw.shape
    L = len(mw.layers)
    hv = host_view(mw)
    t = toks.cpu().numpy()
    if branches is not None:
        t = t[branches]
    _, ex, _, ent_full, hid_full = oracle.verify_forward(hv, oracle_cfg(shape, L), kv.k.cpu(), kv.v.cpu(), t,
                                                         tau, patience)
    return ent_full, hid_full, ex


def _parity(mw, kv, toks, tau, patience, label, branches=None):
    log(f"[{label}] gpu")
    ent, ex, hid = _run_gpu(mw, kv, toks, tau, patience)
    log(f"[{label}] oracle")
    ent_ref, hid_ref, ex_ref = _run_oracle(mw, kv, toks, tau, patience, branches)
    stats = compare_verify(ent, ex, hid, ent_ref, hid_ref, ex_ref, tau, branches=branches, label=label)
    log(f"[{label}] exits gpu={ex.tolist()} oracle={ex_ref.tolist()} {stats}")
    return ent, ex, hid, stats


@pytest.mark.parametrize("name", ["tiny", "tiny_deep"])
def test_tiny_fp32_synthetic_prefix(name):
    wl = workloads.get(name)
    mw, kv, toks = _inputs(wl.model, wl.n_branches, wl.prefix_len, wl.branch_len, seed=42)
    _parity(mw, kv, toks, wl.tau, wl.patience, name)


def test_tiny_deep_fp32_prefill_prefix_and_exits():
    """Prefix cache from the oracle's own root forward (Eq. prefix_fwd); several taus so exits fire."""
    wl = workloads.get("tiny_deep")
    shape = wl.model
    mw = workloads.make_model(shape, seed=7, device=DEV)
    prefix = workloads.make_tokens(wl.prefix_len, shape.vocab, seed=7, name="prefix").numpy()
    pk, pv, _ = oracle.prefill(host_view(mw), shape, prefix)
    kv = workloads.PrefixKV(torch.from_numpy(pk).float().to(DEV), torch.from_numpy(pv).float().to(DEV))
    toks = workloads.make_tokens(wl.n_branches * wl.branch_len, shape.vocab, seed=7,
                                 device=DEV).reshape(wl.n_branches, wl.branch_len).contiguous()
    exits = set()
    for tau, pat in ((wl.tau, wl.patience), (0.3, 1), (1.0, 2), (0.0, 1), (math.inf, 3)):
        _, ex, _, _ = _parity(mw, kv, toks, tau, pat, f"tiny_deep_prefill tau={tau} p={pat}")
        exits |= set(ex.tolist())
    assert len(exits) > 1, "the sweep should produce more than one exit depth"


@pytest.mark.parametrize("shape,B,n,s", [
    (dataclasses.replace(workloads.get("tiny").model, dtype="bf16"), 4, 64, 16),
    (dataclasses.replace(workloads.get("tiny_deep").model, dtype="bf16"), 3, 50, 21),
    (GQA_BF16, 5, 100, 40),
    (G7_BF16, 2, 129, 65),
    # wide batches: 17..32 and 33..64 live columns take the lm_head kernel's
    # two- and four-block variants; 64 is the largest batch the ABI accepts
    (dataclasses.replace(workloads.get("tiny_deep").model, dtype="bf16"), 20, 30, 5),
    (G7_BF16, 37, 9, 2),
    (GQA_BF16, 64, 16, 3),
], ids=["tiny_bf16", "tiny_deep_bf16", "gqa_bf16", "g7_bf16", "tiny_deep_bf16_b20", "g7_bf16_b37", "gqa_bf16_b64"])
def test_small_bf16(shape, B, n, s):
    mw, kv, toks = _inputs(shape, B, n, s, seed=3)
    for tau, pat in ((0.05, 1), (0.5, 1), (0.0, 1)):
        _parity(mw, kv, toks, tau, pat, f"{shape.d_model}x{shape.n_layers} B={B} tau={tau}")


def test_zero_lm_head_gives_log_vocab():
    shape = GQA_BF16
    mw, kv, toks = _inputs(shape, 3, 20, 9, seed=5)
    mw.lm_head = torch.zeros_like(mw.lm_head)
    ent, ex, _ = _run_gpu(mw, kv, toks, 0.0, 1)
    np.testing.assert_allclose(ent, math.log(shape.vocab), rtol=0, atol=2e-5)
    assert (ex == shape.n_layers).all()
    ent, ex, _ = _run_gpu(mw, kv, toks, 1e-3, 2)    # every delta is 0 after layer 1
    assert (ex == 3).all()


def test_tau_extremes_and_nan_fill():
    shape = GQA_BF16
    mw, kv, toks = _inputs(shape, 4, 33, 17, seed=6)
    ent0, ex0, hid0 = _run_gpu(mw, kv, toks, 0.0, 1)
    assert (ex0 == shape.n_layers).all() and not np.isnan(ent0).any() and not np.isnan(hid0).any()
    for pat in (1, 2, 5):
        ent, ex, hid = _run_gpu(mw, kv, toks, math.inf, pat)
        e = min(1 + pat, shape.n_layers)
        assert (ex == e).all()
        np.testing.assert_array_equal(ent[:e], ent0[:e])      # same arithmetic up to the exit
        np.testing.assert_array_equal(hid[:e], hid0[:e])
        assert np.isnan(ent[e:]).all() and np.isnan(hid[e:]).all()


def test_deterministic_and_batch_position_invariant():
    shape = GQA_BF16
    mw, kv, toks = _inputs(shape, 5, 40, 24, seed=8)
    a = _run_gpu(mw, kv, toks, 0.02, 1)
    b = _run_gpu(mw, kv, toks, 0.02, 1)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    perm = torch.tensor([3, 0, 4, 2, 1], device=DEV)
    c = _run_gpu(mw, kv, toks[perm].contiguous(), 0.0, 1)
    ref = _run_gpu(mw, kv, toks, 0.0, 1)
    p = perm.cpu().numpy()
    np.testing.assert_allclose(c[0], ref[0][:, p], atol=1e-5)
    np.testing.assert_allclose(c[2], ref[2][:, p], rtol=1e-5, atol=1e-5)


def test_7b_single_full():
    """The 7B-shape single-branch verify (32 layers, 1024-token prefix, 128 tokens) in full."""
    wl = workloads.get("7b_single")
    mw, kv, toks = _inputs(wl.model, wl.n_branches, wl.prefix_len, wl.branch_len, seed=42)
    _parity(mw, kv, toks, wl.tau, wl.patience, "7b_single")


def test_7b_single_exit_inside_window():
    """The headline shape with its exit firing (Alg. VerifyWithEntropyExit): 32 layers, one branch
    x 128 tokens over the 1024-token prefix, exit windows of 8 layers (the cost model's choice at
    this shape). tau is read off the oracle's deltas so that the branch exits at a layer inside a
    window, with every delta at least 1.1e-2 nats from tau; the exit layer, the entropies and the
    hidden rows up to it match the oracle and the window's layers after it are NaN."""
    wl = workloads.get("7b_single")
    mw, kv, toks = _inputs(wl.model, 1, wl.prefix_len, wl.branch_len, seed=42)
    L, patience = wl.model.n_layers, wl.patience
    win = rk.rksc_verify_window(wl.model, 1, wl.branch_len, wl.prefix_len)
    assert win == 8
    ent_ref, hid_ref, _ = _run_oracle(mw, kv, toks, 0.0, 1)
    deltas = np.sort(np.abs(np.diff(ent_ref[:, 0])))
    tau = None
    for margin in (2.5e-2, 1.5e-2, 1.1e-2):
        for a, b in zip(deltas[:-1], deltas[1:]):
            t = (a + b) / 2
            e = oracle.exit_layer(ent_ref[:, 0], t, patience)
            if b - a > 2 * margin and e < L and e % win:
                tau = t
                break
        if tau is not None:
            break
    assert tau is not None, f"no separable tau in the oracle deltas {deltas}"
    ex_ref = np.array([oracle.exit_layer(ent_ref[:, 0], tau, patience)])
    log(f"[7b_single exit] tau={tau:.4f} oracle exit {ex_ref.tolist()}")
    ent, ex, hid = rk.verify_forward(mw, kv.k, kv.v, toks, tau, patience, return_hidden=True)
    torch.cuda.synchronize()
    ent, ex, hid = to_np(ent), to_np(ex), to_np(hid)
    stats = compare_verify(ent, ex, hid, ent_ref, hid_ref, ex_ref, tau, label=f"7b_single tau={tau:.4f}")
    log(f"[7b_single exit] gpu exit {ex.tolist()} {stats}")
    assert stats["near_threshold"] == 0 and stats["exit_match"] == 1 and ex[0] < L


@pytest.mark.parametrize("name,layers", [("7b_tot", 2), ("7b_large_vocab", 2), ("10b_long", 2), ("10b_decode", 2),
                                         ("7b_paper_verify", 2)])
def test_large_shapes_sampled_branches(name, layers):
    """Full model width, branch count, prefix and span; first layers only; oracle on two branches."""
    wl = workloads.get(name)
    mw, kv, toks = _inputs(wl.model, wl.n_branches, wl.prefix_len, wl.branch_len, seed=42, n_layers=layers)
    branches = [0, wl.n_branches - 1]
    _parity(mw, kv, toks, wl.tau, wl.patience, name, branches=branches)


@pytest.mark.parametrize("B,taus", [(1, (0.3, 0.6, 0.0)), (4, (0.3, 0.0)), (9, (0.3,)), (20, (0.3,)),
                                    (40, (0.3,))])
def test_exit_window_does_not_change_outputs(B, taus):
    """The exit window (layers sharing one lm_head stream) changes only the schedule: entropies,
    exit layers and hidden rows (NaN after each exit, also inside a window) match the oracle
    for every window, and windows of up to 32 columns reproduce the layer-by-layer outputs bit
    for bit (the same stream kernel; each column is computed on its own)."""
    shape = dataclasses.replace(workloads.get("tiny_deep").model, dtype="bf16")
    mw, kv, toks = _inputs(shape, B, 64, 5, 91)
    auto = rk.rksc_verify_window(shape, B, 5, 64)
    for tau in taus:
        ent_ref, hid_ref, ex_ref = _run_oracle(mw, kv, toks, tau, 1)
        base = None
        for win in (1, 2, 3, 4, 8):
            if win * B > 64:
                continue
            ent, ex, hid = rk.verify_forward(mw, kv.k, kv.v, toks, tau, 1, return_hidden=True, window=win)
            torch.cuda.synchronize()
            ent, ex, hid = to_np(ent), to_np(ex), to_np(hid)
            stats = compare_verify(ent, ex, hid, ent_ref, hid_ref, ex_ref, tau, label=f"B={B} tau={tau} win={win}")
            log(f"[window B={B} tau={tau} win={win}] exits {ex.tolist()} {stats}")
            if win == auto:   # the default call takes the cost model's window: the same outputs
                d_ent, d_ex, d_hid = rk.verify_forward(mw, kv.k, kv.v, toks, tau, 1, return_hidden=True)
                torch.cuda.synchronize()
                np.testing.assert_array_equal(to_np(d_ex), ex)
                np.testing.assert_array_equal(to_np(d_ent), ent)
                np.testing.assert_array_equal(to_np(d_hid), hid)
            if base is None:
                base = (ent, ex, hid)
            elif win * B <= 32:
                np.testing.assert_array_equal(ex, base[1])
                np.testing.assert_array_equal(ent, base[0])
                np.testing.assert_array_equal(hid, base[2])


def _pick_tau(ent_ref, patience, L, window):
    """_pick_tau_margin with the widest margin (from 2.5e-2 down to just above the 1e-2 bar) that
    admits a tau."""
    for margin in (2.5e-2, 1.5e-2, 1.1e-2):
        tau = _pick_tau_margin(ent_ref, patience, L, window, margin)
        if tau is not None:
            return tau
    return None


def _pick_tau_margin(ent_ref, patience, L, window, margin):
    """A tau read off the oracle's full-depth entropies [L, Bo] of the sampled branches such that
    (a) no sampled delta |H_l - H_{l-1}| lies within `margin` of it (so the exit layers must agree
    exactly), (b) some sampled branch exits before layer L and some exits later than another
    (different depths), preferring exits inside an exit window (layer % window != 0)."""
    Bo = ent_ref.shape[1]
    deltas = np.sort(np.unique(np.abs(np.diff(ent_ref, axis=0)).ravel()))
    cands = [(a + b) / 2 for a, b in zip(deltas[:-1], deltas[1:]) if b - a > 2 * margin]
    best, best_score = None, -1
    for tau in cands:
        ex = [oracle.exit_layer(ent_ref[:, j], tau, patience) for j in range(Bo)]
        if min(ex) >= L or len(set(ex)) < 2:
            continue
        # distinct depths first, then a sampled branch that survives every layer after the others
        # left (the survivors' rows are gathered), then exits inside a window
        score = len(set(ex)) * 10 + 15 * (max(ex) == L) + sum(1 for e in ex if e < L and e % window)
        if score > best_score:
            best, best_score = tau, score
    return best


def _exit_path_case(name, n_layers, patience, sampled, window_expect, window=None):
    """Full-size kernel plans with exits firing (Alg. VerifyWithEntropyExit; Sec. 2.3
    "Layer-level entropy exit"): the workload's width, branch count, prefix and span over
    n_layers layers; tau is read off the oracle's deltas of the sampled branches so that they
    exit at different layers (some inside an exit window) while every other branch exits
    wherever its own entropies take it, shrinking the live set under the wide GEMM tiles."""
    wl = workloads.get(name)
    mw, kv, toks = _inputs(wl.model, wl.n_branches, wl.prefix_len, wl.branch_len, seed=42, n_layers=n_layers)
    L = n_layers
    win = window or rk.rksc_verify_window(dataclasses.replace(wl.model, n_layers=L), wl.n_branches, wl.branch_len,
                                          wl.prefix_len)
    assert win == window_expect
    log(f"[{name} exit path] oracle on branches {sampled}")
    ent_ref, hid_ref, _ = _run_oracle(mw, kv, toks, 0.0, 1, branches=sampled)
    tau = _pick_tau(ent_ref, patience, L, win)
    assert tau is not None, f"no separable tau in the oracle deltas {np.abs(np.diff(ent_ref, axis=0)).T}"
    ex_ref = np.array([oracle.exit_layer(ent_ref[:, j], tau, patience) for j in range(len(sampled))])
    log(f"[{name} exit path] tau={tau:.4f} patience={patience} oracle exits {ex_ref.tolist()}")
    ent, ex, hid = rk.verify_forward(mw, kv.k, kv.v, toks, tau, patience, return_hidden=True, window=window)
    torch.cuda.synchronize()
    ent, ex, hid = to_np(ent), to_np(ex), to_np(hid)
    stats = compare_verify(ent, ex, hid, ent_ref, hid_ref, ex_ref, tau, branches=sampled,
                           label=f"{name} L={L} tau={tau:.4f} window={win}")
    log(f"[{name} exit path] gpu exits {ex.tolist()} {stats}")
    assert stats["near_threshold"] == 0 and stats["exit_match"] == len(sampled)
    assert (ex < L).sum() >= 1 and len(set(ex.tolist())) >= 2, "the live set must shrink during the call"
    # the same call at tau = 0 runs every layer: entropies and hidden rows at all depths
    ent0, ex0, hid0 = _run_gpu(mw, kv, toks, 0.0, 1)
    assert (ex0 == L).all()
    compare_verify(ent0, ex0, hid0, ent_ref, hid_ref, np.full(len(sampled), L), 0.0, branches=sampled,
                   label=f"{name} L={L} tau=0")


def test_exit_path_full_plans_paper_verify():
    """28 layers of the large-vocab shape, 8 x 128 rows over 1024 prefix tokens: 1024-row
    projections on the 256 x 256 tiles (with K splits), exit windows of 4 layers."""
    _exit_path_case("7b_paper_verify", 28, 2, [0, 3, 6], 4)


def test_exit_path_full_plans_10b_long():
    """6 layers of the 10B long-prefix shape, 32 x 256 rows over 16384 prefix tokens, patience 1:
    8192-row projections, exit windows of 2 layers at 32 live columns (the window the cost model
    takes for the full 48-layer pass; with 6 layers it would take 1, so it is set here)."""
    _exit_path_case("10b_long", 6, 1, [1, 17, 30], 2, window=2)


@pytest.mark.parametrize("shape,B,n,s,cuts", [
    (GQA_BF16, 3, 200, 40, (70, 130)),                 # per-branch (fused) tiles, cuts inside key tiles
    (GQA_BF16, 6, 300, 3, (64, 65, 250)),              # packed tiles (G * s < 64), a one-entry segment
    (G7_BF16, 2, 129, 65, (1,)),
    (workloads.get("tiny_deep").model, 4, 64, 16, (17, 40)),   # fp32 model: the plain kernel
])
def test_prefix_chain_equals_one_cache(shape, B, n, s, cuts):
    """A prefix given as a chain of caches (tree sharing: the ancestors' caches read in place)
    gives bit for bit the outputs of the same prefix as one cache, for the verify pass and for a
    batched decode step over it."""
    mw, kv, toks = _inputs(shape, B, n, s, seed=17)
    bounds = [0, *cuts, n]
    segs = [(kv.k[:, :, a:b].contiguous(), kv.v[:, :, a:b].contiguous()) for a, b in zip(bounds[:-1], bounds[1:])]
    chain = rk.PrefixCache(segs)
    assert chain.n_prefix == n
    for tau in (0.3, 0.0):
        one = rk.verify_forward(mw, kv.k, kv.v, toks, tau, 1, return_hidden=True)
        many = rk.verify_forward(mw, chain, None, toks, tau, 1, return_hidden=True)
        torch.cuda.synchronize()
        for a, b, what in zip(one, many, ("entropy", "exit", "hidden")):
            np.testing.assert_array_equal(to_np(a), to_np(b), err_msg=f"{what} differs (tau={tau})")
    # batched decode: suffix then two steps, over one cache and over the chain
    outs = []
    for pre_k, pre_v in ((kv.k, kv.v), (chain, None)):
        dec = rk.Decoder(mw, pre_k, pre_v, B, s, capacity=s + 2, device=DEV)
        got = [t.clone() for t in dec.suffix(toks)]
        for _ in range(2):
            got += [t.clone() for t in dec.step()]
        torch.cuda.synchronize()
        outs.append([to_np(t) for t in got])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("case", ["gqa_128rows", "gqa_1024rows", "7b_tot_2layers"])
def test_profiled_call_matches_plain_call(case):
    """The measurement variant of the verify call (a HIP event recorded on the stream before and
    after every kernel class at every layer; the gate|up pair closes between the projection and
    a separate SwiGLU combine where the plan has one) leaves the outputs bit-identical to
    rksc_verify_forward's: 128- and 1024-row plans with the separate combine, and 4096 rows of
    the 7B tree shape with the SwiGLU in the projection's epilogue. Every branch exits at layer
    2, so later layers run on no live rows; every recorded pair has a duration."""
    import ctypes
    if case == "7b_tot_2layers":
        wl = workloads.get("7b_tot")
        B, s, n = wl.n_branches, wl.branch_len, wl.prefix_len
        mw, kv, toks = _inputs(wl.model, B, n, s, seed=17, n_layers=2)
    else:
        B, s, n = (1 if case == "gqa_128rows" else 8), 128, 200
        mw, kv, toks = _inputs(GQA_BF16, B, n, s, seed=17)
    shape = mw.shape
    L, d = len(mw.layers), shape.d_model
    tau, patience = 10.0, 1   # every branch exits at layer 2
    ent0, ex0, hid0 = _run_gpu(mw, kv, toks, tau, patience)

    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    per = 12
    evs = []
    for _ in range(per * L):
        e = ctypes.c_void_p()
        assert hip.hipEventCreateWithFlags(ctypes.byref(e), 0x20000000) == 0   # no system fence on record
        evs.append(e.value)
    arr = (ctypes.c_void_p * (per * L))(*evs)
    lib = rk.load_library()
    lib.rksc_verify_forward_profiled.restype = ctypes.c_int32
    lib.rksc_verify_forward_profiled.argtypes = list(lib.rksc_verify_forward.argtypes) + [ctypes.c_void_p]
    ws = torch.empty(rk.rksc_verify_workspace_size(shape, B, s, n), dtype=torch.uint8, device=DEV)
    ent = torch.empty((L, B), dtype=torch.float32, device=DEV)
    ex = torch.empty((B,), dtype=torch.int32, device=DEV)
    hid = torch.empty((L, B, d), dtype=torch.float32, device=DEV)
    w_struct, keep = rk._weights_struct(mw)
    kv_struct = rk.PrefixKV(n, rk._ptr(kv.k), rk._ptr(kv.v))
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = lib.rksc_verify_forward_profiled(ctypes.byref(w_struct), ctypes.byref(kv_struct), rk._ptr(toks), B, s,
                                          tau, patience, rk._ptr(ent), rk._ptr(ex), rk._ptr(hid), rk._ptr(ws),
                                          ws.numel(), stream, ctypes.cast(arr, ctypes.c_void_p))
    assert st == 0, rk.rksc_last_error()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(ex), ex0)
    np.testing.assert_array_equal(to_np(ent), ent0)
    np.testing.assert_array_equal(to_np(hid), hid0)
    assert (ex0 == 2).all(), f"every branch should exit at layer 2 (got {ex0})"
    for l in range(L):
        for a in (0, 2, 4, 6, 8):   # QKV, attention, O, gate|up, down pairs are recorded at every layer
            ms = ctypes.c_float()
            assert hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(evs[per * l + a]),
                                           ctypes.c_void_p(evs[per * l + a + 1])) == 0
            assert ms.value >= 0.0
    for e in evs:
        hip.hipEventDestroy(ctypes.c_void_p(e))
    del keep
