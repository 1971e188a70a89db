"""Pins of the float64 oracle against facts the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, a library routine (scipy, torch), values printed in the paper, or a brute
force recomputation. CPU only.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.spatial.distance
import scipy.special
import scipy.stats
import torch

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- entropy (Eq. entropy)

@pytest.mark.parametrize("V", [2, 7, 4096, 128256])
def test_entropy_uniform_is_log_v(V):
    for c in (0.0, -3.5, 17.0):
        H = oracle.softmax_entropy(np.full(V, c))
        assert abs(H - math.log(V)) < 1e-12 * max(1.0, math.log(V))


def test_entropy_one_hot_is_zero():
    z = np.zeros(4096)
    z[1234] = 1e4
    assert abs(oracle.softmax_entropy(z)) < 1e-12


@pytest.mark.parametrize("a", [-5.0, 0.5, 3.0, 12.0, 40.0])
@pytest.mark.parametrize("pos", [0, 511, 4095])
def test_entropy_two_level_closed_form(a, pos):
    # z = [0,..,a,..,0]: with E = e^a, H = log(E + V - 1) - a E / (E + V - 1)
    V = 4096
    z = np.zeros(V)
    z[pos] = a
    E = math.exp(a)
    ref = math.log(E + V - 1) - a * E / (E + V - 1)
    assert abs(oracle.softmax_entropy(z) - ref) < 1e-11


def test_entropy_matches_scipy_and_invariances():
    rng = np.random.default_rng(0)
    z = 4.0 * rng.standard_normal((5, 3000))
    H = oracle.softmax_entropy(z)
    ref = scipy.stats.entropy(scipy.special.softmax(z, axis=1), axis=1)
    np.testing.assert_allclose(H, ref, rtol=0, atol=1e-10)
    perm = rng.permutation(3000)
    np.testing.assert_allclose(oracle.softmax_entropy(z[:, perm] + 9.0), H, rtol=0, atol=1e-10)


# ----------------------------------------------------------------- exit rule (Sec. 2.3)

def test_exit_tau_zero_never_exits():
    H = np.linspace(5.0, 5.0, 12)          # constant: every delta is 0, still not < 0
    for p in (1, 2, 3):
        assert oracle.exit_layer(H, 0.0, p) == 12


def test_exit_tau_inf_exits_after_patience():
    H = np.random.default_rng(1).standard_normal(10)
    for p in (1, 2, 3, 9, 10, 20):
        assert oracle.exit_layer(H, math.inf, p) == min(1 + p, 10)


def test_exit_streak_resets_and_is_strict():
    # Binary fractions, so every delta below is exact.
    e = 2.0 ** -8
    #        l:  1    2              3    4        5            6            7
    H = np.array([5.0, 5.0 - 2 * e, 4.0, 4.0 - e, 4.0 - 2 * e, 4.0 - 3 * e, 3.0])
    # deltas: inf, 2e, 1-2e, e, e, e, 1-3e
    assert oracle.exit_layer(H, 0.02, 1) == 2
    assert oracle.exit_layer(H, 0.02, 2) == 5          # streak reset by l=3
    assert oracle.exit_layer(H, 0.02, 3) == 6
    assert oracle.exit_layer(H, 0.02, 4) == 7          # never: defaults to L
    assert oracle.exit_layer(H, e, 1) == 7             # |delta| == tau is not < tau
    assert oracle.exit_layer(H, 2 * e, 1) == 4
    assert oracle.exit_layer(np.array([1.0, 1.0]), 1e-9, 1) == 2   # H_0 = +inf


def _trajectory():
    with open(os.path.join(GOLDEN, "entropy_trajectory.json")) as f:
        return json.load(f)


def test_exit_paper_trajectory_delta_reading():
    """The printed delta column puts the first |dH| < 0.02 at layer 19, the paper's l*."""
    g = _trajectory()
    L = g["n_layers"]
    # Unprinted layers take the delta printed at the next printed layer (piecewise constant).
    deltas = np.empty(L)
    printed = dict(zip(g["layers"], g["delta"]))
    nxt = None
    for l in range(L, 0, -1):
        if l in printed and printed[l] is not None:
            nxt = printed[l]
        deltas[l - 1] = nxt if l > 1 else np.inf
    H = np.empty(L)
    H[0] = g["entropy"][0]
    for l in range(2, L + 1):
        H[l - 1] = H[l - 2] - deltas[l - 1]            # entropy decays monotonically
    assert oracle.exit_layer(H, 0.02, 1) == g["claimed_exit_layer"]
    assert oracle.exit_layer(H, 0.02, 2) == 20


def test_exit_paper_trajectory_entropy_reading():
    """Read from the printed entropy column (linear between printed layers) the exit is 21."""
    g = _trajectory()
    L = g["n_layers"]
    H = np.interp(np.arange(1, L + 1), g["layers"], g["entropy"])
    assert oracle.exit_layer(H, 0.02, 1) == 21
    assert oracle.exit_layer(H, 0.07, 1) == 19          # |1.08 - 1.14| = 0.06 < 0.07


# ----------------------------------------------------------------- ASKS (Eq. asks_sim)

def test_asks_weights_closed_form():
    for alpha, L in ((1.5, 28), (0.1, 32), (0.5, 2), (-2.0, 7)):
        w = oracle.asks_weights(alpha, L)
        r = math.exp(alpha / L)
        geo = np.array([r ** l * (r - 1) / (r * (r ** L - 1)) for l in range(1, L + 1)])
        np.testing.assert_allclose(w, geo, rtol=1e-12)
        assert abs(w.sum() - 1.0) < 1e-14
    np.testing.assert_allclose(oracle.asks_weights(0.0, 9), np.full(9, 1 / 9), rtol=1e-15)


def test_asks_single_layer_is_cosine():
    rng = np.random.default_rng(2)
    h = rng.standard_normal((1, 5, 64))
    S = oracle.asks_similarity(h, 0.7)
    for i in range(5):
        for j in range(5):
            assert abs(S[i, j] - (1 - scipy.spatial.distance.cosine(h[0, i], h[0, j]))) < 1e-12


def test_asks_identical_orthogonal_antipodal_zero():
    rng = np.random.default_rng(3)
    L, d = 6, 32
    h = np.zeros((L, 5, d))
    base = rng.standard_normal((L, d))
    h[:, 0] = base
    h[:, 1] = 3.0 * base                     # same direction, other norm
    h[:, 2] = -base                          # antipodal
    for l in range(L):                       # orthogonal to base in every layer
        v = rng.standard_normal(d)
        h[l, 3] = v - (v @ base[l]) / (base[l] @ base[l]) * base[l]
    # h[:, 4] stays zero
    S = oracle.asks_similarity(h, 1.5)
    assert abs(S[0, 1] - 1.0) < 1e-12 and abs(S[0, 0] - 1.0) < 1e-12
    assert abs(S[0, 2] + 1.0) < 1e-12
    assert abs(S[0, 3]) < 1e-12
    assert S[4, 4] == 0.0 and np.all(S[4] == 0.0)


def test_asks_alpha_zero_is_mean_cosine_and_psd():
    rng = np.random.default_rng(4)
    h = rng.standard_normal((4, 6, 48))
    S = oracle.asks_similarity(h, 0.0)
    ref = np.zeros((6, 6))
    for l in range(4):
        ref += 1 - scipy.spatial.distance.cdist(h[l], h[l], "cosine")
    np.testing.assert_allclose(S, ref / 4, atol=1e-12)
    S2 = oracle.asks_similarity(h, 2.0)
    np.testing.assert_allclose(S2, S2.T, atol=0)
    assert np.linalg.eigvalsh(S2).min() > -1e-12
    assert np.all(np.abs(S2) <= 1 + 1e-12)


# ----------------------------------------------------------------- layer pieces

def test_rmsnorm_matches_torch_and_is_scale_invariant():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((7, 96))
    g = rng.standard_normal(96)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.rmsnorm(37.0 * x, g, 0.0), oracle.rmsnorm(x, g, 0.0), rtol=1e-12)


def test_rope_is_complex_rotation_and_relative():
    rng = np.random.default_rng(6)
    hd, base = 64, 1e4
    x = rng.standard_normal((5, 3, hd))
    pos = np.array([0, 1, 17, 1000, 16639])
    out = oracle.apply_rope(x, pos, base)
    # Rotate-half RoPE = multiply (x_j + i x_{j+hd/2}) by exp(i p theta_j).
    theta = base ** (-np.arange(0, hd, 2) / hd)
    zc = (x[..., : hd // 2] + 1j * x[..., hd // 2:]) * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    np.testing.assert_allclose(out[..., : hd // 2], zc.real, atol=1e-10)
    np.testing.assert_allclose(out[..., hd // 2:], zc.imag, atol=1e-10)
    np.testing.assert_allclose(out[0], x[0], atol=0)                       # position 0: identity
    # q(p).k(p') depends only on p - p'
    q = rng.standard_normal((1, 1, hd))
    k = rng.standard_normal((1, 1, hd))
    d1 = (oracle.apply_rope(q, [40], base) * oracle.apply_rope(k, [13], base)).sum()
    d2 = (oracle.apply_rope(q, [1027], base) * oracle.apply_rope(k, [1000], base)).sum()
    assert abs(d1 - d2) < 1e-9


def test_attention_single_key_returns_value():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((1, 4, 16))
    k = rng.standard_normal((2, 1, 16))
    v = rng.standard_normal((2, 1, 16))
    o = oracle.attention(q, k, v, n_prefix=0)
    for h in range(4):
        np.testing.assert_allclose(o[0, h], v[h // 2, 0], atol=1e-15)


def test_attention_matches_torch_sdpa_with_prefix_and_gqa():
    rng = np.random.default_rng(8)
    T, n, H, Hkv, hd = 9, 13, 6, 2, 16
    q = rng.standard_normal((T, H, hd))
    k = rng.standard_normal((Hkv, n + T, hd))
    v = rng.standard_normal((Hkv, n + T, hd))
    o = oracle.attention(q, k, v, n_prefix=n)
    mask = np.ones((T, n + T), dtype=bool)
    mask[:, n:] = np.tril(np.ones((T, T), dtype=bool))
    G = H // Hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]                       # [1, H, T, hd]
    kt = torch.from_numpy(np.repeat(k, G, axis=0))[None]
    vt = torch.from_numpy(np.repeat(v, G, axis=0))[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=torch.from_numpy(mask))
    np.testing.assert_allclose(o, ref[0].permute(1, 0, 2).numpy(), atol=1e-12)


# ----------------------------------------------------------------- whole decoder vs HF Llama

GQA_SHAPE = workloads.ModelShape(n_layers=3, d_model=128, n_heads=8, n_kv_heads=2, head_dim=32,
                                 d_ff=200, vocab=512, dtype="f32", lm_head_scale=8.0)


def _randomise_gains(mw, seed=11):
    g = torch.Generator().manual_seed(seed)
    for lw in mw.layers:
        lw["attn_norm"] = 1.0 + 0.3 * torch.randn(lw["attn_norm"].shape, generator=g)
        lw["ffn_norm"] = 1.0 + 0.3 * torch.randn(lw["ffn_norm"].shape, generator=g)
    mw.final_norm = 1.0 + 0.3 * torch.randn(mw.final_norm.shape, generator=g)
    return mw


def _close(a, b, tol=1e-6):
    """Norm-relative agreement; HF evaluates RoPE's cos/sin in fp32, so exact match is not expected."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    err = np.linalg.norm(a - b) / np.linalg.norm(b)
    assert err < tol, f"relative error {err:.3e}"


def _hf_model(mw, shape):
    transformers = pytest.importorskip("transformers")
    cfg = transformers.LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.d_ff,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
        rope_theta=shape.rope_base, tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
        max_position_embeddings=4096)
    cfg._attn_implementation = "eager"
    m = transformers.LlamaForCausalLM(cfg).double().eval()
    H, Hkv, hd, F = shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.d_ff
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(mw.embed.double())
        for l, lw in enumerate(mw.layers):
            layer = m.model.layers[l]
            wqkv = lw["w_qkv"].double()
            layer.self_attn.q_proj.weight.copy_(wqkv[: H * hd])
            layer.self_attn.k_proj.weight.copy_(wqkv[H * hd: (H + Hkv) * hd])
            layer.self_attn.v_proj.weight.copy_(wqkv[(H + Hkv) * hd:])
            layer.self_attn.o_proj.weight.copy_(lw["w_o"].double())
            layer.mlp.gate_proj.weight.copy_(lw["w_gate_up"][:F].double())
            layer.mlp.up_proj.weight.copy_(lw["w_gate_up"][F:].double())
            layer.mlp.down_proj.weight.copy_(lw["w_down"].double())
            layer.input_layernorm.weight.copy_(lw["attn_norm"].double())
            layer.post_attention_layernorm.weight.copy_(lw["ffn_norm"].double())
        m.model.norm.weight.copy_(mw.final_norm.double())
        m.lm_head.weight.copy_(mw.lm_head.double())
        # HF derives the inverse frequencies in fp32; use the exact float64 values.
        inv = torch.pow(torch.tensor(shape.rope_base, dtype=torch.float64),
                        -torch.arange(0, hd, 2, dtype=torch.float64) / hd)
        m.model.rotary_emb.inv_freq = inv
        if hasattr(m.model.rotary_emb, "original_inv_freq"):
            m.model.rotary_emb.original_inv_freq = inv
    return m


@pytest.mark.parametrize("shape", [GQA_SHAPE, workloads.get("tiny").model], ids=["gqa", "tiny"])
def test_forward_full_matches_hf_llama(shape):
    mw = _randomise_gains(workloads.make_model(shape, seed=3))
    T = 24
    toks = workloads.make_tokens(T, shape.vocab, seed=3).numpy()
    hid = oracle.forward_full(mw, shape, toks)
    m = _hf_model(mw, shape)
    with torch.no_grad():
        out = m(torch.from_numpy(toks.astype(np.int64))[None], output_hidden_states=True)
    L = shape.n_layers
    for l in range(L - 1):
        _close(hid[l], out.hidden_states[l + 1][0].numpy())
    # HF reports the last layer after the final norm.
    last = oracle.rmsnorm(hid[L - 1], mw.final_norm, shape.rms_eps)
    _close(last, out.hidden_states[L][0].numpy())
    z = last @ oracle.f64(mw.lm_head).T
    _close(z, out.logits[0].numpy())


def test_prefix_cache_verify_matches_hf_dynamic_cache():
    """Prefill + shared-cache branch forward vs HF's own KV-cache path (the paper's stack)."""
    transformers = pytest.importorskip("transformers")
    import copy
    shape = GQA_SHAPE
    mw = _randomise_gains(workloads.make_model(shape, seed=4))
    n, s, B = 20, 7, 3
    prefix = workloads.make_tokens(n, shape.vocab, seed=4, name="prefix").numpy()
    branches = workloads.make_tokens(B * s, shape.vocab, seed=4).numpy().reshape(B, s)
    pk, pv, h_root = oracle.prefill(mw, shape, prefix)
    ent, ex, hid, ent_full, h_last = oracle.verify_forward(mw, shape, pk, pv, branches, 0.0, 1)
    m = _hf_model(mw, shape)
    with torch.no_grad():
        pre = m(torch.from_numpy(prefix.astype(np.int64))[None], use_cache=True, output_hidden_states=True)
        cache = pre.past_key_values
        for l in range(shape.n_layers):
            layer_cache = cache.layers[l] if hasattr(cache, "layers") else None
            kk = layer_cache.keys if layer_cache is not None else cache.key_cache[l]
            vv = layer_cache.values if layer_cache is not None else cache.value_cache[l]
            _close(pk[l], kk[0].numpy())
            _close(pv[l], vv[0].numpy())
        for b in range(B):
            out = m(torch.from_numpy(branches[b].astype(np.int64))[None],
                    past_key_values=copy.deepcopy(cache), use_cache=True, output_hidden_states=True)
            for l in range(shape.n_layers - 1):
                _close(h_last[l, b], out.hidden_states[l + 1][0, -1].numpy())
            H_hf = oracle.softmax_entropy(out.logits[0, -1].numpy())
            assert abs(H_hf - ent_full[-1, b]) < 1e-6


# ----------------------------------------------------------------- whole-pass invariants

def _tiny_inputs(name, seed=42):
    wl = workloads.get(name)
    shape = wl.model
    mw = workloads.make_model(shape, seed=seed)
    prefix = workloads.make_tokens(wl.prefix_len, shape.vocab, seed=seed, name="prefix").numpy()
    toks = workloads.make_tokens(wl.n_branches * wl.branch_len, shape.vocab, seed=seed).numpy()
    return wl, mw, prefix, toks.reshape(wl.n_branches, wl.branch_len)


@pytest.mark.parametrize("name", ["tiny", "tiny_deep"])
def test_shared_prefix_equals_recomputation(name):
    """Shared-prefix verify equals a per-branch full forward of [prefix; branch] (brute force)."""
    wl, mw, prefix, toks = _tiny_inputs(name)
    shape = wl.model
    pk, pv, _ = oracle.prefill(mw, shape, prefix)
    _, _, _, ent_full, h_last = oracle.verify_forward(mw, shape, pk, pv, toks, wl.tau, wl.patience)
    for b in range(wl.n_branches):
        full = oracle.forward_full(mw, shape, np.concatenate([prefix, toks[b]]))
        np.testing.assert_allclose(h_last[:, b], full[:, -1], rtol=1e-10, atol=1e-12)
    ref_ent = oracle.layer_entropies(mw, shape, np.stack(
        [oracle.forward_full(mw, shape, np.concatenate([prefix, toks[b]]))[:, -1] for b in range(wl.n_branches)], 1))
    np.testing.assert_allclose(ent_full, ref_ent, atol=1e-10)


def test_tau_zero_is_full_depth_forward():
    wl, mw, prefix, toks = _tiny_inputs("tiny_deep")
    shape = wl.model
    pk, pv, _ = oracle.prefill(mw, shape, prefix)
    ent, ex, hid, ent_full, h_last = oracle.verify_forward(mw, shape, pk, pv, toks, 0.0, 1)
    assert np.all(ex == shape.n_layers)
    assert not np.isnan(ent).any() and not np.isnan(hid).any()
    np.testing.assert_array_equal(ent, ent_full)
    np.testing.assert_array_equal(hid, h_last)
    # With a finite tau, the outputs agree up to each exit and are NaN after it.
    ent2, ex2, hid2, _, _ = oracle.verify_forward(mw, shape, pk, pv, toks, 10.0, 1)
    assert np.all(ex2 == 2)
    np.testing.assert_array_equal(ent2[:2], ent[:2])
    assert np.isnan(ent2[2:]).all() and np.isnan(hid2[2:]).all()


def test_branches_are_independent():
    wl, mw, prefix, toks = _tiny_inputs("tiny")
    shape = wl.model
    pk, pv, _ = oracle.prefill(mw, shape, prefix)
    _, _, _, e1, h1 = oracle.verify_forward(mw, shape, pk, pv, toks, 0.0, 1)
    perm = np.array([2, 0, 3, 1])
    _, _, _, e2, h2 = oracle.verify_forward(mw, shape, pk, pv, toks[perm], 0.0, 1)
    np.testing.assert_allclose(e2, e1[:, perm], atol=1e-12)
    np.testing.assert_allclose(h2, h1[:, perm], atol=1e-12)
    # identical branches -> ASKS similarity 1 between them
    same = np.stack([toks[0], toks[1], toks[0]])
    _, _, _, _, h3 = oracle.verify_forward(mw, shape, pk, pv, same, 0.0, 1)
    S = oracle.asks_similarity(h3, wl.alpha)
    assert abs(S[0, 2] - 1.0) < 1e-12 and S[0, 1] < 0.999


def test_zero_lm_head_gives_log_vocab_every_layer():
    wl, mw, prefix, toks = _tiny_inputs("tiny_deep")
    shape = wl.model
    mw.lm_head = torch.zeros_like(mw.lm_head)
    pk, pv, _ = oracle.prefill(mw, shape, prefix)
    ent, ex, _, _, _ = oracle.verify_forward(mw, shape, pk, pv, toks, 0.0, 1)
    np.testing.assert_allclose(ent, math.log(shape.vocab), rtol=0, atol=1e-12)
    # Every delta is 0 after layer 1, so any tau > 0 exits at 1 + patience.
    _, ex, _, _, _ = oracle.verify_forward(mw, shape, pk, pv, toks, 1e-9, 2)
    assert np.all(ex == 3)


# ----------------------------------------------------------------- root rows (Eq. prefix_fwd, Alg. AsksGate)

def test_unit_rows_norm_direction_and_zero():
    rng = np.random.default_rng(11)
    h = rng.standard_normal((5, 3, 40)) * rng.uniform(0.01, 100.0, (5, 3, 1))
    h[2, 1] = 0.0
    u = oracle.unit_rows(h)
    nrm = np.linalg.norm(u, axis=-1)
    nz = np.linalg.norm(h, axis=-1) > 0
    np.testing.assert_allclose(nrm[nz], 1.0, rtol=1e-14)
    assert np.all(u[2, 1] == 0.0)
    # same direction: h = |h| u
    np.testing.assert_allclose(h, np.linalg.norm(h, axis=-1, keepdims=True) * u, rtol=1e-12, atol=1e-14)


def test_root_similarity_equals_appended_root_row():
    """sigma_b against pre-normalised root rows equals the pairwise S with the root as one more branch."""
    rng = np.random.default_rng(12)
    L, B, d = 7, 4, 24
    hb = rng.standard_normal((L, B, d))
    root = rng.standard_normal((L, d)) * 5.0
    hb[:, 1] = 2.5 * root                        # a branch on the root's direction: sigma = 1
    hb[:, 2] = -root                             # antipodal: sigma = -1
    sig = oracle.root_similarity(hb, oracle.unit_rows(root), 1.5)
    S = oracle.asks_similarity(np.concatenate([hb, root[:, None, :]], axis=1), 1.5)
    np.testing.assert_allclose(sig, S[:B, B], atol=1e-13)
    assert abs(sig[1] - 1.0) < 1e-13 and abs(sig[2] + 1.0) < 1e-13
    # L = 1: plain cosine
    s1 = oracle.root_similarity(hb[:1], oracle.unit_rows(root[:1]), 0.3)
    for b in range(B):
        assert abs(s1[b] - (1 - scipy.spatial.distance.cosine(hb[0, b], root[0]))) < 1e-12


# ----------------------------------------------------------------- decode, Eq. gen_conf, Eq. cgee_gate

def _gate_examples():
    with open(os.path.join(GOLDEN, "cgee_gate_examples.json")) as f:
        return json.load(f)


def _confidences(top, second, B, seed):
    """B confidences whose maximum is `top` and whose second maximum is `second` (the rest below)."""
    rng = np.random.default_rng(seed)
    p = np.concatenate([[top, second], rng.uniform(0.0, second, B - 2)])
    return p[rng.permutation(B)]


def test_cgee_gate_paper_examples():
    g = _gate_examples()
    for ex in g["examples"]:
        for seed in range(5):
            p = _confidences(ex["max"], ex["second"], g["n_branches"], seed)
            r = oracle.cgee_gate(p, g["tau_conf"], g["r_gap"])
            assert r["fired"] == ex["fires"], ex["name"]
            assert r["max"] == ex["max"] and r["second"] == ex["second"]
            assert round(r["gap"], 2) == ex["printed_gap_ratio"]
            assert p[r["winner"]] == ex["max"]
    # The deferred example fails on the absolute threshold, not on the gap.
    d = g["examples"][1]
    r = oracle.cgee_gate(_confidences(d["max"], d["second"], 8, 0), d["max"], g["r_gap"])
    assert r["fired"] and r["gap"] >= g["r_gap"]
    # Under the stricter decode-level thresholds the first example still fires.
    e = g["examples"][0]
    assert oracle.cgee_gate(_confidences(e["max"], e["second"], 8, 1), g["theta_dec"], g["r_dec"])["fired"]


def test_cgee_gate_two_failure_modes():
    """Sec. 2.3: (a) a confident branch with a close competitor and (b) a large relative gap
    between two unconfident branches must both defer; each condition alone would fire."""
    a = np.array([0.80, 0.79, 0.3])
    r = oracle.cgee_gate(a, 0.70, 0.06)
    assert not r["fired"] and r["max"] >= 0.70 and oracle.cgee_gate(a, 0.70, 0.0)["fired"]
    b = np.array([0.10, 0.40, 0.05])
    r = oracle.cgee_gate(b, 0.70, 0.06)
    assert not r["fired"] and r["gap"] >= 0.06 and r["winner"] == 1
    assert oracle.cgee_gate(b, 0.40, 0.06)["fired"]


def test_cgee_gate_brute_force_sorted():
    rng = np.random.default_rng(5)
    for _ in range(300):
        B = int(rng.integers(2, 65))
        p = rng.uniform(0, 1, B)
        if rng.uniform() < 0.3:
            p[rng.integers(0, B)] = p.max()   # a tie at the maximum
        srt = np.sort(p)
        tau, rg = rng.uniform(0.3, 0.9), rng.uniform(0.0, 0.3)
        gap = (srt[-1] - srt[-2]) / srt[-1]
        r = oracle.cgee_gate(p, tau, rg)
        assert r["max"] == srt[-1] and r["second"] == srt[-2]
        assert abs(r["gap"] - gap) < 1e-15
        assert r["fired"] == (srt[-1] >= tau and gap >= rg)
        assert r["winner"] == int(np.flatnonzero(p == srt[-1])[0])


def test_cgee_gate_single_branch_nan_and_zero():
    r = oracle.cgee_gate([0.75], 0.70, 0.06)
    assert r["fired"] and r["second"] == 0.0 and r["gap"] == 1.0
    assert not oracle.cgee_gate([0.65], 0.70, 0.06)["fired"]
    r = oracle.cgee_gate([np.nan, 0.9, np.nan, 0.5], 0.70, 0.06)
    assert r["winner"] == 1 and r["second"] == 0.5
    r = oracle.cgee_gate([np.nan, np.nan], 0.0, 0.0)
    assert not r["fired"] and r["winner"] == -1
    r = oracle.cgee_gate([0.0, 0.0], 0.0, 0.0)
    assert r["gap"] == 0.0 and r["winner"] == 0 and r["fired"]


def test_gen_confidence_is_the_step_mean():
    rng = np.random.default_rng(6)
    pt = rng.uniform(0.1, 1.0, (9, 5))
    for t in (1, 4, 9):
        np.testing.assert_allclose(oracle.gen_confidence(pt[:t]), [sum(pt[j, b] for j in range(t)) / t
                                                                   for b in range(5)], rtol=1e-15)
    np.testing.assert_allclose(oracle.gen_confidence(np.full((7, 3), 0.35)), 0.35, rtol=1e-15)


@pytest.mark.parametrize("a", [-3.0, 0.0, 2.5, 30.0])
def test_top1_two_level_closed_form(a):
    V = 1000
    z = np.zeros((2, V))
    z[0, 17] = a
    z[1, 999] = a
    tok, p = oracle.top1(z)
    ref = math.exp(a) / (math.exp(a) + V - 1)
    if a > 0:
        assert list(tok) == [17, 999]
        np.testing.assert_allclose(p, ref, rtol=1e-13)
    elif a == 0:
        assert list(tok) == [0, 0]          # first of the tied maxima
        np.testing.assert_allclose(p, 1.0 / V, rtol=1e-13)
    else:
        assert list(tok) == [0, 0]
        np.testing.assert_allclose(p, 1.0 / (V - 1 + math.exp(a)), rtol=1e-13)


def test_decode_equals_full_causal_forward():
    """Prefill + suffix + stepwise decode with the branch caches equals one causal forward of
    the concatenated sequence, for every branch: logits of each step and its cached K/V."""
    shape = GQA_SHAPE
    mw = _randomise_gains(workloads.make_model(shape, seed=8))
    n, s, B, steps = 10, 4, 3, 3
    prefix = workloads.make_tokens(n, shape.vocab, seed=8, name="prefix").numpy()
    suffix = workloads.make_tokens(B * s, shape.vocab, seed=8).numpy().reshape(B, s)
    gen = workloads.make_tokens(B * steps, shape.vocab, seed=8, name="decode").numpy().reshape(steps, B)
    pk, pv, _ = oracle.prefill(mw, shape, prefix)
    ck, cv, z = oracle.decode_suffix(mw, shape, pk, pv, suffix)
    zs = [z]
    for j in range(steps):
        k1, v1, z = oracle.decode_step(mw, shape, pk, pv, ck, cv, gen[j])
        ck, cv = np.concatenate([ck, k1], axis=3), np.concatenate([cv, v1], axis=3)
        zs.append(z)
    lm = oracle.f64(mw.lm_head)
    for b in range(B):
        seq = np.concatenate([prefix, suffix[b], gen[:, b]])
        hid, ks, vs = oracle.decoder_stack(mw, shape, seq[None, :], 0)
        zf = oracle.rmsnorm(hid[-1, 0], mw.final_norm, shape.rms_eps) @ lm.T
        for j in range(steps + 1):
            np.testing.assert_allclose(zs[j][b], zf[n + s - 1 + j], rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(ck[:, b], ks[:, 0, :, n:], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(cv[:, b], vs[:, 0, :, n:], rtol=1e-10, atol=1e-12)


def test_decode_matches_hf_kv_cache_generation():
    """Suffix prefill and teacher-forced decode steps vs HF's own KV-cache path."""
    pytest.importorskip("transformers")
    import copy
    shape = GQA_SHAPE
    mw = _randomise_gains(workloads.make_model(shape, seed=9))
    n, s, B, steps = 12, 5, 2, 3
    prefix = workloads.make_tokens(n, shape.vocab, seed=9, name="prefix").numpy()
    suffix = workloads.make_tokens(B * s, shape.vocab, seed=9).numpy().reshape(B, s)
    gen = workloads.make_tokens(B * steps, shape.vocab, seed=9, name="decode").numpy().reshape(steps, B)
    pk, pv, _ = oracle.prefill(mw, shape, prefix)
    ck, cv, z = oracle.decode_suffix(mw, shape, pk, pv, suffix)
    zs, tops = [z], [oracle.top1(z)[1]]
    for j in range(steps):
        k1, v1, z = oracle.decode_step(mw, shape, pk, pv, ck, cv, gen[j])
        ck, cv = np.concatenate([ck, k1], axis=3), np.concatenate([cv, v1], axis=3)
        zs.append(z)
        tops.append(oracle.top1(z)[1])
    m = _hf_model(mw, shape)
    with torch.no_grad():
        pre = m(torch.from_numpy(prefix.astype(np.int64))[None], use_cache=True)
        for b in range(B):
            out = m(torch.from_numpy(suffix[b].astype(np.int64))[None],
                    past_key_values=copy.deepcopy(pre.past_key_values), use_cache=True)
            hf_z = [out.logits[0, -1].numpy()]
            cache = out.past_key_values
            for j in range(steps):
                out = m(torch.tensor([[int(gen[j, b])]]), past_key_values=cache, use_cache=True)
                cache = out.past_key_values
                hf_z.append(out.logits[0, -1].numpy())
            for j in range(steps + 1):
                _close(zs[j][b], hf_z[j])
                p_hf = torch.softmax(torch.from_numpy(hf_z[j]), -1).max().item()
                assert abs(p_hf - tops[j][b]) < 1e-6
    conf = oracle.gen_confidence(np.stack(tops))
    assert conf.shape == (B,) and np.all((conf > 0) & (conf <= 1))


# ----------------------------------------------------------------- RSBCM (Alg. RsbcmEvict), KV probe

def test_rsbcm_stress_test_eviction_count():
    """App. RSBCM validation: capacity 4, B = 8 branch blocks per solve, 20 solves: exactly
    B - N_max = 4 evictions per solve and 80 in total, whatever the scores."""
    rng = np.random.default_rng(12)
    total = 0
    for problem in range(20):
        blocks = [(b, float(rng.uniform(0, 1)), int(rng.integers(0, 3))) for b in range(8)]
        kept, ev = oracle.rsbcm_evict(blocks, 4)
        assert len(ev) == 4 and len(kept) == 4
        total += len(ev)
        # the evicted blocks are the four of least omega
        om = sorted(oracle.rsbcm_omega(s, d) for _, s, d in blocks)
        assert max(oracle.rsbcm_omega(s, d) for i, s, d in blocks if i in ev) <= om[4]
    assert total == 20 * (8 - 4) == 80


def test_rsbcm_order_depth_ties_and_capacity():
    # omega = score / (depth + 1): a deep high-score block goes before a shallow low-score one
    blocks = [(10, 0.9, 8), (11, 0.2, 0), (12, 0.5, 1), (13, 0.5, 1), (14, 0.05, 0)]
    kept, ev = oracle.rsbcm_evict(blocks, 2)
    # omegas: 0.1, 0.2, 0.25, 0.25, 0.05 -> 14, 10, 11 ; ties (12, 13) keep both
    assert ev == [14, 10, 11] and [b[0] for b in kept] == [12, 13]
    _, ev = oracle.rsbcm_evict(blocks, 3)
    assert ev == [14, 10]
    _, ev = oracle.rsbcm_evict(blocks, 4)
    assert ev == [14]
    # equal omegas go in insertion order
    _, ev = oracle.rsbcm_evict([(1, 0.5, 1), (2, 0.25, 0), (3, 1.0, 3), (4, 0.25, 0)], 1)
    assert ev == [1, 2, 3]
    assert oracle.rsbcm_evict(blocks, 0)[1] == [14, 10, 11, 12, 13]
    assert oracle.rsbcm_evict(blocks, 5)[1] == [] and oracle.rsbcm_evict([], 0) == ([], [])


def test_rsbcm_matches_one_at_a_time_eviction():
    """Brute force of the algorithm's loop: while over capacity, recompute every omega and evict the
    first least one. Its sequence equals the oracle's (omega, insertion) order."""
    def one_at_a_time(blocks, cap):
        table, ev = list(blocks), []
        while len(table) > cap:
            om = [s / (d + 1.0) for _, s, d in table]
            j = min(range(len(table)), key=lambda i: (om[i], i))
            ev.append(table.pop(j)[0])
        return table, ev

    rng = np.random.default_rng(13)
    for _ in range(200):
        n = int(rng.integers(0, 40))
        blocks = [(i, float(np.float32(rng.choice([0.25, 0.5, rng.uniform(-1, 2)]))), int(rng.integers(0, 5)))
                  for i in range(n)]
        cap = int(rng.integers(0, 45))
        kept, ev = oracle.rsbcm_evict(blocks, cap)
        kept_bf, ev_bf = one_at_a_time(blocks, cap)
        assert ev == ev_bf
        assert kept == kept_bf


def test_kv_probe_paper_cost_table():
    with open(os.path.join(GOLDEN, "kv_probe_cost_constants.json")) as f:
        g = json.load(f)
    for row in g["rows"]:
        net = row["batch_full"] - row["prefix_fwd"] - row["sfx_kv"]
        assert abs(net - row["net_saved"]) <= 0.1 + 1e-9, row["model"]
        assert oracle.kv_probe_share(row["batch_full"], row["prefix_fwd"], row["sfx_kv"])
        # sharing stops paying once root forward + suffix decode cost what the recompute costs
        assert not oracle.kv_probe_share(row["batch_full"], row["batch_full"] - row["sfx_kv"], row["sfx_kv"])
    assert [oracle.kv_probe_bucket(n) for n in (0, 63, 64, 1023, 1024, 1087, 1088)] == [0, 0, 1, 15, 16, 16, 17]


# ----------------------------------------------------------------- tree sharing, ASKS gate (Alg. AsksGate)

def test_prefix_extend_equals_prefill_of_the_concatenation():
    """A node's cache built on its parent's equals one causal prefill of [root; node] (and two levels
    [root; a; b]); h_node is the last token's rows of that prefill."""
    shape = GQA_SHAPE
    mw = _randomise_gains(workloads.make_model(shape, seed=14))
    root = workloads.make_tokens(11, shape.vocab, seed=14, name="prefix").numpy()
    a = workloads.make_tokens(6, shape.vocab, seed=14, name="node_a").numpy()
    b = workloads.make_tokens(4, shape.vocab, seed=14, name="node_b").numpy()
    pk, pv, _ = oracle.prefill(mw, shape, root)
    ka, va, ha = oracle.prefix_extend(mw, shape, pk, pv, a)
    rk_, rv_, rh_ = oracle.prefill(mw, shape, np.concatenate([root, a]))
    np.testing.assert_allclose(ka, rk_, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(va, rv_, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(ha, rh_, rtol=1e-10, atol=1e-12)
    kb, vb, hb = oracle.prefix_extend(mw, shape, ka, va, b)
    rk2, rv2, rh2 = oracle.prefill(mw, shape, np.concatenate([root, a, b]))
    np.testing.assert_allclose(kb, rk2, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(hb, rh2, rtol=1e-10, atol=1e-12)
    # an empty parent is a plain prefill
    k0, v0, h0 = oracle.prefix_extend(mw, shape, None, None, root)
    np.testing.assert_allclose(k0, pk, rtol=1e-12, atol=1e-14)


def test_asks_gate_threshold_and_identity():
    rng = np.random.default_rng(15)
    L, d = 6, 48
    root = oracle.unit_rows(rng.standard_normal((L, d)))
    same = np.stack([root * 3.0, -root, rng.standard_normal((L, d)), np.zeros((L, d))], axis=1)   # [L, 4, d]
    sigma, shared = oracle.asks_gate(same, root, 1.5, 0.82)
    assert abs(sigma[0] - 1.0) < 1e-12 and abs(sigma[1] + 1.0) < 1e-12 and sigma[3] == 0.0
    assert list(shared) == [True, False, bool(sigma[2] >= 0.82), False]
    # the threshold is inclusive (Alg. AsksGate shares at sigma_b >= tau)
    assert oracle.asks_gate(same, root, 1.5, float(sigma[2]))[1][2]
    # tau = -1 shares everything with a finite sigma, tau above 1 nothing
    assert oracle.asks_gate(same, root, 1.5, -1.0)[1].all()
    assert not oracle.asks_gate(same, root, 1.5, 1.0 + 1e-9)[1].any()
