"""Plain float64 CPU oracle for the RKSC verify pass and the ASKS similarity.

TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this module. The HIP product path never
calls it, and this module imports nothing from the product package.

Everything is computed from the definitions, in float64, with numpy's matmul as
the only library primitive. Weights and KV arrive in their storage precision
(fp32, or bf16 already widened exactly to fp32) and are widened to float64 on
use. No blocking, fusion or reordering beyond what each definition states.

Model (RKSC paper, Sec. 2.1 "Problem Setting"; the decoder itself is the standard
pre-norm Llama-style block the paper runs through HF Transformers, Appendix
"Implementation Details"):
  x_0 = E[token]
  per layer: u = RMSNorm(x; g_attn); q,k,v = u W_q^T, u W_k^T, u W_v^T;
             rotate-half RoPE on q,k at the token's absolute position;
             grouped-query attention (query head h reads KV head floor(h/G)),
             scale 1/sqrt(hd); x += o W_o^T;
             w = RMSNorm(x; g_ffn); x += (silu(w W_g^T) * (w W_u^T)) W_d^T.
Verify pass (Sec. 2.2 "KV broadcast and batched decode", Eq. prefix_fwd):
  every branch's tokens sit at positions n..n+s-1 and attend to the one shared
  prefix cache plus their own earlier tokens.
Layer entropy (Eq. entropy, Alg. VerifyWithEntropyExit): last token of the
  branch, final RMSNorm, lm_head, softmax entropy in nats.
Exit rule (Sec. 2.3 "Layer-level entropy exit"), as (tau, patience): the layer
  delta is |H_l - H_{l-1}| with H_0 = +inf; a streak counts consecutive layers
  with delta < tau (strict); the branch exits at the first layer whose streak
  reaches patience, else at L.
ASKS (Eq. asks_sim with its exponential layer weights): S_ij = sum_l w_l *
  cos(h_i^(l), h_j^(l)), w_l = exp(alpha l/L) / sum_l' exp(alpha l'/L).
Batched decode (Sec. 2.2; the stepwise loop of the implementation notes): a
  suffix prefill of every branch over the shared prefix, then one token per
  branch per step attending to the prefix, the branch's own earlier tokens and
  itself; each step's top-1 probability max_v softmax(z)_v feeds the generation
  confidence p_b (Eq. gen_conf), and Eq. cgee_gate decides on the p_b.
RSBCM (Sec. 2.4, Alg. RsbcmEvict): while the block table holds more than
  N_max blocks, evict the block of least omega = score / (depth + 1).
Tree sharing: a search-tree node's tokens are run once over its parent's cache
  and the resulting cache serves all of its children.
ASKS gate (Alg. AsksGate): a branch receives the shared cache iff sigma_b >= tau.
KV probe (Sec. 2.2, paragraph "KV probe"): per 64-token prefix bucket, share
  the prefix cache iff t(root forward) + t(suffix decode) < t(full recompute).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "f64", "rmsnorm", "rope_inv_freq", "apply_rope", "silu", "attention",
    "decoder_stack", "prefill", "forward_full", "softmax_entropy",
    "layer_entropies", "exit_layer", "verify_forward", "asks_weights",
    "asks_similarity", "unit_rows", "root_similarity",
    "final_logits", "top1", "decode_suffix", "decode_step", "gen_confidence", "cgee_gate",
    "rsbcm_omega", "rsbcm_evict", "kv_probe_bucket", "kv_probe_share", "prefix_extend", "asks_gate",
]


def f64(a) -> np.ndarray:
    """Widen a numpy array or a torch tensor (any float dtype; bf16 is exact via fp32) to float64."""
    if hasattr(a, "detach"):           # torch tensor: bf16 widens exactly through fp32
        a = a.detach().cpu()
        if not a.dtype.is_floating_point or a.element_size() < 4:
            a = a.float()
        a = a.numpy()
    return np.asarray(a, dtype=np.float64)


def rmsnorm(x, gamma, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: gamma * x / sqrt(mean(x^2) + eps)."""
    x = f64(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return f64(gamma) * x / np.sqrt(ms + eps)


def rope_inv_freq(head_dim: int, base: float) -> np.ndarray:
    """theta_j = base^(-2j/hd), j = 0..hd/2-1."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * j / head_dim)


def apply_rope(x, positions, base: float) -> np.ndarray:
    """Rotate-half RoPE. x: [T, nh, hd]; positions: [T] absolute positions.

    For j < hd/2 the pair (x_j, x_{j+hd/2}) is rotated by the angle p*theta_j.
    """
    x = f64(x)
    hd = x.shape[-1]
    half = hd // 2
    ang = np.asarray(positions, dtype=np.float64)[:, None] * rope_inv_freq(hd, base)[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z) -> np.ndarray:
    """silu(z) = z / (1 + exp(-z))."""
    z = f64(z)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def attention(q, k_keys, v_keys, n_prefix: int) -> np.ndarray:
    """Grouped-query attention of one sequence over [shared prefix ; own tokens].

    q:      [T, H, hd]        queries of the sequence's T tokens (post-RoPE)
    k_keys: [Hkv, n+T, hd]    keys: n_prefix shared prefix keys, then the T own keys
    v_keys: [Hkv, n+T, hd]
    Query token i may read every prefix key and own keys 0..i (causal).
    Returns o: [T, H, hd].
    """
    q = f64(q)
    k_keys = f64(k_keys)
    v_keys = f64(v_keys)
    T, H, hd = q.shape
    Hkv = k_keys.shape[0]
    G = H // Hkv
    n_keys = k_keys.shape[1]
    key_pos = np.arange(n_keys)
    allowed = (key_pos[None, :] < n_prefix) | ((key_pos[None, :] - n_prefix) <= np.arange(T)[:, None])
    o = np.empty((T, H, hd), dtype=np.float64)
    for h in range(H):
        g = h // G
        scores = q[:, h, :] @ k_keys[g].T / np.sqrt(hd)          # [T, n_keys]
        scores = np.where(allowed, scores, -np.inf)
        m = scores.max(axis=1, keepdims=True)
        p = np.exp(scores - m)
        p /= p.sum(axis=1, keepdims=True)
        o[:, h, :] = p @ v_keys[g]
    return o


def decoder_stack(weights, cfg, tokens, start_pos: int = 0, prefix_k=None, prefix_v=None):
    """Run all L decoder layers on a batch of independent token sequences.

    weights: object with .embed [V,d], .layers (sequence of mappings with
             attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down), .final_norm, .lm_head
    cfg:     object with n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff,
             rms_eps, rope_base
    tokens:  int [B, T]; token t of every sequence sits at position start_pos + t
    prefix_k, prefix_v: [L, Hkv, n, hd] shared post-RoPE prefix cache (or None)

    Returns (hidden [L, B, T, d], k [L, B, Hkv, T, hd], v [L, B, Hkv, T, hd]):
    hidden[l] is the output of layer l+1 (before any final norm); k is post-RoPE.
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    B, T = tokens.shape
    L, d = cfg.n_layers, cfg.d_model
    H, Hkv, hd, F = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    n = 0 if prefix_k is None else int(prefix_k.shape[2])
    positions = start_pos + np.arange(T)
    embed = weights.embed
    x = np.stack([f64(embed[tokens[b].tolist()]) for b in range(B)])   # [B, T, d]
    hidden = np.empty((L, B, T, d), dtype=np.float64)
    ks = np.empty((L, B, Hkv, T, hd), dtype=np.float64)
    vs = np.empty((L, B, Hkv, T, hd), dtype=np.float64)
    for l in range(L):
        W = weights.layers[l]
        u = rmsnorm(x, W["attn_norm"], cfg.rms_eps)
        qkv = u.reshape(B * T, d) @ f64(W["w_qkv"]).T
        q = qkv[:, : H * hd].reshape(B, T, H, hd)
        k = qkv[:, H * hd: (H + Hkv) * hd].reshape(B, T, Hkv, hd)
        v = qkv[:, (H + Hkv) * hd:].reshape(B, T, Hkv, hd)
        o = np.empty((B, T, H, hd), dtype=np.float64)
        for b in range(B):
            qb = apply_rope(q[b], positions, cfg.rope_base)
            kb = apply_rope(k[b], positions, cfg.rope_base).transpose(1, 0, 2)   # [Hkv, T, hd]
            vb = v[b].transpose(1, 0, 2)
            ks[l, b] = kb
            vs[l, b] = vb
            if n:
                k_keys = np.concatenate([f64(prefix_k[l]), kb], axis=1)
                v_keys = np.concatenate([f64(prefix_v[l]), vb], axis=1)
            else:
                k_keys, v_keys = kb, vb
            o[b] = attention(qb, k_keys, v_keys, n)
        x = x + (o.reshape(B * T, H * hd) @ f64(W["w_o"]).T).reshape(B, T, d)
        w = rmsnorm(x, W["ffn_norm"], cfg.rms_eps)
        gu = w.reshape(B * T, d) @ f64(W["w_gate_up"]).T
        a = silu(gu[:, :F]) * gu[:, F:]
        x = x + (a @ f64(W["w_down"]).T).reshape(B, T, d)
        hidden[l] = x
    return hidden, ks, vs


def prefill(weights, cfg, prefix_tokens):
    """Root forward over the prefix (Eq. prefix_fwd): causal, positions 0..n-1.

    Returns (k [L, Hkv, n, hd], v [L, Hkv, n, hd], h_root [L, d]); h_root is the
    last prefix token's per-layer output.
    """
    hidden, ks, vs = decoder_stack(weights, cfg, np.asarray(prefix_tokens)[None, :], 0)
    return ks[:, 0], vs[:, 0], hidden[:, 0, -1, :]


def unit_rows(h) -> np.ndarray:
    """Rows scaled to unit Euclidean length; a zero row stays zero.

    The root hidden states of Eq. prefix_fwd are stored in this normalised form
    (Sec. 2.2, paragraph "Prefix forward pass").
    """
    h = f64(h)
    nrm = np.sqrt((h * h).sum(axis=-1, keepdims=True))
    return np.where(nrm > 0, h / np.where(nrm > 0, nrm, 1.0), 0.0)


def root_similarity(hidden, h_root_unit, alpha: float) -> np.ndarray:
    """sigma_b of Eq. asks_sim: sum_l w_l <h_b^(l) / |h_b^(l)|, h_root^(l)> for hidden [L, B, d]
    and pre-normalised root rows h_root_unit [L, d] (Alg. AsksGate); a zero branch row contributes 0."""
    hb = unit_rows(hidden)
    w = asks_weights(alpha, hb.shape[0])
    return np.einsum("l,lbd,ld->b", w, hb, f64(h_root_unit))


def forward_full(weights, cfg, tokens):
    """Plain causal forward of one sequence from position 0: hidden [L, T, d]."""
    hidden, _, _ = decoder_stack(weights, cfg, np.asarray(tokens)[None, :], 0)
    return hidden[:, 0]


def softmax_entropy(z) -> np.ndarray:
    """H = -sum_v p_v log p_v, p = softmax(z) over the last axis, in nats (Eq. entropy)."""
    z = f64(z)
    m = z.max(axis=-1, keepdims=True)
    lse = m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True))
    logp = z - lse
    p = np.exp(logp)
    return -(p * logp).sum(axis=-1)


def layer_entropies(weights, cfg, h_last) -> np.ndarray:
    """Per-layer entropy of last-token rows h_last [L, B, d]: final RMSNorm, lm_head, entropy."""
    h_last = f64(h_last)
    L, B, _ = h_last.shape
    lm = f64(weights.lm_head)
    out = np.empty((L, B), dtype=np.float64)
    for l in range(L):
        z = rmsnorm(h_last[l], weights.final_norm, cfg.rms_eps) @ lm.T     # [B, V]
        out[l] = softmax_entropy(z)
    return out


def exit_layer(entropies, tau: float, patience: int) -> int:
    """1-based exit layer of one branch from its full-depth entropy sequence H_1..H_L."""
    L = len(entropies)
    prev = np.inf
    streak = 0
    for l in range(1, L + 1):
        h = float(entropies[l - 1])
        delta = abs(h - prev)
        streak = streak + 1 if delta < tau else 0
        if streak >= patience:
            return l
        prev = h
    return L


def verify_forward(weights, cfg, prefix_k, prefix_v, branch_tokens, tau: float, patience: int):
    """RKSC verify pass with the layer-level entropy exit.

    Branches never attend to each other, so the exit of each branch is a pure
    function of its full-depth entropy sequence: run full depth, then apply the
    rule. Returns (entropy [L,B] with NaN after exit, exit_layer [B] int32,
    hidden_last [L,B,d] with NaN rows after exit, entropy_full [L,B],
    hidden_full [L,B,d]).
    """
    tokens = np.asarray(branch_tokens, dtype=np.int64)
    B, s = tokens.shape
    n = int(prefix_k.shape[2])
    hidden, _, _ = decoder_stack(weights, cfg, tokens, n, prefix_k, prefix_v)
    h_last = hidden[:, :, s - 1, :]                                        # [L, B, d]
    ent = layer_entropies(weights, cfg, h_last)
    exits = np.array([exit_layer(ent[:, b], tau, patience) for b in range(B)], dtype=np.int32)
    L = cfg.n_layers
    after = np.arange(1, L + 1)[:, None] > exits[None, :]                 # [L, B]
    ent_out = np.where(after, np.nan, ent)
    hid_out = np.where(after[:, :, None], np.nan, h_last)
    return ent_out, exits, hid_out, ent, h_last


def asks_weights(alpha: float, L: int) -> np.ndarray:
    """w_l = exp(alpha*l/L) / sum_{l'=1..L} exp(alpha*l'/L), l = 1..L."""
    e = np.exp(float(alpha) * np.arange(1, L + 1, dtype=np.float64) / L)
    return e / e.sum()


def asks_similarity(hidden, alpha: float) -> np.ndarray:
    """S[i,j] = sum_l w_l cos(h_i^(l), h_j^(l)) for hidden [L, B, d]; a zero row has cosine 0."""
    h = f64(hidden)
    L, B, _ = h.shape
    w = asks_weights(alpha, L)
    S = np.zeros((B, B), dtype=np.float64)
    for l in range(L):
        norms = np.sqrt((h[l] * h[l]).sum(axis=1))
        hat = np.zeros_like(h[l])
        nz = norms > 0
        hat[nz] = h[l][nz] / norms[nz, None]
        S += w[l] * (hat @ hat.T)
    return S


def final_logits(weights, cfg, h) -> np.ndarray:
    """z = RMSNorm(h; g_final) W_lm^T for rows h [..., d]: the model's output logits."""
    return rmsnorm(f64(h), weights.final_norm, cfg.rms_eps) @ f64(weights.lm_head).T


def top1(z):
    """(argmax_v z_v, max_v softmax(z)_v) per row of z [..., V]: the next token and
    the term max_v Pr[y_j = v] of Eq. gen_conf. np.argmax takes the first maximum."""
    z = f64(z)
    m = z.max(axis=-1, keepdims=True)
    p = np.exp(z - m)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.argmax(z, axis=-1).astype(np.int64), p.max(axis=-1)


def decode_suffix(weights, cfg, prefix_k, prefix_v, suffix_tokens):
    """Suffix prefill of B branches over the shared prefix (Sec. 2.2): branch b's
    tokens at positions n..n+s-1. Returns (k [L, B, Hkv, s, hd] post-RoPE,
    v [L, B, Hkv, s, hd], z [B, V] logits of each branch's last token)."""
    tokens = np.asarray(suffix_tokens, dtype=np.int64)
    n = 0 if prefix_k is None else int(prefix_k.shape[2])
    hidden, ks, vs = decoder_stack(weights, cfg, tokens, n, prefix_k, prefix_v)
    return ks, vs, final_logits(weights, cfg, hidden[-1, :, -1, :])


def decode_step(weights, cfg, prefix_k, prefix_v, past_k, past_v, tokens):
    """One decode step: token tokens[b] of branch b at position n + len attends to
    the prefix, to the branch's past entries past_k/past_v [L, B, Hkv, len, hd]
    (post-RoPE keys and values of its tokens at n..n+len-1) and to itself.
    Returns (k [L, B, Hkv, 1, hd], v [L, B, Hkv, 1, hd], z [B, V])."""
    tokens = np.asarray(tokens, dtype=np.int64).reshape(-1)
    B = tokens.shape[0]
    n = 0 if prefix_k is None else int(prefix_k.shape[2])
    length = int(past_k.shape[3])
    L, Hkv, hd = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    ks = np.empty((L, B, Hkv, 1, hd))
    vs = np.empty((L, B, Hkv, 1, hd))
    z = np.empty((B, weights.lm_head.shape[0]))
    for b in range(B):
        if n:
            pk = np.concatenate([f64(prefix_k), f64(past_k[:, b])], axis=2)
            pv = np.concatenate([f64(prefix_v), f64(past_v[:, b])], axis=2)
        else:
            pk, pv = f64(past_k[:, b]), f64(past_v[:, b])
        if pk.shape[2] == 0:
            pk = pv = None
        hidden, kb, vb = decoder_stack(weights, cfg, tokens[b:b + 1, None], n + length, pk, pv)
        ks[:, b], vs[:, b] = kb[:, 0], vb[:, 0]
        z[b] = final_logits(weights, cfg, hidden[-1, 0, -1, :])
    return ks, vs, z


def gen_confidence(p_top) -> np.ndarray:
    """Eq. gen_conf: p_b = (1/t) sum_{j=1..t} max_v Pr[y_j^(b) = v] for p_top [t, B]."""
    p_top = f64(p_top)
    return p_top.sum(axis=0) / p_top.shape[0]


def cgee_gate(p, tau_conf: float, r_gap: float) -> dict:
    """Eq. cgee_gate on the generation confidences p [B]: fires iff
    max_b p >= tau_conf and (max_b p - 2nd-max_b p) / max_b p >= r_gap.

    Readings: the winner is the first index holding the maximum; the 2nd max is
    the largest p among the other branches, 0 when there is none; a zero
    maximum gives a gap ratio of 0. NaN entries are left out.
    """
    p = f64(p).reshape(-1)
    idx = [b for b in range(p.shape[0]) if not np.isnan(p[b])]
    if not idx:
        return {"fired": False, "winner": -1, "max": float("nan"), "second": 0.0, "gap": 0.0}
    winner = idx[0]
    for b in idx:
        if p[b] > p[winner]:
            winner = b
    others = [p[b] for b in idx if b != winner]
    top = float(p[winner])
    second = float(max(others)) if others else 0.0
    gap = (top - second) / top if top > 0 else 0.0
    return {"fired": bool(top >= tau_conf and gap >= r_gap), "winner": winner, "max": top, "second": second,
            "gap": gap}


def rsbcm_omega(score, depth) -> float:
    """Importance of a cached block (Sec. 2.4): omega = score / (depth + 1), in double."""
    return float(np.float32(score)) / (float(depth) + 1.0)


def rsbcm_evict(blocks, n_max: int):
    """Alg. RsbcmEvict on a block table given as a list of (id, score, depth) in
    insertion order, keeping at most n_max blocks. A block's omega depends only on
    its own score and depth, so evicting one never changes another's: the evicted
    blocks are the len - n_max smallest by (omega, insertion index), in that order
    (the algorithm takes the first of equal minima). Returns (remaining table in
    insertion order, evicted ids in eviction order)."""
    table = list(blocks)
    n_evict = max(0, len(table) - int(n_max))
    order = sorted(range(len(table)), key=lambda i: (rsbcm_omega(table[i][1], table[i][2]), i))
    gone = set(order[:n_evict])
    return [b for i, b in enumerate(table) if i not in gone], [table[i][0] for i in order[:n_evict]]


def kv_probe_bucket(n_prefix: int) -> int:
    """The probe's prefix-length bucket k = floor(n / 64) (Sec. 2.2, "KV probe")."""
    return int(n_prefix) // 64


def kv_probe_share(t_full: float, t_prefix: float, t_suffix: float) -> bool:
    """Sharing is beneficial iff t(ii) + t(iii) < t(i): root forward plus batched
    suffix decode against batched full recompute (Sec. 2.2, "KV probe")."""
    return t_prefix + t_suffix < t_full


def prefix_extend(weights, cfg, parent_k, parent_v, tokens):
    """A tree node's cache: its m tokens at positions n..n+m-1 attend to the
    parent's n cached entries and causally to each other. Returns (k [L, Hkv, n+m,
    hd], v, h_node [L, d]): the parent's entries followed by the node's, and the
    last node token's layer outputs (not normalised)."""
    tokens = np.asarray(tokens, dtype=np.int64).reshape(1, -1)
    n = 0 if parent_k is None else int(parent_k.shape[2])
    hidden, ks, vs = decoder_stack(weights, cfg, tokens, n, parent_k if n else None, parent_v if n else None)
    if n:
        k = np.concatenate([f64(parent_k), ks[:, 0]], axis=2)
        v = np.concatenate([f64(parent_v), vs[:, 0]], axis=2)
    else:
        k, v = ks[:, 0], vs[:, 0]
    return k, v, hidden[:, 0, -1, :]


def asks_gate(hidden, h_root_unit, alpha: float, tau: float):
    """Alg. AsksGate: sigma_b of Eq. asks_sim against the unit root rows and the
    shared set {b : sigma_b >= tau}, for branch rows hidden [L, B, d]."""
    sigma = root_similarity(hidden, h_root_unit, alpha)
    return sigma, sigma >= tau
