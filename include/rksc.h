/*
 * rksc.h -- C ABI of the RKSC verify-pass library for MI355X (gfx950).
 *
 * RKSC (arXiv 2606.09937) verifies B reasoning branches that share one prefix.
 * This library implements the verify pass of its layer-level early exit
 * (Sec. 2.3 "Layer-level entropy exit", Alg. VerifyWithEntropyExit) over a
 * prefix KV cache that is computed once and read by every branch
 * (Sec. 2.2 "KV broadcast and batched decode"), the root forward that computes
 * that cache and the root hidden states (Eq. prefix_fwd), the batched decode
 * of the branches over it with the generation confidence (Eq. gen_conf) and
 * the CGEE verify-skip gate (Eq. cgee_gate), the layer-weighted cosine
 * similarity of the ASKS gate (Eq. asks_sim, Alg. AsksGate), and the host
 * runtime around them: the RSBCM block table (Alg. RsbcmEvict) and the KV
 * probe.
 *
 * Conventions shared by every entry point:
 *   - Tensor arguments are DEVICE pointers to dense row-major arrays.
 *   - The caller owns all memory. The library allocates no device memory and
 *     keeps no state between calls; the verify pass uses the caller's
 *     workspace.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL is the default
 *     stream). Outputs are valid once the stream is synchronised; inputs must
 *     stay alive until then. Concurrent calls on different streams must use
 *     different workspaces and outputs.
 *   - Arguments are validated before anything is launched. On a non-OK
 *     status nothing has been written and rksc_last_error() describes the
 *     cause. A failing HIP launch returns RKSC_ERR_HIP.
 *   - Results are deterministic: no floating-point atomics are used, so two
 *     calls with the same inputs produce bitwise-identical outputs.
 */
#ifndef RKSC_H_
#define RKSC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RKSC_ABI_VERSION 8

/* Largest number of branches one verify call accepts. */
#define RKSC_MAX_BRANCHES 64

typedef enum {
  RKSC_OK = 0,
  RKSC_ERR_INVALID_ARGUMENT = -1,   /* NULL pointer, bad size or bad value */
  RKSC_ERR_UNSUPPORTED = -2,        /* valid but outside what the kernels handle */
  RKSC_ERR_WORKSPACE_TOO_SMALL = -3,
  RKSC_ERR_HIP = -4                 /* a HIP runtime call or kernel launch failed */
} rksc_status;

/* Storage type of the weight matrices, the embedding, the lm_head and the
 * prefix K/V. RMSNorm gains are always fp32. */
typedef enum { RKSC_F32 = 0, RKSC_BF16 = 1 } rksc_dtype;

/* Decoder shape. Pre-norm Llama-style blocks: RMSNorm, grouped-query attention
 * with rotate-half RoPE, SwiGLU FFN, no biases, untied lm_head.
 * Requirements: head_dim in {64, 128}; n_heads % n_kv_heads == 0;
 * d_model, d_ff and n_heads*head_dim multiples of 8 (16-byte rows). */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t d_ff;
  int32_t vocab;
  float rms_eps;      /* RMSNorm: g * x / sqrt(mean(x^2) + rms_eps) */
  float rope_base;    /* RoPE: theta_j = rope_base^(-2j/head_dim) */
  int32_t dtype;      /* rksc_dtype */
} rksc_model_config;

/* One decoder layer; every pointer is a device pointer. */
typedef struct {
  const float* attn_norm;   /* [d] RMSNorm gain before attention */
  const void* w_qkv;        /* [(H + 2*Hkv)*hd, d]: the q rows, then k rows, then v rows */
  const void* w_o;          /* [d, H*hd] */
  const float* ffn_norm;    /* [d] RMSNorm gain before the FFN */
  const void* w_gate_up;    /* [2*F, d]: the gate rows, then the up rows */
  const void* w_down;       /* [d, F] */
  const void* w_gate_up_tiled;   /* optional (NULL: none): w_gate_up as laid out by
                                    rksc_tile_gate_up, read instead of it where the
                                    gate|up projection runs on the 128-row tiles (the
                                    smaller row counts); outputs are bitwise the same
                                    with or without it */
} rksc_layer_weights;

typedef struct {
  rksc_model_config cfg;
  const void* embed;                 /* [V, d] device */
  const rksc_layer_weights* layers;  /* HOST array of n_layers entries */
  const float* final_norm;           /* [d] device, RMSNorm gain before lm_head */
  const void* lm_head;               /* [V, d] device */
} rksc_weights;

/* The shared prefix cache C = {(K^(l), V^(l))} of Eq. prefix_fwd, computed once
 * for the prefix tokens and read (never copied) by every branch. A cache may
 * continue another one: a search-tree node's cache (rksc_prefix_extend) holds
 * only the node's own entries and names its parent, so that the node's
 * children read the chain root, ..., parent, node in place as one prefix
 * (Sec. 2.2, sharing of intermediate tree nodes). The prefix of a call is the
 * chain ending at the cache passed, in position order; n_prefix counts this
 * cache's entries only, and "the prefix length" below means the chain's total.
 * At most RKSC_MAX_PREFIX_SEGMENTS caches per chain (RKSC_ERR_UNSUPPORTED
 * otherwise; empty caches do not count). */
#define RKSC_MAX_PREFIX_SEGMENTS 8
typedef struct rksc_prefix_kv {
  int32_t n_prefix;   /* entries of this cache, >= 0 */
  const void* k;      /* [L, Hkv, n_prefix, hd], keys after RoPE at positions base..base+n_prefix-1 */
  const void* v;      /* [L, Hkv, n_prefix, hd] */
  const struct rksc_prefix_kv* parent;   /* NULL for a root cache (base = 0), else the cache whose
                                            entries come first (base = the prefix length up to it) */
} rksc_prefix_kv;

/* One branch set's own K/V cache for the decode loop (Sec. 2.2 "KV broadcast
 * and batched decode"): entry j of branch b holds the key (after RoPE) and the
 * value of the branch's token at position n + j (n: the prefix length). Allocated by the
 * caller for a fixed number of branches B; the decode calls append to it and
 * advance `length` (host field) on success. */
typedef struct {
  int32_t capacity;   /* entries allocated per (layer, branch, kv head) */
  int32_t length;     /* entries filled; 0 before rksc_decode_suffix */
  void* k;            /* [L, B, Hkv, capacity, hd] device, storage type */
  void* v;            /* [L, B, Hkv, capacity, hd] device, storage type */
} rksc_branch_kv;

int32_t rksc_abi_version(void);

/*
 * Pre-tiled copy of one layer's gate|up weight (a storage layout only; the
 * FFN's gate/up projection in the verify pass of Sec. 2.3 computes the same
 * products from it).
 *
 * out[((t * (d / 64) + kb) * 256 + r) * 64 + e] = w_gate_up[(256 t + r) * d + 64 kb + e]
 * for t < 2F / 256, kb < d / 64, r < 256, e < 64: every 256-row x 64-column
 * block of the weight becomes one contiguous run, which is how the 128-row
 * projection kernel streams it (a block per pipeline stage). Set the result as
 * the layer's w_gate_up_tiled. bf16 models with d % 64 == 0 and
 * (2 d_ff) % 256 == 0 only (RKSC_ERR_UNSUPPORTED otherwise, and for fp32).
 * w_gate_up and out: device, 2 F d elements of the model dtype each (out_bytes
 * at least rksc_gate_up_tiled_bytes(cfg)), not overlapping. Asynchronous on
 * `stream`; the copy must be complete before a call that reads it, on the same
 * stream or after a synchronisation. */
size_t rksc_gate_up_tiled_bytes(const rksc_model_config* cfg);
rksc_status rksc_tile_gate_up(const rksc_model_config* cfg, const void* w_gate_up, void* out, size_t out_bytes,
                              void* stream);

/* Bytes of workspace rksc_verify_forward needs for this shape (n_branches
 * branches of branch_len tokens over a prefix of n_prefix entries in all); 0 if the
 * shape is invalid (rksc_last_error() says why). */
size_t rksc_verify_workspace_size(const rksc_model_config* cfg, int32_t n_branches,
                                  int32_t branch_len, int32_t n_prefix);

/*
 * Verify pass with the layer-level entropy exit.
 *
 * Every branch b's tokens branch_tokens[b, 0..s-1] sit at positions n..n+s-1;
 * each attends to the whole shared prefix and, causally, to its own earlier
 * tokens (Sec. 2.2). After every layer l (1-based) the last token's hidden row
 * h goes through the final RMSNorm and the lm_head, and its softmax entropy in
 * nats H_l[b] is taken (Eq. entropy; the final norm is applied before the
 * projection so that layer L gives the model's real output distribution).
 * Exit rule (Sec. 2.3, condition (iii) with the entropy-stabilisation
 * tolerance tau and a patience): with H_0 = +inf, a layer counts toward the
 * streak when |H_l - H_{l-1}| < tau (strict) and resets it otherwise; branch b
 * exits at the first layer whose streak reaches `patience` and is not
 * computed beyond it. tau = 0 never exits (plain full-depth forward).
 *
 * branch_tokens  [B, s] int32 device, ids in [0, V) (not checked).
 * n_branches     B in [1, RKSC_MAX_BRANCHES]; branch_len s >= 1.
 * tau            >= 0 and not NaN (+inf allowed); patience >= 1.
 * entropy        [L, B] fp32 device out: H_l[b] in nats, NaN for l > exit_layer[b].
 * exit_layer     [B] int32 device out: 1-based exit layer, L if the rule never fired.
 * hidden_last    [L, B, d] fp32 device out or NULL: layer-l output row of the
 *                branch's last token (before the final norm), NaN rows after exit.
 * workspace      device buffer of at least rksc_verify_workspace_size() bytes,
 *                256-byte aligned; its contents on entry do not matter.
 *
 * Schedule: the probe's lm_head stream is shared by an exit window of
 * rksc_verify_window(cfg, B, s, n) consecutive layers (their rows are extra columns of
 * one read of W_lm). The rule still runs layer by layer, at the window's end;
 * a branch that exits inside a window has its later layers of that window
 * computed and discarded (NaN in the outputs), so every output equals that of
 * a layer-by-layer schedule.
 */
rksc_status rksc_verify_forward(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv,
                                const int32_t* branch_tokens, int32_t n_branches,
                                int32_t branch_len, float tau, int32_t patience,
                                float* entropy, int32_t* exit_layer, float* hidden_last,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * rksc_verify_forward without a workspace argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation). The pass runs on a device array of
 * RKSC_NOALLOC_SCRATCH_BYTES held by the library: each GPU the library runs on
 * gets its own copy, resolved on the first call on that GPU (with that GPU
 * current) and kept until the process ends. The call itself allocates
 * nothing. Arguments, outputs and results are those of rksc_verify_forward
 * (the same kernels); the caller still provides the inputs and outputs.
 *   - A pass whose workspace (rksc_verify_workspace_size) exceeds
 *     RKSC_NOALLOC_SCRATCH_BYTES is refused with RKSC_ERR_WORKSPACE_TOO_SMALL
 *     before anything is launched (use rksc_verify_forward for it).
 *   - `stream` must belong to the current device (RKSC_ERR_INVALID_ARGUMENT
 *     otherwise).
 *   - Every call on one GPU shares that GPU's array, and the pass overwrites
 *     it: calls that overlap on one GPU (other streams, other threads) race.
 *     Serialise them, e.g. on one stream. The array keeps the last call's
 *     contents; the pass initialises everything it reads.
 */
#define RKSC_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
rksc_status rksc_verify_forward_noalloc(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv,
                                        const int32_t* branch_tokens, int32_t n_branches, int32_t branch_len,
                                        float tau, int32_t patience, float* entropy, int32_t* exit_layer,
                                        float* hidden_last, void* stream);

/* The exit window rksc_verify_forward uses for this pass (B = n_branches
 * branches of s = branch_len tokens over an n_prefix-token cache): a power of
 * two in [1, min(8, 64 / B)] from a cost model of the schedule. Over L layers
 * the probe pays L / w streams of W_lm, and an exit, taken as uniformly placed
 * within its window, wastes (w - 1) / 2 computed layers on average; the window
 * nearest sqrt(2 L c_probe / c_layer) minimises the sum, with c_probe the
 * W_lm stream and c_layer a layer's projections, attention and row kernels,
 * both estimated from the shapes. Outputs do not depend on the window.
 * Returns 0 for an invalid shape (rksc_last_error() says why). */
int32_t rksc_verify_window(const rksc_model_config* cfg, int32_t n_branches, int32_t branch_len, int32_t n_prefix);

/* rksc_verify_forward with the exit window chosen by the caller: window = 1 is
 * the layer-by-layer schedule (a branch stops at its exit layer); window in
 * [1, 8] with window * n_branches <= 64. Outputs do not depend on it. */
rksc_status rksc_verify_forward_window(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv,
                                       const int32_t* branch_tokens, int32_t n_branches, int32_t branch_len,
                                       float tau, int32_t patience, float* entropy, int32_t* exit_layer,
                                       float* hidden_last, void* workspace, size_t workspace_bytes, void* stream,
                                       int32_t window);

/* Bytes of workspace rksc_prefill needs for an n_prefix-token prefix; 0 if the
 * shape is invalid (rksc_last_error() says why). */
size_t rksc_prefill_workspace_size(const rksc_model_config* cfg, int32_t n_prefix);

/*
 * Root forward over the shared prefix (Eq. prefix_fwd; the first step of
 * Alg. RKSC): one causal pass of the n prefix tokens at positions 0..n-1
 * through all L layers. It writes the prefix cache C = {(K^(l), V^(l))} that
 * rksc_verify_forward reads (pass k_out/v_out as rksc_prefix_kv.k/.v with
 * n_prefix = n), and the root hidden states H_root = {h_root^(l)}: the layer-l
 * output row of the last prefix token, normalised to unit length once here as
 * the paper stores them (Sec. 2.2; a zero row stays zero).
 *
 * tokens     [n] int32 device, ids in [0, V) (not checked; an id outside gives
 *            NaN rows); n_prefix = n >= 1.
 * k_out      [L, Hkv, n, hd] device out, the model's storage type (bf16 by
 *            round-to-nearest-even for RKSC_BF16): keys after RoPE.
 * v_out      [L, Hkv, n, hd] device out, same type: values.
 * h_root     [L, d] fp32 device out: unit-normalised root hidden states.
 * workspace  device buffer of at least rksc_prefill_workspace_size() bytes,
 *            256-byte aligned; its contents on entry do not matter.
 */
rksc_status rksc_prefill(const rksc_weights* weights, const int32_t* tokens, int32_t n_prefix, void* k_out,
                         void* v_out, float* h_root, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace that rksc_decode_suffix (suffix_len tokens per branch)
 * and rksc_decode_step (one token per branch) need for n_branches branches over
 * an n_prefix-token prefix cache; one buffer of this size serves both. 0 if the
 * shape is invalid (rksc_last_error() says why). */
size_t rksc_decode_workspace_size(const rksc_model_config* cfg, int32_t n_branches, int32_t suffix_len,
                                  int32_t n_prefix);

/*
 * Batched suffix prefill, the first step of the stepwise decode loop
 * (Sec. 2.2: every branch decodes over the shared cache C_B in one batched
 * call; implementation notes, "Stepwise Batched Decode" (1)). Branch b's
 * tokens suffix_tokens[b, 0..s-1] sit at positions n..n+s-1, attend to the
 * whole prefix and causally to each other, and their keys and values of every
 * layer are written to branch_kv entries 0..s-1 (storage type; bf16 by
 * round-to-nearest-even). From the last token's logits
 * z = lm_head . RMSNorm_final(h_L):
 *   next_token[b] = argmax_v z_v (smallest index among equal maxima),
 *   p_top[b]      = max_v softmax(z)_v, the step's term of Eq. gen_conf,
 *   conf[b]       = p_top[b]  (the running sum of Eq. gen_conf, t = 1).
 * A branch whose logits have no finite maximum gets next_token -1, p_top NaN.
 *
 * branch_kv      length must be 0 and capacity >= s; length becomes s.
 * suffix_tokens  [B, s] int32 device, ids in [0, V) (not checked).
 * n_branches     B in [1, RKSC_MAX_BRANCHES]; suffix_len s >= 1.
 * next_token     [B] int32 device out; p_top, conf [B] fp32 device out.
 * workspace      at least rksc_decode_workspace_size() bytes, 256-byte aligned.
 */
rksc_status rksc_decode_suffix(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv,
                               rksc_branch_kv* branch_kv, const int32_t* suffix_tokens, int32_t n_branches,
                               int32_t suffix_len, int32_t* next_token, float* p_top, float* conf, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * One token-by-token decode step (implementation notes, "Stepwise Batched
 * Decode" (2)): tokens[b] at position n + len (len = branch_kv->length) attends
 * to the prefix, to the branch's cached entries 0..len-1 and to itself; its key
 * and value are written to entry len. Outputs as rksc_decode_suffix, except
 * conf[b] += p_top[b] (the running sum of Eq. gen_conf over the steps).
 * tokens and next_token may be the same buffer (feeding the argmax back).
 *
 * branch_kv  capacity >= len + 1; length becomes len + 1.
 * tokens     [B] int32 device, ids in [0, V) (not checked).
 */
rksc_status rksc_decode_step(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv, rksc_branch_kv* branch_kv,
                             const int32_t* tokens, int32_t n_branches, int32_t* next_token, float* p_top,
                             float* conf, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace rksc_prefix_extend needs for n_new tokens on top of a
 * parent prefix of n_parent entries in all (0 if the shape is invalid). */
size_t rksc_prefix_extend_workspace_size(const rksc_model_config* cfg, int32_t n_parent, int32_t n_new);

/*
 * Tree sharing (Sec. 1: siblings share an intermediate node; the same
 * "compute once, broadcast" of Sec. 2.2 one level down): the cache of a
 * search-tree node whose m tokens follow its parent's prefix (the chain ending
 * at `parent`, n entries in all). The node's tokens are computed in one causal
 * pass at positions n..n+m-1 over that prefix, read in place, and k_out/v_out
 * receive only their m entries. Every child of the node then passes
 * {m, k_out, v_out, parent} as its rksc_prefix_kv in rksc_verify_forward /
 * rksc_decode_* (the chain of its ancestors' caches plus the node's: nothing
 * is copied). h_node receives the node's own "root" rows for the next level's
 * ASKS gate: the last new token's layer outputs, unit-normalised (as h_root of
 * rksc_prefill; with n = 0 this call is rksc_prefill).
 *
 * parent     the parent's prefix chain (n >= 0 entries in all, at most
 *            RKSC_MAX_PREFIX_SEGMENTS - 1 caches, so that the children's chain
 *            fits); no cache of it may overlap k_out / v_out.
 * tokens     [m] int32 device (m = n_new >= 1).
 * k_out      [L, Hkv, m, hd] device out, storage type; v_out likewise.
 * h_node     [L, d] fp32 device out, or NULL.
 * workspace  at least rksc_prefix_extend_workspace_size(cfg, n, m) bytes,
 *            256-byte aligned.
 */
rksc_status rksc_prefix_extend(const rksc_weights* weights, const rksc_prefix_kv* parent, const int32_t* tokens,
                               int32_t n_new, void* k_out, void* v_out, float* h_node, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * ASKS gate (Alg. AsksGate; Eq. asks_sim against the root): for each branch b
 *   sigma_b = sum_l w_l < h_b^(l) / |h_b^(l)| , h_root^(l) >,
 *   w_l = exp(alpha l / L) / sum_{l'} exp(alpha l' / L),
 * with h_root the unit rows of rksc_prefill (not normalised again), and
 * shared[b] = 1 iff sigma_b >= tau: the branch receives the shared cache;
 * below tau it falls back to its own recomputation (Sec. 2.2). A zero branch
 * row contributes 0. The decision is taken in fp32.
 *
 * hidden  [L, B, d] fp32 device: the branches' per-layer rows (e.g. the unit
 *         root rows of each branch's own rksc_prefill, or hidden_last of a
 *         verify pass); h_root [L, d] fp32 device.
 * sigma   [B] fp32 device out; shared [B] int32 device out.
 * L, B, d >= 1; L <= 256 and d % 4 == 0 (RKSC_ERR_UNSUPPORTED otherwise);
 * alpha finite; tau not NaN.
 */
rksc_status rksc_asks_gate(const float* hidden, const float* h_root, int32_t n_layers, int32_t n_branches,
                           int32_t d_model, float alpha, float tau, float* sigma, int32_t* shared, void* stream);

/*
 * CGEE gate (Eq. cgee_gate) over the generation confidences
 * p_b = conf[b] / n_steps (Eq. gen_conf, conf being the running sums of the
 * decode calls and n_steps = t the tokens generated): fires when
 *   max_b p_b >= tau_conf  and  (max_b p_b - 2nd-max_b p_b) / max_b p_b >= r_gap.
 * With (tau_conf, r_gap) = (0.70, 0.06) it is the Level-1 verify-skip gate
 * after decoding; with (0.72, 0.10) the decode-level early-termination gate
 * between steps (Sec. 2.3; implementation notes (3)). The 2nd max is the
 * largest p among the branches other than the winner (the smallest index
 * holding the maximum), 0 for a single branch; NaN entries are ignored. The
 * decision is taken in fp32.
 *
 * conf      [B] fp32 device; B in [1, RKSC_MAX_BRANCHES]; n_steps >= 1;
 *           tau_conf, r_gap not NaN.
 * p_mean    [B] fp32 device out or NULL: p_b.
 * fired     [1] int32 device out: 1 if the gate fires, else 0.
 * winner    [1] int32 device out: argmax_b p_b, -1 if every p_b is NaN.
 * stats     [3] fp32 device out or NULL: max, 2nd max, gap ratio.
 */
rksc_status rksc_cgee_gate(const float* conf, int32_t n_branches, int32_t n_steps, float tau_conf, float r_gap,
                           float* p_mean, int32_t* fired, int32_t* winner, float* stats, void* stream);

/*
 * ASKS similarity (Eq. asks_sim with the weights of Alg. AsksGate, generalised
 * from branch-vs-root to all branch pairs):
 *   w_l = exp(alpha*l/L) / sum_{l'=1..L} exp(alpha*l'/L),  l = 1..L
 *   S[i][j] = sum_l w_l * <h_i^(l), h_j^(l)> / (|h_i^(l)| |h_j^(l)|)
 * A zero row has cosine 0 with everything. To get the paper's sigma_b against
 * the root, append the root's rows (h_root of rksc_prefill) as one more
 * "branch".
 * hidden [L, B, d] fp32 device; S [B, B] fp32 device out.
 * L >= 1, B >= 1, d >= 1, alpha finite; L <= 256 (RKSC_ERR_UNSUPPORTED otherwise).
 */
rksc_status rksc_asks_similarity(const float* hidden, int32_t n_layers, int32_t n_branches,
                                 int32_t d_model, float alpha, float* S, void* stream);

/*
 * RSBCM block table (Sec. 2.4 "RSBCM"; Alg. RsbcmEvict): host-side
 * bookkeeping of cached KV blocks under tree search. Each block carries an
 * importance omega = score / (depth + 1), with score the owning branch's score
 * (e.g. its generation confidence) and depth its depth in the search tree.
 * rksc_block_table_evict runs the algorithm: while the table holds more than
 * `capacity` blocks, it removes the block of smallest omega (the earliest
 * inserted among equal omegas, omega evaluated in double). The ids are the
 * caller's (a KV block, a branch-cache slot); the caller releases the memory
 * of the evicted ids. A table is not thread-safe.
 */
typedef struct rksc_block_table rksc_block_table;

/* New empty table (capacity N_max >= 0; the paper's default is 2000); NULL on
 * a bad argument. Destroy with rksc_block_table_destroy. */
rksc_block_table* rksc_block_table_create(int32_t capacity);
void rksc_block_table_destroy(rksc_block_table* table);
/* Adds block_id (not yet in the table) with a finite score and depth >= 0. */
rksc_status rksc_block_table_insert(rksc_block_table* table, int64_t block_id, float score, int32_t depth);
/* Replaces the score of a block in the table (its omega changes with it). */
rksc_status rksc_block_table_set_score(rksc_block_table* table, int64_t block_id, float score);
/* Removes a block without counting an eviction (the caller freed it). */
rksc_status rksc_block_table_remove(rksc_block_table* table, int64_t block_id);
/* Alg. RsbcmEvict: evicts size - capacity blocks (if positive) in ascending
 * omega order, writing their ids to evicted[0 .. *n_evicted) (host array of
 * max_evicted entries; RKSC_ERR_INVALID_ARGUMENT, with nothing evicted, if it
 * is shorter than needed). */
rksc_status rksc_block_table_evict(rksc_block_table* table, int64_t* evicted, int32_t max_evicted,
                                   int32_t* n_evicted);
/* Blocks in the table; evictions so far (-1 for a NULL table). */
int32_t rksc_block_table_size(const rksc_block_table* table);
int64_t rksc_block_table_evicted_total(const rksc_block_table* table);

/*
 * KV probe (Sec. 2.2, paragraph "KV probe"): decides per 64-token
 * prefix-length bucket k = floor(n / 64) whether sharing the prefix cache pays
 * off. At the first decide call of a bucket it times, each as the minimum of
 * `reps` runs (the paper uses 3) with HIP events on `stream`:
 *   (i)   the batched full recompute: every branch's prefix and suffix as one
 *         sequence (rksc_decode_suffix over an empty prefix, B x (n + s) tokens);
 *   (ii)  one root forward over the prefix (rksc_prefill);
 *   (iii) the batched suffix decode over that shared cache (rksc_decode_suffix);
 * and stores share = 1 iff t(ii) + t(iii) < t(i). Later calls in the bucket
 * return the stored verdict and run nothing. A timing call blocks until the
 * stream has run the paths. A probe is not thread-safe.
 */
typedef struct rksc_kv_probe rksc_kv_probe;

rksc_kv_probe* rksc_kv_probe_create(int32_t reps);
void rksc_kv_probe_destroy(rksc_kv_probe* probe);
/* Device workspace the timing runs need (0 if the shape is invalid). */
size_t rksc_kv_probe_workspace_size(const rksc_model_config* cfg, int32_t n_prefix, int32_t n_branches,
                                    int32_t suffix_len);
/*
 * prefix_tokens  [n] int32 device; suffix_tokens [B, s] int32 device.
 * share          host out: 1 share the prefix cache, 0 recompute.
 * times_ms       host out [3] or NULL: t(i), t(ii), t(iii) of the bucket's probe.
 * probed         host out or NULL: 1 if this call ran the timing, 0 if the
 *                bucket's verdict was stored.
 */
rksc_status rksc_kv_probe_decide(rksc_kv_probe* probe, const rksc_weights* weights, const int32_t* prefix_tokens,
                                 int32_t n_prefix, const int32_t* suffix_tokens, int32_t n_branches,
                                 int32_t suffix_len, void* workspace, size_t workspace_bytes, void* stream,
                                 int32_t* share, float* times_ms, int32_t* probed);
/* The stored verdict of n_prefix's bucket: share = -1 if it was never probed. */
rksc_status rksc_kv_probe_lookup(const rksc_kv_probe* probe, int32_t n_prefix, int32_t* share, float* times_ms);

const char* rksc_status_string(rksc_status status);

/* Detail of the last non-OK status returned on this thread ("" if none). */
const char* rksc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RKSC_H_ */
