/*
 * rksc_testing.h -- kernel-level entry points of librksc for unit tests.
 *
 * These expose single kernels of the verify pass so that tests can compare
 * them one by one with a CPU reference. They follow the conventions of
 * rksc.h (device pointers, asynchronous on `stream`, validation before any
 * launch, rksc_last_error() on failure). They are not needed to run the verify
 * pass and make no stability promise beyond RKSC_ABI_VERSION.
 */
#ifndef RKSC_TESTING_H_
#define RKSC_TESTING_H_

#include "rksc.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Dense projection as the verify pass runs it: for split z, P[z][m][n] =
 * sum over the split's K range of A[m][k] * W[n][k], W [N, K] of `dtype`.
 * RKSC_BF16: the activation is given as its bf16 hi/lo planes A and A_lo
 * ([M, K] each, A = hi + lo). RKSC_F32: A is fp32 [M, K], A_lo unused.
 * P is fp32 and must hold 8 * M * N floats. splits = 0 uses the library's
 * own split-K plan for this shape (bf16 with M <= 16, or M <= 32 and
 * K <= 16384, always does: the weight-streaming kernel fixes its splits); the
 * number used is written to
 * *splits_used (host pointer). K % 8 == 0. */
rksc_status rksc_test_gemm(int32_t dtype, const void* A, const void* A_lo, const void* W, float* P, int32_t M,
                           int32_t N, int32_t K, int32_t splits, int32_t* splits_used, void* stream);

/* rksc_test_gemm with the kernel chosen by the caller: kind = -1 the
 * library's own choice for this shape, 0 the 128-row-tile kernel, 1 the
 * 256 x 256-tile kernel, 2 the weight-streaming kernel for at most 32 rows
 * (kinds 1 and 2 bf16 only; kind 2 needs M <= 32, N % 4 == 0, K <= 32768 and,
 * above 16 rows, K <= 16384, and fixes its own splits; RKSC_ERR_UNSUPPORTED
 * otherwise). The verify pass picks kind 1 for projections with many rows and
 * kind 2 for a decode step of at most 32 branches. */
rksc_status rksc_test_gemm_kind(int32_t dtype, const void* A, const void* A_lo, const void* W, float* P,
                                int32_t M, int32_t N, int32_t K, int32_t splits, int32_t kind,
                                int32_t* splits_used, void* stream);

/* rksc_test_gemm_kind with a shrunken live set, as after branch exits in the
 * verify pass (Alg. VerifyWithEntropyExit; Sec. 2.3 "Layer-level entropy
 * exit"): the kernels are launched for M rows (the plan of an M-row call), but
 * a control block in `ctrl_scratch` (a device buffer of at least 4096 bytes,
 * overwritten) says that only live_count branches of branch_len rows are live,
 * so only rows m < live_count * branch_len of P are written; the other rows
 * of P are left as they were. Requires 1 <= live_count <= RKSC_MAX_BRANCHES,
 * branch_len >= 1 and live_count * branch_len <= M. */
rksc_status rksc_test_gemm_live(int32_t dtype, const void* A, const void* A_lo, const void* W, float* P, int32_t M,
                                int32_t N, int32_t K, int32_t splits, int32_t kind, int32_t live_count,
                                int32_t branch_len, void* ctrl_scratch, int32_t* splits_used, void* stream);

/* The gate|up projection with its SwiGLU (the down projection's input), bf16
 * weights: a = silu(A W_gate^T) * (A W_up^T) for W [2F, K] (gate rows, then up
 * rows), the activation given as bf16 hi/lo planes A, A_lo [M, K]. a_out
 * receives a as bf16 hi/lo planes [M, F] (hi at a_out, lo M * F elements
 * later). fused = 1: the 256 x 256 kernel over one K split with the SwiGLU in
 * its epilogue (what the verify pass runs for projections with many rows;
 * RKSC_ERR_UNSUPPORTED if the planner has no such plan for the shape);
 * fused = 0: the 128-row kernel's split partials in P (8 * M * 2F floats)
 * combined by the SwiGLU kernel. */
rksc_status rksc_test_gate_up_swiglu(const void* A, const void* A_lo, const void* W, void* a_out, float* P,
                                     int32_t M, int32_t F, int32_t K, int32_t fused, void* stream);

/* The plan rksc_test_gemm_kind would launch for this shape, without launching
 * anything (host only): plan[0..4] = kernel kind (0, 1 or 2 as above), rows
 * and columns of a workgroup's output tile, number of K splits, K elements per
 * split. The verify pass, the root forward and the decode use the plan of
 * kind = -1, splits = 0 for each projection. */
rksc_status rksc_test_gemm_plan(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t splits, int32_t kind,
                                int32_t* plan);

/* Shared-prefix attention of one layer for B branches of s tokens, with the
 * same split of the prefix across workgroups as the verify pass:
 * q [B*s, H, hd], k_own/v_own [B, Hkv, s, hd] are fp32 and prefix_k/prefix_v
 * [Hkv, n, hd] of `dtype`. The output o [B*s, H*hd] is fp32 for RKSC_F32 and
 * for RKSC_BF16 its bf16 hi/lo planes (hi at o, lo B*s*H*hd elements later:
 * 4 bytes per element in total). `scratch` is a device buffer of at least
 * rksc_test_attention_scratch_size() bytes. */
size_t rksc_test_attention_scratch_size(int32_t dtype, int32_t B, int32_t n, int32_t s, int32_t H, int32_t Hkv,
                                        int32_t hd);
rksc_status rksc_test_attention(int32_t dtype, const void* q, const void* prefix_k, const void* prefix_v,
                                const void* k_own, const void* v_own, void* o, int32_t B, int32_t n,
                                int32_t s, int32_t H, int32_t Hkv, int32_t hd, void* scratch,
                                size_t scratch_bytes, void* stream);

/* Measurement variant of rksc_verify_forward: the same validation, kernels and
 * launches, plus a HIP event recorded on `stream` right before and right after
 * the launches named below, so that a benchmark can time single kernels inside
 * the real sequence with hipEventElapsedTime. `events` is a HOST array of
 * RKSC_PROFILE_EVENTS_PER_LAYER * n_layers hipEvent_t handles created by the
 * caller; NULL entries are skipped. Per layer l the entries at
 * l * RKSC_PROFILE_EVENTS_PER_LAYER + k are, for k =
 *   0/1 QKV projection, 2/3 attention (with its split-KV combine where the
 *   plan splits the prefix), 4/5 O projection, 6/7 gate|up projection (7 is
 *   recorded right after the projection kernel, before the separate SwiGLU /
 *   split-K combine kernel of the 128-row plans), 8/9 down projection,
 *   10/11 fused lm_head-entropy.
 * The lm_head-entropy events are recorded only at the last layer of each exit
 * window (rksc_verify_window), where the stream runs. Events of layers a
 * branch set never reaches are recorded too (their kernels exit at once). */
#define RKSC_PROFILE_EVENTS_PER_LAYER 12
rksc_status rksc_verify_forward_profiled(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv,
                                         const int32_t* branch_tokens, int32_t n_branches, int32_t branch_len,
                                         float tau, int32_t patience, float* entropy, int32_t* exit_layer,
                                         float* hidden_last, void* workspace, size_t workspace_bytes,
                                         void* stream, void* const* events);

/* Precision ablation of the verify pass (Eq. entropy is the quantity the
 * ablation is judged on): rksc_verify_forward with the fp32 value at chosen
 * operand sites carried at bf16 precision instead of as a bf16 hi + lo pair.
 * drop_mask is an OR of the RKSC_DROP_* bits:
 *   QKV_LO, O_LO, GATE_UP_LO, DOWN_LO   the lo plane of that projection's
 *                                       activation is zeroed (bf16 hi alone);
 *   Q_LO, OWN_KV_LO                     the queries / the branch's own keys and
 *                                       values are rounded to bf16 before the
 *                                       attention;
 *   P_LO                                the attention probabilities enter P.V
 *                                       as bf16 alone;
 *   LM_HEAD_LO                          the final-normed rows meet W_lm as bf16
 *                                       alone.
 * bf16 models only (RKSC_ERR_UNSUPPORTED otherwise); drop_mask = 0 is
 * rksc_verify_forward. For measuring which sites the error bars need, not for
 * production use. */
#define RKSC_DROP_QKV_LO 0x01u
#define RKSC_DROP_O_LO 0x02u
#define RKSC_DROP_GATE_UP_LO 0x04u
#define RKSC_DROP_DOWN_LO 0x08u
#define RKSC_DROP_Q_LO 0x10u
#define RKSC_DROP_OWN_KV_LO 0x20u
#define RKSC_DROP_P_LO 0x40u
#define RKSC_DROP_LM_HEAD_LO 0x80u
#define RKSC_DROP_ALL 0xffu
rksc_status rksc_test_verify_precision(const rksc_weights* weights, const rksc_prefix_kv* prefix_kv,
                                       const int32_t* branch_tokens, int32_t n_branches, int32_t branch_len,
                                       float tau, int32_t patience, float* entropy, int32_t* exit_layer,
                                       float* hidden_last, void* workspace, size_t workspace_bytes, void* stream,
                                       uint32_t drop_mask);

#ifdef __cplusplus
}
#endif

#endif /* RKSC_TESTING_H_ */
