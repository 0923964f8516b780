/*
 * streamkl.h -- C ABI of the fused attention-distillation KL primitive for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (paper Sec. 2.1, "KL Divergence"): for every batch b, head h
 * and query row i,
 *
 *     S1 = s1 * Q1[b,h,i] K1[b,h]^T,   S2 = s2 * Q2[b,h,i] K2[b,h]^T,
 *     P_t = softmax(S_t) over the keys row i may attend,
 *     L[b,h,i] = KL(P1 || P2) = sum_j P1_j (log P1_j - log P2_j)   (eq:kl-def)
 *
 * computed in one online pass over key tiles (eq:kl-final, Algorithm 1) that
 * never materialises P1 or P2, and its gradients (eq:kl-case1, eq:kl-case2,
 * Algorithms 2 and 3) recomputed tile by tile from the saved row statistics.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers owned by the caller. The library
 *   never allocates, frees or retains device memory, keeps no per-call state,
 *   and never writes its inputs.
 * - Q1, K1, Q2, K2 are bf16, contiguous, row-major:
 *       Q1 [B, H, N_Q, d1]   K1 [B, H, N_K, d1]
 *       Q2 [B, H, N_Q, d2]   K2 [B, H, N_K, d2]
 *   and must be 16-byte aligned. Row statistics and gradients are fp32,
 *   contiguous, 4-byte aligned: kl, lse1, lse2, dkl are [B, H, N_Q];
 *   dQ1 [B,H,N_Q,d1], dQ2 [B,H,N_Q,d2], dK1 [B,H,N_K,d1], dK2 [B,H,N_K,d2].
 * - s1, s2 are the logit scales (the paper leaves the sqrt(d) factor out of
 *   its formulas; the usual choice is 1/sqrt(d_t)). They must be finite and > 0.
 * - causal = 1 masks with bottom-right alignment: query row i sits at
 *   absolute position N_K - N_Q + i and attends keys j <= that position
 *   (j <= i when N_Q = N_K). Rows left with no key (only when N_Q > N_K)
 *   give KL = 0, LSE = -inf and zero gradients.
 * - direction = STREAMKL_KL_FWD evaluates KL(P1 || P2) (the paper's
 *   objective); STREAMKL_KL_REV evaluates KL(P2 || P1). lse1/lse2 always
 *   belong to (Q1,K1,s1) / (Q2,K2,s2).
 * - Supported head dims: d1, d2 in {32, 64, 96, ..., 256} (multiples of 32).
 *   The kernels are built for multiples of 64; 32, 96, 160 and 224 run those
 *   of the next multiple of 64 with the missing columns read as zeros, so
 *   their matrix work is that of the wider head.
 * - B, H, N_Q, N_K >= 0; a zero extent is a valid call that launches
 *   nothing (N_K = 0 with N_Q > 0 makes every row empty). One head's rows
 *   of any tensor must span less than 4 GiB as fp32 (N * max(d1, d2) * 4 <
 *   2^32), else STREAMKL_ERR_UNSUPPORTED.
 * - Inputs are expected finite, with every raw dot product q.k below 1e29
 *   in magnitude (the kernels stand in -1e30 for the logit of a key a row
 *   may not see). Non-finite values are not detected or reported. Where
 *   they reach: the forward outputs (kl, lse1, lse2) of a query row are
 *   non-finite if the row holds one or attends a key row that does, and
 *   are otherwise bit for bit those of finite inputs. The backward adds a
 *   second route: a row's masked (zero) logit gradients still multiply the
 *   key rows of the 32-key tiles the row's block streams, so a non-finite
 *   entry in column c of key row j can make column c of dQ non-finite for
 *   rows of the same head that do not attend key j (0 x inf), and likewise
 *   column c of dK from a query row. Other heads are never affected.
 * - Work is enqueued on `stream` (NULL = the default stream) and the call
 *   returns before it completes. Asynchronous faults surface at the caller's
 *   next synchronisation, as usual for HIP.
 * - Arguments are checked before anything is enqueued; on a non-zero return
 *   nothing was launched (except STREAMKL_ERR_HIP, see below). No C++
 *   exception crosses this interface. Calls on different streams are
 *   independent and thread-safe.
 */
#ifndef STREAMKL_H
#define STREAMKL_H

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  STREAMKL_OK = 0,
  STREAMKL_ERR_INVALID_ARG = 1, /* NULL pointer, negative extent, bad flag, scale, alignment */
  STREAMKL_ERR_UNSUPPORTED = 2, /* head dim not in {32, 64, ..., 256}, extent too large     */
  STREAMKL_ERR_HIP = 3,         /* a kernel launch was rejected by the HIP runtime          */
  STREAMKL_ERR_SCRATCH_LIMIT = 4 /* streamkl_fwd_split_noalloc: partials exceed its scratch */
} streamkl_status;

typedef enum {
  STREAMKL_KL_FWD = 0, /* L = KL(P1 || P2), eq:kl-def                */
  STREAMKL_KL_REV = 1  /* L = KL(P2 || P1), the two roles swapped    */
} streamkl_direction;

/* Attention-score activations (Sec. 3.1, "Generalizability beyond Softmax"). */
typedef enum {
  STREAMKL_ACT_SOFTMAX = 0, /* P_t = softmax(S_t); L = KL(P1 || P2), eq:kl-def                  */
  STREAMKL_ACT_SIGMOID = 1  /* A_t = sigmoid(S_t), not normalised; L = generalized KL (below)  */
} streamkl_activation;

/* Backward kernel strategies of Sec. 4.2 ("GPU Kernel Design"). */
typedef enum {
  STREAMKL_BWD_AUTO = 0,     /* adaptive selection (streamkl_bwd_choose)          */
  STREAMKL_BWD_SEPARATE = 1, /* query-owned dQ kernel + key-owned dK kernel        */
  STREAMKL_BWD_FUSED = 2     /* one key-owned kernel, dQ added with fp32 atomics   */
} streamkl_bwd_strategy;

/* Gradient request bits of streamkl_bwd_choose. */
enum {
  STREAMKL_GRAD_DQ1 = 1,
  STREAMKL_GRAD_DK1 = 2,
  STREAMKL_GRAD_DQ2 = 4,
  STREAMKL_GRAD_DK2 = 8
};

/*
 * Forward pass (Algorithm 1, Sec. 3.2; eq:kl-final): one tiled pass over the
 * keys per block of query rows keeping the five running row scalars
 * (m1, l1, m2, l2, acc). Writes, for every row,
 *   kl   = L as defined by `direction`,
 *   lse1 = natural-log log-sum-exp of the scaled, masked logits S1,
 *   lse2 = the same for S2
 * and nothing else (the saved state of Sec. 3.2, "Saved state for backward").
 * Required: Q1, K1, Q2, K2, kl, lse1, lse2 (unless the extent is zero).
 */
int streamkl_fwd(const void* Q1, const void* K1, const void* Q2, const void* K2,
                 int B, int H, int N_Q, int N_K, int d1, int d2,
                 float s1, float s2, int causal, int direction,
                 float* kl, float* lse1, float* lse2,
                 hipStream_t stream);

/*
 * Backward pass (Algorithms 2 and 3, Sec. 4): recomputes S1, S2 and
 * P_t = exp(S_t - LSE_t) tile by tile from kl/lse1/lse2 of streamkl_fwd (same
 * inputs, scales, causal flag and direction) and returns the gradients of
 * sum_{b,h,i} dkl[b,h,i] * L[b,h,i]:
 *   FWD: dS2 = g (P2 - P1)                                   (eq:kl-case1)
 *        dS1 = g P1 (r - L), r = (S1 - S2) - (LSE1 - LSE2)   (eq:kl-case2, eq:stable-r)
 *   REV: dS1 = g (P1 - P2),  dS2 = g P2 (r' - L), r' = -r
 *   dQ_t = s_t dS_t K_t,  dK_t = s_t dS_t^T Q_t.
 * dkl: per-row upstream gradient g; NULL means g = 1 for every row.
 * dQ1, dK1, dQ2, dK2: each NULL (not computed) or written in full
 * (overwritten, never accumulated into). At least one must be non-NULL.
 * The outputs must not overlap each other or the inputs. When a dK and a dQ
 * are both requested, the call first writes the dK kernel's per-row
 * statistics into one of the dQ outputs, which the dQ kernel then
 * overwrites: work ordered after the call on `stream` sees only the final
 * dQ, but other streams must not read a dQ output before the call completes.
 * dQ tiles are owned by query blocks and dK tiles by key blocks, so no
 * atomics are used and results are bitwise reproducible run to run (the
 * separate-kernel strategy of Sec. 4.2; streamkl_bwd_ex offers the fused one).
 * Both gradient pairs of a call are formed by one set of kernels while
 * d1 + d2 < 448 (head dims rounded up to multiples of 64); from there on by
 * the second-slot kernels followed by the first-slot ones, each recomputing
 * the logits (one kernel holding both pairs would not fit the registers).
 */
int streamkl_bwd(const void* Q1, const void* K1, const void* Q2, const void* K2,
                 int B, int H, int N_Q, int N_K, int d1, int d2,
                 float s1, float s2, int causal, int direction,
                 const float* kl, const float* lse1, const float* lse2,
                 const float* dkl,
                 float* dQ1, float* dK1, float* dQ2, float* dK2,
                 hipStream_t stream);

/*
 * Backward pass with a choice of kernel strategy (Sec. 4.2, "Separate dQ/dK
 * Kernels", "Fused Backward Kernel", "Adaptive Strategy Selection").
 * Arguments, outputs and errors are those of streamkl_bwd, plus `strategy`:
 *   STREAMKL_BWD_SEPARATE  exactly streamkl_bwd (bitwise reproducible).
 *   STREAMKL_BWD_FUSED     one kernel over (batch*head, 128-key blocks): each
 *                          workgroup recomputes its key block against every
 *                          query tile once, writes dK for its keys and adds
 *                          its share of dQ with fp32 atomic adds. dQ is first
 *                          zeroed on `stream`. The summation order of dQ is
 *                          not fixed, so dQ may differ between runs in the
 *                          last bits (dK does not). Returns
 *                          STREAMKL_ERR_UNSUPPORTED when a dQ is requested
 *                          and the fused kernel's working set does not fit
 *                          in LDS for these head dims (only when gradients
 *                          of both distributions are requested and
 *                          d1 + d2 > 320), or when a head dim is not a
 *                          multiple of 64.
 *   STREAMKL_BWD_AUTO      the strategy streamkl_bwd_choose returns.
 * With no dQ requested every strategy runs the dK kernel alone.
 */
int streamkl_bwd_ex(const void* Q1, const void* K1, const void* Q2, const void* K2,
                    int B, int H, int N_Q, int N_K, int d1, int d2,
                    float s1, float s2, int causal, int direction,
                    const float* kl, const float* lse1, const float* lse2,
                    const float* dkl,
                    float* dQ1, float* dK1, float* dQ2, float* dK2,
                    int strategy, hipStream_t stream);

/*
 * Adaptive strategy selection (Sec. 4.2): with T_Q and T_K the numbers of
 * 128-row query and key tiles per head, returns STREAMKL_BWD_FUSED when
 * T_Q * C <= T_K (dQ small next to dK, so its atomics stay cheap) with C = 8,
 * T_Q <= 4, and the fused kernel exists for the request (head dims that
 * are multiples of 64, working set within LDS); else
 * STREAMKL_BWD_SEPARATE. The constants were measured on MI355X: there the
 * fused kernel loses beyond 512 query rows at any N_K. `grads` is an OR of
 * STREAMKL_GRAD_* bits. Returns 0 for invalid or unsupported arguments.
 */
int streamkl_bwd_choose(int B, int H, int N_Q, int N_K, int d1, int d2,
                        int causal, int direction, int grads);

/*
 * Forward with a choice of score activation (Sec. 3.1, "Generalizability
 * beyond Softmax": activations without softmax's global normalisation need
 * no normalisers). The paper defines neither the scores nor the divergence
 * for that case; this library reads it as:
 *   STREAMKL_ACT_SOFTMAX  exactly streamkl_fwd (stat1, stat2 = lse1, lse2).
 *   STREAMKL_ACT_SIGMOID  A_t[j] = sigmoid(S_t[j]) with no normalisation and
 *       L = sum_j [A1 log(A1 / A2) - A1 + A2] over the keys the row may
 *       attend (the generalized KL divergence of the two score rows: >= 0,
 *       0 iff A1 = A2, eq:kl-def when both rows sum to 1); REV swaps the
 *       roles. stat1, stat2 receive the row masses sum_j A1[j], sum_j A2[j]
 *       (each may be NULL). A row with no visible key gives L = 0. ReLU and
 *       tanh scores are not offered: under this divergence L is infinite
 *       where A2 = 0 < A1 (ReLU) and undefined for negative scores (tanh).
 * Single pass only (no split-K); other arguments, layouts and errors as for
 * streamkl_fwd. An activation outside the enum is STREAMKL_ERR_INVALID_ARG.
 */
int streamkl_fwd_act(const void* Q1, const void* K1, const void* Q2, const void* K2,
                     int B, int H, int N_Q, int N_K, int d1, int d2,
                     float s1, float s2, int causal, int direction, int activation,
                     float* kl, float* stat1, float* stat2,
                     hipStream_t stream);

/*
 * Backward for streamkl_fwd_act's objective sum_{b,h,i} dkl L (separate
 * query- and key-owned kernels; bitwise reproducible).
 *   STREAMKL_ACT_SOFTMAX  exactly streamkl_bwd (kl, stat1, stat2 = kl, lse1,
 *                         lse2 of the forward).
 *   STREAMKL_ACT_SIGMOID  FWD: dS2 = g (A2 - A1)(1 - A2),
 *                              dS1 = g A1 (1 - A1)(log A1 - log A2);
 *                         REV: the roles swapped. No saved statistic is
 *                         needed: kl, stat1, stat2 are not read (may be NULL).
 * dQ_t = s_t dS_t K_t, dK_t = s_t dS_t^T Q_t; other arguments as streamkl_bwd.
 */
int streamkl_bwd_act(const void* Q1, const void* K1, const void* Q2, const void* K2,
                     int B, int H, int N_Q, int N_K, int d1, int d2,
                     float s1, float s2, int causal, int direction, int activation,
                     const float* kl, const float* stat1, const float* stat2,
                     const float* dkl,
                     float* dQ1, float* dK1, float* dQ2, float* dK2,
                     hipStream_t stream);

/*
 * Split-K forward (Sec. 3.3, "Split-K variant" and "Adaptive split
 * selection"): for heads with few query rows, the key range is cut into
 * `splits` contiguous chunks of whole 32-key tiles, each (head, query block,
 * chunk) runs the online pass of streamkl_fwd over its chunk and stores the
 * five row statistics (m1, l1, m2, l2, acc) in `workspace`, and a reduce
 * kernel merges the chunks per row with the rescaling rule of Sec. 3.3
 * (associative, so the result equals streamkl_fwd up to fp32 rounding).
 * Arguments and outputs are those of streamkl_fwd, plus:
 *   splits          >= 1; 1 runs streamkl_fwd itself and needs no workspace.
 *                   streamkl_fwd_split_count gives the paper's adaptive choice.
 *   workspace       device memory owned by the caller, 4-byte aligned, at
 *                   least streamkl_fwd_split_workspace_bytes(B, H, N_Q, splits)
 *                   bytes; its contents on entry are ignored and on return
 *                   are unspecified. Two calls may share it only if they are
 *                   ordered on one stream.
 *   workspace_bytes its size in bytes (smaller than required:
 *                   STREAMKL_ERR_INVALID_ARG, nothing launched).
 */
int streamkl_fwd_split(const void* Q1, const void* K1, const void* Q2, const void* K2,
                       int B, int H, int N_Q, int N_K, int d1, int d2,
                       float s1, float s2, int causal, int direction, int splits,
                       void* workspace, size_t workspace_bytes,
                       float* kl, float* lse1, float* lse2,
                       hipStream_t stream);

/* Bytes of device memory streamkl_fwd_split_noalloc holds on each GPU it runs on. */
#define STREAMKL_NOALLOC_SCRATCH_BYTES (16u << 20)

/*
 * Allocation-free split-K forward, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. Arguments, outputs and results are those of
 * streamkl_fwd_split without the workspace: the partial row statistics go to
 * a static array of STREAMKL_NOALLOC_SCRATCH_BYTES (16 MiB) that the library
 * holds on every GPU it runs on until the process ends. The call allocates
 * and frees nothing.
 *   - A request whose partials need more
 *     (streamkl_fwd_split_workspace_bytes(B, H, N_Q, splits) >
 *     STREAMKL_NOALLOC_SCRATCH_BYTES) returns STREAMKL_ERR_SCRATCH_LIMIT and
 *     launches nothing; splits = 1 needs no scratch.
 *   - Every call on one GPU uses that GPU's one array, which keeps the last
 *     call's contents. Calls whose work may overlap on one GPU (different
 *     streams, or host threads without ordering between them) race on it and
 *     give undefined results; calls ordered on one stream are safe. Nothing
 *     in it needs clearing: every partial is written before it is read.
 *   - `stream` must belong to the current device (else
 *     STREAMKL_ERR_INVALID_ARG). The first call on a device looks up the
 *     array's address there; if HIP fails that lookup, STREAMKL_ERR_HIP.
 */
int streamkl_fwd_split_noalloc(const void* Q1, const void* K1, const void* Q2, const void* K2,
                               int B, int H, int N_Q, int N_K, int d1, int d2,
                               float s1, float s2, int causal, int direction, int splits,
                               float* kl, float* lse1, float* lse2,
                               hipStream_t stream);

/* Workspace bytes streamkl_fwd_split needs: 20 * splits * B * H * N_Q when
   splits > 1, else 0. Returns 0 for negative extents. */
size_t streamkl_fwd_split_workspace_bytes(int B, int H, int N_Q, int splits);

/*
 * Adaptive split count (Sec. 3.3): with P_base the number of workgroups the
 * single-pass forward launches for these shapes and P_target = 512 (two per
 * CU of an MI355X), returns 1 when P_base >= P_target and otherwise
 * min(floor(P_target / P_base), number of 32-key tiles), at least 1.
 * Returns 0 for invalid or unsupported arguments.
 */
int streamkl_fwd_split_count(int B, int H, int N_Q, int N_K, int d1, int d2);

/* Static description of a status code. Never NULL. */
const char* streamkl_strerror(int status);

/* Library version string, e.g. "streamkl 0.1.0 gfx950". Never NULL. */
const char* streamkl_version(void);

/* 1 if d is a supported head dimension, else 0. */
int streamkl_supported_head_dim(int d);

#ifdef __cplusplus
}
#endif

#endif /* STREAMKL_H */
