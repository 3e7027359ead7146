/*
 * cmsd.h - confidence-modulated speculative decoding: the vocabulary-wide logit
 * pass (arXiv 2508.15371, Sec. III.B), as a C ABI over gfx950 HIP kernels.
 *
 * Three calls, in the order one decoding iteration uses them (plus
 * cmsd_draft_sample, which draws sampled drafts from the drafter rows):
 *
 *   cmsd_confidence  per drafter row: softmax normaliser, entropy, top-1/top-2
 *                    margins and the unified confidence C     (Sec. III.B(1))
 *   cmsd_draft_len   per sequence: adaptive draft length k_b from the mean
 *                    confidence, plus packed target-row offsets (Sec. III.B(b))
 *   cmsd_verify      per drafted position: confidence-modulated acceptance,
 *                    accepted-prefix length, and the final token sampled from
 *                    the residual (or bonus) distribution     (Sec. III.A, III.B(c))
 *
 * cmsd_logit_pass does all three in one call (three or four launches, two in GREEDY
 * mode) for a dense target layout; cmsd_logit_pass_fused does it in one launch, for small
 * batches.
 *
 * Conventions shared by every call
 *   - All array pointers are DEVICE pointers (hipMalloc / torch CUDA tensors);
 *     params structs are HOST pointers read during the call.  The caller owns
 *     every buffer and the library allocates no memory.  Its only state is the
 *     overrides of cmsd_set_row_shape and cmsd_set_pass_decisions and, per device, the static
 *     scratch array of cmsd_logit_pass_noalloc.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Calls
 *     only enqueue work and return; results are ready when the stream is.
 *   - Argument errors are detected on the host before anything is enqueued and
 *     returned as CMSD_ERR_ARG / CMSD_ERR_DTYPE; in that case no output is
 *     touched.  CMSD_ERR_LAUNCH reports a failed kernel launch.
 *   - Launch sizes: a kernel launch holds fewer than 2^32 work-items, and a call
 *     whose launches would not returns CMSD_ERR_ARG: cmsd_verify needs
 *     batch*(k_max+1) < 2^26, cmsd_logit_pass and cmsd_logit_pass_noalloc
 *     batch*(2*k_max+1) < 2^26 (cmsd_logit_pass_fused < 2^24), and every call that
 *     samples (cmsd_verify, the single-call passes, cmsd_draft_sample) batch (n_rows)
 *     < 2^24 and batch*S < 2^26 for S = ceil((vocab/4 + 2)/256) vocabulary slices.
 *     cmsd_confidence takes any n_rows < 2^31.
 *   - Device-resident indices (draft lengths, offsets, drafted ids) cannot be
 *     checked on the host; the kernels check them and report a violation per
 *     sequence through the outputs (see cmsd_verify) without reading out of
 *     bounds.
 *   - Logit preconditions (not checked): every row has at least one finite
 *     entry; entries are finite with |z| < 2^96, or -inf (masked tokens); no
 *     NaN or +inf.  Violations give unspecified values, never a fault.  Rows with
 *     -inf entries are read once, like any other.
 *   - Logit dtypes: CMSD_F32 (float) or CMSD_BF16 (raw bfloat16, 2 bytes).
 *     Pointers must be aligned to the element size; rows need no other
 *     alignment (an unaligned head and tail are read element-wise).
 *   - Results are deterministic: fixed reduction orders, no float atomics.
 */
#ifndef CMSD_H
#define CMSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CMSD_OK = 0,
  CMSD_ERR_ARG = 1,    /* invalid size, pointer or parameter            */
  CMSD_ERR_DTYPE = 2,  /* unknown logit dtype                            */
  CMSD_ERR_LAUNCH = 3, /* the HIP runtime refused a launch               */
  CMSD_ERR_SIZE = 4    /* the problem exceeds CMSD_STATIC_SCRATCH_BYTES
                          (cmsd_logit_pass_noalloc only)                  */
} cmsd_status;

/* Size of the static per-device scratch array that cmsd_logit_pass_noalloc uses in
 * place of a caller workspace: 16 MiB, i.e. cmsd_verify_workspace_bytes(batch,
 * k_max, vocab) up to 16 MiB (e.g. batch 1024 at k_max 16, vocab 128256). */
#define CMSD_STATIC_SCRATCH_BYTES (16u << 20)

typedef enum { CMSD_F32 = 0, CMSD_BF16 = 1 } cmsd_dtype;

typedef enum {
  CMSD_MODE_STANDARD = 0, /* standard speculative sampling only                    */
  CMSD_MODE_CM = 1,       /* plus the confidence-modulated gate (OR-ed)            */
  CMSD_MODE_GREEDY = 2    /* the paper's deterministic rule: the target's top token
                             or the gate; the top token after the accepted prefix  */
} cmsd_mode;

/* Weights of the unified confidence, Sec. III.B(1): C = lambda_ent*(1 - H/ln V)
 * + lambda_margin*sigmoid(beta_margin*(z1 - z2)) + lambda_soft*min(1, (P1-P2)/(1-1/V)).
 * Each lambda in [0,1], |sum - 1| <= 1e-6; beta_margin finite and > 0. */
typedef struct {
  float lambda_ent;
  float lambda_margin;
  float lambda_soft;
  float beta_margin;
} cmsd_conf_params;

/* Draft-length clip, Sec. III.B(b): k = min(k_max, max(k_min, floor(alpha*Cbar*k_max))).
 * 1 <= k_min <= k_max <= 4096, 0 < alpha <= 1. */
typedef struct {
  int32_t k_min;
  int32_t k_max;
  float alpha;
} cmsd_draft_params;

/* Verification, Sec. III.B(c): tau_t = tau_base + gamma*(1 - C_t); the gate passes
 * when the drafted token is within the target's top_beta and its log-prob gap to the
 * target's top-1 is <= tau_t.  mode is a cmsd_mode; top_beta >= 0 (0 disables the
 * gate); tau_base, gamma finite (gamma may be negative). */
typedef struct {
  int32_t mode;
  int32_t top_beta;
  float tau_base;
  float gamma;
} cmsd_verify_params;

/* One record per drafter row (32 bytes), written by cmsd_confidence. */
typedef struct {
  float max_logit;    /* z^(1)                                                  */
  float sum_exp;      /* A = sum_v exp(z_v - z^(1)); log-normaliser = max_logit + ln A */
  float entropy;      /* H = -sum p ln p, nats (Sec. III.B(1), entropy)           */
  float margin_soft;  /* P^(1) - P^(2) in [0,1] (softmax margin)                  */
  float margin_logit; /* z^(1) - z^(2) >= 0, +inf with a single finite logit      */
  float conf;         /* unified confidence C_t (Sec. III.B(1), ensemble)         */
  int32_t top1;       /* lowest index attaining z^(1)                             */
  uint32_t flags;     /* bit 0: the row contains -inf entries                     */
} cmsd_row_stats;

/* One record per packed target row (32 bytes), written by cmsd_verify. */
typedef struct {
  float max_logit;    /* max of the target row                                    */
  float sum_exp;      /* sum_v exp(z_v - max)                                     */
  int32_t n_greater;  /* CM/GREEDY: min(#{v : z_v > z_drafted}, top_beta); 0 in
                         STANDARD mode or with top_beta = 0; -1 on the final row   */
  int32_t accept;     /* 1 accepted, 0 rejected, -1 final row, -2 invalid input   */
  int32_t top1;       /* GREEDY mode: lowest index of the row max; else -1        */
  int32_t reserved[3];
} cmsd_target_stats;

/*
 * cmsd_confidence - reduce each logit row to its cmsd_row_stats (Sec. III.B(1):
 * entropy, logit margin, softmax margin, unified confidence).
 *
 *   logits      device, n_rows rows of `vocab` logits; row r starts at element
 *               r*row_stride.  dtype CMSD_F32 or CMSD_BF16.
 *   n_rows      >= 0 (0: nothing is enqueued).  For a draft of k_max positions
 *               over B sequences, n_rows = B*k_max with row b*k_max+i = position i.
 *   vocab       >= 2 and < 2^31; row_stride >= vocab (elements).
 *   params      host; see cmsd_conf_params.
 *   stats       device, n_rows records (output).
 * Errors: CMSD_ERR_ARG (null pointer, bad size, misaligned pointer, bad params),
 *         CMSD_ERR_DTYPE, CMSD_ERR_LAUNCH.
 */
cmsd_status cmsd_confidence(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab,
                            int64_t row_stride, const cmsd_conf_params* params,
                            cmsd_row_stats* stats, void* stream);

/*
 * cmsd_confidence_var - cmsd_confidence plus, per row, the population variance of
 * the row's finite logits: the logit-variance proxy for drafter uncertainty that
 * Sec. I names beside entropy and the top-1/top-2 margin.  The paper gives it no
 * normalisation, so it is reported and does not enter C.  Same arguments and
 * errors as cmsd_confidence, plus:
 *   logit_var   device, n_rows floats (output): sum_v (z_v - mean)^2 / n over the n
 *               finite logits of the row (0 with a single finite logit).
 */
cmsd_status cmsd_confidence_var(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab,
                                int64_t row_stride, const cmsd_conf_params* params,
                                cmsd_row_stats* stats, float* logit_var, void* stream);

/*
 * cmsd_draft_len - adaptive draft length per sequence (Sec. III.B(b)).
 *
 *   stats           device, batch*k_max records from cmsd_confidence (row b*k_max+i).
 *   batch           >= 0.
 *   params          host; k_max must equal the number of drafter rows per sequence.
 *                   The window mean runs over all k_max positions.
 *   draft_len       device, batch int32 (output): k_b in [k_min, k_max].
 *   target_offsets  device, batch+1 int32 (output): exclusive prefix sum of k_b+1,
 *                   i.e. the first packed target row of each sequence; entry
 *                   [batch] is the total number of target rows.
 * The mean and product are formed in double precision, left to right.
 * Errors: CMSD_ERR_ARG, CMSD_ERR_LAUNCH.
 */
cmsd_status cmsd_draft_len(const cmsd_row_stats* stats, int32_t batch, const cmsd_draft_params* params,
                           int32_t* draft_len, int32_t* target_offsets, void* stream);

/*
 * cmsd_verify - confidence-modulated verification (Sec. III.B(c)) of every drafted
 * position, accepted-prefix length (halt at the first rejection, Sec. III.A), and
 * the final token: on a rejection at position c, a sample from the residual
 * max(0, p_t - p_d) of target and drafter rows c; when all k_b drafts pass, a
 * sample from target row k_b.
 *
 * A position is accepted when u < p_t(y)/p_d(y) (standard speculative sampling)
 * or, in CMSD_MODE_CM, when the gate passes: #{v: z_t,v > z_t,y} < top_beta and
 * z_t^(1) - z_t,y <= tau_base + gamma*(1 - C).  In CMSD_MODE_GREEDY a position is
 * accepted iff the draft is the target's top token (lowest index among equal
 * maxima) or the gate passes, and the final token is the target's top token at the
 * first rejected position, or at position k_b; with top_beta = 0 (gate off) this is
 * exact-match verification.
 *
 *   draft_logits    device, batch*k_max drafter rows (row b*k_max+i), stride
 *                   draft_stride >= vocab elements (the rows cmsd_confidence saw).
 *   draft_stats     device, batch*k_max records from cmsd_confidence.
 *   target_logits   device, target_rows packed rows, stride target_stride >= vocab:
 *                   sequence b owns rows target_offsets[b] .. target_offsets[b]+k_b,
 *                   row target_offsets[b]+i scoring position i, the last one the
 *                   row after the final draft.  Dense layouts pass
 *                   target_offsets[b] = b*(k_max+1) and draft_len[b] = k_max.
 *   target_rows     number of rows allocated in target_logits, uniforms and
 *                   target_stats (>= target_offsets[batch]).
 *   target_offsets  device, batch+1 int32 (as written by cmsd_draft_len),
 *                   non-decreasing; a sequence whose own offsets disagree with its
 *                   draft length or target_rows is reported invalid, while
 *                   non-monotone offsets give unspecified (in-bounds) results.
 *   draft_len       device, batch int32, each in [0, k_max].
 *   drafted         device, batch*k_max int32 token ids (entries i >= k_b unused).
 *   uniforms        device, target_rows floats in [0,1), packed like the target rows:
 *                   slot i < k_b is the accept test of position i, slot k_b the
 *                   final sample.  Unused (may be NULL) in CMSD_MODE_GREEDY.
 *   dtype           logit dtype of both logit arrays.
 *   batch >= 0, k_max in [1, 4096], vocab in [2, 2^31).
 *   params          host; see cmsd_verify_params.
 *   target_stats    device, target_rows records (output): the k_b + 1 rows of every
 *                   sequence with a valid draft length and offsets; rows beyond
 *                   target_offsets[batch], and the rows of a sequence reported
 *                   invalid for its draft length or offsets, are not written.
 *   n_accepted      device, batch int32 (output): accepted prefix length c_b in
 *                   [0, k_b]; -1 if the sequence's device inputs are invalid
 *                   (offsets inconsistent with draft_len or target_rows, draft_len
 *                   out of range, drafted id outside [0, vocab)).
 *   next_token      device, batch int32 (output): the final token; -1 when invalid.
 *   workspace       device scratch of at least cmsd_verify_workspace_bytes(batch,
 *                   k_max, vocab) bytes, 8-byte aligned, owned by the caller: the
 *                   target-row results by (sequence, position) and the per-slice
 *                   partial sums of the final-token sample.  Its contents need no
 *                   initialisation and are meaningless after the call.  Calls that
 *                   share a workspace must be ordered (same stream); overlapping
 *                   calls race.
 *   workspace_bytes its size.
 * Errors: CMSD_ERR_ARG, CMSD_ERR_DTYPE, CMSD_ERR_LAUNCH.
 */
cmsd_status cmsd_verify(const void* draft_logits, int64_t draft_stride, const cmsd_row_stats* draft_stats,
                        const void* target_logits, int64_t target_stride, int64_t target_rows,
                        const int32_t* target_offsets, const int32_t* draft_len, const int32_t* drafted,
                        const float* uniforms, int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                        const cmsd_verify_params* params, cmsd_target_stats* target_stats,
                        int32_t* n_accepted, int32_t* next_token, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * cmsd_logit_pass - the whole logit pass of one decoding iteration in one call, for
 * a dense target layout: cmsd_confidence on the drafter rows, cmsd_draft_len's draft
 * length and cmsd_verify on target rows stored k_max + 1 per sequence (Sec. III.B(1)
 * to (c), Sec. III.A), in three or four launches instead of five: one row pass over
 * the drafter and target rows together (they do not depend on each other), then the
 * two final-token kernels.  Each sequence's draft length and accept tests are formed
 * either by one wave per sequence between them (large launches) or by every
 * final-token workgroup from the row results (launches of at most 32 final-token
 * waves per compute unit, one launch fewer); cmsd_set_pass_decisions forces either.
 * In GREEDY mode, whose final token is the row's top token, the decision wave ends
 * the call.
 *
 *   draft_logits    device, batch*k_max drafter rows (row b*k_max+i), stride
 *                   draft_stride >= vocab elements.
 *   target_logits   device, batch*(k_max+1) target rows, stride target_stride >=
 *                   vocab: row b*(k_max+1)+i scores position i, the last row of each
 *                   sequence is the row after its final draft.
 *   drafted         device, batch*k_max int32 token ids; all k_max of a sequence must
 *                   lie in [0, vocab), else the sequence is reported invalid.
 *   uniforms        device, batch*(k_max+1) floats in [0,1), slot b*(k_max+1)+i:
 *                   slot i < k_v the accept test of position i, slot k_v the final
 *                   sample (k_v below).  Unused (may be NULL) in CMSD_MODE_GREEDY.
 *   dtype           logit dtype of both logit arrays.
 *   batch >= 0 (0: nothing is enqueued); k_max in [1, 63]; vocab in [2, 2^31).
 *   conf, draft, verify  host; as for the separate calls (draft->k_max == k_max).
 *   adaptive        0: all k_max drafts are verified (k_v = k_max), as cmsd_verify with
 *                   draft_len[b] = k_max and dense offsets; 1: only the first k_b, the
 *                   draft length computed here (k_v = k_b), and target row k_b is the
 *                   final row.
 *   draft_stats     device, batch*k_max records (output), as cmsd_confidence writes.
 *   draft_len       device, batch int32 (output): k_b, as cmsd_draft_len computes it
 *                   (no packed offsets are formed: the layout is dense).
 *   target_stats    device, batch*(k_max+1) records (output): row i < k_v holds the
 *                   accept test of position i and row k_v has n_greater = accept = -1,
 *                   as cmsd_verify writes them; in adaptive mode rows k_b+1 .. k_max
 *                   hold the tests of the positions beyond the draft, made all the same.
 *   n_accepted      device, batch int32 (output): accepted prefix c_b in [0, k_v];
 *                   -1 when a drafted id of the sequence is outside [0, vocab).
 *   next_token      device, batch int32 (output): the final token; -1 when invalid.
 *   workspace       device scratch of at least cmsd_verify_workspace_bytes(batch,
 *                   k_max, vocab) bytes, 8-byte aligned, owned by the caller, as for
 *                   cmsd_verify (calls sharing it must be ordered).
 *   workspace_bytes its size.
 * The arithmetic is the separate calls': the outputs are bit-identical to theirs
 * whenever the row kernels run with the same workgroup size (chosen from the number
 * of rows in the launch and their length, or forced by cmsd_set_row_shape), else
 * equal up to the rounding of the reduction order.
 * Errors: CMSD_ERR_ARG, CMSD_ERR_DTYPE, CMSD_ERR_LAUNCH.
 */
cmsd_status cmsd_logit_pass(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                            int64_t target_stride, const int32_t* drafted, const float* uniforms,
                            int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                            const cmsd_conf_params* conf, const cmsd_draft_params* draft,
                            const cmsd_verify_params* verify, int32_t adaptive, cmsd_row_stats* draft_stats,
                            int32_t* draft_len, cmsd_target_stats* target_stats, int32_t* n_accepted,
                            int32_t* next_token, void* workspace, size_t workspace_bytes, void* stream);

/*
 * cmsd_set_row_events - a measurement hook, for callers that time the row pass (a
 * benchmark): arms the next cmsd_logit_pass call made by the calling host thread to
 * record row_events[0] on its stream just before its row-pass launch and
 * row_events[1] just after it, so their interval times that bandwidth-bound launch
 * alone (its kernel and the gap before it).  That call disarms the hook whatever its
 * outcome (an argument error or an empty batch records nothing); results never
 * depend on it, and the other calls neither record nor disarm.
 *   row_events      NULL (disarm), or a host array of two hipEvent_t created by the
 *                   caller.
 * Errors: CMSD_ERR_ARG (an array with a NULL event; the hook is left as it was).
 */
cmsd_status cmsd_set_row_events(void* const* row_events);

/*
 * cmsd_logit_pass_fused - cmsd_logit_pass in a single launch, for small batches
 * (Sec. III.B(1) to (c), Sec. III.A, as cmsd_logit_pass; the paper's small-batch
 * latency, Fig. 2, is what it is for).  Every drafter and target row is one
 * 256-thread workgroup; the last row of a sequence to finish (an atomic count per
 * sequence, each row's results published behind a device fence) makes the draft
 * length and the accept tests and samples the final token in the same launch.  The
 * fences serialise across the chip (tens of ns per row), and one workgroup carries each
 * sequence's final token, so the single launch is the faster call only when that work
 * is tiny (one MI355X: 1024-logit rows); at V = 32000 cmsd_logit_pass (three launches
 * for small batches) was faster at every batch measured, 1 to 64.  It is for callers
 * that need exactly one launch.  Arguments, outputs and errors are cmsd_logit_pass's
 * (cmsd_set_row_events does not apply to it), except the workspace:
 *   workspace       device scratch of at least
 *                   cmsd_logit_pass_fused_workspace_bytes(batch, k_max, vocab) bytes,
 *                   8-byte aligned, owned by the caller.  Its last 4*batch bytes
 *                   (ending at workspace_bytes rounded down to a multiple of 4) hold
 *                   one int32 counter per sequence: they must be zero before the first
 *                   call with this workspace (zero the whole buffer once when
 *                   allocating it), and every call leaves them zero, so one workspace
 *                   serves repeated calls of one (batch, k_max, vocab).  A call of
 *                   another shape lays its records over other bytes, which may hold
 *                   the counters of a former shape: zero the workspace again before
 *                   changing batch, k_max or vocab (or keep one workspace per shape),
 *                   and after another call (cmsd_verify, cmsd_logit_pass) has used it.
 *                   Calls sharing a workspace must be ordered (same stream).
 * The outputs are bit-identical to cmsd_logit_pass's when that call's row kernels
 * run with 256 threads: it chooses 256 for rows over 128 KiB and for launches of
 * fewer than 8 rows per compute unit (batch*(2*k_max+1) < 2048 on 256 compute
 * units); cmsd_set_row_shape(256, 0) forces it.
 */
cmsd_status cmsd_logit_pass_fused(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                                  int64_t target_stride, const int32_t* drafted, const float* uniforms,
                                  int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                                  const cmsd_conf_params* conf, const cmsd_draft_params* draft,
                                  const cmsd_verify_params* verify, int32_t adaptive, cmsd_row_stats* draft_stats,
                                  int32_t* draft_len, cmsd_target_stats* target_stats, int32_t* n_accepted,
                                  int32_t* next_token, void* workspace, size_t workspace_bytes, void* stream);

/* Workspace of cmsd_logit_pass_fused: cmsd_verify_workspace_bytes(batch, k_max, vocab)
 * plus 4 bytes per sequence (rounded up to 8) for the counters; 0 for batch <= 0 or
 * an invalid k_max (outside [1, 63]) / vocab. */
size_t cmsd_logit_pass_fused_workspace_bytes(int32_t batch, int32_t k_max, int64_t vocab);

/*
 * cmsd_logit_pass_noalloc - cmsd_logit_pass without a caller workspace, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  It calls no hipMalloc or hipFree and no
 * allocating routine.  Its workspace is a static array of CMSD_STATIC_SCRATCH_BYTES
 * in the library, one per device, held from the first call on that device until the
 * process ends; its device address is looked up once per device (with that device
 * current) and kept.
 *
 * Arguments, outputs and results are those of cmsd_logit_pass without workspace and
 * workspace_bytes (cmsd_set_row_events does not apply): the same kernels on the same
 * workgroup sizes, so
 * the outputs are bit-identical to cmsd_logit_pass's.  Nothing in the scratch needs
 * to start at zero; it keeps the last call's contents.
 * Limits and errors: as cmsd_logit_pass, plus CMSD_ERR_SIZE (nothing enqueued) when
 * cmsd_verify_workspace_bytes(batch, k_max, vocab) > CMSD_STATIC_SCRATCH_BYTES, and
 * CMSD_ERR_LAUNCH if the scratch address cannot be obtained.
 * Every call on one device shares that device's scratch: calls that can overlap on
 * one GPU (concurrent streams, several host threads) race and give wrong results;
 * order them on one stream.
 */
cmsd_status cmsd_logit_pass_noalloc(const void* draft_logits, int64_t draft_stride, const void* target_logits,
                                    int64_t target_stride, const int32_t* drafted, const float* uniforms,
                                    int32_t dtype, int32_t batch, int32_t k_max, int64_t vocab,
                                    const cmsd_conf_params* conf, const cmsd_draft_params* draft,
                                    const cmsd_verify_params* verify, int32_t adaptive,
                                    cmsd_row_stats* draft_stats, int32_t* draft_len,
                                    cmsd_target_stats* target_stats, int32_t* n_accepted,
                                    int32_t* next_token, void* stream);

/*
 * cmsd_set_row_shape - launch shape of the streaming row kernels (one workgroup per
 * logit row: cmsd_confidence, cmsd_confidence_var, cmsd_verify's target rows, the row
 * pass of cmsd_logit_pass / cmsd_logit_pass_noalloc), for tuning and for tests that
 * cover every shape.  Process-wide; applies to launches made after it returns.
 *   threads     0 (chosen per launch from its rows and row length), 64, 128 or 256.
 *   ring_depth  0 (chosen per launch), 2 or 3: rounds of 16-byte loads kept in flight
 *               per thread.  It schedules loads only: results are identical.
 * The workgroup size fixes the reduction order, so outputs are bit-identical across
 * calls with the same size and equal up to rounding otherwise.  cmsd_logit_pass_fused
 * always uses 256 threads.  Errors: CMSD_ERR_ARG for any other value.
 */
cmsd_status cmsd_set_row_shape(int32_t threads, int32_t ring_depth);

/*
 * cmsd_set_pass_decisions - where cmsd_logit_pass (and cmsd_logit_pass_noalloc) forms
 * each sequence's draft length and accept tests outside GREEDY mode, for tuning and
 * for tests that cover both launch sequences.  Process-wide; applies to calls made
 * after it returns.
 *   mode  0: chosen per call from the number of final-token workgroups (default);
 *         1: one decision wave per sequence writes a record the final-token kernels
 *            read (four launches);
 *         2: every final-token workgroup forms the decisions from the row results
 *            (three launches).
 * Both run the same arithmetic: the outputs are bit-identical.
 * Errors: CMSD_ERR_ARG for any other mode.
 */
cmsd_status cmsd_set_pass_decisions(int32_t mode);

/* Workspace cmsd_verify needs for `batch` sequences of up to `k_max` drafts over
 * `vocab`: per sequence, one 32-byte record per vocabulary slice (256 16-byte
 * vectors of a row) and one 32-byte record per target row position (k_max + 1);
 * 0 for batch <= 0 or an invalid k_max / vocab. */
size_t cmsd_verify_workspace_bytes(int32_t batch, int32_t k_max, int64_t vocab);

/*
 * cmsd_draft_sample - one sample per row from the row's softmax: the smallest
 * token y whose cumulative probability (vocabulary order) exceeds u (the
 * inverse-CDF convention of cmsd_verify's final token).  This draws the drafted
 * tokens that standard speculative sampling assumes (x ~ p_d); the paper's own
 * drafter takes the argmax (stats.top1), Sec. III.A step 1.
 *
 *   logits, dtype, n_rows, vocab, row_stride   as for cmsd_confidence.
 *   stats       device, n_rows records from cmsd_confidence on the same logits
 *               (max_logit is the exponent reference).
 *   uniforms    device, n_rows floats in [0,1), one per row.
 *   drafted     device, n_rows int32 (output).
 *   workspace   device scratch of cmsd_draft_sample_workspace_bytes(n_rows, vocab)
 *               bytes, 8-byte aligned, no initialisation needed.
 * Errors: CMSD_ERR_ARG, CMSD_ERR_DTYPE, CMSD_ERR_LAUNCH.
 */
cmsd_status cmsd_draft_sample(const void* logits, int32_t dtype, int64_t n_rows, int64_t vocab, int64_t row_stride,
                              const cmsd_row_stats* stats, const float* uniforms, int32_t* drafted, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Workspace cmsd_draft_sample needs: one 32-byte record per vocabulary slice
 * (256 16-byte vectors) per row; 0 for n_rows <= 0 or an invalid vocab. */
size_t cmsd_draft_sample_workspace_bytes(int64_t n_rows, int64_t vocab);

/* Human-readable name of a status code (static string). */
const char* cmsd_status_string(cmsd_status s);

/* Library ABI version, (major << 16) | minor: 1.7.  1.5 added cmsd_logit_pass_noalloc,
 * cmsd_set_row_shape and CMSD_ERR_SIZE; 1.6 cmsd_set_pass_decisions; 1.7 moved the
 * row-pass timing events out of cmsd_logit_pass's arguments into cmsd_set_row_events. */
int32_t cmsd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CMSD_H */
