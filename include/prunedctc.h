/*
 * prunedctc.h -- C ABI of the Pruned CTC head-and-loss library for MI355X (gfx950).
 *
 * The library evaluates the loss of "Pruned CTC for Memory-Efficient Large-Vocabulary
 * ASR Training" and its gradients with respect to the head input and head weight:
 *
 *   Z = H W^T (logits, never stored), lambda_m = log sum_v exp Z[m, v]      (Eq. lognorm)
 *   L_beta = -sum over alignable utterances of log sum over retained alignments of
 *            prod_t p_{pi_t}(frame)                                          (Eq. pruned-ctc)
 *   dL/dZ[m, v] = scatter_U(G)[m, v] - g_m p_v(m)                              (Eq. vjp)
 *   dH = dZ W,   dW = dZ^T H                                          (App. A, Step 3)
 *
 * following Algorithm 1 ("Pruned CTC"): union of target labels plus blank, online
 * full-vocabulary log-sum-exp over vocabulary chunks, selected-class log-probabilities
 * S, beam-pruned alignment lattice, and a chunk-by-chunk recomputed backward pass.
 *
 * Conventions (Sec. 3.1): a batch holds N utterances; utterance n has T_n >= 1 frames
 * and a blank-free target of U_n >= 0 labels.  The M = sum T_n frames are stacked
 * row-wise, utterance after utterance, without padding.  Class ids are 0-based.
 *
 * Memory: every buffer argument is a HIP device pointer owned by the caller, except the
 * two length arrays, which are host pointers.  The library allocates no device memory in
 * these calls; all scratch comes from the caller's workspace.  The loss is the sum of
 * per-utterance losses (unit weights); gradients are of that sum.
 *
 * Excluded utterances are not errors: an utterance whose target cannot be aligned to
 * its frames (T_n < U_n + r_n, r_n = number of adjacent equal label pairs; App. B.1
 * "Loss aggregation") or whose loss is not finite contributes zero loss, zero dH rows
 * and nothing to dW, and is reported in utt_status.
 *
 * Threading: calls on different streams may run concurrently if they use different
 * workspaces and outputs.  The optional kernel-timing facility (pctc_prof_*) keeps
 * process-wide state and is meant for single-threaded benchmarking.
 */
#ifndef PRUNEDCTC_H
#define PRUNEDCTC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage type of H and W.  Arithmetic: bf16 inputs are multiplied on bf16 matrix cores
 * with fp32 accumulation; f32 inputs on fp32 matrix cores. */
typedef enum { PCTC_F32 = 0, PCTC_BF16 = 1 } pctc_dtype;

typedef enum {
  PCTC_OK = 0,
  PCTC_EINVAL = -1,     /* bad sizes, pointers, blank, beam, chunk or dtype */
  PCTC_ELABEL = -2,     /* a target label is outside [0, V) or equals blank */
  PCTC_ELENGTH = -3,    /* some T_n < 1 or U_n < 0 */
  PCTC_EWORKSPACE = -4, /* workspace_bytes smaller than pctc_workspace_size() */
  PCTC_EHIP = -5,       /* a HIP runtime call failed; see pctc_last_error() */
  PCTC_ETOOLONG = -6    /* a target longer than PCTC_MAX_TARGET labels */
} pctc_status;

/* Per-utterance status codes written to utt_status. */
enum { PCTC_UTT_OK = 0, PCTC_UTT_NOT_ALIGNABLE = 1, PCTC_UTT_NONFINITE = 2 };

/* Limits of this implementation. */
#define PCTC_MAX_TARGET 1023    /* U_n (2U_n+1 lattice states per frame held in one wavefront) */
#define PCTC_MAX_VOCAB 524288   /* V (the largest vocabulary the parity tests cover) */
#define PCTC_MAX_DIM 1048576    /* D (the products address 256-row tiles with 32-bit byte offsets) */

/* Bytes of workspace pruned_ctc_fwd_bwd needs for this batch.  Depends on N, the frame
 * and target lengths, D, the chunk width and (through the union bitmap, the vocabulary
 * chunk and the remap table) linearly on V only in a V-sized int32 table; the dominant
 * terms scale with M*K (selected log-probabilities and their gradient), the lattice
 * size sum_n T_n (2U_n+1), and M*chunk (one recomputed bf16 gradient chunk).
 * chunk: vocabulary columns recomputed per backward step; 0 selects the default (about
 * 512 MiB of recomputed gradient, see pctc_bwd_chunk); a chunk wider than V rounded up to a
 * multiple of 256 is taken as that width.  Returns 0 if the arguments are
 * invalid.  The same workspace serves pruned_ctc_fwd_bwd_ex. */
size_t pctc_workspace_size(pctc_dtype dtype, int32_t N, const int32_t* input_lengths,
                           const int32_t* target_lengths, int32_t D, int32_t V, float beam,
                           int32_t chunk);

/* The same for a call of a stated kind: flags 0 is pctc_workspace_size; PCTC_WS_NO_DW sizes it
 * for calls with dW == NULL (a frozen head, as in the paper's LLM-CTC runs), which need no room
 * for the union classes' weight-gradient slices.  Returns 0 for unknown flags. */
#define PCTC_WS_NO_DW 1
size_t pctc_workspace_size_ex(pctc_dtype dtype, int32_t N, const int32_t* input_lengths,
                              const int32_t* target_lengths, int32_t D, int32_t V, float beam,
                              int32_t chunk, int32_t flags);

/* Vocabulary columns of the first backward chunk whose gradient rows the normaliser pass of a
 * fused call of this shape writes itself (Eq. vjp: the dense part -g_m p_v(m) of that chunk is
 * exp(z) times a per-frame factor formed once lambda is known, so the chunk needs no recomputed
 * logits), or 0 when every chunk is recomputed.  Applies to bf16 calls with a second stream
 * (pruned_ctc_fwd_bwd, pruned_ctc_fwd_bwd_ex without bias and db) asking for dH or dW; at run
 * time the call still recomputes the chunk when some frame's lambda lies outside [-40, 60]
 * (where exp(z) in bf16 would overflow or lose mass).  Arguments as pctc_workspace_size_ex; 0
 * on invalid arguments.  Host only; no device work. */
int32_t pctc_normaliser_chunk_columns(pctc_dtype dtype, int32_t N, const int32_t* input_lengths,
                                      const int32_t* target_lengths, int32_t D, int32_t V, float beam,
                                      int32_t chunk, int32_t flags);

/* Forward and backward pass of Pruned CTC (Algorithm 1).
 *
 * H        [M, D] row-major, dtype; M = sum input_lengths.  D must be a multiple of 8 and at
 *          most PCTC_MAX_DIM.
 * W        [V, D] row-major, dtype (the head weight; a bias: pruned_ctc_fwd_bwd_ex).
 *          H and W are read in 16-byte pieces: both pointers must be 16-byte aligned
 *          (PCTC_EINVAL otherwise; every entry point below that takes H or W checks this).
 * targets  device int32 [sum target_lengths]: concatenated blank-free labels.
 * input_lengths, target_lengths: HOST int32 [N].
 * blank    the blank class id, 0 <= blank < V.  It becomes column 0 of the union.
 * beam     alignment beam in natural-log units (Sec. 3.3, App. B.3).  A finite value
 *          >= 0 prunes every lattice arc whose best complete alignment scores more than
 *          beam below the best alignment; +INF or a negative value keeps all alignments
 *          (unpruned reduced CTC).  NaN is PCTC_EINVAL.  Tolerance: the rule is evaluated
 *          in float32 and arcs up to 1e-3 nats beyond the beam are kept, so that rounding
 *          never drops the best alignment (at beam 0 the best path is always kept).
 * chunk    vocabulary columns per backward recompute step (0 = the default of
 *          pctc_bwd_chunk; otherwise a positive multiple of 256).
 * loss     device double [1]: sum over utterances of the finite per-utterance losses.
 * loss_per_utt  device double [N] or NULL.
 * utt_status    device int32 [N] or NULL (PCTC_UTT_* codes).
 * dH       device float [M, D] or NULL (not computed).
 * dW       device float [V, D] or NULL (frozen head: not computed).
 * workspace/workspace_bytes: device scratch of at least pctc_workspace_size() bytes,
 *          256-byte aligned.  Contents on entry are ignored.
 * stream   hipStream_t to run on (NULL = the default stream).
 *
 * The call is asynchronous except for one stream synchronisation at the end, which
 * reads back the device-side label check.  Host-checkable errors return before any
 * work is queued.  On any error the outputs are unspecified.
 */
int32_t pruned_ctc_fwd_bwd(pctc_dtype dtype, const void* H, int32_t D, const void* W, int32_t V,
                           const int32_t* targets, const int32_t* input_lengths,
                           const int32_t* target_lengths, int32_t N, int32_t blank, float beam,
                           int32_t chunk, double* loss, double* loss_per_utt, int32_t* utt_status,
                           float* dH, float* dW, void* workspace, size_t workspace_bytes,
                           void* stream);

/* The same with a head bias, per-utterance loss weights and the bias gradient (Sec. 2:
 * the head is the affine map (W, b); Algorithm 1 writes the rows of dL/dW and dL/db per
 * vocabulary chunk; the LLM-CTC blank offset eta enters as b = b_pre + eta e_blank, so
 * dL/deta = db[blank]; App. C normalises losses by the batch's target-token count,
 * which is w_n = 1 / sum_n U_n).
 *
 * bias        device float [V] or NULL: logits are H W^T + 1 b^T.
 * utt_weight  device float [N] or NULL (all 1): loss = sum_n w_n L_n over the included
 *             utterances, and dH, dW, db are the gradients of that sum.  loss_per_utt
 *             still receives the unweighted L_n.  A zero weight excludes the utterance
 *             from the gradients.
 * db          device float [V] or NULL: dL/db, the column sums of dL/dZ (bf16 path:
 *             the sums of the bf16-rounded dL/dZ that the dH and dW products also use).
 * Every other argument is as for pruned_ctc_fwd_bwd, which equals this call with three
 * NULLs. */
int32_t pruned_ctc_fwd_bwd_ex(pctc_dtype dtype, const void* H, int32_t D, const void* W,
                              const float* bias, int32_t V, const int32_t* targets,
                              const int32_t* input_lengths, const int32_t* target_lengths,
                              int32_t N, int32_t blank, float beam, int32_t chunk,
                              const float* utt_weight, double* loss, double* loss_per_utt,
                              int32_t* utt_status, float* dH, float* dW, float* db,
                              void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): pruned_ctc_fwd_bwd_ex without a
 * workspace argument.  Its scratch is a file-scope device array of
 * PCTC_NOALLOC_SCRATCH_MIB MiB inside the library, one copy per device, held from the
 * first call on a device until the process ends; the call allocates nothing (no
 * hipMalloc, no events, no second stream: every step runs on `stream` in Algorithm 1's
 * order).  Inputs and outputs are the caller's, as for pruned_ctc_fwd_bwd_ex.
 * chunk 0 selects the widest backward chunk whose layout fits the scratch (results then
 * differ from pruned_ctc_fwd_bwd_ex's only by summation order); a batch that needs more
 * scratch than the array holds even at the narrowest chunk, or an explicit chunk that does
 * not fit, returns PCTC_EWORKSPACE before any work is queued (pctc_last_error() states
 * both sizes).  Every call on a device shares that device's array and leaves its contents
 * behind (nothing is assumed zero on entry): calls that overlap in time on one device,
 * from any streams or threads, race and give unspecified results.  Synchronises `stream`
 * once at the end, like pruned_ctc_fwd_bwd_ex. */
#define PCTC_NOALLOC_SCRATCH_MIB 256
size_t pctc_noalloc_scratch_bytes(void);
int32_t pruned_ctc_fwd_bwd_noalloc(pctc_dtype dtype, const void* H, int32_t D, const void* W,
                                   const float* bias, int32_t V, const int32_t* targets,
                                   const int32_t* input_lengths, const int32_t* target_lengths,
                                   int32_t N, int32_t blank, float beam, int32_t chunk,
                                   const float* utt_weight, double* loss, double* loss_per_utt,
                                   int32_t* utt_status, float* dH, float* dW, float* db,
                                   void* stream);

/* Human-readable text of a status code, and the text of the last HIP error seen by the
 * calling thread. */
const char* pctc_status_string(int32_t status);
const char* pctc_last_error(void);

/* ----------------------------------------------------------------------------------
 * Stage entry points.  Each runs one stage of Algorithm 1 on caller buffers, so that a
 * stage can be checked on its own.  All run asynchronously on `stream` unless stated.
 * ---------------------------------------------------------------------------------- */

/* Union subset and relabelling (Sec. 3.2 "Reformulation"; Algorithm 1).  The selected
 * classes are blank followed by the distinct target labels in increasing id order.
 * remap    device int32 [V]: index of class v in the union, or -1.
 * u_ids    device int32 [1 + sum target_lengths]: the union; entries past K unspecified.
 * y_rel    device int32 [sum target_lengths]: targets relabelled by their union index.
 * K        device int32 [1]: the union size.
 * err      device int32 [1]: set non-zero if a label is out of range or equals blank.
 * scratch  device, pctc_union_scratch_bytes(V) bytes (a membership bitmap and a count per
 *          block of 2048 classes; contents on entry ignored).
 * Synchronous (reads err back); returns PCTC_ELABEL on a bad label. */
size_t pctc_union_scratch_bytes(int32_t V);
int32_t pctc_union_remap(const int32_t* targets, int32_t total_targets, int32_t blank, int32_t V,
                         int32_t* remap, int32_t* u_ids, int32_t* y_rel, int32_t* K, int32_t* err,
                         void* scratch, void* stream);

/* Normaliser and selected-class log-probabilities (Eq. lognorm; Algorithm 1):
 * lam[m] = log sum_v exp (H W^T)[m, v] in double; S[m, j] = float(Z[m, u_ids[j]] - lam[m])
 * with the subtraction in double and one rounding to float, for j < K (K read from the
 * device scalar), S row pitch ldS >= K_max.  K_max bounds K (1 + total targets).
 * partials: device scratch of pctc_lse_scratch_bytes(M, D) bytes (8 bytes per frame and
 * vocabulary partition: 256 partitions, 1024 for D >= 2048; independent of V).  Returns 0
 * for M < 0 or D <= 0. */
size_t pctc_lse_scratch_bytes(int32_t M, int32_t D);
int32_t pctc_lse_select(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W,
                        int32_t V, const int32_t* u_ids, const int32_t* K, int32_t K_max,
                        double* lam, float* S, int32_t ldS, void* partials, void* stream);

/* Alignment stage (Sec. 3.3; Algorithm 1 lattice, total scores and gradient): from the
 * selected log-probabilities S [M, ldS] (column 0 = blank) and the relabelled targets,
 * per-utterance losses, statuses, G = dL/dS [M, ldS] (-occupancy summed over the states
 * of each class; zero on excluded utterances and unused columns) and g[m] = sum_j G[m, j].
 * keep_mask (optional, device uint8 [sum_n T_n (2U_n+1)], utterance-major, frame-major):
 * bit0 self arc kept, bit1 arc from s-1 kept, bit2 arc from s-2 kept (bit0 at t = 0:
 * start arc), bit3 final arc kept (last frame only).  NULL when not wanted.
 * dp_scratch: device scratch of pctc_dp_scratch_bytes() bytes. */
size_t pctc_dp_scratch_bytes(int32_t N, const int32_t* input_lengths, const int32_t* target_lengths,
                             float beam);
int32_t pctc_ctc_dp(const float* S, int32_t ldS, int32_t K_max, const int32_t* y_rel,
                    const int32_t* input_lengths, const int32_t* target_lengths, int32_t N,
                    float beam, double* loss_per_utt, int32_t* utt_status, float* G, float* g,
                    uint8_t* keep_mask, void* dp_scratch, void* stream);

/* Greedy (best-path) recognition with the same head (the inference side of the method):
 * per frame the class with the largest logit H W^T + b over the full vocabulary (the
 * smallest class id on exact ties), computed on the vocabulary-tiled matrix-core products
 * without storing the logits; then per utterance the CTC collapse (Sec. 3.1): repeated ids
 * merged, blanks removed.
 * H, D, W, bias, V, blank: as for pruned_ctc_fwd_bwd_ex.  input_lengths: HOST int32 [N].
 * ids: device int32 [M] or NULL: the per-frame argmax.  tokens: device int32 [M]: utterance
 * n's sequence occupies [o_n, o_n + token_lengths[n]) with o_n = sum of the earlier
 * input_lengths; the rest is unspecified.  token_lengths: device int32 [N].
 * workspace: pctc_greedy_workspace_size(N, M, D) bytes, 256-byte aligned (independent of V).
 * NaN logits give an unspecified id for their frame.  Synchronises the stream. */
size_t pctc_greedy_workspace_size(int32_t N, int32_t M, int32_t D);
int32_t pctc_greedy_decode(pctc_dtype dtype, const void* H, int32_t D, const void* W,
                           const float* bias, int32_t V, const int32_t* input_lengths, int32_t N,
                           int32_t blank, int32_t* ids, int32_t* tokens, int32_t* token_lengths,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Discarded posterior mass (App. B.3): for each beam b and utterance n,
 *   delta[b * N + n] = 1 - (sum over the alignments that the beam retains) /
 *                          (sum over all valid alignments),
 * both sums of prod_t p_{pi_t}(t) on the same scores S (layout as for pctc_ctc_dp).  The
 * retained set is the one pruned_ctc_fwd_bwd uses at that beam.  Two forward recursions run
 * in lockstep in double precision with one shared per-frame scale; the per-frame emission
 * factors are formed once in float and used by both, so their rounding cancels in the
 * ratio.  Estimates carry the rounding of both sums (they are not certified bounds) and
 * can be slightly negative.  Utterances that are not alignable get NaN.
 * beams: HOST float [nbeams], each finite and >= 0.  delta: device double [nbeams * N].
 * dp_scratch: pctc_discarded_mass_scratch_bytes() bytes.  Synchronises the stream. */
size_t pctc_discarded_mass_scratch_bytes(int32_t N, const int32_t* input_lengths,
                                         const int32_t* target_lengths);
int32_t pctc_discarded_mass(const float* S, int32_t ldS, int32_t K_max, const int32_t* y_rel,
                            const int32_t* input_lengths, const int32_t* target_lengths, int32_t N,
                            const float* beams, int32_t nbeams, double* delta, void* dp_scratch,
                            void* stream);

/* Recomputed backward (Eq. vjp; Algorithm 1 backward loop): for each vocabulary chunk,
 * dZ = scatter_U(G) - g p with p = exp(H W^T - lam) recomputed, then dH = sum dZ W and
 * dW = dZ^T H (rows of frames with g[m] == 0 contribute nothing).  remap: device
 * int32 [V] from pctc_union_remap.  dH and/or dW may be NULL.
 * bwd_scratch: device scratch of pctc_bwd_scratch_bytes() bytes (ldG: the row pitch of G,
 * at least the union size K). */
size_t pctc_bwd_scratch_bytes(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t ldG,
                              int32_t chunk);
/* Vocabulary columns per backward step that a call with this chunk argument uses (0 picks
 * the default: the fewest chunks that keep the recomputed gradient within about 512 MiB,
 * made equal and rounded up to a multiple of 256).  Returns 0 for invalid arguments. */
int32_t pctc_bwd_chunk(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t chunk);
int32_t pctc_head_bwd(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W,
                      int32_t V, const double* lam, const float* G, int32_t ldG, const float* g,
                      const int32_t* remap, int32_t chunk, float* dH, float* dW, void* bwd_scratch,
                      void* stream);

/* Grouped logits for a stock CTC (Sec. 3.2, Eq. grouped; Prop. 1; Eq. offsupport).  The
 * selected classes u_ids (device int32 [K], distinct, in [0, V); e.g. the union of
 * pctc_union_remap with its size read back) keep their own logits and every other class is
 * merged into one "other" class whose logit is the log-sum-exp of the remaining logits.  The
 * log softmax of these K + 1 grouped logits is exported; an unmodified CTC loss over K + 1
 * classes (blank at the blank's position in u_ids, targets relabelled by their position) on
 * it gives the full-vocabulary CTC loss exactly, and its gradient maps back to dH, dW, db.
 *
 * pctc_grouped_logprobs: logp device float [M, K + 1] row-major:
 *   logp[m, j] = Z[m, u_ids[j]] - lam[m] (j < K),
 *   logp[m, K] = log sum over the classes not in u_ids of exp Z[m, v] - lam[m]
 *   (-inf when u_ids covers the vocabulary), Z = H W^T + bias (bias device float [V] or NULL);
 * lam device double [M]: the full log normaliser, needed by the backward.  One pass over
 * the vocabulary.
 * pctc_grouped_backward: dlogp device float [M, K + 1]: dL/dlogp as a CTC implementation
 * returns it (either the true gradient or one with a multiple of exp(logp) added per row:
 * the result is the same).  logp and lam as the forward returned them.  dH [M, D], dW [V, D],
 * db [V] device float, each may be NULL; they are overwritten.  chunk: as for
 * pctc_head_bwd (0 = default).
 * workspace: pctc_grouped_workspace_size(dtype, M, D, V, K, chunk) bytes, 256-byte aligned
 * (the forward needs no more than the size for chunk 0).  Both calls check u_ids first and
 * return PCTC_ELABEL for an id outside [0, V) or given twice; both synchronise the stream. */
size_t pctc_grouped_workspace_size(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t K,
                                   int32_t chunk);
int32_t pctc_grouped_logprobs(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W,
                              const float* bias, int32_t V, const int32_t* u_ids, int32_t K,
                              float* logp, double* lam, void* workspace, size_t workspace_bytes,
                              void* stream);
int32_t pctc_grouped_backward(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W,
                              const float* bias, int32_t V, const int32_t* u_ids, int32_t K,
                              const float* logp, const double* lam, const float* dlogp,
                              int32_t chunk, float* dH, float* dW, float* db, void* workspace,
                              size_t workspace_bytes, void* stream);

/* ----------------------------------------------------------------------------------
 * Kernel timing for benchmarks.  When enabled, every kernel the library launches is
 * bracketed by HIP events on its stream; the times are accumulated per kernel name when
 * they are read (pctc_prof_count / pctc_prof_get, which wait for the recorded launches to
 * finish) or reset, so that timing adds no per-call host work beyond the event records.
 * ---------------------------------------------------------------------------------- */
void pctc_prof_enable(int32_t on);
/* Restrict timing to the kernels of one name (as reported by pctc_prof_get); NULL or ""
 * times every kernel again.  Each timed launch is bracketed by two events, which keeps the
 * launches around it from overlapping, so timing fewer kinds disturbs the run less. */
void pctc_prof_select(const char* name);
void pctc_prof_reset(void);
int32_t pctc_prof_count(void);
/* Name, total milliseconds and launch count of the i-th kernel kind; returns 0 if i is
 * out of range. */
int32_t pctc_prof_get(int32_t i, const char** name, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* PRUNEDCTC_H */
