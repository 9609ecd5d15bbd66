/*
 * doloss.h -- C ABI of the DO-loss hot path on MI355X (gfx950).
 *
 * DO-loss ("Function Over Form: Distributional Orthogonalization in
 * Mixture-of-Experts with Replica Expert Mechanism", arXiv 2609.32398)
 * records, for every expert, which tokens of a batch routed to it (its binary
 * load signature) and penalises overlap between experts through the pairwise
 * Hamming distances of those signatures.  This library computes, on one GPU:
 *
 *   1. router Top-K over a token x expert score matrix          (Sec. 3.1.1, Eq. 1)
 *   2. the per-expert N-bit load signatures F_i                  (Sec. 3.1.1)
 *   3. the E x E matrix G_ij = ||F_i - F_j||_1                    (Sec. 3.1.3, Eq. 6)
 *   4. the loss sum_{i != j} G_ij^2 with mean / variance of the
 *      off-diagonal distances                                   (Sec. 3.1.1, Eq. 3; App. C.1)
 *
 * Notation: the paper's m tokens / n experts / K choices are N / E / k here.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument is DEVICE memory of the current HIP device unless
 *   stated otherwise; the caller owns it.  Only do_stream_create allocates.
 * - Calls are asynchronous on `stream` (0 = the null stream).  Results are
 *   valid once the caller synchronises that stream.
 * - Every argument is validated on the host before anything is launched; on
 *   error nothing is enqueued and a do_status other than DO_OK is returned.
 *   do_last_error() gives a message for the calling thread's last error.
 * - Layouts (all row-major, little-endian):
 *     scores  [L][N][E]  fp32 or bf16 (raw bf16 bit patterns)
 *     bits    [L][U][E][8]  uint64 signature words, U = ceil(N / 512) units of
 *                        512 tokens (unit-major).  Word w (tokens 64w .. 64w +
 *                        63) of expert e is element [w / 8][e][w % 8] of its
 *                        layer; token t is bit (t % 64) of word t / 64 (least
 *                        significant bit first); bits past N in word
 *                        ceil(N/64) - 1 are zero.  A layer is E * Wp words,
 *                        Wp = 8 * U ("padded words per expert"); the words
 *                        past ceil(N/64) of the last unit are neither written
 *                        nor read.  One unit of every expert is 64 * E
 *                        contiguous bytes, which the Top-K kernel writes at
 *                        once (Sec. 3.1.1 defines F_i as N bits per expert;
 *                        the tiling is this library's).
 *     D       [L][E][E]  uint32, symmetric, zero diagonal
 *     out     [L]        do_loss_result
 * - Ranking rule for Top-K (the paper gives none; this is the library's reading):
 *   larger score first; equal scores go to the lower expert index; -0.0 and
 *   +0.0 are equal; NaN ranks below every number (including -inf) and all NaNs
 *   are equal.  Scores are ranked exactly as given: no gating is applied.
 * - Limits: 1 <= E <= 1024, 1 <= k <= E, 1 <= N < 2^32, 1 <= L <= 65535 and
 *   E*(E-1)*N^2 < 2^64 (so the sum of squares is exact in 64 bits).
 *   The fast path needs 16-byte aligned scores with E*sizeof(score) a multiple
 *   of 16, E <= 256 and k <= 8; other valid shapes take a slower exact path.
 */
#ifndef DOLOSS_H
#define DOLOSS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DO_OK = 0,
  DO_ERR_INVALID_ARG = 1,       /* null/misaligned pointer, size or range out of limits */
  DO_ERR_UNSUPPORTED_DTYPE = 2, /* dtype is not DO_F32 or DO_BF16 */
  DO_ERR_CAPACITY = 3,          /* a stream append would exceed the history capacity */
  DO_ERR_OVERFLOW = 4,          /* E*(E-1)*N^2 >= 2^64 or N >= 2^32 */
  DO_ERR_HIP = 5,               /* the HIP runtime reported an error */
  DO_ERR_NONFINITE = 6          /* a score is NaN (only with DO_OPT_CHECK_FINITE on) */
} do_status;

typedef enum { DO_F32 = 0, DO_BF16 = 1 } do_dtype;

/* Per-layer result of the loss (device memory, 40 bytes). */
typedef struct {
  uint64_t sum;   /* exact sum over i != j of D_ij (Eq. 2: equals 2*N*k*(E-k)) */
  uint64_t sumsq; /* exact sum over i != j of D_ij^2 (Eq. 3); do_loss saturates it at
                     2^64 - 1 when the sum does not fit (never for distances of signatures) */
  double loss;    /* Eq. 3 as fp64: L_origin_DO = sum_{i != j} ||F_i - F_j||_1^2 (the
                     exact integer sum, rounded; within 2 ulp when sumsq saturates) */
  double mean;    /* sum / (E*(E-1)) */
  double var;     /* population variance of the E*(E-1) off-diagonal D_ij (App. C.1) */
} do_loss_result;

/*
 * Steps 1-2 (Sec. 3.1.1, Eq. 1): Top-k of every token's scores and the packed
 * load signatures.
 *   scores  [L][N][E] device, dtype `dtype`
 *   bits    [L][U][E][8] device (signature layout above); the words of
 *           tokens 0 .. N-1 are overwritten
 */
do_status do_topk_signature(const void* scores, do_dtype dtype, int64_t N, int32_t E, int32_t k, int32_t L,
                            uint64_t* bits, hipStream_t stream);

/*
 * Step 3 (Sec. 3.1.3, Eq. 6 magnitude term; App. C.3 identity): the Hamming
 * distance matrix of existing signatures, computed as
 * D_ij = c_ii + c_jj - 2 c_ij with c_ij = popcount(F_i AND F_j).
 *   bits  [L][U][E][8] device (signature layout); bits past N in the last
 *         word must be zero (else the result is undefined)
 *   D     [L][E][E] device, fully overwritten
 */
do_status do_pairwise_hamming(const uint64_t* bits, int64_t N, int32_t E, int32_t L, uint32_t* D,
                              hipStream_t stream);

/*
 * Step 4 (Sec. 3.1.1, Eq. 3; App. C.1): loss and off-diagonal statistics of
 * any E x E distance matrices (the diagonal is ignored; symmetry is not
 * assumed).  For E = 1 every field is zero.  Any uint32 entries are accepted:
 * the sums are accumulated exactly (the sum of squares in 128 bits, so it
 * never wraps); `sum` is exact, `sumsq` is exact below 2^64 and saturated at
 * 2^64 - 1 above, and loss, mean and var are the exact sums rounded to fp64.
 *   D    [L][E][E] device
 *   out  [L] device
 */
do_status do_loss(const uint32_t* D, int32_t E, int32_t L, do_loss_result* out, hipStream_t stream);

/*
 * Steps 1-4 in a single pass over the scores: signatures stay on chip and are
 * written out only if `bits` is not NULL; the co-occurrence counts are
 * accumulated in `D` itself, which is then turned into distances and reduced
 * to the loss.  Results are identical to do_topk_signature +
 * do_pairwise_hamming + do_loss.
 *   bits  [L][U][E][8] device; may be NULL only for E <= 256 (wider E
 *         re-reads the stored signatures for the Gram: DO_ERR_INVALID_ARG)
 *   D     [L][E][E] device, fully overwritten
 *   out   [L] device
 */
do_status do_fused(const void* scores, do_dtype dtype, int64_t N, int32_t E, int32_t k, int32_t L, uint64_t* bits,
                   uint32_t* D, do_loss_result* out, hipStream_t stream);

/*
 * Surrogate DO-loss (Sec. 3.1.3, Eq. 6-7) and its gradient with respect to the
 * routing probabilities, with the magnitude G and the assignments F detached
 * (stop-gradient, Sec. 3.1.2):
 *   C_ij = sum_t p_it (f_it - f_jt)
 *   loss = scale / (N^2 k) * sum_{i,j} G_ij C_ij
 *   grad_it = dloss/dp_it = scale / (N^2 k) * sum_j G_ij (f_it - f_jt)
 * G is `D`; scale is 1 on one device (Sec. 3.1.4: with G summed over R
 * data-parallel ranks, scale = 1/R gives the averaged magnitude of Eq. 8).
 *   p     [L][N][E] device, fp32 or bf16 routing probabilities (as given),
 *         aligned to two elements
 *   bits  [L][U][E][8] device: the tokens' signatures (f_it = bit)
 *   D     [L][E][E] device
 *   loss  [L] device doubles, overwritten
 *   grad  nullable, [L][N][E] device fp32 (8-byte aligned), overwritten
 * Any set of bits is accepted as a signature; words in which some token has
 * more than 8 set bits (not a top-k with k <= 8) take a slower path.  k only
 * enters the normalisation.
 * Limits: E <= 256 and (E-1)*N < 2^31 (DO_ERR_OVERFLOW otherwise).  The loss
 * is accumulated in fp64 with atomic adds, so its last bits may differ
 * between runs; the gradient is deterministic.
 */
do_status do_surrogate(const void* p, do_dtype dtype, int64_t N, int32_t E, int32_t k, int32_t L, const uint64_t* bits,
                       const uint32_t* D, double scale, double* loss, float* grad, hipStream_t stream);

/* Per-layer load statistics (device memory, 32 bytes). */
typedef struct {
  uint64_t total;    /* sum_i n_i: N*k for Top-K signatures */
  uint32_t max_load; /* max_i n_i */
  uint32_t min_load; /* min_i n_i */
  double lbl;        /* Local-LBL (Sec. 4.2) sum_i f_i P_i, f_i = n_i / (N k), P_i = (1/N) sum_t p_it; 0 without p */
  double maxvio;     /* App. E: max over ranks r of |L_r / tau - 1|, tau the mean rank load; 0 if tau is 0 */
} do_load_stats_result;

/*
 * Load statistics of signatures: the per-expert loads n_i = ||F_i||_1 (the
 * diagonal of the co-occurrence counts, App. C.3), the Local-LBL balance loss
 * of Sec. 4.2 and the MaxVio imbalance of App. E for a placement of the
 * experts on ranks (L_r = sum of the loads of the experts on rank r).
 *   bits         device signatures in the signature layout, the layers
 *                E * ld words apart; ld = padded words per expert, a
 *                multiple of 8 of at least 8 * ceil(N/512) (0 means that
 *                minimum; a stream history passes
 *                do_stream_words_per_expert); bits past N in the last word
 *                must be zero
 *   p            nullable, [L][N][E] device routing probabilities (fp32 or
 *                bf16, aligned to the element); NULL leaves lbl at 0
 *   expert_rank  nullable HOST array [E] of ranks in [0, R), read during the
 *                call; NULL places every expert on its own rank (R = E)
 *   loads        [L][E] device uint32, overwritten
 *   out          [L] device, overwritten
 * Limits as for do_topk_signature; 1 <= R <= 1024.  lbl is accumulated in
 * fp64 with atomic adds, so its last bits may differ between runs; the other
 * fields are exact and deterministic.
 */
do_status do_load_stats(const uint64_t* bits, int64_t N, int64_t ld, int32_t E, int32_t k, int32_t L, const void* p,
                        do_dtype dtype, const int32_t* expert_rank, int32_t R, uint32_t* loads,
                        do_load_stats_result* out, hipStream_t stream);

/*
 * Streaming global-batch history (Sec. 3.1.4: distances over a batch wider
 * than one micro-batch; App. F.2, Table 4: G over gradient-accumulated
 * micro-batches).  A handle owns a
 * signature history of `capacity_tokens` bits per expert and the running
 * co-occurrence counts.  Each append ranks one micro-batch and appends its
 * signatures after the tokens already held (concatenation), so that after any
 * sequence of appends the distances equal those of one batch made of all
 * appended tokens in order.
 */
typedef struct do_stream_s do_stream;

/* Allocates the history (E x 8 * ceil(capacity/512) words, the signature
 * layout of one layer) and the counters on the
 * current device and zeroes them (synchronously).  *out receives the handle,
 * or NULL on failure (DO_ERR_HIP when a device or host allocation fails). */
do_status do_stream_create(int32_t E, int32_t k, int64_t capacity_tokens, do_stream** out);

/* Appends n_tokens >= 0 tokens of scores [n_tokens][E] (device).  Fails with
 * DO_ERR_CAPACITY, leaving the handle unchanged, if the history would overflow.
 * With n_tokens = 0 nothing is read or launched, and scores may be NULL. */
do_status do_stream_append(do_stream* h, const void* scores, do_dtype dtype, int64_t n_tokens, hipStream_t stream);

/* Appends `count` (1..64) micro-batches of n_tokens_each tokens in one launch.
 * `scores` is a HOST array of `count` device pointers, read during the call;
 * with n_tokens_each = 0 the device pointers may be NULL. */
do_status do_stream_append_many(do_stream* h, const void* const* scores, do_dtype dtype, int64_t n_tokens_each,
                                int32_t count, hipStream_t stream);

/* Writes the distances D [E][E] and the loss `out` [1] (both device) of all
 * tokens appended so far (since the last reset).  The history is not
 * modified, and a repeated finalize gives the same result.  Calls on one
 * handle must not overlap in time (use one stream, or synchronise): the
 * handle's counters are moved into its running totals here. */
do_status do_stream_finalize(do_stream* h, uint32_t* D, do_loss_result* out, hipStream_t stream);

/* Empties the history: the next append starts at token 0 and the next
 * finalize counts only tokens appended after the reset.  Bits of earlier
 * tokens are not erased here: the next appends overwrite or clear the words
 * they use (see do_stream_bits).  Enqueues at most one small fill, and none
 * when the previous call on the handle was a finalize. */
do_status do_stream_reset(do_stream* h, hipStream_t stream);

/* Frees the handle after synchronising the device it was created on (the
 * current device is restored).  NULL is accepted. */
do_status do_stream_destroy(do_stream* h);

/* Device pointer to the history: one layer in the signature layout with
 * do_stream_words_per_expert(h) padded words per expert (E times that in
 * total).  Words 0 .. ceil(do_stream_tokens(h) / 64) - 1 of every expert hold
 * the signatures of the appended tokens, with zero bits past the last token;
 * words after them are zero until the first reset and unspecified after it
 * (they may keep bits of tokens appended before the reset).  A prefix of the
 * history is itself a valid signature array for N = do_stream_tokens(h). */
const uint64_t* do_stream_bits(const do_stream* h);
int64_t do_stream_tokens(const do_stream* h);
int64_t do_stream_words_per_expert(const do_stream* h);

/*
 * Benchmark hook: the next do_fused / do_topk_signature / do_stream_append* /
 * do_global_batch_noalloc call made by this thread binds `start` and `stop`
 * to the dispatch of its main score-streaming kernel (hipExtLaunchKernel), so
 * that hipEventElapsedTime gives that kernel's own run time.  do_surrogate
 * records them on its stream right before and after its main kernel.
 * One-shot; both are events of the current device created by the caller
 * (either may be NULL).  Pass NULLs to cancel.
 */
do_status do_profile_next(hipEvent_t start, hipEvent_t stop);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the result
 * of do_stream_create + do_stream_append_many + do_stream_finalize on one
 * global batch of `count` micro-batches, in one call that allocates nothing.
 * The caller owns the history; the running co-occurrence counts and the
 * finalize's partial sums live in a static device buffer of the library
 * (256 KiB + 32 bytes, held on every GPU the library runs on until the
 * process ends), which every call clears before use.
 *   scores         HOST array of `count` (1..64) device pointers, each
 *                  [n_tokens_each][E], read during the call
 *   hist           [U][E][8] device, U = ceil(count * n_tokens_each / 512):
 *                  the signatures of the tokens in order (signature layout,
 *                  as do_stream_bits), overwritten
 *   D, out         as do_stream_finalize
 * Limits: E <= 256 (DO_ERR_INVALID_ARG otherwise), 1 <= k <= E,
 * n_tokens_each >= 1, count * n_tokens_each < 2^32 and the limits of
 * do_topk_signature.  All calls on one GPU share the buffer: calls that may
 * overlap in time (on different streams, or from several threads without
 * ordering) race and give wrong results.
 */
do_status do_global_batch_noalloc(const void* const* scores, do_dtype dtype, int64_t n_tokens_each, int32_t count,
                                  int32_t E, int32_t k, uint64_t* hist, uint32_t* D, do_loss_result* out,
                                  hipStream_t stream);

/*
 * Replica Expert Mechanism (REM) scheduling on the device.  One replica
 * placement (Alg. 1) or one token route (Alg. 2): `tokens` tokens of expert
 * `expert` go from its home rank `src_rank` to its replica on `dst_rank`
 * (24 bytes).
 */
typedef struct {
  int32_t expert;
  int32_t src_rank;
  int32_t dst_rank;
  int32_t reserved; /* 0 */
  int64_t tokens;
} do_rem_move;

/*
 * REM global-batch replica allocation (Sec. 3.2.1, Benefit Score; App. B,
 * Alg. 1), one independent problem per layer.  With tau the mean rank load,
 * the Benefit Score of expert e (home rank r_s) for a replica on r_r is
 *   min(tau - L_r, T_e, L_s - tau)      if L_r < tau < L_s
 *   min(floor((L_s - L_r) / 2), T_e)    if L_r >= tau and L_s > L_r
 *   -1                                  otherwise,
 * the two differences with tau rounded down to whole tokens.  While some rank
 * has fewer than D replicas, the least-loaded such rank (lowest index on
 * ties) receives a replica of the expert with the largest score among the
 * experts homed elsewhere (lowest expert index on ties), and L_r, L_s and T_e
 * move by that score; a largest score <= 0 stops the allocation.
 *   rank_load      nullable, [L][R] device: historical loads L_r; NULL takes
 *                  L_r = sum of expert_tokens over the experts homed on r
 *   expert_tokens  [L][E] device: volumes T_e (e.g. the loads of do_load_stats)
 *   expert_rank    HOST array [E] of home ranks in [0, R), read during the call
 *   moves          [L][R*D] device: the first n_moves[l] entries of layer l
 *                  are the placements in order
 *   n_moves        [L] device; -1 when a load or volume of layer l is negative
 *                  or >= 2^40 (then nothing else of that layer is written)
 *   load_out       nullable, [L][R] device: L_r after the last placement
 *   tokens_out     nullable, [L][E] device: T_e after the last placement
 * Limits: 1 <= E <= 1024, 1 <= R <= 1024, D >= 1 with R*D <= 4096,
 * 1 <= L <= 65535.  Integer results are exact and deterministic.
 */
do_status do_rem_allocate(const int64_t* rank_load, const int64_t* expert_tokens, const int32_t* expert_rank,
                          int32_t E, int32_t R, int32_t D, int32_t L, do_rem_move* moves, int32_t* n_moves,
                          int64_t* load_out, int64_t* tokens_out, hipStream_t stream);

/*
 * REM micro-batch token dispatching (App. B, Alg. 2), one problem per layer.
 * The queue depth Q_r starts as the sum of this micro-batch's volumes T_e
 * over the experts homed on r; tau is their mean.  D passes: each orders the
 * ranks by Q_r ascending (ties by index, no re-sorting within the pass) and,
 * for every rank holding a replica, routes the Benefit Score's number of
 * tokens (with L = Q) through the best of its replicas (earliest in the
 * assignment on ties); a score <= 0 routes nothing.
 *   replicas       [L][replica_stride] device: the assignment, e.g. the moves
 *                  of do_rem_allocate (expert, src_rank = its home rank,
 *                  dst_rank = the replica's rank; `tokens` is ignored)
 *   n_replicas     [L] device: valid entries per layer (a negative count, or
 *                  a replica whose src_rank is not its expert's home rank,
 *                  fails the layer as below)
 *   expert_tokens  [L][E] device: this micro-batch's volumes T_e
 *   expert_rank    HOST array [E] of home ranks in [0, R), read during the call
 *   routes         [L][R*D] device: the first n_routes[l] entries are the routes
 *   n_routes       [L] device; -1 for invalid input of layer l (volumes outside
 *                  [0, 2^40), a bad replica or count)
 *   queue_out      nullable, [L][R] device: Q_r after the last pass
 *   tokens_out     nullable, [L][E] device: T_e after the last pass
 * Limits: as do_rem_allocate, and replica_stride <= 4096.
 */
do_status do_rem_dispatch(const do_rem_move* replicas, const int32_t* n_replicas, int32_t replica_stride,
                          const int64_t* expert_tokens, const int32_t* expert_rank, int32_t E, int32_t R, int32_t D,
                          int32_t L, do_rem_move* routes, int32_t* n_routes, int64_t* queue_out, int64_t* tokens_out,
                          hipStream_t stream);

/*
 * Process-wide options (they take effect at the next call; calls already
 * enqueued are unaffected).  Returns DO_ERR_INVALID_ARG for an unknown option
 * or a value out of range.  The first two override internal choices that
 * never change any result, for tests and benchmarks:
 *   DO_OPT_SCHEDULE      unit schedule of the score pass: -1 (default)
 *                        measures both candidates on the first launches of
 *                        every shape of at least 512 Ki tokens (1,024 units)
 *                        and keeps the faster; 0 fixes the XCD-partitioned
 *                        schedule; 1 fixes one contiguous range of work units
 *                        per block.
 *   DO_OPT_GRAM          co-occurrence Gram for E <= 256: 0 (default) the fp4
 *                        MFMA Gram, 1 the VALU popcount Gram.
 * The third adds an input check.  NaN scores have a defined rank (below -inf,
 * equal to each other), so results are defined without it:
 *   DO_OPT_CHECK_FINITE  0 (default) off; 1: do_topk_signature, do_fused,
 *                        do_stream_append and do_stream_append_many first scan
 *                        their scores for NaN (+-inf are ordinary values), wait
 *                        for the scan on the caller's stream, and return
 *                        DO_ERR_NONFINITE without writing anything (the
 *                        stream handle is unchanged) if one is found.  Such a
 *                        call synchronises the stream, so under stream capture
 *                        it returns DO_ERR_INVALID_ARG.  Check-mode calls of
 *                        one process are serialised by a host lock.
 *                        do_global_batch_noalloc, whose callers cannot wait,
 *                        does not scan.
 */
typedef enum { DO_OPT_SCHEDULE = 0, DO_OPT_GRAM = 1, DO_OPT_CHECK_FINITE = 2 } do_option;
do_status do_set_option(do_option opt, int32_t value);

/* Text of a status code, and the message of the calling thread's last error. */
const char* do_status_string(do_status s);
const char* do_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int32_t do_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DOLOSS_H */
