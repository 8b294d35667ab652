/*
 * asd.h -- C ABI of the MI355X (gfx950) verifier of Approximate Speculative
 * Decoding (ASD).
 *
 * One call verifies a batch of draft blocks against their teacher-forced
 * target logits (Sec. 3.1, Eq. 1: row i of a block holds z_i =
 * Target(h_0, x_{<i}); a block of K drafts has K + 1 rows, the last one giving
 * the bonus token).  For every request it returns the longest feasible prefix
 * of Algorithm 1 (Sec. 3.2, Eq. 12), the recovery or bonus token, and the
 * updated regret ledger (Sec. 3.3, Eq. 13).
 *
 * Equations are numbered as in the paper: 1 target rows, 2 strict prefix,
 * 3 local regret, 5 mismatch indicator, 6 remaining length q_i = K - i + 1,
 * 7 normalized gate r_i / q_i <= g, 8 cumulative regret C_t and count N_t,
 * 9 budget C_t <= B - s, 10 block cap N_t <= M, 11 gate at every accepted
 * mismatch, 12 longest feasible prefix, 13 ledger update s' = s + C_a,
 * 14 feasibility mask.
 *
 * All arrays are caller-owned device memory unless stated otherwise.  Every
 * call is asynchronous on the given HIP stream (NULL = the null stream): it
 * never synchronizes, and its outputs are valid in stream order.
 */
#ifndef ASD_H
#define ASD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of the logits.  A plain 32-bit integer, so that any value a
 * caller passes is well defined; values other than these return ASD_EDTYPE. */
typedef int32_t asd_dtype;
enum {
    ASD_F32 = 0,   /* IEEE binary32 */
    ASD_BF16 = 1   /* bfloat16: the upper 16 bits of a binary32 value */
};

/* Status of a call (a plain 32-bit integer, like asd_dtype). */
typedef int32_t asd_status;
enum {
    ASD_OK = 0,
    ASD_EINVAL = 1,    /* an argument the host can check is invalid; nothing launched */
    ASD_EDTYPE = 2,    /* unknown dtype; nothing launched */
    ASD_ENOMEM = 3,    /* workspace could not be allocated, or too small */
    ASD_EHIP = 4,      /* a HIP runtime call or kernel launch failed */
    ASD_ECAPTURE = 5,  /* the library workspace must grow while the stream is captured */
    ASD_ESCRATCH = 6   /* the call needs more workspace than asd_verify_static's fixed
                          scratch holds; nothing launched */
};

/*
 * Per-request regret ledger (B, s) (Sec. 3.2): total budget B and the regret s
 * already spent by exceptions accepted in earlier rounds.  B = 0 selects exact
 * greedy verification (Algorithm 1, first step; Eq. 2).
 */
typedef struct {
    float total;   /* B */
    float spent;   /* s, updated in place to s' (Eq. 13) */
} asd_budget;

/*
 * asd_verify -- verify a batch of draft blocks (Algorithm 1 on every request).
 *
 * logits          [total_rows, vocab], row-major, dense, dtype elements; the
 *                 base address must be a multiple of the element size.
 * dtype           ASD_F32 or ASD_BF16.
 * vocab           V, 1 <= V < 2^30.
 * num_requests    number of requests (draft blocks) in the batch, >= 0;
 *                 0 returns ASD_OK with nothing launched.
 * total_rows      number of logit rows, num_requests <= total_rows < 2^31.
 * draft_tokens    int32 [total_rows]: row o_i + p - 1 holds draft x_p of
 *                 request i (p = 1..K_i); the entry of each bonus row o_i + K_i
 *                 is ignored.
 * block_lens      int32 [num_requests]: K_i >= 0 (a negative K_i is read as 0
 *                 and reported in the device error word, see asd_device_error).
 * row_offsets     int64 [num_requests]: first row o_i of request i, or NULL for
 *                 the packed layout o_i = sum_{j<i} (max(K_j, 0) + 1).
 * tau             float [num_requests]: the local gate g_i of Eq. 7.
 * exc_cap         int32 [num_requests]: the block cap M_i of Eq. 10
 *                 (INT32_MAX acts as no cap).
 * budget_inout    asd_budget [num_requests]: .total read, .spent read and
 *                 rewritten (left bit-identical when no mismatch is accepted).
 * out_accept_len  int32 [num_requests]: a_i in [0, K_i] (Eq. 12).
 * out_next_token  int32 [num_requests]: y*_{a+1}, the recovery token when
 *                 a_i < K_i and the bonus token y*_{K_i+1} when a_i = K_i.
 * out_argmax      int32 [total_rows] or NULL: y* of every row (Eq. 1), the
 *                 lowest index among equal greatest values.
 * out_regret      float [total_rows] or NULL: for the rows of every verified
 *                 request, r = fl32(z(y*) - z(x)) (Eq. 3) at each draft row
 *                 (+inf for an id outside [0, V)) and +0 at its bonus row.
 *                 Rows outside verified requests are not written.
 * stream          a hipStream_t, or NULL.
 *
 * Semantics (bit-exact with the CPU oracle):
 *  - argmax order: the numeric order with -0 == +0; every NaN, of either sign
 *    and any payload, ranks above +inf and equal to every other NaN, so a
 *    row's first NaN is its argmax (numpy.argmax's convention).  A row whose
 *    greatest logit is NaN has a NaN regret, and a NaN regret never passes
 *    the gate.
 *  - gate r_i <= g_i * q_i is decided exactly (binary64); budget as
 *    fl32(s + C_t) <= B; cap as N_t <= M; C_t is a binary32 running sum in
 *    position order; s' = fl32(s + C_a).
 *  - B == 0 (either sign): exact greedy verification, ledger unchanged.
 *  - a draft id outside [0, V) is a mismatch that is never accepted.
 *  - K_i < 0 is read as K_i = 0: the request's one row is its bonus row,
 *    a_i = 0 and the next token is that row's argmax.
 *  - a request with o_i < 0 or o_i + K_i >= total_rows is not verified:
 *    a_i = 0, next token = -1, ledger untouched.
 *  Both cases also set a bit of the device error word (asd_device_error).
 *
 * Small calls (at most 512 row tiles and 8 requests, the latency-bound
 * regime of single-request decoding) that are not being captured run as one
 * kernel launch instead of two: the last row tile to finish runs the scan.
 * This form needs a zeroed counter, so it runs only with a library workspace
 * (here, asd_verify_ex and asd_verify_commit without a workspace, and
 * asd_verify_static); with a caller's workspace, or during stream capture
 * (where launches are cheap and two kernels are faster), the two-launch form
 * runs.  The results are the same.
 *
 * Outputs must not alias the inputs.  Calls that share the library workspace
 * of one (device, stream) pair are ordered by the stream; calls on different
 * streams use different workspaces.  The first call on a (device, stream)
 * pair, or one that needs a larger workspace, allocates device memory
 * (hipMalloc) and so must not happen during stream capture (ASD_ECAPTURE).
 * A larger workspace is a new buffer of at least twice the size; the buffers
 * it replaces stay allocated until asd_release, so a graph captured with an
 * earlier call stays valid after the workspace grows.
 * Returns ASD_OK once the work is enqueued.
 */
asd_status asd_verify(const void *logits, asd_dtype dtype, int64_t vocab,
                      int32_t num_requests, int64_t total_rows,
                      const int32_t *draft_tokens, const int32_t *block_lens,
                      const int64_t *row_offsets, const float *tau,
                      const int32_t *exc_cap, asd_budget *budget_inout,
                      int32_t *out_accept_len, int32_t *out_next_token,
                      int32_t *out_argmax, float *out_regret, void *stream);

/*
 * asd_workspace_bytes -- device workspace that asd_verify_ws needs for a call
 * of this shape on the current device.  Returns 0 for invalid arguments.
 */
size_t asd_workspace_bytes(asd_dtype dtype, int64_t vocab, int32_t num_requests,
                           int64_t total_rows);

/*
 * asd_verify_ws -- asd_verify with a caller-provided workspace.
 *
 * workspace        device memory of at least asd_workspace_bytes(...) bytes,
 *                  256-byte aligned, with any content: nothing in it is
 *                  carried between calls, so one workspace serves any later
 *                  call that fits, in stream order.  Calls that may overlap
 *                  must use different workspaces.
 * workspace_bytes  its size; too small returns ASD_ENOMEM with nothing launched.
 * Never allocates, so it may be used during stream capture.
 */
asd_status asd_verify_ws(const void *logits, asd_dtype dtype, int64_t vocab,
                         int32_t num_requests, int64_t total_rows,
                         const int32_t *draft_tokens, const int32_t *block_lens,
                         const int64_t *row_offsets, const float *tau,
                         const int32_t *exc_cap, asd_budget *budget_inout,
                         int32_t *out_accept_len, int32_t *out_next_token,
                         int32_t *out_argmax, float *out_regret, void *stream,
                         void *workspace, size_t workspace_bytes);

/* Bytes of the fixed device scratch of asd_verify_static (4 MiB per device). */
#define ASD_STATIC_SCRATCH_BYTES ((size_t)4 << 20)

/*
 * asd_verify_static -- asd_verify that allocates nothing, for callers that
 * cannot allocate device memory: code under stream (graph) capture, tight
 * serving loops, harnesses that forbid hipMalloc.
 *
 * Arguments and outputs are those of asd_verify, with the same results.  The
 * call's workspace is a fixed device array of ASD_STATIC_SCRATCH_BYTES bytes
 * that the library holds on every device it runs on until the process ends;
 * the call never calls hipMalloc or hipFree.  A call whose workspace
 * (asd_workspace_bytes) exceeds that size less 256 bytes returns ASD_ESCRATCH
 * with nothing launched: it needs 8 bytes per request, 8 per row, and 16 per
 * vocabulary split of a row when rows are split (about 500,000 whole rows
 * fit).  Every call on a device shares that device's array, which keeps the
 * last call's contents.  Its first 256 bytes hold the counter of the
 * single-launch form, zero when the library is loaded and left zero by every
 * call; nothing else in it needs to start at zero or is carried from one call
 * to the next.  Calls that may overlap on one device (different streams,
 * or host threads without ordering) race on the array and must not be issued;
 * calls in order on one stream are safe.  The first call on a device looks up
 * the array's address.
 */
asd_status asd_verify_static(const void *logits, asd_dtype dtype, int64_t vocab,
                             int32_t num_requests, int64_t total_rows,
                             const int32_t *draft_tokens, const int32_t *block_lens,
                             const int64_t *row_offsets, const float *tau,
                             const int32_t *exc_cap, asd_budget *budget_inout,
                             int32_t *out_accept_len, int32_t *out_next_token,
                             int32_t *out_argmax, float *out_regret, void *stream);

/* Flags of asd_verify_ex. */
enum {
    ASD_GATE_RAW = 1   /* gate on the raw regret r_i <= g_i instead of Eq. 7's
                          normalized r_i / q_i <= g_i (q_i read as 1) */
};

/*
 * asd_verify_ex -- asd_verify with flags and an optional caller workspace.
 *
 * flags            0 (the paper's gate, Eqs. 7 and 11: identical to asd_verify)
 *                  or ASD_GATE_RAW, a variant that gates every accepted
 *                  mismatch on r_i <= g_i; budget, cap, dispatch and ledger are
 *                  unchanged.  Unknown bits return ASD_EINVAL.
 * workspace        NULL: the library workspace of (device, stream), as for
 *                  asd_verify.  Otherwise as for asd_verify_ws (256-byte
 *                  aligned, workspace_bytes >= asd_workspace_bytes(...)), and
 *                  the call allocates nothing.
 * The other arguments and all outputs are those of asd_verify.
 */
asd_status asd_verify_ex(const void *logits, asd_dtype dtype, int64_t vocab,
                         int32_t num_requests, int64_t total_rows,
                         const int32_t *draft_tokens, const int32_t *block_lens,
                         const int64_t *row_offsets, const float *tau,
                         const int32_t *exc_cap, asd_budget *budget_inout,
                         int32_t *out_accept_len, int32_t *out_next_token,
                         int32_t *out_argmax, float *out_regret, uint32_t flags,
                         void *stream, void *workspace, size_t workspace_bytes);

/* Bits of the device error word. */
enum {
    ASD_DEVERR_NEGATIVE_K = 1,   /* a request had K_i < 0 (read as 0) */
    ASD_DEVERR_ROWS = 2,         /* a request's rows lay outside [0, total_rows)
                                    (not verified, or not committed) */
    ASD_DEVERR_COMMIT = 4        /* a verified request committed nothing: its
                                    tokens did not fit below capacity, seq_len_i
                                    was negative or a_i lay outside [0, K_i] */
};

/*
 * asd_device_error -- read the sticky error word of the current device.
 *
 * The kernels OR ASD_DEVERR_* bits into one word per device when they meet
 * data that has a defined but unusual reading (the calls still complete and
 * return their documented outputs).  The word is shared by every call on the
 * device, from any stream, and keeps its bits until cleared.
 * out_word        host uint32: the word once all work enqueued on `stream` so
 *                 far has completed.
 * clear           nonzero: reset the word to 0 after reading it (in stream
 *                 order; calls on other streams may set bits again at any time).
 * Synchronizes `stream`, so it must not be called during stream capture
 * (ASD_ECAPTURE).  ASD_EINVAL for a NULL out_word.
 */
asd_status asd_device_error(uint32_t *out_word, int32_t clear, void *stream);

/*
 * Vocabulary-sharded (tensor-parallel) verification.  The verifier needs, per
 * row, only the greatest logit, its column and the draft token's logit
 * (Sec. 3.3), so each holder of a column shard can reduce its own columns and
 * only 16 bytes per row need to meet: no K x |V| logit buffer is gathered.
 */

/* One shard's result for one row (16 bytes, 16-byte aligned; contents opaque). */
typedef struct {
    uint32_t opaque[4];
} asd_row_partial;

/*
 * asd_shard_argmax -- the row pass of asd_verify (Eqs. 1 and 3) on one shard.
 *
 * shard_logits    [total_rows, shard_vocab], row-major, dense, dtype elements:
 *                 row r holds columns [vocab_offset, vocab_offset + shard_vocab)
 *                 of the full vocabulary of row r.  Base address a multiple of
 *                 the element size.
 * vocab           V, the full vocabulary size: vocab_offset >= 0,
 *                 shard_vocab >= 1, vocab_offset + shard_vocab <= V < 2^30.
 * total_rows      rows, 1 <= total_rows < 2^31.
 * draft_tokens    int32 [total_rows], global token ids as for asd_verify.
 * out_partials    asd_row_partial [total_rows]: the shard's greatest value and
 *                 its global column (argmax order of asd_verify), and the draft
 *                 token's logit when its id lies in the shard.
 * Allocates nothing and uses no workspace.  Asynchronous on `stream`.
 */
asd_status asd_shard_argmax(const void *shard_logits, asd_dtype dtype, int64_t shard_vocab,
                            int64_t vocab_offset, int64_t vocab, int64_t total_rows,
                            const int32_t *draft_tokens, asd_row_partial *out_partials,
                            void *stream);

/*
 * asd_verify_partials -- finish asd_verify from the partials of all shards.
 *
 * partials        asd_row_partial [num_shards][total_rows] (shard-major), shard k
 *                 written by asd_shard_argmax for columns
 *                 [k * shard_vocab, min((k + 1) * shard_vocab, V)).  With one
 *                 shard per GPU they are gathered to one device first.
 * num_shards      1 <= num_shards <= 4096, and the shards cover V exactly:
 *                 (num_shards - 1) * shard_vocab < V <= num_shards * shard_vocab.
 * The other arguments and every output are those of asd_verify, and the results
 * are bit-identical to asd_verify on the unsharded rows.  When row_offsets is
 * NULL and num_requests > 1024 the packed offsets are computed into the
 * library workspace of this (device, stream) pair (allocated on first use, see
 * asd_verify); otherwise nothing is allocated.
 */
asd_status asd_verify_partials(const asd_row_partial *partials, int32_t num_shards,
                               int64_t shard_vocab, int64_t vocab, int32_t num_requests,
                               int64_t total_rows, const int32_t *draft_tokens,
                               const int32_t *block_lens, const int64_t *row_offsets,
                               const float *tau, const int32_t *exc_cap,
                               asd_budget *budget_inout, int32_t *out_accept_len,
                               int32_t *out_next_token, int32_t *out_argmax,
                               float *out_regret, void *stream);

/*
 * asd_opportunity -- accumulate the opportunity statistic of Sec. 3.1, Eq. 4:
 *   Omega(tau, p) = (1 / |M|) * #{ mismatch (x, i) in M : r_i <= tau,
 *                    i + p <= K, and x_l = y*_l for l = i+1 .. i+p },
 * the share of draft-target mismatches that have low regret and are followed
 * by p target-greedy drafts, over the blocks of one verified batch.
 *
 * draft_tokens, block_lens, row_offsets, num_requests, total_rows, vocab
 *                 as for asd_verify (the batch that was verified); row_offsets
 *                 may be NULL (packed layout) for any number of requests.
 * row_argmax      int32 [total_rows]: the out_argmax of asd_verify on the batch.
 * row_regret      float [total_rows]: the out_regret of asd_verify on the batch.
 * taus            float [num_taus] (raw regret thresholds); ps int32 [num_ps],
 *                 p >= 0; 1 <= num_taus * num_ps <= 1024.
 * counts          uint64 [num_taus][num_ps]: count of contributing mismatches,
 *                 added to in place (the numerator of Omega(taus[a], ps[b])).
 * mismatches      uint64 [1]: |M|, added to in place.
 * A draft id outside [0, V) is a mismatch (its regret is +inf).  Requests that
 * asd_verify does not verify are skipped.  Allocates nothing; asynchronous.
 */
asd_status asd_opportunity(const int32_t *draft_tokens, const int32_t *row_argmax,
                           const float *row_regret, int64_t vocab, int32_t num_requests,
                           int64_t total_rows, const int32_t *block_lens,
                           const int64_t *row_offsets, const float *taus, int32_t num_taus,
                           const int32_t *ps, int32_t num_ps, uint64_t *counts,
                           uint64_t *mismatches, void *stream);

/*
 * asd_commit -- the commit that follows verification (Sec. 3.3): request i
 * emits its accepted drafts x_1..x_a followed by y*_{a+1} (Algorithm 1's
 * return), and its committed sequence -- the extent its target and draft caches
 * keep -- advances along exactly those a + 1 tokens.
 *
 * draft_tokens, block_lens, row_offsets, num_requests, total_rows
 *                 as for the asd_verify call (row_offsets may be NULL, the packed
 *                 layout, for any number of requests).
 * accept_len, next_token   the outputs of that call.
 * tokens          int32 [num_requests][capacity]: entries
 *                 [seq_len_i, seq_len_i + a_i + 1) of row i are written.
 * seq_len         int64 [num_requests]: committed lengths, advanced in place.
 * out_committed   int32 [num_requests] or NULL: a_i + 1, or 0 for a request that
 *                 commits nothing.
 * A negative K_i is read as 0, as asd_verify reads it.  A request commits
 * nothing when its rows do not fit in [0, total_rows), its next_token is
 * negative (not verified), a_i lies outside [0, K_i], seq_len_i is negative, or
 * the a_i + 1 tokens do not fit below capacity; each case but a negative
 * next_token sets a bit of the device error word.  Allocates nothing;
 * asynchronous on `stream`, so it can follow asd_verify in one captured graph.
 */
asd_status asd_commit(const int32_t *draft_tokens, const int32_t *block_lens,
                      const int64_t *row_offsets, int32_t num_requests, int64_t total_rows,
                      const int32_t *accept_len, const int32_t *next_token, int32_t *tokens,
                      int64_t capacity, int64_t *seq_len, int32_t *out_committed, void *stream);

/*
 * asd_verify_commit -- asd_verify followed, in the same pass, by the commit of
 * asd_commit (Sec. 3.3): after request i's scan its wavefront writes the
 * emitted tokens x_1..x_a, y*_{a+1} and advances its committed length, so a
 * decoding round is one call instead of two.
 *
 * The first fifteen arguments are those of asd_verify (here the packed layout,
 * row_offsets == NULL, has no request limit).  tokens, capacity, seq_len and
 * out_committed are those of asd_commit, with the same rules: a request
 * commits nothing when it is not verified, its a_i + 1 tokens do not fit below
 * capacity, or seq_len_i is negative (the last two set ASD_DEVERR_COMMIT).
 * workspace       NULL: the library workspace of (device, stream), allocated on
 *                 first use and never during stream capture, as for asd_verify.
 *                 Otherwise caller memory of workspace_bytes >=
 *                 asd_workspace_bytes(...) bytes, 256-byte aligned, as for
 *                 asd_verify_ws; the call then allocates nothing.
 * Returns ASD_EINVAL also for capacity < 1, missing tokens or seq_len, or
 * num_requests * capacity overflowing int64.
 */
asd_status asd_verify_commit(const void *logits, asd_dtype dtype, int64_t vocab,
                             int32_t num_requests, int64_t total_rows,
                             const int32_t *draft_tokens, const int32_t *block_lens,
                             const int64_t *row_offsets, const float *tau,
                             const int32_t *exc_cap, asd_budget *budget_inout,
                             int32_t *out_accept_len, int32_t *out_next_token,
                             int32_t *out_argmax, float *out_regret, int32_t *tokens,
                             int64_t capacity, int64_t *seq_len, int32_t *out_committed,
                             void *stream, void *workspace, size_t workspace_bytes);

/*
 * asd_lmhead_verify -- asd_verify with the target's output layer fused in: the
 * logit rows z = H W^T are computed on the matrix cores and reduced at once to
 * each row's greatest logit, its column and the draft token's logit, the only
 * values the verifier needs (Sec. 3.3), so the total_rows x V logits are never
 * written to memory.
 *
 * hidden          bf16 [total_rows, d], row-major: the final hidden state of
 *                 every logit row (teacher-forced rows, Sec. 3.1, Eq. 1).
 * weight          bf16 [vocab, d], row-major: the output (LM-head) weights.
 * d               hidden size, a multiple of 128, 128 <= d <= 2^20.  Both base
 *                 addresses 16-byte aligned.
 * Logits are binary32 sums of the bf16 products (accumulated on the matrix
 * cores in an order of their own); a greatest logit of zero is taken as +0.
 * The other arguments and all outputs are those of asd_verify.  Uses the
 * library workspace of (device, stream) like asd_verify (allocated on first
 * use, never during stream capture).
 */
asd_status asd_lmhead_verify(const void *hidden, const void *weight, int64_t d, int64_t vocab,
                             int32_t num_requests, int64_t total_rows,
                             const int32_t *draft_tokens, const int32_t *block_lens,
                             const int64_t *row_offsets, const float *tau,
                             const int32_t *exc_cap, asd_budget *budget_inout,
                             int32_t *out_accept_len, int32_t *out_next_token,
                             int32_t *out_argmax, float *out_regret, void *stream);

/*
 * asd_row_splits -- the number S of column tiles per row that asd_verify cuts
 * `total_rows` rows of `vocab` elements of `dtype` into on the current device
 * (its row pass runs one workgroup per tile).  0 for arguments asd_verify
 * rejects (dtype, vocab outside [1, 2^30), total_rows outside [1, 2^31)).
 */
int32_t asd_row_splits(asd_dtype dtype, int64_t vocab, int64_t total_rows);

/*
 * asd_row_pass -- a measurement helper: the first stage of asd_verify alone
 * (each row's greatest logit with its column, Eq. 1, and the draft token's
 * logit, Eq. 3), as the same row kernel on the same tile grid that asd_verify
 * launches for these rows: S = asd_row_splits(dtype, vocab, total_rows) tiles
 * per row, one workgroup per tile.  Its duration is that stage's duration
 * inside asd_verify; the only difference is that every tile writes a 16-byte
 * partial (asd_verify writes an 8-byte row record when S = 1).
 *
 * logits, dtype, vocab, total_rows, draft_tokens: as for asd_verify (the rows
 *                 are the rows of a packed or explicit-offset batch alike).
 * out_partials    asd_row_partial [total_rows][S], 16-byte aligned: tile s of
 *                 row r in entry r * S + s, with the layout asd_shard_argmax
 *                 writes (opaque).  The tile whose columns hold the draft
 *                 token holds its logit.
 * Returns ASD_EDTYPE or ASD_EINVAL for the argument errors asd_shard_argmax
 * rejects.  Allocates nothing and uses no workspace.  Asynchronous on `stream`.
 */
asd_status asd_row_pass(const void *logits, asd_dtype dtype, int64_t vocab, int64_t total_rows,
                        const int32_t *draft_tokens, asd_row_partial *out_partials,
                        void *stream);

/*
 * asd_read_probe -- a measurement helper: stream `rows` rows of `row_bytes`
 * bytes from `buf` once, with the access pattern of the verifier's row pass
 * (one 256-thread workgroup per row, 16-byte non-temporal loads, four per lane
 * in flight) and no ranking work.  Its duration is the practical read ceiling
 * that the row pass's bandwidth is compared with.
 *
 * buf             device memory, 16-byte aligned, rows * row_bytes bytes.
 * rows            1 <= rows < 2^31.
 * row_bytes       a multiple of 16, >= 16.
 * out_word        device uint32: written only by a lane whose XOR of the words
 *                 it read equals 0x9e3779b9 (so the loads cannot be elided; a
 *                 caller can plant that value to check that the data is read).
 * Allocates nothing; asynchronous on `stream`.
 */
asd_status asd_read_probe(const void *buf, int64_t rows, int64_t row_bytes, uint32_t *out_word,
                          void *stream);

/*
 * asd_mfma_probe -- a measurement helper: the matrix-core work of
 * asd_lmhead_verify with no memory traffic.  Each of `workgroups` workgroups
 * has the LM-head kernel's shape (eight wavefronts, each with 4 x 2 tiles of
 * 32 x 32 binary32 accumulators) and runs `steps` K steps of 64, i.e. 32
 * v_mfma_f32_32x32x16_bf16 per wavefront per step (2^23 flops per workgroup
 * per step), on operand fragments read once from `operands` and held in
 * registers.  The matrix cores' power depends on their operands, so the caller
 * passes data of the distribution it measures.  Run over an LM-head launch's
 * workgroups and steps (steps = d / 64), its duration is the practical
 * matrix-core ceiling of that launch under the chip's power limit.
 *
 * operands        device bf16 values, 16-byte aligned, `vectors` 16-byte
 *                 vectors (>= 6); thread t of workgroup w reads the 6 vectors
 *                 starting at ((w mod 64) * 512 + t) * 6, modulo `vectors`,
 *                 and forms four fragment sets from them.
 * workgroups      1 <= workgroups < 2^31;  steps >= 1.
 * out             device uint32 [workgroups]: the binary32 bits of the sum of
 *                 the accumulators of each workgroup's thread 0 (with every
 *                 operand 1.0 this is 8192 * steps).
 * Allocates nothing; asynchronous on `stream`.
 */
asd_status asd_mfma_probe(const void *operands, int64_t vectors, int64_t workgroups,
                          int64_t steps, uint32_t *out, void *stream);

/* Human-readable name of a status code (static storage). */
const char *asd_status_string(asd_status status);

/* Library version string (static storage), e.g.
 * "asd-mi355x 0.4.0 gfx950 src 0123456789abcdef": the last word is a hash of
 * the sources the library was built from (comments and whitespace ignored). */
const char *asd_version(void);

/*
 * asd_release -- free every library-owned workspace, including the buffers
 * a workspace outgrew.  The caller must make sure no enqueued call that uses
 * a library workspace is still running (synchronize first), and must not
 * replay a graph captured with such a call afterwards.
 */
asd_status asd_release(void);

#ifdef __cplusplus
}
#endif

#endif /* ASD_H */
