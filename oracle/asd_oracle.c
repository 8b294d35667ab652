/*
 * CPU oracle for the verifier of Approximate Speculative Decoding (ASD).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * includes this file; only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark load it.  It shares no code, header or helper
 * with the HIP path.
 *
 * It is a plain, slow, sequential statement of what the verifier computes:
 *
 *   1. For every target logit row z_i the greedy token y*_i = argmax_v z_i(v)
 *      (Sec. 3.1, Eq. 1).  Ties go to the lowest index.
 *   2. For every draft block, its accepted length.  When the request's total
 *      budget B is zero, the paper dispatches to exact greedy verification,
 *      so the length is the strict prefix of Eq. 2.  Otherwise it is the
 *      largest t in 0..K whose prefix x_{1:t} is feasible (Eq. 12), every
 *      candidate t being checked directly against the definitions: the
 *      mismatch indicator d_i (Eq. 5), the regret r_i (Eq. 3), the remaining
 *      length q_i (Eq. 6), the running totals C_t and N_t (Eq. 8), the budget
 *      (Eq. 9), the cap (Eq. 10) and the gate at every mismatch i <= t
 *      (Eqs. 7 and 11).  Then the ledger update s' = s + C_a (Sec. 3.3,
 *      Eq. 13) and the emitted token y*_{a+1}: the recovery token when a < K,
 *      the bonus token y*_{K+1} when a = K (Sec. 3.3).
 *   3. The opportunity statistic of Eq. 4 (Sec. 3.1) from the per-row outputs.
 *   4. The commit of the emitted tokens that keeps the caches on the emitted
 *      sequence (Sec. 3.3).
 *   Equations are numbered in the order the paper numbers them: 1 target rows,
 *   2 strict prefix, 3 local regret, 4 opportunity, 5 mismatch indicator,
 *   6 remaining length, 7 normalized gate, 8 cumulative state, 9 budget,
 *   10 block cap, 11 gate for every mismatch, 12 longest feasible prefix,
 *   13 ledger update, 14 feasibility mask.
 *
 * Readings taken where the paper does not fix a detail (each is listed, with
 * its reason, in the design notes of the repository):
 *   - argmax order: numeric order of the values, with -0 and +0 equal.  A
 *     NaN of either sign ranks above +inf and all NaNs rank equal, so the
 *     first NaN of a row is its argmax (the convention of numpy.argmax).
 *     Lowest index wins among equal values.
 *   - r_i is one binary32 subtraction of the binary32 values (a bf16 logit is
 *     widened to binary32 exactly first); C_i is a binary32 running sum from
 *     +0 in position order; s' is one binary32 addition s + C_a, and s is left
 *     untouched when no mismatch was accepted.
 *   - gate (Eqs. 7, 11) r_i / q_i <= g is decided as the real-number inequality
 *     r_i <= g * q_i, evaluated in binary64 (exact for q_i < 2^29).  A variant
 *     selected by a flag gates on the raw regret instead, r_i <= g (q_i read
 *     as 1); the normalized gate is the default.
 *   - budget (Eq. 9) C_t <= B - s is decided as fl32(s + C_t) <= B, which
 *     makes the paper's s' <= B hold exactly after rounding.
 *   - block cap (Eq. 10) N_t <= M.
 *   - the B = 0 dispatch tests the total budget B (so -0 counts as zero).
 *   - a draft id outside [0, V) is a mismatch that is never feasible, with
 *     r = +inf.
 *   - the bonus row's draft entry is ignored.  The per-row regret output is
 *     written for the rows of verified requests only: r_i at draft rows, +0
 *     at the bonus row.
 *   - a negative K is read as K = 0 (the request owns one row, its bonus
 *     row) and is reported in the error word.  A request whose rows do not
 *     fit in [0, total_rows) is not verified: a = 0, next token = -1, state
 *     untouched, also reported in the error word.
 *
 * Parity unpinned: none of the functions below is unpinned; the seeded input
 * generators live elsewhere and are described with the workloads.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

/* flags of oracle_verify_ex */
#define ORACLE_RAW_GATE 1u          /* gate on r_i <= g instead of r_i / q_i <= g */

/* bits of the error word of oracle_verify_ex */
#define ORACLE_ERR_NEGATIVE_K 1u    /* some K_i < 0, read as 0 */
#define ORACLE_ERR_ROWS 2u          /* some request's rows outside [0, total_rows) */

/* ---------------------------------------------------------------- values */

/* A bf16 value is the upper half of a binary32 value: widening is exact. */
static float bf16_bits_to_float(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static float logit_at(const void *logits, int dtype, int64_t vocab,
                      int64_t row, int64_t col)
{
    int64_t k = row * vocab + col;
    if (dtype == ORACLE_BF16)
        return bf16_bits_to_float(((const uint16_t *)logits)[k]);
    return ((const float *)logits)[k];
}

/*
 * Does value a rank strictly above value b?
 * Two numbers: the ordinary IEEE comparison a > b (so -0 and +0 tie).  A NaN
 * of either sign ranks above every number, and no NaN ranks above another.
 */
int oracle_ranks_above(float a, float b)
{
    if (isnan(b))
        return 0;
    if (isnan(a))
        return 1;
    return a > b;
}

/* Eq. 1: y*_i = argmax_v z_i(v); the first (lowest) index among equals. */
int64_t oracle_row_argmax(const void *logits, int dtype, int64_t vocab,
                          int64_t row)
{
    int64_t best = 0;
    for (int64_t v = 1; v < vocab; ++v)
        if (oracle_ranks_above(logit_at(logits, dtype, vocab, row, v),
                               logit_at(logits, dtype, vocab, row, best)))
            best = v;
    return best;
}

/* Eq. 1 for rows [0, total_rows): out[row] = y*_row. */
void oracle_argmax_rows(const void *logits, int dtype, int64_t vocab,
                        int64_t total_rows, int32_t *out)
{
    for (int64_t row = 0; row < total_rows; ++row)
        out[row] = (int32_t)oracle_row_argmax(logits, dtype, vocab, row);
}

/* ------------------------------------------------- accepted length (Sec. 3.2) */

/*
 * Is the prefix x_{1:t} feasible (Sec. 3.2, Eqs. 9-11)?
 *
 * C_t and N_t are the sums of Eq. 8 over positions 1..t, formed here from
 * scratch for this t: C_t in binary32 from +0, adding d_i r_i in position
 * order (a match adds nothing, whatever its r_i), N_t as an integer count.
 * The gate (Eqs. 7 and 11) must hold at every mismatch i <= t; it is decided
 * as r_i <= g q_i in binary64, with q_i = K - i + 1 (Eq. 6), or q_i = 1 for
 * the raw-gate variant.  A draft id outside the vocabulary is a mismatch that
 * no prefix may contain.  A prefix that holds no mismatch spends nothing and
 * is feasible (the first term of Eq. 14); one that holds a mismatch must also
 * meet the budget (Eq. 9, decided as fl32(s + C_t) <= B) and the cap N_t <= M
 * (Eq. 10).  d, x_valid and r are indexed from 0 (position i is entry i - 1).
 */
static int prefix_is_feasible(int32_t t, int32_t K, const uint8_t *d,
                              const uint8_t *x_valid, const float *r,
                              float B_total, float s, float g, int32_t M,
                              int raw_gate)
{
    float C_t = 0.0f;
    int64_t N_t = 0;
    for (int32_t i = 1; i <= t; ++i) {
        double q_i;
        if (!d[i - 1])
            continue;
        if (!x_valid[i - 1])
            return 0;
        q_i = raw_gate ? 1.0 : (double)(K - i + 1);
        if (!((double)r[i - 1] <= (double)g * q_i))
            return 0;
        C_t = C_t + r[i - 1];
        N_t = N_t + 1;
    }
    if (N_t == 0)
        return 1;
    return (float)(s + C_t) <= B_total && N_t <= (int64_t)M;
}

/*
 * The accepted length of one draft block of length K >= 0, with its emitted
 * token and ledger update.
 *
 * Inputs:
 *   x[0..K-1]        the draft block x_1..x_K (token ids)
 *   x_valid[0..K-1]  1 if x_i is a vocabulary id (0 <= x_i < V), else 0
 *   y[0..K]          the target greedy tokens y*_1..y*_{K+1}
 *   z_y[0..K-1]      the target logits z_i(y*_i)
 *   z_x[0..K-1]      the target logits z_i(x_i) (not read where x_valid == 0)
 *   B_total, *s      the request's ledger (B, s); *s is updated in place
 *   g, M             the local gate and the per-block exception cap
 *   raw_gate         nonzero: gate on r_i <= g (q_i read as 1)
 * Outputs: *a_out (accepted length), *next_out (the emitted token y*_{a+1});
 * r_out[0..K-1] receives r_i when non-NULL.
 *
 * B = 0 is exact greedy verification with the ledger unchanged: a is the
 * largest t with x_i = y*_i for every i <= t (Eq. 2).  Otherwise a is the
 * largest feasible t (Eq. 12), and s' = s + C_a (Eq. 13) when the accepted
 * prefix holds a mismatch (s is left untouched when it holds none).
 */
void oracle_block(int32_t K, const int32_t *x, const uint8_t *x_valid,
                  const int32_t *y, const float *z_y, const float *z_x,
                  float B_total, float *s, float g, int32_t M, int raw_gate,
                  int32_t *a_out, int32_t *next_out, float *r_out)
{
    size_t n = (size_t)(K > 0 ? K : 1);
    uint8_t *d = (uint8_t *)malloc(n);
    float *r = (float *)malloc(sizeof(float) * n);
    int32_t a = 0;

    for (int32_t i = 1; i <= K; ++i) {
        /* Eq. 5 on token ids; a non-vocabulary id equals no greedy token */
        d[i - 1] = (x_valid[i - 1] && x[i - 1] == y[i - 1]) ? 0 : 1;
        /* Eq. 3: one binary32 subtraction; +inf for a non-vocabulary id */
        r[i - 1] = x_valid[i - 1] ? z_y[i - 1] - z_x[i - 1] : INFINITY;
        if (r_out)
            r_out[i - 1] = r[i - 1];
    }

    if (B_total == 0.0f) {
        /* Eq. 2: the largest t whose drafts all equal the greedy tokens */
        for (int32_t t = 0; t <= K; ++t) {
            int all_equal = 1;
            for (int32_t i = 1; i <= t; ++i)
                if (d[i - 1])
                    all_equal = 0;
            if (all_equal)
                a = t;
        }
    } else {
        float C_a = 0.0f;
        int64_t N_a = 0;
        /* Eq. 12: the largest feasible t */
        for (int32_t t = 0; t <= K; ++t)
            if (prefix_is_feasible(t, K, d, x_valid, r, B_total, *s, g, M,
                                   raw_gate))
                a = t;
        /* Eq. 13 with the totals of Eq. 8 over the accepted prefix */
        for (int32_t i = 1; i <= a; ++i)
            if (d[i - 1]) {
                C_a = C_a + r[i - 1];
                N_a = N_a + 1;
            }
        if (N_a > 0)
            *s = *s + C_a;
    }

    *a_out = a;
    *next_out = y[a];   /* y*_{a+1}: recovery if a < K, bonus if a = K */
    free(d);
    free(r);
}

/* ------------------------------------------------------- whole verifier call */

/*
 * The whole verification call over a batch, on host arrays.
 *
 * logits        [total_rows, vocab] row-major; binary32 (dtype 0) or bf16 bit
 *               patterns (dtype 1)
 * draft         [total_rows]; row o_i + p - 1 holds draft x_p of request i;
 *               the bonus row's entry is ignored
 * block_lens    [num_requests] K_i
 * row_offsets   [num_requests] first row o_i of each request, or NULL for the
 *               packed layout o_i = sum_{j<i} (max(K_j, 0) + 1)
 * tau           [num_requests] local gate g of each request
 * exc_cap       [num_requests] block cap M of each request
 * budget        [num_requests][2] = (B, s); s updated in place
 * out_accept_len, out_next_token [num_requests]
 * out_argmax    [total_rows] or NULL: y* of every row
 * out_regret    [total_rows] or NULL: r of every draft row of a verified
 *               request, +0 for its bonus row; other rows are not written
 * flags         0, or ORACLE_RAW_GATE
 * error_word    NULL, or ORed with ORACLE_ERR_* for the requests that have them
 * Returns 0, or 1 for an argument the call cannot work with.
 */
int oracle_verify_ex(const void *logits, int dtype, int64_t vocab,
                     int32_t num_requests, int64_t total_rows,
                     const int32_t *draft, const int32_t *block_lens,
                     const int64_t *row_offsets, const float *tau,
                     const int32_t *exc_cap, float *budget,
                     int32_t *out_accept_len, int32_t *out_next_token,
                     int32_t *out_argmax, float *out_regret,
                     uint32_t flags, uint32_t *error_word)
{
    int32_t *y_all;
    int64_t packed_offset = 0;

    if (vocab < 1 || num_requests < 0 || total_rows < 0 ||
        (dtype != ORACLE_F32 && dtype != ORACLE_BF16))
        return 1;

    y_all = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total_rows > 0 ? total_rows : 1));
    for (int64_t row = 0; row < total_rows; ++row) {
        y_all[row] = (int32_t)oracle_row_argmax(logits, dtype, vocab, row);
        if (out_argmax)
            out_argmax[row] = y_all[row];
    }

    for (int32_t i = 0; i < num_requests; ++i) {
        int32_t K = block_lens[i] > 0 ? block_lens[i] : 0;
        int64_t o = row_offsets ? row_offsets[i] : packed_offset;
        packed_offset += (int64_t)K + 1;

        if (block_lens[i] < 0 && error_word)
            *error_word |= ORACLE_ERR_NEGATIVE_K;
        if (o < 0 || o + (int64_t)K >= total_rows) {
            out_accept_len[i] = 0;
            out_next_token[i] = -1;
            if (error_word)
                *error_word |= ORACLE_ERR_ROWS;
            continue;
        }

        {
            int32_t *x = (int32_t *)malloc(sizeof(int32_t) * (size_t)(K > 0 ? K : 1));
            uint8_t *x_valid = (uint8_t *)malloc((size_t)(K > 0 ? K : 1));
            float *z_y = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
            float *z_x = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
            float *r = (float *)malloc(sizeof(float) * (size_t)(K > 0 ? K : 1));
            const int32_t *y = y_all + o;
            int32_t a = 0, next = -1;
            float s = budget[2 * i + 1];

            for (int32_t p = 0; p < K; ++p) {
                int64_t row = o + p;
                x[p] = draft[row];
                x_valid[p] = (x[p] >= 0 && (int64_t)x[p] < vocab) ? 1 : 0;
                z_y[p] = logit_at(logits, dtype, vocab, row, y[p]);
                z_x[p] = x_valid[p] ? logit_at(logits, dtype, vocab, row, x[p]) : 0.0f;
            }

            oracle_block(K, x, x_valid, y, z_y, z_x, budget[2 * i], &s,
                         tau[i], exc_cap[i], (flags & ORACLE_RAW_GATE) != 0,
                         &a, &next, r);

            budget[2 * i + 1] = s;
            out_accept_len[i] = a;
            out_next_token[i] = next;
            if (out_regret) {
                for (int32_t p = 0; p < K; ++p)
                    out_regret[o + p] = r[p];
                out_regret[o + K] = 0.0f;
            }
            free(x);
            free(x_valid);
            free(z_y);
            free(z_x);
            free(r);
        }
    }

    free(y_all);
    return 0;
}

/* oracle_verify_ex with the normalized gate and no error word. */
int oracle_verify(const void *logits, int dtype, int64_t vocab,
                  int32_t num_requests, int64_t total_rows,
                  const int32_t *draft, const int32_t *block_lens,
                  const int64_t *row_offsets, const float *tau,
                  const int32_t *exc_cap, float *budget,
                  int32_t *out_accept_len, int32_t *out_next_token,
                  int32_t *out_argmax, float *out_regret)
{
    return oracle_verify_ex(logits, dtype, vocab, num_requests, total_rows,
                            draft, block_lens, row_offsets, tau, exc_cap,
                            budget, out_accept_len, out_next_token,
                            out_argmax, out_regret, 0u, NULL);
}

/* -------------------------------------------- opportunity statistic (Eq. 4) */

/*
 * Counts of the opportunity statistic of Sec. 3.1, Eq. 4, over the blocks of one
 * batch, accumulated into counts[a * num_ps + b] (numerator of
 * Omega(taus[a], ps[b])) and *mismatches (|M|).  Omega = numerator / |M|.
 *
 * M is the set of draft positions i (1-based, 1 <= i <= K) with x_i != y*_i
 * (Eq. 5; a draft id outside [0, V) is a mismatch).  A mismatch contributes to
 * (tau, p) when r_i <= tau, i + p <= K, and x_l = y*_l for every l in
 * i+1 .. i+p.  y* and r are the per-row argmax and regret of a verifier call
 * on the same batch (its out_argmax / out_regret).  A negative K is read as 0
 * (no draft positions); requests whose rows do not fit in [0, total_rows) are
 * not evaluated.
 */
void oracle_opportunity(const int32_t *draft, const int32_t *row_argmax,
                        const float *row_regret, int64_t vocab,
                        int32_t num_requests, int64_t total_rows,
                        const int32_t *block_lens, const int64_t *row_offsets,
                        const float *taus, int32_t num_taus,
                        const int32_t *ps, int32_t num_ps,
                        uint64_t *counts, uint64_t *mismatches)
{
    int64_t packed_offset = 0;
    for (int32_t req = 0; req < num_requests; ++req) {
        int32_t K = block_lens[req] > 0 ? block_lens[req] : 0;
        int64_t o = row_offsets ? row_offsets[req] : packed_offset;
        packed_offset += (int64_t)K + 1;
        if (o < 0 || o + (int64_t)K >= total_rows)
            continue;
        for (int32_t i = 1; i <= K; ++i) {
            int64_t row = o + i - 1;
            int32_t x = draft[row];
            int is_mismatch = !(x >= 0 && (int64_t)x < vocab) || x != row_argmax[row];
            if (!is_mismatch)
                continue;
            *mismatches += 1;
            for (int32_t a = 0; a < num_taus; ++a) {
                if (!(row_regret[row] <= taus[a]))
                    continue;
                for (int32_t b = 0; b < num_ps; ++b) {
                    int32_t p = ps[b];
                    int all_greedy = 1;
                    if (!((int64_t)i + p <= (int64_t)K))
                        continue;
                    for (int32_t l = i + 1; l <= i + p; ++l) {
                        int64_t lrow = o + l - 1;
                        if (draft[lrow] != row_argmax[lrow]) {
                            all_greedy = 0;
                            break;
                        }
                    }
                    if (all_greedy)
                        counts[(int64_t)a * num_ps + b] += 1;
                }
            }
        }
    }
}

/* ------------------------------------------------------- commit (Sec. 3.3) */

/*
 * The commit that follows verification (Sec. 3.3): request i emits its
 * accepted drafts x_1..x_a followed by y*_{a+1} (Algorithm 1's return), and
 * its committed sequence -- the length that the target and draft caches keep
 * -- advances along exactly those a + 1 tokens.
 *
 * tokens     [num_requests][capacity] committed tokens of each request
 * seq_len    [num_requests] committed length, advanced in place by a + 1
 * committed  [num_requests] or NULL: tokens committed this round (a + 1), or 0
 * A negative K is read as 0, as the verifier reads it.  A request whose rows
 * do not fit in [0, total_rows), with next_token < 0 (not verified), with a
 * outside [0, K], with seq_len < 0, or whose a + 1 tokens do not fit in
 * [seq_len, capacity), commits nothing.
 */
void oracle_commit(const int32_t *draft, const int32_t *block_lens,
                   const int64_t *row_offsets, int32_t num_requests,
                   int64_t total_rows,
                   const int32_t *accept_len, const int32_t *next_token,
                   int32_t *tokens, int64_t capacity, int64_t *seq_len,
                   int32_t *committed)
{
    int64_t packed_offset = 0;
    for (int32_t i = 0; i < num_requests; ++i) {
        int32_t K = block_lens[i] > 0 ? block_lens[i] : 0;
        int64_t o = row_offsets ? row_offsets[i] : packed_offset;
        int32_t a = accept_len[i];
        int64_t L = seq_len[i];
        packed_offset += (int64_t)K + 1;
        if (committed)
            committed[i] = 0;
        if (o < 0 || o + (int64_t)K >= total_rows)
            continue;                          /* rows of a request asd_verify skips */
        if (next_token[i] < 0 || L < 0 || a < 0 || a > K || L + a + 1 > capacity)
            continue;
        for (int32_t p = 0; p < a; ++p)
            tokens[(int64_t)i * capacity + L + p] = draft[o + p];
        tokens[(int64_t)i * capacity + L + a] = next_token[i];
        seq_len[i] = L + a + 1;
        if (committed)
            committed[i] = a + 1;
    }
}
