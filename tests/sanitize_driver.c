/*
 * Host sanitizer driver for the CPU oracle and the seeded input generator.
 *
 * Built by tests/test_sanitizers.py with -fsanitize=address,undefined: it runs
 * every oracle entry point and both generator routines on a few hundred small
 * randomized cases, with every buffer allocated to its exact size, so an
 * out-of-bounds access, a use of uninitialized heap memory that reaches a
 * sanitizer check, or undefined arithmetic stops the run.  The cases cover
 * the edge conditions the verifier defines: K = 0 and K < 0, requests whose
 * rows do not fit, explicit offsets with gaps, draft ids outside [0, V),
 * NaN / infinity / signed-zero logits, g in {-1, 0, 0.25, inf, NaN},
 * M in {0, 1, INT32_MAX}, B in {0, -0, tiny, inf} and s = B, with and without
 * the raw-gate flag and the error word.
 */
#include "../oracle/asd_oracle.c"
#include "../workloads/gen.c"

#include <stdio.h>

static uint64_t lcg_state = 0x9E3779B97F4A7C15ull;

static uint32_t next_u32(void)
{
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(lcg_state >> 33);
}

static int64_t pick(int64_t n) { return (int64_t)(next_u32() % (uint32_t)n); }

static void *exact_alloc(size_t bytes)
{
    void *p = malloc(bytes > 0 ? bytes : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static const uint32_t special_bits[] = {
    0x00000000u, 0x80000000u, 0x00000001u, 0x80000001u, 0x3f800000u, 0xbf800000u,
    0x7f800000u, 0xff800000u, 0x7fc00000u, 0xffc00000u, 0x7f800001u, 0xff800001u,
};

static float random_logit(void)
{
    if (pick(4) == 0) {
        uint32_t b = special_bits[pick(sizeof special_bits / sizeof special_bits[0])];
        float f;
        memcpy(&f, &b, sizeof f);
        return f;
    }
    return (float)(pick(13) - 6) / 4.0f;
}

static void run_case(int c)
{
    const int64_t vocabs[] = {1, 2, 5, 64, 300};
    const float taus[] = {-1.0f, 0.0f, 0.25f, 1.0f, INFINITY, NAN};
    const int32_t caps[] = {0, 1, 3, 2147483647};
    const float totals[] = {0.0f, -0.0f, 1e-30f, 0.5f, 2.0f, INFINITY};

    const int64_t vocab = vocabs[pick(5)];
    const int dtype = (int)pick(2);
    const int32_t nreq = (int32_t)pick(7);
    int32_t *lens = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)nreq);
    int64_t rows = 0;
    for (int32_t i = 0; i < nreq; ++i) {
        lens[i] = (int32_t)pick(12) - 1;                 /* -1 .. 10 */
        rows += (lens[i] > 0 ? lens[i] : 0) + 1;
    }
    rows += pick(3);                                     /* sometimes spare rows */
    int64_t *offs = NULL;
    if (pick(2)) {                                       /* explicit offsets, some invalid */
        offs = (int64_t *)exact_alloc(sizeof(int64_t) * (size_t)nreq);
        for (int32_t i = 0; i < nreq; ++i)
            offs[i] = pick(5) == 0 ? -3 : pick(rows + 2);
    }

    const size_t esize = dtype == ORACLE_F32 ? 4 : 2;
    void *logits = exact_alloc(esize * (size_t)(rows * vocab));
    for (int64_t k = 0; k < rows * vocab; ++k) {
        float f = random_logit();
        if (dtype == ORACLE_F32) {
            ((float *)logits)[k] = f;
        } else {
            uint32_t b;
            memcpy(&b, &f, sizeof b);
            ((uint16_t *)logits)[k] = (uint16_t)(b >> 16);
        }
    }
    int32_t *draft = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)rows);
    for (int64_t r = 0; r < rows; ++r)
        draft[r] = (int32_t)(pick(vocab + 4) - 2);
    float *tau = (float *)exact_alloc(sizeof(float) * (size_t)nreq);
    int32_t *cap = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)nreq);
    float *budget = (float *)exact_alloc(sizeof(float) * 2 * (size_t)nreq);
    for (int32_t i = 0; i < nreq; ++i) {
        tau[i] = taus[pick(6)];
        cap[i] = caps[pick(4)];
        budget[2 * i] = totals[pick(6)];
        budget[2 * i + 1] = pick(3) == 0 ? budget[2 * i] : 0.0f;   /* s = B sometimes */
    }
    int32_t *acc = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)nreq);
    int32_t *nxt = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)nreq);
    int32_t *amax = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)rows);
    float *regret = (float *)exact_alloc(sizeof(float) * (size_t)rows);
    for (int64_t r = 0; r < rows; ++r) {
        amax[r] = -1;
        regret[r] = 0.0f;
    }
    const int with_rows = (int)pick(2);
    uint32_t err = 0;
    const uint32_t flags = pick(3) == 0 ? ORACLE_RAW_GATE : 0u;
    if (oracle_verify_ex(logits, dtype, vocab, nreq, rows, draft, lens, offs, tau, cap, budget,
                         acc, nxt, with_rows ? amax : NULL, with_rows ? regret : NULL, flags,
                         pick(2) ? &err : NULL) != 0) {
        fprintf(stderr, "case %d: oracle_verify_ex rejected valid arguments\n", c);
        exit(1);
    }
    if (err & ~(ORACLE_ERR_NEGATIVE_K | ORACLE_ERR_ROWS)) {
        fprintf(stderr, "case %d: unknown error bits %u\n", c, err);
        exit(1);
    }
    for (int32_t i = 0; i < nreq; ++i) {
        if (acc[i] < 0 || (lens[i] >= 0 && acc[i] > lens[i])) {
            fprintf(stderr, "case %d: accept length %d outside [0, K]\n", c, acc[i]);
            exit(1);
        }
    }

    /* opportunity statistic on the per-row outputs */
    oracle_argmax_rows(logits, dtype, vocab, rows, amax);
    const float otau[] = {0.0f, 0.5f, INFINITY};
    const int32_t ops[] = {0, 1, 4};
    uint64_t counts[9] = {0};
    uint64_t mism = 0;
    oracle_opportunity(draft, amax, regret, vocab, nreq, rows, lens, offs, otau, 3, ops, 3,
                       counts, &mism);

    /* commit into exact-size token buffers */
    const int64_t capacity = 1 + pick(20);
    int32_t *tokens = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)(nreq * capacity));
    int64_t *seq_len = (int64_t *)exact_alloc(sizeof(int64_t) * (size_t)nreq);
    int32_t *done = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)nreq);
    for (int64_t k = 0; k < nreq * capacity; ++k)
        tokens[k] = 0;
    for (int32_t i = 0; i < nreq; ++i)
        seq_len[i] = pick(4) == 0 ? -1 : pick(capacity + 2);
    oracle_commit(draft, lens, offs, nreq, rows, acc, nxt, tokens, capacity, seq_len, done);

    /* single-row helpers */
    if (rows > 0) {
        (void)oracle_row_argmax(logits, dtype, vocab, pick(rows));
        (void)oracle_ranks_above(random_logit(), random_logit());
    }

    free(lens); free(offs); free(logits); free(draft); free(tau); free(cap); free(budget);
    free(acc); free(nxt); free(amax); free(regret); free(tokens); free(seq_len); free(done);
}

static void run_generator(int c)
{
    const int64_t vocab = 1 + pick(40);
    const int64_t nrows = 1 + pick(5);
    const int dtype = (int)pick(2);
    const size_t esize = dtype == 0 ? 4 : 2;
    void *rows = exact_alloc(esize * (size_t)(nrows * vocab));
    gen_normal_rows((uint64_t)c, dtype, vocab, pick(100), nrows, 2.0, rows);
    int64_t *peak = (int64_t *)exact_alloc(sizeof(int64_t) * (size_t)nrows);
    float *margin = (float *)exact_alloc(sizeof(float) * (size_t)nrows);
    int32_t *runner = (int32_t *)exact_alloc(sizeof(int32_t) * (size_t)nrows);
    for (int64_t r = 0; r < nrows; ++r) {
        peak[r] = pick(vocab);
        margin[r] = pick(3) == 0 ? 0.0f : 0.5f;
    }
    gen_plant_rows(dtype, vocab, nrows, rows, peak, margin, runner);
    double u[7];
    gen_u01((uint64_t)c, 3, 7, u);
    free(rows); free(peak); free(margin); free(runner);
}

int main(void)
{
    const int cases = 400;
    for (int c = 0; c < cases; ++c) {
        run_case(c);
        if (c % 4 == 0)
            run_generator(c);
    }
    printf("sanitized cases: %d\n", cases);
    return 0;
}
