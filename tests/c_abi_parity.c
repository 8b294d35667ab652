/*
 * A pure C consumer of the library's C ABI: seeded batches are verified with
 * asd_verify on the GPU through the HIP runtime API alone (no C++, no Python,
 * no torch), and every output is compared bit for bit with the CPU oracle.
 *
 * Test infrastructure, like the oracle it links: __graft_entry__.build()
 * compiles it with gcc, and tests/test_c_abi_gpu.py runs it.  Exit status 0
 * when every case matches, 1 on a mismatch, 2 on a setup error.
 *
 * Usage: c_abi_parity [cases]   (default 40)
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "asd.h"

/* The oracle's entry points (oracle/asd_oracle.c); dtype 0 = binary32, 1 = bf16. */
int oracle_verify(const void *logits, int dtype, int64_t vocab, int32_t num_requests,
                  int64_t total_rows, const int32_t *draft, const int32_t *block_lens,
                  const int64_t *row_offsets, const float *tau, const int32_t *exc_cap,
                  float *budget, int32_t *out_accept_len, int32_t *out_next_token,
                  int32_t *out_argmax, float *out_regret);
int64_t oracle_row_argmax(const void *logits, int dtype, int64_t vocab, int64_t row);

/* xorshift64* for the inputs (any seeded generator serves: the inputs are data). */
static uint64_t g_state;
static uint64_t next_u64(void)
{
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return g_state * 0x2545f4914f6cdd1dull;
}
static int64_t uniform(int64_t n) { return (int64_t)(next_u64() % (uint64_t)n); }

static uint32_t f32_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return u;
}

/* A logit: mostly small dyadic values (many ties), sometimes a special value. */
static uint32_t logit_bits(int specials)
{
    static const uint32_t special[] = {0x00000000u, 0x80000000u, 0x7f800000u, 0xff800000u,
                                       0x7fc00000u, 0xffc00000u, 0x00000001u, 0x3f800000u};
    if (specials && uniform(50) == 0)
        return special[uniform(8)];
    return f32_bits((float)(uniform(25) - 12) / 4.0f);
}

#define CHECK_HIP(x)                                                                   \
    do {                                                                               \
        hipError_t e_ = (x);                                                           \
        if (e_ != hipSuccess) {                                                        \
            fprintf(stderr, "HIP error %d at line %d\n", (int)e_, __LINE__);            \
            exit(2);                                                                   \
        }                                                                              \
    } while (0)

/* Device memory of `bytes` bytes, filled from `host` unless that is NULL. */
static void *to_device(const void *host, size_t bytes)
{
    void *d = NULL;
    CHECK_HIP(hipMalloc(&d, bytes > 0 ? bytes : 16));
    if (host != NULL && bytes > 0)
        CHECK_HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
    return d;
}

static int same_f32(float a, float b)
{
    if (isnan(a) && isnan(b))
        return 1;
    return f32_bits(a) == f32_bits(b);
}

/* One seeded batch; returns the number of mismatching outputs. */
static int run_case(int index)
{
    const int bf16 = (int)uniform(2);
    static const int64_t vocabs[] = {7, 129, 1000, 5003, 32000, 151936};
    const int64_t vocab = vocabs[uniform(6)];
    const int32_t n = (int32_t)(vocab >= 32000 ? 1 + uniform(4) : 1 + uniform(48));
    const int explicit_offsets = (int)uniform(3) == 0;
    const int specials = (int)uniform(2);
    const size_t eb = bf16 ? 2 : 4;

    int32_t *lens = malloc(sizeof(int32_t) * (size_t)n);
    int64_t *offsets = malloc(sizeof(int64_t) * (size_t)n);
    float *tau = malloc(sizeof(float) * (size_t)n);
    int32_t *cap = malloc(sizeof(int32_t) * (size_t)n);
    float *budget = malloc(sizeof(float) * 2 * (size_t)n);
    int64_t rows = 0;
    for (int32_t i = 0; i < n; ++i) {
        static const float taus[] = {0.25f, 1.0f, 2.0f, INFINITY};
        static const float budgets[] = {0.0f, 1.0f, 4.0f, 16.0f};
        lens[i] = (int32_t)uniform(vocab >= 32000 ? 9 : 17);
        if (explicit_offsets)
            rows += uniform(2);               /* a gap row before some requests */
        offsets[i] = rows;
        rows += lens[i] + 1;
        tau[i] = taus[uniform(4)];
        cap[i] = (int32_t)uniform(4);
        budget[2 * i] = budgets[uniform(4)];
        budget[2 * i + 1] = (float)uniform(3) / 2.0f;
    }

    unsigned char *logits = malloc((size_t)rows * (size_t)vocab * eb);
    for (int64_t k = 0; k < rows * vocab; ++k) {
        const uint32_t b = logit_bits(specials);
        if (bf16) {
            const uint16_t h = (uint16_t)(b >> 16);
            memcpy(logits + k * 2, &h, 2);
        } else {
            memcpy(logits + k * 4, &b, 4);
        }
    }
    int32_t *draft = malloc(sizeof(int32_t) * (size_t)rows);
    for (int64_t r = 0; r < rows; ++r) {
        const int64_t u = uniform(10);
        if (u < 6)
            draft[r] = (int32_t)oracle_row_argmax(logits, bf16, vocab, r);
        else if (u < 9)
            draft[r] = (int32_t)uniform(vocab);
        else
            draft[r] = uniform(2) ? -1 : (int32_t)vocab;      /* outside [0, V) */
    }

    /* device side */
    void *d_logits = to_device(logits, (size_t)rows * (size_t)vocab * eb);
    int32_t *d_draft = to_device(draft, sizeof(int32_t) * (size_t)rows);
    int32_t *d_lens = to_device(lens, sizeof(int32_t) * (size_t)n);
    int64_t *d_off = explicit_offsets ? to_device(offsets, sizeof(int64_t) * (size_t)n) : NULL;
    float *d_tau = to_device(tau, sizeof(float) * (size_t)n);
    int32_t *d_cap = to_device(cap, sizeof(int32_t) * (size_t)n);
    asd_budget *d_budget = to_device(budget, sizeof(float) * 2 * (size_t)n);
    int32_t *d_acc = to_device(NULL, sizeof(int32_t) * (size_t)n);
    int32_t *d_next = to_device(NULL, sizeof(int32_t) * (size_t)n);
    int32_t *d_amax = to_device(NULL, sizeof(int32_t) * (size_t)rows);
    float *d_regret = to_device(NULL, sizeof(float) * (size_t)rows);
    CHECK_HIP(hipMemset(d_regret, 0xff, sizeof(float) * (size_t)rows));   /* NaN where unwritten */

    const asd_status st = asd_verify(d_logits, bf16 ? ASD_BF16 : ASD_F32, vocab, n, rows, d_draft,
                                     d_lens, d_off, d_tau, d_cap, d_budget, d_acc, d_next, d_amax,
                                     d_regret, NULL);
    if (st != ASD_OK) {
        fprintf(stderr, "case %d: asd_verify returned %s\n", index, asd_status_string(st));
        exit(2);
    }
    CHECK_HIP(hipDeviceSynchronize());

    int32_t *g_acc = malloc(sizeof(int32_t) * (size_t)n), *g_next = malloc(sizeof(int32_t) * (size_t)n);
    int32_t *g_amax = malloc(sizeof(int32_t) * (size_t)rows);
    float *g_regret = malloc(sizeof(float) * (size_t)rows), *g_budget = malloc(sizeof(float) * 2 * (size_t)n);
    CHECK_HIP(hipMemcpy(g_acc, d_acc, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(g_next, d_next, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(g_amax, d_amax, sizeof(int32_t) * (size_t)rows, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(g_regret, d_regret, sizeof(float) * (size_t)rows, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(g_budget, d_budget, sizeof(float) * 2 * (size_t)n, hipMemcpyDeviceToHost));

    /* the oracle on the same inputs */
    int32_t *r_acc = malloc(sizeof(int32_t) * (size_t)n), *r_next = malloc(sizeof(int32_t) * (size_t)n);
    int32_t *r_amax = malloc(sizeof(int32_t) * (size_t)rows);
    float *r_regret = malloc(sizeof(float) * (size_t)rows);
    for (int64_t r = 0; r < rows; ++r)
        r_regret[r] = NAN;
    if (oracle_verify(logits, bf16, vocab, n, rows, draft, lens, explicit_offsets ? offsets : NULL,
                      tau, cap, budget, r_acc, r_next, r_amax, r_regret) != 0) {
        fprintf(stderr, "case %d: the oracle rejected the batch\n", index);
        exit(2);
    }

    int bad = 0;
    for (int32_t i = 0; i < n; ++i) {
        bad += g_acc[i] != r_acc[i];
        bad += g_next[i] != r_next[i];
        bad += f32_bits(g_budget[2 * i + 1]) != f32_bits(budget[2 * i + 1]);
    }
    for (int64_t r = 0; r < rows; ++r) {
        bad += g_amax[r] != r_amax[r];
        bad += !same_f32(g_regret[r], r_regret[r]);
    }
    printf("case %d: %s V %lld, %d requests, %lld rows, %s offsets%s: %s\n", index,
           bf16 ? "bf16" : "f32", (long long)vocab, (int)n, (long long)rows,
           explicit_offsets ? "explicit" : "packed", specials ? ", special values" : "",
           bad ? "MISMATCH" : "ok");
    fflush(stdout);

    hipFree(d_logits); hipFree(d_draft); hipFree(d_lens); hipFree(d_off); hipFree(d_tau);
    hipFree(d_cap); hipFree(d_budget); hipFree(d_acc); hipFree(d_next); hipFree(d_amax);
    hipFree(d_regret);
    free(lens); free(offsets); free(tau); free(cap); free(budget); free(logits); free(draft);
    free(g_acc); free(g_next); free(g_amax); free(g_regret); free(g_budget);
    free(r_acc); free(r_next); free(r_amax); free(r_regret);
    return bad;
}

int main(int argc, char **argv)
{
    const int cases = argc > 1 ? atoi(argv[1]) : 40;
    int failed = 0;
    printf("%s\n", asd_version());
    g_state = 0x9e3779b97f4a7c15ull;
    for (int c = 0; c < cases; ++c)
        failed += run_case(c) != 0;
    printf("%d of %d cases matched the oracle\n", cases - failed, cases);
    return failed ? 1 : 0;
}
