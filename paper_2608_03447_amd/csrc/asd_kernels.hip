// gfx950 kernels of the ASD verifier.
//
// Stage 1 (asd_row_kernel): one workgroup per (row, vocabulary split) tile
// streams the tile's logits once from HBM with 16-byte non-temporal loads and
// keeps, per lane, the greatest logit seen so far (Eq. 1).  Logits are compared
// as order-preserving integer keys, so the whole reduction is integer max work
// with no rounding.  The tile that owns the draft token's column also gathers
// z(x) (Eq. 3).  The last tile of a row to finish combines the split partials,
// forms the regret r = fl32(z(y*) - z(x)) and the mismatch bit d (Eq. 5), and
// writes the row's record.
//
// Stage 2 (asd_scan_kernel): one thread per request runs Algorithm 1 over the
// row records of its block: the B = 0 dispatch to exact greedy verification
// (Eq. 2), otherwise the left-to-right scan that accepts a mismatch only while
// the gate r <= g q (Eqs. 7, 11), the budget fl32(s + C) <= B (Eq. 9) and the
// cap N <= M (Eq. 10) hold, stopping at the first infeasible position (the
// longest feasible prefix, Eq. 12); then the ledger update (Eq. 13) and the
// recovery or bonus token.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asd_plan.h"

namespace asd {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// 16-byte vectors per lane per group in the streaming loop.
constexpr int kUnroll = 4;
constexpr int kGroupVecs = kRowThreads * kUnroll;
constexpr int kWaves = kRowThreads / 64;

// ------------------------------------------------------------ integer keys
//
// key(x) is an integer that orders logits the way the argmax must: numeric
// order with -0 == +0, positive NaNs above +inf and negative NaNs below -inf
// (IEEE totalOrder for NaNs).  For a sign-magnitude pattern: key = magnitude
// when the sign is clear, key = -magnitude when it is set.

// Two bf16 keys at once, one per 16-bit half (packed 16-bit integer ops).
__device__ __forceinline__ uint32_t bf16x2_keys(uint32_t w) {
    const u16x2 v = __builtin_bit_cast(u16x2, w);
    const u16x2 neg = (u16x2)(unsigned short)0x8000 - v;       // -magnitude, mod 2^16
    const u16x2 sign = __builtin_bit_cast(u16x2, __builtin_bit_cast(s16x2, v) >> (s16x2)15);
    return __builtin_bit_cast(uint32_t, (neg & sign) | (v & ~sign));
}

__device__ __forceinline__ int32_t f32_key(uint32_t u) {
    const uint32_t sign = (uint32_t)((int32_t)u >> 31);
    return (int32_t)(((0x80000000u - u) & sign) | (u & ~sign));
}

__device__ __forceinline__ int32_t bf16_key(uint32_t h16) {
    return (int32_t)(int16_t)(bf16x2_keys(h16) & 0xffffu);
}

__device__ __forceinline__ uint32_t pkmax16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2, a),
                                                                  __builtin_bit_cast(s16x2, b)));
}

// Smallest key of each dtype: below every key a real logit can have.
template <int EB> struct KeyTraits;
template <> struct KeyTraits<2> {
    static constexpr int32_t kNone = -0x8000;         // bf16 keys lie in [-0x7fff, 0x7fff]
    static constexpr uint32_t kNonePacked = 0x80008000u;
};
template <> struct KeyTraits<4> {
    static constexpr int32_t kNone = (int32_t)0x80000000;   // f32 keys >= -0x7fffffff
};

// Max key over the 16-byte vectors of one group (per-dtype).
template <int EB, bool kMasked>
__device__ __forceinline__ int32_t group_max_key(const u32x4 (&raw)[kUnroll], int nvalid) {
    if constexpr (EB == 2) {
        uint32_t acc = KeyTraits<2>::kNonePacked;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            uint32_t k0 = bf16x2_keys(raw[u].x), k1 = bf16x2_keys(raw[u].y);
            uint32_t k2 = bf16x2_keys(raw[u].z), k3 = bf16x2_keys(raw[u].w);
            uint32_t m = pkmax16(pkmax16(k0, k1), pkmax16(k2, k3));
            if (kMasked && u >= nvalid) m = KeyTraits<2>::kNonePacked;
            acc = pkmax16(acc, m);
        }
        const int32_t lo = (int32_t)(int16_t)(acc & 0xffffu);
        const int32_t hi = (int32_t)acc >> 16;
        return lo > hi ? lo : hi;
    } else {
        int32_t acc = KeyTraits<4>::kNone;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            int32_t m = max(max(f32_key(raw[u].x), f32_key(raw[u].y)),
                            max(f32_key(raw[u].z), f32_key(raw[u].w)));
            if (kMasked && u >= nvalid) m = KeyTraits<4>::kNone;
            acc = max(acc, m);
        }
        return acc;
    }
}

// Element e of a 16-byte vector as (key, binary32 bits).
template <int EB>
__device__ __forceinline__ void element_of(const u32x4& v, int e, int32_t& key, uint32_t& bits) {
    if constexpr (EB == 2) {
        const uint32_t w = v[e >> 1];
        const uint32_t h = (e & 1) ? (w >> 16) : (w & 0xffffu);
        key = bf16_key(h);
        bits = h << 16;
    } else {
        bits = v[e];
        key = f32_key(bits);
    }
}

template <int EB>
__device__ __forceinline__ void load_scalar(const unsigned char* p, int32_t& key, uint32_t& bits) {
    if constexpr (EB == 2) {
        const uint32_t h = *(const unsigned short*)p;
        key = bf16_key(h);
        bits = h << 16;
    } else {
        bits = *(const uint32_t*)p;
        key = f32_key(bits);
    }
}

// Pack (key, column) so that the unsigned maximum is the greatest key with the
// lowest column.
__device__ __forceinline__ unsigned long long pack_kc(int32_t key, int64_t col) {
    return ((unsigned long long)((uint32_t)key ^ 0x80000000u) << 32) |
           (unsigned long long)(0xffffffffu - (uint32_t)col);
}
__device__ __forceinline__ int32_t packed_col(unsigned long long p) {
    return (int32_t)(0xffffffffu - (uint32_t)(p & 0xffffffffull));
}

__device__ __forceinline__ void take_better(unsigned long long& p, uint32_t& bits,
                                            unsigned long long q, uint32_t qbits) {
    if (q > p) {
        p = q;
        bits = qbits;
    }
}

// Workgroup-wide maximum of (packed, bits); the result is valid in thread 0.
__device__ __forceinline__ void block_reduce(unsigned long long& p, uint32_t& bits) {
    __shared__ unsigned long long s_p[kWaves];
    __shared__ uint32_t s_b[kWaves];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const unsigned long long q = __shfl_xor(p, off, 64);
        const uint32_t qb = __shfl_xor(bits, off, 64);
        take_better(p, bits, q, qb);
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        s_p[wave] = p;
        s_b[wave] = bits;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 1; w < kWaves; ++w) take_better(p, bits, s_p[w], s_b[w]);
    }
}

__device__ __forceinline__ float bits_to_float(uint32_t b) { return __builtin_bit_cast(float, b); }

// Row geometry: elements [0, head) and [tail, V) are read one by one; the
// 16-byte aligned middle as nvec vectors.
struct RowGeom {
    int64_t head, nvec, tail;
};

template <int EB>
__device__ __forceinline__ RowGeom row_geom(const unsigned char* row_ptr, int64_t vocab) {
    constexpr int kEpv = 16 / EB;
    RowGeom g;
    const int64_t mis = (int64_t)((16 - ((uintptr_t)row_ptr & 15)) & 15) / EB;
    g.head = mis < vocab ? mis : vocab;
    g.nvec = (vocab - g.head) / kEpv;
    g.tail = g.head + g.nvec * kEpv;
    return g;
}

// Split that owns column c.
__device__ __forceinline__ int owner_split(int64_t c, const RowGeom& g, int64_t chunk_cols,
                                           int splits) {
    if (c < g.head) return 0;
    const int64_t s = (c - g.head) / chunk_cols;
    return s < splits - 1 ? (int)s : splits - 1;
}

// ----------------------------------------------------------- stage 1 kernel

template <int EB>
__global__ __launch_bounds__(kRowThreads) void asd_row_kernel(
    const unsigned char* __restrict__ logits, int64_t vocab, int splits, int64_t chunk_vecs,
    const int32_t* __restrict__ draft_tokens, TilePartial* __restrict__ partials,
    int32_t* __restrict__ row_counters, RowRecord* __restrict__ records,
    int32_t* __restrict__ out_argmax, float* __restrict__ out_regret) {
    constexpr int kEpv = 16 / EB;
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x / splits;
    const int split = (int)(blockIdx.x - row * splits);
    const unsigned char* row_ptr = logits + row * vocab * EB;
    const RowGeom geom = row_geom<EB>(row_ptr, vocab);
    const int64_t chunk_cols = chunk_vecs * kEpv;

    // Draft token of this row (uniform); the owning tile gathers z(x) early so
    // the load overlaps the stream.
    const int32_t x = draft_tokens[row];
    const bool x_valid = x >= 0 && (int64_t)x < vocab;
    const bool owns_x = x_valid && owner_split(x, geom, chunk_cols, splits) == split;
    uint32_t draft_bits = 0;
    if (owns_x && tid == 0) {
        int32_t k_unused;
        load_scalar<EB>(row_ptr + (int64_t)x * EB, k_unused, draft_bits);
    }

    // ---- stream this tile's 16-byte vectors
    const u32x4* vec = (const u32x4*)(row_ptr + geom.head * EB);
    const int64_t v0 = (int64_t)split * chunk_vecs;
    const int64_t v1 = min(v0 + chunk_vecs, geom.nvec);
    const int64_t nv = v1 > v0 ? v1 - v0 : 0;
    const int64_t nfull = nv / kGroupVecs;

    int32_t best_key = KeyTraits<EB>::kNone;
    int64_t best_group = -1;
    int best_nvalid = 0;
    u32x4 saved[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) saved[u] = (u32x4)(0u);

    for (int64_t g = 0; g < nfull; ++g) {
        const u32x4* p = vec + v0 + g * kGroupVecs + tid;
        u32x4 raw[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) raw[u] = __builtin_nontemporal_load(p + u * kRowThreads);
        const int32_t gk = group_max_key<EB, false>(raw, kUnroll);
        const bool better = gk > best_key;
        best_key = better ? gk : best_key;
        best_group = better ? g : best_group;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) saved[u] = better ? raw[u] : saved[u];
    }
    best_nvalid = best_group >= 0 ? kUnroll : 0;

    if (nv > nfull * kGroupVecs) {       // the tile's last, partial group
        const int64_t g = nfull;
        const int64_t first = v0 + g * kGroupVecs + tid;
        int nvalid = 0;
        u32x4 raw[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            raw[u] = (u32x4)(0u);
            if (first + u * kRowThreads < v1) {
                raw[u] = __builtin_nontemporal_load(vec + first + u * kRowThreads);
                ++nvalid;
            }
        }
        const int32_t gk = group_max_key<EB, true>(raw, nvalid);
        if (gk > best_key) {
            best_key = gk;
            best_group = g;
            best_nvalid = nvalid;
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) saved[u] = raw[u];
        }
    }

    // ---- this lane's first element holding best_key
    unsigned long long packed = pack_kc(KeyTraits<4>::kNone, 0x7fffffff);
    uint32_t bits = 0;
    if (best_group >= 0) {
        bool found = false;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
            for (int e = 0; e < kEpv; ++e) {
                int32_t k;
                uint32_t b;
                element_of<EB>(saved[u], e, k, b);
                if (!found && u < best_nvalid && k == best_key) {
                    found = true;
                    const int64_t vi = v0 + best_group * kGroupVecs + u * kRowThreads + tid;
                    packed = pack_kc(k, geom.head + vi * kEpv + e);
                    bits = b;
                }
            }
        }
    }

    // ---- unaligned head and tail elements (at most 16 / EB - 1 of each)
    if (split == 0 && tid < geom.head) {
        int32_t k;
        uint32_t b;
        load_scalar<EB>(row_ptr + (int64_t)tid * EB, k, b);
        take_better(packed, bits, pack_kc(k, tid), b);
    }
    if (split == splits - 1 && tid < vocab - geom.tail) {
        const int64_t c = geom.tail + tid;
        int32_t k;
        uint32_t b;
        load_scalar<EB>(row_ptr + c * EB, k, b);
        take_better(packed, bits, pack_kc(k, c), b);
    }

    block_reduce(packed, bits);
    if (tid != 0) return;

    // ---- combine the splits of this row (the last tile to finish does it)
    if (splits > 1) {
        TilePartial* mine = partials + row * splits;
        TilePartial tp;
        tp.packed = packed;
        tp.bits = bits;
        tp.draft_bits = draft_bits;
        mine[split] = tp;
        const int32_t done = __hip_atomic_fetch_add(row_counters + row, 1, __ATOMIC_ACQ_REL,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        if (done != splits - 1) return;
        row_counters[row] = 0;            // ready for the next call
        if (x_valid) draft_bits = mine[owner_split(x, geom, chunk_cols, splits)].draft_bits;
        for (int s = 0; s < splits; ++s) {
            if (s == split) continue;
            const TilePartial o = mine[s];
            take_better(packed, bits, o.packed, o.bits);
        }
    }

    // ---- row record: argmax, mismatch bit, regret (one binary32 subtraction)
    const int32_t y = packed_col(packed);
    float r;
    uint32_t flags;
    if (x_valid) {
        r = bits_to_float(bits) - bits_to_float(draft_bits);
        flags = (x != y) ? kMismatchBit : 0u;
    } else {
        r = __builtin_huge_valf();
        flags = kMismatchBit | kBadDraftBit;
    }
    RowRecord rec;
    rec.y_flags = (uint32_t)y | flags;
    rec.regret = r;
    records[row] = rec;
    if (out_argmax) out_argmax[row] = y;
    if (out_regret) out_regret[row] = r;
}

// ----------------------------------------------------------- stage 2 kernel

// Records read ahead per scan window: one window covers K <= 31 and the bonus row.
constexpr int kScanWindow = 32;

// Algorithm 1 for request i whose rows start at o (validated by the caller).
__device__ __forceinline__ void scan_request(int32_t i, int64_t o, int32_t K, const float* tau,
                                             const int32_t* exc_cap, float2* budget,
                                             const RowRecord* records, int32_t* out_accept_len,
                                             int32_t* out_next_token, float* out_regret) {
    const float2 ledger = budget[i];
    const float B = ledger.x;
    float s = ledger.y;
    const float g = tau[i];
    const int32_t M = exc_cap[i];
    const bool strict = (B == 0.0f);      // Algorithm 1: B = 0 -> exact greedy verification

    int32_t a = 0, N = 0, next = -1;
    float C = 0.0f;
    bool stop = false;
    for (int64_t w0 = 0; w0 <= K && !stop; w0 += kScanWindow) {
        RowRecord rec[kScanWindow];
#pragma unroll
        for (int j = 0; j < kScanWindow; ++j)
            if (w0 + j <= K) rec[j] = records[o + w0 + j];
#pragma unroll
        for (int j = 0; j < kScanWindow; ++j) {
            const int64_t p = w0 + j;                 // 0-based position; p == K: bonus row
            if (!stop && p <= K) {
                const uint32_t yf = rec[j].y_flags;
                bool accept = (p < K) && (yf & kMismatchBit) == 0u;   // exact match
                if (p < K && !accept && !strict && (yf & kBadDraftBit) == 0u) {
                    const float r = rec[j].regret;
                    const int32_t q = K - (int32_t)p;  // q_i = K - i + 1 with i = p + 1
                    const bool gate = (double)r <= (double)g * (double)q;
                    const float C_new = C + r;
                    const int32_t N_new = N + 1;
                    const float s_new = s + C_new;
                    if (gate && s_new <= B && N_new <= M) {
                        C = C_new;
                        N = N_new;
                        accept = true;
                    }
                }
                if (accept) {
                    a = (int32_t)p + 1;
                } else {
                    // First infeasible position, or the bonus row after a
                    // fully accepted block: emit y*_{a+1}.
                    next = (int32_t)(yf & kArgmaxMask);
                    stop = true;
                }
            }
        }
    }
    if (N > 0) {
        s = s + C;                                    // s' = s + C_a
        budget[i].y = s;
    }
    out_accept_len[i] = a;
    out_next_token[i] = next;
    if (out_regret) out_regret[o + K] = 0.0f;
}

// Per-request validity: rows [o, o + K] inside [0, total_rows).
__device__ __forceinline__ bool request_ok(int64_t o, int32_t K, int64_t total_rows) {
    return K >= 0 && o >= 0 && o + (int64_t)K < total_rows;
}

// Requests with explicit row offsets: one thread per request, any grid.
__global__ __launch_bounds__(kScanThreads) void asd_scan_offsets_kernel(
    int32_t num_requests, int64_t total_rows, const int32_t* __restrict__ block_lens,
    const int64_t* __restrict__ row_offsets, const float* __restrict__ tau,
    const int32_t* __restrict__ exc_cap, float2* __restrict__ budget,
    const RowRecord* __restrict__ records, int32_t* __restrict__ out_accept_len,
    int32_t* __restrict__ out_next_token, float* __restrict__ out_regret) {
    const int64_t i = (int64_t)blockIdx.x * kScanThreads + threadIdx.x;
    if (i >= num_requests) return;
    const int32_t K = block_lens[i];
    const int64_t o = row_offsets[i];
    if (!request_ok(o, K, total_rows)) {
        out_accept_len[i] = 0;
        out_next_token[i] = -1;
        return;
    }
    scan_request((int32_t)i, o, K, tau, exc_cap, budget, records, out_accept_len, out_next_token,
                 out_regret);
}

// Packed layout o_i = sum_{j<i} (max(K_j, 0) + 1): one workgroup walks the
// requests in chunks, an exclusive scan of the row counts giving each offset.
__global__ __launch_bounds__(kScanThreads) void asd_scan_packed_kernel(
    int32_t num_requests, int64_t total_rows, const int32_t* __restrict__ block_lens,
    const float* __restrict__ tau, const int32_t* __restrict__ exc_cap,
    float2* __restrict__ budget, const RowRecord* __restrict__ records,
    int32_t* __restrict__ out_accept_len, int32_t* __restrict__ out_next_token,
    float* __restrict__ out_regret) {
    __shared__ long long s_wave[kScanThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    long long carry = 0;
    for (int64_t c0 = 0; c0 < num_requests; c0 += kScanThreads) {
        const int64_t i = c0 + tid;
        const int32_t K = i < num_requests ? block_lens[i] : 0;
        const long long n = i < num_requests ? (long long)(K > 0 ? K : 0) + 1 : 0;
        // inclusive scan within the wavefront
        long long incl = n;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const long long t = __shfl_up(incl, off, 64);
            if (lane >= off) incl += t;
        }
        if (lane == 63) s_wave[wave] = incl;
        __syncthreads();
        long long before = 0, chunk_total = 0;
#pragma unroll
        for (int w = 0; w < kScanThreads / 64; ++w) {
            const long long t = s_wave[w];
            before += (w < wave) ? t : 0;
            chunk_total += t;
        }
        __syncthreads();
        const int64_t o = carry + before + incl - n;
        carry += chunk_total;
        if (i < num_requests) {
            if (!request_ok(o, K, total_rows)) {
                out_accept_len[i] = 0;
                out_next_token[i] = -1;
            } else {
                scan_request((int32_t)i, o, K, tau, exc_cap, budget, records, out_accept_len,
                             out_next_token, out_regret);
            }
        }
    }
}

}  // namespace

// ------------------------------------------------------------------ launch

hipError_t launch_verify(const Plan& plan, const CallArgs& a, void* workspace,
                         hipStream_t stream) {
    unsigned char* ws = (unsigned char*)workspace;
    RowRecord* records = (RowRecord*)(ws + plan.off_records);
    TilePartial* partials = plan.splits > 1 ? (TilePartial*)(ws + plan.off_partials) : nullptr;
    int32_t* counters = plan.splits > 1 ? (int32_t*)(ws + plan.off_counters) : nullptr;

    const dim3 grid((unsigned)(plan.rows * plan.splits));
    if (plan.elem_bytes == 2)
        asd_row_kernel<2><<<grid, kRowThreads, 0, stream>>>(
            (const unsigned char*)a.logits, plan.vocab, plan.splits, plan.chunk_vecs,
            a.draft_tokens, partials, counters, records, a.out_argmax, a.out_regret);
    else
        asd_row_kernel<4><<<grid, kRowThreads, 0, stream>>>(
            (const unsigned char*)a.logits, plan.vocab, plan.splits, plan.chunk_vecs,
            a.draft_tokens, partials, counters, records, a.out_argmax, a.out_regret);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;

    if (a.row_offsets) {
        const unsigned blocks = (unsigned)((a.num_requests + kScanThreads - 1) / kScanThreads);
        asd_scan_offsets_kernel<<<blocks, kScanThreads, 0, stream>>>(
            a.num_requests, plan.rows, a.block_lens, a.row_offsets, a.tau, a.exc_cap, a.budget,
            records, a.out_accept_len, a.out_next_token, a.out_regret);
    } else {
        asd_scan_packed_kernel<<<1, kScanThreads, 0, stream>>>(
            a.num_requests, plan.rows, a.block_lens, a.tau, a.exc_cap, a.budget, records,
            a.out_accept_len, a.out_next_token, a.out_regret);
    }
    return hipGetLastError();
}

}  // namespace asd
