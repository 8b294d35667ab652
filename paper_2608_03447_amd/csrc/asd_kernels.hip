// gfx950 kernels of the ASD verifier.
//
// Stage 1 (asd_row_kernel): one workgroup per (row, vocabulary split) tile
// streams the tile's logits once from HBM with 16-byte non-temporal loads and
// keeps, per lane, the greatest logit seen so far (Eq. 1).  Logits are compared
// as order-preserving integer keys, so the whole reduction is integer max work
// with no rounding.  The tile that owns the draft token's column also gathers
// z(x) (Eq. 3).  With one tile per row the tile writes the row's record:
// argmax, mismatch bit d (Eq. 5) and regret r = fl32(z(y*) - z(x)).  With
// several tiles per row each tile writes a partial; no workgroup waits for or
// signals another.  Block 0 also writes the packed row offsets of the requests.
//
// Stage 2 (asd_scan_kernel): one wavefront per request runs Algorithm 1 with
// lanes = block positions.  Each lane forms its row's record (or combines the
// row's split partials), then the wavefront ballots the mismatches and walks
// only those, in position order: the B = 0 dispatch stops at the first one
// (Eq. 2); otherwise a mismatch is accepted while the gate r <= g q (Eqs. 7,
// 11), the budget fl32(s + C) <= B (Eq. 9) and the cap N <= M (Eq. 10) hold,
// and the first that fails ends the longest feasible prefix (Eq. 12).  Exact
// matches in between are feasible by Eq. 14's first term.  The running sum C
// is accumulated in position order, one binary32 addition per accepted
// mismatch, exactly as the sequential definition does.  Then the ledger update
// (Eq. 13) and the recovery or bonus token.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <mutex>

#include "asd_plan.h"

// Workspace of asd_verify_static, for callers that cannot allocate: one fixed
// array per device, held until the process ends.  In host code its name is
// only a stand-in for the symbol, not a device address; host code uses the
// address static_scratch_address returns for the current device.
static __device__ __align__(256) unsigned char scratch[asd::kStaticScratchBytes];

namespace asd {

hipError_t static_scratch_address(void** ptr) {
    static std::mutex m;
    static std::map<int, void*> by_device;   // each device holds its own copy
    int device = 0;
    hipError_t err = hipGetDevice(&device);
    if (err != hipSuccess) return err;
    std::lock_guard<std::mutex> lock(m);
    auto it = by_device.find(device);
    if (it == by_device.end()) {
        void* p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return err;
        if (p == nullptr) return hipErrorInvalidSymbol;
        it = by_device.emplace(device, p).first;
    }
    *ptr = it->second;
    return hipSuccess;
}

// Sticky error word of this device: the kernels OR in kErr* bits when they meet
// data that the verifier reads in a defined but unusual way.
__device__ uint32_t asd_error_word;

hipError_t error_word_address(uint32_t** ptr) {
    return hipGetSymbolAddress((void**)ptr, HIP_SYMBOL(asd_error_word));
}

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
// order with -0 == +0, and every NaN, of either sign and any payload, above
// +inf and equal to every other NaN (so a row's first NaN is its argmax).  For
// a number's sign-magnitude pattern: key = magnitude when the sign is clear,
// key = -magnitude when it is set; every NaN has the key kNan, one above +inf's.

// Smallest key of each dtype (below every key a real logit can have), the key
// of +inf, the key of every NaN, and the greatest pattern that is not a NaN
// with the sign bit set (-inf's).
template <int EB> struct KeyTraits;
template <> struct KeyTraits<2> {
    static constexpr uint32_t kNonePacked = 0x80008000u;   // bf16 keys lie in [-0x7f80, 0x7f81]
    static constexpr int32_t kInf = 0x7f80;
    static constexpr int32_t kNan = 0x7f81;
    static constexpr uint32_t kNegInfPattern = 0xff80u;
};
template <> struct KeyTraits<4> {
    static constexpr int32_t kNone = (int32_t)0x80000000;   // f32 keys >= -0x7f800000
    static constexpr int32_t kInf = 0x7f800000;
    static constexpr int32_t kNan = 0x7f800001;
    static constexpr uint32_t kNegInfPattern = 0xff800000u;
};

// The key of every binary32 pattern (used where one pass must rank anything).
__device__ __forceinline__ int32_t f32_key(uint32_t u) {
    const uint32_t mag = u & 0x7fffffffu;
    const int32_t key = (int32_t)u < 0 ? -(int32_t)mag : (int32_t)mag;
    return mag > 0x7f800000u ? KeyTraits<4>::kNan : key;
}

// Three ways to rank logits, cheapest first.
//  kKeysRaw:   the raw bit patterns read as signed integers.  For every pattern
//              with the sign bit clear that is neither +0 nor a NaN this equals
//              the key, and every pattern with the sign bit set reads as
//              negative.  So among elements that include a number in [1, +inf]
//              and no NaN, the raw maximum is the exact maximum, found with one
//              integer max per element.
//  kKeysExact: sign-magnitude keys, exact for every number.
//  kKeysNan:   min(magnitude, kNan): every NaN gets kNan and every number a
//              smaller key, so in a tile known to hold a NaN the greatest key
//              is kNan and its first element is the tile's first NaN.
// With raw and sign-magnitude keys a NaN's key is not kNan.  Those passes keep
// the greatest pattern read as unsigned, which exceeds -inf's exactly when a
// NaN with the sign bit set is present; a NaN with it clear shows as a greatest
// key above +inf's.  Either sends the tile to a NaN pass.
constexpr int kKeysRaw = 0, kKeysExact = 1, kKeysNan = 2;
constexpr int32_t kRawExactFrom = 1;

// Two bf16 sign-magnitude keys at once, one per 16-bit half.
__device__ __forceinline__ uint32_t bf16x2_keys(uint32_t w) {
    const u16x2 v = __builtin_bit_cast(u16x2, w);
    const u16x2 neg = (u16x2)(unsigned short)0x8000 - v;       // -magnitude, mod 2^16
    const u16x2 sign = __builtin_bit_cast(u16x2, __builtin_bit_cast(s16x2, v) >> (s16x2)15);
    return __builtin_bit_cast(uint32_t, (neg & sign) | (v & ~sign));
}

__device__ __forceinline__ uint32_t pkmax16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2, a),
                                                                  __builtin_bit_cast(s16x2, b)));
}

__device__ __forceinline__ uint32_t pkmaxu16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, a),
                                                                  __builtin_bit_cast(u16x2, b)));
}

__device__ __forceinline__ uint32_t pkminu16(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_min(__builtin_bit_cast(u16x2, a),
                                                                  __builtin_bit_cast(u16x2, b)));
}

template <int EB, int kMode>
__device__ __forceinline__ uint32_t dword_keys(uint32_t w) {
    if constexpr (kMode == kKeysRaw) {
        return w;
    } else if constexpr (kMode == kKeysExact) {
        if constexpr (EB == 2) return bf16x2_keys(w);
        else return (int32_t)w < 0 ? 0x80000000u - w : w;
    } else {
        if constexpr (EB == 2) return pkminu16(w & 0x7fff7fffu, (uint32_t)KeyTraits<2>::kNan * 0x10001u);
        else return min(w & 0x7fffffffu, (uint32_t)KeyTraits<4>::kNan);
    }
}

// Max key over the 16-byte vectors of one group.  With raw and sign-magnitude
// keys `umax` also takes the greatest pattern read as unsigned (per 16-bit half
// for bf16).
template <int EB, int kMode>
__device__ __forceinline__ int32_t group_max_key(const u32x4 (&raw)[kUnroll], uint32_t& umax) {
    if constexpr (EB == 2) {
        uint32_t acc = KeyTraits<2>::kNonePacked;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint32_t k0 = dword_keys<2, kMode>(raw[u].x), k1 = dword_keys<2, kMode>(raw[u].y);
            const uint32_t k2 = dword_keys<2, kMode>(raw[u].z), k3 = dword_keys<2, kMode>(raw[u].w);
            uint32_t m = pkmax16(pkmax16(k0, k1), pkmax16(k2, k3));
            acc = pkmax16(acc, m);
            if constexpr (kMode != kKeysNan)
                umax = pkmaxu16(umax, pkmaxu16(pkmaxu16(raw[u].x, raw[u].y),
                                               pkmaxu16(raw[u].z, raw[u].w)));
        }
        const int32_t lo = (int32_t)(int16_t)(acc & 0xffffu);
        const int32_t hi = (int32_t)acc >> 16;
        return lo > hi ? lo : hi;
    } else {
        int32_t acc = KeyTraits<4>::kNone;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            int32_t m = max(max((int32_t)dword_keys<4, kMode>(raw[u].x),
                                (int32_t)dword_keys<4, kMode>(raw[u].y)),
                            max((int32_t)dword_keys<4, kMode>(raw[u].z),
                                (int32_t)dword_keys<4, kMode>(raw[u].w)));
            acc = max(acc, m);
            if constexpr (kMode != kKeysNan)
                umax = max(umax, max(max(raw[u].x, raw[u].y), max(raw[u].z, raw[u].w)));
        }
        return acc;
    }
}

// Key of a bf16 bit pattern (low 16 bits of h16) or f32 bit pattern.
template <int EB, int kMode>
__device__ __forceinline__ int32_t key_of(uint32_t pattern) {
    if constexpr (EB == 2) return (int32_t)(int16_t)(dword_keys<2, kMode>(pattern) & 0xffffu);
    else return (int32_t)dword_keys<4, kMode>(pattern);
}

// Greatest key among the elements of one dword (two bf16 or one f32).
template <int EB, int kMode>
__device__ __forceinline__ int32_t dword_max_key(uint32_t w) {
    const uint32_t k = dword_keys<EB, kMode>(w);
    if constexpr (EB == 2) {
        const int32_t lo = (int32_t)(int16_t)(k & 0xffffu), hi = (int32_t)k >> 16;
        return lo > hi ? lo : hi;
    } else {
        return (int32_t)k;
    }
}

template <int EB, int kMode>
__device__ __forceinline__ void load_scalar(const unsigned char* p, int32_t& key, uint32_t& bits) {
    if constexpr (EB == 2) {
        const uint32_t h = *(const unsigned short*)p;
        key = key_of<2, kMode>(h);
        bits = h << 16;
    } else {
        bits = *(const uint32_t*)p;
        key = key_of<4, kMode>(bits);
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
__device__ __forceinline__ int32_t packed_key(unsigned long long p) {
    return (int32_t)((uint32_t)(p >> 32) ^ 0x80000000u);
}

__device__ __forceinline__ void take_better(unsigned long long& p, uint32_t& bits,
                                            unsigned long long q, uint32_t qbits) {
    if (q > p) {
        p = q;
        bits = qbits;
    }
}

// One step of a wavefront maximum of (packed, bits) by DPP: each lane takes
// the pair of the lane that `kCtrl` names when it is greater.  A lane with no
// source lane in the step (or in a row that kRowMask leaves out) reads 0,
// which ranks below every packed pair.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ void dpp_max_step(unsigned long long& p, uint32_t& bits) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)p, kCtrl, kRowMask,
                                                              0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(p >> 32), kCtrl,
                                                              kRowMask, 0xf, false);
    const uint32_t qb = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)bits, kCtrl, kRowMask, 0xf,
                                                              false);
    const unsigned long long q = ((unsigned long long)hi << 32) | lo;
    const bool take = q > p;
    p = take ? q : p;
    bits = take ? qb : bits;
}

// Unsigned 64-bit maximum of a lane's value and that of the lane `kCtrl`
// names (a DPP pattern in which every lane has a source).
template <int kCtrl>
__device__ __forceinline__ unsigned long long dpp_umax64(unsigned long long p) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)p, kCtrl, 0xf, 0xf,
                                                              false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(p >> 32), kCtrl,
                                                              0xf, 0xf, false);
    const unsigned long long q = ((unsigned long long)hi << 32) | lo;
    return q > p ? q : p;
}

// Workgroup-wide maximum of (packed, bits), and the OR of one flag per
// wavefront; every thread returns with both.  Within a wavefront, shifts of 1,
// 2, 4 and 8 lanes make lane 15 of each 16-lane row hold the row's maximum,
// and the broadcasts of lanes 15 and 31 carry it on, so that lane 63 holds the
// wavefront's.  No cross-lane step waits on LDS.  The wavefronts' results meet
// in LDS behind one barrier.
__device__ __forceinline__ bool block_reduce(unsigned long long& p, uint32_t& bits, bool flag) {
    __shared__ unsigned long long s_p[kWaves];
    __shared__ uint32_t s_b[kWaves];
    __shared__ int s_f[kWaves];
    dpp_max_step<0x111, 0xf>(p, bits);   // row_shr:1
    dpp_max_step<0x112, 0xf>(p, bits);   // row_shr:2
    dpp_max_step<0x114, 0xf>(p, bits);   // row_shr:4
    dpp_max_step<0x118, 0xf>(p, bits);   // row_shr:8
    dpp_max_step<0x142, 0xa>(p, bits);   // row_bcast:15 into rows 1 and 3
    dpp_max_step<0x143, 0xc>(p, bits);   // row_bcast:31 into rows 2 and 3
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 63) {
        s_p[wave] = p;
        s_b[wave] = bits;
        s_f[wave] = flag;
    }
    __syncthreads();
    p = s_p[0];
    bits = s_b[0];
    int any = s_f[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) {
        take_better(p, bits, s_p[w], s_b[w]);
        any |= s_f[w];
    }
    return any != 0;
}

__device__ __forceinline__ float bits_to_float(uint32_t b) { return __builtin_bit_cast(float, b); }

// Row geometry: elements [0, head) and [tail, V) are read one by one; the
// 16-byte aligned middle as nvec vectors.
struct RowGeom {
    int64_t head, nvec, tail;
};

__device__ __forceinline__ RowGeom row_geom(const unsigned char* row_ptr, int64_t vocab, int eb) {
    RowGeom g;
    const int64_t mis = (int64_t)((16 - ((uintptr_t)row_ptr & 15)) & 15) / eb;
    g.head = mis < vocab ? mis : vocab;
    g.nvec = (vocab - g.head) * eb / 16;
    g.tail = g.head + g.nvec * (16 / eb);
    return g;
}

// Split that owns column c.
__device__ __forceinline__ int owner_split(int64_t c, const RowGeom& g, int64_t chunk_cols,
                                           int splits) {
    if (c < g.head) return 0;
    const int64_t s = (uint32_t)(c - g.head) / (uint32_t)chunk_cols;   // both below 2^31
    return s < splits - 1 ? (int)s : splits - 1;
}

// Packed layout o_i = sum_{j<i} (max(K_j, 0) + 1), written by one workgroup:
// an exclusive scan of the row counts in chunks of kRowThreads requests.
__device__ void write_packed_offsets(int32_t num_requests, const int32_t* __restrict__ block_lens,
                                     int64_t* __restrict__ offsets) {
    __shared__ long long s_wave[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    long long carry = 0;
    for (int64_t c0 = 0; c0 < num_requests; c0 += kRowThreads) {
        const int64_t i = c0 + tid;
        const int32_t K = i < num_requests ? block_lens[i] : 0;
        const long long n = i < num_requests ? (long long)(K > 0 ? K : 0) + 1 : 0;
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
        for (int w = 0; w < kWaves; ++w) {
            const long long t = s_wave[w];
            before += (w < wave) ? t : 0;
            chunk_total += t;
        }
        __syncthreads();
        if (i < num_requests) offsets[i] = carry + before + incl - n;
        carry += chunk_total;
    }
}

// Row offsets of one workgroup's requests [first, first + count), count <=
// kScanThreads, into s_off: row_offsets[i] when given, else the packed layout
// o_i = sum_{j<i} (max(K_j, 0) + 1).  For the packed layout the whole workgroup
// sums the row counts of the requests before `first`, then scans its own, so
// no request count is too large and nothing is written to global memory.
// Ends with a barrier.
__device__ void block_offsets(int32_t num_requests, const int32_t* __restrict__ block_lens,
                              const int64_t* __restrict__ row_offsets, int64_t first, int count,
                              int64_t* s_off) {
    __shared__ long long s_before[kWaves];
    __shared__ long long s_mine[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (row_offsets) {
        if (tid < count) s_off[tid] = row_offsets[first + tid];
        __syncthreads();
        return;
    }
    long long before = 0;
    for (int64_t j = tid; j < first; j += blockDim.x) {
        const int32_t K = block_lens[j];
        before += (long long)(K > 0 ? K : 0) + 1;
    }
    const int32_t Km = tid < count ? block_lens[first + tid] : 0;
    const long long mine = tid < count ? (long long)(Km > 0 ? Km : 0) + 1 : 0;
    long long incl = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const long long t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
        before += __shfl_xor(before, off, 64);
    }
    if (lane == 63) s_mine[wave] = incl;
    if (lane == 0) s_before[wave] = before;
    __syncthreads();
    long long base = 0, earlier = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
        base += s_before[w];
        earlier += (w < wave) ? s_mine[w] : 0;
    }
    if (tid < count) s_off[tid] = base + earlier + incl - mine;
    __syncthreads();
}

// Where one lane's share of a tile lies: 16-byte vectors [v0, v1) of the row's
// aligned middle, in ngroups groups of kGroupVecs vectors (the last one padded
// with copies, see load_group).
struct TileSpan {
    const u32x4* vec;
    int32_t v0, v1, nv, ngroups;  // vector counts: a row has fewer than 2^28 vectors
    int tid;
};

// Group g of the lane's share.  In the tile's last group a vector past the
// tile's end is read as a copy of the tile's last vector: a copy adds no new
// value, and its column (past the end) is greater than the original's, so the
// tile's first greatest element is unchanged.  Every group is then whole, and
// the last one is loaded in the pipeline like the others.
__device__ __forceinline__ void load_group(const TileSpan& t, u32x4 (&r)[kUnroll], int32_t g) {
    const int32_t i0 = t.v0 + g * kGroupVecs + t.tid;
    const unsigned char* base = (const unsigned char*)t.vec;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        // a 32-bit byte offset from the row (a row is under 2^32 bytes)
        const uint32_t off = (uint32_t)min(i0 + u * kRowThreads, t.v1 - 1) << 4;
        r[u] = __builtin_nontemporal_load((const u32x4*)(base + off));
    }
}

// The lane's first element holding `key` in a saved group, narrowed level by
// level in column order: the first vector whose greatest key is `key`, then
// that vector's first such dword, then (bf16) the half.  Returns the element's
// index within the group's vectors' elements and its binary32 bits.
template <int EB, int kMode>
__device__ __forceinline__ void find_first(const u32x4 (&saved)[kUnroll], int32_t key, int& su,
                                           int& e, uint32_t& bits) {
    su = 0;
    u32x4 sv = saved[0];
    bool hit = false;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int32_t mk = max(max(dword_max_key<EB, kMode>(saved[u].x),
                                   dword_max_key<EB, kMode>(saved[u].y)),
                               max(dword_max_key<EB, kMode>(saved[u].z),
                                   dword_max_key<EB, kMode>(saved[u].w)));
        const bool take = !hit && mk == key;
        su = take ? u : su;
        sv = take ? saved[u] : sv;
        hit = hit || take;
    }
    int d = 3;
    uint32_t w = sv.w;
#pragma unroll
    for (int j = 2; j >= 0; --j) {                 // the first dword holding key wins
        const bool take = dword_max_key<EB, kMode>(sv[j]) == key;
        d = take ? j : d;
        w = take ? sv[j] : w;
    }
    if constexpr (EB == 2) {
        const bool low = key_of<2, kMode>(w & 0xffffu) == key;
        e = 2 * d + (low ? 0 : 1);
        bits = (low ? (w & 0xffffu) : (w >> 16)) << 16;
    } else {
        e = d;
        bits = w;
    }
}

// Key modes of rank_share beyond the three key kinds: choose raw or
// sign-magnitude keys from the first whole group (see tile_best).
constexpr int kKeysChoose = 3;

// One lane's ranking of its share of a tile: the greatest key, the first
// element holding it (as a packed (key, column)) and that element's binary32
// bits.  `mode` is uniform across the wavefront; the loop is shared and each
// group's ranking branches on it.  With kKeysChoose the wavefront ranks its
// first whole group with raw keys and keeps them if that group holds a number
// in [1, +inf] in any lane, else switches to sign-magnitude keys (ranking the
// group again from its registers).  Except with NaN keys, `umax` takes the
// greatest pattern read as unsigned (per 16-bit half for bf16).
template <int EB, typename Hook>
__device__ __forceinline__ void rank_share(const TileSpan& t, int mode, int64_t col_base,
                                           unsigned long long& packed, uint32_t& bits,
                                           uint32_t& umax, Hook&& after_first_loads) {
    constexpr int kEpv = 16 / EB;
    int32_t best_key = KeyTraits<4>::kNone;
    int32_t best_group = -1;
    u32x4 saved[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) saved[u] = (u32x4)(0u);

    auto rank_group = [&](const u32x4 (&r)[kUnroll], int32_t g) {
        int32_t gk;
        if (mode == kKeysNan) {
            gk = group_max_key<EB, kKeysNan>(r, umax);
        } else if (mode == kKeysExact) {
            gk = group_max_key<EB, kKeysExact>(r, umax);
        } else {
            gk = group_max_key<EB, kKeysRaw>(r, umax);
            if (mode == kKeysChoose) {
                const int raw_ok =
                    __ballot(gk >= kRawExactFrom && gk <= KeyTraits<EB>::kInf) != 0ull;
                mode = __builtin_amdgcn_readfirstlane(raw_ok) ? kKeysRaw : kKeysExact;
                if (mode == kKeysExact) gk = group_max_key<EB, kKeysExact>(r, umax);
            }
        }
        const bool better = gk > best_key;
        best_key = better ? gk : best_key;
        best_group = better ? g : best_group;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) saved[u] = better ? r[u] : saved[u];
    };
    // Whole groups through two register buffers in ping-pong: a group's four
    // loads are issued before the previous group is ranked, so each wavefront
    // keeps eight 16-byte loads per lane in flight while it computes.  The
    // first two groups are issued before anything else that reads memory (the
    // hook), so a tile's first data is requested as soon as it starts.  The
    // scheduling barriers keep the compiler from moving ranking work (and its
    // waits) ahead of the loads.
    if (t.ngroups > 0) {
        u32x4 ra[kUnroll], rb[kUnroll];
        load_group(t, ra, 0);
        __builtin_amdgcn_sched_barrier(0);
        after_first_loads();
        __builtin_amdgcn_sched_barrier(0);
        int32_t g = 0;
        for (; g + 2 < t.ngroups; g += 2) {
            load_group(t, rb, g + 1);
            __builtin_amdgcn_sched_barrier(0);
            rank_group(ra, g);
            load_group(t, ra, g + 2);
            __builtin_amdgcn_sched_barrier(0);
            rank_group(rb, g + 1);
        }
        if (g + 1 < t.ngroups) {
            load_group(t, rb, g + 1);
            __builtin_amdgcn_sched_barrier(0);
            rank_group(ra, g);
            rank_group(rb, g + 1);
        } else {
            rank_group(ra, g);
        }
    } else {
        after_first_loads();
    }
    if (mode == kKeysChoose) mode = kKeysExact;      // no group: sign-magnitude keys

    packed = pack_kc(KeyTraits<4>::kNone, 0x7fffffff);
    bits = 0;
    if (best_group >= 0) {
        int su, e;
        if (mode == kKeysRaw) find_first<EB, kKeysRaw>(saved, best_key, su, e, bits);
        else if (mode == kKeysExact)
            find_first<EB, kKeysExact>(saved, best_key, su, e, bits);
        else find_first<EB, kKeysNan>(saved, best_key, su, e, bits);
        const int64_t vi = (int64_t)t.v0 + best_group * kGroupVecs + su * kRowThreads + t.tid;
        packed = pack_kc(best_key, col_base + vi * kEpv + e);
    }
}

// One lane's best (key, column) and bits over its share of a tile: the
// tile's 16-byte vectors [split * chunk_vecs, ...) of the row's aligned middle,
// plus the row's unaligned head (split 0) and tail (last split) elements.
//
// kNanPass = false, the first pass.  Each wavefront ranks its first group with
// raw keys; if that group holds a number in [1, +inf] in any lane, raw keys
// rank the wavefront's whole share (every key that can win is then exact),
// else sign-magnitude keys do.  So the tile's greatest key is exact unless the
// tile holds a NaN, and `nan_seen` tells whether the lane's share holds one
// that the greatest key does not show (one with the sign bit set, or any NaN
// among the head and tail elements).
// kNanPass = true: NaN keys, for a tile known to hold a NaN.
template <int EB, bool kNanPass, typename Hook>
__device__ __forceinline__ void tile_best(const unsigned char* row_ptr, const RowGeom& geom,
                                          int64_t vocab, int64_t col_offset, int split,
                                          int splits, int64_t chunk_vecs, int tid,
                                          unsigned long long& packed, uint32_t& bits,
                                          bool& nan_seen, Hook&& after_first_loads) {
    constexpr int kScalarMode = kNanPass ? kKeysNan : kKeysExact;
    TileSpan t;
    t.vec = (const u32x4*)(row_ptr + geom.head * EB);
    t.v0 = (int32_t)(split * chunk_vecs);
    t.v1 = (int32_t)min(split * chunk_vecs + chunk_vecs, geom.nvec);
    t.nv = t.v1 > t.v0 ? t.v1 - t.v0 : 0;
    t.ngroups = (t.nv + kGroupVecs - 1) / kGroupVecs;
    t.tid = tid;
    const int64_t col_base = col_offset + geom.head;

    uint32_t umax = 0;
    if constexpr (kNanPass) {
        rank_share<EB>(t, kKeysNan, col_base, packed, bits, umax, after_first_loads);
    } else {
        rank_share<EB>(t, kKeysChoose, col_base, packed, bits, umax, after_first_loads);
        if constexpr (EB == 2)
            nan_seen = max(umax & 0xffffu, umax >> 16) > KeyTraits<2>::kNegInfPattern;
        else
            nan_seen = umax > KeyTraits<4>::kNegInfPattern;
    }

    // unaligned head and tail elements (at most 16 / EB - 1 of each)
    if (split == 0 && tid < geom.head) {
        int32_t k;
        uint32_t b;
        load_scalar<EB, kScalarMode>(row_ptr + (int64_t)tid * EB, k, b);
        take_better(packed, bits, pack_kc(k, col_offset + tid), b);
        if constexpr (!kNanPass) nan_seen = nan_seen || (b & 0x7fffffffu) > 0x7f800000u;
    }
    if (split == splits - 1 && tid < vocab - geom.tail) {
        const int64_t c = geom.tail + tid;
        int32_t k;
        uint32_t b;
        load_scalar<EB, kScalarMode>(row_ptr + c * EB, k, b);
        take_better(packed, bits, pack_kc(k, col_offset + c), b);
        if constexpr (!kNanPass) nan_seen = nan_seen || (b & 0x7fffffffu) > 0x7f800000u;
    }
}

// ----------------------------------------------------------- stage 1 kernel

// One tile of the row pass, the body of the row kernels.  `logits` rows hold
// columns [col_offset, col_offset + vocab) of the full vocabulary (col_offset
// = 0 and vocab = V unless the rows are one tensor-parallel shard); columns are
// reported globally.  With `partials` set the tile writes a partial (split
// rows, or one shard of each row); otherwise the row is one tile and writes its
// record.  `pre` runs once, right after the tile's first loads are issued (for
// the caller's own loads).  Thread 0 writes; every thread returns.
template <int EB, typename Pre>
__device__ __forceinline__ void row_tile(
    const unsigned char* __restrict__ logits, int64_t vocab, int64_t col_offset, int splits,
    int64_t chunk_vecs, const int32_t* __restrict__ draft_tokens,
    TilePartial* __restrict__ partials, RowRecord* __restrict__ records,
    int32_t* __restrict__ out_argmax, Pre&& pre) {
    constexpr int kEpv = 16 / EB;
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x / splits;
    const int split = (int)(blockIdx.x - row * splits);
    const unsigned char* row_ptr = logits + row * vocab * EB;
    const RowGeom geom = row_geom(row_ptr, vocab, EB);
    const int64_t chunk_cols = chunk_vecs * kEpv;

    // The row's draft token x (uniform) and, in the tile that owns its column,
    // the pattern of z(x).  Both are read after the tile's first loads are
    // issued.  Every lane reads the pattern from one uniform address (the row's
    // first element when the tile does not own x): with no branch around the
    // load nothing waits for it before the ranking, so it overlaps the stream.
    int32_t x = 0;
    bool x_here = false, owns_x = false;
    uint32_t draft_raw = 0;
    auto after_first_loads = [&]() {
        x = draft_tokens[row];
        const int64_t x_local = (int64_t)x - col_offset;
        x_here = x_local >= 0 && x_local < vocab;
        owns_x = x_here && owner_split(x_local, geom, chunk_cols, splits) == split;
        const unsigned char* p = row_ptr + (owns_x ? x_local * EB : 0);
        if constexpr (EB == 2) draft_raw = *(const unsigned short*)p;
        else draft_raw = *(const uint32_t*)p;
        pre();
    };

    // ---- rank the tile (first pass); if it holds a NaN, rank it again to find
    // its first NaN.
    unsigned long long packed;
    uint32_t bits;
    bool nan_seen = false;
    tile_best<EB, false>(row_ptr, geom, vocab, col_offset, split, splits, chunk_vecs, tid, packed,
                         bits, nan_seen, after_first_loads);
    // Every thread learns the tile's best pair and whether any wavefront saw a
    // NaN, so every thread takes the same decision without a second barrier.
    const bool wave_nan = __ballot(nan_seen) != 0ull;
    const bool any_nan = block_reduce(packed, bits, wave_nan);
    if (any_nan || packed_key(packed) > KeyTraits<EB>::kInf) {
        __syncthreads();                 // every thread has read the first reduction
        tile_best<EB, true>(row_ptr, geom, vocab, col_offset, split, splits, chunk_vecs, tid,
                            packed, bits, nan_seen, [] {});
        block_reduce(packed, bits, false);
    }
    if (tid != 0) return;
    const uint32_t draft_bits = owns_x ? (EB == 2 ? draft_raw << 16 : draft_raw) : 0u;

    if (partials != nullptr) {           // combined by the scan
        TilePartial tp;
        tp.packed = packed;
        tp.bits = bits;
        tp.draft_bits = draft_bits;      // meaningful in the owning tile only
        partials[blockIdx.x] = tp;
        return;
    }

    // ---- one tile per row: the row record (one binary32 subtraction)
    const int32_t y = packed_col(packed);
    RowRecord rec;
    if (x_here) {                        // the whole vocabulary: x_here = x in [0, V)
        rec.regret = bits_to_float(bits) - bits_to_float(draft_bits);
        rec.y_flags = (uint32_t)y | ((x != y) ? kMismatchBit : 0u);
    } else {
        rec.regret = __builtin_huge_valf();
        rec.y_flags = (uint32_t)y | kMismatchBit | kBadDraftBit;
    }
    records[row] = rec;
    if (out_argmax) out_argmax[row] = y;
}

// The row pass as its own kernel, followed by the scan kernel.  Block 0 also
// writes the packed row offsets of the requests when `packed_offsets` is set,
// after its first loads are issued: a test of that argument ahead of the row
// pass would make every tile wait for its arguments twice before its first
// load.  Five wavefronts per SIMD: the two load buffers and the clamped offsets
// of the last group fit in 96 VGPRs with no spill (at six, 80 VGPRs, an
// earlier form spilled to scratch and ran 25% slower).
template <int EB>
__global__ __launch_bounds__(kRowThreads) __attribute__((amdgpu_waves_per_eu(5))) void asd_row_kernel(
    const unsigned char* __restrict__ logits, int64_t vocab, int64_t col_offset, int splits,
    int64_t chunk_vecs, const int32_t* __restrict__ draft_tokens,
    TilePartial* __restrict__ partials, RowRecord* __restrict__ records,
    int32_t* __restrict__ out_argmax, int32_t num_requests,
    const int32_t* __restrict__ block_lens, int64_t* __restrict__ packed_offsets) {
    row_tile<EB>(logits, vocab, col_offset, splits, chunk_vecs, draft_tokens, partials, records,
                 out_argmax, [&] {
                     if (blockIdx.x == 0 && packed_offsets != nullptr)
                         write_packed_offsets(num_requests, block_lens, packed_offsets);
                 });
}

// ----------------------------------------------------------- stage 2 kernel

struct ScanArgs {
    int32_t num_requests;
    int32_t request_blocks;      // workgroups that scan requests; the rest write argmax rows
    int64_t total_rows;
    int64_t vocab;
    int elem_bytes;
    int splits;
    int64_t chunk_vecs;
    const unsigned char* logits; // row addresses only (alignment -> split ownership)
    const int32_t* draft_tokens;
    const int32_t* block_lens;
    const int64_t* offsets;
    const float* tau;
    const int32_t* exc_cap;
    float2* budget;
    const RowRecord* records;    // splits == 1 and no shards
    const TilePartial* partials; // split rows: [row][split]; shards: [shard][row]
    int64_t shard_vocab;         // > 0: partials come from vocabulary shards of this width
    const unsigned long long* row_best;   // LM-head pass: each row's greatest (key, column)
    const uint32_t* row_draft_bits;       // LM-head pass: each row's draft logit
    int32_t* commit_tokens;               // commit in the same pass, or nullptr
    int64_t commit_capacity;
    int64_t* commit_seq_len;
    int32_t* commit_done;
    int raw_gate;                         // gate on r <= g (q read as 1)
    int32_t* out_accept_len;
    int32_t* out_next_token;
    float* out_regret;
    int32_t* out_argmax;
};

// Greatest (key, column) of a row's split partials and the gathered draft logit.
__device__ __forceinline__ void combine_row(const ScanArgs& A, int64_t row, int32_t x,
                                            unsigned long long& packed, uint32_t& bits,
                                            uint32_t& draft_bits) {
    const bool x_valid = x >= 0 && (int64_t)x < A.vocab;
    if (A.row_best) {                    // LM-head pass: value bits from the exact key
        packed = A.row_best[row];
        const int32_t key = packed_key(packed);
        bits = key >= 0 ? (uint32_t)key : (0x80000000u | (uint32_t)(-(int64_t)key));
        draft_bits = x_valid ? A.row_draft_bits[row] : 0u;
        return;
    }
    const TilePartial* parts;
    int64_t stride;
    int owner = -1;
    if (A.shard_vocab > 0) {             // shard k holds columns [k W, (k + 1) W)
        parts = A.partials + row;
        stride = A.total_rows;
        if (x_valid) owner = (int)min((int64_t)x / A.shard_vocab, (int64_t)A.splits - 1);
    } else {                             // tiles of one row
        parts = A.partials + row * A.splits;
        stride = 1;
        const unsigned char* row_ptr = A.logits + row * A.vocab * A.elem_bytes;
        const RowGeom geom = row_geom(row_ptr, A.vocab, A.elem_bytes);
        if (x_valid) owner = owner_split(x, geom, A.chunk_vecs * (16 / A.elem_bytes), A.splits);
    }
    packed = 0;
    bits = 0;
    draft_bits = 0;
    // Partials are read eight at a time so that their loads are in flight together.
    for (int s0 = 0; s0 < A.splits; s0 += 8) {
        TilePartial tp[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (s0 + j < A.splits) tp[j] = parts[(s0 + j) * stride];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (s0 + j < A.splits) {
                take_better(packed, bits, tp[j].packed, tp[j].bits);
                if (s0 + j == owner) draft_bits = tp[j].draft_bits;
            }
        }
    }
}

__device__ __forceinline__ uint32_t lane_u32(uint32_t v, int lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// Algorithm 1 for request i, whose rows start at o, by one wavefront: lanes
// are block positions.  Each lane forms its row's record (or combines the
// row's partials); the wavefront walks the mismatches in position order.
// Wave-uniform: every lane of the wavefront calls it with the same i and o.
// The per-request inputs of Algorithm 1 (block length, ledger, gate, cap and
// committed length), loaded together so that their loads are in flight at
// once, ahead of the rows.
struct RequestIn {
    int32_t K_given;
    int32_t M;
    float2 ledger;
    float g;
    int64_t L;
};

__device__ __forceinline__ RequestIn load_request(const ScanArgs& A, int64_t i) {
    RequestIn q;
    q.K_given = A.block_lens[i];
    q.ledger = A.budget[i];
    q.g = A.tau[i];
    q.M = A.exc_cap[i];
    q.L = A.commit_tokens ? A.commit_seq_len[i] : 0;
    return q;
}

__device__ __forceinline__ void scan_request(const ScanArgs& A, int64_t i, int64_t o,
                                             const RequestIn& q) {
    const int lane = threadIdx.x & 63;
    const int32_t K_given = q.K_given;
    const int32_t K = K_given > 0 ? K_given : 0;      // a negative K is read as 0
    const int64_t L = q.L;
    if (K_given < 0 && lane == 0) atomicOr(&asd_error_word, kErrNegativeK);
    if (!(o >= 0 && o + (int64_t)K < A.total_rows)) {
        if (lane == 0) {
            A.out_accept_len[i] = 0;
            A.out_next_token[i] = -1;
            if (A.commit_tokens && A.commit_done) A.commit_done[i] = 0;
            atomicOr(&asd_error_word, kErrRows);
        }
        return;
    }
    const float B = q.ledger.x;
    const float s = q.ledger.y;
    const float g = q.g;
    const int32_t M = q.M;
    const bool strict = (B == 0.0f);   // Algorithm 1: B = 0 -> exact greedy verification

    int32_t a = 0, N = 0, next = -1;
    float C = 0.0f;
    bool done = false;
    for (int64_t c0 = 0; c0 <= K; c0 += 64) {
        const int64_t p = c0 + lane;                  // 0-based position; p == K: bonus row
        const bool have = p <= K;
        const bool is_draft = p < K;
        uint32_t y = 0;
        bool mism = false, bad = false;
        float r = 0.0f;
        if (have) {
            const int64_t row = o + p;
            if (A.records != nullptr) {
                const RowRecord rec = A.records[row];
                y = rec.y_flags & kArgmaxMask;
                mism = (rec.y_flags & kMismatchBit) != 0u;
                bad = (rec.y_flags & kBadDraftBit) != 0u;
                r = rec.regret;
            } else {
                const int32_t x = A.draft_tokens[row];
                unsigned long long packed;
                uint32_t bits, draft_bits;
                combine_row(A, row, x, packed, bits, draft_bits);
                y = (uint32_t)packed_col(packed);
                bad = !(x >= 0 && (int64_t)x < A.vocab);
                mism = bad || (uint32_t)x != y;
                r = bad ? __builtin_huge_valf() : bits_to_float(bits) - bits_to_float(draft_bits);
            }
            if (A.out_regret) A.out_regret[row] = is_draft ? r : 0.0f;
        }
        if (done) continue;

        // Mismatches among this chunk's draft positions, and those that pass
        // the local gate r <= g q (q = K - p, i.e. K - i + 1 for i = p + 1;
        // q = 1 for the raw-gate variant).
        const int32_t q = A.raw_gate ? 1 : K - (int32_t)p;
        const bool gate = (double)r <= (double)g * (double)q;
        const unsigned long long mism_mask = __ballot(is_draft && mism);
        const unsigned long long ok_mask = __ballot(is_draft && mism && !bad && gate);
        int stop = -1;
        if (strict) {
            if (mism_mask) stop = __builtin_ctzll(mism_mask);
        } else {
            for (unsigned long long m = mism_mask; m != 0ull; m &= m - 1ull) {
                const int j = __builtin_ctzll(m);
                const float rj = __builtin_bit_cast(float, lane_u32(__builtin_bit_cast(uint32_t, r), j));
                const float C_new = C + rj;
                const int32_t N_new = N + 1;
                const float s_new = s + C_new;
                if (!(((ok_mask >> j) & 1ull) && s_new <= B && N_new <= M)) {
                    stop = j;
                    break;
                }
                C = C_new;
                N = N_new;
            }
        }
        if (stop >= 0) {                              // first infeasible position
            a = (int32_t)(c0 + stop);
            next = (int32_t)lane_u32(y, stop);         // recovery token y*_{a+1}
            done = true;
        } else if (K - c0 < 64) {                     // the bonus row is in this chunk
            a = K;
            next = (int32_t)lane_u32(y, (int)(K - c0));
            done = true;
        }
    }
    if (lane == 0) {
        if (N > 0) A.budget[i].y = s + C;             // s' = s + C_a
        A.out_accept_len[i] = a;
        A.out_next_token[i] = next;
    }
    if (A.commit_tokens) {
        // The commit (Sec. 3.3): x_1..x_a then y*_{a+1} at the request's
        // committed length, when they fit below capacity.
        const bool ok = next >= 0 && L >= 0 && L + (int64_t)a + 1 <= A.commit_capacity;
        if (ok) {
            int32_t* dst = A.commit_tokens + i * A.commit_capacity + L;
            for (int64_t j = lane; j <= a; j += 64) dst[j] = j < a ? A.draft_tokens[o + j] : next;
        }
        if (lane == 0) {
            if (ok) A.commit_seq_len[i] = L + (int64_t)a + 1;
            if (A.commit_done) A.commit_done[i] = ok ? a + 1 : 0;
            if (!ok) atomicOr(&asd_error_word, kErrCommit);
        }
    }
}

__global__ __launch_bounds__(kScanThreads) void asd_scan_kernel(const ScanArgs A) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    if ((int32_t)blockIdx.x >= A.request_blocks) {
        // Argmax of every row when rows were split (one lane per row).
        const int64_t row = (int64_t)(blockIdx.x - A.request_blocks) * kScanThreads + tid;
        if (row < A.total_rows) {
            unsigned long long packed;
            uint32_t bits, draft_bits;
            combine_row(A, row, -1, packed, bits, draft_bits);
            A.out_argmax[row] = packed_col(packed);
        }
        return;
    }

    const int64_t i = (int64_t)blockIdx.x * (kScanThreads / 64) + wave;   // wave-uniform
    if (i >= A.num_requests) return;
    const RequestIn q = load_request(A, i);
    int64_t o;
    if (A.offsets) {
        o = A.offsets[i];
    } else {
        // Packed layout, few requests: this wavefront sums the row counts of
        // the requests before it.
        long long part = 0;
#pragma unroll 4
        for (int64_t j = lane; j < i; j += 64) {
            const int32_t Kj = A.block_lens[j];
            part += (long long)(Kj > 0 ? Kj : 0) + 1;
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
        o = part;
    }
    scan_request(A, i, o, q);
}

// ---------------------------------------------- single-launch verification
//
// For plans with few tiles and few requests the call is bound by latency, and
// the second launch of the scan is a large share of it.  Here the row pass and
// the scan run in one launch: every tile counts itself done on a counter, with
// release order after its record or partial, and the one tile that finds
// itself last (acquire order) runs Algorithm 1 for every request, one
// wavefront per request, writes the argmax of split rows and resets the
// counter to zero for the next call.  No tile waits for another.  The counter
// must be zero when the call starts: it lives in a header of the library's
// workspaces that is zeroed when they are allocated, and every call leaves it
// at zero.
// Small plans have at most two tiles per CU, so the kernel takes the registers
// it needs (no occupancy bound).
static_assert(kSingleLaunchMaxRequests <= 2 * kWaves, "two requests per wavefront at most");

template <int EB>
__global__ __launch_bounds__(kRowThreads) void asd_row_scan_kernel(const unsigned char* __restrict__ logits, int64_t vocab, int splits,
                    int64_t chunk_vecs, TilePartial* __restrict__ partials,
                    RowRecord* __restrict__ records, unsigned* __restrict__ counter,
                    const ScanArgs A) {
    // Every tile loads the requests' inputs and row offsets during its row pass,
    // right after its first loads are issued (the few requests of a
    // single-launch plan: wavefront w takes requests w and w + 4), so that the
    // last tile's scan waits only for the rows.
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    RequestIn q[2];
    int64_t o[2];
    auto preload = [&]() {
        const int n = A.num_requests;            // <= kSingleLaunchMaxRequests <= 64
        const int32_t Kl = lane < n ? A.block_lens[lane] : 0;
        long long incl = lane < n ? (long long)(Kl > 0 ? Kl : 0) + 1 : 0;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const long long t = __shfl_up(incl, off, 64);
            if (lane >= off) incl += t;
        }
        const long long excl = incl - (lane < n ? (long long)(Kl > 0 ? Kl : 0) + 1 : 0);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int k = wave + 4 * j;
            if (k < n) {
                q[j] = load_request(A, k);
                o[j] = A.offsets ? A.offsets[k] : (int64_t)__shfl(excl, k, 64);
            }
        }
    };
    row_tile<EB>(logits, vocab, 0, splits, chunk_vecs, A.draft_tokens, partials, records,
                 splits == 1 ? A.out_argmax : nullptr, preload);
    __shared__ int s_last;
    if (threadIdx.x == 0) {
        const unsigned prev =
            __hip_atomic_fetch_add(counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        s_last = prev == gridDim.x - 1;
    }
    __syncthreads();
    if (!s_last) return;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");   // every tile's output, for every thread

#pragma unroll
    for (int j = 0; j < 2; ++j)
        if (wave + 4 * j < A.num_requests) scan_request(A, wave + 4 * j, o[j], q[j]);
    if (splits > 1 && A.out_argmax) {
        for (int64_t row = threadIdx.x; row < A.total_rows; row += kRowThreads) {
            unsigned long long packed;
            uint32_t bits, draft_bits;
            combine_row(A, row, -1, packed, bits, draft_bits);
            A.out_argmax[row] = packed_col(packed);
        }
    }
    if (threadIdx.x == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Packed row offsets for the calls that have no row kernel before the scan.
__global__ __launch_bounds__(kRowThreads) void asd_offsets_kernel(
    int32_t num_requests, const int32_t* __restrict__ block_lens, int64_t* __restrict__ offsets) {
    write_packed_offsets(num_requests, block_lens, offsets);
}

ScanArgs scan_args(const CallArgs& a, int64_t rows, int64_t vocab, int elem_bytes) {
    ScanArgs A{};
    A.num_requests = a.num_requests;
    A.request_blocks = (int32_t)((a.num_requests + kScanThreads / 64 - 1) / (kScanThreads / 64));
    A.total_rows = rows;
    A.vocab = vocab;
    A.elem_bytes = elem_bytes;
    A.logits = (const unsigned char*)a.logits;
    A.draft_tokens = a.draft_tokens;
    A.block_lens = a.block_lens;
    A.offsets = a.row_offsets;
    A.tau = a.tau;
    A.exc_cap = a.exc_cap;
    A.budget = a.budget;
    A.out_accept_len = a.out_accept_len;
    A.out_next_token = a.out_next_token;
    A.out_regret = a.out_regret;
    A.out_argmax = a.out_argmax;
    A.commit_tokens = a.commit_tokens;
    A.commit_capacity = a.commit_capacity;
    A.commit_seq_len = a.commit_seq_len;
    A.commit_done = a.commit_done;
    A.raw_gate = a.raw_gate ? 1 : 0;
    return A;
}

hipError_t launch_scan(const ScanArgs& A, bool argmax_rows, hipStream_t stream) {
    const int64_t row_blocks =
        (argmax_rows && A.out_argmax) ? (A.total_rows + kScanThreads - 1) / kScanThreads : 0;
    asd_scan_kernel<<<(unsigned)(A.request_blocks + row_blocks), kScanThreads, 0, stream>>>(A);
    return hipGetLastError();
}

template <typename... Args>
hipError_t launch_row(int elem_bytes, dim3 grid, hipStream_t stream, Args... args) {
    if (elem_bytes == 2)
        asd_row_kernel<2><<<grid, kRowThreads, 0, stream>>>(args...);
    else
        asd_row_kernel<4><<<grid, kRowThreads, 0, stream>>>(args...);
    return hipGetLastError();
}

// --------------------------------------------- opportunity statistic (Eq. 4)

// Counts of Eq. 4 over one batch, one wavefront per request with lanes =
// draft positions.  The ballot of target-greedy drafts gives, for every
// position, the length of the run of greedy drafts that follows it (trailing
// ones of the mask above the position, carried across 64-position chunks from
// the block's end).  A mismatch at position i with r_i <= tau and a following
// run of at least p greedy drafts (which also gives i + p <= K) counts for
// (tau, p); each (tau, p) count of a chunk is one ballot's popcount.  Counts
// gather in LDS, then in the caller's uint64 accumulators.
__global__ __launch_bounds__(kScanThreads) void asd_opportunity_kernel(
    const int32_t* __restrict__ draft_tokens, const int32_t* __restrict__ row_argmax,
    const float* __restrict__ row_regret, int64_t vocab, int32_t num_requests,
    int64_t total_rows, const int32_t* __restrict__ block_lens,
    const int64_t* __restrict__ row_offsets, const float* __restrict__ taus, int32_t num_taus,
    const int32_t* __restrict__ ps, int32_t num_ps, unsigned long long* __restrict__ counts,
    unsigned long long* __restrict__ mismatches, int per_block) {
    __shared__ uint32_t s_counts[kMaxOpportunityPairs];
    __shared__ uint32_t s_mism;
    __shared__ int64_t s_off[kScanThreads];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int pairs = num_taus * num_ps;
    for (int k = tid; k < pairs; k += kScanThreads) s_counts[k] = 0u;
    if (tid == 0) s_mism = 0u;
    const int64_t first = (int64_t)blockIdx.x * per_block;
    const int count = (int)min((int64_t)per_block, (int64_t)num_requests - first);
    block_offsets(num_requests, block_lens, row_offsets, first, count, s_off);   // + barrier

    for (int kq = wave; kq < count; kq += kScanThreads / 64) {    // wave-uniform
        const int64_t i = first + kq;
        const int32_t K = block_lens[i];
        const int64_t o = s_off[kq];
        if (K >= 0 && o >= 0 && o + (int64_t)K < total_rows) {
            // Chunks from the block's end: `carry` = greedy run starting at the
            // first position after the chunk.
            int64_t carry = 0;
            uint32_t mism_total = 0;
            const int64_t nchunks = ((int64_t)K + 63) / 64;
            for (int64_t c = nchunks - 1; c >= 0; --c) {
                const int64_t p = c * 64 + lane;      // 0-based draft position
                const bool have = p < K;
                bool match = false;
                float r = 0.0f;
                if (have) {
                    const int32_t x = draft_tokens[o + p];
                    match = x >= 0 && (int64_t)x < vocab && x == row_argmax[o + p];
                    r = row_regret[o + p];
                }
                const unsigned long long m = __ballot(have && match);
                const int n_here = (int)min((int64_t)64, (int64_t)K - c * 64);
                // trailing ones of the mask above this lane, within the chunk
                const unsigned long long above = lane < 63 ? (m >> (lane + 1)) : 0ull;
                const int ones = (int)__builtin_ctzll(~above);   // < 64 - lane
                const int64_t run = (lane + 1 + ones >= n_here) ? (int64_t)(n_here - 1 - lane) + carry
                                                                : (int64_t)ones;
                const bool mism = have && !match;
                const unsigned long long mm = __ballot(mism);
                mism_total += (uint32_t)__builtin_popcountll(mm);
                if (mm) {
                    for (int a = 0; a < num_taus; ++a) {
                        const float t = taus[a];
                        const unsigned long long ma = __ballot(mism && r <= t);
                        if (!ma) continue;
                        for (int b = 0; b < num_ps; ++b) {
                            const int64_t need = ps[b];
                            const unsigned long long mab = __ballot(mism && r <= t && run >= need);
                            if (lane == 0 && mab)
                                atomicAdd(&s_counts[a * num_ps + b],
                                          (uint32_t)__builtin_popcountll(mab));
                        }
                    }
                }
                // greedy run starting at this chunk's first position
                const int lead = m == ~0ull ? 64 : (int)__builtin_ctzll(~m);
                carry = lead >= n_here ? (int64_t)n_here + carry : (int64_t)lead;
            }
            if (lane == 0 && mism_total) atomicAdd(&s_mism, mism_total);
        }
    }
    __syncthreads();
    for (int k = tid; k < pairs; k += kScanThreads)
        if (s_counts[k]) atomicAdd(counts + k, (unsigned long long)s_counts[k]);
    if (tid == 0 && s_mism) atomicAdd(mismatches, (unsigned long long)s_mism);
}

// --------------------------------------------------------- commit (Sec. 3.3)

// The commit after verification: request i appends its emitted tokens x_1..x_a
// and y*_{a+1} to its token buffer at its committed length and advances that
// length (the extent the target and draft caches keep) by a + 1.  Each
// workgroup takes `per_block` consecutive requests, one wavefront per request
// at a time, lanes writing consecutive tokens.
__global__ __launch_bounds__(kScanThreads) void asd_commit_kernel(
    const int32_t* __restrict__ draft_tokens, const int32_t* __restrict__ block_lens,
    const int64_t* __restrict__ row_offsets, int32_t num_requests, int64_t total_rows,
    const int32_t* __restrict__ accept_len, const int32_t* __restrict__ next_token,
    int32_t* __restrict__ tokens, int64_t capacity, int64_t* __restrict__ seq_len,
    int32_t* __restrict__ committed, int per_block) {
    __shared__ int64_t s_off[kScanThreads];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t first = (int64_t)blockIdx.x * per_block;
    const int count = (int)min((int64_t)per_block, (int64_t)num_requests - first);
    block_offsets(num_requests, block_lens, row_offsets, first, count, s_off);
    for (int k = wave; k < count; k += kScanThreads / 64) {       // wave-uniform
        const int64_t i = first + k;
        const int32_t K_given = block_lens[i];
        const int32_t K = K_given > 0 ? K_given : 0;  // a negative K is read as 0
        const int64_t o = s_off[k];
        const int32_t a = accept_len[i];
        const int32_t next = next_token[i];
        const int64_t L = seq_len[i];
        const bool rows_ok = o >= 0 && o + (int64_t)K < total_rows;
        const bool ok = rows_ok && next >= 0 && L >= 0 && a >= 0 && a <= K &&
                        L + (int64_t)a + 1 <= capacity;
        if (ok) {
            int32_t* dst = tokens + i * capacity + L;
            for (int64_t j = lane; j <= a; j += 64) dst[j] = j < a ? draft_tokens[o + j] : next;
        }
        if (lane == 0) {
            if (ok) seq_len[i] = L + (int64_t)a + 1;
            if (committed) committed[i] = ok ? a + 1 : 0;
            const uint32_t err = (K_given < 0 ? kErrNegativeK : 0u) | (rows_ok ? 0u : kErrRows) |
                                 (rows_ok && next >= 0 && !ok ? kErrCommit : 0u);
            if (err) atomicOr(&asd_error_word, err);
        }
    }
}

// ------------------------------------------- LM-head-fused row pass (MFMA)
//
// z = H W^T for hidden states H [M, K] and output weights W [N, K] (both bf16,
// K-contiguous), in binary32 on v_mfma_f32_32x32x16_bf16, reduced at once to
// each row's greatest (key, column) and the draft token's logit: the M x N
// logits never reach memory.
//
// One workgroup of eight wavefronts per 256 x 256 output tile, two per SIMD:
// wavefront w covers rows 128 (w / 4) .. + 128 and columns 64 (w % 4) .. + 64
// as 4 x 2 MFMA tiles whose 128 accumulators per lane live in AGPRs.  With
// two wavefronts per SIMD one issues while the other waits on its LDS reads or
// at the barrier.  MFMA operand layout (lane l, element e): A row l % 32,
// k = 8 (l / 32) + e; B column l % 32, same k; accumulator v of lane l is row
// 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32.
//
// K steps of 64 go through two LDS stages per operand, each [256 rows][128 B].
// Global -> LDS copies are buffer loads that write LDS directly (no VGPR
// staging); rows past M or N read as zero from the buffer resource.  The 16-B
// chunk c of row r is stored at chunk c ^ lm_swz(r), which keeps both the
// copies and the fragment reads free of bank conflicts.  The two stages are
// distinct arrays so the compiler can tell that a copy into one stage does not
// alias the fragment reads from the other.
//
// Software pipeline of one wavefront: the fragments of the next k-slice are
// read while the current slice's 8 MFMAs issue (one LDS read per MFMA), and
// the barrier that publishes the next stage sits before the last slice's
// MFMAs, so the next stage's first reads and copies overlap them.
constexpr int kLmTile = 256;
constexpr int kLmK = 64;
constexpr int kLmThreads = 512;
constexpr int kLmGroup = kLmheadGroup;   // weight tiles that share a hidden-state row tile

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;
#define ASD_LDS __attribute__((address_space(3)))

constexpr int kRsrcWord3 = 0x00020000;   // raw buffer, 32-bit data format

__device__ __forceinline__ int lm_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// One stage of one operand: tile rows 0..255, columns [k0b / 2, k0b / 2 + 64).
// Row r of the tile starts at byte r * K2 of the buffer.  Wavefronts 0..3, one
// per SIMD, copy; wavefront w copies the 1-KB blocks w, w + 4, ..., w + 28,
// each 8 rows, and lane l fills 16-B position l % 8 of row l / 8 with k-chunk
// (l % 8) ^ lm_swz(row).  The other wavefront of each SIMD issues none, so it
// keeps the matrix core busy while its partner's copies are issued (measured
// faster than all eight wavefronts copying four blocks each).
__device__ __forceinline__ void lm_copy_stage(rsrc_t rs, int K2, int k0b, int wave, int lane,
                                              __bf16* lds) {
    if (wave >= 4) return;
    const int c = (lane & 7) ^ (lane >> 3) ^ (wave & 1);   // (lane & 7) ^ lm_swz(row)
    const int voff = (wave * 8 + (lane >> 3)) * K2 + c * 16;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int blk = u * 4 + wave;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (void ASD_LDS*)(lds + blk * 512), 16,
                                                 voff + u * 32 * K2, k0b, 0, 0);
    }
}

__device__ __forceinline__ void lm_frags(const __bf16* Ar, const __bf16* Br, int p,
                                         bf16x8 (&a)[4], bf16x8 (&b)[2]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *(const bf16x8*)(Ar + i * 32 * kLmK + p);
#pragma unroll
    for (int j = 0; j < 2; ++j) b[j] = *(const bf16x8*)(Br + j * 32 * kLmK + p);
}

__device__ __forceinline__ void lm_mfma8(const bf16x8 (&a)[4], const bf16x8 (&b)[2],
                                         f32x16 (&acc)[4][2]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
}

// Interleave: one MFMA, then one LDS read, six times, then two MFMAs; the
// variant for the stage boundary also spreads a copying wavefront's buffer
// copies.
#define LM_SCHED_READS()                                                     \
    do {                                                                     \
        _Pragma("unroll") for (int t_ = 0; t_ < 6; ++t_) {                   \
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);               \
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);               \
        }                                                                    \
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);                   \
    } while (0)
#define LM_SCHED_READS_COPIES()                                              \
    do {                                                                     \
        _Pragma("unroll") for (int t_ = 0; t_ < 6; ++t_) {                   \
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);               \
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);               \
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);               \
        }                                                                    \
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);                   \
        __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);                   \
    } while (0)

struct LmCtx {
    rsrc_t rh, rw;
    int K2, wave, lane, offA, offB, h, sw;
};

// One K step on stage (Ac, Bc).  Slices 0..2 prefetch the next slice's
// fragments.  Before slice 3 all wavefronts meet: the next stage (An, Bn) is
// complete, (Ac, Bc) is no longer read, so the stage after next is copied into
// it (k0b) and the next stage's first fragments are read.
__device__ __forceinline__ void lm_step(const LmCtx& x, const __bf16* Ac, const __bf16* Bc,
                                        const __bf16* An, const __bf16* Bn, int k0b,
                                        bf16x8 (&fa)[2][4], bf16x8 (&fb)[2][2],
                                        f32x16 (&acc)[4][2]) {
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
        lm_frags(Ac + x.offA, Bc + x.offB, ((2 * (kk + 1) + x.h) ^ x.sw) * 8, fa[(kk + 1) & 1],
                 fb[(kk + 1) & 1]);
        lm_mfma8(fa[kk & 1], fb[kk & 1], acc);
        LM_SCHED_READS();
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this lane's copies of (An, Bn)
    __syncthreads();
    lm_copy_stage(x.rh, x.K2, k0b, x.wave, x.lane, (__bf16*)Ac);
    lm_copy_stage(x.rw, x.K2, k0b, x.wave, x.lane, (__bf16*)Bc);
    lm_frags(An + x.offA, Bn + x.offB, (x.h ^ x.sw) * 8, fa[0], fb[0]);
    lm_mfma8(fa[1], fb[1], acc);
    LM_SCHED_READS_COPIES();
}

__global__ __launch_bounds__(kLmThreads) void asd_lmhead_kernel(
    const unsigned char* __restrict__ hidden, const unsigned char* __restrict__ weight,
    int64_t M, int64_t N, int64_t K, int64_t tiles_m, int64_t tiles,
    const int32_t* __restrict__ draft_tokens, unsigned long long* __restrict__ row_best,
    uint32_t* __restrict__ row_draft_bits) {
    __shared__ __attribute__((aligned(1024))) __bf16 A0[kLmTile * kLmK];
    __shared__ __attribute__((aligned(1024))) __bf16 B0[kLmTile * kLmK];
    __shared__ __attribute__((aligned(1024))) __bf16 A1[kLmTile * kLmK];
    __shared__ __attribute__((aligned(1024))) __bf16 B1[kLmTile * kLmK];
    __shared__ int32_t s_draft[kLmTile];

    // XCD-aware order: workgroup i runs on XCD i % 8, and each XCD takes a run
    // of consecutive positions.  Positions run over groups of kLmGroup weight
    // tiles (slowest), row tiles, then the weight tiles of the group (fastest):
    // the tiles of a group start together and read each hidden-state slice
    // once between them from L2, and a group of weight tiles serves the row
    // tiles that the XCD runs alongside it.
    const int64_t per_xcd = gridDim.x / 8;
    const int64_t linear = (int64_t)(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    const int64_t tiles_n = (N + kLmTile - 1) / kLmTile;
    const int64_t group = linear / (kLmGroup * tiles_m), within = linear % (kLmGroup * tiles_m);
    const int64_t rt = within / kLmGroup, ct = group * kLmGroup + within % kLmGroup;
    if (linear >= tiles || ct >= tiles_n) return;
    const int64_t row0 = rt * kLmTile, col0 = ct * kLmTile;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar LDS targets
    const int wm = wave >> 2, wn = wave & 3, h = lane >> 5;
    if (tid < kLmTile) s_draft[tid] = row0 + tid < M ? draft_tokens[row0 + tid] : -1;

    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = (f32x16)(0.0f);

    LmCtx x;
    x.K2 = (int)(K * 2);
    x.rh = __builtin_amdgcn_make_buffer_rsrc((void*)(hidden + row0 * x.K2), (short)0,
                                             (int)(min((int64_t)kLmTile, M - row0) * x.K2),
                                             kRsrcWord3);
    x.rw = __builtin_amdgcn_make_buffer_rsrc((void*)(weight + col0 * x.K2), (short)0,
                                             (int)(min((int64_t)kLmTile, N - col0) * x.K2),
                                             kRsrcWord3);
    x.wave = wave;
    x.lane = lane;
    x.h = h;
    x.sw = lm_swz(lane & 31);
    x.offA = (wm * 128 + (lane & 31)) * kLmK;
    x.offB = (wn * 64 + (lane & 31)) * kLmK;

    // K / 64 is even.  Copies past the last stage are clamped to it: they
    // refill a stage that is no longer read, and the fragments read after the
    // last stage are never used.
    const int64_t KT = K / kLmK;
    bf16x8 fa[2][4], fb[2][2];
    lm_copy_stage(x.rh, x.K2, 0, wave, lane, A0);
    lm_copy_stage(x.rw, x.K2, 0, wave, lane, B0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    lm_copy_stage(x.rh, x.K2, 2 * kLmK, wave, lane, A1);
    lm_copy_stage(x.rw, x.K2, 2 * kLmK, wave, lane, B1);
    lm_frags(A0 + x.offA, B0 + x.offB, (h ^ x.sw) * 8, fa[0], fb[0]);
    for (int64_t s = 0; s < KT; s += 2) {
        lm_step(x, A0, B0, A1, B1, (int)(min(s + 2, KT - 1) * 2 * kLmK), fa, fb, acc);
        lm_step(x, A1, B1, A0, B0, (int)(min(s + 3, KT - 1) * 2 * kLmK), fa, fb, acc);
    }

    // ---- epilogue, through LDS (the stages are free now).  Four passes, one
    // per 32-row slice i of each wavefront; pass i uses the stage pair i % 2,
    // so one barrier per pass separates its stores from its scans.  E0 holds
    // the slice rows of wm = 0, E1 those of wm = 1, each [32 rows][256
    // columns] of logit bits, with the 16-B chunk c of row lr at chunk c ^
    // ((c >> 4) & 3) ^ 4 (lr & 3) ^ 8 ((lr >> 2) & 1), which keeps the stores
    // free of bank conflicts.  Eight threads then scan each of the 64 rows, 32
    // columns each.
    //
    // A scan ranks raw patterns read as signed integers: per 16-B chunk a
    // signed and an unsigned maximum, and the first chunk with the greatest
    // signed maximum.  When that maximum is a number in [1, +inf] and the
    // unsigned maximum shows no NaN with the sign bit set, it is the exact
    // maximum of the 32 columns and the winning chunk's first element equal
    // to it is their first maximum.  Otherwise (a NaN, no positive number, or
    // columns past N, which take no part in the ranking) the thread ranks its
    // columns again with exact keys.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no copy outlives the main loop
    int wbase[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int col = wn * 64 + j * 32 + (lane & 31);
        const int cl = col >> 2;
        wbase[j] = 4 * 256 * h + ((cl ^ ((cl >> 4) & 3) ^ (h << 3)) << 2) + (col & 3);
    }
    const int rr = tid >> 3, q = tid & 7;                 // scan: slice row, column eighth
    const int lrr = rr & 31;
    const int xr = ((lrr & 3) << 2) ^ (((lrr >> 2) & 1) << 3);
    const int64_t qcol0 = col0 + q * 32;                  // first column of the eighth
    const bool qfull = qcol0 + 32 <= N;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t* const E0 = (uint32_t*)((i & 1) ? A1 : A0);
        uint32_t* const E1 = (uint32_t*)((i & 1) ? B1 : B0);
        uint32_t* const Ew = wm ? E1 : E0;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                // The element is copied out before its bits are taken: a bit
                // cast of the vector element itself read element 0 for every v.
                const float val = acc[i][j][v];
                Ew[(wbase[j] ^ ((v & 3) << 4)) + 256 * (8 * (v >> 2) + (v & 3))] =
                    __float_as_uint(val);
            }
        __syncthreads();
        const int r = (rr >> 5) * 128 + i * 32 + lrr;      // tile row
        const uint32_t* const Er = (rr < 32 ? E0 : E1) + lrr * 256;
        auto chunk = [&](int c) {                          // chunk c of this thread's eighth
            const int cl = q * 8 + c;
            return *(const uint4*)(Er + ((cl ^ ((cl >> 4) & 3) ^ xr) << 2));
        };
        unsigned long long best = 0;                       // ranks below every key
        if (row0 + r < M) {
            int32_t bm = (int32_t)0x80000000;
            uint32_t um = 0;
            int bch = 0;
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const uint4 f = chunk(c);
                const int32_t m = max(max((int32_t)f.x, (int32_t)f.y), max((int32_t)f.z, (int32_t)f.w));
                um = max(um, max(max(f.x, f.y), max(f.z, f.w)));
                if (m > bm) {                              // strict: first chunk on ties
                    bm = m;
                    bch = c;
                }
            }
            int32_t bk;
            int bc;
            if (qfull && bm >= 1 && bm <= KeyTraits<4>::kInf && um <= KeyTraits<4>::kNegInfPattern) {
                const uint4 f = chunk(bch);
                const int e = (int32_t)f.x == bm ? 0 : (int32_t)f.y == bm ? 1 : (int32_t)f.z == bm ? 2 : 3;
                bk = bm;                                   // a positive number's key is its pattern
                bc = bch * 4 + e;
            } else {
                bk = (int32_t)0x80000000;
                bc = 0;
                for (int c = 0; c < 8; ++c) {
                    const uint4 f = chunk(c);
                    const uint32_t fv[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int k = qcol0 + c * 4 + e < N ? f32_key(fv[e]) : (int32_t)0x80000000;
                        if (k > bk) {                      // strict: lowest column on ties
                            bk = k;
                            bc = c * 4 + e;
                        }
                    }
                }
            }
            best = pack_kc(bk, qcol0 + bc);
            const int64_t xo = (int64_t)s_draft[r] - qcol0;
            if (xo >= 0 && xo < 32 && qcol0 + xo < N) {
                const uint4 f = chunk((int)xo >> 2);
                const uint32_t fv[4] = {f.x, f.y, f.z, f.w};
                row_draft_bits[row0 + r] = fv[(int)xo & 3];
            }
        }
        // The eight threads of a row (lanes 8k .. 8k + 7) combine by DPP: the
        // lane pairs and quad pairs of quad_perm, then the mirror within each
        // eight-lane half row.
        best = dpp_umax64<0xb1>(best);                     // quad_perm [1, 0, 3, 2]
        best = dpp_umax64<0x4e>(best);                     // quad_perm [2, 3, 0, 1]
        best = dpp_umax64<0x141>(best);                    // row_half_mirror
        if (q == 0 && row0 + r < M) atomicMax(row_best + row0 + r, best);
    }
}

__global__ void asd_fill_u64_kernel(unsigned long long* p, int64_t n, unsigned long long v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// ------------------------------------------------------- matrix-core probe
//
// The matrix-core work of asd_lmhead_kernel with no memory traffic: a
// workgroup of eight wavefronts, each wavefront issuing 32
// v_mfma_f32_32x32x16_bf16 per K step of 64 into its 4 x 2 accumulator tiles,
// as the LM-head kernel does, with operand fragments held in registers.  Each
// thread reads six fragments once from the caller's buffer and forms four
// fragment sets from them (the elements rotated within each fragment), which
// the steps cycle through, so that the matrix cores see data of the caller's
// distribution (the power a matrix core draws depends on its operands' bits).
// Workgroup w reads the data of workgroup w % 64, which then stays in the
// cache.  Run over as many workgroups and steps as an LM-head launch, its
// duration is the practical matrix-core ceiling of that launch under the
// chip's power limit.  Thread 0 of each workgroup writes the binary32 bits of
// the sum of its accumulators.
constexpr int kProbeSets = 4;
constexpr int kProbeVecs = 6;                  // 16-byte fragments read per thread

template <int R>
__device__ __forceinline__ bf16x8 rotate_elements(bf16x8 v) {
    return __builtin_shufflevector(v, v, R % 8, (R + 1) % 8, (R + 2) % 8, (R + 3) % 8,
                                   (R + 4) % 8, (R + 5) % 8, (R + 6) % 8, (R + 7) % 8);
}

__global__ __launch_bounds__(kLmThreads) void asd_mfma_probe_kernel(
    const bf16x8* __restrict__ operands, int64_t vectors, int64_t steps,
    uint32_t* __restrict__ out) {
    bf16x8 a[kProbeSets][4], b[kProbeSets][2];
    const int64_t first = ((int64_t)(blockIdx.x % 64) * kLmThreads + threadIdx.x) * kProbeVecs;
    bf16x8 f[kProbeVecs];
#pragma unroll
    for (int k = 0; k < kProbeVecs; ++k) f[k] = operands[(first + k) % vectors];
#pragma unroll
    for (int k = 0; k < 6; ++k) {
        bf16x8* const dst0 = k < 4 ? &a[0][k] : &b[0][k - 4];
        bf16x8* const dst1 = k < 4 ? &a[1][k] : &b[1][k - 4];
        bf16x8* const dst2 = k < 4 ? &a[2][k] : &b[2][k - 4];
        bf16x8* const dst3 = k < 4 ? &a[3][k] : &b[3][k - 4];
        *dst0 = f[k];
        *dst1 = rotate_elements<1>(f[k]);
        *dst2 = rotate_elements<2>(f[k]);
        *dst3 = rotate_elements<3>(f[k]);
    }
    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = (f32x16)(0.0f);
    for (int64_t s = 0; s < steps; ++s) {
#pragma unroll
        for (int t = 0; t < kProbeSets; ++t) lm_mfma8(a[t], b[t], acc);
    }
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float x = acc[i][j][v];
                sum += x;
            }
    if (threadIdx.x == 0) out[blockIdx.x] = __float_as_uint(sum);
}

// ------------------------------------------------------- read probe
//
// The row kernel's access pattern with no ranking: one workgroup per row,
// groups of four 16-byte non-temporal loads per lane issued before any wait,
// each vector folded into a per-lane XOR.  Its duration is the practical read
// ceiling of that pattern.  A lane whose fold equals kProbeMark stores it to
// *out (keeps the loads live; callers can plant the mark to check the read).
constexpr uint32_t kProbeMark = 0x9e3779b9u;

__global__ __launch_bounds__(kRowThreads) __attribute__((amdgpu_waves_per_eu(8))) void
asd_read_probe_kernel(const unsigned char* __restrict__ buf, int64_t row_bytes,
                      uint32_t* __restrict__ out) {
    const u32x4* vec = (const u32x4*)(buf + (int64_t)blockIdx.x * row_bytes);
    const int64_t nvec = row_bytes / 16;
    uint32_t acc = 0;
    int64_t i = threadIdx.x;
    for (; i + (kUnroll - 1) * kRowThreads < nvec; i += kGroupVecs) {
        u32x4 r[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) r[u] = __builtin_nontemporal_load(vec + i + u * kRowThreads);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc ^= r[u].x ^ r[u].y ^ r[u].z ^ r[u].w;
    }
    for (; i < nvec; i += kRowThreads) {
        const u32x4 v = __builtin_nontemporal_load(vec + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == kProbeMark) *out = acc;
}

}  // namespace

// ------------------------------------------------------------------ launch

hipError_t launch_verify(const Plan& plan, const CallArgs& a, void* workspace,
                         unsigned* counter, hipStream_t stream) {
    unsigned char* ws = (unsigned char*)workspace;
    RowRecord* records = (RowRecord*)(ws + plan.off_records);
    TilePartial* partials = plan.splits > 1 ? (TilePartial*)(ws + plan.off_partials) : nullptr;

    if (counter != nullptr && single_launch(plan)) {
        ScanArgs A = scan_args(a, plan.rows, plan.vocab, plan.elem_bytes);
        A.splits = plan.splits;
        A.chunk_vecs = plan.chunk_vecs;
        A.offsets = a.row_offsets;                      // NULL: packed, formed in LDS
        A.records = plan.splits == 1 ? records : nullptr;
        A.partials = partials;
        A.shard_vocab = 0;
        const dim3 grid((unsigned)(plan.rows * plan.splits));
        if (plan.elem_bytes == 2)
            asd_row_scan_kernel<2><<<grid, kRowThreads, 0, stream>>>(
                (const unsigned char*)a.logits, plan.vocab, plan.splits, plan.chunk_vecs, partials,
                records, counter, A);
        else
            asd_row_scan_kernel<4><<<grid, kRowThreads, 0, stream>>>(
                (const unsigned char*)a.logits, plan.vocab, plan.splits, plan.chunk_vecs, partials,
                records, counter, A);
        return hipGetLastError();
    }

    int64_t* packed = a.row_offsets ? nullptr : (int64_t*)(ws + plan.off_offsets);

    const dim3 grid((unsigned)(plan.rows * plan.splits));
    int32_t* row_argmax = plan.splits == 1 ? a.out_argmax : nullptr;
    hipError_t err = launch_row(plan.elem_bytes, grid, stream, (const unsigned char*)a.logits,
                                plan.vocab, (int64_t)0, plan.splits, plan.chunk_vecs,
                                a.draft_tokens, partials, records, row_argmax, a.num_requests,
                                a.block_lens, packed);
    if (err != hipSuccess) return err;

    ScanArgs A = scan_args(a, plan.rows, plan.vocab, plan.elem_bytes);
    A.splits = plan.splits;
    A.chunk_vecs = plan.chunk_vecs;
    A.offsets = a.row_offsets ? a.row_offsets : packed;
    A.records = plan.splits == 1 ? records : nullptr;   // record mode only when rows are whole
    A.partials = partials;
    A.shard_vocab = 0;
    return launch_scan(A, plan.splits > 1, stream);
}

hipError_t launch_row_pass(const Plan& plan, const void* logits, const int32_t* draft_tokens,
                          void* out_partials, hipStream_t stream) {
    return launch_row(plan.elem_bytes, dim3((unsigned)(plan.rows * plan.splits)), stream,
                      (const unsigned char*)logits, plan.vocab, (int64_t)0, plan.splits,
                      plan.chunk_vecs, draft_tokens, (TilePartial*)out_partials,
                      (RowRecord*)nullptr, (int32_t*)nullptr, (int32_t)0,
                      (const int32_t*)nullptr, (int64_t*)nullptr);
}

hipError_t launch_shard_argmax(int elem_bytes, const void* shard_logits, int64_t shard_vocab,
                               int64_t vocab_offset, int64_t rows, const int32_t* draft_tokens,
                               void* out_partials, hipStream_t stream) {
    const int64_t nvec = shard_vocab * elem_bytes / 16;
    int64_t chunk = (nvec + kRowThreads - 1) / kRowThreads * kRowThreads;
    if (chunk < kRowThreads) chunk = kRowThreads;
    return launch_row(elem_bytes, dim3((unsigned)rows), stream,
                      (const unsigned char*)shard_logits, shard_vocab, vocab_offset, 1, chunk,
                      draft_tokens, (TilePartial*)out_partials, (RowRecord*)nullptr,
                      (int32_t*)nullptr, (int32_t)0, (const int32_t*)nullptr,
                      (int64_t*)nullptr);
}

hipError_t launch_verify_partials(const void* partials, int num_shards, int64_t shard_vocab,
                                  int64_t vocab, int64_t rows, const CallArgs& a,
                                  int64_t* packed_offsets, hipStream_t stream) {
    if (!a.row_offsets && packed_offsets) {
        asd_offsets_kernel<<<1, kRowThreads, 0, stream>>>(a.num_requests, a.block_lens,
                                                          packed_offsets);
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    ScanArgs A = scan_args(a, rows, vocab, 2);
    A.splits = num_shards;
    A.chunk_vecs = 0;
    A.offsets = a.row_offsets ? a.row_offsets : packed_offsets;   // NULL: summed per wavefront
    A.records = nullptr;
    A.partials = (const TilePartial*)partials;
    A.shard_vocab = shard_vocab;
    return launch_scan(A, true, stream);
}

// Requests per workgroup of the commit and opportunity kernels: one per
// wavefront while the packed layout's per-workgroup prefix sums stay short
// (at most 8,192 requests before a workgroup), else 64, so that those sums
// total about n^2 / 128 loads.
static int requests_per_block(int32_t num_requests, const int64_t* row_offsets) {
    return (row_offsets || num_requests <= 8192) ? kScanThreads / 64 : 64;
}

hipError_t launch_opportunity(const int32_t* draft_tokens, const int32_t* row_argmax,
                              const float* row_regret, int64_t vocab, int32_t num_requests,
                              int64_t total_rows, const int32_t* block_lens,
                              const int64_t* row_offsets, const float* taus, int32_t num_taus,
                              const int32_t* ps, int32_t num_ps, unsigned long long* counts,
                              unsigned long long* mismatches, hipStream_t stream) {
    const int per_block = requests_per_block(num_requests, row_offsets);
    const unsigned blocks = (unsigned)((num_requests + per_block - 1) / per_block);
    asd_opportunity_kernel<<<blocks, kScanThreads, 0, stream>>>(
        draft_tokens, row_argmax, row_regret, vocab, num_requests, total_rows, block_lens,
        row_offsets, taus, num_taus, ps, num_ps, counts, mismatches, per_block);
    return hipGetLastError();
}

hipError_t launch_commit(const int32_t* draft_tokens, const int32_t* block_lens,
                         const int64_t* row_offsets, int32_t num_requests, int64_t total_rows,
                         const int32_t* accept_len, const int32_t* next_token, int32_t* tokens,
                         int64_t capacity, int64_t* seq_len, int32_t* committed,
                         hipStream_t stream) {
    const int per_block = requests_per_block(num_requests, row_offsets);
    const unsigned blocks = (unsigned)((num_requests + per_block - 1) / per_block);
    asd_commit_kernel<<<blocks, kScanThreads, 0, stream>>>(
        draft_tokens, block_lens, row_offsets, num_requests, total_rows, accept_len, next_token,
        tokens, capacity, seq_len, committed, per_block);
    return hipGetLastError();
}

hipError_t launch_lmhead_verify(const void* hidden, const void* weight, int64_t d,
                                int64_t vocab, int64_t rows, const CallArgs& a, void* workspace,
                                hipStream_t stream) {
    unsigned char* ws = (unsigned char*)workspace;
    unsigned long long* best = (unsigned long long*)ws;
    uint32_t* draft_bits = (uint32_t*)(ws + lmhead_draft_offset(rows));
    asd_fill_u64_kernel<<<(unsigned)((rows + 255) / 256), 256, 0, stream>>>(best, rows, 0ull);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const int64_t tiles_m = (rows + kLmTile - 1) / kLmTile;
    // positions: row tiles x the weight tiles rounded up to whole groups
    const int64_t tiles =
        tiles_m * kLmGroup * (((vocab + kLmTile - 1) / kLmTile + kLmGroup - 1) / kLmGroup);
    const int64_t grid = (tiles + 7) / 8 * 8;
    asd_lmhead_kernel<<<(unsigned)grid, kLmThreads, 0, stream>>>(
        (const unsigned char*)hidden, (const unsigned char*)weight, rows, vocab, d, tiles_m,
        tiles, a.draft_tokens, best, draft_bits);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    ScanArgs A = scan_args(a, rows, vocab, 2);
    A.splits = 1;
    A.chunk_vecs = 0;
    A.offsets = a.row_offsets;
    if (!A.offsets && a.num_requests > kWaveOffsetsMaxRequests) {
        int64_t* packed = (int64_t*)(ws + lmhead_offsets_offset(rows));
        asd_offsets_kernel<<<1, kRowThreads, 0, stream>>>(a.num_requests, a.block_lens, packed);
        if ((err = hipGetLastError()) != hipSuccess) return err;
        A.offsets = packed;
    }
    A.records = nullptr;
    A.partials = nullptr;
    A.shard_vocab = 0;
    A.row_best = best;
    A.row_draft_bits = draft_bits;
    return launch_scan(A, true, stream);
}

hipError_t launch_mfma_probe(const void* operands, int64_t vectors, int64_t workgroups,
                             int64_t steps, uint32_t* out, hipStream_t stream) {
    asd_mfma_probe_kernel<<<(unsigned)workgroups, kLmThreads, 0, stream>>>(
        (const bf16x8*)operands, vectors, steps, out);
    return hipGetLastError();
}

hipError_t launch_read_probe(const void* buf, int64_t rows, int64_t row_bytes, uint32_t* out,
                             hipStream_t stream) {
    asd_read_probe_kernel<<<(unsigned)rows, kRowThreads, 0, stream>>>(
        (const unsigned char*)buf, row_bytes, out);
    return hipGetLastError();
}

}  // namespace asd
