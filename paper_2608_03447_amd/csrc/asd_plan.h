// Launch plan and workspace layout shared by the C-ABI host code and the
// gfx950 kernels of the ASD verifier.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace asd {

// Threads per workgroup of the row kernel: four 64-wide wavefronts.
constexpr int kRowThreads = 256;
// Threads of the per-request scan kernel.
constexpr int kScanThreads = 256;
// Largest number of vocabulary splits of one row.
constexpr int kMaxSplits = 64;

// One tile's best candidate when a row is split over several workgroups:
// (key, column) packed so that a larger value means a greater logit and, among
// equal logits, a lower column; the logit's binary32 bit pattern; and, in the
// tile that owns the draft token's column, that column's logit.
struct alignas(16) TilePartial {
    unsigned long long packed;
    uint32_t bits;
    uint32_t draft_bits;
};

// Per-row result consumed by the per-request scan: argmax in the low 30 bits,
// bit 31 = mismatch (draft != argmax), bit 30 = draft id outside [0, V);
// and the regret r = fl32(z(y*) - z(x)).
struct alignas(8) RowRecord {
    uint32_t y_flags;
    float regret;
};

// Bits of the sticky per-device error word (the values of ASD_DEVERR_*).
constexpr uint32_t kErrNegativeK = 1u;   // a request with K < 0, read as K = 0
constexpr uint32_t kErrRows = 2u;        // a request whose rows lie outside the batch
constexpr uint32_t kErrCommit = 4u;      // a verified request whose tokens were not committed

// Address of this device's error word (device memory, 4 bytes), valid on the
// device current at the call.
hipError_t error_word_address(uint32_t** ptr);

// Size of the fixed per-device workspace of asd_verify_static (the value of
// ASD_STATIC_SCRATCH_BYTES).
constexpr size_t kStaticScratchBytes = (size_t)4 << 20;

// Device address of that workspace on the device current at the call, looked
// up once per device and cached.
hipError_t static_scratch_address(void** ptr);

constexpr uint32_t kMismatchBit = 0x80000000u;
constexpr uint32_t kBadDraftBit = 0x40000000u;
constexpr uint32_t kArgmaxMask = 0x3fffffffu;

struct Plan {
    int elem_bytes;          // 2 (bf16) or 4 (f32)
    int64_t vocab;
    int64_t rows;
    int32_t num_requests;
    int splits;              // S >= 1 vocabulary splits per row
    int64_t chunk_vecs;      // 16-byte vectors per split (multiple of kRowThreads)
    // Workspace layout (byte offsets from the workspace base; 256-byte aligned).
    // Nothing in it is carried from one call to the next.
    size_t off_offsets;      // int64 [num_requests]: packed row offsets
    size_t off_records;      // RowRecord [rows] (splits == 1)
    size_t off_partials;     // TilePartial [rows * splits] (splits > 1)
    size_t ws_bytes;
};

// Arguments of one verifier call after host validation.
struct CallArgs {
    const void* logits = nullptr;
    int32_t num_requests = 0;
    const int32_t* draft_tokens = nullptr;
    const int32_t* block_lens = nullptr;
    const int64_t* row_offsets = nullptr;
    const float* tau = nullptr;
    const int32_t* exc_cap = nullptr;
    float2* budget = nullptr;          // (B, s) per request
    int32_t* out_accept_len = nullptr;
    int32_t* out_next_token = nullptr;
    int32_t* out_argmax = nullptr;
    float* out_regret = nullptr;
    bool raw_gate = false;             // gate on r <= g instead of r / q <= g
    // Commit in the same pass (asd_verify_commit); tokens == nullptr: none.
    int32_t* commit_tokens = nullptr;  // [num_requests][commit_capacity]
    int64_t commit_capacity = 0;
    int64_t* commit_seq_len = nullptr; // [num_requests], advanced in place
    int32_t* commit_done = nullptr;    // [num_requests] or nullptr
};

Plan make_plan(int elem_bytes, int64_t vocab, int64_t rows, int32_t num_requests,
               int num_cus);

// Plans small enough for one launch (row pass and scan in one kernel; see
// asd_row_scan_kernel): few tiles, and few requests, since the last tile scans
// every request with its four wavefronts.
constexpr int64_t kSingleLaunchMaxTiles = 512;
constexpr int32_t kSingleLaunchMaxRequests = 8;   // two per wavefront of the last tile
inline bool single_launch(const Plan& p) {
    return p.rows * p.splits <= kSingleLaunchMaxTiles &&
           p.num_requests <= kSingleLaunchMaxRequests;
}

// Bytes of the header in front of every library-owned workspace (and of the
// fixed scratch): the counter of single-launch calls, zero between calls.
constexpr size_t kCounterHeaderBytes = 256;

// `counter`: a zero counter the call may use for the single-launch form (it
// leaves it zero), or nullptr for the two-kernel form.
hipError_t launch_verify(const Plan& plan, const CallArgs& args, void* workspace,
                         unsigned* counter, hipStream_t stream);

// The row pass of `plan` alone: the row kernel on the plan's tile grid, every
// tile writing its TilePartial at out_partials[row * splits + split].
hipError_t launch_row_pass(const Plan& plan, const void* logits, const int32_t* draft_tokens,
                          void* out_partials, hipStream_t stream);

// One vocabulary shard: rows of `shard_vocab` columns that are columns
// [vocab_offset, vocab_offset + shard_vocab) of the full vocabulary.  Writes one
// TilePartial per row.
hipError_t launch_shard_argmax(int elem_bytes, const void* shard_logits, int64_t shard_vocab,
                               int64_t vocab_offset, int64_t rows, const int32_t* draft_tokens,
                               void* out_partials, hipStream_t stream);

// Combine the partials of `num_shards` shards ([shard][row], shard k holding
// columns [k shard_vocab, (k + 1) shard_vocab)) and run Algorithm 1.
// `packed_offsets` (int64 [num_requests]) is scratch for the packed layout; when
// it is NULL too, each scan wavefront sums its request's offset itself (meant
// for at most kWaveOffsetsMaxRequests requests).
constexpr int32_t kWaveOffsetsMaxRequests = 1024;
hipError_t launch_verify_partials(const void* partials, int num_shards, int64_t shard_vocab,
                                  int64_t vocab, int64_t rows, const CallArgs& args,
                                  int64_t* packed_offsets, hipStream_t stream);

// Opportunity statistic (Eq. 4): at most this many (tau, p) pairs per call.
constexpr int kMaxOpportunityPairs = 1024;

hipError_t launch_opportunity(const int32_t* draft_tokens, const int32_t* row_argmax,
                              const float* row_regret, int64_t vocab, int32_t num_requests,
                              int64_t total_rows, const int32_t* block_lens,
                              const int64_t* row_offsets, const float* taus, int32_t num_taus,
                              const int32_t* ps, int32_t num_ps, unsigned long long* counts,
                              unsigned long long* mismatches, hipStream_t stream);

hipError_t launch_commit(const int32_t* draft_tokens, const int32_t* block_lens,
                         const int64_t* row_offsets, int32_t num_requests, int64_t total_rows,
                         const int32_t* accept_len, const int32_t* next_token, int32_t* tokens,
                         int64_t capacity, int64_t* seq_len, int32_t* committed,
                         hipStream_t stream);

// LM-head-fused verification: workspace = uint64 best [rows], uint32 draft
// logits [rows] at lmhead_draft_offset(rows), int64 packed offsets
// [num_requests] at lmhead_offsets_offset(rows).
inline size_t lmhead_draft_offset(int64_t rows) {
    return ((size_t)rows * 8 + 255) / 256 * 256;
}
inline size_t lmhead_offsets_offset(int64_t rows) {
    return lmhead_draft_offset(rows) + ((size_t)rows * 4 + 255) / 256 * 256;
}
inline size_t lmhead_workspace_bytes(int64_t rows, int32_t num_requests) {
    return lmhead_offsets_offset(rows) + ((size_t)num_requests * 8 + 255) / 256 * 256;
}
// LM-head tiles are 256 x 256; grid positions run over whole groups of
// kLmheadGroup weight tiles (the kernel's tile order).
constexpr int kLmheadGroup = 4;
hipError_t launch_lmhead_verify(const void* hidden, const void* weight, int64_t d,
                                int64_t vocab, int64_t rows, const CallArgs& a, void* workspace,
                                hipStream_t stream);

// Matrix-core probe: `workgroups` workgroups of the LM-head kernel's shape, each
// running `steps` K steps of its MFMA work on operands held in registers.
hipError_t launch_mfma_probe(const void* operands, int64_t vectors, int64_t workgroups,
                             int64_t steps, uint32_t* out, hipStream_t stream);

// Read probe: `rows` workgroups each streaming `row_bytes` (a multiple of 16)
// from a 16-byte aligned buffer.
hipError_t launch_read_probe(const void* buf, int64_t rows, int64_t row_bytes, uint32_t* out,
                             hipStream_t stream);

}  // namespace asd
