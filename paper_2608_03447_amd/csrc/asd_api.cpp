// C ABI of the ASD verifier: host-side argument checks, the launch plan, and
// the library-owned per-(device, stream) workspaces.  Kernels are in
// asd_kernels.hip.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>
#include <utility>
#include <vector>

#include "../../include/asd.h"
#include "asd_plan.h"

namespace asd {

static_assert(kStaticScratchBytes == ASD_STATIC_SCRATCH_BYTES,
              "the fixed scratch size of the header and the kernels must agree");

namespace {

size_t align_up(size_t n, size_t a) { return (n + a - 1) / a * a; }

// Tiles the row kernel aims for: at least two rounds of the resident 256-thread
// workgroups per CU (five at the kernel's register budget), so that the last
// round's stragglers are a small share of the stream (measured on MI355X: 4,352 whole rows of 297 KB
// stream best unsplit; 2,112 rows of 607 KB gain 5% from two splits).
constexpr int kTilesPerCu = 16;
// Smallest split worth its own workgroup, in vectors of 16 bytes.  With at
// least as many rows as CUs, 64 KiB: smaller tiles cost more in per-workgroup
// overhead than they recover in balance (544 rows of 297 KB: 4 splits beat 8
// by 4%, cold).  With fewer rows than CUs the call is bound by latency and
// more parallel streams win: 16 KiB (9 rows of 128 KB: 7 splits take 5.2 us,
// whole rows 9.4 us).
constexpr int64_t kMinChunkVecs = 4096;
constexpr int64_t kMinChunkVecsFewRows = 1024;

}  // namespace

Plan make_plan(int elem_bytes, int64_t vocab, int64_t rows, int32_t num_requests,
               int num_cus) {
    Plan p{};
    p.elem_bytes = elem_bytes;
    p.vocab = vocab;
    p.rows = rows;
    p.num_requests = num_requests;
    const int64_t nvec_max = vocab * elem_bytes / 16;
    int64_t splits = 1;
    if (rows > 0) {
        const int64_t want = ((int64_t)num_cus * kTilesPerCu + rows - 1) / rows;
        const int64_t most = nvec_max / (rows < num_cus ? kMinChunkVecsFewRows : kMinChunkVecs);
        splits = want < most ? want : most;
        if (splits > kMaxSplits) splits = kMaxSplits;
        if (splits < 1) splits = 1;
    }
    int64_t chunk = (nvec_max + splits - 1) / splits;
    chunk = (chunk + kRowThreads - 1) / kRowThreads * kRowThreads;
    if (chunk < kRowThreads) chunk = kRowThreads;
    splits = (nvec_max + chunk - 1) / chunk;
    if (splits < 1) splits = 1;
    p.splits = (int)splits;
    p.chunk_vecs = chunk;

    size_t off = 0;
    p.off_offsets = off;
    off = align_up(off + (size_t)num_requests * sizeof(int64_t), 256);
    p.off_records = off;
    off = align_up(off + (size_t)rows * sizeof(RowRecord), 256);
    p.off_partials = off;
    if (p.splits > 1) off = align_up(off + (size_t)rows * p.splits * sizeof(TilePartial), 256);
    p.ws_bytes = off > 0 ? off : 256;
    return p;
}

namespace {

// A library workspace grows by allocating a larger buffer.  The buffers it
// outgrew stay allocated until asd_release: a graph captured earlier may still
// hold their addresses, and work already enqueued may still use them.
struct Workspace {
    void* ptr = nullptr;
    size_t bytes = 0;
    std::vector<void*> retired;
};

std::mutex g_mutex;
std::map<std::pair<int, hipStream_t>, Workspace> g_workspaces;
std::map<int, int> g_cu_count;
std::map<int, uint32_t*> g_error_words;   // device -> address of its error word

asd_status cu_count(int device, int* out) {
    auto it = g_cu_count.find(device);
    if (it != g_cu_count.end()) {
        *out = it->second;
        return ASD_OK;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
        n <= 0)
        return ASD_EHIP;
    g_cu_count[device] = n;
    *out = n;
    return ASD_OK;
}

int elem_bytes_of(asd_dtype dtype) {
    switch (dtype) {
        case ASD_F32: return 4;
        case ASD_BF16: return 2;
        default: return 0;
    }
}

// Checks every argument the host can see; nothing is launched on failure.
asd_status check_args(const void* logits, asd_dtype dtype, int64_t vocab, int32_t num_requests,
                      int64_t total_rows, const int32_t* draft_tokens, const int32_t* block_lens,
                      const float* tau, const int32_t* exc_cap, const asd_budget* budget,
                      const int32_t* out_accept_len, const int32_t* out_next_token) {
    const int eb = elem_bytes_of(dtype);
    if (eb == 0) return ASD_EDTYPE;
    if (vocab < 1 || vocab >= ((int64_t)1 << 30)) return ASD_EINVAL;
    if (num_requests < 0 || total_rows < (int64_t)num_requests) return ASD_EINVAL;
    if (total_rows >= ((int64_t)1 << 31)) return ASD_EINVAL;
    if (num_requests == 0) return ASD_OK;
    if (!logits || !draft_tokens || !block_lens || !tau || !exc_cap || !budget ||
        !out_accept_len || !out_next_token)
        return ASD_EINVAL;
    if (((uintptr_t)logits % (uintptr_t)eb) != 0) return ASD_EINVAL;
    if (total_rows > INT64_MAX / vocab / eb) return ASD_EINVAL;
    return ASD_OK;
}

// The counter of the single-launch form for a call on stream `s`, or nullptr
// for the two-launch form.  Eager small calls are bound by host launches, so
// one launch wins (workload 1, eager: 12.6 against 15.3 us per call); inside a
// captured graph launches cost little and the two kernels are faster than one
// whose last tile runs the scan after every tile's release (7.7 against 9.4
// us per round), so a call being captured takes two launches.
unsigned* single_launch_counter(hipStream_t s, unsigned* counter) {
    if (counter == nullptr) return nullptr;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone)
        return nullptr;
    return counter;
}

asd_status enqueue(const void* logits, asd_dtype dtype, int64_t vocab, int32_t num_requests,
                   int64_t total_rows, const int32_t* draft_tokens, const int32_t* block_lens,
                   const int64_t* row_offsets, const float* tau, const int32_t* exc_cap,
                   asd_budget* budget, int32_t* out_accept_len, int32_t* out_next_token,
                   int32_t* out_argmax, float* out_regret, hipStream_t stream, const Plan& plan,
                   void* workspace, unsigned* counter, int32_t* commit_tokens = nullptr,
                   int64_t commit_capacity = 0,
                   int64_t* commit_seq_len = nullptr, int32_t* commit_done = nullptr,
                   bool raw_gate = false) {
    CallArgs a;
    a.logits = logits;
    a.num_requests = num_requests;
    a.draft_tokens = draft_tokens;
    a.block_lens = block_lens;
    a.row_offsets = row_offsets;
    a.tau = tau;
    a.exc_cap = exc_cap;
    a.budget = reinterpret_cast<float2*>(budget);
    a.out_accept_len = out_accept_len;
    a.out_next_token = out_next_token;
    a.out_argmax = out_argmax;
    a.out_regret = out_regret;
    a.commit_tokens = commit_tokens;
    a.commit_capacity = commit_capacity;
    a.commit_seq_len = commit_seq_len;
    a.commit_done = commit_done;
    a.raw_gate = raw_gate;
    (void)dtype;
    (void)vocab;
    (void)total_rows;
    return launch_verify(plan, a, workspace, single_launch_counter(stream, counter), stream) ==
                   hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status plan_for(asd_dtype dtype, int64_t vocab, int32_t num_requests, int64_t total_rows,
                    Plan* plan) {
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return ASD_EHIP;
    int cus = 0;
    asd_status st;
    {
        std::lock_guard<std::mutex> lock(g_mutex);
        st = cu_count(device, &cus);
    }
    if (st != ASD_OK) return st;
    *plan = make_plan(elem_bytes_of(dtype), vocab, total_rows, num_requests, cus);
    if ((int64_t)plan->rows * plan->splits >= ((int64_t)1 << 31)) return ASD_EINVAL;
    return ASD_OK;
}

// The library-owned workspace of (current device, stream), grown to at least
// `bytes` (and at least doubled, so the retired buffers total less than the
// current one); growth (hipMalloc) is refused during stream capture.  Every
// buffer starts with a header that holds the counter of single-launch calls,
// zeroed when the buffer is allocated (calls leave it zero); `out` is the
// memory after it, `counter` (optional) the header.
asd_status library_workspace(hipStream_t s, size_t bytes, void** out,
                             unsigned** counter = nullptr) {
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return ASD_EHIP;
    std::lock_guard<std::mutex> lock(g_mutex);
    Workspace& w = g_workspaces[std::make_pair(device, s)];
    if (w.bytes < bytes) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(s, &cap) != hipSuccess) return ASD_EHIP;
        if (cap != hipStreamCaptureStatusNone) return ASD_ECAPTURE;
        size_t want = bytes < ((size_t)1 << 20) ? ((size_t)1 << 20) : bytes;
        if (want < 2 * w.bytes) want = 2 * w.bytes;
        want = align_up(want, (size_t)1 << 20);
        void* p = nullptr;
        if (hipMalloc(&p, want + kCounterHeaderBytes) != hipSuccess) return ASD_ENOMEM;
        if (hipMemsetAsync(p, 0, kCounterHeaderBytes, s) != hipSuccess) {
            (void)hipFree(p);
            return ASD_EHIP;
        }
        if (w.ptr) w.retired.push_back(w.ptr);
        w.ptr = p;
        w.bytes = want;
    }
    *out = (unsigned char*)w.ptr + kCounterHeaderBytes;
    if (counter) *counter = (unsigned*)w.ptr;
    return ASD_OK;
}

// The caller's workspace when given (size checked; its alignment is checked
// with the other host arguments), else the library's.
// A caller's workspace has any content, so it gets no counter (the two-kernel
// form runs).
asd_status resolve_workspace(hipStream_t s, const Plan& plan, void* workspace,
                             size_t workspace_bytes, void** out, unsigned** counter) {
    if (workspace) {
        if (workspace_bytes < plan.ws_bytes) return ASD_ENOMEM;
        *out = workspace;
        *counter = nullptr;
        return ASD_OK;
    }
    return library_workspace(s, plan.ws_bytes, out, counter);
}

}  // namespace
}  // namespace asd

using namespace asd;

extern "C" {

asd_status asd_verify(const void* logits, asd_dtype dtype, int64_t vocab, int32_t num_requests,
                      int64_t total_rows, const int32_t* draft_tokens, const int32_t* block_lens,
                      const int64_t* row_offsets, const float* tau, const int32_t* exc_cap,
                      asd_budget* budget_inout, int32_t* out_accept_len,
                      int32_t* out_next_token, int32_t* out_argmax, float* out_regret,
                      void* stream) {
    asd_status st = check_args(logits, dtype, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK || num_requests == 0) return st;
    Plan plan;
    if ((st = plan_for(dtype, vocab, num_requests, total_rows, &plan)) != ASD_OK) return st;

    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    unsigned* counter = nullptr;
    if ((st = library_workspace(s, plan.ws_bytes, &ws, &counter)) != ASD_OK) return st;
    return enqueue(logits, dtype, vocab, num_requests, total_rows, draft_tokens, block_lens,
                   row_offsets, tau, exc_cap, budget_inout, out_accept_len, out_next_token,
                   out_argmax, out_regret, s, plan, ws, counter);
}

size_t asd_workspace_bytes(asd_dtype dtype, int64_t vocab, int32_t num_requests,
                           int64_t total_rows) {
    if (elem_bytes_of(dtype) == 0 || vocab < 1 || vocab >= ((int64_t)1 << 30) ||
        num_requests < 0 || total_rows < (int64_t)num_requests ||
        total_rows >= ((int64_t)1 << 31))
        return 0;
    Plan plan;
    if (plan_for(dtype, vocab, num_requests, total_rows, &plan) != ASD_OK) return 0;
    return plan.ws_bytes;
}

asd_status asd_verify_ws(const void* logits, asd_dtype dtype, int64_t vocab,
                         int32_t num_requests, int64_t total_rows, const int32_t* draft_tokens,
                         const int32_t* block_lens, const int64_t* row_offsets, const float* tau,
                         const int32_t* exc_cap, asd_budget* budget_inout,
                         int32_t* out_accept_len, int32_t* out_next_token, int32_t* out_argmax,
                         float* out_regret, void* stream, void* workspace,
                         size_t workspace_bytes) {
    asd_status st = check_args(logits, dtype, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK || num_requests == 0) return st;
    if (!workspace || ((uintptr_t)workspace & 255) != 0) return ASD_EINVAL;
    Plan plan;
    if ((st = plan_for(dtype, vocab, num_requests, total_rows, &plan)) != ASD_OK) return st;
    if (workspace_bytes < plan.ws_bytes) return ASD_ENOMEM;
    return enqueue(logits, dtype, vocab, num_requests, total_rows, draft_tokens, block_lens,
                   row_offsets, tau, exc_cap, budget_inout, out_accept_len, out_next_token,
                   out_argmax, out_regret, (hipStream_t)stream, plan, workspace, nullptr);
}

asd_status asd_verify_ex(const void* logits, asd_dtype dtype, int64_t vocab,
                         int32_t num_requests, int64_t total_rows, const int32_t* draft_tokens,
                         const int32_t* block_lens, const int64_t* row_offsets, const float* tau,
                         const int32_t* exc_cap, asd_budget* budget_inout,
                         int32_t* out_accept_len, int32_t* out_next_token, int32_t* out_argmax,
                         float* out_regret, uint32_t flags, void* stream, void* workspace,
                         size_t workspace_bytes) {
    asd_status st = check_args(logits, dtype, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK) return st;
    if ((flags & ~(uint32_t)ASD_GATE_RAW) != 0) return ASD_EINVAL;
    if (num_requests == 0) return ASD_OK;
    if (workspace && ((uintptr_t)workspace & 255) != 0) return ASD_EINVAL;
    Plan plan;
    if ((st = plan_for(dtype, vocab, num_requests, total_rows, &plan)) != ASD_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    unsigned* counter = nullptr;
    if ((st = resolve_workspace(s, plan, workspace, workspace_bytes, &ws, &counter)) != ASD_OK)
        return st;
    return enqueue(logits, dtype, vocab, num_requests, total_rows, draft_tokens, block_lens,
                   row_offsets, tau, exc_cap, budget_inout, out_accept_len, out_next_token,
                   out_argmax, out_regret, s, plan, ws, counter, nullptr, 0, nullptr, nullptr,
                   (flags & ASD_GATE_RAW) != 0);
}

asd_status asd_verify_static(const void* logits, asd_dtype dtype, int64_t vocab,
                             int32_t num_requests, int64_t total_rows,
                             const int32_t* draft_tokens, const int32_t* block_lens,
                             const int64_t* row_offsets, const float* tau,
                             const int32_t* exc_cap, asd_budget* budget_inout,
                             int32_t* out_accept_len, int32_t* out_next_token,
                             int32_t* out_argmax, float* out_regret, void* stream) {
    asd_status st = check_args(logits, dtype, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK || num_requests == 0) return st;
    Plan plan;
    if ((st = plan_for(dtype, vocab, num_requests, total_rows, &plan)) != ASD_OK) return st;
    if (plan.ws_bytes > kStaticScratchBytes - kCounterHeaderBytes) return ASD_ESCRATCH;
    void* base = nullptr;
    if (static_scratch_address(&base) != hipSuccess) return ASD_EHIP;
    // the scratch starts with the single-launch counter (zero at load, left
    // zero by every call), then the call's workspace
    return enqueue(logits, dtype, vocab, num_requests, total_rows, draft_tokens, block_lens,
                   row_offsets, tau, exc_cap, budget_inout, out_accept_len, out_next_token,
                   out_argmax, out_regret, (hipStream_t)stream, plan,
                   (unsigned char*)base + kCounterHeaderBytes, (unsigned*)base);
}

asd_status asd_device_error(uint32_t* out_word, int32_t clear, void* stream) {
    if (!out_word) return ASD_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess) return ASD_EHIP;
    if (cap != hipStreamCaptureStatusNone) return ASD_ECAPTURE;
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return ASD_EHIP;
    uint32_t* word = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_mutex);
        auto it = g_error_words.find(device);
        if (it == g_error_words.end()) {
            if (error_word_address(&word) != hipSuccess || !word) return ASD_EHIP;
            g_error_words[device] = word;
        } else {
            word = it->second;
        }
    }
    uint32_t host = 0;
    if (hipMemcpyAsync(&host, word, sizeof host, hipMemcpyDeviceToHost, s) != hipSuccess)
        return ASD_EHIP;
    if (clear && hipMemsetAsync(word, 0, sizeof host, s) != hipSuccess) return ASD_EHIP;
    if (hipStreamSynchronize(s) != hipSuccess) return ASD_EHIP;
    *out_word = host;
    return ASD_OK;
}

asd_status asd_shard_argmax(const void* shard_logits, asd_dtype dtype, int64_t shard_vocab,
                            int64_t vocab_offset, int64_t vocab, int64_t total_rows,
                            const int32_t* draft_tokens, asd_row_partial* out_partials,
                            void* stream) {
    const int eb = elem_bytes_of(dtype);
    if (eb == 0) return ASD_EDTYPE;
    if (vocab < 1 || vocab >= ((int64_t)1 << 30) || shard_vocab < 1 || vocab_offset < 0 ||
        vocab_offset + shard_vocab > vocab)
        return ASD_EINVAL;
    if (total_rows < 1 || total_rows >= ((int64_t)1 << 31)) return ASD_EINVAL;
    if (!shard_logits || !draft_tokens || !out_partials) return ASD_EINVAL;
    if (((uintptr_t)shard_logits % (uintptr_t)eb) != 0 || ((uintptr_t)out_partials & 15) != 0)
        return ASD_EINVAL;
    return launch_shard_argmax(eb, shard_logits, shard_vocab, vocab_offset, total_rows,
                               draft_tokens, out_partials, (hipStream_t)stream) == hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

int32_t asd_row_splits(asd_dtype dtype, int64_t vocab, int64_t total_rows) {
    if (elem_bytes_of(dtype) == 0 || vocab < 1 || vocab >= ((int64_t)1 << 30) ||
        total_rows < 1 || total_rows >= ((int64_t)1 << 31))
        return 0;
    Plan plan;
    if (plan_for(dtype, vocab, 0, total_rows, &plan) != ASD_OK) return 0;
    return plan.splits;
}

asd_status asd_row_pass(const void* logits, asd_dtype dtype, int64_t vocab, int64_t total_rows,
                        const int32_t* draft_tokens, asd_row_partial* out_partials,
                        void* stream) {
    const int eb = elem_bytes_of(dtype);
    if (eb == 0) return ASD_EDTYPE;
    if (vocab < 1 || vocab >= ((int64_t)1 << 30)) return ASD_EINVAL;
    if (total_rows < 1 || total_rows >= ((int64_t)1 << 31)) return ASD_EINVAL;
    if (!logits || !draft_tokens || !out_partials) return ASD_EINVAL;
    if (((uintptr_t)logits % (uintptr_t)eb) != 0 || ((uintptr_t)out_partials & 15) != 0)
        return ASD_EINVAL;
    Plan plan;
    asd_status st;
    if ((st = plan_for(dtype, vocab, 0, total_rows, &plan)) != ASD_OK) return st;
    return launch_row_pass(plan, logits, draft_tokens, out_partials, (hipStream_t)stream) ==
                   hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status asd_verify_partials(const asd_row_partial* partials, int32_t num_shards,
                               int64_t shard_vocab, int64_t vocab, int32_t num_requests,
                               int64_t total_rows, const int32_t* draft_tokens,
                               const int32_t* block_lens, const int64_t* row_offsets,
                               const float* tau, const int32_t* exc_cap,
                               asd_budget* budget_inout, int32_t* out_accept_len,
                               int32_t* out_next_token, int32_t* out_argmax, float* out_regret,
                               void* stream) {
    asd_status st = check_args(partials, ASD_F32, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK || num_requests == 0) return st;
    if (num_shards < 1 || num_shards > 4096 || shard_vocab < 1 ||
        (int64_t)(num_shards - 1) * shard_vocab >= vocab ||
        (int64_t)num_shards * shard_vocab < vocab)
        return ASD_EINVAL;
    if (((uintptr_t)partials & 15) != 0) return ASD_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    if (!row_offsets && num_requests > kWaveOffsetsMaxRequests) {
        if ((st = library_workspace(s, align_up((size_t)num_requests * sizeof(int64_t), 256),
                                    &ws)) != ASD_OK)
            return st;
    }
    CallArgs a{};
    a.logits = nullptr;
    a.num_requests = num_requests;
    a.draft_tokens = draft_tokens;
    a.block_lens = block_lens;
    a.row_offsets = row_offsets;
    a.tau = tau;
    a.exc_cap = exc_cap;
    a.budget = reinterpret_cast<float2*>(budget_inout);
    a.out_accept_len = out_accept_len;
    a.out_next_token = out_next_token;
    a.out_argmax = out_argmax;
    a.out_regret = out_regret;
    return launch_verify_partials(partials, num_shards, shard_vocab, vocab, total_rows, a,
                                  (int64_t*)ws, s) == hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status asd_opportunity(const int32_t* draft_tokens, const int32_t* row_argmax,
                           const float* row_regret, int64_t vocab, int32_t num_requests,
                           int64_t total_rows, const int32_t* block_lens,
                           const int64_t* row_offsets, const float* taus, int32_t num_taus,
                           const int32_t* ps, int32_t num_ps, uint64_t* counts,
                           uint64_t* mismatches, void* stream) {
    if (vocab < 1 || vocab >= ((int64_t)1 << 30)) return ASD_EINVAL;
    if (num_requests < 0 || total_rows < (int64_t)num_requests ||
        total_rows >= ((int64_t)1 << 31))
        return ASD_EINVAL;
    if (num_taus < 1 || num_ps < 1 || (int64_t)num_taus * num_ps > kMaxOpportunityPairs)
        return ASD_EINVAL;
    if (num_requests == 0) return ASD_OK;
    if (!draft_tokens || !row_argmax || !row_regret || !block_lens || !taus || !ps || !counts ||
        !mismatches)
        return ASD_EINVAL;
    return launch_opportunity(draft_tokens, row_argmax, row_regret, vocab, num_requests,
                              total_rows, block_lens, row_offsets, taus, num_taus, ps, num_ps,
                              (unsigned long long*)counts, (unsigned long long*)mismatches,
                              (hipStream_t)stream) == hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status asd_commit(const int32_t* draft_tokens, const int32_t* block_lens,
                      const int64_t* row_offsets, int32_t num_requests, int64_t total_rows,
                      const int32_t* accept_len, const int32_t* next_token, int32_t* tokens,
                      int64_t capacity, int64_t* seq_len, int32_t* out_committed, void* stream) {
    if (num_requests < 0 || total_rows < (int64_t)num_requests ||
        total_rows >= ((int64_t)1 << 31) || capacity < 1)
        return ASD_EINVAL;
    if (num_requests == 0) return ASD_OK;
    if (!draft_tokens || !block_lens || !accept_len || !next_token || !tokens || !seq_len)
        return ASD_EINVAL;
    if (capacity > INT64_MAX / num_requests) return ASD_EINVAL;
    return launch_commit(draft_tokens, block_lens, row_offsets, num_requests, total_rows,
                         accept_len, next_token, tokens, capacity, seq_len, out_committed,
                         (hipStream_t)stream) == hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status asd_verify_commit(const void* logits, asd_dtype dtype, int64_t vocab,
                             int32_t num_requests, int64_t total_rows,
                             const int32_t* draft_tokens, const int32_t* block_lens,
                             const int64_t* row_offsets, const float* tau,
                             const int32_t* exc_cap, asd_budget* budget_inout,
                             int32_t* out_accept_len, int32_t* out_next_token,
                             int32_t* out_argmax, float* out_regret, int32_t* tokens,
                             int64_t capacity, int64_t* seq_len, int32_t* out_committed,
                             void* stream, void* workspace, size_t workspace_bytes) {
    asd_status st = check_args(logits, dtype, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK) return st;
    if (capacity < 1) return ASD_EINVAL;
    if (num_requests == 0) return ASD_OK;
    if (!tokens || !seq_len || capacity > INT64_MAX / num_requests) return ASD_EINVAL;
    if (workspace && ((uintptr_t)workspace & 255) != 0) return ASD_EINVAL;
    Plan plan;
    if ((st = plan_for(dtype, vocab, num_requests, total_rows, &plan)) != ASD_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    unsigned* counter = nullptr;
    if ((st = resolve_workspace(s, plan, workspace, workspace_bytes, &ws, &counter)) != ASD_OK)
        return st;
    return enqueue(logits, dtype, vocab, num_requests, total_rows, draft_tokens, block_lens,
                   row_offsets, tau, exc_cap, budget_inout, out_accept_len, out_next_token,
                   out_argmax, out_regret, s, plan, ws, counter, tokens, capacity, seq_len,
                   out_committed);
}

asd_status asd_lmhead_verify(const void* hidden, const void* weight, int64_t d, int64_t vocab,
                             int32_t num_requests, int64_t total_rows,
                             const int32_t* draft_tokens, const int32_t* block_lens,
                             const int64_t* row_offsets, const float* tau,
                             const int32_t* exc_cap, asd_budget* budget_inout,
                             int32_t* out_accept_len, int32_t* out_next_token,
                             int32_t* out_argmax, float* out_regret, void* stream) {
    asd_status st = check_args(hidden, ASD_BF16, vocab, num_requests, total_rows, draft_tokens,
                               block_lens, tau, exc_cap, budget_inout, out_accept_len,
                               out_next_token);
    if (st != ASD_OK || num_requests == 0) return st;
    if (!weight || d < 128 || d % 128 != 0 || d > ((int64_t)1 << 20)) return ASD_EINVAL;
    if (((uintptr_t)hidden & 15) != 0 || ((uintptr_t)weight & 15) != 0) return ASD_EINVAL;
    // grid positions: row tiles x weight tiles rounded up to whole groups
    const int64_t tiles = ((total_rows + 255) / 256) * kLmheadGroup *
                          (((vocab + 255) / 256 + kLmheadGroup - 1) / kLmheadGroup);
    if (tiles >= ((int64_t)1 << 31) - 8) return ASD_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    void* ws = nullptr;
    if ((st = library_workspace(s, lmhead_workspace_bytes(total_rows, num_requests), &ws)) !=
        ASD_OK)
        return st;
    CallArgs a{};
    a.logits = nullptr;
    a.num_requests = num_requests;
    a.draft_tokens = draft_tokens;
    a.block_lens = block_lens;
    a.row_offsets = row_offsets;
    a.tau = tau;
    a.exc_cap = exc_cap;
    a.budget = reinterpret_cast<float2*>(budget_inout);
    a.out_accept_len = out_accept_len;
    a.out_next_token = out_next_token;
    a.out_argmax = out_argmax;
    a.out_regret = out_regret;
    return launch_lmhead_verify(hidden, weight, d, vocab, total_rows, a, ws, s) == hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status asd_mfma_probe(const void* operands, int64_t vectors, int64_t workgroups,
                          int64_t steps, uint32_t* out, void* stream) {
    if (!operands || !out || ((uintptr_t)operands & 15) != 0) return ASD_EINVAL;
    if (vectors < 6 || workgroups < 1 || workgroups >= ((int64_t)1 << 31) || steps < 1)
        return ASD_EINVAL;
    return launch_mfma_probe(operands, vectors, workgroups, steps, out, (hipStream_t)stream) ==
                   hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

asd_status asd_read_probe(const void* buf, int64_t rows, int64_t row_bytes, uint32_t* out_word,
                          void* stream) {
    if (!buf || !out_word || ((uintptr_t)buf & 15) != 0) return ASD_EINVAL;
    if (rows < 1 || rows >= ((int64_t)1 << 31) || row_bytes < 16 || row_bytes % 16 != 0 ||
        row_bytes > INT64_MAX / rows)
        return ASD_EINVAL;
    return launch_read_probe(buf, rows, row_bytes, out_word, (hipStream_t)stream) == hipSuccess
               ? ASD_OK
               : ASD_EHIP;
}

const char* asd_status_string(asd_status status) {
    switch (status) {
        case ASD_OK: return "ASD_OK";
        case ASD_EINVAL: return "ASD_EINVAL: invalid argument";
        case ASD_EDTYPE: return "ASD_EDTYPE: unknown logits dtype";
        case ASD_ENOMEM: return "ASD_ENOMEM: workspace allocation failed or too small";
        case ASD_EHIP: return "ASD_EHIP: HIP runtime error";
        case ASD_ECAPTURE: return "ASD_ECAPTURE: workspace must grow during stream capture";
        case ASD_ESCRATCH:
            return "ASD_ESCRATCH: the call needs more workspace than the fixed scratch of "
                   "asd_verify_static holds";
        default: return "ASD: unknown status";
    }
}

// The build passes the hash of the sources it compiled; the binding compares
// it with the sources beside the library.
#ifndef ASD_SOURCE_HASH
#define ASD_SOURCE_HASH "unhashed"
#endif
const char* asd_version(void) { return "asd-mi355x 0.4.0 gfx950 src " ASD_SOURCE_HASH; }

asd_status asd_release(void) {
    std::lock_guard<std::mutex> lock(g_mutex);
    asd_status st = ASD_OK;
    for (auto& kv : g_workspaces) {
        if (kv.second.ptr && hipFree(kv.second.ptr) != hipSuccess) st = ASD_EHIP;
        for (void* old : kv.second.retired)
            if (hipFree(old) != hipSuccess) st = ASD_EHIP;
    }
    g_workspaces.clear();
    return st;
}

}  // extern "C"
