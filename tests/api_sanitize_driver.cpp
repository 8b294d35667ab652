// Host sanitizer driver for the C ABI (include/asd.h).
//
// Built by tests/test_sanitizers.py with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code only.  It calls every entry
// point with each class of argument the host checks reject (all return before
// any HIP call), the size helpers over a range of shapes, and the status and
// version strings.  Only when the process sees no GPU does it also make
// well-formed calls: they then reach the runtime, fail there and must report
// ASD_EHIP or ASD_ENOMEM without touching the (fake) device pointers.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "asd.h"

namespace {

int failures = 0;

void expect(asd_status got, asd_status want, const char* what) {
    if (got != want) {
        std::fprintf(stderr, "%s: got %s, want %s\n", what, asd_status_string(got),
                     asd_status_string(want));
        ++failures;
    }
}

template <typename T>
T* fake(uintptr_t a) {
    return reinterpret_cast<T*>(a);
}

}  // namespace

int main() {
    const void* L = fake<const void>(0x10000);
    const int32_t* D = fake<const int32_t>(0x20000);
    const int32_t* K = fake<const int32_t>(0x30000);
    const float* T = fake<const float>(0x40000);
    const int32_t* M = fake<const int32_t>(0x50000);
    asd_budget* B = fake<asd_budget>(0x60000);
    int32_t* A = fake<int32_t>(0x70000);
    int32_t* X = fake<int32_t>(0x80000);

    // asd_verify: host-checkable errors, nothing launched
    expect(asd_verify(nullptr, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr,
                      nullptr, nullptr), ASD_EINVAL, "verify null logits");
    expect(asd_verify(L, -1, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                      nullptr), ASD_EDTYPE, "verify dtype -1");
    expect(asd_verify(L, ASD_F32, 0, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                      nullptr), ASD_EINVAL, "verify vocab 0");
    expect(asd_verify(L, ASD_F32, 100, 3, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                      nullptr), ASD_EINVAL, "verify rows < requests");
    expect(asd_verify(fake<const void>(0x10002), ASD_F32, 100, 1, 2, D, K, nullptr, T, M, B, A,
                      X, nullptr, nullptr, nullptr), ASD_EINVAL, "verify f32 base not 4-aligned");
    expect(asd_verify(fake<const void>(0x10001), ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A,
                      X, nullptr, nullptr, nullptr), ASD_EINVAL, "verify bf16 base odd");
    expect(asd_verify(L, ASD_F32, 100, 1, 2, nullptr, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                      nullptr), ASD_EINVAL, "verify null draft");
    expect(asd_verify(L, ASD_F32, 100, 0, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                      nullptr, nullptr, nullptr, nullptr, nullptr), ASD_OK, "verify empty");
    expect(asd_verify_ws(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                         nullptr, nullptr, 1 << 20), ASD_EINVAL, "verify_ws null workspace");

    // flags and the device error word
    expect(asd_verify_ex(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                         2u, nullptr, nullptr, 0), ASD_EINVAL, "verify_ex unknown flag");
    expect(asd_verify_ex(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                         ASD_GATE_RAW, nullptr, fake<void>(0x90010), 1 << 20), ASD_EINVAL,
           "verify_ex misaligned workspace");
    expect(asd_verify_ex(L, ASD_BF16, 100, 0, 0, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                         ASD_GATE_RAW, nullptr, nullptr, 0), ASD_OK, "verify_ex empty");
    expect(asd_device_error(nullptr, 1, nullptr), ASD_EINVAL, "device_error null output");
    expect(asd_verify_static(nullptr, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr,
                             nullptr, nullptr),
           ASD_EINVAL, "verify_static null logits");
    expect(asd_verify_static(L, 9, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                             nullptr),
           ASD_EDTYPE, "verify_static bad dtype");
    expect(asd_verify_static(L, ASD_F32, 100, 0, 0, nullptr, nullptr, nullptr, nullptr, nullptr,
                             nullptr, nullptr, nullptr, nullptr, nullptr, nullptr),
           ASD_OK, "verify_static empty batch");
    expect(asd_mfma_probe(nullptr, 24, 1, 1, fake<uint32_t>(0xe0000), nullptr), ASD_EINVAL,
           "mfma_probe null operands");
    expect(asd_mfma_probe(fake<const void>(0x10008), 24, 1, 1, fake<uint32_t>(0xe0000), nullptr),
           ASD_EINVAL, "mfma_probe misaligned");
    expect(asd_mfma_probe(L, 5, 1, 1, fake<uint32_t>(0xe0000), nullptr), ASD_EINVAL,
           "mfma_probe too few vectors");
    expect(asd_mfma_probe(L, 24, 1, 0, fake<uint32_t>(0xe0000), nullptr), ASD_EINVAL,
           "mfma_probe no steps");

    // sharded form
    expect(asd_shard_argmax(L, ASD_BF16, 0, 0, 100, 2, D, fake<asd_row_partial>(0xa0000),
                            nullptr), ASD_EINVAL, "shard width 0");
    expect(asd_shard_argmax(L, ASD_BF16, 50, 60, 100, 2, D, fake<asd_row_partial>(0xa0000),
                            nullptr), ASD_EINVAL, "shard past V");
    expect(asd_verify_partials(nullptr, 2, 50, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr,
                               nullptr, nullptr), ASD_EINVAL, "partials null");

    // the row pass alone
    expect(asd_row_pass(L, ASD_BF16, 0, 2, D, fake<asd_row_partial>(0xa0000), nullptr),
           ASD_EINVAL, "row pass vocab 0");
    expect(asd_row_pass(L, ASD_BF16, 100, 2, D, fake<asd_row_partial>(0xa0008), nullptr),
           ASD_EINVAL, "row pass misaligned partials");
    expect(asd_row_pass(L, (asd_dtype)7, 100, 2, D, fake<asd_row_partial>(0xa0000), nullptr),
           ASD_EDTYPE, "row pass dtype");
    if (asd_row_splits((asd_dtype)7, 100, 2) != 0 || asd_row_splits(ASD_BF16, 100, 0) != 0) {
        std::fprintf(stderr, "FAIL row splits of invalid shapes\n");
        return 1;
    }

    // opportunity and commit
    const float taus[2] = {0.5f, 1.0f};
    const int32_t ps[2] = {0, 1};
    expect(asd_opportunity(D, D, T, 100, 1, 2, K, nullptr, taus, 0, ps, 2,
                           fake<uint64_t>(0xb0000), fake<uint64_t>(0xc0000), nullptr),
           ASD_EINVAL, "opportunity no taus");
    expect(asd_commit(D, K, nullptr, 1, 2, A, X, fake<int32_t>(0xd0000), 0,
                      fake<int64_t>(0xe0000), nullptr, nullptr), ASD_EINVAL, "commit capacity 0");

    // fused output layer
    expect(asd_lmhead_verify(L, L, 64, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr,
                             nullptr), ASD_EINVAL, "lmhead d 64");
    expect(asd_lmhead_verify(L, fake<const void>(0x10008), 256, 100, 1, 2, D, K, nullptr, T, M,
                             B, A, X, nullptr, nullptr, nullptr), ASD_EINVAL, "lmhead misaligned");

    // size helpers: invalid shapes give 0; valid ones need the device's CU count
    if (asd_workspace_bytes(ASD_BF16, 0, 1, 2) != 0 || asd_workspace_bytes(99, 100, 1, 2) != 0 ||
        asd_workspace_bytes(ASD_F32, 100, 3, 2) != 0) {
        std::fprintf(stderr, "workspace_bytes accepted an invalid shape\n");
        ++failures;
    }
    for (int64_t v : {1, 7, 8, 32000, 151936})
        for (int64_t rows : {1, 9, 544, 4352})
            (void)asd_workspace_bytes(ASD_BF16, v, (int32_t)(rows > 4 ? rows / 4 : 1), rows);
    for (int c = -1; c <= 7; ++c) (void)asd_status_string(c);
    expect(asd_verify(L, 7, 100, 1, 2, D, K, nullptr, T, M, B, A, X, nullptr, nullptr, nullptr),
           ASD_EDTYPE, "verify dtype 7");
    (void)asd_version();

    int devices = 0;
    if (hipGetDeviceCount(&devices) != hipSuccess) devices = 0;
    if (devices == 0) {
        // Well-formed calls reach the runtime, which has no device.
        const asd_status s = asd_verify(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X,
                                        nullptr, nullptr, nullptr);
        const asd_status w = asd_verify_ws(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X,
                                           nullptr, nullptr, nullptr, fake<void>(0x90000), 16);
        if (w != ASD_EHIP && w != ASD_ENOMEM) {
            std::fprintf(stderr, "verify_ws without a device returned %s\n", asd_status_string(w));
            ++failures;
        }
        if (s != ASD_EHIP && s != ASD_ENOMEM) {
            std::fprintf(stderr, "verify without a device returned %s\n", asd_status_string(s));
            ++failures;
        }
        const asd_status x = asd_verify_ex(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A, X,
                                           nullptr, nullptr, ASD_GATE_RAW, nullptr, nullptr, 0);
        if (x != ASD_EHIP && x != ASD_ENOMEM) {
            std::fprintf(stderr, "verify_ex without a device returned %s\n", asd_status_string(x));
            ++failures;
        }
        uint32_t word = 0;
        const asd_status e = asd_device_error(&word, 1, nullptr);
        if (e != ASD_EHIP) {
            std::fprintf(stderr, "device_error without a device returned %s\n",
                         asd_status_string(e));
            ++failures;
        }
        const asd_status v = asd_verify_static(L, ASD_BF16, 100, 1, 2, D, K, nullptr, T, M, B, A,
                                               X, nullptr, nullptr, nullptr);
        if (v != ASD_EHIP) {
            std::fprintf(stderr, "verify_static without a device returned %s\n",
                         asd_status_string(v));
            ++failures;
        }
        const asd_status t = asd_lmhead_verify(L, L, 256, 100, 1, 2, D, K, nullptr, T, M, B, A,
                                               X, nullptr, nullptr, nullptr);
        if (t != ASD_EHIP && t != ASD_ENOMEM) {
            std::fprintf(stderr, "lmhead without a device returned %s\n", asd_status_string(t));
            ++failures;
        }
    }
    expect(asd_release(), ASD_OK, "release");
    std::printf("api sanitizer driver: %d failures (devices %d)\n", failures, devices);
    return failures == 0 ? 0 : 1;
}
