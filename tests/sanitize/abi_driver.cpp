/*
 * Host-code check of the C-ABI library under AddressSanitizer and
 * UndefinedBehaviorSanitizer (built by tests/test_sanitizers.py with the
 * sanitizers on the host compilation only, linked with the library's own
 * source).  Every call here is refused by host validation before any HIP
 * call, so no GPU is needed and no pointer is dereferenced: it exercises the
 * argument checks, the status strings and the thread-local error messages
 * of every entry point, and the workspace-pool and profiling calls that need
 * no device.  Exit status 0 when every call returned what it should.
 */
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <thread>

#include "gt_attn.h"

static int failures = 0;
#define EXPECT(cond)                                                        \
    do {                                                                    \
        if (!(cond)) {                                                      \
            std::fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                     \
        }                                                                   \
    } while (0)

namespace {
// never dereferenced: each call below fails validation first
template <typename T>
T* fake(uintptr_t off) {
    return reinterpret_cast<T*>(uintptr_t(0x10000) + off);
}

gt_status fwd(gt_dtype dt, int64_t N, int64_t E, int32_t H, int32_t D, float scale, uintptr_t qoff = 0,
              uintptr_t ooff = 0x300000, float* lse = nullptr, const gt_tuning* tu = nullptr, bool noalloc = false) {
    auto f = noalloc ? gt_attn_fwd_noalloc : gt_attn_fwd_ex;
    return f(dt, fake<int64_t>(0), fake<int32_t>(0), fake<void>(qoff), fake<void>(0x100000), fake<void>(0x200000),
             fake<void>(ooff), lse, N, E, H, D, scale, tu, nullptr);
}
}  // namespace

int main() {
    // shapes and sizes
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 3, 32, 0.1f) == GT_ERROR_NOT_SUPPORTED);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 512, 0.1f) == GT_ERROR_NOT_SUPPORTED);
    EXPECT(fwd(GT_DTYPE_BF16, 10, 20, 8, 512, 0.1f) == GT_ERROR_NOT_SUPPORTED);
    EXPECT(fwd(static_cast<gt_dtype>(7), 10, 20, 4, 32, 0.1f) == GT_ERROR_NOT_SUPPORTED);
    EXPECT(fwd(GT_DTYPE_F32, -1, 20, 4, 32, 0.1f) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, int64_t(1) << 31, 4, 32, 0.1f) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, int64_t(1) << 31, 20, 4, 32, 0.1f) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, NAN) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, INFINITY) == GT_ERROR_INVALID_VALUE);
    // alignment and aliasing
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 8) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 0, 0x200000 + 1024) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 0, 0, nullptr) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 0, 0x300000, fake<float>(0x300000 + 4)) == GT_ERROR_INVALID_VALUE);
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 0, 0x300000, fake<float>(0x400002)) == GT_ERROR_INVALID_VALUE);
    // tuning fields near INT32_MAX
    gt_tuning tu;
    std::memset(&tu, 0, sizeof tu);
    tu.chunk_edges = INT32_MAX;
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 0, 0x300000, nullptr, &tu) == GT_ERROR_INVALID_VALUE);
    EXPECT(std::strstr(gt_last_error_message(), "tuning") != nullptr);
    tu.chunk_edges = 0;
    tu.light_max_deg = INT32_MAX;
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 4, 32, 0.1f, 0, 0x300000, nullptr, &tu) == GT_ERROR_INVALID_VALUE);
    // the allocation-free entry point validates the same way
    EXPECT(fwd(GT_DTYPE_F32, 10, 20, 3, 32, 0.1f, 0, 0x300000, nullptr, nullptr, true) == GT_ERROR_NOT_SUPPORTED);
    EXPECT(fwd(GT_DTYPE_BF16, 10, 20, 4, 32, 0.1f, 0, 0, nullptr, nullptr, true) == GT_ERROR_INVALID_VALUE);
    // N == 0 enqueues nothing and succeeds
    EXPECT(fwd(GT_DTYPE_F32, 0, 0, 4, 32, 0.1f) == GT_SUCCESS);
    EXPECT(std::strcmp(gt_last_error_message(), "") == 0);
    // the contract entry points
    EXPECT(gt_attn_fwd(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 10, 20, 4, 32, 0.1f, nullptr) ==
           GT_ERROR_INVALID_VALUE);
    EXPECT(gt_attn_fwd_bf16(fake<int64_t>(0), fake<int32_t>(0), nullptr, nullptr, nullptr, nullptr, 10, 20, 4, 32,
                            0.1f, nullptr) == GT_ERROR_INVALID_VALUE);
    // GATv2
    EXPECT(gt_gatv2_fwd(GT_DTYPE_F32, fake<int64_t>(0), fake<int32_t>(0), fake<void>(0), fake<void>(0x100000),
                        nullptr, 0.2f, fake<void>(0x300000), nullptr, 10, 20, 4, 32, nullptr, nullptr) ==
           GT_ERROR_INVALID_VALUE);
    EXPECT(gt_gatv2_fwd(GT_DTYPE_F32, fake<int64_t>(0), fake<int32_t>(0), fake<void>(0), fake<void>(0x100000),
                        fake<float>(0x500000), NAN, fake<void>(0x300000), nullptr, 10, 20, 4, 32, nullptr,
                        nullptr) == GT_ERROR_INVALID_VALUE);
    // backward
    EXPECT(gt_attn_bwd(GT_DTYPE_F32, fake<int64_t>(0), fake<int32_t>(0), fake<int64_t>(0), fake<int32_t>(0),
                       fake<void>(0), fake<void>(0x100000), fake<void>(0x200000), fake<void>(0x300000),
                       fake<void>(0x400000), nullptr, fake<void>(0x500000), fake<void>(0x600000),
                       fake<void>(0x700000), 10, 20, 4, 32, 0.1f, nullptr) == GT_ERROR_INVALID_VALUE);
    EXPECT(gt_attn_bwd(GT_DTYPE_BF16, fake<int64_t>(0), fake<int32_t>(0), fake<int64_t>(0), fake<int32_t>(0),
                       fake<void>(0), fake<void>(0x100000), fake<void>(0x200000), fake<void>(0x300000),
                       fake<void>(0x400000), fake<float>(0x800000), fake<void>(0x500000), fake<void>(0x500000),
                       fake<void>(0x700000), 10, 20, 4, 32, 0.1f, nullptr) == GT_ERROR_INVALID_VALUE);
    // reduction and the locality microbenchmark
    EXPECT(gt_segment_reduce(GT_DTYPE_F32, GT_REDUCE_MIN, fake<int64_t>(0), fake<int32_t>(0), fake<void>(0),
                             fake<void>(0x100000), fake<int32_t>(0x200000), 10, 20, 48, nullptr, nullptr) ==
           GT_ERROR_NOT_SUPPORTED);
    EXPECT(gt_segment_reduce(GT_DTYPE_F32, static_cast<gt_reduce_op>(5), fake<int64_t>(0), fake<int32_t>(0),
                             fake<void>(0), fake<void>(0x100000), nullptr, 10, 20, 64, nullptr, nullptr) ==
           GT_ERROR_NOT_SUPPORTED);
    EXPECT(gt_dot_aggr(fake<int64_t>(0), fake<int32_t>(0), fake<float>(0), fake<float>(0x100000), 10, 20, 32, 2, 16,
                       nullptr) == GT_ERROR_NOT_SUPPORTED);
    int32_t valid = 7;
    EXPECT(gt_csr_validate(nullptr, nullptr, 10, 20, &valid, nullptr) == GT_ERROR_INVALID_VALUE && valid == 0);
    // status strings, pool and profiler calls that need no device
    for (int c = 0; c < 5; ++c) EXPECT(std::strlen(gt_status_string(static_cast<gt_status>(c))) > 0);
    uint64_t reserved = 1, used = 1;
    EXPECT(gt_workspace_pool_stats(0, &reserved, &used) == GT_SUCCESS && reserved == 0 && used == 0);
    EXPECT(gt_workspace_pool_stats(-1, &reserved, &used) == GT_ERROR_INVALID_VALUE);
    EXPECT(gt_workspace_release() == GT_SUCCESS);
    EXPECT(gt_profile_enable(1) == GT_SUCCESS);
    double ms[3];
    int64_t calls = -1;
    EXPECT(gt_profile_collect(ms, &calls) == GT_SUCCESS && calls == 0);
    EXPECT(gt_profile_enable(0) == GT_SUCCESS);
    // error messages are per thread
    std::thread t([] { EXPECT(fwd(GT_DTYPE_F32, 10, 20, 3, 32, 0.1f) == GT_ERROR_NOT_SUPPORTED); });
    t.join();
    EXPECT(std::strcmp(gt_last_error_message(), "") == 0);
    std::printf("abi driver: %d failure(s)\n", failures);
    return failures ? 1 : 0;
}
