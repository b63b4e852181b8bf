// Host-only checks of the kernel-dispatch predicates in wq_limits.h at the
// 32-bit buffer-offset boundaries (built with g++ by tests/test_host_logic.py).
#include <cstdio>
#include <cstdlib>

#include "wq_limits.h"

static int failures = 0;

static void expect(bool got, bool want, const char* what) {
    if (got != want) {
        std::printf("FAIL %s: got %d, want %d\n", what, (int)got, (int)want);
        ++failures;
    }
}

int main() {
    using wq::fits_rsrc;
    using wq::prefill_fits;
    const int64_t out = (int64_t)wq::kPrefillOutOffset;
    // Prompt-sized shapes of the decoders.
    expect(prefill_fits(16384, 3072, 2048), true, "3B gate_up, 2048 tokens");
    expect(prefill_fits(128256, 3072, 2048), true, "3B lm_head, 2048 tokens");
    // x of exactly 4 GiB (M = 128, K = 2^24): its byte offsets wrap in 32 bits.
    expect(prefill_fits(256, (int64_t)1 << 24, 128), false, "x of 4 GiB");
    // x just at the out-of-range offset, and one 32-element group past it.
    const int64_t k_at = out / 2 / 128 / 32 * 32;  // largest K with 128 * K * 2 <= out
    expect(prefill_fits(256, k_at, 128), true, "x at the out-of-range offset");
    expect(prefill_fits(256, k_at + 32, 128), false, "x one group past it");
    // Codes of 4 GiB (N = 2^20 rows of K = 8192): 2^20 * 256 * 16 = 2^32.
    expect(prefill_fits((int64_t)1 << 20, 8192, 128), false, "codes of 4 GiB");
    expect(prefill_fits(((int64_t)1 << 20) - 1, 8192, 128), true, "codes one row below 4 GiB");
    // int32 limits on the sizes themselves.
    expect(prefill_fits((int64_t)1 << 31, 32, 128), false, "N above INT32_MAX");
    expect(prefill_fits(0, 32, 128), false, "empty N");
    // Buffer-resource reach of the batch-1 and small-batch kernels.
    expect(fits_rsrc(((int64_t)1 << 28) - 1, 1), true, "codes one group below 4 GiB");
    expect(fits_rsrc((int64_t)1 << 28, 1), false, "codes of 4 GiB");
    expect(fits_rsrc(128256, 96), true, "3B lm_head");
    if (failures) return 1;
    std::printf("ok\n");
    return 0;
}
