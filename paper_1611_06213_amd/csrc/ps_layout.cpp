// Buffer placement and front choice; see ps_layout.h.
#include "ps_layout.h"

namespace gadei {

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

char *align_up(void *p, size_t a) {
    return reinterpret_cast<char *>(round_up(reinterpret_cast<uintptr_t>(p), a));
}

size_t velocity_offset(size_t w_bytes) { return round_up(w_bytes, kRowAlign) + kRowStagger; }

RowLayout row_layout(size_t row_bytes, int count) {
    RowLayout r;
    if (row_bytes < kRowAlign) {
        // packed on 4 KiB boundaries (their phases differ anyway, and rounding
        // each up to 2 MiB would waste memory)
        r.head = 2 * kPhase;
        r.stride = round_up(row_bytes, kPhase);
    } else {
        r.head = 2 * kRowStagger;
        r.stride = round_up(row_bytes, kRowAlign) + kRowStagger;
    }
    r.span = r.head + (static_cast<size_t>(count) - 1) * r.stride + row_bytes;
    return r;
}

int fronts_log2_for(const void *const *ptrs, int count) {
    constexpr int kMaxStreams = 66;   // PS_MAX_QUEUE_DEPTH gradients + w + v
    uintptr_t ph[kMaxStreams];
    int streams = 0;
    for (int i = 0; i < count && streams < kMaxStreams; ++i) {
        if (ptrs[i] == nullptr) continue;
        ph[streams++] = (reinterpret_cast<uintptr_t>(ptrs[i]) % kRowAlign) / kPhase;
    }
    int most = 0;   // the largest number of streams sharing one phase
    for (int i = 0; i < streams; ++i) {
        int same = 0;
        for (int j = 0; j < streams; ++j) same += ph[j] == ph[i];
        most = same > most ? same : most;
    }
    return (streams >= 8 && 2 * most > streams) ? 2 : 0;
}

ApplyShape apply_shape(int k, bool momentum, bool bf16, size_t n) {
    // Measured at 138,357,544 fp32 / 200,000,000 bf16 parameters for the
    // depths 1, 2, 3, 4, 6, 8, 12, 16, 20, 24, 32, 36, 40, 44, 48 and 64
    // (bf16: from 8); the depths between take a neighbour's shape. A group of
    // 24 or 32 pays only from its own depth on: below it the w/v loads would
    // be waited for before the first (smaller) group.
    if (bf16) {
        if (momentum) {
            if (k <= 11) return {2, 0, 16};
            if (k <= 23) return {1, 0, 16};
            if (k <= 44) return {1, 0, 24};
            return {1, 0, 16};
        }
        if (k <= 11) return {2, 0, 8};
        if (k <= 23) return {1, 0, 16};
        if (k <= 31) return {1, 0, 24};
        if (k <= 47) return {1, 0, 32};
        if (k <= 56) return {1, 0, 16};
        return {1, 0, 8};
    }
    if (momentum) {
        if (k <= 1) return {4, 0, 16};
        if (k == 2) return {3, 0, 4};
        if (k <= 9) return {2, 0, 4};
        if (k <= 13) return {1, 0, 12};
        if (k <= 17) return {1, 0, 16};
        if (k <= 21) return {1, 0, 12};
        if (k <= 31) return {1, 0, 16};
        if (k <= 44) return {1, 0, 32};
        return {1, 0, 8};
    }
    if (k <= 2) return {0, 0, 16};
    if (k <= 6) return {3, 0, 4};
    if (k <= 13) return n < kSmallVector ? ApplyShape{3, 0, 4} : ApplyShape{2, 0, 4};
    if (k <= 17) return {1, 0, 16};
    if (k <= 21) return {2, 0, 4};
    return {1, 0, 8};
}

ApplyShape sync_shape(int k, bool momentum, bool bf16) {
    // Measured at 138,357,544 fp32 / 200,000,000 bf16 parameters with one
    // gradient per learner, for 4, 8, 12, 16, 20, 24 and 32 learners; the
    // counts between take the next measured one's shape.
    if (bf16) {
        if (momentum) {
            if (k <= 4) return {3, 0, 16};
            if (k <= 8) return {2, 0, 12};
            if (k <= 12) return {2, 0, 4};
            if (k <= 16) return {1, 0, 16};
            if (k <= 20) return {1, 0, 12};
            if (k <= 24) return {1, 0, 16};
            return {1, 0, 8};
        }
        if (k <= 4) return {3, 0, 4};
        if (k <= 16) return {2, 0, 4};
        return {1, 0, 12};
    }
    if (momentum) {
        if (k <= 4) return {2, 0, 16};
        if (k <= 8) return {2, 0, 4};
        if (k <= 12) return {1, 0, 12};
        if (k <= 16) return {1, 0, 16};
        if (k <= 20) return {1, 0, 12};
        if (k <= 24) return {1, 0, 16};
        return {1, 0, 8};
    }
    if (k <= 4) return {3, 0, 16};
    if (k <= 12) return {2, 0, 4};
    return {1, 0, 16};
}

bool fuse_replicas(int r, int k, size_t n) {
    return r <= 1 || (r <= 4 && k <= 16) || (r <= 6 && k <= 8 && n < kSmallVector);
}

}  // namespace gadei
