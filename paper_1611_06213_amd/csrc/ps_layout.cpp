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
    r.head = 2 * kRowStagger;
    // rows under 2 MiB are packed on 4 KiB boundaries (their phases differ
    // anyway, and rounding each up to 2 MiB would waste memory)
    r.stride = row_bytes < kRowAlign ? round_up(row_bytes, kRowStagger)
                                     : round_up(row_bytes, kRowAlign) + kRowStagger;
    r.span = r.head + (static_cast<size_t>(count) - 1) * r.stride + row_bytes;
    return r;
}

int fronts_log2_for(const void *const *ptrs, int count) {
    constexpr int kMaxStreams = 66;   // PS_MAX_QUEUE_DEPTH gradients + w + v
    uintptr_t seen[kMaxStreams];
    int distinct = 0, streams = 0;
    for (int i = 0; i < count && streams < kMaxStreams; ++i) {
        if (ptrs[i] == nullptr) continue;
        ++streams;
        const uintptr_t ph = (reinterpret_cast<uintptr_t>(ptrs[i]) % kRowAlign) / kRowStagger;
        bool dup = false;
        for (int j = 0; j < distinct; ++j) dup = dup || seen[j] == ph;
        if (!dup) seen[distinct++] = ph;
    }
    return (streams >= 8 && 2 * distinct < streams) ? 2 : 0;
}

}  // namespace gadei
