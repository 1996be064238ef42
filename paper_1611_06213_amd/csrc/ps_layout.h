// Where the server puts its buffers, and how the apply kernels sweep
// buffers it did not place. Host-only; ps_server.cpp uses it, and it builds
// on its own for host tests.
//
// DRAM serves many concurrent streams fastest when they start at different
// offsets within 2 MiB. The server's own buffers (w, v and the rows of
// ps_alloc_rows) start on 2 MiB boundaries plus distinct multiples of 4 KiB.
// Buffers allocated one by one all start at one such offset; for them the
// kernels sweep several fronts instead of one (fronts_log2_for).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace gadei {

constexpr size_t kRowAlign = size_t(2) << 20;
constexpr size_t kRowStagger = 4096;

size_t round_up(size_t x, size_t a);
char *align_up(void *p, size_t a);

// Offset of v from w (w at a 2 MiB boundary): one stagger past w's
// 2 MiB-rounded end.
size_t velocity_offset(size_t w_bytes);

// A set of `count` rows of row_bytes each, from a 2 MiB-aligned base: row i
// at head + i * stride. Rows of 2 MiB or more step by their 2 MiB-rounded
// size plus 4 KiB, so row i sits at offset (i + 2) * 4 KiB within 2 MiB (w
// and v take the first two offsets); smaller rows are packed on 4 KiB
// boundaries. `span` = bytes from the base to the end of the last row.
struct RowLayout {
    size_t head;
    size_t stride;
    size_t span;
};
RowLayout row_layout(size_t row_bytes, int count);

// Fronts (log2) an apply over these streams (gradients, w, v; null entries
// are skipped) should sweep: 2 (four fronts) when at least 8 streams and
// fewer than half of them start at distinct 4 KiB offsets within 2 MiB,
// else 0 (one front). Measured on 34 streams of 553 MB: same-offset buffers
// 3.97-4.27 ms with one front, 3.42-3.54 ms with four; staggered buffers
// 3.09-3.31 ms with one front and no better with four.
int fronts_log2_for(const void *const *ptrs, int count);

}  // namespace gadei
