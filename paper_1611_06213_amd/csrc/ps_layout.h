// Where the server puts its buffers, and how the apply kernels sweep
// buffers it did not place. Host-only; ps_server.cpp uses it, and it builds
// on its own for host tests.
//
// DRAM serves many concurrent streams fastest when they do not start at one
// offset within 2 MiB (their "phase"), and the distance between them matters
// beyond that: the apply reads 32 or more rows in lockstep, and how their
// addresses spread over HBM channels and banks depends on higher address bits
// too. The server's own large buffers (w, v and the rows of ps_alloc_rows)
// therefore start 1.75 MiB apart beyond their 2 MiB-rounded sizes, so
// consecutive rows step through the eight 256 KiB phases downwards. Buffers
// allocated one by one all start at one phase; for them the kernels sweep
// several fronts instead of one (fronts_log2_for).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace gadei {

constexpr size_t kRowAlign = size_t(2) << 20;
// Phase granularity: rows under 2 MiB are packed on it, and the front choice
// compares buffer phases at it.
constexpr size_t kPhase = 4096;
// Step between large rows (and from w to v) beyond their 2 MiB-rounded size.
// Measured on the VGG-16 (fp32) and Mixed (bf16) applies from 32 rows, over
// steps of 4 KiB and 64 KiB .. 2 MiB: 64-256 KiB were worst (up to 20%
// slower than 4 KiB), steps near 1 MiB were bad for the bf16 rows, and
// 1.75 MiB was among the best for both. Whole bench steps against 4 KiB:
// VGG-16 7,111-7,119 vs 6,953-6,961 pushes/s, Mixed +2.8%, AlexNet +0.9%.
// The gain is at the default depth: for applies of 16 or fewer gradients
// with momentum, 4 KiB steps measured 1.5-3.7 points of peak faster.
constexpr size_t kRowStagger = size_t(7) << 18;

size_t round_up(size_t x, size_t a);
char *align_up(void *p, size_t a);

// Offset of v from w (w at a 2 MiB boundary): one kRowStagger past w's
// 2 MiB-rounded end.
size_t velocity_offset(size_t w_bytes);

// A set of `count` rows of row_bytes each, from a 2 MiB-aligned base: row i
// at head + i * stride. Rows of 2 MiB or more start two kRowStagger in and
// step by their 2 MiB-rounded size plus kRowStagger, so row i sits at phase
// ((i + 2) * kRowStagger) mod 2 MiB (w, v and the rows of one set cycle
// through the eight 256 KiB phases); smaller rows are packed on kPhase
// boundaries after a head of 2 * kPhase. `span` = bytes from the base to the
// end of the last row.
struct RowLayout {
    size_t head;
    size_t stride;
    size_t span;
};
RowLayout row_layout(size_t row_bytes, int count);

// Fronts (log2) an apply over these streams (gradients, w, v; null entries
// are skipped) should sweep: 2 (four fronts) when there are at least 8
// streams and more than half of them share one phase (compared at kPhase),
// else 0 (one front). Measured on 34 streams of 553 MB: same-phase buffers
// 3.97-4.27 ms with one front, 3.42-3.54 ms with four; staggered buffers
// no better with four.
int fronts_log2_for(const void *const *ptrs, int count);

// Launch shape of an apply of k gradients (fp32, or bf16): how many 256-thread
// blocks one compute unit may hold (0 = as many as fit), for buffers at
// distinct phases (where fronts_log2_for gives 0) how many fronts to sweep
// (log2), and how many gradients each lane loads at once (4, 8, 12, 16, 24 or
// 32; the synchronous step's table stops at 16).
// Fewer resident blocks and smaller groups keep fewer DRAM pages and address
// translations live across the k + 2 streams; too few loads in flight starve
// the memory system. Chosen from sweeps at the VGG-16 (fp32) and Mixed (bf16)
// sizes from server rows, % of 8 TB/s: fp32 with momentum, k = 32: one group
// of 32 at one block per CU 82.2, groups of 16 81.7, groups of 4 at two blocks
// 76.2; k = 4: groups of 4 at two blocks 82.9, groups of 16 at three 80.0;
// bf16 with momentum, k = 24: groups of 24 at one block 79.9, of 16 77.9.
struct ApplyShape {
    int blocks_per_cu;
    int fronts_log2;
    int group;
};
// n is the vector's length: below kSmallVector coordinates a shallow fp32
// apply without momentum (7..13 gradients) keeps three blocks per CU instead
// of two (Text-CNN-sized vectors, 10M and 17.3M: 77.3-77.7 and 76.2% vs
// 76.2-76.4 and 74.7; from 24M two are best, 80.4 vs 79.2).
constexpr size_t kSmallVector = 20000000;
ApplyShape apply_shape(int k, bool momentum, bool bf16, size_t n);

// The same for a synchronous step over k gradients (one per learner; no
// fronts choice beyond the phase rule: fronts_log2 is 0).
ApplyShape sync_shape(int k, bool momentum, bool bf16);

// Whether ps_apply_pull writes its r replicas from the apply pass over k
// gradients of an n-coordinate vector (else the apply is followed by the
// tiled fan-out): one replica always; up to 4 when at most 16 gradients are
// folded; up to 6 when at most 8 are folded into a vector of fewer than
// kSmallVector coordinates (10M, k = 8: r = 5 0.100 vs 0.104 ms, r = 6 0.108
// vs 0.110; at 30M and above 5 or 6 are even or slower, 138M r = 6 1.50 vs
// 1.44 ms). Writing replicas from
// the apply adds write streams to its read streams, which costs more than a
// separate fan-out once there are many of either; for few of both it saves
// the fan-out's launch and its second read of w. Measured from server rows
// (apply+pull time, fused vs separate): k = 8, r = 2: 10M coordinates
// 0.079 vs 0.086 ms, 138M 1.07 vs 1.10 ms; k = 16, r = 2: 138M 1.89-1.90 vs
// 1.93-1.94 ms; k = 16, r = 8: 138M 2.47 vs 2.42-2.43 ms; k = 32, r = 2:
// 61M 1.55 vs 1.51 ms.
bool fuse_replicas(int r, int k, size_t n);

}  // namespace gadei
