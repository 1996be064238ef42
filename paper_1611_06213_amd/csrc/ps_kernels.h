// Internal interface between the host library (ps_server.cpp) and the HIP
// kernels (ps_kernels.hip). Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "ps.h"

namespace gadei {

// Kernel argument block of one fused apply (and optional pull fan-out).
// Passed by value, so the K gradient and R replica pointers travel in the
// kernel-argument segment and are read with scalar loads.
struct ApplyArgs {
    float *w;                 // n fp32 weights, updated in place
    float *v;                 // n fp32 velocities (momentum only)
    uint64_t n;
    float lr;
    float m;
    int k;                    // gradients to fold, 1..PS_MAX_QUEUE_DEPTH
    int r;                    // replicas to write after the update, 0..PS_MAX_REPLICAS
    int fronts_log2;          // blocks sweep 2^fronts_log2 evenly spaced fronts (front_block)
    const void *g[PS_MAX_QUEUE_DEPTH];   // oldest first
    void *dst[PS_MAX_REPLICAS];
};

struct PullArgs {
    const float *w;
    uint64_t n;
    int r;
    void *dst[PS_MAX_REPLICAS];
};

// Launch geometry: blocks are 256 threads; max_blocks caps the grid (the
// kernels then stride over the remaining chunks). 0 = one chunk per lane.
// fp32-gradient kernels reserve LDS so that only a few blocks fit per
// compute unit: occupancy_cap_lds leaves room for one, occupancy_cap2_lds
// for two (0 = no reservation; both chosen at server creation for the
// current device). Asynchronous applies take two blocks per CU from
// occupancy_cap2_min_k gradients on, one from occupancy_cap_min_k_momentum
// on when they carry momentum; synchronous steps take one from
// occupancy_cap_min_k on.
struct Geometry {
    int max_blocks = 0;
    int fronts_log2 = -1;   // -1: chosen per apply (fronts_log2_for, ps_layout.h)
    unsigned occupancy_cap_lds = 0;
    unsigned occupancy_cap2_lds = 0;
    int occupancy_cap_min_k = 16;
    int occupancy_cap2_min_k = 8;
    int occupancy_cap_min_k_momentum = 24;
};

// LDS bytes that leave room for exactly `blocks` (1 or 2) blocks per compute
// unit on the current device, or 0 if the device does not allow such a
// reservation.
unsigned blocks_per_cu_lds(int blocks);


// grad_dtype: PS_F32 | PS_BF16. pull_dtype: -1 (no replicas), PS_F32, PS_BF16.
// level: 2 = every buffer 16-byte aligned; 1 = fp32 buffers 16-byte and bf16
// buffers 8-byte aligned; 0 = anything else (scalar kernels).
hipError_t launch_apply(const ApplyArgs &a, int grad_dtype, int pull_dtype, int level,
                        const Geometry &geo, hipStream_t s);
hipError_t launch_pull(const PullArgs &a, int pull_dtype, int level, const Geometry &geo,
                       hipStream_t s);
// Synchronous step over a.k gradients of one dtype (no replicas).
hipError_t launch_sync(const ApplyArgs &a, int grad_dtype, int level, const Geometry &geo,
                       hipStream_t s);
hipError_t launch_zero(float *p, uint64_t n, hipStream_t s);

}  // namespace gadei
