// HIP kernels of the parameter server for gfx950 (CDNA4).
//
// The kernels are pure streams over HBM: every byte is read or written once
// per launch and there is no reuse to stage in LDS and no contraction for
// the matrix cores. What matters is that each lane moves whole, aligned
// 16-byte chunks (4 fp32 or 8 bf16 values; narrower only for misaligned
// buffers), that enough loads are in flight, that nothing is re-read, and
// which coordinates the resident blocks work on at the same time (the DRAM
// serves some access patterns faster than others: see front_block,
// pull_tiled and pull_slices).
//
// apply:  for each coordinate i and each pending gradient k = 0..K-1, oldest
//         first, one ASGD step (Eq. "asgd" with the step of Eq. "gd"):
//           momentum == 0: p = lr*g; w = w - p
//           momentum != 0: t = m*v; v = t + g; p = lr*v; w = w - p
//         w (and v) are loaded once, the K gradients streamed past them in
//         registers, and the result stored once: K sequential steps cost one
//         pass over w instead of K. Optionally the same pass writes R replica
//         copies of the new w (a fused pull).
// sync:   the synchronous step (Eq. "ssgd"): the K pending gradients summed
//         per coordinate in push order, divided by K, applied as one step.
// pull:   write w to R replica buffers (fp32, or bf16 rounded to nearest
//         even). One replica: a streaming copy. Several: a tiled fan-out that
//         keeps each tile of w in cache while the replicas are written one
//         after another, each XCD writing its own contiguous slice of the
//         tile (see pull_tiled and pull_slices).
//
// Every product and sum is rounded on its own (no fused multiply-add), so
// the result is bit-identical to sequential binary32 steps. Built with
// PS_FP_CONTRACT defined, the compiler may fuse them instead (the
// contraction-allowed flavour, libgadeips_fma.so), which stays within 1e-6
// relative of the sequential result.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "ps_kernels.h"

#ifdef PS_FP_CONTRACT
#pragma clang fp contract(fast)
#else
#pragma clang fp contract(off)
#endif

namespace gadei {
namespace {

#ifndef PS_BLOCK
#define PS_BLOCK 256
#endif
#ifndef PS_GROUP
#define PS_GROUP 16
#endif
#ifndef PS_NT_WV
#define PS_NT_WV 1
#endif

constexpr int kBlock = PS_BLOCK;

// Compact kernel argument blocks for launches of at most kCompact gradients
// and kCompact replicas: the fields of ApplyArgs / PullArgs with 8-entry
// pointer arrays (176 and 88 bytes instead of 1064 and 536). The host
// enqueues a launch faster the smaller its argument segment (back-to-back
// launches of an empty kernel: 4.5 us with a 1 KiB argument, 2.9 us with 64
// bytes, each beside the runtime's implicit arguments), and that cost sets
// the rate of launch-bound loops such as one gradient and one replica per
// step. The kernels are the same templates over either block.
constexpr int kCompact = 8;
struct ApplyArgsC {
    float *w;
    float *v;
    uint64_t n;
    float lr;
    float m;
    int k;
    int r;
    int fronts_log2;
    const void *g[kCompact];
    void *dst[kCompact];
};
struct PullArgsC {
    const float *w;
    uint64_t n;
    int r;
    void *dst[kCompact];
};
template <class A>
constexpr bool kCompactArgs = std::is_same_v<A, ApplyArgsC>;      // threads per block (waves of 64 lanes)
// Gradients whose loads are issued together: the vector kernels take the
// group size their launcher chooses (4, 8, 12, 16, 24 or 32 for the apply,
// up to 16 for the synchronous step); the scalar paths take kGroup. Full
// groups, then one of 16 (groups above 16), one of 8 (groups above 8) and
// the remainder (at most 7) cover every K.
constexpr int kGroup = PS_GROUP;
static_assert(kGroup >= 1 && kGroup <= 16, "gradient group size must be 1..16");
// w and v are read once and written once per launch and are not touched
// again until the next apply, after tens of GB of other traffic: stream them
// with the non-temporal hint too.
constexpr bool kNtWV = PS_NT_WV != 0;
// The same choice for the 8-coordinate chunks of bf16-gradient applies, for
// loads and stores separately.
#ifndef PS_NT_WV_LD8
#define PS_NT_WV_LD8 PS_NT_WV
#endif
#ifndef PS_NT_WV_ST8
#define PS_NT_WV_ST8 PS_NT_WV
#endif
template <int E>
constexpr bool nt_wv_ld() { return E == 8 ? PS_NT_WV_LD8 != 0 : kNtWV; }
template <int E>
constexpr bool nt_wv_st() { return E == 8 ? PS_NT_WV_ST8 != 0 : kNtWV; }

// A launch's work-items (blocks * threads) must stay below 2^32.
constexpr uint64_t kMaxBlocks = 0xffffffffull / kBlock;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- loads

// E consecutive fp32 values starting at p (E = 4: one 16-byte load; E = 8:
// two adjacent ones).
template <int E, bool NT>
__device__ __forceinline__ void ld_f32(float (&x)[E], const float *p) {
    if constexpr (E == 1) {
        x[0] = NT ? __builtin_nontemporal_load(p) : *p;
    } else {
#pragma unroll
        for (int h = 0; h < E / 4; ++h) {
            const f32x4 *q = reinterpret_cast<const f32x4 *>(p) + h;
            f32x4 t = NT ? __builtin_nontemporal_load(q) : *q;
            x[4 * h] = t.x; x[4 * h + 1] = t.y; x[4 * h + 2] = t.z; x[4 * h + 3] = t.w;
        }
    }
}

template <int E, bool NT>
__device__ __forceinline__ void st_f32(float *p, const float (&x)[E]) {
    if constexpr (E == 1) {
        if constexpr (NT) __builtin_nontemporal_store(x[0], p); else *p = x[0];
    } else {
#pragma unroll
        for (int h = 0; h < E / 4; ++h) {
            f32x4 t = {x[4 * h], x[4 * h + 1], x[4 * h + 2], x[4 * h + 3]};
            f32x4 *q = reinterpret_cast<f32x4 *>(p) + h;
            if constexpr (NT) __builtin_nontemporal_store(t, q); else *q = t;
        }
    }
}

// bf16 -> fp32 is exact: the bf16 bits are the upper half of the fp32 bits.
__device__ __forceinline__ float lo_bf16(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// Gradient lanes for coordinates i .. i+E-1 (i is a multiple of E) as
// loaded: fp32 chunks are 4 values (16 bytes); bf16 chunks are 8 values (16
// bytes) or 4 (8 bytes) when a buffer is only 8-byte aligned. Gradients are
// read exactly once per launch, so the loads carry the non-temporal hint.
// Loading and widening are separate steps so that a group's loads can all be
// issued before the first of its values is widened.
template <int GDT, int E> struct GradBits;
template <> struct GradBits<PS_F32, 4> { f32x4 u; };
template <> struct GradBits<PS_F32, 1> { float u; };
template <> struct GradBits<PS_BF16, 8> { u32x4 u; };
template <> struct GradBits<PS_BF16, 4> { u32x2 u; };
template <> struct GradBits<PS_BF16, 1> { uint32_t u; };

template <int GDT, int E>
__device__ __forceinline__ GradBits<GDT, E> ld_bits(const void *g, uint64_t i) {
    GradBits<GDT, E> r;
    if constexpr (GDT == PS_F32) {
        if constexpr (E == 1) {
            r.u = static_cast<const float *>(g)[i];
        } else {
            r.u = __builtin_nontemporal_load(
                reinterpret_cast<const f32x4 *>(static_cast<const float *>(g) + i));
        }
    } else {
        if constexpr (E == 8) {
            r.u = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(g) + (i >> 3));
        } else if constexpr (E == 4) {
            r.u = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(g) + (i >> 2));
        } else {
            r.u = static_cast<const uint16_t *>(g)[i];
        }
    }
    return r;
}

template <int GDT, int E>
__device__ __forceinline__ void widen(float (&x)[E], const GradBits<GDT, E> &r) {
    if constexpr (GDT == PS_F32) {
        if constexpr (E == 1) {
            x[0] = r.u;
        } else {
            x[0] = r.u.x; x[1] = r.u.y; x[2] = r.u.z; x[3] = r.u.w;
        }
    } else {
        if constexpr (E == 8) {
            x[0] = lo_bf16(r.u.x); x[1] = hi_bf16(r.u.x);
            x[2] = lo_bf16(r.u.y); x[3] = hi_bf16(r.u.y);
            x[4] = lo_bf16(r.u.z); x[5] = hi_bf16(r.u.z);
            x[6] = lo_bf16(r.u.w); x[7] = hi_bf16(r.u.w);
        } else if constexpr (E == 4) {
            x[0] = lo_bf16(r.u.x); x[1] = hi_bf16(r.u.x);
            x[2] = lo_bf16(r.u.y); x[3] = hi_bf16(r.u.y);
        } else {
            x[0] = lo_bf16(r.u);
        }
    }
}

template <int GDT, int E>
__device__ __forceinline__ void ld_grad(float (&x)[E], const void *g, uint64_t i) {
    widen<GDT, E>(x, ld_bits<GDT, E>(g, i));
}

// Two fp32 values -> two bf16 in one 32-bit word (a in the low half), each
// rounded to nearest, ties to even; a NaN keeps its sign and the top of its
// payload and gets the quiet bit. This is gfx950's packed conversion
// (v_cvt_pk_bf16_f32), one instruction per pair. Under the kernels' float
// mode (round to nearest even, fp32 denormals kept) it equals, for all 2^32
// inputs (checked exhaustively on the device), the bit-level definition:
// r = (u + 0x7fff + ((u >> 16) & 1)) >> 16 for non-NaN bits u, and
// (u >> 16) | 0x40 for NaN.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16x2_rne(float a, float b) {
    const f32x2 x = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
}

// One replica's values for coordinates i .. i+E-1 (i a multiple of E).
// Replicas are not read back by the server, so the stores carry the
// non-temporal hint.
template <int PDT, int E>
__device__ __forceinline__ void st_dst(void *d, uint64_t i, const float (&x)[E]) {
    if constexpr (PDT == PS_F32) {
        if constexpr (E == 1) {
            static_cast<float *>(d)[i] = x[0];
        } else {
            st_f32<E, true>(static_cast<float *>(d) + i, x);
        }
    } else {
        if constexpr (E == 8) {
            u32x4 t;
            t.x = bf16x2_rne(x[0], x[1]);
            t.y = bf16x2_rne(x[2], x[3]);
            t.z = bf16x2_rne(x[4], x[5]);
            t.w = bf16x2_rne(x[6], x[7]);
            __builtin_nontemporal_store(t, reinterpret_cast<u32x4 *>(d) + (i >> 3));
        } else if constexpr (E == 4) {
            u32x2 t;
            t.x = bf16x2_rne(x[0], x[1]);
            t.y = bf16x2_rne(x[2], x[3]);
            __builtin_nontemporal_store(t, reinterpret_cast<u32x2 *>(d) + (i >> 2));
        } else {
            static_cast<uint16_t *>(d)[i] = static_cast<uint16_t>(bf16x2_rne(x[0], 0.0f));
        }
    }
}

// ---------------------------------------------------------------- apply

// One ASGD step (Eq. "asgd" with the step of Eq. "gd") on E coordinates.
template <bool MOM, int E>
__device__ __forceinline__ void step(float (&w)[E], float (&v)[E], const float (&g)[E], float lr,
                                     float m) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
        if constexpr (MOM) {
            float t = m * v[e];
            v[e] = t + g[e];
            float p = lr * v[e];
            w[e] = w[e] - p;
        } else {
            float p = lr * g[e];
            w[e] = w[e] - p;
        }
    }
}

// Coordinates i .. i+E-1 through all K pending gradients, oldest first, in
// groups whose loads are all issued before the group's updates, so each lane
// keeps G independent loads in flight. The scheduling barrier keeps the
// compiler from pulling the updates (and the bf16 widening) up between the
// loads, which would make the later loads of a group wait for the earlier
// ones to arrive.
template <bool MOM, int GDT, int E, int G, class A>
__device__ __forceinline__ void apply_group(const A &a, int k0, uint64_t i, float (&w)[E],
                                            float (&v)[E], float lr, float m) {
    GradBits<GDT, E> r[G];
#pragma unroll
    for (int j = 0; j < G; ++j) r[j] = ld_bits<GDT, E>(a.g[k0 + j], i);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < G; ++j) {
        float g[E];
        widen<GDT, E>(g, r[j]);
        step<MOM, E>(w, v, g, lr, m);
    }
}

// The first group is straight-line code after the w/v loads, so its loads
// overlap theirs (the compiler waits for every outstanding load a loop reads
// before entering the loop). The remainder after the full groups (and one
// group of 8) is one straight-line group of its exact size: loads under
// per-gradient conditions would each wait for the memory in turn.
template <bool MOM, int GDT, int PDT, int E, int G, class A>
__device__ __forceinline__ void apply_chunk(const A &a, uint64_t i) {
    static_assert(G >= 1 && G <= 32, "gradient group size must be 1..32");
    float w[E], v[E];
    ld_f32<E, nt_wv_ld<E>()>(w, a.w + i);
    if constexpr (MOM) ld_f32<E, nt_wv_ld<E>()>(v, a.v + i);
    const float lr = a.lr;
    const float m = a.m;
    const int k = a.k;
    int k0 = 0;
    if (k >= G) {
        apply_group<MOM, GDT, E, G>(a, 0, i, w, v, lr, m);
        k0 = G;
    }
    for (; k0 + G <= k; k0 += G) apply_group<MOM, GDT, E, G>(a, k0, i, w, v, lr, m);
    if constexpr (G > 16) {
        if (k0 + 16 <= k) {
            apply_group<MOM, GDT, E, 16>(a, k0, i, w, v, lr, m);
            k0 += 16;
        }
    }
    if constexpr (G > 8) {
        if (k0 + 8 <= k) {
            apply_group<MOM, GDT, E, 8>(a, k0, i, w, v, lr, m);
            k0 += 8;
        }
    }
    switch (k - k0) {
        case 1: apply_group<MOM, GDT, E, 1>(a, k0, i, w, v, lr, m); break;
        case 2: apply_group<MOM, GDT, E, 2>(a, k0, i, w, v, lr, m); break;
        case 3: apply_group<MOM, GDT, E, 3>(a, k0, i, w, v, lr, m); break;
        case 4: apply_group<MOM, GDT, E, 4>(a, k0, i, w, v, lr, m); break;
        case 5: apply_group<MOM, GDT, E, 5>(a, k0, i, w, v, lr, m); break;
        case 6: apply_group<MOM, GDT, E, 6>(a, k0, i, w, v, lr, m); break;
        case 7: apply_group<MOM, GDT, E, 7>(a, k0, i, w, v, lr, m); break;
        default: break;
    }
    st_f32<E, nt_wv_st<E>()>(a.w + i, w);
    if constexpr (MOM) st_f32<E, nt_wv_st<E>()>(a.v + i, v);
    if constexpr (PDT >= 0) {
        for (int r = 0; r < a.r; ++r) st_dst<PDT, E>(a.dst[r], i, w);
    }
}

// Synchronous SGD (Eq. "ssgd"): the K pending gradients (one per learner)
// are summed per coordinate in push order from +0, divided by K (correctly
// rounded division), and the average is applied as one step. Same streams
// and gradient groups as the apply, loaded and waited for as the compiler
// schedules them (the apply's load arrangement measured no faster here), the
// remainder as one predicated group.
template <int GDT, int E, int G, class A>
__device__ __forceinline__ void sum_group(const A &a, int k0, uint64_t i, float (&s)[E]) {
    float g[G][E];
#pragma unroll
    for (int j = 0; j < G; ++j) ld_grad<GDT, E>(g[j], a.g[k0 + j], i);
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
        for (int e = 0; e < E; ++e) s[e] = s[e] + g[j][e];
}

template <bool MOM, int GDT, int E, int G, class A>
__device__ __forceinline__ void sync_chunk(const A &a, uint64_t i) {
    static_assert(G >= 1 && G <= 16, "gradient group size must be 1..16");
    float w[E], v[E], s[E];
    ld_f32<E, nt_wv_ld<E>()>(w, a.w + i);
    if constexpr (MOM) ld_f32<E, nt_wv_ld<E>()>(v, a.v + i);
#pragma unroll
    for (int e = 0; e < E; ++e) s[e] = 0.0f;
    const int k = a.k;
    int k0 = 0;
    for (; k0 + G <= k; k0 += G) sum_group<GDT, E, G>(a, k0, i, s);
    if constexpr (G > 8) {
        if (k0 + 8 <= k) {
            sum_group<GDT, E, 8>(a, k0, i, s);
            k0 += 8;
        }
    }
    if (k0 < k) {
        float g[8][E];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (k0 + j < k) ld_grad<GDT, E>(g[j], a.g[k0 + j], i);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (k0 + j < k)
#pragma unroll
                for (int e = 0; e < E; ++e) s[e] = s[e] + g[j][e];
    }
    const float kf = static_cast<float>(k);
    float avg[E];
#pragma unroll
    for (int e = 0; e < E; ++e) avg[e] = s[e] / kf;
    step<MOM, E>(w, v, avg, a.lr, a.m);
    st_f32<E, nt_wv_st<E>()>(a.w + i, w);
    if constexpr (MOM) st_f32<E, nt_wv_st<E>()>(a.v + i, v);
}

// Blocks are dispatched in index order. With F = 2^f fronts, block b works
// at position b / F of front b % F, the fronts spaced evenly over the grid's
// blocks: at any moment the resident blocks sit in F regions far apart
// instead of one. A bijection on the first F * floor(nb / F) blocks, the
// identity on the rest, so every chunk is still covered exactly once.
__device__ __forceinline__ uint64_t front_block(unsigned b, unsigned nb, int f) {
    const unsigned q = nb >> f;
    if (f > 0 && b < (q << f)) return static_cast<uint64_t>(b & ((1u << f) - 1)) * q + (b >> f);
    return b;
}

template <bool MOM, int GDT, int E, int G, class A>
__global__ void __launch_bounds__(kBlock) sync_vec(const A a) {
    const uint64_t chunks = a.n / E;
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t vtid = front_block(blockIdx.x, gridDim.x, a.fronts_log2) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t c = vtid; c < chunks; c += stride) sync_chunk<MOM, GDT, E, G>(a, c * E);
    if (tid < a.n - chunks * E) sync_chunk<MOM, GDT, 1, G>(a, chunks * E + tid);
}

// Vector path: lane t of the grid owns E-coordinate chunks t', t' + stride,
// ... where t' is t with its block renumbered by front_block. The n mod E
// trailing coordinates go to the first lanes of the grid.
template <bool MOM, int GDT, int PDT, int E, int G, class A>
__global__ void __launch_bounds__(kBlock) apply_vec(const A a) {
    const uint64_t chunks = a.n / E;
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t vtid = front_block(blockIdx.x, gridDim.x, a.fronts_log2) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t c = vtid; c < chunks; c += stride) apply_chunk<MOM, GDT, PDT, E, G>(a, c * E);
    if (tid < a.n - chunks * E) apply_chunk<MOM, GDT, PDT, 1, G>(a, chunks * E + tid);
}

// Scalar path for buffers without vector alignment: one coordinate per lane.
template <bool MOM, int GDT, int PDT, class A>
__global__ void __launch_bounds__(kBlock) apply_scalar(const A a) {
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t i = tid; i < a.n; i += stride) apply_chunk<MOM, GDT, PDT, 1, kGroup>(a, i);
}

// ---------------------------------------------------------------- pull

template <int PDT, int E, bool NT, class P>
__device__ __forceinline__ void pull_chunk(const P &a, uint64_t i) {
    float w[E];
    ld_f32<E, NT>(w, a.w + i);
    for (int r = 0; r < a.r; ++r) st_dst<PDT, E>(a.dst[r], i, w);
}

// One pass: each lane reads its chunk of w once and writes it to every
// replica. Used for a single replica (a plain streaming copy).
template <int PDT, class P>
__global__ void __launch_bounds__(kBlock) pull_vec(const P a) {
    const uint64_t chunks = a.n >> 2;
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t c = tid; c < chunks; c += stride) pull_chunk<PDT, 4, true>(a, c << 2);
    if (tid < a.n - (chunks << 2)) pull_chunk<PDT, 1, true>(a, (chunks << 2) + tid);
}

// Tiled fan-outs for R >= 2 replicas. w is cut into tiles; blocks enumerate
// (tile, replica, block within the tile) with the last fastest, so in-order
// dispatch walks replica 0 of tile 0, replica 1 of tile 0, ... The R
// re-reads of a tile then hit the memory-side cache (the tile is loaded with
// ordinary, allocating loads) and HBM sees one replica's write stream at a
// time instead of R interleaved ones, which the memory system serves
// markedly faster. HBM traffic stays one read of w plus the R replica
// writes. One 16-byte chunk of w per lane (4 fp32 or 8 bf16 values): two
// chunks per lane measured 4-5% slower for bf16 replicas.
//
// pull_tiled: 4 Mi-coordinate tiles on a 1-D grid (4096 blocks per tile and
// replica). Blocks are dispatched round-robin over the chip's 8 XCDs (block
// index mod 8); when a group's block count is a multiple of 8, block b of the
// group works on slice (b mod 8) * (bpt / 8) + b / 8, so each XCD writes one
// contiguous eighth of the tile per replica instead of 4 KiB pieces
// interleaved with the other seven, and re-reads only its own eighth of the
// tile from its own L2. Used for fp32 replicas of 8 or more tiles, where it
// measured faster in whole steps (AlexNet's pulls 0.422 vs 0.426 ms, VGG-16's
// 16 replicas 1.36-1.37 vs 1.38 ms); pull_slices below elsewhere.
constexpr uint64_t kTiledCoords = uint64_t(4) << 20;
constexpr unsigned kTileBlocks = 4096;      // most blocks per (tile, replica)

template <int PDT, int E, class P>
__global__ void __launch_bounds__(kBlock) pull_tiled(const P a, unsigned bpt) {
    constexpr uint64_t kTileChunksE = kTiledCoords / E;
    const uint64_t chunks = a.n / E;
    const unsigned b0 = blockIdx.x % bpt;
    const unsigned b = (bpt & 7u) == 0 ? (b0 & 7u) * (bpt >> 3) + (b0 >> 3) : b0;
    const unsigned tr = blockIdx.x / bpt;
    const int r = static_cast<int>(tr % static_cast<unsigned>(a.r));
    const uint64_t t = tr / static_cast<unsigned>(a.r);
    const uint64_t c0 = t * kTileChunksE;
    const uint64_t c1 = c0 + kTileChunksE < chunks ? c0 + kTileChunksE : chunks;
    void *d = a.dst[r];
    for (uint64_t c = c0 + static_cast<uint64_t>(b) * kBlock + threadIdx.x; c < c1;
         c += static_cast<uint64_t>(bpt) * kBlock) {
        float w[E];
        ld_f32<E, false>(w, a.w + c * E);
        st_dst<PDT, E>(d, c * E, w);
    }
    if (t == 0 && b == 0 && threadIdx.x < a.n - chunks * E) {
        const uint64_t i = chunks * E + threadIdx.x;
        float w[1];
        ld_f32<1, false>(w, a.w + i);
        st_dst<PDT, 1>(d, i, w);
    }
}

// pull_slices: the same fan-out over 2 Mi-coordinate tiles on a 3-D grid
// (x: block within the tile, y: replica, z: tile; dispatch order x
// fastest). Each tile is cut into 8 contiguous slices, whole multiples of
// kBlock chunks (the last slices short or empty for a short tile), and the
// blocks of XCD x (x = block mod 8, the grid's x extent being a multiple of
// 8) stride through slice x. This keeps each XCD's writes in one contiguous
// slice and spreads a short last tile over all 8 XCDs. Used for bf16
// replicas (Mixed's 32: 1.98 ms; 2.08 ms with two chunks per lane) and for
// vectors of fewer than 8 tiles of pull_tiled, where its smaller tiles and
// short-tile spreading pay (the 17.3M-coordinate shard's 16 fp32 replicas:
// 0.172 vs 0.185 ms).
constexpr uint64_t kSliceTileCoords = uint64_t(2) << 20;

template <int PDT, int E, class P>
__global__ void __launch_bounds__(kBlock) pull_slices(const P a) {
    constexpr uint64_t kTileChunksE = kSliceTileCoords / E;
    const uint64_t chunks = a.n / E;
    const unsigned b = blockIdx.x;
    const uint64_t t = blockIdx.z;
    const uint64_t c0 = t * kTileChunksE;
    const uint64_t c1 = c0 + kTileChunksE < chunks ? c0 + kTileChunksE : chunks;
    uint64_t lo = c0, hi = c1, j = b, nj = gridDim.x;
    if ((gridDim.x & 7u) == 0) {
        const uint64_t per = (c1 - c0 + 8 * kBlock - 1) / (8 * kBlock) * kBlock;
        const uint64_t x = b & 7u;
        lo = c0 + x * per < c1 ? c0 + x * per : c1;
        hi = lo + per < c1 ? lo + per : c1;
        j = b >> 3;
        nj = gridDim.x >> 3;
    }
    void *d = a.dst[blockIdx.y];
    const uint64_t step = nj * kBlock;
    for (uint64_t c = lo + j * kBlock + threadIdx.x; c < hi; c += step) {
        float w[E];
        ld_f32<E, false>(w, a.w + c * E);
        st_dst<PDT, E>(d, c * E, w);
    }
    if (t == 0 && b == 0 && threadIdx.x < a.n - chunks * E) {
        const uint64_t i = chunks * E + threadIdx.x;
        float w[1];
        ld_f32<1, false>(w, a.w + i);
        st_dst<PDT, 1>(d, i, w);
    }
}

// Scalar path for replicas without vector alignment.
template <int PDT, class P>
__global__ void __launch_bounds__(kBlock) pull_scalar(const P a) {
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t i = tid; i < a.n; i += stride) pull_chunk<PDT, 1, false>(a, i);
}

__global__ void __launch_bounds__(kBlock) zero_f32(float *p, uint64_t n) {
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t i = tid; i < n; i += stride) p[i] = 0.0f;
}

// ---------------------------------------------------------------- launch

unsigned grid_for(uint64_t items, const Geometry &geo) {
    uint64_t blocks = (items + kBlock - 1) / kBlock;
    if (blocks == 0) blocks = 1;
    uint64_t cap = geo.max_blocks > 0 ? static_cast<uint64_t>(geo.max_blocks) : kMaxBlocks;
    if (cap > kMaxBlocks) cap = kMaxBlocks;
    return static_cast<unsigned>(blocks < cap ? blocks : cap);
}

template <bool MOM, int GDT, int PDT, int E, int G, class A>
hipError_t launch_vec(const A &a, unsigned lds, const Geometry &geo, hipStream_t s) {
    hipLaunchKernelGGL((apply_vec<MOM, GDT, PDT, E, G, A>), dim3(grid_for(a.n / E, geo)),
                       dim3(kBlock), lds, s, a);
    return hipGetLastError();
}

template <bool MOM, int GDT, int PDT, int E, class A>
hipError_t launch_vec_g(const A &a, int group, unsigned lds, const Geometry &geo,
                        hipStream_t s) {
    if constexpr (kCompactArgs<A>) {
        // at most kCompact gradients: groups above 8 all take one group of 8
        // and the exact remainder, so 16 stands for 12, 24 and 32
        if (group == 4) return launch_vec<MOM, GDT, PDT, E, 4>(a, lds, geo, s);
        if (group == 8) return launch_vec<MOM, GDT, PDT, E, 8>(a, lds, geo, s);
        return launch_vec<MOM, GDT, PDT, E, 16>(a, lds, geo, s);
    } else {
        switch (group) {
            case 4: return launch_vec<MOM, GDT, PDT, E, 4>(a, lds, geo, s);
            case 8: return launch_vec<MOM, GDT, PDT, E, 8>(a, lds, geo, s);
            case 12: return launch_vec<MOM, GDT, PDT, E, 12>(a, lds, geo, s);
            case 24: return launch_vec<MOM, GDT, PDT, E, 24>(a, lds, geo, s);
            case 32: return launch_vec<MOM, GDT, PDT, E, 32>(a, lds, geo, s);
            default: return launch_vec<MOM, GDT, PDT, E, 16>(a, lds, geo, s);
        }
    }
}

template <bool MOM, int GDT, int PDT, class A>
hipError_t go_apply(const A &a, int level, const Shape &sh, const Geometry &geo,
                    hipStream_t s) {
    if (level == 0) {
        hipLaunchKernelGGL((apply_scalar<MOM, GDT, PDT, A>), dim3(grid_for(a.n, geo)),
                           dim3(kBlock), 0, s, a);
        return hipGetLastError();
    }
    // Residency as the caller asks (apply_shape, ps_layout.h), reserved via
    // dynamic LDS that the kernel does not use; 0 blocks = as many as fit.
    const unsigned lds =
        (sh.blocks_per_cu >= 1 && sh.blocks_per_cu <= 4) ? geo.lds_for_blocks[sh.blocks_per_cu] : 0;
    // bf16 gradients move 16 bytes per lane as 8 values when every buffer is
    // 16-byte aligned; otherwise (and for fp32) a lane's chunk is 4 values.
    if constexpr (GDT == PS_BF16) {
        if (level == 2) return launch_vec_g<MOM, GDT, PDT, 8>(a, sh.group, lds, geo, s);
    }
    return launch_vec_g<MOM, GDT, PDT, 4>(a, sh.group, lds, geo, s);
}

template <bool MOM, int GDT, int E, int G>
hipError_t launch_sync_vec(const ApplyArgs &a, unsigned lds, const Geometry &geo, hipStream_t s) {
    hipLaunchKernelGGL((sync_vec<MOM, GDT, E, G, ApplyArgs>), dim3(grid_for(a.n / E, geo)),
                       dim3(kBlock), lds, s, a);
    return hipGetLastError();
}

template <bool MOM, int GDT, int E>
hipError_t launch_sync_g(const ApplyArgs &a, int group, unsigned lds, const Geometry &geo,
                         hipStream_t s) {
    switch (group) {
        case 4: return launch_sync_vec<MOM, GDT, E, 4>(a, lds, geo, s);
        case 8: return launch_sync_vec<MOM, GDT, E, 8>(a, lds, geo, s);
        case 12: return launch_sync_vec<MOM, GDT, E, 12>(a, lds, geo, s);
        default: return launch_sync_vec<MOM, GDT, E, 16>(a, lds, geo, s);
    }
}

template <bool MOM, int GDT>
hipError_t go_sync(const ApplyArgs &a, int level, const Shape &sh, const Geometry &geo,
                   hipStream_t s) {
    if (level == 0) return launch_sync_vec<MOM, GDT, 1, kGroup>(a, 0, geo, s);
    const unsigned lds =
        (sh.blocks_per_cu >= 1 && sh.blocks_per_cu <= 4) ? geo.lds_for_blocks[sh.blocks_per_cu] : 0;
    if constexpr (GDT == PS_BF16) {
        if (level == 2) return launch_sync_g<MOM, GDT, 8>(a, sh.group, lds, geo, s);
    }
    return launch_sync_g<MOM, GDT, 4>(a, sh.group, lds, geo, s);
}

template <bool MOM, int GDT, class A>
hipError_t go_apply_p(const A &a, int pdt, int level, const Shape &sh, const Geometry &geo,
                      hipStream_t s) {
    if (pdt == PS_F32) return go_apply<MOM, GDT, PS_F32>(a, level, sh, geo, s);
    if (pdt == PS_BF16) return go_apply<MOM, GDT, PS_BF16>(a, level, sh, geo, s);
    return go_apply<MOM, GDT, -1>(a, level, sh, geo, s);
}

template <bool MOM, class A>
hipError_t go_apply_g(const A &a, int gdt, int pdt, int level, const Shape &sh,
                      const Geometry &geo, hipStream_t s) {
    if (gdt == PS_BF16) return go_apply_p<MOM, PS_BF16>(a, pdt, level, sh, geo, s);
    return go_apply_p<MOM, PS_F32>(a, pdt, level, sh, geo, s);
}

}  // namespace

hipError_t launch_apply(const ApplyArgs &a, int grad_dtype, int pull_dtype, int level,
                        const Shape &shape, const Geometry &geo, hipStream_t s) {
    if (a.r == 0) pull_dtype = -1;
    if (a.k <= kCompact && a.r <= kCompact) {
        ApplyArgsC c;
        c.w = a.w;
        c.v = a.v;
        c.n = a.n;
        c.lr = a.lr;
        c.m = a.m;
        c.k = a.k;
        c.r = a.r;
        c.fronts_log2 = a.fronts_log2;
        for (int j = 0; j < kCompact; ++j) {
            c.g[j] = j < a.k ? a.g[j] : nullptr;
            c.dst[j] = j < a.r ? a.dst[j] : nullptr;
        }
        if (c.v != nullptr) return go_apply_g<true>(c, grad_dtype, pull_dtype, level, shape, geo, s);
        return go_apply_g<false>(c, grad_dtype, pull_dtype, level, shape, geo, s);
    }
    if (a.v != nullptr) return go_apply_g<true>(a, grad_dtype, pull_dtype, level, shape, geo, s);
    return go_apply_g<false>(a, grad_dtype, pull_dtype, level, shape, geo, s);
}

template <int PDT, int E, class P>
void go_pull_tiled(const P &a, const Geometry &geo, hipStream_t s) {
    const uint64_t chunks = a.n / E;
    const bool one_d = PDT == PS_F32 && chunks / (kTiledCoords / E) >= 8;
    if (!one_d) {
        // tiles * R * bx blocks, the x extent a multiple of 8 once there are
        // more than 8 blocks per tile
        constexpr uint64_t kTileChunksE = kSliceTileCoords / E;
        const uint64_t tiles = chunks == 0 ? 1 : (chunks + kTileChunksE - 1) / kTileChunksE;
        const uint64_t per_tile = chunks < kTileChunksE ? chunks : kTileChunksE;
        uint64_t bx = (per_tile + kBlock - 1) / kBlock;
        if (bx < 1) bx = 1;
        if (bx > 8) bx = (bx + 7) / 8 * 8;
        if (tiles <= 65535 && bx * tiles * static_cast<uint64_t>(a.r) <= kMaxBlocks) {
            hipLaunchKernelGGL((pull_slices<PDT, E, P>),
                               dim3(static_cast<unsigned>(bx), static_cast<unsigned>(a.r),
                                    static_cast<unsigned>(tiles)),
                               dim3(kBlock), 0, s, a);
            return;
        }
    }
    // tiles * R * bpt blocks; a tile smaller than a full one needs fewer blocks
    constexpr uint64_t kTileChunksE = kTiledCoords / E;
    const uint64_t tiles = chunks == 0 ? 1 : (chunks + kTileChunksE - 1) / kTileChunksE;
    const uint64_t per_tile = chunks < kTileChunksE ? chunks : kTileChunksE;
    uint64_t bpt = (per_tile + kBlock - 1) / kBlock;
    if (bpt < 1) bpt = 1;
    if (bpt > kTileBlocks) bpt = kTileBlocks;
    const uint64_t groups = tiles * static_cast<uint64_t>(a.r);
    if (groups * bpt > kMaxBlocks) bpt = kMaxBlocks / groups;   // lanes stride further
    if (bpt < 1) {
        // more (tile, replica) pairs than a grid can hold: one pass per lane
        hipLaunchKernelGGL((pull_vec<PDT, P>), dim3(grid_for(a.n >> 2, geo)), dim3(kBlock), 0, s,
                           a);
        return;
    }
    hipLaunchKernelGGL((pull_tiled<PDT, E, P>), dim3(static_cast<unsigned>(groups * bpt)),
                       dim3(kBlock), 0, s, a, static_cast<unsigned>(bpt));
}

template <int PDT, class P>
void go_pull(const P &a, int level, const Geometry &geo, hipStream_t s) {
    if (level == 0) {
        hipLaunchKernelGGL((pull_scalar<PDT, P>), dim3(grid_for(a.n, geo)), dim3(kBlock), 0, s, a);
    } else if (a.r == 1) {
        hipLaunchKernelGGL((pull_vec<PDT, P>), dim3(grid_for(a.n >> 2, geo)), dim3(kBlock), 0, s,
                           a);
    } else if (PDT == PS_BF16 && level == 2) {
        go_pull_tiled<PDT, 8>(a, geo, s);
    } else {
        go_pull_tiled<PDT, 4>(a, geo, s);
    }
}

hipError_t launch_sync(const ApplyArgs &a, int grad_dtype, int level, const Shape &shape,
                       const Geometry &geo, hipStream_t s) {
    if (a.v != nullptr) {
        return grad_dtype == PS_BF16 ? go_sync<true, PS_BF16>(a, level, shape, geo, s)
                                     : go_sync<true, PS_F32>(a, level, shape, geo, s);
    }
    return grad_dtype == PS_BF16 ? go_sync<false, PS_BF16>(a, level, shape, geo, s)
                                 : go_sync<false, PS_F32>(a, level, shape, geo, s);
}

hipError_t launch_pull(const PullArgs &a, int pull_dtype, int level, const Geometry &geo,
                       hipStream_t s) {
    if (a.r <= kCompact) {
        PullArgsC c;
        c.w = a.w;
        c.n = a.n;
        c.r = a.r;
        for (int j = 0; j < kCompact; ++j) c.dst[j] = j < a.r ? a.dst[j] : nullptr;
        if (pull_dtype == PS_BF16) go_pull<PS_BF16>(c, level, geo, s);
        else go_pull<PS_F32>(c, level, geo, s);
        return hipGetLastError();
    }
    if (pull_dtype == PS_BF16) go_pull<PS_BF16>(a, level, geo, s);
    else go_pull<PS_F32>(a, level, geo, s);
    return hipGetLastError();
}

unsigned blocks_per_cu_lds(int blocks) {
    int dev = 0, per_cu = 0, per_block = 0;
    if (blocks < 1) return 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
            hipSuccess ||
        hipDeviceGetAttribute(&per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
            hipSuccess)
        return 0;
    // `blocks` reservations fit, one more does not
    const unsigned want = static_cast<unsigned>(per_cu) / static_cast<unsigned>(blocks + 1) + 1024;
    return want <= static_cast<unsigned>(per_block) ? want : 0;
}

hipError_t launch_zero(float *p, uint64_t n, hipStream_t s) {
    Geometry geo;
    geo.max_blocks = 4096;
    hipLaunchKernelGGL(zero_f32, dim3(grid_for(n, geo)), dim3(kBlock), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace gadei
