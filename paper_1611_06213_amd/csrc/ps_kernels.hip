// HIP kernels of the parameter server for gfx950 (CDNA4).
//
// All three kernels are pure streams over HBM: every byte is read or written
// once per launch and there is no reuse to stage in LDS and no contraction
// for the matrix cores. What matters is that each wave moves whole, aligned
// 16-byte (fp32) or 8-byte (bf16) lanes, that enough loads are in flight per
// wave, and that nothing is re-read.
//
// apply:  for each coordinate i and each pending gradient k = 0..K-1, oldest
//         first, one ASGD step (Eq. "asgd" with the step of Eq. "gd"):
//           momentum == 0: p = lr*g; w = w - p
//           momentum != 0: t = m*v; v = t + g; p = lr*v; w = w - p
//         w (and v) are loaded once, the K gradients streamed past them in
//         registers, and the result stored once: K sequential steps cost one
//         pass over w instead of K. Optionally the same pass writes R replica
//         copies of the new w (a fused pull).
// pull:   load w once, write it to R replica buffers (fp32, or bf16 rounded
//         to nearest even).
//
// Every product and sum is rounded on its own (no fused multiply-add), so
// the result is bit-identical to sequential binary32 steps.
#include <hip/hip_runtime.h>

#include "ps_kernels.h"

#pragma clang fp contract(off)

namespace gadei {
namespace {

constexpr int kBlock = 256;   // 4 waves of 64 lanes
constexpr int kGroup = 8;     // gradients whose loads are issued together

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- loads

// E consecutive fp32 values starting at p (E = 4: one 16-byte load).
template <int E>
__device__ __forceinline__ void ld_f32(float (&x)[E], const float *p) {
    if constexpr (E == 4) {
        f32x4 t = *reinterpret_cast<const f32x4 *>(p);
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    } else {
        x[0] = *p;
    }
}

template <int E>
__device__ __forceinline__ void st_f32(float *p, const float (&x)[E]) {
    if constexpr (E == 4) {
        f32x4 t = {x[0], x[1], x[2], x[3]};
        *reinterpret_cast<f32x4 *>(p) = t;
    } else {
        *p = x[0];
    }
}

// bf16 -> fp32 is exact: the bf16 bits are the upper half of the fp32 bits.
__device__ __forceinline__ float lo_bf16(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

// Gradient values for coordinates i .. i+E-1. Gradients are read exactly once
// per launch, so the loads carry the non-temporal hint.
template <int GDT, int E>
__device__ __forceinline__ void ld_grad(float (&x)[E], const void *g, uint64_t i) {
    if constexpr (GDT == PS_F32) {
        if constexpr (E == 4) {
            f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(g) + (i >> 2));
            x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
        } else {
            x[0] = static_cast<const float *>(g)[i];
        }
    } else {
        if constexpr (E == 4) {
            u32x2 u = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(g) + (i >> 2));
            x[0] = lo_bf16(u.x); x[1] = hi_bf16(u.x);
            x[2] = lo_bf16(u.y); x[3] = hi_bf16(u.y);
        } else {
            x[0] = lo_bf16(static_cast<const uint16_t *>(g)[i]);
        }
    }
}

// fp32 -> bf16 bits, round to nearest, ties to even. Adding 0x7fff plus the
// lowest kept bit carries into the kept half exactly when the discarded half
// is above one half, or equal to it with an odd kept half. NaN keeps its sign
// and gets the quiet bit.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    uint32_t r = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    return ((u & 0x7fffffffu) > 0x7f800000u) ? ((u >> 16) | 0x40u) : r;
}

// One replica's values for coordinates i .. i+E-1. Replicas are not read
// back by the server, so the stores carry the non-temporal hint.
template <int PDT, int E>
__device__ __forceinline__ void st_dst(void *d, uint64_t i, const float (&x)[E]) {
    if constexpr (PDT == PS_F32) {
        if constexpr (E == 4) {
            f32x4 t = {x[0], x[1], x[2], x[3]};
            __builtin_nontemporal_store(t, reinterpret_cast<f32x4 *>(d) + (i >> 2));
        } else {
            static_cast<float *>(d)[i] = x[0];
        }
    } else {
        if constexpr (E == 4) {
            u32x2 t;
            t.x = bf16_rne(x[0]) | (bf16_rne(x[1]) << 16);
            t.y = bf16_rne(x[2]) | (bf16_rne(x[3]) << 16);
            __builtin_nontemporal_store(t, reinterpret_cast<u32x2 *>(d) + (i >> 2));
        } else {
            static_cast<uint16_t *>(d)[i] = static_cast<uint16_t>(bf16_rne(x[0]));
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

// Coordinates i .. i+E-1 through all K pending gradients, oldest first.
// Gradients go in groups of kGroup whose loads are all issued before the
// group's updates, so each lane keeps kGroup independent loads in flight;
// full groups carry no predicates (their pointer loads batch and the waits
// count down one load at a time), the last partial group is predicated.
template <bool MOM, int GDT, int PDT, int E>
__device__ __forceinline__ void apply_chunk(const ApplyArgs &a, uint64_t i) {
    float w[E], v[E];
    ld_f32<E>(w, a.w + i);
    if constexpr (MOM) ld_f32<E>(v, a.v + i);
    const float lr = a.lr;
    const float m = a.m;
    const int k = a.k;
    int k0 = 0;
    for (; k0 + kGroup <= k; k0 += kGroup) {
        float g[kGroup][E];
#pragma unroll
        for (int j = 0; j < kGroup; ++j) ld_grad<GDT, E>(g[j], a.g[k0 + j], i);
#pragma unroll
        for (int j = 0; j < kGroup; ++j) step<MOM, E>(w, v, g[j], lr, m);
    }
    if (k0 < k) {
        float g[kGroup][E];
#pragma unroll
        for (int j = 0; j < kGroup; ++j)
            if (k0 + j < k) ld_grad<GDT, E>(g[j], a.g[k0 + j], i);
#pragma unroll
        for (int j = 0; j < kGroup; ++j)
            if (k0 + j < k) step<MOM, E>(w, v, g[j], lr, m);
    }
    st_f32<E>(a.w + i, w);
    if constexpr (MOM) st_f32<E>(a.v + i, v);
    if constexpr (PDT >= 0) {
        for (int r = 0; r < a.r; ++r) st_dst<PDT, E>(a.dst[r], i, w);
    }
}

// Vector path: lane t of the grid owns 4-coordinate chunks t, t + stride, ...
// The n mod 4 trailing coordinates go to the first lanes of the grid.
template <bool MOM, int GDT, int PDT>
__global__ void __launch_bounds__(kBlock) apply_vec(const ApplyArgs a) {
    const uint64_t chunks = a.n >> 2;
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t c = tid; c < chunks; c += stride) apply_chunk<MOM, GDT, PDT, 4>(a, c << 2);
    if (tid < a.n - (chunks << 2)) apply_chunk<MOM, GDT, PDT, 1>(a, (chunks << 2) + tid);
}

// Scalar path for buffers without vector alignment: one coordinate per lane.
template <bool MOM, int GDT, int PDT>
__global__ void __launch_bounds__(kBlock) apply_scalar(const ApplyArgs a) {
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t i = tid; i < a.n; i += stride) apply_chunk<MOM, GDT, PDT, 1>(a, i);
}

// ---------------------------------------------------------------- pull

template <int PDT, int E>
__device__ __forceinline__ void pull_chunk(const PullArgs &a, uint64_t i) {
    float w[E];
    ld_f32<E>(w, a.w + i);
    for (int r = 0; r < a.r; ++r) st_dst<PDT, E>(a.dst[r], i, w);
}

template <int PDT>
__global__ void __launch_bounds__(kBlock) pull_vec(const PullArgs a) {
    const uint64_t chunks = a.n >> 2;
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t c = tid; c < chunks; c += stride) pull_chunk<PDT, 4>(a, c << 2);
    if (tid < a.n - (chunks << 2)) pull_chunk<PDT, 1>(a, (chunks << 2) + tid);
}

template <int PDT>
__global__ void __launch_bounds__(kBlock) pull_scalar(const PullArgs a) {
    const uint64_t tid = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kBlock;
    for (uint64_t i = tid; i < a.n; i += stride) pull_chunk<PDT, 1>(a, i);
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
    const uint64_t cap = geo.max_blocks > 0 ? static_cast<uint64_t>(geo.max_blocks) : 0x7fffffffull;
    return static_cast<unsigned>(blocks < cap ? blocks : cap);
}

template <bool MOM, int GDT, int PDT>
hipError_t go_apply(const ApplyArgs &a, bool vec, const Geometry &geo, hipStream_t s) {
    if (vec) {
        hipLaunchKernelGGL((apply_vec<MOM, GDT, PDT>), dim3(grid_for(a.n >> 2, geo)), dim3(kBlock),
                           0, s, a);
    } else {
        hipLaunchKernelGGL((apply_scalar<MOM, GDT, PDT>), dim3(grid_for(a.n, geo)), dim3(kBlock),
                           0, s, a);
    }
    return hipGetLastError();
}

template <bool MOM, int GDT>
hipError_t go_apply_p(const ApplyArgs &a, int pdt, bool vec, const Geometry &geo, hipStream_t s) {
    if (pdt == PS_F32) return go_apply<MOM, GDT, PS_F32>(a, vec, geo, s);
    if (pdt == PS_BF16) return go_apply<MOM, GDT, PS_BF16>(a, vec, geo, s);
    return go_apply<MOM, GDT, -1>(a, vec, geo, s);
}

template <bool MOM>
hipError_t go_apply_g(const ApplyArgs &a, int gdt, int pdt, bool vec, const Geometry &geo,
                      hipStream_t s) {
    if (gdt == PS_BF16) return go_apply_p<MOM, PS_BF16>(a, pdt, vec, geo, s);
    return go_apply_p<MOM, PS_F32>(a, pdt, vec, geo, s);
}

}  // namespace

hipError_t launch_apply(const ApplyArgs &a, int grad_dtype, int pull_dtype, bool vec,
                        const Geometry &geo, hipStream_t s) {
    if (a.r == 0) pull_dtype = -1;
    if (a.v != nullptr) return go_apply_g<true>(a, grad_dtype, pull_dtype, vec, geo, s);
    return go_apply_g<false>(a, grad_dtype, pull_dtype, vec, geo, s);
}

hipError_t launch_pull(const PullArgs &a, int pull_dtype, bool vec, const Geometry &geo,
                       hipStream_t s) {
    const uint64_t items = vec ? (a.n >> 2) : a.n;
    const dim3 grid(grid_for(items, geo)), block(kBlock);
    if (pull_dtype == PS_BF16) {
        if (vec) hipLaunchKernelGGL(pull_vec<PS_BF16>, grid, block, 0, s, a);
        else hipLaunchKernelGGL(pull_scalar<PS_BF16>, grid, block, 0, s, a);
    } else {
        if (vec) hipLaunchKernelGGL(pull_vec<PS_F32>, grid, block, 0, s, a);
        else hipLaunchKernelGGL(pull_scalar<PS_F32>, grid, block, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_zero(float *p, uint64_t n, hipStream_t s) {
    Geometry geo;
    geo.max_blocks = 4096;
    hipLaunchKernelGGL(zero_f32, dim3(grid_for(n, geo)), dim3(kBlock), 0, s, p, n);
    return hipGetLastError();
}

}  // namespace gadei
