// HBM streams with the access pattern of the optimizer's kernels and none of
// their arithmetic: the attainable bandwidth for each kernel's traffic (see
// include/stream_probe.h). Each workgroup of 256 threads streams one tile of
// `tile` elements, two float4 groups per thread in flight, with nontemporal
// 16-byte loads and stores (8-byte loads for bf16 g), like the kernels. A
// partial last float4 group is skipped (the probe measures rates, n is large).

#include <hip/hip_runtime.h>

#include "stream_probe.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
#define PROBE_GLOBAL __attribute__((address_space(1)))

constexpr int kThreads = 256;
constexpr int kUnroll = 2;

__device__ __forceinline__ f32x4 ld4(const float *p) {
    return __builtin_nontemporal_load((PROBE_GLOBAL const f32x4 *)p);
}
__device__ __forceinline__ void st4(float *p, f32x4 v) {
    __builtin_nontemporal_store(v, (PROBE_GLOBAL f32x4 *)p);
}

template <bool kBf16>
__device__ __forceinline__ f32x4 ldg(const void *g, int64_t i) {
    if constexpr (kBf16) {
        const u32x2 w = __builtin_nontemporal_load(
            (PROBE_GLOBAL const u32x2 *)(static_cast<const uint16_t *>(g) + i));
        return f32x4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                     __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u)};
    } else {
        return ld4(static_cast<const float *>(g) + i);
    }
}

// kR*: the array is read; kW*: it is written. Written values are the read
// values plus a term built from every loaded value whose bits are masked by
// `keep`, which is 0 at run time: the term is then exactly -0.0, so every
// array keeps its values (NaN payloads aside) while the compiler cannot drop
// a load or a store.
// Element offset of float4 group q of workgroup b: contiguous tiles, or,
// with `layer_tiles` > 0, the layer-cyclic deal of the single-pass kernel
// (the array cut into layers of layer_tiles tiles; tile i of a layer holds
// its 1024-element blocks i, i + layer_tiles, ...).
__device__ __forceinline__ int64_t element(int64_t b, int q, int32_t tile, int32_t layer_tiles) {
    if (layer_tiles <= 0)
        return b * tile + 4 * int64_t(q);
    const int64_t layer = b / layer_tiles, i = b % layer_tiles;
    const int64_t block = int64_t(q / kThreads) * layer_tiles + i;
    return (layer * layer_tiles) * int64_t(tile) + block * (4 * kThreads) + 4 * (q % kThreads);
}

template <bool kBf16, bool kRX, bool kWX, bool kRM, bool kWM, bool kRV, bool kWV, bool kRG>
__global__ __launch_bounds__(kThreads) void stream_kernel(float *x, float *m, float *v,
                                                        const void *g, int64_t n, int32_t tile,
                                                        int32_t layer_tiles, uint32_t keep,
                                                        float *sink) {
    const int n4 = tile >> 2;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int base = threadIdx.x; base < n4; base += kThreads * kUnroll) {
        f32x4 xr[kUnroll], mr[kUnroll], vr[kUnroll], gr[kUnroll];
        int64_t at[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kThreads;
            at[k] = element(blockIdx.x, q, tile, layer_tiles);
            xr[k] = mr[k] = vr[k] = gr[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            if (q < n4 && at[k] + 4 <= n) {
                const int64_t i = at[k];
                if constexpr (kRX) xr[k] = ld4(x + i);
                if constexpr (kRM) mr[k] = ld4(m + i);
                if constexpr (kRV) vr[k] = ld4(v + i);
                if constexpr (kRG) gr[k] = ldg<kBf16>(g, i);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kThreads;
            if (q < n4 && at[k] + 4 <= n) {
                const int64_t i = at[k];
                const f32x4 sum = xr[k] + mr[k] + vr[k] + gr[k];
                f32x4 t;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    t[e] = __uint_as_float((__float_as_uint(sum[e]) & keep) | 0x80000000u);
                if constexpr (kWX) st4(x + i, (kRX ? xr[k] : mr[k]) + t);
                if constexpr (kWM) st4(m + i, mr[k] + t);
                if constexpr (kWV) st4(v + i, vr[k] + t);
                acc += sum;
            }
        }
    }
    // Read-only streams: keep the loads alive through a store that never happens.
    if (keep != 0u && sink)
        sink[blockIdx.x * kThreads + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

template <bool kBf16>
const void *pick(int pattern) {
    switch (pattern) {
    case STREAM_SINGLE_PASS:
        return reinterpret_cast<const void *>(
            &stream_kernel<kBf16, true, true, true, true, true, true, true>);
    case STREAM_MOMENTS:
        return reinterpret_cast<const void *>(
            &stream_kernel<kBf16, true, false, true, true, true, true, true>);
    case STREAM_APPLY:
        return reinterpret_cast<const void *>(
            &stream_kernel<kBf16, true, true, true, false, true, false, false>);
    case STREAM_READ:
        return reinterpret_cast<const void *>(
            &stream_kernel<kBf16, true, false, true, false, true, false, true>);
    default:
        return reinterpret_cast<const void *>(
            &stream_kernel<kBf16, false, true, true, false, false, false, false>);
    }
}

}  // namespace

extern "C" int stream_probe(int32_t pattern, float *x, float *m, float *v, const void *g,
                            int32_t g_bf16, int64_t n, int32_t tile, int32_t layer_tiles,
                            void *stream) {
    if (pattern < STREAM_SINGLE_PASS || pattern > STREAM_COPY || n < 1 || tile < 8 ||
        tile > (1 << 24) || tile % 8 != 0 || (g_bf16 != 0 && g_bf16 != 1) || layer_tiles < 0 ||
        (layer_tiles > 0 && tile % (4 * kThreads) != 0))
        return -1;
    const bool reads_g =
        pattern == STREAM_SINGLE_PASS || pattern == STREAM_MOMENTS || pattern == STREAM_READ;
    if (!x || !m || (pattern != STREAM_COPY && !v) || (reads_g && !g))
        return -1;
    const uintptr_t mask = reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(m) |
                           reinterpret_cast<uintptr_t>(v) | reinterpret_cast<uintptr_t>(g);
    if (mask & 15u)
        return -1;
    int64_t blocks = (n + tile - 1) / tile;
    if (layer_tiles > 0)  // whole layers: tiles past the end find no element
        blocks = (blocks + layer_tiles - 1) / layer_tiles * layer_tiles;
    if (blocks > 0x7fffffff)
        return -1;
    uint32_t keep = 0u;
    float *sink = nullptr;
    void *params[] = {&x, &m, &v, &g, &n, &tile, &layer_tiles, &keep, &sink};
    const void *fn = g_bf16 ? pick<true>(pattern) : pick<false>(pattern);
    hipError_t err = hipLaunchKernel(fn, dim3(unsigned(blocks)), dim3(kThreads), params, 0,
                                     static_cast<hipStream_t>(stream));
    return err == hipSuccess ? 0 : -5;
}
