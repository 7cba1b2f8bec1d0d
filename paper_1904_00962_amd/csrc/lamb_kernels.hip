// HIP kernels of the multi-tensor LAMB / LARS step for gfx950 (MI355X).
//
// You et al., "Large Batch Optimization for Deep Learning" (arXiv:1904.00962):
// LAMB is Algorithm 2, LARS is Algorithm 1, phi is defined in Section 3.
//
// The step needs every per-layer norm ||u_i|| before any x_i may move, so it
// is two streaming passes over HBM with a tiny reduction between them:
//
//   moments  (one workgroup per chunk): read x, g, m, v; write the new m, v;
//            write the chunk's sums of x^2 and u^2 to a fixed slot.
//   finalize (one wave64 per tensor):  sum the tensor's chunk slots in a
//            fixed order, form ||x_i||, ||u_i||, phi, the trust ratio and the
//            step scale lr * ratio.
//   apply    (one workgroup per chunk): read x and the new m, v; recompute u
//            with the same inline function the moment pass used (so it is
//            bit-identical) and write x - scale_i * u.
//
// Recomputing u instead of storing it saves 4 bytes per parameter of HBM
// traffic. There are no float atomics: every sum has a fixed order, so a step
// is bitwise reproducible for a given chunk size. Every global access of the
// vector loops is a 16-byte (fp32) or 8-byte (bf16) load or store, and the
// lanes of a wave touch consecutive addresses, so one instruction moves 1 KiB
// (fp32) or 512 B (bf16) of contiguous memory. This path has no dense
// contraction, so it uses no MFMA; it is bound by HBM bandwidth.

#include <hip/hip_runtime.h>

#include "lamb_internal.h"

namespace lamb_mi355x {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Tensor addresses come out of the descriptor table, so the compiler cannot
// tell they are global memory and would emit flat instructions. Every access
// goes through these global-address-space views instead.
#define LAMB_GLOBAL __attribute__((address_space(1)))
typedef LAMB_GLOBAL float gfloat;
typedef LAMB_GLOBAL const float gcfloat;
typedef LAMB_GLOBAL const uint16_t gcbf16;

__device__ __forceinline__ gfloat *global_view(float *p) { return (gfloat *)p; }
__device__ __forceinline__ gcfloat *global_view(const float *p) { return (gcfloat *)p; }

// Tuning knobs (compile-time; the defaults are the measured best on MI355X).
// LAMB_UNROLL: float4 groups each thread keeps in flight per loop trip.
// LAMB_NONTEMPORAL: stream x, g, m, v with nontemporal loads and stores; the
//   data is touched once per pass, so it should not displace cache lines.
// LAMB_APPLY_REVERSE: the apply pass walks chunks last-to-first, so its first
//   reads are the lines the moment pass touched last (still in the caches).
#ifndef LAMB_UNROLL
#define LAMB_UNROLL 2
#endif
#ifndef LAMB_NONTEMPORAL
#define LAMB_NONTEMPORAL 1
#endif
#ifndef LAMB_APPLY_REVERSE
#define LAMB_APPLY_REVERSE 1
#endif
#ifndef LAMB_XCD_CONTIGUOUS
#define LAMB_XCD_CONTIGUOUS 0
#endif
constexpr int kUnroll = LAMB_UNROLL;

template <typename T>
__device__ __forceinline__ T stream_load(LAMB_GLOBAL const T *p) {
#if LAMB_NONTEMPORAL
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void stream_store(LAMB_GLOBAL T *p, T v) {
#if LAMB_NONTEMPORAL
    __builtin_nontemporal_store(v, p);
#else
    *p = v;
#endif
}

__device__ __forceinline__ f32x4 load4(gcfloat *p) {
    return stream_load((LAMB_GLOBAL const f32x4 *)p);
}

__device__ __forceinline__ void store4(gfloat *p, f32x4 v) {
    stream_store((LAMB_GLOBAL f32x4 *)p, v);
}

// The gradient of one chunk: fp32, or bf16 bit patterns that widen exactly
// (a bf16 is the top half of an fp32).
template <bool kBf16>
struct GradView {
    const void *base;
    __device__ __forceinline__ GradView(const void *g, int64_t start)
        : base(kBf16 ? static_cast<const void *>(static_cast<const uint16_t *>(g) + start)
                     : static_cast<const void *>(static_cast<const float *>(g) + start)) {}

    __device__ __forceinline__ float at(int i) const {
        if constexpr (kBf16)
            return __uint_as_float(uint32_t(((gcbf16 *)base)[i]) << 16);
        else
            return ((gcfloat *)base)[i];
    }

    // elements i..i+3, i a multiple of 4
    __device__ __forceinline__ f32x4 at4(int i) const {
        if constexpr (kBf16) {
            const u32x2 w = stream_load((LAMB_GLOBAL const u32x2 *)((gcbf16 *)base + i));
            f32x4 r;
            r.x = __uint_as_float(w.x << 16);
            r.y = __uint_as_float(w.x & 0xffff0000u);
            r.z = __uint_as_float(w.y << 16);
            r.w = __uint_as_float(w.y & 0xffff0000u);
            return r;
        } else {
            return load4((gcfloat *)base + i);
        }
    }
};

// ---------------------------------------------------------------------------
// Elementwise arithmetic of Algorithm 2 (LAMB) and Algorithm 1 (LARS).
// ---------------------------------------------------------------------------

// m_t = beta1 m_{t-1} + (1 - beta1) g_t
__device__ __forceinline__ float lamb_first_moment(float m, float g, const LambArgs &a) {
    return fmaf(a.beta1, m, a.one_minus_beta1 * g);
}

// v_t = beta2 v_{t-1} + (1 - beta2) g_t^2
__device__ __forceinline__ float lamb_second_moment(float v, float g, const LambArgs &a) {
    return fmaf(a.beta2, v, a.one_minus_beta2 * (g * g));
}

// u = r + lambda x with r = m_hat / (sqrt(v_hat) + eps), from the NEW moments
// m = m_t, v = v_t. Algorithm 2 corrects by 1 / (1 - beta^t); Algorithms 3
// and 4 add the Nesterov gradient terms, which is why their apply pass also
// reads g. The moment and apply passes both call this, so their u agree bit
// for bit; division and square root are the correctly rounded IEEE
// operations.
template <int kVariant>
__device__ __forceinline__ float lamb_update(float x, float g, float m, float v, float lam,
                                             const LambArgs &a) {
    float m_hat, v_hat;
    if constexpr (kVariant == kLamb) {
        m_hat = m * a.m_scale;
        v_hat = v * a.v_scale;
    } else {
        m_hat = fmaf(a.m_scale, m, a.m_grad * g);
        if constexpr (kVariant == kNNLamb)
            v_hat = fmaf(a.v_scale, v, a.v_grad * (g * g));
        else
            v_hat = v * a.v_scale;
    }
    const float r = __fdiv_rn(m_hat, __fadd_rn(__fsqrt_rn(v_hat), a.eps));
    return fmaf(lam, x, r);
}

// m_t = beta1 m_{t-1} + (1 - beta1) (g_t + lambda x_t)
__device__ __forceinline__ float lars_momentum(float m, float g, float x, float lam,
                                               const LarsArgs &a) {
    return fmaf(a.beta1, m, a.one_minus_beta1 * fmaf(lam, x, g));
}

// ---------------------------------------------------------------------------
// Deterministic reductions.
// ---------------------------------------------------------------------------

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v += __shfl_xor(v, off, 64);
    return v;
}

// Sum (a, b) over a workgroup of kNumWaves wave64s in a fixed tree and store
// it at `out` (thread 0 writes).
template <int kNumWaves>
__device__ __forceinline__ void block_sums(double a, double b, Partial *out) {
    __shared__ double red_a[kNumWaves];
    __shared__ double red_b[kNumWaves];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    a = wave_sum(a);
    b = wave_sum(b);
    if (lane == 0) {
        red_a[wave] = a;
        red_b[wave] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double sa = red_a[0], sb = red_b[0];
#pragma unroll
        for (int w = 1; w < kNumWaves; ++w) {
            sa += red_a[w];
            sb += red_b[w];
        }
        out->sum_xx = sa;
        out->sum_uu = sb;
    }
}

// Workgroups are dispatched round-robin over the 8 XCDs. With
// LAMB_XCD_CONTIGUOUS each XCD takes one contiguous eighth of the chunk list
// instead of every eighth chunk.
__device__ __forceinline__ uint32_t dispatch_rank() {
#if LAMB_XCD_CONTIGUOUS
    const uint32_t n = gridDim.x, b = blockIdx.x;
    const uint32_t per = n / 8, extra = n % 8;  // XCDs 0..extra-1 get one more
    const uint32_t xcd = b % 8, k = b / 8;
    const uint32_t first = xcd * per + (xcd < extra ? xcd : extra);
    return first + k;
#else
    return blockIdx.x;
#endif
}

// Chunk handled by this workgroup of a moment pass.
__device__ __forceinline__ uint32_t chunk_index() { return dispatch_rank(); }

// Chunk handled by this workgroup of an apply pass.
__device__ __forceinline__ uint32_t apply_chunk_index() {
#if LAMB_APPLY_REVERSE
    return gridDim.x - 1 - dispatch_rank();
#else
    return dispatch_rank();
#endif
}

// ---------------------------------------------------------------------------
// LAMB passes.
// ---------------------------------------------------------------------------

template <bool kBf16, int kVariant>
__global__ __launch_bounds__(kBlock) void lamb_moments_kernel(
    const TensorDesc *__restrict__ tensors, const ChunkDesc *__restrict__ chunks,
    Partial *__restrict__ partials, LambArgs a) {
    const ChunkDesc c = chunks[chunk_index()];
    const TensorDesc &t = tensors[c.tensor];
    gcfloat *x = global_view(t.x + c.start);
    gfloat *m = global_view(t.m + c.start);
    gfloat *v = global_view(t.v + c.start);
    const GradView<kBf16> g(t.g, c.start);
    const float lam = t.wd ? a.weight_decay : 0.0f;

    double sum_xx = 0.0, sum_uu = 0.0;
    const int n4 = c.len >> 2;
    for (int base = threadIdx.x; base < n4; base += kBlock * kUnroll) {
        f32x4 xr[kUnroll], gr[kUnroll], mr[kUnroll], vr[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                xr[k] = load4(x + 4 * q);
                gr[k] = g.at4(4 * q);
                mr[k] = load4(m + 4 * q);
                vr[k] = load4(v + 4 * q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                f32x4 mn, vn;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    mn[e] = lamb_first_moment(mr[k][e], gr[k][e], a);
                    vn[e] = lamb_second_moment(vr[k][e], gr[k][e], a);
                    const float u = lamb_update<kVariant>(xr[k][e], gr[k][e], mn[e], vn[e], lam, a);
                    const double xd = xr[k][e], ud = u;
                    sum_xx = fma(xd, xd, sum_xx);
                    sum_uu = fma(ud, ud, sum_uu);
                }
                store4(m + 4 * q, mn);
                store4(v + 4 * q, vn);
            }
        }
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len) {
        const float xj = x[tail];
        const float gj = g.at(tail);
        const float mj = lamb_first_moment(m[tail], gj, a);
        const float vj = lamb_second_moment(v[tail], gj, a);
        const float u = lamb_update<kVariant>(xj, gj, mj, vj, lam, a);
        m[tail] = mj;
        v[tail] = vj;
        const double xd = xj, ud = u;
        sum_xx = fma(xd, xd, sum_xx);
        sum_uu = fma(ud, ud, sum_uu);
    }
    block_sums<kWaves>(sum_xx, sum_uu, partials + chunk_index());
}

// kVariant = kLamb never reads g (the template flag kBf16 is then unused).
template <bool kBf16, int kVariant>
__global__ __launch_bounds__(kBlock) void lamb_apply_kernel(
    const TensorDesc *__restrict__ tensors, const ChunkDesc *__restrict__ chunks,
    const float *__restrict__ scale, LambArgs a) {
    constexpr bool kReadsGrad = kVariant != kLamb;
    const ChunkDesc c = chunks[apply_chunk_index()];
    const TensorDesc &t = tensors[c.tensor];
    gfloat *x = global_view(t.x + c.start);
    gcfloat *m = global_view(static_cast<const float *>(t.m) + c.start);
    gcfloat *v = global_view(static_cast<const float *>(t.v) + c.start);
    const GradView<kBf16> g(t.g, c.start);
    const float lam = t.wd ? a.weight_decay : 0.0f;
    const float s = scale[c.tensor];

    const int n4 = c.len >> 2;
    for (int base = threadIdx.x; base < n4; base += kBlock * kUnroll) {
        f32x4 xr[kUnroll], gr[kUnroll], mr[kUnroll], vr[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                xr[k] = load4(x + 4 * q);
                if constexpr (kReadsGrad)
                    gr[k] = g.at4(4 * q);
                else
                    gr[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                mr[k] = load4(m + 4 * q);
                vr[k] = load4(v + 4 * q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                f32x4 xn;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    xn[e] = fmaf(-s, lamb_update<kVariant>(xr[k][e], gr[k][e], mr[k][e],
                                                           vr[k][e], lam, a),
                                 xr[k][e]);
                store4(x + 4 * q, xn);
            }
        }
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len) {
        const float gj = kReadsGrad ? g.at(tail) : 0.0f;
        x[tail] = fmaf(-s, lamb_update<kVariant>(x[tail], gj, m[tail], v[tail], lam, a), x[tail]);
    }
}

// ---------------------------------------------------------------------------
// LARS passes.
// ---------------------------------------------------------------------------

template <bool kBf16>
__global__ __launch_bounds__(kBlock) void lars_moments_kernel(
    const TensorDesc *__restrict__ tensors, const ChunkDesc *__restrict__ chunks,
    Partial *__restrict__ partials, LarsArgs a) {
    const ChunkDesc c = chunks[chunk_index()];
    const TensorDesc &t = tensors[c.tensor];
    gcfloat *x = global_view(static_cast<const float *>(t.x) + c.start);
    gfloat *m = global_view(t.m + c.start);
    const GradView<kBf16> g(t.g, c.start);
    const float lam = t.wd ? a.weight_decay : 0.0f;

    double sum_xx = 0.0, sum_mm = 0.0;
    const int n4 = c.len >> 2;
    for (int base = threadIdx.x; base < n4; base += kBlock * kUnroll) {
        f32x4 xr[kUnroll], gr[kUnroll], mr[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                xr[k] = load4(x + 4 * q);
                gr[k] = g.at4(4 * q);
                mr[k] = load4(m + 4 * q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                f32x4 mn;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    mn[e] = lars_momentum(mr[k][e], gr[k][e], xr[k][e], lam, a);
                    const double xd = xr[k][e], md = mn[e];
                    sum_xx = fma(xd, xd, sum_xx);
                    sum_mm = fma(md, md, sum_mm);
                }
                store4(m + 4 * q, mn);
            }
        }
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len) {
        const float xj = x[tail];
        const float mj = lars_momentum(m[tail], g.at(tail), xj, lam, a);
        m[tail] = mj;
        const double xd = xj, md = mj;
        sum_xx = fma(xd, xd, sum_xx);
        sum_mm = fma(md, md, sum_mm);
    }
    block_sums<kWaves>(sum_xx, sum_mm, partials + chunk_index());
}

__global__ __launch_bounds__(kBlock) void lars_apply_kernel(
    const TensorDesc *__restrict__ tensors, const ChunkDesc *__restrict__ chunks,
    const float *__restrict__ scale) {
    const ChunkDesc c = chunks[apply_chunk_index()];
    const TensorDesc &t = tensors[c.tensor];
    gfloat *x = global_view(t.x + c.start);
    gcfloat *m = global_view(static_cast<const float *>(t.m) + c.start);
    const float s = scale[c.tensor];

    const int n4 = c.len >> 2;
    for (int base = threadIdx.x; base < n4; base += kBlock * kUnroll) {
        f32x4 xr[kUnroll], mr[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                xr[k] = load4(x + 4 * q);
                mr[k] = load4(m + 4 * q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * kBlock;
            if (q < n4) {
                f32x4 xn;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    xn[e] = fmaf(-s, mr[k][e], xr[k][e]);
                store4(x + 4 * q, xn);
            }
        }
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len)
        x[tail] = fmaf(-s, m[tail], x[tail]);
}

// ---------------------------------------------------------------------------
// Per-tensor finalize: norms, phi, trust ratio, step scale. One workgroup of
// kFinalizeBlock threads per tensor. Thread k owns slots k + j*kFinalizeBlock
// and sums them into kFinalizeLanes independent accumulators (so several
// loads are in flight), which it then adds in a fixed order; the fixed
// wave/LDS tree combines the threads. The order never depends on timing.
// ---------------------------------------------------------------------------

constexpr int kFinalizeBlock = 1024;
constexpr int kFinalizeLanes = 16;

__global__ __launch_bounds__(kFinalizeBlock) void finalize_kernel(
    const TensorDesc *__restrict__ tensors, const Partial *__restrict__ partials,
    FinalizeArgs a, float *__restrict__ scale, double *__restrict__ ratio_out,
    double *__restrict__ norms_out) {
    const int i = blockIdx.x;
    const TensorDesc &t = tensors[i];
    const Partial *p = partials + t.first_chunk;
    const int n = t.n_chunks;
    double sx[kFinalizeLanes] = {}, su[kFinalizeLanes] = {};
    int k = threadIdx.x;
    for (; k + (kFinalizeLanes - 1) * kFinalizeBlock < n; k += kFinalizeLanes * kFinalizeBlock) {
#pragma unroll
        for (int j = 0; j < kFinalizeLanes; ++j) {
            const Partial q = p[k + j * kFinalizeBlock];
            sx[j] += q.sum_xx;
            su[j] += q.sum_uu;
        }
    }
#pragma unroll
    for (int j = 0; j < kFinalizeLanes - 1; ++j) {
        if (k + j * kFinalizeBlock < n) {
            const Partial q = p[k + j * kFinalizeBlock];
            sx[j] += q.sum_xx;
            su[j] += q.sum_uu;
        }
    }
#pragma unroll
    for (int j = 1; j < kFinalizeLanes; ++j) {
        sx[0] += sx[j];
        su[0] += su[j];
    }
    __shared__ Partial total;
    block_sums<kFinalizeBlock / 64>(sx[0], su[0], &total);
    __syncthreads();
    if (threadIdx.x == 0) {
        const double norm_x = sqrt(total.sum_xx);
        const double norm_u = sqrt(total.sum_uu);
        // phi(z) = min(max(z, gamma_l), gamma_u), Section 3; comparisons keep NaN.
        double phi = norm_x;
        if (phi < a.gamma_l)
            phi = a.gamma_l;
        if (phi > a.gamma_u)
            phi = a.gamma_u;
        // A zero update norm means a zero update: report ratio 0, move nothing.
        const double ratio = (norm_u == 0.0) ? 0.0 : a.trust_coef * phi / norm_u;
        scale[i] = static_cast<float>(a.lr * ratio);
        if (ratio_out)
            ratio_out[i] = ratio;
        if (norms_out) {
            norms_out[2 * i] = norm_x;
            norms_out[2 * i + 1] = norm_u;
        }
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------

template <int kVariant>
const void *moments_fn(bool bf16) {
    return bf16 ? reinterpret_cast<const void *>(&lamb_moments_kernel<true, kVariant>)
                : reinterpret_cast<const void *>(&lamb_moments_kernel<false, kVariant>);
}

hipError_t launch_lamb_moments(const TensorDesc *tensors, const ChunkDesc *chunks,
                               Partial *partials, int32_t n_chunks, bool bf16_grad,
                               LambVariant variant, const LambArgs &args, hipStream_t stream) {
    LambArgs a = args;
    void *params[] = {&tensors, &chunks, &partials, &a};
    const void *fn = variant == kNLamb    ? moments_fn<kNLamb>(bf16_grad)
                     : variant == kNNLamb ? moments_fn<kNNLamb>(bf16_grad)
                                          : moments_fn<kLamb>(bf16_grad);
    return hipLaunchKernel(fn, dim3(n_chunks), dim3(kBlock), params, 0, stream);
}

hipError_t launch_lamb_apply(const TensorDesc *tensors, const ChunkDesc *chunks,
                             const float *scale, int32_t n_chunks, bool bf16_grad,
                             LambVariant variant, const LambArgs &args, hipStream_t stream) {
    LambArgs a = args;
    void *params[] = {&tensors, &chunks, &scale, &a};
    const void *fn;
    if (variant == kNLamb)
        fn = bf16_grad ? reinterpret_cast<const void *>(&lamb_apply_kernel<true, kNLamb>)
                       : reinterpret_cast<const void *>(&lamb_apply_kernel<false, kNLamb>);
    else if (variant == kNNLamb)
        fn = bf16_grad ? reinterpret_cast<const void *>(&lamb_apply_kernel<true, kNNLamb>)
                       : reinterpret_cast<const void *>(&lamb_apply_kernel<false, kNNLamb>);
    else
        fn = reinterpret_cast<const void *>(&lamb_apply_kernel<false, kLamb>);
    return hipLaunchKernel(fn, dim3(n_chunks), dim3(kBlock), params, 0, stream);
}

hipError_t launch_lars_moments(const TensorDesc *tensors, const ChunkDesc *chunks,
                               Partial *partials, int32_t n_chunks, bool bf16_grad,
                               const LarsArgs &args, hipStream_t stream) {
    LarsArgs a = args;
    void *params[] = {&tensors, &chunks, &partials, &a};
    const void *fn = bf16_grad ? reinterpret_cast<const void *>(&lars_moments_kernel<true>)
                               : reinterpret_cast<const void *>(&lars_moments_kernel<false>);
    return hipLaunchKernel(fn, dim3(n_chunks), dim3(kBlock), params, 0, stream);
}

hipError_t launch_lars_apply(const TensorDesc *tensors, const ChunkDesc *chunks,
                             const float *scale, int32_t n_chunks, hipStream_t stream) {
    void *params[] = {&tensors, &chunks, &scale};
    return hipLaunchKernel(reinterpret_cast<const void *>(&lars_apply_kernel), dim3(n_chunks),
                           dim3(kBlock), params, 0, stream);
}

hipError_t launch_finalize(const TensorDesc *tensors, int32_t n_tensors,
                           const Partial *partials, const FinalizeArgs &args, float *scale,
                           double *ratio_out, double *norms_out, hipStream_t stream) {
    FinalizeArgs a = args;
    void *params[] = {&tensors, &partials, &a, &scale, &ratio_out, &norms_out};
    return hipLaunchKernel(reinterpret_cast<const void *>(&finalize_kernel), dim3(n_tensors),
                           dim3(kFinalizeBlock), params, 0, stream);
}

}  // namespace lamb_mi355x
