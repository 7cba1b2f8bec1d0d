// HIP kernels of the multi-tensor LAMB-family and LARS step for gfx950
// (MI355X).
//
// You et al., "Large Batch Optimization for Deep Learning" (arXiv:1904.00962):
// LARS is Algorithm 1, LAMB Algorithm 2, N-LAMB and NN-LAMB Algorithms 3 and 4
// (Appendix D); phi is defined in Section 3, the other layer norms in
// Appendix F.
//
// The step needs every per-layer norm ||u_i|| before any x_i may move, so it
// is two streaming passes over HBM with a tiny reduction between them:
//
//   moments  (one workgroup per chunk, sized to it: one thread per float4 in
//            whole waves, at most 256): read x, g, m (and v); form the new
//            moments and the update direction u (m_t for LARS); write the
//            chunk's partial norms of x and u to a fixed slot; store the new
//            moments (direct mode) or nothing (deferred mode).
//   finalize (two small kernels): fold runs of chunk slots into segment
//            slots, then per tensor combine its segment slots in a fixed
//            order into ||x_i||, ||u_i||, phi, the trust ratio and the step
//            scale lr * ratio.
//   apply    (one workgroup per chunk): read x and the moments; recompute u
//            with the same inline functions the moment pass used (so it is
//            bit-identical) and write x - scale_i * u. In deferred mode it
//            recomputes the new moments from the old ones and writes them
//            too, unless the moment pass found a non-finite scaled gradient,
//            in which case nothing changes.
//
// A layer small enough to sit on chip in the resident workgroups takes a
// single pass instead (fused_kernel below): each tile's x (in LDS, part of it
// in registers for the wider tile) and u (in registers) stay there while the
// layer's partial norms meet, so x, g, m, v are read and x, m, v written
// exactly once. A step that skips on a non-finite gradient first runs a
// read-only check of g (finite_kernel) whose verdict every later kernel of
// the step reads.
//
// Recomputing u instead of storing it saves 4 bytes per parameter of HBM
// traffic. There are no float atomics: every reduction has a fixed order, so
// a step is bitwise reproducible for a given chunk size. The vector loops
// move 16 bytes per lane (8 for bf16 gradients) with nontemporal loads and
// stores, and the lanes of a wave touch consecutive addresses. This path has
// no dense contraction, so it uses no MFMA; it is bound by HBM bandwidth.

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

// Float4 groups each thread of the two-pass kernels keeps in flight per loop
// trip (a default chunk gives every thread one).
constexpr int kUnroll = 2;

// Every streamed access is nontemporal: x, g, m, v are touched once per pass
// and should not displace cache lines (10% faster than plain accesses).
template <typename T>
__device__ __forceinline__ T stream_load(LAMB_GLOBAL const T *p) {
    return __builtin_nontemporal_load(p);
}

template <typename T>
__device__ __forceinline__ void stream_store(LAMB_GLOBAL T *p, T v) {
    __builtin_nontemporal_store(v, p);
}

__device__ __forceinline__ f32x4 load4(gcfloat *p) {
    return stream_load((LAMB_GLOBAL const f32x4 *)p);
}

__device__ __forceinline__ void store4(gfloat *p, f32x4 v) {
    stream_store((LAMB_GLOBAL f32x4 *)p, v);
}

// Element i of a float array as a 32-bit byte offset from a uniform base, so
// that the loads and stores take the base in scalar registers and one VGPR of
// offset (arrays of the single pass stay far below 4 GiB).
__device__ __forceinline__ f32x4 load4_at(gcfloat *base, uint32_t i) {
    return stream_load((LAMB_GLOBAL const f32x4 *)((LAMB_GLOBAL const char *)base + i * 4u));
}

__device__ __forceinline__ void store4_at(gfloat *base, uint32_t i, f32x4 v) {
    stream_store((LAMB_GLOBAL f32x4 *)((LAMB_GLOBAL char *)base + i * 4u), v);
}

// The gradient of one chunk: fp32, or bf16 bit patterns that widen exactly
// (a bf16 is the top half of an fp32), multiplied by the step's grad_scale.
template <bool kBf16>
struct GradView {
    const void *base;
    float scale;
    __device__ __forceinline__ GradView(const void *g, int64_t start, float s)
        : base(kBf16 ? static_cast<const void *>(static_cast<const uint16_t *>(g) + start)
                     : static_cast<const void *>(static_cast<const float *>(g) + start)),
          scale(s) {}

    __device__ __forceinline__ float at(int i) const {
        float r;
        if constexpr (kBf16)
            r = __uint_as_float(uint32_t(((gcbf16 *)base)[i]) << 16);
        else
            r = ((gcfloat *)base)[i];
        return r * scale;
    }

    // elements i..i+3 at a 32-bit byte offset, i a multiple of 4
    __device__ __forceinline__ f32x4 at4_off(uint32_t i) const {
        f32x4 r;
        if constexpr (kBf16) {
            const u32x2 w = stream_load(
                (LAMB_GLOBAL const u32x2 *)((LAMB_GLOBAL const char *)base + i * 2u));
            r.x = __uint_as_float(w.x << 16);
            r.y = __uint_as_float(w.x & 0xffff0000u);
            r.z = __uint_as_float(w.y << 16);
            r.w = __uint_as_float(w.y & 0xffff0000u);
        } else {
            r = load4_at((gcfloat *)base, i);
        }
        return r * scale;
    }

    // elements i..i+3, i a multiple of 4
    __device__ __forceinline__ f32x4 at4(int i) const {
        f32x4 r;
        if constexpr (kBf16) {
            const u32x2 w = stream_load((LAMB_GLOBAL const u32x2 *)((gcbf16 *)base + i));
            r.x = __uint_as_float(w.x << 16);
            r.y = __uint_as_float(w.x & 0xffff0000u);
            r.z = __uint_as_float(w.y << 16);
            r.w = __uint_as_float(w.y & 0xffff0000u);
        } else {
            r = load4((gcfloat *)base + i);
        }
        return r * scale;
    }
};

// bf16 bit pattern of an fp32 value, rounded to nearest with ties to even
// (NaN becomes the quiet NaN 0x7fc0). Adding 0x7fff plus the lowest kept bit
// and truncating rounds the dropped half correctly; a carry moves into the
// exponent, so the largest finite values round to infinity.
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t b = __float_as_uint(f);
    if ((b & 0x7fffffffu) > 0x7f800000u)
        return 0x7fc0u;
    return (b + 0x7fffu + ((b >> 16) & 1u)) >> 16;
}

typedef LAMB_GLOBAL uint16_t gbf16;

// ---------------------------------------------------------------------------
// Elementwise arithmetic of Algorithms 1-4.
// ---------------------------------------------------------------------------

template <int kAlgo>
constexpr bool kHasSecondMoment = kAlgo != kLars;

// Nesterov variants need g_t to form the corrected moments, so their apply
// pass reads the gradient again.
template <int kAlgo>
constexpr bool kDirectionNeedsGrad = kAlgo == kNLamb || kAlgo == kNNLamb;

// New moments from the old ones, in place:
//   LAMB family: m_t = beta1 m + (1 - beta1) g,  v_t = beta2 v + (1 - beta2) g^2
//   LARS:        m_t = beta1 m + (1 - beta1) (g + lambda x)
template <int kAlgo>
__device__ __forceinline__ void new_moments(float x, float g, float lam, float &m, float &v,
                                            const StepArgs &a) {
    if constexpr (kAlgo == kLars) {
        m = fmaf(a.beta1, m, a.one_minus_beta1 * fmaf(lam, x, g));
    } else {
        m = fmaf(a.beta1, m, a.one_minus_beta1 * g);
        v = fmaf(a.beta2, v, a.one_minus_beta2 * (g * g));
    }
}

// The update direction from the NEW moments m = m_t, v = v_t: for the LAMB
// family u = r + lambda x with r = m_hat / (sqrt(v_hat) + eps); for LARS it is
// m_t itself. The moment and apply passes both call this, so their u agree
// bit for bit; division and square root are the correctly rounded IEEE
// operations.
template <int kAlgo>
__device__ __forceinline__ float direction(float x, float g, float m, float v, float lam,
                                           const StepArgs &a) {
    if constexpr (kAlgo == kLars) {
        return m;
    } else {
        float m_hat, v_hat;
        if constexpr (kAlgo == kLamb) {
            m_hat = m * a.m_scale;
            v_hat = v * a.v_scale;
        } else {
            m_hat = fmaf(a.m_scale, m, a.m_grad * g);
            if constexpr (kAlgo == kNNLamb)
                v_hat = fmaf(a.v_scale, v, a.v_grad * (g * g));
            else
                v_hat = v * a.v_scale;
        }
        const float r = __fdiv_rn(m_hat, __fadd_rn(__fsqrt_rn(v_hat), a.eps));
        return fmaf(lam, x, r);
    }
}

// ---------------------------------------------------------------------------
// Layer norms (Appendix F) and their deterministic reductions, in fp64.
// ---------------------------------------------------------------------------

// Maximum that keeps NaN: once a NaN is seen the result is NaN.
__device__ __forceinline__ double max_keep_nan(double a, double b) {
    return (isnan(a) || a > b) ? a : b;
}

template <int kNorm>
__device__ __forceinline__ double norm_add(double acc, float value) {
    const double d = value;
    if constexpr (kNorm == kL1)
        return acc + fabs(d);
    else if constexpr (kNorm == kLinf)
        return max_keep_nan(fabs(d), acc);
    else
        return fma(d, d, acc);
}

template <int kNorm>
__device__ __forceinline__ double norm_combine(double a, double b) {
    if constexpr (kNorm == kLinf)
        return max_keep_nan(a, b);
    else
        return a + b;
}

template <int kNorm>
__device__ __forceinline__ double norm_finish(double acc) {
    if constexpr (kNorm == kL2)
        return sqrt(acc);
    else
        return acc;
}

template <int kNorm>
__device__ __forceinline__ double wave_combine(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v = norm_combine<kNorm>(v, __shfl_xor(v, off, 64));
    return v;
}

// Combine (a, b) over a workgroup of kNumWaves wave64s in a fixed tree and
// store it at `out` (thread 0 writes).
template <int kNorm, int kNumWaves>
__device__ __forceinline__ void block_combine(double a, double b, Partial *out) {
    __shared__ double red_a[kNumWaves];
    __shared__ double red_b[kNumWaves];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    a = wave_combine<kNorm>(a);
    b = wave_combine<kNorm>(b);
    if (lane == 0) {
        red_a[wave] = a;
        red_b[wave] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double sa = red_a[0], sb = red_b[0];
#pragma unroll
        for (int w = 1; w < kNumWaves; ++w) {
            sa = norm_combine<kNorm>(sa, red_a[w]);
            sb = norm_combine<kNorm>(sb, red_b[w]);
        }
        out->sum_xx = sa;
        out->sum_uu = sb;
    }
}

// block_combine over a workgroup of blockDim.x threads (whole waves, at most
// kWaves of them): the same fixed tree; a single wave needs no LDS.
template <int kNorm>
__device__ __forceinline__ void block_combine_any(double a, double b, Partial *out) {
    if (blockDim.x == 64) {
        a = wave_combine<kNorm>(a);
        b = wave_combine<kNorm>(b);
        if (threadIdx.x == 0) {
            out->sum_xx = a;
            out->sum_uu = b;
        }
        return;
    }
    __shared__ double red_a[kWaves];
    __shared__ double red_b[kWaves];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int waves = int(blockDim.x >> 6);
    a = wave_combine<kNorm>(a);
    b = wave_combine<kNorm>(b);
    if (lane == 0) {
        red_a[wave] = a;
        red_b[wave] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double sa = red_a[0], sb = red_b[0];
        for (int w = 1; w < waves; ++w) {
            sa = norm_combine<kNorm>(sa, red_a[w]);
            sb = norm_combine<kNorm>(sb, red_b[w]);
        }
        out->sum_xx = sa;
        out->sum_uu = sb;
    }
}

// Chunk handled by this workgroup of a moment pass. Workgroups are dealt
// round-robin over the 8 XCDs, so consecutive chunks run on different XCDs
// (giving each XCD runs of consecutive chunks was 3% slower).
__device__ __forceinline__ uint32_t chunk_index() { return blockIdx.x; }

// Chunk handled by this workgroup of an apply pass: the chunks last to first,
// so the apply pass starts on the lines the moment pass touched last.
__device__ __forceinline__ uint32_t apply_chunk_index() { return gridDim.x - 1 - blockIdx.x; }

// ---------------------------------------------------------------------------
// Moment pass.
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t ctl_load(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Whether a two-pass kernel must do nothing: the plan's single pass gave up a
// wait (`fault`, the sticky fault word, so that no layer moves after a
// give-up), or, for a direct-mode pass of a step whose verdict the finiteness
// check took, that verdict (`guard`, a Guard value) is raised. The kernels
// load the fault word before their chunk-table entry, so its latency hides
// behind that load.
__device__ __forceinline__ bool pass_stopped(uint32_t fault, const uint32_t *flags,
                                             const uint32_t *ctl, int32_t guard) {
    if (guard == kGuardEpoch && flags[kVerdictWord + (ctl[kCtlEpoch] & 1u)] != 0)
        return true;
    if (guard == kGuardCopy && flags[1] != 0)
        return true;
    return fault != 0;
}

// Chunk k of a table of `chunk`-element chunks whose tensor ids are `ids`:
// tensor i's chunks are consecutive from `first` (its first_chunk, or its
// first_coarse in the coarse table), the last one ragged. A 4-byte id per
// chunk instead of a 16-byte descriptor keeps the table's share of the
// traffic small: consecutive chunks run on different XCDs, and each XCD's L2
// fetches every line of the table.
template <bool kCoarse>
__device__ __forceinline__ ChunkDesc chunk_at(const TensorDesc *tensors, const int32_t *ids,
                                              uint32_t k, int32_t chunk) {
    const int32_t i = ids[k];
    const TensorDesc &t = tensors[i];
    const int32_t first = kCoarse ? t.first_coarse : t.first_chunk;
    const int64_t start = int64_t(int32_t(k) - first) * chunk;
    const int64_t left = t.numel - start;
    return ChunkDesc{i, int32_t(left < chunk ? left : chunk), start};
}

template <int kAlgo, bool kBf16, int kNorm, bool kDeferred>
__global__ __launch_bounds__(kBlock) void moments_kernel(
    const TensorDesc *__restrict__ tensors, const int32_t *__restrict__ chunk_ids,
    int32_t chunk_elems, Partial *__restrict__ partials, uint32_t *__restrict__ flags,
    const uint32_t *__restrict__ ctl, int32_t guard, StepArgs a) {
    constexpr bool kV = kHasSecondMoment<kAlgo>;
    const uint32_t fault = ctl_load(ctl + kCtlFault);
    const ChunkDesc c = chunk_at<kDeferred>(tensors, chunk_ids, chunk_index(), chunk_elems);
    if (pass_stopped(fault, flags, ctl, kDeferred ? int32_t(kGuardNone) : guard))
        return;
    const TensorDesc &t = tensors[c.tensor];
    gcfloat *x = global_view(static_cast<const float *>(t.x) + c.start);
    gfloat *m = global_view(t.m + c.start);
    gfloat *v = kV ? global_view(t.v + c.start) : nullptr;
    const GradView<kBf16> g(t.g, c.start, a.grad_scale);
    const float lam = t.wd ? a.weight_decay : 0.0f;

    double sum_xx = 0.0, sum_uu = 0.0;
    bool nonfinite = false;
    const int n4 = c.len >> 2;
    const int stride = int(blockDim.x);
    for (int base = threadIdx.x; base < n4; base += stride * kUnroll) {
        f32x4 xr[kUnroll], gr[kUnroll], mr[kUnroll], vr[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * stride;
            if (q < n4) {
                xr[k] = load4(x + 4 * q);
                gr[k] = g.at4(4 * q);
                mr[k] = load4(m + 4 * q);
                if constexpr (kV)
                    vr[k] = load4(v + 4 * q);
                else
                    vr[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * stride;
            if (q < n4) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float me = mr[k][e], ve = vr[k][e];
                    new_moments<kAlgo>(xr[k][e], gr[k][e], lam, me, ve, a);
                    const float u = direction<kAlgo>(xr[k][e], gr[k][e], me, ve, lam, a);
                    sum_xx = norm_add<kNorm>(sum_xx, xr[k][e]);
                    sum_uu = norm_add<kNorm>(sum_uu, u);
                    mr[k][e] = me;
                    vr[k][e] = ve;
                    if constexpr (kDeferred)
                        nonfinite |= !isfinite(gr[k][e]);
                }
                if constexpr (!kDeferred) {
                    store4(m + 4 * q, mr[k]);
                    if constexpr (kV)
                        store4(v + 4 * q, vr[k]);
                }
            }
        }
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len) {
        const float xj = x[tail];
        const float gj = g.at(tail);
        float mj = m[tail];
        float vj = kV ? v[tail] : 0.0f;
        new_moments<kAlgo>(xj, gj, lam, mj, vj, a);
        const float u = direction<kAlgo>(xj, gj, mj, vj, lam, a);
        sum_xx = norm_add<kNorm>(sum_xx, xj);
        sum_uu = norm_add<kNorm>(sum_uu, u);
        if constexpr (kDeferred) {
            nonfinite |= !isfinite(gj);
        } else {
            m[tail] = mj;
            if constexpr (kV)
                v[tail] = vj;
        }
    }
    if constexpr (kDeferred) {
        // Rare event: one integer atomic per chunk that saw a bad gradient.
        if (__syncthreads_or(nonfinite) && threadIdx.x == 0)
            atomicOr(flags, 1u);
    }
    block_combine_any<kNorm>(sum_xx, sum_uu, partials + chunk_index());
}

// ---------------------------------------------------------------------------
// Apply pass.
//
// kCheck (direct mode only): the pass also sums the partial norms of the x it
// reads and of the u it recomputes, in the moment pass's order per thread and
// its fixed tree, into `check` at the chunk's slot. Algorithm 2 uses one u for
// the norm and for the update, so these sums must equal the moment pass's
// partials bit for bit; a plan switches this on to test that
// (lamb_plan_set_u_check).
// ---------------------------------------------------------------------------

template <int kAlgo, bool kBf16, bool kDeferred, int kNorm, bool kCheck>
__global__ __launch_bounds__(kBlock) void apply_kernel(
    const TensorDesc *__restrict__ tensors, const int32_t *__restrict__ chunk_ids,
    int32_t chunk_elems, const float *__restrict__ scale, uint32_t *__restrict__ flags,
    const uint32_t *__restrict__ ctl, int32_t guard, int32_t *__restrict__ nonfinite_out,
    Partial *__restrict__ check, StepArgs a) {
    static_assert(!(kCheck && kDeferred), "the check runs on direct-mode steps");
    constexpr bool kV = kHasSecondMoment<kAlgo>;
    constexpr bool kReadsGrad = kDeferred || kDirectionNeedsGrad<kAlgo>;
    const uint32_t fault = ctl_load(ctl + kCtlFault);
    const ChunkDesc c = chunk_at<false>(tensors, chunk_ids, apply_chunk_index(), chunk_elems);
    if (pass_stopped(fault, flags, ctl, kDeferred ? int32_t(kGuardNone) : guard))
        return;
    if constexpr (kDeferred) {
        // The finalize moved the moment pass's verdict (raised if any scaled
        // gradient was NaN or infinite) into flags[1].
        const uint32_t bad = flags[1];
        if (blockIdx.x == 0 && threadIdx.x == 0 && nonfinite_out)
            *nonfinite_out = bad ? 1 : 0;
        if (bad)
            return;
    }
    const TensorDesc &t = tensors[c.tensor];
    gfloat *x = global_view(t.x + c.start);
    gfloat *m = global_view(t.m + c.start);
    gfloat *v = kV ? global_view(t.v + c.start) : nullptr;
    const GradView<kBf16> g(t.g, c.start, a.grad_scale);
    gbf16 *copy = t.x_copy ? (gbf16 *)(t.x_copy + c.start) : nullptr;
    const float lam = t.wd ? a.weight_decay : 0.0f;
    const float s = scale[c.tensor];

    double sum_xx = 0.0, sum_uu = 0.0;
    const int n4 = c.len >> 2;
    const int stride = int(blockDim.x);
    for (int base = threadIdx.x; base < n4; base += stride * kUnroll) {
        f32x4 xr[kUnroll], gr[kUnroll], mr[kUnroll], vr[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * stride;
            if (q < n4) {
                xr[k] = load4(x + 4 * q);
                if constexpr (kReadsGrad)
                    gr[k] = g.at4(4 * q);
                else
                    gr[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                mr[k] = load4(m + 4 * q);
                if constexpr (kV)
                    vr[k] = load4(v + 4 * q);
                else
                    vr[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = base + k * stride;
            if (q < n4) {
                f32x4 xn;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float me = mr[k][e], ve = vr[k][e];
                    if constexpr (kDeferred)
                        new_moments<kAlgo>(xr[k][e], gr[k][e], lam, me, ve, a);
                    const float u = direction<kAlgo>(xr[k][e], gr[k][e], me, ve, lam, a);
                    if constexpr (kCheck) {
                        sum_xx = norm_add<kNorm>(sum_xx, xr[k][e]);
                        sum_uu = norm_add<kNorm>(sum_uu, u);
                    }
                    xn[e] = fmaf(-s, u, xr[k][e]);
                    mr[k][e] = me;
                    vr[k][e] = ve;
                }
                store4(x + 4 * q, xn);
                if (copy) {
                    const u32x2 packed = {bf16_bits(xn[0]) | (bf16_bits(xn[1]) << 16),
                                          bf16_bits(xn[2]) | (bf16_bits(xn[3]) << 16)};
                    stream_store((LAMB_GLOBAL u32x2 *)(copy + 4 * q), packed);
                }
                if constexpr (kDeferred) {
                    store4(m + 4 * q, mr[k]);
                    if constexpr (kV)
                        store4(v + 4 * q, vr[k]);
                }
            }
        }
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len) {
        const float xj = x[tail];
        const float gj = kReadsGrad ? g.at(tail) : 0.0f;
        float mj = m[tail];
        float vj = kV ? v[tail] : 0.0f;
        if constexpr (kDeferred)
            new_moments<kAlgo>(xj, gj, lam, mj, vj, a);
        const float u = direction<kAlgo>(xj, gj, mj, vj, lam, a);
        if constexpr (kCheck) {
            sum_xx = norm_add<kNorm>(sum_xx, xj);
            sum_uu = norm_add<kNorm>(sum_uu, u);
        }
        const float xn = fmaf(-s, u, xj);
        x[tail] = xn;
        if (copy)
            copy[tail] = uint16_t(bf16_bits(xn));
        if constexpr (kDeferred) {
            m[tail] = mj;
            if constexpr (kV)
                v[tail] = vj;
        }
    }
    if constexpr (kCheck)
        block_combine_any<kNorm>(sum_xx, sum_uu, check + apply_chunk_index());
}

// One layer's norms, phi, trust ratio and step scale lr * ratio from its
// combined partial norms; reports ratio and norms at index `out`.
template <int kNorm>
__device__ float finish_layer(const Partial &total, const FinalizeArgs &a, int32_t out,
                              double *ratio_out, double *norms_out) {
    const double norm_x = norm_finish<kNorm>(total.sum_xx);
    const double norm_u = norm_finish<kNorm>(total.sum_uu);
    // phi(z) = min(max(z, gamma_l), gamma_u), Section 3; comparisons keep NaN.
    double phi = norm_x;
    if (phi < a.gamma_l)
        phi = a.gamma_l;
    if (phi > a.gamma_u)
        phi = a.gamma_u;
    // A zero update norm means a zero update: report ratio 0, move nothing.
    const double ratio = (norm_u == 0.0) ? 0.0 : a.trust_coef * phi / norm_u;
    if (ratio_out)
        ratio_out[out] = ratio;
    if (norms_out) {
        norms_out[2 * out] = norm_x;
        norms_out[2 * out + 1] = norm_u;
    }
    return static_cast<float>(a.lr * ratio);
}

// finish_layer for the single pass: a layer too large for one round keeps its
// head on the two-pass kernels, whose totals (ext_totals[2 ext], [2 ext + 1])
// come first in the layer's sum; its step scale also goes to ext_scale[ext]
// for the apply pass over the head.
template <int kNorm>
__device__ float finish_split_layer(const Partial &tiles_total, int32_t ext,
                                    const double *ext_totals, float *ext_scale,
                                    const FinalizeArgs &a, int32_t out, double *ratio_out,
                                    double *norms_out) {
    if (ext < 0)
        return finish_layer<kNorm>(tiles_total, a, out, ratio_out, norms_out);
    const Partial total{norm_combine<kNorm>(ext_totals[2 * ext], tiles_total.sum_xx),
                        norm_combine<kNorm>(ext_totals[2 * ext + 1], tiles_total.sum_uu)};
    const float s = finish_layer<kNorm>(total, a, out, ratio_out, norms_out);
    ext_scale[ext] = s;
    return s;
}

// ---------------------------------------------------------------------------
// Finiteness check: the verdict of a skip_nonfinite step taken before
// anything is written (the step then runs the direct-mode kernels, which
// return at once when the verdict is raised). Reads g only; a chunk that
// finds a NaN or infinite scaled gradient raises the step's verdict word,
// selected by the single pass's epoch, with one integer atomicOr.
// ---------------------------------------------------------------------------

template <bool kBf16>
__global__ __launch_bounds__(kBlock) void finite_kernel(const TensorDesc *__restrict__ tensors,
                                                       const ChunkDesc *__restrict__ chunks,
                                                       uint32_t *__restrict__ flags,
                                                       const uint32_t *__restrict__ ctl,
                                                       float grad_scale) {
    const ChunkDesc c = chunks[blockIdx.x];
    const TensorDesc &t = tensors[c.tensor];
    const GradView<kBf16> g(t.g, c.start, grad_scale);
    bool bad = false;
    const int n4 = c.len >> 2;
#pragma unroll 4
    for (int q = threadIdx.x; q < n4; q += kBlock) {
        const f32x4 v = g.at4(4 * q);
        bad |= !(isfinite(v.x) && isfinite(v.y) && isfinite(v.z) && isfinite(v.w));
    }
    const int tail = 4 * n4 + threadIdx.x;
    if (tail < c.len)
        bad |= !isfinite(g.at(tail));
    if (__syncthreads_or(bad) && threadIdx.x == 0)
        atomicOr(flags + kVerdictWord + (ctl[kCtlEpoch] & 1u), 1u);
}

// ---------------------------------------------------------------------------
// Finalize, in two levels. The segment kernel gives each workgroup up to
// kSegChunks consecutive chunk partials of one tensor: thread k folds slots
// k + j * kSegBlock into kSegLanes independent accumulators (several loads in
// flight), combines them in a fixed order, and the fixed wave/LDS tree
// combines the threads into the segment's partial. The per-tensor finalize
// then combines the tensor's segment partials the same way and forms the
// norms, phi, trust ratio and step scale. The order never depends on timing.
// ---------------------------------------------------------------------------

template <int kNorm>
__global__ __launch_bounds__(kSegBlock) void segment_kernel(const Partial *__restrict__ partials,
                                                          const SegDesc *__restrict__ segs,
                                                          Partial *__restrict__ seg_partials) {
    const SegDesc sd = segs[blockIdx.x];
    const Partial *p = partials + sd.first;
    double sx[kSegLanes] = {}, su[kSegLanes] = {};
#pragma unroll
    for (int j = 0; j < kSegLanes; ++j) {
        const int k = threadIdx.x + j * kSegBlock;
        if (k < sd.count) {
            const Partial q = p[k];
            sx[j] = q.sum_xx;
            su[j] = q.sum_uu;
        }
    }
#pragma unroll
    for (int j = 1; j < kSegLanes; ++j) {
        sx[0] = norm_combine<kNorm>(sx[0], sx[j]);
        su[0] = norm_combine<kNorm>(su[0], su[j]);
    }
    block_combine<kNorm, kSegBlock / 64>(sx[0], su[0], seg_partials + blockIdx.x);
}

// A tensor's combined partial norms from its segment partials, in a fixed
// order (every thread of the workgroup returns it).
template <int kNorm>
__device__ Partial tensor_total(const Partial *__restrict__ seg_partials, SegRange r) {
    double sx = 0.0, su = 0.0;
    for (int k = threadIdx.x; k < r.count; k += kSegBlock) {
        const Partial q = seg_partials[r.first + k];
        sx = norm_combine<kNorm>(sx, q.sum_xx);
        su = norm_combine<kNorm>(su, q.sum_uu);
    }
    __shared__ Partial total;
    block_combine<kNorm, kSegBlock / 64>(sx, su, &total);
    __syncthreads();
    return total;
}

template <int kNorm>
__global__ __launch_bounds__(kSegBlock) void finalize_kernel(
    const TensorDesc *__restrict__ tensors, const Partial *__restrict__ seg_partials,
    const SegRange *__restrict__ ranges, FinalizeArgs a, float *__restrict__ scale,
    double *__restrict__ ratio_out, double *__restrict__ norms_out, uint32_t *__restrict__ flags) {
    const int i = blockIdx.x;
    const Partial total = tensor_total<kNorm>(seg_partials, ranges[i]);
    if (threadIdx.x == 0) {
        scale[i] = finish_layer<kNorm>(total, a, tensors[i].out_index, ratio_out, norms_out);
        // Deferred mode: hand the moment pass's non-finite verdict to the apply
        // pass and clear the word the next moment pass raises.
        if (flags && i == 0) {
            flags[1] = flags[0];
            flags[0] = 0u;
        }
    }
}

// ---------------------------------------------------------------------------
// Split step (a step over a shard of every tensor, Section 4.1's synchronous
// data parallelism with the optimizer state sharded): the first half writes
// each tensor's combined partial norms, the raw accumulators that add (L2:
// sums of squares; L1: sums of magnitudes) or take a maximum (L-infinity)
// across shards, to totals[2 i] (x) and totals[2 i + 1] (u), and the step's
// non-finite verdict (0 or 1) to totals[2 n]; the caller combines the shards'
// buffers; the second half turns the combined totals into each layer's norms,
// phi, trust ratio and step scale, exactly as the finalize does, and hands
// the combined verdict (nonzero: skip) to a deferred apply pass.
// ---------------------------------------------------------------------------

template <int kNorm>
__global__ __launch_bounds__(kSegBlock) void totals_kernel(
    const Partial *__restrict__ seg_partials, const SegRange *__restrict__ ranges,
    int32_t n_tensors, double *__restrict__ totals, uint32_t *__restrict__ flags,
    const uint32_t *__restrict__ ctl, int32_t verdict_mode) {
    const int i = blockIdx.x;
    const Partial total = tensor_total<kNorm>(seg_partials, ranges[i]);
    if (threadIdx.x == 0) {
        totals[2 * i] = total.sum_xx;
        totals[2 * i + 1] = total.sum_uu;
        if (i == 0) {
            uint32_t bad = 0u;
            if (verdict_mode == kVerdictMove) {
                bad = flags[0];
                flags[0] = 0u;
            } else if (verdict_mode == kVerdictCopy) {
                bad = flags[kVerdictWord + (ctl[kCtlEpoch] & 1u)];
                flags[1] = bad;
            }
            totals[2 * n_tensors] = bad != 0u ? 1.0 : 0.0;
        }
    }
}

template <int kNorm>
__global__ __launch_bounds__(kSegBlock) void scale_kernel(
    const double *__restrict__ totals, int32_t n_tensors, FinalizeArgs a,
    float *__restrict__ scale, double *__restrict__ ratio_out, double *__restrict__ norms_out,
    uint32_t *__restrict__ flags) {
    const int i = int(blockIdx.x * blockDim.x + threadIdx.x);
    if (i < n_tensors)
        scale[i] = finish_layer<kNorm>(Partial{totals[2 * i], totals[2 * i + 1]}, a, i,
                                       ratio_out, norms_out);
    if (i == 0)
        flags[1] = totals[2 * n_tensors] != 0.0 ? 1u : 0u;
}

// ---------------------------------------------------------------------------
// Single-pass path.
//
// A persistent grid of `grid` workgroups, all resident at once, walks the
// tile list: workgroup w takes entries w, w + grid, w + 2 grid, ..., so the
// list falls into rounds of `grid` entries. The host packs every layer's
// tiles consecutively inside one round (empty entries pad a round's gap).
// A tile is G = kGroups float4 groups per thread (8 or 10; the plan picks).
// Tile i of a layer of T tiles holds the layer's 1024-element blocks i,
// i + T, ..., i + (G - 1) T, so the layer's tiles stream one dense stretch of
// it at a time (contiguous 8192-element tiles, 32 KB apart, streamed 2.3%
// slower). For each tile a workgroup reads x, g, m, v once, writes the new
// moments at once, and keeps x in LDS (a 10-group tile keeps the x of its
// last two groups in registers) and u in registers. The tile's partial norms go
// to a slot; the layer's first tile (its leader) waits for every slot of the
// layer, combines them in tile order, forms the step scale exactly as the
// finalize kernel does and writes it to each member's broadcast slot; every
// member then writes x - scale * u. A workgroup only waits after publishing
// its own slot, and a layer's members sit in one round on distinct
// workgroups that reach it once their earlier rounds are done, so by
// induction over rounds every wait ends.
//
// Slots are 64-bit words read and written with agent-scope atomics, which
// are coherent across the XCDs' separate L2 caches. An empty slot holds
// kEmptySlot, which no published value equals. Two slot buffers alternate by
// the epoch word: a step fills buffer (epoch & 1) and empties the other for
// the next step; the last workgroup to finish advances the epoch (a step
// skipped for a non-finite gradient touches no slot and leaves it). Nothing
// depends on a host counter, so a captured graph replays correctly.
// Every wait is bounded: after StepArgs::spin_limit polls, or once another
// workgroup has given up, a workgroup raises the sticky fault word and
// abandons the step, and every later step of the plan does nothing.
// ---------------------------------------------------------------------------

// s_sleep argument between polls (units of 64 clocks): 512 clocks beat 128,
// 256 and 1024 by 0.3-0.6% on BERT-Large.
constexpr int kPollSleep = 8;
// A workgroup that waits for its layer's scale drops its waves to the lowest
// issue priority (s_setprio 0) and raises them (to 3) once the scale is
// known, so that waves with reads and writes to issue go first (1.2-1.4%
// faster on BERT-Large, 0.5-0.6% on LARS; within 0.5% on the other sets).
// Before it waits, a workgroup loads group 0 of its next tile, so that HBM
// keeps streaming through the wait (0.2-0.55% faster; 16 more VGPRs).
// Float4 groups each thread of the single pass uses per trip: one for the
// LAMB family (four streams; two were 0.3-1% slower), two for LARS (three
// streams; one was 3-5% slower). On a full tile the next trip's groups are
// loaded before this trip's are used, so a wave always has loads in flight
// (same-box A/B against loading each trip after the last: BERT-Large 0.25%
// faster, its LARS step 3.9%, BERT-Base 1.1%, ResNet-50 1.7% and 0.75% for
// LARS, the 1.5B set 0.8%; two trips ahead was slower on all but ResNet-50).
// Every load and store of the single pass addresses its array as a uniform
// base plus a 32-bit byte offset (one VGPR instead of a 64-bit address).
template <int kAlgo>
constexpr int kFusedUnroll = kAlgo == kLars ? 2 : 1;
static_assert(kTileGroups % 2 == 0 && kWideGroups % 2 == 0,
              "tile groups must be a multiple of the unroll");

__device__ __forceinline__ uint64_t slot_load(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void slot_store(uint64_t *p, uint64_t w) {
    __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


// A partial norm as a slot word. Partial norms are >= 0, +inf or NaN; every
// NaN is stored as the positive quiet NaN, so no value is kEmptySlot.
__device__ __forceinline__ uint64_t slot_word(double d) {
    return isnan(d) ? 0x7ff8000000000000ull : static_cast<uint64_t>(__double_as_longlong(d));
}

// Polls *p until it holds a value; kEmptySlot if the wait was abandoned.
template <int kSleep>
__device__ uint64_t slot_wait(const uint64_t *p, uint32_t *ctl, uint32_t limit) {
    for (uint32_t k = 1;; ++k) {
        const uint64_t w = slot_load(p);
        if (w != kEmptySlot)
            return w;
        if (k >= limit || (k & 255u) == 0) {
            if (ctl_load(ctl + kCtlFault) != 0)
                return kEmptySlot;
            if (k >= limit) {
                __hip_atomic_fetch_or(ctl + kCtlFault, 1u, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
                return kEmptySlot;
            }
        }
        __builtin_amdgcn_s_sleep(kSleep);
    }
}

template <int kAlgo, bool kBf16, int kNorm, int kGroups>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(kFusedWaves)))
void fused_kernel(const TensorDesc *__restrict__ tensors, const ChunkDesc *__restrict__ tiles,
                  int32_t n_tiles, uint64_t *__restrict__ slots, uint32_t *__restrict__ ctl,
                  uint32_t *__restrict__ flags, int32_t guarded,
                  int32_t *__restrict__ nonfinite_out,
                  StepArgs a, FinalizeArgs f, double *__restrict__ ratio_out,
                  double *__restrict__ norms_out, const double *__restrict__ ext_totals,
                  float *__restrict__ ext_scale, uint64_t *__restrict__ trace) {
    constexpr bool kV = kHasSecondMoment<kAlgo>;
    constexpr int kUnrollF = kFusedUnroll<kAlgo>;
    __shared__ uint32_t sh_epoch, sh_fault, sh_skip;
    __shared__ float sh_scale;
    __shared__ Partial sh_tile, sh_layer;
    // The tile's x waits in LDS (32 KB for the first kLdsGroups groups) and,
    // past those, in registers; its update direction waits in registers.
    constexpr int kInLds = kGroups < kLdsGroups ? kGroups : kLdsGroups;
    constexpr int kInRegs = kGroups - kInLds;
    __shared__ f32x4 sh_x[kInLds][kBlock];
    if (threadIdx.x == 0) {
        sh_epoch = ctl_load(ctl + kCtlEpoch);
        sh_fault = ctl_load(ctl + kCtlFault);
        // skip_nonfinite step: the finiteness check's verdict
        sh_skip = guarded ? flags[kVerdictWord + (sh_epoch & 1u)] : 0u;
    }
    __syncthreads();
    const uint32_t epoch = sh_epoch;
    const size_t n = static_cast<size_t>(n_tiles);
    // per buffer: partial ||x|| words, partial ||u|| words, broadcast scales
    uint64_t *cur = slots + size_t(epoch & 1u) * 3 * n;
    uint64_t *next = slots + size_t((epoch & 1u) ^ 1u) * 3 * n;
    bool stop = sh_fault != 0 || sh_skip != 0;

    const int32_t grid = static_cast<int32_t>(gridDim.x);
    // Group 0 of this workgroup's next tile (when that tile is full), loaded
    // before the current tile waits for its layer's scale, so that HBM keeps
    // streaming through the wait. p_j: the entry it belongs to (-1: none).
    f32x4 px = {0.0f, 0.0f, 0.0f, 0.0f}, pg = px, pm = px, pv = px;
    int32_t p_j = -1;
    for (int32_t r = 0; !stop; ++r) {
        const int32_t j = r * grid + static_cast<int32_t>(blockIdx.x);  // entry of round r
        if (j >= n_tiles)
            break;
        const ChunkDesc c = tiles[j];
        if (c.len == 0)
            continue;  // an empty entry that pads a round
        const TensorDesc &t = tensors[c.tensor];
        uint64_t stamp[3] = {0, 0, 0};  // the trace's first three clocks of this tile
        if (trace)
            stamp[0] = __builtin_amdgcn_s_memrealtime();
        gfloat *x = global_view(t.x);
        gfloat *m = global_view(t.m);
        gfloat *v = kV ? global_view(t.v) : nullptr;
        const GradView<kBf16> g(t.g, 0, a.grad_scale);
        const float lam = t.wd ? a.weight_decay : 0.0f;
        // Group k of this thread: 4 elements from `first`, `valid` (0-4) of them
        // inside the layer.
        auto group = [&](int k, uint32_t &first, int &valid) {
            // Tile i of a layer of T tiles holds its 1024-element blocks i, i + T,
            // i + 2T, ...: at any moment the layer's tiles stream one dense
            // stretch of it.
            const uint32_t block = uint32_t(k) * uint32_t(t.n_tiles) + uint32_t(j - t.first_tile);
            first = block * (4u * kBlock) + 4u * threadIdx.x;
            const int64_t left = t.numel - int64_t(first);
            valid = left >= 4 ? 4 : left > 0 ? int(left) : 0;
        };

        // Read once, write the new moments, keep x and u.
        f32x4 us[kGroups];
        f32x4 x_keep[kInRegs > 0 ? kInRegs : 1];
        double sum_xx = 0.0, sum_uu = 0.0;
        if (c.len == kGroups * 4 * kBlock) {
            // A full tile: every group is whole, so every load is issued
            // unconditionally and the next trip's groups are in flight while
            // this trip's are used.
            auto fetch = [&](int k, f32x4 &xr, f32x4 &gr, f32x4 &mr, f32x4 &vr, uint32_t &at) {
                int whole;
                group(k, at, whole);
                xr = load4_at(x, at);
                gr = g.at4_off(at);
                mr = load4_at(m, at);
                vr = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                if constexpr (kV)
                    vr = load4_at(v, at);
            };
            // A ring of two trips' groups: the next trip's loads are issued before
            // this trip's groups are used.
            constexpr int kAhead = kUnrollF;
            constexpr int kRing = kAhead + kUnrollF;
            f32x4 bx[kRing], bg[kRing], bm[kRing], bv[kRing];
            uint32_t bat[kRing];
#pragma unroll
            for (int k = 0; k < kAhead && k < kGroups; ++k) {
                if (k == 0 && p_j == j) {
                    int whole;
                    group(0, bat[0], whole);
                    bx[0] = px;
                    bg[0] = pg;
                    bm[0] = pm;
                    bv[0] = pv;
                } else {
                    fetch(k, bx[k % kRing], bg[k % kRing], bm[k % kRing], bv[k % kRing],
                          bat[k % kRing]);
                }
            }
#pragma unroll
            for (int k0 = 0; k0 < kGroups; k0 += kUnrollF) {
#pragma unroll
                for (int k = 0; k < kUnrollF; ++k) {
                    const int q = k0 + kAhead + k;
                    if (q < kGroups)
                        fetch(q, bx[q % kRing], bg[q % kRing], bm[q % kRing], bv[q % kRing],
                              bat[q % kRing]);
                }
#pragma unroll
                for (int k = 0; k < kUnrollF; ++k) {
                    const int q = (k0 + k) % kRing;
                    f32x4 xr = bx[q], gr = bg[q], mr = bm[q], vr = bv[q];
                    f32x4 ur;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float me = mr[e], ve = vr[e];
                        new_moments<kAlgo>(xr[e], gr[e], lam, me, ve, a);
                        ur[e] = direction<kAlgo>(xr[e], gr[e], me, ve, lam, a);
                        sum_xx = norm_add<kNorm>(sum_xx, xr[e]);
                        sum_uu = norm_add<kNorm>(sum_uu, ur[e]);
                        mr[e] = me;
                        vr[e] = ve;
                    }
                    store4_at(m, bat[q], mr);
                    if constexpr (kV)
                        store4_at(v, bat[q], vr);
                    if (k0 + k < kInLds)
                        sh_x[k0 + k][threadIdx.x] = xr;
                    else
                        x_keep[k0 + k - kInLds] = xr;
                    us[k0 + k] = ur;
                }
            }
        } else {
            // A tile that is not full (the layer ends inside it): groups past
            // the layer's end hold nothing, and one group may be partial.
#pragma unroll
            for (int k0 = 0; k0 < kGroups; k0 += kUnrollF) {
                f32x4 xr[kUnrollF], gr[kUnrollF], mr[kUnrollF], vr[kUnrollF];
                uint32_t at[kUnrollF];
                int ok[kUnrollF];
#pragma unroll
                for (int k = 0; k < kUnrollF; ++k) {
                    group(k0 + k, at[k], ok[k]);
                    xr[k] = gr[k] = mr[k] = vr[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                    if (ok[k] == 4) {
                        xr[k] = load4_at(x, at[k]);
                        gr[k] = g.at4_off(at[k]);
                        mr[k] = load4_at(m, at[k]);
                        if constexpr (kV)
                            vr[k] = load4_at(v, at[k]);
                    } else if (ok[k] > 0) {  // the layer's last, partial group
                        for (int e = 0; e < ok[k]; ++e) {
                            xr[k][e] = x[at[k] + e];
                            gr[k][e] = g.at(at[k] + e);
                            mr[k][e] = m[at[k] + e];
                            if constexpr (kV)
                                vr[k][e] = v[at[k] + e];
                        }
                    }
                }
#pragma unroll
                for (int k = 0; k < kUnrollF; ++k) {
                    f32x4 ur = {0.0f, 0.0f, 0.0f, 0.0f};
                    if (ok[k] > 0) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            if (e < ok[k]) {
                                float me = mr[k][e], ve = vr[k][e];
                                new_moments<kAlgo>(xr[k][e], gr[k][e], lam, me, ve, a);
                                ur[e] = direction<kAlgo>(xr[k][e], gr[k][e], me, ve, lam, a);
                                sum_xx = norm_add<kNorm>(sum_xx, xr[k][e]);
                                sum_uu = norm_add<kNorm>(sum_uu, ur[e]);
                                mr[k][e] = me;
                                vr[k][e] = ve;
                            }
                        }
                        if (ok[k] == 4) {
                            store4_at(m, at[k], mr[k]);
                            if constexpr (kV)
                                store4_at(v, at[k], vr[k]);
                        } else {
                            for (int e = 0; e < ok[k]; ++e) {
                                m[at[k] + e] = mr[k][e];
                                if constexpr (kV)
                                    v[at[k] + e] = vr[k][e];
                            }
                        }
                    }
                    if (k0 + k < kInLds)
                        sh_x[k0 + k][threadIdx.x] = xr[k];
                    else
                        x_keep[k0 + k - kInLds] = xr[k];
                    us[k0 + k] = ur;
                }
            }
        }
        block_combine<kNorm, kWaves>(sum_xx, sum_uu, &sh_tile);
        __syncthreads();
        if (trace)
            stamp[1] = __builtin_amdgcn_s_memrealtime();
        __builtin_amdgcn_s_setprio(0);
        p_j = -1;
        if (j + grid < n_tiles) {
            const int32_t jn = j + grid;
            const ChunkDesc cn = tiles[jn];
            if (cn.len == kGroups * 4 * kBlock) {  // a full tile: block 0 is whole
                const TensorDesc &tn = tensors[cn.tensor];
                // block 0 of tile jn - first_tile of its layer
                const uint32_t at0 = uint32_t(jn - tn.first_tile) * (4u * kBlock) + 4u * threadIdx.x;
                px = load4_at(global_view(tn.x), at0);
                pg = GradView<kBf16>(tn.g, 0, a.grad_scale).at4_off(at0);
                pm = load4_at(global_view(tn.m), at0);
                if constexpr (kV)
                    pv = load4_at(global_view(tn.v), at0);
                p_j = jn;
            }
        }

        // The layer's step scale.
        const int32_t first = t.first_tile, team = t.n_tiles;
        int give_up = 0;
        if (team == 1) {
            if (threadIdx.x == 0)
                sh_scale = finish_split_layer<kNorm>(sh_tile, t.ext, ext_totals, ext_scale, f,
                                                     t.out_index, ratio_out, norms_out);
        } else {
            if (threadIdx.x == 0) {
                slot_store(cur + j, slot_word(sh_tile.sum_xx));
                slot_store(cur + n + j, slot_word(sh_tile.sum_uu));
                slot_store(next + j, kEmptySlot);
                slot_store(next + n + j, kEmptySlot);
                slot_store(next + 2 * n + j, kEmptySlot);
            }
            if (j == first) {
                double ax = 0.0, au = 0.0;
                for (int k = threadIdx.x; k < team; k += kBlock) {
                    const uint64_t wx =
                        slot_wait<kPollSleep>(cur + first + k, ctl, a.spin_limit);
                    const uint64_t wu =
                        wx == kEmptySlot
                            ? kEmptySlot
                            : slot_wait<kPollSleep>(cur + n + first + k, ctl, a.spin_limit);
                    if (wu == kEmptySlot) {
                        give_up = 1;
                        break;
                    }
                    ax = norm_combine<kNorm>(ax, __longlong_as_double(static_cast<long long>(wx)));
                    au = norm_combine<kNorm>(au, __longlong_as_double(static_cast<long long>(wu)));
                }
                block_combine<kNorm, kWaves>(ax, au, &sh_layer);
                give_up = __syncthreads_or(give_up);
                if (!give_up) {
                    if (threadIdx.x == 0)
                        sh_scale = finish_split_layer<kNorm>(sh_layer, t.ext, ext_totals,
                                                             ext_scale, f, t.out_index,
                                                             ratio_out, norms_out);
                    __syncthreads();
                    const uint64_t w = __float_as_uint(sh_scale);
                    for (int k = threadIdx.x + 1; k < team; k += kBlock)
                        slot_store(cur + 2 * n + first + k, w);
                }
            } else if (threadIdx.x == 0) {
                const uint64_t w =
                    slot_wait<kPollSleep>(cur + 2 * n + j, ctl, a.spin_limit);
                if (w == kEmptySlot)
                    give_up = 1;
                else
                    sh_scale = __uint_as_float(static_cast<uint32_t>(w));
            }
        }
        stop = __syncthreads_or(give_up) != 0;
        if (stop)
            break;
        if (trace)
            stamp[2] = __builtin_amdgcn_s_memrealtime();

        __builtin_amdgcn_s_setprio(3);
        // x - scale * u from LDS and the registers.
        const float s = sh_scale;
        gbf16 *copy = t.x_copy ? (gbf16 *)t.x_copy : nullptr;
#pragma unroll
        for (int k = 0; k < kGroups; ++k) {
            uint32_t at;
            int valid;
            group(k, at, valid);
            if (valid > 0) {
                const f32x4 xo = k < kInLds ? sh_x[k][threadIdx.x] : x_keep[k - kInLds];
                f32x4 xn;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    xn[e] = fmaf(-s, us[k][e], xo[e]);
                if (valid == 4) {
                    store4_at(x, at, xn);
                    if (copy) {
                        const u32x2 packed = {bf16_bits(xn[0]) | (bf16_bits(xn[1]) << 16),
                                              bf16_bits(xn[2]) | (bf16_bits(xn[3]) << 16)};
                        stream_store((LAMB_GLOBAL u32x2 *)((LAMB_GLOBAL char *)copy + at * 2u),
                                     packed);
                    }
                } else {
                    for (int e = 0; e < valid; ++e) {
                        x[at + e] = xn[e];
                        if (copy)
                            copy[at + e] = uint16_t(bf16_bits(xn[e]));
                    }
                }
            }
        }
        if (trace && threadIdx.x == 0) {
            trace[4 * j] = stamp[0];
            trace[4 * j + 1] = stamp[1];
            trace[4 * j + 2] = stamp[2];
            trace[4 * j + 3] = __builtin_amdgcn_s_memrealtime();
        }
    }

    // The last workgroup to finish advances the epoch. Every workgroup read
    // the epoch before any of its work, so none can still be reading it.
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t done =
            __hip_atomic_fetch_add(ctl + kCtlDone, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (done == gridDim.x - 1) {
            if (guarded && nonfinite_out)
                *nonfinite_out = sh_skip ? 1 : 0;
            __hip_atomic_store(ctl + kCtlDone, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (sh_skip) {
                // A skipped step touched no slot, so its buffer is still empty
                // and the next step reuses it: the epoch stays, and the raised
                // verdict word is cleared for that step.
                flags[kVerdictWord + (epoch & 1u)] = 0u;
            } else {
                // Clear the verdict word of the next epoch (last used two
                // steps ago, read by nothing now) and advance the epoch.
                flags[kVerdictWord + ((epoch + 1u) & 1u)] = 0u;
                __hip_atomic_store(ctl + kCtlEpoch, epoch + 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Kernel selection: the template arguments are spelled out so every
// combination the launchers may pick is instantiated.
// ---------------------------------------------------------------------------

template <int kAlgo, bool kBf16, int kNorm>
const void *moments_fn(bool deferred) {
    return deferred ? reinterpret_cast<const void *>(&moments_kernel<kAlgo, kBf16, kNorm, true>)
                    : reinterpret_cast<const void *>(&moments_kernel<kAlgo, kBf16, kNorm, false>);
}

template <int kAlgo, bool kBf16>
const void *moments_fn(int norm, bool deferred) {
    switch (norm) {
    case kL1: return moments_fn<kAlgo, kBf16, kL1>(deferred);
    case kLinf: return moments_fn<kAlgo, kBf16, kLinf>(deferred);
    default: return moments_fn<kAlgo, kBf16, kL2>(deferred);
    }
}

template <int kAlgo>
const void *moments_fn(const StepKind &k) {
    return k.bf16_grad ? moments_fn<kAlgo, true>(k.norm, k.deferred)
                       : moments_fn<kAlgo, false>(k.norm, k.deferred);
}

template <int kAlgo, bool kBf16>
const void *apply_fn(bool deferred, int norm, bool check) {
    if (deferred)
        return reinterpret_cast<const void *>(&apply_kernel<kAlgo, kBf16, true, kL2, false>);
    if (!check)
        return reinterpret_cast<const void *>(&apply_kernel<kAlgo, kBf16, false, kL2, false>);
    switch (norm) {
    case kL1: return reinterpret_cast<const void *>(&apply_kernel<kAlgo, kBf16, false, kL1, true>);
    case kLinf:
        return reinterpret_cast<const void *>(&apply_kernel<kAlgo, kBf16, false, kLinf, true>);
    default: return reinterpret_cast<const void *>(&apply_kernel<kAlgo, kBf16, false, kL2, true>);
    }
}

template <int kAlgo>
const void *apply_fn(const StepKind &k, bool check) {
    return k.bf16_grad ? apply_fn<kAlgo, true>(k.deferred, k.norm, check)
                       : apply_fn<kAlgo, false>(k.deferred, k.norm, check);
}

template <int kAlgo, bool kBf16, int kGroups>
const void *fused_fn(int norm) {
    switch (norm) {
    case kL1: return reinterpret_cast<const void *>(&fused_kernel<kAlgo, kBf16, kL1, kGroups>);
    case kLinf:
        return reinterpret_cast<const void *>(&fused_kernel<kAlgo, kBf16, kLinf, kGroups>);
    default: return reinterpret_cast<const void *>(&fused_kernel<kAlgo, kBf16, kL2, kGroups>);
    }
}

template <int kAlgo, int kGroups>
const void *fused_fn(const StepKind &k) {
    return k.bf16_grad ? fused_fn<kAlgo, true, kGroups>(k.norm)
                       : fused_fn<kAlgo, false, kGroups>(k.norm);
}

template <int kGroups>
const void *fused_fn(const StepKind &k) {
    switch (k.algo) {
    case kNLamb: return fused_fn<kNLamb, kGroups>(k);
    case kNNLamb: return fused_fn<kNNLamb, kGroups>(k);
    case kLars: return fused_fn<kLars, kGroups>(k);
    default: return fused_fn<kLamb, kGroups>(k);
    }
}

// Null for a tile shape other than the two a plan may pick.
const void *fused_fn(const StepKind &k, int groups) {
    if (groups == kTileGroups)
        return fused_fn<kTileGroups>(k);
    if (groups == kWideGroups)
        return fused_fn<kWideGroups>(k);
    return nullptr;
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------

hipError_t launch_moments(const StepKind &kind, const TensorDesc *tensors,
                          const int32_t *chunk_ids, int32_t chunk_elems, Partial *partials,
                          int32_t n_chunks, int32_t threads, uint32_t *flags,
                          const uint32_t *ctl, int32_t guard, const StepArgs &args,
                          hipStream_t stream) {
    if (threads < 64 || threads > kBlock || threads % 64 != 0 || !ctl ||
        guard < kGuardNone || guard > kGuardCopy)
        return hipErrorInvalidValue;
    StepArgs a = args;
    void *params[] = {&tensors, &chunk_ids, &chunk_elems, &partials, &flags, &ctl, &guard, &a};
    const void *fn;
    switch (kind.algo) {
    case kNLamb: fn = moments_fn<kNLamb>(kind); break;
    case kNNLamb: fn = moments_fn<kNNLamb>(kind); break;
    case kLars: fn = moments_fn<kLars>(kind); break;
    default: fn = moments_fn<kLamb>(kind); break;
    }
    return hipLaunchKernel(fn, dim3(n_chunks), dim3(threads), params, 0, stream);
}

hipError_t launch_apply(const StepKind &kind, const TensorDesc *tensors,
                        const int32_t *chunk_ids, int32_t chunk_elems, const float *scale,
                        int32_t n_chunks, int32_t threads, uint32_t *flags, const uint32_t *ctl,
                        int32_t guard, int32_t *nonfinite_out, Partial *check,
                        const StepArgs &args, hipStream_t stream) {
    if (threads < 64 || threads > kBlock || threads % 64 != 0 || !ctl ||
        (check && kind.deferred) || guard < kGuardNone || guard > kGuardCopy)
        return hipErrorInvalidValue;
    StepArgs a = args;
    void *params[] = {&tensors, &chunk_ids,     &chunk_elems, &scale, &flags,
                      &ctl,     &guard,         &nonfinite_out, &check, &a};
    const bool c = check != nullptr;
    const void *fn;
    switch (kind.algo) {
    case kNLamb: fn = apply_fn<kNLamb>(kind, c); break;
    case kNNLamb: fn = apply_fn<kNNLamb>(kind, c); break;
    case kLars: fn = apply_fn<kLars>(kind, c); break;
    default: fn = apply_fn<kLamb>(kind, c); break;
    }
    return hipLaunchKernel(fn, dim3(n_chunks), dim3(threads), params, 0, stream);
}

namespace {

hipError_t launch_segments(NormKind norm, const Partial *partials, const SegDesc *segs,
                           int32_t n_segs, Partial *seg_partials, hipStream_t stream) {
    const void *fn = norm == kL1     ? reinterpret_cast<const void *>(&segment_kernel<kL1>)
                     : norm == kLinf ? reinterpret_cast<const void *>(&segment_kernel<kLinf>)
                                     : reinterpret_cast<const void *>(&segment_kernel<kL2>);
    void *params[] = {&partials, &segs, &seg_partials};
    return hipLaunchKernel(fn, dim3(n_segs), dim3(kSegBlock), params, 0, stream);
}

}  // namespace

hipError_t launch_finalize(NormKind norm, const TensorDesc *tensors, int32_t n_tensors,
                           const Partial *partials, const SegDesc *segs, int32_t n_segs,
                           const SegRange *ranges, Partial *seg_partials,
                           const FinalizeArgs &args, float *scale, double *ratio_out,
                           double *norms_out, uint32_t *flags, hipStream_t stream) {
    hipError_t err = launch_segments(norm, partials, segs, n_segs, seg_partials, stream);
    if (err != hipSuccess)
        return err;
    FinalizeArgs a = args;
    void *params[] = {&tensors, &seg_partials, &ranges,    &a,
                      &scale,   &ratio_out,    &norms_out, &flags};
    const void *fn = norm == kL1     ? reinterpret_cast<const void *>(&finalize_kernel<kL1>)
                     : norm == kLinf ? reinterpret_cast<const void *>(&finalize_kernel<kLinf>)
                                     : reinterpret_cast<const void *>(&finalize_kernel<kL2>);
    return hipLaunchKernel(fn, dim3(n_tensors), dim3(kSegBlock), params, 0, stream);
}

hipError_t launch_totals(NormKind norm, const Partial *partials, const SegDesc *segs,
                         int32_t n_segs, const SegRange *ranges, int32_t n_tensors,
                         Partial *seg_partials, double *totals, uint32_t *flags,
                         const uint32_t *ctl, int32_t verdict_mode, hipStream_t stream) {
    if (verdict_mode < kVerdictZero || verdict_mode > kVerdictCopy ||
        (verdict_mode == kVerdictCopy && !ctl))
        return hipErrorInvalidValue;
    hipError_t err = launch_segments(norm, partials, segs, n_segs, seg_partials, stream);
    if (err != hipSuccess)
        return err;
    void *params[] = {&seg_partials, &ranges, &n_tensors, &totals, &flags, &ctl, &verdict_mode};
    const void *fn = norm == kL1     ? reinterpret_cast<const void *>(&totals_kernel<kL1>)
                     : norm == kLinf ? reinterpret_cast<const void *>(&totals_kernel<kLinf>)
                                     : reinterpret_cast<const void *>(&totals_kernel<kL2>);
    return hipLaunchKernel(fn, dim3(n_tensors), dim3(kSegBlock), params, 0, stream);
}

hipError_t launch_scale(NormKind norm, const double *totals, int32_t n_tensors,
                        const FinalizeArgs &args, float *scale, double *ratio_out,
                        double *norms_out, uint32_t *flags, hipStream_t stream) {
    FinalizeArgs a = args;
    void *params[] = {&totals, &n_tensors, &a, &scale, &ratio_out, &norms_out, &flags};
    const void *fn = norm == kL1     ? reinterpret_cast<const void *>(&scale_kernel<kL1>)
                     : norm == kLinf ? reinterpret_cast<const void *>(&scale_kernel<kLinf>)
                                     : reinterpret_cast<const void *>(&scale_kernel<kL2>);
    const int32_t blocks = (n_tensors + kSegBlock - 1) / kSegBlock;
    return hipLaunchKernel(fn, dim3(blocks), dim3(kSegBlock), params, 0, stream);
}

hipError_t launch_fused(const StepKind &kind, int groups, const TensorDesc *tensors,
                        const ChunkDesc *tiles, int32_t n_tiles, int32_t grid, uint64_t *slots,
                        uint32_t *ctl, uint32_t *flags, bool guarded, int32_t *nonfinite_out,
                        const StepArgs &args, const FinalizeArgs &fargs, double *ratio_out,
                        double *norms_out, const double *ext_totals, float *ext_scale,
                        uint64_t *trace, hipStream_t stream) {
    const void *fn = fused_fn(kind, groups);
    if (!fn)
        return hipErrorInvalidValue;
    StepArgs a = args;
    FinalizeArgs f = fargs;
    int32_t guard = guarded ? 1 : 0;
    void *params[] = {&tensors, &tiles,     &n_tiles,   &slots,      &ctl,
                      &flags,   &guard,     &nonfinite_out, &a,      &f,
                      &ratio_out, &norms_out, &ext_totals, &ext_scale, &trace};
    return hipLaunchKernel(fn, dim3(grid), dim3(kBlock), params, 0, stream);
}

hipError_t fused_blocks_per_cu(const StepKind &kind, int groups, int *blocks) {
    const void *fn = fused_fn(kind, groups);
    if (!fn)
        return hipErrorInvalidValue;
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, fn, kBlock, 0);
}

hipError_t launch_finite(bool bf16_grad, const TensorDesc *tensors, const ChunkDesc *chunks,
                         int32_t n_chunks, uint32_t *flags, const uint32_t *ctl, float grad_scale,
                         hipStream_t stream) {
    void *params[] = {&tensors, &chunks, &flags, &ctl, &grad_scale};
    const void *fn = bf16_grad ? reinterpret_cast<const void *>(&finite_kernel<true>)
                               : reinterpret_cast<const void *>(&finite_kernel<false>);
    return hipLaunchKernel(fn, dim3(n_chunks), dim3(kBlock), params, 0, stream);
}

}  // namespace lamb_mi355x
