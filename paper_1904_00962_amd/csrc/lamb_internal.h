// Internal layout shared by the HIP kernels (lamb_kernels.hip) and the host
// side of the C ABI (lamb_api.cpp). Not installed; the public interface is
// include/lamb_mi355x.h.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace lamb_mi355x {

// Work is cut into chunks of at most `chunk_elems` elements of one tensor;
// one workgroup of kBlock threads handles one chunk. kBlock = 4 wave64s.
#ifndef LAMB_BLOCK
#define LAMB_BLOCK 256
#endif
#ifndef LAMB_DEFAULT_CHUNK
#define LAMB_DEFAULT_CHUNK 512
#endif
constexpr int kBlock = LAMB_BLOCK;
constexpr int kWaves = kBlock / 64;
constexpr int32_t kDefaultChunkElems = LAMB_DEFAULT_CHUNK;

// One layer block x^(i) (Section 2) as the kernels see it. 64 bytes.
struct TensorDesc {
    float *x;
    const void *g;
    float *m;
    float *v;
    int64_t numel;
    int32_t wd;           // 1: lambda applies, 0: lambda = 0
    int32_t first_chunk;  // this tensor's chunks are [first_chunk, first_chunk + n_chunks)
    int32_t n_chunks;
    int32_t pad0;
    int64_t pad1;
};
static_assert(sizeof(TensorDesc) == 64, "TensorDesc layout");

// One chunk: `len` elements of tensor `tensor` starting at element `start`.
struct ChunkDesc {
    int32_t tensor;
    int32_t len;
    int64_t start;
};
static_assert(sizeof(ChunkDesc) == 16, "ChunkDesc layout");

// Per-chunk partial sums of squares, written once per step at a fixed slot.
struct Partial {
    double sum_xx;  // sum of x^2 over the chunk
    double sum_uu;  // sum of u^2 (LAMB) or m_t^2 (LARS) over the chunk
};

// Which corrected moments the update uses.
enum LambVariant : int {
    kLamb = 0,    // Algorithm 2: m_hat = m_t / c1, v_hat = v_t / c2
    kNLamb = 1,   // Algorithm 3: Nesterov m_hat, v_hat = beta2 v_t / c2
    kNNLamb = 2,  // Algorithm 4: Nesterov m_hat and v_hat
};

// fp32 scalars of the elementwise LAMB-family passes. The corrected moments
// are m_hat = m_scale * m_t + m_grad * g_t and v_hat = v_scale * v_t +
// v_grad * g_t^2; Algorithm 2 has m_grad = v_grad = 0.
struct LambArgs {
    float beta1, one_minus_beta1;
    float beta2, one_minus_beta2;
    float m_scale, m_grad;
    float v_scale, v_grad;
    float eps;
    float weight_decay;
};

// fp32 scalars of the elementwise LARS passes (Algorithm 1).
struct LarsArgs {
    float beta1, one_minus_beta1;
    float weight_decay;
};

// Scalars of the per-tensor finalize (trust ratio and step scale).
struct FinalizeArgs {
    double lr;
    double gamma_l, gamma_u;
    double trust_coef;  // 1 for LAMB
};

// Kernel launchers (lamb_kernels.hip). Each returns the launch status.
hipError_t launch_lamb_moments(const TensorDesc *tensors, const ChunkDesc *chunks,
                               Partial *partials, int32_t n_chunks, bool bf16_grad,
                               LambVariant variant, const LambArgs &args, hipStream_t stream);
hipError_t launch_lamb_apply(const TensorDesc *tensors, const ChunkDesc *chunks,
                             const float *scale, int32_t n_chunks, bool bf16_grad,
                             LambVariant variant, const LambArgs &args, hipStream_t stream);
hipError_t launch_lars_moments(const TensorDesc *tensors, const ChunkDesc *chunks,
                               Partial *partials, int32_t n_chunks, bool bf16_grad,
                               const LarsArgs &args, hipStream_t stream);
hipError_t launch_lars_apply(const TensorDesc *tensors, const ChunkDesc *chunks,
                             const float *scale, int32_t n_chunks, hipStream_t stream);
hipError_t launch_finalize(const TensorDesc *tensors, int32_t n_tensors,
                           const Partial *partials, const FinalizeArgs &args, float *scale,
                           double *ratio_out, double *norms_out, hipStream_t stream);

}  // namespace lamb_mi355x
