// Internal layout shared by the HIP kernels (lamb_kernels.hip) and the host
// side of the C ABI (lamb_api.cpp). Not installed; the public interface is
// include/lamb_mi355x.h.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace lamb_mi355x {

// Work is cut into chunks of at most `chunk_elems` elements of one tensor;
// one workgroup of two_pass_threads(chunk_elems) threads (at most kBlock)
// handles one chunk.
constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int32_t kDefaultChunkElems = 256;

// Threads per workgroup of the moment and apply passes over chunks of `chunk`
// elements: one float4 group per thread, whole waves, at least one wave and
// at most kBlock threads. A default chunk is one wave's float4 each: no thread
// of the workgroup idles.
constexpr int32_t two_pass_threads(int64_t chunk) {
    const int64_t threads = (chunk + 3) / 4;
    const int64_t waves = (threads + 63) / 64;
    return int32_t(waves < 1 ? 64 : waves * 64 > kBlock ? kBlock : waves * 64);
}

// A plan cuts every tensor twice: into fine chunks of chunk_elems elements
// (direct-mode moment passes and every apply pass) and into coarse chunks of
// kCoarseFactor times as many (deferred-mode moment passes, which only read
// and run faster with more work per workgroup).
constexpr int32_t kCoarseFactor = 8;

// Single-pass path: with tiles of G float4 groups per thread, a layer of n
// elements takes T = ceil(n / (G * kBlockElems)) tiles; tile i holds the
// layer's (4 * kBlock)-element blocks i, i + T, ..., i + (G - 1) T. One
// workgroup keeps a tile's x (the first kLdsGroups groups in LDS, any others
// in registers) and update direction (in registers) until the layer's step
// scale is known. The persistent grid keeps kFusedBlocksPerCu workgroups on
// every CU, so a layer of up to kFusedBlocksPerCu * (compute units) tiles can
// have every tile resident at once. A plan uses kTileGroups, or kWideGroups
// when the wider tile puts more parameters on the single pass.
constexpr int kTileGroups = 8;
constexpr int kWideGroups = 10;
constexpr int kLdsGroups = kTileGroups;
static_assert(kWideGroups > kTileGroups, "the wide tile is the larger one");
constexpr int32_t kBlockElems = kBlock * 4;  // one float4 per thread
constexpr int64_t tile_elems(int groups) { return int64_t(groups) * kBlockElems; }
constexpr int kFusedWaves = 4;  // waves per SIMD
constexpr int kFusedBlocksPerCu = kFusedWaves * 4 / kWaves;  // 4 SIMDs per CU
// Polls before a single-pass wait gives up (about a second); a plan reads an
// override from the environment variable LAMB_MI355X_SPIN_LIMIT.
constexpr uint32_t kDefaultSpinLimit = 1u << 22;

// Synchronisation words of the single-pass path (per plan).
enum FusedCtl : int {
    kCtlEpoch = 0,  // single-pass steps completed; its low bit selects the slot buffer
    kCtlDone = 1,   // workgroups of the running step that have finished
    kCtlFault = 2,  // sticky: a wait ran out of time and the step was abandoned
};

// One layer block x^(i) (Section 2) as the kernels see it. 80 bytes.
struct TensorDesc {
    float *x;
    const void *g;
    float *m;
    float *v;              // null for LARS plans
    uint16_t *x_copy;      // bf16 working copy written by the apply pass, or null
    int64_t numel;
    int32_t wd;            // 1: lambda applies, 0: lambda = 0
    int32_t first_chunk;   // fine chunks [first_chunk, first_chunk + n_chunks)
    int32_t n_chunks;
    int32_t first_coarse;  // coarse chunks [first_coarse, first_coarse + n_coarse)
    int32_t n_coarse;
    int32_t first_tile;    // single-pass tiles [first_tile, first_tile + n_tiles);
    int32_t n_tiles;       //   n_tiles = 0: the layer takes the two-pass path
    int32_t out_index;     // the layer's index in ratio_out / norms_out
    int32_t ext;           // single-pass table: the index of the layer's head in the
                           // two-pass table (its partial-norm totals and its step
                           // scale), or -1 when the whole layer is in the tiles
};
static_assert(sizeof(TensorDesc) == 88, "TensorDesc layout");

// One chunk: `len` elements of tensor `tensor` starting at element `start`.
struct ChunkDesc {
    int32_t tensor;
    int32_t len;
    int64_t start;
};
static_assert(sizeof(ChunkDesc) == 16, "ChunkDesc layout");

// The finalize runs in two levels: a segment kernel folds each run of up to
// kSegChunks consecutive chunk partials of one tensor into one segment
// partial, then the per-tensor finalize combines the tensor's segment
// partials. Both in a fixed order.
constexpr int kSegBlock = 256;
constexpr int kSegLanes = 8;
constexpr int32_t kSegChunks = kSegBlock * kSegLanes;

// One segment: chunk partials [first, first + count) of one tensor.
struct SegDesc {
    int32_t first;
    int32_t count;
};

// A tensor's segments: [first, first + count) of the segment list.
struct SegRange {
    int32_t first;
    int32_t count;
};

// Per-chunk partial norms of x and of the update direction u (LAMB family)
// or m_t (LARS), written once per step at a fixed slot: sums of squares (L2),
// sums of magnitudes (L1) or maxima of magnitudes (L-infinity).
struct Partial {
    double sum_xx;
    double sum_uu;
};

// Algorithms (the kernels' template argument).
enum Algo : int {
    kLamb = 0,    // Algorithm 2: m_hat = m_t / c1, v_hat = v_t / c2
    kNLamb = 1,   // Algorithm 3: Nesterov m_hat, v_hat = beta2 v_t / c2
    kNNLamb = 2,  // Algorithm 4: Nesterov m_hat and v_hat
    kLars = 3,    // Algorithm 1: momentum with weight decay
};

// Layer norms (Appendix F).
enum NormKind : int { kL2 = 0, kL1 = 1, kLinf = 2 };

// fp32 scalars of the elementwise passes. For the LAMB family the corrected
// moments are m_hat = m_scale * m_t + m_grad * g_t and v_hat = v_scale * v_t +
// v_grad * g_t^2 (Algorithm 2 has m_grad = v_grad = 0). LARS uses beta1 as its
// momentum. Every gradient element is multiplied by grad_scale first.
struct StepArgs {
    float beta1, one_minus_beta1;
    float beta2, one_minus_beta2;
    float m_scale, m_grad;
    float v_scale, v_grad;
    float eps;
    float weight_decay;
    float grad_scale;
    uint32_t spin_limit;  // single pass: polls before a wait gives up (>= 1)
};

// Scalars of the per-tensor finalize (trust ratio and step scale).
struct FinalizeArgs {
    double lr;
    double gamma_l, gamma_u;
    double trust_coef;  // 1 for the LAMB family
};

// What one step launches.
struct StepKind {
    Algo algo;
    NormKind norm;
    bool bf16_grad;
    bool deferred;  // moment pass writes nothing; apply pass recomputes and
                    // writes x, m, v unless a scaled gradient was non-finite
};

// The plan's flag words: [0] raised by a deferred-mode moment pass, [1] the
// verdict the finalize hands to the deferred apply pass; [2] and [3] the
// verdict of a skip_nonfinite step that checks the gradient first, selected
// by the single pass's epoch (kVerdictWord + (epoch & 1)).
constexpr int kVerdictWord = 2;
// Elements per chunk of the finiteness check.
constexpr int32_t kCheckElems = 16384;

// Kernel launchers (lamb_kernels.hip). Each returns the launch status.
// `flags` points at the plan's two non-finite words (deferred mode only): the
// moment pass raises flags[0], the finalize moves it to flags[1] and clears
// flags[0], the apply pass reads flags[1]. Nothing depends on a host counter,
// so a captured graph replays correctly. `nonfinite_out` may be null.
// `guard_ctl` non-null (direct mode only): return at once when the verdict
// word of the epoch in guard_ctl is raised. The moment and apply passes take
// a chunk table as one tensor id per chunk (`chunk_ids`) and its chunk size;
// the moment pass of deferred mode reads the coarse table (tensors'
// first_coarse), every other pass a fine one (first_chunk).
// Which verdict a direct-mode pass of a skip_nonfinite step obeys (it returns
// at once when that word is raised).
enum Guard : int32_t {
    kGuardNone = 0,   // not a skip_nonfinite step (or deferred mode)
    kGuardEpoch = 1,  // the verdict word of the epoch in ctl (kVerdictWord + (epoch & 1))
    kGuardCopy = 2,   // flags[1], the copy the totals kernel took before the single
                      // pass (which rewrites the epoch's words as it ends)
};

// `ctl` is the plan's FusedCtl words: every pass returns at once while the
// sticky fault word is raised, so that after a single-pass give-up no layer
// moves; `guard` is a Guard value.
hipError_t launch_moments(const StepKind &kind, const TensorDesc *tensors,
                          const int32_t *chunk_ids, int32_t chunk_elems, Partial *partials,
                          int32_t n_chunks, int32_t threads, uint32_t *flags,
                          const uint32_t *ctl, int32_t guard, const StepArgs &args,
                          hipStream_t stream);
// Both levels of the finalize: `segs` (n_segs entries) over `partials` into
// `seg_partials`, then per tensor over its `ranges` entry of the segments.
hipError_t launch_finalize(NormKind norm, const TensorDesc *tensors, int32_t n_tensors,
                           const Partial *partials, const SegDesc *segs, int32_t n_segs,
                           const SegRange *ranges, Partial *seg_partials,
                           const FinalizeArgs &args, float *scale, double *ratio_out,
                           double *norms_out, uint32_t *flags, hipStream_t stream);
// `check` non-null (direct mode only): also re-sum the partial norms of every
// chunk from the x read and the u recomputed, into check[chunk].
hipError_t launch_apply(const StepKind &kind, const TensorDesc *tensors,
                        const int32_t *chunk_ids, int32_t chunk_elems, const float *scale,
                        int32_t n_chunks, int32_t threads, uint32_t *flags, const uint32_t *ctl,
                        int32_t guard, int32_t *nonfinite_out, Partial *check,
                        const StepArgs &args, hipStream_t stream);
// What the totals kernel does with the step's non-finite verdict.
enum VerdictMode : int32_t {
    kVerdictZero = 0,   // totals[2 n] = 0 (a direct-mode step)
    kVerdictMove = 1,   // totals[2 n] = the deferred moment pass's flags[0], then cleared
    kVerdictCopy = 2,   // flags[1] = totals[2 n] = the epoch's verdict word (kGuardCopy)
};
// Per tensor its combined partial norms into totals[2 i], totals[2 i + 1]
// after the segment level over `partials`, and the verdict into totals[2 n]
// (a VerdictMode). The split step's first half, and the totals of the heads
// of layers split between the two paths.
hipError_t launch_totals(NormKind norm, const Partial *partials, const SegDesc *segs,
                         int32_t n_segs, const SegRange *ranges, int32_t n_tensors,
                         Partial *seg_partials, double *totals, uint32_t *flags,
                         const uint32_t *ctl, int32_t verdict_mode, hipStream_t stream);
// Split step, second half: per tensor the norms, phi, ratio and scale from
// combined totals; flags[1] receives the combined verdict for a deferred
// apply pass.
hipError_t launch_scale(NormKind norm, const double *totals, int32_t n_tensors,
                        const FinalizeArgs &args, float *scale, double *ratio_out,
                        double *norms_out, uint32_t *flags, hipStream_t stream);
// The finiteness check over `chunks` (all tensors, kCheckElems each).
hipError_t launch_finite(bool bf16_grad, const TensorDesc *tensors, const ChunkDesc *chunks,
                         int32_t n_chunks, uint32_t *flags, const uint32_t *ctl, float grad_scale,
                         hipStream_t stream);

// Single-pass kernel over the `n_tiles` tiles of the layers with n_tiles > 0,
// on a persistent grid of `grid` workgroups. `slots` holds 2 x 3 x n_tiles
// words (two buffers of partial norms and broadcast scales, alternating per
// step by the epoch in `ctl`), all initialised to kEmptySlot; `ctl` holds the
// FusedCtl words, initialised to 0.
constexpr uint64_t kEmptySlot = ~uint64_t(0);
// `guarded`: a skip_nonfinite step, whose verdict word the finiteness check
// raised or not; the last workgroup writes it to `nonfinite_out` (may be
// null). Every step's last workgroup clears the verdict word of the next
// epoch.
// `trace` non-null: every tile j of the step writes trace[4 j .. 4 j + 3], the
// device's constant 100 MHz clock when the tile starts, when its reads and
// partial norms are done, when its layer's scale is known and when its writes
// are issued.
// `groups` is the plan's tile shape, kTileGroups or kWideGroups. A layer
// whose descriptor has ext >= 0 (the last part of a layer too large for one
// round) combines the totals of its head, ext_totals[2 ext] and
// ext_totals[2 ext + 1], before its own tiles' partials, and writes its step
// scale to ext_scale[ext] for the apply pass over the head.
hipError_t launch_fused(const StepKind &kind, int groups, const TensorDesc *tensors,
                        const ChunkDesc *tiles, int32_t n_tiles, int32_t grid, uint64_t *slots,
                        uint32_t *ctl, uint32_t *flags, bool guarded, int32_t *nonfinite_out,
                        const StepArgs &args, const FinalizeArgs &fargs, double *ratio_out,
                        double *norms_out, const double *ext_totals, float *ext_scale,
                        uint64_t *trace, hipStream_t stream);
// Workgroups of the single-pass kernel for `kind` and tile shape `groups`
// that fit on one CU at once.
hipError_t fused_blocks_per_cu(const StepKind &kind, int groups, int *blocks);

}  // namespace lamb_mi355x
