// A planless two-pass step (lamb_step_static, include/lamb_mi355x.h) for
// callers that cannot allocate: code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc. It runs the same moment, finalize
// and apply kernels as a plan on LAMB_PATH_TWO_PASS, but keeps the tables,
// partial norms, scales and flags in one fixed device array of the library,
// and brings the tensor table to the device as kernel arguments of a small
// table kernel, so a call allocates no memory and copies nothing from the
// host.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>

#include "lamb_host.h"
#include "lamb_internal.h"

namespace lamb_mi355x {
namespace {

// ---------------------------------------------------------------------------
// Planless two-pass steps (lamb_step_static): every table, partial and flag
// lives in one fixed device array of the library, one per device, sized for
// at most kStaticMaxTensors tensors and kStaticMaxChunks fine chunks.
// ---------------------------------------------------------------------------
constexpr int32_t kStaticMaxTensors = 4096;
constexpr int32_t kStaticMaxChunks = 1 << 19;
// ceil(n / 8C) <= ceil(n / C) / 8 + 1 per tensor, and likewise for segments
constexpr int32_t kStaticMaxCoarse = kStaticMaxChunks / kCoarseFactor + kStaticMaxTensors;
constexpr int32_t kStaticMaxSegs = kStaticMaxChunks / kSegChunks + kStaticMaxTensors;
constexpr size_t static_round(size_t b) { return (b + 255) & ~size_t(255); }
constexpr size_t kStaticTensorsAt = 0;
constexpr size_t kStaticIdsAt =
    kStaticTensorsAt + static_round(sizeof(TensorDesc) * kStaticMaxTensors);
constexpr size_t kStaticCoarseIdsAt = kStaticIdsAt + static_round(4u * kStaticMaxChunks);
constexpr size_t kStaticPartialsAt = kStaticCoarseIdsAt + static_round(4u * kStaticMaxCoarse);
constexpr size_t kStaticSegsAt =
    kStaticPartialsAt + static_round(sizeof(Partial) * kStaticMaxChunks);
constexpr size_t kStaticRangesAt = kStaticSegsAt + 2 * static_round(sizeof(SegDesc) * kStaticMaxSegs);
constexpr size_t kStaticSegPartialsAt =
    kStaticRangesAt + 2 * static_round(sizeof(SegRange) * kStaticMaxTensors);
constexpr size_t kStaticScaleAt =
    kStaticSegPartialsAt + static_round(sizeof(Partial) * kStaticMaxSegs);
constexpr size_t kStaticFlagsAt = kStaticScaleAt + static_round(4u * kStaticMaxTensors);
constexpr size_t kStaticCtlAt = kStaticFlagsAt + 256;
constexpr size_t kStaticScratchBytes = kStaticCtlAt + 256;

// Views into one device's array (base: its device address).
struct StaticTables {
    TensorDesc *tensors;
    int32_t *ids;         // fine chunk table
    int32_t *coarse_ids;  // coarse chunk table
    Partial *partials;
    SegDesc *segs[2];     // finalize segments of the fine and the coarse table
    SegRange *ranges[2];
    Partial *seg_partials;
    float *scale;
    uint32_t *flags;      // the non-finite words, as a plan's
    uint32_t *ctl;        // FusedCtl words, all 0 (no single pass)
};

inline StaticTables static_tables(char *base) {
    StaticTables t;
    t.tensors = reinterpret_cast<TensorDesc *>(base + kStaticTensorsAt);
    t.ids = reinterpret_cast<int32_t *>(base + kStaticIdsAt);
    t.coarse_ids = reinterpret_cast<int32_t *>(base + kStaticCoarseIdsAt);
    t.partials = reinterpret_cast<Partial *>(base + kStaticPartialsAt);
    t.segs[0] = reinterpret_cast<SegDesc *>(base + kStaticSegsAt);
    t.segs[1] = reinterpret_cast<SegDesc *>(base + kStaticSegsAt +
                                            static_round(sizeof(SegDesc) * kStaticMaxSegs));
    t.ranges[0] = reinterpret_cast<SegRange *>(base + kStaticRangesAt);
    t.ranges[1] = reinterpret_cast<SegRange *>(base + kStaticRangesAt +
                                               static_round(sizeof(SegRange) * kStaticMaxTensors));
    t.seg_partials = reinterpret_cast<Partial *>(base + kStaticSegPartialsAt);
    t.scale = reinterpret_cast<float *>(base + kStaticScaleAt);
    t.flags = reinterpret_cast<uint32_t *>(base + kStaticFlagsAt);
    t.ctl = reinterpret_cast<uint32_t *>(base + kStaticCtlAt);
    return t;
}

// One tensor of a table batch: the caller's buffers plus where its chunks
// and segments start in the fine and the coarse table (host-computed
// prefixes). 64 bytes.
struct TableEntry {
    float *x;
    const void *g;
    float *m;
    float *v;
    int64_t numel;
    int32_t wd;
    int32_t first_chunk;
    int32_t first_coarse;
    int32_t first_seg;
    int32_t first_cseg;
    int32_t reserved;
};
static_assert(sizeof(TableEntry) == 64, "TableEntry layout");

// Up to kTableBatch tensors, passed to the table kernel by value (3 KB of
// kernel arguments): the step's tables reach the device with no copy and no
// buffer of their own.
constexpr int kTableBatch = 48;
struct TableBatch {
    TableEntry e[kTableBatch];
    int32_t count;        // entries used
    int32_t first_index;  // table index of e[0]
    int32_t chunk_elems;
    int32_t coarse_elems;
};

}  // namespace
}  // namespace lamb_mi355x

// Tables, partials and flags of planless steps: one array per device, held
// from the library's load on that device until the process ends. Host code
// never passes this name to a kernel (on the host it only stands for the
// device symbol); it uses the device address static_scratch() looks up.
static __device__ __align__(256) unsigned char scratch[lamb_mi355x::kStaticScratchBytes];

namespace lamb_mi355x {
namespace {

// ---------------------------------------------------------------------------
// Tables of a planless step, written from a batch passed by value: workgroup
// e writes tensor first_index + e's descriptor and segment ranges and fills
// its stretch of the fine and coarse chunk tables and of both segment lists.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void table_kernel(TableBatch b, StaticTables t) {
    const int e = blockIdx.x;
    const TableEntry &r = b.e[e];
    const int32_t i = b.first_index + e;
    const int32_t nc = int32_t((r.numel + b.chunk_elems - 1) / b.chunk_elems);
    const int32_t ncc = int32_t((r.numel + b.coarse_elems - 1) / b.coarse_elems);
    const int32_t ns = (nc + kSegChunks - 1) / kSegChunks;
    const int32_t ncs = (ncc + kSegChunks - 1) / kSegChunks;
    if (threadIdx.x == 0) {
        TensorDesc d;
        d.x = r.x;
        d.g = r.g;
        d.m = r.m;
        d.v = r.v;
        d.x_copy = nullptr;
        d.numel = r.numel;
        d.wd = r.wd;
        d.first_chunk = r.first_chunk;
        d.n_chunks = nc;
        d.first_coarse = r.first_coarse;
        d.n_coarse = ncc;
        d.first_tile = 0;
        d.n_tiles = 0;
        d.out_index = i;
        d.ext = -1;
        t.tensors[i] = d;
        t.ranges[0][i] = SegRange{r.first_seg, ns};
        t.ranges[1][i] = SegRange{r.first_cseg, ncs};
    }
    if (i == 0 && threadIdx.x < 64) {
        t.flags[threadIdx.x] = 0u;
        t.ctl[threadIdx.x] = 0u;
    }
    for (int32_t k = threadIdx.x; k < nc; k += kBlock)
        t.ids[r.first_chunk + k] = i;
    for (int32_t k = threadIdx.x; k < ncc; k += kBlock)
        t.coarse_ids[r.first_coarse + k] = i;
    for (int32_t k = threadIdx.x; k < ns; k += kBlock) {
        const int32_t left = nc - k * kSegChunks;
        t.segs[0][r.first_seg + k] =
            SegDesc{r.first_chunk + k * kSegChunks, left < kSegChunks ? left : kSegChunks};
    }
    for (int32_t k = threadIdx.x; k < ncs; k += kBlock) {
        const int32_t left = ncc - k * kSegChunks;
        t.segs[1][r.first_cseg + k] =
            SegDesc{r.first_coarse + k * kSegChunks, left < kSegChunks ? left : kSegChunks};
    }
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
char *g_scratch[kMaxDevices] = {};  // device address of `scratch`, by device

// Device address of the static array on the current device: looked up once
// per device, with that device current, and kept (each device holds its own
// copy of the array at its own address).
hipError_t static_scratch(char **base) {
    int device = 0;
    hipError_t err = hipGetDevice(&device);
    if (err != hipSuccess)
        return err;
    if (device < 0 || device >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch[device]) {
        void *p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(::scratch));
        if (err != hipSuccess)
            return err;
        if (!p)
            return hipErrorInvalidSymbol;
        g_scratch[device] = static_cast<char *>(p);
    }
    *base = g_scratch[device];
    return hipSuccess;
}

// Writes the batch's tensors into the tables at `t`: descriptors, chunk ids,
// segments and segment ranges of both tables; the batch holding tensor 0
// also clears the flag and control words.
hipError_t launch_table(const TableBatch &batch, const StaticTables &t, hipStream_t stream) {
    if (batch.count < 1 || batch.count > kTableBatch)
        return hipErrorInvalidValue;
    TableBatch b = batch;
    StaticTables tables = t;
    void *params[] = {&b, &tables};
    return hipLaunchKernel(reinterpret_cast<const void *>(&table_kernel), dim3(b.count),
                           dim3(kBlock), params, 0, stream);
}

// Room for the overlap check of planless steps (no allocation per call).
std::mutex g_static_mutex;
BufferRange g_static_ranges[4 * kStaticMaxTensors];

}  // namespace
}  // namespace lamb_mi355x

using namespace lamb_mi355x;

extern "C" {

lamb_status lamb_step_static(const lamb_tensor *tensors, int32_t n_tensors, int32_t g_dtype_in,
                             int32_t chunk_elems, const lamb_hparams *hp, void *stream,
                             double *ratio_out, double *norms_out, int32_t *nonfinite_out) {
    if (!tensors)
        return fail(LAMB_ENULL, "tensors must not be NULL");
    if (n_tensors < 1 || n_tensors > kStaticMaxTensors)
        return fail(LAMB_EINVAL, "n_tensors = %d, need 1 to %d", n_tensors, kStaticMaxTensors);
    if (g_dtype_in != LAMB_GRAD_F32 && g_dtype_in != LAMB_GRAD_BF16)
        return fail(LAMB_EINVAL, "unknown gradient dtype %d", g_dtype_in);
    const lamb_grad_dtype g_dtype = static_cast<lamb_grad_dtype>(g_dtype_in);
    int32_t chunk = 0;
    lamb_status st = resolve_chunk_elems(chunk_elems, &chunk);
    if (st != LAMB_OK)
        return st;
    st = check_hparams(nullptr, hp, nonfinite_out);
    if (st != LAMB_OK)
        return st;
    const bool needs_v = hp->variant != LAMB_VARIANT_LARS;
    {
        std::lock_guard<std::mutex> lock(g_static_mutex);
        int32_t n_ranges = 0;
        st = check_table(tensors, n_tensors, g_dtype, needs_v, g_static_ranges, &n_ranges);
        if (st != LAMB_OK)
            return st;
    }
    const int32_t coarse =
        int32_t(std::min<int64_t>(int64_t(chunk) * kCoarseFactor, kMaxChunkElems));
    int64_t n_chunks = 0, n_coarse = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        n_chunks += (tensors[i].numel + chunk - 1) / chunk;
        n_coarse += (tensors[i].numel + coarse - 1) / coarse;
        if (n_chunks > kStaticMaxChunks)
            return fail(LAMB_EINVAL, "more than %d chunks of %d elements (at most %d chunks "
                        "without a plan); raise chunk_elems", kStaticMaxChunks, chunk,
                        kStaticMaxChunks);
    }
    if (n_coarse > kStaticMaxCoarse)
        return fail(LAMB_EINVAL, "more than %d coarse chunks", kStaticMaxCoarse);
    const StepKind kind = step_kind(*hp, g_dtype);
    StepArgs a = step_args(*hp);
    const FinalizeArgs f = finalize_args(*hp);
    char *base = nullptr;
    hipError_t err = static_scratch(&base);
    if (err != hipSuccess)
        return fail_hip(err, "looking up the static device array");
    const StaticTables t = static_tables(base);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // The tables, batch by batch, as kernel arguments.
    TableBatch b;
    std::memset(&b, 0, sizeof b);
    b.chunk_elems = chunk;
    b.coarse_elems = coarse;
    int32_t first_chunk = 0, first_coarse = 0, first_seg = 0, first_cseg = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        const lamb_tensor &src = tensors[i];
        if (b.count == 0)
            b.first_index = i;
        const int32_t nc = int32_t((src.numel + chunk - 1) / chunk);
        const int32_t ncc = int32_t((src.numel + coarse - 1) / coarse);
        TableEntry &e = b.e[b.count++];
        e.x = src.x;
        e.g = src.g;
        e.m = src.m;
        e.v = needs_v ? src.v : nullptr;
        e.numel = src.numel;
        e.wd = src.wd;
        e.first_chunk = first_chunk;
        e.first_coarse = first_coarse;
        e.first_seg = first_seg;
        e.first_cseg = first_cseg;
        e.reserved = 0;
        first_chunk += nc;
        first_coarse += ncc;
        first_seg += (nc + kSegChunks - 1) / kSegChunks;
        first_cseg += (ncc + kSegChunks - 1) / kSegChunks;
        if (b.count == kTableBatch || i == n_tensors - 1) {
            err = launch_table(b, t, s);
            if (err != hipSuccess)
                return fail_hip(err, "launching the table kernel");
            b.count = 0;
        }
    }
    const int32_t *moment_ids = kind.deferred ? t.coarse_ids : t.ids;
    const int32_t n_moment = kind.deferred ? int32_t(n_coarse) : int32_t(n_chunks);
    const int32_t moment_elems = kind.deferred ? coarse : chunk;
    err = launch_moments(kind, t.tensors, moment_ids, moment_elems, t.partials, n_moment,
                         two_pass_threads(moment_elems), t.flags, t.ctl, kGuardNone, a, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the moment kernel");
    const int seg = kind.deferred ? 1 : 0;
    err = launch_finalize(kind.norm, t.tensors, n_tensors, t.partials, t.segs[seg],
                          kind.deferred ? first_cseg : first_seg, t.ranges[seg], t.seg_partials,
                          f, t.scale, ratio_out, norms_out, kind.deferred ? t.flags : nullptr, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the finalize kernel");
    err = launch_apply(kind, t.tensors, t.ids, chunk, t.scale, int32_t(n_chunks),
                       two_pass_threads(chunk), t.flags, t.ctl, kGuardNone,
                       kind.deferred ? nonfinite_out : nullptr, nullptr, a, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the apply kernel");
    return LAMB_OK;
}

}  // extern "C"
