// Host side of the C ABI declared in include/lamb_mi355x.h: argument
// validation, the chunk tables and the single-pass schedule (Section 2's
// layer blocks cut into work units), plan buffers, per-step scalars, kernel
// launches and timing hooks.

#include "lamb_mi355x.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "lamb_host.h"
#include "lamb_internal.h"

using namespace lamb_mi355x;

struct lamb_plan {
    int device = 0;
    lamb_algo algo = LAMB_ALGO_LAMB;
    lamb_grad_dtype g_dtype = LAMB_GRAD_F32;
    int32_t n_tensors = 0;
    int32_t n_chunks = 0;
    int32_t chunk_elems = 0;
    int32_t coarse_elems = 0;       // elements per coarse chunk
    void *device_block = nullptr;  // one allocation holding every device buffer below
    int32_t n_coarse = 0;       // coarse chunks (kCoarseFactor * chunk_elems each)
    TensorDesc *tensors = nullptr;
    int32_t *chunk_ids = nullptr;   // tensor id of every fine chunk
    int32_t *coarse_ids = nullptr;  // tensor id of every coarse chunk
    Partial *partials = nullptr;
    float *scale = nullptr;
    uint32_t *flags = nullptr;     // the four non-finite words (kVerdictWord)
    // Single-pass path: the tiles of the layers that fit, and a second tensor
    // and chunk table holding only the other layers (their two-pass work).
    lamb_path path = LAMB_PATH_AUTO;
    int32_t cu_count = 0;
    int32_t round = 0;             // single-pass grid: workgroups per round of the tile list
    int32_t tile_groups = kTileGroups;  // single-pass tile shape (float4 groups per thread)
    uint32_t spin_limit = kDefaultSpinLimit;
    int32_t n_tiles = 0;
    int32_t n_rest = 0;            // layers outside the single pass
    int32_t n_rest_chunks = 0;
    ChunkDesc *tiles = nullptr;
    uint64_t *slots = nullptr;     // 2 x 3 x n_tiles slot words
    uint32_t *ctl = nullptr;       // FusedCtl words
    // Layers of more than one round of tiles keep a head on the two-pass
    // kernels (rest_tensors) and put their tail on the single pass.
    TensorDesc *rest_tensors = nullptr;
    int32_t *rest_ids = nullptr;    // tensor id (in rest_tensors) of every fine chunk of the heads
    TensorDesc *fused_tensors = nullptr;  // the single pass's table: tails at their offsets
    double *ext_totals = nullptr;   // the heads' partial-norm totals (2 per head, then a verdict)
    // Finalize segments of the fine, the coarse and the other-layers table.
    SegDesc *segs[3] = {};
    SegRange *seg_ranges[3] = {};
    int32_t n_segs[3] = {};
    Partial *seg_partials = nullptr;
    int fused_per_cu[4][2][3] = {};  // single-pass workgroups per CU by algo, bf16, norm
    std::vector<TensorDesc> host_tensors;  // host image of the tensor table
    std::vector<TensorDesc> host_rest;     // host image of the heads' table
    std::vector<TensorDesc> host_fused;    // host image of the single pass's table
    std::vector<int64_t> single_elems;     // elements of each layer on the single pass
    std::vector<std::pair<uintptr_t, uintptr_t>> ranges;  // sorted buffer ranges of the table
    // finiteness check of skip_nonfinite steps that take the single pass
    ChunkDesc *check_chunks = nullptr;
    int32_t n_check = 0;
    // u-consistency check (lamb_plan_set_u_check): the apply pass's re-summed
    // partial norms, and the chunk count of the last step that filled them
    Partial *u_check = nullptr;
    int32_t u_check_chunks = 0;
    uint64_t *trace = nullptr;      // caller's per-tile clock stamps (lamb_plan_set_trace)
    // timing hooks: up to kEvents events per recorded step, in launch order,
    // with the kernel kind of each interval
    std::vector<hipEvent_t> events;
    std::vector<uint8_t> timing_kinds;
    std::vector<uint8_t> timing_count;
    int timing_next = 0;
    int32_t timing_capacity = 0;
    int32_t timing_used = 0;
    int32_t timing_every = 1;      // record one step in timing_every
    int64_t timing_seen = 0;       // steps enqueued since timing was enabled
    bool timing_this_step = false;
};

namespace lamb_mi355x {

// Kernel kinds of the timing hooks (the index in lamb_plan_timing's output).
enum TimedKernel : uint8_t { kTimedMoments = 0, kTimedFinalize = 1, kTimedApply = 2,
                             kTimedSingle = 3, kTimedCheck = 4, kTimedKinds = 5 };
constexpr int kEvents = kTimedKinds + 1;  // at most one interval per kind

thread_local char g_last_error[512] = "";

lamb_status fail(lamb_status status, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

lamb_status fail_hip(hipError_t err, const char *what) {
    return fail(LAMB_EHIP, "%s: %s", what, hipGetErrorString(err));
}

bool aligned16(const void *p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}


// Every size in [1, kMaxNumel]: chunk and tile counts then stay far from
// int64 overflow.
lamb_status check_numel(const int64_t *numel, int32_t n) {
    for (int32_t i = 0; i < n; ++i)
        if (numel[i] < 1 || numel[i] > kMaxNumel)
            return fail(LAMB_EINVAL, "tensor %d has numel %lld, need 1 to 2^40", i,
                        static_cast<long long>(numel[i]));
    return LAMB_OK;
}

lamb_status resolve_chunk_elems(int32_t requested, int32_t *out) {
    if (requested == 0) {
        *out = kDefaultChunkElems;
        return LAMB_OK;
    }
    if (requested < 8 || requested > kMaxChunkElems || requested % 8 != 0)
        return fail(LAMB_EINVAL, "chunk_elems %d must be 0 or a multiple of 8 in [8, 2^30]",
                    requested);
    *out = requested;
    return LAMB_OK;
}

// Number of chunks of the table, or -1 if it exceeds the grid limit.
int64_t count_chunks(const int64_t *numel, int32_t n, int32_t chunk) {
    int64_t total = 0;
    for (int32_t i = 0; i < n; ++i) {
        total += (numel[i] + chunk - 1) / chunk;
        if (total > INT32_MAX)
            return -1;
    }
    return total;
}

// Scoped switch to the plan's device.
struct DeviceGuard {
    int previous = -1;
    hipError_t status = hipSuccess;
    explicit DeviceGuard(int device) {
        status = hipGetDevice(&previous);
        if (status == hipSuccess && previous != device)
            status = hipSetDevice(device);
        else if (status == hipSuccess)
            previous = -1;
    }
    ~DeviceGuard() {
        if (previous >= 0)
            (void)hipSetDevice(previous);
    }
};

bool finite(float a) { return std::isfinite(a); }

lamb_status check_phi_bounds(float gamma_l, float gamma_u) {
    if (!(gamma_l >= 0.0f) || !finite(gamma_l) || !(gamma_u >= gamma_l))
        return fail(LAMB_EINVAL, "need 0 <= gamma_l <= gamma_u (gamma_l finite), got %g, %g",
                    double(gamma_l), double(gamma_u));
    return LAMB_OK;
}

// Timing hooks: begin_timing decides whether this step is recorded and
// records its first event; mark() records the event after a kernel.
void begin_timing(lamb_plan *plan, hipStream_t stream) {
    plan->timing_this_step = plan->timing_used < plan->timing_capacity &&
                             plan->timing_seen % plan->timing_every == 0;
    ++plan->timing_seen;
    plan->timing_next = 0;
    if (plan->timing_this_step)
        (void)hipEventRecord(plan->events[size_t(plan->timing_used) * kEvents], stream);
}

void mark(lamb_plan *plan, TimedKernel kind, hipStream_t stream) {
    if (!plan->timing_this_step || plan->timing_next >= kEvents - 1)
        return;
    const size_t k = size_t(plan->timing_used);
    plan->timing_kinds[k * (kEvents - 1) + size_t(plan->timing_next)] = kind;
    ++plan->timing_next;
    (void)hipEventRecord(plan->events[k * kEvents + size_t(plan->timing_next)], stream);
}

// Single-pass launches of one process on one device run one at a time: each
// persistent grid needs the whole device resident, and two such grids on
// different streams could each hold part of it and wait on each other. A
// launch on another stream than the previous one first waits for the
// previous launch. Graph capture skips the gate (the replay order is the
// caller's).
struct FusedGate {
    hipEvent_t done = nullptr;
    hipStream_t stream = nullptr;
    bool used = false;
};
std::mutex g_gate_mutex;
std::vector<FusedGate> g_gates;  // by device; events live until the process ends

hipError_t gated_fused_launch(int device, hipStream_t stream, const StepKind &kind,
                              const lamb_plan *plan, int32_t grid, bool guarded,
                              int32_t *nonfinite_out, const StepArgs &a, const FinalizeArgs &f,
                              double *ratio_out, double *norms_out) {
    hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
    hipError_t err = hipStreamIsCapturing(stream, &capture);
    if (err != hipSuccess)
        return err;
    if (capture != hipStreamCaptureStatusNone)
        return launch_fused(kind, plan->tile_groups, plan->fused_tensors, plan->tiles,
                            plan->n_tiles, grid, plan->slots, plan->ctl, plan->flags, guarded,
                            nonfinite_out, a, f, ratio_out, norms_out, plan->ext_totals,
                            plan->scale, plan->trace, stream);
    std::lock_guard<std::mutex> lock(g_gate_mutex);
    if (g_gates.size() <= size_t(device))
        g_gates.resize(size_t(device) + 1);
    FusedGate &gate = g_gates[size_t(device)];
    if (!gate.done) {
        // only orders kernels of this device: no system-scope fence (which
        // writes back the caches and cost about 1.7 us per step)
        err = hipEventCreateWithFlags(&gate.done,
                                      hipEventDisableTiming | hipEventDisableSystemFence);
        if (err != hipSuccess)
            return err;
    }
    if (gate.used && gate.stream != stream) {
        err = hipStreamWaitEvent(stream, gate.done, 0);
        if (err != hipSuccess)
            return err;
    }
    err = launch_fused(kind, plan->tile_groups, plan->fused_tensors, plan->tiles, plan->n_tiles,
                       grid, plan->slots, plan->ctl, plan->flags, guarded, nonfinite_out, a, f,
                       ratio_out, norms_out, plan->ext_totals, plan->scale, plan->trace, stream);
    if (err != hipSuccess)
        return err;
    err = hipEventRecord(gate.done, stream);
    if (err != hipSuccess)
        return err;
    gate.stream = stream;
    gate.used = true;
    return hipSuccess;
}

void end_timing(lamb_plan *plan) {
    if (plan->timing_this_step) {
        plan->timing_count[size_t(plan->timing_used)] = uint8_t(plan->timing_next);
        ++plan->timing_used;
    }
    plan->timing_this_step = false;
}

// The chunk table of `numel` at `chunk` elements per chunk (lamb_chunk_table).
lamb_status build_chunks(const std::vector<int64_t> &numel, int32_t chunk, int32_t n_chunks,
                         std::vector<ChunkDesc> *out);

void release_events(lamb_plan *plan) {
    for (hipEvent_t e : plan->events)
        (void)hipEventDestroy(e);
    plan->events.clear();
    plan->timing_capacity = 0;
    plan->timing_used = 0;
    plan->timing_every = 1;
    plan->timing_seen = 0;
}

}  // namespace lamb_mi355x

extern "C" {

const char *lamb_status_str(int32_t status) {
    switch (status) {
    case LAMB_OK: return "ok";
    case LAMB_EINVAL: return "invalid argument";
    case LAMB_ENULL: return "null pointer";
    case LAMB_EALIGN: return "tensor not 16-byte aligned";
    case LAMB_EOVERLAP: return "tensor buffers overlap";
    case LAMB_EHIP: return "HIP runtime error";
    case LAMB_ENOMEM: return "out of memory";
    case LAMB_EPLAN: return "plan built for the other algorithm";
    case LAMB_ESYNC: return "a single-pass step abandoned a wait";
    }
    return "unknown status";
}

const char *lamb_last_error(void) { return g_last_error; }

lamb_status lamb_chunk_table(const int64_t *numel, int32_t n_tensors, int32_t chunk_elems,
                             int32_t capacity, int32_t *chunk_tensor, int64_t *chunk_start,
                             int32_t *chunk_len, int32_t *n_chunks) {
    if (!numel || !n_chunks)
        return fail(LAMB_ENULL, "numel and n_chunks must not be NULL");
    if (n_tensors < 1)
        return fail(LAMB_EINVAL, "n_tensors = %d, need >= 1", n_tensors);
    int32_t chunk = 0;
    lamb_status st = resolve_chunk_elems(chunk_elems, &chunk);
    if (st != LAMB_OK)
        return st;
    st = check_numel(numel, n_tensors);
    if (st != LAMB_OK)
        return st;
    const int64_t total = count_chunks(numel, n_tensors, chunk);
    if (total < 0)
        return fail(LAMB_EINVAL, "more than 2^31-1 chunks; raise chunk_elems");
    *n_chunks = int32_t(total);
    if (capacity == 0 && !chunk_tensor && !chunk_start && !chunk_len)
        return LAMB_OK;
    if (capacity < total)
        return fail(LAMB_EINVAL, "capacity %d < %lld chunks", capacity,
                    static_cast<long long>(total));
    if (!chunk_tensor || !chunk_start || !chunk_len)
        return fail(LAMB_ENULL, "chunk output arrays must not be NULL");
    int32_t k = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        for (int64_t s = 0; s < numel[i]; s += chunk) {
            chunk_tensor[k] = i;
            chunk_start[k] = s;
            chunk_len[k] = int32_t(std::min<int64_t>(chunk, numel[i] - s));
            ++k;
        }
    }
    return LAMB_OK;
}

namespace {

// Parameters a tile shape of `groups` puts on the single pass: those of the
// layers of at most `max_round` tiles.
int64_t single_pass_params(const int64_t *numel, int32_t n_tensors, int32_t max_round,
                           int groups) {
    const int64_t te = tile_elems(groups);
    int64_t total = 0;
    for (int32_t i = 0; i < n_tensors; ++i)
        if ((numel[i] + te - 1) / te <= max_round)
            total += numel[i];
    return total;
}

}  // namespace

lamb_status lamb_tile_schedule(const int64_t *numel, int32_t n_tensors, int32_t max_round,
                               int32_t tile_groups, int32_t capacity, int32_t *entry_tensor,
                               int64_t *entry_start, int32_t *entry_len, int32_t *first_tile,
                               int32_t *tiles, int32_t *n_entries, int32_t *round_out,
                               int32_t *groups_out) {
    if (!numel || !n_entries || !first_tile || !tiles || !round_out)
        return fail(LAMB_ENULL,
                    "numel, first_tile, tiles, n_entries and round_out must not be NULL");
    if (n_tensors < 1)
        return fail(LAMB_EINVAL, "n_tensors = %d, need >= 1", n_tensors);
    if (max_round < 1)
        return fail(LAMB_EINVAL, "max_round = %d, need >= 1", max_round);
    if (tile_groups != 0 && tile_groups != kTileGroups && tile_groups != kWideGroups)
        return fail(LAMB_EINVAL, "tile_groups = %d, need 0, %d or %d", tile_groups, kTileGroups,
                    kWideGroups);
    const lamb_status st = check_numel(numel, n_tensors);
    if (st != LAMB_OK)
        return st;
    // A plan's choice: the wide tile only if it puts more parameters on the
    // single pass (with as many, the narrow tile streams slightly faster).
    int groups = tile_groups;
    if (groups == 0)
        groups = single_pass_params(numel, n_tensors, max_round, kWideGroups) >
                         single_pass_params(numel, n_tensors, max_round, kTileGroups)
                     ? kWideGroups
                     : kTileGroups;
    if (groups_out)
        *groups_out = groups;
    const int64_t te = tile_elems(groups);
    // Layers of at most `max_round` tiles, in decreasing tile count (ties in
    // table order).
    std::vector<std::pair<int64_t, int32_t>> teams;
    int64_t total_tiles = 0, largest = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        const int64_t nt = (numel[i] + te - 1) / te;
        first_tile[i] = 0;
        tiles[i] = 0;
        if (nt <= max_round) {
            teams.emplace_back(nt, i);
            total_tiles += nt;
            largest = std::max(largest, nt);
        }
    }
    using Team = std::pair<int64_t, int32_t>;
    std::stable_sort(teams.begin(), teams.end(),
                     [](const Team &a, const Team &b) { return a.first > b.first; });
    // First-fit into rounds of `width` entries.
    std::vector<int64_t> fill;
    std::vector<std::vector<int32_t>> members;
    auto pack = [&](int64_t width) {
        fill.clear();
        members.clear();
        for (const auto &team : teams) {
            size_t r = 0;
            while (r < fill.size() && fill[r] + team.first > width)
                ++r;
            if (r == fill.size()) {
                fill.push_back(0);
                members.emplace_back();
            }
            fill[r] += team.first;
            members[r].push_back(team.second);
        }
    };
    // The fewest rounds, at the narrowest width that still needs no more:
    // the rounds come out about equally full instead of full rounds and a
    // short last one.
    // Binary search over the width (at most ~10 packings): the smallest width
    // in [lower bound, max_round] whose packing needs no more rounds.
    pack(max_round);
    const size_t n_rounds = fill.size();
    int64_t round = max_round;
    if (n_rounds > 0) {
        int64_t lo = std::max(largest, (total_tiles + int64_t(n_rounds) - 1) / int64_t(n_rounds));
        int64_t hi = max_round;  // packs into n_rounds
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            pack(mid);
            if (fill.size() <= n_rounds)
                hi = mid;
            else
                lo = mid + 1;
        }
        round = hi;
        pack(round);
    }
    *round_out = int32_t(round);
    const int64_t total =
        fill.empty() ? 0 : int64_t(round) * int64_t(fill.size() - 1) + fill.back();
    if (total > INT32_MAX / 8)
        return fail(LAMB_EINVAL, "too many single-pass tiles");
    *n_entries = int32_t(total);
    const bool write = capacity != 0 || entry_tensor || entry_start || entry_len;
    if (write && capacity < total)
        return fail(LAMB_EINVAL, "capacity %d < %lld entries", capacity,
                    static_cast<long long>(total));
    if (write && (!entry_tensor || !entry_start || !entry_len))
        return fail(LAMB_ENULL, "entry output arrays must not be NULL");
    int32_t k = 0;
    for (size_t r = 0; r < fill.size(); ++r) {
        for (int32_t i : members[r]) {
            const int64_t nt = (numel[i] + te - 1) / te;
            first_tile[i] = k;
            tiles[i] = int32_t(nt);
            for (int64_t j = 0; j < nt; ++j, ++k) {
                if (!write)
                    continue;
                // tile j holds the blocks j, j + nt, ... of kBlockElems each
                int64_t held = 0;
                for (int64_t b = j; b < int64_t(groups) * nt; b += nt)
                    held += std::max<int64_t>(0, std::min<int64_t>(kBlockElems,
                                                                   numel[i] - b * kBlockElems));
                entry_tensor[k] = i;
                entry_start[k] = j * kBlockElems;
                entry_len[k] = int32_t(held);
            }
        }
        if (r + 1 < fill.size()) {
            for (int64_t j = fill[r]; j < round; ++j, ++k) {
                if (!write)
                    continue;
                entry_tensor[k] = -1;
                entry_start[k] = 0;
                entry_len[k] = 0;
            }
        }
    }
    return LAMB_OK;
}

}  // extern "C"

namespace lamb_mi355x {

lamb_status build_chunks(const std::vector<int64_t> &numel, int32_t chunk, int32_t n_chunks,
                         std::vector<ChunkDesc> *out) {
    std::vector<int32_t> ct(static_cast<size_t>(n_chunks)), cl(static_cast<size_t>(n_chunks));
    std::vector<int64_t> cs(static_cast<size_t>(n_chunks));
    int32_t count = 0;
    lamb_status st = lamb_chunk_table(numel.data(), int32_t(numel.size()), chunk, n_chunks,
                                      ct.data(), cs.data(), cl.data(), &count);
    if (st != LAMB_OK)
        return st;
    out->resize(static_cast<size_t>(n_chunks));
    for (int32_t k = 0; k < n_chunks; ++k)
        (*out)[size_t(k)] = ChunkDesc{ct[size_t(k)], cl[size_t(k)], cs[size_t(k)]};
    return LAMB_OK;
}

// Validates a table of blocks (as lamb_plan_create documents) using the
// caller's room for 4 * n ranges, which it leaves sorted; allocates nothing.
lamb_status check_table(const lamb_tensor *tensors, int32_t n_tensors, lamb_grad_dtype g_dtype,
                        bool needs_v, BufferRange *ranges, int32_t *n_ranges) {
    const size_t g_size = g_dtype == LAMB_GRAD_BF16 ? 2 : 4;
    int32_t k = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        const lamb_tensor &t = tensors[i];
        if (!t.x || !t.g || !t.m || (needs_v && !t.v))
            return fail(LAMB_ENULL, "tensor %d: x, g, m%s must not be NULL", i,
                        needs_v ? ", v" : "");
        if (t.numel < 1 || t.numel > kMaxNumel)
            return fail(LAMB_EINVAL, "tensor %d: numel %lld, need 1 to 2^40", i,
                        static_cast<long long>(t.numel));
        if (t.wd != 0 && t.wd != 1)
            return fail(LAMB_EINVAL, "tensor %d: wd must be 0 or 1", i);
        if (t.reserved != 0)
            return fail(LAMB_EINVAL, "tensor %d: reserved field must be 0", i);
        if (!aligned16(t.x) || !aligned16(t.g) || !aligned16(t.m) || (needs_v && !aligned16(t.v)))
            return fail(LAMB_EALIGN, "tensor %d: every buffer must be 16-byte aligned", i);
        const uintptr_t f32_bytes = uintptr_t(t.numel) * 4u;
        auto add = [&](const void *p, uintptr_t bytes, const char *what) {
            const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
            ranges[k++] = BufferRange{lo, lo + bytes, i, what};
        };
        add(t.x, f32_bytes, "x");
        add(t.g, uintptr_t(t.numel) * g_size, "g");
        add(t.m, f32_bytes, "m");
        if (needs_v)
            add(t.v, f32_bytes, "v");
    }
    std::sort(ranges, ranges + k,
              [](const BufferRange &a, const BufferRange &b) { return a.lo < b.lo; });
    for (int32_t j = 1; j < k; ++j)
        if (ranges[j].lo < ranges[j - 1].hi)
            return fail(LAMB_EOVERLAP, "tensor %d %s overlaps tensor %d %s", ranges[j].tensor,
                        ranges[j].what, ranges[j - 1].tensor, ranges[j - 1].what);
    *n_ranges = k;
    return LAMB_OK;
}

enum SegTable { kSegFine = 0, kSegCoarse = 1, kSegRest = 2 };

// The tensor id of every chunk of a table (what the moment and apply passes
// read; start and length follow from the tensor and the chunk size).
std::vector<int32_t> ids_of(const std::vector<ChunkDesc> &chunks) {
    std::vector<int32_t> ids(chunks.size());
    for (size_t k = 0; k < chunks.size(); ++k)
        ids[k] = chunks[k].tensor;
    return ids;
}

// Finalize segments of a chunk table: tensor k's chunk partials
// [first_k, first_k + count_k) cut into runs of kSegChunks.
void build_segments(const std::vector<std::pair<int32_t, int32_t>> &tensor_chunks,
                    std::vector<SegDesc> *segs, std::vector<SegRange> *ranges) {
    segs->clear();
    ranges->clear();
    for (const auto &tc : tensor_chunks) {
        const int32_t first_seg = int32_t(segs->size());
        for (int32_t k = 0; k < tc.second; k += kSegChunks)
            segs->push_back(SegDesc{tc.first + k, std::min(kSegChunks, tc.second - k)});
        ranges->push_back(SegRange{first_seg, int32_t(segs->size()) - first_seg});
    }
}

}  // namespace lamb_mi355x

extern "C" {

lamb_status lamb_plan_create(const lamb_tensor *tensors, int32_t n_tensors,
                             int32_t g_dtype_in, int32_t algo_in, int32_t chunk_elems,
                             lamb_plan **out) {
    if (!out)
        return fail(LAMB_ENULL, "out must not be NULL");
    *out = nullptr;
    if (!tensors)
        return fail(LAMB_ENULL, "tensors must not be NULL");
    if (n_tensors < 1)
        return fail(LAMB_EINVAL, "n_tensors = %d, need >= 1", n_tensors);
    if (g_dtype_in != LAMB_GRAD_F32 && g_dtype_in != LAMB_GRAD_BF16)
        return fail(LAMB_EINVAL, "unknown gradient dtype %d", g_dtype_in);
    if (algo_in != LAMB_ALGO_LAMB && algo_in != LAMB_ALGO_LARS)
        return fail(LAMB_EINVAL, "unknown algorithm %d", algo_in);
    const lamb_grad_dtype g_dtype = static_cast<lamb_grad_dtype>(g_dtype_in);
    const lamb_algo algo = static_cast<lamb_algo>(algo_in);
    int32_t chunk = 0;
    lamb_status st = resolve_chunk_elems(chunk_elems, &chunk);
    if (st != LAMB_OK)
        return st;

    const bool needs_v = algo == LAMB_ALGO_LAMB;
    std::vector<int64_t> numel(size_t(n_tensors), 0);
    std::vector<BufferRange> ranges(size_t(n_tensors) * 4);
    int32_t n_ranges = 0;
    st = check_table(tensors, n_tensors, g_dtype, needs_v, ranges.data(), &n_ranges);
    if (st != LAMB_OK)
        return st;
    ranges.resize(size_t(n_ranges));
    for (int32_t i = 0; i < n_tensors; ++i)
        numel[size_t(i)] = tensors[i].numel;

    const int64_t total = count_chunks(numel.data(), n_tensors, chunk);
    if (total < 0)
        return fail(LAMB_EINVAL, "more than 2^31-1 chunks; raise chunk_elems");
    const int32_t n_chunks = int32_t(total);
    const int32_t coarse = int32_t(std::min<int64_t>(int64_t(chunk) * kCoarseFactor,
                                                     kMaxChunkElems));
    const int32_t n_coarse = int32_t(count_chunks(numel.data(), n_tensors, coarse));

    // Host images of the tables: the fine and the coarse chunk table, and the
    // tensor table with each tensor's range in both.
    std::vector<TensorDesc> host_tensors(static_cast<size_t>(n_tensors));
    std::vector<ChunkDesc> host_chunks;
    std::vector<ChunkDesc> host_coarse;
    st = build_chunks(numel, chunk, n_chunks, &host_chunks);
    if (st == LAMB_OK)
        st = build_chunks(numel, coarse, n_coarse, &host_coarse);
    std::vector<ChunkDesc> host_check;
    const int64_t n_check64 = count_chunks(numel.data(), n_tensors, kCheckElems);
    if (st == LAMB_OK && n_check64 < 0)
        st = fail(LAMB_EINVAL, "too many finiteness-check chunks");
    if (st == LAMB_OK)
        st = build_chunks(numel, kCheckElems, int32_t(n_check64), &host_check);
    if (st != LAMB_OK)
        return st;
    int device = 0, cu_count = 0;
    hipError_t err = hipGetDevice(&device);
    if (err == hipSuccess)
        err = hipDeviceGetAttribute(&cu_count, hipDeviceAttributeMultiprocessorCount, device);
    if (err != hipSuccess)
        return fail_hip(err, "querying the current device");
    // Single-pass schedule (lamb_tile_schedule): rounds of one tile per
    // workgroup of the persistent grid, which keeps kFusedBlocksPerCu
    // workgroups on every CU.
    const int32_t max_round = int32_t(std::max<int64_t>(1, int64_t(kFusedBlocksPerCu) * cu_count));
    std::vector<int32_t> first_tile(static_cast<size_t>(n_tensors)),
        tile_count(static_cast<size_t>(n_tensors));
    uint32_t spin_limit = kDefaultSpinLimit;
    if (const char *env = std::getenv("LAMB_MI355X_SPIN_LIMIT")) {
        char *end = nullptr;
        const long long v = std::strtoll(env, &end, 10);
        if (end == env || *end != '\0' || v < 1)
            return fail(LAMB_EINVAL, "LAMB_MI355X_SPIN_LIMIT = \"%s\", need a positive integer",
                        env);
        spin_limit = uint32_t(std::min<long long>(v, 1LL << 30));
    }
    int32_t n_entries = 0, round = 0, groups = 0;
    if (const char *env = std::getenv("LAMB_MI355X_TILE_GROUPS")) {
        char *end = nullptr;
        const long v = std::strtol(env, &end, 10);
        if (end == env || *end != '\0' || (v != kTileGroups && v != kWideGroups))
            return fail(LAMB_EINVAL, "LAMB_MI355X_TILE_GROUPS = \"%s\", need %d or %d", env,
                        kTileGroups, kWideGroups);
        groups = int32_t(v);
    }
    // The tile shape (lamb_tile_schedule's rule over whole layers), then the
    // schedule: a layer of more tiles than a round keeps a head on the
    // two-pass kernels and puts its last elements on the single pass, from a
    // multiple of kBlockElems, in as many tiles as the largest layer that
    // fits whole (one round if none does). Every tile of a layer must be
    // resident at once, and work on other streams can withhold residency; a
    // tail no larger than the plan's largest layer keeps that demand as it
    // was (a tail of a whole round, on a plan whose layers take half of one,
    // gave up its waits beside fp32 matrix products on another stream).
    st = lamb_tile_schedule(numel.data(), n_tensors, max_round, groups, 0, nullptr, nullptr,
                            nullptr, first_tile.data(), tile_count.data(), &n_entries, &round,
                            &groups);
    if (st != LAMB_OK)
        return st;
    int64_t largest = 0;
    for (int32_t i = 0; i < n_tensors; ++i)
        largest = std::max<int64_t>(largest, tile_count[size_t(i)]);
    const int64_t round_elems = int64_t(max_round) * tile_elems(groups);
    // the single pass addresses a layer's elements with 32-bit byte offsets
    if (round_elems > (int64_t(1) << 29))
        return fail(LAMB_EINVAL, "%d single-pass workgroups: a round of tiles exceeds 2^29 elements",
                    max_round);
    const int64_t tail_elems = (largest > 0 ? largest : max_round) * tile_elems(groups);
    std::vector<int64_t> head(size_t(n_tensors), 0), tail(size_t(n_tensors), 0);
    for (int32_t i = 0; i < n_tensors; ++i) {
        const int64_t n = numel[size_t(i)];
        if (n > round_elems)
            head[size_t(i)] = (n - tail_elems + kBlockElems - 1) / kBlockElems * kBlockElems;
        tail[size_t(i)] = n - head[size_t(i)];
    }
    st = lamb_tile_schedule(tail.data(), n_tensors, max_round, groups, 0, nullptr, nullptr,
                            nullptr, first_tile.data(), tile_count.data(), &n_entries, &round,
                            nullptr);
    std::vector<int32_t> entry_tensor(static_cast<size_t>(n_entries)),
        entry_len(static_cast<size_t>(n_entries));
    std::vector<int64_t> entry_start(static_cast<size_t>(n_entries));
    if (st == LAMB_OK)
        st = lamb_tile_schedule(tail.data(), n_tensors, max_round, groups, n_entries,
                                entry_tensor.data(), entry_start.data(), entry_len.data(),
                                first_tile.data(), tile_count.data(), &n_entries, &round,
                                nullptr);
    if (st != LAMB_OK)
        return st;
    std::vector<ChunkDesc> host_tiles(static_cast<size_t>(n_entries));
    for (int32_t k = 0; k < n_entries; ++k)
        host_tiles[size_t(k)] =
            ChunkDesc{entry_tensor[size_t(k)], entry_len[size_t(k)], entry_start[size_t(k)]};
    // Three tensor tables: every layer whole (the two-pass path and the split
    // step), the single pass's (tails at their offsets), and the heads.
    std::vector<TensorDesc> host_fused(static_cast<size_t>(n_tensors));
    std::vector<TensorDesc> host_rest;
    std::vector<int32_t> host_rest_ids;
    {
        int32_t first = 0, first_coarse = 0;
        for (int32_t i = 0; i < n_tensors; ++i) {
            const lamb_tensor &t = tensors[i];
            const int32_t nc = int32_t((t.numel + chunk - 1) / chunk);
            const int32_t ncc = int32_t((t.numel + coarse - 1) / coarse);
            TensorDesc d{t.x,          t.g,          t.m,   needs_v ? t.v : nullptr,
                         nullptr,      t.numel,      t.wd,  first,
                         nc,           first_coarse, ncc,   first_tile[size_t(i)],
                         tile_count[size_t(i)], i,   -1};
            host_tensors[size_t(i)] = d;
            const int64_t h = head[size_t(i)];
            TensorDesc f = d;
            f.first_chunk = f.n_chunks = f.first_coarse = f.n_coarse = 0;
            if (h > 0) {
                const size_t g_size = g_dtype == LAMB_GRAD_BF16 ? 2 : 4;
                f.x = t.x + h;
                f.g = static_cast<const char *>(t.g) + h * int64_t(g_size);
                f.m = t.m + h;
                f.v = needs_v ? t.v + h : nullptr;
                f.numel = tail[size_t(i)];
                f.ext = int32_t(host_rest.size());
                TensorDesc r = d;
                r.numel = h;
                r.first_chunk = int32_t(host_rest_ids.size());
                r.n_chunks = int32_t((h + chunk - 1) / chunk);
                r.first_coarse = r.n_coarse = 0;
                r.first_tile = r.n_tiles = 0;
                for (int32_t k = 0; k < r.n_chunks; ++k)
                    host_rest_ids.push_back(f.ext);
                host_rest.push_back(r);
            }
            host_fused[size_t(i)] = f;
            first += nc;
            first_coarse += ncc;
        }
    }
    const int32_t n_tiles = int32_t(host_tiles.size());
    const int32_t n_rest = int32_t(host_rest.size());
    const int32_t n_rest_chunks = int32_t(host_rest_ids.size());
    std::vector<SegDesc> host_segs[3];
    std::vector<SegRange> host_ranges[3];
    {
        std::vector<std::pair<int32_t, int32_t>> fine, coarse_tc, rest;
        for (const TensorDesc &d : host_tensors) {
            fine.emplace_back(d.first_chunk, d.n_chunks);
            coarse_tc.emplace_back(d.first_coarse, d.n_coarse);
        }
        for (const TensorDesc &d : host_rest)
            rest.emplace_back(d.first_chunk, d.n_chunks);
        build_segments(fine, &host_segs[kSegFine], &host_ranges[kSegFine]);
        build_segments(coarse_tc, &host_segs[kSegCoarse], &host_ranges[kSegCoarse]);
        build_segments(rest, &host_segs[kSegRest], &host_ranges[kSegRest]);
    }
    size_t max_segs = 1;
    for (const auto &v : host_segs)
        max_segs = std::max(max_segs, v.size());

    lamb_plan *plan = new (std::nothrow) lamb_plan();
    if (!plan)
        return fail(LAMB_ENOMEM, "host allocation of the plan failed");
    plan->device = device;
    plan->cu_count = cu_count;
    plan->round = round;
    plan->tile_groups = groups;
    plan->spin_limit = spin_limit;
    auto round256 = [](size_t b) { return (b + 255) & ~size_t(255); };
    const size_t tensors_bytes = round256(sizeof(TensorDesc) * size_t(n_tensors));
    const size_t chunks_bytes = round256(sizeof(int32_t) * size_t(n_chunks));
    const size_t coarse_bytes = round256(sizeof(int32_t) * size_t(n_coarse));
    const size_t partial_bytes = round256(sizeof(Partial) * size_t(n_chunks));
    const size_t scale_bytes = round256(sizeof(float) * size_t(n_tensors));
    const size_t flag_bytes = 256;
    const size_t tiles_bytes = round256(sizeof(ChunkDesc) * size_t(n_tiles));
    const size_t slot_bytes = round256(sizeof(uint64_t) * 6 * size_t(n_tiles));
    const size_t ctl_bytes = 256;
    const size_t rest_bytes = round256(sizeof(TensorDesc) * size_t(n_rest));
    const size_t rest_chunk_bytes = round256(sizeof(int32_t) * size_t(n_rest_chunks));
    const size_t fused_bytes = round256(sizeof(TensorDesc) * size_t(n_tensors));
    const size_t ext_bytes = round256(sizeof(double) * (2 * size_t(n_rest) + 1));
    size_t seg_bytes[3], range_bytes[3];
    for (int k = 0; k < 3; ++k) {
        seg_bytes[k] = round256(sizeof(SegDesc) * host_segs[k].size());
        range_bytes[k] = round256(sizeof(SegRange) * host_ranges[k].size());
    }
    const size_t seg_partial_bytes = round256(sizeof(Partial) * max_segs);
    const size_t check_bytes = round256(sizeof(ChunkDesc) * host_check.size());
    err = hipMalloc(&plan->device_block,
                    tensors_bytes + chunks_bytes + coarse_bytes + partial_bytes + scale_bytes +
                        flag_bytes + tiles_bytes + slot_bytes + ctl_bytes + rest_bytes +
                        rest_chunk_bytes + fused_bytes + ext_bytes + seg_bytes[0] +
                        seg_bytes[1] + seg_bytes[2] +
                        range_bytes[0] + range_bytes[1] + range_bytes[2] + seg_partial_bytes +
                        check_bytes);
    if (err != hipSuccess) {
        delete plan;
        if (err == hipErrorOutOfMemory)
            return fail(LAMB_ENOMEM, "hipMalloc of plan buffers: %s", hipGetErrorString(err));
        return fail_hip(err, "hipMalloc");
    }
    char *base = static_cast<char *>(plan->device_block);
    plan->tensors = reinterpret_cast<TensorDesc *>(base);
    base += tensors_bytes;
    plan->chunk_ids = reinterpret_cast<int32_t *>(base);
    base += chunks_bytes;
    plan->coarse_ids = reinterpret_cast<int32_t *>(base);
    base += coarse_bytes;
    plan->partials = reinterpret_cast<Partial *>(base);  // sized for the fine table
    base += partial_bytes;
    plan->scale = reinterpret_cast<float *>(base);
    base += scale_bytes;
    plan->flags = reinterpret_cast<uint32_t *>(base);
    base += flag_bytes;
    plan->tiles = reinterpret_cast<ChunkDesc *>(base);
    base += tiles_bytes;
    plan->slots = reinterpret_cast<uint64_t *>(base);
    base += slot_bytes;
    plan->ctl = reinterpret_cast<uint32_t *>(base);
    base += ctl_bytes;
    plan->rest_tensors = reinterpret_cast<TensorDesc *>(base);
    base += rest_bytes;
    plan->rest_ids = reinterpret_cast<int32_t *>(base);
    base += rest_chunk_bytes;
    plan->fused_tensors = reinterpret_cast<TensorDesc *>(base);
    base += fused_bytes;
    plan->ext_totals = reinterpret_cast<double *>(base);
    base += ext_bytes;
    for (int k = 0; k < 3; ++k) {
        plan->segs[k] = reinterpret_cast<SegDesc *>(base);
        base += seg_bytes[k];
        plan->seg_ranges[k] = reinterpret_cast<SegRange *>(base);
        base += range_bytes[k];
        plan->n_segs[k] = int32_t(host_segs[k].size());
    }
    plan->seg_partials = reinterpret_cast<Partial *>(base);
    base += seg_partial_bytes;
    plan->check_chunks = reinterpret_cast<ChunkDesc *>(base);
    plan->n_check = int32_t(host_check.size());
    err = hipMemcpy(plan->tensors, host_tensors.data(), sizeof(TensorDesc) * size_t(n_tensors),
                    hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipMemcpy(plan->chunk_ids, ids_of(host_chunks).data(),
                        sizeof(int32_t) * size_t(n_chunks), hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipMemcpy(plan->coarse_ids, ids_of(host_coarse).data(),
                        sizeof(int32_t) * size_t(n_coarse), hipMemcpyHostToDevice);
    if (err == hipSuccess && n_tiles > 0)
        err = hipMemcpy(plan->tiles, host_tiles.data(), sizeof(ChunkDesc) * size_t(n_tiles),
                        hipMemcpyHostToDevice);
    if (err == hipSuccess && n_rest > 0)
        err = hipMemcpy(plan->rest_tensors, host_rest.data(), sizeof(TensorDesc) * size_t(n_rest),
                        hipMemcpyHostToDevice);
    if (err == hipSuccess && n_rest > 0)
        err = hipMemcpy(plan->rest_ids, host_rest_ids.data(),
                        sizeof(int32_t) * size_t(n_rest_chunks), hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipMemcpy(plan->fused_tensors, host_fused.data(),
                        sizeof(TensorDesc) * size_t(n_tensors), hipMemcpyHostToDevice);
    for (int k = 0; k < 3 && err == hipSuccess; ++k) {
        if (!host_segs[k].empty())
            err = hipMemcpy(plan->segs[k], host_segs[k].data(),
                            sizeof(SegDesc) * host_segs[k].size(), hipMemcpyHostToDevice);
        if (err == hipSuccess && !host_ranges[k].empty())
            err = hipMemcpy(plan->seg_ranges[k], host_ranges[k].data(),
                            sizeof(SegRange) * host_ranges[k].size(), hipMemcpyHostToDevice);
    }
    if (err == hipSuccess)
        err = hipMemcpy(plan->check_chunks, host_check.data(),
                        sizeof(ChunkDesc) * host_check.size(), hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipMemset(plan->flags, 0, flag_bytes);
    if (err == hipSuccess && slot_bytes > 0)
        err = hipMemset(plan->slots, 0xff, slot_bytes);  // every slot kEmptySlot
    if (err == hipSuccess)
        err = hipMemset(plan->ctl, 0, ctl_bytes);
    if (err == hipSuccess)
        err = hipDeviceSynchronize();
    if (err != hipSuccess) {
        (void)hipFree(plan->device_block);
        delete plan;
        return fail_hip(err, "hipMemcpy of plan tables");
    }
    // Occupancy of every single-pass kernel a step of this plan may pick, so
    // that a step makes no HIP query (it may be under graph capture).
    if (n_tiles > 0) {
        const Algo algos[3] = {kLamb, kNLamb, kNNLamb};
        const int n_algos = algo == LAMB_ALGO_LARS ? 1 : 3;
        for (int ai = 0; ai < n_algos && err == hipSuccess; ++ai) {
            for (int nk = 0; nk < 3 && err == hipSuccess; ++nk) {
                StepKind kind;
                kind.algo = algo == LAMB_ALGO_LARS ? kLars : algos[ai];
                kind.norm = static_cast<NormKind>(nk);
                kind.bf16_grad = g_dtype == LAMB_GRAD_BF16;
                kind.deferred = false;
                int per_cu = 0;
                err = fused_blocks_per_cu(kind, plan->tile_groups, &per_cu);
                plan->fused_per_cu[int(kind.algo)][kind.bf16_grad ? 1 : 0][nk] = per_cu;
            }
        }
        if (err != hipSuccess) {
            (void)hipFree(plan->device_block);
            delete plan;
            return fail_hip(err, "occupancy of the single-pass kernel");
        }
    }
    plan->algo = algo;
    plan->g_dtype = g_dtype;
    plan->n_tensors = n_tensors;
    plan->n_chunks = n_chunks;
    plan->n_coarse = n_coarse;
    plan->n_tiles = n_tiles;
    plan->n_rest = n_rest;
    plan->n_rest_chunks = n_rest_chunks;
    plan->host_tensors = std::move(host_tensors);
    plan->host_fused = std::move(host_fused);
    plan->host_rest = std::move(host_rest);
    plan->single_elems = std::move(tail);
    for (const BufferRange &r : ranges)
        plan->ranges.emplace_back(r.lo, r.hi);
    plan->chunk_elems = chunk;
    plan->coarse_elems = coarse;
    *out = plan;
    return LAMB_OK;
}

lamb_status lamb_plan_destroy(lamb_plan *plan) {
    if (!plan)
        return LAMB_OK;
    DeviceGuard guard(plan->device);
    release_events(plan);
    hipError_t err = hipFree(plan->device_block);
    if (plan->u_check) {
        const hipError_t e2 = hipFree(plan->u_check);
        if (err == hipSuccess)
            err = e2;
    }
    delete plan;
    if (err != hipSuccess)
        return fail_hip(err, "hipFree");
    return LAMB_OK;
}

lamb_status lamb_plan_info(const lamb_plan *plan, int32_t *n_tensors, int32_t *n_chunks,
                           int32_t *chunk_elems) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (n_tensors)
        *n_tensors = plan->n_tensors;
    if (n_chunks)
        *n_chunks = plan->n_chunks;
    if (chunk_elems)
        *chunk_elems = plan->chunk_elems;
    return LAMB_OK;
}

}  // extern "C"

namespace lamb_mi355x {

bool valid_beta(float beta) { return beta >= 0.0f && beta < 1.0f; }

// Host-side validation of one step's hyperparameters (all before any HIP
// call); `plan` may be null (a planless step).
lamb_status check_hparams(const lamb_plan *plan, const lamb_hparams *hp,
                          const int32_t *nonfinite_out) {
    if (!hp)
        return fail(LAMB_ENULL, "hparams must not be NULL");
    if (hp->reserved != 0)
        return fail(LAMB_EINVAL, "hparams.reserved must be 0");
    const int32_t variant = hp->variant;
    if (variant < LAMB_VARIANT_LAMB || variant > LAMB_VARIANT_LARS)
        return fail(LAMB_EINVAL, "unknown variant %d", variant);
    const bool lars = variant == LAMB_VARIANT_LARS;
    if (plan && lars != (plan->algo == LAMB_ALGO_LARS))
        return fail(LAMB_EPLAN, "%s needs a plan created for %s", lars ? "LARS" : "the LAMB family",
                    lars ? "LARS" : "LAMB");
    if (hp->norm < LAMB_NORM_L2 || hp->norm > LAMB_NORM_LINF)
        return fail(LAMB_EINVAL, "unknown norm %d", hp->norm);
    if (!valid_beta(hp->beta1))
        return fail(LAMB_EINVAL, "%s = %g outside [0, 1)", lars ? "momentum" : "beta1",
                    double(hp->beta1));
    if (!finite(hp->lr) || !finite(hp->weight_decay) || !finite(hp->grad_scale))
        return fail(LAMB_EINVAL, "lr, weight_decay and grad_scale must be finite");
    lamb_status st = check_phi_bounds(hp->gamma_l, hp->gamma_u);
    if (st != LAMB_OK)
        return st;
    if (hp->skip_nonfinite != 0 && hp->skip_nonfinite != 1)
        return fail(LAMB_EINVAL, "skip_nonfinite must be 0 or 1");
    if (nonfinite_out && !hp->skip_nonfinite)
        return fail(LAMB_EINVAL, "nonfinite_out needs skip_nonfinite = 1");
    if (lars) {
        if (!finite(hp->trust_coef))
            return fail(LAMB_EINVAL, "trust_coef must be finite");
        return LAMB_OK;
    }
    if (hp->step < 1)
        return fail(LAMB_EINVAL, "step = %lld, need >= 1", static_cast<long long>(hp->step));
    if (!valid_beta(hp->beta2))
        return fail(LAMB_EINVAL, "beta2 = %g outside [0, 1)", double(hp->beta2));
    if (!(hp->eps >= 0.0f) || !finite(hp->eps))
        return fail(LAMB_EINVAL, "eps = %g, need finite and >= 0", double(hp->eps));
    if (hp->bias_correction != 0 && hp->bias_correction != 1)
        return fail(LAMB_EINVAL, "bias_correction must be 0 or 1");
    if (variant != LAMB_VARIANT_LAMB && !hp->bias_correction)
        return fail(LAMB_EINVAL, "N-LAMB and NN-LAMB carry their own bias correction");
    return LAMB_OK;
}

// fp32 kernel scalars of a validated step. The LAMB family's correction
// coefficients are computed in double and rounded once.
StepArgs step_args(const lamb_hparams &hp) {
    StepArgs a;
    a.beta1 = hp.beta1;
    a.one_minus_beta1 = float(1.0 - double(hp.beta1));
    a.beta2 = hp.beta2;
    a.one_minus_beta2 = float(1.0 - double(hp.beta2));
    a.m_scale = a.v_scale = 1.0f;
    a.m_grad = a.v_grad = 0.0f;
    a.eps = hp.eps;
    a.weight_decay = hp.weight_decay;
    a.grad_scale = hp.grad_scale;
    a.spin_limit = kDefaultSpinLimit;
    const double b1 = hp.beta1, b2 = hp.beta2, t = double(hp.step);
    switch (hp.variant) {
    case LAMB_VARIANT_LAMB:
        // Algorithm 2: m_hat = m_t / (1 - beta1^t), v_hat = v_t / (1 - beta2^t)
        if (hp.bias_correction) {
            a.m_scale = float(1.0 / (1.0 - std::pow(b1, t)));
            a.v_scale = float(1.0 / (1.0 - std::pow(b2, t)));
        }
        break;
    case LAMB_VARIANT_NLAMB:
    case LAMB_VARIANT_NNLAMB:
        // Algorithms 3 and 4 with the constant sequence beta1^t = beta1,
        // whose running products are powers.
        a.m_scale = float(b1 / (1.0 - std::pow(b1, t + 1.0)));
        a.m_grad = float((1.0 - b1) / (1.0 - std::pow(b1, t)));
        if (hp.variant == LAMB_VARIANT_NNLAMB) {
            a.v_scale = float(b2 / (1.0 - std::pow(b2, t + 1.0)));
            a.v_grad = float((1.0 - b2) / (1.0 - std::pow(b2, t)));
        } else {
            a.v_scale = float(b2 / (1.0 - std::pow(b2, t)));
        }
        break;
    default:
        break;
    }
    return a;
}

// What a validated step launches.
StepKind step_kind(const lamb_hparams &hp, lamb_grad_dtype g_dtype) {
    StepKind kind;
    kind.algo = static_cast<Algo>(hp.variant);
    kind.norm = static_cast<NormKind>(hp.norm);
    kind.bf16_grad = g_dtype == LAMB_GRAD_BF16;
    kind.deferred = hp.skip_nonfinite != 0;
    return kind;
}

FinalizeArgs finalize_args(const lamb_hparams &hp) {
    const bool lars = hp.variant == LAMB_VARIANT_LARS;
    return FinalizeArgs{double(hp.lr), double(hp.gamma_l), double(hp.gamma_u),
                        lars ? double(hp.trust_coef) : 1.0};
}

}  // namespace lamb_mi355x

extern "C" {

lamb_status lamb_hparams_init(lamb_hparams *hp, int32_t variant) {
    if (!hp)
        return fail(LAMB_ENULL, "hparams must not be NULL");
    if (variant < LAMB_VARIANT_LAMB || variant > LAMB_VARIANT_LARS)
        return fail(LAMB_EINVAL, "unknown variant %d", variant);
    *hp = lamb_hparams{};
    hp->variant = variant;
    hp->norm = LAMB_NORM_L2;
    hp->step = 1;
    hp->lr = 1e-3f;
    hp->weight_decay = 0.01f;
    hp->gamma_l = 0.0f;
    hp->gamma_u = 10.0f;
    hp->trust_coef = 1.0f;
    hp->grad_scale = 1.0f;
    hp->bias_correction = 1;
    hp->skip_nonfinite = 0;
    switch (variant) {
    case LAMB_VARIANT_LAMB:  // Section 4 and Appendix H
        hp->beta1 = 0.9f;
        hp->beta2 = 0.999f;
        hp->eps = 1e-6f;
        break;
    case LAMB_VARIANT_NLAMB:  // Appendix D, after Nadam
    case LAMB_VARIANT_NNLAMB:
        hp->beta1 = 0.975f;
        hp->beta2 = 0.999f;
        hp->eps = 1e-8f;
        break;
    default:  // LARS: heavy-ball momentum
        hp->beta1 = 0.9f;
        hp->beta2 = 0.0f;
        hp->eps = 0.0f;
        break;
    }
    return LAMB_OK;
}

lamb_status lamb_step_ex(lamb_plan *plan, const lamb_hparams *hp, void *stream,
                         double *ratio_out, double *norms_out, int32_t *nonfinite_out) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    lamb_status st = check_hparams(plan, hp, nonfinite_out);
    if (st != LAMB_OK)
        return st;
    const StepKind kind = step_kind(*hp, plan->g_dtype);
    StepArgs a = step_args(*hp);
    a.spin_limit = plan->spin_limit;
    const FinalizeArgs f = finalize_args(*hp);
    // On LAMB_PATH_AUTO the single pass serves every layer of at most one
    // round of tiles and the tails of larger ones, whose heads take a moment
    // pass and a totals kernel before it and an apply pass after it (the
    // single pass adds the heads' totals into those layers' norms and writes
    // their scales). LAMB_PATH_TWO_PASS runs everything on the two-pass
    // kernels. A skip_nonfinite step on the single pass first takes its
    // verdict with a read-only check of g; the kernels before the single pass
    // obey the epoch's verdict word, the apply pass after it a copy the totals
    // kernel takes (the single pass rewrites the epoch's words as it ends).
    const bool single = plan->path == LAMB_PATH_AUTO && plan->n_tiles > 0;
    const bool checked = single && kind.deferred;
    const bool heads = single && plan->n_rest > 0;
    StepKind direct = kind;
    direct.deferred = false;

    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    int32_t grid = 0;
    if (single) {
        const int per_cu =
            plan->fused_per_cu[int(kind.algo)][kind.bf16_grad ? 1 : 0][int(kind.norm)];
        // The tile list was packed in rounds of at most kFusedBlocksPerCu * CUs
        // entries; the grid is one round, so it must all be resident at once.
        if (per_cu < kFusedBlocksPerCu)
            return fail(LAMB_EHIP,
                        "single-pass kernel keeps %d workgroups per CU resident, needs %d", per_cu,
                        kFusedBlocksPerCu);
        grid = std::min(plan->n_tiles, plan->round);
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    begin_timing(plan, s);
    hipError_t err = hipSuccess;
    if (checked) {
        err = launch_finite(kind.bf16_grad, plan->tensors, plan->check_chunks, plan->n_check,
                            plan->flags, plan->ctl, a.grad_scale, s);
        if (err != hipSuccess)
            return fail_hip(err, "launching the finiteness check");
        mark(plan, kTimedCheck, s);
    }
    if (single) {
        if (heads) {
            err = launch_moments(direct, plan->rest_tensors, plan->rest_ids, plan->chunk_elems,
                                 plan->partials, plan->n_rest_chunks,
                                 two_pass_threads(plan->chunk_elems), plan->flags, plan->ctl,
                                 checked ? kGuardEpoch : kGuardNone, a, s);
            if (err != hipSuccess)
                return fail_hip(err, "launching the moment kernel");
            mark(plan, kTimedMoments, s);
            err = launch_totals(direct.norm, plan->partials, plan->segs[kSegRest],
                                plan->n_segs[kSegRest], plan->seg_ranges[kSegRest], plan->n_rest,
                                plan->seg_partials, plan->ext_totals, plan->flags, plan->ctl,
                                checked ? kVerdictCopy : kVerdictZero, s);
            if (err != hipSuccess)
                return fail_hip(err, "launching the totals kernel");
            mark(plan, kTimedFinalize, s);
        }
        err = gated_fused_launch(plan->device, s, direct, plan, grid, checked,
                                 checked ? nonfinite_out : nullptr, a, f, ratio_out, norms_out);
        if (err != hipSuccess)
            return fail_hip(err, "launching the single-pass kernel");
        mark(plan, kTimedSingle, s);
        plan->u_check_chunks = 0;
        if (heads) {
            err = launch_apply(direct, plan->rest_tensors, plan->rest_ids, plan->chunk_elems,
                               plan->scale, plan->n_rest_chunks,
                               two_pass_threads(plan->chunk_elems), plan->flags, plan->ctl,
                               checked ? kGuardCopy : kGuardNone, nullptr, plan->u_check, a, s);
            if (err != hipSuccess)
                return fail_hip(err, "launching the apply kernel");
            mark(plan, kTimedApply, s);
            plan->u_check_chunks = plan->u_check ? plan->n_rest_chunks : 0;
        }
    } else {
        // Deferred moment passes only read, and use the coarse chunk table.
        const int32_t *moment_ids = kind.deferred ? plan->coarse_ids : plan->chunk_ids;
        const int32_t n_moment_chunks = kind.deferred ? plan->n_coarse : plan->n_chunks;
        const int32_t moment_elems = kind.deferred ? plan->coarse_elems : plan->chunk_elems;
        err = launch_moments(kind, plan->tensors, moment_ids, moment_elems, plan->partials,
                             n_moment_chunks, two_pass_threads(moment_elems), plan->flags,
                             plan->ctl, kGuardNone, a, s);
        if (err != hipSuccess)
            return fail_hip(err, "launching the moment kernel");
        mark(plan, kTimedMoments, s);
        const int seg = kind.deferred ? kSegCoarse : kSegFine;
        err = launch_finalize(kind.norm, plan->tensors, plan->n_tensors, plan->partials,
                              plan->segs[seg], plan->n_segs[seg], plan->seg_ranges[seg],
                              plan->seg_partials, f, plan->scale, ratio_out, norms_out,
                              kind.deferred ? plan->flags : nullptr, s);
        if (err != hipSuccess)
            return fail_hip(err, "launching the finalize kernel");
        mark(plan, kTimedFinalize, s);
        Partial *check = kind.deferred ? nullptr : plan->u_check;
        err = launch_apply(kind, plan->tensors, plan->chunk_ids, plan->chunk_elems, plan->scale,
                           plan->n_chunks, two_pass_threads(plan->chunk_elems), plan->flags,
                           plan->ctl, kGuardNone, kind.deferred ? nonfinite_out : nullptr, check,
                           a, s);
        if (err != hipSuccess)
            return fail_hip(err, "launching the apply kernel");
        mark(plan, kTimedApply, s);
        plan->u_check_chunks = check ? plan->n_chunks : 0;
    }
    end_timing(plan);
    return LAMB_OK;
}

lamb_status lamb_step(lamb_plan *plan, float lr, float beta1, float beta2, float eps,
                      float weight_decay, float gamma_l, float gamma_u, int64_t step,
                      int32_t bias_correction, void *stream, double *ratio_out,
                      double *norms_out) {
    lamb_hparams hp;
    lamb_hparams_init(&hp, LAMB_VARIANT_LAMB);
    hp.lr = lr;
    hp.beta1 = beta1;
    hp.beta2 = beta2;
    hp.eps = eps;
    hp.weight_decay = weight_decay;
    hp.gamma_l = gamma_l;
    hp.gamma_u = gamma_u;
    hp.step = step;
    hp.bias_correction = bias_correction;
    return lamb_step_ex(plan, &hp, stream, ratio_out, norms_out, nullptr);
}

lamb_status nlamb_step(lamb_plan *plan, float lr, float beta1, float beta2, float eps,
                       float weight_decay, float gamma_l, float gamma_u, int64_t step,
                       int32_t nesterov_v, void *stream, double *ratio_out,
                       double *norms_out) {
    if (nesterov_v != 0 && nesterov_v != 1)
        return fail(LAMB_EINVAL, "nesterov_v must be 0 or 1");
    lamb_hparams hp;
    lamb_hparams_init(&hp, nesterov_v ? LAMB_VARIANT_NNLAMB : LAMB_VARIANT_NLAMB);
    hp.lr = lr;
    hp.beta1 = beta1;
    hp.beta2 = beta2;
    hp.eps = eps;
    hp.weight_decay = weight_decay;
    hp.gamma_l = gamma_l;
    hp.gamma_u = gamma_u;
    hp.step = step;
    return lamb_step_ex(plan, &hp, stream, ratio_out, norms_out, nullptr);
}

lamb_status lars_step(lamb_plan *plan, float lr, float momentum, float weight_decay,
                      float gamma_l, float gamma_u, float trust_coef, void *stream,
                      double *ratio_out, double *norms_out) {
    lamb_hparams hp;
    lamb_hparams_init(&hp, LAMB_VARIANT_LARS);
    hp.lr = lr;
    hp.beta1 = momentum;
    hp.weight_decay = weight_decay;
    hp.gamma_l = gamma_l;
    hp.gamma_u = gamma_u;
    hp.trust_coef = trust_coef;
    return lamb_step_ex(plan, &hp, stream, ratio_out, norms_out, nullptr);
}

lamb_status lamb_plan_set_bf16_copies(lamb_plan *plan, void *const *copies) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    std::vector<TensorDesc> next = plan->host_tensors;
    std::vector<std::pair<uintptr_t, uintptr_t>> mine;
    for (int32_t i = 0; i < plan->n_tensors; ++i) {
        uint16_t *c = copies ? static_cast<uint16_t *>(copies[i]) : nullptr;
        next[size_t(i)].x_copy = c;
        if (!c)
            continue;
        if (!aligned16(c))
            return fail(LAMB_EALIGN, "copy %d must be 16-byte aligned", i);
        const uintptr_t lo = reinterpret_cast<uintptr_t>(c);
        mine.emplace_back(lo, lo + uintptr_t(next[size_t(i)].numel) * 2u);
    }
    // Copies may overlap neither each other nor any buffer of the table.
    std::vector<std::pair<uintptr_t, uintptr_t>> all = plan->ranges;
    all.insert(all.end(), mine.begin(), mine.end());
    std::sort(all.begin(), all.end());
    for (size_t k = 1; k < all.size(); ++k)
        if (all[k].first < all[k - 1].second)
            return fail(LAMB_EOVERLAP, "a bf16 copy overlaps another buffer of the plan");
    std::vector<TensorDesc> next_rest = plan->host_rest;
    for (TensorDesc &r : next_rest)
        r.x_copy = next[size_t(r.out_index)].x_copy;
    // the single pass's table holds the tails of split layers at an offset
    std::vector<TensorDesc> next_fused = plan->host_fused;
    for (int32_t i = 0; i < plan->n_tensors; ++i) {
        uint16_t *c = next[size_t(i)].x_copy;
        const int64_t head = next[size_t(i)].numel - next_fused[size_t(i)].numel;
        next_fused[size_t(i)].x_copy = c ? c + head : nullptr;
    }
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipError_t err = hipMemcpy(plan->tensors, next.data(),
                               sizeof(TensorDesc) * size_t(plan->n_tensors), hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipMemcpy(plan->fused_tensors, next_fused.data(),
                        sizeof(TensorDesc) * size_t(plan->n_tensors), hipMemcpyHostToDevice);
    if (err == hipSuccess && plan->n_rest > 0)
        err = hipMemcpy(plan->rest_tensors, next_rest.data(),
                        sizeof(TensorDesc) * size_t(plan->n_rest), hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipDeviceSynchronize();
    if (err != hipSuccess)
        return fail_hip(err, "hipMemcpy of the tensor table");
    plan->host_tensors = std::move(next);
    plan->host_fused = std::move(next_fused);
    plan->host_rest = std::move(next_rest);
    return LAMB_OK;
}

lamb_status lamb_plan_set_path(lamb_plan *plan, int32_t path) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (path != LAMB_PATH_AUTO && path != LAMB_PATH_TWO_PASS)
        return fail(LAMB_EINVAL, "unknown path %d", path);
    plan->path = static_cast<lamb_path>(path);
    return LAMB_OK;
}

lamb_status lamb_plan_tiles(const lamb_plan *plan, int32_t *tiles_per_tensor, int32_t *n_tiles,
                            int32_t *tile_groups, int64_t *single_elems) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (tiles_per_tensor)
        for (int32_t i = 0; i < plan->n_tensors; ++i)
            tiles_per_tensor[i] = plan->host_fused[size_t(i)].n_tiles;
    if (single_elems)
        for (int32_t i = 0; i < plan->n_tensors; ++i)
            single_elems[i] = plan->single_elems[size_t(i)];
    if (n_tiles)
        *n_tiles = plan->n_tiles;
    if (tile_groups)
        *tile_groups = plan->tile_groups;
    return LAMB_OK;
}

lamb_status lamb_plan_check(lamb_plan *plan, void *stream) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t *host = nullptr;
    hipError_t err = hipHostMalloc(reinterpret_cast<void **>(&host), 4 * sizeof(uint32_t), 0);
    if (err != hipSuccess)
        return fail_hip(err, "hipHostMalloc");
    err = hipMemcpyAsync(host, plan->ctl, 4 * sizeof(uint32_t), hipMemcpyDeviceToHost, s);
    if (err == hipSuccess)
        err = hipStreamSynchronize(s);
    const uint32_t fault = host[kCtlFault];
    (void)hipHostFree(host);
    if (err != hipSuccess)
        return fail_hip(err, "reading the plan's synchronisation words");
    if (fault)
        return fail(LAMB_ESYNC, "a single-pass step of this plan abandoned a wait; the plan's "
                                "single pass is disabled and the state of that step is undefined");
    return LAMB_OK;
}

lamb_status lamb_lr_at(const lamb_lr_stage *stages, int32_t n_stages, int64_t step,
                       double *lr_out) {
    if (!stages || !lr_out)
        return fail(LAMB_ENULL, "stages and lr_out must not be NULL");
    if (n_stages < 1 || step < 1)
        return fail(LAMB_EINVAL, "need n_stages >= 1 and step >= 1");
    for (int32_t k = 0; k < n_stages; ++k) {
        const lamb_lr_stage &s = stages[k];
        if (s.steps < 1 || s.warmup_steps < 0 || s.warmup_steps > s.steps ||
            !(s.peak_lr >= 0.0) || !std::isfinite(s.peak_lr) || !(s.power >= 0.0) ||
            !std::isfinite(s.power))
            return fail(LAMB_EINVAL, "stage %d out of range", k);
    }
    int64_t tau = step - 1;  // steps already taken, counted from the first stage
    for (int32_t k = 0; k < n_stages; ++k) {
        const lamb_lr_stage &s = stages[k];
        if (tau < s.steps) {
            if (tau < s.warmup_steps)
                *lr_out = s.peak_lr * double(tau + 1) / double(s.warmup_steps);
            else
                *lr_out = s.peak_lr * std::pow(1.0 - double(tau) / double(s.steps), s.power);
            return LAMB_OK;
        }
        tau -= s.steps;
    }
    *lr_out = 0.0;
    return LAMB_OK;
}

lamb_status lamb_sqrt_scaled_lr(double base_lr, int64_t base_batch, int64_t batch,
                                double *lr_out) {
    if (!lr_out)
        return fail(LAMB_ENULL, "lr_out must not be NULL");
    if (base_batch < 1 || batch < 1 || !(base_lr >= 0.0) || !std::isfinite(base_lr))
        return fail(LAMB_EINVAL, "need positive batch sizes and a finite base_lr >= 0");
    *lr_out = base_lr * std::sqrt(double(batch) / double(base_batch));
    return LAMB_OK;
}

lamb_status lamb_plan_set_timing(lamb_plan *plan, int32_t max_steps, int32_t every) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (max_steps < 0 || max_steps > (1 << 20))
        return fail(LAMB_EINVAL, "max_steps = %d outside [0, 2^20]", max_steps);
    if (every < 1)
        return fail(LAMB_EINVAL, "every = %d, need >= 1", every);
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    release_events(plan);
    if (max_steps == 0)
        return LAMB_OK;
    plan->events.assign(size_t(max_steps) * kEvents, nullptr);
    plan->timing_kinds.assign(size_t(max_steps) * (kEvents - 1), uint8_t(0));
    plan->timing_count.assign(size_t(max_steps), uint8_t(0));
    for (size_t k = 0; k < plan->events.size(); ++k) {
        // timing only: no system-scope fence, which would perturb the step
        hipError_t err = hipEventCreateWithFlags(&plan->events[k], hipEventDisableSystemFence);
        if (err != hipSuccess) {
            plan->events.resize(k);
            release_events(plan);
            return fail_hip(err, "hipEventCreate");
        }
    }
    plan->timing_capacity = max_steps;
    plan->timing_used = 0;
    plan->timing_every = every;
    plan->timing_seen = 0;
    return LAMB_OK;
}

lamb_status lamb_plan_timing(lamb_plan *plan, double *kernel_ms, int64_t *steps) {
    if (!plan || !kernel_ms || !steps)
        return fail(LAMB_ENULL, "plan, kernel_ms and steps must not be NULL");
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    for (int j = 0; j < kTimedKinds; ++j)
        kernel_ms[j] = 0.0;
    for (int32_t k = 0; k < plan->timing_used; ++k) {
        hipEvent_t *e = &plan->events[size_t(k) * kEvents];
        const int n = plan->timing_count[size_t(k)];
        hipError_t err = hipEventSynchronize(e[n]);
        if (err != hipSuccess)
            return fail_hip(err, "hipEventSynchronize");
        for (int j = 0; j < n; ++j) {
            float ms = 0.0f;
            err = hipEventElapsedTime(&ms, e[j], e[j + 1]);
            if (err != hipSuccess)
                return fail_hip(err, "hipEventElapsedTime");
            kernel_ms[plan->timing_kinds[size_t(k) * (kEvents - 1) + size_t(j)]] += ms;
        }
    }
    *steps = plan->timing_used;
    plan->timing_used = 0;
    return LAMB_OK;
}

lamb_status lamb_step_partials(lamb_plan *plan, const lamb_hparams *hp, void *stream,
                               double *totals) {
    if (!plan || !totals)
        return fail(LAMB_ENULL, "plan and totals must not be NULL");
    lamb_status st = check_hparams(plan, hp, nullptr);
    if (st != LAMB_OK)
        return st;
    const StepKind kind = step_kind(*hp, plan->g_dtype);
    StepArgs a = step_args(*hp);
    a.spin_limit = plan->spin_limit;
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    // Every layer takes the moment pass: a deferred one (read only, coarse
    // chunks) when the step may be skipped, since the verdict is only known
    // once the shards' totals are combined.
    const int32_t *ids = kind.deferred ? plan->coarse_ids : plan->chunk_ids;
    const int32_t n = kind.deferred ? plan->n_coarse : plan->n_chunks;
    const int32_t elems = kind.deferred ? plan->coarse_elems : plan->chunk_elems;
    hipError_t err = launch_moments(kind, plan->tensors, ids, elems, plan->partials, n,
                                    two_pass_threads(elems), plan->flags, plan->ctl, kGuardNone,
                                    a, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the moment kernel");
    const int seg = kind.deferred ? kSegCoarse : kSegFine;
    err = launch_totals(kind.norm, plan->partials, plan->segs[seg], plan->n_segs[seg],
                        plan->seg_ranges[seg], plan->n_tensors, plan->seg_partials, totals,
                        plan->flags, plan->ctl, kind.deferred ? kVerdictMove : kVerdictZero, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the totals kernel");
    plan->u_check_chunks = 0;
    return LAMB_OK;
}

lamb_status lamb_step_finish(lamb_plan *plan, const lamb_hparams *hp, void *stream,
                             const double *totals, double *ratio_out, double *norms_out,
                             int32_t *nonfinite_out) {
    if (!plan || !totals)
        return fail(LAMB_ENULL, "plan and totals must not be NULL");
    lamb_status st = check_hparams(plan, hp, nonfinite_out);
    if (st != LAMB_OK)
        return st;
    const StepKind kind = step_kind(*hp, plan->g_dtype);
    StepArgs a = step_args(*hp);
    a.spin_limit = plan->spin_limit;
    const FinalizeArgs f = finalize_args(*hp);
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t err = launch_scale(kind.norm, totals, plan->n_tensors, f, plan->scale, ratio_out,
                                  norms_out, plan->flags, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the scale kernel");
    Partial *check = kind.deferred ? nullptr : plan->u_check;
    err = launch_apply(kind, plan->tensors, plan->chunk_ids, plan->chunk_elems, plan->scale,
                       plan->n_chunks, two_pass_threads(plan->chunk_elems), plan->flags,
                       plan->ctl, kGuardNone, kind.deferred ? nonfinite_out : nullptr, check, a,
                       s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the apply kernel");
    plan->u_check_chunks = check ? plan->n_chunks : 0;
    return LAMB_OK;
}

lamb_status lamb_plan_set_u_check(lamb_plan *plan, int32_t enable) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (enable != 0 && enable != 1)
        return fail(LAMB_EINVAL, "enable must be 0 or 1");
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    if (!enable) {
        hipError_t err = plan->u_check ? hipFree(plan->u_check) : hipSuccess;
        plan->u_check = nullptr;
        plan->u_check_chunks = 0;
        if (err != hipSuccess)
            return fail_hip(err, "hipFree");
        return LAMB_OK;
    }
    if (plan->u_check)
        return LAMB_OK;
    void *p = nullptr;
    hipError_t err = hipMalloc(&p, sizeof(Partial) * size_t(plan->n_chunks));
    if (err != hipSuccess)
        return err == hipErrorOutOfMemory ? fail(LAMB_ENOMEM, "hipMalloc of the check buffer")
                                          : fail_hip(err, "hipMalloc");
    plan->u_check = static_cast<Partial *>(p);
    plan->u_check_chunks = 0;
    return LAMB_OK;
}

lamb_status lamb_plan_u_partials(lamb_plan *plan, void *stream, int32_t capacity,
                                 double *moment_out, double *apply_out, int32_t *n_out) {
    if (!plan || !n_out)
        return fail(LAMB_ENULL, "plan and n_out must not be NULL");
    const int32_t n = plan->u_check ? plan->u_check_chunks : 0;
    *n_out = n;
    if (n == 0)
        return LAMB_OK;
    if (capacity < n)
        return fail(LAMB_EINVAL, "capacity %d < %d chunks", capacity, n);
    if (!moment_out || !apply_out)
        return fail(LAMB_ENULL, "moment_out and apply_out must not be NULL");
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t bytes = sizeof(Partial) * size_t(n);
    hipError_t err = hipMemcpyAsync(moment_out, plan->partials, bytes, hipMemcpyDeviceToHost, s);
    if (err == hipSuccess)
        err = hipMemcpyAsync(apply_out, plan->u_check, bytes, hipMemcpyDeviceToHost, s);
    if (err == hipSuccess)
        err = hipStreamSynchronize(s);
    if (err != hipSuccess)
        return fail_hip(err, "copying the partial norms");
    return LAMB_OK;
}

lamb_status lamb_plan_set_trace(lamb_plan *plan, uint64_t *trace) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (trace && (reinterpret_cast<uintptr_t>(trace) & 7u) != 0)
        return fail(LAMB_EALIGN, "the trace buffer must be 8-byte aligned");
    plan->trace = trace;
    return LAMB_OK;
}

}  // extern "C"
