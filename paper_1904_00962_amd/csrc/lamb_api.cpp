// Host side of the C ABI declared in include/lamb_mi355x.h: argument
// validation, the chunk table (Section 2's layer blocks cut into work
// chunks), plan buffers, per-step scalars and kernel launches.

#include "lamb_mi355x.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "lamb_internal.h"

using namespace lamb_mi355x;

struct lamb_plan {
    int device = 0;
    lamb_algo algo = LAMB_ALGO_LAMB;
    lamb_grad_dtype g_dtype = LAMB_GRAD_F32;
    int32_t n_tensors = 0;
    int32_t n_chunks = 0;
    int32_t chunk_elems = 0;
    void *device_block = nullptr;  // one allocation holding the four buffers below
    TensorDesc *tensors = nullptr;
    ChunkDesc *chunks = nullptr;
    Partial *partials = nullptr;
    float *scale = nullptr;
    // timing hooks: 4 events per recorded step
    std::vector<hipEvent_t> events;
    int32_t timing_capacity = 0;
    int32_t timing_used = 0;
};

namespace {

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

constexpr int64_t kMaxChunkElems = int64_t(1) << 30;

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

lamb_status check_beta(float beta, const char *name) {
    if (!(beta >= 0.0f && beta < 1.0f))
        return fail(LAMB_EINVAL, "%s = %g outside [0, 1)", name, double(beta));
    return LAMB_OK;
}

void record(lamb_plan *plan, int slot, hipStream_t stream) {
    if (plan->timing_used < plan->timing_capacity)
        (void)hipEventRecord(plan->events[size_t(plan->timing_used) * 4 + slot], stream);
}

void release_events(lamb_plan *plan) {
    for (hipEvent_t e : plan->events)
        (void)hipEventDestroy(e);
    plan->events.clear();
    plan->timing_capacity = 0;
    plan->timing_used = 0;
}

}  // namespace

extern "C" {

const char *lamb_status_str(lamb_status status) {
    switch (status) {
    case LAMB_OK: return "ok";
    case LAMB_EINVAL: return "invalid argument";
    case LAMB_ENULL: return "null pointer";
    case LAMB_EALIGN: return "tensor not 16-byte aligned";
    case LAMB_EOVERLAP: return "tensor buffers overlap";
    case LAMB_EHIP: return "HIP runtime error";
    case LAMB_ENOMEM: return "out of memory";
    case LAMB_EPLAN: return "plan built for the other algorithm";
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
    for (int32_t i = 0; i < n_tensors; ++i)
        if (numel[i] < 1)
            return fail(LAMB_EINVAL, "tensor %d has numel %lld, need >= 1", i,
                        static_cast<long long>(numel[i]));
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

lamb_status lamb_plan_create(const lamb_tensor *tensors, int32_t n_tensors,
                             lamb_grad_dtype g_dtype, lamb_algo algo, int32_t chunk_elems,
                             lamb_plan **out) {
    if (!out)
        return fail(LAMB_ENULL, "out must not be NULL");
    *out = nullptr;
    if (!tensors)
        return fail(LAMB_ENULL, "tensors must not be NULL");
    if (n_tensors < 1)
        return fail(LAMB_EINVAL, "n_tensors = %d, need >= 1", n_tensors);
    if (g_dtype != LAMB_GRAD_F32 && g_dtype != LAMB_GRAD_BF16)
        return fail(LAMB_EINVAL, "unknown gradient dtype %d", int(g_dtype));
    if (algo != LAMB_ALGO_LAMB && algo != LAMB_ALGO_LARS)
        return fail(LAMB_EINVAL, "unknown algorithm %d", int(algo));
    int32_t chunk = 0;
    lamb_status st = resolve_chunk_elems(chunk_elems, &chunk);
    if (st != LAMB_OK)
        return st;

    const bool needs_v = algo == LAMB_ALGO_LAMB;
    const size_t g_size = g_dtype == LAMB_GRAD_BF16 ? 2 : 4;
    struct Range {
        uintptr_t lo, hi;
        int32_t tensor;
        const char *what;
    };
    std::vector<Range> ranges;
    std::vector<int64_t> numel(size_t(n_tensors), 0);
    ranges.reserve(size_t(n_tensors) * 4);
    for (int32_t i = 0; i < n_tensors; ++i) {
        const lamb_tensor &t = tensors[i];
        if (!t.x || !t.g || !t.m || (needs_v && !t.v))
            return fail(LAMB_ENULL, "tensor %d: x, g, m%s must not be NULL", i,
                        needs_v ? ", v" : "");
        if (t.numel < 1)
            return fail(LAMB_EINVAL, "tensor %d: numel %lld, need >= 1", i,
                        static_cast<long long>(t.numel));
        if (t.numel > (int64_t(1) << 40))
            return fail(LAMB_EINVAL, "tensor %d: numel %lld too large", i,
                        static_cast<long long>(t.numel));
        if (t.wd != 0 && t.wd != 1)
            return fail(LAMB_EINVAL, "tensor %d: wd must be 0 or 1", i);
        if (t.reserved != 0)
            return fail(LAMB_EINVAL, "tensor %d: reserved field must be 0", i);
        if (!aligned16(t.x) || !aligned16(t.g) || !aligned16(t.m) || (needs_v && !aligned16(t.v)))
            return fail(LAMB_EALIGN, "tensor %d: every buffer must be 16-byte aligned", i);
        numel[size_t(i)] = t.numel;
        const uintptr_t f32_bytes = uintptr_t(t.numel) * 4u;
        ranges.push_back({reinterpret_cast<uintptr_t>(t.x), reinterpret_cast<uintptr_t>(t.x) + f32_bytes, i, "x"});
        ranges.push_back({reinterpret_cast<uintptr_t>(t.g),
                          reinterpret_cast<uintptr_t>(t.g) + uintptr_t(t.numel) * g_size, i, "g"});
        ranges.push_back({reinterpret_cast<uintptr_t>(t.m), reinterpret_cast<uintptr_t>(t.m) + f32_bytes, i, "m"});
        if (needs_v)
            ranges.push_back({reinterpret_cast<uintptr_t>(t.v), reinterpret_cast<uintptr_t>(t.v) + f32_bytes, i, "v"});
    }
    std::sort(ranges.begin(), ranges.end(),
              [](const Range &a, const Range &b) { return a.lo < b.lo; });
    for (size_t k = 1; k < ranges.size(); ++k)
        if (ranges[k].lo < ranges[k - 1].hi)
            return fail(LAMB_EOVERLAP, "tensor %d %s overlaps tensor %d %s", ranges[k].tensor,
                        ranges[k].what, ranges[k - 1].tensor, ranges[k - 1].what);

    const int64_t total = count_chunks(numel.data(), n_tensors, chunk);
    if (total < 0)
        return fail(LAMB_EINVAL, "more than 2^31-1 chunks; raise chunk_elems");
    const int32_t n_chunks = int32_t(total);

    // Host images of the tables.
    std::vector<TensorDesc> host_tensors(static_cast<size_t>(n_tensors));
    std::vector<ChunkDesc> host_chunks(static_cast<size_t>(n_chunks));
    {
        std::vector<int32_t> ct(static_cast<size_t>(n_chunks)), cl(static_cast<size_t>(n_chunks));
        std::vector<int64_t> cs(static_cast<size_t>(n_chunks));
        int32_t count = 0;
        st = lamb_chunk_table(numel.data(), n_tensors, chunk, n_chunks, ct.data(), cs.data(),
                              cl.data(), &count);
        if (st != LAMB_OK)
            return st;
        for (int32_t k = 0; k < n_chunks; ++k)
            host_chunks[size_t(k)] = ChunkDesc{ct[size_t(k)], cl[size_t(k)], cs[size_t(k)]};
        int32_t first = 0;
        for (int32_t i = 0; i < n_tensors; ++i) {
            const lamb_tensor &t = tensors[i];
            const int32_t nc = int32_t((t.numel + chunk - 1) / chunk);
            host_tensors[size_t(i)] = TensorDesc{t.x, t.g, t.m, needs_v ? t.v : nullptr, t.numel,
                                                 t.wd, first, nc, 0, 0};
            first += nc;
        }
    }

    lamb_plan *plan = new (std::nothrow) lamb_plan();
    if (!plan)
        return fail(LAMB_ENOMEM, "host allocation of the plan failed");
    hipError_t err = hipGetDevice(&plan->device);
    if (err != hipSuccess) {
        delete plan;
        return fail_hip(err, "hipGetDevice");
    }
    auto round256 = [](size_t b) { return (b + 255) & ~size_t(255); };
    const size_t tensors_bytes = round256(sizeof(TensorDesc) * size_t(n_tensors));
    const size_t chunks_bytes = round256(sizeof(ChunkDesc) * size_t(n_chunks));
    const size_t partial_bytes = round256(sizeof(Partial) * size_t(n_chunks));
    const size_t scale_bytes = round256(sizeof(float) * size_t(n_tensors));
    err = hipMalloc(&plan->device_block, tensors_bytes + chunks_bytes + partial_bytes + scale_bytes);
    if (err != hipSuccess) {
        delete plan;
        if (err == hipErrorOutOfMemory)
            return fail(LAMB_ENOMEM, "hipMalloc of plan buffers: %s", hipGetErrorString(err));
        return fail_hip(err, "hipMalloc");
    }
    char *base = static_cast<char *>(plan->device_block);
    plan->tensors = reinterpret_cast<TensorDesc *>(base);
    plan->chunks = reinterpret_cast<ChunkDesc *>(base + tensors_bytes);
    plan->partials = reinterpret_cast<Partial *>(base + tensors_bytes + chunks_bytes);
    plan->scale = reinterpret_cast<float *>(base + tensors_bytes + chunks_bytes + partial_bytes);
    err = hipMemcpy(plan->tensors, host_tensors.data(), sizeof(TensorDesc) * size_t(n_tensors),
                    hipMemcpyHostToDevice);
    if (err == hipSuccess)
        err = hipMemcpy(plan->chunks, host_chunks.data(), sizeof(ChunkDesc) * size_t(n_chunks),
                        hipMemcpyHostToDevice);
    if (err != hipSuccess) {
        (void)hipFree(plan->device_block);
        delete plan;
        return fail_hip(err, "hipMemcpy of plan tables");
    }
    plan->algo = algo;
    plan->g_dtype = g_dtype;
    plan->n_tensors = n_tensors;
    plan->n_chunks = n_chunks;
    plan->chunk_elems = chunk;
    *out = plan;
    return LAMB_OK;
}

lamb_status lamb_plan_destroy(lamb_plan *plan) {
    if (!plan)
        return LAMB_OK;
    DeviceGuard guard(plan->device);
    release_events(plan);
    hipError_t err = hipFree(plan->device_block);
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

namespace {

// Scalar checks shared by the LAMB family (Algorithms 2, 3 and 4).
lamb_status check_lamb_scalars(const lamb_plan *plan, float lr, float beta1, float beta2,
                               float eps, float weight_decay, float gamma_l, float gamma_u,
                               int64_t step) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (plan->algo != LAMB_ALGO_LAMB)
        return fail(LAMB_EPLAN, "the LAMB family needs a plan created for LAMB");
    if (step < 1)
        return fail(LAMB_EINVAL, "step = %lld, need >= 1", static_cast<long long>(step));
    lamb_status st = check_beta(beta1, "beta1");
    if (st == LAMB_OK)
        st = check_beta(beta2, "beta2");
    if (st != LAMB_OK)
        return st;
    if (!(eps >= 0.0f) || !finite(eps))
        return fail(LAMB_EINVAL, "eps = %g, need finite and >= 0", double(eps));
    if (!finite(lr) || !finite(weight_decay))
        return fail(LAMB_EINVAL, "lr and weight_decay must be finite");
    return check_phi_bounds(gamma_l, gamma_u);
}

LambArgs lamb_args(float beta1, float beta2, float eps, float weight_decay) {
    LambArgs a;
    a.beta1 = beta1;
    a.one_minus_beta1 = float(1.0 - double(beta1));
    a.beta2 = beta2;
    a.one_minus_beta2 = float(1.0 - double(beta2));
    a.m_scale = a.v_scale = 1.0f;
    a.m_grad = a.v_grad = 0.0f;
    a.eps = eps;
    a.weight_decay = weight_decay;
    return a;
}

// Enqueue moment pass, finalize and apply pass of the LAMB family.
lamb_status launch_lamb_family(lamb_plan *plan, LambVariant variant, const LambArgs &a,
                               const FinalizeArgs &f, void *stream, double *ratio_out,
                               double *norms_out) {
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bf16 = plan->g_dtype == LAMB_GRAD_BF16;
    record(plan, 0, s);
    hipError_t err = launch_lamb_moments(plan->tensors, plan->chunks, plan->partials,
                                         plan->n_chunks, bf16, variant, a, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the LAMB moment kernel");
    record(plan, 1, s);
    err = launch_finalize(plan->tensors, plan->n_tensors, plan->partials, f, plan->scale,
                          ratio_out, norms_out, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the finalize kernel");
    record(plan, 2, s);
    err = launch_lamb_apply(plan->tensors, plan->chunks, plan->scale, plan->n_chunks, bf16,
                            variant, a, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the LAMB apply kernel");
    record(plan, 3, s);
    if (plan->timing_used < plan->timing_capacity)
        ++plan->timing_used;
    return LAMB_OK;
}

}  // namespace

extern "C" {

lamb_status lamb_step(lamb_plan *plan, float lr, float beta1, float beta2, float eps,
                      float weight_decay, float gamma_l, float gamma_u, int64_t step,
                      int32_t bias_correction, void *stream, double *ratio_out,
                      double *norms_out) {
    lamb_status st = check_lamb_scalars(plan, lr, beta1, beta2, eps, weight_decay, gamma_l,
                                        gamma_u, step);
    if (st != LAMB_OK)
        return st;
    if (bias_correction != 0 && bias_correction != 1)
        return fail(LAMB_EINVAL, "bias_correction must be 0 or 1");
    // Bias-correction denominators 1 - beta^t in double (Algorithm 2).
    double c1 = 1.0, c2 = 1.0;
    if (bias_correction) {
        c1 = 1.0 - std::pow(double(beta1), double(step));
        c2 = 1.0 - std::pow(double(beta2), double(step));
    }
    LambArgs a = lamb_args(beta1, beta2, eps, weight_decay);
    a.m_scale = float(1.0 / c1);
    a.v_scale = float(1.0 / c2);
    const FinalizeArgs f{double(lr), double(gamma_l), double(gamma_u), 1.0};
    return launch_lamb_family(plan, kLamb, a, f, stream, ratio_out, norms_out);
}

lamb_status nlamb_step(lamb_plan *plan, float lr, float beta1, float beta2, float eps,
                       float weight_decay, float gamma_l, float gamma_u, int64_t step,
                       int32_t nesterov_v, void *stream, double *ratio_out,
                       double *norms_out) {
    lamb_status st = check_lamb_scalars(plan, lr, beta1, beta2, eps, weight_decay, gamma_l,
                                        gamma_u, step);
    if (st != LAMB_OK)
        return st;
    if (nesterov_v != 0 && nesterov_v != 1)
        return fail(LAMB_EINVAL, "nesterov_v must be 0 or 1");
    // Algorithms 3 and 4 with the constant sequence beta1^t = beta1, whose
    // products are powers: coefficients in double, rounded once to fp32.
    const double b1 = beta1, b2 = beta2, t = double(step);
    const double b1_t = std::pow(b1, t), b1_next = std::pow(b1, t + 1.0);
    const double b2_t = std::pow(b2, t), b2_next = std::pow(b2, t + 1.0);
    LambArgs a = lamb_args(beta1, beta2, eps, weight_decay);
    a.m_scale = float(b1 / (1.0 - b1_next));
    a.m_grad = float((1.0 - b1) / (1.0 - b1_t));
    if (nesterov_v) {
        a.v_scale = float(b2 / (1.0 - b2_next));
        a.v_grad = float((1.0 - b2) / (1.0 - b2_t));
    } else {
        a.v_scale = float(b2 / (1.0 - b2_t));
    }
    const FinalizeArgs f{double(lr), double(gamma_l), double(gamma_u), 1.0};
    return launch_lamb_family(plan, nesterov_v ? kNNLamb : kNLamb, a, f, stream, ratio_out,
                              norms_out);
}

lamb_status lars_step(lamb_plan *plan, float lr, float momentum, float weight_decay,
                      float gamma_l, float gamma_u, float trust_coef, void *stream,
                      double *ratio_out, double *norms_out) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (plan->algo != LAMB_ALGO_LARS)
        return fail(LAMB_EPLAN, "lars_step needs a plan created for LARS");
    lamb_status st = check_beta(momentum, "momentum");
    if (st != LAMB_OK)
        return st;
    if (!finite(lr) || !finite(weight_decay) || !finite(trust_coef))
        return fail(LAMB_EINVAL, "lr, weight_decay and trust_coef must be finite");
    st = check_phi_bounds(gamma_l, gamma_u);
    if (st != LAMB_OK)
        return st;

    LarsArgs a;
    a.beta1 = momentum;
    a.one_minus_beta1 = float(1.0 - double(momentum));
    a.weight_decay = weight_decay;
    FinalizeArgs f{double(lr), double(gamma_l), double(gamma_u), double(trust_coef)};

    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bf16 = plan->g_dtype == LAMB_GRAD_BF16;
    record(plan, 0, s);
    hipError_t err = launch_lars_moments(plan->tensors, plan->chunks, plan->partials,
                                         plan->n_chunks, bf16, a, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the LARS momentum kernel");
    record(plan, 1, s);
    err = launch_finalize(plan->tensors, plan->n_tensors, plan->partials, f, plan->scale,
                          ratio_out, norms_out, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the finalize kernel");
    record(plan, 2, s);
    err = launch_lars_apply(plan->tensors, plan->chunks, plan->scale, plan->n_chunks, s);
    if (err != hipSuccess)
        return fail_hip(err, "launching the LARS apply kernel");
    record(plan, 3, s);
    if (plan->timing_used < plan->timing_capacity)
        ++plan->timing_used;
    return LAMB_OK;
}

lamb_status lamb_plan_set_timing(lamb_plan *plan, int32_t max_steps) {
    if (!plan)
        return fail(LAMB_ENULL, "plan must not be NULL");
    if (max_steps < 0 || max_steps > (1 << 20))
        return fail(LAMB_EINVAL, "max_steps = %d outside [0, 2^20]", max_steps);
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    release_events(plan);
    if (max_steps == 0)
        return LAMB_OK;
    plan->events.assign(size_t(max_steps) * 4, nullptr);
    for (size_t k = 0; k < plan->events.size(); ++k) {
        hipError_t err = hipEventCreate(&plan->events[k]);
        if (err != hipSuccess) {
            plan->events.resize(k);
            release_events(plan);
            return fail_hip(err, "hipEventCreate");
        }
    }
    plan->timing_capacity = max_steps;
    plan->timing_used = 0;
    return LAMB_OK;
}

lamb_status lamb_plan_timing(lamb_plan *plan, double *kernel_ms, int64_t *steps) {
    if (!plan || !kernel_ms || !steps)
        return fail(LAMB_ENULL, "plan, kernel_ms and steps must not be NULL");
    DeviceGuard guard(plan->device);
    if (guard.status != hipSuccess)
        return fail_hip(guard.status, "selecting the plan's device");
    kernel_ms[0] = kernel_ms[1] = kernel_ms[2] = 0.0;
    for (int32_t k = 0; k < plan->timing_used; ++k) {
        hipEvent_t *e = &plan->events[size_t(k) * 4];
        hipError_t err = hipEventSynchronize(e[3]);
        if (err != hipSuccess)
            return fail_hip(err, "hipEventSynchronize");
        for (int j = 0; j < 3; ++j) {
            float ms = 0.0f;
            err = hipEventElapsedTime(&ms, e[j], e[j + 1]);
            if (err != hipSuccess)
                return fail_hip(err, "hipEventElapsedTime");
            kernel_ms[j] += ms;
        }
    }
    *steps = plan->timing_used;
    plan->timing_used = 0;
    return LAMB_OK;
}

}  // extern "C"
