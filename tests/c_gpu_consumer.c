/*
 * The optimizer step end to end from plain C: device buffers from the HIP
 * runtime, the step through include/lamb_mi355x.h, and every result checked
 * against the CPU oracle (oracle/lamb_oracle.c, a separate library) on the
 * same inputs. No Python and no torch are involved.
 *
 * Three LAMB steps (Algorithm 2) on both paths and with fp32 and bf16
 * gradients, then three LARS steps (Algorithm 1), over tensors of ragged
 * sizes. x, m and v must agree element by element to 1e-5 relative to
 * max(|oracle|, the oracle's RMS of that tensor), and the trust ratios to
 * 1e-6 relative (exactly 0 where the oracle's is 0).
 *
 * Prints one line per failed check and exits non-zero on any failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "lamb_mi355x.h"

/* The oracle's entry points (oracle/lamb_oracle.c). */
int oracle_lamb_layer(int64_t d, float *x, const void *g, int g_is_bf16, float *m, float *v,
                      double lr, double beta1, double beta2, double eps, double weight_decay,
                      int wd, double gamma_l, double gamma_u, int64_t t, int bias_correction,
                      double grad_scale, int norm, double *out);
int oracle_lars_layer(int64_t d, float *x, const void *g, int g_is_bf16, float *m, double lr,
                      double beta1, double weight_decay, int wd, double gamma_l, double gamma_u,
                      double trust_coef, double grad_scale, int norm, double *out);

#define N_TENSORS 7
static const int64_t kSizes[N_TENSORS] = {1, 3, 1000, 4096, 3 * 8192 + 5, 100003, 1 << 20};

static int failures = 0;

#define HIP_OK(call)                                                            \
    do {                                                                        \
        hipError_t e_ = (call);                                                 \
        if (e_ != hipSuccess) {                                                 \
            printf("HIP error %s at line %d: %s\n", hipGetErrorString(e_),      \
                   __LINE__, #call);                                            \
            exit(2);                                                            \
        }                                                                       \
    } while (0)

/* Inputs: splitmix64 draws turned into normal deviates (Box-Muller). */
static uint64_t rng_state;

static double uniform01(void) {
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return ((double)(z >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

static float normal(double sigma) {
    const double two_pi = 6.283185307179586;
    double a = uniform01(), b = uniform01();
    return (float)(sigma * sqrt(-2.0 * log(a)) * cos(two_pi * b));
}

/* The high half of an fp32: the same bf16 bits go to both sides. */
static uint16_t bf16_bits(float f) {
    uint32_t w;
    memcpy(&w, &f, sizeof w);
    return (uint16_t)(w >> 16);
}

typedef struct {
    float *x, *m, *v;   /* host: the oracle's state */
    void *g;            /* host gradient (fp32 or bf16 bits) */
    float *dx, *dm, *dv; /* device: the library's state */
    void *dg;
} Tensor;

static void check_close(const char *what, int tensor, int step, const float *got,
                        const float *want, int64_t n) {
    double ss = 0.0, worst = 0.0;
    int64_t j, at = 0;
    for (j = 0; j < n; ++j)
        ss += (double)want[j] * (double)want[j];
    {
        const double rms = sqrt(ss / (double)n);
        for (j = 0; j < n; ++j) {
            const double b = want[j], a = got[j];
            const double scale = fabs(b) > rms ? fabs(b) : rms;
            const double err = scale > 0.0 ? fabs(a - b) / scale : fabs(a - b);
            if (!(err <= worst)) {
                worst = err;
                at = j;
            }
        }
    }
    if (!(worst <= 1e-5)) {
        printf("FAILED %s of tensor %d at step %d: element %lld error %.3g (got %.9g, want %.9g)\n",
               what, tensor, step, (long long)at, worst, got[at], want[at]);
        ++failures;
    }
}

static void check_ratio(int tensor, int step, double got, double want) {
    const int ok = want == 0.0 ? got == 0.0 : fabs(got - want) <= 1e-6 * fabs(want);
    if (!ok) {
        printf("FAILED ratio of tensor %d at step %d: got %.17g, want %.17g\n", tensor, step, got,
               want);
        ++failures;
    }
}

/* Draw x ~ N(0, 0.02), zero moments, and copy them to the device. */
static void init_tensors(Tensor *ts, int bf16, uint64_t seed) {
    int i;
    int64_t j;
    rng_state = seed;
    for (i = 0; i < N_TENSORS; ++i) {
        const int64_t n = kSizes[i];
        Tensor *t = &ts[i];
        t->x = (float *)malloc((size_t)n * sizeof(float));
        t->m = (float *)calloc((size_t)n, sizeof(float));
        t->v = (float *)calloc((size_t)n, sizeof(float));
        t->g = malloc((size_t)n * (bf16 ? 2 : 4));
        if (!t->x || !t->m || !t->v || !t->g) {
            printf("host allocation failed\n");
            exit(2);
        }
        for (j = 0; j < n; ++j)
            t->x[j] = normal(0.02);
        HIP_OK(hipMalloc((void **)&t->dx, (size_t)n * sizeof(float)));
        HIP_OK(hipMalloc((void **)&t->dm, (size_t)n * sizeof(float)));
        HIP_OK(hipMalloc((void **)&t->dv, (size_t)n * sizeof(float)));
        HIP_OK(hipMalloc(&t->dg, (size_t)n * (bf16 ? 2 : 4)));
        HIP_OK(hipMemcpy(t->dx, t->x, (size_t)n * sizeof(float), hipMemcpyHostToDevice));
        HIP_OK(hipMemset(t->dm, 0, (size_t)n * sizeof(float)));
        HIP_OK(hipMemset(t->dv, 0, (size_t)n * sizeof(float)));
    }
}

/* Gradient of one step, g ~ N(0, 1e-3), on both sides. */
static void draw_grads(Tensor *ts, int bf16) {
    int i;
    int64_t j;
    for (i = 0; i < N_TENSORS; ++i) {
        const int64_t n = kSizes[i];
        for (j = 0; j < n; ++j) {
            const float f = normal(1e-3);
            if (bf16)
                ((uint16_t *)ts[i].g)[j] = bf16_bits(f);
            else
                ((float *)ts[i].g)[j] = f;
        }
        HIP_OK(hipMemcpy(ts[i].dg, ts[i].g, (size_t)n * (bf16 ? 2 : 4), hipMemcpyHostToDevice));
    }
}

static void compare_state(Tensor *ts, int with_v, int step, const double *ratios,
                          const double *want_ratios) {
    int i;
    for (i = 0; i < N_TENSORS; ++i) {
        const int64_t n = kSizes[i];
        float *buf = (float *)malloc((size_t)n * sizeof(float));
        if (!buf) {
            printf("host allocation failed\n");
            exit(2);
        }
        HIP_OK(hipMemcpy(buf, ts[i].dx, (size_t)n * sizeof(float), hipMemcpyDeviceToHost));
        check_close("x", i, step, buf, ts[i].x, n);
        HIP_OK(hipMemcpy(buf, ts[i].dm, (size_t)n * sizeof(float), hipMemcpyDeviceToHost));
        check_close("m", i, step, buf, ts[i].m, n);
        if (with_v) {
            HIP_OK(hipMemcpy(buf, ts[i].dv, (size_t)n * sizeof(float), hipMemcpyDeviceToHost));
            check_close("v", i, step, buf, ts[i].v, n);
        }
        check_ratio(i, step, ratios[i], want_ratios[i]);
        free(buf);
    }
}

static void free_tensors(Tensor *ts) {
    int i;
    for (i = 0; i < N_TENSORS; ++i) {
        free(ts[i].x);
        free(ts[i].m);
        free(ts[i].v);
        free(ts[i].g);
        HIP_OK(hipFree(ts[i].dx));
        HIP_OK(hipFree(ts[i].dm));
        HIP_OK(hipFree(ts[i].dv));
        HIP_OK(hipFree(ts[i].dg));
    }
}

static lamb_plan *make_plan(Tensor *ts, int bf16, int algo) {
    lamb_tensor rows[N_TENSORS];
    lamb_plan *plan = NULL;
    int i;
    for (i = 0; i < N_TENSORS; ++i) {
        rows[i].x = ts[i].dx;
        rows[i].g = ts[i].dg;
        rows[i].m = ts[i].dm;
        rows[i].v = algo == LAMB_ALGO_LAMB ? ts[i].dv : NULL;
        rows[i].numel = kSizes[i];
        rows[i].wd = kSizes[i] > 1000; /* the small ones play biases */
        rows[i].reserved = 0;
    }
    if (lamb_plan_create(rows, N_TENSORS, bf16 ? LAMB_GRAD_BF16 : LAMB_GRAD_F32, algo, 0,
                         &plan) != LAMB_OK) {
        printf("lamb_plan_create failed: %s\n", lamb_last_error());
        exit(2);
    }
    return plan;
}

static void run_lamb(int bf16, int path, uint64_t seed) {
    Tensor ts[N_TENSORS];
    double *d_ratio = NULL, ratio[N_TENSORS], want[N_TENSORS], out[3];
    const float lr = 6e-3f, b1 = 0.9f, b2 = 0.999f, eps = 1e-6f, wd = 0.01f, gl = 0.0f,
                gu = 10.0f;
    lamb_plan *plan;
    int i, t;
    init_tensors(ts, bf16, seed);
    plan = make_plan(ts, bf16, LAMB_ALGO_LAMB);
    if (lamb_plan_set_path(plan, path) != LAMB_OK) {
        printf("lamb_plan_set_path failed: %s\n", lamb_last_error());
        exit(2);
    }
    HIP_OK(hipMalloc((void **)&d_ratio, N_TENSORS * sizeof(double)));
    for (t = 1; t <= 3; ++t) {
        draw_grads(ts, bf16);
        if (lamb_step(plan, lr, b1, b2, eps, wd, gl, gu, t, 1, NULL, d_ratio, NULL) != LAMB_OK) {
            printf("lamb_step failed: %s\n", lamb_last_error());
            exit(2);
        }
        for (i = 0; i < N_TENSORS; ++i) {
            if (oracle_lamb_layer(kSizes[i], ts[i].x, ts[i].g, bf16, ts[i].m, ts[i].v, lr, b1,
                                  b2, eps, wd, kSizes[i] > 1000, gl, gu, t, 1, 1.0, 0,
                                  out) != 0) {
                printf("oracle failed\n");
                exit(2);
            }
            want[i] = out[0];
        }
        HIP_OK(hipDeviceSynchronize());
        HIP_OK(hipMemcpy(ratio, d_ratio, sizeof ratio, hipMemcpyDeviceToHost));
        compare_state(ts, 1, t, ratio, want);
    }
    if (lamb_plan_check(plan, NULL) != LAMB_OK) {
        printf("FAILED lamb_plan_check: %s\n", lamb_last_error());
        ++failures;
    }
    lamb_plan_destroy(plan);
    HIP_OK(hipFree(d_ratio));
    free_tensors(ts);
    printf("LAMB %s gradients, %s path: 3 steps compared\n", bf16 ? "bf16" : "fp32",
           path == LAMB_PATH_AUTO ? "default" : "two-pass");
}

static void run_lars(uint64_t seed) {
    Tensor ts[N_TENSORS];
    double *d_ratio = NULL, ratio[N_TENSORS], want[N_TENSORS], out[3];
    const float lr = 1e-3f, mom = 0.9f, wd = 1e-4f, gl = 0.0f, gu = 10.0f, kappa = 1e-3f;
    lamb_plan *plan;
    int i, t;
    init_tensors(ts, 0, seed);
    plan = make_plan(ts, 0, LAMB_ALGO_LARS);
    HIP_OK(hipMalloc((void **)&d_ratio, N_TENSORS * sizeof(double)));
    for (t = 1; t <= 3; ++t) {
        draw_grads(ts, 0);
        if (lars_step(plan, lr, mom, wd, gl, gu, kappa, NULL, d_ratio, NULL) != LAMB_OK) {
            printf("lars_step failed: %s\n", lamb_last_error());
            exit(2);
        }
        for (i = 0; i < N_TENSORS; ++i) {
            if (oracle_lars_layer(kSizes[i], ts[i].x, ts[i].g, 0, ts[i].m, lr, mom, wd,
                                  kSizes[i] > 1000, gl, gu, kappa, 1.0, 0, out) != 0) {
                printf("oracle failed\n");
                exit(2);
            }
            want[i] = out[0];
        }
        HIP_OK(hipDeviceSynchronize());
        HIP_OK(hipMemcpy(ratio, d_ratio, sizeof ratio, hipMemcpyDeviceToHost));
        compare_state(ts, 0, t, ratio, want);
    }
    lamb_plan_destroy(plan);
    HIP_OK(hipFree(d_ratio));
    free_tensors(ts);
    printf("LARS fp32 gradients, default path: 3 steps compared\n");
}

int main(void) {
    run_lamb(0, LAMB_PATH_AUTO, 11);
    run_lamb(1, LAMB_PATH_AUTO, 12);
    run_lamb(1, LAMB_PATH_TWO_PASS, 13);
    run_lars(14);
    if (failures == 0)
        printf("c gpu consumer: all checks passed\n");
    return failures == 0 ? 0 : 1;
}
