/*
 * stream_probe.h -- HBM streams with the per-element access pattern of the
 * optimizer's kernels and none of their arithmetic (measurement only).
 *
 * The LAMB step is bound by HBM bandwidth, and what a bandwidth-bound kernel
 * can reach depends on its mix of reads and writes. These streams read and
 * write the same arrays, in the same 16-byte (8-byte for bf16) per-lane
 * accesses, with the same nontemporal hints and the same number of elements
 * per workgroup as the kernel they stand for, so their rate is the
 * attainable bandwidth for that kernel's traffic. They are not part of the
 * optimizer (include/lamb_mi355x.h); bench.py uses them.
 *
 * All pointers are device pointers to `n` elements, 16-byte aligned (x, m, v
 * fp32; g fp32 or bf16). A stream writes x, m and v back unchanged (it adds
 * -0.0, built at run time from the loaded values so that no access can be
 * optimised away), so it may run over live data; NaN payloads may be
 * quieted. Errors: -1 for an invalid argument (checked on the host before any
 * launch), -5 for a failed launch.
 */
#ifndef STREAM_PROBE_H
#define STREAM_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define PROBE_API __attribute__((visibility("default")))
#else
#define PROBE_API
#endif

typedef enum stream_pattern {
    STREAM_SINGLE_PASS = 0, /* read x g m v, write x m v (the single-pass kernel) */
    STREAM_MOMENTS = 1,     /* read x g m v, write m v (the moment kernel)         */
    STREAM_APPLY = 2,       /* read x m v, write x (the apply kernel)              */
    STREAM_READ = 3,        /* read x g m v                                        */
    STREAM_COPY = 4         /* read m, write x                                     */
} stream_pattern;

/*
 * One stream of `pattern` over n elements, `tile` elements per workgroup of
 * 256 threads (a multiple of 8 in [8, 2^24]; the single-pass kernel uses
 * 8192, the moment and apply kernels the plan's chunk size, 256 by default),
 * enqueued on `stream` (hipStream_t, NULL = null stream). g_bf16: 1 if g
 * holds bf16.
 * layer_tiles = 0: each workgroup streams a contiguous tile. layer_tiles > 0
 * (tile a multiple of 1024): the single-pass kernel's layout, the array cut
 * into layers of layer_tiles tiles, tile i of a layer holding the layer's
 * 1024-element blocks i, i + layer_tiles, ....
 */
PROBE_API int stream_probe(int32_t pattern, float *x, float *m, float *v, const void *g,
                           int32_t g_bf16, int64_t n, int32_t tile, int32_t layer_tiles,
                           void *stream);

#ifdef __cplusplus
}
#endif

#endif /* STREAM_PROBE_H */
