/*
 * madd_ceiling.h -- C ABI of libmadd_ceiling.so, a measurement probe for
 * AMD Instinct MI355X (gfx950).  Not part of the optimizer.
 *
 * The M+Adam step (include/madd.h) is bound by HBM bandwidth: per element it
 * streams the weight code, the gradient and the three moments in and the
 * weight code and the three moments out (for bf16 weights and fp32 moments
 * 18 bytes read and 14 written).  This probe moves exactly those bytes with
 * the step kernel's work mapping (2048 elements per 256-thread workgroup,
 * four consecutive elements per thread and 1024-element sub-tile,
 * non-temporal 8/16-byte accesses) and no arithmetic, so its bandwidth is the
 * empirical ceiling of the step's memory traffic on the same buffers.
 *
 * Every buffer is written back unchanged (each value is XORed with the
 * gradient's bits masked by a runtime zero), so the probe can run on live
 * optimizer state.
 */
#ifndef MADD_CEILING_H
#define MADD_CEILING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One pass over n elements: read w (bf16 codes), g (fp32), m, v, ve
 * (state_bytes = 4: fp32, 2: bf16 codes), write w, m, v, ve.
 * All pointers are DEVICE pointers, 16-byte aligned, owned by the caller;
 * n >= 0.  Enqueued on `stream` (hipStream_t as void*).
 * Returns 0 on success, -1 for an invalid argument (NULL pointer, n < 0,
 * state_bytes not 2 or 4), -2 for an unaligned pointer, -4 when the launch
 * fails; nothing is launched on an error. */
int32_t madd_ceiling_stream(void* w, const float* g, void* m, void* v, void* ve,
                            int32_t state_bytes, int64_t n, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MADD_CEILING_H */
