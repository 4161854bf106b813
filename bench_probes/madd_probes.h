/*
 * madd_probes.h -- C ABI of libmadd_probes.so: device probes for AMD
 * Instinct MI355X (gfx950) that the benchmark and the tests use.  Not part
 * of the optimizer.
 *
 * madd_ceiling_stream: the empirical bandwidth ceiling of the M+Adam step.
 * The step (include/madd.h) is bound by HBM bandwidth: per element it
 * streams the weight code, the gradient and the three moments in and the
 * weight code and the three moments out (for bf16 weights and fp32 moments
 * 18 bytes read and 14 written).  The probe moves exactly those bytes with
 * the step kernel's work mapping (2048 elements per 256-thread workgroup,
 * four consecutive elements per thread and 1024-element sub-tile,
 * non-temporal 8/16-byte accesses) and no arithmetic.  Every buffer is
 * written back unchanged (each value is XORed with the gradient's bits
 * masked by a runtime zero), so the probe can run on live optimizer state.
 *
 * madd_stream_modes: plain streams in the same access shape (a 256-thread
 * workgroup per 8 KiB tile, 16 bytes per thread in each 4 KiB half,
 * non-temporal): read only, write only, or copy.  Together with the
 * ceiling probe they place the step between what HBM delivers for reads
 * alone, for writes alone and for the step's own read:write mix.
 *
 * madd_probe_bf16_rounding: the step kernel rounds fp32 to bf16 with the
 * v_cvt_pk_bf16_f32 (round to nearest-even) and v_cvt_sr_bf16_f32
 * (stochastic) instructions.  The probe runs both on all 2^32 fp32 bit
 * patterns and counts disagreements with the integer definitions of the
 * two roundings: RNE(u) = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 and
 * SR(u, r16) = (u + r16) >> 16 with the draw r16 in the high half of the
 * instruction's random operand, and checks that the canonical quiet NaN
 * 0x7FC00000 converts to 0x7FC0 under both.
 */
#ifndef MADD_PROBES_H
#define MADD_PROBES_H

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

/* One pass of a plain stream over `bytes` bytes (a positive multiple of
 * 8192): mode 0 reads a (and writes at most the first 4 KiB of b, and only
 * when an XOR of what it read equals a fixed key, which keeps the loads
 * alive), mode 1 writes b, mode 2 copies a to b.  DEVICE pointers, 16-byte
 * aligned, owned by the caller; a may be NULL in mode 1.  Enqueued on
 * `stream`.  Returns 0, -1 for an invalid argument (unknown mode, bad size,
 * NULL pointer), -2 for an unaligned pointer, -4 when the launch fails;
 * nothing is launched on an error. */
int32_t madd_stream_modes(int32_t mode, const void* a, void* b, int64_t bytes, void* stream);

/* Exhaustive check of the two bf16 conversion instructions.
 * counters: DEVICE array of 4 uint64 values owned by the caller, which the
 * caller zeroes before the call; on completion they hold
 *   [0] non-NaN inputs where v_cvt_pk_bf16_f32 differs from RNE(u),
 *   [1] non-NaN inputs where v_cvt_sr_bf16_f32 differs from SR(u, r16)
 *       (r16: a fixed hash of u, so every input meets a different draw),
 *   [2] conversions of 0x7FC00000 (both instructions, with every draw of a
 *       sample of 2^16 draws) that do not give 0x7FC0,
 *   [3] the number of inputs examined (2^32).
 * Enqueued on `stream`.  Returns 0, -1 for a NULL pointer, -4 when the
 * launch fails. */
int32_t madd_probe_bf16_rounding(uint64_t* counters, void* stream);

/* madd_probe_delay: one wave on `stream` that sleeps `sleeps` times (each
 * s_sleep 127, about 8k cycles, ~3.5 us) and exits.  The benchmark enqueues
 * it ahead of a run of short steps so that the host has queued them all
 * before the first starts, and the events between steps time the GPU alone.
 * Returns -1 for sleeps outside [0, 2^20], -3 if the launch fails. */
int32_t madd_probe_delay(int32_t sleeps, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MADD_PROBES_H */
