/*
 * madd.h -- C ABI of the M+Adam optimizer-step library for AMD Instinct
 * MI355X (gfx950).
 *
 * The library applies one step of M+Adam, the additive-multiplicative
 * optimizer of arXiv 2607.10611, to weights kept only in a low-precision
 * storage format (no FP32 master copy):
 *
 *   additive branch (Algorithm 1; Section 3.1)
 *       m  <- b1 m + (1 - b1) g            v <- b2 v + (1 - b2) g^2
 *       u_a = -eta_a m^ / (sqrt(v^) + eps),  m^ = m/(1-b1^t), v^ = v/(1-b2^t)
 *   multiplicative branch (Algorithm 1; Section 3.1)
 *       g_e = ln2 * w * g                  (gradient w.r.t. the exponent)
 *       ve <- b2 ve + (1 - b2) g_e^2
 *       ut = -eta_m clamp_{g_max}(g_e / (sqrt(ve^) + eps)),  ve^ = ve/(1-b2^t)
 *       u_m = clip(ut / max(|w|, tau))     clip: [-(r_max - eps0), r_max] and
 *                                          |log2(1 + u_m)| <= d_mult_max
 *                                          (clamps of Algorithm 2, Appendix A)
 *   combine
 *       w <- clamp_{w_max}(w + w u_m + u_a), rounded into the storage format
 *       (the FP32-step / low-precision-storage round trip of Appendix B),
 *       to nearest-even or stochastically.  Storage: bf16, FP8 (unscaled or
 *       with FP16 scales per 128 elements), MXFP4 and NVFP4 (Section 4.2's
 *       4-bit master weights), FP32 for testing.
 *
 * The step is computed in FP32 in one fixed operation order; results are
 * bit-reproducible across launches, shardings and tensor groupings.
 *
 * Conventions common to every entry point
 *   - Buffer pointers (weights, gradients, moments, scales) are DEVICE
 *     pointers owned by the caller.  Pointer arrays, numel arrays and the
 *     hyper-parameter struct are HOST memory, read during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued asynchronously on it; no call synchronizes the host
 *     or the device.  The only device allocations are those of
 *     madd_multi_tensor_step's descriptor-table cache (see that function).
 *   - A failed launch is reported as MADD_EDEVICE from the launch's own
 *     return status; the calling thread's HIP last-error state is neither
 *     read nor cleared.
 *   - Updates are in place on w, m, v, ve and scales; g is read-only
 *     (except for NVFP4_CURRENT tensors, whose step writes w' over g).
 *     Buffers must not alias each other: each call checks that the byte
 *     ranges of the arrays it takes for one tensor (weights, scales, compute
 *     copy, gradient, moments; input and output of an encoding) are
 *     pairwise disjoint, from their formats and sizes, and returns
 *     MADD_EINVAL otherwise.  Overlap between different tensors of a list is
 *     not checked.  Concurrent calls that touch the same buffers race.
 *   - Arguments are validated before any device work; on any status other
 *     than MADD_OK no buffer has been touched.  A tensor holds at most 2^60
 *     elements (larger sizes are MADD_EINVAL).
 *   - Every status is a madd_status value; madd_status_string() names it.
 */
#ifndef MADD_H
#define MADD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
typedef enum madd_status {
  MADD_OK = 0,
  MADD_EINVAL = -1,      /* invalid argument (NULL pointer, size, range, enum) */
  MADD_EALIGN = -2,      /* block-scaled buffers not 16-byte aligned          */
  MADD_EUNSUPPORTED = -3,/* valid request the library does not implement      */
  MADD_EDEVICE = -4,     /* a HIP runtime call or kernel launch failed         */
  MADD_ENOMEM = -5,      /* device allocation for the descriptor table failed  */
  MADD_ECAPTURE = -6,    /* a multi-tensor list seen for the first time while
                            its stream is capturing a graph                    */
  MADD_ESCRATCH = -7     /* more tensors than madd_multi_tensor_step_noalloc's
                            fixed descriptor table holds                       */
} madd_status;

/* Weight storage formats.
 *   BF16     : IEEE-style bfloat16; RNE overflows to Inf; NaN stored as
 *              0x7FC0.
 *   FP8_E4M3 : OCP E4M3 (bias 7, max 448, no Inf, NaN = S.1111.111).
 *   FP8_E5M2 : OCP E5M2 (bias 15, max 57344).
 *              Both FP8 formats saturate finite overflow and Inf to +-max and
 *              store NaN as 0x7F.
 *   FP32     : passthrough (no rounding); for testing the unrounded step.
 *              NaN stored as 0x7FC00000.
 *   MXFP4    : 4-bit block-scaled storage, the OCP Microscaling (MX) v1.0
 *              format MXFP4 -- the paper's 4-bit master-weight regime
 *              (Section 4.2, the NVFP4/FP8 setting) names a 4-bit block
 *              format without defining it.  Elements are OCP E2M1 (values
 *              0, 0.5, 1, 1.5, 2, 3, 4, 6 and negatives), packed two per
 *              byte, element 2k in the low nibble of byte k (w holds n/2
 *              bytes).  Blocks of 32 contiguous elements share one E8M0
 *              scale X = 2^(code - 127) (code 255 = NaN); the weight is
 *              E2M1 value * X.  Always block-scaled (scales required).
 *   NVFP4    : 4-bit two-level block scaling, NVIDIA's NVFP4 (the format the
 *              paper's 4-bit runs name): E2M1 payloads packed as for MXFP4;
 *              blocks of 16 elements, each with an OCP E4M3 scale code c
 *              (unsigned; 0x7F = NaN); one fp32 scale st per tensor.  The
 *              weight is E2M1 value * fp32(E4M3(c) * st).  The scale array
 *              holds st in its first 4 bytes (fp32, 4-byte aligned), then
 *              the n/16 block codes.  Always block-scaled.  A step keeps st.
 *   NVFP4_CURRENT : NVFP4 whose per-tensor scale is derived anew from the
 *              updated tensor at every step (current scaling), as the
 *              dequantize / FP32 step / quantize round trip of the paper's
 *              NVFP4 prototype (Section 4.2, Appendix G) does.  Payloads and
 *              block codes as NVFP4; the scale array holds st (4 bytes), one
 *              4-byte word that a step sets to the bits of the tensor's
 *              largest finite |w'|, then the n/16 block codes (8 + n/16
 *              bytes, 4-byte aligned).  The step needs fp32 gradients and
 *              overwrites them with the updated weights w' (fp32): the
 *              second of its two passes re-encodes them once the new st is
 *              known. */
typedef enum madd_wfmt {
  MADD_W_BF16 = 0,
  MADD_W_FP8_E4M3 = 1,
  MADD_W_FP8_E5M2 = 2,
  MADD_W_FP32 = 3,
  MADD_W_MXFP4 = 4,
  MADD_W_NVFP4 = 5,
  MADD_W_NVFP4_CURRENT = 6
} madd_wfmt;

/* Gradient formats (decoded exactly to FP32). */
typedef enum madd_gfmt { MADD_G_FP32 = 0, MADD_G_BF16 = 1 } madd_gfmt;

/* Storage of the moments m, v, v_e.
 *   FP32    : float arrays.
 *   BF16    : bfloat16 codes -- the precision of the optimizer states in the
 *             paper's per-parameter memory accounting (Appendix, memory
 *             comparison table).  A step decodes them exactly, computes in
 *             FP32, uses the FP32 results within the step and stores them
 *             rounded to nearest (ties to even).
 *   BF16_SR : bfloat16 codes as BF16, stored with stochastic rounding (the
 *             rule of madd_round) instead; m, v and v_e of the element with
 *             global index i draw from Philox streams 1, 2 and 3 (counter
 *             word 3) at the step's seed and t, independently of the weight's
 *             stream 0 and of hp->rounding. */
typedef enum madd_sfmt { MADD_S_FP32 = 0, MADD_S_BF16 = 1, MADD_S_BF16_SR = 2 } madd_sfmt;

/* Rounding of the new weight into its storage format.
 *   RNE : round to nearest, ties to even.
 *   SR  : stochastic.  For |x| between adjacent grid points lo < |x| < hi,
 *         rounds up iff floor((|x|-lo)/(hi-lo) * 2^16) + r16 >= 2^16, where
 *         r16 is the element's 16-bit draw; the sign is restored afterwards.
 *         For BF16 this gives P(up) = (|x|-lo)/(hi-lo) exactly.
 *         r16 for global element index i at step t is the 16-bit lane
 *         (i & 7) -- bits 16*(i&1)..+15 of word (i&7)>>1 -- of
 *         Philox4x32-10 (Salmon et al., SC'11) with key (seed lo32, seed
 *         hi32) and counter ((i>>3) lo32, (i>>3) hi32, t, 0).  The paper cites
 *         stochastic rounding without defining it. */
typedef enum madd_round { MADD_ROUND_RNE = 0, MADD_ROUND_SR = 1 } madd_round;

/* Hyper-parameters of one step (inputs of Algorithms 1 and 2).
 * The library evaluates the derived scalars in double and rounds each once
 * to float: b1, b2, 1-b1, 1-b2, eta_a/(1-b1^t) (or eta_a), 1/(1-b2^t) (or 1),
 * eta_m, eps, tau, g_max, w_max, and the u_m clip bounds
 * max(-(r_max-eps0), 2^-d - 1), min(r_max, 2^d - 1) with d = d_mult_max.
 * Valid ranges (else MADD_EINVAL):
 *   0 <= beta1 < 1, 0 <= beta2 < 1, eps >= 0, tau > 0, 0 < r_max < 1,
 *   0 <= eps0 < r_max, g_max > 0, d_mult_max > 0, w_max > 0 (+INFINITY turns
 *   the clamp off), bias_correction in {0, 1}, rounding a madd_round,
 *   1 <= step <= 2^32 - 1. */
typedef struct madd_hparams {
  double lr_add;          /* eta_a: additive step size                         */
  double lr_mul;          /* eta_m: multiplicative step size                   */
  double beta1, beta2;    /* moment decay rates                                */
  double eps;             /* stabiliser in both denominators                   */
  double tau;             /* rho = max(|w|, tau)                               */
  double r_max;           /* u_m clip: [-(r_max - eps0), r_max]; paper: 0.75   */
  double eps0;            /* asymmetry of the lower clip bound; 0 = symmetric  */
  double g_max;           /* clamp of the normalised multiplicative direction  */
  double d_mult_max;      /* cap on |log2(1 + u_m)|                            */
  double w_max;           /* final weight clamp                                */
  int32_t bias_correction;/* 1: Algorithm 1 (bias-corrected); 0: Algorithm 2   */
  int32_t rounding;       /* madd_round                                        */
  uint64_t seed;          /* stochastic-rounding key                           */
  int64_t step;           /* t, starting at 1; the caller increments it        */
} madd_hparams;

/* Zero the optimizer state (Algorithm 1: moments start at 0).
 * m, v, ve: device arrays of n elements stored as sfmt (a madd_sfmt); n >= 0,
 * NULL allowed when n == 0.  Enqueued on `stream`. */
int32_t madd_init_state(void* m, void* v, void* ve, int32_t sfmt, int64_t n, void* stream);

/* Round n fp32 values x into weight storage w with round-to-nearest-even.
 * w: device codes of format wfmt (2, 1, 1, 4 or 1/2 bytes per element).
 * scales: NULL for unscaled storage, else a device array of block scales:
 *   - block-scaled FP8 (wfmt E4M3 or E5M2): n/128 FP16 codes (uint16),
 *     n % 128 == 0.  Block b is elements [128b, 128b+128); its scale is
 *     RNE_fp16(max|x| / FMAX) (1.0 when the block is all zero, smallest FP16
 *     subnormal on underflow, largest finite FP16 on overflow, FP16 NaN when
 *     the block holds a non-finite value) and its payloads are
 *     encode(x / scale).
 *   - MXFP4 (required): n/32 E8M0 codes (uint8), n % 32 == 0.  Block b is
 *     elements [32b, 32b+32); its scale is 2^s with s = floor(log2 max|x|)
 *     - 2 (2 = exponent of E2M1's largest value 6), clamped to [-127, 127]
 *     (the OCP MX conversion rule); s = 0 for an all-zero block; the NaN
 *     scale, with zero payloads, for a block holding a non-finite value.
 *     Payloads are x / 2^s rounded onto E2M1, saturating at +-6.
 *   - NVFP4 (required): 4 + n/16 bytes, 4-byte aligned, n % 16 == 0.  The
 *     per-tensor scale is st = fp32(amax / 2688) over the finite |x| (2688 =
 *     6 * 448, E2M1's largest value times E4M3's; st = 1 when no value is
 *     finite and nonzero); block b's code is RNE_E4M3(fp32(amax_b /
 *     fp32(6 st))) saturating at 448 (NaN when the block holds a non-finite
 *     value); payloads are fp32(x / D_b), D_b = fp32(E4M3(code) * st),
 *     rounded onto E2M1 saturating at +-6, and 0 when D_b is 0 or the block
 *     is NaN.  Four launches on `stream` (the amax reduction uses the first
 *     scale word).
 *   - NVFP4_CURRENT (required): 8 + n/16 bytes, 4-byte aligned: st and the
 *     block codes as for NVFP4, with the second word set to 0. */
int32_t madd_encode_weights(const float* x, void* w, int32_t wfmt, void* scales, int64_t n,
                            void* stream);

/* One M+Adam step on one tensor of n elements (Algorithm 1 with the optional
 * clamps of Algorithm 2).
 * w       : device weight codes of format wfmt, updated in place.
 * copy    : NULL, or a device array of n bf16 codes that receives the compute
 *           copy of the new weights: each new stored value (payload x scale
 *           when block-scaled) rounded to nearest-even -- the BF16 copy the
 *           next step's GEMMs read, which the paper's FP8-master dataflow
 *           (Appendix figure) rebuilds from the stored weights after every
 *           update; here the same pass writes it.  16-byte aligned for the
 *           fast path.
 * scales  : NULL, or the block scales of block-scaled FP8, MXFP4 or NVFP4
 *           as in madd_encode_weights (required for the 4-bit formats): the
 *           weight is payload * scale (fp32 product); after the update each
 *           block's scale is recomputed from the new weights by the same rule
 *           and the payloads re-encoded with hp->rounding.  NVFP4's
 *           per-tensor scale st is read and kept (re-encode to refresh it);
 *           NVFP4_CURRENT derives st' = fp32(amax / 2688) over the finite
 *           |w'| of the whole tensor (1 when none is nonzero), stores it and
 *           the amax bits, and re-encodes every block with st'.  It runs
 *           in two passes: pass 1 (the FP32 step: moments stored, w' written
 *           over g, amax folded in with atomics) and pass 2 (block codes and
 *           payloads from w' and st'), after a launch that clears the amax
 *           words.  In a multi-tensor call, pass 2 of one group of tensors
 *           runs in the same launch as pass 1 of the next group.  gfmt must
 *           be FP32 (else MADD_EINVAL) and g is overwritten.
 *           Requires n % 128 == 0 (FP8), n % 32 == 0 (MXFP4) or n % 16 == 0
 *           (NVFP4, NVFP4_CURRENT) and 16-byte-aligned w, g, m, v, ve and
 *           copy, and a 4-byte-aligned NVFP4 scale array (else MADD_EINVAL /
 *           MADD_EALIGN).
 * g       : device gradient of format gfmt (read only, except for
 *           NVFP4_CURRENT, which overwrites it with w').
 * m, v, ve: device moments (first, second, multiplicative second) stored as
 *           sfmt (a madd_sfmt), updated in place.
 * index_base: global index of element 0 (keys the stochastic-rounding draw);
 *           a loop of madd_step calls whose bases are the prefix sums of the
 *           sizes is bit-identical to one madd_multi_tensor_step call, and to
 *           any split of the index space (sharding).
 * Unaligned unscaled buffers are accepted and take a slower path with
 * identical results. */
int32_t madd_step(void* w, int32_t wfmt, void* scales, uint16_t* copy, const void* g,
                  int32_t gfmt, void* m, void* v, void* ve, int32_t sfmt, int64_t n,
                  int64_t index_base, const madd_hparams* hp, void* stream);

/* One M+Adam step on a list of tensors in as few launches as the formats
 * allow (one per distinct (format, scaled) pair).
 * ntensors >= 0; w, wfmt, g, m, v, ve, numel: host arrays of ntensors
 * entries; gfmt and sfmt apply to every tensor (gfmt must be FP32 when the
 * list holds a nonempty NVFP4_CURRENT tensor, whose gradient the step
 * overwrites with w'); scales: NULL (no tensor
 * block-scaled) or a host array whose entry i is NULL or tensor i's scale
 * array (never NULL for an MXFP4, NVFP4 or NVFP4_CURRENT tensor); copy: NULL (no compute copies) or a host array whose entry i is NULL
 * or tensor i's bf16 compute-copy array (as in madd_step).  Tensors of
 * different weight formats may be mixed -- e.g. block-scaled FP8 linear
 * layers (or MXFP4 / NVFP4 ones) with BF16 embeddings, norms and head, the paper's
 * FP8-master (4-bit-master) setting (Section 4.2).  Tensor i's elements have global
 * indices index_base + sum_{j<i} numel[j] + local index.
 * Descriptor tables.  The kernels read a device table of the list (88 bytes
 * per tensor: pointers, sizes, index bases) that the library caches by
 * content, per device:
 *   - The first call with a given list (same pointers and sizes) allocates
 *     the table's device memory (hipMalloc) and writes it on `stream` with a
 *     small kernel (asynchronous); later calls with the same list enqueue
 *     only the step kernels.  Nothing records events, waits on the host or
 *     frees memory.
 *   - Up to 32 lists per (device, stream) are cached besides pinned ones; a
 *     new list past that rewrites the least recently used table whose latest
 *     use was on the same stream, so the rewrite is queued behind every
 *     launch that read it there (launches of it on other streams came
 *     earlier and were ordered before that one by the caller, who must order
 *     two steps of the same tensors anyway).  Otherwise a new table is
 *     allocated.
 *   - Graph capture.  A call made while `stream` is capturing a graph only
 *     enqueues kernels, and its tables are pinned: never rewritten or freed
 *     until the process ends, so every replay of the graph reads a live,
 *     unchanged table.  A list must have been stepped once outside the
 *     capture; a list first seen during a capture returns MADD_ECAPTURE and
 *     enqueues nothing (no allocation or upload inside a capture; the
 *     allocation-free entry point below has no such restriction).  No call
 *     records a memset.  The hyper-parameters, step counter included, are
 *     kernel arguments fixed at capture (see madd_multi_tensor_step_dev for
 *     replaying successive steps). */
int32_t madd_multi_tensor_step(int32_t ntensors, void* const* w, const int32_t* wfmt,
                               void* const* scales, uint16_t* const* copy,
                               const void* const* g, int32_t gfmt,
                               void* const* m, void* const* v, void* const* ve, int32_t sfmt,
                               const int64_t* numel, int64_t index_base, const madd_hparams* hp,
                               void* stream);

/* madd_multi_tensor_step without any device allocation, for callers that
 * cannot allocate device memory (code running under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  Same arguments, results
 * (bit for bit) and validation as madd_multi_tensor_step.  The descriptor
 * tables of the call are written into a fixed device array that the library
 * holds on each GPU until the process ends (4096 descriptors of 88 bytes,
 * 352 KiB per GPU), with small kernels on `stream` ahead of the step kernels:
 * nothing is cached, allocated, freed or waited for, and a captured call
 * records the table writes too, so its replays need no earlier eager call.
 * Limits: at most 4096 nonempty tensors per call (else MADD_ESCRATCH, nothing
 * enqueued).  Every call on one GPU shares that array: calls on one GPU that
 * can run at the same time (different streams or threads, or graphs replayed
 * concurrently) race and must be ordered by the caller.  The first call on a
 * GPU looks up the array's device address (hipGetSymbolAddress) with that GPU
 * current; make that first call outside a graph capture. */
int32_t madd_multi_tensor_step_noalloc(int32_t ntensors, void* const* w, const int32_t* wfmt,
                                       void* const* scales, uint16_t* const* copy,
                                       const void* const* g, int32_t gfmt, void* const* m,
                                       void* const* v, void* const* ve, int32_t sfmt,
                                       const int64_t* numel, int64_t index_base,
                                       const madd_hparams* hp, void* stream);

/* Hyper-parameters read from device memory when the kernels run, so that a
 * captured step (HIP graph) can be replayed step after step: the caller
 * updates the device copy between replays instead of capturing again.
 *
 * madd_scalars_bytes(): size in bytes of the prepared scalars (the fp32
 *   coefficients of Algorithm 2 for one step -- beta1, beta2, 1 - beta1,
 *   1 - beta2, the bias-corrected eta_a / (1 - beta1^t) and 1 / (1 - beta2^t),
 *   eta_m, eps, tau, g_max, the u_m clip bounds, w_max -- and the Philox key
 *   and counter word: seed and t); the layout is internal to the library.
 * madd_prepare_scalars(hp, out): validates hp as the step entry points do and
 *   writes its scalars to `out` (HOST memory of madd_scalars_bytes() bytes),
 *   computed exactly as madd_step computes them, so a step that reads them
 *   gives the same bits as one passed hp.  MADD_EINVAL for a NULL `out` or
 *   an invalid hp.
 * madd_multi_tensor_step_dev(...): madd_multi_tensor_step, except that the
 *   kernels read the scalars from `dev_scalars` (DEVICE memory, 4-byte
 *   aligned, madd_scalars_bytes() bytes written from madd_prepare_scalars'
 *   output) at run time.  `hp` is still validated and fixes what selects the
 *   kernels -- the rounding mode and whether g_max / w_max are finite -- which
 *   the prepared scalars must share; its other fields are not used.  The
 *   caller keeps dev_scalars allocated while launches that read it are in
 *   flight.  MADD_EINVAL for a NULL dev_scalars, MADD_EALIGN when it is not
 *   4-byte aligned; otherwise as madd_multi_tensor_step. */
int64_t madd_scalars_bytes(void);
int32_t madd_prepare_scalars(const madd_hparams* hp, void* out);
int32_t madd_multi_tensor_step_dev(int32_t ntensors, void* const* w, const int32_t* wfmt,
                                   void* const* scales, uint16_t* const* copy,
                                   const void* const* g, int32_t gfmt,
                                   void* const* m, void* const* v, void* const* ve,
                                   int32_t sfmt, const int64_t* numel, int64_t index_base,
                                   const madd_hparams* hp, const void* dev_scalars,
                                   void* stream);

/* One step of the moment-free update rules of Appendix B's BF16-stored
 * matrix-fitting diagnostic, on one tensor of n elements:
 *   additive        u_a = -eta_a g
 *   multiplicative  u_m = clip(-eta_m g_e / max(|w|, tau)),  g_e = ln2 w g,
 *                   clip to [-(r_max - eps0), r_max] and the d_mult_max cap
 *   combined        w <- clamp_{w_max}(w + w u_m + u_a), rounded into wfmt
 * (eta_m = 0 gives the additive rule, eta_a = 0 the multiplicative one).
 * No optimizer state.  w: device weight codes of format wfmt, in place;
 * g: device gradient of format gfmt; index_base, rounding and seed as in
 * madd_step; hp's beta1, beta2, eps, g_max and bias_correction are validated
 * but unused.  Unscaled formats only (MXFP4, NVFP4, NVFP4_CURRENT:
 * MADD_EINVAL).  Errors as in
 * madd_step. */
int32_t madd_plain_step(void* w, int32_t wfmt, const void* g, int32_t gfmt, int64_t n,
                        int64_t index_base, const madd_hparams* hp, void* stream);

/* Gradient of Appendix B's diagnostic loss on sampled entries: the loss is
 * (1/B) sum over the B sampled entries k of c_i (w_i - w*_i)^4 (i the entry
 * drawn as sample k, with replacement), whose gradient is
 *   g_i = ((s_i d_i) d_i) d_i,  d_i = w_i - w*_i,  s_i = (fp32(4/B) cnt_i) c_i,
 * cnt_i = number of samples equal to i, evaluated in fp32 in this order.
 * w      : device weight codes of format wfmt (BF16, FP8 E4M3 / E5M2 or FP32;
 *          4-bit formats are MADD_EINVAL), n elements, decoded exactly.
 * target, c : device fp32 arrays of n elements (w* and the per-entry scale).
 * idx    : device int64 array of the B = batch sampled entries (the random
 *          draws are the caller's); entries outside [0, n) are skipped.
 * counts : device int32 workspace of n elements (overwritten with cnt).
 * g      : device fp32 output of n elements.
 * Three launches on `stream` (clear counts, count with integer atomics, the
 * gradient); results do not depend on the order of the samples.  Arrays
 * must not overlap (MADD_EINVAL). */
int32_t madd_toy_gradient(const void* w, int32_t wfmt, const float* target, const float* c,
                          const int64_t* idx, int64_t batch, int64_t n, int32_t* counts,
                          float* g, void* stream);

/* Human-readable name of a status code (static storage; never NULL). */
const char* madd_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* MADD_H */
