// M+Adam optimizer step for AMD Instinct MI355X (gfx950): HIP kernels and the
// C ABI declared in include/madd.h.
//
// One fused, HBM-bound elementwise pass per step.  Per element it reads the
// weight code, the gradient and the three moments (fp32 or bf16), updates them,
// forms the additive update u_a and the multiplicative update u_m
// (Algorithm 1, with the optional clamps of Algorithm 2), combines
// w + w u_m + u_a, and rounds the result back into the storage format (the
// FP32-step / low-precision-storage round trip of Appendix B), to nearest-even
// or stochastically with a Philox4x32-10 draw keyed by (seed, step, element).
// Storage formats: bf16, FP8 E4M3 / E5M2 (optionally with FP16 scales per
// 128-element block), and for the 4-bit master-weight setting of Section 4.2
// NVFP4 (E2M1 with an E4M3 scale per 16 elements and an fp32 scale per
// tensor) and MXFP4 (E2M1 with an E8M0 scale per 32 elements).
//
// Layout of work: a launch covers a list of tensors.  The element space of
// each tensor is cut into chunks; one workgroup (256 threads, four wave64s)
// owns one chunk.  A chunk is made of tiles of 2048 elements, each split into
// two sub-tiles of 1024; thread t handles the four consecutive elements
// [4t, 4t+4) of both sub-tiles, so every load and store instruction of a
// wave covers one contiguous span (1 KiB for fp32 arrays); a tile's loads
// are issued together, and in whole tiles the arithmetic of sub-tile A waits
// only for A's loads.  A workgroup finds its
// tensor by a binary search over the descriptor table (uniform, scalar
// loads).  Loads and stores of the streamed arrays are non-temporal global
// accesses: nothing is reused within a step.
//
// Random draws: the eight elements of an aligned group share one Philox
// block.  Lanes 2k and 2k+1 cover one group of sub-tile A and one of
// sub-tile B; the even lane computes the A block, the odd lane the B block,
// and each hands the half its partner needs across a DPP lane swap, so a
// block is computed once per eight elements.
//
// Arithmetic: FP32, one fixed operation order (step_elem), built with
// -ffp-contract=off so that only the written fmaf calls fuse; division and
// square root are the correctly rounded IEEE operations; fp32 denormals are
// kept.  The result is bit-identical on every launch shape.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <cmath>
#include <string.h>

#include <atomic>
#include <mutex>
#include <tuple>
#include <utility>
#include <vector>

#include "madd.h"
#include "table_cache.h"

// The library is built from this one source compiled as several parts
// (-DMADD_PART=k, in parallel): part 0 holds the host code, the ABI and the
// set-up kernels; parts 1-8 each instantiate the step kernels of one weight
// format (block-scaled FP8 separately from unscaled), part 9 those of NVFP4
// with current scaling.  Without MADD_PART everything is compiled as one
// unit.
#ifndef MADD_PART
#define MADD_PART -1
#endif
#define MADD_IN_PART(k) (MADD_PART < 0 || MADD_PART == (k))

namespace madd_detail {

constexpr int kThreads = 256;
constexpr int kQuad = 4;                     // consecutive elements per thread and sub-tile
constexpr int kSub = kThreads * kQuad;       // 1024 elements per sub-tile
constexpr int kTile = 2 * kSub;              // sub-tiles A and B
constexpr int kTilesPerChunk = 1;
constexpr int64_t kChunk = (int64_t)kTile * kTilesPerChunk;
constexpr int kBlock = 128;                  // block-scaled FP8 block length
constexpr int kMxBlock = 32;                 // MXFP4 block length (OCP MX)
constexpr int kNvBlock = 16;                 // NVFP4 block length

// ---------------------------------------------------------------------------
// Scalars and descriptors
// ---------------------------------------------------------------------------

struct Scalars {
  float B1, B2, OMB1, OMB2;  // b1, b2, 1-b1, 1-b2
  float SA;                  // eta_a / (1 - b1^t)   (eta_a without bias correction)
  float IBC2;                // 1 / (1 - b2^t)       (1 without bias correction)
  float LRM, EPS, TAU, GMAX; // eta_m, eps, tau, g_max
  float ULO, UHI;            // u_m clip bounds
  float WMAX;                // final weight clamp
  uint32_t key0, key1;       // Philox key = seed
  uint32_t t;                // step (Philox counter word 2)
};

struct TensorDesc {
  void* w;
  const void* g;
  void* m;   // moments: fp32, or bf16 codes
  void* v;
  void* ve;
  void* scales;    // FP16 codes (block FP8), E8M0 codes (MXFP4), or fp32 tensor
                   // scale then E4M3 codes (NVFP4)
  uint16_t* copy;  // optional bf16 compute copy of the new weights
  int64_t n;       // elements
  int64_t gbase;   // global index of element 0
  int64_t chunk0;  // first chunk of this tensor within the launch
  int32_t vec_ok;  // buffers 16-byte aligned and gbase a multiple of 8
  int32_t pad;
};

// Chunk ranges of one launch of NVFP4 current scaling (nvcs_step_kernel):
// pass 1 over [a1, a1 + n1), pass 2 over [a2, a2 + n2).
struct NvcsSpan {
  int64_t a1, n1, a2, n2;
};

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw; SC'11)
// ---------------------------------------------------------------------------

__device__ __forceinline__ u4 philox10(u4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;  // one v_mad_u64_u32 each
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = u4{(uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1,
           (uint32_t)p0};
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// 128 random bits for the group of eight elements j = idx >> 3 on a stream:
// 0 rounds the weights, 1, 2, 3 the stochastically rounded bf16 moments
// m, v, v_e.
__device__ __forceinline__ u4 draw_group(uint64_t j, const Scalars& s, uint32_t stream = 0u) {
  return philox10(u4{(uint32_t)j, (uint32_t)(j >> 32), s.t, stream}, s.key0, s.key1);
}

__device__ __forceinline__ uint32_t lane16(u4 r, uint32_t lane) {
  const uint32_t word = (lane < 2) ? r.x : (lane < 4) ? r.y : (lane < 6) ? r.z : r.w;
  return (lane & 1u) ? (word >> 16) : (word & 0xFFFFu);
}

// 16-bit draw of a single element.
__device__ __forceinline__ uint32_t draw_one(uint64_t idx, const Scalars& s, uint32_t stream = 0u) {
  return lane16(draw_group(idx >> 3, s, stream), (uint32_t)(idx & 7u));
}

// ---------------------------------------------------------------------------
// Storage-format codecs (bit level)
// ---------------------------------------------------------------------------

enum : int { WF_BF16 = 0, WF_E4M3 = 1, WF_E5M2 = 2, WF_FP32 = 3, WF_MXFP4 = 4, WF_NVFP4 = 5 };
enum : int { GF_FP32 = 0, GF_BF16 = 1 };
// storage of the moments: fp32, bf16 rounded to nearest-even, bf16 rounded
// stochastically (streams 1, 2, 3)
enum : int { SF_FP32 = 0, SF_BF16 = 1, SF_BF16_SR = 2 };

__device__ __forceinline__ float dec_bf16(uint32_t c) { return __uint_as_float(c << 16); }

// BF16 encoding with gfx950's conversion instructions.  v_cvt_pk_bf16_f32
// rounds to nearest-even; v_cvt_sr_bf16_f32 adds the high 16 bits of its
// random operand to the 16 discarded bits and truncates, which with the draw
// placed there is the stochastic rule above (carry into the kept half with
// probability low16 / 2^16).  Both match the integer definitions bit for bit
// on every non-NaN fp32 (checked exhaustively on the device) and turn a NaN
// into a quieted truncation of it, so a NaN is first replaced by the
// canonical 0x7FC00000, whose conversion is the canonical code 0x7FC0.
typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
typedef short s2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float canon_nan(float x) {
  return (x == x) ? x : __uint_as_float(0x7FC00000u);
}

// Two values, `a` in the low half.
__device__ __forceinline__ uint32_t enc_bf16x2(float a, float b, bool sr, uint32_t ra,
                                               uint32_t rb) {
  if (sr) {
    s2v r = __builtin_amdgcn_cvt_sr_bf16_f32(s2v{0, 0}, canon_nan(a), ra << 16, false);
    r = __builtin_amdgcn_cvt_sr_bf16_f32(r, canon_nan(b), rb << 16, true);
    return __builtin_bit_cast(uint32_t, r);
  }
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2v{canon_nan(a), canon_nan(b)}, bf2v));
}

__device__ __forceinline__ uint32_t enc_bf16(float x, bool sr, uint32_t r16) {
  if (sr) {
    const s2v r = __builtin_amdgcn_cvt_sr_bf16_f32(s2v{0, 0}, canon_nan(x), r16 << 16, false);
    return __builtin_bit_cast(uint32_t, r) & 0xFFFFu;
  }
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)canon_nan(x));
}

// Minifloat description: M mantissa bits, exponent bias, minimum normal
// exponent, largest finite magnitude and its code, NaN code.
template <int WF>
struct Mini;
template <>
struct Mini<WF_E4M3> {
  static constexpr int M = 3, BIAS = 7, EMIN = -6;
  static constexpr float MAXV = 448.0f;
  static constexpr uint32_t MAXCODE = 0x7Eu, NANCODE = 0x7Fu;
  static constexpr uint32_t RESCALE_BITS = (127u + 127u - 7u) << 23;  // 2^(127 - BIAS)
};
template <>
struct Mini<WF_E5M2> {
  static constexpr int M = 2, BIAS = 15, EMIN = -14;
  static constexpr float MAXV = 57344.0f;
  static constexpr uint32_t MAXCODE = 0x7Bu, NANCODE = 0x7Fu;
  static constexpr uint32_t RESCALE_BITS = (127u + 127u - 15u) << 23;
};

// Branch-free decode: the code's exponent and mantissa fields, placed at the
// top of an fp32's exponent and mantissa fields, read as 2^(E-127) (1.M) for
// E > 0 and as the fp32 subnormal M 2^(-149+23-M) for E = 0; one multiply by
// 2^(127 - BIAS) rescales both exactly (fp32 denormals are kept).
template <int WF>
__device__ __forceinline__ float dec_fp8(uint32_t c) {
  using F = Mini<WF>;
  const uint32_t mag = c & 0x7Fu;
  float v = __uint_as_float(mag << (23 - F::M)) * __uint_as_float(F::RESCALE_BITS);
  if constexpr (WF == WF_E4M3) {
    v = (mag == 0x7Fu) ? __uint_as_float(0x7FC00000u) : v;
  } else {  // E5M2: all-ones exponent is Inf (mantissa 0) or NaN
    v = (mag >= 0x7Cu) ? __uint_as_float((mag & 3u) ? 0x7FC00000u : 0x7F800000u) : v;
  }
  return __uint_as_float(__float_as_uint(v) | ((c & 0x80u) << 24));
}

// Value-domain rounding onto a minifloat grid: scale |x| so that the grid
// spacing of its binade is 1, round to an integer k (ties to even, or
// stochastically), and assemble the code from the spacing exponent and k.
// A k that reaches the next power of two lands on the next binade's code.
// `val` receives the rounded magnitude k 2^se (exact), for callers that need
// the stored value as well as its code.
template <int M, int BIAS, int EMIN>
__device__ __forceinline__ uint32_t round_mini(float a, bool sr, uint32_t r16, float& val) {
  const int e = (int)((__float_as_uint(a) >> 23) & 0xFFu) - 127;
  const int se = (e > EMIN ? e : EMIN) - M;  // exponent of the grid spacing
  const float q = ldexpf(a, -se);            // exact; q < 2^(M+1)
  float k;
  if (sr) {
    k = floorf(q);
    const uint32_t f16 = (uint32_t)((q - k) * 65536.0f);  // exact
    if (f16 + r16 >= 65536u) k += 1.0f;
  } else {
    k = rintf(q);
  }
  val = ldexpf(k, se);
  return ((uint32_t)(se + M + BIAS - 1) << M) + (uint32_t)k;
}
template <int M, int BIAS, int EMIN>
__device__ __forceinline__ uint32_t round_mini(float a, bool sr, uint32_t r16) {
  float unused;
  return round_mini<M, BIAS, EMIN>(a, sr, r16, unused);
}

// Branch-free: |x| is first clamped to the largest finite value (Inf and
// finite overflow saturate; a NaN takes the clamp's value and is replaced by
// the NaN code at the end).  The largest value is a grid point of its binade,
// whose spacing then bounds every rounding of a clamped |x| by it, so no
// code beyond the largest finite one can arise.
// `val` receives the value of the returned code.
template <int WF>
__device__ __forceinline__ uint32_t enc_fp8(float x, bool sr, uint32_t r16, float& val) {
  using F = Mini<WF>;
  const uint32_t sign = (__float_as_uint(x) >> 24) & 0x80u;
  float a = fabsf(x);
  a = a < F::MAXV ? a : F::MAXV;
  float mag;
  const uint32_t c = round_mini<F::M, F::BIAS, F::EMIN>(a, sr, r16, mag);
  val = (x == x) ? __uint_as_float(__float_as_uint(mag) | (sign << 24)) : x;
  return (x == x) ? (sign | c) : F::NANCODE;
}
template <int WF>
__device__ __forceinline__ uint32_t enc_fp8(float x, bool sr, uint32_t r16) {
  float unused;
  return enc_fp8<WF>(x, sr, r16, unused);
}

// FP16 codes of the block scales (IEEE: RNE, overflow to Inf).
__device__ __forceinline__ float dec_fp16(uint32_t c) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)c);
}

__device__ __forceinline__ uint32_t enc_fp16_rne(float x) {
  const uint32_t sign = (__float_as_uint(x) >> 16) & 0x8000u;
  const float a = fabsf(x);
  if (!(a == a)) return 0x7E00u;
  if (a >= 65536.0f) return sign | 0x7C00u;
  uint32_t c = round_mini<10, 15, -14>(a, false, 0u);
  c = c > 0x7C00u ? 0x7C00u : c;
  return sign | c;
}

// MXFP4 (OCP Microscaling): E2M1 elements sharing an E8M0 power-of-two scale.
// E2M1 magnitudes of codes 0..7, doubled (0 1 2 3 4 6 8 12), one per nibble.
__device__ __forceinline__ float dec_e2m1(uint32_t c) {
  const float mag = (float)((0xC8643210u >> (4u * (c & 7u))) & 0xFu) * 0.5f;
  return (c & 8u) ? -mag : mag;
}

// x already divided by the block scale and finite; saturates at +-6 (6 is a
// grid point, so rounding a clamped |x| never passes code 7).
// `val` receives the value of the returned code.
__device__ __forceinline__ uint32_t enc_e2m1(float x, bool sr, uint32_t r16, float& val) {
  const uint32_t sign = (__float_as_uint(x) >> 28) & 0x8u;
  float a = fabsf(x);
  a = a < 6.0f ? a : 6.0f;
  float mag;
  const uint32_t c = round_mini<1, 1, 0>(a, sr, r16, mag);  // 1 mantissa bit, bias 1, min exponent 0
  val = __uint_as_float(__float_as_uint(mag) | (sign << 28));
  return sign | c;
}
__device__ __forceinline__ uint32_t enc_e2m1(float x, bool sr, uint32_t r16) {
  float unused;
  return enc_e2m1(x, sr, r16, unused);
}

// E8M0: 2^(c - 127); code 0 is the fp32 subnormal 2^-127; code 255 is NaN.
__device__ __forceinline__ float dec_e8m0(uint32_t c) {
  if (c == 0xFFu) return __uint_as_float(0x7FC00000u);
  return __uint_as_float(c == 0u ? 0x00400000u : (c << 23));
}

// Scale code of a block whose largest |w'| has the raw bits amax_bits:
// s = floor(log2 amax) - 2 clamped to [-127, 127] (code s + 127); 1.0 for an
// all-zero block; NaN when the block holds a non-finite value.  For a normal
// amax floor(log2 amax) is its unbiased exponent field, so the code is the
// biased field minus 2; a subnormal amax clamps to code 0.
__device__ __forceinline__ uint32_t mx_scale(uint32_t amax_bits) {
  if (amax_bits >= 0x7F800000u) return 0xFFu;
  if (amax_bits == 0u) return 127u;
  const uint32_t ef = amax_bits >> 23;
  return ef > 2u ? ef - 2u : 0u;
}

// 2^-s for a finite scale code (a normal float for every code the rule
// produces, 0..252), so that w' * 2^-s is the exact quotient w' / 2^s.
__device__ __forceinline__ float mx_inv_scale(uint32_t code) {
  return __uint_as_float((code < 0xFFu ? 254u - code : 127u) << 23);
}

template <int WF>
__device__ __forceinline__ uint32_t encode(float x, bool sr, uint32_t r16) {
  if constexpr (WF == WF_BF16) return enc_bf16(x, sr, r16);
  else if constexpr (WF == WF_FP32) return (x == x) ? __float_as_uint(x) : 0x7FC00000u;
  else return enc_fp8<WF>(x, sr, r16);
}

template <int WF>
__device__ __forceinline__ float decode(uint32_t c) {
  if constexpr (WF == WF_BF16) return dec_bf16(c);
  else if constexpr (WF == WF_FP32) return __uint_as_float(c);
  else if constexpr (WF == WF_MXFP4 || WF == WF_NVFP4) return dec_e2m1(c);  // before the scale
  else return dec_fp8<WF>(c);
}

// Block-scale rule: scale = RNE_fp16(amax / FMAX), with 1.0 for an all-zero
// block, the smallest subnormal on underflow, the largest finite value on
// overflow and NaN for a block holding a non-finite value.  `amax_bits` is the
// largest |w'| as raw bits (unsigned order = magnitude order, NaN above Inf).
template <int WF>
__device__ __forceinline__ uint32_t block_scale(uint32_t amax_bits) {
  if (amax_bits >= 0x7F800000u) return 0x7E00u;
  if (amax_bits == 0u) return 0x3C00u;
  uint32_t s = enc_fp16_rne(__uint_as_float(amax_bits) / Mini<WF>::MAXV);
  if (s == 0u) s = 1u;
  if (s == 0x7C00u) s = 0x7BFFu;
  return s;
}

// ---------------------------------------------------------------------------
// The per-element step (fixed FP32 operation order)
// ---------------------------------------------------------------------------

__device__ __forceinline__ float clampf(float x, float lo, float hi) {
  return x < lo ? lo : (x > hi ? hi : x);  // NaN passes through
}

// CLAMP = false drops the g_max and w_max clamps; the host selects it only
// when both bounds are +infinity, where the clamps are the identity (also for
// NaN and infinite arguments), so the results are the same bits.
template <bool CLAMP>
__device__ __forceinline__ float step_elem(float w, float g, float& m, float& v, float& ve,
                                           const Scalars& s) {
  const float LN2 = 0.693147182464599609375f;  // fp32(ln 2)
  // additive branch
  m = fmaf(s.B1, m, s.OMB1 * g);
  v = fmaf(s.B2, v, s.OMB2 * (g * g));
  const float ua = -((s.SA * m) / (sqrtf(v * s.IBC2) + s.EPS));
  // multiplicative branch: exponent gradient and its second moment
  const float ge = (LN2 * w) * g;
  ve = fmaf(s.B2, ve, s.OMB2 * (ge * ge));
  float r = ge / (sqrtf(ve * s.IBC2) + s.EPS);
  if (CLAMP) r = clampf(r, -s.GMAX, s.GMAX);
  const float ut = -(s.LRM * r);
  // relative conversion and clip
  const float aw = fabsf(w);
  const float rho = aw > s.TAU ? aw : s.TAU;
  const float um = clampf(ut / rho, s.ULO, s.UHI);
  // combine, optional final clamp
  const float wn = fmaf(w, um, w) + ua;
  return CLAMP ? clampf(wn, -s.WMAX, s.WMAX) : wn;
}

// ---------------------------------------------------------------------------
// Global-memory accesses of four consecutive elements
// ---------------------------------------------------------------------------

#define GLOBAL __attribute__((address_space(1)))

template <typename T>
__device__ __forceinline__ T ldg(const void* p) {
  return __builtin_nontemporal_load((const GLOBAL T*)p);
}
template <typename T>
__device__ __forceinline__ void stg(void* p, T x) {
  __builtin_nontemporal_store(x, (GLOBAL T*)p);
}

template <int WF>
struct WQuad;
template <>
struct WQuad<WF_BF16> {  // 4 x 16 bits
  u2 raw;
  __device__ __forceinline__ void load(const void* p, int64_t e) { raw = ldg<u2>((const uint16_t*)p + e); }
  __device__ __forceinline__ uint32_t code(int k) const { return (raw[k >> 1] >> (16 * (k & 1))) & 0xFFFFu; }
  __device__ __forceinline__ void set(int k, uint32_t c) {
    raw[k >> 1] = (k & 1) ? ((raw[k >> 1] & 0xFFFFu) | (c << 16)) : ((raw[k >> 1] & 0xFFFF0000u) | c);
  }
  __device__ __forceinline__ void store(void* p, int64_t e) const { stg<u2>((uint16_t*)p + e, raw); }
};
template <int WF>
struct WQuad8 {  // 4 x 8 bits
  uint32_t raw;
  __device__ __forceinline__ void load(const void* p, int64_t e) { raw = ldg<uint32_t>((const uint8_t*)p + e); }
  __device__ __forceinline__ uint32_t code(int k) const { return (raw >> (8 * k)) & 0xFFu; }
  __device__ __forceinline__ void set(int k, uint32_t c) { raw = (raw & ~(0xFFu << (8 * k))) | (c << (8 * k)); }
  __device__ __forceinline__ void store(void* p, int64_t e) const { stg<uint32_t>((uint8_t*)p + e, raw); }
};
template <>
struct WQuad<WF_E4M3> : WQuad8<WF_E4M3> {};
template <>
struct WQuad<WF_E5M2> : WQuad8<WF_E5M2> {};
template <>
struct WQuad<WF_MXFP4> {  // 4 x 4 bits: two bytes, element 2k in the low nibble of byte k
  uint32_t raw;
  __device__ __forceinline__ void load(const void* p, int64_t e) {
    raw = ldg<uint16_t>((const uint8_t*)p + (e >> 1));
  }
  __device__ __forceinline__ uint32_t code(int k) const { return (raw >> (4 * k)) & 0xFu; }
  __device__ __forceinline__ void set(int k, uint32_t c) { raw = (raw & ~(0xFu << (4 * k))) | (c << (4 * k)); }
  __device__ __forceinline__ void store(void* p, int64_t e) const {
    stg<uint16_t>((uint8_t*)p + (e >> 1), (uint16_t)raw);
  }
};
template <>
struct WQuad<WF_NVFP4> : WQuad<WF_MXFP4> {};  // the same packed E2M1 payloads
template <>
struct WQuad<WF_FP32> {  // 4 x 32 bits
  u4 raw;
  __device__ __forceinline__ void load(const void* p, int64_t e) { raw = ldg<u4>((const uint32_t*)p + e); }
  __device__ __forceinline__ uint32_t code(int k) const { return raw[k]; }
  __device__ __forceinline__ void set(int k, uint32_t c) { raw[k] = c; }
  __device__ __forceinline__ void store(void* p, int64_t e) const { stg<u4>((uint32_t*)p + e, raw); }
};

template <int GF>
__device__ __forceinline__ f4 ld4g(const void* p, int64_t e) {
  if constexpr (GF == GF_FP32) {
    return ldg<f4>((const float*)p + e);
  } else {
    const u2 r = ldg<u2>((const uint16_t*)p + e);
    return f4{dec_bf16(r.x & 0xFFFFu), dec_bf16(r.x >> 16), dec_bf16(r.y & 0xFFFFu),
              dec_bf16(r.y >> 16)};
  }
}

template <int GF>
__device__ __forceinline__ float ld1g(const void* p, int64_t e) {
  if constexpr (GF == GF_FP32) return ((const float*)p)[e];
  else return dec_bf16(((const uint16_t*)p)[e]);
}

template <int WF>
__device__ __forceinline__ uint32_t ld1w(const void* p, int64_t e) {
  if constexpr (WF == WF_BF16) return ((const uint16_t*)p)[e];
  else if constexpr (WF == WF_FP32) return ((const uint32_t*)p)[e];
  else return ((const uint8_t*)p)[e];
}
template <int WF>
__device__ __forceinline__ void st1w(void* p, int64_t e, uint32_t c) {
  if constexpr (WF == WF_BF16) ((uint16_t*)p)[e] = (uint16_t)c;
  else if constexpr (WF == WF_FP32) ((uint32_t*)p)[e] = c;
  else ((uint8_t*)p)[e] = (uint8_t)c;
}

// Moments as stored: fp32, or bf16 codes (decoded exactly; stored rounded to
// nearest, ties to even, or stochastically with the given draws).
template <int SF>
__device__ __forceinline__ f4 ld4s(const void* p, int64_t e) {
  if constexpr (SF == SF_FP32) {
    return ldg<f4>((const float*)p + e);
  } else {
    const u2 r = ldg<u2>((const uint16_t*)p + e);
    return f4{dec_bf16(r.x & 0xFFFFu), dec_bf16(r.x >> 16), dec_bf16(r.y & 0xFFFFu),
              dec_bf16(r.y >> 16)};
  }
}
template <int SF>
__device__ __forceinline__ void st4s(void* p, int64_t e, f4 x, const uint32_t (&r16)[4]) {
  if constexpr (SF == SF_FP32) {
    stg<f4>((float*)p + e, x);
  } else {
    constexpr bool sr = SF == SF_BF16_SR;
    const u2 r = u2{enc_bf16x2(x.x, x.y, sr, r16[0], r16[1]),
                    enc_bf16x2(x.z, x.w, sr, r16[2], r16[3])};
    stg<u2>((uint16_t*)p + e, r);
  }
}
template <int SF>
__device__ __forceinline__ float ld1s(const void* p, int64_t e) {
  if constexpr (SF == SF_FP32) return ((const float*)p)[e];
  else return dec_bf16(((const uint16_t*)p)[e]);
}
template <int SF>
__device__ __forceinline__ void st1s(void* p, int64_t e, float x, uint32_t r16) {
  if constexpr (SF == SF_FP32) ((float*)p)[e] = x;
  else ((uint16_t*)p)[e] = (uint16_t)enc_bf16(x, SF == SF_BF16_SR, r16);
}

// The draws of the three moments of four elements (stochastic bf16 moments).
struct MDraws {
  uint32_t m[4], v[4], ve[4];
};

// One sub-tile's worth of a thread's inputs: four consecutive elements.
template <int WF>
struct Quad {
  WQuad<WF> w;
  f4 g, m, v, ve;
};

template <int WF, int GF, int SF>
__device__ __forceinline__ void load_quad(Quad<WF>& q, const TensorDesc& d, int64_t e) {
  q.w.load(d.w, e);
  q.g = ld4g<GF>(d.g, e);
  q.m = ld4s<SF>(d.m, e);
  q.v = ld4s<SF>(d.v, e);
  q.ve = ld4s<SF>(d.ve, e);
}

template <int WF, int SF>
__device__ __forceinline__ void store_quad(const Quad<WF>& q, const TensorDesc& d, int64_t e,
                                           const MDraws& md) {
  q.w.store(d.w, e);
  st4s<SF>(d.m, e, q.m, md.m);
  st4s<SF>(d.v, e, q.v, md.v);
  st4s<SF>(d.ve, e, q.ve, md.ve);
}

// The bf16 compute copy (rounded to nearest-even) of four new stored weights,
// given as values (block-scaled: payload value already multiplied by the
// block's factor).
__device__ __forceinline__ void store_copy_values(const float (&v)[4], uint16_t* copy, int64_t e) {
  stg<u2>(copy + e, u2{enc_bf16x2(v[0], v[1], false, 0u, 0u), enc_bf16x2(v[2], v[3], false, 0u, 0u)});
}

template <int WF>
__device__ __forceinline__ void store_copy(const WQuad<WF>& w, uint16_t* copy, int64_t e) {
  float v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) v[k] = decode<WF>(w.code(k));
  store_copy_values(v, copy, e);
}

// Swap a value with the neighbouring lane (DPP quad_perm [1,0,3,2]).
__device__ __forceinline__ uint32_t swap_lane_pair(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);
}

// The 16-bit draws of a thread's four A elements and four B elements when
// the groups are 8-aligned in the global index (gA = global index of the
// pair's first A element, a multiple of 8; the pair's B group is gA + 1024).
// Every lane of the wave must call this (lane swap).
template <bool SR>
__device__ __forceinline__ void draws_aligned(uint64_t gA, const Scalars& s, uint32_t (&rA)[4],
                                              uint32_t (&rB)[4], uint32_t stream = 0u) {
  if constexpr (!SR) {
#pragma unroll
    for (int k = 0; k < 4; ++k) rA[k] = rB[k] = 0u;
  } else {
    const bool odd = (threadIdx.x & 1u) != 0u;
    const u4 P = draw_group((gA >> 3) + (odd ? (uint64_t)(kSub / 8) : 0u), s, stream);
    // even lane keeps words x,y of its A block and sends z,w; odd lane keeps
    // z,w of its B block and sends x,y
    const uint32_t r0 = swap_lane_pair(odd ? P.x : P.z);
    const uint32_t r1 = swap_lane_pair(odd ? P.y : P.w);
    const uint32_t a0 = odd ? r0 : P.x, a1 = odd ? r1 : P.y;
    const uint32_t b0 = odd ? P.z : r0, b1 = odd ? P.w : r1;
    rA[0] = a0 & 0xFFFFu; rA[1] = a0 >> 16; rA[2] = a1 & 0xFFFFu; rA[3] = a1 >> 16;
    rB[0] = b0 & 0xFFFFu; rB[1] = b0 >> 16; rB[2] = b1 & 0xFFFFu; rB[3] = b1 >> 16;
  }
}

// Draws of four consecutive elements starting at an arbitrary global index.
template <bool SR>
__device__ __forceinline__ void draws_any(uint64_t g0, const Scalars& s, uint32_t (&r)[4],
                                          uint32_t stream = 0u) {
  if constexpr (!SR) {
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = 0u;
  } else {
    const uint32_t off = (uint32_t)(g0 & 7u);
    const u4 a = draw_group(g0 >> 3, s, stream);
    if (off <= 4u) {
#pragma unroll
      for (int k = 0; k < 4; ++k) r[k] = lane16(a, off + (uint32_t)k);
    } else {
      const u4 b = draw_group((g0 >> 3) + 1u, s, stream);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t l = off + (uint32_t)k;
        r[k] = l < 8u ? lane16(a, l) : lane16(b, l - 8u);
      }
    }
  }
}

// Moment draws of a lane pair's A and B groups (see draws_aligned; every lane
// of the pair must call), or of four elements at any index.
template <int SF>
__device__ __forceinline__ void mdraws_aligned(uint64_t gA, const Scalars& s, MDraws& a, MDraws& b) {
  if constexpr (SF == SF_BF16_SR) {
    draws_aligned<true>(gA, s, a.m, b.m, 1u);
    draws_aligned<true>(gA, s, a.v, b.v, 2u);
    draws_aligned<true>(gA, s, a.ve, b.ve, 3u);
  }
}
template <int SF>
__device__ __forceinline__ void mdraws_any(uint64_t g0, const Scalars& s, MDraws& a) {
  if constexpr (SF == SF_BF16_SR) {
    draws_any<true>(g0, s, a.m, 1u);
    draws_any<true>(g0, s, a.v, 2u);
    draws_any<true>(g0, s, a.ve, 3u);
  }
}

template <int WF, bool SR, bool CLAMP>
__device__ __forceinline__ void step_quad(Quad<WF>& q, const uint32_t (&r)[4], const Scalars& s) {
  float wn[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float m = q.m[k], v = q.v[k], ve = q.ve[k];
    wn[k] = step_elem<CLAMP>(decode<WF>(q.w.code(k)), q.g[k], m, v, ve, s);
    q.m[k] = m;
    q.v[k] = v;
    q.ve[k] = ve;
  }
  if constexpr (WF == WF_BF16) {  // two codes per conversion
    q.w.raw = u2{enc_bf16x2(wn[0], wn[1], SR, r[0], r[1]), enc_bf16x2(wn[2], wn[3], SR, r[2], r[3])};
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) q.w.set(k, encode<WF>(wn[k], SR, r[k]));
  }
}

// ---------------------------------------------------------------------------
// Step kernel
// ---------------------------------------------------------------------------

__device__ __forceinline__ TensorDesc find_tensor(const TensorDesc* __restrict__ table, int ntab,
                                                  const TensorDesc& single, int64_t chunk) {
  if (ntab == 0) return single;
  int lo = 0, hi = ntab - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (table[mid].chunk0 <= chunk) lo = mid;
    else hi = mid - 1;
  }
  return table[lo];
}

// Elements [b, e) one at a time (tails and unaligned buffers).
template <int WF, int GF, int SF, bool SR, bool CLAMP, bool COPY>
__device__ __forceinline__ void step_scalar_range(const TensorDesc& d, int64_t b, int64_t e,
                                                  const Scalars& s) {
  for (int64_t i = b; i < e; ++i) {
    float m = ld1s<SF>(d.m, i), v = ld1s<SF>(d.v, i), ve = ld1s<SF>(d.ve, i);
    const float w = decode<WF>(ld1w<WF>(d.w, i));
    const float g = ld1g<GF>(d.g, i);
    const float wn = step_elem<CLAMP>(w, g, m, v, ve, s);
    const uint64_t gi = (uint64_t)(d.gbase + i);
    const uint32_t r16 = SR ? draw_one(gi, s) : 0u;
    const uint32_t code = encode<WF>(wn, SR, r16);
    st1w<WF>(d.w, i, code);
    if (COPY && d.copy) d.copy[i] = (uint16_t)enc_bf16(decode<WF>(code), false, 0u);
    constexpr bool ssr = SF == SF_BF16_SR;
    st1s<SF>(d.m, i, m, ssr ? draw_one(gi, s, 1u) : 0u);
    st1s<SF>(d.v, i, v, ssr ? draw_one(gi, s, 2u) : 0u);
    st1s<SF>(d.ve, i, ve, ssr ? draw_one(gi, s, 3u) : 0u);
  }
}

// Waves per SIMD the step kernel asks the compiler for: with bf16 moments
// (rounded to nearest, no compute copy) the step is bound by VALU issue and
// fits a fifth wave (at most 96 VGPRs) without spilling; elsewhere the
// compiler's own choice stands (a tighter bound spills).
template <int SF, bool COPY>
constexpr int kStepWaves = (SF == SF_BF16 && !COPY) ? 5 : 1;

template <int WF, int GF, int SF, bool SR, bool CLAMP, bool COPY>
__global__ __launch_bounds__(kThreads, (kStepWaves<SF, COPY>)) void madd_step_kernel(const TensorDesc* __restrict__ table,
                                                             int ntab, TensorDesc single,
                                                             Scalars s_arg,
                                                             const Scalars* __restrict__ sdev) {
  const Scalars s = sdev ? *sdev : s_arg;  // uniform: device-resident hyper-parameters
  const int64_t chunk = blockIdx.x;
  const TensorDesc d = find_tensor(table, ntab, single, chunk);
  const int64_t c0 = (chunk - d.chunk0) * kChunk;
  const int64_t cend = (c0 + kChunk < d.n) ? c0 + kChunk : d.n;
#pragma unroll 1
  for (int tile = 0; tile < kTilesPerChunk; ++tile) {
    const int64_t tb = c0 + (int64_t)tile * kTile;
    if (tb >= cend) break;  // uniform
    const int64_t eA = tb + (int64_t)threadIdx.x * kQuad, eB = eA + kSub;
    if (!d.vec_ok) {  // uniform: unaligned buffers or index base
      if (eA < cend) step_scalar_range<WF, GF, SF, SR, CLAMP, COPY>(d, eA, eA + kQuad < cend ? eA + kQuad : cend, s);
      if (eB < cend) step_scalar_range<WF, GF, SF, SR, CLAMP, COPY>(d, eB, eB + kQuad < cend ? eB + kQuad : cend, s);
      continue;
    }
    // Whole quads, decided per lane pair: lanes 2k and 2k+1 exchange halves of
    // their Philox blocks over a DPP swap, so both must take the same branch.
    const int64_t pA = tb + 2 * kQuad * (int64_t)(threadIdx.x >> 1), pB = pA + kSub;
    const bool fullA = pA + 2 * kQuad <= cend, fullB = pB + 2 * kQuad <= cend;
    const uint64_t gpair = (uint64_t)(d.gbase + tb) + 8u * (threadIdx.x >> 1);
    Quad<WF> qa, qb;
    MDraws mA, mB;
    if (tb + kTile <= cend) {  // uniform
      // The whole tile lies in the tensor (every tile but a tensor's last).
      // A uniform branch keeps this path straight-line, so the compiler waits
      // for sub-tile A's loads alone before A's arithmetic and B's arithmetic
      // does not wait for A's stores (1024x1024 step 7.60 -> 7.51 us, 7B list
      // 34.38 -> 34.26 ms, same process; the same split of the block-scaled
      // kernel made it 7-10% slower).  Loads grouped by array, so a wave's
      // two requests to one array are adjacent spans.
      qa.w.load(d.w, eA);
      qb.w.load(d.w, eB);
      qa.g = ld4g<GF>(d.g, eA);
      qb.g = ld4g<GF>(d.g, eB);
      qa.m = ld4s<SF>(d.m, eA);
      qb.m = ld4s<SF>(d.m, eB);
      qa.v = ld4s<SF>(d.v, eA);
      qb.v = ld4s<SF>(d.v, eB);
      qa.ve = ld4s<SF>(d.ve, eA);
      qb.ve = ld4s<SF>(d.ve, eB);
      uint32_t rA[4], rB[4];
      draws_aligned<SR>(gpair, s, rA, rB);
      mdraws_aligned<SF>(gpair, s, mA, mB);
      step_quad<WF, SR, CLAMP>(qa, rA, s);
      store_quad<WF, SF>(qa, d, eA, mA);
      if (COPY && d.copy) store_copy<WF>(qa.w, d.copy, eA);
      step_quad<WF, SR, CLAMP>(qb, rB, s);
      store_quad<WF, SF>(qb, d, eB, mB);
      if (COPY && d.copy) store_copy<WF>(qb.w, d.copy, eB);
      continue;
    }
    if (fullA) load_quad<WF, GF, SF>(qa, d, eA);
    if (fullB) load_quad<WF, GF, SF>(qb, d, eB);
    uint32_t rA[4], rB[4];
    draws_aligned<SR>(gpair, s, rA, rB);
    mdraws_aligned<SF>(gpair, s, mA, mB);
    if (fullA) {
      step_quad<WF, SR, CLAMP>(qa, rA, s);
      store_quad<WF, SF>(qa, d, eA, mA);
      if (COPY && d.copy) store_copy<WF>(qa.w, d.copy, eA);
    } else if (eA < cend) {
      step_scalar_range<WF, GF, SF, SR, CLAMP, COPY>(d, eA, eA + kQuad < cend ? eA + kQuad : cend, s);
    }
    if (fullB) {
      step_quad<WF, SR, CLAMP>(qb, rB, s);
      store_quad<WF, SF>(qb, d, eB, mB);
      if (COPY && d.copy) store_copy<WF>(qb.w, d.copy, eB);
    } else if (eB < cend) {
      step_scalar_range<WF, GF, SF, SR, CLAMP, COPY>(d, eB, eB + kQuad < cend ? eB + kQuad : cend, s);
    }
  }
}

// Block-scaled storage: the kBlk / 4 consecutive lanes that hold one block of
// a sub-tile (32 lanes for a 128-element FP8 block, 8 for a 32-element MXFP4
// block, 4 for a 16-element NVFP4 block) combine the block's max |w'| with
// lane shuffles.  The launch requires n to be a multiple of the block length,
// so a block is never split and whole lane groups are active or inactive
// together; every lane runs the shuffles and the draw exchange.
template <int WF>
constexpr int block_len() {
  return WF == WF_MXFP4 ? kMxBlock : (WF == WF_NVFP4 ? kNvBlock : kBlock);
}

// Max over aligned groups of LANES lanes (4, 8 or 32): lane swaps within quads
// (DPP quad_perm [1,0,3,2] and [2,3,0,1]), the mirrored quad of each half row
// (row_half_mirror), the mirrored half of each row (row_mirror) and the
// other row of each 32-lane half (ds_swizzle, xor 16).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, false);
}
template <int LANES>
__device__ __forceinline__ uint32_t block_amax(uint32_t a) {
  static_assert(LANES == 4 || LANES == 8 || LANES == 32, "block lane groups are 4, 8 or 32 lanes");
  uint32_t o = dpp_u32<0xB1>(a);
  a = o > a ? o : a;
  o = dpp_u32<0x4E>(a);
  a = o > a ? o : a;
  if constexpr (LANES == 4) return a;
  o = dpp_u32<0x141>(a);
  a = o > a ? o : a;
  if constexpr (LANES == 32) {
    o = dpp_u32<0x140>(a);
    a = o > a ? o : a;
    o = (uint32_t)__builtin_amdgcn_ds_swizzle((int)a, 0x401F);  // and 0x1F, xor 0x10
    a = o > a ? o : a;
  }
  return a;
}

// The block's dequantization factor from its scale code; `st` is NVFP4's
// per-tensor scale (unused by the other formats).  NVFP4's scale array holds
// st in its first 4 bytes, then one E4M3 code per block.
template <int WF>
__device__ __forceinline__ float scale_value(uint32_t code, float st) {
  if constexpr (WF == WF_MXFP4) return dec_e8m0(code);
  else if constexpr (WF == WF_NVFP4) return dec_fp8<WF_E4M3>(code) * st;
  else return dec_fp16(code);
}
template <int WF>
__device__ __forceinline__ uint32_t load_scale(const void* scales, int64_t b) {
  if constexpr (WF == WF_MXFP4) return ((const uint8_t*)scales)[b];
  else if constexpr (WF == WF_NVFP4) return ((const uint8_t*)scales)[4 + b];
  else return ((const uint16_t*)scales)[b];
}
template <int WF>
__device__ __forceinline__ void store_scale(void* scales, int64_t b, uint32_t code) {
  if constexpr (WF == WF_MXFP4) ((uint8_t*)scales)[b] = (uint8_t)code;
  else if constexpr (WF == WF_NVFP4) ((uint8_t*)scales)[4 + b] = (uint8_t)code;
  else ((uint16_t*)scales)[b] = (uint16_t)code;
}

// NVFP4 block code: RNE_E4M3(amax / fp32(6 st)), saturating at 448; the E4M3
// NaN code for a block holding a non-finite value.
__device__ __forceinline__ uint32_t nv_block_code(uint32_t amax_bits, float st) {
  if (amax_bits >= 0x7F800000u) return 0x7Fu;
  const float six_st = 6.0f * st;
  return enc_fp8<WF_E4M3>(__uint_as_float(amax_bits) / six_st, false, 0u);
}

template <int WF, bool SR, bool CLAMP>
__device__ __forceinline__ uint32_t step_quad_unrounded(Quad<WF>& q, float sold, float (&wn)[4],
                                                        const Scalars& s) {
  uint32_t amax = 0u;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float m = q.m[k], v = q.v[k], ve = q.ve[k];
    wn[k] = step_elem<CLAMP>(decode<WF>(q.w.code(k)) * sold, q.g[k], m, v, ve, s);
    q.m[k] = m;
    q.v[k] = v;
    q.ve[k] = ve;
    const uint32_t ab = __float_as_uint(wn[k]) & 0x7FFFFFFFu;
    amax = ab > amax ? ab : amax;
  }
  return amax;
}

// Re-quantize four new weights of one block; `cv` receives their stored
// values (payload value x scale) for the compute copy.
template <int WF, bool SR>
__device__ __forceinline__ uint32_t requant_quad(Quad<WF>& q, const float (&wn)[4], uint32_t amax,
                                                 const uint32_t (&r)[4], float (&cv)[4], float st) {
  if constexpr (WF == WF_NVFP4) {
    const uint32_t sc = nv_block_code(amax, st);
    const float den = dec_fp8<WF_E4M3>(sc) * st;
    const bool zero = sc == 0x7Fu || den == 0.0f;  // NaN block, or a factor of 0
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float v;
      const uint32_t c = enc_e2m1(wn[k] / den, SR, r[k], v);
      q.w.set(k, zero ? 0u : c);
      cv[k] = (zero ? 0.0f : v) * den;
    }
    return sc;
  } else if constexpr (WF == WF_MXFP4) {
    const uint32_t sc = mx_scale(amax);
    const float inv = mx_inv_scale(sc), X = dec_e8m0(sc);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float v;
      const uint32_t c = enc_e2m1(wn[k] * inv, SR, r[k], v);
      q.w.set(k, sc == 0xFFu ? 0u : c);
      cv[k] = (sc == 0xFFu ? 0.0f : v) * X;
    }
    return sc;
  } else {
    const uint32_t sc = block_scale<WF>(amax);
    const float sf = dec_fp16(sc);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float v;
      q.w.set(k, enc_fp8<WF>(wn[k] / sf, SR, r[k], v));
      cv[k] = v * sf;
    }
    return sc;
  }
}

template <int WF, int GF, int SF, bool SR, bool CLAMP, bool COPY>
__global__ __launch_bounds__(kThreads) void madd_step_block_kernel(
    const TensorDesc* __restrict__ table, int ntab, TensorDesc single, Scalars s_arg,
    const Scalars* __restrict__ sdev) {
  const Scalars s = sdev ? *sdev : s_arg;
  constexpr int kBlk = block_len<WF>();
  constexpr int kLanes = kBlk / kQuad;
  const int64_t chunk = blockIdx.x;
  const TensorDesc d = find_tensor(table, ntab, single, chunk);
  const float st = WF == WF_NVFP4 ? *(const float*)d.scales : 1.0f;  // NVFP4 tensor scale
  const int64_t c0 = (chunk - d.chunk0) * kChunk;
  const int64_t cend = (c0 + kChunk < d.n) ? c0 + kChunk : d.n;
#pragma unroll 1
  for (int tile = 0; tile < kTilesPerChunk; ++tile) {
    const int64_t tb = c0 + (int64_t)tile * kTile;
    if (tb >= cend) break;
    const int64_t eA = tb + (int64_t)threadIdx.x * kQuad, eB = eA + kSub;
    const bool actA = eA < cend, actB = eB < cend;  // whole lane groups of a block agree
    Quad<WF> qa, qb;
    float wa[4], wb[4];
    uint32_t amaxA = 0u, amaxB = 0u;
    if (actA) load_quad<WF, GF, SF>(qa, d, eA);
    if (actB) load_quad<WF, GF, SF>(qb, d, eB);
    uint32_t rA[4], rB[4];
    MDraws mA, mB;
    if (d.vec_ok) {  // uniform: index base a multiple of 8
      const uint64_t gpair = (uint64_t)(d.gbase + tb) + 8u * (threadIdx.x >> 1);
      draws_aligned<SR>(gpair, s, rA, rB);
      mdraws_aligned<SF>(gpair, s, mA, mB);
    } else {
      draws_any<SR>((uint64_t)(d.gbase + eA), s, rA);
      draws_any<SR>((uint64_t)(d.gbase + eB), s, rB);
      mdraws_any<SF>((uint64_t)(d.gbase + eA), s, mA);
      mdraws_any<SF>((uint64_t)(d.gbase + eB), s, mB);
    }
    if (actA)
      amaxA = step_quad_unrounded<WF, SR, CLAMP>(
          qa, scale_value<WF>(load_scale<WF>(d.scales, (int64_t)((uint64_t)eA / kBlk)), st), wa, s);
    if (actB)
      amaxB = step_quad_unrounded<WF, SR, CLAMP>(
          qb, scale_value<WF>(load_scale<WF>(d.scales, (int64_t)((uint64_t)eB / kBlk)), st), wb, s);
    amaxA = block_amax<kLanes>(amaxA);
    amaxB = block_amax<kLanes>(amaxB);
    float cv[4];
    if (actA) {
      const uint32_t sc = requant_quad<WF, SR>(qa, wa, amaxA, rA, cv, st);
      store_quad<WF, SF>(qa, d, eA, mA);
      if (COPY && d.copy) store_copy_values(cv, d.copy, eA);
      if ((threadIdx.x & (kLanes - 1)) == 0u) store_scale<WF>(d.scales, (int64_t)((uint64_t)eA / kBlk), sc);
    }
    if (actB) {
      const uint32_t sc = requant_quad<WF, SR>(qb, wb, amaxB, rB, cv, st);
      store_quad<WF, SF>(qb, d, eB, mB);
      if (COPY && d.copy) store_copy_values(cv, d.copy, eB);
      if ((threadIdx.x & (kLanes - 1)) == 0u) store_scale<WF>(d.scales, (int64_t)((uint64_t)eB / kBlk), sc);
    }
  }
}


// ---------------------------------------------------------------------------
// NVFP4 with current scaling: the per-tensor scale derived anew from the
// updated tensor at every step.  A launch clears each tensor's amax word;
// pass 1 takes the FP32 step (moments stored, w' written over the fp32
// gradient, the largest finite |w'| folded into the amax word); pass 2
// derives s_t' = fp32(amax / 2688) and re-encodes every block of w' with it.
// The amax is a reduction over a whole tensor, so pass 2 of a tensor must
// follow its pass 1 in a later launch; the launches pipeline the two passes
// over groups of tensors (nvcs_step_kernel).
// Scale array: s_t (fp32), the amax word, then one E4M3 code per 16 elements.
// ---------------------------------------------------------------------------

#if MADD_IN_PART(9)
__global__ __launch_bounds__(kThreads) void nvcs_clear_kernel(const TensorDesc* __restrict__ table,
                                                              int ntab, TensorDesc single,
                                                              Scalars, const Scalars*) {
  const int i = (int)(blockIdx.x * kThreads + threadIdx.x);
  if (i >= (ntab == 0 ? 1 : ntab)) return;
  void* scales = ntab == 0 ? single.scales : table[i].scales;
  ((uint32_t*)scales)[1] = 0u;
}

// |x| as raw bits when x is finite, else 0.
__device__ __forceinline__ uint32_t finite_abs_bits(float x) {
  const uint32_t b = __float_as_uint(x) & 0x7FFFFFFFu;
  return b < 0x7F800000u ? b : 0u;
}

template <int SF, bool CLAMP>
__device__ __forceinline__ uint32_t nvcs_step_quad(const TensorDesc& d, int64_t e, float st,
                                                   const MDraws& md, const Scalars& s) {
  Quad<WF_NVFP4> q;
  load_quad<WF_NVFP4, GF_FP32, SF>(q, d, e);
  const float den = scale_value<WF_NVFP4>(
      load_scale<WF_NVFP4>((const uint8_t*)d.scales + 4, (int64_t)((uint64_t)e / kNvBlock)), st);
  f4 wn;
  uint32_t amax = 0u;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float m = q.m[k], v = q.v[k], ve = q.ve[k];
    wn[k] = step_elem<CLAMP>(decode<WF_NVFP4>(q.w.code(k)) * den, q.g[k], m, v, ve, s);
    q.m[k] = m;
    q.v[k] = v;
    q.ve[k] = ve;
    const uint32_t ab = finite_abs_bits(wn[k]);
    amax = ab > amax ? ab : amax;
  }
  st4s<SF>(d.m, e, q.m, md.m);
  st4s<SF>(d.v, e, q.v, md.v);
  st4s<SF>(d.ve, e, q.ve, md.ve);
  stg<f4>((float*)d.g + e, wn);  // w' replaces the gradient
  return amax;
}

// Pass 1 on one chunk: the FP32 step, moments stored, w' over the gradient,
// the chunk's largest finite |w'| folded into its tensor's amax word.
template <int SF, bool CLAMP>
__device__ __forceinline__ void nvcs_pass1_chunk(const TensorDesc* __restrict__ table, int ntab,
                                                 const TensorDesc& single, int64_t chunk,
                                                 const Scalars& s) {
  const TensorDesc d = find_tensor(table, ntab, single, chunk);
  const float st = *(const float*)d.scales;
  const int64_t c0 = (chunk - d.chunk0) * kChunk;
  const int64_t cend = (c0 + kChunk < d.n) ? c0 + kChunk : d.n;
  const int64_t eA = c0 + (int64_t)threadIdx.x * kQuad, eB = eA + kSub;
  MDraws mA, mB;
  if (d.vec_ok) {  // uniform: index base a multiple of 8
    mdraws_aligned<SF>((uint64_t)(d.gbase + c0) + 8u * (threadIdx.x >> 1), s, mA, mB);
  } else {
    mdraws_any<SF>((uint64_t)(d.gbase + eA), s, mA);
    mdraws_any<SF>((uint64_t)(d.gbase + eB), s, mB);
  }
  uint32_t amax = 0u;
  if (eA < cend) amax = nvcs_step_quad<SF, CLAMP>(d, eA, st, mA, s);  // n % 16 == 0: whole quads
  if (eB < cend) {
    const uint32_t b = nvcs_step_quad<SF, CLAMP>(d, eB, st, mB, s);
    amax = b > amax ? b : amax;
  }
  // the wave's largest finite |w'|, folded into the tensor's amax word; a
  // wave whose value is not above the word's current one skips the atomic
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)amax, off);
    amax = o > amax ? o : amax;
  }
  if ((threadIdx.x & 63u) == 0u && amax != 0u) {
    uint32_t* word = (uint32_t*)d.scales + 1;
    if (amax > __atomic_load_n(word, __ATOMIC_RELAXED)) atomicMax(word, amax);
  }
}

template <bool SR, bool COPY>
__device__ __forceinline__ void nvcs_requant(const TensorDesc& d, int64_t e, f4 w,
                                             uint32_t amax, const uint32_t (&r)[4], float st) {
  Quad<WF_NVFP4> q;
  q.w.raw = 0u;
  const float wn[4] = {w.x, w.y, w.z, w.w};
  float cv[4];
  const uint32_t sc = requant_quad<WF_NVFP4, SR>(q, wn, amax, r, cv, st);
  q.w.store(d.w, e);
  if (COPY && d.copy) store_copy_values(cv, d.copy, e);
  if ((threadIdx.x & 3u) == 0u)
    store_scale<WF_NVFP4>((uint8_t*)d.scales + 4, (int64_t)((uint64_t)e / kNvBlock), sc);
}

// Pass 2 on one chunk: the tensor scale from its complete amax word, then
// every block of the chunk re-encoded from w'.
template <bool SR, bool COPY>
__device__ __forceinline__ void nvcs_pass2_chunk(const TensorDesc* __restrict__ table, int ntab,
                                                 const TensorDesc& single, int64_t chunk,
                                                 const Scalars& s) {
  const TensorDesc d = find_tensor(table, ntab, single, chunk);
  const float amax_t = __uint_as_float(((const uint32_t*)d.scales)[1]);
  const float st = amax_t > 0.0f ? amax_t / 2688.0f : 1.0f;
  if (chunk == d.chunk0 && threadIdx.x == 0) *(float*)d.scales = st;  // pass 2 reads only the amax word
  const int64_t c0 = (chunk - d.chunk0) * kChunk;
  const int64_t cend = (c0 + kChunk < d.n) ? c0 + kChunk : d.n;
  const int64_t eA = c0 + (int64_t)threadIdx.x * kQuad, eB = eA + kSub;
  const bool actA = eA < cend, actB = eB < cend;  // whole lane groups of a block agree
  f4 wa = f4{0.0f, 0.0f, 0.0f, 0.0f}, wb = wa;
  if (actA) wa = ldg<f4>((const float*)d.g + eA);
  if (actB) wb = ldg<f4>((const float*)d.g + eB);
  uint32_t rA[4], rB[4];
  if (d.vec_ok) {
    draws_aligned<SR>((uint64_t)(d.gbase + c0) + 8u * (threadIdx.x >> 1), s, rA, rB);
  } else {
    draws_any<SR>((uint64_t)(d.gbase + eA), s, rA);
    draws_any<SR>((uint64_t)(d.gbase + eB), s, rB);
  }
  uint32_t amaxA = 0u, amaxB = 0u;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t a = __float_as_uint(wa[k]) & 0x7FFFFFFFu, b = __float_as_uint(wb[k]) & 0x7FFFFFFFu;
    amaxA = a > amaxA ? a : amaxA;
    amaxB = b > amaxB ? b : amaxB;
  }
  amaxA = block_amax<4>(amaxA);
  amaxB = block_amax<4>(amaxB);
  if (actA) nvcs_requant<SR, COPY>(d, eA, wa, amaxA, rA, st);
  if (actB) nvcs_requant<SR, COPY>(d, eB, wb, amaxB, rB, st);
}

// One launch of the pipelined current-scaling step: pass 1 over the chunks
// [a1, a1 + n1) of one group of tensors and pass 2 over the chunks
// [a2, a2 + n2) of the previous group, whose amax words the previous launch
// completed.  The two kinds of workgroup are spread evenly over the grid
// (n1 + n2 workgroups), so that the arithmetic-heavy re-encoding of one group
// runs while the memory-heavy first pass of the next one streams.

template <int SF, bool CLAMP, bool SR, bool COPY>
__global__ __launch_bounds__(kThreads) void nvcs_step_kernel(const TensorDesc* __restrict__ table,
                                                             int ntab, TensorDesc single,
                                                             Scalars s_arg,
                                                             const Scalars* __restrict__ sdev,
                                                             NvcsSpan sp) {
  const Scalars s = sdev ? *sdev : s_arg;
  const int64_t b = blockIdx.x, n = sp.n1 + sp.n2;
  const int64_t before = (b * sp.n2) / n;  // pass-2 workgroups ahead of this one
  if (((b + 1) * sp.n2) / n > before)       // uniform per workgroup
    nvcs_pass2_chunk<SR, COPY>(table, ntab, single, sp.a2 + before, s);
  else
    nvcs_pass1_chunk<SF, CLAMP>(table, ntab, single, sp.a1 + (b - before), s);
}
#endif  // MADD_IN_PART(9)

// ---------------------------------------------------------------------------
// The moment-free rules of Appendix B's diagnostic
// ---------------------------------------------------------------------------

// Additive u_a = -eta_a g; multiplicative ut = -eta_m g_e with g_e = ln2 w g,
// u_m = clip(ut / max(|w|, tau)); combined w + w u_m + u_a.  Same FP32
// conventions as step_elem.
__device__ __forceinline__ float plain_elem(float w, float g, float lra, const Scalars& s) {
  const float LN2 = 0.693147182464599609375f;
  const float ua = -(lra * g);
  const float ge = (LN2 * w) * g;
  const float ut = -(s.LRM * ge);
  const float aw = fabsf(w);
  const float rho = aw > s.TAU ? aw : s.TAU;
  const float um = clampf(ut / rho, s.ULO, s.UHI);
  return clampf(fmaf(w, um, w) + ua, -s.WMAX, s.WMAX);
}

// Four consecutive elements per thread, grid-stride (diagnostic-sized work).
template <int WF, int GF, bool SR>
__global__ __launch_bounds__(kThreads) void madd_plain_kernel(void* w, const void* g, int64_t n,
                                                              int64_t gbase, float lra,
                                                              Scalars s) {
  const int64_t stride = (int64_t)gridDim.x * kThreads * kQuad;
  for (int64_t e0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kQuad; e0 < n; e0 += stride) {
    const int64_t e1 = e0 + kQuad < n ? e0 + kQuad : n;
    for (int64_t i = e0; i < e1; ++i) {
      const float wn = plain_elem(decode<WF>(ld1w<WF>(w, i)), ld1g<GF>(g, i), lra, s);
      const uint32_t r16 = SR ? draw_one((uint64_t)(gbase + i), s) : 0u;
      st1w<WF>(w, i, encode<WF>(wn, SR, r16));
    }
  }
}

typedef void (*plain_fn)(void*, const void*, int64_t, int64_t, float, Scalars);

template <int WF, int GF>
plain_fn pick_plain_sr(bool sr) {
  return sr ? madd_plain_kernel<WF, GF, true> : madd_plain_kernel<WF, GF, false>;
}
template <int WF>
plain_fn pick_plain_gf(int gf, bool sr) {
  return gf == GF_FP32 ? pick_plain_sr<WF, GF_FP32>(sr) : pick_plain_sr<WF, GF_BF16>(sr);
}

// ---------------------------------------------------------------------------
// Auxiliary kernels: zero state, encode weights
// ---------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(kThreads) void zero_kernel(T* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) p[i] = T(0);
}

template <int WF>
__global__ __launch_bounds__(kThreads) void encode_kernel(const float* __restrict__ x, void* w,
                                                          int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
    st1w<WF>(w, i, encode<WF>(x[i], false, 0u));
}

// One thread per 128-element block.
template <int WF>
__global__ __launch_bounds__(kThreads) void encode_block_kernel(const float* __restrict__ x,
                                                                uint8_t* q, uint16_t* scales,
                                                                int64_t nblocks) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < nblocks; b += stride) {
    const float* xb = x + b * kBlock;
    uint32_t amax = 0u;
    for (int k = 0; k < kBlock; ++k) {
      const uint32_t ab = __float_as_uint(xb[k]) & 0x7FFFFFFFu;
      amax = ab > amax ? ab : amax;
    }
    const uint32_t sc = block_scale<WF>(amax);
    const float sf = dec_fp16(sc);
    for (int k = 0; k < kBlock; ++k) q[b * kBlock + k] = (uint8_t)enc_fp8<WF>(xb[k] / sf, false, 0u);
    scales[b] = (uint16_t)sc;
  }
}

#if MADD_IN_PART(0)
// ---------------------------------------------------------------------------
// Appendix B's diagnostic: the gradient of its sampled quartic loss
// ---------------------------------------------------------------------------

// counts[i] = number of sampled entries equal to i (entries outside [0, n)
// are skipped).  Integer atomics: the counts do not depend on their order.
__global__ __launch_bounds__(kThreads) void toy_count_kernel(const int64_t* __restrict__ idx,
                                                             int64_t batch, int64_t n,
                                                             int32_t* __restrict__ counts) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x; k < batch; k += stride) {
    const int64_t i = idx[k];
    if (i >= 0 && i < n) atomicAdd(&counts[i], 1);
  }
}

// g_i = ((s d) d) d with d = w_i - target_i and s = (fob cnt_i) c_i, fob =
// fp32(4 / B): the derivative of (1/B) sum_k c_i (w_i - target_i)^4 over the
// B sampled entries, in this fixed fp32 order.
template <int WF>
__global__ __launch_bounds__(kThreads) void toy_grad_kernel(const void* w,
                                                            const float* __restrict__ target,
                                                            const float* __restrict__ c,
                                                            const int32_t* __restrict__ counts,
                                                            int64_t n, float fob,
                                                            float* __restrict__ g) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
    const float d = decode<WF>(ld1w<WF>(w, i)) - target[i];
    const float s = (fob * (float)counts[i]) * c[i];
    g[i] = ((s * d) * d) * d;
  }
}

// One thread per 32-element MXFP4 block.
__global__ __launch_bounds__(kThreads) void encode_mx_kernel(const float* __restrict__ x,
                                                             uint8_t* q, uint8_t* scales,
                                                             int64_t nblocks) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < nblocks; b += stride) {
    const float* xb = x + b * kMxBlock;
    uint32_t amax = 0u;
    for (int k = 0; k < kMxBlock; ++k) {
      const uint32_t ab = __float_as_uint(xb[k]) & 0x7FFFFFFFu;
      amax = ab > amax ? ab : amax;
    }
    const uint32_t sc = mx_scale(amax);
    const float inv = mx_inv_scale(sc);
    for (int k = 0; k < kMxBlock; k += 2) {
      const uint32_t lo = sc == 0xFFu ? 0u : enc_e2m1(xb[k] * inv, false, 0u);
      const uint32_t hi = sc == 0xFFu ? 0u : enc_e2m1(xb[k + 1] * inv, false, 0u);
      q[b * (kMxBlock / 2) + k / 2] = (uint8_t)(lo | (hi << 4));
    }
    scales[b] = (uint8_t)sc;
  }
}

// NVFP4 encoding, three stages on the stream: the largest finite |x| of the
// tensor into the scale array's first word (as fp32 bits; non-negative floats
// order like their bits), that word turned into the per-tensor scale
// st = amax / 2688 (1 when amax is 0), then one thread per 16-element block.
__global__ __launch_bounds__(kThreads) void nv_amax_kernel(const float* __restrict__ x, int64_t n,
                                                           uint32_t* slot) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  uint32_t m = 0u;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
    const uint32_t b = __float_as_uint(x[i]) & 0x7FFFFFFFu;
    m = (b < 0x7F800000u && b > m) ? b : m;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)m, off);
    m = o > m ? o : m;
  }
  if ((threadIdx.x & 63u) == 0u && m != 0u) atomicMax(slot, m);
}

__global__ void nv_scale_kernel(uint32_t* slot) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const float amax = __uint_as_float(*slot);
    *slot = __float_as_uint(amax > 0.0f ? amax / 2688.0f : 1.0f);
  }
}

// Zero the first `words` 32-bit words of a scale array.
__global__ void nv_clear_kernel(uint32_t* slot, int words) {
  if (blockIdx.x == 0 && (int)threadIdx.x < words) slot[threadIdx.x] = 0u;
}

// `scales` holds st in its first word; the block codes start `head` bytes in
// (4 for NVFP4, 8 for NVFP4 with current scaling).
__global__ __launch_bounds__(kThreads) void encode_nv_kernel(const float* __restrict__ x,
                                                             uint8_t* q, uint8_t* scales,
                                                             int64_t nblocks, int head) {
  const float st = *(const float*)scales;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t b = (int64_t)blockIdx.x * kThreads + threadIdx.x; b < nblocks; b += stride) {
    const float* xb = x + b * kNvBlock;
    uint32_t amax = 0u;
    for (int k = 0; k < kNvBlock; ++k) {
      const uint32_t ab = __float_as_uint(xb[k]) & 0x7FFFFFFFu;
      amax = ab > amax ? ab : amax;
    }
    const uint32_t sc = nv_block_code(amax, st);
    const float den = dec_fp8<WF_E4M3>(sc) * st;
    const bool zero = sc == 0x7Fu || den == 0.0f;
    for (int k = 0; k < kNvBlock; k += 2) {
      const uint32_t lo = zero ? 0u : enc_e2m1(xb[k] / den, false, 0u);
      const uint32_t hi = zero ? 0u : enc_e2m1(xb[k + 1] / den, false, 0u);
      q[b * (kNvBlock / 2) + k / 2] = (uint8_t)(lo | (hi << 4));
    }
    scales[head + b] = (uint8_t)sc;
  }
}
#endif  // MADD_IN_PART(0)

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

typedef void (*step_fn)(const TensorDesc*, int, TensorDesc, Scalars, const Scalars*);

// Kernel instantiation for (weight format, block-scaled; gradient and moment
// formats, rounding, optional clamps present, compute copies present).
template <int WF, bool BLK, int GF, int SF, bool SR, bool CLAMP>
step_fn pick_copy(bool copy) {
  if constexpr (BLK)
    return copy ? madd_step_block_kernel<WF, GF, SF, SR, CLAMP, true>
                : madd_step_block_kernel<WF, GF, SF, SR, CLAMP, false>;
  else
    return copy ? madd_step_kernel<WF, GF, SF, SR, CLAMP, true>
                : madd_step_kernel<WF, GF, SF, SR, CLAMP, false>;
}
template <int WF, bool BLK, int GF, int SF, bool SR>
step_fn pick_clamp(bool clamp, bool copy) {
  return clamp ? pick_copy<WF, BLK, GF, SF, SR, true>(copy)
               : pick_copy<WF, BLK, GF, SF, SR, false>(copy);
}
template <int WF, bool BLK, int GF, int SF>
step_fn pick_sr(bool sr, bool clamp, bool copy) {
  return sr ? pick_clamp<WF, BLK, GF, SF, true>(clamp, copy)
            : pick_clamp<WF, BLK, GF, SF, false>(clamp, copy);
}
template <int WF, bool BLK, int GF>
step_fn pick_sf(int sf, bool sr, bool clamp, bool copy) {
  switch (sf) {
    case SF_FP32: return pick_sr<WF, BLK, GF, SF_FP32>(sr, clamp, copy);
    case SF_BF16: return pick_sr<WF, BLK, GF, SF_BF16>(sr, clamp, copy);
    case SF_BF16_SR: return pick_sr<WF, BLK, GF, SF_BF16_SR>(sr, clamp, copy);
    default: return nullptr;
  }
}
template <int WF, bool BLK>
step_fn pick_gf(int gf, int sf, bool sr, bool clamp, bool copy) {
  return gf == GF_FP32 ? pick_sf<WF, BLK, GF_FP32>(sf, sr, clamp, copy)
                       : pick_sf<WF, BLK, GF_BF16>(sf, sr, clamp, copy);
}

// One entry point per part; each instantiates one (weight format, scaled)
// family of step kernels.
step_fn pick_part1(int gf, int sf, bool sr, bool clamp, bool copy);  // bf16
step_fn pick_part2(int gf, int sf, bool sr, bool clamp, bool copy);  // e4m3
step_fn pick_part3(int gf, int sf, bool sr, bool clamp, bool copy);  // e4m3, block-scaled
step_fn pick_part4(int gf, int sf, bool sr, bool clamp, bool copy);  // e5m2
step_fn pick_part5(int gf, int sf, bool sr, bool clamp, bool copy);  // e5m2, block-scaled
step_fn pick_part6(int gf, int sf, bool sr, bool clamp, bool copy);  // fp32 passthrough
step_fn pick_part7(int gf, int sf, bool sr, bool clamp, bool copy);  // mxfp4 (block-scaled)
step_fn pick_part8(int gf, int sf, bool sr, bool clamp, bool copy);  // nvfp4 (block-scaled)

// NVFP4 with current scaling: the amax-word clear and the pipelined step.
typedef void (*nvcs_fn)(const TensorDesc*, int, TensorDesc, Scalars, const Scalars*, NvcsSpan);
struct NvcsKernels {
  step_fn clear;
  nvcs_fn step;
};
NvcsKernels pick_part9(int sf, bool sr, bool clamp, bool copy);

#if MADD_IN_PART(1)
step_fn pick_part1(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_BF16, false>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(2)
step_fn pick_part2(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_E4M3, false>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(3)
step_fn pick_part3(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_E4M3, true>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(4)
step_fn pick_part4(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_E5M2, false>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(5)
step_fn pick_part5(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_E5M2, true>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(6)
step_fn pick_part6(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_FP32, false>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(7)
step_fn pick_part7(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_MXFP4, true>(gf, sf, sr, clamp, copy);
}
#endif
#if MADD_IN_PART(8)
step_fn pick_part8(int gf, int sf, bool sr, bool clamp, bool copy) {
  return pick_gf<WF_NVFP4, true>(gf, sf, sr, clamp, copy);
}
#endif

#if MADD_IN_PART(9)
template <int SF, bool CLAMP>
nvcs_fn pick_nvcs_rounding(bool sr, bool copy) {
  return sr ? (copy ? nvcs_step_kernel<SF, CLAMP, true, true> : nvcs_step_kernel<SF, CLAMP, true, false>)
            : (copy ? nvcs_step_kernel<SF, CLAMP, false, true>
                    : nvcs_step_kernel<SF, CLAMP, false, false>);
}
template <int SF>
NvcsKernels pick_nvcs(bool sr, bool clamp, bool copy) {
  NvcsKernels k;
  k.clear = nvcs_clear_kernel;
  k.step = clamp ? pick_nvcs_rounding<SF, true>(sr, copy) : pick_nvcs_rounding<SF, false>(sr, copy);
  return k;
}
NvcsKernels pick_part9(int sf, bool sr, bool clamp, bool copy) {
  switch (sf) {
    case SF_FP32: return pick_nvcs<SF_FP32>(sr, clamp, copy);
    case SF_BF16: return pick_nvcs<SF_BF16>(sr, clamp, copy);
    default: return pick_nvcs<SF_BF16_SR>(sr, clamp, copy);
  }
}
#endif

#if MADD_IN_PART(0)
// The step kernel for (weight, gradient and moment formats, rounding,
// optional clamps present, compute copies present, block-scaled); nullptr for
// combinations that do not exist (block scaling is for FP8, MXFP4 and NVFP4
// only, and the 4-bit formats are always block-scaled).
step_fn pick_kernel(int wf, int gf, int sf, bool sr, bool clamp, bool copy, bool blk) {
  switch (wf) {
    case WF_BF16: return blk ? nullptr : pick_part1(gf, sf, sr, clamp, copy);
    case WF_E4M3: return blk ? pick_part3(gf, sf, sr, clamp, copy) : pick_part2(gf, sf, sr, clamp, copy);
    case WF_E5M2: return blk ? pick_part5(gf, sf, sr, clamp, copy) : pick_part4(gf, sf, sr, clamp, copy);
    case WF_FP32: return blk ? nullptr : pick_part6(gf, sf, sr, clamp, copy);
    case WF_MXFP4: return blk ? pick_part7(gf, sf, sr, clamp, copy) : nullptr;
    case WF_NVFP4: return blk ? pick_part8(gf, sf, sr, clamp, copy) : nullptr;
    default: return nullptr;
  }
}

bool needs_clamp(const madd_hparams& hp) {
  return !(std::isinf(hp.g_max) && hp.g_max > 0) || !(std::isinf(hp.w_max) && hp.w_max > 0);
}

bool valid_wfmt(int32_t f) { return f >= MADD_W_BF16 && f <= MADD_W_NVFP4_CURRENT; }
bool nv_fmt(int32_t f) { return f == MADD_W_NVFP4 || f == MADD_W_NVFP4_CURRENT; }
bool fp4_fmt(int32_t f) { return f == MADD_W_MXFP4 || nv_fmt(f); }
bool valid_gfmt(int32_t f) { return f == MADD_G_FP32 || f == MADD_G_BF16; }
bool valid_sfmt(int32_t f) { return f == MADD_S_FP32 || f == MADD_S_BF16 || f == MADD_S_BF16_SR; }
bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int32_t check_hparams(const madd_hparams* hp) {
  if (!hp) return MADD_EINVAL;
  if (!(hp->beta1 >= 0.0 && hp->beta1 < 1.0)) return MADD_EINVAL;
  if (!(hp->beta2 >= 0.0 && hp->beta2 < 1.0)) return MADD_EINVAL;
  if (!(hp->eps >= 0.0)) return MADD_EINVAL;
  if (!(hp->tau > 0.0)) return MADD_EINVAL;
  if (!(hp->r_max > 0.0 && hp->r_max < 1.0)) return MADD_EINVAL;
  if (!(hp->eps0 >= 0.0 && hp->eps0 < hp->r_max)) return MADD_EINVAL;
  if (!(hp->g_max > 0.0) || !(hp->d_mult_max > 0.0) || !(hp->w_max > 0.0)) return MADD_EINVAL;
  if (hp->bias_correction != 0 && hp->bias_correction != 1) return MADD_EINVAL;
  if (hp->rounding != MADD_ROUND_RNE && hp->rounding != MADD_ROUND_SR) return MADD_EINVAL;
  if (hp->step < 1 || hp->step > (int64_t)0xFFFFFFFFll) return MADD_EINVAL;
  if (std::isnan(hp->lr_add) || std::isnan(hp->lr_mul)) return MADD_EINVAL;
  return MADD_OK;
}

Scalars make_scalars(const madd_hparams& hp) {
  Scalars s;
  const double t = (double)hp.step;
  s.B1 = (float)hp.beta1;
  s.B2 = (float)hp.beta2;
  s.OMB1 = (float)(1.0 - hp.beta1);
  s.OMB2 = (float)(1.0 - hp.beta2);
  if (hp.bias_correction) {
    s.SA = (float)(hp.lr_add / (1.0 - pow(hp.beta1, t)));
    s.IBC2 = (float)(1.0 / (1.0 - pow(hp.beta2, t)));
  } else {
    s.SA = (float)hp.lr_add;
    s.IBC2 = 1.0f;
  }
  s.LRM = (float)hp.lr_mul;
  s.EPS = (float)hp.eps;
  s.TAU = (float)hp.tau;
  s.GMAX = (float)hp.g_max;
  double lo = -(hp.r_max - hp.eps0), hi = hp.r_max;
  if (std::isfinite(hp.d_mult_max)) {
    lo = std::fmax(lo, exp2(-hp.d_mult_max) - 1.0);
    hi = std::fmin(hi, exp2(hp.d_mult_max) - 1.0);
  }
  s.ULO = (float)lo;
  s.UHI = (float)hi;
  s.WMAX = (float)hp.w_max;
  s.key0 = (uint32_t)hp.seed;
  s.key1 = (uint32_t)(hp.seed >> 32);
  s.t = (uint32_t)hp.step;
  return s;
}

int64_t chunks_of(int64_t n) { return (n + kChunk - 1) / kChunk; }

// Kernel launch that reports the launch's own status.  hipLaunchKernel
// returns it directly, so the thread's last-error state, which belongs to
// the caller, is neither read nor cleared.
template <typename Tuple, size_t... I>
void kernel_argv(void** argv, Tuple& t, std::index_sequence<I...>) {
  ((argv[I] = (void*)&std::get<I>(t)), ...);
}
template <typename... P, typename... A>
int32_t launch_k(void (*k)(P...), dim3 grid, dim3 block, hipStream_t stream, A&&... a) {
  std::tuple<P...> args(std::forward<A>(a)...);
  void* argv[sizeof...(P) > 0 ? sizeof...(P) : 1];
  kernel_argv(argv, args, std::index_sequence_for<P...>{});
  return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, argv, 0, stream) ==
                 hipSuccess
             ? MADD_OK
             : MADD_EDEVICE;
}

// Device tables are written by a kernel that carries the bytes in its
// arguments: stream-ordered, asynchronous, free of host-memory lifetimes
// (the arguments are copied at launch) and recordable in a graph.
constexpr int kFillWords = 352;  // 16 descriptors of 88 bytes per launch
constexpr int kFillThreads = 384;
struct FillArgs {
  uint32_t nwords;
  uint32_t word[kFillWords];
};
static_assert(sizeof(TensorDesc) == 88, "descriptor layout");
static_assert(sizeof(TensorDesc) % 4 == 0, "descriptors are whole words");

__global__ __launch_bounds__(kFillThreads) void table_fill_kernel(uint32_t* dst, FillArgs a) {
  const uint32_t i = threadIdx.x;
  if (i < a.nwords) dst[i] = a.word[i];
}

// Copy `bytes` (a multiple of 4) from host memory to device memory `dst`
// on `stream`.
int32_t fill_device(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  const uint32_t* w = (const uint32_t*)src;
  const size_t nw = bytes / 4;
  for (size_t off = 0; off < nw; off += kFillWords) {
    FillArgs a;
    a.nwords = (uint32_t)(nw - off < (size_t)kFillWords ? nw - off : (size_t)kFillWords);
    memcpy(a.word, w + off, a.nwords * 4u);
    const int32_t rc = launch_k(table_fill_kernel, dim3(1), dim3(kFillThreads), stream,
                                (uint32_t*)dst + off, a);
    if (rc != MADD_OK) return rc;
  }
  return MADD_OK;
}

// The HIP side of the descriptor-table cache (policy in table_cache.h).
struct HipTables {
  bool alloc(size_t bytes, void** p) { return hipMalloc(p, bytes) == hipSuccess; }
  bool upload(void* dst, const void* src, size_t bytes, void* stream) {
    return fill_device(dst, src, bytes, (hipStream_t)stream) == MADD_OK;
  }
};
HipTables g_hip_tables;
madd_cache::TableCache<HipTables> g_tables;

// Descriptor tables of madd_multi_tensor_step_noalloc: a fixed device array,
// one per GPU the library runs on, held until the process ends.  Every call on
// a GPU rewrites it on its stream before its launches read it, so calls on one
// GPU that overlap in time (other streams, other threads) race.
constexpr int kScratchTensors = 4096;
static __device__ __align__(256) TensorDesc scratch[kScratchTensors];

// The array's device address on each GPU (host code must not pass the
// array's name to a kernel: that is a host-side stand-in).  Looked up once per
// device, with that device current.
std::mutex g_scratch_mu;
std::vector<TensorDesc*> g_scratch_ptr;

int32_t scratch_on_device(int dev, TensorDesc** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (dev < 0) return MADD_EDEVICE;
  if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize((size_t)dev + 1, nullptr);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MADD_EDEVICE;
    g_scratch_ptr[dev] = (TensorDesc*)p;
  }
  *out = g_scratch_ptr[dev];
  return MADD_OK;
}

int32_t cache_status(int rc) {
  switch (rc) {
    case madd_cache::kOk: return MADD_OK;
    case madd_cache::kCaptureMiss: return MADD_ECAPTURE;
    case madd_cache::kNoMem: return MADD_ENOMEM;
    default: return MADD_EDEVICE;
  }
}

// Identity of a stream for the cache: its handle, except for the per-thread
// default stream, whose one handle names a different stream in every thread.
uint64_t stream_key(hipStream_t stream) {
  if (stream != hipStreamPerThread) return (uint64_t)(uintptr_t)stream;
  static std::atomic<uint64_t> next{1};
  thread_local const uint64_t id = (1ull << 63) | next.fetch_add(1);
  return id;
}

// Whether `stream` is capturing a graph.
int32_t capturing(hipStream_t stream, bool* cap) {
  hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &st) != hipSuccess) return MADD_EDEVICE;
  *cap = st != hipStreamCaptureStatusNone;
  return MADD_OK;
}

int32_t launch(step_fn fn, const TensorDesc* table, int ntab, const TensorDesc& single,
               int64_t nchunks, const Scalars& s, const Scalars* sdev, hipStream_t stream) {
  if (nchunks <= 0) return MADD_OK;
  if (nchunks > 0x7FFFFFFFll) return MADD_EUNSUPPORTED;
  return launch_k(fn, dim3((unsigned)nchunks), dim3(kThreads), stream, table, ntab, single, s,
                  sdev);
}

// NVFP4 with current scaling: clear the amax words (one thread per tensor),
// then the passes.  Consecutive tensors form groups of at least
// `group_chunks` chunks; launch j runs pass 1 of group j together with
// pass 2 of group j - 1 (whose amax words launch j - 1 completed), so a
// list of G groups takes G + 1 launches after the clear.  `descs` holds the
// launch's tensors in table order (null for the single tensor of madd_step).
//
// Measured on the 7B list's NVFP4 linear layers (same process): with fp32
// moments pass 1 is bound by HBM and pass 2 by VALU, and overlapping them
// takes the step from 47.2 ms (one group) to 43.8 ms with groups of at
// least 40960 chunks (two groups per transformer layer; 36864-49152: within
// 0.2 ms; 57344 and 65536: 45.2-45.5; 16384: 49.0, launch tails).  Keeping
// w' in the Infinity Cache between the passes (temporal stores and loads,
// pass 2 reading its group newest first) gained at most 0.3% more.  With
// bf16 moments both passes are VALU bound, and the same groups take the
// step from 39.3 ms (one group) to 38.8 ms (65536: 40.9; 98304: 43.7).
constexpr int64_t kNvcsGroupChunks = 40960;

int32_t launch_nvcs(const NvcsKernels& k, const TensorDesc* table, int ntab,
                    const TensorDesc& single, const std::vector<TensorDesc>* descs,
                    int64_t group_chunks, int64_t nchunks, const Scalars& s, const Scalars* sdev,
                    hipStream_t stream) {
  if (nchunks <= 0) return MADD_OK;
  if (nchunks > 0x7FFFFFFFll) return MADD_EUNSUPPORTED;
  std::vector<int64_t> cut{0};  // group boundaries in chunk space
  if (descs) {
    for (size_t i = 0; i < descs->size(); ++i) {
      const int64_t end = (*descs)[i].chunk0 + chunks_of((*descs)[i].n);
      if (end - cut.back() >= group_chunks || i + 1 == descs->size()) cut.push_back(end);
    }
  } else {
    cut.push_back(nchunks);
  }
  const unsigned clear_grid = (unsigned)(((ntab == 0 ? 1 : ntab) + kThreads - 1) / kThreads);
  int32_t rc = launch_k(k.clear, dim3(clear_grid), dim3(kThreads), stream, table, ntab, single, s,
                        sdev);
  const size_t groups = cut.size() - 1;
  for (size_t j = 0; j <= groups && rc == MADD_OK; ++j) {
    NvcsSpan sp = {0, 0, 0, 0};
    if (j < groups) {
      sp.a1 = cut[j];
      sp.n1 = cut[j + 1] - cut[j];
    }
    if (j > 0) {
      sp.a2 = cut[j - 1];
      sp.n2 = cut[j] - cut[j - 1];
    }
    rc = launch_k(k.step, dim3((unsigned)(sp.n1 + sp.n2)), dim3(kThreads), stream, table, ntab,
                  single, s, sdev, sp);
  }
  return rc;
}

TensorDesc make_desc(void* w, void* scales, uint16_t* copy, const void* g, void* m, void* v,
                     void* ve, int64_t n, int64_t gbase) {
  TensorDesc d;
  memset(&d, 0, sizeof(d));
  d.w = w;
  d.g = g;
  d.m = m;
  d.v = v;
  d.ve = ve;
  d.scales = scales;
  d.copy = copy;
  d.n = n;
  d.gbase = gbase;
  d.chunk0 = 0;
  d.vec_ok = al16(w) && al16(g) && al16(m) && al16(v) && al16(ve) && (!copy || al16(copy)) &&
             (gbase & 7) == 0;
  return d;
}

bool block_scaled_fmt(int32_t f) {
  return f == MADD_W_FP8_E4M3 || f == MADD_W_FP8_E5M2 || fp4_fmt(f);
}
int64_t block_len_of(int32_t f) {
  return f == MADD_W_MXFP4 ? kMxBlock : (nv_fmt(f) ? kNvBlock : kBlock);
}

constexpr int64_t kMaxN = (int64_t)1 << 60;  // elements per tensor (byte sizes fit 64 bits)

// Bytes one tensor of n elements occupies in each of its buffers.
uint64_t code_bytes(int32_t wfmt, int64_t n) {
  switch (wfmt) {
    case MADD_W_BF16: return 2ull * (uint64_t)n;
    case MADD_W_FP32: return 4ull * (uint64_t)n;
    case MADD_W_FP8_E4M3:
    case MADD_W_FP8_E5M2: return (uint64_t)n;
    default: return ((uint64_t)n + 1u) / 2u;  // two E2M1 codes per byte
  }
}
uint64_t scale_bytes(int32_t wfmt, int64_t n) {
  const uint64_t u = (uint64_t)n;
  switch (wfmt) {
    case MADD_W_MXFP4: return u / kMxBlock;
    case MADD_W_NVFP4: return 4u + u / kNvBlock;
    case MADD_W_NVFP4_CURRENT: return 8u + u / kNvBlock;
    default: return 2u * (u / kBlock);
  }
}

// The buffers of one tensor must be pairwise disjoint byte ranges (the
// kernels read and write them in place, in no fixed order between arrays).
bool disjoint(const void* const* p, const uint64_t* bytes, int k) {
  for (int i = 0; i < k; ++i) {
    if (!p[i] || bytes[i] == 0) continue;
    const uintptr_t a0 = (uintptr_t)p[i], a1 = a0 + bytes[i];
    for (int j = i + 1; j < k; ++j) {
      if (!p[j] || bytes[j] == 0) continue;
      const uintptr_t b0 = (uintptr_t)p[j], b1 = b0 + bytes[j];
      if (a0 < b1 && b0 < a1) return false;
    }
  }
  return true;
}

int32_t check_tensor(void* w, int32_t wfmt, void* scales, uint16_t* copy, const void* g,
                     int32_t gfmt, void* m, void* v, void* ve, int32_t sfmt, int64_t n) {
  if (n < 0 || n > kMaxN) return MADD_EINVAL;
  if (n == 0) return MADD_OK;
  if (!w || !g || !m || !v || !ve) return MADD_EINVAL;
  if (!valid_wfmt(wfmt)) return MADD_EINVAL;
  if (fp4_fmt(wfmt) && !scales) return MADD_EINVAL;
  if (scales) {
    if (!block_scaled_fmt(wfmt)) return MADD_EINVAL;
    if (n % block_len_of(wfmt) != 0) return MADD_EINVAL;
    if (nv_fmt(wfmt) && ((uintptr_t)scales & 3u) != 0) return MADD_EALIGN;
    if (!(al16(w) && al16(g) && al16(m) && al16(v) && al16(ve) && (!copy || al16(copy))))
      return MADD_EALIGN;
  }
  const uint64_t u = (uint64_t)n;
  const uint64_t sb = (sfmt == MADD_S_FP32 ? 4u : 2u) * u;
  const void* const p[7] = {w, scales, copy, g, m, v, ve};
  const uint64_t b[7] = {code_bytes(wfmt, n), scales ? scale_bytes(wfmt, n) : 0u, 2u * u,
                         (gfmt == MADD_G_FP32 ? 4u : 2u) * u, sb, sb, sb};
  if (!disjoint(p, b, 7)) return MADD_EINVAL;
  return MADD_OK;
}

#endif  // MADD_IN_PART(0)
}  // namespace madd_detail

#if MADD_IN_PART(0)
// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

using namespace madd_detail;

// The multi-tensor step; `sdev`, when not null, is the device copy of the
// hyper-parameter scalars the kernels read when they run (`hp` then only
// selects the kernels: rounding mode and whether the clamps apply).
static int32_t multi_tensor_step(int32_t ntensors, void* const* w, const int32_t* wfmt,
                                 void* const* scales, uint16_t* const* copy,
                                 const void* const* g, int32_t gfmt,
                                 void* const* m, void* const* v, void* const* ve, int32_t sfmt,
                                 const int64_t* numel, int64_t index_base,
                                 const madd_hparams* hp, const Scalars* sdev, void* stream,
                                 bool noalloc = false) {
  int32_t rc = check_hparams(hp);
  if (rc != MADD_OK) return rc;
  if (ntensors < 0 || !valid_gfmt(gfmt) || !valid_sfmt(sfmt) || index_base < 0)
    return MADD_EINVAL;
  if (ntensors == 0) return MADD_OK;
  if (!w || !wfmt || !g || !m || !v || !ve || !numel) return MADD_EINVAL;
  int64_t total = 0;
  for (int32_t i = 0; i < ntensors; ++i) {
    if (!valid_wfmt(wfmt[i])) return MADD_EINVAL;
    if (wfmt[i] == MADD_W_NVFP4_CURRENT && gfmt != MADD_G_FP32 && numel[i] > 0)
      return MADD_EINVAL;  // w' is written over the fp32 gradient
    rc = check_tensor(w[i], wfmt[i], scales ? scales[i] : nullptr, copy ? copy[i] : nullptr, g[i],
                      gfmt, m[i], v[i], ve[i], sfmt, numel[i]);
    if (rc != MADD_OK) return rc;
    if (numel[i] > INT64_MAX - index_base - total) return MADD_EINVAL;
    total += numel[i];
  }
  const Scalars s = make_scalars(*hp);
  const bool sr = hp->rounding == MADD_ROUND_SR;
  // One launch per (format, scaled) group; global indices follow list order.
  // All tables are prepared before the first launch.
  struct Group {
    step_fn fn;  // null for NVFP4 with current scaling, which launches `nvcs`
    NvcsKernels nvcs;
    std::vector<TensorDesc> descs;
    int64_t nchunks;
    const TensorDesc* table;
    size_t slot;
  };
  std::vector<Group> groups;
  for (int wf = MADD_W_BF16; wf <= MADD_W_NVFP4_CURRENT; ++wf) {
    for (int blk = 0; blk <= 1; ++blk) {
      std::vector<TensorDesc> descs;
      int64_t gbase = index_base, nch = 0;
      for (int32_t i = 0; i < ntensors; ++i) {
        const bool is_blk = scales && scales[i];
        if (wfmt[i] == wf && (int)is_blk == blk && numel[i] > 0) {
          TensorDesc d = make_desc(w[i], is_blk ? scales[i] : nullptr, copy ? copy[i] : nullptr,
                                   g[i], m[i], v[i], ve[i], numel[i], gbase);
          d.chunk0 = nch;
          nch += chunks_of(numel[i]);
          descs.push_back(d);
        }
        gbase += numel[i];
      }
      if (descs.empty()) continue;
      if (nch > 0x7FFFFFFFll) return MADD_EUNSUPPORTED;
      bool any_copy = false;
      for (const TensorDesc& d : descs) any_copy = any_copy || d.copy != nullptr;
      step_fn fn = nullptr;
      NvcsKernels nvcs = {nullptr, nullptr};
      if (wf == MADD_W_NVFP4_CURRENT) {
        nvcs = pick_part9(sfmt, sr, needs_clamp(*hp), any_copy);
      } else {
        fn = pick_kernel(wf, gfmt, sfmt, sr, needs_clamp(*hp), any_copy, blk != 0);
        if (!fn) return MADD_EUNSUPPORTED;
      }
      groups.push_back(Group{fn, nvcs, std::move(descs), nch, nullptr, 0});
    }
  }
  hipStream_t st = (hipStream_t)stream;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MADD_EDEVICE;
  TensorDesc none;
  memset(&none, 0, sizeof(none));
  if (noalloc) {
    // The tables of every group, back to back in this GPU's scratch array,
    // written on the stream ahead of the launches that read them.
    size_t total = 0;
    for (const Group& gr : groups) total += gr.descs.size();
    if (total > (size_t)kScratchTensors) return MADD_ESCRATCH;
    TensorDesc* base = nullptr;
    rc = scratch_on_device(dev, &base);
    if (rc != MADD_OK) return rc;
    size_t off = 0;
    for (Group& gr : groups) {
      gr.table = base + off;
      off += gr.descs.size();
    }
    for (const Group& gr : groups) {
      rc = fill_device((void*)gr.table, gr.descs.data(), gr.descs.size() * sizeof(TensorDesc), st);
      if (rc != MADD_OK) return rc;
    }
    for (const Group& gr : groups) {
      const int ntab = (int)gr.descs.size();
      rc = gr.fn ? launch(gr.fn, gr.table, ntab, none, gr.nchunks, s, sdev, st)
                 : launch_nvcs(gr.nvcs, gr.table, ntab, none, &gr.descs, kNvcsGroupChunks,
                               gr.nchunks, s, sdev, st);
      if (rc != MADD_OK) return rc;
    }
    return MADD_OK;
  }
  bool cap = false;
  rc = capturing(st, &cap);
  if (rc != MADD_OK) return rc;
  size_t acquired = 0;
  for (; acquired < groups.size(); ++acquired) {
    Group& gr = groups[acquired];
    void* t = nullptr;
    rc = cache_status(g_tables.acquire(g_hip_tables, dev, stream_key(st), gr.descs.data(),
                                       gr.descs.size() * sizeof(TensorDesc), cap, st, &t,
                                       &gr.slot));
    if (rc != MADD_OK) break;
    gr.table = (const TensorDesc*)t;
  }
  for (size_t k = 0; k < acquired && rc == MADD_OK; ++k) {
    const Group& gr = groups[k];
    const int ntab = (int)gr.descs.size();
    rc = gr.fn ? launch(gr.fn, gr.table, ntab, none, gr.nchunks, s, sdev, st)
               : launch_nvcs(gr.nvcs, gr.table, ntab, none, &gr.descs, kNvcsGroupChunks,
                             gr.nchunks, s, sdev, st);
  }
  for (size_t k = 0; k < acquired; ++k) g_tables.release(groups[k].slot);
  return rc;
}


extern "C" {

const char* madd_status_string(int32_t status) {
  switch (status) {
    case MADD_OK: return "MADD_OK";
    case MADD_EINVAL: return "MADD_EINVAL: invalid argument";
    case MADD_EALIGN: return "MADD_EALIGN: block-scaled buffers must be 16-byte aligned";
    case MADD_EUNSUPPORTED: return "MADD_EUNSUPPORTED: request not implemented";
    case MADD_EDEVICE: return "MADD_EDEVICE: HIP runtime or launch failure";
    case MADD_ENOMEM: return "MADD_ENOMEM: device allocation failed";
    case MADD_ESCRATCH:
      return "MADD_ESCRATCH: more tensors than the allocation-free step's fixed table holds "
             "(4096)";
    case MADD_ECAPTURE:
      return "MADD_ECAPTURE: a tensor list's first step cannot run inside a graph capture "
             "(step it once outside the capture)";
    default: return "unknown madd status";
  }
}

int32_t madd_init_state(void* m, void* v, void* ve, int32_t sfmt, int64_t n, void* stream) {
  if (n < 0 || n > kMaxN || !valid_sfmt(sfmt)) return MADD_EINVAL;
  if (n == 0) return MADD_OK;
  if (!m || !v || !ve) return MADD_EINVAL;
  {
    const uint64_t sb = (sfmt == MADD_S_FP32 ? 4u : 2u) * (uint64_t)n;
    const void* const p[3] = {m, v, ve};
    const uint64_t b[3] = {sb, sb, sb};
    if (!disjoint(p, b, 3)) return MADD_EINVAL;
  }
  const int64_t want = (n + kThreads - 1) / kThreads;
  const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
  hipStream_t st = (hipStream_t)stream;
  void* arr[3] = {m, v, ve};
  for (void* p : arr) {
    const int32_t rc =
        sfmt == MADD_S_FP32
            ? launch_k(zero_kernel<float>, dim3(grid), dim3(kThreads), st, (float*)p, n)
            : launch_k(zero_kernel<uint16_t>, dim3(grid), dim3(kThreads), st, (uint16_t*)p, n);
    if (rc != MADD_OK) return rc;
  }
  return MADD_OK;
}

int32_t madd_encode_weights(const float* x, void* w, int32_t wfmt, void* scales, int64_t n,
                            void* stream) {
  if (n < 0 || n > kMaxN || !valid_wfmt(wfmt)) return MADD_EINVAL;
  if (n == 0) return MADD_OK;
  if (!x || !w) return MADD_EINVAL;
  if (fp4_fmt(wfmt) && !scales) return MADD_EINVAL;
  if (nv_fmt(wfmt)) {
    if (n % kNvBlock != 0) return MADD_EINVAL;
    if (((uintptr_t)scales & 3u) != 0) return MADD_EALIGN;
  } else if (wfmt == MADD_W_MXFP4) {
    if (n % kMxBlock != 0) return MADD_EINVAL;
  } else if (scales) {
    if (wfmt != MADD_W_FP8_E4M3 && wfmt != MADD_W_FP8_E5M2) return MADD_EINVAL;
    if (n % kBlock != 0) return MADD_EINVAL;
  }
  {
    const void* const p[3] = {x, w, scales};
    const uint64_t b[3] = {4u * (uint64_t)n, code_bytes(wfmt, n),
                           scales ? scale_bytes(wfmt, n) : 0u};
    if (!disjoint(p, b, 3)) return MADD_EINVAL;
  }
  hipStream_t st = (hipStream_t)stream;
  if (nv_fmt(wfmt)) {
    uint32_t* slot = (uint32_t*)scales;
    const int head = wfmt == MADD_W_NVFP4 ? 4 : 8;  // current scaling: st, amax word
    const int64_t nb = n / kNvBlock;
    const int64_t want_x = (n + kThreads - 1) / kThreads, want_b = (nb + kThreads - 1) / kThreads;
    const unsigned grid_x = (unsigned)(want_x < 4096 ? want_x : 4096);
    const unsigned grid_b = (unsigned)(want_b < 65536 ? want_b : 65536);
    int32_t rc = launch_k(nv_clear_kernel, dim3(1), dim3(64), st, slot, head / 4);
    if (rc == MADD_OK) rc = launch_k(nv_amax_kernel, dim3(grid_x), dim3(kThreads), st, x, n, slot);
    if (rc == MADD_OK) rc = launch_k(nv_scale_kernel, dim3(1), dim3(64), st, slot);
    if (rc == MADD_OK)
      rc = launch_k(encode_nv_kernel, dim3(grid_b), dim3(kThreads), st, x, (uint8_t*)w,
                    (uint8_t*)scales, nb, head);
    return rc;
  }
  if (wfmt == MADD_W_MXFP4) {
    const int64_t nb = n / kMxBlock;
    const int64_t want = (nb + kThreads - 1) / kThreads;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    return launch_k(encode_mx_kernel, dim3(grid), dim3(kThreads), st, x, (uint8_t*)w,
                    (uint8_t*)scales, nb);
  }
  if (scales) {
    const int64_t nb = n / kBlock;
    const int64_t want = (nb + kThreads - 1) / kThreads;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    return wfmt == MADD_W_FP8_E4M3
               ? launch_k(encode_block_kernel<WF_E4M3>, dim3(grid), dim3(kThreads), st, x,
                          (uint8_t*)w, (uint16_t*)scales, nb)
               : launch_k(encode_block_kernel<WF_E5M2>, dim3(grid), dim3(kThreads), st, x,
                          (uint8_t*)w, (uint16_t*)scales, nb);
  }
  const int64_t want = (n + kThreads - 1) / kThreads;
  const dim3 grid((unsigned)(want < 65536 ? want : 65536)), block(kThreads);
  switch (wfmt) {
    case MADD_W_BF16: return launch_k(encode_kernel<WF_BF16>, grid, block, st, x, w, n);
    case MADD_W_FP8_E4M3: return launch_k(encode_kernel<WF_E4M3>, grid, block, st, x, w, n);
    case MADD_W_FP8_E5M2: return launch_k(encode_kernel<WF_E5M2>, grid, block, st, x, w, n);
    default: return launch_k(encode_kernel<WF_FP32>, grid, block, st, x, w, n);
  }
}

int32_t madd_step(void* w, int32_t wfmt, void* scales, uint16_t* copy, const void* g,
                  int32_t gfmt, void* m, void* v, void* ve, int32_t sfmt, int64_t n,
                  int64_t index_base, const madd_hparams* hp, void* stream) {
  int32_t rc = check_hparams(hp);
  if (rc != MADD_OK) return rc;
  if (!valid_wfmt(wfmt) || !valid_gfmt(gfmt) || !valid_sfmt(sfmt) || index_base < 0)
    return MADD_EINVAL;
  rc = check_tensor(w, wfmt, scales, copy, g, gfmt, m, v, ve, sfmt, n);
  if (rc != MADD_OK) return rc;
  if (n == 0) return MADD_OK;
  if (n > INT64_MAX - index_base) return MADD_EINVAL;
  const Scalars s = make_scalars(*hp);
  if (wfmt == MADD_W_NVFP4_CURRENT) {
    if (gfmt != MADD_G_FP32) return MADD_EINVAL;  // w' is written over the fp32 gradient
    const NvcsKernels k = pick_part9(sfmt, hp->rounding == MADD_ROUND_SR, needs_clamp(*hp),
                                     copy != nullptr);
    const TensorDesc d = make_desc(w, scales, copy, g, m, v, ve, n, index_base);
    return launch_nvcs(k, nullptr, 0, d, nullptr, INT64_MAX, chunks_of(n), s, nullptr,
                       (hipStream_t)stream);
  }
  step_fn fn = pick_kernel(wfmt, gfmt, sfmt, hp->rounding == MADD_ROUND_SR, needs_clamp(*hp),
                           copy != nullptr, scales != nullptr);
  if (!fn) return MADD_EUNSUPPORTED;
  const TensorDesc d = make_desc(w, scales, copy, g, m, v, ve, n, index_base);
  return launch(fn, nullptr, 0, d, chunks_of(n), s, nullptr, (hipStream_t)stream);
}

int32_t madd_plain_step(void* w, int32_t wfmt, const void* g, int32_t gfmt, int64_t n,
                        int64_t index_base, const madd_hparams* hp, void* stream) {
  int32_t rc = check_hparams(hp);
  if (rc != MADD_OK) return rc;
  if (!valid_wfmt(wfmt) || !valid_gfmt(gfmt) || index_base < 0 || n < 0 || n > kMaxN)
    return MADD_EINVAL;
  if (fp4_fmt(wfmt)) return MADD_EINVAL;  // block-scaled: no scale argument here
  if (n == 0) return MADD_OK;
  if (!w || !g) return MADD_EINVAL;
  if (n > INT64_MAX - index_base) return MADD_EINVAL;
  {
    const void* const p[2] = {w, g};
    const uint64_t b[2] = {code_bytes(wfmt, n), (gfmt == MADD_G_FP32 ? 4u : 2u) * (uint64_t)n};
    if (!disjoint(p, b, 2)) return MADD_EINVAL;
  }
  const Scalars s = make_scalars(*hp);
  const bool sr = hp->rounding == MADD_ROUND_SR;
  plain_fn fn = nullptr;
  switch (wfmt) {
    case MADD_W_BF16: fn = pick_plain_gf<WF_BF16>(gfmt, sr); break;
    case MADD_W_FP8_E4M3: fn = pick_plain_gf<WF_E4M3>(gfmt, sr); break;
    case MADD_W_FP8_E5M2: fn = pick_plain_gf<WF_E5M2>(gfmt, sr); break;
    default: fn = pick_plain_gf<WF_FP32>(gfmt, sr); break;
  }
  const int64_t want = (n + (int64_t)kThreads * kQuad - 1) / ((int64_t)kThreads * kQuad);
  const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
  return launch_k(fn, dim3(grid), dim3(kThreads), (hipStream_t)stream, w, g, n, index_base,
                  (float)hp->lr_add, s);
}

int32_t madd_toy_gradient(const void* w, int32_t wfmt, const float* target, const float* c,
                          const int64_t* idx, int64_t batch, int64_t n, int32_t* counts,
                          float* g, void* stream) {
  if (n < 0 || n > kMaxN || batch < 0 || batch > kMaxN) return MADD_EINVAL;
  if (!valid_wfmt(wfmt) || fp4_fmt(wfmt)) return MADD_EINVAL;
  if (n == 0) return MADD_OK;
  if (!w || !target || !c || !counts || !g || (batch > 0 && !idx)) return MADD_EINVAL;
  {
    const uint64_t u = (uint64_t)n;
    const void* const p[6] = {w, target, c, counts, g, idx};
    const uint64_t b[6] = {code_bytes(wfmt, n), 4u * u, 4u * u, 4u * u, 4u * u,
                           8u * (uint64_t)batch};
    if (!disjoint(p, b, 6)) return MADD_EINVAL;
  }
  hipStream_t st = (hipStream_t)stream;
  const int64_t want = (n + kThreads - 1) / kThreads;
  const dim3 grid((unsigned)(want < 65536 ? want : 65536)), block(kThreads);
  int32_t rc = launch_k(zero_kernel<uint32_t>, grid, block, st, (uint32_t*)counts, n);
  if (rc == MADD_OK && batch > 0) {
    const int64_t wb = (batch + kThreads - 1) / kThreads;
    rc = launch_k(toy_count_kernel, dim3((unsigned)(wb < 65536 ? wb : 65536)), block, st, idx,
                  batch, n, counts);
  }
  if (rc != MADD_OK) return rc;
  const float fob = (float)(4.0 / (double)(batch > 0 ? batch : 1));
  switch (wfmt) {
    case MADD_W_BF16:
      return launch_k(toy_grad_kernel<WF_BF16>, grid, block, st, w, target, c, counts, n, fob, g);
    case MADD_W_FP8_E4M3:
      return launch_k(toy_grad_kernel<WF_E4M3>, grid, block, st, w, target, c, counts, n, fob, g);
    case MADD_W_FP8_E5M2:
      return launch_k(toy_grad_kernel<WF_E5M2>, grid, block, st, w, target, c, counts, n, fob, g);
    default:
      return launch_k(toy_grad_kernel<WF_FP32>, grid, block, st, w, target, c, counts, n, fob, g);
  }
}

int32_t madd_multi_tensor_step(int32_t ntensors, void* const* w, const int32_t* wfmt,
                               void* const* scales, uint16_t* const* copy,
                               const void* const* g, int32_t gfmt,
                               void* const* m, void* const* v, void* const* ve, int32_t sfmt,
                               const int64_t* numel, int64_t index_base, const madd_hparams* hp,
                               void* stream) {
  return multi_tensor_step(ntensors, w, wfmt, scales, copy, g, gfmt, m, v, ve, sfmt, numel,
                           index_base, hp, nullptr, stream);
}

int64_t madd_scalars_bytes(void) { return (int64_t)sizeof(Scalars); }

int32_t madd_prepare_scalars(const madd_hparams* hp, void* out) {
  const int32_t rc = check_hparams(hp);
  if (rc != MADD_OK) return rc;
  if (!out) return MADD_EINVAL;
  const Scalars s = make_scalars(*hp);
  memcpy(out, &s, sizeof(s));
  return MADD_OK;
}

int32_t madd_multi_tensor_step_dev(int32_t ntensors, void* const* w, const int32_t* wfmt,
                                   void* const* scales, uint16_t* const* copy,
                                   const void* const* g, int32_t gfmt,
                                   void* const* m, void* const* v, void* const* ve,
                                   int32_t sfmt, const int64_t* numel, int64_t index_base,
                                   const madd_hparams* hp, const void* dev_scalars,
                                   void* stream) {
  if (!dev_scalars) return MADD_EINVAL;
  if (((uintptr_t)dev_scalars & 3u) != 0) return MADD_EALIGN;
  return multi_tensor_step(ntensors, w, wfmt, scales, copy, g, gfmt, m, v, ve, sfmt, numel,
                           index_base, hp, (const Scalars*)dev_scalars, stream);
}

int32_t madd_multi_tensor_step_noalloc(int32_t ntensors, void* const* w, const int32_t* wfmt,
                                       void* const* scales, uint16_t* const* copy,
                                       const void* const* g, int32_t gfmt, void* const* m,
                                       void* const* v, void* const* ve, int32_t sfmt,
                                       const int64_t* numel, int64_t index_base,
                                       const madd_hparams* hp, void* stream) {
  return multi_tensor_step(ntensors, w, wfmt, scales, copy, g, gfmt, m, v, ve, sfmt, numel,
                           index_base, hp, nullptr, stream, true);
}

}  // extern "C"
#endif  // MADD_IN_PART(0)
