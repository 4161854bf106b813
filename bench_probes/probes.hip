// Device probes declared in madd_probes.h (measurement only; not part of the
// optimizer library).
//
// Plain read-only, write-only and copy streams (madd_stream_modes) measure
// what HBM delivers for each direction alone in the same access shape.
//
// Streaming-ceiling probe for the M+Adam step: the step kernel's bytes and
// work mapping without its arithmetic.  A workgroup of 256 threads owns 2048 elements; thread t
// moves elements [4t, 4t+4) of both 1024-element sub-tiles, all loads of a
// tile issued before any store, every access non-temporal.  Values are
// XORed with gradient bits masked by a runtime zero, so the stores write
// back what was read while the compiler must keep every load and store.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "madd_probes.h"

namespace {

constexpr int kThreads = 256;
constexpr int kQuad = 4;
constexpr int kSub = kThreads * kQuad;
constexpr int kTile = 2 * kSub;

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));

#define GLOBAL __attribute__((address_space(1)))

template <typename T>
__device__ __forceinline__ T ldg(const void* p) {
  return __builtin_nontemporal_load((const GLOBAL T*)p);
}
template <typename T>
__device__ __forceinline__ void stg(void* p, T x) {
  __builtin_nontemporal_store(x, (GLOBAL T*)p);
}

// State lanes of four elements: fp32 (u4) or bf16 codes (u2).
template <int SB>
struct StateT;
template <>
struct StateT<4> {
  typedef u4 T;
  static __device__ __forceinline__ T mix(T x, u4 g, uint32_t mask) { return x ^ (g & mask); }
};
template <>
struct StateT<2> {
  typedef u2 T;
  static __device__ __forceinline__ T mix(T x, u4 g, uint32_t mask) {
    return x ^ (u2{g.x ^ g.y, g.z ^ g.w} & mask);
  }
};

template <int SB>
__global__ __launch_bounds__(kThreads) void ceiling_kernel(void* w, const float* g, void* m,
                                                           void* v, void* ve, int64_t n,
                                                           uint32_t mask) {
  typedef typename StateT<SB>::T S;
  const int64_t tb = (int64_t)blockIdx.x * kTile;
  const int64_t eA = tb + (int64_t)threadIdx.x * kQuad, eB = eA + kSub;
  if (eB + kQuad <= n) {
    u2 wa = ldg<u2>((const uint16_t*)w + eA), wb = ldg<u2>((const uint16_t*)w + eB);
    const u4 ga = ldg<u4>(g + eA), gb = ldg<u4>(g + eB);
    S ma = ldg<S>((const uint8_t*)m + eA * SB), mb = ldg<S>((const uint8_t*)m + eB * SB);
    S va = ldg<S>((const uint8_t*)v + eA * SB), vb = ldg<S>((const uint8_t*)v + eB * SB);
    S ea = ldg<S>((const uint8_t*)ve + eA * SB), eb = ldg<S>((const uint8_t*)ve + eB * SB);
    wa ^= u2{ga.x, ga.z} & mask;
    wb ^= u2{gb.x, gb.z} & mask;
    stg<u2>((uint16_t*)w + eA, wa);
    stg<S>((uint8_t*)m + eA * SB, StateT<SB>::mix(ma, ga, mask));
    stg<S>((uint8_t*)v + eA * SB, StateT<SB>::mix(va, ga, mask));
    stg<S>((uint8_t*)ve + eA * SB, StateT<SB>::mix(ea, ga, mask));
    stg<u2>((uint16_t*)w + eB, wb);
    stg<S>((uint8_t*)m + eB * SB, StateT<SB>::mix(mb, gb, mask));
    stg<S>((uint8_t*)v + eB * SB, StateT<SB>::mix(vb, gb, mask));
    stg<S>((uint8_t*)ve + eB * SB, StateT<SB>::mix(eb, gb, mask));
    return;
  }
  // the last, partial tile: element by element
  for (int half = 0; half < 2; ++half) {
    const int64_t e0 = half ? eB : eA;
    for (int64_t i = e0; i < e0 + kQuad && i < n; ++i) {
      const uint32_t gi = __float_as_uint(g[i]) & mask;
      ((uint16_t*)w)[i] ^= (uint16_t)gi;
      if (SB == 4) {
        ((uint32_t*)m)[i] ^= gi;
        ((uint32_t*)v)[i] ^= gi;
        ((uint32_t*)ve)[i] ^= gi;
      } else {
        ((uint16_t*)m)[i] ^= (uint16_t)gi;
        ((uint16_t*)v)[i] ^= (uint16_t)gi;
        ((uint16_t*)ve)[i] ^= (uint16_t)gi;
      }
    }
  }
}

bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// bf16 conversion instructions against the integer definitions.
typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
typedef short s2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t hash32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return x;
}

// 65536 workgroups x 256 threads x 256 inputs = 2^32 inputs.
__global__ __launch_bounds__(256) void bf16_rounding_kernel(unsigned long long* c) {
  const uint32_t base = ((uint32_t)blockIdx.x * 256u + threadIdx.x) * 256u;
  unsigned long long rne_bad = 0, sr_bad = 0, nan_bad = 0;
  for (uint32_t j = 0; j < 256u; ++j) {
    const uint32_t u = base + j;
    const float x = __uint_as_float(u);
    const uint32_t r16 = hash32(u) & 0xFFFFu;
    const uint32_t hw = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2v{x, x}, bf2v)) & 0xFFFFu;
    const uint32_t hs = __builtin_bit_cast(
        uint32_t, __builtin_amdgcn_cvt_sr_bf16_f32(s2v{0, 0}, x, r16 << 16, false)) & 0xFFFFu;
    if ((u & 0x7FFFFFFFu) <= 0x7F800000u) {
      rne_bad += hw != ((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
      sr_bad += hs != ((u + r16) >> 16);
    }
  }
  if (blockIdx.x == 0) {  // the canonical NaN under every 16-bit draw
    const float q = __uint_as_float(0x7FC00000u);
    for (uint32_t r = threadIdx.x; r < 65536u; r += 256u) {
      const uint32_t hw = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2v{q, q}, bf2v)) & 0xFFFFu;
      const uint32_t hs = __builtin_bit_cast(
          uint32_t, __builtin_amdgcn_cvt_sr_bf16_f32(s2v{0, 0}, q, r << 16, false)) & 0xFFFFu;
      nan_bad += (hw != 0x7FC0u) + (hs != 0x7FC0u);
    }
  }
  if (rne_bad) atomicAdd(&c[0], rne_bad);
  if (sr_bad) atomicAdd(&c[1], sr_bad);
  if (nan_bad) atomicAdd(&c[2], nan_bad);
  if (threadIdx.x == 0) atomicAdd(&c[3], 256ull * 256ull);  // this workgroup's inputs
}

// Plain streams in the step's access shape: a 256-thread workgroup owns one
// 8 KiB tile and thread t moves 16 bytes at offset 16 t of each 4 KiB half,
// non-temporal.  Read: the loads feed an XOR that is stored (to the sink's
// first 4 KiB) only if it equals `key`, so the compiler keeps every load.
constexpr int64_t kStreamTile = 8192;
constexpr int kHalf16 = 256;  // 16-byte words per half tile

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u4* a, u4* sink, uint32_t key) {
  const int64_t i = (int64_t)blockIdx.x * (2 * kHalf16) + threadIdx.x;
  const u4 x = ldg<u4>(a + i), y = ldg<u4>(a + i + kHalf16);
  const u4 z = x ^ y;
  if ((z.x ^ z.y ^ z.z ^ z.w) == key) sink[threadIdx.x] = z;
}
__global__ __launch_bounds__(kThreads) void stream_write_kernel(u4* b) {
  const int64_t i = (int64_t)blockIdx.x * (2 * kHalf16) + threadIdx.x;
  const uint32_t v = (uint32_t)i, u = v + (uint32_t)kHalf16;  // word k holds k
  stg<u4>(b + i, u4{v, v, v, v});
  stg<u4>(b + i + kHalf16, u4{u, u, u, u});
}
__global__ __launch_bounds__(kThreads) void stream_copy_kernel(const u4* a, u4* b) {
  const int64_t i = (int64_t)blockIdx.x * (2 * kHalf16) + threadIdx.x;
  const u4 x = ldg<u4>(a + i), y = ldg<u4>(a + i + kHalf16);
  stg<u4>(b + i, x);
  stg<u4>(b + i + kHalf16, y);
}

}  // namespace

extern "C" int32_t madd_stream_modes(int32_t mode, const void* a, void* b, int64_t bytes,
                                     void* stream) {
  if (mode < 0 || mode > 2 || bytes <= 0 || bytes % kStreamTile != 0) return -1;
  if (!b || (mode != 1 && !a)) return -1;
  if (!al16(b) || (mode != 1 && !al16(a))) return -2;
  const int64_t tiles = bytes / kStreamTile;
  if (tiles > 0x7FFFFFFFll) return -1;
  hipStream_t st = (hipStream_t)stream;
  const dim3 grid((unsigned)tiles);
  if (mode == 0)
    hipLaunchKernelGGL(stream_read_kernel, grid, dim3(kThreads), 0, st, (const u4*)a, (u4*)b,
                       0x9E3779B9u);
  else if (mode == 1)
    hipLaunchKernelGGL(stream_write_kernel, grid, dim3(kThreads), 0, st, (u4*)b);
  else
    hipLaunchKernelGGL(stream_copy_kernel, grid, dim3(kThreads), 0, st, (const u4*)a, (u4*)b);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// One wave that sleeps `sleeps` times (s_sleep 127: about 8k cycles each)
// and exits: a bounded wait that keeps the stream busy.
__global__ __launch_bounds__(64) void delay_kernel(int32_t sleeps) {
  for (int32_t i = 0; i < sleeps; ++i) __builtin_amdgcn_s_sleep(127);
}

extern "C" int32_t madd_probe_delay(int32_t sleeps, void* stream) {
  if (sleeps < 0 || sleeps > (1 << 20)) return -1;
  hipLaunchKernelGGL(delay_kernel, dim3(1), dim3(64), 0, (hipStream_t)stream, sleeps);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int32_t madd_probe_bf16_rounding(uint64_t* counters, void* stream) {
  if (!counters) return -1;
  hipLaunchKernelGGL(bf16_rounding_kernel, dim3(65536), dim3(256), 0, (hipStream_t)stream,
                     (unsigned long long*)counters);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

extern "C" int32_t madd_ceiling_stream(void* w, const float* g, void* m, void* v, void* ve,
                                       int32_t state_bytes, int64_t n, void* stream) {
  if (n < 0 || (state_bytes != 2 && state_bytes != 4)) return -1;
  if (n == 0) return 0;
  if (!w || !g || !m || !v || !ve) return -1;
  if (!(al16(w) && al16(g) && al16(m) && al16(v) && al16(ve))) return -2;
  const int64_t tiles = (n + kTile - 1) / kTile;
  if (tiles > 0x7FFFFFFFll) return -1;
  hipStream_t st = (hipStream_t)stream;
  if (state_bytes == 4)
    hipLaunchKernelGGL(ceiling_kernel<4>, dim3((unsigned)tiles), dim3(kThreads), 0, st, w, g, m,
                       v, ve, n, 0u);
  else
    hipLaunchKernelGGL(ceiling_kernel<2>, dim3((unsigned)tiles), dim3(kThreads), 0, st, w, g, m,
                       v, ve, n, 0u);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
