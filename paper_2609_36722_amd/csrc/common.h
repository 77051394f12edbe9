// Device-side helpers shared by the gfx950 kernels of libattuner.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attuner {

typedef uint16_t bf16_t;  // raw bfloat16 bits in memory

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---- bounds-checked build ----------------------------------------------------
// Compiled with -DATTUNER_CHECKED (libattuner_checked.so), the kernels test
// every block-table entry, page id and key range against the extents of their
// launch before they use it.  A failed test sets its bit (kViol*) in the
// violation word of the kernel's source file and the access is skipped (a
// workgroup whose whole range is wrong returns before its first barrier), so a
// bad table shows up as a flag instead of a memory fault.  In the ordinary
// build the tests compile away.
#ifdef ATTUNER_CHECKED
constexpr bool kChecked = true;
#else
constexpr bool kChecked = false;
#endif
constexpr unsigned kViolGatherPage = 1u << 0;  // gather: page id past its pool (or that pool absent)
constexpr unsigned kViolGatherRows = 1u << 1;  // gather: n_valid past a page, or rows past the cache plane
constexpr unsigned kViolStorePage = 1u << 2;   // store: page id past the pool
constexpr unsigned kViolAttnRange = 1u << 3;   // attention: q rows or key range past its buffers
constexpr unsigned kViolCopyEntry = 1u << 4;   // attention's page copy: entry out of its pool or cache plane
constexpr unsigned kViolDecodeRange = 1u << 5; // decode: key range past the cache plane

// One violation word per source file, and the host function that reads (and
// optionally clears) it on the current device; the ordinary build reads 0.
#ifdef ATTUNER_CHECKED
#define ATTUNER_VIOLATION_WORD(word, reader)                                           \
  __device__ unsigned int word = 0;                                                   \
  hipError_t reader(unsigned int* bits, bool reset) {                                 \
    unsigned int v = 0;                                                               \
    hipError_t e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(word), sizeof v, 0, hipMemcpyDeviceToHost); \
    if (e != hipSuccess) return e;                                                    \
    *bits |= v;                                                                       \
    if (reset && v != 0) {                                                            \
      const unsigned int zero = 0;                                                    \
      e = hipMemcpyToSymbol(HIP_SYMBOL(word), &zero, sizeof zero, 0, hipMemcpyHostToDevice); \
    }                                                                                 \
    return e;                                                                         \
  }
#define ATTUNER_VIOLATE(word, bit) atomicOr(&(word), (bit))
#else
#define ATTUNER_VIOLATION_WORD(word, reader) \
  hipError_t reader(unsigned int*, bool) { return hipSuccess; }
#define ATTUNER_VIOLATE(word, bit) ((void)0)
#endif

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even: one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f)); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v;
  v[0] = static_cast<__bf16>(lo);
  v[1] = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// 32x32x16 bf16 MFMA, fp32 accumulate.
// Lane l supplies A[l%32][8*(l/32) .. +8) and B[8*(l/32) .. +8)[l%32];
// the accumulator element v of lane l is C[8*(v/4) + 4*(l/32) + v%4][l%32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}

// ---- RMSNorm pieces shared by every kernel that normalises a row ------------
// Sum of squares of 8 bf16 values added to ss in order, and the scaled
// bf16 values of a row chunk.

__device__ __forceinline__ float accum_squares(float ss, u32x4 v) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float lo = __uint_as_float(v[e] << 16), hi = __uint_as_float(v[e] & 0xFFFF0000u);
    ss += lo * lo + hi * hi;
  }
  return ss;
}

// bf16(x * inv * gamma) for 8 values
__device__ __forceinline__ u32x4 norm_chunk(u32x4 v, u32x4 g, float inv) {
  u32x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float lo = __uint_as_float(v[e] << 16) * inv * __uint_as_float(g[e] << 16);
    const float hi = __uint_as_float(v[e] & 0xFFFF0000u) * inv * __uint_as_float(g[e] & 0xFFFF0000u);
    o[e] = pack_bf16x2(lo, hi);
  }
  return o;
}

// Per-head RMSNorm over 128 dims + RoPE (rotate-half: dim i pairs with
// 64 + i) held by an 8-lane group: lane j has dims 8j .. 8j + 7 in xa and
// 64 + 8j .. 64 + 8j + 7 in xb, gamma likewise in ga / gb, and cs[e] =
// (cos, sin) of pairs 8j + 2e and 8j + 2e + 1 at the token's position.  The
// head's sum of squares is the lane's plus three exchanges in the group.
__device__ __forceinline__ void head_norm_rope(u32x4 xa, u32x4 xb, u32x4 ga, u32x4 gb, const f32x4 cs[4], float eps,
                                               u32x4& oa, u32x4& ob) {
  float x0[8], x1[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x0[2 * e] = __uint_as_float(xa[e] << 16);
    x0[2 * e + 1] = __uint_as_float(xa[e] & 0xFFFF0000u);
    x1[2 * e] = __uint_as_float(xb[e] << 16);
    x1[2 * e + 1] = __uint_as_float(xb[e] & 0xFFFF0000u);
  }
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) ss += x0[e] * x0[e] + x1[e] * x1[e];
  ss += __shfl_xor(ss, 1, 8);
  ss += __shfl_xor(ss, 2, 8);
  ss += __shfl_xor(ss, 4, 8);
  const float inv = 1.0f / sqrtf(ss * (1.0f / 128) + eps);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float o0[2], o1[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = 2 * e + u;
      const float g0 = __uint_as_float(u ? (ga[e] & 0xFFFF0000u) : (ga[e] << 16));
      const float g1 = __uint_as_float(u ? (gb[e] & 0xFFFF0000u) : (gb[e] << 16));
      const float y0 = x0[k] * inv * g0;
      const float y1 = x1[k] * inv * g1;
      const float c = cs[e][2 * u], sn = cs[e][2 * u + 1];
      o0[u] = y0 * c - y1 * sn;
      o1[u] = y1 * c + y0 * sn;
    }
    oa[e] = pack_bf16x2(o0[0], o0[1]);
    ob[e] = pack_bf16x2(o1[0], o1[1]);
  }
}

// ---- direct global -> LDS copies ------------------------------------------

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding and leaves the other counters alone (gfx9 layout:
// vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14, expcnt 6:4, lgkmcnt 11:8).
__host__ __device__ constexpr int vmcnt_wait(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// One 16-byte-per-lane global -> LDS copy (global_load_lds_dwordx4): lane i's
// 16 bytes land at LDS byte lds_base + 16 i (lds_base wave-uniform, in M0).
// Issued as inline assembly so the compiler does not track these LDS writes
// (its tracking would add a full vmcnt(0) wait before every LDS read); the
// caller orders them with an explicit vmcnt wait and a barrier.  The LDS
// base is an input operand bound to M0 ("{m0}"), so the compiler writes M0
// itself and knows the register is live there; the asm only adds one wait
// state between that write and the load.
__device__ __forceinline__ void lds_dma16(const void* gaddr, uint32_t lds_base) {
  asm volatile(
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(gaddr), "{m0}"(__builtin_amdgcn_readfirstlane(lds_base))
      : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

// Workgroup barrier without a memory fence: LDS DMA completion is covered by
// the explicit vmcnt wait before it; the empty asm statements keep the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void barrier_no_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace attuner
