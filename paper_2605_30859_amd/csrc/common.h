// Shared device helpers for the gfx950 rollout kernels: bf16 conversion,
// Philox4x32-10, the float32 logarithm used for Gumbel noise, wavefront
// reductions.  Device code only; host launchers live in each kernel file.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace darts {

typedef uint16_t bf16_t;                       // raw bfloat16 bits
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kPage = 16;
constexpr uint32_t kTagWeight = 1, kTagSample = 2, kTagSweep = 3;

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}
// round to nearest even (finite inputs; NaN kept as a quiet NaN)
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t b = __float_as_uint(f);
  if ((b & 0x7fffffffu) > 0x7f800000u) return (bf16_t)0x7fc0;
  uint32_t lsb = (b >> 16) & 1u;
  return (bf16_t)((b + 0x7fffu + lsb) >> 16);
}

// Philox4x32-10 (Salmon et al., SC'11): 10 rounds of two 32x32->64 products
// with word permutation and key XOR; key bumped by the Weyl constants.
struct Philox4 { uint32_t x[4]; };
__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // 64-bit products: one v_mad_u64_u32 each instead of separate low and
    // high multiplies
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += 0x9E3779B9u; k1 += 0xBB67AE85u;
  }
  Philox4 r; r.x[0] = c0; r.x[1] = c1; r.x[2] = c2; r.x[3] = c3;
  return r;
}

// ((w >> 8) | 1) * 2^-23 - 1: exact float32 in (-1, 1)
__device__ __forceinline__ float signed_unit(uint32_t w) {
  return (float)((w >> 8) | 1u) * 1.1920928955078125e-07f - 1.0f;
}
// ((w >> 8) | 1) * 2^-24: exact float32 in (0, 1)
__device__ __forceinline__ float open_unit(uint32_t w) {
  return (float)((w >> 8) | 1u) * 5.9604644775390625e-08f;
}

// Natural log of a positive normal float32 as a fixed sequence of correctly
// rounded float32 operations (no contraction), atanh series on the reduced
// mantissa: x = 2^e m, m in (sqrt(1/2), sqrt(2)], t = (m-1)/(m+1),
// ln m = 2t(1 + t^2/3 + ... + t^10/11), ln x = e*ln2_hi + (e*ln2_lo + ln m),
// ln2_hi = 45426/65536 (exact products), ln2_lo its float32 tail.
__device__ __forceinline__ float own_ln(float x) {
#pragma clang fp contract(off)
  const uint32_t bits = __float_as_uint(x);
  int e = (int)((bits >> 23) & 0xffu) - 127;
  float m = __uint_as_float((bits & 0x007fffffu) | 0x3f800000u);
  if (m > __uint_as_float(0x3fb504f3u)) { m = m * 0.5f; e += 1; }   // fl32(sqrt 2)
  const float f = m - 1.0f;
  const float den = 2.0f + f;
  const float t = __fdiv_rn(f, den);
  const float t2 = t * t;
  float p = __uint_as_float(0x3dba2e8cu);                 // fl32(1/11)
  p = p * t2; p = p + __uint_as_float(0x3de38e39u);        // fl32(1/9)
  p = p * t2; p = p + __uint_as_float(0x3e124925u);        // fl32(1/7)
  p = p * t2; p = p + __uint_as_float(0x3e4ccccdu);        // fl32(1/5)
  p = p * t2; p = p + __uint_as_float(0x3eaaaaabu);        // fl32(1/3)
  p = p * t2; p = p + 1.0f;
  const float lnm = (t + t) * p;
  const float ef = (float)e;
  float lo = ef * __uint_as_float(0x35bfbe8eu);            // fl32(fl64(ln 2) - ln2_hi)
  lo = lo + lnm;
  const float hi = ef * 0.693145751953125f;                 // ln2_hi = 45426/65536
  return hi + lo;
}
__device__ __forceinline__ float gumbel_of(float u) {
  const float a = -own_ln(u);
  return -own_ln(a);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace darts

namespace darts {
// Paged KV pool layout (one pool per layer, page = 16 token slots, hd a
// multiple of 32):
//   K page of kv head h: [hd/32][slot][32]  (token-major within each 32-dim
//   block: the MFMA B operand of q.k^T for one 32-wide K step is 1 KB
//   contiguous, 16 B per lane)
//   V page of kv head h: [slot/8][hd][slot%8]  (8 consecutive tokens of one
//   dim contiguous; MFMA B operand of p.V with the contraction over tokens)
__host__ __device__ __forceinline__ int64_t k_off(int64_t page, int h, int slot, int d, int hkv,
                                                  int hd) {
  return (page * hkv + h) * (int64_t)kPage * hd + ((int64_t)(d >> 5) * kPage + slot) * 32 + (d & 31);
}
__host__ __device__ __forceinline__ int64_t v_off(int64_t page, int h, int slot, int d, int hkv,
                                                  int hd) {
  return (page * hkv + h) * (int64_t)kPage * hd + ((int64_t)(slot >> 3) * hd + d) * 8 + (slot & 7);
}
}  // namespace darts
