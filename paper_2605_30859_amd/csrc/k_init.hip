// Initialisation kernels: Philox random-init weights, RoPE cos/sin table,
// sweep fills, free-list initialisation.
#include "common.h"
#include "kernels.h"

namespace darts {

RowMap rowmap_plain(int64_t n_out, int64_t row_off) {
  RowMap m;
  m.grp_outer = n_out > 0 ? n_out : 1;
  m.stride_outer = 0;
  m.grp_inner = m.grp_outer;
  m.stride_inner = 0;
  m.row_off = row_off;
  return m;
}

__device__ __forceinline__ int64_t map_row(const RowMap& m, int64_t r) {
  const int64_t o = r / m.grp_outer, w = r % m.grp_outer;
  return o * m.stride_outer + (w / m.grp_inner) * m.stride_inner + (w % m.grp_inner) + m.row_off;
}

// Element idx of the logical [n_out][n_in] tensor takes word idx&3 of
// Philox(counter=(idx>>2, tensor, layer, TAG_WEIGHT), key=seed); the value is
// fl32(((w>>8)|1)*2^-23 - 1) * a) with a = fl32(sqrt(3/fan_in)), then bf16.
template <bool BF16>
__global__ void init_weights_kernel(void* dst, int64_t n_out, int64_t n_in, float a,
                                    uint32_t tensor, uint32_t layer, uint32_t k0, uint32_t k1,
                                    RowMap map) {
  const int64_t total4 = (n_out * n_in + 3) >> 2;
  for (int64_t blk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; blk < total4;
       blk += (int64_t)gridDim.x * blockDim.x) {
    const Philox4 p = philox4x32_10((uint32_t)blk, tensor, layer, kTagWeight, k0, k1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t idx = blk * 4 + j;
      if (idx >= n_out * n_in) break;
      const float v = signed_unit(p.x[j]) * a;
      const int64_t r = idx / n_in, c = idx % n_in;
      const int64_t off = map_row(map, r) * n_in + c;
      if (BF16) ((bf16_t*)dst)[off] = f32_to_bf16(v);
      else ((float*)dst)[off] = v;
    }
  }
}

hipError_t launch_init_weights(void* dst, bool bf16, int64_t n_out, int64_t n_in, int64_t fan_in,
                               uint32_t tensor_id, uint32_t layer, uint64_t seed, RowMap map,
                               hipStream_t st) {
  const float a = (float)sqrt(3.0 / (double)fan_in);
  const int64_t total4 = (n_out * n_in + 3) >> 2;
  int64_t blocks = (total4 + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  if (bf16)
    hipLaunchKernelGGL(init_weights_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, dst,
                       n_out, n_in, a, tensor_id, layer, k0, k1, map);
  else
    hipLaunchKernelGGL(init_weights_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, dst,
                       n_out, n_in, a, tensor_id, layer, k0, k1, map);
  return hipGetLastError();
}

// One thread per element of the logical [n_out][n_in] tensor (grid stride);
// the copy is made once, when a context takes the caller's weights.
template <typename T>
__global__ void copy_rows_kernel(T* __restrict__ dst, const T* __restrict__ src, int64_t n_out,
                                 int64_t n_in, RowMap map) {
  const int64_t total = n_out * n_in;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = idx / n_in, c = idx % n_in;
    dst[map_row(map, r) * n_in + c] = src[idx];
  }
}

hipError_t launch_copy_rows(void* dst, const void* src, bool bf16, int64_t n_out, int64_t n_in, RowMap map,
                            hipStream_t st) {
  const int64_t total = n_out * n_in;
  if (total <= 0) return hipSuccess;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    hipLaunchKernelGGL(copy_rows_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, st, (bf16_t*)dst,
                       (const bf16_t*)src, n_out, n_in, map);
  else
    hipLaunchKernelGGL(copy_rows_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st, (float*)dst,
                       (const float*)src, n_out, n_in, map);
  return hipGetLastError();
}

// table[p][i] = (cos(p * theta^(-2i/hd)), sin(...)) evaluated in float64.
__global__ void rope_table_kernel(float2* table, int max_pos, int half, int hd, double theta) {
  const int64_t n = (int64_t)max_pos * half;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int p = (int)(t / half), i = (int)(t % half);
    const double inv = pow(theta, -2.0 * (double)i / (double)hd);
    const double ang = (double)p * inv;
    table[t] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

hipError_t launch_rope_table(float2* table, int max_pos, int hd, double theta, hipStream_t st) {
  const int half = hd / 2;
  int64_t blocks = ((int64_t)max_pos * half + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)blocks), dim3(256), 0, st, table, max_pos,
                     half, hd, theta);
  return hipGetLastError();
}

template <bool BF16>
__global__ void fill_uniform_kernel(void* dst, uint64_t n, uint32_t tensor, uint32_t k0,
                                    uint32_t k1) {
  const uint64_t n4 = (n + 3) >> 2;
  for (uint64_t blk = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; blk < n4;
       blk += (uint64_t)gridDim.x * blockDim.x) {
    const Philox4 p = philox4x32_10((uint32_t)blk, tensor, 0, kTagSweep, k0, k1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint64_t idx = blk * 4 + j;
      if (idx >= n) break;
      const bf16_t h = f32_to_bf16(signed_unit(p.x[j]));
      if (BF16) ((bf16_t*)dst)[idx] = h;
      else ((float*)dst)[idx] = bf16_to_f32(h);
    }
  }
}

hipError_t launch_fill_uniform(void* dst, uint64_t n, uint32_t tensor, uint64_t seed, bool bf16,
                               hipStream_t st) {
  uint64_t blocks = ((n + 3) / 4 + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (bf16)
    hipLaunchKernelGGL(fill_uniform_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, dst, n,
                       tensor, (uint32_t)seed, (uint32_t)(seed >> 32));
  else
    hipLaunchKernelGGL(fill_uniform_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, dst, n,
                       tensor, (uint32_t)seed, (uint32_t)(seed >> 32));
  return hipGetLastError();
}

// Streaming read of n16 16-byte words (the HBM read rate that the attention
// kernel's roofline is compared with): grid-stride float4 loads, one sum per
// wavefront written to sink so the loads are not dead.
__global__ void __launch_bounds__(256) stream_read_kernel(const float4* __restrict__ src, int64_t n16,
                                                          float* __restrict__ sink) {
  float s = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (int64_t)gridDim.x * 256) {
    // non-temporal: 7.0 TB/s over 8 GiB against 6.3 TB/s with plain loads
    const f32x4_t v = __builtin_nontemporal_load((const f32x4_t*)src + i);
    s += (v[0] + v[1]) + (v[2] + v[3]);
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

hipError_t launch_stream_read(const void* src, int64_t n16, float* sink, hipStream_t st) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(kStreamReadBlocks), dim3(256), 0, st,
                     (const float4*)src, n16, sink);
  return hipGetLastError();
}

// Logical index ((page*Hkv + h)*16 + slot)*hd + d  ->  physical pool layouts.
template <bool BF16>
__global__ void fill_kv_kernel(void* k, void* v, int64_t n_pages, int hkv, int hd, uint32_t k0,
                               uint32_t k1) {
  const int64_t n = n_pages * hkv * kPage * hd;
  const int64_t n4 = n >> 2;   // hd is a multiple of 4
  for (int64_t blk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; blk < n4;
       blk += (int64_t)gridDim.x * blockDim.x) {
    const Philox4 pk = philox4x32_10((uint32_t)blk, 1u, 0u, kTagSweep, k0, k1);
    const Philox4 pv = philox4x32_10((uint32_t)blk, 2u, 0u, kTagSweep, k0, k1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t idx = blk * 4 + j;
      const int d = (int)(idx % hd);
      const int64_t t = idx / hd;
      const int slot = (int)(t % kPage);
      const int64_t ph = t / kPage;
      const int h = (int)(ph % hkv);
      const int64_t page = ph / hkv;
      const bf16_t hk = f32_to_bf16(signed_unit(pk.x[j])), hv = f32_to_bf16(signed_unit(pv.x[j]));
      const int64_t ok = k_off(page, h, slot, d, hkv, hd), ov = v_off(page, h, slot, d, hkv, hd);
      if (BF16) { ((bf16_t*)k)[ok] = hk; ((bf16_t*)v)[ov] = hv; }
      else { ((float*)k)[ok] = bf16_to_f32(hk); ((float*)v)[ov] = bf16_to_f32(hv); }
    }
  }
}

hipError_t launch_fill_kv_pool(void* k, void* v, int64_t n_pages, int hkv, int hd, uint64_t seed,
                               bool bf16, hipStream_t st) {
  const int64_t n4 = n_pages * hkv * kPage * hd / 4;
  int64_t blocks = (n4 + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (bf16)
    hipLaunchKernelGGL(fill_kv_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, k, v,
                       n_pages, hkv, hd, (uint32_t)seed, (uint32_t)(seed >> 32));
  else
    hipLaunchKernelGGL(fill_kv_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, k, v,
                       n_pages, hkv, hd, (uint32_t)seed, (uint32_t)(seed >> 32));
  return hipGetLastError();
}

// Free-list stack: stack[t] = t, or a seeded permutation (Feistel-free
// approach: sort-free "random key" permutation would need a sort, so the
// permutation is an affine map t -> (a*t + b) mod n with gcd(a, n) = 1).
__global__ void iota_perm_kernel(int32_t* stack, int64_t n, uint64_t a, uint64_t b) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
       t += (int64_t)gridDim.x * blockDim.x)
    stack[t] = (int32_t)((a * (uint64_t)t + b) % (uint64_t)n);
}

static uint64_t gcd_u64(uint64_t x, uint64_t y) {
  while (y) { uint64_t t = x % y; x = y; y = t; }
  return x;
}

hipError_t launch_iota_perm(int32_t* stack, int64_t n, uint64_t perm_seed, bool permute,
                            hipStream_t st) {
  uint64_t a = 1, b = 0;
  if (permute && n > 1) {
    uint64_t s = perm_seed * 0x9E3779B97F4A7C15ull + 0x632BE59BD9B4E019ull;
    a = (s >> 11) % (uint64_t)n;
    if (a < 2) a = 2;
    while (gcd_u64(a, (uint64_t)n) != 1) ++a;
    b = (s >> 3) % (uint64_t)n;
  }
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(iota_perm_kernel, dim3((unsigned)blocks), dim3(256), 0, st, stack, n, a % n,
                     b);
  return hipGetLastError();
}

}  // namespace darts
