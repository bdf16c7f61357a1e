// Elementwise kernels of the decoder step: embedding gather, RMSNorm,
// RoPE + paged KV append, row gather.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace darts {

// x[r][:] = E[tokens[rows_traj ? rows_traj[r] : r]][:]   (fp32 residual stream)
template <bool BF16>
__global__ void embed_kernel(const void* __restrict__ table, const int32_t* __restrict__ tokens,
                             const int32_t* __restrict__ rows_traj, int d, int vocab,
                             float* __restrict__ x) {
  const int r = blockIdx.x;
  const int src = rows_traj ? rows_traj[r] : r;
  int tok = tokens[src];
  tok = tok < 0 ? 0 : (tok >= vocab ? vocab - 1 : tok);
  float* xr = x + (int64_t)r * d;
  if (BF16 && (d & 7) == 0) {
    // 8 bf16 (16 bytes) per thread and step
    const uint4* er = (const uint4*)((const bf16_t*)table + (int64_t)tok * d);
    for (int c = threadIdx.x; c < d / 8; c += blockDim.x) {
      const uint4 w = er[c];
      const uint32_t q[4] = {w.x, w.y, w.z, w.w};
      float4 lo, hi;
      lo.x = __uint_as_float(q[0] << 16); lo.y = __uint_as_float(q[0] & 0xffff0000u);
      lo.z = __uint_as_float(q[1] << 16); lo.w = __uint_as_float(q[1] & 0xffff0000u);
      hi.x = __uint_as_float(q[2] << 16); hi.y = __uint_as_float(q[2] & 0xffff0000u);
      hi.z = __uint_as_float(q[3] << 16); hi.w = __uint_as_float(q[3] & 0xffff0000u);
      *(float4*)(xr + 8 * c) = lo;
      *(float4*)(xr + 8 * c + 4) = hi;
    }
    return;
  }
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float v;
    if (BF16) v = bf16_to_f32(((const bf16_t*)table)[(int64_t)tok * d + c]);
    else v = ((const float*)table)[(int64_t)tok * d + c];
    xr[c] = v;
  }
}

hipError_t launch_embed_v(const void* table, bool bf16, const int32_t* tokens,
                          const int32_t* rows_traj, int n_rows, int d, int vocab, float* x,
                          hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(embed_kernel<true>, dim3(n_rows), dim3(256), 0, st, table, tokens,
                       rows_traj, d, vocab, x);
  else
    hipLaunchKernelGGL(embed_kernel<false>, dim3(n_rows), dim3(256), 0, st, table, tokens,
                       rows_traj, d, vocab, x);
  return hipGetLastError();
}

// Embedding gather fused with the first RMSNorm (bf16 tables, d % 8 == 0,
// d <= 4096): x[r] = E[tok] (fp32), xn[r] = bf16(x[r] / sqrt(mean(x^2) + eps)).
constexpr int kEmbVec = 2;                      // 8 bf16 per step, d <= 256 * 8 * 2
__global__ void __launch_bounds__(256) embed_norm_kernel(const bf16_t* __restrict__ table,
                                                         const int32_t* __restrict__ tokens,
                                                         const int32_t* __restrict__ rows_traj,
                                                         int d, int vocab, float eps,
                                                         float* __restrict__ x,
                                                         bf16_t* __restrict__ xn) {
  __shared__ float red[4];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int src = rows_traj ? rows_traj[r] : r;
  int tok = tokens[src];
  tok = tok < 0 ? 0 : (tok >= vocab ? vocab - 1 : tok);
  const uint4* er = (const uint4*)(table + (int64_t)tok * d);
  float* xr = x + (int64_t)r * d;
  float v[kEmbVec][8];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kEmbVec; ++j) {
    const int c = tid + 256 * j;
    uint4 w = c < d / 8 ? er[c] : make_uint4(0u, 0u, 0u, 0u);
    const uint32_t q[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[j][2 * e] = __uint_as_float(q[e] << 16);
      v[j][2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(v[j][e], v[j][e], ss);
    if (c < d / 8) {
      *(float4*)(xr + 8 * c) = make_float4(v[j][0], v[j][1], v[j][2], v[j][3]);
      *(float4*)(xr + 8 * c + 4) = make_float4(v[j][4], v[j][5], v[j][6], v[j][7]);
    }
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
#pragma unroll
  for (int j = 0; j < kEmbVec; ++j) {
    const int c = tid + 256 * j;
    if (c >= d / 8) break;
    uint4 p;
    p.x = (uint32_t)f32_to_bf16(v[j][0] * inv) | ((uint32_t)f32_to_bf16(v[j][1] * inv) << 16);
    p.y = (uint32_t)f32_to_bf16(v[j][2] * inv) | ((uint32_t)f32_to_bf16(v[j][3] * inv) << 16);
    p.z = (uint32_t)f32_to_bf16(v[j][4] * inv) | ((uint32_t)f32_to_bf16(v[j][5] * inv) << 16);
    p.w = (uint32_t)f32_to_bf16(v[j][6] * inv) | ((uint32_t)f32_to_bf16(v[j][7] * inv) << 16);
    *(uint4*)(xn + (int64_t)r * d + 8 * c) = p;
  }
}

// out[r] = x[r] / sqrt(mean(x[r]^2) + eps), one block of 256 per row.  Rows
// with d % 4 == 0 and d <= 4096 are read once as float4 and kept in registers
// between the sum of squares and the scaled store.
constexpr int kRmsVec = 4;                      // float4 per thread: d <= 256 * 4 * 4
template <bool BF16>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x, int d, float eps,
                                                      void* __restrict__ out) {
  __shared__ float red[4];
  const int r = blockIdx.x, tid = threadIdx.x;
  const float* xr = x + (int64_t)r * d;
  const bool vec = (d & 3) == 0 && d <= 256 * 4 * kRmsVec;
  float4 v[kRmsVec];
  float ss = 0.f;
  if (vec) {
#pragma unroll
    for (int j = 0; j < kRmsVec; ++j) {
      const int c = (tid + 256 * j) * 4;
      v[j] = c < d ? *(const float4*)(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      ss = fmaf(v[j].x, v[j].x, ss);
      ss = fmaf(v[j].y, v[j].y, ss);
      ss = fmaf(v[j].z, v[j].z, ss);
      ss = fmaf(v[j].w, v[j].w, ss);
    }
  } else {
    for (int c = tid; c < d; c += 256) ss = fmaf(xr[c], xr[c], ss);
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  if (vec) {
#pragma unroll
    for (int j = 0; j < kRmsVec; ++j) {
      const int c = (tid + 256 * j) * 4;
      if (c >= d) break;
      const float4 o = make_float4(v[j].x * inv, v[j].y * inv, v[j].z * inv, v[j].w * inv);
      if (BF16) {
        uint2 p;
        p.x = (uint32_t)f32_to_bf16(o.x) | ((uint32_t)f32_to_bf16(o.y) << 16);
        p.y = (uint32_t)f32_to_bf16(o.z) | ((uint32_t)f32_to_bf16(o.w) << 16);
        *(uint2*)((bf16_t*)out + (int64_t)r * d + c) = p;
      } else {
        *(float4*)((float*)out + (int64_t)r * d + c) = o;
      }
    }
  } else {
    for (int c = tid; c < d; c += 256) {
      const float o = xr[c] * inv;
      if (BF16) ((bf16_t*)out)[(int64_t)r * d + c] = f32_to_bf16(o);
      else ((float*)out)[(int64_t)r * d + c] = o;
    }
  }
}

hipError_t launch_embed_norm(const void* table, const int32_t* tokens, const int32_t* rows_traj,
                             int n_rows, int d, int vocab, float eps, float* x, void* xn,
                             hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (d % 8 != 0 || d > 256 * 8 * kEmbVec) {
    hipError_t e = launch_embed_v(table, true, tokens, rows_traj, n_rows, d, vocab, x, st);
    return e != hipSuccess ? e : launch_rmsnorm(x, n_rows, d, eps, xn, true, st);
  }
  hipLaunchKernelGGL(embed_norm_kernel, dim3(n_rows), dim3(256), 0, st, (const bf16_t*)table, tokens,
                     rows_traj, d, vocab, eps, x, (bf16_t*)xn);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* x, int n_rows, int d, float eps, void* out, bool bf16,
                          hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(rmsnorm_kernel<true>, dim3(n_rows), dim3(256), 0, st, x, d, eps, out);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<false>, dim3(n_rows), dim3(256), 0, st, x, d, eps, out);
  return hipGetLastError();
}

// qkv[r] = [q (hq*hd) | k (hkv*hd) | v (hkv*hd)] fp32, the sum of n_split
// planes split_stride floats apart (split-K partials of the QKV projection,
// summed here in plane order; n_split = 1 for a plain result).  Rotate-half RoPE on q
// and k with the cos/sin table, write q (activation dtype) and append k, v
// at position pos(r) into the pages of page-table row pt(r).
//   pos(r) = pos_mod ? r % pos_mod + pos_base : pos_base
template <bool BF16>
__global__ void rope_append_kernel(const float* __restrict__ qkv, int n_split, int64_t split_stride,
                                   int hq, int hkv, int hd,
                                   const int32_t* __restrict__ row_pt, int pos_mod, int pos_base,
                                   const int32_t* __restrict__ page_table, int pt_stride,
                                   int64_t n_pages, const float2* __restrict__ rope,
                                   void* __restrict__ q_out, void* __restrict__ k_pool,
                                   void* __restrict__ v_pool) {
  const int r = blockIdx.x;
  const int half = hd / 2;
  const int pos = (pos_mod ? r % pos_mod : 0) + pos_base;
  const int ptr = row_pt ? row_pt[r] : r;
  int page = page_table[(int64_t)ptr * pt_stride + pos / kPage];
  page = page < 0 ? 0 : (page >= n_pages ? (int)(n_pages - 1) : page);
  const int slot = pos % kPage;
  const int width = (hq + 2 * hkv) * hd;
  const float* src = qkv + (int64_t)r * width;
  const float2* cs = rope + (int64_t)pos * half;
  // rotated heads: hq query heads then hkv key heads; four consecutive
  // rotation pairs (i .. i+3 with partners i+half ..) per thread
  const int q4 = half / 4;
  // blockIdx.y splits a row's work over several blocks (small batches)
  const int t0 = blockIdx.y * blockDim.x + threadIdx.x, tstep = gridDim.y * blockDim.x;
  for (int t = t0; t < (hq + hkv) * q4; t += tstep) {
    const int h = t / q4, i = (t % q4) * 4;
    const float* v = src + h * hd;
    float4 a = *(const float4*)(v + i), b = *(const float4*)(v + i + half);
    for (int z = 1; z < n_split; ++z) {
      const float4 a2 = *(const float4*)(v + z * split_stride + i);
      const float4 b2 = *(const float4*)(v + z * split_stride + i + half);
      a.x += a2.x; a.y += a2.y; a.z += a2.z; a.w += a2.w;
      b.x += b2.x; b.y += b2.y; b.z += b2.z; b.w += b2.w;
    }
    const float4 c01 = *(const float4*)(cs + i), c23 = *(const float4*)(cs + i + 2);
    const float ca[4] = {c01.x, c01.z, c23.x, c23.z}, sa[4] = {c01.y, c01.w, c23.y, c23.w};
    const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
    float o1[4], o2[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o1[e] = av[e] * ca[e] - bv[e] * sa[e];
      o2[e] = bv[e] * ca[e] + av[e] * sa[e];
    }
    int64_t oa, ob;
    void* dst;
    if (h < hq) {
      oa = ((int64_t)r * hq + h) * hd + i;
      ob = oa + half;
      dst = q_out;
    } else {
      const int kh = h - hq;
      oa = k_off(page, kh, slot, i, hkv, hd);
      ob = k_off(page, kh, slot, i + half, hkv, hd);
      dst = k_pool;
    }
    if (BF16) {
      uint2 p1, p2;
      p1.x = (uint32_t)f32_to_bf16(o1[0]) | ((uint32_t)f32_to_bf16(o1[1]) << 16);
      p1.y = (uint32_t)f32_to_bf16(o1[2]) | ((uint32_t)f32_to_bf16(o1[3]) << 16);
      p2.x = (uint32_t)f32_to_bf16(o2[0]) | ((uint32_t)f32_to_bf16(o2[1]) << 16);
      p2.y = (uint32_t)f32_to_bf16(o2[2]) | ((uint32_t)f32_to_bf16(o2[3]) << 16);
      *(uint2*)((bf16_t*)dst + oa) = p1;
      *(uint2*)((bf16_t*)dst + ob) = p2;
    } else {
      *(float4*)((float*)dst + oa) = make_float4(o1[0], o1[1], o1[2], o1[3]);
      *(float4*)((float*)dst + ob) = make_float4(o2[0], o2[1], o2[2], o2[3]);
    }
  }
  for (int t = t0; t < hkv * hd; t += tstep) {
    const int h = t / hd, dd = t % hd;
    float v = src[(hq + hkv) * hd + t];
    for (int z = 1; z < n_split; ++z) v += src[z * split_stride + (hq + hkv) * hd + t];
    const int64_t o = v_off(page, h, slot, dd, hkv, hd);
    if (pos_mod == 0 && slot == 0) {
      // A decode append that opens a page (slot 0; the row owns the page) also
      // clears the page's later value slots.  Attention weighs keys at or past
      // the row's context by 0 but still multiplies their values in the P.V
      // product, so those slots must hold finite values, whatever the memory
      // held before (0 x NaN is NaN).  Key slots need nothing: their scores
      // are replaced, not multiplied.  A prefill writes whole pages itself.
      // Slots 0-7 and 8-15 of one dim are 8 consecutive elements each: two
      // aligned vector stores write this slot's value and the zeros.
      static_assert(kPage == 16, "two groups of 8 value slots per page");
      const int64_t o8 = v_off(page, h, 8, dd, hkv, hd);
      if (BF16) {
        *(uint4*)((bf16_t*)v_pool + o) = make_uint4((uint32_t)f32_to_bf16(v), 0u, 0u, 0u);
        *(uint4*)((bf16_t*)v_pool + o8) = make_uint4(0u, 0u, 0u, 0u);
      } else {
        float4* p0 = (float4*)((float*)v_pool + o);
        float4* p8 = (float4*)((float*)v_pool + o8);
        p0[0] = make_float4(v, 0.f, 0.f, 0.f);
        p0[1] = make_float4(0.f, 0.f, 0.f, 0.f);
        p8[0] = make_float4(0.f, 0.f, 0.f, 0.f);
        p8[1] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    } else if (BF16) {
      ((bf16_t*)v_pool)[o] = f32_to_bf16(v);
    } else {
      ((float*)v_pool)[o] = v;
    }
  }
}

hipError_t launch_rope_append2(const float* qkv, int n_split, int64_t split_stride, int n_rows,
                               int hq, int hkv, int hd, const int32_t* row_pt, int pos_mod,
                               int pos_base, const int32_t* page_table, int pt_stride,
                               int64_t n_pages, const float2* rope, void* q_out, void* k_pool,
                               void* v_pool, bool bf16, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (n_split < 1) return hipErrorInvalidValue;
  // at least ~512 blocks when rows are few, at most one block per 256 items
  const int items = std::max((hq + hkv) * (hd / 8), hkv * hd);
  const int ymax = std::max(1, (items + 255) / 256);
  const int y = std::min(ymax, std::max(1, (512 + n_rows - 1) / n_rows));
  const dim3 grid(n_rows, y);
  if (bf16)
    hipLaunchKernelGGL(rope_append_kernel<true>, grid, dim3(256), 0, st, qkv, n_split,
                       split_stride, hq, hkv, hd, row_pt, pos_mod, pos_base, page_table, pt_stride,
                       n_pages, rope, q_out, k_pool, v_pool);
  else
    hipLaunchKernelGGL(rope_append_kernel<false>, grid, dim3(256), 0, st, qkv, n_split,
                       split_stride, hq, hkv, hd, row_pt, pos_mod, pos_base, page_table, pt_stride,
                       n_pages, rope, q_out, k_pool, v_pool);
  return hipGetLastError();
}

// dst[i] = src[rows[i]]  (fp32 rows of width d)
__global__ void gather_rows_kernel(const float* __restrict__ src, const int32_t* __restrict__ rows,
                                   int d, float* __restrict__ dst) {
  const int i = blockIdx.x;
  const int r = rows[i];
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[(int64_t)i * d + c] = src[(int64_t)r * d + c];
}

hipError_t launch_gather_rows(const float* src, const int32_t* rows, int n, int d, float* dst,
                              hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(n), dim3(256), 0, st, src, rows, d, dst);
  return hipGetLastError();
}

}  // namespace darts
