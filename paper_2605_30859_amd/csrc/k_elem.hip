// Elementwise kernels of the decoder step: embedding gather, RMSNorm,
// RoPE + paged KV append, row gather.
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
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float v;
    if (BF16) v = bf16_to_f32(((const bf16_t*)table)[(int64_t)tok * d + c]);
    else v = ((const float*)table)[(int64_t)tok * d + c];
    x[(int64_t)r * d + c] = v;
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

// out[r] = x[r] / sqrt(mean(x[r]^2) + eps), one block of 256 per row
template <bool BF16>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x, int d, float eps,
                                                      void* __restrict__ out) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const float* xr = x + (int64_t)r * d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += 256) ss = fmaf(xr[c], xr[c], ss);
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += 256) {
    const float v = xr[c] * inv;
    if (BF16) ((bf16_t*)out)[(int64_t)r * d + c] = f32_to_bf16(v);
    else ((float*)out)[(int64_t)r * d + c] = v;
  }
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

// qkv[r] = [q (hq*hd) | k (hkv*hd) | v (hkv*hd)] fp32.  Rotate-half RoPE on q
// and k with the cos/sin table, write q (activation dtype) and append k, v
// at position pos(r) into the pages of page-table row pt(r).
//   pos(r) = pos_mod ? r % pos_mod + pos_base : pos_base
template <bool BF16>
__global__ void rope_append_kernel(const float* __restrict__ qkv, int hq, int hkv, int hd,
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
  // rotated heads: hq query heads then hkv key heads
  for (int t = threadIdx.x; t < (hq + hkv) * half; t += blockDim.x) {
    const int h = t / half, i = t % half;
    const float* v = src + h * hd;
    const float a = v[i], b = v[i + half];
    const float2 c = cs[i];
    const float o1 = a * c.x - b * c.y;
    const float o2 = b * c.x + a * c.y;
    if (h < hq) {
      const int64_t base = ((int64_t)r * hq + h) * hd;
      if (BF16) {
        ((bf16_t*)q_out)[base + i] = f32_to_bf16(o1);
        ((bf16_t*)q_out)[base + i + half] = f32_to_bf16(o2);
      } else {
        ((float*)q_out)[base + i] = o1;
        ((float*)q_out)[base + i + half] = o2;
      }
    } else {
      const int kh = h - hq;
      const int64_t o_a = k_off(page, kh, slot, i, hkv, hd), o_b = k_off(page, kh, slot, i + half, hkv, hd);
      if (BF16) {
        ((bf16_t*)k_pool)[o_a] = f32_to_bf16(o1);
        ((bf16_t*)k_pool)[o_b] = f32_to_bf16(o2);
      } else {
        ((float*)k_pool)[o_a] = o1;
        ((float*)k_pool)[o_b] = o2;
      }
    }
  }
  for (int t = threadIdx.x; t < hkv * hd; t += blockDim.x) {
    const int h = t / hd, dd = t % hd;
    const float v = src[(hq + hkv) * hd + t];
    const int64_t o = v_off(page, h, slot, dd, hkv, hd);
    if (BF16) ((bf16_t*)v_pool)[o] = f32_to_bf16(v);
    else ((float*)v_pool)[o] = v;
  }
}

hipError_t launch_rope_append2(const float* qkv, int n_rows, int hq, int hkv, int hd,
                               const int32_t* row_pt, int pos_mod, int pos_base,
                               const int32_t* page_table, int pt_stride, int64_t n_pages,
                               const float2* rope, void* q_out, void* k_pool, void* v_pool,
                               bool bf16, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(rope_append_kernel<true>, dim3(n_rows), dim3(256), 0, st, qkv, hq, hkv, hd,
                       row_pt, pos_mod, pos_base, page_table, pt_stride, n_pages, rope, q_out,
                       k_pool, v_pool);
  else
    hipLaunchKernelGGL(rope_append_kernel<false>, dim3(n_rows), dim3(256), 0, st, qkv, hq, hkv, hd,
                       row_pt, pos_mod, pos_base, page_table, pt_stride, n_pages, rope, q_out,
                       k_pool, v_pool);
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
