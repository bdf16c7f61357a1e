// Mixture-of-experts FFN of the decoder (top-k of E experts, renormalised).
//
//   route:    r = softmax(W_router h); the k largest (ties to the lower
//             expert id); weights renormalised over the k; per-expert counts
//   offsets:  exclusive scan of the counts
//   scatter:  every (row, slot) pair gets a position in its expert's segment
//             and its normalised input row is copied there
//   experts:  grouped GEMMs per expert segment: gate/up (+ SwiGLU), down
//   combine:  x[row] += sum_j w[row][j] * y[pos(row, j)]   (slot order)
// Positions inside a segment come from atomics, so their order varies from
// run to run, but no value depends on it: every output row of an expert GEMM
// depends only on its own input row, and the combine sums in slot order.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace darts {

// One block (256 threads) per row: router logits (E dot products over d),
// fp32 softmax, top-k selection by repeated argmax, renormalisation.
__global__ void __launch_bounds__(256) moe_route_kernel(const bf16_t* __restrict__ xn, int d,
                                                        const bf16_t* __restrict__ wr, int E, int k,
                                                        int32_t* __restrict__ topk_id,
                                                        float* __restrict__ topk_w,
                                                        int32_t* __restrict__ counts) {
  extern __shared__ float sm[];          // [d] input row, then [E] probabilities
  float* xs = sm;
  float* pr = sm + d;
  __shared__ float red_v[4];
  __shared__ int red_i[4];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int c = tid; c < d; c += 256) xs[c] = bf16_to_f32(xn[(int64_t)r * d + c]);
  __syncthreads();
  // each wavefront computes experts w, w+4, ...: lanes split d, shuffle-reduce
  for (int e = w; e < E; e += 4) {
    const bf16_t* we = wr + (int64_t)e * d;
    float s = 0.f;
    for (int c = lane; c < d; c += 64) s = fmaf(xs[c], bf16_to_f32(we[c]), s);
    s = wave_sum(s);
    if (lane == 0) pr[e] = s;
  }
  __syncthreads();
  // softmax over E (max, sum of exp) in one wavefront
  if (w == 0) {
    float mx = -INFINITY;
    for (int e = lane; e < E; e += 64) mx = fmaxf(mx, pr[e]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int e = lane; e < E; e += 64) {
      const float v = __expf(pr[e] - mx);
      pr[e] = v;
      sum += v;
    }
    sum = wave_sum(sum);
    const float inv = 1.0f / sum;
    for (int e = lane; e < E; e += 64) pr[e] *= inv;
  }
  __syncthreads();
  // top-k: k rounds of block argmax (value desc, id asc), selected entries removed
  float wsum = 0.f;
  for (int j = 0; j < k; ++j) {
    float bv = -1.0f;
    int bi = 0x7fffffff;
    for (int e = tid; e < E; e += 256) {
      const float v = pr[e];
      if (v > bv || (v == bv && e < bi)) { bv = v; bi = e; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    if (lane == 0) { red_v[w] = bv; red_i[w] = bi; }
    __syncthreads();
    if (tid == 0) {
      for (int q = 1; q < 4; ++q)
        if (red_v[q] > red_v[0] || (red_v[q] == red_v[0] && red_i[q] < red_i[0])) {
          red_v[0] = red_v[q];
          red_i[0] = red_i[q];
        }
      topk_id[(int64_t)r * k + j] = red_i[0];
      topk_w[(int64_t)r * k + j] = red_v[0];
      wsum += red_v[0];
      pr[red_i[0]] = -2.0f;                 // removed
      atomicAdd(&counts[red_i[0]], 1);
    }
    __syncthreads();
  }
  if (tid == 0) {
    const float inv = 1.0f / wsum;
    for (int j = 0; j < k; ++j) topk_w[(int64_t)r * k + j] *= inv;
  }
}

// Exclusive scan of E counts (E <= 1024) into offsets; cursors reset to 0.
__global__ void __launch_bounds__(1024) moe_offsets_kernel(const int32_t* __restrict__ counts, int E,
                                                           int32_t* __restrict__ offsets,
                                                           int32_t* __restrict__ cursors) {
  __shared__ int32_t sh[1024];
  const int tid = threadIdx.x;
  const int v = tid < E ? counts[tid] : 0;
  sh[tid] = v;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int x = tid >= o ? sh[tid - o] : 0;
    __syncthreads();
    sh[tid] += x;
    __syncthreads();
  }
  if (tid < E) {
    offsets[tid] = sh[tid] - v;
    cursors[tid] = 0;
  }
}

// One block per row: place its k pairs and copy the input row into each.
__global__ void __launch_bounds__(256) moe_scatter_kernel(const bf16_t* __restrict__ xn, int d, int k,
                                                          const int32_t* __restrict__ topk_id,
                                                          const int32_t* __restrict__ offsets,
                                                          int32_t* __restrict__ cursors,
                                                          int32_t* __restrict__ pos_of,
                                                          bf16_t* __restrict__ a_perm) {
  __shared__ int32_t pos[64];
  const int r = blockIdx.x, tid = threadIdx.x;
  if (tid < k) {
    const int e = topk_id[(int64_t)r * k + tid];
    const int p = offsets[e] + atomicAdd(&cursors[e], 1);
    pos[tid] = p;
    pos_of[(int64_t)r * k + tid] = p;
  }
  __syncthreads();
  const uint32_t* src = (const uint32_t*)(xn + (int64_t)r * d);
  for (int j = 0; j < k; ++j) {
    uint32_t* dst = (uint32_t*)(a_perm + (int64_t)pos[j] * d);
    for (int c = tid; c < d / 2; c += 256) dst[c] = src[c];
  }
}

// Grouped GEMM over expert segments: for expert e, rows [off, off+cnt) of A
// times W_e^T (W_e = W + e * w_stride, [N][K]).  Block: 8 wavefronts, NS*16
// output columns of one expert, K split over the wavefronts; rows in tiles of
// 16*MT.  Operand fragments go straight from memory to MFMA registers.
//   SWIGLU: W rows interleaved gate/up in groups of 16, out bf16 [.][N/2]
//   else:   out fp32 [.][N]
template <int MT, int NS, bool SWIGLU>
__global__ void __launch_bounds__(512) moe_gemm_kernel(const bf16_t* __restrict__ A, int K,
                                                       const bf16_t* __restrict__ W,
                                                       int64_t w_stride, int N,
                                                       const int32_t* __restrict__ offsets,
                                                       const int32_t* __restrict__ counts,
                                                       void* __restrict__ out) {
  __shared__ f32x4_t red[8][MT * NS][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nslabs = N / (NS * 16);
  const int e = blockIdx.x / nslabs, slab = blockIdx.x % nslabs;
  const int cnt = counts[e];
  if (cnt == 0) return;
  const int off = offsets[e];
  const int n0 = slab * NS * 16;
  const int kw = K / 8, kbeg = wave * kw;
  const int kq = (lane >> 4) * 8, rr = lane & 15;
  const bf16_t* We = W + (int64_t)e * w_stride;
  for (int m0 = 0; m0 < cnt; m0 += 16 * MT) {
    f32x4_t acc[MT][NS];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NS; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    const bf16_t* wp[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) wp[j] = We + (int64_t)(n0 + 16 * j + rr) * K + kbeg + kq;
    const bf16_t* ap[MT];
    bool av[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int row = m0 + 16 * i + rr;
      av[i] = row < cnt;
      ap[i] = A + (int64_t)(off + (av[i] ? row : 0)) * K + kbeg + kq;
    }
#pragma unroll 2
    for (int kk = 0; kk < kw; kk += 32) {
      bf16x8_t a[MT], b[NS];
#pragma unroll
      for (int j = 0; j < NS; ++j) b[j] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(wp[j] + kk));
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        u32x4_t v = *(const u32x4_t*)(ap[i] + kk);
        if (!av[i]) v = (u32x4_t){0u, 0u, 0u, 0u};
        a[i] = __builtin_bit_cast(bf16x8_t, v);
      }
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NS; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();   // red[] of the previous row tile has been consumed
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NS; ++j) red[wave][i * NS + j][lane] = acc[i][j];
    __syncthreads();
    for (int t = wave; t < MT * NS; t += 8) {
      f32x4_t s = red[0][t][lane];
#pragma unroll
      for (int q = 1; q < 8; ++q) s += red[q][t][lane];
      red[0][t][lane] = s;
    }
    __syncthreads();
    if constexpr (SWIGLU) {
      bf16_t* H = (bf16_t*)out;
      const int F = N / 2;
      for (int t = wave; t < MT * (NS / 2); t += 8) {
        const int i = t / (NS / 2), jp = t % (NS / 2);
        const f32x4_t g = red[0][i * NS + 2 * jp][lane], u = red[0][i * NS + 2 * jp + 1][lane];
        const int col = ((n0 + 32 * jp) >> 5) * 16 + (lane & 15);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = m0 + 16 * i + 4 * (lane >> 4) + q;
          if (row < cnt) {
            const float gv = g[q];
            H[(int64_t)(off + row) * F + col] = f32_to_bf16(gv / (1.0f + __expf(-gv)) * u[q]);
          }
        }
      }
    } else {
      float* Y = (float*)out;
      for (int t = wave; t < MT * NS; t += 8) {
        const int i = t / NS, j = t % NS;
        const f32x4_t v = red[0][t][lane];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = m0 + 16 * i + 4 * (lane >> 4) + q;
          if (row < cnt) Y[(int64_t)(off + row) * N + n0 + 16 * j + (lane & 15)] = v[q];
        }
      }
    }
  }
}

// x[r] += sum_j w[r][j] * y[pos(r, j)]   (slot order)
__global__ void __launch_bounds__(256) moe_combine_kernel(const float* __restrict__ y, int d, int k,
                                                          const int32_t* __restrict__ pos_of,
                                                          const float* __restrict__ topk_w,
                                                          float* __restrict__ x) {
  const int r = blockIdx.x;
  for (int c = threadIdx.x; c < d; c += 256) {
    float s = 0.f;
    for (int j = 0; j < k; ++j)
      s = fmaf(topk_w[(int64_t)r * k + j], y[(int64_t)pos_of[(int64_t)r * k + j] * d + c], s);
    x[(int64_t)r * d + c] += s;
  }
}

__global__ void zero_i32_kernel(int32_t* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

hipError_t launch_moe_ffn(const MoeArgs& a, hipStream_t st) {
  if (a.n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(1024), 0, st, a.counts, a.E);
  hipLaunchKernelGGL(moe_route_kernel, dim3(a.n_rows), dim3(256), (size_t)(a.d + a.E) * 4, st, a.xn,
                     a.d, a.w_router, a.E, a.k, a.topk_id, a.topk_w, a.counts);
  hipLaunchKernelGGL(moe_offsets_kernel, dim3(1), dim3(1024), 0, st, a.counts, a.E, a.offsets,
                     a.cursors);
  hipLaunchKernelGGL(moe_scatter_kernel, dim3(a.n_rows), dim3(256), 0, st, a.xn, a.d, a.k, a.topk_id,
                     a.offsets, a.cursors, a.pos_of, a.a_perm);
  const int Fe = a.Fe, d = a.d;
  // gate/up: N = 2*Fe, K = d; down: N = d, K = Fe
  hipLaunchKernelGGL((moe_gemm_kernel<4, 2, true>), dim3(a.E * (2 * Fe / 32)), dim3(512), 0, st,
                     a.a_perm, d, a.w_gu, (int64_t)2 * Fe * d, 2 * Fe, a.offsets, a.counts,
                     (void*)a.h_perm);
  hipLaunchKernelGGL((moe_gemm_kernel<4, 2, false>), dim3(a.E * (d / 32)), dim3(512), 0, st,
                     a.h_perm, Fe, a.w_down, (int64_t)d * Fe, d, a.offsets, a.counts, (void*)a.y_perm);
  hipLaunchKernelGGL(moe_combine_kernel, dim3(a.n_rows), dim3(256), 0, st, a.y_perm, d, a.k,
                     a.pos_of, a.topk_w, a.x);
  return hipGetLastError();
}

}  // namespace darts
