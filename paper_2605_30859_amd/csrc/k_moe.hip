// Mixture-of-experts FFN of the decoder (top-k of E experts, renormalised).
//
//   route:    router logits = h W_router^T on the dense GEMM path (router rows
//             zero-padded to a multiple of 128); per row r = softmax over the E
//             logits, the k largest (ties to the lower expert id), weights
//             renormalised over the k
//   offsets:  per-expert counts (block histogram), their exclusive scan, one
//             list of expert row tiles per projection, and a position in its
//             expert's segment for every (row, slot) pair
//   experts:  grouped GEMMs over the expert segments: gate/up (+ SwiGLU
//             epilogue; its A rows are gathered from the normalised input
//             through the position -> row list; strip-packed weights, in
//             decode batches streamed straight into MFMA registers), then down
//   combine:  x[row] += sum_j w[row][j] * y[pos(row, j)]   (slot order),
//             then the next RMSNorm of the updated row
// Positions inside a segment come from atomics, so their order varies from
// run to run, but no value depends on it: every output row of an expert GEMM
// depends only on its own input row, and the combine sums in slot order.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace darts {

// One wavefront per row: softmax over the E router logits (fp32); the k
// largest probabilities (value descending, expert id ascending) are found by
// rank: the row's sort keys go to LDS, every lane counts for each of its
// experts how many experts come before it in that order, and the experts of
// rank < k are written to their rank's slot.  This gives the order k rounds
// of wavefront argmax would (a probability that is NaN ranks after every
// number), without their chain of dependent cross-lane steps.  The weights
// are renormalised over the k, summed in rank order.  NPL logits per lane
// (E <= 64 * NPL).  The logits are the sum of n_split split-K partial planes
// split_stride apart, added in plane order (the dense reduce's order), so the
// router GEMM needs no separate reduce.
constexpr int kMoeMaxPerLane = 16;   // E <= 1024
constexpr int kMoeMaxSplits = 8;     // router GEMM K splits the top-k kernel sums
// DBG (verification only): the router's own ids are exported, and a row whose
// key has k forced ids in [0, E) combines those experts instead, with their
// own softmax probabilities renormalised over the k.
template <int NPL, bool DBG>
__global__ void __launch_bounds__(256) moe_topk_kernel(const float* __restrict__ logits, int ld,
                                                       int n_split, int64_t split_stride,
                                                       int n_rows, int E, int k,
                                                       int32_t* __restrict__ topk_id,
                                                       float* __restrict__ topk_w, MoeArgs dbg) {
  // each wavefront's row of sort keys: (order-preserving probability bits,
  // 0xffff - expert id); a larger key ranks first, and keys are distinct
  __shared__ __attribute__((aligned(16))) uint64_t sk[4][64 * NPL];
  __shared__ float sv[4][64];            // selected probabilities by rank
  __shared__ int32_t si[4][64];          // selected expert ids by rank
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = blockIdx.x * 4 + w;
  if (r >= n_rows) return;
  const float* lg = logits + (int64_t)r * ld;
  float p[NPL];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int e = lane + 64 * j;
    float v = -INFINITY;
    if (e < E) {
      // all planes' loads issued before the adds (in plane order)
      float pz[kMoeMaxSplits];
#pragma unroll
      for (int z = 0; z < kMoeMaxSplits; ++z) pz[z] = z < n_split ? lg[z * split_stride + e] : 0.f;
      v = 0.f;
#pragma unroll
      for (int z = 0; z < kMoeMaxSplits; ++z)
        if (z < n_split) v += pz[z];
    }
    p[j] = v;
    mx = fmaxf(mx, p[j]);
  }
  mx = wave_max(mx);
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int e = lane + 64 * j;
    const float v = e < E ? __expf(p[j] - mx) : 0.f;
    p[j] = v;
    sum += v;
  }
  sum = wave_sum(sum);
  const float inv = 1.0f / sum;
  // probabilities (>= 0, so their bits order as unsigned integers); a NaN
  // ranks after every number, the padding past E after everything
  uint64_t key[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int e = lane + 64 * j;
    p[j] *= inv;
    const uint32_t ok = e < E ? (p[j] == p[j] ? __float_as_uint(p[j]) + 2u : 1u) : 0u;
    key[j] = ((uint64_t)ok << 32) | (uint32_t)(0xffff - e);
    sk[w][e] = key[j];
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);    // lgkmcnt(0): this wavefront's LDS writes are done
  __builtin_amdgcn_wave_barrier();
  int rank[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) rank[j] = 0;
  const int E2 = (E + 1) & ~1;
  // unrolled so that several LDS reads are in flight
#pragma unroll 8
  for (int y = 0; y < E2; y += 2) {
    const uint4 q = *(const uint4*)&sk[w][y];             // the same address in every lane
    const uint64_t q0 = ((uint64_t)q.y << 32) | q.x, q1 = ((uint64_t)q.w << 32) | q.z;
#pragma unroll
    for (int j = 0; j < NPL; ++j) rank[j] += (q0 > key[j]) + (q1 > key[j]);
  }
  float p0[DBG ? NPL : 1];
  if (DBG) {
#pragma unroll
    for (int j = 0; j < NPL; ++j) p0[j] = p[j];
  }
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int e = lane + 64 * j;
    if (e < E && rank[j] < k) {
      sv[w][rank[j]] = p[j];
      si[w][rank[j]] = e;
    }
  }
  __builtin_amdgcn_s_waitcnt(0xc07f);
  __builtin_amdgcn_wave_barrier();
  float wsum = 0.f;
#pragma unroll 8
  for (int t = 0; t < k; ++t) wsum += sv[w][t];        // rank order
  float my_w = lane < k ? sv[w][lane] : 0.f;
  int my_id = lane < k ? si[w][lane] : 0;
  if (DBG) {
    const int64_t rk = dbg.route_key ? (int64_t)dbg.route_key[r] : (int64_t)r;
    if (dbg.own_ids_out && lane < k) dbg.own_ids_out[rk * dbg.dbg_stride + lane] = my_id;
    if (dbg.force_ids) {
      const int32_t* f = dbg.force_ids + rk * dbg.dbg_stride;
      const int fid = lane < k ? f[lane] : 0;
      const bool forced = f[0] >= 0 && __all(fid >= 0 && fid < E);
      if (forced) {
        // probability of expert fid: lane fid % 64 holds it in slot fid / 64
        float pf = 0.f;
#pragma unroll
        for (int j = 0; j < NPL; ++j) {
          const float v = __shfl(p0[j], fid & 63, 64);
          if ((fid >> 6) == j) pf = v;
        }
        my_id = fid;
        my_w = pf;
        wsum = wave_sum(lane < k ? pf : 0.f);
      }
    }
    if (dbg.used_p_out && lane < k) dbg.used_p_out[rk * dbg.dbg_stride + lane] = my_w;
  }
  if (lane < k) {
    topk_id[(int64_t)r * k + lane] = my_id;
    topk_w[(int64_t)r * k + lane] = my_w * (1.0f / wsum);
  }
}

// Exclusive scan of one int per thread over a 1024-thread block: inclusive
// scans inside each wavefront (shuffles), the 16 wavefront totals scanned by
// the first wavefront through LDS, then added back.  sh holds >= 16 ints.
__device__ __forceinline__ int block_excl_scan1024(int v, int32_t* sh, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int x = __shfl_up(incl, o, 64);
    if (lane >= o) incl += x;
  }
  if (lane == 63) sh[w] = incl;
  __syncthreads();
  if (w == 0) {
    int t = lane < 16 ? sh[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int x = __shfl_up(t, o, 64);
      if (lane >= o) t += x;
    }
    if (lane < 16) sh[16 + lane] = t;    // inclusive totals of wavefronts 0..lane
  }
  __syncthreads();
  const int before = w > 0 ? sh[16 + w - 1] : 0;
  *total = sh[16 + 15];
  __syncthreads();                      // sh may be reused by the next scan
  return before + incl - v;
}

// Single block: per-expert counts of the n_pairs routed (row, slot) pairs
// (LDS histogram), their exclusive scan into offsets, cursors reset to 0, the
// list of non-empty expert row tiles (e << 16 | tile) for the grouped GEMMs,
// and every pair's position (pos_of) with its inverse (row_of).
__global__ void __launch_bounds__(1024) moe_offsets_kernel(const int32_t* __restrict__ topk_id,
                                                           int n_pairs, int E, int k,
                                                           int32_t* __restrict__ counts,
                                                           int32_t* __restrict__ offsets,
                                                           int32_t* __restrict__ cursors,
                                                           int32_t* __restrict__ mtiles,
                                                           int32_t* __restrict__ n_mtiles,
                                                           int32_t* __restrict__ mtiles2,
                                                           int32_t* __restrict__ n_mtiles2,
                                                           int32_t* __restrict__ pos_of,
                                                           int32_t* __restrict__ row_of,
                                                           int32_t* __restrict__ touched_out,
                                                           int tile_rows, int tile_rows2) {
  __shared__ int32_t hist[1024];
  __shared__ int32_t sh[1024];
  const int tid = threadIdx.x;
  hist[tid] = 0;
  __syncthreads();
  for (int i = tid; i < n_pairs; i += 1024) {
    const int e = topk_id[i];
    if (e >= 0 && e < E) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  const int v = tid < E ? hist[tid] : 0;
  int total;
  const int ex = block_excl_scan1024(v, sh, &total);
  const int nt = (v + tile_rows - 1) / tile_rows;
  int ntiles;
  const int tex = block_excl_scan1024(nt, sh, &ntiles);
  if (tid < E) {
    counts[tid] = v;
    offsets[tid] = ex;
    cursors[tid] = 0;
    for (int j = 0; j < nt; ++j) mtiles[tex + j] = (tid << 16) | j;
  }
  if (tid == 0) *n_mtiles = ntiles;
  // the second list (another row tile for the other projection)
  const int nt2 = (v + tile_rows2 - 1) / tile_rows2;
  int ntiles2;
  const int tex2 = block_excl_scan1024(nt2, sh, &ntiles2);
  if (tid < E)
    for (int j = 0; j < nt2; ++j) mtiles2[tex2 + j] = (tid << 16) | j;
  if (tid == 0) *n_mtiles2 = ntiles2;
  if (touched_out) {
    const int nz = __syncthreads_count(v > 0);
    if (tid == 0) *touched_out = nz;
  }
  // positions: pair i (row i / k) takes the next free slot of its expert's
  // segment; hist becomes the per-expert cursor
  hist[tid] = tid < E ? ex : 0;
  __syncthreads();
  for (int i = tid; i < n_pairs; i += 1024) {
    const int e = topk_id[i];
    if (e < 0 || e >= E) continue;
    const int p = atomicAdd(&hist[e], 1);
    pos_of[i] = p;
    row_of[p] = i / k;
  }
}

// x[r] += sum_j w[r][j] * y[pos(r, j)]   (slot order, y in bf16, the sum in
// fp32), 8 columns per thread: the k expert rows of a column chunk are
// loaded (16 bytes each) before any is summed, so their latencies overlap;
// with xn (d <= 4096) also xn[r] = bf16(x[r] / sqrt(mean(x[r]^2) + eps)).
constexpr int kCombCols = 8;
constexpr int kCombIters = 2;
constexpr int kCombBatch = 8;   // expert rows loaded before summing

__device__ __forceinline__ void comb_fma8(float* s, float w, const uint4& v) {
  s[0] = fmaf(w, bf16_to_f32((bf16_t)(v.x & 0xffffu)), s[0]);
  s[1] = fmaf(w, bf16_to_f32((bf16_t)(v.x >> 16)), s[1]);
  s[2] = fmaf(w, bf16_to_f32((bf16_t)(v.y & 0xffffu)), s[2]);
  s[3] = fmaf(w, bf16_to_f32((bf16_t)(v.y >> 16)), s[3]);
  s[4] = fmaf(w, bf16_to_f32((bf16_t)(v.z & 0xffffu)), s[4]);
  s[5] = fmaf(w, bf16_to_f32((bf16_t)(v.z >> 16)), s[5]);
  s[6] = fmaf(w, bf16_to_f32((bf16_t)(v.w & 0xffffu)), s[6]);
  s[7] = fmaf(w, bf16_to_f32((bf16_t)(v.w >> 16)), s[7]);
}

__global__ void __launch_bounds__(256) moe_combine_kernel(const bf16_t* __restrict__ y, int d, int k,
                                                          const int32_t* __restrict__ pos_of,
                                                          const float* __restrict__ topk_w,
                                                          float* __restrict__ x, float eps,
                                                          bf16_t* __restrict__ xn) {
  __shared__ int32_t sp[64];
  __shared__ float sw[64];
  __shared__ float red[4];
  const int r = blockIdx.x, tid = threadIdx.x;
  if (tid < k) {
    sp[tid] = pos_of[(int64_t)r * k + tid];
    sw[tid] = topk_w[(int64_t)r * k + tid];
  }
  __syncthreads();
  // one chunk: sum the k expert rows, add into x, return the new x values
  auto chunk = [&](int c, float* xv) {
    float s[kCombCols];
#pragma unroll
    for (int u = 0; u < kCombCols; ++u) s[u] = 0.f;
    for (int j0 = 0; j0 < k; j0 += kCombBatch) {
      uint4 v[kCombBatch];
#pragma unroll
      for (int u = 0; u < kCombBatch; ++u)
        if (j0 + u < k) v[u] = *(const uint4*)(y + (int64_t)sp[j0 + u] * d + c);
#pragma unroll
      for (int u = 0; u < kCombBatch; ++u)
        if (j0 + u < k) comb_fma8(s, sw[j0 + u], v[u]);
    }
    float4* xp = (float4*)(x + (int64_t)r * d + c);
    float4 x0 = xp[0], x1 = xp[1];
    x0.x += s[0]; x0.y += s[1]; x0.z += s[2]; x0.w += s[3];
    x1.x += s[4]; x1.y += s[5]; x1.z += s[6]; x1.w += s[7];
    xp[0] = x0;
    xp[1] = x1;
    xv[0] = x0.x; xv[1] = x0.y; xv[2] = x0.z; xv[3] = x0.w;
    xv[4] = x1.x; xv[5] = x1.y; xv[6] = x1.z; xv[7] = x1.w;
  };
  if (xn == nullptr) {
    float xv[kCombCols];
    for (int c = tid * kCombCols; c < d; c += 256 * kCombCols) chunk(c, xv);
    return;
  }
  // fused RMSNorm (d <= 256 * kCombCols * kCombIters): x stays in registers
  float keep[kCombIters][kCombCols];
  float ss = 0.f;
#pragma unroll
  for (int t = 0; t < kCombIters; ++t) {
    const int c = (tid + 256 * t) * kCombCols;
    if (c < d) {
      chunk(c, keep[t]);
#pragma unroll
      for (int u = 0; u < kCombCols; ++u) ss = fmaf(keep[t][u], keep[t][u], ss);
    }
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)d + eps);
#pragma unroll
  for (int t = 0; t < kCombIters; ++t) {
    const int c = (tid + 256 * t) * kCombCols;
    if (c >= d) continue;
    uint4 q;
    q.x = (uint32_t)f32_to_bf16(keep[t][0] * inv) | ((uint32_t)f32_to_bf16(keep[t][1] * inv) << 16);
    q.y = (uint32_t)f32_to_bf16(keep[t][2] * inv) | ((uint32_t)f32_to_bf16(keep[t][3] * inv) << 16);
    q.z = (uint32_t)f32_to_bf16(keep[t][4] * inv) | ((uint32_t)f32_to_bf16(keep[t][5] * inv) << 16);
    q.w = (uint32_t)f32_to_bf16(keep[t][6] * inv) | ((uint32_t)f32_to_bf16(keep[t][7] * inv) << 16);
    *(uint4*)(xn + (int64_t)r * d + c) = q;
  }
}

hipError_t launch_moe_ffn(const MoeArgs& a, hipStream_t st, bool* normed) {
  *normed = false;
  if (a.n_rows <= 0) return hipSuccess;
  if (a.E > 64 * kMoeMaxPerLane || a.E > 1024 || a.k > 64 || a.k > a.E || a.d % kCombCols ||
      a.n_rows > 65536 * kGroupedTileRowsMin)
    return hipErrorInvalidValue;
  // router logits, or their split-K partial planes (summed by the top-k kernel)
  int n_split = 1;
  hipError_t e = launch_gemm_f32_or_partials(a.xn, a.d, a.w_router, a.d, a.logits, a.E_pad, a.n_rows,
                                             a.E_pad, a.d, a.gemm_ws, a.gemm_ws_bytes, st, &n_split);
  if (e != hipSuccess) return e;
  if (n_split > kMoeMaxSplits) return hipErrorInvalidValue;
  const float* lg = n_split > 1 ? (const float*)a.gemm_ws : a.logits;
  const int64_t zs = (int64_t)a.n_rows * a.E_pad;
  const dim3 gtk((a.n_rows + 3) / 4), btk(256);
  const GroupedPlan plan_gu = grouped_plan((int64_t)a.n_rows * a.k, a.E, true);
  const GroupedPlan plan_dn = grouped_plan((int64_t)a.n_rows * a.k, a.E, false);
  const bool dbg = a.force_ids || a.own_ids_out || a.used_p_out;
#define DARTS_TOPK(NPL)                                                                          \
  if (dbg)                                                                                       \
    hipLaunchKernelGGL((moe_topk_kernel<NPL, true>), gtk, btk, 0, st, lg, a.E_pad, n_split, zs,  \
                       a.n_rows, a.E, a.k, a.topk_id, a.topk_w, a);                              \
  else                                                                                           \
    hipLaunchKernelGGL((moe_topk_kernel<NPL, false>), gtk, btk, 0, st, lg, a.E_pad, n_split, zs, \
                       a.n_rows, a.E, a.k, a.topk_id, a.topk_w, a);
  if (a.E <= 128) {
    DARTS_TOPK(2)
  } else if (a.E <= 256) {
    DARTS_TOPK(4)
  } else {
    DARTS_TOPK(kMoeMaxPerLane)
  }
#undef DARTS_TOPK
  hipLaunchKernelGGL(moe_offsets_kernel, dim3(1), dim3(1024), 0, st, a.topk_id, a.n_rows * a.k, a.E, a.k,
                     a.counts, a.offsets, a.cursors, a.mtiles, a.n_mtiles, a.mtiles_dn, a.n_mtiles_dn,
                     a.pos_of, a.row_of, a.touched_out, plan_gu.tile_rows, plan_dn.tile_rows);
  const int Fe = a.Fe, d = a.d;
  // gate/up: N = 2*Fe, K = d (SwiGLU into h_perm), A rows gathered from xn;
  // down: N = d, K = Fe
  if (a.ev_gu0 && (e = hipEventRecord(a.ev_gu0, st)) != hipSuccess) return e;
  e = launch_gemm_grouped(a.xn, d, a.w_gu, (int64_t)2 * Fe * d, d, a.h_perm, Fe, 2 * Fe, d,
                          EPI_SWIGLU, a.offsets, a.counts, a.mtiles, a.n_mtiles, a.row_of, plan_gu,
                          true, st);
  if (e != hipSuccess) return e;
  if (a.ev_gu1 && (e = hipEventRecord(a.ev_gu1, st)) != hipSuccess) return e;
  if (a.ev_down0 && (e = hipEventRecord(a.ev_down0, st)) != hipSuccess) return e;
  e = launch_gemm_grouped(a.h_perm, Fe, a.w_down, (int64_t)d * Fe, Fe, a.y_perm, d, d, Fe, EPI_BF16,
                          a.offsets, a.counts, a.mtiles_dn, a.n_mtiles_dn, nullptr, plan_dn, false, st);
  if (e != hipSuccess) return e;
  if (a.ev_down1 && (e = hipEventRecord(a.ev_down1, st)) != hipSuccess) return e;
  const bool fuse = d <= 256 * kCombCols * kCombIters;
  hipLaunchKernelGGL(moe_combine_kernel, dim3(a.n_rows), dim3(256), 0, st, a.y_perm, d, a.k,
                     a.pos_of, a.topk_w, a.x, a.eps, fuse ? a.xn : nullptr);
  e = hipGetLastError();
  if (e == hipSuccess) *normed = fuse;
  return e;
}

}  // namespace darts
