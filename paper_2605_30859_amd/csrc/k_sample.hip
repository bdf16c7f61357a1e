// Fused sampler: one pass over a logits row computes
//   * the Gumbel-max token  argmax_i fl32(z_i + g_i),  z = logits / T,
//     g_i = -ln(-ln u_i), u_i from Philox(counter=(i>>2, traj, step, TAG_SAMPLE),
//     key=seed), ties to the smallest index;
//   * log-sum-exp and entropy with an online (max, sum e^(z-m), sum e^(z-m)(z-m))
//     state merged across lanes and wavefronts;
// then the log-prob of the taken token.  In the stateful form the same block
// applies the exogenous termination rule (forced end-of-sequence length,
// truncation at cap) and accumulates the trajectory's score.  When few rows
// are live (given room for partials), a row's vocabulary is split into
// slices, one block each, and a finalize kernel merges the slices' states
// and winners before finishing the row.
//
// Filtered argmax.  g_i is defined by the library's exact float32 logarithm
// (two per element, each with a correctly rounded division), which would
// dominate the kernel's arithmetic.  The scan instead scores every element
// with a fast map (two hardware log2 evaluations) whose distance from the
// exact map is at most kGumbelFastBound over all 2^23 possible u (checked
// exhaustively on the device by the test suite), and each thread keeps its
// two best fast scores.  If they are further apart than twice the bound on
// |fast score - exact score| (noise error plus the float32 roundings of the
// two sums), the thread's exact winner is its fast winner, whose exact score
// is then computed once; otherwise (a near tie, probability ~1e-5 per thread)
// the thread re-scans its elements with the exact map.  The token is
// therefore the exact-map argmax, bit for bit, in every case.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace darts {

struct SoftState {
  float m, s, t;   // max, sum e^(z-m), sum e^(z-m)(z-m)
};
__device__ __forceinline__ SoftState soft_merge(SoftState a, SoftState b) {
  if (a.m == -INFINITY) return b;
  if (b.m == -INFINITY) return a;
  const float m = fmaxf(a.m, b.m);
  const float ea = __expf(a.m - m), eb = __expf(b.m - m);
  SoftState r;
  r.m = m;
  r.s = a.s * ea + b.s * eb;
  r.t = ea * (a.t + a.s * (a.m - m)) + eb * (b.t + b.s * (b.m - m));
  return r;
}
struct Best {
  float v;
  int i;
};
__device__ __forceinline__ Best best_merge(Best a, Best b) {
  if (b.v > a.v || (b.v == a.v && b.i < a.i)) return b;
  return a;
}

template <bool BF16>
__device__ __forceinline__ void load4(const void* row, int j, float z[4]) {
  if (BF16) {
    const uint2 v = ((const uint2*)row)[j];
    z[0] = __uint_as_float(v.x << 16);
    z[1] = __uint_as_float(v.x & 0xffff0000u);
    z[2] = __uint_as_float(v.y << 16);
    z[3] = __uint_as_float(v.y & 0xffff0000u);
  } else {
    const float4 v = ((const float4*)row)[j];
    z[0] = v.x; z[1] = v.y; z[2] = v.z; z[3] = v.w;
  }
}

// Fast Gumbel map: -ln(-ln u) from two hardware log2 evaluations (the only
// approximation; products by ln 2 in float32).  u in [2^-24, 1 - 2^-24]
// keeps both log2 arguments normal.
__device__ __forceinline__ float gumbel_fast(float u) {
  constexpr float kLn2 = 0.693147180559945309f;
  const float a = -kLn2 * __builtin_amdgcn_logf(u);
  return -kLn2 * __builtin_amdgcn_logf(a);
}
// |gumbel_fast(u) - gumbel_of(u)| <= kGumbelFastBound for every u the sampler
// draws (measured maximum 1.9e-6; the bound is 2^-17)
constexpr float kGumbelFastBound = 7.62939453125e-06f;

template <bool BF16>
__device__ __forceinline__ float logit_at(const void* row, int i, bool tscale, float temperature) {
  float z = BF16 ? bf16_to_f32(((const bf16_t*)row)[i]) : ((const float*)row)[i];
  return tscale ? __fdiv_rn(z, temperature) : z;
}

// Per-row values every part of a row shares.
struct RowCtx {
  int g, step;
  const void* row;
};
template <bool BF16, bool STATEFUL>
__device__ __forceinline__ RowCtx row_ctx(const SampleArgs& a, int r) {
  RowCtx c;
  c.g = a.traj[r];
  const int lrow = a.row_logit ? a.row_logit[r] : (a.logit_div > 0 ? c.g / a.logit_div : r);
  c.row = BF16 ? (const void*)((const bf16_t*)a.logits + (int64_t)lrow * a.vocab)
               : (const void*)((const float*)a.logits + (int64_t)lrow * a.vocab);
  c.step = STATEFUL ? a.gen[c.g] : a.step[r];
  return c;
}

// Row r's result from its merged softmax state and Gumbel-max winner: the
// taken token (forced end of sequence, teacher forcing), its log-prob, the
// entropy and, in the stateful form, termination and score accumulation.
template <bool BF16, bool STATEFUL>
__device__ __forceinline__ void finish_row(const SampleArgs& a, int r, const RowCtx& c, SoftState st,
                                           Best best) {
  const int g = c.g, step = c.step;
  // A row with no finite perturbed score (every logit -inf or NaN) has no
  // Gumbel-max winner: token 0 stands in (the lowest index, as for equal
  // scores), and its log-prob and entropy are NaN.
  const bool has_winner = best.i >= 0 && best.i < a.vocab;
  const float lse = st.m + logf(st.s);
  const float ent = has_winner ? logf(st.s) - st.t / st.s : NAN;
  const int sampled = has_winner ? best.i : 0;
  int taken = sampled;
  uint8_t fin = 0;
  if (STATEFUL) {
    const int s_new = step + 1;
    const int d = a.forced_len[g];
    if (d <= a.cap && s_new == d) { taken = a.eos; fin = 1; }
    else {
      if (a.force && a.force[g] >= 0) taken = a.force[g];
      if (s_new >= a.cap) fin = 2;
    }
  } else if (a.force && a.force[r] >= 0) {
    taken = a.force[r];
  }
  if (taken < 0 || taken >= a.vocab) taken = sampled;   // sampled is in [0, vocab)
  const float zt = logit_at<BF16>(c.row, taken, a.temperature != 1.0f, a.temperature);
  const float lp = has_winner ? zt - lse : NAN;
  if (a.token_out) a.token_out[r] = taken;
  if (a.sampled_out) a.sampled_out[r] = sampled;
  if (a.logprob_out) a.logprob_out[r] = lp;
  if (a.entropy_out) a.entropy_out[r] = ent;
  if (STATEFUL) {
    if (a.hist_tok && step < a.cap) {
      a.hist_tok[(int64_t)g * a.cap + step] = taken;
      a.hist_lp[(int64_t)g * a.cap + step] = lp;
    }
    a.gen[g] = step + 1;
    a.sum_lp[g] = a.sum_lp[g] + lp;
    a.last_tok[g] = taken;
    if (fin) a.status[g] = fin;
    if (a.finished_out) a.finished_out[r] = fin;
    if (a.traj_out) a.traj_out[r] = g;
  }
}

// Block (r, part): part `part` of the a.parts contiguous slices of row r's
// vocabulary.  With one part the block finishes the row; with several it
// writes its partial (softmax state, winner) and the finalize kernel merges
// the parts.
template <bool BF16, bool STATEFUL>
__global__ void __launch_bounds__(256) sample_kernel(SampleArgs a) {
  __shared__ SoftState ss[4];
  __shared__ Best sb[4];
  const int parts = a.parts > 1 ? a.parts : 1;
  const int r = blockIdx.x / parts, part = blockIdx.x - r * parts;
  const int tid = threadIdx.x;
  const RowCtx c = row_ctx<BF16, STATEFUL>(a, r);
  const int g = c.g, step = c.step;
  const uint32_t gc = (uint32_t)g + (uint32_t)a.traj_base;   // the counter's (global) trajectory id
  const void* row = c.row;
  const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
  const bool tscale = a.temperature != 1.0f;
  SoftState st = {-INFINITY, 0.f, 0.f};
  float b1 = -INFINITY, b2 = -INFINITY;   // this thread's two best fast scores
  int i1 = 0x7fffffff;                     // index of the best
  const int n4 = a.vocab >> 2;
  const int span = (n4 + parts - 1) / parts;
  const int jb = part * span, je = min(n4, jb + span);
  for (int j = jb + tid; j < je; j += 256) {
    float z[4];
    load4<BF16>(row, j, z);
    if (tscale) {
#pragma unroll
      for (int e = 0; e < 4; ++e) z[e] = __fdiv_rn(z[e], a.temperature);
    }
    const Philox4 p = philox4x32_10((uint32_t)j, gc, (uint32_t)step, kTagSample, k0, k1);
    float lm = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    if (lm > st.m) {
      if (st.s > 0.f) {   // rescale the running sums to the new maximum
        const float sc = __expf(st.m - lm);
        st.t = sc * (st.t + st.s * (st.m - lm));
        st.s = st.s * sc;
      }
      st.m = lm;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      // masked (-inf) logits add nothing: d clamps to -FLT_MAX (also when the
      // running max is still -inf), so e^d = 0 and the entropy term 0 * d = 0
      const float d = fmaxf(z[e] - st.m, -3.40282347e+38f);
      const float ez = __expf(d);
      st.s += ez;
      st.t = fmaf(ez, d, st.t);
      const float sf = z[e] + gumbel_fast(open_unit(p.x[e]));
      const bool c1 = sf > b1, c2 = sf > b2;
      b2 = c1 ? b1 : (c2 ? sf : b2);
      b1 = c1 ? sf : b1;
      i1 = c1 ? 4 * j + e : i1;
    }
  }
  // exact score of this thread's winner, or an exact re-scan on a near tie
  Best best = {-INFINITY, 0x7fffffff};
  const float margin =
      2.0f * (kGumbelFastBound + 2.384185791015625e-07f * fmaxf(fabsf(b1), fabsf(b2)));   // 2^-22 |s|
  if (b1 - b2 > margin) {
    const int j = i1 >> 2, e = i1 & 3;
    const Philox4 p = philox4x32_10((uint32_t)j, gc, (uint32_t)step, kTagSample, k0, k1);
    best.v = logit_at<BF16>(row, i1, tscale, a.temperature) + gumbel_of(open_unit(p.x[e]));
    best.i = i1;
  } else {
    for (int j = jb + tid; j < je; j += 256) {
      float z[4];
      load4<BF16>(row, j, z);
      const Philox4 p = philox4x32_10((uint32_t)j, gc, (uint32_t)step, kTagSample, k0, k1);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float zz = tscale ? __fdiv_rn(z[e], a.temperature) : z[e];
        const float sc = zz + gumbel_of(open_unit(p.x[e]));
        if (sc > best.v) { best.v = sc; best.i = 4 * j + e; }
      }
    }
  }
  // wavefront merge
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    SoftState other = {__shfl_xor(st.m, o, 64), __shfl_xor(st.s, o, 64), __shfl_xor(st.t, o, 64)};
    st = soft_merge(st, other);
    Best ob = {__shfl_xor(best.v, o, 64), __shfl_xor(best.i, o, 64)};
    best = best_merge(best, ob);
  }
  if ((tid & 63) == 0) { ss[tid >> 6] = st; sb[tid >> 6] = best; }
  __syncthreads();
  if (tid != 0) return;
  st = soft_merge(soft_merge(ss[0], ss[1]), soft_merge(ss[2], ss[3]));
  best = best_merge(best_merge(sb[0], sb[1]), best_merge(sb[2], sb[3]));
  if (parts > 1) {
    SamplePart o;
    o.m = st.m; o.s = st.s; o.t = st.t; o.v = best.v; o.i = best.i;
    a.part_out[blockIdx.x] = o;
    return;
  }
  finish_row<BF16, STATEFUL>(a, r, c, st, best);
}

// One wavefront per row: lane l merges parts l, l + 64 (in that order), the
// lanes are then merged by a fixed butterfly (a fixed order, so the result
// is reproducible), and lane 0 finishes the row.
template <bool BF16, bool STATEFUL>
__global__ void __launch_bounds__(256) sample_finalize_kernel(SampleArgs a) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= a.n_rows) return;
  SoftState st = {-INFINITY, 0.f, 0.f};
  Best best = {-INFINITY, 0x7fffffff};
  for (int p = lane; p < a.parts; p += 64) {
    const SamplePart o = a.part_out[(int64_t)r * a.parts + p];
    st = soft_merge(st, SoftState{o.m, o.s, o.t});
    best = best_merge(best, Best{o.v, o.i});
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    SoftState other = {__shfl_xor(st.m, o, 64), __shfl_xor(st.s, o, 64), __shfl_xor(st.t, o, 64)};
    st = soft_merge(st, other);
    Best ob = {__shfl_xor(best.v, o, 64), __shfl_xor(best.i, o, 64)};
    best = best_merge(best, ob);
  }
  if (lane == 0) finish_row<BF16, STATEFUL>(a, r, row_ctx<BF16, STATEFUL>(a, r), st, best);
}

int sample_parts(int n_rows, int vocab) {
  // about kSampleBlocks blocks in all, each part at least kSampleMinGroups
  // groups of 4 logits (two per thread), at most kSampleMaxParts per row
  const int n4 = vocab >> 2;
  int parts = (kSampleBlocks + n_rows - 1) / n_rows;
  parts = std::min(parts, std::max(1, n4 / kSampleMinGroups));
  return std::max(1, std::min(parts, kSampleMaxParts));
}

hipError_t launch_sample(const SampleArgs& a0, hipStream_t st) {
  if (a0.n_rows <= 0) return hipSuccess;
  SampleArgs a = a0;
  a.parts = a.part_out ? sample_parts(a.n_rows, a.vocab) : 1;
  if (a.parts > 1 && (int64_t)a.n_rows * a.parts > a.part_cap) a.parts = 1;
  const bool stateful = a.gen != nullptr;
  const dim3 grid((unsigned)(a.n_rows * a.parts)), blk(256);
  const dim3 gfin((unsigned)((a.n_rows + 3) / 4));
  if (a.bf16) {
    if (stateful) hipLaunchKernelGGL((sample_kernel<true, true>), grid, blk, 0, st, a);
    else hipLaunchKernelGGL((sample_kernel<true, false>), grid, blk, 0, st, a);
    if (a.parts > 1) {
      if (stateful) hipLaunchKernelGGL((sample_finalize_kernel<true, true>), gfin, blk, 0, st, a);
      else hipLaunchKernelGGL((sample_finalize_kernel<true, false>), gfin, blk, 0, st, a);
    }
  } else {
    if (stateful) hipLaunchKernelGGL((sample_kernel<false, true>), grid, blk, 0, st, a);
    else hipLaunchKernelGGL((sample_kernel<false, false>), grid, blk, 0, st, a);
    if (a.parts > 1) {
      if (stateful) hipLaunchKernelGGL((sample_finalize_kernel<false, true>), gfin, blk, 0, st, a);
      else hipLaunchKernelGGL((sample_finalize_kernel<false, false>), gfin, blk, 0, st, a);
    }
  }
  return hipGetLastError();
}

}  // namespace darts

namespace darts {
__global__ void gumbel_map_kernel(const float* __restrict__ u, float* __restrict__ g, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    g[i] = gumbel_of(u[i]);
}
__global__ void gumbel_fast_map_kernel(const float* __restrict__ u, float* __restrict__ g, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    g[i] = gumbel_fast(u[i]);
}
hipError_t launch_gumbel_map(const float* u, float* g, int64_t n, bool fast, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (fast) hipLaunchKernelGGL(gumbel_fast_map_kernel, dim3((unsigned)blocks), dim3(256), 0, st, u, g, n);
  else hipLaunchKernelGGL(gumbel_map_kernel, dim3((unsigned)blocks), dim3(256), 0, st, u, g, n);
  return hipGetLastError();
}
float gumbel_fast_bound() { return kGumbelFastBound; }
}  // namespace darts
