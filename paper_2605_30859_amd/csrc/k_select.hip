// Distribution-aware selection (paper Sec. 4.1.2, Sec. 4.3.1, Alg. 2) and
// KV page bookkeeping.
//
// One wavefront decides one prompt group of m <= 64 trajectories (lane j =
// member j).  Orders are packed into 64-bit keys compared as integers:
//   shortest-first: (truncated, length, -mean_logprob, member)
//   longest-first:  (2^20-1-length, -mean_logprob, member)   [valid only]
// -mean_logprob is mapped to an order-preserving uint32 (NaN -> +inf, -0 -> +0).
// Shortest-only mode (m >= m_up) with early stop completes as soon as k
// members ended validly: the k first valid ones are kept, live members are
// aborted.  Otherwise a group completes when no member is live; shortest-only
// keeps the k first of all members, dual-end keeps the K = k-L first, then
// the L first remaining valid members by longest-first, then fills any
// deficit from the remaining members in shortest-first order.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace darts {

enum { ST_LIVE = 0, ST_EOS = 1, ST_TRUNC = 2, ST_ABORT = 3, ST_ABSENT = 4 };

__device__ __forceinline__ uint32_t ord_neg(float x) {
  float y = -x;
  if (x != x) y = INFINITY;
  if (y == 0.0f) y = 0.0f;           // -0 -> +0
  const uint32_t b = __float_as_uint(y);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src, 64), hi = __shfl((uint32_t)(v >> 32), src, 64);
  return ((uint64_t)hi << 32) | lo;
}

// rank of this lane's key among lanes in `pool` (mask) with a smaller key
__device__ __forceinline__ int rank_in(uint64_t key, uint64_t pool, int m) {
  int r = 0;
  for (int i = 0; i < m; ++i) {
    const uint64_t ki = shfl_u64(key, i);
    if (((pool >> i) & 1ull) && ki < key) ++r;
  }
  return r;
}

// Decide one group.  Returns true if it completed now (kept written, live
// members marked aborted in *st).  All lanes of the wave call this.
__device__ bool decide_group(int lane, int m, int k, int L, int m_up, int early_stop, uint8_t* st,
                             int len, float mlp, int g, int32_t* kept_row) {
  const bool act = lane < m;
  const uint8_t s = act ? *st : (uint8_t)ST_ABORT;
  const uint64_t live_m = __ballot(act && s == ST_LIVE);
  const uint64_t valid_m = __ballot(act && s == ST_EOS);
  const uint64_t all_m = __ballot(act);
  const int n_live = __popcll(live_m), n_valid = __popcll(valid_m);
  const uint32_t ln = (uint32_t)min(max(len, 0), (1 << 20) - 1);
  const uint64_t kshort = ((uint64_t)(s == ST_TRUNC) << 58) | ((uint64_t)ln << 38) |
                          ((uint64_t)ord_neg(mlp) << 6) | (uint64_t)lane;
  const uint64_t klong = ((uint64_t)((1u << 20) - 1 - ln) << 38) | ((uint64_t)ord_neg(mlp) << 6) |
                         (uint64_t)lane;
  if (m >= m_up) {
    uint64_t pool;
    bool abort_live;
    if (early_stop && n_valid >= k) { pool = valid_m; abort_live = true; }
    else if (n_live == 0) { pool = all_m; abort_live = false; }
    else return false;
    const int r = rank_in(kshort, pool, m);
    if (act && ((pool >> lane) & 1ull) && r < k) kept_row[r] = g;
    if (abort_live && act && s == ST_LIVE) *st = ST_ABORT;
    return true;
  }
  if (n_live != 0) return false;
  const int K = k - L;
  const int rs = rank_in(kshort, all_m, m);
  const bool in_short = act && rs < K;
  if (in_short) kept_row[rs] = g;
  const uint64_t elig = __ballot(act && s == ST_EOS && !in_short);
  const int rl = rank_in(klong, elig, m);
  const bool in_long = act && ((elig >> lane) & 1ull) && rl < L;
  if (in_long) kept_row[K + rl] = g;
  const int n_long = min(L, __popcll(elig));
  const uint64_t rest = __ballot(act && !in_short && !in_long);
  const int need = k - K - n_long;
  if (need > 0) {
    const int rf = rank_in(kshort, rest, m);
    if (act && ((rest >> lane) & 1ull) && rf < need) kept_row[K + n_long + rf] = g;
  }
  return true;
}

// Stateless: one wavefront per group, 4 groups per block.
__global__ void select_groups_kernel(uint8_t* status, const int32_t* len, const float* mean_lp,
                                     int n_groups, int m, int k, int L, int m_up, int early_stop,
                                     int32_t* kept, uint8_t* complete) {
  const int lane = threadIdx.x & 63;
  const int grp = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (grp >= n_groups) return;
  const int g = grp * m + lane;
  const bool act = lane < m;
  uint8_t dummy = ST_ABORT;
  uint8_t* stp = act ? &status[g] : &dummy;
  const int ln = act ? len[g] : 0;
  const float ml = act ? mean_lp[g] : 0.f;
  const bool c = decide_group(lane, m, k, L, m_up, early_stop, stp, ln, ml, g, kept + (int64_t)grp * k);
  if (lane == 0) complete[grp] = c ? 1 : 0;
}

// Page reclaim after a stateless selection, step 1 (single block): each
// group's freed count (all its members' pages if it completed, else 0), their
// exclusive scan into work[0 .. n_groups) and the total into work[n_groups]
// and *n_free.
__global__ void __launch_bounds__(1024) reclaim_scan_kernel(const uint8_t* __restrict__ complete,
                                                            const int32_t* __restrict__ page_off,
                                                            int n_groups, int m,
                                                            int32_t* __restrict__ work,
                                                            int32_t* __restrict__ n_free) {
  __shared__ int32_t sums[1024];
  __shared__ int32_t running;
  const int tid = threadIdx.x;
  if (tid == 0) running = 0;
  __syncthreads();
  for (int base = 0; base < n_groups; base += 1024) {
    const int grp = base + tid;
    const int c = (grp < n_groups && complete[grp])
                      ? page_off[(int64_t)(grp + 1) * m] - page_off[(int64_t)grp * m] : 0;
    sums[tid] = c;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {     // inclusive Hillis-Steele scan
      const int v = tid >= o ? sums[tid - o] : 0;
      __syncthreads();
      sums[tid] += v;
      __syncthreads();
    }
    if (grp < n_groups) work[grp] = running + sums[tid] - c;
    __syncthreads();
    if (tid == 1023) running += sums[1023];
    __syncthreads();
  }
  if (tid == 0) {
    work[n_groups] = running;
    *n_free = running;
  }
}

// Step 2: one block per group copies a completed group's page ids (its
// members' lists are contiguous in the page array) to its slot of free_out.
__global__ void __launch_bounds__(256) reclaim_copy_kernel(const uint8_t* __restrict__ complete,
                                                           const int32_t* __restrict__ page_off,
                                                           const int32_t* __restrict__ pages, int m,
                                                           const int32_t* __restrict__ work,
                                                           int32_t* __restrict__ free_out) {
  const int grp = blockIdx.x;
  if (!complete[grp]) return;
  const int64_t b = page_off[(int64_t)grp * m], e = page_off[(int64_t)(grp + 1) * m];
  int32_t* dst = free_out + work[grp] - b;
  for (int64_t i = b + threadIdx.x; i < e; i += 256) dst[i] = pages[i];
}

hipError_t launch_select(const GroupArgs& a, hipStream_t st) {
  if (a.n_groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(select_groups_kernel, dim3((a.n_groups + 3) / 4), dim3(256), 0, st, a.status,
                     a.len, a.mean_lp, a.n_groups, a.m, a.k, a.L, a.m_up, a.early_stop, a.kept,
                     a.complete);
  if (a.page_off) {
    hipLaunchKernelGGL(reclaim_scan_kernel, dim3(1), dim3(1024), 0, st, a.complete, a.page_off, a.n_groups,
                       a.m, a.work, a.n_free);
    hipLaunchKernelGGL(reclaim_copy_kernel, dim3(a.n_groups), dim3(256), 0, st, a.complete, a.page_off,
                       a.pages, a.m, a.work, a.free_out);
  }
  return hipGetLastError();
}

// Group-normalised advantages of the kept groups (Sec. 3.1, Eq. 2): one
// wavefront per group, lane j = kept slot j; mean and population standard
// deviation by wavefront sums.  A group with an id outside [0, n_traj) (not
// complete yet) gets NaN.
__global__ void advantage_kernel(const int32_t* kept, int n_groups, int k, const float* reward,
                                 int n_traj, float eps, float* adv) {
  const int lane = threadIdx.x & 63;
  const int grp = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (grp >= n_groups) return;
  const bool act = lane < k;
  const int g = act ? kept[(int64_t)grp * k + lane] : 0;
  const bool bad = __ballot(act && (g < 0 || g >= n_traj)) != 0ull;
  const float r = (act && !bad) ? reward[g] : 0.f;
  const float mu = wave_sum(r) / (float)k;
  const float dv = act ? r - mu : 0.f;
  const float sd = sqrtf(wave_sum(dv * dv) / (float)k);
  if (act) adv[(int64_t)grp * k + lane] = bad ? __int_as_float(0x7fc00000) : dv / (sd + eps);
}

hipError_t launch_advantages(const int32_t* kept, int n_groups, int k, const float* reward,
                             int n_traj, float eps, float* adv, hipStream_t st) {
  if (n_groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(advantage_kernel, dim3((n_groups + 3) / 4), dim3(256), 0, st, kept, n_groups,
                     k, reward, n_traj, eps, adv);
  return hipGetLastError();
}

// ---------------------------------------------------------------- stateful
// One block of 1024 threads (16 wavefronts) does the whole select-and-prune
// step: decide every open group, free the pages of members that ended or
// were aborted (and a prompt's shared pages when its last member is done),
// push them on the free stack in group order, compact the live list.
__device__ __forceinline__ int block_excl_scan(int v, int32_t* sh, int* total) {
  const int tid = threadIdx.x;
  sh[tid] = v;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int x = tid >= o ? sh[tid - o] : 0;
    __syncthreads();
    sh[tid] += x;
    __syncthreads();
  }
  const int incl = sh[tid];
  *total = sh[1023];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(1024) prune_kernel(PruneArgs a) {
  __shared__ int32_t sh[1024];
  __shared__ int32_t s_base;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // phase 1: decisions; pages each member / group releases now
  for (int grp = wv; grp < a.n_groups; grp += 16) {
    const int g = grp * a.m + lane;
    const int mi = a.grp_m[grp];              // this group's candidate count M'_i
    const bool act = lane < mi;
    if (!a.group_done[grp]) {
      uint8_t dummy = ST_ABORT;
      uint8_t* stp = act ? &a.status[g] : &dummy;
      const int ln = act ? a.gen[g] : 0;
      const float ml = (act && ln > 0) ? __fdiv_rn(a.sum_lp[g], (float)ln) : 0.f;
      const bool c = decide_group(lane, mi, a.k, a.L, a.m_up, a.early_stop, stp, ln, ml, g,
                                  a.kept + (int64_t)grp * a.k);
      if (c && lane == 0) { a.group_done[grp] = 1; a.done_step[grp] = a.step; }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    const bool now = act && a.status[g] != ST_LIVE && !a.freed[g];
    const int gn = act ? a.gen[g] : 0;
    const int priv = now ? (gn > 1 ? (gn - 1 + kPage - 1) / kPage : 0) : 0;
    if (act) a.trj_cnt[g] = priv;
    const int n_now = __popcll(__ballot(now));
    int tot = priv;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) tot += __shfl_xor(tot, o, 64);
    if (lane == 0) {
      int rel = 0;
      if (n_now > 0) {
        const int rc = a.refcnt[grp] - n_now;
        a.refcnt[grp] = rc;
        rel = (rc == 0) ? 1 : 0;
      }
      a.grp_rel[grp] = rel;
      a.grp_cnt[grp] = tot + (rel ? a.prompt_pages : 0);
    }
    if (now) a.freed[g] = 1;
  }
  __syncthreads();
  // phase 2: each group's start offset on the free stack (scan in group order)
  if (tid == 0) s_base = *a.free_top;
  __syncthreads();
  const int top0 = s_base;
  int running = 0;
  for (int base = 0; base < a.n_groups; base += 1024) {
    const int grp = base + tid;
    const int v = grp < a.n_groups ? a.grp_cnt[grp] : 0;
    int total;
    const int ex = block_excl_scan(v, sh, &total);
    if (grp < a.n_groups) a.grp_cnt[grp] = top0 + running + ex;
    running += total;
  }
  const int top1 = top0 + running;
  __syncthreads();
  // phase 3: push page ids: members in order, then the prompt's shared pages
  for (int grp = wv; grp < a.n_groups; grp += 16) {
    const int g = grp * a.m + lane;
    const bool act = lane < a.grp_m[grp];
    const int c = act ? a.trj_cnt[g] : 0;
    int incl = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int x = __shfl_up(incl, o, 64);
      if (lane >= o) incl += x;
    }
    const int start = a.grp_cnt[grp];
    const int off = start + incl - c;
    if (act) {
      const int32_t* ptr = a.page_table + (int64_t)g * a.pt_stride + a.prompt_pages;
      for (int t = 0; t < c; ++t)
        if (off + t < a.n_pages) a.free_stack[off + t] = ptr[t];
    }
    const int mem_tot = __shfl(incl, 63, 64);
    if (a.grp_rel[grp]) {
      const int32_t* pp = a.page_table + (int64_t)(grp * a.m) * a.pt_stride;
      for (int t = lane; t < a.prompt_pages; t += 64)
        if (start + mem_tot + t < a.n_pages) a.free_stack[start + mem_tot + t] = pp[t];
    }
  }
  __syncthreads();
  // phase 4: stable live-list compaction and counters
  running = 0;
  for (int base = 0; base < a.n_live_in; base += 1024) {
    const int i = base + tid;
    const int g = i < a.n_live_in ? a.live_in[i] : 0;
    const int keep = (i < a.n_live_in && a.status[g] == ST_LIVE) ? 1 : 0;
    int total;
    const int ex = block_excl_scan(keep, sh, &total);
    if (keep) a.live_out[running + ex] = g;
    running += total;
  }
  int nd = 0;
  for (int grp = tid; grp < a.n_groups; grp += 1024) nd += a.group_done[grp] ? 1 : 0;
  int total_done;
  (void)block_excl_scan(nd, sh, &total_done);
  if (tid == 0) {
    *a.free_top = min(top1, a.n_pages);
    a.info[0] = running;
    a.info[1] = total_done;
    a.info[2] = top1;
  }
}

hipError_t launch_prune(const PruneArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(prune_kernel, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}

// Token-chunk streaming (Sec. 4.3.2, producer side): one block of 1024
// threads.  Pending tokens of trajectory g are those generated since its last
// dispatch (gen[g] - streamed[g]); when their total reaches the threshold (or
// on a flush) every trajectory with pending tokens, or that ended and has not
// been marked final yet, gets one descriptor (ascending g) and its tokens are
// copied, in descriptor order, into the output buffers.
__global__ void __launch_bounds__(1024) stream_kernel(StreamArgs a) {
  __shared__ int32_t sh[1024];
  __shared__ int s_emit, s_ndesc;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // pass 1: pending total and whether some trajectory still owes a final mark
  int64_t pend_tot = 0;
  int owes = 0;
  for (int base = 0; base < a.n_traj; base += 1024) {
    const int g = base + tid;
    int pend = 0, fin = 0;
    if (g < a.n_traj && a.status[g] != ST_ABSENT) {
      pend = a.gen[g] - a.streamed[g];
      fin = (a.status[g] >= ST_EOS && a.status[g] <= ST_ABORT && !a.fin_sent[g]) ? 1 : 0;
    }
    int total, tf;
    (void)block_excl_scan(pend, sh, &total);
    (void)block_excl_scan(fin, sh, &tf);
    pend_tot += total;
    owes += tf;
  }
  if (tid == 0) {
    const bool emit = pend_tot >= a.threshold || (a.flush && (pend_tot > 0 || owes > 0));
    s_emit = !emit ? 0 : (pend_tot > a.out_cap ? -1 : 1);
    if (s_emit <= 0) { a.info[0] = s_emit < 0 ? -1 : 0; a.info[1] = (int32_t)pend_tot; }
  }
  __syncthreads();
  if (s_emit <= 0) return;
  // pass 2: descriptors, token offsets, dispatch bookkeeping
  int run_desc = 0, run_tok = 0;
  for (int base = 0; base < a.n_traj; base += 1024) {
    const int g = base + tid;
    int pend = 0, fin = 0, stv = 0, start = 0;
    if (g < a.n_traj && a.status[g] != ST_ABSENT) {
      stv = a.status[g];
      start = a.streamed[g];
      pend = a.gen[g] - start;
      fin = (stv >= ST_EOS && stv <= ST_ABORT && !a.fin_sent[g]) ? 1 : 0;
    }
    const int want = (pend > 0 || fin) ? 1 : 0;
    int nd, nt;
    const int di = block_excl_scan(want, sh, &nd);
    const int to = block_excl_scan(pend, sh, &nt);
    if (want) {
      const int i = run_desc + di;
      a.desc[4 * i] = g;
      a.desc[4 * i + 1] = start;
      a.desc[4 * i + 2] = pend;
      a.desc[4 * i + 3] = fin ? stv : 0;
      a.off[i] = run_tok + to;
      a.streamed[g] = start + pend;
      if (fin) a.fin_sent[g] = 1;
    }
    run_desc += nd;
    run_tok += nt;
  }
  if (tid == 0) { s_ndesc = run_desc; a.info[0] = run_desc; a.info[1] = run_tok; }
  __syncthreads();
  // pass 3: copy each descriptor's tokens (one wavefront per descriptor)
  for (int i = wv; i < s_ndesc; i += 16) {
    const int g = a.desc[4 * i], start = a.desc[4 * i + 1], cnt = a.desc[4 * i + 2];
    const int o = a.off[i];
    const int64_t src = (int64_t)g * a.cap + start;
    for (int t = lane; t < cnt; t += 64) {
      a.tok_out[o + t] = a.hist_tok[src + t];
      a.lp_out[o + t] = a.hist_lp[src + t];
    }
  }
}

hipError_t launch_stream(const StreamArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(stream_kernel, dim3(1), dim3(1024), 0, st, a);
  return hipGetLastError();
}

// Pop a page for every live row whose next key/value write starts a page:
// the token written this step has 0-based index gen-1 among the generated
// tokens, so a page is needed when (gen-1) % 16 == 0.  Pages are taken from
// the top of the stack in live-list order.  If the stack holds fewer pages
// than needed nothing is popped and info[3] is set.
__global__ void __launch_bounds__(1024) alloc_pages_kernel(const int32_t* live, int n_live,
                                                           const int32_t* gen, int prompt_pages,
                                                           int32_t* page_table, int pt_stride,
                                                           int32_t* free_stack, int32_t* free_top,
                                                           int32_t* info) {
  __shared__ int32_t sh[1024];
  __shared__ int32_t s_need;
  const int tid = threadIdx.x;
  int need = 0;
  for (int base = 0; base < n_live; base += 1024) {
    const int i = base + tid;
    const int v = (i < n_live && ((gen[live[i]] - 1) % kPage) == 0) ? 1 : 0;
    int total;
    (void)block_excl_scan(v, sh, &total);
    need += total;
  }
  if (tid == 0) s_need = need;
  __syncthreads();
  const int top = *free_top;
  if (s_need > top) {
    if (tid == 0) info[3] = 1;
    return;
  }
  int running = 0;
  for (int base = 0; base < n_live; base += 1024) {
    const int i = base + tid;
    const int g = i < n_live ? live[i] : 0;
    const int gn = i < n_live ? gen[g] : 1;
    const int v = (i < n_live && ((gn - 1) % kPage) == 0) ? 1 : 0;
    int total;
    const int ex = block_excl_scan(v, sh, &total);
    if (v) {
      const int page = free_stack[top - 1 - (running + ex)];
      page_table[(int64_t)g * pt_stride + prompt_pages + (gn - 1) / kPage] = page;
    }
    running += total;
  }
  __syncthreads();
  if (tid == 0) { *free_top = top - s_need; info[3] = 0; }
}

hipError_t launch_alloc_pages(const int32_t* live, int n_live, const int32_t* gen, int prompt_pages,
                              int32_t* page_table, int pt_stride, int32_t* free_stack,
                              int32_t* free_top, int32_t* info, hipStream_t st) {
  hipLaunchKernelGGL(alloc_pages_kernel, dim3(1), dim3(1024), 0, st, live, n_live, gen,
                     prompt_pages, page_table, pt_stride, free_stack, free_top, info);
  return hipGetLastError();
}

// Prefill: prompt i takes pages top-1-(i*pp + t), t < pp; every member's
// page-table row starts with them; refcount = the prompt's candidate count.
// Caller guarantees the stack holds n_prompts*pp pages.
__global__ void prefill_pages_kernel(int n_prompts, int m, const int32_t* grp_m, int pp,
                                     int32_t* page_table, int pt_stride,
                                     const int32_t* free_stack, const int32_t* free_top,
                                     int32_t* refcnt) {
  const int top = *free_top;
  const int64_t n = (int64_t)n_prompts * m * pp;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(t % pp);
    const int64_t gm = t / pp;
    const int g = (int)gm;
    const int i = g / m;
    page_table[(int64_t)g * pt_stride + j] = free_stack[top - 1 - (i * pp + j)];
    if (j == 0 && g % m == 0) refcnt[i] = grp_m[i];
  }
}
__global__ void set_top_kernel(int32_t* free_top, int delta) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *free_top += delta;
}

hipError_t launch_prefill_pages(int n_prompts, int m, const int32_t* grp_m, int prompt_pages,
                                int32_t* page_table, int pt_stride, int32_t* free_stack,
                                int32_t* free_top, int32_t* refcnt, hipStream_t st) {
  const int64_t n = (int64_t)n_prompts * m * prompt_pages;
  int64_t blocks = (n + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(prefill_pages_kernel, dim3((unsigned)blocks), dim3(256), 0, st, n_prompts, m,
                     grp_m, prompt_pages, page_table, pt_stride, free_stack, free_top, refcnt);
  hipLaunchKernelGGL(set_top_kernel, dim3(1), dim3(64), 0, st, free_top, -n_prompts * prompt_pages);
  return hipGetLastError();
}

}  // namespace darts
