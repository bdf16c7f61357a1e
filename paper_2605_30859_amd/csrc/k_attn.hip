// Paged GQA decode attention on gfx950.
//
// out[r][h] = sum_j softmax_j(q[r][h] . k_j / sqrt(hd)) v_j over the row's ctx
// keys; key j sits in page page_table[pt_row][j/16], slot j%16, kv head
// h / G (G = Hq/Hkv).
//
// Work unit = (row, kv head, chunk of C pages), one wavefront each, with a
// grid-stride loop; the wavefront attends 16 query vectors (MFMA rows) to a
// run of pages with an online softmax (attn_page_loop).  Rows of equal context
// (every decode step) map units arithmetically; ragged contexts use a work
// list built on the device (no host round trip, no idle blocks).  Contexts
// are split into chunks only when there are too few (row, kv head) units to
// fill the GPU; chunk partials (o, max, sum) are merged by a combine kernel.
//
// Shared prompt prefix (the rollout): the m trajectories of a prompt share
// its prompt pages.  A prefix kernel stacks the query vectors of a group's
// members 16 to a wavefront and reads each prefix page once per 16 query
// vectors (the per-row kernel fills only G of its 16 MFMA rows); the per-row
// kernel then covers the keys after the prefix, starting from the prefix
// partials.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace darts {

struct CtxSpec {
  const int32_t* ctx_len;  // per-row context, or NULL
  int mod, base;           // ctx(r) = ctx_len ? ctx_len[r] : (mod ? r % mod : 0) + base
  const int32_t* row_pt;   // page-table row of row r, or NULL (identity)
  int max_ctx;             // contexts are clamped to max_ctx (memory safety)
  int64_t n_pages;         // page ids are clamped into [0, n_pages)
  int skip;                // keys [0, skip) are attended by the shared-prefix kernel (a
                           // multiple of 16; 0 when prefixes are not shared)
  int pt_rows;             // row_pt values are clamped into [0, pt_rows) when > 0
};
__device__ __forceinline__ int pt_row(const CtxSpec& c, int r) {
  if (!c.row_pt) return r;
  const int v = c.row_pt[r];
  return c.pt_rows > 0 ? min(max(v, 0), c.pt_rows - 1) : v;
}
__device__ __forceinline__ int ctx_of(const CtxSpec& c, int r) {
  const int v = c.ctx_len ? c.ctx_len[r] : (c.mod ? r % c.mod : 0) + c.base;
  return min(v, c.max_ctx);
}
// keys the per-row kernel covers: those after the shared prefix
__device__ __forceinline__ int span_of(const CtxSpec& c, int r) { return max(ctx_of(c, r) - c.skip, 0); }
__device__ __forceinline__ int clamp_page(const CtxSpec& c, int p) {
  return (int)min((int64_t)max(p, 0), c.n_pages - 1);
}

// Single block: per-row chunk counts -> exclusive offsets and the work list.
__global__ void attn_plan_kernel(CtxSpec cs, int n_rows, int chunk_tokens, int32_t* chunk_off,
                                 int2* work, int32_t* info) {
  __shared__ int32_t sums[1024];
  __shared__ int32_t running;
  const int tid = threadIdx.x;
  if (tid == 0) running = 0;
  __syncthreads();
  for (int base = 0; base < n_rows; base += 1024) {
    const int r = base + tid;
    const int c = r < n_rows ? (span_of(cs, r) + chunk_tokens - 1) / chunk_tokens : 0;
    sums[tid] = c;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {     // inclusive Hillis-Steele scan
      const int v = tid >= o ? sums[tid - o] : 0;
      __syncthreads();
      sums[tid] += v;
      __syncthreads();
    }
    const int excl = running + sums[tid] - c;
    if (r < n_rows) {
      chunk_off[r] = excl;
      for (int j = 0; j < c; ++j) work[excl + j] = make_int2(r, j);
    }
    __syncthreads();
    if (tid == 1023) running += sums[1023];
    __syncthreads();
  }
  if (tid == 0) info[0] = running;
}

// Single block: row ranges of the prompt groups in a row list sorted by
// group (group of row r = traj[r] / m): grp_row0[i], grp_n[i], *n_groups.
__global__ void attn_groups_kernel(const int32_t* __restrict__ traj, int n_rows, int m,
                                   int32_t* __restrict__ grp_row0, int32_t* __restrict__ grp_n,
                                   int32_t* __restrict__ n_groups, int32_t* __restrict__ n_groups_out) {
  __shared__ int32_t sums[1024];
  __shared__ int32_t running;
  const int tid = threadIdx.x;
  if (tid == 0) running = 0;
  __syncthreads();
  for (int base = 0; base < n_rows; base += 1024) {
    const int r = base + tid;
    const int st = (r < n_rows && (r == 0 || traj[r] / m != traj[r - 1] / m)) ? 1 : 0;
    sums[tid] = st;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
      const int v = tid >= o ? sums[tid - o] : 0;
      __syncthreads();
      sums[tid] += v;
      __syncthreads();
    }
    if (st) grp_row0[running + sums[tid] - 1] = r;
    __syncthreads();
    if (tid == 1023) running += sums[1023];
    __syncthreads();
  }
  const int ng = running;
  for (int i = tid; i < ng; i += 1024) grp_n[i] = (i + 1 < ng ? grp_row0[i + 1] : n_rows) - grp_row0[i];
  if (tid == 0) {
    *n_groups = ng;
    if (n_groups_out) *n_groups_out = ng;
  }
}

struct AttnBf16Args {
  const bf16_t* q; const bf16_t* kpool; const bf16_t* vpool;
  const int32_t* page_table; int pt_stride; CtxSpec cs; int hq, hkv, chunk_pages;
  int n_rows;
  int uniform_nch;            // > 0: every row has this many chunks, no work list
  const int2* work; const int32_t* chunk_off; const int32_t* info;
  float* ws_o; float2* ws_ml; bf16_t* out;
  // shared-prefix partials of each (row, q head): pre_nch (o, max, sum) sets
  // that chunk 0 of the row starts from; pre_nch == 0 when there are none
  const float* pre_o; const float2* pre_ml; int pre_nch;
};

struct AttnPrefixArgs {
  const bf16_t* q; const bf16_t* kpool; const bf16_t* vpool;
  const int32_t* page_table; int pt_stride; CtxSpec cs; int hq, hkv;
  int prefix_pages;           // shared pages at the front of every member's page list
  int chunk_pages;            // prefix pages per wavefront
  int pre_nch;                // ceil(prefix_pages / chunk_pages)
  int qblocks;                // 16-query blocks per (group, kv head)
  const int32_t* grp_row0; const int32_t* grp_n; const int32_t* n_groups;
  float* pre_o; float2* pre_ml;
};

// K and V of one pair of pages (32 keys) for one kv head, in MFMA operand layout
template <int HD>
struct PagePair {
  bf16x8_t ka[HD / 32], kb[HD / 32], vv[HD / 16];
  bool hasb;
};

// Online-softmax state of one wavefront's 16 query vectors (the MFMA rows):
// lane (quad, col) holds, for query vector 4*quad+i, the running max m[i],
// its share l[i] of the denominator (summed over the 16 lanes at the end) and
// output dims nb*16+col in O[nb][i].
template <int HD>
struct AttnAcc {
  float m[4], l[4];
  f32x4_t O[HD / 16];
};

constexpr int kPst = 40;   // P row stride in LDS (bf16): 80 bytes

// Attend the wavefront's 16 query vectors (A operand qa) to the keys of pages
// [pbeg, pend) of page list pt (kv head kvh); keys at or after ctx are masked.
//   S[16 x 32]  = Q[16 x hd] . K^T      MFMA 16x16x32 bf16 per pair of pages
//   online softmax per query row (16-lane shuffles)
//   O[16 x hd] += P[16 x 32] . V[32 x hd]   MFMA 16x16x32 bf16, P via LDS
// K is read token-major straight into the MFMA B operand (16 B per lane, one
// contiguous 1 KB block of the page per 32-wide K step);
// V pages store 8 consecutive tokens of one dim contiguously, so the P.V
// B operand is also one 16 B load per lane.  Page ids of the next pair are
// fetched one iteration ahead so that the page-id -> key/value load chain is
// not serial.  With DB the loads of the next pair are issued before the
// current pair is computed (two pairs in flight; the 128-dim kernel then
// needs all 256 registers a wavefront may hold at two per SIMD): faster with
// many rows (5-8% from 64 live rows up), slower with few.
template <int HD, bool DB>
__device__ __forceinline__ void attn_page_loop(const bf16x8_t (&qa)[HD / 32], const bf16_t* kpool,
                                               const bf16_t* vpool, const CtxSpec& cs,
                                               const int32_t* pt, int pbeg, int pend, int ctx,
                                               int kvh, int hkv, bf16_t* P, AttnAcc<HD>& acc) {
  constexpr int NKK = HD / 32, NNB = HD / 16;
  const int lane = threadIdx.x & 63;
  const int quad = lane >> 4, col = lane & 15;
  const float scale = 1.0f / sqrtf((float)HD);
  auto load = [&](int p, PagePair<HD>& F, int ida, int idb) {
    const int pa = clamp_page(cs, ida);
    F.hasb = (p + 1) < pend;
    const int pb = F.hasb ? clamp_page(cs, idb) : pa;
    const bf16_t* kpa = kpool + k_off(pa, kvh, col, quad * 8, hkv, HD);
    const bf16_t* kpb = kpool + k_off(pb, kvh, col, quad * 8, hkv, HD);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      F.ka[kk] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(kpa + kk * kPage * 32));
      F.kb[kk] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(kpb + kk * kPage * 32));
    }
    const int vpage = quad < 2 ? pa : pb;
    const bf16_t* vb = vpool + v_off(vpage, kvh, (quad & 1) * 8, col, hkv, HD);
#pragma unroll
    for (int nb = 0; nb < NNB; ++nb)
      F.vv[nb] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(vb + nb * 16 * 8));
  };
  auto compute = [&](int p, const PagePair<HD>& F) {
    f32x4_t sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kk], F.ka[kk], sa, 0, 0, 0);
      sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kk], F.kb[kk], sb, 0, 0, 0);
    }
    // lane holds S[query 4*quad+i][key p*16+col] (sa) and [(p+1)*16+col] (sb)
    const bool va = p * kPage + col < ctx;
    const bool vb2 = F.hasb && ((p + 1) * kPage + col < ctx);
    float pva[4], pvb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float s1 = va ? sa[i] * scale : -INFINITY;
      const float s2 = vb2 ? sb[i] * scale : -INFINITY;
      float mx = fmaxf(s1, s2);
      mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 4, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 8, 64));
      const float mnew = fmaxf(acc.m[i], mx);
      const float alpha = __expf(acc.m[i] - mnew);
      // the denominator sums the same bf16-rounded weights that multiply V
      pva[i] = bf16_to_f32(f32_to_bf16(__expf(s1 - mnew)));
      pvb[i] = bf16_to_f32(f32_to_bf16(__expf(s2 - mnew)));
      acc.l[i] = acc.l[i] * alpha + pva[i] + pvb[i];
      acc.m[i] = mnew;
#pragma unroll
      for (int nb = 0; nb < NNB; ++nb) acc.O[nb][i] *= alpha;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      P[(4 * quad + i) * kPst + col] = f32_to_bf16(pva[i]);
      P[(4 * quad + i) * kPst + 16 + col] = f32_to_bf16(pvb[i]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const bf16x8_t pa8 = *(const bf16x8_t*)(&P[col * kPst + quad * 8]);
#pragma unroll
    for (int nb = 0; nb < NNB; ++nb)
      acc.O[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa8, F.vv[nb], acc.O[nb], 0, 0, 0);
    __builtin_amdgcn_wave_barrier();   // P is rewritten by the next pair
  };
  if constexpr (DB) {
    auto ids = [&](int p, int& a, int& b) {
      a = pt[p];
      b = p + 1 < pend ? pt[p + 1] : a;
    };
    if (pbeg >= pend) return;
    PagePair<HD> F0, F1;
    int ia, ib;
    ids(pbeg, ia, ib);
    load(pbeg, F0, ia, ib);
    if (pbeg + 2 < pend) ids(pbeg + 2, ia, ib);
    for (int p = pbeg; p < pend; p += 4) {
      if (p + 2 < pend) {
        load(p + 2, F1, ia, ib);
        if (p + 4 < pend) ids(p + 4, ia, ib);
      }
      compute(p, F0);
      if (p + 2 >= pend) break;
      if (p + 4 < pend) {
        load(p + 4, F0, ia, ib);
        if (p + 6 < pend) ids(p + 6, ia, ib);
      }
      compute(p + 2, F1);
    }
  } else {
    PagePair<HD> F;
    int nxa = pbeg < pend ? pt[pbeg] : 0;
    int nxb = pbeg + 1 < pend ? pt[pbeg + 1] : nxa;
    for (int p = pbeg; p < pend; p += 2) {
      const int ca = nxa, cb = nxb;
      if (p + 2 < pend) {
        nxa = pt[p + 2];
        nxb = p + 3 < pend ? pt[p + 3] : nxa;
      }
      load(p, F, ca, cb);
      compute(p, F);
    }
  }
}

// sum of a lane-partial over the 16 lanes of a query row
__device__ __forceinline__ float row16_sum(float l) {
  l += __shfl_xor(l, 1, 64);
  l += __shfl_xor(l, 2, 64);
  l += __shfl_xor(l, 4, 64);
  l += __shfl_xor(l, 8, 64);
  return l;
}

// Per-row decode attention.  Work unit = (row, kv head, chunk of C pages),
// one wavefront each, grid-stride loop; the G query heads sharing the kv head
// fill MFMA rows 0..G-1.  Rows of equal context (every decode step) map units
// arithmetically; ragged contexts use a work list built on the device.  A row
// whose keys span several chunks writes unnormalised partials (o, max, sum)
// and the combine kernel merges them.  With a shared prefix the row's keys
// start at cs.skip and chunk 0 starts from the prefix partials.
template <int HD, bool DB>
__device__ __forceinline__ void attn_bf16_body(const AttnBf16Args& A) {
  constexpr int NKK = HD / 32, NNB = HD / 16;
  __shared__ __attribute__((aligned(16))) bf16_t plds[4][16 * kPst];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int hq = A.hq, hkv = A.hkv;
  const int G = hq / hkv;
  const int quad = lane >> 4, col = lane & 15;
  const int total = (A.uniform_nch > 0 ? A.n_rows * A.uniform_nch : A.info[0]) * hkv;
  const int skip_pages = A.cs.skip / kPage;
  bf16_t* P = plds[w];
  for (int item = blockIdx.x * 4 + w; item < total; item += gridDim.x * 4) {
    const int wi = item / hkv, kvh = item - wi * hkv;
    int row, chunk, cid;
    if (A.uniform_nch > 0) {
      row = wi / A.uniform_nch; chunk = wi - row * A.uniform_nch; cid = wi;
    } else {
      const int2 rc = A.work[wi];
      row = rc.x; chunk = rc.y; cid = A.chunk_off[row] + chunk;
    }
    const int ctx = ctx_of(A.cs, row);
    const int32_t* pt = A.page_table + (int64_t)pt_row(A.cs, row) * A.pt_stride;
    const int npg = (ctx + kPage - 1) / kPage;
    const int nch = (npg - skip_pages + A.chunk_pages - 1) / A.chunk_pages;
    const int pbeg = skip_pages + chunk * A.chunk_pages;
    const int pend = min(pbeg + A.chunk_pages, npg);

    bf16x8_t qa[NKK];
    {
      const bool valid = col < G;
      const bf16_t* qrow = A.q + ((int64_t)row * hq + kvh * G + (valid ? col : 0)) * HD + quad * 8;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        u32x4_t v = valid ? *(const u32x4_t*)(qrow + 32 * kk) : (u32x4_t){0u, 0u, 0u, 0u};
        qa[kk] = __builtin_bit_cast(bf16x8_t, v);
      }
    }
    AttnAcc<HD> acc;
#pragma unroll
    for (int i = 0; i < 4; ++i) { acc.m[i] = -INFINITY; acc.l[i] = 0.f; }
#pragma unroll
    for (int nb = 0; nb < NNB; ++nb) acc.O[nb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    if (A.pre_nch > 0 && chunk == 0) {
      // start from the merged prefix partials of this row's heads
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h = 4 * quad + i;
        if (h >= G) continue;
        const int64_t base = ((int64_t)row * hq + kvh * G + h) * A.pre_nch;
        float M = -INFINITY;
        for (int c = 0; c < A.pre_nch; ++c) M = fmaxf(M, A.pre_ml[base + c].x);
        float L = 0.f;
        for (int c = 0; c < A.pre_nch; ++c) {
          const float2 ml = A.pre_ml[base + c];
          const float f = __expf(ml.x - M);
          L += ml.y * f;
#pragma unroll
          for (int nb = 0; nb < NNB; ++nb) acc.O[nb][i] += A.pre_o[(base + c) * HD + nb * 16 + col] * f;
        }
        acc.m[i] = M;
        acc.l[i] = col == 0 ? L : 0.f;
      }
    }
    attn_page_loop<HD, DB>(qa, A.kpool, A.vpool, A.cs, pt, pbeg, pend, ctx, kvh, hkv, P, acc);

    float lrow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) lrow[i] = row16_sum(acc.l[i]);
    if (nch == 1) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h = 4 * quad + i;
        if (h >= G) continue;
        const float inv = 1.0f / lrow[i];
        bf16_t* orow = A.out + ((int64_t)row * hq + kvh * G + h) * HD + col;
#pragma unroll
        for (int nb = 0; nb < NNB; ++nb) orow[nb * 16] = f32_to_bf16(acc.O[nb][i] * inv);
      }
      continue;
    }
    // several chunks: write this chunk's unnormalised partial; the combine
    // kernel merges the chunks of a row
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * quad + i;
      if (h >= G) continue;
      const int qh = kvh * G + h;
      float* po = A.ws_o + ((int64_t)cid * hq + qh) * HD + col;
#pragma unroll
      for (int nb = 0; nb < NNB; ++nb) po[nb * 16] = acc.O[nb][i];
      if (col == 0) A.ws_ml[(int64_t)cid * hq + qh] = make_float2(acc.m[i], lrow[i]);
    }
  }
}

// Entry points: one page pair in flight per wavefront (registers as the code
// needs them), or two (double-buffered), held to two wavefronts per SIMD,
// i.e. at most 256 registers.
template <int HD>
__global__ void __launch_bounds__(256) attn_bf16_kernel(AttnBf16Args A) {
  attn_bf16_body<HD, false>(A);
}
template <int HD>
__global__ void __launch_bounds__(256, 2) attn_bf16_db_kernel(AttnBf16Args A) {
  attn_bf16_body<HD, true>(A);
}

// Shared-prefix attention.  The members of a prompt group (consecutive rows
// of one group) share their first prefix_pages pages, so their query vectors
// (rows x G heads) are stacked 16 to a wavefront as the MFMA rows and attend
// to the prefix keys together: each prefix key and value is read once per
// 16 query vectors instead of once per G.  Work unit = (group, kv head,
// 16-query block, chunk of chunk_pages prefix pages); it writes the
// unnormalised partial (o, max, sum) of each of its query vectors.
template <int HD>
__global__ void __launch_bounds__(256) attn_prefix_kernel(AttnPrefixArgs A) {
  constexpr int NKK = HD / 32, NNB = HD / 16;
  __shared__ __attribute__((aligned(16))) bf16_t plds[4][16 * kPst];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int hq = A.hq, hkv = A.hkv;
  const int G = hq / hkv;
  const int quad = lane >> 4, col = lane & 15;
  const int total = A.n_groups[0] * hkv * A.qblocks * A.pre_nch;
  const int ctx = A.prefix_pages * kPage;
  bf16_t* P = plds[w];
  for (int item = blockIdx.x * 4 + w; item < total; item += gridDim.x * 4) {
    int t = item;
    const int pc = t % A.pre_nch; t /= A.pre_nch;
    const int qb = t % A.qblocks; t /= A.qblocks;
    const int kvh = t % hkv;
    const int gi = t / hkv;
    const int r0 = A.grp_row0[gi], ng = A.grp_n[gi];
    bf16x8_t qa[NKK];
    {
      const int qv = qb * 16 + col, rl = qv / G, h = qv - rl * G;
      const bool valid = rl < ng;
      const bf16_t* qrow = A.q + ((int64_t)(r0 + (valid ? rl : 0)) * hq + kvh * G + h) * HD + quad * 8;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        u32x4_t v = valid ? *(const u32x4_t*)(qrow + 32 * kk) : (u32x4_t){0u, 0u, 0u, 0u};
        qa[kk] = __builtin_bit_cast(bf16x8_t, v);
      }
    }
    const int32_t* pt = A.page_table + (int64_t)pt_row(A.cs, r0) * A.pt_stride;
    const int pbeg = pc * A.chunk_pages;
    const int pend = min(pbeg + A.chunk_pages, A.prefix_pages);
    AttnAcc<HD> acc;
#pragma unroll
    for (int i = 0; i < 4; ++i) { acc.m[i] = -INFINITY; acc.l[i] = 0.f; }
#pragma unroll
    for (int nb = 0; nb < NNB; ++nb) acc.O[nb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    attn_page_loop<HD, false>(qa, A.kpool, A.vpool, A.cs, pt, pbeg, pend, ctx, kvh, hkv, P, acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float l = row16_sum(acc.l[i]);
      const int qv = qb * 16 + 4 * quad + i, rl = qv / G, h = qv - rl * G;
      if (rl >= ng) continue;
      const int64_t idx = ((int64_t)(r0 + rl) * hq + kvh * G + h) * A.pre_nch + pc;
      float* po = A.pre_o + idx * HD + col;
#pragma unroll
      for (int nb = 0; nb < NNB; ++nb) po[nb * 16] = acc.O[nb][i];
      if (col == 0) A.pre_ml[idx] = make_float2(acc.m[i], l);
    }
  }
}

// fp32 attention (fp32 models): one wavefront per (row, q head, chunk).
template <int HD>
__global__ void __launch_bounds__(256) attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kpool, const float* __restrict__ vpool,
    const int32_t* __restrict__ page_table, int pt_stride, CtxSpec cs, int hq, int hkv,
    int chunk_pages, const int2* __restrict__ work, const int32_t* __restrict__ chunk_off,
    const int32_t* __restrict__ info, float* __restrict__ ws_o, float2* __restrict__ ws_ml,
    float* __restrict__ out) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = hq / hkv;
  const float scale = 1.0f / sqrtf((float)HD);
  const int total = info[0] * hq;
  for (int item = blockIdx.x * 4 + w; item < total; item += gridDim.x * 4) {
    const int wi = item / hq, qh = item - wi * hq, kvh = qh / G;
    const int2 rc = work[wi];
    const int row = rc.x, chunk = rc.y;
    const int ctx = ctx_of(cs, row);
    const int32_t* pt = page_table + (int64_t)pt_row(cs, row) * pt_stride;
    const int tbeg = chunk * chunk_pages * kPage;
    const int tend = min(tbeg + chunk_pages * kPage, ctx);
    const float* qv = q + ((int64_t)row * hq + qh) * HD;
    float qreg[HD];
#pragma unroll
    for (int d = 0; d < HD; ++d) qreg[d] = qv[d];
    float m = -INFINITY, l = 0.f, o[HD];
#pragma unroll
    for (int d = 0; d < HD; ++d) o[d] = 0.f;
    for (int j = tbeg + lane; j < tend; j += 64) {
      const int page = clamp_page(cs, pt[j / kPage]), slot = j % kPage;
      const float* kp = kpool + k_off(page, kvh, slot, 0, hkv, HD);
      float s = 0.f;
#pragma unroll
      for (int d = 0; d < HD; ++d) s = fmaf(qreg[d], kp[(d >> 5) * kPage * 32 + (d & 31)], s);
      s *= scale;
      const float mn = fmaxf(m, s);
      const float a = __expf(m - mn), pj = __expf(s - mn);
      l = l * a + pj;
#pragma unroll
      for (int d = 0; d < HD; ++d) o[d] = o[d] * a + pj * vpool[v_off(page, kvh, slot, d, hkv, HD)];
      m = mn;
    }
    const float mw = wave_max(m);
    const float a = (m == -INFINITY) ? 0.f : __expf(m - mw);
    const float lw = wave_sum(l * a);
    const int nch = ((ctx + kPage - 1) / kPage + chunk_pages - 1) / chunk_pages;
    const int cid = chunk_off[row] + chunk;
#pragma unroll
    for (int d = 0; d < HD; ++d) {
      const float v = wave_sum(o[d] * a);
      if ((d & 63) == lane) {
        if (nch == 1) out[((int64_t)row * hq + qh) * HD + d] = v / lw;
        else ws_o[((int64_t)cid * hq + qh) * HD + d] = v;
      }
    }
    if (nch > 1 && lane == 0) ws_ml[(int64_t)cid * hq + qh] = make_float2(mw, lw);
  }
}

// Merge chunk partials: one wavefront per (row, q head); rows with a single
// chunk were written directly by the attention kernel.  The chunk maxima and
// denominators are reduced across lanes (lane = chunk), then each lane
// accumulates its output dims over the chunks, taking each chunk's weight
// exp(m_c - M) from the lane that computed it.  The first batch of partial
// outputs and the lane's own chunk statistics are loaded together, before
// any reduction, so a row of up to kCB chunks costs one round trip to memory.
template <typename OUT>
__global__ void attn_combine_kernel(CtxSpec cs, int n_rows, int hq, int hd, int chunk_tokens,
                                    int uniform_nch, const int32_t* __restrict__ chunk_off,
                                    const float* __restrict__ ws_o, const float2* __restrict__ ws_ml,
                                    OUT* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= n_rows * hq) return;
  const int row = item / hq, qh = item % hq;
  const int nch = (span_of(cs, row) + chunk_tokens - 1) / chunk_tokens;
  if (nch <= 1) return;
  // equal contexts (no work list): row r's chunks are partial sets r*nch ..
  const int c0 = uniform_nch > 0 ? row * uniform_nch : chunk_off[row];
  const float2* ml = ws_ml + (int64_t)c0 * hq + qh;          // chunk c at ml[c * hq]
  const int nd = (hd + 63) / 64;                             // output dims per lane: lane + 64 t
  const float* ob = ws_o + ((int64_t)c0 * hq + qh) * hd + lane;   // chunk c at ob[c * hq * hd]
  const int64_t cstride = (int64_t)hq * hd;
  // batches of up to kCB chunks: every partial of the batch is loaded before
  // any is accumulated, so a lane keeps 2 * kCB loads in flight
  constexpr int kCB = 16;
  float o0[kCB], o1[kCB];
  auto load_batch = [&](int c) {
#pragma unroll
    for (int j = 0; j < kCB; ++j) {
      const float* o = ob + (int64_t)(c + j) * cstride;
      const bool ok = c + j < nch;
      o0[j] = (ok && lane < hd) ? o[0] : 0.f;
      o1[j] = (ok && nd > 1) ? o[64] : 0.f;
    }
  };
  load_batch(0);
  const float2 v0 = lane < nch ? ml[(int64_t)lane * hq] : make_float2(-INFINITY, 0.f);
  float M = v0.x;
  for (int c = lane + 64; c < nch; c += 64) M = fmaxf(M, ml[(int64_t)c * hq].x);
  M = wave_max(M);
  float L = lane < nch ? v0.y * __expf(v0.x - M) : 0.f;
  for (int c = lane + 64; c < nch; c += 64) {
    const float2 v = ml[(int64_t)c * hq];
    L += v.y * __expf(v.x - M);
  }
  L = wave_sum(L);
  const float invL = 1.0f / L;
  float acc[2] = {0.f, 0.f};
  for (int base = 0; base < nch; base += 64) {
    const int nb = min(64, nch - base);
    const float w = lane < nb ? __expf((base == 0 ? v0.x : ml[(int64_t)(base + lane) * hq].x) - M) : 0.f;
    for (int j0 = 0; j0 < nb; j0 += kCB) {
      if (base + j0 > 0) load_batch(base + j0);
#pragma unroll
      for (int j = 0; j < kCB; ++j) {
        const float wj = __shfl(w, (j0 + j) & 63, 64);
        acc[0] += wj * o0[j];
        acc[1] += wj * o1[j];
      }
    }
  }
  for (int t = 0; t < nd; ++t) {
    const int d = lane + 64 * t;
    if (d >= hd) break;
    const float v = acc[t] * invL;
    if constexpr (sizeof(OUT) == 2) out[((int64_t)row * hq + qh) * hd + d] = f32_to_bf16(v);
    else out[((int64_t)row * hq + qh) * hd + d] = v;
  }
}

// Resident wavefronts of the per-row bf16 kernel on MI355X: 256 CUs times its
// occupancy (a property of the compiled kernel).  Fixed CU count: the chunking,
// and with it the summation order, depends on the shapes only.
constexpr int kAttnMaxSlots = 256 * 16;
static int attn_slots(int hd) {
  static int cached[3] = {0, 0, 0};
  const int i = hd == 128 ? 0 : (hd == 64 ? 1 : 2);
  if (cached[i] == 0) {
    int nb = 0;
    hipError_t e = hd == 128 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_bf16_kernel<128>, 256, 0)
                 : hd == 64  ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_bf16_kernel<64>, 256, 0)
                             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, attn_bf16_kernel<32>, 256, 0);
    if (e != hipSuccess || nb < 1) nb = 2;
    cached[i] = std::min(256 * 4 * nb, kAttnMaxSlots);
  }
  return cached[i];
}

// Pages per chunk.  Ragged contexts: 128 pages (2048 keys), so that the
// longest rows are spread over many wavefronts instead of one while short rows
// stay whole (on the sweep's lognormal contexts, 32 / 64 / 128 / 256 pages
// took 1.85 / 1.76 / 1.72 / 1.82 ms: fewer chunks mean fewer partial sums and
// less per-item work, more mean better balance).  Equal contexts: the
// chunk count that minimises the kernel's makespan, rounds of resident
// wavefronts times pages per chunk (plus a page of fixed work per item), plus
// the partial-sum round trip and combine launch when rows are split; at most
// ~4 rounds of items and chunks of at least 4 pages.
constexpr int kRaggedChunkPages = 128;
// equal-context launches with at least this many rows keep two page pairs in
// flight per wavefront (measured on the Qwen3-8B-shaped rollout: 4-8% faster
// from 64 live rows up, 3-5% slower below)
constexpr int kAttnDbMinRows = 64;
static int choose_chunk_pages(int n_rows, int hkv, int max_ctx, bool uniform, int hd) {
  const int64_t units = (int64_t)n_rows * hkv;
  const int npg = (max_ctx + kPage - 1) / kPage;
  if (!uniform) return npg <= kRaggedChunkPages ? npg + (npg & 1) : kRaggedChunkPages;
  const int slots = attn_slots(hd);
  const int64_t nmax = std::max<int64_t>(1, (4 * (int64_t)slots + units - 1) / units);
  double best = 1e30;
  int best_c = npg;
  for (int64_t n = 1; n <= std::min<int64_t>(nmax, npg); ++n) {
    const int c = (int)((npg + n - 1) / n);
    const int64_t nch = (npg + c - 1) / c;
    if (nch != n) continue;                 // same split as a smaller n
    if (n > 1 && c < 4) break;              // chunks of at least 4 pages (64 keys)
    const double items = (double)units * nch;
    const double rounds = std::ceil(items / slots);
    double t = rounds * (c + 1.0);
    if (nch > 1) t += 0.5 * items / slots + 3.0;
    if (t < best) { best = t; best_c = c; }
  }
  return best_c;
}

constexpr int kPrefixChunkPages = 8;   // shared-prefix pages per wavefront (128 keys)

struct AttnWs {
  int32_t* chunk_off; int2* work; int32_t* info; float* ws_o; float2* ws_ml;
  int64_t max_chunks;          // partial sets the workspace holds
  float* pre_o; float2* pre_ml; int32_t* grp_row0; int32_t* grp_n; int32_t* n_groups;
};
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
// Workspace: [chunk_off | work list | info | partial o | partial (m, l)], then
// with a shared prefix [prefix partial o | prefix (m, l) | group row0 | group n | n_groups].
static size_t ws_layout(int n_rows, int hq, int hkv, int hd, int max_ctx, int prefix_pages, char* base,
                        AttnWs* w) {
  // partial sets for either chunking: ragged rows split into kRaggedChunkPages chunks;
  // equal contexts into at most max(1, ceil(4 * slots / units)) chunks per row
  // (choose_chunk_pages), i.e. at most n_rows + 4 * kAttnMaxSlots / hkv sets
  const int npg = (max_ctx + kPage - 1) / kPage;
  const int64_t ragged = (int64_t)n_rows * ((npg + kRaggedChunkPages - 1) / kRaggedChunkPages);
  const int64_t equal = (int64_t)n_rows + (4 * (int64_t)kAttnMaxSlots + hkv - 1) / hkv;
  const int64_t maxch = std::max(ragged, std::min<int64_t>(equal, (int64_t)n_rows * npg));
  (void)prefix_pages;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align256(off + bytes); return base ? base + o : nullptr; };
  char* a = take((size_t)n_rows * 4);
  char* b = take((size_t)maxch * sizeof(int2));
  char* c = take(64);
  char* d = take((size_t)maxch * hq * hd * sizeof(float));
  char* e = take((size_t)maxch * hq * sizeof(float2));
  char *f = nullptr, *g = nullptr, *h = nullptr, *i = nullptr, *j = nullptr;
  if (prefix_pages > 0) {
    const int64_t pn = (prefix_pages + kPrefixChunkPages - 1) / kPrefixChunkPages;
    f = take((size_t)n_rows * hq * pn * hd * sizeof(float));
    g = take((size_t)n_rows * hq * pn * sizeof(float2));
    h = take((size_t)n_rows * 4);
    i = take((size_t)n_rows * 4);
    j = take(64);
  }
  if (w) {
    w->chunk_off = (int32_t*)a; w->work = (int2*)b; w->info = (int32_t*)c;
    w->ws_o = (float*)d; w->ws_ml = (float2*)e; w->max_chunks = maxch;
    w->pre_o = (float*)f; w->pre_ml = (float2*)g; w->grp_row0 = (int32_t*)h; w->grp_n = (int32_t*)i;
    w->n_groups = (int32_t*)j;
  }
  return off;
}

size_t attn_workspace_bytes(int n_rows, int hq, int hkv, int hd, int max_ctx) {
  return ws_layout(n_rows, hq, hkv, hd, max_ctx, 0, nullptr, nullptr);
}
size_t attn_shared_workspace_bytes(int n_rows, int hq, int hkv, int hd, int ctx, int prefix_pages) {
  return ws_layout(n_rows, hq, hkv, hd, ctx, prefix_pages, nullptr, nullptr);
}

template <int HD>
static void attn_f32_go(dim3 grid, hipStream_t st, const void* q, const void* k, const void* v,
                        const int32_t* pt, int pts, CtxSpec cs, int hq, int hkv, int cp, AttnWs w,
                        void* out) {
  hipLaunchKernelGGL(attn_f32_kernel<HD>, grid, dim3(256), 0, st, (const float*)q,
                     (const float*)k, (const float*)v, pt, pts, cs, hq, hkv, cp, w.work,
                     w.chunk_off, w.info, w.ws_o, w.ws_ml, (float*)out);
}

// uniform: every row has the same context (cs.ctx_len == NULL, cs.mod == 0)
hipError_t launch_attention_spec(const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* page_table, int pt_stride, CtxSpec cs, int n_rows,
                                 int hq, int hkv, int hd, int max_ctx, bool bf16, void* out,
                                 void* ws, size_t ws_bytes, hipStream_t st, hipEvent_t ev0,
                                 hipEvent_t ev1) {
  if (n_rows <= 0) return hipSuccess;
  cs.max_ctx = max_ctx;
  cs.skip = 0;
  AttnWs w;
  const size_t need = ws_layout(n_rows, hq, hkv, hd, max_ctx, 0, (char*)ws, &w);
  if (ws == nullptr || ws_bytes < need) return hipErrorInvalidValue;
  const bool uniform = bf16 && cs.ctx_len == nullptr && cs.mod == 0;
  const int cp = choose_chunk_pages(n_rows, hkv, max_ctx, uniform, hd);
  const int uni_nch = uniform ? ((min(cs.base, max_ctx) + cp * kPage - 1) / (cp * kPage)) : 0;
  if (!uniform)
    hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(1024), 0, st, cs, n_rows, cp * kPage,
                       w.chunk_off, w.work, w.info);
  const int64_t maxch = uniform ? (int64_t)n_rows * uni_nch
                                : (int64_t)n_rows * ((max_ctx + cp * kPage - 1) / (cp * kPage));
  const int64_t items = maxch * (bf16 ? hkv : hq);
  int64_t blocks = (items + 3) / 4;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  const dim3 grid((unsigned)blocks);
  if (bf16) {
    AttnBf16Args a;
    a.q = (const bf16_t*)q; a.kpool = (const bf16_t*)k_pool; a.vpool = (const bf16_t*)v_pool;
    a.page_table = page_table; a.pt_stride = pt_stride; a.cs = cs; a.hq = hq; a.hkv = hkv;
    a.chunk_pages = cp; a.n_rows = n_rows; a.uniform_nch = uni_nch;
    a.work = w.work; a.chunk_off = w.chunk_off; a.info = w.info;
    a.ws_o = w.ws_o; a.ws_ml = w.ws_ml; a.out = (bf16_t*)out;
    a.pre_o = nullptr; a.pre_ml = nullptr; a.pre_nch = 0;
    if (ev0) (void)hipEventRecord(ev0, st);
    // two page pairs in flight for decode batches of 64 rows or more
    const bool db = uniform && n_rows >= kAttnDbMinRows;
    if (hd == 128) {
      if (db) hipLaunchKernelGGL(attn_bf16_db_kernel<128>, grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(256), 0, st, a);
    } else if (hd == 64) {
      if (db) hipLaunchKernelGGL(attn_bf16_db_kernel<64>, grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(256), 0, st, a);
    } else if (hd == 32) {
      if (db) hipLaunchKernelGGL(attn_bf16_db_kernel<32>, grid, dim3(256), 0, st, a);
      else hipLaunchKernelGGL(attn_bf16_kernel<32>, grid, dim3(256), 0, st, a);
    }
    else return hipErrorInvalidValue;
    if (ev1) (void)hipEventRecord(ev1, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((uniform ? uni_nch : (max_ctx + cp * kPage - 1) / (cp * kPage)) > 1) {
      const int64_t nb = ((int64_t)n_rows * hq + 3) / 4;
      hipLaunchKernelGGL(attn_combine_kernel<bf16_t>, dim3((unsigned)nb), dim3(256), 0, st, cs,
                         n_rows, hq, hd, cp * kPage, uni_nch, w.chunk_off, w.ws_o, w.ws_ml,
                         (bf16_t*)out);
      e = hipGetLastError();
    }
    return e;
  }
  if (hd == 128) attn_f32_go<128>(grid, st, q, k_pool, v_pool, page_table, pt_stride, cs, hq, hkv, cp, w, out);
  else if (hd == 64) attn_f32_go<64>(grid, st, q, k_pool, v_pool, page_table, pt_stride, cs, hq, hkv, cp, w, out);
  else if (hd == 32) attn_f32_go<32>(grid, st, q, k_pool, v_pool, page_table, pt_stride, cs, hq, hkv, cp, w, out);
  else return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((max_ctx + cp * kPage - 1) / (cp * kPage) > 1) {
    const int64_t nb = ((int64_t)n_rows * hq + 3) / 4;
    hipLaunchKernelGGL(attn_combine_kernel<float>, dim3((unsigned)nb), dim3(256), 0, st, cs,
                       n_rows, hq, hd, cp * kPage, 0, w.chunk_off, w.ws_o, w.ws_ml, (float*)out);
    e = hipGetLastError();
  }
  return e;
}

template <int HD>
static void attn_shared_go(dim3 gpre, dim3 grow, hipStream_t st, const AttnPrefixArgs& p,
                           const AttnBf16Args& a) {
  hipLaunchKernelGGL(attn_prefix_kernel<HD>, gpre, dim3(256), 0, st, p);
  hipLaunchKernelGGL(attn_bf16_kernel<HD>, grow, dim3(256), 0, st, a);
}

hipError_t launch_attention_shared(const void* q, const void* k_pool, const void* v_pool,
                                   int64_t n_pages, const int32_t* page_table, int pt_stride,
                                   const int32_t* row_traj, int pt_rows, int m, int prefix_pages,
                                   bool build_groups, int ctx, int n_rows, int hq, int hkv, int hd,
                                   void* out, void* ws, size_t ws_bytes, hipStream_t st,
                                   hipEvent_t ev0, hipEvent_t ev1, int32_t* n_groups_out) {
  if (n_rows <= 0) return hipSuccess;
  const int G = hq / hkv;
  if (prefix_pages < 1 || ctx <= prefix_pages * kPage || m < 1 || G < 1 || G > 16 || hq % hkv)
    return hipErrorInvalidValue;
  if (!(hd == 32 || hd == 64 || hd == 128)) return hipErrorInvalidValue;
  AttnWs w;
  const size_t need = ws_layout(n_rows, hq, hkv, hd, ctx, prefix_pages, (char*)ws, &w);
  if (ws == nullptr || ws_bytes < need) return hipErrorInvalidValue;
  CtxSpec cs;
  cs.ctx_len = nullptr; cs.mod = 0; cs.base = ctx; cs.row_pt = row_traj; cs.max_ctx = ctx;
  cs.n_pages = n_pages; cs.skip = prefix_pages * kPage; cs.pt_rows = pt_rows;
  if (build_groups)
    hipLaunchKernelGGL(attn_groups_kernel, dim3(1), dim3(1024), 0, st, row_traj, n_rows, m, w.grp_row0,
                       w.grp_n, w.n_groups, n_groups_out);
  AttnPrefixArgs p;
  p.q = (const bf16_t*)q; p.kpool = (const bf16_t*)k_pool; p.vpool = (const bf16_t*)v_pool;
  p.page_table = page_table; p.pt_stride = pt_stride; p.cs = cs; p.hq = hq; p.hkv = hkv;
  p.prefix_pages = prefix_pages; p.chunk_pages = kPrefixChunkPages;
  p.pre_nch = (prefix_pages + kPrefixChunkPages - 1) / kPrefixChunkPages;
  p.qblocks = (m * G + 15) / 16;
  p.grp_row0 = w.grp_row0; p.grp_n = w.grp_n; p.n_groups = w.n_groups;
  p.pre_o = w.pre_o; p.pre_ml = w.pre_ml;
  // at most n_rows groups
  int64_t pre_items = (int64_t)std::min(n_rows, (n_rows + m - 1) / m + n_rows) * hkv * p.qblocks * p.pre_nch;
  int64_t gpre = std::min<int64_t>(std::max<int64_t>((pre_items + 3) / 4, 1), 2048);
  // per-row kernel over the keys after the prefix
  const int span = ctx - cs.skip;
  const int cp = choose_chunk_pages(n_rows, hkv, span, true, hd);
  const int nch = (span + cp * kPage - 1) / (cp * kPage);
  if ((int64_t)n_rows * nch > w.max_chunks) return hipErrorInvalidValue;
  AttnBf16Args a;
  a.q = (const bf16_t*)q; a.kpool = (const bf16_t*)k_pool; a.vpool = (const bf16_t*)v_pool;
  a.page_table = page_table; a.pt_stride = pt_stride; a.cs = cs; a.hq = hq; a.hkv = hkv;
  a.chunk_pages = cp; a.n_rows = n_rows; a.uniform_nch = nch;
  a.work = w.work; a.chunk_off = w.chunk_off; a.info = w.info;
  a.ws_o = w.ws_o; a.ws_ml = w.ws_ml; a.out = (bf16_t*)out;
  a.pre_o = w.pre_o; a.pre_ml = w.pre_ml; a.pre_nch = p.pre_nch;
  const int64_t items = (int64_t)n_rows * nch * hkv;
  const int64_t grow = std::min<int64_t>(std::max<int64_t>((items + 3) / 4, 1), 2048);
  if (ev0) (void)hipEventRecord(ev0, st);
  if (hd == 128) attn_shared_go<128>(dim3((unsigned)gpre), dim3((unsigned)grow), st, p, a);
  else if (hd == 64) attn_shared_go<64>(dim3((unsigned)gpre), dim3((unsigned)grow), st, p, a);
  else attn_shared_go<32>(dim3((unsigned)gpre), dim3((unsigned)grow), st, p, a);
  if (ev1) (void)hipEventRecord(ev1, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (nch > 1) {
    const int64_t nb = ((int64_t)n_rows * hq + 3) / 4;
    hipLaunchKernelGGL(attn_combine_kernel<bf16_t>, dim3((unsigned)nb), dim3(256), 0, st, cs,
                       n_rows, hq, hd, cp * kPage, nch, w.chunk_off, w.ws_o, w.ws_ml, (bf16_t*)out);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_attention(const void* q, const void* k_pool, const void* v_pool,
                            int64_t n_pages, const int32_t* page_table, int pt_stride,
                            const int32_t* row_pt, const int32_t* ctx_len, int ctx_mod,
                            int ctx_base, int n_rows, int hq, int hkv, int hd, int max_ctx,
                            bool bf16, void* out, void* ws, size_t ws_bytes, hipStream_t st,
                            hipEvent_t ev0, hipEvent_t ev1) {
  CtxSpec cs;
  cs.ctx_len = ctx_len; cs.mod = ctx_mod; cs.base = ctx_base; cs.row_pt = row_pt;
  cs.max_ctx = max_ctx; cs.n_pages = n_pages; cs.skip = 0; cs.pt_rows = 0;
  return launch_attention_spec(q, k_pool, v_pool, page_table, pt_stride, cs, n_rows, hq, hkv, hd,
                               max_ctx, bf16, out, ws, ws_bytes, st, ev0, ev1);
}

}  // namespace darts
