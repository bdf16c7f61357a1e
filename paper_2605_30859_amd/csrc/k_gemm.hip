// Dense GEMMs of the decoder: C[M,N] (op)= A[M,K] * W[N,K]^T.
// bf16 operands on gfx950 MFMA (v_mfma_f32_16x16x32_bf16), fp32 accumulate.
// Epilogues: store fp32, store bf16, add into an fp32 residual, SwiGLU
// (W rows interleaved in groups of 16: 16 gate rows then the 16 matching up
// rows; output silu(gate) * up as bf16).
//
// Two kernel families, chosen per launch from (M, N, K):
//  * tiled: BM x BN block tile whose A and W slices are copied global -> LDS
//    by direct loads (no register staging) through a ring of 2-4 LDS stages;
//    4 or 8 wavefronts each own a WM x WN register tile.  Blocks are
//    renumbered so that the blocks an XCD runs are neighbours in (m, n) and
//    share operand tiles in that XCD's L2.  Configs: 128x128 with 2 stages
//    (64 KB, two blocks per CU: one block's barrier wait is covered by the
//    other), 128x128 with 4 stages (one block per CU, deepest prefetch: for
//    weight streaming over very wide N), 256x128, 256x192 and 256x256 with 8
//    wavefronts (half the operand bytes per flop: large M), and 64- or
//    128-row tiles 64 or 96 wide with 4 stages for small batches, where they
//    give exactly one block per CU.
//  * skinny (M <= 32 with small W): no LDS for operands; each wavefront loads
//    W and A fragments straight into MFMA operand registers, 8 wavefronts of a
//    block split K and are reduced through LDS.
// Either family may split K across blocks; partial sums then go to a
// workspace and a reduce kernel adds them in a fixed order (bitwise
// deterministic).  The plan is a pure function of (M, N, K), so results do
// not depend on the device or on earlier calls.
//
// Grouped GEMMs (mixture of experts) run the tiled kernel over a device-built
// list of expert row tiles, or, for the gate/up projection in decode batches,
// a kernel that streams strip-packed weights straight into MFMA registers
// (see the strip layout below); a plan per launch (grouped_plan) picks the
// row tile and the kernel from the routed pairs per expert.
#include <algorithm>
#include <cmath>

#include "common.h"
#include "kernels.h"

namespace darts {


__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

template <int EPI>
__device__ __forceinline__ void epi_store(void* C, int ldc, int M, int m, int n, float v) {
  if (m >= M) return;
  if (EPI == EPI_F32) ((float*)C)[(int64_t)m * ldc + n] = v;
  else if (EPI == EPI_BF16) ((bf16_t*)C)[(int64_t)m * ldc + n] = f32_to_bf16(v);
  else if (EPI == EPI_ADD_F32) ((float*)C)[(int64_t)m * ldc + n] += v;
}

// Write a 16x16 MFMA output tile pair / single tile.  acc layout: lane holds
// rows r0 + 4*(lane/16) + i, column c0 + lane%16.
template <int EPI>
__device__ __forceinline__ void store_tile(void* C, int ldc, int M, int r0, int c0, int lane,
                                           const f32x4_t& v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) epi_store<EPI>(C, ldc, M, r0 + 4 * (lane >> 4) + i, c0 + (lane & 15), v[i]);
}
// gate tile (physical cols 32g..32g+15) and up tile (32g+16..32g+31) -> H cols 16g..16g+15
__device__ __forceinline__ void store_swiglu(bf16_t* H, int ldc, int M, int r0, int pc0, int lane,
                                             const f32x4_t& g, const f32x4_t& u) {
  const int col = (pc0 >> 5) * 16 + (lane & 15);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = r0 + 4 * (lane >> 4) + i;
    if (m < M) H[(int64_t)m * ldc + col] = f32_to_bf16(silu_f(g[i]) * u[i]);
  }
}
__device__ __forceinline__ void store_partial(float* P, int M, int N, int r0, int c0, int lane,
                                              const f32x4_t& v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = r0 + 4 * (lane >> 4) + i;
    if (m < M) P[(int64_t)m * N + c0 + (lane & 15)] = v[i];
  }
}

// ------------------------------------------------------------ strip layout
// Strip-packed weights: a [N][K] matrix (N % 16 == 0, K % 32 == 0) is stored
// as N/16 strips of 16 consecutive rows; strip g holds K/32 blocks of 64 x 8
// bf16, and lane l of block s holds W[16g + l%16][32s + 8(l/16), +8), the B
// operand of v_mfma_f32_16x16x32_bf16 for that strip and K step.  A strip
// occupies the same 16*K elements as in the row-major layout, only reordered.
// Element offset of the 8-element chunk W[n][k, k+8), k % 8 == 0:
__device__ __forceinline__ int64_t strip_off(int n, int k, int K) {
  return (((int64_t)(n >> 4) * (K >> 5) + (k >> 5)) * 64 + (n & 15) + 16 * ((k >> 3) & 3)) * 8;
}

// In-place repack of a row-major [16 * gridDim.x][K] bf16 matrix into the
// strip layout: one block per strip, staged through 16*K*2 bytes of LDS.
__global__ void __launch_bounds__(256) pack_strips_kernel(bf16_t* __restrict__ W, int K) {
  extern __shared__ __attribute__((aligned(16))) bf16_t strip[];
  bf16_t* base = W + (int64_t)blockIdx.x * 16 * K;
  const int nch = 2 * K;                     // 16-byte chunks per strip
  for (int c = threadIdx.x; c < nch; c += blockDim.x)
    *(u32x4_t*)(strip + c * 8) = *(const u32x4_t*)(base + (int64_t)c * 8);
  __syncthreads();
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    const int s = c >> 6, l = c & 63;        // block s, lane l: row l%16, K 32s + 8(l/16)
    *(u32x4_t*)(base + (int64_t)c * 8) = *(const u32x4_t*)(strip + (l & 15) * K + 32 * s + 8 * (l >> 4));
  }
}

// ------------------------------------------------------------------ tiled
// Operand tiles travel global -> LDS with direct 16-byte LDS loads (no
// staging registers) through a STAGES-deep ring of LDS buffers.  A KB-wide K
// slice of a row is KB/8 chunks of 16 bytes, stored in a swizzled chunk order
// (dma_swz) so that the 16-byte fragment reads of consecutive rows hit
// distinct banks.  Rows of A past M load row M-1 (their results are never
// stored).  Each wavefront owns a (BM/WGM) x (BN/WGN) register tile of
// 16x16 MFMA accumulators.
// s_waitcnt vmcnt(N) (gfx9 encoding: vmcnt bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their "don't wait" maxima)
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Cache-policy operand of the direct LDS loads that marks them non-temporal
// (the nt bit of gfx950's global loads).  A streaming read of 8 GiB measured
// 7.0 TB/s with non-temporal 16-byte loads against 6.3 TB/s with plain ones;
// the weight streams of the MoE expert GEMMs gain 4-13% from it wherever each
// weight tile is read once per launch.
constexpr int kNtLoad = 2;

// LDS chunk swizzle for a tile row of KB bf16 (KB/8 chunks of 16 bytes): the
// chunk order of row r is permuted so that the 8 rows a 16-byte fragment read
// touches in one LDS pass land in distinct banks.
template <int KB>
__device__ __forceinline__ int dma_swz(int r) {
  if constexpr (KB == 64) return r & 7;
  else return (r >> 1) & 3;
}

// One BM x BN output tile (rows m0.., cols n0.., K range [z*k_chunk, +k_chunk)).
// arow != NULL: row r of the tile's A operand is row arow[r] of A (a gather).
// PW: W is strip-packed (pack_strips_kernel; ldw = K): the same LDS tile is
// filled from the packed addresses, so results are bitwise those of the
// row-major layout.  WAUX: cache policy of the W loads (kNtLoad: non-temporal,
// for weights a launch reads once).
template <int BM, int BN, int KB, int WGM, int WGN, int STAGES, int EPI, bool SPLIT, bool PW = false,
          int WAUX = 0>
__device__ __forceinline__ void dma_gemm_tile(const bf16_t* __restrict__ A, int lda,
                                              const bf16_t* __restrict__ W, int ldw,
                                              void* __restrict__ C, int ldc, int M, int N,
                                              int k_chunk, int mi, int ni, int z,
                                              float* __restrict__ ws,
                                              const int32_t* __restrict__ arow = nullptr) {
  static_assert(KB == 32 || KB == 64, "K tile");
  constexpr int NW = WGM * WGN;                    // wavefronts per block
  constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 16, TN = WN / 16;
  constexpr int CH = KB / 8, RPI = 64 / CH;        // chunks per row, rows per 1 KB load instruction
  constexpr int AI = BM / (RPI * NW), WI = BN / (RPI * NW);   // load instructions per wave per stage
  static_assert(AI * RPI * NW == BM && WI * RPI * NW == BN, "tile rows must split over the waves");
  constexpr int KH = KB / 32;                      // 32-wide MFMA K steps per tile
  constexpr int STAGE_ELEMS = (BM + BN) * KB;      // bf16 elements per stage
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int m0 = mi * BM, n0 = ni * BN;
  const int kbeg = z * k_chunk;
  const int nk = k_chunk / KB;

  // per-lane global source rows for this wave's load instructions: lane i fills
  // LDS bytes [16i, 16i+16) of the instruction's RPI rows, which hold source
  // chunk (i % CH) ^ swizzle(row)
  const int lrow = lane / CH;
  const int gchunk = (lane % CH) ^ dma_swz<KB>(lrow);
  const bf16_t* asrc[AI];
  const bf16_t* wsrc[WI];
#pragma unroll
  for (int j = 0; j < AI; ++j) {
    int r = m0 + wave * (BM / NW) + RPI * j + lrow;
    r = r < M ? r : M - 1;
    if (arow) r = arow[r];
    asrc[j] = A + (int64_t)r * lda + kbeg + gchunk * 8;
  }
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int n = n0 + wave * (BN / NW) + RPI * j + lrow;
    if constexpr (PW) wsrc[j] = W + strip_off(n, kbeg + gchunk * 8, ldw);
    else wsrc[j] = W + (int64_t)n * ldw + kbeg + gchunk * 8;
  }
  // one KB-wide K step moves a row-major source KB elements on, a packed one
  // KB/32 blocks of 512 elements
  constexpr int WSTEP = PW ? KB * 16 : KB;

  auto issue = [&](int kt, int buf) {
    bf16_t* sa = smem + buf * STAGE_ELEMS;
    bf16_t* sw = sa + BM * KB;
#pragma unroll
    for (int j = 0; j < AI; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[j] + kt * KB),
                                       (lds_void_t*)(sa + (wave * (BM / NW) + RPI * j) * KB), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < WI; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(wsrc[j] + kt * WSTEP),
                                       (lds_void_t*)(sw + (wave * (BN / NW) + RPI * j) * KB), 16, 0, WAUX);
  };

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s, s);

  const int fr = lane & 15, fq = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    // this wave's loads of stage kt are done once at most the (STAGES-2) later
    // stages' loads are outstanding (all outstanding in the last stages); the
    // raw barrier then publishes every wave's stage kt (no memory fence: it
    // would drain the prefetches still in flight)
    if (kt + STAGES - 2 < nk) vm_wait<(STAGES - 2) * (AI + WI)>();
    else vm_wait<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    const bf16_t* sa = smem + (kt % STAGES) * STAGE_ELEMS;
    const bf16_t* sw = sa + BM * KB;
    // fragments of every 32-wide K step are read before the first MFMA, so
    // LDS latency overlaps matrix work
    bf16x8_t a[KH][TM], bb[KH][TN];
#pragma unroll
    for (int ks = 0; ks < KH; ++ks) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WM + 16 * i + fr;
        a[ks][i] = *(const bf16x8_t*)(sa + r * KB + (((ks * 4 + fq) ^ dma_swz<KB>(r)) * 8));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WN + 16 * j + fr;
        bb[ks][j] = *(const bf16x8_t*)(sw + r * KB + (((ks * 4 + fq) ^ dma_swz<KB>(r)) * 8));
      }
    }
#pragma unroll
    for (int ks = 0; ks < KH; ++ks)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][i], bb[ks][j], acc[i][j], 0, 0, 0);
  }

  const int rb = m0 + wm * WM, cb = n0 + wn * WN;
  if constexpr (SPLIT) {
    float* P = ws + (int64_t)z * M * N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) store_partial(P, M, N, rb + 16 * i, cb + 16 * j, lane, acc[i][j]);
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; j += 2)
        store_swiglu((bf16_t*)C, ldc, M, rb + 16 * i, cb + 16 * j, lane, acc[i][j], acc[i][j + 1]);
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) store_tile<EPI>(C, ldc, M, rb + 16 * i, cb + 16 * j, lane, acc[i][j]);
  }
}

// Blocks are renumbered so that the blocks one XCD runs (dispatch is round
// robin over the 8 XCDs) are consecutive tiles and share operands in its L2.
__device__ __forceinline__ int xcd_block() {
  const int nb = gridDim.x;
  int b = blockIdx.x;
  const int full = (nb / 8) * 8;
  if (b < full) b = (b % 8) * (full / 8) + b / 8;
  return b;
}

template <int BM, int BN, int KB, int WGM, int WGN, int STAGES, int EPI, bool SPLIT>
__global__ void __launch_bounds__(64 * WGM * WGN) gemm_dma_kernel(const bf16_t* __restrict__ A, int lda,
                                                       const bf16_t* __restrict__ W, int ldw,
                                                       void* __restrict__ C, int ldc, int M,
                                                       int N, int /*K*/, int k_chunk, int mt, int nt,
                                                       float* __restrict__ ws) {
  const int b = xcd_block();
  const int mi = b % mt, ni = (b / mt) % nt, z = b / (mt * nt);
  dma_gemm_tile<BM, BN, KB, WGM, WGN, STAGES, EPI, SPLIT>(A, lda, W, ldw, C, ldc, M, N, k_chunk, mi,
                                                          ni, z, ws);
}

// Grouped GEMM (mixture-of-experts): group e owns rows [off[e], off[e] +
// cnt[e]) of C (and of A, or of the gather list arow into A) and the weight
// matrix W + e * w_stride ([N][K]).  The
// non-empty row tiles are listed on the device (mtiles[i] = e << 16 | m tile,
// *n_mtiles of them); persistent blocks take items (row tile, n tile), n tile
// fastest, in a grid-stride loop.  PW: W strip-packed; WAUX: W cache policy.
template <int BM, int BN, int KB, int WGM, int WGN, int STAGES, int EPI, bool PW, int WAUX>
__global__ void __launch_bounds__(64 * WGM * WGN) gemm_dma_grouped_kernel(
    const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ W, int64_t w_stride, int ldw,
    void* __restrict__ C, int ldc, int N, int K, const int32_t* __restrict__ g_off,
    const int32_t* __restrict__ g_cnt, const int32_t* __restrict__ mtiles,
    const int32_t* __restrict__ n_mtiles, int nt, const int32_t* __restrict__ arow) {
  const int total = n_mtiles[0] * nt;
  constexpr int esz = (EPI == EPI_F32 || EPI == EPI_ADD_F32) ? 4 : 2;
  // Items are (row tile, column tile) in row-tile order.  With gathered A
  // rows, each XCD takes one contiguous eighth of the items (blocks are dealt
  // to the 8 XCDs round robin, block b on XCD b % 8), so the column tiles of
  // one expert row tile run on one XCD and find its gathered input rows in
  // that XCD's L2; the grid is a multiple of 8 blocks and the eighths
  // partition [0, total).  Otherwise items go to blocks round robin (the
  // down projection measured no gain from the XCD split).
  const bool by_xcd = arow != nullptr;
  const int chunk = (total + 7) >> 3;
  const int lo = by_xcd ? (int)(blockIdx.x & 7) * chunk : 0;
  const int hi = by_xcd ? min(total, lo + chunk) : total;
  const int step = by_xcd ? (int)(gridDim.x >> 3) : (int)gridDim.x;
  for (int it = by_xcd ? lo + (int)(blockIdx.x >> 3) : (int)blockIdx.x; it < hi; it += step) {
    const int mt = mtiles[it / nt], ni = it % nt;
    const int e = mt >> 16, mi = mt & 0xffff;
    const int cnt = g_cnt[e];
    const int64_t off = g_off[e];
    // other waves may still read the previous item's last LDS stage: a raw
    // barrier (their LDS reads have retired once their MFMAs issued); no
    // memory fence, which would also wait for the previous item's stores
    __builtin_amdgcn_s_barrier();
    void* Ce = (char*)C + off * ldc * esz;
    // with arow, A rows are gathered: segment row r is A row arow[off + r]
    dma_gemm_tile<BM, BN, KB, WGM, WGN, STAGES, EPI, false, PW, WAUX>(arow ? A : A + off * lda, lda,
                                                            W + (int64_t)e * w_stride, ldw, Ce, ldc,
                                                            cnt, N, K, mi, ni, 0, nullptr,
                                                            arow ? arow + off : nullptr);
  }
}

// ------------------------------------------- grouped, weights into registers
// Grouped GEMM for decode batches with strip-packed W (the MoE gate/up
// projection).  Block = 4 wavefronts over an item (expert row tile of BM
// rows, slab of 4 x CPW columns); wavefront w owns CPW columns and loads
// their W blocks (one 1 KB block per 16-column strip and 32-wide K step)
// straight from memory into MFMA B-operand registers, P K steps of 64
// ahead (non-temporal loads: each block is read once), so W never passes
// through LDS.  The BM x 64 A tiles of the
// expert's rows (gathered through arow when given; rows past the expert's
// count repeat its last row) go through a P-stage LDS ring shared by the
// four wavefronts, filled by direct 16-byte LDS loads in the swizzled layout
// of the tiled kernel.  Per output tile the MFMAs run over K in order, as in
// the tiled kernel, so results are bitwise those of the tiled kernel.
// Items are dealt XCD by XCD as in the tiled grouped kernel.
template <int BM, int CPW, int P, int EPI>
__global__ void __launch_bounds__(256, 2) gemm_wd_grouped_kernel(
    const bf16_t* __restrict__ A, int lda, const bf16_t* Wp, int64_t w_stride,
    void* __restrict__ C, int ldc, int N, int K, const int32_t* __restrict__ g_off,
    const int32_t* __restrict__ g_cnt, const int32_t* __restrict__ mtiles,
    const int32_t* __restrict__ n_mtiles, const int32_t* __restrict__ arow) {
  constexpr int NW = 4, KB = 64, CH = KB / 8, RPI = 64 / CH;
  constexpr int AI = BM / (RPI * NW);                 // A load instructions per wave per stage
  static_assert(AI * RPI * NW == BM, "A tile rows must split over the waves");
  static_assert(CPW % 32 == 0 || EPI != EPI_SWIGLU, "SwiGLU pairs gate and up strips");
  constexpr int TM = BM / 16, TN = CPW / 16;
  constexpr int WL = 2 * TN;                          // W loads per wave per 64-wide K step
  constexpr int STAGE = BM * KB;
  constexpr int SLAB = NW * CPW;
  constexpr int esz = (EPI == EPI_F32 || EPI == EPI_ADD_F32) ? 4 : 2;
  __shared__ __attribute__((aligned(16))) bf16_t sA[P * STAGE];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nt = N / SLAB;
  const int total = n_mtiles[0] * nt;
  const int nk = K / KB;                              // a multiple of P
  const int k32 = K >> 5;
  const int chunk = (total + 7) >> 3;
  const int lo = (int)(blockIdx.x & 7) * chunk;
  const int hi = min(total, lo + chunk);
  const int step = (int)(gridDim.x >> 3);
  const int lrow = lane / CH;
  const int gchunk = (lane % CH) ^ dma_swz<KB>(lrow);
  const int fr = lane & 15, fq = lane >> 4;
  for (int it = lo + (int)(blockIdx.x >> 3); it < hi; it += step) {
    const int mt = mtiles[it / nt], ni = it % nt;
    const int e = mt >> 16, mi = mt & 0xffff;
    const int cnt = g_cnt[e];
    const int64_t off = g_off[e];
    // the previous item's last LDS stage may still be read by other waves
    __builtin_amdgcn_s_barrier();
    const bf16_t* asrc[AI];
#pragma unroll
    for (int j = 0; j < AI; ++j) {
      int r = mi * BM + wave * (BM / NW) + RPI * j + lrow;
      r = r < cnt ? r : cnt - 1;
      const int64_t row = arow ? (int64_t)arow[off + r] : off + r;
      asrc[j] = A + row * lda + gchunk * 8;
    }
    // this wave's first strip; block (strip g0 + j, K step q) at (j*k32 + q)*512
    const int g0 = (ni * SLAB + wave * CPW) >> 4;
    const bf16_t* wsrc = Wp + (int64_t)e * w_stride + (int64_t)g0 * k32 * 512 + lane * 8;
    f32x4_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    bf16x8_t wr[P][2][TN];   // register ring: slot u holds K step k0 + u
#define DARTS_WD_ISSUE(KT, SLOT)                                                                  \
    {                                                                                            \
      bf16_t* sa_ = sA + (SLOT) * STAGE;                                                         \
      _Pragma("unroll") for (int j = 0; j < AI; ++j)                                             \
        __builtin_amdgcn_global_load_lds((const void*)(asrc[j] + (KT) * KB),                    \
                                         (lds_void_t*)(sa_ + (wave * (BM / NW) + RPI * j) * KB), \
                                         16, 0, 0);                                              \
      _Pragma("unroll") for (int h = 0; h < 2; ++h)                                              \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                           \
          wr[SLOT][h][j] = __builtin_bit_cast(                                                  \
              bf16x8_t, __builtin_nontemporal_load(                                              \
                            (const u32x4_t*)(wsrc + ((int64_t)j * k32 + 2 * (KT) + h) * 512)));  \
    }
#pragma unroll
    for (int u = 0; u < P - 1; ++u)
      if (u < nk) DARTS_WD_ISSUE(u, u)
    for (int k0 = 0; k0 < nk; k0 += P) {
#pragma unroll
      for (int u = 0; u < P; ++u) {
        const int kt = k0 + u;
        // K step kt's A and W loads are done once at most the loads of the
        // (P - 2) later steps are outstanding (whatever the order of the A
        // and W loads inside a step); the raw barrier then publishes every
        // wave's A stage kt, and the scheduling barrier keeps the next
        // step's loads from moving above it
        if (kt + P - 2 < nk) vm_wait<(P - 2) * (AI + WL)>();
        else vm_wait<0>();
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        const int kn = kt + P - 1;
        if (kn < nk) DARTS_WD_ISSUE(kn, (u + P - 1) % P)
        const bf16_t* sa = sA + u * STAGE;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          bf16x8_t a[TM];
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = 16 * i + fr;
            a[i] = *(const bf16x8_t*)(sa + r * KB + (((h * 4 + fq) ^ dma_swz<KB>(r)) * 8));
          }
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], wr[u][h][j], acc[i][j], 0, 0, 0);
        }
      }
    }
#undef DARTS_WD_ISSUE
    void* Ce = (char*)C + off * ldc * esz;
    const int r0 = mi * BM, c0 = ni * SLAB + wave * CPW;
    if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; j += 2)
          store_swiglu((bf16_t*)Ce, ldc, cnt, r0 + 16 * i, c0 + 16 * j, lane, acc[i][j], acc[i][j + 1]);
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) store_tile<EPI>(Ce, ldc, cnt, r0 + 16 * i, c0 + 16 * j, lane, acc[i][j]);
    }
  }
}

// ----------------------------------------------------------------- skinny
// Block: 8 wavefronts, NS*16 output columns, all M <= 16*MT rows.  Wavefront
// w handles K range [kbeg + w*kw, kbeg + (w+1)*kw).
template <int MT, int NS, int EPI, bool SPLIT>
__global__ void __launch_bounds__(512) gemm_skinny_kernel(const bf16_t* __restrict__ A, int lda,
                                                          const bf16_t* __restrict__ W, int ldw,
                                                          void* __restrict__ C, int ldc, int M,
                                                          int N, int /*K*/, int k_chunk, int nt,
                                                          float* __restrict__ ws) {
  __shared__ f32x4_t red[8][MT * NS][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ni = blockIdx.x % nt, z = blockIdx.x / nt;
  const int n0 = ni * NS * 16;
  const int kw = k_chunk / 8;
  const int kbeg = z * k_chunk + wave * kw;
  const int kq = (lane >> 4) * 8, r = lane & 15;
  f32x4_t acc[MT][NS];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  const bf16_t* wp[NS];
#pragma unroll
  for (int j = 0; j < NS; ++j) wp[j] = W + (int64_t)(n0 + 16 * j + r) * ldw + kbeg + kq;
  const bf16_t* ap[MT];
  bool av[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    av[i] = (16 * i + r) < M;
    ap[i] = A + (int64_t)(av[i] ? 16 * i + r : 0) * lda + kbeg + kq;
  }
  for (int k = 0; k < kw; k += 32) {
    bf16x8_t a[MT], b[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) b[j] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(wp[j] + k));
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      u32x4_t v = *(const u32x4_t*)(ap[i] + k);
      if (!av[i]) v = (u32x4_t){0u, 0u, 0u, 0u};
      a[i] = __builtin_bit_cast(bf16x8_t, v);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NS; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NS; ++j) red[wave][i * NS + j][lane] = acc[i][j];
  __syncthreads();
  // wave t sums tile t (in wave order 0..7) and stores it
  for (int t = wave; t < MT * NS; t += 8) {
    f32x4_t s = red[0][t][lane];
#pragma unroll
    for (int w = 1; w < 8; ++w) s += red[w][t][lane];
    red[0][t][lane] = s;
  }
  __syncthreads();
  if constexpr (SPLIT) {
    float* P = ws + (int64_t)z * M * N;
    for (int t = wave; t < MT * NS; t += 8)
      store_partial(P, M, N, 16 * (t / NS), n0 + 16 * (t % NS), lane, red[0][t][lane]);
  } else if constexpr (EPI == EPI_SWIGLU) {
    for (int t = wave; t < MT * NS / 2; t += 8) {
      const int i = t / (NS / 2), jp = t % (NS / 2);
      store_swiglu((bf16_t*)C, ldc, M, 16 * i, n0 + 32 * jp, lane, red[0][i * NS + 2 * jp][lane],
                   red[0][i * NS + 2 * jp + 1][lane]);
    }
  } else {
    for (int t = wave; t < MT * NS; t += 8)
      store_tile<EPI>(C, ldc, M, 16 * (t / NS), n0 + 16 * (t % NS), lane, red[0][t][lane]);
  }
}

// Sum split-K partials in order z = 0..S-1 and apply the epilogue.
template <int EPI>
__global__ void splitk_reduce_kernel(const float* __restrict__ ws, int S, int M, int N, void* C,
                                     int ldc) {
  // four consecutive output columns per thread (N % 128 == 0 and, for SwiGLU,
  // four consecutive hidden columns stay inside one 16-column gate/up group)
  const int64_t ncol = (EPI == EPI_SWIGLU) ? N / 2 : N;
  const int64_t nout4 = (int64_t)M * ncol / 4;
  const int64_t zs = (int64_t)M * N;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nout4;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(t / (ncol / 4));
    const int c = (int)(t % (ncol / 4)) * 4;
    if constexpr (EPI == EPI_SWIGLU) {
      const int pg = (c >> 4) * 32 + (c & 15), pu = pg + 16;
      float4 g = make_float4(0.f, 0.f, 0.f, 0.f), u = g;
      for (int z = 0; z < S; ++z) {
        const float4 a = *(const float4*)(ws + z * zs + (int64_t)m * N + pg);
        const float4 b = *(const float4*)(ws + z * zs + (int64_t)m * N + pu);
        g.x += a.x; g.y += a.y; g.z += a.z; g.w += a.w;
        u.x += b.x; u.y += b.y; u.z += b.z; u.w += b.w;
      }
      uint2 p;
      p.x = (uint32_t)f32_to_bf16(silu_f(g.x) * u.x) | ((uint32_t)f32_to_bf16(silu_f(g.y) * u.y) << 16);
      p.y = (uint32_t)f32_to_bf16(silu_f(g.z) * u.z) | ((uint32_t)f32_to_bf16(silu_f(g.w) * u.w) << 16);
      *(uint2*)((bf16_t*)C + (int64_t)m * ldc + c) = p;
    } else {
      float4 s4 = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int z = 0; z < S; ++z) {
        const float4 a = *(const float4*)(ws + z * zs + (int64_t)m * N + c);
        s4.x += a.x; s4.y += a.y; s4.z += a.z; s4.w += a.w;
      }
      if constexpr (EPI == EPI_F32) {
        *(float4*)((float*)C + (int64_t)m * ldc + c) = s4;
      } else if constexpr (EPI == EPI_ADD_F32) {
        float4* o = (float4*)((float*)C + (int64_t)m * ldc + c);
        const float4 x = *o;
        *o = make_float4(x.x + s4.x, x.y + s4.y, x.z + s4.z, x.w + s4.w);
      } else {
        uint2 p;
        p.x = (uint32_t)f32_to_bf16(s4.x) | ((uint32_t)f32_to_bf16(s4.y) << 16);
        p.y = (uint32_t)f32_to_bf16(s4.z) | ((uint32_t)f32_to_bf16(s4.w) << 16);
        *(uint2*)((bf16_t*)C + (int64_t)m * ldc + c) = p;
      }
    }
  }
}

// Split-K reduce fused with the residual add and the next RMSNorm: one block
// of 1024 threads per row, one float4 of the row per thread (N % 4 == 0,
// N <= 4096); x[m] += sum_z ws[z][m] in z order (all S partial loads issued
// together), then xn[m] = bf16(x[m] / sqrt(mean(x[m]^2) + eps)).
constexpr int kAddNormMaxN = 4096;
constexpr int kMaxSplits = 8;
__global__ void __launch_bounds__(1024) splitk_add_norm_kernel(const float* __restrict__ ws, int S,
                                                               int M, int N, float* __restrict__ x,
                                                               int ldx, float eps,
                                                               bf16_t* __restrict__ xn) {
  __shared__ float red[16];
  const int m = blockIdx.x, tid = threadIdx.x;
  const int64_t zs = (int64_t)M * N;
  const int c = tid * 4;
  const bool act = c < N;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  if (act) {
    float4 p[kMaxSplits];
#pragma unroll
    for (int z = 0; z < kMaxSplits; ++z)
      p[z] = z < S ? *(const float4*)(ws + z * zs + (int64_t)m * N + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    a = *(const float4*)(x + (int64_t)m * ldx + c);
#pragma unroll
    for (int z = 0; z < kMaxSplits; ++z) {
      a.x += p[z].x; a.y += p[z].y; a.z += p[z].z; a.w += p[z].w;
    }
    *(float4*)(x + (int64_t)m * ldx + c) = a;
  }
  float ss = a.x * a.x;
  ss = fmaf(a.y, a.y, ss);
  ss = fmaf(a.z, a.z, ss);
  ss = fmaf(a.w, a.w, ss);
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)N + eps);
  if (act) {
    uint2 q;
    q.x = (uint32_t)f32_to_bf16(a.x * inv) | ((uint32_t)f32_to_bf16(a.y * inv) << 16);
    q.y = (uint32_t)f32_to_bf16(a.z * inv) | ((uint32_t)f32_to_bf16(a.w * inv) << 16);
    *(uint2*)(xn + (int64_t)m * N + c) = q;
  }
}

// fp32 GEMM (fp32 models): 16x16 output tile per block, K in steps of 16.
template <int EPI>
__global__ void __launch_bounds__(256) gemm_f32_kernel(const float* __restrict__ A, int lda,
                                                       const float* __restrict__ W, int ldw, void* C,
                                                       int ldc, int M, int N, int K) {
  __shared__ float As[16][17], Ws2[16][17];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m = blockIdx.y * 16 + ty, n = blockIdx.x * 16 + tx;
  const int wrow = blockIdx.x * 16 + ty;
  float acc = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    As[ty][tx] = (m < M && k0 + tx < K) ? A[(int64_t)m * lda + k0 + tx] : 0.f;
    Ws2[ty][tx] = (wrow < N && k0 + tx < K) ? W[(int64_t)wrow * ldw + k0 + tx] : 0.f;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) acc = fmaf(As[ty][kk], Ws2[tx][kk], acc);
    __syncthreads();
  }
  if (m >= M || n >= N) return;
  if (EPI == EPI_F32) ((float*)C)[(int64_t)m * ldc + n] = acc;
  else if (EPI == EPI_ADD_F32) ((float*)C)[(int64_t)m * ldc + n] += acc;
}

// fp32 SwiGLU: one thread per output (m, c): reads the gate and up rows directly.
__global__ void gemm_f32_swiglu_kernel(const float* __restrict__ A, int lda, const float* __restrict__ W,
                                       int ldw, float* H, int ldc, int M, int F, int K) {
  const int64_t n = (int64_t)M * F;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(t / F), c = (int)(t % F);
    const int pg = (c >> 4) * 32 + (c & 15), pu = pg + 16;
    const float* a = A + (int64_t)m * lda;
    const float* wg = W + (int64_t)pg * ldw;
    const float* wu = W + (int64_t)pu * ldw;
    float g = 0.f, u = 0.f;
    for (int k = 0; k < K; ++k) {
      g = fmaf(a[k], wg[k], g);
      u = fmaf(a[k], wu[k], u);
    }
    H[(int64_t)m * ldc + c] = silu_f(g) * u;
  }
}

// ------------------------------------------------------------ dispatch
struct Plan {
  int kind;        // 0 skinny; tiled: 1 = 128x128 4 stages, 2 = 128x128 2 stages,
                   // 3 = 256x128 8 waves, 4 = 256x256 8 waves, 5 = 256x192 8 waves,
                   // exact-fill tiles with 4 stages and 4 waves: 6 = 128x96 (4x1),
                   // 7 = 128x64 (4x1), 8 = 64x64 (2x2), 9 = 64x96 (4x1)
  int mt, nt, S;   // tiles and K splits
  int MT, NS;      // skinny shape
};

// Planning assumes MI355X's 256 CUs whatever device runs the call, so a
// shape always gets the same plan (and the same summation order).
static constexpr int kCus = 256;

static void set_tiled(Plan& p, int kind, int bm, int bn, int M, int N, int S) {
  p.kind = kind; p.mt = (M + bm - 1) / bm; p.nt = N / bn; p.S = S;
}

// Tiled configs with the throughput model fitted to MI355X timings of every
// projection of the supported models (M = 1..512, weights streamed from HBM,
// not cache-resident): per-CU MFMA rate of one block (TFLOP/s), the weight
// streaming rate (GB/s) and blocks resident per CU.
struct TileCfg {
  int kind, bm, bn, occ;
  double rate, bw;
};
// The 256x192 tile (4 x 2 wavefronts of 64 x 96) fills all 256 CUs at
// M in (256, 512] for the gate/up projection of the 8B shape (N = 128 * 192);
// its rate is the 256x256 tile's scaled by their measured cache-cold ratio.
static const TileCfg kTileCfgs[5] = {
    {1, 128, 128, 1, 3.38, 6425.0},
    {2, 128, 128, 2, 2.26, 6423.0},
    {3, 256, 128, 1, 4.89, 6325.0},
    {4, 256, 256, 1, 6.68, 6298.0},
    {5, 256, 192, 1, 5.84, 6298.0},
};
static constexpr double kOcc2Gain = 1.76;   // CU throughput with two co-resident blocks / one block
static constexpr double kLaunchUs = 0.16;
static constexpr double kSplitGBs = 4106.0;  // partial sums: written once, read once by the reduce
static constexpr double kReduceUs = 3.19;

// Estimated time (us): rounds of resident blocks at the config's rate, at
// least the weight bytes at its streaming rate, plus the K-split partial-sum
// round trip and reduce launch.
static double tile_estimate(const TileCfg& c, int S, int M, int N, int K) {
  const int mt = (M + c.bm - 1) / c.bm, nt = N / c.bn;
  const double blocks = (double)mt * nt * S;
  const double mflop = 2.0 * c.bm * c.bn * ((double)K / S) * 1e-6;
  double t;
  if (blocks <= kCus) t = mflop / c.rate;
  else {
    const double rounds = std::ceil(blocks / (c.occ * kCus));
    t = rounds * c.occ * mflop / (c.occ == 2 ? c.rate * kOcc2Gain : c.rate);
  }
  t = std::max(t, 2.0 * N * (double)K / (c.bw * 1e3)) + kLaunchUs;
  if (S > 1) t += 2.0 * S * (double)M * N * 4.0 / (kSplitGBs * 1e3) + kReduceUs;
  return t;
}

// Small batches stream the weights once: what matters is that every CU
// streams an equal share.  Up to 128 rows, a tile of the batch's height
// (64 or 128 rows) and a K split whose block count is exactly one per CU is
// used when one exists (fewest splits, then the wider tile; a 64-column tile
// with 128 rows only for blocks of at most 1024 of K, where the 128x128
// tile's better reuse does not pay).  Measured on the Qwen3-8B projections
// (cache-cold weights), 8-20% faster than the best of the other configs up
// to 64 rows and up to 12% up to 128.
static bool exact_fill_plan(int M, int N, int K, Plan& p) {
  if (M > 128) return false;
  struct T { int kind, bm, bn; };
  static const T small[2] = {{9, 64, 96}, {8, 64, 64}};
  static const T mid[2] = {{6, 128, 96}, {7, 128, 64}};
  const T* cand = M <= 64 ? small : mid;
  for (int S = 1; S <= 8; S *= 2) {
    if (K % (S * 256) != 0 || K / S < 256) break;
    for (int i = 0; i < 2; ++i) {
      const T& t = cand[i];
      if (N % t.bn != 0 || (N / t.bn) * S != kCus) continue;
      if (M > 64 && t.bn == 64 && K / S > 1024) continue;
      set_tiled(p, t.kind, t.bm, t.bn, M, N, S);
      return true;
    }
  }
  return false;
}

//  * up to 128 rows: the exact-fill tile when one exists;
//  * M <= 32 with W up to 40 MB (and K <= 2048 beyond 16 rows): skinny;
//  * otherwise the tiled config and K split with the least estimated time
//    (256-row tiles only above 128 rows).
static Plan plan_gemm(int M, int N, int K) {
  Plan p{};
  if (exact_fill_plan(M, N, K, p)) return p;
  const double wbytes = 2.0 * N * K;
  if (M <= 32 && wbytes <= 40e6 && (M <= 16 || K <= 2048) && N % 32 == 0) {
    p.kind = 0;
    p.MT = (M + 15) / 16;
    p.NS = (M <= 16) ? 2 : 4;
    if (N % (p.NS * 16) != 0) p.NS = 2;
    p.nt = N / (p.NS * 16);
    p.mt = 1;
    // split K across blocks until there are ~2 blocks per CU (each wave keeps >= 256 of K)
    p.S = 1;
    while (p.nt * p.S < 2 * kCus && K % (p.S * 2 * 8 * 32) == 0 && K / (p.S * 2) >= 8 * 256) p.S *= 2;
    return p;
  }
  double best = 1e30;
  for (const TileCfg& c : kTileCfgs) {
    if (N % c.bn != 0 || (c.bm > 128 && M <= 128)) continue;
    for (int S = 1; S <= 8; S *= 2) {
      if (K % (S * 256) != 0 || K / S < 256) break;
      const double t = tile_estimate(c, S, M, N, K);
      if (t < best) { best = t; set_tiled(p, c.kind, c.bm, c.bn, M, N, S); }
    }
  }
  return p;
}

size_t gemm_workspace_bytes(int M, int N, int K) {
  const Plan p = plan_gemm(M, N, K);
  return p.S > 1 ? (size_t)p.S * M * N * sizeof(float) : 0;
}

template <int EPI>
static hipError_t reduce_launch(const void* ws, int S, int M, int N, void* C, int ldc,
                                hipStream_t st) {
  const int64_t nout = ((EPI == EPI_SWIGLU) ? (int64_t)M * (N / 2) : (int64_t)M * N) / 4;
  int64_t blocks = (nout + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(splitk_reduce_kernel<EPI>, dim3((unsigned)blocks), dim3(256), 0, st,
                     (const float*)ws, S, M, N, C, ldc);
  return hipGetLastError();
}

template <int EPI, int MT, int NS>
static void skinny_go(const Plan& p, const void* A, int lda, const void* W, int ldw, void* C,
                      int ldc, int M, int N, int K, void* ws, hipStream_t st) {
  const dim3 grid(p.nt * p.S), blk(512);
  if (p.S == 1)
    hipLaunchKernelGGL((gemm_skinny_kernel<MT, NS, EPI, false>), grid, blk, 0, st, (const bf16_t*)A,
                       lda, (const bf16_t*)W, ldw, C, ldc, M, N, K, K, p.nt, (float*)nullptr);
  else
    hipLaunchKernelGGL((gemm_skinny_kernel<MT, NS, EPI, true>), grid, blk, 0, st, (const bf16_t*)A,
                       lda, (const bf16_t*)W, ldw, C, ldc, M, N, K, K / p.S, p.nt, (float*)ws);
}

template <int EPI, int BM_, int BN_, int KB, int WGM, int WGN, int ST>
static void dma_go(const Plan& p, const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                   int M, int N, int K, void* ws, hipStream_t st) {
  const dim3 grid(p.mt * p.nt * p.S), blk(64 * WGM * WGN);
  const size_t lds = (size_t)ST * (BM_ + BN_) * KB * sizeof(bf16_t);
  static bool attr_done[2] = {false, false};
  if (p.S == 1) {
    auto kern = gemm_dma_kernel<BM_, BN_, KB, WGM, WGN, ST, EPI, false>;
    if (!attr_done[0]) {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      attr_done[0] = true;
    }
    hipLaunchKernelGGL(kern, grid, blk, lds, st, (const bf16_t*)A, lda, (const bf16_t*)W, ldw, C,
                       ldc, M, N, K, K, p.mt, p.nt, (float*)nullptr);
  } else {
    auto kern = gemm_dma_kernel<BM_, BN_, KB, WGM, WGN, ST, EPI, true>;
    if (!attr_done[1]) {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      attr_done[1] = true;
    }
    hipLaunchKernelGGL(kern, grid, blk, lds, st, (const bf16_t*)A, lda, (const bf16_t*)W, ldw, C,
                       ldc, M, N, K, K / p.S, p.mt, p.nt, (float*)ws);
  }
}

GroupedPlan grouped_plan(int64_t n_pairs, int E, bool gate_up) {
  if (n_pairs > (int64_t)96 * E) return {kGroupedTileRows, false, false};
  if (!gate_up) return {kGroupedTileRowsMin, false, n_pairs <= (int64_t)48 * E};
  if (n_pairs > (int64_t)48 * E) return {kGroupedTileRowsGU, true, true};
  return {kGroupedTileRowsMin, n_pairs >= (int64_t)2 * E, true};
}

hipError_t launch_pack_strips(void* W, int64_t rows, int K, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (rows % 16 || K % 32 || K < 32 || (size_t)16 * K * 2 > 160 * 1024 || rows / 16 > INT32_MAX)
    return hipErrorInvalidValue;
  const size_t lds = (size_t)16 * K * sizeof(bf16_t);
  static bool attr_done = false;
  if (!attr_done) {
    (void)hipFuncSetAttribute((const void*)pack_strips_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                              160 * 1024);
    attr_done = true;
  }
  hipLaunchKernelGGL(pack_strips_kernel, dim3((unsigned)(rows / 16)), dim3(256), lds, st, (bf16_t*)W, K);
  return hipGetLastError();
}

// Persistent blocks over (row tile, n tile) items.  128-row tiles (the
// prefill): 128x128 with a 4-stage ring, one block per CU.  64-row tiles
// (decode batches, where the expert weights are streamed): two blocks per
// CU, so one block's loads stream while the other waits at its barrier or
// refills its ring at an item boundary; 64x64 tiles with a 4-stage ring for
// the gate/up projection (K = d), 64x128 tiles with a 3-stage ring for the
// down projection (K = expert FFN).  Measured on the Qwen3-30B-A3B expert
// shapes from 1 to 1024 rows against one block per CU with 64x128 tiles and
// a 6-stage ring: 6-18% faster for gate/up, 10-18% for down.  96-row tiles:
// 96x128 with a 3-stage ring, one block per CU.  At 64 rows per expert about
// half the experts exceed 64 rows, and a 64-row tile list streams their
// weights twice; the 96-row tile streams them once (171-180 us per launch at
// 1024 rows against 222 us).  The gate/up plan now runs its 96-row (and most
// of its 64-row) tiles on the weights-into-registers kernel below, which is
// faster still; the down projection gains nothing from 96-row tiles (its
// second pass mostly hits in cache) and keeps 64-row tiles up to 96 rows per
// expert.
template <int BM_, int ST, int EPI, int BN_, int BPC, bool PW, int WAUX>
static hipError_t grouped_launch(const void* A, int lda, const void* W, int64_t w_stride, int ldw,
                                 void* C, int ldc, int N, int K, const int32_t* g_off,
                                 const int32_t* g_cnt, const int32_t* mtiles,
                                 const int32_t* n_mtiles, const int32_t* arow, hipStream_t st) {
  constexpr int KB = 64;
  if (N % BN_ != 0) return hipErrorInvalidValue;
  if (PW && (ldw != K || K % 32 != 0)) return hipErrorInvalidValue;
  const int nt = N / BN_;
  const size_t lds = (size_t)ST * (BM_ + BN_) * KB * sizeof(bf16_t);
  auto kern = gemm_dma_grouped_kernel<BM_, BN_, KB, 2, 2, ST, EPI, PW, WAUX>;
  static bool attr_done = false;
  if (!attr_done) {
    (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr_done = true;
  }
  static_assert((kCus * BPC) % 8 == 0, "the grouped kernel deals items to 8 XCDs");
  hipLaunchKernelGGL(kern, dim3(kCus * BPC), dim3(256), lds, st, (const bf16_t*)A, lda, (const bf16_t*)W,
                     w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles, n_mtiles, nt, arow);
  return hipGetLastError();
}

template <int EPI, bool PW, int WAUX>
static hipError_t grouped_by_rows_aux(int tile_rows, const void* A, int lda, const void* W, int64_t w_stride,
                                      int ldw, void* C, int ldc, int N, int K, const int32_t* g_off,
                                      const int32_t* g_cnt, const int32_t* mtiles, const int32_t* n_mtiles,
                                      const int32_t* arow, hipStream_t st) {
  if (tile_rows == kGroupedTileRowsMin) {
    if constexpr (EPI == EPI_SWIGLU)
      return grouped_launch<kGroupedTileRowsMin, 4, EPI, 64, 2, PW, WAUX>(A, lda, W, w_stride, ldw, C, ldc, N, K,
                                                                          g_off, g_cnt, mtiles, n_mtiles, arow, st);
    else
      return grouped_launch<kGroupedTileRowsMin, 3, EPI, 128, 2, PW, WAUX>(A, lda, W, w_stride, ldw, C, ldc, N, K,
                                                                           g_off, g_cnt, mtiles, n_mtiles, arow, st);
  }
  if (tile_rows == kGroupedTileRowsGU)
    return grouped_launch<kGroupedTileRowsGU, 3, EPI, 128, 1, PW, WAUX>(A, lda, W, w_stride, ldw, C, ldc, N, K,
                                                                        g_off, g_cnt, mtiles, n_mtiles, arow, st);
  if (tile_rows == kGroupedTileRows)
    return grouped_launch<kGroupedTileRows, 4, EPI, 128, 1, PW, WAUX>(A, lda, W, w_stride, ldw, C, ldc, N, K,
                                                                      g_off, g_cnt, mtiles, n_mtiles, arow, st);
  return hipErrorInvalidValue;
}

template <int EPI, bool PW>
static hipError_t grouped_by_rows(int tile_rows, bool nt_w, const void* A, int lda, const void* W,
                                  int64_t w_stride, int ldw, void* C, int ldc, int N, int K,
                                  const int32_t* g_off, const int32_t* g_cnt, const int32_t* mtiles,
                                  const int32_t* n_mtiles, const int32_t* arow, hipStream_t st) {
  return nt_w ? grouped_by_rows_aux<EPI, PW, kNtLoad>(tile_rows, A, lda, W, w_stride, ldw, C, ldc, N, K, g_off,
                                                      g_cnt, mtiles, n_mtiles, arow, st)
              : grouped_by_rows_aux<EPI, PW, 0>(tile_rows, A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt,
                                                mtiles, n_mtiles, arow, st);
}

// Weights into registers: 32 columns per wavefront (a 128-column slab per
// block), a 2-step register ring and 2-stage A ring, two blocks per CU.
// Measured against the tiled kernel on the Qwen3-30B-A3B gate/up shape
// (random routings, weights cache-cold, outputs bitwise equal), per launch:
// 96-row tiles 154 against 178 us at 1024 rows and 147 against 170 us at
// 768; 64-row tiles 139 against 150 us at 512, 132 against 138 at 256,
// 128 against 132 at 64 and 86 against 88 at 16; below 2 rows per expert
// (8 live rows) the tiled kernel is faster (67 against 73 us).
template <int BM>
static hipError_t wd_launch(const void* A, int lda, const void* W, int64_t w_stride, int ldw, void* C, int ldc,
                            int N, int K, const int32_t* g_off, const int32_t* g_cnt, const int32_t* mtiles,
                            const int32_t* n_mtiles, const int32_t* arow, hipStream_t st) {
  constexpr int CPW = 32, P = 2, BPC = 2;
  if (N % (4 * CPW) != 0 || ldw != K || (K / 64) % P != 0) return hipErrorInvalidValue;
  static_assert((kCus * BPC) % 8 == 0, "the grouped kernel deals items to 8 XCDs");
  hipLaunchKernelGGL((gemm_wd_grouped_kernel<BM, CPW, P, EPI_SWIGLU>), dim3(kCus * BPC), dim3(256), 0, st,
                     (const bf16_t*)A, lda, (const bf16_t*)W, w_stride, C, ldc, N, K, g_off, g_cnt, mtiles,
                     n_mtiles, arow);
  return hipGetLastError();
}

hipError_t launch_gemm_grouped(const void* A, int lda, const void* W, int64_t w_stride, int ldw,
                               void* C, int ldc, int N, int K, int epi, const int32_t* g_off,
                               const int32_t* g_cnt, const int32_t* mtiles, const int32_t* n_mtiles,
                               const int32_t* arow, GroupedPlan plan, bool packed_w, hipStream_t st) {
  if (N % 128 != 0 || K % 64 != 0 || K < 64) return hipErrorInvalidValue;
  const int tile_rows = plan.tile_rows;
  if (packed_w) {
    // strip-packed weights: the gate/up projection
    if (epi != EPI_SWIGLU) return hipErrorInvalidValue;
    if (plan.wdirect) {
      if (tile_rows == kGroupedTileRowsMin)
        return wd_launch<kGroupedTileRowsMin>(A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles,
                                              n_mtiles, arow, st);
      if (tile_rows == kGroupedTileRowsGU)
        return wd_launch<kGroupedTileRowsGU>(A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles,
                                             n_mtiles, arow, st);
      return hipErrorInvalidValue;
    }
    return grouped_by_rows<EPI_SWIGLU, true>(tile_rows, plan.nt_w, A, lda, W, w_stride, ldw, C, ldc, N, K,
                                             g_off, g_cnt, mtiles, n_mtiles, arow, st);
  }
  if (plan.wdirect) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_F32: return grouped_by_rows<EPI_F32, false>(tile_rows, plan.nt_w, A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles, n_mtiles, arow, st);
    case EPI_BF16: return grouped_by_rows<EPI_BF16, false>(tile_rows, plan.nt_w, A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles, n_mtiles, arow, st);
    case EPI_ADD_F32: return grouped_by_rows<EPI_ADD_F32, false>(tile_rows, plan.nt_w, A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles, n_mtiles, arow, st);
    case EPI_SWIGLU: return grouped_by_rows<EPI_SWIGLU, false>(tile_rows, plan.nt_w, A, lda, W, w_stride, ldw, C, ldc, N, K, g_off, g_cnt, mtiles, n_mtiles, arow, st);
    default: return hipErrorInvalidValue;
  }
}

// Launch the GEMM kernel of plan p (partial sums into ws when p.S > 1).
template <int EPI>
static hipError_t launch_plan(const Plan& p, const void* A, int lda, const void* W, int ldw, void* C,
                              int ldc, int M, int N, int K, void* ws, hipStream_t st) {
  if (p.kind == 0) {
    if (p.NS == 2) {
      switch (p.MT) {
        case 1: skinny_go<EPI, 1, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
        case 2: skinny_go<EPI, 2, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
        case 3: skinny_go<EPI, 3, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
        default: skinny_go<EPI, 4, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      }
    } else {
      switch (p.MT) {
        case 1: skinny_go<EPI, 1, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
        case 2: skinny_go<EPI, 2, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
        case 3: skinny_go<EPI, 3, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
        default: skinny_go<EPI, 4, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      }
    }
  } else {
    switch (p.kind) {
      case 1: dma_go<EPI, 128, 128, 64, 2, 2, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 2: dma_go<EPI, 128, 128, 64, 2, 2, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 3: dma_go<EPI, 256, 128, 64, 4, 2, 3>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 4: dma_go<EPI, 256, 256, 64, 2, 4, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 5: dma_go<EPI, 256, 192, 64, 4, 2, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 6: dma_go<EPI, 128, 96, 64, 4, 1, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 7: dma_go<EPI, 128, 64, 64, 4, 1, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 8: dma_go<EPI, 64, 64, 64, 2, 2, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      default: dma_go<EPI, 64, 96, 64, 4, 1, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
    }
  }
  return hipGetLastError();
}

template <int EPI>
static hipError_t gemm_bf16_launch(const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                                   int M, int N, int K, void* ws, size_t ws_bytes, hipStream_t st) {
  const Plan p = plan_gemm(M, N, K);
  if (p.S > 1 && (ws == nullptr || ws_bytes < (size_t)p.S * M * N * sizeof(float)))
    return hipErrorInvalidValue;
  hipError_t e = launch_plan<EPI>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st);
  if (e != hipSuccess || p.S == 1) return e;
  return reduce_launch<EPI>(ws, p.S, M, N, C, ldc, st);
}

template <int EPI>
static hipError_t gemm_f32_launch(const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                                  int M, int N, int K, hipStream_t st) {
  if constexpr (EPI == EPI_SWIGLU) {
    const int F = N / 2;
    int64_t blocks = ((int64_t)M * F + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(gemm_f32_swiglu_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                       (const float*)A, lda, (const float*)W, ldw, (float*)C, ldc, M, F, K);
    return hipGetLastError();
  } else {
    dim3 grid((N + 15) / 16, (M + 15) / 16);
    hipLaunchKernelGGL(gemm_f32_kernel<EPI>, grid, dim3(256), 0, st, (const float*)A, lda,
                       (const float*)W, ldw, C, ldc, M, N, K);
    return hipGetLastError();
  }
}

hipError_t launch_gemm(bool bf16, const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                       int M, int N, int K, int epi, void* ws, size_t ws_bytes, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!bf16) {
    switch (epi) {
      case EPI_F32: return gemm_f32_launch<EPI_F32>(A, lda, W, ldw, C, ldc, M, N, K, st);
      case EPI_BF16: return gemm_f32_launch<EPI_F32>(A, lda, W, ldw, C, ldc, M, N, K, st);
      case EPI_ADD_F32: return gemm_f32_launch<EPI_ADD_F32>(A, lda, W, ldw, C, ldc, M, N, K, st);
      case EPI_SWIGLU: return gemm_f32_launch<EPI_SWIGLU>(A, lda, W, ldw, C, ldc, M, N, K, st);
    }
    return hipErrorInvalidValue;
  }
  if (N % 128 != 0 || K % 256 != 0) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_F32: return gemm_bf16_launch<EPI_F32>(A, lda, W, ldw, C, ldc, M, N, K, ws, ws_bytes, st);
    case EPI_BF16: return gemm_bf16_launch<EPI_BF16>(A, lda, W, ldw, C, ldc, M, N, K, ws, ws_bytes, st);
    case EPI_ADD_F32:
      return gemm_bf16_launch<EPI_ADD_F32>(A, lda, W, ldw, C, ldc, M, N, K, ws, ws_bytes, st);
    case EPI_SWIGLU:
      return gemm_bf16_launch<EPI_SWIGLU>(A, lda, W, ldw, C, ldc, M, N, K, ws, ws_bytes, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_f32_or_partials(const void* A, int lda, const void* W, int ldw, float* C,
                                       int ldc, int M, int N, int K, void* ws, size_t ws_bytes,
                                       hipStream_t st, int* n_split) {
  *n_split = 1;
  if (M <= 0) return hipSuccess;
  if (N % 128 != 0 || K % 256 != 0) return hipErrorInvalidValue;
  const Plan p = plan_gemm(M, N, K);
  if (p.S == 1) return launch_plan<EPI_F32>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st);
  if (ws == nullptr || ws_bytes < (size_t)p.S * M * N * sizeof(float)) return hipErrorInvalidValue;
  *n_split = p.S;
  return launch_plan<EPI_F32>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st);
}

// x[M, N] += A . W^T followed by xn = bf16(RMSNorm(x)).  When the plan splits
// K the add and the norm are fused into the reduce (returns *fused = true);
// otherwise the GEMM adds in its epilogue and the caller normalises.
hipError_t launch_gemm_add_norm(const void* A, int lda, const void* W, int ldw, float* x, int ldx,
                                int M, int N, int K, void* ws, size_t ws_bytes, float eps,
                                void* xn, hipStream_t st, bool* fused) {
  *fused = false;
  if (M <= 0) return hipSuccess;
  if (N % 128 != 0 || K % 256 != 0) return hipErrorInvalidValue;
  const Plan p = plan_gemm(M, N, K);
  if (p.S == 1 || p.S > kMaxSplits || N > kAddNormMaxN)
    return gemm_bf16_launch<EPI_ADD_F32>(A, lda, W, ldw, x, ldx, M, N, K, ws, ws_bytes, st);
  if (ws == nullptr || ws_bytes < (size_t)p.S * M * N * sizeof(float)) return hipErrorInvalidValue;
  // the partial-sum GEMM of the plan, then the fused reduce
  hipError_t e = launch_plan<EPI_ADD_F32>(p, A, lda, W, ldw, x, ldx, M, N, K, ws, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(splitk_add_norm_kernel, dim3(M), dim3(1024), 0, st, (const float*)ws, p.S, M, N,
                     x, ldx, eps, (bf16_t*)xn);
  *fused = true;
  return hipGetLastError();
}

}  // namespace darts
