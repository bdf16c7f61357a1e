// Dense GEMMs of the decoder: C[M,N] (op)= A[M,K] * W[N,K]^T.
// bf16 operands on gfx950 MFMA (v_mfma_f32_16x16x32_bf16), fp32 accumulate.
// Epilogues: store fp32, store bf16, add into an fp32 residual, SwiGLU
// (W rows interleaved in groups of 16: 16 gate rows then the 16 matching up
// rows; output silu(gate) * up as bf16).
//
// Two kernel families, chosen per launch from (M, N, K):
//  * tiled: BM x BN block tile staged through LDS, 4 wavefronts each owning
//    a WM x WN register tile; blocks are renumbered so that the blocks an XCD
//    runs are neighbours in (m, n) and share operand tiles in that XCD's L2.
//    The 64x128 tile uses a register-staged double buffer; the larger tiles
//    use direct global->LDS loads through a 3-4 deep ring of LDS stages.
//  * skinny (M <= 32, weight-bandwidth bound): no LDS for operands; each
//    wavefront loads W and A fragments straight into MFMA operand registers,
//    8 wavefronts of a block split K and are reduced through LDS.
// Either family may split K across blocks; partial sums then go to a
// workspace and a reduce kernel adds them in a fixed order (bitwise
// deterministic).
#include "common.h"
#include "kernels.h"

namespace darts {

constexpr int BK = 64, LDSK = BK + 8;  // +8 bf16 row pad: conflict-free 16-byte fragment reads

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

// ------------------------------------------------------------------ tiled
template <int BM, int BN, int WGM, int WGN, int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemm_tiled_kernel(const bf16_t* __restrict__ A, int lda,
                                                         const bf16_t* __restrict__ W, int ldw,
                                                         void* __restrict__ C, int ldc, int M,
                                                         int N, int K, int k_chunk, int mt, int nt,
                                                         float* __restrict__ ws) {
  constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 16, TN = WN / 16;
  constexpr int ALD = BM / 32, WLD = BN / 32;   // 16-byte chunks per thread per k-tile
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDSK];
  __shared__ __attribute__((aligned(16))) bf16_t Ws[2][BN * LDSK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  // XCD-aware renumbering: hardware block b runs on XCD b % 8; give each XCD a
  // contiguous range of logical tiles (m fastest, then n, then the K split).
  const int nb = gridDim.x;
  int b = blockIdx.x;
  const int full = (nb / 8) * 8;
  if (b < full) b = (b % 8) * (full / 8) + b / 8;
  const int mi = b % mt, ni = (b / mt) % nt, z = b / (mt * nt);
  const int m0 = mi * BM, n0 = ni * BN;
  const int kbeg = z * k_chunk;
  const int nk = k_chunk / BK;

  const int lr = tid >> 3, lc = (tid & 7) * 8;
  u32x4_t ra[ALD], rw[WLD];
  auto gload = [&](int kt) {
    const int kk = kbeg + kt * BK + lc;
#pragma unroll
    for (int i = 0; i < ALD; ++i) {
      const int r = m0 + lr + 32 * i;
      ra[i] = r < M ? *(const u32x4_t*)(A + (int64_t)r * lda + kk) : (u32x4_t){0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < WLD; ++i) rw[i] = *(const u32x4_t*)(W + (int64_t)(n0 + lr + 32 * i) * ldw + kk);
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ALD; ++i) *(u32x4_t*)(&As[buf][(lr + 32 * i) * LDSK + lc]) = ra[i];
#pragma unroll
    for (int i = 0; i < WLD; ++i) *(u32x4_t*)(&Ws[buf][(lr + 32 * i) * LDSK + lc]) = rw[i];
  };

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  gload(0);
  sstore(0);
  __syncthreads();
  const int arow = wm * WM + (lane & 15), brow = wn * WN + (lane & 15), kq = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      bf16x8_t a[TM], bb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = *(const bf16x8_t*)(&As[buf][(arow + 16 * i) * LDSK + ks + kq]);
#pragma unroll
      for (int j = 0; j < TN; ++j) bb[j] = *(const bf16x8_t*)(&Ws[buf][(brow + 16 * j) * LDSK + ks + kq]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      sstore(buf ^ 1);
      __syncthreads();
    }
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

// ------------------------------------------------------- tiled, LDS DMA
// Same tile math as above, but operand tiles travel global -> LDS with
// direct 16-byte LDS loads (no staging registers) through a STAGES-deep ring
// of LDS buffers.  A 64-wide K slice of a row is 8 chunks of 16 bytes; chunk
// c of row r is stored at chunk position c ^ (r & 7) of that row so that the
// 16-byte fragment reads of 8 consecutive rows hit distinct banks.  Rows of A
// past M load row M-1 (their results are never stored).
// s_waitcnt vmcnt(N) (gfx9 encoding: vmcnt bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their "don't wait" maxima)
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef __attribute__((address_space(3))) void lds_void_t;

template <int BM, int BN, int WGM, int WGN, int STAGES, int EPI, bool SPLIT>
__global__ void __launch_bounds__(64 * WGM * WGN) gemm_dma_kernel(const bf16_t* __restrict__ A, int lda,
                                                       const bf16_t* __restrict__ W, int ldw,
                                                       void* __restrict__ C, int ldc, int M,
                                                       int N, int K, int k_chunk, int mt, int nt,
                                                       float* __restrict__ ws) {
  constexpr int NW = WGM * WGN;                    // wavefronts per block
  constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 16, TN = WN / 16;
  constexpr int AI = BM / (8 * NW), WI = BN / (8 * NW);   // 1 KB load instructions per wave per stage
  static_assert(AI * 8 * NW == BM && WI * 8 * NW == BN, "tile rows must split over the waves");
  constexpr int STAGE_ELEMS = (BM + BN) * BK;      // bf16 elements per stage
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int nb = gridDim.x;
  int b = blockIdx.x;
  const int full = (nb / 8) * 8;
  if (b < full) b = (b % 8) * (full / 8) + b / 8;
  const int mi = b % mt, ni = (b / mt) % nt, z = b / (mt * nt);
  const int m0 = mi * BM, n0 = ni * BN;
  const int kbeg = z * k_chunk;
  const int nk = k_chunk / BK;

  // per-lane global source rows for this wave's load instructions
  const int lrow = lane >> 3;                     // row within an 8-row instruction
  const int gchunk = (lane & 7) ^ lrow;           // swizzled source chunk
  const bf16_t* asrc[AI];
  const bf16_t* wsrc[WI];
#pragma unroll
  for (int j = 0; j < AI; ++j) {
    int r = m0 + wave * (BM / NW) + 8 * j + lrow;
    r = r < M ? r : M - 1;
    asrc[j] = A + (int64_t)r * lda + kbeg + gchunk * 8;
  }
#pragma unroll
  for (int j = 0; j < WI; ++j)
    wsrc[j] = W + (int64_t)(n0 + wave * (BN / NW) + 8 * j + lrow) * ldw + kbeg + gchunk * 8;

  auto issue = [&](int kt, int buf) {
    bf16_t* sa = smem + buf * STAGE_ELEMS;
    bf16_t* sw = sa + BM * BK;
#pragma unroll
    for (int j = 0; j < AI; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[j] + kt * BK),
                                       (lds_void_t*)(sa + (wave * (BM / NW) + 8 * j) * BK), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < WI; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(wsrc[j] + kt * BK),
                                       (lds_void_t*)(sw + (wave * (BN / NW) + 8 * j) * BK), 16, 0, 0);
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
    const bf16_t* sw = sa + BM * BK;
    // fragments of both 32-wide K halves are read before the MFMAs of the
    // first half, so LDS latency overlaps matrix work
    bf16x8_t a[2][TM], bb[2][TN];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WM + 16 * i + fr;
        a[ks][i] = *(const bf16x8_t*)(sa + r * BK + (((ks * 4 + fq) ^ (r & 7)) * 8));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WN + 16 * j + fr;
        bb[ks][j] = *(const bf16x8_t*)(sw + r * BK + (((ks * 4 + fq) ^ (r & 7)) * 8));
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
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

// ----------------------------------------------------------------- skinny
// Block: 8 wavefronts, NS*16 output columns, all M <= 16*MT rows.  Wavefront
// w handles K range [kbeg + w*kw, kbeg + (w+1)*kw).
template <int MT, int NS, int EPI, bool SPLIT>
__global__ void __launch_bounds__(512) gemm_skinny_kernel(const bf16_t* __restrict__ A, int lda,
                                                          const bf16_t* __restrict__ W, int ldw,
                                                          void* __restrict__ C, int ldc, int M,
                                                          int N, int K, int k_chunk, int nt,
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
#pragma unroll 4
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
  const int64_t nout = (EPI == EPI_SWIGLU) ? (int64_t)M * (N / 2) : (int64_t)M * N;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nout;
       t += (int64_t)gridDim.x * blockDim.x) {
    if constexpr (EPI == EPI_SWIGLU) {
      const int F = N / 2;
      const int m = (int)(t / F), c = (int)(t % F);
      const int pg = (c >> 4) * 32 + (c & 15), pu = pg + 16;
      float g = 0.f, u = 0.f;
      for (int z = 0; z < S; ++z) {
        g += ws[((int64_t)z * M + m) * N + pg];
        u += ws[((int64_t)z * M + m) * N + pu];
      }
      ((bf16_t*)C)[(int64_t)m * ldc + c] = f32_to_bf16(silu_f(g) * u);
    } else {
      const int m = (int)(t / N), n = (int)(t % N);
      float s = 0.f;
      for (int z = 0; z < S; ++z) s += ws[((int64_t)z * M + m) * N + n];
      epi_store<EPI>(C, ldc, M, m, n, s);
    }
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
  int kind;        // 0 skinny, 1..4 tiled configs
  int mt, nt, S;   // tiles and K splits
  int MT, NS;      // skinny shape
};

static int cu_count() { return 256; }

// Tiled configs: (BM, BN)
static const int kTiles[5][2] = {{64, 128}, {128, 128}, {128, 256}, {256, 128}, {256, 256}};

static Plan plan_gemm(int M, int N, int K) {
  Plan p{};
  const int cus = cu_count();
  if (M <= 32) {
    p.kind = 0;
    p.MT = (M + 15) / 16;
    p.NS = (M <= 16) ? 2 : 4;
    if (N % (p.NS * 16) != 0) p.NS = 2;
    p.nt = N / (p.NS * 16);
    p.mt = 1;
    // split K across blocks until there are ~2 blocks per CU (each wave keeps >= 256 of K)
    p.S = 1;
    while (p.nt * p.S < 2 * cus && K % (p.S * 2 * 8 * 32) == 0 && K / (p.S * 2) >= 8 * 256) p.S *= 2;
    return p;
  }
  // tiled: estimated time (us) = rounds * tile time at the config's measured
  // per-CU MFMA efficiency, plus, for a K split, the partial-sum round trip
  // through HBM (S*M*N fp32 written and read) and the reduce launch.
  const double cu_tflops = 2500.0 / cus;                    // dense bf16 per CU
  const double eff[5] = {0.12, 0.35, 0.42, 0.42, 0.55};   // measured on MI355X (decode shapes)
  double best = 1e30;
  for (int c = 0; c < 5; ++c) {
    const int BMc = kTiles[c][0], BNc = kTiles[c][1];
    if (N % BNc) continue;
    if (BMc > 128 && M <= 128) continue;
    const int mt = (M + BMc - 1) / BMc, nt = N / BNc;
    for (int S = 1; S <= 8; S *= 2) {
      if (K % (S * BK) || K / S < 4 * BK) break;
      const int tiles = mt * nt * S;
      const int rounds = (tiles + cus - 1) / cus;
      double t = rounds * (2.0 * BMc * BNc * (K / S)) / (cu_tflops * eff[c] * 1e6);
      if (S > 1) t += (2.0 * S * (double)M * N * 4.0) / 4.0e6 + 4.0;
      if (t < best * 0.97) {
        best = t;
        p.kind = 1 + c; p.mt = mt; p.nt = nt; p.S = S;
      }
    }
  }
  if (p.kind == 0) { p.kind = 1; p.mt = (M + 63) / 64; p.nt = N / 128; p.S = 1; }
  return p;
}

size_t gemm_workspace_bytes(int M, int N, int K) {
  const Plan p = plan_gemm(M, N, K);
  return p.S > 1 ? (size_t)p.S * M * N * sizeof(float) : 0;
}

template <int EPI>
static hipError_t reduce_launch(const void* ws, int S, int M, int N, void* C, int ldc,
                                hipStream_t st) {
  const int64_t nout = (EPI == EPI_SWIGLU) ? (int64_t)M * (N / 2) : (int64_t)M * N;
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

template <int EPI, int BM_, int BN_, int WGM, int WGN, int ST>
static void dma_go(const Plan& p, const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                   int M, int N, int K, void* ws, hipStream_t st) {
  const dim3 grid(p.mt * p.nt * p.S), blk(64 * WGM * WGN);
  const size_t lds = (size_t)ST * (BM_ + BN_) * BK * sizeof(bf16_t);
  static bool attr_done[2] = {false, false};
  if (p.S == 1) {
    auto kern = gemm_dma_kernel<BM_, BN_, WGM, WGN, ST, EPI, false>;
    if (!attr_done[0]) {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      attr_done[0] = true;
    }
    hipLaunchKernelGGL(kern, grid, blk, lds, st, (const bf16_t*)A, lda, (const bf16_t*)W, ldw, C,
                       ldc, M, N, K, K, p.mt, p.nt, (float*)nullptr);
  } else {
    auto kern = gemm_dma_kernel<BM_, BN_, WGM, WGN, ST, EPI, true>;
    if (!attr_done[1]) {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      attr_done[1] = true;
    }
    hipLaunchKernelGGL(kern, grid, blk, lds, st, (const bf16_t*)A, lda, (const bf16_t*)W, ldw, C,
                       ldc, M, N, K, K / p.S, p.mt, p.nt, (float*)ws);
  }
}

template <int EPI, int BM_, int BN_, int WGM, int WGN>
static void tiled_go(const Plan& p, const void* A, int lda, const void* W, int ldw, void* C,
                     int ldc, int M, int N, int K, void* ws, hipStream_t st) {
  const dim3 grid(p.mt * p.nt * p.S), blk(256);
  if (p.S == 1)
    hipLaunchKernelGGL((gemm_tiled_kernel<BM_, BN_, WGM, WGN, EPI, false>), grid, blk, 0, st,
                       (const bf16_t*)A, lda, (const bf16_t*)W, ldw, C, ldc, M, N, K, K, p.mt, p.nt,
                       (float*)nullptr);
  else
    hipLaunchKernelGGL((gemm_tiled_kernel<BM_, BN_, WGM, WGN, EPI, true>), grid, blk, 0, st,
                       (const bf16_t*)A, lda, (const bf16_t*)W, ldw, C, ldc, M, N, K, K / p.S, p.mt,
                       p.nt, (float*)ws);
}

template <int EPI>
static hipError_t gemm_bf16_launch(const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                                   int M, int N, int K, void* ws, size_t ws_bytes, hipStream_t st) {
  Plan p = plan_gemm(M, N, K);
  if (p.S > 1 && (ws == nullptr || ws_bytes < (size_t)p.S * M * N * sizeof(float)))
    return hipErrorInvalidValue;
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
      case 1: tiled_go<EPI, 64, 128, 1, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 2: dma_go<EPI, 128, 128, 2, 2, 4>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 3: dma_go<EPI, 128, 256, 2, 2, 3>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      case 4: dma_go<EPI, 256, 128, 2, 2, 3>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
      default: dma_go<EPI, 256, 256, 2, 4, 2>(p, A, lda, W, ldw, C, ldc, M, N, K, ws, st); break;
    }
  }
  hipError_t e = hipGetLastError();
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

}  // namespace darts
