// Dense GEMMs of the decoder: C[M,N] (op)= A[M,K] * W[N,K]^T.
// bf16 operands on gfx950 MFMA (v_mfma_f32_16x16x32_bf16), fp32 accumulate.
// Epilogues: store fp32, store bf16, add into an fp32 residual, SwiGLU
// (W rows interleaved in groups of 16: 16 gate rows then the 16 matching up
// rows, output silu(gate) * up as bf16).  Small-M launches split K across
// blocks; partial sums go to a workspace and a second kernel reduces them in
// a fixed order (bitwise deterministic).
#include "common.h"
#include "kernels.h"

namespace darts {

constexpr int BM = 64, BN = 128, BK = 64, LDSK = BK + 8;  // +8 bf16 pad: conflict-free b128 reads

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

template <int EPI>
__device__ __forceinline__ void epi_store(void* C, int ldc, int M, int m, int n, float v) {
  if (m >= M) return;
  if (EPI == EPI_F32) ((float*)C)[(int64_t)m * ldc + n] = v;
  else if (EPI == EPI_BF16) ((bf16_t*)C)[(int64_t)m * ldc + n] = f32_to_bf16(v);
  else if (EPI == EPI_ADD_F32) ((float*)C)[(int64_t)m * ldc + n] += v;
}

// SPLIT: write raw fp32 partials to ws[z][M][N] instead of the epilogue.
template <int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(const bf16_t* __restrict__ A, int lda,
                                                        const bf16_t* __restrict__ W, int ldw,
                                                        void* __restrict__ C, int ldc, int M, int N,
                                                        int K, int k_chunk, float* __restrict__ ws) {
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDSK];
  __shared__ __attribute__((aligned(16))) bf16_t Ws[2][BN * LDSK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * k_chunk;
  const int nk = k_chunk / BK;

  // global -> register staging: A 2 x 16B, W 4 x 16B per thread
  const int lr = tid >> 3, lc = (tid & 7) * 8;
  uint4 ra[2], rw[4];
  auto gload = [&](int kt) {
    const int kk = kbeg + kt * BK + lc;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = m0 + lr + 32 * i;
      if (r < M) ra[i] = *(const uint4*)(A + (int64_t)r * lda + kk);
      else ra[i] = make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = n0 + lr + 32 * i;
      rw[i] = *(const uint4*)(W + (int64_t)r * ldw + kk);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) *(uint4*)(&As[buf][(lr + 32 * i) * LDSK + lc]) = ra[i];
#pragma unroll
    for (int i = 0; i < 4; ++i) *(uint4*)(&Ws[buf][(lr + 32 * i) * LDSK + lc]) = rw[i];
  };

  f32x4_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  gload(0);
  sstore(0);
  __syncthreads();
  const int arow = wm * 32 + (lane & 15), brow = wn * 64 + (lane & 15), kq = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      bf16x8_t a[2], b[4];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = *(const bf16x8_t*)(&As[buf][(arow + 16 * i) * LDSK + ks + kq]);
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = *(const bf16x8_t*)(&Ws[buf][(brow + 16 * j) * LDSK + ks + kq]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      sstore(buf ^ 1);
      __syncthreads();
    }
  }

  // lane holds C[row = base + 4*(lane/16) + r][col = base + lane%16]
  const int rbase = m0 + wm * 32 + 4 * (lane >> 4);
  const int cbase = n0 + wn * 64 + (lane & 15);
  if (SPLIT) {
    float* P = ws + (int64_t)blockIdx.z * M * N;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = rbase + 16 * i + r;
          if (m < M) P[(int64_t)m * N + cbase + 16 * j] = acc[i][j][r];
        }
    return;
  }
  if (EPI == EPI_SWIGLU) {
    // tiles j=0,1 are (gate, up) of one 16-feature group, tiles 2,3 the next
    bf16_t* H = (bf16_t*)C;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int jp = 0; jp < 2; ++jp) {
        const int grp = (n0 + wn * 64 + 32 * jp) >> 5;
        const int col = grp * 16 + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = rbase + 16 * i + r;
          if (m < M) {
            const float g = acc[i][2 * jp][r], u = acc[i][2 * jp + 1][r];
            H[(int64_t)m * ldc + col] = f32_to_bf16(silu_f(g) * u);
          }
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) epi_store<EPI>(C, ldc, M, rbase + 16 * i + r, cbase + 16 * j, acc[i][j][r]);
}

// Sum split-K partials in order z = 0..S-1 and apply the epilogue.
template <int EPI>
__global__ void splitk_reduce_kernel(const float* __restrict__ ws, int S, int M, int N, void* C,
                                     int ldc) {
  const int64_t nout = (EPI == EPI_SWIGLU) ? (int64_t)M * (N / 2) : (int64_t)M * N;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < nout;
       t += (int64_t)gridDim.x * blockDim.x) {
    if (EPI == EPI_SWIGLU) {
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

// fp32 GEMM (used by fp32 models): 16x16 output tile per block, K in steps of 16.
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
  else if (EPI == EPI_BF16) ((bf16_t*)C)[(int64_t)m * ldc + n] = f32_to_bf16(acc);
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

static int choose_splits(int M, int N, int K) {
  const int blocks = ((M + BM - 1) / BM) * (N / BN);
  int s = 1;
  while (blocks * s < 512 && s < 8 && (K / (BK * 2 * s)) >= 2 && (K % (BK * 2 * s)) == 0) s *= 2;
  return s;
}

size_t gemm_workspace_bytes(int M, int N, int K) {
  const int s = choose_splits(M, N, K);
  return s > 1 ? (size_t)s * M * N * sizeof(float) : 0;
}

template <int EPI>
static hipError_t gemm_bf16_launch(const void* A, int lda, const void* W, int ldw, void* C, int ldc,
                                   int M, int N, int K, void* ws, size_t ws_bytes, hipStream_t st) {
  int S = choose_splits(M, N, K);
  if (S > 1 && (ws == nullptr || ws_bytes < (size_t)S * M * N * sizeof(float))) S = 1;
  dim3 grid(N / BN, (M + BM - 1) / BM, S);
  if (S == 1) {
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI, false>), grid, dim3(256), 0, st, (const bf16_t*)A,
                       lda, (const bf16_t*)W, ldw, C, ldc, M, N, K, K, (float*)nullptr);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((gemm_bf16_kernel<EPI, true>), grid, dim3(256), 0, st, (const bf16_t*)A, lda,
                     (const bf16_t*)W, ldw, C, ldc, M, N, K, K / S, (float*)ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nout = (EPI == EPI_SWIGLU) ? (int64_t)M * (N / 2) : (int64_t)M * N;
  int64_t blocks = (nout + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(splitk_reduce_kernel<EPI>, dim3((unsigned)blocks), dim3(256), 0, st,
                     (const float*)ws, S, M, N, C, ldc);
  return hipGetLastError();
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
  if (N % BN != 0 || K % BK != 0) return hipErrorInvalidValue;
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
