// float32 GEMM for the float32 MLP workload (batch 32, widths <= 512): the
// products are a few MFLOP, so the kernel is latency-bound and kept simple:
// 64x64 block tiles staged through LDS, 4x4 outputs per thread, plain FMA.
#include "layup_internal.h"

namespace layup {

namespace {
constexpr int TB = 64, TK = 16;

template <bool AK, bool BKM>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ B, float* C,
                                                       const float* bias, const float* aux,
                                                       int64_t M, int64_t N, int64_t K,
                                                       int64_t lda, int64_t ldb, int64_t ldc) {
  __shared__ float sA[TK][TB + 4];
  __shared__ float sB[TK][TB + 4];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t m0 = (int64_t)blockIdx.y * TB, n0 = (int64_t)blockIdx.x * TB;
  float acc[4][4] = {};
  for (int64_t k0 = 0; k0 < K; k0 += TK) {
    for (int e = threadIdx.x; e < TK * TB; e += 256) {
      int kk, r;
      if (AK) { r = e / TK; kk = e % TK; } else { kk = e / TB; r = e % TB; }
      int64_t gm = m0 + r, gk = k0 + kk;
      float va = 0.f;
      if (gm < M && gk < K) va = AK ? A[gm * lda + gk] : A[gk * lda + gm];
      sA[kk][r] = va;
      if (BKM) { r = e / TK; kk = e % TK; } else { kk = e / TB; r = e % TB; }
      int64_t gn = n0 + r;
      gk = k0 + kk;
      float vb = 0.f;
      if (gn < N && gk < K) vb = BKM ? B[gn * ldb + gk] : B[gk * ldb + gn];
      sB[kk][r] = vb;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int64_t m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int64_t n = n0 + tx * 4 + j;
      if (n >= N) continue;
      float v = acc[i][j];
      if (bias) v += bias[n];
      if (aux) v += aux[m * ldc + n];
      C[m * ldc + n] = v;
    }
  }
}
}  // namespace

hipError_t launch_gemm_f32(const Gemm& g, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  if (g.batch != 1) return hipErrorInvalidValue;
  dim3 grid((unsigned)cdiv(g.N, TB), (unsigned)cdiv(g.M, TB));
  const float* A = (const float*)g.A;
  const float* B = (const float*)g.B;
  float* C = (float*)g.C;
  const float* aux = (const float*)g.aux;
#define LAUNCH(ak, bk)                                                                         \
  gemm_f32_kernel<ak, bk><<<grid, 256, 0, s>>>(A, B, C, g.bias, aux, g.M, g.N, g.K, g.lda, \
                                               g.ldb, g.ldc)
  if (g.a_kmajor && g.b_kmajor) LAUNCH(true, true);
  else if (g.a_kmajor) LAUNCH(true, false);
  else if (g.b_kmajor) LAUNCH(false, true);
  else LAUNCH(false, false);
#undef LAUNCH
  return hipGetLastError();
}

}  // namespace layup
