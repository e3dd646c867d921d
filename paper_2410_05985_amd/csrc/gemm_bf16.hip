// bfloat16 GEMM on the CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16), float32
// accumulation.  This is the one dense contraction of the layer-wise step:
// the dX = dY W and dW = dY^T X products of every linear layer's backward
// (LayUp Algorithm 1, "Backward pass at layer l"), plus the forward and the
// attention products that produce what the backward reads.
//
// Structure: 256 threads = 4 wave64s in a 2x2 grid; a BM x BN block tile,
// each wave a (BM/2) x (BN/2) tile of 32x32 MFMA blocks.  K advances in
// steps of 64 through double-buffered LDS (one barrier per step); the next
// step's global loads are in flight while the current step's MFMAs run.
// Operands land in LDS k-contiguous ([row][k], padded rows) whatever their
// layout in HBM: a k-contiguous operand is copied with 128-bit loads/stores;
// an m/n-contiguous operand (the transposed operands of dW = dY^T X) is
// loaded as 4(k) x 8(m) blocks with 128-bit loads and transposed in
// registers before 64-bit LDS stores.  Each lane then reads its 8 k-values
// of an MFMA operand with one 128-bit LDS read.
//
// Block tiles are remapped so that consecutive tiles of one output row band
// run on the same XCD (workgroups are dealt round-robin over the 8 XCDs,
// each with its own L2), then grouped along M for L2 reuse of B.
// Split-K (float32 partials + fixed-order reduction, deterministic) is used
// when the output has too few tiles to fill 256 CUs.
#include "layup_internal.h"

namespace layup {

namespace {

constexpr int BK = 64;
constexpr int LDS_PAD = 8;           // bf16 elements of padding per LDS row
constexpr int LDK = BK + LDS_PAD;    // LDS row stride (elements)
constexpr int THREADS = 256;

struct KArgs {
  const bf16_t* A;
  const bf16_t* B;
  void* C;
  void* C2;
  const void* aux;
  const float* bias;
  float* partial;
  int64_t M, N, K, lda, ldb, ldc;
  int64_t a_outer, a_inner, b_outer, b_inner, c_outer, c_inner;
  int32_t inner, splits, tiles_m, tiles_n;
  int64_t k_per_split;
};

__device__ __forceinline__ float gelu_tanh_f(float x) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  float u = c * fmaf(0.044715f * x, x * x, x);
  return 0.5f * x * (1.0f + tanhf(u));
}

__device__ __forceinline__ float gelu_tanh_grad_f(float x) {
  const float c = 0.7978845608028654f;
  float u = c * fmaf(0.044715f * x, x * x, x);
  float t = tanhf(u);
  return 0.5f * (1.0f + t) + 0.5f * x * (1.0f - t * t) * c * fmaf(3.0f * 0.044715f, x * x, 1.0f);
}

// Loads of one operand tile (rows x BK) into registers.
// KMAJOR: element (r, k) at base[r*ld + k]; else at base[k*ld + r].
template <int ROWS, bool KMAJOR>
struct TileLoader {
  // k-major: ROWS*BK/8 vectors of 8 bf16, ROWS/32 per thread
  // r-major: (BK/4)*(ROWS/8) blocks of 4(k) x 8(r), ROWS/128 per thread (ROWS >= 128)
  //          or one block per thread for the first 16*ROWS/8 threads (ROWS = 64)
  static constexpr int NV = KMAJOR ? ROWS / 32 : (ROWS >= 128 ? ROWS / 128 : 1);
  u32x4 reg[KMAJOR ? NV : NV * 4];

  __device__ __forceinline__ void load(const bf16_t* base, int64_t ld, int64_t r0, int64_t k0,
                                       int64_t R, int64_t K, bool guard) {
    const int t = threadIdx.x;
    if (KMAJOR) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int L = t + THREADS * i;
        int row = L >> 3, kc = (L & 7) * 8;
        int64_t gr = r0 + row, gk = k0 + kc;
        if (!guard || (gr < R && gk < K))
          reg[i] = *reinterpret_cast<const u32x4*>(base + gr * ld + gk);
        else
          reg[i] = u32x4{0, 0, 0, 0};
      }
    } else {
      constexpr int RG = ROWS / 8;  // 8-wide row groups
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int L = t + THREADS * i;
        int rg = L % RG, kg = L / RG;
        bool active = kg < BK / 4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          int64_t gk = k0 + kg * 4 + r, gr = r0 + rg * 8;
          if (active && (!guard || (gk < K && gr < R)))
            reg[i * 4 + r] = *reinterpret_cast<const u32x4*>(base + gk * ld + gr);
          else
            reg[i * 4 + r] = u32x4{0, 0, 0, 0};
        }
      }
    }
  }

  __device__ __forceinline__ void store(bf16_t* lds) const {
    const int t = threadIdx.x;
    if (KMAJOR) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int L = t + THREADS * i;
        int row = L >> 3, kc = (L & 7) * 8;
        *reinterpret_cast<u32x4*>(lds + row * LDK + kc) = reg[i];
      }
    } else {
      constexpr int RG = ROWS / 8;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int L = t + THREADS * i;
        int rg = L % RG, kg = L / RG;
        if (kg >= BK / 4) continue;
        const u32x4* q = &reg[i * 4];
#pragma unroll
        for (int mm = 0; mm < 8; ++mm) {
          const int w = mm >> 1;
          uint32_t e0, e1;
          if (mm & 1) {
            e0 = (q[0][w] >> 16) | (q[1][w] & 0xffff0000u);
            e1 = (q[2][w] >> 16) | (q[3][w] & 0xffff0000u);
          } else {
            e0 = (q[0][w] & 0xffffu) | (q[1][w] << 16);
            e1 = (q[2][w] & 0xffffu) | (q[3][w] << 16);
          }
          *reinterpret_cast<u32x2*>(lds + (rg * 8 + mm) * LDK + kg * 4) = u32x2{e0, e1};
        }
      }
    }
  }
};

template <int BM, int BN, bool AK, bool BKM, int EPI, bool SPLIT>
__global__ __launch_bounds__(THREADS, 2) void gemm_bf16_kernel(const KArgs P) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 32, TN = WN / 32;
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (BM + BN) * LDK];
  // buffer b: A tile at smem + b*(BM+BN)*LDK, B tile right after it
  constexpr int BUF = (BM + BN) * LDK;

  // ---- tile mapping: XCD-aware remap, then group along M
  const int n_tiles = P.tiles_m * P.tiles_n;
  int id = blockIdx.x;
  if ((n_tiles & 7) == 0) id = (id & 7) * (n_tiles >> 3) + (id >> 3);
  constexpr int GROUP = 8;
  const int width = GROUP * P.tiles_n;
  const int grp = id / width;
  const int first_m = grp * GROUP;
  const int gsz = min(P.tiles_m - first_m, GROUP);
  const int tm = first_m + (id % width) % gsz;
  const int tn = (id % width) / gsz;

  const int z = SPLIT ? 0 : blockIdx.y;
  const int split = SPLIT ? blockIdx.y : 0;
  const int zo = z / P.inner, zi = z % P.inner;
  const bf16_t* Ab = P.A + zo * P.a_outer + zi * P.a_inner;
  const bf16_t* Bb = P.B + zo * P.b_outer + zi * P.b_inner;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  int64_t kb = 0, ke = P.K;
  if (SPLIT) {
    kb = split * P.k_per_split;
    ke = min(P.K, kb + P.k_per_split);
  }
  const bool guard = (m0 + BM > P.M) || (n0 + BN > P.N) || ((ke - kb) % BK != 0);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  TileLoader<BM, AK> la;
  TileLoader<BN, BKM> lb;
  const int nk = (int)((ke - kb + BK - 1) / BK);
  if (nk > 0) {
    la.load(Ab, P.lda, m0, kb, P.M, ke, guard);
    lb.load(Bb, P.ldb, n0, kb, P.N, ke, guard);
    la.store(smem);
    lb.store(smem + BM * LDK);
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(Ab, P.lda, m0, kb + (int64_t)(kt + 1) * BK, P.M, ke, guard);
      lb.load(Bb, P.ldb, n0, kb + (int64_t)(kt + 1) * BK, P.N, ke, guard);
    }
    const bf16_t* a_s = smem + cur * BUF + (wm * WM + (lane & 31)) * LDK + (lane >> 5) * 8;
    const bf16_t* b_s = smem + cur * BUF + BM * LDK + (wn * WN + (lane & 31)) * LDK + (lane >> 5) * 8;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(a_s + i * 32 * LDK + ks * 16);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(b_s + j * 32 * LDK + ks * 16);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      la.store(smem + (cur ^ 1) * BUF);
      lb.store(smem + (cur ^ 1) * BUF + BM * LDK);
    }
    __syncthreads();
  }

  // ---- epilogue.  32x32 accumulator layout: lane l, register r holds
  // row (r/4)*8 + (l/32)*4 + r%4, column l%32 of the 32x32 block.
  const int64_t c_off = zo * P.c_outer + zi * P.c_inner;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t n = n0 + wn * WN + j * 32 + (lane & 31);
      if (n >= P.N) continue;
      float bn = 0.f;
      if (!SPLIT && P.bias && (EPI == EPI_F32 || EPI == EPI_BF16 || EPI == EPI_GELU)) bn = P.bias[n];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * WM + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (m >= P.M) continue;
        float v = acc[i][j][r];
        if (SPLIT) {
          P.partial[(int64_t)split * P.M * P.N + m * P.N + n] = v;
          continue;
        }
        const int64_t off = c_off + m * P.ldc + n;
        if (EPI == EPI_F32) {
          v += bn;
          if (P.aux) v += reinterpret_cast<const float*>(P.aux)[off];
          reinterpret_cast<float*>(P.C)[off] = v;
        } else if (EPI == EPI_BF16) {
          reinterpret_cast<bf16_t*>(P.C)[off] = f2bf(v + bn);
        } else if (EPI == EPI_GELU) {
          v += bn;
          reinterpret_cast<bf16_t*>(P.C)[off] = f2bf(v);
          reinterpret_cast<bf16_t*>(P.C2)[off] = f2bf(gelu_tanh_f(v));
        } else {  // EPI_DGELU
          float f = bf2f(reinterpret_cast<const bf16_t*>(P.aux)[off]);
          reinterpret_cast<bf16_t*>(P.C)[off] = f2bf(v * gelu_tanh_grad_f(f));
        }
      }
    }
  }
}

// Fixed-order sum of split-K partials plus the epilogue.
template <int EPI>
__global__ void splitk_reduce_kernel(const KArgs P) {
  const int64_t total = P.M * P.N;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = idx / P.N, n = idx % P.N;
    float v = 0.f;
    for (int s = 0; s < P.splits; ++s) v += P.partial[(int64_t)s * total + idx];
    const int64_t off = m * P.ldc + n;
    float bn = P.bias ? P.bias[n] : 0.f;
    if (EPI == EPI_F32) {
      v += bn;
      if (P.aux) v += reinterpret_cast<const float*>(P.aux)[off];
      reinterpret_cast<float*>(P.C)[off] = v;
    } else if (EPI == EPI_BF16) {
      reinterpret_cast<bf16_t*>(P.C)[off] = f2bf(v + bn);
    } else if (EPI == EPI_GELU) {
      v += bn;
      reinterpret_cast<bf16_t*>(P.C)[off] = f2bf(v);
      reinterpret_cast<bf16_t*>(P.C2)[off] = f2bf(gelu_tanh_f(v));
    } else {
      float f = bf2f(reinterpret_cast<const bf16_t*>(P.aux)[off]);
      reinterpret_cast<bf16_t*>(P.C)[off] = f2bf(v * gelu_tanh_grad_f(f));
    }
  }
}

template <int BM, int BN, bool AK, bool BKM, int EPI>
hipError_t launch_tiles(const KArgs& P, int batch, hipStream_t s) {
  dim3 grid(P.tiles_m * P.tiles_n, P.splits > 1 ? P.splits : batch);
  if (P.splits > 1) {
    gemm_bf16_kernel<BM, BN, AK, BKM, EPI, true><<<grid, THREADS, 0, s>>>(P);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int64_t total = P.M * P.N;
    int blocks = (int)std::min<int64_t>(cdiv(total, 256), 4096);
    splitk_reduce_kernel<EPI><<<blocks, 256, 0, s>>>(P);
  } else {
    gemm_bf16_kernel<BM, BN, AK, BKM, EPI, false><<<grid, THREADS, 0, s>>>(P);
  }
  return hipGetLastError();
}

template <int BM, int BN, int EPI>
hipError_t dispatch_layout(const Gemm& g, const KArgs& P, hipStream_t s) {
  if (g.a_kmajor && g.b_kmajor) return launch_tiles<BM, BN, true, true, EPI>(P, g.batch, s);
  if (g.a_kmajor && !g.b_kmajor) return launch_tiles<BM, BN, true, false, EPI>(P, g.batch, s);
  if (!g.a_kmajor && !g.b_kmajor) return launch_tiles<BM, BN, false, false, EPI>(P, g.batch, s);
  return launch_tiles<BM, BN, false, true, EPI>(P, g.batch, s);
}

template <int BM, int BN>
hipError_t dispatch_epi(const Gemm& g, const KArgs& P, hipStream_t s) {
  switch (g.epi) {
    case EPI_F32: return dispatch_layout<BM, BN, EPI_F32>(g, P, s);
    case EPI_BF16: return dispatch_layout<BM, BN, EPI_BF16>(g, P, s);
    case EPI_GELU: return dispatch_layout<BM, BN, EPI_GELU>(g, P, s);
    default: return dispatch_layout<BM, BN, EPI_DGELU>(g, P, s);
  }
}

}  // namespace

std::string gemm_check(const Gemm& g, bool f32_operands) {
  if (g.M < 0 || g.N < 0 || g.K < 0) return "negative GEMM dimension";
  if (g.batch < 1 || g.inner < 1) return "batch and inner must be >= 1";
  if (!g.A || !g.B || !g.C) return "null GEMM operand";
  if (g.epi == EPI_GELU && !g.C2) return "GELU epilogue needs a second output";
  if (g.epi == EPI_DGELU && !g.aux) return "GELU-backward epilogue needs the pre-activation";
  const int64_t a_contig0 = g.a_kmajor ? g.K : g.M;
  const int64_t b_contig0 = g.b_kmajor ? g.K : g.N;
  if (g.lda < a_contig0 || g.ldb < b_contig0 || g.ldc < g.N) return "leading dimension smaller than the row";
  if (f32_operands) return "";  // scalar loads: no alignment rules
  const int64_t q = 8;
  // contiguous dimension of each operand and all leading dims multiples of q
  const int64_t a_contig = g.a_kmajor ? g.K : g.M;
  const int64_t b_contig = g.b_kmajor ? g.K : g.N;
  if (a_contig % q || b_contig % q) return "contiguous GEMM dimensions must be multiples of 8 (bf16) / 4 (f32)";
  if (g.lda % q || g.ldb % q) return "leading dimensions of A and B must be multiples of 8 (bf16) / 4 (f32)";
  if (((uintptr_t)g.A | (uintptr_t)g.B) & 15) return "A and B must be 16-byte aligned";
  if ((g.a_outer | g.a_inner | g.b_outer | g.b_inner) % q) return "batch strides must keep 16-byte alignment";
  return "";
}

hipError_t launch_gemm_bf16(const Gemm& g, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  KArgs P;
  memset(&P, 0, sizeof(P));
  P.A = (const bf16_t*)g.A;
  P.B = (const bf16_t*)g.B;
  P.C = g.C;
  P.C2 = g.C2;
  P.aux = g.aux;
  P.bias = g.bias;
  P.M = g.M;
  P.N = g.N;
  P.K = g.K;
  P.lda = g.lda;
  P.ldb = g.ldb;
  P.ldc = g.ldc;
  P.a_outer = g.a_outer;
  P.a_inner = g.a_inner;
  P.b_outer = g.b_outer;
  P.b_inner = g.b_inner;
  P.c_outer = g.c_outer;
  P.c_inner = g.c_inner;
  P.inner = g.inner;
  P.splits = 1;
  const bool narrow = g.N <= 64;
  const int BM = 128, BN = narrow ? 64 : 128;
  P.tiles_m = (int)cdiv(g.M, BM);
  P.tiles_n = (int)cdiv(g.N, BN);
  const int64_t tiles = (int64_t)P.tiles_m * P.tiles_n * g.batch;
  // split-K when the output tiles cannot fill the machine and K is long
  if (g.batch == 1 && tiles < 240 && g.K >= 1024 && g.splitk_ws) {
    int splits = (int)std::min<int64_t>(std::max<int64_t>(1, 512 / tiles), g.K / 512);
    while (splits > 1 && (size_t)splits * g.M * g.N * 4 > g.splitk_ws_bytes) --splits;
    if (splits > 1) {
      P.splits = splits;
      P.k_per_split = cdiv(cdiv(g.K, splits), BK) * BK;
      P.splits = (int)cdiv(g.K, P.k_per_split);
      P.partial = g.splitk_ws;
    }
  }
  if (narrow) return dispatch_epi<128, 64>(g, P, s);
  return dispatch_epi<128, 128>(g, P, s);
}

}  // namespace layup
