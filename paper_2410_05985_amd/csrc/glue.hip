// Non-GEMM kernels of the GPT and MLP forward/backward: embedding gather and
// deterministic scatter, LayerNorm, causal softmax, cross-entropy, column
// sums (bias gradients), conversions.  All are HBM-bound elementwise or
// row-reduction kernels; math is float32 in registers, storage as the caller
// chooses (bf16 activations, f32 residual stream and gradients).  Every
// reduction has a fixed order, so results are bitwise reproducible.
#include "layup_internal.h"

namespace layup {

// ------------------------------------------------------------- embedding
// x[b,t,:] = wte[tokens[b, t], :] + wpe[t, :]; tokens has seq+1 columns.
// A token outside [0, V) gathers no embedding row (only the position row).
__global__ void embed_fwd_kernel(const int32_t* tokens, const float* wte, const float* wpe,
                                 float* x, int T, int d, int V) {
  const int row = blockIdx.x;  // b*T + t
  const int b = row / T, t = row % T;
  const int tok = tokens[(int64_t)b * (T + 1) + t];
  const bool ok = tok >= 0 && tok < V;
  const f32x4* e = reinterpret_cast<const f32x4*>(wte + (int64_t)(ok ? tok : 0) * d);
  const f32x4* p = reinterpret_cast<const f32x4*>(wpe + (int64_t)t * d);
  f32x4* o = reinterpret_cast<f32x4*>(x + (int64_t)row * d);
  for (int i = threadIdx.x; i < d / 4; i += blockDim.x) o[i] = ok ? e[i] + p[i] : p[i];
}

hipError_t launch_embed_fwd(const int32_t* tokens, const float* wte, const float* wpe, float* x,
                            int B, int T, int d, int V, hipStream_t s) {
  embed_fwd_kernel<<<B * T, 64, 0, s>>>(tokens, wte, wpe, x, T, d, V);
  return hipGetLastError();
}

// Sort the B*T (token, position) pairs by token, then position, in one
// workgroup (bitonic sort of packed 32-bit keys token<<14 | position in LDS).
// Positions with the same token are then contiguous and in increasing order.
constexpr int SORT_MAX = 8192;
// Tokens outside [0, V) get the sentinel V and are skipped by the scatter.
__global__ __launch_bounds__(1024) void token_sort_kernel(const int32_t* tokens, int B, int T,
                                                          int V, uint32_t* sorted) {
  __shared__ uint32_t key[SORT_MAX];
  const int n = B * T;
  int np = 1;
  while (np < n) np <<= 1;
  for (int i = threadIdx.x; i < np; i += blockDim.x) {
    if (i < n) {
      int b = i / T, t = i % T;
      int tok = tokens[(int64_t)b * (T + 1) + t];
      if (tok < 0 || tok >= V) tok = V;
      key[i] = ((uint32_t)tok << 14) | (uint32_t)i;
    } else {
      key[i] = 0xffffffffu;
    }
  }
  __syncthreads();
  for (int k = 2; k <= np; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < np; i += blockDim.x) {
        int ixj = i ^ j;
        if (ixj > i) {
          uint32_t a = key[i], c = key[ixj];
          bool up = (i & k) == 0;
          if ((a > c) == up) {
            key[i] = c;
            key[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < n; i += blockDim.x) sorted[i] = key[i];
}

hipError_t launch_token_sort(const int32_t* tokens, int B, int T, int V, int32_t* counts,
                             int32_t* sorted_pos, int32_t* seg_start, int32_t* seg_token,
                             int32_t* n_seg, hipStream_t s) {
  (void)counts; (void)seg_start; (void)seg_token; (void)n_seg;
  if (B * T > SORT_MAX || V >= (1 << 17)) return hipErrorInvalidValue;
  token_sort_kernel<<<1, 1024, 0, s>>>(tokens, B, T, V, reinterpret_cast<uint32_t*>(sorted_pos));
  return hipGetLastError();
}

// dwte[token] += sum over that token's positions (increasing) of dx[pos];
// one block per sorted slot, active only at the first slot of a token.
// dwpe[t] = sum over b (increasing) of dx[b, t]: blocks N.. N+T-1.
__global__ void embed_bwd_kernel(const float* dx, const uint32_t* sorted, float* dwte,
                                 float* dwpe, int B, int T, int d, int V) {
  const int n = B * T;
  const int i = blockIdx.x;
  if (i < n) {
    const uint32_t tok = sorted[i] >> 14;
    if (tok >= (uint32_t)V) return;
    if (i > 0 && (sorted[i - 1] >> 14) == tok) return;
    for (int c = threadIdx.x; c < d / 4; c += blockDim.x) {
      f32x4 acc = reinterpret_cast<const f32x4*>(dwte + (int64_t)tok * d)[c];
      for (int j = i; j < n && (sorted[j] >> 14) == tok; ++j) {
        const int pos = sorted[j] & 0x3fff;
        acc += reinterpret_cast<const f32x4*>(dx + (int64_t)pos * d)[c];
      }
      reinterpret_cast<f32x4*>(dwte + (int64_t)tok * d)[c] = acc;
    }
  } else {
    const int t = i - n;
    for (int c = threadIdx.x; c < d / 4; c += blockDim.x) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int b = 0; b < B; ++b) acc += reinterpret_cast<const f32x4*>(dx + ((int64_t)b * T + t) * d)[c];
      reinterpret_cast<f32x4*>(dwpe + (int64_t)t * d)[c] = acc;
    }
  }
}

hipError_t launch_embed_bwd(const float* dx, const int32_t* sorted_pos, float* dwte, float* dwpe,
                            int B, int T, int d, int V, hipStream_t s) {
  embed_bwd_kernel<<<B * T + T, 64, 0, s>>>(dx, reinterpret_cast<const uint32_t*>(sorted_pos), dwte,
                                            dwpe, B, T, d, V);
  return hipGetLastError();
}

// ------------------------------------------------------------- LayerNorm
// One wave64 per row, 4 rows per block.  y = (x - mean) * rstd * g + b in
// bf16; mean and rstd (1/sqrt(var + 1e-5), biased variance) kept for the
// backward.  The row is read once into registers (NVL float4 groups per
// lane, d <= 256*NVL); the mean and the variance are two passes over them.
template <int NVL>
__global__ __launch_bounds__(256) void layernorm_fwd_kernel(const float* x, const float* g,
                                                            const float* b, bf16_t* y,
                                                            float* mean, float* rstd,
                                                            int64_t rows, int d) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const f32x4* xr = reinterpret_cast<const f32x4*>(x + row * d);
  const int nv = d / 4;
  // the row, gain and bias are all requested before the first reduction
  f32x4 v[NVL], gg[NVL], bb[NVL];
#pragma unroll
  for (int j = 0; j < NVL; ++j) {
    const int i = lane + 64 * j;
    if (i < nv) {
      v[j] = xr[i];
      gg[j] = reinterpret_cast<const f32x4*>(g)[i];
      bb[j] = reinterpret_cast<const f32x4*>(b)[i];
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NVL; ++j)
    if (lane + 64 * j < nv) s += (v[j][0] + v[j][1]) + (v[j][2] + v[j][3]);
  const float mu = warp_sum(s) / d;
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NVL; ++j) {
    if (lane + 64 * j >= nv) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float c = v[j][e] - mu;
      ss = fmaf(c, c, ss);
    }
  }
  const float var = warp_sum(ss) / d;
  const float r = 1.0f / sqrtf(var + 1e-5f);
#pragma unroll
  for (int j = 0; j < NVL; ++j) {
    const int i = lane + 64 * j;
    if (i >= nv) continue;
    u32x2 o;
    o[0] = pack_bf2((v[j][0] - mu) * r * gg[j][0] + bb[j][0], (v[j][1] - mu) * r * gg[j][1] + bb[j][1]);
    o[1] = pack_bf2((v[j][2] - mu) * r * gg[j][2] + bb[j][2], (v[j][3] - mu) * r * gg[j][3] + bb[j][3]);
    reinterpret_cast<u32x2*>(y + row * d)[i] = o;
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = r;
  }
}

hipError_t launch_layernorm_fwd(const float* x, const float* g, const float* b, bf16_t* y,
                                float* mean, float* rstd, int64_t rows, int d, hipStream_t s) {
  if (d % 4 != 0 || d > 256 * 8 || rows <= 0) return hipErrorInvalidValue;
  const unsigned nb = (unsigned)cdiv(rows, 4);
  const int nvl = (int)cdiv(d / 4, 64);
  if (nvl <= 1) layernorm_fwd_kernel<1><<<nb, 256, 0, s>>>(x, g, b, y, mean, rstd, rows, d);
  else if (nvl == 2) layernorm_fwd_kernel<2><<<nb, 256, 0, s>>>(x, g, b, y, mean, rstd, rows, d);
  else if (nvl == 3) layernorm_fwd_kernel<3><<<nb, 256, 0, s>>>(x, g, b, y, mean, rstd, rows, d);
  else if (nvl == 4) layernorm_fwd_kernel<4><<<nb, 256, 0, s>>>(x, g, b, y, mean, rstd, rows, d);
  else layernorm_fwd_kernel<8><<<nb, 256, 0, s>>>(x, g, b, y, mean, rstd, rows, d);
  return hipGetLastError();
}

// LayerNorm backward.  dx = dres + r*(dxh - mean(dxh) - xh*mean(dxh*xh)) with
// xh = (x-mean)*r and dxh = dy*g.  A block of LN_WAVES waves takes LN_ROWS
// rows; wave w takes rows w, w + LN_WAVES, ... and loads its next row while it
// works on the current one, every operand of a row held in registers (NVL
// float4 groups per lane, d <= 256*NVL; wider rows are read twice, and the
// next-row prefetch is used while two rows fit in registers).  dg and db (column sums of dy*xh and
// dy) are summed per wave in row order, then over the waves in wave order,
// into one partial row per block; ln_partial_sum_kernel adds the partial rows
// in a fixed order.
constexpr int LN_WAVES = 8;
constexpr int LN_ROWS = 32;

struct LnRow {
  float mu, r;
};

template <int NVL>
__device__ __forceinline__ void ln_load_row(const float* dy, const float* x, const float* dres,
                                            const float* mean, const float* rstd, int64_t row,
                                            int d, int lane, f32x4 (&a)[NVL], f32x4 (&xv)[NVL],
                                            f32x4 (&o)[NVL], LnRow& st) {
  const int nv = d / 4;
  st.mu = mean[row];
  st.r = rstd[row];
#pragma unroll
  for (int j = 0; j < NVL; ++j) {
    const int i = lane + 64 * j;
    const f32x4 z{0.f, 0.f, 0.f, 0.f};
    a[j] = i < nv ? reinterpret_cast<const f32x4*>(dy + row * d)[i] : z;
    xv[j] = i < nv ? reinterpret_cast<const f32x4*>(x + row * d)[i] : z;
    o[j] = (dres && i < nv) ? reinterpret_cast<const f32x4*>(dres + row * d)[i] : z;
  }
}

template <int NVL>
__global__ __launch_bounds__(64 * LN_WAVES) void layernorm_bwd_kernel(
    const float* dy, const float* x, const float* mean, const float* rstd, const float* g,
    const float* dres, float* dx, bf16_t* dx16, float* part, int64_t rows, int d) {
  extern __shared__ f32x4 ln_red[];  // [2][LN_WAVES][nv]
  // HOLD: the row stays in registers between the two passes (else it is read
  // again, from cache); PF: the next row is loaded during the current one.
  constexpr bool HOLD = NVL <= 4, PF = NVL <= 3;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nv = d / 4;
  const float inv_d = 1.0f / (float)d;
  const f32x4 z{0.f, 0.f, 0.f, 0.f};
  f32x4 gg[NVL], ag[NVL], ab[NVL];
#pragma unroll
  for (int j = 0; j < NVL; ++j) {
    const int i = lane + 64 * j;
    gg[j] = i < nv ? reinterpret_cast<const f32x4*>(g)[i] : z;
    ag[j] = ab[j] = z;
  }
  const int64_t r0 = (int64_t)blockIdx.x * LN_ROWS + w;
  f32x4 a[HOLD ? NVL : 1], xv[HOLD ? NVL : 1], o[HOLD ? NVL : 1];
  LnRow st{0.f, 0.f};
  if constexpr (PF) {
    if (r0 < rows) ln_load_row<NVL>(dy, x, dres, mean, rstd, r0, d, lane, a, xv, o, st);
  }
#pragma unroll
  for (int k = 0; k < LN_ROWS / LN_WAVES; ++k) {
    const int64_t row = r0 + (int64_t)k * LN_WAVES;
    if (row >= rows) break;
    const f32x4* dyr = reinterpret_cast<const f32x4*>(dy + row * d);
    const f32x4* xr = reinterpret_cast<const f32x4*>(x + row * d);
    float s1 = 0.f, s2 = 0.f;
    if constexpr (HOLD) {
      if constexpr (!PF) ln_load_row<NVL>(dy, x, dres, mean, rstd, row, d, lane, a, xv, o, st);
      f32x4 a1[PF ? NVL : 1], x1[PF ? NVL : 1], o1[PF ? NVL : 1];
      LnRow st1{0.f, 0.f};
      const bool more = PF && k + 1 < LN_ROWS / LN_WAVES && row + LN_WAVES < rows;
      if constexpr (PF) {
        if (more) ln_load_row<NVL>(dy, x, dres, mean, rstd, row + LN_WAVES, d, lane, a1, x1, o1, st1);
      }
#pragma unroll
      for (int j = 0; j < NVL; ++j) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float xh = (xv[j][e] - st.mu) * st.r;
          const float dxh = a[j][e] * gg[j][e];
          s1 += dxh;
          s2 = fmaf(dxh, xh, s2);
          ag[j][e] = fmaf(a[j][e], xh, ag[j][e]);
          ab[j][e] += a[j][e];
        }
      }
      s1 = warp_sum(s1) * inv_d;
      s2 = warp_sum(s2) * inv_d;
#pragma unroll
      for (int j = 0; j < NVL; ++j) {
        const int i = lane + 64 * j;
        if (i >= nv) break;
        f32x4 v = o[j];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float xh = (xv[j][e] - st.mu) * st.r;
          v[e] += st.r * (a[j][e] * gg[j][e] - s1 - xh * s2);
        }
        reinterpret_cast<f32x4*>(dx + row * d)[i] = v;
        if (dx16) reinterpret_cast<u32x2*>(dx16 + row * d)[i] = u32x2{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
      }
      if constexpr (PF) {
        if (more) {
#pragma unroll
          for (int j = 0; j < NVL; ++j) {
            a[j] = a1[j];
            xv[j] = x1[j];
            o[j] = o1[j];
          }
          st = st1;
        }
      }
    } else {
      st.mu = mean[row];
      st.r = rstd[row];
#pragma unroll
      for (int j = 0; j < NVL; ++j) {
        const int i = lane + 64 * j;
        const f32x4 av = i < nv ? dyr[i] : z, xx = i < nv ? xr[i] : z;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float xh = (xx[e] - st.mu) * st.r;
          const float dxh = av[e] * gg[j][e];
          s1 += dxh;
          s2 = fmaf(dxh, xh, s2);
          ag[j][e] = fmaf(av[e], xh, ag[j][e]);
          ab[j][e] += av[e];
        }
      }
      s1 = warp_sum(s1) * inv_d;
      s2 = warp_sum(s2) * inv_d;
#pragma unroll
      for (int j = 0; j < NVL; ++j) {
        const int i = lane + 64 * j;
        if (i >= nv) break;
        const f32x4 av = dyr[i], xx = xr[i];
        f32x4 v = dres ? reinterpret_cast<const f32x4*>(dres + row * d)[i] : z;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float xh = (xx[e] - st.mu) * st.r;
          v[e] += st.r * (av[e] * gg[j][e] - s1 - xh * s2);
        }
        reinterpret_cast<f32x4*>(dx + row * d)[i] = v;
        if (dx16) reinterpret_cast<u32x2*>(dx16 + row * d)[i] = u32x2{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3])};
      }
    }
  }
  f32x4* red_g = ln_red;
  f32x4* red_b = ln_red + LN_WAVES * nv;
#pragma unroll
  for (int j = 0; j < NVL; ++j) {
    const int i = lane + 64 * j;
    if (i < nv) {
      red_g[w * nv + i] = ag[j];
      red_b[w * nv + i] = ab[j];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nv; i += 64 * LN_WAVES) {
    f32x4 sg = red_g[i], sb = red_b[i];
    for (int k = 1; k < LN_WAVES; ++k) {
      sg += red_g[k * nv + i];
      sb += red_b[k * nv + i];
    }
    // partial row of this block: [dg (d) | db (d)]
    reinterpret_cast<f32x4*>(part + (int64_t)blockIdx.x * 2 * d)[i] = sg;
    reinterpret_cast<f32x4*>(part + (int64_t)blockIdx.x * 2 * d + d)[i] = sb;
  }
}

// dg | db = the nb partial rows [nb][2d] summed in a fixed order.  A block
// covers 16 columns (4 float4 groups) with 64 row lanes: lane l adds rows l,
// l+64, ... in order (all of its loads in flight at once for nb <= 256), then
// the 64 lane sums are added pairwise in a fixed tree (lane l += lane l+h for
// h = 32, 16, ..., 1).  96 blocks for d = 768, so the pass is one memory
// round trip rather than a serial walk down the partial rows.
constexpr int LNP_COLS = 4;    // float4 column groups per block
constexpr int LNP_LANES = 64;  // row lanes per block
__global__ __launch_bounds__(LNP_COLS * LNP_LANES) void ln_partial_sum_kernel(const float* part, int64_t nb,
                                                                               int d, float* dg, float* db) {
  __shared__ f32x4 red[LNP_LANES][LNP_COLS];
  const int cg = threadIdx.x % LNP_COLS, rl = threadIdx.x / LNP_COLS;
  const int64_t cols = 2 * (int64_t)d;
  const int64_t c = ((int64_t)blockIdx.x * LNP_COLS + cg) * 4;
  f32x4 s{0.f, 0.f, 0.f, 0.f};
  if (c < cols) {
#pragma unroll 4
    for (int64_t r = rl; r < nb; r += LNP_LANES) s += *reinterpret_cast<const f32x4*>(part + r * cols + c);
  }
  red[rl][cg] = s;
  __syncthreads();
#pragma unroll
  for (int h = LNP_LANES / 2; h >= 1; h >>= 1) {
    if (rl < h) red[rl][cg] += red[rl + h][cg];
    __syncthreads();
  }
  if (rl == 0 && c < cols) {
    float* out = c < d ? dg + c : db + (c - d);
    *reinterpret_cast<f32x4*>(out) = red[0][cg];
  }
}

template <int NVL>
static hipError_t ln_bwd_launch(const float* dy, const float* x, const float* mean, const float* rstd,
                                const float* g, const float* dres, float* dx, bf16_t* dx16, float* part,
                                int64_t rows, int d, unsigned nb, hipStream_t s) {
  const size_t lds = (size_t)2 * LN_WAVES * (d / 4) * sizeof(f32x4);
  layernorm_bwd_kernel<NVL><<<nb, 64 * LN_WAVES, lds, s>>>(dy, x, mean, rstd, g, dres, dx, dx16, part,
                                                           rows, d);
  return hipGetLastError();
}

int64_t layernorm_bwd_partial_floats(int64_t rows, int d) { return cdiv(rows, LN_ROWS) * 2 * (int64_t)d; }

hipError_t launch_layernorm_bwd(const float* dy, const float* x, const float* mean,
                                const float* rstd, const float* g, const float* dres, float* dx,
                                bf16_t* dx16, float* part, float* dg, float* db, int64_t rows, int d,
                                hipStream_t s) {
  if (d % 4 != 0 || d > 256 * 8 || rows <= 0) return hipErrorInvalidValue;
  const unsigned nb = (unsigned)cdiv(rows, LN_ROWS);
  const int nvl = (int)cdiv(d / 4, 64);
  hipError_t e;
  if (nvl <= 1) e = ln_bwd_launch<1>(dy, x, mean, rstd, g, dres, dx, dx16, part, rows, d, nb, s);
  else if (nvl == 2) e = ln_bwd_launch<2>(dy, x, mean, rstd, g, dres, dx, dx16, part, rows, d, nb, s);
  else if (nvl == 3) e = ln_bwd_launch<3>(dy, x, mean, rstd, g, dres, dx, dx16, part, rows, d, nb, s);
  else if (nvl == 4) e = ln_bwd_launch<4>(dy, x, mean, rstd, g, dres, dx, dx16, part, rows, d, nb, s);
  else e = ln_bwd_launch<8>(dy, x, mean, rstd, g, dres, dx, dx16, part, rows, d, nb, s);
  if (e != hipSuccess) return e;
  ln_partial_sum_kernel<<<(unsigned)cdiv(2 * (int64_t)d, 4 * LNP_COLS), LNP_COLS * LNP_LANES, 0, s>>>(part, nb, d, dg,
                                                                                                 db);
  return hipGetLastError();
}

// ------------------------------------------------------------ column sums
// out[c] = sum over rows of x[r*ld + c] in a fixed order: stage 1 sums
// chunks of CS_ROWS rows (inside a chunk: rows r = l, l+8, ... per row lane
// l, then the 8 row lanes in order) into partial rows, stage 2 sums the
// partial rows in chunk order.  Stage 1 reads 16 bytes per thread per row,
// coalesced across the 32 column groups of a block.  Columns >= split go to
// out2[c - split] when out2 is given.
constexpr int CS_ROWS = 128;

template <typename T>
__device__ __forceinline__ void load_vec(const T* p, float* out);
template <>
__device__ __forceinline__ void load_vec<bf16_t>(const bf16_t* p, float* out) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __builtin_bit_cast(float, v[i] << 16);
    out[2 * i + 1] = __builtin_bit_cast(float, v[i] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void load_vec<float>(const float* p, float* out) {
  const f32x4 v = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = v[i];
}

template <typename T>
__global__ __launch_bounds__(256) void colsum_stage1(const T* x, int64_t rows, int64_t cols, int64_t ld,
                                                     float* partial) {
  constexpr int VEC = 16 / sizeof(T);
  __shared__ float red[8][32 * VEC];
  const int cg = threadIdx.x & 31, rl = threadIdx.x >> 5;
  const int64_t c0 = ((int64_t)blockIdx.x * 32 + cg) * VEC;
  const int64_t r0 = (int64_t)blockIdx.y * CS_ROWS;
  const int64_t r1 = min(rows, r0 + CS_ROWS);
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
  if (c0 < cols) {
    for (int64_t r = r0 + rl; r < r1; r += 8) {
      float v[VEC];
      load_vec<T>(x + r * ld + c0, v);
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += v[e];
    }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) red[rl][cg * VEC + e] = acc[e];
  __syncthreads();
  for (int i = threadIdx.x; i < 32 * VEC; i += 256) {
    const int64_t c = (int64_t)blockIdx.x * 32 * VEC + i;
    if (c >= cols) continue;
    float t = red[0][i];
    for (int l = 1; l < 8; ++l) t += red[l][i];
    partial[(int64_t)blockIdx.y * cols + c] = t;
  }
}

// Scalar stage 1 for narrow or unaligned inputs (the float32 MLP's 10 classes).
template <typename T>
__global__ void colsum_scalar(const T* x, int64_t rows, int64_t cols, int64_t ld, float* partial) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= cols) return;
  const int64_t r0 = (int64_t)blockIdx.y * CS_ROWS;
  const int64_t r1 = min(rows, r0 + CS_ROWS);
  float s = 0.f;
  for (int64_t r = r0; r < r1; ++r) {
    if constexpr (sizeof(T) == 2) s += bf2f(x[r * ld + c]);
    else s += x[r * ld + c];
  }
  partial[(int64_t)blockIdx.y * cols + c] = s;
}

// 64 columns x 4 chunk lanes per block: lane l sums chunks l, l+4, ... in
// order, then the four lane sums are added in lane order.
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* partial, int64_t chunks,
                                                           int64_t cols, float* out, float* out2,
                                                           int64_t split) {
  __shared__ float red[4][64];
  const int cl = threadIdx.x & 63, l = threadIdx.x >> 6;
  const int64_t c = (int64_t)blockIdx.x * 64 + cl;
  float s = 0.f;
  if (c < cols)
    for (int64_t k = l; k < chunks; k += 4) s += partial[k * cols + c];
  red[l][cl] = s;
  __syncthreads();
  if (l == 0 && c < cols) {
    const float t = (red[0][cl] + red[1][cl]) + (red[2][cl] + red[3][cl]);
    if (out2 && c >= split) out2[c - split] = t;
    else out[c] = t;
  }
}

template <typename T>
hipError_t colsum2(const T* x, int64_t rows, int64_t cols, int64_t ld, const ColsumScratch& cs,
                   float* out, float* out2, int64_t split, hipStream_t s) {
  constexpr int VEC = 16 / sizeof(T);
  const int64_t chunks = cdiv(rows, CS_ROWS);
  if (chunks > 65535 || chunks * cols > cs.partial_floats) return hipErrorInvalidValue;
  const bool vec = cols % VEC == 0 && ld % VEC == 0 && ((uintptr_t)x & 15) == 0;
  if (vec) {
    dim3 g1((unsigned)cdiv(cols, 32 * VEC), (unsigned)chunks);
    colsum_stage1<T><<<g1, 256, 0, s>>>(x, rows, cols, ld, cs.partial);
  } else {
    dim3 g1((unsigned)cdiv(cols, 256), (unsigned)chunks);
    colsum_scalar<T><<<g1, 256, 0, s>>>(x, rows, cols, ld, cs.partial);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  colsum_final_kernel<<<(unsigned)cdiv(cols, 64), 256, 0, s>>>(cs.partial, chunks, cols, out, out2, split);
  return hipGetLastError();
}

hipError_t launch_colsum_f32(const float* x, int64_t rows, int64_t cols, int64_t ld,
                             const ColsumScratch& cs, float* out, hipStream_t s) {
  return colsum2<float>(x, rows, cols, ld, cs, out, nullptr, 0, s);
}

// ------------------------------------------------------- causal softmax
// P[i, j] = exp(scale*S[i,j] - max) / sum for j <= i, 0 for j > i.  One wave64
// per row; 16-byte loads of S; only the unmasked part of S is read.
__global__ __launch_bounds__(256) void softmax_fwd_kernel(const float* S, bf16_t* P,
                                                          int64_t n_rows, int T, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int i = (int)(row % T);
  const f32x4* s = reinterpret_cast<const f32x4*>(S + row * T);
  u32x2* p = reinterpret_cast<u32x2*>(P + row * T);
  const int nv = i / 4 + 1;  // vectors holding columns 0..i
  float mx = -INFINITY;
  for (int v = lane; v < nv; v += 64) {
    const f32x4 x = s[v];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (4 * v + e <= i) mx = fmaxf(mx, x[e] * scale);
  }
  mx = warp_max(mx);
  float sum = 0.f;
  for (int v = lane; v < nv; v += 64) {
    const f32x4 x = s[v];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (4 * v + e <= i) sum += expf(x[e] * scale - mx);
  }
  sum = warp_sum(sum);
  const float inv = 1.0f / sum;
  for (int v = lane; v < T / 4; v += 64) {
    u32x2 o = {0u, 0u};
    if (v < nv) {
      const f32x4 x = s[v];
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = (4 * v + e <= i) ? expf(x[e] * scale - mx) * inv : 0.f;
      o[0] = pack_bf2(y[0], y[1]);
      o[1] = pack_bf2(y[2], y[3]);
    }
    p[v] = o;
  }
}

hipError_t launch_softmax_fwd(const float* S, bf16_t* P, int64_t n_mat, int T, float scale,
                              hipStream_t s) {
  if (T % 4) return hipErrorInvalidValue;
  const int64_t rows = n_mat * T;
  softmax_fwd_kernel<<<(unsigned)cdiv(rows, 4), 256, 0, s>>>(S, P, rows, T, scale);
  return hipGetLastError();
}

// dS[i, j] = scale * P[i,j] * (dP[i,j] - sum_k dP[i,k] P[i,k]); zero above
// the diagonal (P is zero there).  One wave64 per row, unmasked part read.
__global__ __launch_bounds__(256) void softmax_bwd_kernel(const float* dP, const bf16_t* P,
                                                          bf16_t* dS, int64_t n_rows, int T,
                                                          float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int i = (int)(row % T);
  const f32x4* dp = reinterpret_cast<const f32x4*>(dP + row * T);
  const u32x2* p = reinterpret_cast<const u32x2*>(P + row * T);
  u32x2* ds = reinterpret_cast<u32x2*>(dS + row * T);
  const int nv = i / 4 + 1;
  float acc = 0.f;
  for (int v = lane; v < nv; v += 64) {
    const f32x4 g = dp[v];
    const u32x2 pv = p[v];
    const float pe[4] = {__builtin_bit_cast(float, pv[0] << 16), __builtin_bit_cast(float, pv[0] & 0xffff0000u),
                         __builtin_bit_cast(float, pv[1] << 16), __builtin_bit_cast(float, pv[1] & 0xffff0000u)};
#pragma unroll
    for (int e = 0; e < 4; ++e) acc = fmaf(g[e], pe[e], acc);  // P is 0 beyond the diagonal
  }
  const float D = warp_sum(acc);
  for (int v = lane; v < T / 4; v += 64) {
    u32x2 o = {0u, 0u};
    if (v < nv) {
      const f32x4 g = dp[v];
      const u32x2 pv = p[v];
      const float pe[4] = {__builtin_bit_cast(float, pv[0] << 16), __builtin_bit_cast(float, pv[0] & 0xffff0000u),
                           __builtin_bit_cast(float, pv[1] << 16), __builtin_bit_cast(float, pv[1] & 0xffff0000u)};
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = scale * pe[e] * (g[e] - D);
      o[0] = pack_bf2(y[0], y[1]);
      o[1] = pack_bf2(y[2], y[3]);
    }
    ds[v] = o;
  }
}

hipError_t launch_softmax_bwd(const float* dP, const bf16_t* P, bf16_t* dS, int64_t n_mat, int T,
                              float scale, hipStream_t s) {
  if (T % 4) return hipErrorInvalidValue;
  const int64_t rows = n_mat * T;
  softmax_bwd_kernel<<<(unsigned)cdiv(rows, 4), 256, 0, s>>>(dP, P, dS, rows, T, scale);
  return hipGetLastError();
}

// ----------------------------------------------------------- cross-entropy
// Row r = b*T + t of the bf16 logits (logical vocabulary V, storage ld, a
// multiple of 8); target tokens[b, t+1].  loss_rows[r] = logsumexp(z) - z[y];
// dlogits = bf16((softmax(z) - onehot) / (B*T)) for columns < V, 0 beyond.
// Pass 1 keeps a running (max, sum of exp) per thread over 16-byte vectors,
// combined across the block in a fixed order; pass 2 writes the gradient
// (in place over the logits is allowed: each element is read before it is
// written, by the same thread).
__global__ __launch_bounds__(256) void ce_kernel(const bf16_t* z, int64_t ld, const int32_t* tokens,
                                                 int T, int V, int64_t n_rows, bf16_t* dz,
                                                 float* loss_rows) {
  __shared__ float rm[4], rs[4];
  const int64_t row = blockIdx.x;
  const int b = (int)(row / T), t = (int)(row % T);
  int tgt = tokens[(int64_t)b * (T + 1) + t + 1];
  const bool valid = tgt >= 0 && tgt < V;  // an invalid target adds no loss and no gradient
  if (!valid) tgt = 0;
  const u32x4* zr = reinterpret_cast<const u32x4*>(z + row * ld);
  const int nv = (int)(ld / 8);
  float m = -INFINITY, sum = 0.f;
  for (int v = threadIdx.x; v < nv; v += blockDim.x) {
    const u32x4 w = zr[v];
    float x[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[2 * k] = __builtin_bit_cast(float, w[k] << 16);
      x[2 * k + 1] = __builtin_bit_cast(float, w[k] & 0xffff0000u);
    }
    float lm = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (8 * v + e < V) lm = fmaxf(lm, x[e]);
    if (lm == -INFINITY) continue;
    const float mn = fmaxf(m, lm);
    float acc = sum * expf(m - mn);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (8 * v + e < V) acc += expf(x[e] - mn);
    m = mn;
    sum = acc;
  }
  // combine (m, sum) across lanes, then across the four waves, in fixed order
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o, 64), os = __shfl_xor(sum, o, 64);
    const float mn = fmaxf(m, om);
    sum = (m == -INFINITY ? 0.f : sum * expf(m - mn)) + (om == -INFINITY ? 0.f : os * expf(om - mn));
    m = mn;
  }
  if ((threadIdx.x & 63) == 0) {
    rm[threadIdx.x >> 6] = m;
    rs[threadIdx.x >> 6] = sum;
  }
  __syncthreads();
  float M = rm[0];
  for (int w = 1; w < 4; ++w) M = fmaxf(M, rm[w]);
  float Ssum = 0.f;
  for (int w = 0; w < 4; ++w) Ssum += rs[w] * expf(rm[w] - M);
  const float inv = 1.0f / Ssum;
  const float scale = 1.0f / (float)n_rows;
  const float zt = bf2f(z[row * ld + tgt]);
  __syncthreads();
  u32x4* dr = reinterpret_cast<u32x4*>(dz + row * ld);
  for (int v = threadIdx.x; v < nv; v += blockDim.x) {
    const u32x4 w = zr[v];
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float g[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int j = 8 * v + 2 * k + h;
        const float x = __builtin_bit_cast(float, h ? (w[k] & 0xffff0000u) : (w[k] << 16));
        g[h] = (j < V && valid) ? (expf(x - M) * inv - (j == tgt ? 1.0f : 0.0f)) * scale : 0.f;
      }
      o[k] = pack_bf2(g[0], g[1]);
    }
    dr[v] = o;
  }
  if (threadIdx.x == 0) loss_rows[row] = valid ? logf(Ssum) + M - zt : 0.0f;
}

__global__ void mean_kernel(const float* x, int64_t n, float* out) {
  __shared__ float red[16];
  float s = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) s += x[i];
  s = block_sum(s, red);
  if (threadIdx.x == 0) *out = s / (float)n;
}

// Register-resident form for rows of at most CE_T x CE_CH 16-byte vectors
// (V <= 53248; wider rows take ce_kernel): each of CE_T threads loads its
// vectors once (all loads in flight together), so the row is read from HBM
// once.  The maximum M is exact.  e^(z - M) is taken as 2^(z log2(e) - Ms)
// with Ms = M log2(e) rounded to float: one fused multiply-add and the
// hardware exponential per element; the rounding of Ms scales every term by
// the same factor c, which cancels in the probabilities and is removed from
// the loss (log c computed in double precision).  The sum is accumulated in
// double precision in a fixed order (per thread, a shuffle tree, the waves
// in order).  Only vectors that reach past V test each column.  The
// exponentials are taken again for the gradient; the target's -1 is
// applied by the one thread holding it.  Deterministic.
constexpr int CE_T = 512;
template <int CE_CH>
__global__ __launch_bounds__(CE_T) void ce_regs_kernel(const bf16_t* z, int64_t ld, const int32_t* tokens,
                                                       int T, int V, int64_t n_rows, bf16_t* dz,
                                                       float* loss_rows) {
  constexpr int NW = CE_T / 64;
  constexpr float L2E = 1.4426950408889634f;
  __shared__ float rmax[NW];
  __shared__ double rsum[NW];
  const int64_t row = blockIdx.x;
  const int b = (int)(row / T), t = (int)(row % T);
  int tgt = tokens[(int64_t)b * (T + 1) + t + 1];
  const bool valid = tgt >= 0 && tgt < V;  // an invalid target adds no loss and no gradient
  if (!valid) tgt = 0;
  const u32x4* zr = reinterpret_cast<const u32x4*>(z + row * ld);
  const int nv = (int)(ld / 8);
  const float zt = bf2f(z[row * ld + tgt]);
  u32x4 w[CE_CH];
#pragma unroll
  for (int c = 0; c < CE_CH; ++c) {
    const int v = threadIdx.x + CE_T * c;
    if (v < nv) w[c] = zr[v];
  }
  auto raw = [&](int c, int e) {  // element e of this thread's vector c
    const uint32_t u = w[c][e >> 1];
    return __builtin_bit_cast(float, (e & 1) ? (u & 0xffff0000u) : (u << 16));
  };
  float m = -INFINITY;
#pragma unroll
  for (int c = 0; c < CE_CH; ++c) {
    const int v = threadIdx.x + CE_T * c;
    if (v >= nv) continue;
    if (8 * v + 8 <= V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) m = fmaxf(m, raw(c, e));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * v + e < V) m = fmaxf(m, raw(c, e));
    }
  }
  m = warp_max(m);
  if ((threadIdx.x & 63) == 0) rmax[threadIdx.x >> 6] = m;
  __syncthreads();
  float M = rmax[0];
#pragma unroll
  for (int q = 1; q < NW; ++q) M = fmaxf(M, rmax[q]);
  const float Ms = M * L2E;
  // c * e^(z - M) for column j < V (bitwise the same in both uses), 0 past V
  auto prob = [&](int c, int e, bool full) {
    const int j = 8 * (threadIdx.x + CE_T * c) + e;
    const float p = __builtin_amdgcn_exp2f(fmaf(raw(c, e), L2E, -Ms));
    return (full || j < V) ? p : 0.f;
  };
  double sum = 0.0;
#pragma unroll
  for (int c = 0; c < CE_CH; ++c) {
    const int v = threadIdx.x + CE_T * c;
    if (v >= nv) continue;
    const bool full = 8 * v + 8 <= V;
#pragma unroll
    for (int e = 0; e < 8; ++e) sum += (double)prob(c, e, full);
  }
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
  if ((threadIdx.x & 63) == 0) rsum[threadIdx.x >> 6] = sum;
  __syncthreads();
  double S = 0.0;
#pragma unroll
  for (int q = 0; q < NW; ++q) S += rsum[q];
  const float scale = 1.0f / (float)n_rows;
  const float ks = (float)(1.0 / S) * scale;
  u32x4* dr = reinterpret_cast<u32x4*>(dz + row * ld);
  const int tv = tgt >> 3, te = tgt & 7;
#pragma unroll
  for (int c = 0; c < CE_CH; ++c) {
    const int v = threadIdx.x + CE_T * c;
    if (v >= nv) continue;
    const bool full = 8 * v + 8 <= V;
    float g[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) g[e] = valid ? prob(c, e, full) * ks : 0.f;
    if (valid && v == tv) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (e == te) g[e] -= scale;
    }
    dr[v] = u32x4{pack_bf2(g[0], g[1]), pack_bf2(g[2], g[3]), pack_bf2(g[4], g[5]), pack_bf2(g[6], g[7])};
  }
  if (threadIdx.x == 0) {
    // S = c * sum e^(z - M) with c = 2^(M log2(e) - Ms)
    const double log_c = ((double)M * 1.4426950408889634 - (double)Ms) * 0.6931471805599453;
    loss_rows[row] = valid ? (float)(log(S) - log_c + (double)M - (double)zt) : 0.0f;
  }
}

hipError_t launch_ce_fwd_bwd(const bf16_t* logits, int64_t ld, const int32_t* tokens, int B, int T,
                             int V, bf16_t* dlogits, float* loss_rows, float* loss_out,
                             hipStream_t s, int64_t mean_rows) {
  if (ld % 8 || ld < V) return hipErrorInvalidValue;
  const int64_t rows = (int64_t)B * T;
  const int64_t mr = mean_rows > 0 ? mean_rows : rows;  // rows of the mean the gradient is of
  const int64_t nv = ld / 8;
  if (nv <= CE_T * 4)
    ce_regs_kernel<4><<<(unsigned)rows, CE_T, 0, s>>>(logits, ld, tokens, T, V, mr, dlogits, loss_rows);
  else if (nv <= CE_T * 13)  // GPT-2's 50304-column logits
    ce_regs_kernel<13><<<(unsigned)rows, CE_T, 0, s>>>(logits, ld, tokens, T, V, mr, dlogits, loss_rows);
  else
    ce_kernel<<<(unsigned)rows, 256, 0, s>>>(logits, ld, tokens, T, V, mr, dlogits, loss_rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !loss_out) return e;
  mean_kernel<<<1, 1024, 0, s>>>(loss_rows, rows, loss_out);
  return hipGetLastError();
}

hipError_t launch_row_mean(const float* x, int64_t n, float* out, hipStream_t s) {
  mean_kernel<<<1, 1024, 0, s>>>(x, n, out);
  return hipGetLastError();
}

// float32 logits [rows, V] with labels: loss = mean(lse - z[y]),
// dz = (softmax - onehot) / rows.  One wave64 per row.
__global__ void ce_f32_kernel(const float* z, const int32_t* labels, int rows, int V, float* dz,
                              float* loss_rows) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float* zr = z + (int64_t)row * V;
  float mx = -INFINITY;
  for (int j = lane; j < V; j += 64) mx = fmaxf(mx, zr[j]);
  mx = warp_max(mx);
  float s = 0.f;
  for (int j = lane; j < V; j += 64) s += expf(zr[j] - mx);
  s = warp_sum(s);
  const int y = labels[row];
  const bool valid = y >= 0 && y < V;  // an invalid label adds no loss and no gradient
  for (int j = lane; j < V; j += 64)
    dz[(int64_t)row * V + j] = valid ? (expf(zr[j] - mx) / s - (j == y ? 1.f : 0.f)) / (float)rows : 0.f;
  if (lane == 0) loss_rows[row] = valid ? logf(s) + mx - zr[y] : 0.f;
}

hipError_t launch_ce_f32(const float* logits, const int32_t* labels, int rows, int V, float* dlogits,
                         float* loss_rows, float* loss_out, hipStream_t s) {
  ce_f32_kernel<<<(unsigned)cdiv(rows, 4), 256, 0, s>>>(logits, labels, rows, V, dlogits, loss_rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !loss_out) return e;
  mean_kernel<<<1, 256, 0, s>>>(loss_rows, rows, loss_out);
  return hipGetLastError();
}

// --------------------------------------------------------- elementwise
__global__ void f32_to_bf16_kernel(const float* x, bf16_t* y, int64_t n) {
  const int64_t n4 = n / 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * blockDim.x) {
    f32x4 v = reinterpret_cast<const f32x4*>(x)[i];
    u32x2 o;
    o[0] = pack_bf2(v[0], v[1]);
    o[1] = pack_bf2(v[2], v[3]);
    reinterpret_cast<u32x2*>(y)[i] = o;
  }
  for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    y[i] = f2bf(x[i]);
}

hipError_t launch_f32_to_bf16(const float* x, bf16_t* y, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  unsigned blocks = (unsigned)std::min<int64_t>(cdiv(n / 4 + 1, 256), 8192);
  f32_to_bf16_kernel<<<blocks, 256, 0, s>>>(x, y, n);
  return hipGetLastError();
}

__global__ void relu_kernel(float* x, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    x[i] = x[i] > 0.f ? x[i] : 0.f;
}

__global__ void relu_bwd_kernel(float* dy, const float* y, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dy[i] = y[i] > 0.f ? dy[i] : 0.f;
}

hipError_t launch_relu_inplace(float* x, int64_t n, hipStream_t s) {
  relu_kernel<<<(unsigned)std::min<int64_t>(cdiv(n, 256), 4096), 256, 0, s>>>(x, n);
  return hipGetLastError();
}

hipError_t launch_relu_bwd_inplace(float* dy, const float* y, int64_t n, hipStream_t s) {
  relu_bwd_kernel<<<(unsigned)std::min<int64_t>(cdiv(n, 256), 4096), 256, 0, s>>>(dy, y, n);
  return hipGetLastError();
}

}  // namespace layup
