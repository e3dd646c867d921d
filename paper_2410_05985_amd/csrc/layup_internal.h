// Internal declarations shared by the LayUp HIP translation units.
#pragma once
#include <math.h>
#include <string.h>

#include <algorithm>
#include <string>

#include "../../include/layup.h"
#include "common.h"

namespace layup {

// ------------------------------------------------------------ update+mix
constexpr int UM_MAX_TENSORS = 16;
constexpr int64_t UM_MAX_BLOCKS = 16384;  // grid cap; also the partial-sum scratch size

struct UMTensor {
  float* p;
  const float* g;
  float* m;
  float* v;
  float* q;      // peer copy: read (pull) or mixed in place (push)
  bf16_t* p16;   // bfloat16 copy of p (nullable)
  bf16_t* q16;   // push: bfloat16 copy of the peer (nullable)
  int64_t n;
  int32_t decay;
  int32_t pad;
};

struct TraceInfo {
  int32_t* trace = nullptr;
  int32_t* counter = nullptr;
  int32_t capacity = 0;
  int32_t step = 0;
  int32_t unit = 0;
};

// push = false: p <- (1-alpha) p1 + alpha q (the worker absorbs the peer);
// push = true:  p <- p1 and q <- (1-alpha) q + alpha p1 (the worker writes its
// update into the receiving replica), with p1 the locally updated layer.
hipError_t launch_update_mix(const UMTensor* ts, int n, const layup_hparams& hp, float alpha,
                             float* dis_out, float* dis_partial, const TraceInfo& tr,
                             hipStream_t stream, bool push = false);

// Several units whose gradients are all ready, in one launch: up to
// UMF_MAX_TENSORS tensors that share one flat layout (update_mix_flat_layout),
// listed unit by unit in the order the units are visited; units[i] is tensor
// i's unit.  One trace entry per unit (tr.unit unused).  No disagreement.
constexpr int UMF_MAX_TENSORS = 192;
bool update_mix_flat_layout(const UMTensor* ts, int n, bool adamw, bool push, int* base_index);
hipError_t launch_update_mix_flat(const UMTensor* ts, const int32_t* units, int n, const layup_hparams& hp,
                                  float alpha, const TraceInfo& tr, hipStream_t stream, bool push);

// ------------------------------------------------------------------ GEMM
enum Epilogue : int {
  EPI_F32 = 0,    // C(f32) = acc + bias (+ aux residual f32)
  EPI_BF16 = 1,   // C(bf16) = acc + bias
  EPI_GELU = 2,   // C(bf16) = acc + bias; C2(bf16) = gelu_tanh(acc + bias)
  EPI_DGELU = 3,  // C(bf16) = acc * gelu_tanh'(aux bf16)
  EPI_UPDATE = 4, // acc is dW: local update + peer average of the weight (no C)
};

// Local optimizer update + peer average of one weight matrix, applied by the
// dW GEMM (or its split-K sum) to the element it has just finished: the
// weight gradient never goes to HBM.  Weight, optimizer state and peer copy
// share the dW layout (row m, column n at m*ldc + n).
struct UpdArgs {
  float* p;
  float* m;
  float* v;        // AdamW only
  const float* q;  // peer copy (pull form)
  bf16_t* p16;     // bfloat16 copy of the weight
  int32_t adamw;
  float lr, mu, wd, b1, b2, eps, step_size, inv_sqrt_bc2, a, b, dfac, wdc;
};
// Scalars of the update for hyperparameters hp, mixing weight alpha and the
// tensor's decay flag (bias corrections in double precision on the host).
UpdArgs make_upd_args(const layup_hparams& hp, float alpha, bool decay);

// The element update shared by the fused dW epilogues (same arithmetic as the
// update+mix kernel: LibTorch SGD momentum or AdamW, then p <- a p1 + b q).
__device__ __forceinline__ void apply_update(const UpdArgs& U, int64_t off, float g) {
  float p = U.p[off], m = U.m[off], p1;
  if (U.adamw) {
    float v = U.v[off];
    const float pd = p * U.dfac;
    m = fmaf(U.b1, m, (1.0f - U.b1) * g);
    v = fmaf(U.b2, v, (1.0f - U.b2) * (g * g));
    const float den = fmaf(__builtin_amdgcn_sqrtf(v), U.inv_sqrt_bc2, U.eps);
    p1 = fmaf(-U.step_size, m * __builtin_amdgcn_rcpf(den), pd);
    U.v[off] = v;
  } else {
    const float gg = fmaf(U.wdc, p, g);
    m = fmaf(U.mu, m, gg);
    p1 = fmaf(-U.lr, m, p);
  }
  const float p2 = fmaf(U.a, p1, U.b * U.q[off]);
  U.p[off] = p2;
  U.m[off] = m;
  if (U.p16) U.p16[off] = f2bf(p2);
}

// Four consecutive elements with 128-bit accesses (off a multiple of 4 and
// every pointer 16-byte aligned; the bf16 copy 8-byte aligned).
__device__ __forceinline__ void apply_update4(const UpdArgs& U, int64_t off, f32x4 g) {
  f32x4 p = *reinterpret_cast<const f32x4*>(U.p + off), m = *reinterpret_cast<const f32x4*>(U.m + off);
  const f32x4 q = *reinterpret_cast<const f32x4*>(U.q + off);
  f32x4 p2;
  if (U.adamw) {
    f32x4 v = *reinterpret_cast<const f32x4*>(U.v + off);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float pd = p[e] * U.dfac;
      m[e] = fmaf(U.b1, m[e], (1.0f - U.b1) * g[e]);
      v[e] = fmaf(U.b2, v[e], (1.0f - U.b2) * (g[e] * g[e]));
      const float den = fmaf(__builtin_amdgcn_sqrtf(v[e]), U.inv_sqrt_bc2, U.eps);
      p2[e] = fmaf(U.a, fmaf(-U.step_size, m[e] * __builtin_amdgcn_rcpf(den), pd), U.b * q[e]);
    }
    *reinterpret_cast<f32x4*>(U.v + off) = v;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      m[e] = fmaf(U.mu, m[e], fmaf(U.wdc, p[e], g[e]));
      p2[e] = fmaf(U.a, fmaf(-U.lr, m[e], p[e]), U.b * q[e]);
    }
  }
  *reinterpret_cast<f32x4*>(U.p + off) = p2;
  *reinterpret_cast<f32x4*>(U.m + off) = m;
  if (U.p16) *reinterpret_cast<u32x2*>(U.p16 + off) = u32x2{pack_bf2(p2[0], p2[1]), pack_bf2(p2[2], p2[3])};
}

struct Gemm {
  bool a_kmajor = true, b_kmajor = true;
  int64_t M = 0, N = 0, K = 0;
  const void* A = nullptr;
  int64_t lda = 0;
  const void* B = nullptr;
  int64_t ldb = 0;
  void* C = nullptr;
  int64_t ldc = 0;
  void* C2 = nullptr;         // second output (EPI_GELU)
  const void* aux = nullptr;  // residual (EPI_F32) or pre-activation (EPI_DGELU), ld = ldc
  const float* bias = nullptr;
  int epi = EPI_F32;
  int batch = 1, inner = 1;
  int64_t a_outer = 0, a_inner = 0, b_outer = 0, b_inner = 0, c_outer = 0, c_inner = 0;
  float* splitk_ws = nullptr;  // float32 partials for split-K (batch 1 only)
  size_t splitk_ws_bytes = 0;
  // Causal structure of square attention products (M = N or M = K = T):
  //   CAUSAL_OUT_LOWER: only outputs with n <= m are needed (S, dP); tiles
  //     strictly above the diagonal are skipped and left unwritten.
  //   CAUSAL_A_LOWER: A(m, k) = 0 for k > m (P V, dS K): K stops at the tile's last row.
  //   CAUSAL_A_UPPER: A(m, k) = 0 for k < m (P^T dO, dS^T Q): K starts at the tile's first row.
  int causal = 0;
  UpdArgs upd{};  // EPI_UPDATE
  // m-major A only (dW = dY^T X): rowsum[m] = sum over k of A(m, k), the
  // bias gradient, accumulated from the A fragments the MFMAs consume
  float* rowsum = nullptr;
};
enum Causal : int { CAUSAL_NONE = 0, CAUSAL_OUT_LOWER = 1, CAUSAL_A_LOWER = 2, CAUSAL_A_UPPER = 3 };

// Validates shapes/alignment; returns a message or empty string.
std::string gemm_check(const Gemm& g, bool f32_operands);
hipError_t launch_gemm_bf16(const Gemm& g, hipStream_t stream);
// explicit tile configuration (0 = 256x256 K64, 1 = 128x128 K32, 2 = 128x64 K32, 3 = 128x128 K64,
// 4 = 256x256 K32 four stages, 5 = 256x128 K32)
hipError_t launch_gemm_bf16_cfg(const Gemm& g, int cfg, int splits, hipStream_t stream);
hipError_t launch_gemm_f32(const Gemm& g, hipStream_t stream);

// ------------------------------------------------------------ glue kernels
hipError_t launch_embed_fwd(const int32_t* tokens, const float* wte, const float* wpe, float* x,
                            int B, int T, int d, int V, hipStream_t s);
hipError_t launch_layernorm_fwd(const float* x, const float* g, const float* b, bf16_t* y,
                                float* mean, float* rstd, int64_t rows, int d, hipStream_t s);
// Scratch of the column sums: partial rows, ceil(rows/128) x cols floats.
struct ColsumScratch {
  float* partial;
  int64_t partial_floats;
};
// LayerNorm backward: dx (float32) and optionally its bfloat16 copy dx16;
// per-block partial sums of dg and db go to part
// (layernorm_bwd_partial_floats(rows, d) floats) and are added into dg, db
// in a fixed order.  d a multiple of 4, at most 2048.
int64_t layernorm_bwd_partial_floats(int64_t rows, int d);
hipError_t launch_layernorm_bwd(const float* dy, const float* x, const float* mean,
                                const float* rstd, const float* g, const float* dres,
                                float* dx, bf16_t* dx16, float* part, float* dg, float* db,
                                int64_t rows, int d, hipStream_t s);
hipError_t launch_softmax_fwd(const float* S, bf16_t* P, int64_t n_mat, int T, float scale,
                              hipStream_t s);
hipError_t launch_softmax_bwd(const float* dP, const bf16_t* P, bf16_t* dS, int64_t n_mat, int T,
                              float scale, hipStream_t s);
// Fused causal attention (head width 32, 64 or 128).  Forward: O (bf16),
// O in float32 and the base-2 log-sum-exp of each query's scaled scores
// (lse, [B][H][T]) from qkv.  Backward: dQ, dK, dV into the q, k, v columns
// of dqkv from qkv, lse, dO and the float32 O; D ([B][H][T]) receives
// rowsum(dP P) = dO . O.
bool attention_fused_supported(int dh);
hipError_t launch_attention_fwd(const bf16_t* qkv, float* lse, bf16_t* O, float* Of, int B, int H,
                                int T, int dh, float scale, hipStream_t s);
hipError_t launch_attention_bwd(const bf16_t* qkv, const float* lse, const bf16_t* dO, const float* Of,
                                float* D, bf16_t* dqkv, int B, int H, int T, int dh, float scale,
                                hipStream_t s);
// Cross-entropy over rows [B*T] of logits (row r = b*T + t predicts token
// t + 1 of sequence b) with its gradient written to dlogits (may alias the
// logits); the gradient is of the mean over mean_rows rows (0: the B*T rows
// of this call, so a batch can be taken in parts); loss_out, when given,
// receives the mean of this call's loss rows.
hipError_t launch_ce_fwd_bwd(const bf16_t* logits, int64_t ld, const int32_t* tokens, int B,
                             int T, int V, bf16_t* dlogits, float* loss_rows, float* loss_out,
                             hipStream_t s, int64_t mean_rows = 0);
hipError_t launch_row_mean(const float* x, int64_t n, float* out, hipStream_t s);
hipError_t launch_f32_to_bf16(const float* x, bf16_t* y, int64_t n, hipStream_t s);
hipError_t launch_colsum_f32(const float* x, int64_t rows, int64_t cols, int64_t ld,
                             const ColsumScratch& cs, float* out, hipStream_t s);
hipError_t launch_embed_bwd(const float* dx, const int32_t* sorted_pos, float* dwte, float* dwpe,
                            int B, int T, int d, int V, hipStream_t s);
hipError_t launch_token_sort(const int32_t* tokens, int B, int T, int V, int32_t* counts,
                             int32_t* sorted_pos, int32_t* seg_start, int32_t* seg_token,
                             int32_t* n_seg, hipStream_t s);
hipError_t launch_relu_bwd_inplace(float* dy, const float* y, int64_t n, hipStream_t s);
hipError_t launch_relu_inplace(float* x, int64_t n, hipStream_t s);
hipError_t launch_ce_f32(const float* logits, const int32_t* labels, int rows, int V,
                         float* dlogits, float* loss_rows, float* loss_out, hipStream_t s);

}  // namespace layup
