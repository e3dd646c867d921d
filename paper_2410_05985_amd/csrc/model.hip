// The layer-wise LayUp step of one worker and the C ABI around it.
//
// Scheduling (LayUp Algorithm 1 and section 3.2): after the forward pass,
// units are visited from the output back to the input.  Unit u's backward
// runs on the compute stream and ends by recording the unit's event (the
// "notify" of Algorithm 1); the update stream waits for that event and runs
// the fused local update + peer average of unit u while the compute stream
// already runs unit u-1's backward.  A unit's backward reads only its own
// weights (which its own update has not touched yet), so the overlap has no
// hazard; the tied token embedding is updated last because its gradient is
// complete only after the embedding backward.  The next forward waits for
// the last update (join).
//
// Memory: every parameter-shaped buffer (params, grads, m, v, peers, bf16
// copy) is one flat caller-owned allocation with the layout built here, so
// a unit is one or two contiguous ranges and its update is one launch.
// Activations saved by the forward, gradient scratch and split-K partials
// live in one caller-owned workspace carved by the context.
#include <mutex>
#include <vector>

#include "layup_internal.h"

using namespace layup;

namespace {

thread_local std::string g_err;

struct TensorInfo {
  std::string name;
  int64_t off = 0, numel = 0;
  int rows = 0, cols = 1, padded_rows = 0, unit = 0, decay = 0;
};

struct Layout {
  std::vector<TensorInfo> t;
  int n_units = 0;
  int64_t total = 0;
  std::vector<std::vector<int>> unit_tensors;
};

int64_t align64(int64_t x) { return (x + 63) / 64 * 64; }

std::string check_config(const layup_config& c) {
  if (c.model == LAYUP_MODEL_MLP_F32) {
    if (c.n_mlp_layers < 1 || c.n_mlp_layers > LAYUP_MAX_MLP_LAYERS) return "n_mlp_layers out of range";
    for (int i = 0; i <= c.n_mlp_layers; ++i)
      if (c.mlp_dims[i] < 1) return "mlp_dims must be positive";
    if (c.batch < 1) return "batch must be >= 1";
  } else if (c.model == LAYUP_MODEL_GPT_BF16) {
    if (c.n_layer < 1 || c.d_model < 8 || c.n_head < 1 || c.d_ff < 8 || c.seq < 1 || c.vocab < 2 ||
        c.batch < 1)
      return "GPT dimensions must be positive";
    if (c.d_model % c.n_head) return "d_model must be a multiple of n_head";
    if ((c.d_model / c.n_head) % 8) return "head width must be a multiple of 8";
    if (c.d_model % 8 || c.d_ff % 8 || c.seq % 8) return "d_model, d_ff and seq must be multiples of 8";
    if (c.d_model > 2048) return "d_model above 2048 is not supported";
    if ((int64_t)c.batch * c.seq > 8192) return "batch*seq above 8192 is not supported";
    if (c.vocab >= (1 << 17)) return "vocab must be below 131072";
  } else {
    return "unknown model kind";
  }
  if (c.n_peers < 1) return "n_peers must be >= 1";
  return "";
}

Layout build_layout(const layup_config& c) {
  Layout L;
  auto add = [&](const std::string& n, int rows, int cols, int unit, int decay, int padded = 0) {
    TensorInfo ti;
    ti.name = n;
    ti.rows = rows;
    ti.cols = cols;
    ti.padded_rows = padded ? padded : rows;
    ti.numel = (int64_t)rows * cols;
    ti.unit = unit;
    ti.decay = decay;
    ti.off = L.total;
    L.total = align64(L.total + (int64_t)ti.padded_rows * cols);
    L.t.push_back(ti);
  };
  if (c.model == LAYUP_MODEL_MLP_F32) {
    L.n_units = c.n_mlp_layers;
    for (int i = 0; i < c.n_mlp_layers; ++i) {
      add("fc" + std::to_string(i + 1) + ".w", c.mlp_dims[i + 1], c.mlp_dims[i], i, 1);
      add("fc" + std::to_string(i + 1) + ".b", c.mlp_dims[i + 1], 1, i, 1);
    }
  } else {
    const int d = c.d_model, f = c.d_ff;
    L.n_units = c.n_layer + 2;
    add("wpe", c.seq, d, 0, 1);
    add("wte", c.vocab, d, 0, 1, (int)align64(c.vocab));
    for (int l = 0; l < c.n_layer; ++l) {
      const std::string p = "h" + std::to_string(l) + ".";
      const int u = l + 1;
      add(p + "qkv.w", 3 * d, d, u, 1);
      add(p + "proj.w", d, d, u, 1);
      add(p + "fc.w", f, d, u, 1);
      add(p + "mproj.w", d, f, u, 1);
      add(p + "ln1.g", d, 1, u, 0);
      add(p + "ln1.b", d, 1, u, 0);
      add(p + "qkv.b", 3 * d, 1, u, 0);
      add(p + "proj.b", d, 1, u, 0);
      add(p + "ln2.g", d, 1, u, 0);
      add(p + "ln2.b", d, 1, u, 0);
      add(p + "fc.b", f, 1, u, 0);
      add(p + "mproj.b", d, 1, u, 0);
    }
    add("lnf.g", d, 1, c.n_layer + 1, 0);
    add("lnf.b", d, 1, c.n_layer + 1, 0);
  }
  L.unit_tensors.resize(L.n_units);
  for (int i = 0; i < (int)L.t.size(); ++i) L.unit_tensors[L.t[i].unit].push_back(i);
  return L;
}

// Workspace carving: a bump allocator over the caller's buffer.
struct Carver {
  char* base;
  size_t used = 0;
  template <class T>
  T* take(int64_t n) {
    used = (used + 255) / 256 * 256;
    T* p = base ? reinterpret_cast<T*>(base + used) : nullptr;
    used += (size_t)n * sizeof(T);
    return p;
  }
};

struct BlockActs {
  float *x, *h, *mean1, *rstd1, *mean2, *rstd2;
  bf16_t *a, *qkv, *P, *o, *a2, *f, *gl;  // P: softmax probabilities (unfused attention only)
  float* of;   // fused attention: float32 O (rowsum(dP P) = dO . O in the backward)
  float* lse;  // fused attention: base-2 log-sum-exp of each query's scaled scores
};

// Fused attention kernels cover head widths 32, 64 and 128; other widths use
// the score GEMM + softmax + GEMM kernels.
bool fused_attention(const layup_config& g) {
  return g.model == LAYUP_MODEL_GPT_BF16 && attention_fused_supported(g.d_model / g.n_head);
}

}  // namespace

struct layup_ctx {
  layup_config cfg;
  Layout L;
  layup_buffers buf;
  hipStream_t sc = nullptr, su = nullptr;
  std::vector<hipEvent_t> ev_unit;     // gradient of unit u ready (compute stream)
  std::vector<hipEvent_t> ev_applied;  // update+mix of unit u done (update stream)
  hipEvent_t ev_start = nullptr;       // start of the step's forward pass
  hipEvent_t ev_fwd_end = nullptr;     // end of the forward pass (loss gradient formed)
  hipEvent_t ev_join = nullptr;
  bool timeline_valid = false;
  // fused dW update (schedule LAYUP_SCHEDULE_FUSED_DW) of the step in flight
  bool fused_dw = false;
  layup_hparams fused_hp{};
  float fused_alpha = 0.f;
  const float* fused_peer = nullptr;
  // optional timing of the linear layers' backward GEMMs (events around each)
  bool gemm_timing = false;
  std::vector<hipEvent_t> gt_events;  // start/stop pairs
  int gt_used = 0;
  double gt_flops = 0.0;
  bool have_join = false;
  std::string err;
  int device = 0;
  // state machine of one step
  bool forward_done = false;
  int next_backward = -1;
  std::vector<char> backward_done;
  int32_t step_index = 0;  // value written to the trace
  bool dx_valid = false;   // dx[cur_dx] holds the input gradient of the last backwarded unit
  // workspace
  size_t ws_bytes = 0;
  std::vector<BlockActs> acts;
  float *xL = nullptr, *meanf = nullptr, *rstdf = nullptr;
  bf16_t* xf = nullptr;
  bf16_t* logits = nullptr;  // logits, then the logit gradient in place
  float* loss_rows = nullptr;
  uint32_t* sorted = nullptr;
  float* S = nullptr;       // scores, then dP
  bf16_t* dS = nullptr;      // unfused attention: score gradient
  float* att_D = nullptr;    // fused attention: rowsum(dP P) per query
  float* dx[2] = {nullptr, nullptr};
  float* dh = nullptr;
  float* da = nullptr;
  bf16_t* do16 = nullptr;
  // The operands a linear layer's dW GEMM and bias sum read (dY), double-
  // buffered by block parity: when the update stream differs from the
  // compute stream, those dW GEMMs and sums run on the update stream,
  // concurrently with the next layers' backward on the compute stream.
  //   dyA: bf16 of the block's output gradient (MLP output projection)
  //   dfb: GELU backward (MLP input projection)
  //   dyB: bf16 of the gradient after the attention residual (attention proj)
  //   dqb: dQ, dK, dV (qkv projection)
  bf16_t *dyA[2] = {nullptr, nullptr}, *dfb[2] = {nullptr, nullptr};
  bf16_t *dyB[2] = {nullptr, nullptr}, *dqb[2] = {nullptr, nullptr};
  // ev_mid[p]: the first half of block parity p's operands written (dfb, dyB;
  // compute stream) -- the others (dyA, dqb) are covered by the unit events;
  // ev_rd[k][p]: operand k's dW GEMM and bias sum done (update stream);
  hipEvent_t ev_mid[2] = {}, ev_rd[4][2] = {};
  hipEvent_t ev_head = nullptr;  // the head's dW done (update stream)
  hipEvent_t ev_sort = nullptr;  // the token sort done (update stream)
  hipEvent_t ev_fwd_half = nullptr;  // the forward's second half done (update stream)
  bool unit_recorded = false;  // the backward recorded its unit event itself
  float *ln_part = nullptr, *cs_part = nullptr;
  int64_t cs_part_floats = 0;
  ColsumScratch cs() const { return ColsumScratch{cs_part, cs_part_floats}; }
  float *splitk = nullptr, *splitk_su = nullptr;
  size_t splitk_bytes = 0, splitk_su_bytes = 0;
  bool dw_side() const { return su != sc; }
  float* dis_partial = nullptr;
  // MLP
  std::vector<float*> mlp_act;  // input copy not kept: act[0] = x pointer of the step
  float *mlp_dz = nullptr, *mlp_dh = nullptr;
  const float* mlp_x = nullptr;
  const int32_t* tokens = nullptr;
  int cur_dx = 0;
};

namespace {

constexpr size_t SPLITK_BYTES = 256u << 20;  // room for an 8-way split of an 8192 x 768 float32 output
constexpr size_t SPLITK_SU_BYTES = 128u << 20;  // split-K of the dW GEMMs on the update stream

size_t carve(layup_ctx* c, char* base) {
  Carver cv{base};
  const layup_config& g = c->cfg;
  if (g.model == LAYUP_MODEL_GPT_BF16) {
    const int64_t N = (int64_t)g.batch * g.seq, d = g.d_model, F = g.d_ff, H = g.n_head, T = g.seq;
    const int64_t Vp = align64(g.vocab);
    const bool fused = fused_attention(g);
    c->acts.assign(g.n_layer, BlockActs{});
    for (int l = 0; l < g.n_layer; ++l) {
      BlockActs& A = c->acts[l];
      A.x = cv.take<float>(N * d);
      A.h = cv.take<float>(N * d);
      A.mean1 = cv.take<float>(N);
      A.rstd1 = cv.take<float>(N);
      A.mean2 = cv.take<float>(N);
      A.rstd2 = cv.take<float>(N);
      A.a = cv.take<bf16_t>(N * d);
      A.qkv = cv.take<bf16_t>(N * 3 * d);
      A.P = fused ? nullptr : cv.take<bf16_t>(g.batch * H * T * T);
      A.o = cv.take<bf16_t>(N * d);
      A.a2 = cv.take<bf16_t>(N * d);
      A.f = cv.take<bf16_t>(N * F);
      A.gl = cv.take<bf16_t>(N * F);
      A.of = fused ? cv.take<float>(N * d) : nullptr;
      A.lse = fused ? cv.take<float>(g.batch * H * T) : nullptr;
    }
    c->xL = cv.take<float>(N * d);
    c->meanf = cv.take<float>(N);
    c->rstdf = cv.take<float>(N);
    c->xf = cv.take<bf16_t>(N * d);
    c->logits = cv.take<bf16_t>(N * Vp);
    c->loss_rows = cv.take<float>(N);
    c->sorted = cv.take<uint32_t>(N);
    c->S = fused ? nullptr : cv.take<float>(g.batch * H * T * T);
    c->dS = fused ? nullptr : cv.take<bf16_t>(g.batch * H * T * T);
    c->att_D = fused ? cv.take<float>(g.batch * H * T) : nullptr;
    c->dx[0] = cv.take<float>(N * d);
    c->dx[1] = cv.take<float>(N * d);
    c->dh = cv.take<float>(N * d);
    c->da = cv.take<float>(N * d);
    for (int q = 0; q < 2; ++q) {
      c->dyA[q] = cv.take<bf16_t>(N * d);
      c->dfb[q] = cv.take<bf16_t>(N * F);
      c->dyB[q] = cv.take<bf16_t>(N * d);
      c->dqb[q] = cv.take<bf16_t>(N * 3 * d);
    }
    c->do16 = cv.take<bf16_t>(N * d);
    c->ln_part = cv.take<float>(layernorm_bwd_partial_floats(N, (int)d));
    c->splitk = cv.take<float>(SPLITK_BYTES / 4);
    c->splitk_bytes = SPLITK_BYTES;
    c->splitk_su = cv.take<float>(SPLITK_SU_BYTES / 4);
    c->splitk_su_bytes = SPLITK_SU_BYTES;
  } else {
    const int n = g.n_mlp_layers;
    c->mlp_act.assign(n + 1, nullptr);
    for (int i = 1; i <= n; ++i) c->mlp_act[i] = cv.take<float>((int64_t)g.batch * g.mlp_dims[i]);
    int64_t wmax = 0;
    for (int i = 0; i <= n; ++i) wmax = std::max<int64_t>(wmax, g.mlp_dims[i]);
    c->mlp_dz = cv.take<float>(g.batch * wmax);
    c->mlp_dh = cv.take<float>(g.batch * wmax);
    c->loss_rows = cv.take<float>(g.batch);
    c->cs_part_floats = cdiv(g.batch, 128) * wmax;
    c->cs_part = cv.take<float>(c->cs_part_floats);
  }
  c->dis_partial = cv.take<float>(UM_MAX_BLOCKS);
  return cv.used + 256;
}

layup_status fail(layup_ctx* c, layup_status st, const std::string& msg) {
  if (c) c->err = msg;
  g_err = msg;
  return st;
}

layup_status hip_fail(layup_ctx* c, hipError_t e, const char* what) {
  return fail(c, LAYUP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIPCHK(c, expr, what)                     \
  do {                                            \
    hipError_t e_ = (expr);                       \
    if (e_ != hipSuccess) return hip_fail(c, e_, what); \
  } while (0)

const TensorInfo* find(const layup_ctx* c, const std::string& n) {
  for (const auto& t : c->L.t)
    if (t.name == n) return &t;
  return nullptr;
}

// pointers into the flat buffers
struct Flat {
  layup_ctx* c;
  float* p(const std::string& n) const { return c->buf.params + find(c, n)->off; }
  float* g(const std::string& n) const { return c->buf.grads + find(c, n)->off; }
  bf16_t* w16(const std::string& n) const { return c->buf.params_bf16 + find(c, n)->off; }
};

// dW GEMM of weight matrix `name`: writes the gradient (EPI_F32), or, in the
// fused schedule, applies the local update and peer average to the weight in
// its epilogue (EPI_UPDATE; the gradient is not stored).
Gemm dw_gemm(layup_ctx* c, Gemm g, const std::string& name) {
  if (!c->fused_dw) return g;
  const int64_t off = find(c, name)->off;
  g.epi = EPI_UPDATE;
  g.C = nullptr;
  g.upd = make_upd_args(c->fused_hp, c->fused_alpha, true);
  g.upd.p = c->buf.params + off;
  g.upd.m = c->buf.m + off;
  g.upd.v = c->buf.v ? c->buf.v + off : nullptr;
  g.upd.q = c->fused_peer + off;
  g.upd.p16 = c->buf.params_bf16 ? c->buf.params_bf16 + off : nullptr;
  return g;
}

Gemm mk(bool ak, bool bk, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* B,
        int64_t ldb, void* C, int64_t ldc, int epi) {
  Gemm g;
  g.a_kmajor = ak;
  g.b_kmajor = bk;
  g.M = M;
  g.N = N;
  g.K = K;
  g.A = A;
  g.lda = lda;
  g.B = B;
  g.ldb = ldb;
  g.C = C;
  g.ldc = ldc;
  g.epi = epi;
  return g;
}

// timed: one of a block's linear-layer backward GEMMs (dX or dW); with GEMM
// timing on, HIP events on its stream bracket the launch (and its split-K sum)
layup_status run_gemm(layup_ctx* c, Gemm g, hipStream_t s, const char* what, bool timed = false) {
  const bool side = s != c->sc;  // the update stream has a split-K workspace of its own
  g.splitk_ws = side ? c->splitk_su : c->splitk;
  g.splitk_ws_bytes = side ? c->splitk_su_bytes : c->splitk_bytes;
  std::string m = gemm_check(g, false);
  if (!m.empty()) return fail(c, LAYUP_ERR_SHAPE, std::string(what) + ": " + m);
  timed = timed && c->gemm_timing;
  if (timed) {
    if ((size_t)c->gt_used + 2 > c->gt_events.size()) {
      hipEvent_t e[2];
      if (hipEventCreate(&e[0]) != hipSuccess || hipEventCreate(&e[1]) != hipSuccess)
        return fail(c, LAYUP_ERR_HIP, "event creation failed");
      c->gt_events.push_back(e[0]);
      c->gt_events.push_back(e[1]);
    }
    HIPCHK(c, hipEventRecord(c->gt_events[c->gt_used], s), "GEMM timing event");
  }
  HIPCHK(c, launch_gemm_bf16(g, s), what);
  if (timed) {
    HIPCHK(c, hipEventRecord(c->gt_events[c->gt_used + 1], s), "GEMM timing event");
    c->gt_used += 2;
    c->gt_flops += 2.0 * (double)g.M * (double)g.N * (double)g.K * g.batch;
  }
  return LAYUP_OK;
}

#define TRY(x)                         \
  do {                                 \
    layup_status st_ = (x);            \
    if (st_ != LAYUP_OK) return st_;   \
  } while (0)

// ---------------------------------------------------------------- GPT
layup_status gpt_forward(layup_ctx* c, const int32_t* tokens, float* loss_out) {
  const layup_config& g = c->cfg;
  const hipStream_t s = c->sc;
  const int64_t B = g.batch, T = g.seq, N = B * T, d = g.d_model, F = g.d_ff, H = g.n_head,
                dh = d / H, Vp = align64(g.vocab);
  const float scale = 1.0f / sqrtf((float)dh);
  Flat fl{c};
  // The forward of sequences [b0, b0 + nb) on stream st, in three pieces
  // (embedding, block l, final LayerNorm + head + loss).  With an update
  // stream (idle during the forward) the batch is taken in two halves, the
  // second there, and the two halves' pieces are enqueued alternately so
  // that both streams have work from the start; every row's arithmetic is
  // the same either way.
  auto embed = [&](int64_t b0, int64_t nb, hipStream_t st) -> layup_status {
    const int64_t r0 = b0 * T;
    const int32_t* tk = tokens + b0 * (T + 1);
    HIPCHK(c, launch_embed_fwd(tk, fl.p("wte"), fl.p("wpe"), c->acts[0].x + r0 * d, (int)nb, (int)T, (int)d,
                               g.vocab, st), "embedding");
    return LAYUP_OK;
  };
  auto block = [&](int l, int64_t b0, int64_t nb, hipStream_t st) -> layup_status {
    const int64_t r0 = b0 * T, n = nb * T;
    {
      BlockActs& A = c->acts[l];
      const std::string p = "h" + std::to_string(l) + ".";
      float* x_next = ((l + 1 < g.n_layer) ? c->acts[l + 1].x : c->xL) + r0 * d;
      bf16_t* qkv = A.qkv + r0 * 3 * d;
      bf16_t* o = A.o + r0 * d;
      HIPCHK(c, launch_layernorm_fwd(A.x + r0 * d, fl.p(p + "ln1.g"), fl.p(p + "ln1.b"), A.a + r0 * d,
                                     A.mean1 + r0, A.rstd1 + r0, n, (int)d, st), "ln1");
      Gemm q = mk(true, true, n, 3 * d, d, A.a + r0 * d, d, fl.w16(p + "qkv.w"), d, qkv, 3 * d, EPI_BF16);
      q.bias = fl.p(p + "qkv.b");
      TRY(run_gemm(c, q, st, "qkv forward"));
      if (A.of) {
        HIPCHK(c, launch_attention_fwd(qkv, A.lse + b0 * H * T, o, A.of + r0 * d, (int)nb, (int)H, (int)T,
                                       (int)dh, scale, st), "attention");
      } else {
        // scores S[z] = Q_h K_h^T, z = b*H + h
        float* S = c->S + b0 * H * T * T;
        bf16_t* P = A.P + b0 * H * T * T;
        Gemm sg = mk(true, true, T, T, dh, qkv, 3 * d, qkv + d, 3 * d, S, T, EPI_F32);
        sg.batch = (int)(nb * H);
        sg.inner = (int)H;
        sg.a_outer = sg.b_outer = T * 3 * d;
        sg.a_inner = sg.b_inner = dh;
        sg.c_outer = H * T * T;
        sg.c_inner = T * T;
        sg.causal = CAUSAL_OUT_LOWER;
        TRY(run_gemm(c, sg, st, "scores"));
        HIPCHK(c, launch_softmax_fwd(S, P, nb * H, (int)T, scale, st), "softmax");
        // o_h = P V_h
        Gemm pv = mk(true, false, T, dh, T, P, T, qkv + 2 * d, 3 * d, o, d, EPI_BF16);
        pv.batch = (int)(nb * H);
        pv.inner = (int)H;
        pv.a_outer = H * T * T;
        pv.a_inner = T * T;
        pv.b_outer = T * 3 * d;
        pv.b_inner = dh;
        pv.c_outer = T * d;
        pv.c_inner = dh;
        pv.causal = CAUSAL_A_LOWER;
        TRY(run_gemm(c, pv, st, "attention output"));
      }
      Gemm pr = mk(true, true, n, d, d, o, d, fl.w16(p + "proj.w"), d, A.h + r0 * d, d, EPI_F32);
      pr.bias = fl.p(p + "proj.b");
      pr.aux = A.x + r0 * d;
      TRY(run_gemm(c, pr, st, "proj forward"));
      HIPCHK(c, launch_layernorm_fwd(A.h + r0 * d, fl.p(p + "ln2.g"), fl.p(p + "ln2.b"), A.a2 + r0 * d,
                                     A.mean2 + r0, A.rstd2 + r0, n, (int)d, st), "ln2");
      Gemm fc = mk(true, true, n, F, d, A.a2 + r0 * d, d, fl.w16(p + "fc.w"), d, A.f + r0 * F, F, EPI_GELU);
      fc.bias = fl.p(p + "fc.b");
      fc.C2 = A.gl + r0 * F;
      TRY(run_gemm(c, fc, st, "fc forward"));
      Gemm mp = mk(true, true, n, d, F, A.gl + r0 * F, F, fl.w16(p + "mproj.w"), F, x_next, d, EPI_F32);
      mp.bias = fl.p(p + "mproj.b");
      mp.aux = A.h + r0 * d;
      TRY(run_gemm(c, mp, st, "mproj forward"));
    }
    return LAYUP_OK;
  };
  auto tail = [&](int64_t b0, int64_t nb, hipStream_t st) -> layup_status {
    const int64_t r0 = b0 * T, n = nb * T;
    const int32_t* tk = tokens + b0 * (T + 1);
    HIPCHK(c, launch_layernorm_fwd(c->xL + r0 * d, fl.p("lnf.g"), fl.p("lnf.b"), c->xf + r0 * d, c->meanf + r0,
                                   c->rstdf + r0, n, (int)d, st), "lnf");
    Gemm hd = mk(true, true, n, Vp, d, c->xf + r0 * d, d, fl.w16("wte"), d, c->logits + r0 * Vp, Vp, EPI_BF16);
    TRY(run_gemm(c, hd, st, "head forward"));
    HIPCHK(c, launch_ce_fwd_bwd(c->logits + r0 * Vp, Vp, tk, (int)nb, (int)T, g.vocab, c->logits + r0 * Vp,
                                c->loss_rows + r0, nullptr, st, N), "cross-entropy");
    return LAYUP_OK;
  };
  const bool side = c->dw_side();
  const hipStream_t s2 = side ? c->su : s;
  // the update stream starts after everything the compute stream had done
  // when the step started (the previous step's updates and backward)
  if (side) HIPCHK(c, hipStreamWaitEvent(s2, c->ev_start, 0), "wait step start");
  // one stream: the whole batch at once (half-size products are less efficient)
  const int64_t nb0 = (side && B >= 2) ? B / 2 : B;
  const bool two = nb0 < B;
  TRY(embed(0, nb0, s));
  if (two) TRY(embed(nb0, B - nb0, s2));
  for (int l = 0; l < g.n_layer; ++l) {
    TRY(block(l, 0, nb0, s));
    if (two) TRY(block(l, nb0, B - nb0, s2));
  }
  TRY(tail(0, nb0, s));
  if (two) TRY(tail(nb0, B - nb0, s2));
  if (side) {
    HIPCHK(c, hipEventRecord(c->ev_fwd_half, s2), "record forward half");
    HIPCHK(c, hipStreamWaitEvent(s, c->ev_fwd_half, 0), "wait forward half");
  }
  if (loss_out) HIPCHK(c, launch_row_mean(c->loss_rows, N, loss_out, s), "loss mean");
  // the token positions sorted by token (for the embedding backward at the
  // end of the step): on the update stream, off the critical path (the
  // embedding backward waits for it); the previous step's embedding
  // backward, which read the list, finished before the step started
  HIPCHK(c, launch_token_sort(tokens, (int)B, (int)T, g.vocab, nullptr, (int32_t*)c->sorted, nullptr,
                              nullptr, nullptr, s2), "token sort");
  if (side) HIPCHK(c, hipEventRecord(c->ev_sort, s2), "record token sort");
  return LAYUP_OK;
}

layup_status gpt_backward(layup_ctx* c, int u) {
  const layup_config& g = c->cfg;
  const hipStream_t s = c->sc;
  const int64_t B = g.batch, T = g.seq, N = B * T, d = g.d_model, F = g.d_ff, H = g.n_head,
                dh = d / H, Vp = align64(g.vocab);
  const float scale = 1.0f / sqrtf((float)dh);
  Flat fl{c};
  // dW GEMMs and bias sums go to the update stream when it is a different
  // stream (sw); the events order them against the compute stream (s): an
  // operand is read there only after s wrote it, and s overwrites it only
  // after those reads (two blocks later, by parity)
  const bool side = c->dw_side();
  const hipStream_t sw = c->su;
  auto rec = [&](hipEvent_t e, hipStream_t st) { return side ? hipEventRecord(e, st) : hipSuccess; };
  auto wait = [&](hipStream_t st, hipEvent_t e) { return side ? hipStreamWaitEvent(st, e, 0) : hipSuccess; };
  enum { OP_A = 0, OP_F = 1, OP_B = 2, OP_Q = 3 };
  // The head's dW (the tied wte's gradient, needed only by the embedding
  // backward at the very end).  With a separate update stream it runs there
  // after the top block's dW GEMMs, filling that stream's slack instead of
  // taking 0.7 ms of the compute stream (measured: 1 % faster steps; next to
  // the head's dX, the two largest GEMMs of the step slowed each other, and
  // four vocabulary slices of it were slower than one GEMM).
  auto head_dw = [&](hipStream_t st) -> layup_status {
    Gemm dw = mk(false, false, Vp, d, N, c->logits, Vp, c->xf, d, fl.g("wte"), d, EPI_F32);
    return run_gemm(c, dw, st, "head dW");
  };
  if (u == g.n_layer + 1) {
    // output head (tied wte) and final LayerNorm
    Gemm dx = mk(true, false, N, d, Vp, c->logits, Vp, fl.w16("wte"), d, c->da, d, EPI_F32);
    TRY(run_gemm(c, dx, s, "head dX"));
    if (!side) TRY(head_dw(s));
    c->cur_dx = 0;
    const int q = (g.n_layer - 1) & 1;  // the last block's output-gradient operand
    HIPCHK(c, wait(s, c->ev_rd[OP_A][q]), "wait operand free");
    HIPCHK(c, launch_layernorm_bwd(c->da, c->xL, c->meanf, c->rstdf, fl.p("lnf.g"), nullptr,
                                   c->dx[0], c->dyA[q], c->ln_part, fl.g("lnf.g"), fl.g("lnf.b"), N,
                                   (int)d, s), "lnf backward");
    return LAYUP_OK;  // the unit event orders dyA for the update stream
  }
  if (u == 0) {
    HIPCHK(c, wait(s, c->ev_head), "wait head dW");  // the embedding adds into the wte gradient
    HIPCHK(c, wait(s, c->ev_sort), "wait token sort");
    HIPCHK(c, launch_embed_bwd(c->dx[c->cur_dx], (const int32_t*)c->sorted, fl.g("wte"), fl.g("wpe"),
                               (int)B, (int)T, (int)d, g.vocab, s), "embedding backward");
    return LAYUP_OK;
  }
  const int l = u - 1;
  const int pq = l & 1;
  const BlockActs& A = c->acts[l];
  const std::string p = "h" + std::to_string(l) + ".";
  float* dxo = c->dx[c->cur_dx];
  float* dxi = c->dx[c->cur_dx ^ 1];
  bf16_t *dyA = c->dyA[pq], *df16 = c->dfb[pq], *dyB = c->dyB[pq], *dq16 = c->dqb[pq];
  // Every linear layer: dX on the compute stream (the critical path), then
  // dW and db.  In the fused schedule the dW GEMM updates the weight in
  // place, so it must follow the layer's dX (which reads the weight first):
  // the MLP output projection's dW is issued after the event that follows
  // the MLP's dX GEMMs (ev_mid) and the attention projection's after the
  // unit event, the same events the other dW GEMMs wait for (an extra event
  // record per layer on the compute stream costs it a few microseconds of
  // idle time each).
  const bool fz = c->fused_dw;
  // The bias gradient (column sums of dY) comes out of the same dW GEMM: its
  // A operand is dY^T, whose row sums it accumulates from the fragments.
  auto weight_grads = [&](int op, Gemm dw, const std::string& wname, const char* bname,
                          const char* what) -> layup_status {
    dw.rowsum = fl.g(p + bname);
    TRY(run_gemm(c, dw_gemm(c, dw, wname), sw, what, true));
    HIPCHK(c, rec(c->ev_rd[op][pq], sw), "record operand read");
    return LAYUP_OK;
  };
  // MLP output projection: dY = dyA (written by the LayerNorm backward that produced dxo)
  Gemm dg = mk(true, false, N, F, d, dyA, d, fl.w16(p + "mproj.w"), F, df16, F, EPI_DGELU);
  dg.aux = A.f;
  HIPCHK(c, wait(s, c->ev_rd[OP_F][pq]), "wait operand free");
  TRY(run_gemm(c, dg, s, "mproj dX + gelu backward", true));
  // dyA was written before the previous unit event, which the update stream
  // has waited for
  const Gemm mproj_dw = mk(false, false, d, F, N, dyA, d, A.gl, F, fl.g(p + "mproj.w"), F, EPI_F32);
  if (!fz) TRY(weight_grads(OP_A, mproj_dw, p + "mproj.w", "mproj.b", "mproj dW + db"));
  // MLP input projection: dY = df16
  Gemm fcx = mk(true, false, N, d, F, df16, F, fl.w16(p + "fc.w"), d, c->da, d, EPI_F32);
  TRY(run_gemm(c, fcx, s, "fc dX", true));
  HIPCHK(c, wait(s, c->ev_rd[OP_B][pq]), "wait operand free");
  HIPCHK(c, launch_layernorm_bwd(c->da, A.h, A.mean2, A.rstd2, fl.p(p + "ln2.g"), dxo, c->dh,
                                 dyB, c->ln_part, fl.g(p + "ln2.g"), fl.g(p + "ln2.b"), N, (int)d,
                                 s), "ln2 backward");
  // one event for df16 and dyB (each event record on the compute stream
  // costs a few microseconds of idle time there)
  HIPCHK(c, rec(c->ev_mid[pq], s), "record operands written");
  HIPCHK(c, wait(sw, c->ev_mid[pq]), "wait operands written");
  if (fz) TRY(weight_grads(OP_A, mproj_dw, p + "mproj.w", "mproj.b", "mproj dW + db"));
  TRY(weight_grads(OP_F, mk(false, false, F, d, N, df16, F, A.a2, d, fl.g(p + "fc.w"), d, EPI_F32),
                   p + "fc.w", "fc.b", "fc dW + db"));
  // attention output projection: dY = dyB = bf16(dh) from the LayerNorm backward above
  Gemm prx = mk(true, false, N, d, d, dyB, d, fl.w16(p + "proj.w"), d, c->do16, d, EPI_BF16);
  TRY(run_gemm(c, prx, s, "proj dX", true));
  const Gemm proj_dw = mk(false, false, d, d, N, dyB, d, A.o, d, fl.g(p + "proj.w"), d, EPI_F32);
  if (!fz) TRY(weight_grads(OP_B, proj_dw, p + "proj.w", "proj.b", "proj dW + db"));
  HIPCHK(c, wait(s, c->ev_rd[OP_Q][pq]), "wait operand free");
  if (A.of) {
    // attention core, fused: dQ, dK, dV from recomputed scores (P and dS stay
    // in registers)
    HIPCHK(c, launch_attention_bwd(A.qkv, A.lse, c->do16, A.of, c->att_D, dq16, (int)B, (int)H,
                                   (int)T, (int)dh, scale, s), "attention backward");
  } else {
    // attention core, batched over z = b*H + h
    auto batched = [&](Gemm gm, int64_t ao, int64_t ai, int64_t bo, int64_t bi, int64_t co,
                       int64_t ci, int causal) {
      gm.causal = causal;
      gm.batch = (int)(B * H);
      gm.inner = (int)H;
      gm.a_outer = ao;
      gm.a_inner = ai;
      gm.b_outer = bo;
      gm.b_inner = bi;
      gm.c_outer = co;
      gm.c_inner = ci;
      return gm;
    };
    const int64_t TT = T * T;
    // dP = dO_h V_h^T
    TRY(run_gemm(c, batched(mk(true, true, T, T, dh, c->do16, d, A.qkv + 2 * d, 3 * d, c->S, T, EPI_F32),
                            T * d, dh, T * 3 * d, dh, H * TT, TT, CAUSAL_OUT_LOWER), s, "dP"));
    // dV_h = P^T dO_h
    TRY(run_gemm(c, batched(mk(false, false, T, dh, T, A.P, T, c->do16, d, dq16 + 2 * d, 3 * d,
                               EPI_BF16), H * TT, TT, T * d, dh, T * 3 * d, dh, CAUSAL_A_UPPER), s, "dV"));
    HIPCHK(c, launch_softmax_bwd(c->S, A.P, c->dS, B * H, (int)T, scale, s), "softmax backward");
    // dQ_h = dS K_h
    TRY(run_gemm(c, batched(mk(true, false, T, dh, T, c->dS, T, A.qkv + d, 3 * d, dq16, 3 * d,
                               EPI_BF16), H * TT, TT, T * 3 * d, dh, T * 3 * d, dh, CAUSAL_A_LOWER), s, "dQ"));
    // dK_h = dS^T Q_h
    TRY(run_gemm(c, batched(mk(false, false, T, dh, T, c->dS, T, A.qkv, 3 * d, dq16 + d, 3 * d,
                               EPI_BF16), H * TT, TT, T * 3 * d, dh, T * 3 * d, dh, CAUSAL_A_UPPER), s, "dK"));
  }
  // qkv projection: dY = dq16
  Gemm qx = mk(true, false, N, d, 3 * d, dq16, 3 * d, fl.w16(p + "qkv.w"), d, c->da, d, EPI_F32);
  TRY(run_gemm(c, qx, s, "qkv dX", true));
  // LayerNorm 1; its bf16 dx is the next block's output-gradient operand
  const int nq = pq ^ 1;
  if (l > 0) HIPCHK(c, wait(s, c->ev_rd[OP_A][nq]), "wait operand free");
  HIPCHK(c, launch_layernorm_bwd(c->da, A.x, A.mean1, A.rstd1, fl.p(p + "ln1.g"), c->dh, dxi,
                                 l > 0 ? c->dyA[nq] : nullptr, c->ln_part, fl.g(p + "ln1.g"),
                                 fl.g(p + "ln1.b"), N, (int)d,
                                 s), "ln1 backward");
  if (side) {
    // the unit event (compute stream's part of the unit done) also orders
    // dq16 and the next block's dyA for the update stream; the qkv dW GEMM
    // follows it there, ahead of the unit's update
    HIPCHK(c, hipEventRecord(c->ev_unit[u], s), "record unit event");
    HIPCHK(c, hipStreamWaitEvent(sw, c->ev_unit[u], 0), "wait unit event");
    c->unit_recorded = true;
  }
  if (fz) TRY(weight_grads(OP_B, proj_dw, p + "proj.w", "proj.b", "proj dW + db"));
  TRY(weight_grads(OP_Q, mk(false, false, 3 * d, d, N, dq16, 3 * d, A.a, d, fl.g(p + "qkv.w"), d, EPI_F32),
                   p + "qkv.w", "qkv.b", "qkv dW + db"));
  if (side && l == (int)g.n_layer - 1) {
    TRY(head_dw(sw));
    HIPCHK(c, rec(c->ev_head, sw), "record head dW done");
  }
  c->cur_dx ^= 1;
  return LAYUP_OK;
}

// ---------------------------------------------------------------- MLP
layup_status mlp_gemm(layup_ctx* c, Gemm g, const char* what) {
  std::string m = gemm_check(g, true);
  if (!m.empty()) return fail(c, LAYUP_ERR_SHAPE, std::string(what) + ": " + m);
  HIPCHK(c, launch_gemm_f32(g, c->sc), what);
  return LAYUP_OK;
}

layup_status mlp_forward(layup_ctx* c, const int32_t* labels, const float* x, float* loss_out) {
  const layup_config& g = c->cfg;
  const int n = g.n_mlp_layers, Bt = g.batch;
  Flat fl{c};
  c->mlp_x = x;
  const float* h = x;
  for (int i = 0; i < n; ++i) {
    const std::string p = "fc" + std::to_string(i + 1) + ".";
    const int in = g.mlp_dims[i], out = g.mlp_dims[i + 1];
    Gemm gm = mk(true, true, Bt, out, in, h, in, fl.p(p + "w"), in, c->mlp_act[i + 1], out, EPI_F32);
    gm.bias = fl.p(p + "b");
    TRY(mlp_gemm(c, gm, "mlp forward"));
    if (i + 1 < n) HIPCHK(c, launch_relu_inplace(c->mlp_act[i + 1], (int64_t)Bt * out, c->sc), "relu");
    h = c->mlp_act[i + 1];
  }
  HIPCHK(c, launch_ce_f32(c->mlp_act[n], labels, Bt, g.mlp_dims[n], c->mlp_dz, c->loss_rows, loss_out,
                          c->sc), "cross-entropy");
  return LAYUP_OK;
}

layup_status mlp_backward(layup_ctx* c, int u) {
  const layup_config& g = c->cfg;
  const int Bt = g.batch, in = g.mlp_dims[u], out = g.mlp_dims[u + 1];
  Flat fl{c};
  const std::string p = "fc" + std::to_string(u + 1) + ".";
  const float* hin = u == 0 ? c->mlp_x : c->mlp_act[u];
  TRY(mlp_gemm(c, mk(false, false, out, in, Bt, c->mlp_dz, out, hin, in, fl.g(p + "w"), in, EPI_F32),
               "mlp dW"));
  HIPCHK(c, launch_colsum_f32(c->mlp_dz, Bt, out, out, c->cs(), fl.g(p + "b"), c->sc), "mlp db");
  if (u > 0) {
    TRY(mlp_gemm(c, mk(true, false, Bt, in, out, c->mlp_dz, out, fl.p(p + "w"), in, c->mlp_dh, in,
                       EPI_F32), "mlp dX"));
    HIPCHK(c, launch_relu_bwd_inplace(c->mlp_dh, c->mlp_act[u], (int64_t)Bt * in, c->sc), "relu bwd");
    std::swap(c->mlp_dz, c->mlp_dh);
  }
  return LAYUP_OK;
}

// ------------------------------------------------------------ update+mix
// peer: flat buffer of the peer copy (a resident slot or a receiving
// replica); peer16: its bfloat16 copy (push mode, nullable).
void unit_tensors(layup_ctx* c, int u, float* peer, bf16_t* peer16, std::vector<UMTensor>& out) {
  out.clear();
  // fused schedule: a block's weight matrices were updated by their dW GEMMs
  const bool skip_mats = c->fused_dw && c->cfg.model == LAYUP_MODEL_GPT_BF16 && u >= 1 && u <= c->cfg.n_layer;
  for (int ti : c->L.unit_tensors[u]) {
    const TensorInfo& t = c->L.t[ti];
    if (skip_mats && t.decay) continue;
    if (!out.empty()) {
      UMTensor& last = out.back();
      if (last.decay == t.decay && last.p + last.n == c->buf.params + t.off) {
        last.n += t.numel;
        continue;
      }
    }
    UMTensor m;
    m.p = c->buf.params + t.off;
    m.g = c->buf.grads + t.off;
    m.m = c->buf.m + t.off;
    m.v = c->buf.v ? c->buf.v + t.off : nullptr;
    m.q = peer + t.off;
    m.p16 = c->buf.params_bf16 ? c->buf.params_bf16 + t.off : nullptr;
    m.q16 = peer16 ? peer16 + t.off : nullptr;
    m.n = t.numel;
    m.decay = t.decay;
    m.pad = 0;
    out.push_back(m);
  }
}

std::string check_hp(const layup_hparams* hp) {
  if (!hp) return "null hparams";
  if (hp->kind != LAYUP_SGD_MOMENTUM && hp->kind != LAYUP_ADAMW) return "unknown optimizer";
  if (hp->kind == LAYUP_ADAMW && hp->step < 1) return "AdamW step must be >= 1";
  if (!std::isfinite(hp->lr) || !std::isfinite(hp->weight_decay)) return "non-finite hyperparameter";
  return "";
}

// Update+mix of unit u against the peer copy `peer` (pull) or into the
// receiving replica `peer` (push).
layup_status unit_update(layup_ctx* c, int u, const layup_hparams* hp, float alpha, float* peer,
                         bf16_t* peer16, bool push, float* dis) {
  std::string m = check_hp(hp);
  if (!m.empty()) return fail(c, LAYUP_ERR_INVALID_ARG, m);
  if (u < 0 || u >= c->L.n_units) return fail(c, LAYUP_ERR_INVALID_ARG, "unit index out of range");
  if (hp->kind == LAYUP_ADAMW && !c->buf.v) return fail(c, LAYUP_ERR_INVALID_ARG, "AdamW needs the v buffer");
  if (!c->backward_done[u]) return fail(c, LAYUP_ERR_STATE, "unit updated before its backward");
  std::vector<UMTensor> ts;
  unit_tensors(c, u, peer, peer16, ts);
  HIPCHK(c, hipStreamWaitEvent(c->su, c->ev_unit[u], 0), "wait for unit gradient");
  TraceInfo tr;
  tr.trace = c->buf.trace;
  tr.counter = c->buf.trace_counter;
  tr.capacity = c->buf.trace_capacity;
  tr.step = c->step_index;
  tr.unit = u;
  for (size_t i = 0; i < ts.size(); i += UM_MAX_TENSORS) {
    int n = (int)std::min<size_t>(UM_MAX_TENSORS, ts.size() - i);
    TraceInfo t2 = tr;
    if (i > 0) t2.trace = nullptr;  // one trace entry per unit
    HIPCHK(c, launch_update_mix(&ts[i], n, *hp, alpha, (i == 0) ? dis : nullptr, c->dis_partial, t2, c->su,
                                push),
           "update+mix");
  }
  HIPCHK(c, hipEventRecord(c->ev_applied[u], c->su), "record unit applied");
  c->backward_done[u] = 0;
  if (u == 0) {
    HIPCHK(c, hipEventRecord(c->ev_join, c->su), "record join");
    c->have_join = true;
    c->timeline_valid = true;
    c->step_index++;
  }
  return LAYUP_OK;
}

float* slot_ptr(layup_ctx* c, int slot) {
  return const_cast<float*>(c->buf.peers) + (int64_t)slot * c->L.total;
}

// push target checks: a whole flat buffer of this configuration that is not
// one of the context's own
std::string check_push_target(layup_ctx* c, const float* peer, const uint16_t* peer16) {
  if (!peer) return "push mode needs the receiving replica's parameters";
  if ((uintptr_t)peer & 15) return "receiving replica must be 16-byte aligned";
  if ((uintptr_t)peer16 & 7) return "receiving replica's bf16 copy must be 8-byte aligned";
  const float* own = c->buf.params;
  if (peer < own + c->L.total && own < peer + c->L.total)
    return "receiving replica overlaps the worker's own parameters";
  return "";
}

// Update+mix of caller-described tensors (layup_layer_update_mix and its
// allocation-free variant): checks every tensor, then one launch per 16
// tensors.  part: the disagreement partial sums (one float per workgroup),
// part_floats of them.
// Checks caller-described tensors and converts them to kernel descriptors.
layup_status collect_tensors(layup_ctx* ctx, const layup_tensor* tensors, int32_t n_tensors,
                             const layup_hparams* hp, int32_t mix_mode, std::vector<UMTensor>& ts) {
  if (!tensors || n_tensors < 1) return fail(ctx, LAYUP_ERR_INVALID_ARG, "no tensors");
  if (mix_mode != LAYUP_MIX_PULL && mix_mode != LAYUP_MIX_PUSH)
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "unknown mix mode");
  const bool push = mix_mode == LAYUP_MIX_PUSH;
  std::string m = check_hp(hp);
  if (!m.empty()) return fail(ctx, LAYUP_ERR_INVALID_ARG, m);
  ts.assign(n_tensors, UMTensor{});
  for (int i = 0; i < n_tensors; ++i) {
    const layup_tensor& t = tensors[i];
    if (t.numel < 0) return fail(ctx, LAYUP_ERR_INVALID_ARG, "tensor " + std::to_string(i) + ": negative size");
    if (t.numel == 0) {  // nothing to read or write: the pointers are not used
      ts[i] = UMTensor{};
      continue;
    }
    if (!t.param || !t.grad || !t.state0 || !t.peer)
      return fail(ctx, LAYUP_ERR_INVALID_ARG, "tensor " + std::to_string(i) + ": null pointer");
    if (hp->kind == LAYUP_ADAMW && !t.state1)
      return fail(ctx, LAYUP_ERR_INVALID_ARG, "tensor " + std::to_string(i) + ": AdamW needs state1");
    uintptr_t al = (uintptr_t)t.param | (uintptr_t)t.grad | (uintptr_t)t.state0 | (uintptr_t)t.peer |
                   (uintptr_t)(hp->kind == LAYUP_ADAMW ? t.state1 : nullptr);
    if (al & 15) return fail(ctx, LAYUP_ERR_ALIGN, "tensor " + std::to_string(i) + ": pointers must be 16-byte aligned");
    if (((uintptr_t)t.param_bf16 | (uintptr_t)(push ? t.peer_bf16 : nullptr)) & 7)
      return fail(ctx, LAYUP_ERR_ALIGN, "tensor " + std::to_string(i) + ": bf16 copies must be 8-byte aligned");
    if ((const void*)t.param == (const void*)t.peer || (const void*)t.param == (const void*)t.grad)
      return fail(ctx, LAYUP_ERR_INVALID_ARG, "tensor " + std::to_string(i) + ": param aliases grad or peer");
    UMTensor& u = ts[i];
    u.p = t.param;
    u.g = t.grad;
    u.m = t.state0;
    u.v = hp->kind == LAYUP_ADAMW ? t.state1 : nullptr;
    u.q = t.peer;
    u.p16 = t.param_bf16;
    u.q16 = push ? t.peer_bf16 : nullptr;
    u.n = t.numel;
    u.decay = t.decay ? 1 : 0;
    u.pad = 0;
  }
  return LAYUP_OK;
}

layup_status tensors_update_mix(layup_ctx* ctx, const layup_tensor* tensors, int32_t n_tensors,
                                const layup_hparams* hp, float alpha, int32_t mix_mode,
                                float* disagreement, float* part, int64_t part_floats, hipStream_t s) {
  std::vector<UMTensor> ts;
  TRY(collect_tensors(ctx, tensors, n_tensors, hp, mix_mode, ts));
  const bool push = mix_mode == LAYUP_MIX_PUSH;
  if (disagreement && n_tensors > UM_MAX_TENSORS)
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "the disagreement output supports at most 16 tensors per call");
  // the launcher caps its grid at UM_MAX_BLOCKS workgroups, one partial each
  if (disagreement && (!part || part_floats < UM_MAX_BLOCKS))
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "disagreement scratch smaller than the update+mix grid");
  TraceInfo tr;
  for (int i = 0; i < n_tensors; i += UM_MAX_TENSORS) {
    int n = std::min(UM_MAX_TENSORS, n_tensors - i);
    hipError_t e = launch_update_mix(&ts[i], n, *hp, alpha, disagreement, part, tr, s, push);
    if (e != hipSuccess) return hip_fail(ctx, e, "update+mix");
  }
  return LAYUP_OK;
}

// Scratch of layup_layer_update_mix_static, for callers that cannot allocate
// device memory: the disagreement's per-workgroup partial sums.  Each GPU
// holds its own copy for the life of the process.  In host code the array's
// name is not a device address: its address on the current device comes from
// hipGetSymbolAddress, taken once per device and kept.
constexpr int64_t STATIC_SCRATCH_FLOATS = UM_MAX_BLOCKS;  // 64 KiB
static __device__ __align__(256) float scratch[STATIC_SCRATCH_FLOATS];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[MAX_DEVICES] = {};

// The current device's address of `scratch`; an error message on failure.
std::string static_scratch(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return std::string("hipGetDevice: ") + hipGetErrorString(e);
  if (dev < 0 || dev >= MAX_DEVICES) return "device index beyond the scratch table";
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return "";
}

}  // namespace

// ===================================================================== ABI
extern "C" {

const char* layup_global_error(void) { return g_err.c_str(); }

const char* layup_last_error(const layup_ctx* ctx) { return ctx ? ctx->err.c_str() : g_err.c_str(); }

layup_status layup_param_layout(const layup_config* cfg, int32_t* n_tensors, int32_t* n_units,
                                int64_t* total) {
  if (!cfg) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null config");
  std::string m = check_config(*cfg);
  if (!m.empty()) return fail(nullptr, LAYUP_ERR_SHAPE, m);
  Layout L = build_layout(*cfg);
  if (n_tensors) *n_tensors = (int32_t)L.t.size();
  if (n_units) *n_units = L.n_units;
  if (total) *total = L.total;
  return LAYUP_OK;
}

layup_status layup_tensor_layout(const layup_config* cfg, int32_t index, layup_tensor_info* out) {
  if (!cfg || !out) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null argument");
  std::string m = check_config(*cfg);
  if (!m.empty()) return fail(nullptr, LAYUP_ERR_SHAPE, m);
  Layout L = build_layout(*cfg);
  if (index < 0 || index >= (int)L.t.size()) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "tensor index out of range");
  const TensorInfo& t = L.t[index];
  memset(out, 0, sizeof(*out));
  strncpy(out->name, t.name.c_str(), sizeof(out->name) - 1);
  out->offset = t.off;
  out->numel = t.numel;
  out->rows = t.rows;
  out->cols = t.cols;
  out->padded_rows = t.padded_rows;
  out->unit = t.unit;
  out->decay = t.decay;
  return LAYUP_OK;
}

layup_status layup_workspace_size(const layup_config* cfg, size_t* bytes) {
  if (!cfg || !bytes) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null argument");
  std::string m = check_config(*cfg);
  if (!m.empty()) return fail(nullptr, LAYUP_ERR_SHAPE, m);
  layup_ctx tmp;
  tmp.cfg = *cfg;
  *bytes = carve(&tmp, nullptr);
  return LAYUP_OK;
}

layup_status layup_init(layup_ctx** out, const layup_config* cfg, const layup_buffers* bufs,
                        void* workspace, size_t workspace_bytes, void* compute_stream,
                        void* update_stream) {
  if (!out || !cfg || !bufs || !workspace) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  std::string m = check_config(*cfg);
  if (!m.empty()) return fail(nullptr, LAYUP_ERR_SHAPE, m);
  if (!bufs->params || !bufs->grads || !bufs->m || !bufs->peers)
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "params, grads, m and peers are required");
  if (cfg->model == LAYUP_MODEL_GPT_BF16 && !bufs->params_bf16)
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "the GPT model needs the bf16 parameter copy");
  if (bufs->trace && (!bufs->trace_counter || bufs->trace_capacity < 1))
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "trace needs a counter and a positive capacity");
  const uintptr_t al = (uintptr_t)bufs->params | (uintptr_t)bufs->grads | (uintptr_t)bufs->m |
                       (uintptr_t)bufs->v | (uintptr_t)bufs->peers | (uintptr_t)bufs->params_bf16;
  if (al & 15) return fail(nullptr, LAYUP_ERR_ALIGN, "flat buffers must be 16-byte aligned");
  if ((uintptr_t)workspace & 255) return fail(nullptr, LAYUP_ERR_ALIGN, "workspace must be 256-byte aligned");
  layup_ctx* c = new layup_ctx();
  c->cfg = *cfg;
  c->L = build_layout(*cfg);
  c->buf = *bufs;
  size_t need = carve(c, nullptr);
  if (workspace_bytes < need) {
    delete c;
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "workspace smaller than layup_workspace_size");
  }
  c->ws_bytes = carve(c, (char*)workspace);
  if (cfg->model == LAYUP_MODEL_GPT_BF16 && !fused_attention(*cfg)) {
    // probabilities and score gradients above the diagonal are zero and no
    // kernel writes them: clear both matrices once
    const size_t pm = (size_t)cfg->batch * cfg->n_head * cfg->seq * cfg->seq * sizeof(bf16_t);
    bool ok = true;
    for (auto& A : c->acts) ok = ok && hipMemsetAsync(A.P, 0, pm, (hipStream_t)compute_stream) == hipSuccess;
    ok = ok && hipMemsetAsync(c->dS, 0, pm, (hipStream_t)compute_stream) == hipSuccess;
    if (!ok) {
      delete c;
      return fail(nullptr, LAYUP_ERR_HIP, "clearing the attention matrices failed");
    }
  }
  c->sc = (hipStream_t)compute_stream;
  c->su = update_stream ? (hipStream_t)update_stream : c->sc;
  hipGetDevice(&c->device);
  c->ev_unit.assign(c->L.n_units, nullptr);
  c->ev_applied.assign(c->L.n_units, nullptr);
  c->backward_done.assign(c->L.n_units, 0);
  // unit events carry timestamps (the per-unit timeline); the join does not
  for (int u = 0; u < c->L.n_units; ++u) {
    if (hipEventCreate(&c->ev_unit[u]) != hipSuccess || hipEventCreate(&c->ev_applied[u]) != hipSuccess) {
      layup_destroy(c);
      return fail(nullptr, LAYUP_ERR_HIP, "event creation failed");
    }
  }
  if (hipEventCreate(&c->ev_start) != hipSuccess || hipEventCreate(&c->ev_fwd_end) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming) != hipSuccess) {
    layup_destroy(c);
    return fail(nullptr, LAYUP_ERR_HIP, "event creation failed");
  }
  // ordering events between the compute stream and the update stream's dW work
  bool ev_ok = hipEventCreateWithFlags(&c->ev_head, hipEventDisableTiming) == hipSuccess &&
          hipEventCreateWithFlags(&c->ev_sort, hipEventDisableTiming) == hipSuccess &&
          hipEventCreateWithFlags(&c->ev_fwd_half, hipEventDisableTiming) == hipSuccess;
  for (int q = 0; q < 2; ++q) {
    ev_ok = ev_ok && hipEventCreateWithFlags(&c->ev_mid[q], hipEventDisableTiming) == hipSuccess;
    for (int k = 0; k < 4; ++k)
      ev_ok = ev_ok && hipEventCreateWithFlags(&c->ev_rd[k][q], hipEventDisableTiming) == hipSuccess;
  }
  if (!ev_ok) {
    layup_destroy(c);
    return fail(nullptr, LAYUP_ERR_HIP, "event creation failed");
  }
  *out = c;
  return LAYUP_OK;
}

void layup_destroy(layup_ctx* ctx) {
  if (!ctx) return;
  for (auto e : ctx->ev_unit)
    if (e) hipEventDestroy(e);
  for (auto e : ctx->ev_applied)
    if (e) hipEventDestroy(e);
  for (auto e : ctx->gt_events) hipEventDestroy(e);
  if (ctx->ev_start) hipEventDestroy(ctx->ev_start);
  if (ctx->ev_fwd_end) hipEventDestroy(ctx->ev_fwd_end);
  if (ctx->ev_join) hipEventDestroy(ctx->ev_join);
  for (auto e : ctx->ev_mid)
    if (e) hipEventDestroy(e);
  for (auto& row : ctx->ev_rd)
    for (auto e : row)
      if (e) hipEventDestroy(e);
  if (ctx->ev_head) hipEventDestroy(ctx->ev_head);
  if (ctx->ev_sort) hipEventDestroy(ctx->ev_sort);
  if (ctx->ev_fwd_half) hipEventDestroy(ctx->ev_fwd_half);
  delete ctx;
}

layup_status layup_synchronize(layup_ctx* ctx) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  HIPCHK(ctx, hipStreamSynchronize(ctx->sc), "synchronize compute stream");
  HIPCHK(ctx, hipStreamSynchronize(ctx->su), "synchronize update stream");
  return LAYUP_OK;
}

layup_status layup_refresh_shadow(layup_ctx* ctx) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  if (!ctx->buf.params_bf16) return LAYUP_OK;
  if (ctx->have_join) HIPCHK(ctx, hipStreamWaitEvent(ctx->sc, ctx->ev_join, 0), "wait join");
  HIPCHK(ctx, launch_f32_to_bf16(ctx->buf.params, ctx->buf.params_bf16, ctx->L.total, ctx->sc),
         "bf16 copy");
  return LAYUP_OK;
}

layup_status layup_forward(layup_ctx* ctx, const int32_t* tokens, const float* x, float* loss_out) {
  if (!ctx || !tokens) return fail(ctx, LAYUP_ERR_INVALID_ARG, "null argument");
  if (ctx->cfg.model == LAYUP_MODEL_MLP_F32 && !x) return fail(ctx, LAYUP_ERR_INVALID_ARG, "the MLP needs x");
  if (ctx->cfg.model == LAYUP_MODEL_GPT_BF16 && x) return fail(ctx, LAYUP_ERR_INVALID_ARG, "the GPT takes no x");
  for (char b : ctx->backward_done)
    if (b) return fail(ctx, LAYUP_ERR_STATE, "forward called while a unit awaits its update");
  // the forward reads every unit's weights: wait for the previous step's updates
  if (ctx->have_join) HIPCHK(ctx, hipStreamWaitEvent(ctx->sc, ctx->ev_join, 0), "wait join");
  HIPCHK(ctx, hipEventRecord(ctx->ev_start, ctx->sc), "record step start");
  ctx->timeline_valid = false;
  ctx->dx_valid = false;
  ctx->tokens = tokens;
  layup_status st = ctx->cfg.model == LAYUP_MODEL_GPT_BF16 ? gpt_forward(ctx, tokens, loss_out)
                                                            : mlp_forward(ctx, tokens, x, loss_out);
  if (st != LAYUP_OK) return st;
  HIPCHK(ctx, hipEventRecord(ctx->ev_fwd_end, ctx->sc), "record forward end");
  ctx->forward_done = true;
  ctx->next_backward = ctx->L.n_units - 1;
  return LAYUP_OK;
}

layup_status layup_layer_backward(layup_ctx* ctx, int32_t unit) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  if (!ctx->forward_done) return fail(ctx, LAYUP_ERR_STATE, "backward before forward");
  if (unit != ctx->next_backward)
    return fail(ctx, LAYUP_ERR_STATE, "units must be backpropagated in reverse order, expected " +
                                          std::to_string(ctx->next_backward));
  ctx->unit_recorded = false;
  layup_status st = ctx->cfg.model == LAYUP_MODEL_GPT_BF16 ? gpt_backward(ctx, unit) : mlp_backward(ctx, unit);
  if (st != LAYUP_OK) return st;
  if (!ctx->unit_recorded) HIPCHK(ctx, hipEventRecord(ctx->ev_unit[unit], ctx->sc), "record unit event");
  if (ctx->dw_side()) {
    // the unit's gradients are complete once both streams' parts are: the
    // event is re-recorded on the update stream behind the compute stream's
    HIPCHK(ctx, hipStreamWaitEvent(ctx->su, ctx->ev_unit[unit], 0), "wait unit event");
    HIPCHK(ctx, hipEventRecord(ctx->ev_unit[unit], ctx->su), "record unit event");
  }
  ctx->backward_done[unit] = 1;
  ctx->dx_valid = ctx->cfg.model == LAYUP_MODEL_GPT_BF16 && unit >= 1;
  ctx->next_backward--;
  if (ctx->next_backward < 0) ctx->forward_done = false;
  return LAYUP_OK;
}

layup_status layup_unit_update_mix(layup_ctx* ctx, int32_t unit, const layup_hparams* hp, float alpha,
                                   int32_t peer_slot, float* disagreement) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  if (peer_slot < 0 || peer_slot >= ctx->cfg.n_peers)
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "peer slot out of range");
  return unit_update(ctx, unit, hp, alpha, slot_ptr(ctx, peer_slot), nullptr, false, disagreement);
}

layup_status layup_unit_update_push(layup_ctx* ctx, int32_t unit, const layup_hparams* hp, float alpha,
                                    float* peer_params, uint16_t* peer_params_bf16, float* disagreement) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  std::string m = check_push_target(ctx, peer_params, peer_params_bf16);
  if (!m.empty()) return fail(ctx, m.find("aligned") != std::string::npos ? LAYUP_ERR_ALIGN : LAYUP_ERR_INVALID_ARG, m);
  return unit_update(ctx, unit, hp, alpha, peer_params, peer_params_bf16, true, disagreement);
}

layup_status layup_layer_update_mix(layup_ctx* ctx, const layup_tensor* tensors, int32_t n_tensors,
                                    const layup_hparams* hp, float alpha, int32_t mix_mode,
                                    float* disagreement, void* stream) {
  if (disagreement && !ctx)
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "the disagreement output needs a context (its partial sums live in the workspace)");
  hipStream_t s = stream ? (hipStream_t)stream : (ctx ? ctx->su : nullptr);
  return tensors_update_mix(ctx, tensors, n_tensors, hp, alpha, mix_mode, disagreement,
                            ctx ? ctx->dis_partial : nullptr, UM_MAX_BLOCKS, s);
}

layup_status layup_layer_update_mix_static(const layup_tensor* tensors, int32_t n_tensors,
                                           const layup_hparams* hp, float alpha, int32_t mix_mode,
                                           float* disagreement, void* stream) {
  float* part = nullptr;
  if (disagreement && n_tensors > UM_MAX_TENSORS)
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "the disagreement output supports at most 16 tensors per call");
  if (disagreement && tensors && n_tensors >= 1) {
    std::string m = static_scratch(&part);
    if (!m.empty()) return fail(nullptr, LAYUP_ERR_HIP, m);
  }
  return tensors_update_mix(nullptr, tensors, n_tensors, hp, alpha, mix_mode, disagreement, part,
                            STATIC_SCRATCH_FLOATS, (hipStream_t)stream);
}

layup_status layup_units_update_mix(const layup_tensor* tensors, const int32_t* units, int32_t n_tensors,
                                    const layup_hparams* hp, float alpha, int32_t mix_mode, int32_t* trace,
                                    int32_t* trace_counter, int32_t trace_capacity, int32_t trace_step,
                                    void* stream) {
  std::vector<UMTensor> ts;
  TRY(collect_tensors(nullptr, tensors, n_tensors, hp, mix_mode, ts));
  if (!units) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null unit list");
  if (trace && (!trace_counter || trace_capacity < 1))
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "trace needs a counter and a positive capacity");
  // a unit's tensors are adjacent: a unit id that reappears after another unit is refused
  std::vector<int32_t> seen;
  for (int i = 0; i < n_tensors; ++i) {
    if (units[i] < 0 || units[i] >= (1 << 30)) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "unit id out of range");
    if (i > 0 && units[i] == units[i - 1]) continue;
    if (std::find(seen.begin(), seen.end(), units[i]) != seen.end())
      return fail(nullptr, LAYUP_ERR_INVALID_ARG, "the tensors of a unit must be adjacent");
    seen.push_back(units[i]);
  }
  const bool push = mix_mode == LAYUP_MIX_PUSH;
  const hipStream_t s = (hipStream_t)stream;
  TraceInfo tr;
  tr.trace = trace;
  tr.counter = trace_counter;
  tr.capacity = trace_capacity;
  tr.step = trace_step;
  int dummy = 0;
  const bool flat = update_mix_flat_layout(ts.data(), n_tensors, hp->kind == LAYUP_ADAMW, push, &dummy);
  // whole units, in order, grouped into launches of up to UMF_MAX_TENSORS
  // tensors (flat layout), else one unit at a time
  int i = 0;
  while (i < n_tensors) {
    int j = i;  // end of the group
    while (j < n_tensors) {
      int k = j + 1;
      while (k < n_tensors && units[k] == units[j]) ++k;  // end of unit at j
      if (flat && k - i <= UMF_MAX_TENSORS) {
        j = k;
        continue;
      }
      if (j == i) j = k;  // a unit alone
      break;
    }
    hipError_t e;
    if (flat && j - i <= UMF_MAX_TENSORS) {
      e = launch_update_mix_flat(&ts[i], units + i, j - i, *hp, alpha, tr, s, push);
    } else {
      // one unit: launches of up to 16 tensors, the trace entry with the first
      e = hipSuccess;
      for (int a = i; a < j && e == hipSuccess; a += UM_MAX_TENSORS) {
        TraceInfo t2 = tr;
        t2.unit = units[i];
        if (a > i) t2.trace = nullptr;
        e = launch_update_mix(&ts[a], std::min(UM_MAX_TENSORS, j - a), *hp, alpha, nullptr, nullptr, t2, s, push);
      }
    }
    if (e != hipSuccess) return hip_fail(nullptr, e, "update+mix of several units");
    i = j;
  }
  return LAYUP_OK;
}

layup_status layup_step_ex(layup_ctx* ctx, const layup_step_args* a) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  if (!a) return fail(ctx, LAYUP_ERR_INVALID_ARG, "null step arguments");
  std::string m = check_hp(a->hp);
  if (!m.empty()) return fail(ctx, LAYUP_ERR_INVALID_ARG, m);
  if (a->schedule != LAYUP_SCHEDULE_LAYERWISE && a->schedule != LAYUP_SCHEDULE_AFTER_BACKWARD &&
      a->schedule != LAYUP_SCHEDULE_FUSED_DW)
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "unknown schedule");
  const bool fused = a->schedule == LAYUP_SCHEDULE_FUSED_DW;
  if (fused && ctx->cfg.model != LAYUP_MODEL_GPT_BF16)
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "the fused dW schedule is for the GPT model");
  if (fused && (a->mix_mode != LAYUP_MIX_PULL || a->disagreement))
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "the fused dW schedule mixes in pull form and reports no disagreement");
  float* peer = nullptr;
  bf16_t* peer16 = nullptr;
  const bool push = a->mix_mode == LAYUP_MIX_PUSH;
  if (a->mix_mode == LAYUP_MIX_PULL) {
    if (a->peer_slot < 0 || a->peer_slot >= ctx->cfg.n_peers)
      return fail(ctx, LAYUP_ERR_INVALID_ARG, "peer slot out of range");
    peer = slot_ptr(ctx, a->peer_slot);
  } else if (push) {
    m = check_push_target(ctx, a->push_params, a->push_params_bf16);
    if (!m.empty()) return fail(ctx, m.find("aligned") != std::string::npos ? LAYUP_ERR_ALIGN : LAYUP_ERR_INVALID_ARG, m);
    peer = a->push_params;
    peer16 = a->push_params_bf16;
  } else {
    return fail(ctx, LAYUP_ERR_INVALID_ARG, "unknown mix mode");
  }
  TRY(layup_forward(ctx, a->tokens, a->x, a->loss_out));
  const int U = ctx->L.n_units;
  ctx->fused_dw = fused;
  ctx->fused_hp = *a->hp;
  ctx->fused_alpha = a->alpha;
  ctx->fused_peer = peer;
  struct Reset {
    layup_ctx* c;
    ~Reset() { c->fused_dw = false; }
  } reset{ctx};
  auto dis = [&](int u) { return a->disagreement ? a->disagreement + u : nullptr; };
  if (a->schedule != LAYUP_SCHEDULE_AFTER_BACKWARD) {
    for (int u = U - 1; u >= 0; --u) {
      TRY(layup_layer_backward(ctx, u));
      TRY(unit_update(ctx, u, a->hp, a->alpha, peer, peer16, push, dis(u)));
    }
  } else {
    for (int u = U - 1; u >= 0; --u) TRY(layup_layer_backward(ctx, u));
    // every update waits for the end of the whole backward pass (unit 0's
    // gradient is the last one produced)
    HIPCHK(ctx, hipStreamWaitEvent(ctx->su, ctx->ev_unit[0], 0), "wait for the end of the backward pass");
    for (int u = U - 1; u >= 0; --u) TRY(unit_update(ctx, u, a->hp, a->alpha, peer, peer16, push, dis(u)));
  }
  // join: the compute stream continues only after the last update
  HIPCHK(ctx, hipStreamWaitEvent(ctx->sc, ctx->ev_join, 0), "join");
  return LAYUP_OK;
}

layup_status layup_step(layup_ctx* ctx, const int32_t* tokens, const float* x, const layup_hparams* hp,
                        float alpha, int32_t peer_slot, float* loss_out, float* disagreement) {
  layup_step_args a;
  memset(&a, 0, sizeof(a));
  a.tokens = tokens;
  a.x = x;
  a.hp = hp;
  a.alpha = alpha;
  a.schedule = LAYUP_SCHEDULE_LAYERWISE;
  a.mix_mode = LAYUP_MIX_PULL;
  a.peer_slot = peer_slot;
  a.loss_out = loss_out;
  a.disagreement = disagreement;
  return layup_step_ex(ctx, &a);
}

layup_status layup_unit_timeline(layup_ctx* ctx, float* forward_ms, float* ready_ms, float* applied_ms) {
  if (!ctx || !ready_ms || !applied_ms) return fail(ctx, LAYUP_ERR_INVALID_ARG, "null argument");
  if (!ctx->timeline_valid) return fail(ctx, LAYUP_ERR_STATE, "no whole step has run since the last forward");
  TRY(layup_synchronize(ctx));
  if (forward_ms) HIPCHK(ctx, hipEventElapsedTime(forward_ms, ctx->ev_start, ctx->ev_fwd_end), "forward time");
  for (int u = 0; u < ctx->L.n_units; ++u) {
    HIPCHK(ctx, hipEventElapsedTime(&ready_ms[u], ctx->ev_start, ctx->ev_unit[u]), "unit ready time");
    HIPCHK(ctx, hipEventElapsedTime(&applied_ms[u], ctx->ev_start, ctx->ev_applied[u]), "unit applied time");
  }
  return LAYUP_OK;
}

layup_status layup_gemm_timing(layup_ctx* ctx, int32_t enable) {
  if (!ctx) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null context");
  TRY(layup_synchronize(ctx));
  ctx->gemm_timing = enable != 0;
  ctx->gt_used = 0;
  ctx->gt_flops = 0.0;
  return LAYUP_OK;
}

layup_status layup_gemm_timing_read(layup_ctx* ctx, float* total_ms, int32_t* launches, double* flops) {
  if (!ctx || !total_ms || !launches || !flops) return fail(ctx, LAYUP_ERR_INVALID_ARG, "null argument");
  TRY(layup_synchronize(ctx));
  float tot = 0.f;
  for (int i = 0; i < ctx->gt_used; i += 2) {
    float ms = 0.f;
    HIPCHK(ctx, hipEventElapsedTime(&ms, ctx->gt_events[i], ctx->gt_events[i + 1]), "GEMM timing");
    tot += ms;
  }
  *total_ms = tot;
  *launches = ctx->gt_used / 2;
  *flops = ctx->gt_flops;
  return LAYUP_OK;
}

layup_status layup_push_sum_send(double* w, int32_t n_workers, int32_t sender, int32_t receiver,
                                 float* alpha_out) {
  if (!w || !alpha_out) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null argument");
  if (n_workers < 2) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "push-sum needs at least two workers");
  if (sender < 0 || sender >= n_workers || receiver < 0 || receiver >= n_workers)
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "worker index out of range");
  if (sender == receiver) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "a worker does not send to itself");
  if (!(w[sender] > 0.0) || !(w[receiver] > 0.0) || !std::isfinite(w[sender]) || !std::isfinite(w[receiver]))
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "push-sum weights must be positive and finite");
  w[sender] *= 0.5;
  *alpha_out = (float)(w[sender] / (w[sender] + w[receiver]));
  return LAYUP_OK;
}

layup_status layup_push_sum_receive(double* w, int32_t n_workers, int32_t sender, int32_t receiver) {
  if (!w) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null argument");
  if (n_workers < 2) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "push-sum needs at least two workers");
  if (sender < 0 || sender >= n_workers || receiver < 0 || receiver >= n_workers)
    return fail(nullptr, LAYUP_ERR_INVALID_ARG, "worker index out of range");
  if (sender == receiver) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "a worker does not send to itself");
  w[receiver] += w[sender];
  return LAYUP_OK;
}

layup_status layup_activation(layup_ctx* ctx, int32_t which, int32_t layer, const void** ptr,
                              int64_t* numel, int32_t* dtype_out) {
  if (!ctx || !ptr) return fail(ctx, LAYUP_ERR_INVALID_ARG, "null argument");
  if (ctx->cfg.model != LAYUP_MODEL_GPT_BF16) return fail(ctx, LAYUP_ERR_DTYPE, "activations are exposed for the GPT model");
  const layup_config& g = ctx->cfg;
  const int64_t N = (int64_t)g.batch * g.seq, d = g.d_model, F = g.d_ff;
  const int64_t PT = (int64_t)g.batch * g.n_head * g.seq * g.seq;
  const bool per_layer = which <= 8 || which == 12;
  if (per_layer && (layer < 0 || layer >= g.n_layer)) return fail(ctx, LAYUP_ERR_INVALID_ARG, "layer out of range");
  const BlockActs* A = per_layer ? &ctx->acts[layer] : nullptr;
  const void* p = nullptr;
  int64_t n = 0;
  int dt = 0;
  switch (which) {
    case 0: p = A->x; n = N * d; dt = 0; break;
    case 1: p = A->a; n = N * d; dt = 1; break;
    case 2: p = A->qkv; n = N * 3 * d; dt = 1; break;
    case 3:
      if (!A->P) return fail(ctx, LAYUP_ERR_INVALID_ARG, "attention probabilities are not stored by the fused attention (head width 32, 64 or 128); its log-sum-exp is activation 12");
      p = A->P; n = PT; dt = 1; break;
    case 4: p = A->o; n = N * d; dt = 1; break;
    case 5: p = A->h; n = N * d; dt = 0; break;
    case 6: p = A->a2; n = N * d; dt = 1; break;
    case 7: p = A->f; n = N * F; dt = 1; break;
    case 8: p = A->gl; n = N * F; dt = 1; break;
    case 9: p = ctx->xf; n = N * d; dt = 1; break;
    case 10: p = ctx->logits; n = N * align64(g.vocab); dt = 1; break;
    case 11: p = ctx->xL; n = N * d; dt = 0; break;
    case 12:
      if (!A->lse) return fail(ctx, LAYUP_ERR_INVALID_ARG, "the log-sum-exp is stored by the fused attention only (head width 32, 64 or 128)");
      p = A->lse; n = (int64_t)g.batch * g.n_head * g.seq; dt = 0; break;
    case 13:
      if (!ctx->dx_valid)
        return fail(ctx, LAYUP_ERR_STATE, "no unit above the embeddings has been backpropagated since the forward");
      p = ctx->dx[ctx->cur_dx]; n = N * d; dt = 0; break;
    default: return fail(ctx, LAYUP_ERR_INVALID_ARG, "unknown activation");
  }
  *ptr = p;
  if (numel) *numel = n;
  if (dtype_out) *dtype_out = dt;
  return LAYUP_OK;
}

static layup_status gemm_abi(const layup_gemm_desc* d, void* stream, bool f32) {
  if (!d) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "null descriptor");
  Gemm g;
  g.a_kmajor = d->a_kmajor != 0;
  g.b_kmajor = d->b_kmajor != 0;
  g.M = d->M;
  g.N = d->N;
  g.K = d->K;
  g.A = d->A;
  g.lda = d->lda;
  g.B = d->B;
  g.ldb = d->ldb;
  g.C = d->C;
  g.ldc = d->ldc;
  g.bias = d->bias;
  g.batch = d->batch < 1 ? 1 : d->batch;
  g.inner = d->inner < 1 ? 1 : d->inner;
  g.a_outer = d->a_outer;
  g.a_inner = d->a_inner;
  g.b_outer = d->b_outer;
  g.b_inner = d->b_inner;
  g.c_outer = d->c_outer;
  g.c_inner = d->c_inner;
  g.epi = (f32 || d->c_f32) ? EPI_F32 : EPI_BF16;
  g.splitk_ws = (float*)d->workspace;
  g.splitk_ws_bytes = d->workspace_bytes;
  g.rowsum = d->a_rowsum;
  if (f32 && d->a_rowsum) return fail(nullptr, LAYUP_ERR_INVALID_ARG, "row sums of A only on the bf16 path");
  if (f32 && !d->c_f32) return fail(nullptr, LAYUP_ERR_DTYPE, "the float32 GEMM writes float32");
  if (f32 && g.batch != 1) return fail(nullptr, LAYUP_ERR_SHAPE, "the float32 GEMM is not batched");
  if (d->workspace && ((uintptr_t)d->workspace & 15)) return fail(nullptr, LAYUP_ERR_ALIGN, "workspace must be 16-byte aligned");
  std::string m = gemm_check(g, f32);
  if (!m.empty()) return fail(nullptr, m.find("aligned") != std::string::npos || m.find("multiple") != std::string::npos
                                           ? LAYUP_ERR_ALIGN : LAYUP_ERR_SHAPE, m);
  hipError_t e = f32 ? launch_gemm_f32(g, (hipStream_t)stream) : launch_gemm_bf16(g, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(nullptr, e, "gemm");
  return LAYUP_OK;
}

layup_status layup_gemm_bf16(const layup_gemm_desc* d, void* stream) { return gemm_abi(d, stream, false); }
layup_status layup_gemm_f32(const layup_gemm_desc* d, void* stream) { return gemm_abi(d, stream, true); }

}  // extern "C"
