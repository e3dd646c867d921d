// Fused local update + gossip mix, one HBM pass (LayUp Algorithm 1, "Local
// Update" followed by "Peer Update").
//
// Per element, SGD momentum (LibTorch semantics, coupled decay):
//   g' = g + wd*p;  m = mu*m + g';  p1 = p - lr*m
// or AdamW (decoupled decay, bias-corrected):
//   p' = p*(1 - lr*wd);  m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*g*g;
//   p1 = p' - (lr/bc1) * m / (sqrt(v)/sqrt(bc2) + eps)
// then the peer average with a = 1-alpha, b = alpha, in one of two forms:
//   pull:  p2 = a*p1 + b*q          (the worker's copy absorbs the peer's)
//   push:  p2 = p1, q2 = a*q + b*p1 (Algorithm 1 as written: the sender keeps
//          its update and overwrites the receiving replica's layer)
// optionally the bfloat16 copies of the written tensors and the disagreement
// sum((p1-q)^2).
//
// Each tensor is read once and written once (streaming loads and stores):
// pull 24 B/param for SGD momentum (read p,g,m,q; write p,m), 32 B/param for
// AdamW (read p,g,m,v,q; write p,m,v), +2 B with the bfloat16 copy; push adds
// the write of q (+4 B) and its bfloat16 copy (+2 B).  Loads and stores are
// 128-bit; the grid walks (tensor, chunk) pairs of a multi-tensor table so a
// layer of many small tensors is one launch.
#include "layup_internal.h"

namespace layup {

constexpr int UM_THREADS = 256;
constexpr int UM_CHUNK = 2048;  // elements per (block, chunk) = 2 x 4 per thread (measured best)
static_assert(UM_CHUNK == 8 * UM_THREADS, "one pass of two 4-element groups per thread");

struct UMArgs {
  UMTensor t[UM_MAX_TENSORS];
  int64_t chunk_prefix[UM_MAX_TENSORS + 1];
  int32_t n_tensors;
  int32_t trace_step, trace_unit, trace_cap;
  float lr, mu, wd, b1, b2, eps, step_size, inv_sqrt_bc2, a, b;
  float* dis_partial;
  int32_t* trace;
  int32_t* trace_counter;
};

template <int OPT, bool PUSH>
__device__ __forceinline__ void um_elem(float& p, float g, float& m, float& v, float q, float dfac,
                                        float wdc, const UMArgs& A, float& dis, float& p_out,
                                        float& q_out) {
  float p1;
  if (OPT == 0) {
    float gg = fmaf(wdc, p, g);                 // g + wd*p (wdc = 0 without decay)
    m = fmaf(A.mu, m, gg);
    p1 = fmaf(-A.lr, m, p);
  } else {
    float pd = p * dfac;                        // p * (1 - lr*wd)
    m = fmaf(A.b1, m, (1.0f - A.b1) * g);
    v = fmaf(A.b2, v, (1.0f - A.b2) * (g * g));
    // hardware square root and reciprocal (1 ulp each): the exact-division
    // sequence costs registers that would cut the waves per SIMD from 8 to 7
    float den = fmaf(__builtin_amdgcn_sqrtf(v), A.inv_sqrt_bc2, A.eps);
    p1 = fmaf(-A.step_size, m * __builtin_amdgcn_rcpf(den), pd);
  }
  float d = p1 - q;
  dis = fmaf(d, d, dis);
  if (PUSH) {
    p_out = p1;
    q_out = fmaf(A.a, q, A.b * p1);
  } else {
    p_out = fmaf(A.a, p1, A.b * q);
    q_out = q;
  }
}

template <int OPT, bool DIS, bool PUSH>
__global__ __launch_bounds__(UM_THREADS) void update_mix_kernel(const UMArgs A, int64_t total_chunks) {
  __shared__ float red[16];
  float dis = 0.f;
  for (int64_t c = blockIdx.x; c < total_chunks; c += gridDim.x) {
    int ti = 0;
    while (ti + 1 < A.n_tensors && A.chunk_prefix[ti + 1] <= c) ++ti;
    const UMTensor T = A.t[ti];
    const int64_t begin = (c - A.chunk_prefix[ti]) * UM_CHUNK;
    const int64_t end = min(begin + (int64_t)UM_CHUNK, T.n);
    const float dfac = T.decay ? (1.0f - A.lr * A.wd) : 1.0f;
    const float wdc = T.decay ? A.wd : 0.0f;
    // chunk base pointers are uniform (scalar registers); lanes use 32-bit
    // offsets, which keeps the kernel at 8 waves per SIMD
    const int cnt = (int)(end - begin);   // <= UM_CHUNK
    const int vcnt = cnt & ~3;
    float* __restrict__ pp = T.p + begin;
    const float* __restrict__ gp = T.g + begin;
    float* __restrict__ mp = T.m + begin;
    float* __restrict__ vp = OPT == 1 ? T.v + begin : nullptr;
    float* __restrict__ qp = T.q + begin;
    bf16_t* __restrict__ hp = T.p16 ? T.p16 + begin : nullptr;
    bf16_t* __restrict__ hq = PUSH && T.q16 ? T.q16 + begin : nullptr;
    // two 4-element groups per thread, all loads issued before any math;
    // streaming (nontemporal) loads and stores: every byte is used once
    f32x4 p[2], g[2], m[2], v[2], q[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const uint32_t i = 4u * threadIdx.x + u * 4u * UM_THREADS;
      if (i < (uint32_t)vcnt) {
        p[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(pp + i));
        g[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(gp + i));
        m[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(mp + i));
        q[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(qp + i));
        v[u] = OPT == 1 ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(vp + i))
                        : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const uint32_t i = 4u * threadIdx.x + u * 4u * UM_THREADS;
      if (i >= (uint32_t)vcnt) continue;
      f32x4 po, qo;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float pj = p[u][j], mj = m[u][j], vj = v[u][j], o, oq;
        um_elem<OPT, PUSH>(pj, g[u][j], mj, vj, q[u][j], dfac, wdc, A, dis, o, oq);
        m[u][j] = mj;
        v[u][j] = vj;
        po[j] = o;
        qo[j] = oq;
      }
      __builtin_nontemporal_store(po, reinterpret_cast<f32x4*>(pp + i));
      if (PUSH) {
        __builtin_nontemporal_store(qo, reinterpret_cast<f32x4*>(qp + i));
        if (hq) {
          u32x2 w;
          w[0] = pack_bf2(qo[0], qo[1]);
          w[1] = pack_bf2(qo[2], qo[3]);
          __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(hq + i));
        }
      }
      __builtin_nontemporal_store(m[u], reinterpret_cast<f32x4*>(mp + i));
      if (OPT == 1) __builtin_nontemporal_store(v[u], reinterpret_cast<f32x4*>(vp + i));
      if (hp) {
        u32x2 w;
        w[0] = pack_bf2(po[0], po[1]);
        w[1] = pack_bf2(po[2], po[3]);
        __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(hp + i));
      }
    }
    // ragged tail of the tensor (fewer than 4 elements)
    for (uint32_t i = (uint32_t)vcnt + threadIdx.x; i < (uint32_t)cnt; i += UM_THREADS) {
      float pv = pp[i], mv = mp[i], vv = OPT == 1 ? vp[i] : 0.f, o, oq;
      um_elem<OPT, PUSH>(pv, gp[i], mv, vv, qp[i], dfac, wdc, A, dis, o, oq);
      pp[i] = o;
      if (PUSH) {
        qp[i] = oq;
        if (hq) hq[i] = f2bf(oq);
      }
      mp[i] = mv;
      if (OPT == 1) vp[i] = vv;
      if (hp) hp[i] = f2bf(o);
    }
  }
  if (DIS) {
    float s = block_sum(dis, red);
    if (threadIdx.x == 0) A.dis_partial[blockIdx.x] = s;
  }
  if (A.trace && blockIdx.x == 0 && threadIdx.x == 0) {
    int idx = atomicAdd(A.trace_counter, 1);
    if (idx < A.trace_cap) {
      A.trace[2 * idx] = A.trace_step;
      A.trace[2 * idx + 1] = A.trace_unit;
    }
  }
}

// Sum of the per-block partials in block order (deterministic).
__global__ void sum_partials_kernel(const float* part, int n, float* out) {
  __shared__ float red[16];
  float s = 0.f;
  // each thread sums a strided subset in fixed order, then a fixed tree
  for (int i = threadIdx.x; i < n; i += blockDim.x) s += part[i];
  s = block_sum(s, red);
  if (threadIdx.x == 0) *out = s;
}

int64_t update_mix_max_blocks() { return UM_MAX_BLOCKS; }

UpdArgs make_upd_args(const layup_hparams& hp, float alpha, bool decay) {
  UpdArgs U;
  memset(&U, 0, sizeof(U));
  U.adamw = hp.kind == LAYUP_ADAMW;
  U.lr = hp.lr;
  U.mu = hp.momentum;
  U.wd = hp.weight_decay;
  U.b1 = hp.beta1;
  U.b2 = hp.beta2;
  U.eps = hp.eps;
  if (U.adamw) {
    const double t = (double)hp.step;
    U.step_size = (float)((double)hp.lr / (1.0 - pow((double)hp.beta1, t)));
    U.inv_sqrt_bc2 = (float)(1.0 / sqrt(1.0 - pow((double)hp.beta2, t)));
  }
  U.a = (float)(1.0 - (double)alpha);
  U.b = alpha;
  U.dfac = decay ? (1.0f - hp.lr * hp.weight_decay) : 1.0f;
  U.wdc = decay ? hp.weight_decay : 0.0f;
  return U;
}

template <int OPT, bool DIS>
static void launch_um(bool push, int64_t grid, const UMArgs& A, int64_t chunks, hipStream_t stream) {
  if (push) update_mix_kernel<OPT, DIS, true><<<grid, UM_THREADS, 0, stream>>>(A, chunks);
  else update_mix_kernel<OPT, DIS, false><<<grid, UM_THREADS, 0, stream>>>(A, chunks);
}

hipError_t launch_update_mix(const UMTensor* ts, int n, const layup_hparams& hp, float alpha,
                             float* dis_out, float* dis_partial, const TraceInfo& tr,
                             hipStream_t stream, bool push) {
  UMArgs A;
  memset(&A, 0, sizeof(A));
  int64_t chunks = 0;
  for (int i = 0; i < n; ++i) {
    A.t[i] = ts[i];
    A.chunk_prefix[i] = chunks;
    chunks += cdiv(ts[i].n, UM_CHUNK);
  }
  A.chunk_prefix[n] = chunks;
  A.n_tensors = n;
  A.lr = hp.lr;
  A.mu = hp.momentum;
  A.wd = hp.weight_decay;
  A.b1 = hp.beta1;
  A.b2 = hp.beta2;
  A.eps = hp.eps;
  if (hp.kind == LAYUP_ADAMW) {
    double t = (double)hp.step;
    double bc1 = 1.0 - pow((double)hp.beta1, t);
    double bc2 = 1.0 - pow((double)hp.beta2, t);
    A.step_size = (float)((double)hp.lr / bc1);
    A.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
  }
  A.a = (float)(1.0 - (double)alpha);
  A.b = alpha;
  A.dis_partial = dis_partial;
  A.trace = tr.trace;
  A.trace_counter = tr.counter;
  A.trace_cap = tr.capacity;
  A.trace_step = tr.step;
  A.trace_unit = tr.unit;
  // at least one block even when every tensor is empty: it still writes the
  // disagreement partial (zero) and appends the order-trace entry
  const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(chunks, UM_MAX_BLOCKS));
  const bool dis = dis_out != nullptr;
  if (hp.kind == LAYUP_ADAMW) {
    if (dis) launch_um<1, true>(push, grid, A, chunks, stream);
    else launch_um<1, false>(push, grid, A, chunks, stream);
  } else {
    if (dis) launch_um<0, true>(push, grid, A, chunks, stream);
    else launch_um<0, false>(push, grid, A, chunks, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (dis) {
    sum_partials_kernel<<<1, 1024, 0, stream>>>(dis_partial, (int)grid, dis_out);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace layup
