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

// Scalars of one update+mix launch (bias corrections and mixing
// coefficients formed on the host).
struct UMScalars {
  float lr, mu, wd, b1, b2, eps, step_size, inv_sqrt_bc2, a, b;
};

struct UMArgs {
  UMTensor t[UM_MAX_TENSORS];
  int64_t chunk_prefix[UM_MAX_TENSORS + 1];
  int32_t n_tensors;
  int32_t trace_step, trace_unit, trace_cap;
  UMScalars s;
  float* dis_partial;
  int32_t* trace;
  int32_t* trace_counter;
};

// Several units in one launch, tensors given as offsets from common base
// pointers (every tensor at the same place in the param, grad, state and peer
// buffers: the flat layout of a model).  Up to UMF_MAX_TENSORS tensors fit in
// the kernel arguments; tag = unit << 1 | decay.
struct UMFlatArgs {
  float* p;
  const float* g;
  float* m;
  float* v;
  float* q;
  bf16_t* p16;
  bf16_t* q16;
  UMScalars s;
  int32_t* trace;
  int32_t* trace_counter;
  int32_t n_tensors, trace_step, trace_cap, pad;
  int32_t off[UMF_MAX_TENSORS];
  int32_t n[UMF_MAX_TENSORS];
  int32_t prefix[UMF_MAX_TENSORS + 1];
  int32_t tag[UMF_MAX_TENSORS];
};
static_assert(sizeof(UMFlatArgs) <= 3584, "kernel arguments of the multi-unit update+mix");

template <int OPT, bool PUSH>
__device__ __forceinline__ void um_elem(float& p, float g, float& m, float& v, float q, float dfac,
                                        float wdc, const UMScalars& A, float& dis, float& p_out,
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

// One chunk of up to UM_CHUNK consecutive elements of one tensor: two
// 4-element groups per thread, all loads issued before any math; streaming
// (nontemporal) loads and stores, every byte is used once; chunk base
// pointers are uniform (scalar registers) and lanes use 32-bit offsets,
// which keeps the kernel at 8 waves per SIMD.
template <int OPT, bool PUSH>
__device__ __forceinline__ void um_chunk(float* __restrict__ pp, const float* __restrict__ gp,
                                         float* __restrict__ mp, float* __restrict__ vp,
                                         float* __restrict__ qp, bf16_t* __restrict__ hp,
                                         bf16_t* __restrict__ hq, int cnt, bool decay, const UMScalars& S,
                                         float& dis) {
  const float dfac = decay ? (1.0f - S.lr * S.wd) : 1.0f;
  const float wdc = decay ? S.wd : 0.0f;
  const int vcnt = cnt & ~3;
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
      um_elem<OPT, PUSH>(pj, g[u][j], mj, vj, q[u][j], dfac, wdc, S, dis, o, oq);
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
    um_elem<OPT, PUSH>(pv, gp[i], mv, vv, qp[i], dfac, wdc, S, dis, o, oq);
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

template <int OPT, bool DIS, bool PUSH>
__global__ __launch_bounds__(UM_THREADS) void update_mix_kernel(const UMArgs A, int64_t total_chunks) {
  __shared__ float red[16];
  float dis = 0.f;
  for (int64_t c = blockIdx.x; c < total_chunks; c += gridDim.x) {
    int ti = 0;
    while (ti + 1 < A.n_tensors && A.chunk_prefix[ti + 1] <= c) ++ti;
    const UMTensor T = A.t[ti];
    const int64_t begin = (c - A.chunk_prefix[ti]) * UM_CHUNK;
    const int cnt = (int)(min(begin + (int64_t)UM_CHUNK, T.n) - begin);   // <= UM_CHUNK
    um_chunk<OPT, PUSH>(T.p + begin, T.g + begin, T.m + begin, OPT == 1 ? T.v + begin : nullptr,
                        T.q + begin, T.p16 ? T.p16 + begin : nullptr,
                        PUSH && T.q16 ? T.q16 + begin : nullptr, cnt, T.decay != 0, A.s, dis);
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

// Several units in one pass: the chunks are numbered unit by unit in the
// table's order (the order the units are visited), so workgroups, which
// start in order, take the units in that order.  Workgroup 0 appends one
// trace entry per unit, in table order.
template <int OPT, bool PUSH>
__global__ __launch_bounds__(UM_THREADS) void update_mix_flat_kernel(const UMFlatArgs A, int total_chunks) {
  float dis = 0.f;  // no disagreement output in this form
  for (int c = blockIdx.x; c < total_chunks; c += gridDim.x) {
    // the last tensor whose first chunk is <= c (empty tensors share their
    // successor's first chunk and are passed over)
    int lo = 0, hi = A.n_tensors - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (A.prefix[mid] <= c) lo = mid;
      else hi = mid - 1;
    }
    const int64_t begin = (int64_t)(c - A.prefix[lo]) * UM_CHUNK;
    const int cnt = (int)min((int64_t)UM_CHUNK, (int64_t)A.n[lo] - begin);
    const int64_t o = (int64_t)A.off[lo] + begin;
    um_chunk<OPT, PUSH>(A.p + o, A.g + o, A.m + o, OPT == 1 ? A.v + o : nullptr, A.q + o,
                        A.p16 ? A.p16 + o : nullptr, PUSH && A.q16 ? A.q16 + o : nullptr, cnt,
                        (A.tag[lo] & 1) != 0, A.s, dis);
  }
  if (A.trace && blockIdx.x == 0 && threadIdx.x == 0) {
    for (int i = 0; i < A.n_tensors; ++i) {
      if (i > 0 && (A.tag[i] >> 1) == (A.tag[i - 1] >> 1)) continue;
      const int idx = atomicAdd(A.trace_counter, 1);
      if (idx < A.trace_cap) {
        A.trace[2 * idx] = A.trace_step;
        A.trace[2 * idx + 1] = A.tag[i] >> 1;
      }
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

static UMScalars um_scalars(const layup_hparams& hp, float alpha) {
  UMScalars S;
  memset(&S, 0, sizeof(S));
  S.lr = hp.lr;
  S.mu = hp.momentum;
  S.wd = hp.weight_decay;
  S.b1 = hp.beta1;
  S.b2 = hp.beta2;
  S.eps = hp.eps;
  if (hp.kind == LAYUP_ADAMW) {
    const double t = (double)hp.step;
    const double bc1 = 1.0 - pow((double)hp.beta1, t);
    const double bc2 = 1.0 - pow((double)hp.beta2, t);
    S.step_size = (float)((double)hp.lr / bc1);
    S.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
  }
  S.a = (float)(1.0 - (double)alpha);
  S.b = alpha;
  return S;
}

// Do the (non-empty) tensors share one flat layout: the same byte distance
// from param to grad, state0, state1 and peer for every tensor, bf16 copies
// at the param's element offset, and element offsets from the lowest param
// that fit in 31 bits?  base_index: the tensor with the lowest param.
bool update_mix_flat_layout(const UMTensor* ts, int n, bool adamw, bool push, int* base_index) {
  int b = -1;
  for (int i = 0; i < n; ++i)
    if (ts[i].n > 0 && (b < 0 || ts[i].p < ts[b].p)) b = i;
  if (b < 0) return false;
  const UMTensor& B = ts[b];
  auto dist = [](const void* x, const void* y) { return (intptr_t)x - (intptr_t)y; };
  for (int i = 0; i < n; ++i) {
    const UMTensor& T = ts[i];
    if (T.n == 0) continue;
    const int64_t off = (T.p - B.p);
    if (off < 0 || off + T.n >= (1ll << 31) || T.n >= (1ll << 31)) return false;
    if (dist(T.g, T.p) != dist(B.g, B.p) || dist(T.m, T.p) != dist(B.m, B.p) ||
        dist(T.q, T.p) != dist(B.q, B.p))
      return false;
    if (adamw && dist(T.v, T.p) != dist(B.v, B.p)) return false;
    if ((T.p16 == nullptr) != (B.p16 == nullptr) || (T.p16 && T.p16 - B.p16 != off)) return false;
    if (push && ((T.q16 == nullptr) != (B.q16 == nullptr) || (T.q16 && T.q16 - B.q16 != off))) return false;
  }
  *base_index = b;
  return true;
}

hipError_t launch_update_mix_flat(const UMTensor* ts, const int32_t* units, int n, const layup_hparams& hp,
                                  float alpha, const TraceInfo& tr, hipStream_t stream, bool push) {
  if (n < 1 || n > UMF_MAX_TENSORS) return hipErrorInvalidValue;
  int b = 0;
  const bool adamw = hp.kind == LAYUP_ADAMW;
  if (!update_mix_flat_layout(ts, n, adamw, push, &b)) return hipErrorInvalidValue;
  UMFlatArgs A;
  memset(&A, 0, sizeof(A));
  const UMTensor& B = ts[b];
  A.p = B.p;
  A.g = B.g;
  A.m = B.m;
  A.v = adamw ? B.v : nullptr;
  A.q = B.q;
  A.p16 = B.p16;
  A.q16 = push ? B.q16 : nullptr;
  A.s = um_scalars(hp, alpha);
  A.trace = tr.trace;
  A.trace_counter = tr.counter;
  A.trace_cap = tr.capacity;
  A.trace_step = tr.step;
  A.n_tensors = n;
  int64_t chunks = 0;
  for (int i = 0; i < n; ++i) {
    A.off[i] = ts[i].n > 0 ? (int32_t)(ts[i].p - B.p) : 0;
    A.n[i] = (int32_t)ts[i].n;
    A.prefix[i] = (int32_t)chunks;
    A.tag[i] = (units[i] << 1) | (ts[i].decay ? 1 : 0);
    chunks += cdiv(ts[i].n, UM_CHUNK);
  }
  A.prefix[n] = (int32_t)chunks;
  if (chunks >= (1ll << 31)) return hipErrorInvalidValue;
  // at least one workgroup even when every tensor is empty (trace entries)
  const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(chunks, UM_MAX_BLOCKS));
  if (adamw) {
    if (push) update_mix_flat_kernel<1, true><<<grid, UM_THREADS, 0, stream>>>(A, (int)chunks);
    else update_mix_flat_kernel<1, false><<<grid, UM_THREADS, 0, stream>>>(A, (int)chunks);
  } else {
    if (push) update_mix_flat_kernel<0, true><<<grid, UM_THREADS, 0, stream>>>(A, (int)chunks);
    else update_mix_flat_kernel<0, false><<<grid, UM_THREADS, 0, stream>>>(A, (int)chunks);
  }
  return hipGetLastError();
}

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
  A.s = um_scalars(hp, alpha);
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
