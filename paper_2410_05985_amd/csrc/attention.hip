// Fused causal attention core of a GPT block on the CDNA4 matrix cores,
// flash-attention style: the score matrix S = Q K^T / sqrt(dh), its softmax P
// and, in the backward, dP = dO V^T and dS = P (dP - rowsum(dP P)) / sqrt(dh)
// live only in registers; no T x T matrix is stored.
//
//  - Forward: one pass over the keys with the running (online) row maximum
//    and sum; O accumulates unnormalised and is divided by the row sum at the
//    end.  Stored: O (bf16, the next GEMM's operand), O in float32 and the
//    base-2 log-sum-exp of each query's scaled scores.
//  - Backward, two kernels, every output written by one workgroup in a fixed
//    order (deterministic): (1) per block of queries, P and dS are recomputed
//    from Q, K, V, dO and the log-sum-exp and dQ = dS K accumulates; this
//    kernel also stores D = rowsum(dP P) = dO . O (from the float32 O).
//    (2) per block of keys, P and dS are recomputed again and dV = P^T dO and
//    dK = dS^T Q accumulate.
//
// A workgroup of four waves owns 128 consecutive queries (forward, dQ) or
// keys (dK/dV) of one (batch, head), 32 per wave, and walks the other
// operand in steps of 64 rows (two 32-row sub-tiles), staged through
// registers into double-buffered LDS and shared by the four waves.  Products
// use v_mfma_f32_32x32x16_bf16.  The score block is computed so that every
// lane owns one of the wave's 32 rows (a query in the forward and dQ
// kernels, S^T = K Q^T; a key in the dK/dV kernel, S = Q K^T) and 16 of the
// sub-tile's other index; those registers, rounded to bfloat16, are directly
// the B operand of the next product (O^T = V^T P^T, dQ^T = K^T dS^T,
// dV^T = dO^T P, dK^T = Q^T dS): lane half h holds indices 4h..4h+3 and
// 8+4h..8+4h+3 of each 16-step, and the A operand is read from its LDS tile
// with the transposing LDS read in exactly that order.
//
// Exponentials are base 2 on scores pre-multiplied by scale * log2(e).  The
// backward recomputes P in float32 and rounds it to bfloat16 before both of
// its uses (dV = P^T dO and dS = P (dP - D)), the precision at which an
// unfused implementation would have stored it.
#include "layup_internal.h"

namespace layup {

namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define AT_LDS(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int AT_WAVES = 4;              // waves per workgroup, 32 rows each
constexpr int AT_THREADS = 64 * AT_WAVES;
constexpr int AT_STEP = 64;              // rows of the walked operand per step (two sub-tiles)
// Workgroups per CU each kernel is compiled for (the register budget per
// lane is 512 / occupancy); the LDS of that many workgroups fits in 160 KB.
#define AT_OCC_FWD(DH) ((DH) <= 64 ? 3 : 2)
#define AT_OCC_DQ(DH) ((DH) <= 64 ? 3 : 1)
#define AT_OCC_DKV(DH) ((DH) <= 64 ? 2 : 1)

// LDS tile of AT_STEP rows x DH columns (rows of 2*DH bytes) in one of two
// layouts, both swizzling 16-byte chunks within a row:
//  - row-read tile (A operand whose rows are the tile rows; lane reads 16
//    bytes of row lane % 32 of a sub-tile): chunk c of row r at
//    c ^ ((r / (128/DH)) % (DH/8)), so 16 consecutive rows cover the 256-byte
//    bank cycle once;
//  - transposed-read tile (A operand whose rows are the tile columns): chunk
//    c of row r at c ^ (((r & 3) << 2) & (DH/8 - 1)), so the four rows of one
//    transposing read fall on different banks.
// Both swizzles repeat every 32 rows, so a sub-tile is a fixed offset.
template <int DH>
__device__ __forceinline__ int row_off(int r, int c) {
  return r * 2 * DH + 16 * (c ^ ((r / (128 / DH)) % (DH / 8)));
}
template <int DH>
__device__ __forceinline__ int tr_off(int r, int c) {
  return r * 2 * DH + 16 * (c ^ (((r & 3) << 2) & (DH / 8 - 1)));
}

// One tile of ROWS rows staged in registers by the whole workgroup: 16-byte
// chunk idx = thread + AT_THREADS * i is chunk idx % (DH/8) of row idx / (DH/8).
template <int DH, int ROWS>
struct Stage {
  static constexpr int LPR = DH / 8;
  static constexpr int CHUNKS = ROWS * LPR;
  static constexpr int PER = (CHUNKS + AT_THREADS - 1) / AT_THREADS;
  u32x4 v[PER];
};

// rows r0.. of a row-major matrix with leading dimension ld (rows past T
// read row T - 1; they only feed masked products)
template <int DH, int ROWS>
__device__ __forceinline__ void fetch(Stage<DH, ROWS>& st, const bf16_t* m, int64_t ld, int r0, int T) {
#pragma unroll
  for (int i = 0; i < Stage<DH, ROWS>::PER; ++i) {
    const int idx = threadIdx.x + AT_THREADS * i;
    // the guard is compiled out when the chunks fill every thread's slots
    // (branch-free loads keep the compiler's wait counts exact)
    if (Stage<DH, ROWS>::CHUNKS % AT_THREADS == 0 || idx < Stage<DH, ROWS>::CHUNKS) {
      const int r = idx / Stage<DH, ROWS>::LPR, c = idx % Stage<DH, ROWS>::LPR;
      st.v[i] = *reinterpret_cast<const u32x4*>(m + (int64_t)min(r0 + r, T - 1) * ld + 8 * c);
    }
  }
}

template <int DH, int ROWS, bool TR>
__device__ __forceinline__ void put(const Stage<DH, ROWS>& st, char* lds) {
#pragma unroll
  for (int i = 0; i < Stage<DH, ROWS>::PER; ++i) {
    const int idx = threadIdx.x + AT_THREADS * i;
    if (Stage<DH, ROWS>::CHUNKS % AT_THREADS == 0 || idx < Stage<DH, ROWS>::CHUNKS) {
      const int r = idx / Stage<DH, ROWS>::LPR, c = idx % Stage<DH, ROWS>::LPR;
      *reinterpret_cast<u32x4*>(lds + (TR ? tr_off<DH>(r, c) : row_off<DH>(r, c))) = st.v[i];
    }
  }
}

// Before the step loop: every load issued so far (the wave's own operand
// rows and the first tile) complete, so the compiler's wait counting enters
// the loop with nothing outstanding and waits inside it only for what the
// loop issues.
__device__ __forceinline__ void loop_entry_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) expcnt(0) lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// LDS stores of this wave done, then the workgroup barrier (no wait on the
// vector-memory counter: the next tile's loads stay in flight).
__device__ __forceinline__ void tile_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// A operand from a row-read tile: row 32*sub + lane % 32 of the tile,
// columns 16 ks + 8 (lane / 32) .. +7.
template <int DH>
__device__ __forceinline__ bf16x8 row_frag(const char* lds, int sub, int ks, int lane) {
  return *reinterpret_cast<const bf16x8*>(lds + row_off<DH>(32 * sub + (lane & 31), 2 * ks + (lane >> 5)));
}

// A operand (rows m = tile columns rb..rb+31; k = 16 tile rows of step ks,
// ks = 0..3 over the 64-row tile) from a transposed-read tile, in the row
// order of a score accumulator: lane half h takes rows ks*16 + 4h + 0..3 and
// ks*16 + 8 + 4h + 0..3.  Transposing read: lane s of a 16-lane group
// addresses tile row kb + s/4, columns m..m+3, and receives column
// rb + 16*(group & 1) + s of four consecutive tile rows.
template <int DH>
__device__ __forceinline__ bf16x8 tr_frag(const char* lds, int rb, int ks, int lane) {
  const int g = lane >> 4, s = lane & 15;
  const int kb = ks * 16 + 4 * (g >> 1) + (s >> 2);
  const int m = rb + 16 * (g & 1) + 4 * (s & 3);
  const int c = m >> 3, half = (m & 7) * 2;
  v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)AT_LDS(lds + tr_off<DH>(kb, c) + half));
  v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)AT_LDS(lds + tr_off<DH>(kb + 8, c) + half));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ bf16x8 pack8(const float* v) {
  u32x4 w;
  w[0] = pack_bf2(v[0], v[1]);
  w[1] = pack_bf2(v[2], v[3]);
  w[2] = pack_bf2(v[4], v[5]);
  w[3] = pack_bf2(v[6], v[7]);
  return __builtin_bit_cast(bf16x8, w);
}

template <int V>
struct AtC {
  static constexpr int value = V;
};

// The two bfloat16 halves of a packed pair, as floats.
__device__ __forceinline__ float bf_lo(uint32_t u) { return __builtin_bit_cast(float, u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __builtin_bit_cast(float, u & 0xffff0000u); }

// Key (or query) of accumulator register r for lane half h, relative to the
// 32-row sub-tile start.
__device__ __forceinline__ int acc_key(int r, int h) { return (r >> 2) * 8 + 4 * h + (r & 3); }

// ---- workgroup items
// Forward and dQ: 128 queries of one (batch, head), heaviest (last) first.
struct QItem {
  int qb;    // this wave's 32-query block
  int nst;   // key steps the workgroup walks
  int mine;  // key steps this wave computes (0 past the sequence end)
  int b, hh;
};
__device__ __forceinline__ bool q_item(int T, int B, int H, QItem& it) {
  const int nqb = (T + 31) / 32, nqg = (nqb + AT_WAVES - 1) / AT_WAVES;
  const int64_t id = blockIdx.x;
  if (id >= (int64_t)nqg * B * H) return false;
  const int z = (int)(id % (B * H));
  const int qg = nqg - 1 - (int)(id / (B * H));
  it.qb = qg * AT_WAVES + (int)(threadIdx.x >> 6);
  it.nst = (min(T, (qg + 1) * AT_WAVES * 32) - 1) / AT_STEP + 1;
  it.mine = it.qb < nqb ? (min(T, it.qb * 32 + 32) - 1) / AT_STEP + 1 : 0;
  it.b = z / H;
  it.hh = z % H;
  return true;
}
// dK/dV: 128 keys of one (batch, head), heaviest (first) first.
struct KItem {
  int kb;     // this wave's 32-key block
  int first;  // first query step of the workgroup
  int mine;   // first query step this wave computes
  int nst;    // query steps (to the end of the sequence)
  bool active;
  int b, hh;
};
__device__ __forceinline__ bool k_item(int T, int B, int H, KItem& it) {
  const int nkb = (T + 31) / 32, nkg = (nkb + AT_WAVES - 1) / AT_WAVES;
  const int64_t id = blockIdx.x;
  if (id >= (int64_t)nkg * B * H) return false;
  const int z = (int)(id % (B * H));
  const int kg = (int)(id / (B * H));
  it.kb = kg * AT_WAVES + (int)(threadIdx.x >> 6);
  it.first = kg * AT_WAVES * 32 / AT_STEP;
  it.mine = it.kb * 32 / AT_STEP;
  it.nst = (T + AT_STEP - 1) / AT_STEP;
  it.active = it.kb < nkb;
  it.b = z / H;
  it.hh = z % H;
  return true;
}

// Store a 32 x DH accumulator block held transposed (lane: row of the
// output, registers: columns db*32 + acc_key(r, h)) as bfloat16 (and
// optionally float32) with 8-byte (16-byte) segments.
template <int DB>
__device__ __forceinline__ void store_rows(const f32x16 (&acc)[DB], float mul, bf16_t* out16, float* out32,
                                           int h) {
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c = db * 32 + g * 8 + 4 * h;
      const float a0 = acc[db][4 * g] * mul, a1 = acc[db][4 * g + 1] * mul;
      const float a2 = acc[db][4 * g + 2] * mul, a3 = acc[db][4 * g + 3] * mul;
      *reinterpret_cast<u32x2*>(out16 + c) = u32x2{pack_bf2(a0, a1), pack_bf2(a2, a3)};
      if (out32) *reinterpret_cast<f32x4*>(out32 + c) = f32x4{a0, a1, a2, a3};
    }
  }
}

// ---- forward
template <int DH>
__global__ __launch_bounds__(AT_THREADS, AT_OCC_FWD(DH)) void attn_fwd_kernel(const bf16_t* __restrict__ qkv,
                                                              bf16_t* __restrict__ O,
                                                              float* __restrict__ Of,
                                                              float* __restrict__ lse, int B, int H,
                                                              int T, float scale) {
  constexpr int KS = DH / 16, DB = DH / 32, TB = AT_STEP * DH * 2;
  __shared__ __attribute__((aligned(1024))) char kbuf[2][TB];
  __shared__ __attribute__((aligned(1024))) char vbuf[2][TB];
  QItem it;
  if (!q_item(T, B, H, it)) return;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  const int d = H * DH;
  const int64_t ld = 3 * (int64_t)d;
  const bf16_t* Qp = qkv + (int64_t)it.b * T * ld + it.hh * DH;
  const bf16_t* Kp = Qp + d;
  const bf16_t* Vp = Qp + 2 * d;
  const int qlo = it.qb * 32, q = qlo + col, qc = min(q, T - 1);
  const float c2 = scale * 1.4426950408889634f;  // scale * log2(e)
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(Qp + qc * ld + 16 * ks + 8 * h);
  f32x16 oacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  // running maximum (shared by the two lane halves of a query) and this
  // lane's partial sum; the first key of every computed step is <= q, so
  // the maximum is finite after the first step
  float m = -INFINITY, l = 0.f;
  Stage<DH, AT_STEP> sk, sv;
  fetch<DH, AT_STEP>(sk, Kp, ld, 0, T);
  fetch<DH, AT_STEP>(sv, Vp, ld, 0, T);
  put<DH, AT_STEP, false>(sk, kbuf[0]);
  put<DH, AT_STEP, true>(sv, vbuf[0]);
  loop_entry_barrier();
  for (int st = 0; st < it.nst; ++st) {
    if (st + 1 < it.nst) {
      fetch<DH, AT_STEP>(sk, Kp, ld, (st + 1) * AT_STEP, T);
      fetch<DH, AT_STEP>(sv, Vp, ld, (st + 1) * AT_STEP, T);
    }
    if (st < it.mine) {
      const char* kt = kbuf[st & 1];
      const char* vt = vbuf[st & 1];
      f32x16 s0, s1;
#pragma unroll
      for (int r = 0; r < 16; ++r) s0[r] = s1[r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(kt, 0, ks, lane), qf[ks], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(kt, 1, ks, lane), qf[ks], s1, 0, 0, 0);
      }
      const int k0 = st * AT_STEP;
      // raw scores; the scale c2 > 0 is applied after the maximum (rounding
      // is monotone, so max(s) c2 = max(s c2)) inside the exponent's fma
      float x[32];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        x[r] = s0[r];
        x[16 + r] = s1[r];
      }
      if (k0 + AT_STEP - 1 > qlo || k0 + AT_STEP > T) {  // diagonal or last step: mask
#pragma unroll
        for (int r = 0; r < 32; ++r) {
          const int key = k0 + 32 * (r >> 4) + acc_key(r & 15, h);
          if (!(key <= q && key < T)) x[r] = -INFINITY;
        }
      }
      float tmax = x[0];
#pragma unroll
      for (int r = 1; r < 32; ++r) tmax = fmaxf(tmax, x[r]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64)) * c2;
      const float mn = fmaxf(m, tmax);
      const float alpha = __builtin_amdgcn_exp2f(m - mn);  // 0 on the first step
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 32; ++r) {
        x[r] = __builtin_amdgcn_exp2f(fmaf(x[r], c2, -mn));
        ps += x[r];
      }
      l = fmaf(l, alpha, ps);
      m = mn;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
      bf16x8 pb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) pb[k] = pack8(x + 8 * k);
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int db = 0; db < DB; ++db)
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(vt, db * 32, k, lane), pb[k], oacc[db], 0, 0, 0);
    }
    if (st + 1 < it.nst) {
      put<DH, AT_STEP, false>(sk, kbuf[(st + 1) & 1]);
      put<DH, AT_STEP, true>(sv, vbuf[(st + 1) & 1]);
    }
    tile_barrier();
  }
  if (q >= T) return;
  const float lt = l + __shfl_xor(l, 32, 64);
  const int64_t orow = ((int64_t)it.b * T + q) * d + it.hh * DH;
  store_rows<DB>(oacc, 1.0f / lt, O + orow, Of + orow, h);
  if (h == 0) lse[((int64_t)it.b * H + it.hh) * T + q] = m + log2f(lt);
}

// ---- backward (1): dQ and D, per block of queries
template <int DH>
__global__ __launch_bounds__(AT_THREADS, AT_OCC_DQ(DH)) void attn_bwd_dq_kernel(
    const bf16_t* __restrict__ qkv, const float* __restrict__ lse, const bf16_t* __restrict__ dO,
    const float* __restrict__ Of, float* __restrict__ Dout, bf16_t* __restrict__ dqkv, int B, int H,
    int T, float scale) {
  constexpr int KS = DH / 16, DB = DH / 32, TB = AT_STEP * DH * 2;
  __shared__ __attribute__((aligned(1024))) char krow[2][TB];
  __shared__ __attribute__((aligned(1024))) char ktr[2][TB];
  __shared__ __attribute__((aligned(1024))) char vrow[2][TB];
  QItem it;
  if (!q_item(T, B, H, it)) return;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  const int d = H * DH;
  const int64_t ld = 3 * (int64_t)d;
  const bf16_t* Qp = qkv + (int64_t)it.b * T * ld + it.hh * DH;
  const bf16_t* Kp = Qp + d;
  const bf16_t* Vp = Qp + 2 * d;
  const int qlo = it.qb * 32, q = qlo + col, qc = min(q, T - 1);
  const float c2 = scale * 1.4426950408889634f;
  const int64_t z = (int64_t)it.b * H + it.hh;
  const int64_t orow = ((int64_t)it.b * T + qc) * d + it.hh * DH;
  // Q^T and dO^T operands; D = dO . O over this lane's half of the columns
  bf16x8 qf[KS], df[KS];
  float part = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = *reinterpret_cast<const bf16x8*>(Qp + qc * ld + 16 * ks + 8 * h);
    df[ks] = *reinterpret_cast<const bf16x8*>(dO + orow + 16 * ks + 8 * h);
    const f32x4 o0 = *reinterpret_cast<const f32x4*>(Of + orow + 16 * ks + 8 * h);
    const f32x4 o1 = *reinterpret_cast<const f32x4*>(Of + orow + 16 * ks + 8 * h + 4);
    const u32x4 w = __builtin_bit_cast(u32x4, df[ks]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __builtin_bit_cast(float, w[e] << 16), hi = __builtin_bit_cast(float, w[e] & 0xffff0000u);
      const float oa = e < 2 ? o0[2 * e] : o1[2 * e - 4], ob = e < 2 ? o0[2 * e + 1] : o1[2 * e - 3];
      part = fmaf(lo, oa, part);
      part = fmaf(hi, ob, part);
    }
  }
  const float D = part + __shfl_xor(part, 32, 64);
  const float Ds = D * scale;
  const float ls = lse[z * T + qc];
  if (q < T && h == 0 && it.mine > 0) Dout[z * T + q] = D;
  f32x16 qacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) qacc[i][r] = 0.f;
  Stage<DH, AT_STEP> sk, sv;
  fetch<DH, AT_STEP>(sk, Kp, ld, 0, T);
  fetch<DH, AT_STEP>(sv, Vp, ld, 0, T);
  put<DH, AT_STEP, false>(sk, krow[0]);
  put<DH, AT_STEP, true>(sk, ktr[0]);
  put<DH, AT_STEP, false>(sv, vrow[0]);
  loop_entry_barrier();
  for (int st = 0; st < it.nst; ++st) {
    if (st + 1 < it.nst) {
      fetch<DH, AT_STEP>(sk, Kp, ld, (st + 1) * AT_STEP, T);
      fetch<DH, AT_STEP>(sv, Vp, ld, (st + 1) * AT_STEP, T);
    }
    if (st < it.mine) {
      const char* kr = krow[st & 1];
      const char* kt = ktr[st & 1];
      const char* vr = vrow[st & 1];
      const int k0 = st * AT_STEP;
      const bool edge = k0 + AT_STEP - 1 > qlo || k0 + AT_STEP > T;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        f32x16 sa, pa;
#pragma unroll
        for (int r = 0; r < 16; ++r) sa[r] = pa[r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(kr, sub, ks, lane), qf[ks], sa, 0, 0, 0);
          pa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(vr, sub, ks, lane), df[ks], pa, 0, 0, 0);
        }
        // P at its bfloat16 storage precision (the value dV = P^T dO uses),
        // dS = P (dP - D) / sqrt(dh); masked entries (diagonal and tail
        // steps only): exp2(-inf) = 0
        float ds[16];
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          float a0 = fmaf(sa[r], c2, -ls), a1 = fmaf(sa[r + 1], c2, -ls);
          if (edge) {
            const int key = k0 + 32 * sub + acc_key(r, h);  // key of r + 1 is key + 1
            a0 = ((key <= q) & (key < T)) ? a0 : -INFINITY;
            a1 = ((key + 1 <= q) & (key + 1 < T)) ? a1 : -INFINITY;
          }
          const uint32_t u = pack_bf2(__builtin_amdgcn_exp2f(a0), __builtin_amdgcn_exp2f(a1));
          ds[r] = bf_lo(u) * fmaf(pa[r], scale, -Ds);
          ds[r + 1] = bf_hi(u) * fmaf(pa[r + 1], scale, -Ds);
        }
        const bf16x8 d0 = pack8(ds), d1 = pack8(ds + 8);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          qacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(kt, db * 32, 2 * sub, lane), d0, qacc[db], 0, 0, 0);
          qacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(kt, db * 32, 2 * sub + 1, lane), d1, qacc[db], 0, 0, 0);
        }
      }
    }
    if (st + 1 < it.nst) {
      put<DH, AT_STEP, false>(sk, krow[(st + 1) & 1]);
      put<DH, AT_STEP, true>(sk, ktr[(st + 1) & 1]);
      put<DH, AT_STEP, false>(sv, vrow[(st + 1) & 1]);
    }
    tile_barrier();
  }
  if (q >= T) return;
  store_rows<DB>(qacc, 1.0f, dqkv + ((int64_t)it.b * T + q) * ld + it.hh * DH, nullptr, h);
}

// ---- backward (2): dK and dV, per block of keys
template <int DH>
__global__ __launch_bounds__(AT_THREADS, AT_OCC_DKV(DH)) void attn_bwd_dkv_kernel(
    const bf16_t* __restrict__ qkv, const float* __restrict__ lse, const bf16_t* __restrict__ dO,
    const float* __restrict__ Din, bf16_t* __restrict__ dqkv, int B, int H, int T, float scale) {
  constexpr int KS = DH / 16, DB = DH / 32, TB = AT_STEP * DH * 2;
  __shared__ __attribute__((aligned(1024))) char qrow[2][TB];
  __shared__ __attribute__((aligned(1024))) char qtr[2][TB];
  __shared__ __attribute__((aligned(1024))) char orow_t[2][TB];
  __shared__ __attribute__((aligned(1024))) char otr[2][TB];
  __shared__ __attribute__((aligned(16))) float lsd[2][2][AT_STEP];  // [stage][lse, D/sqrt(dh)][query]
  KItem it;
  if (!k_item(T, B, H, it)) return;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  const int d = H * DH;
  const int64_t ld = 3 * (int64_t)d;
  const bf16_t* Qp = qkv + (int64_t)it.b * T * ld + it.hh * DH;
  const bf16_t* dOp = dO + (int64_t)it.b * T * d + it.hh * DH;
  const int64_t z = (int64_t)it.b * H + it.hh;
  const float* lsep = lse + z * T;
  const float* Dp = Din + z * T;
  const int key = it.kb * 32 + col, kc = min(key, T - 1);
  const float c2 = scale * 1.4426950408889634f;
  // K^T and V^T operands of this lane's key
  bf16x8 kf[KS], vf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kf[ks] = *reinterpret_cast<const bf16x8*>(Qp + kc * ld + d + 16 * ks + 8 * h);
    vf[ks] = *reinterpret_cast<const bf16x8*>(Qp + kc * ld + 2 * d + 16 * ks + 8 * h);
  }
  f32x16 kacc[DB], vacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) kacc[i][r] = vacc[i][r] = 0.f;
  // Q and dO tiles (and the lse and D values) of a query step are loaded into
  // registers two steps ahead (slots by step parity, as the LDS stages), so a
  // load has two steps' compute to land before its stores into LDS.
  Stage<DH, AT_STEP> sq[2], so[2];
  float sl[2] = {0.f, 0.f};  // one lse or D value per thread of the first 128
  auto fetch_step = [&](auto S, int st) {
    constexpr int k = decltype(S)::value;
    fetch<DH, AT_STEP>(sq[k], Qp, ld, st * AT_STEP, T);
    fetch<DH, AT_STEP>(so[k], dOp, d, st * AT_STEP, T);
    const int t = threadIdx.x & (2 * AT_STEP - 1);  // every thread loads (one wait count for all)
    sl[k] = (t < AT_STEP ? lsep : Dp)[min(st * AT_STEP + (t % AT_STEP), T - 1)];
  };
  auto put_step = [&](auto S) {
    constexpr int k = decltype(S)::value;
    put<DH, AT_STEP, false>(sq[k], qrow[k]);
    put<DH, AT_STEP, true>(sq[k], qtr[k]);
    put<DH, AT_STEP, false>(so[k], orow_t[k]);
    put<DH, AT_STEP, true>(so[k], otr[k]);
    const int t = threadIdx.x;
    if (t < 2 * AT_STEP) lsd[k][t / AT_STEP][t % AT_STEP] = t < AT_STEP ? sl[k] : sl[k] * scale;
  };
  fetch_step(AtC<0>{}, it.first);
  put_step(AtC<0>{});
  if (it.first + 1 < it.nst) fetch_step(AtC<1>{}, it.first + 1);
  loop_entry_barrier();
  // step st: its tiles in LDS stage P = (st - first) % 2, the next step's in
  // register slot P ^ 1; slot P is free for step st + 2
  auto step = [&](auto PC, int st) {
    constexpr int P = decltype(PC)::value;
    // issued on every step (a step past the end reloads the last one, never
    // stored) so that the wait before the stores below counts the same
    // loads on every path
    fetch_step(AtC<P>{}, min(st + 2, it.nst - 1));
    if (it.active && st >= it.mine) {
      const int qs = st * AT_STEP;
      const bool edge = qs < it.kb * 32 + 32 || qs + AT_STEP > T;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        f32x16 sa, pa;
#pragma unroll
        for (int r = 0; r < 16; ++r) sa[r] = pa[r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(qrow[P], sub, ks, lane), kf[ks], sa, 0, 0, 0);
          pa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(orow_t[P], sub, ks, lane), vf[ks], pa, 0, 0, 0);
        }
        // P in bfloat16 (packed pairs: directly the dV operand), dS = P (dP - D)
        // / sqrt(dh); masked entries (diagonal and tail steps only): 0
        uint32_t pu[8];
        float ds[16];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int qi = 32 * sub + 8 * g + 4 * h;  // query of registers 4g..4g+3, within the step
          const f32x4 lv = *reinterpret_cast<const f32x4*>(&lsd[P][0][qi]);
          const f32x4 dv = *reinterpret_cast<const f32x4*>(&lsd[P][1][qi]);
#pragma unroll
          for (int e = 0; e < 4; e += 2) {
            const int r = 4 * g + e, qq = qs + qi + e;
            float a0 = fmaf(sa[r], c2, -lv[e]), a1 = fmaf(sa[r + 1], c2, -lv[e + 1]);
            if (edge) {
              a0 = ((qq >= key) & (qq < T)) ? a0 : -INFINITY;
              a1 = ((qq + 1 >= key) & (qq + 1 < T)) ? a1 : -INFINITY;
            }
            const uint32_t u = pack_bf2(__builtin_amdgcn_exp2f(a0), __builtin_amdgcn_exp2f(a1));
            pu[r >> 1] = u;
            ds[r] = bf_lo(u) * fmaf(pa[r], scale, -dv[e]);
            ds[r + 1] = bf_hi(u) * fmaf(pa[r + 1], scale, -dv[e + 1]);
          }
        }
        const bf16x8 p0 = __builtin_bit_cast(bf16x8, u32x4{pu[0], pu[1], pu[2], pu[3]});
        const bf16x8 p1 = __builtin_bit_cast(bf16x8, u32x4{pu[4], pu[5], pu[6], pu[7]});
        const bf16x8 d0 = pack8(ds), d1 = pack8(ds + 8);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          vacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(otr[P], db * 32, 2 * sub, lane), p0, vacc[db], 0, 0, 0);
          vacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(otr[P], db * 32, 2 * sub + 1, lane), p1, vacc[db], 0, 0, 0);
          kacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(qtr[P], db * 32, 2 * sub, lane), d0, kacc[db], 0, 0, 0);
          kacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(qtr[P], db * 32, 2 * sub + 1, lane), d1, kacc[db], 0, 0, 0);
        }
      }
    }
    if (st + 1 < it.nst) put_step(AtC<P ^ 1>{});
    tile_barrier();
  };
  for (int st = it.first; st < it.nst; st += 2) {
    step(AtC<0>{}, st);
    if (st + 1 < it.nst) step(AtC<1>{}, st + 1);
  }
  if (!it.active || key >= T) return;
  bf16_t* rowp = dqkv + ((int64_t)it.b * T + key) * ld + it.hh * DH;
  store_rows<DB>(kacc, 1.0f, rowp + d, nullptr, h);
  store_rows<DB>(vacc, 1.0f, rowp + 2 * d, nullptr, h);
}

}  // namespace

bool attention_fused_supported(int dh) { return dh == 32 || dh == 64 || dh == 128; }

hipError_t launch_attention_fwd(const bf16_t* qkv, float* lse, bf16_t* O, float* Of, int B, int H,
                                int T, int dh, float scale, hipStream_t s) {
  if (T % 8 || T <= 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(cdiv(cdiv(T, 32), AT_WAVES) * B * H));
  switch (dh) {
    case 32: attn_fwd_kernel<32><<<grid, AT_THREADS, 0, s>>>(qkv, O, Of, lse, B, H, T, scale); break;
    case 64: attn_fwd_kernel<64><<<grid, AT_THREADS, 0, s>>>(qkv, O, Of, lse, B, H, T, scale); break;
    case 128: attn_fwd_kernel<128><<<grid, AT_THREADS, 0, s>>>(qkv, O, Of, lse, B, H, T, scale); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention_bwd(const bf16_t* qkv, const float* lse, const bf16_t* dO, const float* Of,
                                float* D, bf16_t* dqkv, int B, int H, int T, int dh, float scale,
                                hipStream_t s) {
  if (T % 8 || T <= 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(cdiv(cdiv(T, 32), AT_WAVES) * B * H));
  switch (dh) {
    case 32:
      attn_bwd_dq_kernel<32><<<grid, AT_THREADS, 0, s>>>(qkv, lse, dO, Of, D, dqkv, B, H, T, scale);
      attn_bwd_dkv_kernel<32><<<grid, AT_THREADS, 0, s>>>(qkv, lse, dO, D, dqkv, B, H, T, scale);
      break;
    case 64:
      attn_bwd_dq_kernel<64><<<grid, AT_THREADS, 0, s>>>(qkv, lse, dO, Of, D, dqkv, B, H, T, scale);
      attn_bwd_dkv_kernel<64><<<grid, AT_THREADS, 0, s>>>(qkv, lse, dO, D, dqkv, B, H, T, scale);
      break;
    case 128:
      attn_bwd_dq_kernel<128><<<grid, AT_THREADS, 0, s>>>(qkv, lse, dO, Of, D, dqkv, B, H, T, scale);
      attn_bwd_dkv_kernel<128><<<grid, AT_THREADS, 0, s>>>(qkv, lse, dO, D, dqkv, B, H, T, scale);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace layup
