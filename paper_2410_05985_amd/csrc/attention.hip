// Fused causal attention core of a GPT block on the CDNA4 matrix cores: the
// forward P = softmax(Q K^T / sqrt(dh)), O = P V and the backward part that
// needs the score matrix, dS = P (dP - rowsum(dP P)) / sqrt(dh) with
// dP = dO V^T, and dQ = dS K.  The score and dP matrices live only in
// registers; P (the saved activation) and dS (read by the dK = dS^T Q GEMM)
// are written once in bfloat16, at the same rounding points as the unfused
// kernels (P and dS rounded after normalisation/scaling, O and dQ rounded
// from float32 accumulations).
//
// A workgroup of four waves owns 128 consecutive queries of one (batch,
// head), one wave per 32 queries, and walks the key tiles of 32 keys up to
// its last diagonal.  Each K and V tile is loaded once per workgroup
// (coalesced, through registers) into double-buffered LDS and read by all
// four waves; a wave computes only the tiles up to its own diagonal.
//
// Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
// in the accumulator every lane then holds one query (lane % 32) and 16 of
// the tile's keys, so the row statistics of a query are a reduction over the
// lane's registers plus one exchange with lane l ^ 32.  The same registers,
// rounded to bfloat16, are the B operand of the next product O^T = V^T P^T
// (and dQ^T = K^T dS^T): lane half h holds keys 4h..4h+3 and 8+4h..8+4h+3 of
// each 16-key step, and the A operand (V^T or K^T) is read from its LDS tile
// with the transposing LDS read in exactly that key order.  The outputs O^T
// and dQ^T again give each lane one query, stored with 8-byte row segments.
//
// The forward makes two passes over the keys: row maximum and sum first,
// then the normalised P, which is stored and multiplied with V.  The
// backward takes rowsum(dP P) as dO . O from the float32 O the forward keeps
// (equal in exact arithmetic, since O = P V).  Entries above the diagonal,
// up to the end of the query's 128-row band, are written as zeros: the
// batched dV = P^T dO and dK = dS^T Q GEMMs read whole 128-wide diagonal
// tiles.
#include "layup_internal.h"

namespace layup {

namespace {

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define AT_LDS(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int AT_WAVES = 4;              // waves per workgroup, 32 queries each
constexpr int AT_THREADS = 64 * AT_WAVES;
constexpr int AT_ZERO_BAND = 128;        // row band of the batched attention GEMMs' tiles

// LDS tile of 32 keys x DH columns (key rows of 2*DH bytes) in one of two
// layouts, both swizzling 16-byte chunks within a row:
//  - row-read tile (A operand of S^T = K Q^T and dP^T = V dO^T; lane reads
//    16 bytes of key row lane % 32): chunk c of row r at c ^ ((r / (128/DH)) % (DH/8)),
//    so 16 consecutive rows cover the 256-byte bank cycle once;
//  - transposed-read tile (A operand of O^T = V^T P^T and dQ^T = K^T dS^T):
//    chunk c of row r at c ^ (((r & 3) << 2) & (DH/8 - 1)), so the four rows
//    of one transposing read fall on different banks.
template <int DH>
__device__ __forceinline__ int row_off(int r, int c) {
  return r * 2 * DH + 16 * (c ^ ((r / (128 / DH)) % (DH / 8)));
}
template <int DH>
__device__ __forceinline__ int tr_off(int r, int c) {
  return r * 2 * DH + 16 * (c ^ (((r & 3) << 2) & (DH / 8 - 1)));
}

// One 32-key tile staged in registers by the whole workgroup: 16-byte chunk
// idx = thread + AT_THREADS * i is chunk idx % (DH/8) of key row idx / (DH/8).
template <int DH>
struct Stage {
  static constexpr int LPR = DH / 8;
  static constexpr int CHUNKS = 32 * LPR;
  static constexpr int PER = (CHUNKS + AT_THREADS - 1) / AT_THREADS;
  u32x4 v[PER];
};

template <int DH>
__device__ __forceinline__ void fetch(Stage<DH>& st, const bf16_t* m, int64_t ld, int k0, int T) {
#pragma unroll
  for (int i = 0; i < Stage<DH>::PER; ++i) {
    const int idx = threadIdx.x + AT_THREADS * i;
    if (idx < Stage<DH>::CHUNKS) {
      const int r = idx / Stage<DH>::LPR, c = idx % Stage<DH>::LPR;
      st.v[i] = *reinterpret_cast<const u32x4*>(m + (int64_t)min(k0 + r, T - 1) * ld + 8 * c);
    }
  }
}

template <int DH, bool TR>
__device__ __forceinline__ void put(const Stage<DH>& st, char* lds) {
#pragma unroll
  for (int i = 0; i < Stage<DH>::PER; ++i) {
    const int idx = threadIdx.x + AT_THREADS * i;
    if (idx < Stage<DH>::CHUNKS) {
      const int r = idx / Stage<DH>::LPR, c = idx % Stage<DH>::LPR;
      *reinterpret_cast<u32x4*>(lds + (TR ? tr_off<DH>(r, c) : row_off<DH>(r, c))) = st.v[i];
    }
  }
}

// LDS stores of this wave done, then the workgroup barrier (no wait on the
// vector-memory counter: outstanding P/dS stores are left in flight).
__device__ __forceinline__ void tile_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// A operand of S^T = K Q^T (or dP^T = V dO^T) from a row-read tile: key row
// lane % 32, columns 16 ks + 8 (lane / 32) .. +7.
template <int DH>
__device__ __forceinline__ bf16x8 row_frag(const char* lds, int ks, int lane) {
  return *reinterpret_cast<const bf16x8*>(lds + row_off<DH>(lane & 31, 2 * ks + (lane >> 5)));
}

// A operand (rows m = tile columns rb..rb+31; k = 16 keys of step ks) from a
// transposed-read tile, in the key order of the S^T accumulator: lane half h
// takes keys ks*16 + 4h + 0..3 and ks*16 + 8 + 4h + 0..3.  Transposing read:
// lane s of a 16-lane group addresses key row kb + s/4, columns m..m+3, and
// receives column rb + 16*(group & 1) + s of four consecutive key rows.
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

// Key of accumulator register r for lane half h, relative to the tile start.
__device__ __forceinline__ int acc_key(int r, int h) { return (r >> 2) * 8 + 4 * h + (r & 3); }

// Work of a workgroup: 128 queries of one (batch, head), heaviest first.
struct Item {
  int qb;    // this wave's 32-query block
  int nkt;   // key tiles the workgroup walks
  int mine;  // key tiles this wave computes (0 past the sequence end)
  int b, hh;
};
__device__ __forceinline__ bool item_of(int T, int B, int H, Item& it) {
  const int nqb = (T + 31) / 32, nqg = (nqb + AT_WAVES - 1) / AT_WAVES;
  const int64_t id = blockIdx.x;
  if (id >= (int64_t)nqg * B * H) return false;
  const int z = (int)(id % (B * H));
  const int qg = nqg - 1 - (int)(id / (B * H));
  it.qb = qg * AT_WAVES + (int)(threadIdx.x >> 6);
  it.nkt = min(nqb, (qg + 1) * AT_WAVES);
  it.mine = it.qb < nqb ? it.qb + 1 : 0;
  it.b = z / H;
  it.hh = z % H;
  return true;
}

// Zero 4-key groups [kbeg, kend) of one row of a [T][T] bf16 matrix (this
// lane's half of every 8-key group).
__device__ __forceinline__ void zero_row(bf16_t* row, int kbeg, int kend, int h) {
  for (int k = kbeg + 4 * h; k < kend; k += 8) *reinterpret_cast<u32x2*>(row + k) = u32x2{0u, 0u};
}

// Forward.  Exponentials are taken base 2 on scores pre-multiplied by
// scale * log2(e) (the hardware exp2); P is rounded to bfloat16 after
// normalisation.  While a tile is used, the workgroup fetches the next one.
template <int DH>
__global__ __launch_bounds__(AT_THREADS) void attn_fwd_kernel(const bf16_t* __restrict__ qkv,
                                                              bf16_t* __restrict__ P,
                                                              bf16_t* __restrict__ O,
                                                              float* __restrict__ Of, int B, int H,
                                                              int T, float scale) {
  constexpr int KS = DH / 16, DB = DH / 32, TB = 32 * DH * 2;
  __shared__ __attribute__((aligned(1024))) char kbuf[2][TB];
  __shared__ __attribute__((aligned(1024))) char vbuf[2][TB];
  Item it;
  if (!item_of(T, B, H, it)) return;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  const int d = H * DH;
  const int64_t ld = 3 * (int64_t)d;
  const bf16_t* Qp = qkv + (int64_t)it.b * T * ld + it.hh * DH;
  const bf16_t* Kp = Qp + d;
  const bf16_t* Vp = Qp + 2 * d;
  const int q = it.qb * 32 + col, qc = min(q, T - 1);
  const float c2 = scale * 1.4426950408889634f;  // scale * log2(e)
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(Qp + qc * ld + 16 * ks + 8 * h);
  auto valid = [&](int key) { return key <= q && key < T; };
  auto scores = [&](const char* kt_lds) {
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(kt_lds, ks, lane), qf[ks], acc, 0, 0, 0);
    return acc;
  };
  Stage<DH> sk, sv;
  // pass 1: row maximum and sum of exponentials over this lane's keys
  float mx = -INFINITY, sm = 0.f;
  fetch<DH>(sk, Kp, ld, 0, T);
  put<DH, false>(sk, kbuf[0]);
  tile_barrier();
  for (int kt = 0; kt < it.nkt; ++kt) {
    if (kt + 1 < it.nkt) fetch<DH>(sk, Kp, ld, (kt + 1) * 32, T);
    if (kt < it.mine) {
      const f32x16 s = scores(kbuf[kt & 1]);
      float tmax = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (valid(kt * 32 + acc_key(r, h))) tmax = fmaxf(tmax, s[r] * c2);
      if (tmax > -INFINITY) {
        const float mn = fmaxf(mx, tmax);
        float acc = (mx > -INFINITY) ? sm * __builtin_amdgcn_exp2f(mx - mn) : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (valid(kt * 32 + acc_key(r, h))) acc += __builtin_amdgcn_exp2f(fmaf(s[r], c2, -mn));
        sm = acc;
        mx = mn;
      }
    }
    if (kt + 1 < it.nkt) put<DH, false>(sk, kbuf[(kt + 1) & 1]);
    tile_barrier();
  }
  // combine the two lane halves of the query
  const float mo = __shfl_xor(mx, 32, 64), so = __shfl_xor(sm, 32, 64);
  const float m = fmaxf(mx, mo);
  const float l = ((mx > -INFINITY) ? sm * __builtin_amdgcn_exp2f(mx - m) : 0.f) +
                  ((mo > -INFINITY) ? so * __builtin_amdgcn_exp2f(mo - m) : 0.f);
  const float inv = 1.0f / l;
  // pass 2: normalised P (stored), O^T += V^T P^T
  f32x16 oacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  const int64_t z = (int64_t)it.b * H + it.hh;
  bf16_t* Prow = P + (z * T + qc) * (int64_t)T;
  fetch<DH>(sk, Kp, ld, 0, T);
  fetch<DH>(sv, Vp, ld, 0, T);
  put<DH, false>(sk, kbuf[0]);
  put<DH, true>(sv, vbuf[0]);
  tile_barrier();
  for (int kt = 0; kt < it.nkt; ++kt) {
    if (kt + 1 < it.nkt) {
      fetch<DH>(sk, Kp, ld, (kt + 1) * 32, T);
      fetch<DH>(sv, Vp, ld, (kt + 1) * 32, T);
    }
    if (kt < it.mine) {
      const f32x16 s = scores(kbuf[kt & 1]);
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r)
        p[r] = valid(kt * 32 + acc_key(r, h)) ? __builtin_amdgcn_exp2f(fmaf(s[r], c2, -m)) * inv : 0.f;
      const bf16x8 pb0 = pack8(p), pb1 = pack8(p + 8);
      const char* vt = vbuf[kt & 1];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(vt, db * 32, 0, lane), pb0, oacc[db], 0, 0, 0);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(vt, db * 32, 1, lane), pb1, oacc[db], 0, 0, 0);
      }
      if (q < T) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int key = kt * 32 + g * 8 + 4 * h;
          if (key < T) {
            u32x2 w;
            w[0] = pack_bf2(p[4 * g], p[4 * g + 1]);
            w[1] = pack_bf2(p[4 * g + 2], p[4 * g + 3]);
            *reinterpret_cast<u32x2*>(Prow + key) = w;
          }
        }
      }
    }
    if (kt + 1 < it.nkt) {
      put<DH, false>(sk, kbuf[(kt + 1) & 1]);
      put<DH, true>(sv, vbuf[(kt + 1) & 1]);
    }
    tile_barrier();
  }
  if (q >= T) return;
  // zeros above the diagonal up to the end of the query's 128-row band
  zero_row(Prow, it.mine * 32, min(T, (it.qb * 32 / AT_ZERO_BAND + 1) * AT_ZERO_BAND), h);
  // O (bf16) and its float32 copy: lane holds query q, columns db*32 + acc_key(r, h)
  const int64_t orow = ((int64_t)it.b * T + q) * d + it.hh * DH;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c = db * 32 + g * 8 + 4 * h;
      u32x2 w;
      w[0] = pack_bf2(oacc[db][4 * g], oacc[db][4 * g + 1]);
      w[1] = pack_bf2(oacc[db][4 * g + 2], oacc[db][4 * g + 3]);
      *reinterpret_cast<u32x2*>(O + orow + c) = w;
      f32x4 f = {oacc[db][4 * g], oacc[db][4 * g + 1], oacc[db][4 * g + 2], oacc[db][4 * g + 3]};
      *reinterpret_cast<f32x4*>(Of + orow + c) = f;
    }
  }
}

// Backward: dS and dQ, with the same workgroup structure: V tiles (row read,
// for dP^T = V dO^T) and K tiles (transposed read, for dQ^T = K^T dS^T) are
// shared through LDS; each wave reads its own rows of P.
template <int DH>
__global__ __launch_bounds__(AT_THREADS) void attn_bwd_kernel(
    const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ P, const bf16_t* __restrict__ dO,
    const float* __restrict__ Of, bf16_t* __restrict__ dS, bf16_t* __restrict__ dQ, int B, int H,
    int T, float scale) {
  constexpr int KS = DH / 16, DB = DH / 32, TB = 32 * DH * 2;
  __shared__ __attribute__((aligned(1024))) char kbuf[2][TB];
  __shared__ __attribute__((aligned(1024))) char vbuf[2][TB];
  Item it;
  if (!item_of(T, B, H, it)) return;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, col = lane & 31;
  const int d = H * DH;
  const int64_t ld = 3 * (int64_t)d;
  const bf16_t* Kp = qkv + (int64_t)it.b * T * ld + d + it.hh * DH;
  const bf16_t* Vp = Kp + d;
  const int q = it.qb * 32 + col, qc = min(q, T - 1);
  const int64_t orow = ((int64_t)it.b * T + qc) * d + it.hh * DH;
  // dO^T operand and rowsum(dP * P) = dO . O (this lane's half of the columns)
  bf16x8 df[KS];
  float part = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
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
  const int64_t z = (int64_t)it.b * H + it.hh;
  const bf16_t* Prow = P + (z * T + qc) * (int64_t)T;
  bf16_t* dSrow = dS + (z * T + qc) * (int64_t)T;
  f32x16 qacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) qacc[i][r] = 0.f;
  auto load_p = [&](u32x2 (&pw)[4], int kt) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
      pw[g] = *reinterpret_cast<const u32x2*>(Prow + min(kt * 32 + g * 8 + 4 * h, T - 4));
  };
  u32x2 pw[4];
  Stage<DH> sk, sv;
  if (it.mine > 0) load_p(pw, 0);
  fetch<DH>(sk, Kp, ld, 0, T);
  fetch<DH>(sv, Vp, ld, 0, T);
  put<DH, true>(sk, kbuf[0]);
  put<DH, false>(sv, vbuf[0]);
  tile_barrier();
  for (int kt = 0; kt < it.nkt; ++kt) {
    if (kt + 1 < it.nkt) {
      fetch<DH>(sk, Kp, ld, (kt + 1) * 32, T);
      fetch<DH>(sv, Vp, ld, (kt + 1) * 32, T);
    }
    if (kt < it.mine) {
      // dP^T = V dO^T for this tile
      f32x16 acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
      const char* vt = vbuf[kt & 1];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<DH>(vt, ks, lane), df[ks], acc, 0, 0, 0);
      float ds[16];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int key = kt * 32 + g * 8 + 4 * h;
        const float pv[4] = {__builtin_bit_cast(float, pw[g][0] << 16), __builtin_bit_cast(float, pw[g][0] & 0xffff0000u),
                             __builtin_bit_cast(float, pw[g][1] << 16), __builtin_bit_cast(float, pw[g][1] & 0xffff0000u)};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          ds[4 * g + e] = (key + e <= q && key + e < T) ? scale * pv[e] * (acc[4 * g + e] - D) : 0.f;
      }
      if (kt + 1 < it.mine) load_p(pw, kt + 1);
      const bf16x8 sb0 = pack8(ds), sb1 = pack8(ds + 8);
      const char* ktl = kbuf[kt & 1];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        qacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(ktl, db * 32, 0, lane), sb0, qacc[db], 0, 0, 0);
        qacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_frag<DH>(ktl, db * 32, 1, lane), sb1, qacc[db], 0, 0, 0);
      }
      if (q < T) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int key = kt * 32 + g * 8 + 4 * h;
          if (key < T) {
            u32x2 w;
            w[0] = pack_bf2(ds[4 * g], ds[4 * g + 1]);
            w[1] = pack_bf2(ds[4 * g + 2], ds[4 * g + 3]);
            *reinterpret_cast<u32x2*>(dSrow + key) = w;
          }
        }
      }
    }
    if (kt + 1 < it.nkt) {
      put<DH, true>(sk, kbuf[(kt + 1) & 1]);
      put<DH, false>(sv, vbuf[(kt + 1) & 1]);
    }
    tile_barrier();
  }
  if (q >= T) return;
  zero_row(dSrow, it.mine * 32, min(T, (it.qb * 32 / AT_ZERO_BAND + 1) * AT_ZERO_BAND), h);
  // dQ (bf16) into the q columns of the dqkv rows
  const int64_t qrow = ((int64_t)it.b * T + q) * ld + it.hh * DH;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c = db * 32 + g * 8 + 4 * h;
      u32x2 w;
      w[0] = pack_bf2(qacc[db][4 * g], qacc[db][4 * g + 1]);
      w[1] = pack_bf2(qacc[db][4 * g + 2], qacc[db][4 * g + 3]);
      *reinterpret_cast<u32x2*>(dQ + qrow + c) = w;
    }
  }
}

}  // namespace

bool attention_fused_supported(int dh) { return dh == 32 || dh == 64 || dh == 128; }

hipError_t launch_attention_fwd(const bf16_t* qkv, bf16_t* P, bf16_t* O, float* Of, int B, int H,
                                int T, int dh, float scale, hipStream_t s) {
  if (T % 8) return hipErrorInvalidValue;
  const int64_t groups = cdiv(cdiv(T, 32), AT_WAVES) * B * H;
  const dim3 grid((unsigned)groups);
  switch (dh) {
    case 32: attn_fwd_kernel<32><<<grid, AT_THREADS, 0, s>>>(qkv, P, O, Of, B, H, T, scale); break;
    case 64: attn_fwd_kernel<64><<<grid, AT_THREADS, 0, s>>>(qkv, P, O, Of, B, H, T, scale); break;
    case 128: attn_fwd_kernel<128><<<grid, AT_THREADS, 0, s>>>(qkv, P, O, Of, B, H, T, scale); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention_bwd(const bf16_t* qkv, const bf16_t* P, const bf16_t* dO, const float* Of,
                                bf16_t* dS, bf16_t* dqkv, int B, int H, int T, int dh, float scale,
                                hipStream_t s) {
  if (T % 8) return hipErrorInvalidValue;
  const int64_t groups = cdiv(cdiv(T, 32), AT_WAVES) * B * H;
  const dim3 grid((unsigned)groups);
  switch (dh) {
    case 32: attn_bwd_kernel<32><<<grid, AT_THREADS, 0, s>>>(qkv, P, dO, Of, dS, dqkv, B, H, T, scale); break;
    case 64: attn_bwd_kernel<64><<<grid, AT_THREADS, 0, s>>>(qkv, P, dO, Of, dS, dqkv, B, H, T, scale); break;
    case 128: attn_bwd_kernel<128><<<grid, AT_THREADS, 0, s>>>(qkv, P, dO, Of, dS, dqkv, B, H, T, scale); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace layup
