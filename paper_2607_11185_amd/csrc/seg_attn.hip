// Masked GQA attention over packed VCS segments, forward and backward
// (the policy-update attention of Sec. 3.3 training items), bf16 MFMA on gfx950.
//
// Every segment is an independent attention unit.  A query row sees the keys of
// its segment that are not after it, except screenshot tokens more than W-1
// turns older than its own turn.  The layout's tile map lists, per 128-row
// q-tile, the k-tiles that hold at least one visible pair (CSR) and marks them
// FULL (every pair visible: no predicate) or PARTIAL (per-element predicate).
//
// MFMA v_mfma_f32_32x32x16_bf16 lane layout used throughout (lane l, c = l%32,
// h = l/32):  A[i][k]: i = c, k = 8h + 0..7;  B[k][j]: j = c, k = 8h + 0..7;
// D[i][j] (16 regs r): j = c, i = 8*(r/4) + 4h + r%4.
// Products that contract over the rows held in accumulator registers read the
// other operand from "transposed tiles" T[tile][head][d][128] whose positions
// follow kperm() inside each 16-row chunk (see common.h).
#include <climits>
#include <cmath>

#include "common.h"

namespace seg {
namespace {

constexpr int TQ = 128;  // tile edge
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

struct TileRows {
  int start, len, qbase, i, row0, nrows;  // row0 is segment-relative
};

__device__ __forceinline__ TileRows tile_rows(const int32_t *seg_info, const int32_t *tile_seg,
                                              int g) {
  TileRows t;
  const int s = tile_seg[g];
  const int32_t *si = seg_info + (long)s * SEG_INFO_FIELDS;
  t.start = si[SEG_INFO_START];
  t.len = si[SEG_INFO_LEN];
  t.qbase = si[SEG_INFO_QTILE_BASE];
  t.i = g - t.qbase;
  t.row0 = t.i * TQ;
  t.nrows = min(TQ, t.len - t.row0);
  return t;
}

__device__ __forceinline__ int key_expiry(int meta, int W) {
  return ((meta & 3) == SEG_KIND_IMAGE) ? (meta >> 2) + W : INT_MAX;
}

__device__ __forceinline__ bf16x8 lds8(const unsigned short *p) {
  return *reinterpret_cast<const bf16x8 *>(p);
}

__device__ __forceinline__ bf16x8 pack8(const f32x16 &v, int base) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)v[base + j];
  return r;
}

__device__ __forceinline__ u16x8 load8_bf(const unsigned short *p) {
  return *reinterpret_cast<const u16x8 *>(p);
}
__device__ __forceinline__ u16x8 load8_bf(const float *p) {
  const f32x4 a = *reinterpret_cast<const f32x4 *>(p);
  const f32x4 b = *reinterpret_cast<const f32x4 *>(p + 4);
  u16x8 r;
  r[0] = f2bf_bits(a[0]); r[1] = f2bf_bits(a[1]); r[2] = f2bf_bits(a[2]); r[3] = f2bf_bits(a[3]);
  r[4] = f2bf_bits(b[0]); r[5] = f2bf_bits(b[1]); r[6] = f2bf_bits(b[2]); r[7] = f2bf_bits(b[3]);
  return r;
}

// ------------------------------------------------------------- prep kernels

// Transposed tiles: T[(g*nh + h)][d][p] = X[row of position p][h][d] (bf16),
// zero beyond the tile's rows.
template <class TI, int D>
__global__ void __launch_bounds__(256) k_transpose_tiles(const TI *__restrict__ x, int nh,
                                                         const int32_t *__restrict__ seg_info,
                                                         const int32_t *__restrict__ tile_seg,
                                                         unsigned short *__restrict__ out) {
  constexpr int LD = D + 8;
  __shared__ unsigned short t[TQ * LD];
  const int g = blockIdx.x / nh, h = blockIdx.x % nh;
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  for (int c = threadIdx.x; c < TQ * D / 8; c += 256) {
    const int row = c / (D / 8), ch = c % (D / 8);
    u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
    if (row < tr.nrows)
      v = load8_bf(x + ((long)(tr.start + tr.row0 + row) * nh + h) * D + ch * 8);
    *reinterpret_cast<u16x8 *>(&t[row * LD + ch * 8]) = v;
  }
  __syncthreads();
  unsigned short *o = out + ((long)g * nh + h) * D * TQ;
  for (int c = threadIdx.x; c < D * TQ / 8; c += 256) {
    const int d = c / (TQ / 8), pc = c % (TQ / 8);
    u16x8 v;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int p = pc * 8 + j;
      v[j] = t[((p & ~15) | kperm(p & 15)) * LD + d];
    }
    *reinterpret_cast<u16x8 *>(o + d * TQ + pc * 8) = v;
  }
}

// fp32 -> bf16 copy (row-major, any shape)
__global__ void k_f32_to_bf16(const float *__restrict__ x, unsigned short *__restrict__ y, long n) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    y[i] = f2bf_bits(x[i]);
}

// Delta[h][row] = sum_d dO[row][h][d] * O[row][h][d]  (D/8 lanes per (row, head))
template <class TI, int D>
__global__ void __launch_bounds__(256) k_delta(const TI *__restrict__ o, const TI *__restrict__ dout,
                                               int hq, long P, float *__restrict__ delta) {
  constexpr int LPR = D / 8;  // lanes per (row, head)
  const long gid = (long)blockIdx.x * 256 + threadIdx.x;
  const long pair = gid / LPR;
  const int part = (int)(gid % LPR);
  const bool ok = pair < P * hq;
  float acc = 0.f;
  if (ok) {
    const long base = pair * D + part * 8;  // pair = row * hq + h
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float a, b;
      if constexpr (sizeof(TI) == 2) {
        a = bf_bits2f(((const unsigned short *)o)[base + j]);
        b = bf_bits2f(((const unsigned short *)dout)[base + j]);
      } else {
        a = ((const float *)o)[base + j];
        b = ((const float *)dout)[base + j];
      }
      acc += a * b;
    }
  }
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (ok && part == 0) {
    const long row = pair / hq;
    const int h = (int)(pair % hq);
    delta[(long)h * P + row] = acc;
  }
}

// ------------------------------------------------------------- forward

// One block = one q-tile x one query head; 4 waves of 32 query rows.
// S^T = K Q^T (keys on accumulator rows, queries on lanes), online softmax in
// the exp2 domain, O^T += V^T P^T with V^T from transposed tiles.
template <int D, class TO>
__global__ void __launch_bounds__(256, 2) k_attn_fwd(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ vt, const int32_t *__restrict__ seg_info,
    const int32_t *__restrict__ tile_seg, const int32_t *__restrict__ tok_meta,
    const int32_t *__restrict__ qt_ptr, const int32_t *__restrict__ qt_col,
    const uint8_t *__restrict__ qt_cls, const int32_t *__restrict__ work_order, int hq, int hkv,
    int W, float scale_log2, long P, TO *__restrict__ o, float *__restrict__ lse) {
  constexpr int KK = D / 16;   // k-steps over the head dim
  constexpr int CPR = D / 8;   // 16-byte chunks per K row
  constexpr int DB = D / 32;   // 32-row blocks of the head dim
  __shared__ unsigned short sK[TQ * D];
  __shared__ unsigned short sV[D * TQ];
  __shared__ int sKexp[TQ];

  const int g = work_order[blockIdx.x / hq];
  const int h = blockIdx.x % hq;
  const int hk = h / (hq / hkv);
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int qloc = wave * 32 + col;
  const bool qvalid = qloc < tr.nrows;
  const int qr = tr.row0 + qloc;  // segment-relative query row
  const int qstep = qvalid ? (tok_meta[tr.start + qr] >> 2) : 0;

  bf16x8 qf[KK];
  {
    const unsigned short *qrow = q + ((long)(tr.start + (qvalid ? qr : tr.row0)) * hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = lds8(qrow + kk * 16 + hh * 8);
      if (!qvalid) qf[kk] = bf16x8{};
    }
  }
  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  const int e0 = qt_ptr[g], e1 = qt_ptr[g + 1];
  for (int e = e0; e < e1; ++e) {
    const int gk = qt_col[e];
    const bool partial = qt_cls[e] == SEG_TILE_PARTIAL;
    const int k0 = (gk - tr.qbase) * TQ;
    const int krows = min(TQ, tr.len - k0);
    __syncthreads();
    for (int c = threadIdx.x; c < TQ * CPR; c += 256) {
      const int row = c / CPR, ch = c % CPR;
      u16x8 val = {0, 0, 0, 0, 0, 0, 0, 0};
      if (row < krows) val = load8_bf(k + ((long)(tr.start + k0 + row) * hkv + hk) * D + ch * 8);
      *reinterpret_cast<u16x8 *>(&sK[row * D + ((ch ^ (row & (CPR - 1))) * 8)]) = val;
    }
    {
      const unsigned short *vsrc = vt + ((long)gk * hkv + hk) * D * TQ;
      for (int c = threadIdx.x; c < D * 16; c += 256) {
        const int row = c >> 4, ch = c & 15;
        *reinterpret_cast<u16x8 *>(&sV[row * TQ + ((ch ^ (row & 15)) * 8)]) =
            load8_bf(vsrc + row * TQ + ch * 8);
      }
    }
    if (threadIdx.x < TQ) {
      const int kr = threadIdx.x;
      sKexp[kr] = kr < krows ? key_expiry(tok_meta[tr.start + k0 + kr], W) : INT_MIN;
    }
    __syncthreads();

    f32x16 sacc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      sacc[kb] = f32x16{};
      const int key = kb * 32 + col;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const int ch = kk * 2 + hh;
        sacc[kb] = mfma32(lds8(&sK[key * D + ((ch ^ (key & (CPR - 1))) * 8)]), qf[kk], sacc[kb]);
      }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float sv = sacc[kb][r] * scale_log2;
        if (partial) {
          const int key = kb * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
          const bool vis = qvalid && (k0 + key <= qr) && (qstep < sKexp[key]);
          sv = vis ? sv : -INFINITY;
        }
        sacc[kb][r] = sv;
        mloc = fmaxf(mloc, sv);
      }
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_run, mloc);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float rsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = exp2f(sacc[kb][r] - m_use);
        sacc[kb][r] = pv;
        rsum += pv;
      }
    }
    rsum += __shfl_xor(rsum, 32, 64);
    l_run = l_run * alpha + rsum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        const bf16x8 pf = pack8(sacc[kb], c2 * 8);
        const int chunk = kb * 4 + c2 * 2 + hh;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int dd = db * 32 + col;
          oacc[db] = mfma32(lds8(&sV[dd * TQ + ((chunk ^ (dd & 15)) * 8)]), pf, oacc[db]);
        }
      }
    }
  }

  if (qvalid) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    const long row = tr.start + qr;
    TO *orow = o + (row * hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = db * 32 + 8 * r4 + 4 * hh;
#pragma unroll
        for (int j = 0; j < 4; ++j) store_val(orow, d0 + j, oacc[db][r4 * 4 + j] * inv);
      }
    }
    if (hh == 0) lse[(long)h * P + row] = (m_run + log2f(l_run)) * LN2;
  }
}

// ------------------------------------------------------------- backward

// dK/dV: one block = one k-tile x one kv head; wave w owns keys 32w..32w+31.
// Loops over the q-tiles of the transposed CSR column and over the query heads
// of the group, in 64-row halves.  S = Q K^T has queries on accumulator rows
// and keys on lanes, so P and dS feed dV += P^T dO and dK += dS^T Q directly,
// with dO^T and Q^T from transposed tiles.
template <int D, class TO>
__global__ void __launch_bounds__(256, 1) k_attn_bwd_dkdv(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const unsigned short *__restrict__ dout,
    const unsigned short *__restrict__ qt, const unsigned short *__restrict__ dot,
    const float *__restrict__ lse, const float *__restrict__ delta,
    const int32_t *__restrict__ seg_info, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ tok_meta, const int32_t *__restrict__ kt_ptr,
    const int32_t *__restrict__ kt_row, const uint8_t *__restrict__ kt_cls, int hq, int hkv,
    int W, float scale_log2, float scale, long P, TO *__restrict__ dk, TO *__restrict__ dv) {
  constexpr int KK = D / 16, CPR = D / 8, DB = D / 32;
  constexpr int HQ = 64;  // query rows per half
  __shared__ unsigned short sQ[HQ * D];
  __shared__ unsigned short sdO[HQ * D];
  __shared__ unsigned short sQt[D * HQ];
  __shared__ unsigned short sdOt[D * HQ];
  __shared__ float sLse[HQ], sDelta[HQ];
  __shared__ int sQstep[HQ], sQrow[HQ];

  // k-tiles in natural order: within a segment the earliest k-tiles have the
  // longest transposed-CSR columns, so they start first.
  const int g = blockIdx.x / hkv;
  const int hk = blockIdx.x % hkv;
  const int grp = hq / hkv;
  const TileRows tr = tile_rows(seg_info, tile_seg, g);  // this k-tile
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int kloc = wave * 32 + col;
  const bool kvalid = kloc < tr.nrows;
  const int kr = tr.row0 + kloc;  // segment-relative key row
  const int kexp = kvalid ? key_expiry(tok_meta[tr.start + kr], W) : INT_MIN;

  bf16x8 kf[KK], vf[KK];
  {
    const long row = tr.start + (kvalid ? kr : tr.row0);
    const unsigned short *krow = k + (row * hkv + hk) * D;
    const unsigned short *vrow = v + (row * hkv + hk) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kf[kk] = lds8(krow + kk * 16 + hh * 8);
      vf[kk] = lds8(vrow + kk * 16 + hh * 8);
      if (!kvalid) {
        kf[kk] = bf16x8{};
        vf[kk] = bf16x8{};
      }
    }
  }
  f32x16 dkacc[DB], dvacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dkacc[db] = f32x16{};
    dvacc[db] = f32x16{};
  }

  const int e0 = kt_ptr[g], e1 = kt_ptr[g + 1];
  for (int e = e0; e < e1; ++e) {
    const int gq = kt_row[e];
    const bool partial = kt_cls[e] == SEG_TILE_PARTIAL;
    const int q0 = (gq - tr.qbase) * TQ;
    const int qrows = min(TQ, tr.len - q0);
    for (int hi = 0; hi < grp; ++hi) {
      const int h = hk * grp + hi;
      for (int half = 0; half < 2; ++half) {
        const int hq0 = half * HQ;  // first row of this half inside the q-tile
        if (hq0 >= qrows) break;
        __syncthreads();
        for (int c = threadIdx.x; c < HQ * CPR; c += 256) {
          const int row = c / CPR, ch = c % CPR;
          u16x8 a = {0, 0, 0, 0, 0, 0, 0, 0}, b = a;
          if (hq0 + row < qrows) {
            const long off = ((long)(tr.start + q0 + hq0 + row) * hq + h) * D + ch * 8;
            a = load8_bf(q + off);
            b = load8_bf(dout + off);
          }
          const int sw = (ch ^ (row & (CPR - 1))) * 8;
          *reinterpret_cast<u16x8 *>(&sQ[row * D + sw]) = a;
          *reinterpret_cast<u16x8 *>(&sdO[row * D + sw]) = b;
        }
        {
          const long tb = ((long)gq * hq + h) * D * TQ + hq0;
          for (int c = threadIdx.x; c < D * (HQ / 8); c += 256) {
            const int row = c / (HQ / 8), ch = c % (HQ / 8);
            const int sw = (ch ^ (row & 7)) * 8;
            *reinterpret_cast<u16x8 *>(&sQt[row * HQ + sw]) = load8_bf(qt + tb + row * TQ + ch * 8);
            *reinterpret_cast<u16x8 *>(&sdOt[row * HQ + sw]) = load8_bf(dot + tb + row * TQ + ch * 8);
          }
        }
        if (threadIdx.x < HQ) {
          const int r = threadIdx.x;
          const bool ok = hq0 + r < qrows;
          const long row = tr.start + q0 + hq0 + r;
          sLse[r] = ok ? lse[(long)h * P + row] * LOG2E : INFINITY;
          sDelta[r] = ok ? delta[(long)h * P + row] : 0.f;
          sQstep[r] = ok ? (tok_meta[row] >> 2) : INT_MAX;
          sQrow[r] = ok ? (q0 + hq0 + r) : -1;
        }
        __syncthreads();

#pragma unroll
        for (int qb = 0; qb < HQ / 32; ++qb) {
          f32x16 s = f32x16{}, dp = f32x16{};
          const int qrow = qb * 32 + col;
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            const int ch = kk * 2 + hh;
            const int sw = (ch ^ (qrow & (CPR - 1))) * 8;
            s = mfma32(lds8(&sQ[qrow * D + sw]), kf[kk], s);
            dp = mfma32(lds8(&sdO[qrow * D + sw]), vf[kk], dp);
          }
          // P and dS; accumulator row r holds query qb*32 + 8*(r/4) + 4*hh + r%4
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int ql = qb * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
            float pv = exp2f(s[r] * scale_log2 - sLse[ql]);
            bool vis = kvalid && sQrow[ql] >= 0;
            if (partial) vis = vis && (kr <= sQrow[ql]) && (sQstep[ql] < kexp);
            pv = vis ? pv : 0.f;
            s[r] = pv;
            dp[r] = pv * (dp[r] - sDelta[ql]);
          }
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) {
            const bf16x8 pa = pack8(s, c2 * 8);
            const bf16x8 dsa = pack8(dp, c2 * 8);
            const int chunk = qb * 4 + c2 * 2 + hh;  // 16-byte chunk of the transposed row
#pragma unroll
            for (int db = 0; db < DB; ++db) {
              const int dd = db * 32 + col;
              const int sw = (chunk ^ (dd & 7)) * 8;
              dvacc[db] = mfma32(pa, lds8(&sdOt[dd * HQ + sw]), dvacc[db]);
              dkacc[db] = mfma32(dsa, lds8(&sQt[dd * HQ + sw]), dkacc[db]);
            }
          }
        }
      }
    }
  }

  // accumulator D[i = key][j = d]: lane holds d = db*32 + col, rows are keys
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int dd = db * 32 + col;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int kl = wave * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
      if (kl < tr.nrows) {
        const long row = tr.start + tr.row0 + kl;
        store_val(dk, (row * hkv + hk) * D + dd, dkacc[db][r] * scale);
        store_val(dv, (row * hkv + hk) * D + dd, dvacc[db][r]);
      }
    }
  }
}

// dQ: one block = one q-tile x one query head; 4 waves of 32 query rows.
// Recomputes S^T = K Q^T and dP^T = V dO^T per 64-key half of each listed
// k-tile, then dQ^T += K^T dS^T with K^T from transposed tiles.
template <int D, class TO>
__global__ void __launch_bounds__(256, 2) k_attn_bwd_dq(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const unsigned short *__restrict__ dout,
    const unsigned short *__restrict__ kt, const float *__restrict__ lse,
    const float *__restrict__ delta, const int32_t *__restrict__ seg_info,
    const int32_t *__restrict__ tile_seg, const int32_t *__restrict__ tok_meta,
    const int32_t *__restrict__ qt_ptr, const int32_t *__restrict__ qt_col,
    const uint8_t *__restrict__ qt_cls, const int32_t *__restrict__ work_order, int hq, int hkv,
    int W, float scale_log2, float scale, long P, TO *__restrict__ dq) {
  constexpr int KK = D / 16, CPR = D / 8, DB = D / 32;
  constexpr int HK = 64;  // keys per half
  __shared__ unsigned short sK[HK * D];
  __shared__ unsigned short sV[HK * D];
  __shared__ unsigned short sKt[D * HK];
  __shared__ int sKexp[HK];

  const int g = work_order[blockIdx.x / hq];
  const int h = blockIdx.x % hq;
  const int hk = h / (hq / hkv);
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int qloc = wave * 32 + col;
  const bool qvalid = qloc < tr.nrows;
  const int qr = tr.row0 + qloc;
  const long qrow_abs = tr.start + (qvalid ? qr : tr.row0);
  const int qstep = qvalid ? (tok_meta[tr.start + qr] >> 2) : 0;
  const float lse2 = qvalid ? lse[(long)h * P + qrow_abs] * LOG2E : INFINITY;
  const float dlt = qvalid ? delta[(long)h * P + qrow_abs] : 0.f;

  bf16x8 qf[KK], df[KK];
  {
    const unsigned short *qp = q + (qrow_abs * hq + h) * D;
    const unsigned short *dp = dout + (qrow_abs * hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = lds8(qp + kk * 16 + hh * 8);
      df[kk] = lds8(dp + kk * 16 + hh * 8);
      if (!qvalid) {
        qf[kk] = bf16x8{};
        df[kk] = bf16x8{};
      }
    }
  }
  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dqacc[db] = f32x16{};

  const int e0 = qt_ptr[g], e1 = qt_ptr[g + 1];
  for (int e = e0; e < e1; ++e) {
    const int gk = qt_col[e];
    const bool partial = qt_cls[e] == SEG_TILE_PARTIAL;
    const int k0 = (gk - tr.qbase) * TQ;
    const int krows = min(TQ, tr.len - k0);
    for (int half = 0; half < 2; ++half) {
      const int hk0 = half * HK;
      if (hk0 >= krows) break;
      __syncthreads();
      for (int c = threadIdx.x; c < HK * CPR; c += 256) {
        const int row = c / CPR, ch = c % CPR;
        u16x8 a = {0, 0, 0, 0, 0, 0, 0, 0}, b = a;
        if (hk0 + row < krows) {
          const long off = ((long)(tr.start + k0 + hk0 + row) * hkv + hk) * D + ch * 8;
          a = load8_bf(k + off);
          b = load8_bf(v + off);
        }
        const int sw = (ch ^ (row & (CPR - 1))) * 8;
        *reinterpret_cast<u16x8 *>(&sK[row * D + sw]) = a;
        *reinterpret_cast<u16x8 *>(&sV[row * D + sw]) = b;
      }
      {
        const long tb = ((long)gk * hkv + hk) * D * TQ + hk0;
        for (int c = threadIdx.x; c < D * (HK / 8); c += 256) {
          const int row = c / (HK / 8), ch = c % (HK / 8);
          *reinterpret_cast<u16x8 *>(&sKt[row * HK + ((ch ^ (row & 7)) * 8)]) =
              load8_bf(kt + tb + row * TQ + ch * 8);
        }
      }
      if (threadIdx.x < HK) {
        const int r = threadIdx.x;
        sKexp[r] = hk0 + r < krows ? key_expiry(tok_meta[tr.start + k0 + hk0 + r], W) : INT_MIN;
      }
      __syncthreads();

#pragma unroll
      for (int kb = 0; kb < HK / 32; ++kb) {
        f32x16 s = f32x16{}, dp = f32x16{};
        const int key = kb * 32 + col;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          const int ch = kk * 2 + hh;
          const int sw = (ch ^ (key & (CPR - 1))) * 8;
          s = mfma32(lds8(&sK[key * D + sw]), qf[kk], s);
          dp = mfma32(lds8(&sV[key * D + sw]), df[kk], dp);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kl = kb * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
          float pv = exp2f(s[r] * scale_log2 - lse2);
          bool vis = qvalid && (sKexp[kl] != INT_MIN);
          if (partial) vis = vis && (k0 + hk0 + kl <= qr) && (qstep < sKexp[kl]);
          pv = vis ? pv : 0.f;
          s[r] = pv * (dp[r] - dlt);  // dS^T
        }
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          const bf16x8 dsb = pack8(s, c2 * 8);
          const int chunk = kb * 4 + c2 * 2 + hh;
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const int dd = db * 32 + col;
            dqacc[db] = mfma32(lds8(&sKt[dd * HK + ((chunk ^ (dd & 7)) * 8)]), dsb, dqacc[db]);
          }
        }
      }
    }
  }

  if (qvalid) {
    TO *qrowp = dq + (qrow_abs * hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = db * 32 + 8 * r4 + 4 * hh;
#pragma unroll
        for (int j = 0; j < 4; ++j) store_val(qrowp, d0 + j, dqacc[db][r4 * 4 + j] * scale);
      }
    }
  }
}

// ------------------------------------------------------------- host side

struct AttnWs {
  size_t vt, kt, qt, dot, delta, qb, kb, vb, ob, dob, total;
};

AttnWs attn_ws(const seg_sizes &sz, seg_dtype dt, int hq, int hkv, int d, int bwd) {
  AttnWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t G = (size_t)std::max(1, sz.num_qtiles);
  const size_t P = (size_t)std::max<int64_t>(1, sz.packed_tokens);
  const size_t tkv = G * hkv * d * TQ * 2, tq = G * hq * d * TQ * 2;
  if (!bwd) {
    w.vt = take(tkv);
  } else {
    w.kt = take(tkv);
    w.qt = take(tq);
    w.dot = take(tq);
    w.delta = take(P * hq * sizeof(float));
  }
  if (dt == SEG_F32) {
    w.qb = take(P * hq * d * 2);
    w.kb = take(P * hkv * d * 2);
    w.vb = take(P * hkv * d * 2);
    if (bwd) w.dob = take(P * hq * d * 2);
  }
  w.total = off;
  return w;
}

void check_common(const seg_layout *L, const seg_sizes *sz, seg_dtype dt, int hq, int hkv, int d) {
  SEG_CHECK(L && sz, SEG_ERR_ARG, "layout or sizes is NULL");
  SEG_CHECK(dt == SEG_BF16 || dt == SEG_F32, SEG_ERR_ARG, "unknown dtype %d", (int)dt);
  SEG_CHECK(hq >= 1 && hkv >= 1 && hq % hkv == 0, SEG_ERR_UNSUPPORTED,
            "need hq %% hkv == 0 (hq=%d, hkv=%d)", hq, hkv);
  SEG_CHECK(d == 64 || d == 128, SEG_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", d);
  SEG_CHECK(L->tile == TQ, SEG_ERR_UNSUPPORTED, "attention needs a layout with tile 128 (got %d)",
            L->tile);
  SEG_CHECK(L->window >= 1, SEG_ERR_ARG, "layout window not set (build the layout first)");
  SEG_CHECK((long)sz->packed_tokens * hq * d < (1L << 40), SEG_ERR_CAPACITY, "tensor too large");
}

template <class TI, int D>
void launch_transpose(const TI *x, int nh, const seg_layout *L, int G, unsigned short *out,
                      hipStream_t st) {
  ProfScope prof("attn_prep", st);
  k_transpose_tiles<TI, D><<<G * nh, 256, 0, st>>>(x, nh, L->seg_info, L->tile_seg, out);
  SEG_LAUNCH_CHECK();
}

template <class TI>
void transpose_any(int d, const TI *x, int nh, const seg_layout *L, int G, unsigned short *out,
                   hipStream_t st) {
  if (d == 128) launch_transpose<TI, 128>(x, nh, L, G, out, st);
  else launch_transpose<TI, 64>(x, nh, L, G, out, st);
}

void to_bf16(const void *x, unsigned short *y, long n, hipStream_t st) {
  int grid = (int)std::min<long>(65536, (n + 255) / 256);
  ProfScope prof("attn_prep", st);
  k_f32_to_bf16<<<std::max(1, grid), 256, 0, st>>>(static_cast<const float *>(x), y, n);
  SEG_LAUNCH_CHECK();
}

template <int D, class TO>
void fwd_impl(const seg_layout *L, const seg_sizes *sz, int hq, int hkv, float scale,
              const unsigned short *q, const unsigned short *k, const unsigned short *vt, void *o,
              float *lse, hipStream_t st) {
  const int G = sz->num_qtiles;
  ProfScope prof("attn_fwd", st);
  k_attn_fwd<D, TO><<<G * hq, 256, 0, st>>>(q, k, vt, L->seg_info, L->tile_seg, L->tok_meta,
                                            L->qt_ptr, L->qt_col, L->qt_cls, L->work_order, hq,
                                            hkv, L->window, scale * LOG2E, sz->packed_tokens,
                                            static_cast<TO *>(o), lse);
  SEG_LAUNCH_CHECK();
}

template <int D, class TO, class TI>
void bwd_impl(const seg_layout *L, const seg_sizes *sz, int hq, int hkv, float scale,
              const unsigned short *q, const unsigned short *k, const unsigned short *v,
              const unsigned short *dout, const TI *o_raw, const TI *dout_raw,
              const float *lse, unsigned short *kt, unsigned short *qt, unsigned short *dot,
              float *delta, void *dq, void *dk, void *dv, hipStream_t st) {
  const int G = sz->num_qtiles;
  const long P = sz->packed_tokens;
  {
    const long threads = P * hq * (D / 8);
    ProfScope prof("attn_delta", st);
    k_delta<TI, D><<<(int)((threads + 255) / 256), 256, 0, st>>>(o_raw, dout_raw, hq, P, delta);
    SEG_LAUNCH_CHECK();
  }
  launch_transpose<unsigned short, D>(k, hkv, L, G, kt, st);
  launch_transpose<unsigned short, D>(q, hq, L, G, qt, st);
  launch_transpose<unsigned short, D>(dout, hq, L, G, dot, st);
  {
  ProfScope prof("attn_bwd_dkdv", st);
  k_attn_bwd_dkdv<D, TO><<<G * hkv, 256, 0, st>>>(
      q, k, v, dout, qt, dot, lse, delta, L->seg_info, L->tile_seg, L->tok_meta, L->kt_ptr,
      L->kt_row, L->kt_cls, hq, hkv, L->window, scale * LOG2E, scale, P,
      static_cast<TO *>(dk), static_cast<TO *>(dv));
  SEG_LAUNCH_CHECK();
  }
  ProfScope prof("attn_bwd_dq", st);
  k_attn_bwd_dq<D, TO><<<G * hq, 256, 0, st>>>(
      q, k, v, dout, kt, lse, delta, L->seg_info, L->tile_seg, L->tok_meta, L->qt_ptr, L->qt_col,
      L->qt_cls, L->work_order, hq, hkv, L->window, scale * LOG2E, scale, P,
      static_cast<TO *>(dq));
  SEG_LAUNCH_CHECK();
}

}  // namespace
}  // namespace seg

using namespace seg;

extern "C" size_t seg_attn_workspace_bytes(const seg_sizes *sz, seg_dtype dt, int32_t hq,
                                           int32_t hkv, int32_t d, int32_t bwd) {
  if (!sz || hq < 1 || hkv < 1) return 0;
  return attn_ws(*sz, dt, hq, hkv, d, bwd).total;
}

extern "C" seg_status seg_attn_fwd(const seg_layout *L, const seg_sizes *sz, seg_dtype dt,
                                   int32_t hq, int32_t hkv, int32_t d, float softmax_scale,
                                   const void *q, const void *k, const void *v, void *o,
                                   float *lse, void *ws, size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    check_common(L, sz, dt, hq, hkv, d);
    const AttnWs w = attn_ws(*sz, dt, hq, hkv, d, 0);
    SEG_CHECK(ws_bytes >= w.total, SEG_ERR_WORKSPACE, "workspace of %zu bytes < required %zu",
              ws_bytes, w.total);
    if (sz->num_qtiles == 0) return;
    SEG_CHECK(q && k && v && o && lse && ws, SEG_ERR_ARG, "a tensor pointer is NULL");
    SEG_CHECK(std::isfinite(softmax_scale), SEG_ERR_ARG, "softmax_scale is not finite");
    char *base = static_cast<char *>(ws);
    const int G = sz->num_qtiles;
    const long P = sz->packed_tokens;
    unsigned short *vt = reinterpret_cast<unsigned short *>(base + w.vt);
    const unsigned short *qb, *kb;
    if (dt == SEG_F32) {
      unsigned short *q2 = reinterpret_cast<unsigned short *>(base + w.qb);
      unsigned short *k2 = reinterpret_cast<unsigned short *>(base + w.kb);
      to_bf16(q, q2, P * hq * d, stream);
      to_bf16(k, k2, P * hkv * d, stream);
      transpose_any(d, static_cast<const float *>(v), hkv, L, G, vt, stream);
      qb = q2;
      kb = k2;
    } else {
      transpose_any(d, static_cast<const unsigned short *>(v), hkv, L, G, vt, stream);
      qb = static_cast<const unsigned short *>(q);
      kb = static_cast<const unsigned short *>(k);
    }
    if (d == 128) {
      if (dt == SEG_F32) fwd_impl<128, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vt, o, lse, stream);
      else fwd_impl<128, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vt, o, lse, stream);
    } else {
      if (dt == SEG_F32) fwd_impl<64, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vt, o, lse, stream);
      else fwd_impl<64, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vt, o, lse, stream);
    }
  });
}

extern "C" seg_status seg_attn_bwd(const seg_layout *L, const seg_sizes *sz, seg_dtype dt,
                                   int32_t hq, int32_t hkv, int32_t d, float softmax_scale,
                                   const void *q, const void *k, const void *v, const void *o,
                                   const float *lse, const void *d_o, void *dq, void *dk, void *dv,
                                   void *ws, size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    check_common(L, sz, dt, hq, hkv, d);
    const AttnWs w = attn_ws(*sz, dt, hq, hkv, d, 1);
    SEG_CHECK(ws_bytes >= w.total, SEG_ERR_WORKSPACE, "workspace of %zu bytes < required %zu",
              ws_bytes, w.total);
    if (sz->num_qtiles == 0) return;
    SEG_CHECK(q && k && v && o && lse && d_o && dq && dk && dv && ws, SEG_ERR_ARG,
              "a tensor pointer is NULL");
    SEG_CHECK(std::isfinite(softmax_scale), SEG_ERR_ARG, "softmax_scale is not finite");
    char *base = static_cast<char *>(ws);
    const long P = sz->packed_tokens;
    unsigned short *kt = reinterpret_cast<unsigned short *>(base + w.kt);
    unsigned short *qt = reinterpret_cast<unsigned short *>(base + w.qt);
    unsigned short *dot = reinterpret_cast<unsigned short *>(base + w.dot);
    float *delta = reinterpret_cast<float *>(base + w.delta);
    const unsigned short *qb, *kb, *vb, *dob;
    if (dt == SEG_F32) {
      unsigned short *q2 = reinterpret_cast<unsigned short *>(base + w.qb);
      unsigned short *k2 = reinterpret_cast<unsigned short *>(base + w.kb);
      unsigned short *v2 = reinterpret_cast<unsigned short *>(base + w.vb);
      unsigned short *do2 = reinterpret_cast<unsigned short *>(base + w.dob);
      to_bf16(q, q2, P * hq * d, stream);
      to_bf16(k, k2, P * hkv * d, stream);
      to_bf16(v, v2, P * hkv * d, stream);
      to_bf16(d_o, do2, P * hq * d, stream);
      qb = q2; kb = k2; vb = v2; dob = do2;
      const float *o32 = static_cast<const float *>(o), *do32 = static_cast<const float *>(d_o);
      if (d == 128)
        bwd_impl<128, float, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, dob, o32, do32,
                                    lse, kt, qt, dot, delta, dq, dk, dv, stream);
      else
        bwd_impl<64, float, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, dob, o32, do32, lse,
                                   kt, qt, dot, delta, dq, dk, dv, stream);
    } else {
      qb = static_cast<const unsigned short *>(q);
      kb = static_cast<const unsigned short *>(k);
      vb = static_cast<const unsigned short *>(v);
      dob = static_cast<const unsigned short *>(d_o);
      const unsigned short *o16 = static_cast<const unsigned short *>(o);
      if (d == 128)
        bwd_impl<128, unsigned short, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb,
                                                      dob, o16, dob, lse, kt, qt, dot, delta, dq,
                                                      dk, dv, stream);
      else
        bwd_impl<64, unsigned short, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb,
                                                     dob, o16, dob, lse, kt, qt, dot, delta, dq,
                                                     dk, dv, stream);
    }
  });
}
