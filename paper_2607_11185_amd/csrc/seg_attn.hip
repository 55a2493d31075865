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
// Products that contract over the rows held in accumulator registers take
// their other operand from LDS through transpose reads in the same row order
// (kperm() in common.h).
#include <climits>
#include <cmath>
#include <mutex>
#include <type_traits>

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

// The window test of a key's turn/kind word (turn << 2 | kind) in one
// unsigned compare: with the kind bits xored with IMAGE and rotated to the
// top, an image key reads as its turn tau and any other kind as >= 2^30.  A
// query of turn t sees an image key iff t < tau + W, i.e. iff the rotated
// word is >= max(t - W + 1, 0).
__device__ __forceinline__ unsigned window_word(int meta) {
  return __builtin_rotateright32((unsigned)meta ^ SEG_KIND_IMAGE, 2);
}
__device__ __forceinline__ unsigned window_floor(int qstep, int W) {
  return (unsigned)max(qstep - W + 1, 0);
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

// fp32 -> bf16 copy (row-major, any shape)
__global__ void k_f32_to_bf16(const float *__restrict__ x, unsigned short *__restrict__ y, long n) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    y[i] = f2bf_bits(x[i]);
}

// Delta[h][row] = sum_d dO[row][h][d] * O[row][h][d]  (D/8 lanes per (row, head)),
// stored negated (the backward kernels start their dP accumulators from
// -Delta, so dP - Delta costs no instruction), and the row's log-sum-exp in
// log2 units for the backward kernels.
template <class TI, int D>
__global__ void __launch_bounds__(256) k_delta(const TI *__restrict__ o, const TI *__restrict__ dout,
                                               const float *__restrict__ lse, int hq, long P,
                                               float *__restrict__ delta, float *__restrict__ lse2) {
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
    delta[(long)h * P + row] = -acc;
    lse2[(long)h * P + row] = lse[(long)h * P + row] * LOG2E;
  }
}

// Largest squared key norm of each (segment, kv head), a bound on the
// forward's scores: |q . k| <= |q| |k|.  One block per (k-tile, kv head), two
// lanes per row; squared norms are >= 0, so their float bits order as
// unsigned integers and the maximum is an integer atomic (any order gives
// the same result).  The targets start at 0.
template <int D>
__global__ void __launch_bounds__(256) k_key_norm(const unsigned short *__restrict__ k,
                                                  const int32_t *__restrict__ seg_info,
                                                  const int32_t *__restrict__ tile_seg, int hkv,
                                                  unsigned *__restrict__ kn2) {
  constexpr int LPR = 256 / TQ, PER = D / LPR;
  const int g = blockIdx.x, hk = blockIdx.y;
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int r = threadIdx.x / LPR, part = threadIdx.x % LPR;
  float n2 = 0.f;
  if (r < tr.nrows) {
    const unsigned short *src = k + ((long)(tr.start + tr.row0 + r) * hkv + hk) * D + part * PER;
#pragma unroll
    for (int i = 0; i < PER; i += 8) {
      const bf16x8 x = lds8(src + i);
#pragma unroll
      for (int j = 0; j < 8; ++j) n2 = fmaf((float)x[j], (float)x[j], n2);
    }
  }
  n2 += __shfl_xor(n2, 1, 64);
#pragma unroll
  for (int off = 2; off < 64; off <<= 1) n2 = fmaxf(n2, __shfl_xor(n2, off, 64));
  __shared__ float wmax[4];
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = n2;
  __syncthreads();
  if (threadIdx.x == 0)
    atomicMax(kn2 + (long)tile_seg[g] * hkv + hk,
              __float_as_uint(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]))));
}

// ------------------------------------------------------------- pipelined kernels
//
// Tiles of 64 rows x d (row-major, bf16) are multi-buffered in LDS: the
// loads of the next unit are in flight while the current one is computed.
// Every kernel fills them with direct 16-byte buffer->LDS loads (see the
// note on wait counts below).  All tile loads go through buffer resources
// that start at the segment's first row, so a lane's offset inside a tile is
// fixed for the kernel and a unit adds one scalar; rows past the segment read
// as zeros.  Rows are stored with a 16-byte-chunk swizzle that keeps both
// 16-byte row reads (MFMA operands contracting over d; 16 lanes per LDS
// cycle) and 4x16 transpose reads (ds_read_b64_tr_b16: operands contracting
// over the rows; 32 lanes per cycle) free of bank conflicts on 64 four-byte
// banks, so no transposed copy of any tensor is needed.  Every lane's swizzled offsets are computed once;
// inside the loops a read is a register offset plus an immediate.

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

// 16-byte chunk swizzle of row `row`: a bijection on row % 16 (a 16-lane row
// read of one logical chunk hits 16 distinct chunks), and rows 4m..4m+3 differ
// in bits 2-3 (a 32-lane transpose read of 4 rows x 4 chunks hits 16 distinct
// chunks).  For d = 64 two rows share one 256-byte bank line, so the same two
// properties are built from row / 2.
template <int D>
__device__ __forceinline__ int swz(int row) {
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}

// element offset of (row, col) in a swizzled row-major tile of d columns
template <int D>
__device__ __forceinline__ int toff(int row, int col) {
  return row * D + (((col >> 3) ^ swz<D>(row)) << 3) + (col & 7);
}

// Per-lane byte offsets into a 64-row tile, valid for any row block R that is
// a multiple of 16 (the swizzle depends on row % 16 only).
template <int D>
struct LaneOffsets {
  static constexpr int KK = D / 16, DB = D / 32;
  int row[KK];     // 16-byte read of row R + lane%32, chunk 2*kk + lane/32
  int tra[DB];     // transpose reads: rows R + 4h + (lane%16)/4 (+8 for trb),
  int trb[DB];     // columns nb0 + 32*db + 16*((lane/16)%2) + 4*(lane%4)
  __device__ __forceinline__ void init(int lane, int nb0) {
    const int col = lane & 31, hh = lane >> 5, l16 = lane & 15, g = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) row[kk] = toff<D>(col, (kk * 2 + hh) * 8) * 2;
    const int r = 4 * hh + (l16 >> 2);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int c = nb0 + db * 32 + 16 * (g & 1) + 4 * (l16 & 3);
      tra[db] = toff<D>(r, c) * 2;
      trb[db] = toff<D>(r + 8, c) * 2;
    }
  }
};

template <int D>
__device__ __forceinline__ bf16x8 frag_row(const char *tile, int R, int off) {
  return *reinterpret_cast<const bf16x8 *>(tile + R * D * 2 + off);
}

// Operand fragment contracting over tile rows: lane l receives column
// n(l) of rows R + kperm(8h + j), j = 0..7 (h = l/32), the MFMA k-order of
// accumulator-held operands.
// `bias` is a constant already added to offa and offb (see the dK/dV kernel).
template <int D>
__device__ __forceinline__ bf16x8 frag_tr(const char *tile, int R, int offa, int offb,
                                          int bias = 0) {
  const v4i16 a =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)(tile + (R * D * 2 - bias + offa)));
  const v4i16 b =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)(tile + (R * D * 2 - bias + offb)));
  const bf16x4 a4 = __builtin_bit_cast(bf16x4, a), b4 = __builtin_bit_cast(bf16x4, b);
  bf16x8 r;
  r[0] = a4[0]; r[1] = a4[1]; r[2] = a4[2]; r[3] = a4[3];
  r[4] = b4[0]; r[5] = b4[1]; r[6] = b4[2]; r[7] = b4[3];
  return r;
}

// Raw buffer resource over [base, base + bytes): loads past the end return
// zeros, so a tile fill needs no clamping of its rows.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// Direct buffer->LDS fill of a 64-row tile by NW waves: per-lane byte offsets
// are fixed for the kernel (tile row * row stride + swizzled chunk); a unit
// only adds its first row's byte offset (a scalar).
template <int D, int NW>
struct BufFill {
  static constexpr int CPR = D / 8, PW = 64 * CPR / (64 * NW);
  int voff[PW];
  __device__ __forceinline__ void init(int wave, int lane, int row_bytes) {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int s = (wave * PW + i) * 64 + lane;
      const int row = s / CPR;
      voff[i] = row * row_bytes + ((s % CPR) ^ swz<D>(row)) * 16;
    }
  }
  __device__ __forceinline__ void issue(unsigned short *tile, __amdgpu_buffer_rsrc_t rs, int soff,
                                        int wave) const {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
    for (int i = 0; i < PW; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void *)(tile + (wave * PW + i) * 64 * 8), 16,
          voff[i], soff, 0, 0);
#endif
  }
};

// one dword per lane (lane l: byte l*4 + soff) into 64 consecutive dwords of LDS
__device__ __forceinline__ void buf64_dw(void *dst, __amdgpu_buffer_rsrc_t rs, int lane, int soff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void *)dst, 4,
                                           lane * 4, soff, 0, 0);
#endif
}

// Software pipelining over units.  The loads of unit n+1 are issued, then
// unit n is computed from the other buffer, then a barrier ends the step.
// With direct loads, both happen inside one always-inline step whose LDS
// buffers are distinct __restrict__ parameters: a direct load's LDS write is
// counted with the global loads, and without the no-alias facts the compiler
// would wait for the loads in flight before the first LDS read of the
// compute.  Every LDS access of a step goes through those parameters (an
// access without them, such as one indexed by a run-time buffer number, waits
// for every direct load in flight).  While a direct load is in flight the
// compiler also gives up counted LDS waits (every wait becomes lgkmcnt(0)),
// which serialises read-ahead.

__device__ __forceinline__ void wait_all_and_sync() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// sum of 8 bf16 values (fp32 accumulation)
__device__ __forceinline__ float sum8(const bf16x8 &v, float acc) {
  const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
  for (int i = 0; i < 4; ++i)
    acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v[2 * i], v[2 * i + 1]}, one, acc, false);
  return acc;
}

// XCD-aware block mapping.  Blocks are dispatched round-robin over the 8
// XCDs (block b runs on XCD b % 8), each with its own L2.  XCD x takes the
// contiguous tile range [r.b[x], r.b[x+1]) chosen by the layout so that the
// ranges hold about equal work (the kernel ends with the slowest XCD), and
// runs it kv head by kv head, with the grp query heads of one tile back to
// back: those heads read the same key/value tiles, and neighbouring tiles of
// a segment read mostly the same ones, so the blocks resident on one XCD
// share one kv head's tiles in its L2 (the whole range of one kv head before
// the next measured 1.5-2% faster for the forward and dQ than all nh heads
// of a tile back to back).  `reverse` walks the range from its end (the
// longest rows of each segment first).  The grid is 8 * max range * nh
// blocks; blocks past their XCD's range exit at once.
struct XcdRanges {
  int32_t b[9];
};

__device__ __forceinline__ bool xcd_block(const XcdRanges &r, int nh, int grp, bool reverse,
                                          int &tile, int &head) {
  const int bx = blockIdx.x, x = bx & 7, i = bx >> 3;
  const int lo = r.b[x], C = r.b[x + 1] - lo;
  const int per = C * grp;  // blocks of one kv head's query heads over the range
  if (per == 0) return false;
  const int hk = i / per;
  if (hk >= nh / grp) return false;
  const int rem = i - hk * per;
  const int t = rem / grp;
  head = hk * grp + (rem - t * grp);
  tile = lo + (reverse ? C - 1 - t : t);
  return true;
}

inline XcdRanges xcd_ranges(const int32_t (&b)[9]) {
  XcdRanges r;
  for (int i = 0; i < 9; ++i) r.b[i] = b[i];
  return r;
}

inline int xcd_grid(const XcdRanges &r, int nh) {
  int c = 0;
  for (int x = 0; x < 8; ++x) c = std::max(c, r.b[x + 1] - r.b[x]);
  return std::max(1, 8 * c * nh);
}

// A unit of work: 64 rows (half of a 128-row tile) of the tile listed at CSR
// entry e.
struct Unit {
  int e, half;
  int r0;       // segment-relative first row of the unit
  int vrows;    // valid rows (1..64)
  int partial;  // PARTIAL tile (an int: a struct without padding bytes is
                // copied field by field, never through private memory)
};

// Unit (e, half) of a q-tile's walking order (`qt_ord`: the global k-tile
// index, bit 31 set for PARTIAL), read as a uniform load through the scalar
// cache (which measured faster than staging the entries in LDS).
__device__ __forceinline__ Unit make_unit(const int32_t *ord, int e, int half, int qbase,
                                          int seg_len) {
  Unit u;
  u.e = e;
  u.half = half;
  const unsigned x = (unsigned)ord[e];
  const int t0 = ((int)(x & 0x7fffffffu) - qbase) * TQ;
  u.r0 = t0 + half * 64;
  u.vrows = min(64, seg_len - u.r0);
  u.partial = (int)(x >> 31);
  return u;
}

// next unit: the second half of the same tile when it has rows, else the next entry
__device__ __forceinline__ bool next_unit(const Unit &u, int e1, const int32_t *ord, int qbase,
                                          int seg_len, Unit &nu) {
  if (u.half == 0 && u.r0 + 64 < seg_len) {
    nu = make_unit(ord, u.e, 1, qbase, seg_len);
    return true;
  }
  if (u.e + 1 < e1) {
    nu = make_unit(ord, u.e + 1, 0, qbase, seg_len);
    return true;
  }
  return false;
}

// The q-tile-stationary kernels walk a q-tile's units in the order of
// `qt_ord`, every FULL unit first and the PARTIAL ones after (measured about
// 3% faster for dQ and 1.5% for the forward than ascending k-tiles, where
// the PARTIAL units of expired turns' text sit between FULL ones; running
// the FULL units in a loop of their own, without the masking branch, gained
// nothing more).  Units alternate between two LDS buffers; `step(u, more,
// nu, current..., next...)` issues the loads of `nu` and computes `u`.
template <class Step, class Issue, class Next>
__device__ __forceinline__ void walk_units(Unit u, const Step &step, const Issue &issue,
                                           const Next &next, unsigned short *__restrict__ k0,
                                           unsigned short *__restrict__ v0, int *__restrict__ m0,
                                           unsigned short *__restrict__ k1,
                                           unsigned short *__restrict__ v1, int *__restrict__ m1) {
  Unit nu;
  issue(u, k0, v0, m0);
  wait_all_and_sync();
  for (;;) {
    bool more = next(u, nu);
    step(u, more, nu, k0, v0, m0, k1, v1, m1);
    __syncthreads();
    if (!more) return;
    u = nu;
    more = next(u, nu);
    step(u, more, nu, k1, v1, m1, k0, v0, m0);
    __syncthreads();
    if (!more) return;
    u = nu;
  }
}

// Forward: one block = one q-tile x one query head, 4 waves of 32 query rows;
// units are 64-key halves of the listed k-tiles.  S^T = K Q^T keeps one query
// per lane, so the online softmax is in-lane (plus one exchange with the
// other half-wave); O^T += V^T P^T with V^T by transpose reads.
template <int D, class TO>
__global__ void __launch_bounds__(256, 2) k_attn_fwd(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const int32_t *__restrict__ seg_info,
    const int32_t *__restrict__ tile_seg, const int32_t *__restrict__ tok_meta,
    const int32_t *__restrict__ qt_ptr, const int32_t *__restrict__ qt_ord,
    const float *__restrict__ kn2, const XcdRanges xr, int hq, int hkv, int W, float scale_log2,
    long P, TO *__restrict__ o, float *__restrict__ lse) {
  constexpr int KK = D / 16, DB = D / 32, T64 = 64 * D;
  __shared__ __attribute__((aligned(16))) unsigned short sK0[T64], sK1[T64], sV0[T64], sV1[T64];
  __shared__ __attribute__((aligned(16))) int sM0[64], sM1[64];

  int g, h;
  if (!xcd_block(xr, hq, hq / hkv, true, g, h)) return;
  const int hk = h / (hq / hkv);
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int qloc = wave * 32 + col;
  const bool qvalid = qloc < tr.nrows;
  const int qr = tr.row0 + (qvalid ? qloc : 0);
  const int qstep = tok_meta[tr.start + qr] >> 2;

  bf16x8 qf[KK];
  {
    const unsigned short *qrow = q + ((long)(tr.start + qr) * hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = lds8(qrow + kk * 16 + hh * 8);
  }
  // Fixed offset: when |q| max|k| * scale * log2(e) <= 64 for every row of
  // the wave (max over the segment's keys), every score in log2 units lies
  // in [-64, 64], so P = exp2(S) needs no running max (P and its sums stay
  // within fp32 and bf16 range, and relative precision does not depend on
  // the offset).  Other waves keep the lazily rescaled running max.
  bool zoff;
  {
    float qn2 = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int j = 0; j < 8; ++j) qn2 = fmaf((float)qf[kk][j], (float)qf[kk][j], qn2);
    qn2 += __shfl_xor(qn2, 32, 64);
    const float kmax2 = kn2[(long)tile_seg[g] * hkv + hk];
    zoff = __all(!qvalid || qn2 * kmax2 * (scale_log2 * scale_log2) <= 4096.f);
  }
  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = zoff ? 0.f : -INFINITY, l_run = 0.f;

  LaneOffsets<D> lo;
  lo.init(lane, 0);
  const long kv_stride = (long)hkv * D;
  const int row_bytes = (int)(kv_stride * 2);
  BufFill<D, 4> fp;
  fp.init(wave, lane, row_bytes);
  // the segment's rows of this kv head; rows past the segment read as zeros
  const __amdgpu_buffer_rsrc_t rK =
      make_rsrc(k + (long)hk * D + (long)tr.start * kv_stride, (unsigned)tr.len * row_bytes);
  const __amdgpu_buffer_rsrc_t rV =
      make_rsrc(v + (long)hk * D + (long)tr.start * kv_stride, (unsigned)tr.len * row_bytes);
  const __amdgpu_buffer_rsrc_t rM = make_rsrc(tok_meta + tr.start, (unsigned)tr.len * 4);

  auto issue = [&](const Unit &u, unsigned short *__restrict__ nK, unsigned short *__restrict__ nV,
                   int *__restrict__ nM) __attribute__((always_inline)) {
    fp.issue(nK, rK, u.r0 * row_bytes, wave);
    fp.issue(nV, rV, u.r0 * row_bytes, wave);
    if (wave == 0) buf64_dw(nM, rM, lane, u.r0 * 4);
  };
  auto compute = [&](const Unit &u, const char *__restrict__ sK, const char *__restrict__ sV,
                     const int *__restrict__ sM) __attribute__((always_inline)) {
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 ak[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) ak[kk] = frag_row<D>(sK, kb * 32, lo.row[kk]);
      sacc[kb] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) sacc[kb] = mfma32(ak[kk], qf[kk], sacc[kb]);
    }
    // raw scores; masked entries -inf (scale > 0 keeps the order).  The
    // forward keeps the direct per-element test: with the cheaper form of
    // the backward kernels the compiler schedules the unmasked path of this
    // kernel less well (the forward ran 1% slower in measurement).
    if (__builtin_expect(u.partial, 0)) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int kb0 = kb * 32 + 8 * rg + 4 * hh;
          const i32x4 M4 = *reinterpret_cast<const i32x4 *>(sM + kb0);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // bitwise, not short-circuit: no branch per element
            const int key = kb0 + j;
            const bool vis = qvalid & (key < u.vrows) & (u.r0 + key <= qr) &
                             (qstep < key_expiry(M4[j], W));
            sacc[kb][rg * 4 + j] = vis ? sacc[kb][rg * 4 + j] : -INFINITY;
          }
        }
    }
    if (!zoff) {
      float mloc = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sacc[kb][r]);
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * scale_log2;
      // Lazy rescaling: the running max (log2 units) only moves when a row's
      // tile max exceeds it by more than 8, so unnormalised P stays below 2^8.
      const bool grow = mloc > m_run + 8.f;
      if (__any(grow)) {
        // lanes that keep their max keep alpha = 1: with an unset (-inf)
        // max, exp2(m_run - m_new) would be exp2(NaN)
        const float m_new = grow ? mloc : m_run;
        const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
        m_run = m_new;
      }
    }
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    bf16x8 pf[2][2];
    float rsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sacc[kb][r] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][r], scale_log2, -m_use));
      pf[kb][0] = pack8(sacc[kb], 0);
      pf[kb][1] = pack8(sacc[kb], 8);
      rsum = sum8(pf[kb][0], rsum);
      rsum = sum8(pf[kb][1], rsum);
    }
    // l_run holds the sum over this lane's keys only: both half-waves of a
    // row share its max and rescale factors, so their sums are combined once
    // at the end
    l_run += rsum;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        bf16x8 av[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db)
          av[db] = frag_tr<D>(sV, kb * 32 + c2 * 16, lo.tra[db], lo.trb[db]);
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] = mfma32(av[db], pf[kb][c2], oacc[db]);
      }
  };
  auto step = [&](const Unit &u, const bool more, const Unit &nu,
                  const unsigned short *__restrict__ cK, const unsigned short *__restrict__ cV,
                  const int *__restrict__ cM, unsigned short *__restrict__ nK,
                  unsigned short *__restrict__ nV, int *__restrict__ nM)
                  __attribute__((always_inline)) {
    if (more) issue(nu, nK, nV, nM);
    compute(u, reinterpret_cast<const char *>(cK), reinterpret_cast<const char *>(cV), cM);
  };

  const int e0 = qt_ptr[g], e1 = qt_ptr[g + 1];
  auto next = [&](const Unit &u, Unit &n) __attribute__((always_inline)) -> bool {
    return next_unit(u, e1, qt_ord, tr.qbase, tr.len, n);
  };
  walk_units(make_unit(qt_ord, e0, 0, tr.qbase, tr.len), step, issue, next, sK0, sV0, sM0,
             sK1, sV1, sM1);

  l_run += __shfl_xor(l_run, 32, 64);
  if (qvalid) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    const long row = tr.start + qr;
    TO *orow = o + (row * hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = db * 32 + 8 * r4 + 4 * hh;
#pragma unroll
        for (int j = 0; j < 4; ++j) store_val(orow, d0 + j, oacc[db][r4 * 4 + j] * inv);
      }
    if (hh == 0) lse[(long)h * P + row] = (m_run + log2f(l_run)) * LN2;
  }
}

// dK/dV: one block = one k-tile x one kv head, 8 waves, two per SIMD.  Waves
// 0-3 (the P side) each hold K of 32 keys and their dV accumulator; waves
// 4-7 (the dS side) hold V of the same 32 keys and their dK accumulator.  A
// unit is 64 rows of one query head; per 32-row block:
//   P side:  S = Q K^T, P = exp2(S * scale - lse) (masked pairs give 0),
//            P -> LDS, dV += P^T dO
//   dS side: dP = dO V^T, P <- LDS, dS = P (dP - Delta), dK += dS^T Q
// The dS side works one unit behind the P side, so the P of a unit crosses
// the barrier that ends a step; Q/dO tiles therefore live in three buffers
// (the P side's unit, the dS side's unit, and the next unit being loaded;
// the step is unrolled three ways so that each is a compile-time buffer).
// Units are 64-row halves of the listed q-tiles, for every query head of the
// group, in the order of `kt_ord` (FULL q-tiles first, then the PARTIAL
// ones, each from the segment's last q-tile down).  No atomics.
template <int D, class TO>
__global__ void __launch_bounds__(512, 1) k_attn_bwd_dkdv(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const unsigned short *__restrict__ dout,
    const float *__restrict__ lse2, const float *__restrict__ delta,
    const int32_t *__restrict__ seg_info, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ tok_meta, const int32_t *__restrict__ kt_ptr,
    const int32_t *__restrict__ kt_ord, const XcdRanges xr,
    int hq, int hkv, int W,
    float scale_log2, float scale, long P, TO *__restrict__ dk, TO *__restrict__ dv) {
  constexpr int KK = D / 16, T64 = 64 * D, DB = D / 32, NB = 3;
  // three Q/dO buffers (and their per-row values) as distinct objects, so
  // that the direct loads into one provably write other LDS than the reads
  // of the other two
  // Q/dO tiles first (LDS is laid out by decreasing alignment), buffers 0
  // and 1 in the low 64 KB and buffer 2 above it
  __shared__ __attribute__((aligned(1024))) unsigned short sQ0[T64], sQ1[T64], sD0[T64], sD1[T64];
  __shared__ __attribute__((aligned(512))) unsigned short sQ2[T64], sD2[T64];
  __shared__ __attribute__((aligned(16))) unsigned short sP[2][64 * TQ];
  __shared__ __attribute__((aligned(16))) float sL0[64], sL1[64], sL2[64];
  __shared__ __attribute__((aligned(16))) float sE0[64], sE1[64], sE2[64];
  __shared__ __attribute__((aligned(16))) int sM0[64], sM1[64], sM2[64];

  int g, hk;
  {
    // XCD x takes the tiles of its range in order and runs them kv head by
    // kv head, so the blocks resident on one XCD are neighbouring k-tiles of
    // one kv head: they walk the same q-tiles of a segment and share their
    // Q/dO tiles in L2 (ordering the range longest column first instead mixes
    // segments and was 7% slower)
    const int bx = blockIdx.x, x = bx & 7, i = bx >> 3;
    const int lo = xr.b[x], C = xr.b[x + 1] - lo;
    if (C == 0) return;
    hk = i / C;
    if (hk >= hkv) return;
    g = lo + (i - hk * C);
  }
  const int grp = hq / hkv;
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int side = wave >> 2, kg = wave & 3;  // side 0: P, dV; side 1: dS, dK
  const int col = lane & 31, hh = lane >> 5;
  const int kloc = kg * 32 + col;
  const bool kvalid = kloc < tr.nrows;
  const int kr = tr.row0 + (kvalid ? kloc : 0);
  // a query row sees the lane's key only if its turn/kind word is below
  // kexp4 = 4 x (the key's expiry turn), INT_MAX for keys that never expire
  const int kexp = key_expiry(tok_meta[tr.start + kr], W);
  const int kexp4 = kexp >= (1 << 29) ? INT_MAX : kexp << 2;

  // K fragments (P side) or V fragments (dS side) of the wave's 32 keys
  bf16x8 xf[KK];
  {
    const long row = tr.start + kr;
    const unsigned short *src = (side == 0 ? k : v) + (row * hkv + hk) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) xf[kk] = lds8(src + kk * 16 + hh * 8);
  }
  f32x16 acc[DB];  // dV (P side) or dK (dS side): D[i = key][j = d]
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};

  LaneOffsets<D> lo;
  lo.init(lane, 0);
  // Transposed-read offsets with 64 KB added, hidden from the compiler: for
  // d = 128 a tile of buffer 2 lies above the 64 KB that an LDS
  // instruction's offset field reaches, and with these its reads carry the
  // tile's address in that field instead of adding it to the lane offset per
  // read.
  constexpr int HIBUF = 2, HIBIAS = 65536;
  constexpr bool HIGH2 = 4 * T64 * 2 >= HIBIAS;  // buffers 0 and 1 fill the low 64 KB
  int trah[DB], trbh[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    trah[db] = lo.tra[db] + HIBIAS;
    trbh[db] = lo.trb[db] + HIBIAS;
    asm volatile("" : "+v"(trah[db]), "+v"(trbh[db]));
  }
  const long q_stride = (long)hq * D;
  const int e0 = kt_ptr[g], e1 = kt_ptr[g + 1];

  // Fill of one unit by all 8 waves with direct buffer->LDS loads: Q and dO
  // rows, and one per-row value by waves 0-2 (log2-sum-exp, Delta, turn).
  // The Q/dO resources start at the segment's first row of the group's first
  // head and a unit adds a scalar byte offset; the per-row resources cover
  // one head's rows of the segment, so rows past the segment (the next
  // segment's, or buffer padding whose log-sum-exp and Delta were never
  // computed) read as zeros and no non-finite value can reach dS = P (dP -
  // Delta) through a masked P = 0.
  const int qrow_bytes = (int)(q_stride * 2);
  BufFill<D, 8> fq;
  fq.init(wave, lane, qrow_bytes);
  const long hbase = (long)hk * grp * D + (long)tr.start * q_stride;
  const unsigned qbytes = (unsigned)(tr.len * (long)qrow_bytes);
  const __amdgpu_buffer_rsrc_t rQ = make_rsrc(q + hbase, qbytes);
  const __amdgpu_buffer_rsrc_t rO = make_rsrc(dout + hbase, qbytes);
  // the wave index as a scalar: the resources and the direct loads' LDS
  // addresses are then built in scalar registers (a resource held in vector
  // registers needs a waterfall loop around every load)
  const int swave = __builtin_amdgcn_readfirstlane(wave);
  const unsigned rbytes = (unsigned)tr.len * 4;
  auto issue = [&](int r0, int hi, unsigned short *__restrict__ nQ, unsigned short *__restrict__ nD,
                   float *__restrict__ nL, float *__restrict__ nE, int *__restrict__ nM)
                   __attribute__((always_inline)) {
    const int so = r0 * qrow_bytes + hi * D * 2;
    fq.issue(nQ, rQ, so, swave);
    fq.issue(nD, rO, so, swave);
    if (swave < 3) {
      const long hrow = (long)(hk * grp + hi) * P + tr.start;
      const __amdgpu_buffer_rsrc_t rS =
          make_rsrc(swave == 0 ? (const void *)(lse2 + hrow)
                    : swave == 1 ? (const void *)(delta + hrow)
                                 : (const void *)(tok_meta + tr.start),
                    rbytes);
      buf64_dw(swave == 0 ? (void *)nL : swave == 1 ? (void *)nE : (void *)nM, rS, lane, r0 * 4);
    }
  };

  // P side: one unit (rows r0 .. r0 + vrows - 1, PARTIAL or ragged if masked)
  auto p_side = [&](auto hi_tag, const int r0, const int vrows, const bool masked,
                    const unsigned short *__restrict__ bQ, const unsigned short *__restrict__ bD,
                    const float *__restrict__ bL, const int *__restrict__ bM,
                    unsigned short *__restrict__ bP) __attribute__((always_inline)) {
    const char *cQ = reinterpret_cast<const char *>(bQ);
    const char *cD = reinterpret_cast<const char *>(bD);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      bf16x8 aq[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) aq[kk] = frag_row<D>(cQ, qb * 32, lo.row[kk]);
      f32x16 s = f32x16{};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) s = mfma32(aq[kk], xf[kk], s);
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const f32x4 L4 = *reinterpret_cast<const f32x4 *>(&bL[qb * 32 + 8 * rg + 4 * hh]);
#pragma unroll
        for (int j = 0; j < 4; ++j) s[rg * 4 + j] = fmaf(s[rg * 4 + j], scale_log2, -L4[j]);
      }
      if (masked) {  // uniform branch: only the exponents change
        // the lane's query rows qc + 4 hh in [qlo, qhi) are inside the unit
        // and not before its key
        const int qhi = vrows - 4 * hh;
        const int qlo = kvalid ? kr - r0 - 4 * hh : qhi;
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int qc0 = qb * 32 + 8 * rg;
          const i32x4 M4 = *reinterpret_cast<const i32x4 *>(&bM[qc0 + 4 * hh]);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int qc = qc0 + j;
            const bool vis = (qc >= qlo) & (qc < qhi) & (M4[j] < kexp4);
            s[rg * 4 + j] = vis ? s[rg * 4 + j] : -INFINITY;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = __builtin_amdgcn_exp2f(s[r]);
      bf16x8 pa[2];
      pa[0] = pack8(s, 0);
      pa[1] = pack8(s, 8);
      // P in the accumulator's lane order, read back by the dS wave of the same keys
      bf16x8 *pdst = reinterpret_cast<bf16x8 *>(bP) + ((qb * 4 + kg) * 2) * 64 + lane;
      pdst[0] = pa[0];
      pdst[64] = pa[1];
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        bf16x8 bo[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db)
          bo[db] = decltype(hi_tag)::value
                       ? frag_tr<D>(cD, qb * 32 + c2 * 16, trah[db], trbh[db], HIBIAS)
                       : frag_tr<D>(cD, qb * 32 + c2 * 16, lo.tra[db], lo.trb[db]);
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] = mfma32(pa[c2], bo[db], acc[db]);
      }
    }
  };
  // dS side: one unit, whose P was written in the previous step
  auto ds_side = [&](auto hi_tag, const unsigned short *__restrict__ bQ,
                     const unsigned short *__restrict__ bD,
                     const float *__restrict__ bE, const unsigned short *__restrict__ bP)
                     __attribute__((always_inline)) {
    const char *cQ = reinterpret_cast<const char *>(bQ);
    const char *cD = reinterpret_cast<const char *>(bD);
    f32x16 dpb[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      bf16x8 ad[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) ad[kk] = frag_row<D>(cD, qb * 32, lo.row[kk]);
      // dP - Delta: the chain starts from the rows' -Delta
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const f32x4 N4 = *reinterpret_cast<const f32x4 *>(&bE[qb * 32 + 8 * rg + 4 * hh]);
#pragma unroll
        for (int j = 0; j < 4; ++j) dpb[qb][rg * 4 + j] = N4[j];
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) dpb[qb] = mfma32(ad[kk], xf[kk], dpb[qb]);
    }
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      f32x16 dp = dpb[qb];
      const bf16x8 *psrc = reinterpret_cast<const bf16x8 *>(bP) + ((qb * 4 + kg) * 2) * 64 + lane;
      const bf16x8 p0 = psrc[0], p1 = psrc[64];
#pragma unroll
      for (int r = 0; r < 16; ++r) dp[r] *= (float)(r < 8 ? p0[r] : p1[r - 8]);
      bf16x8 dsa[2];
      dsa[0] = pack8(dp, 0);
      dsa[1] = pack8(dp, 8);
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        bf16x8 bq[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db)
          bq[db] = decltype(hi_tag)::value
                       ? frag_tr<D>(cQ, qb * 32 + c2 * 16, trah[db], trbh[db], HIBIAS)
                       : frag_tr<D>(cQ, qb * 32 + c2 * 16, lo.tra[db], lo.trb[db]);
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] = mfma32(dsa[c2], bq[db], acc[db]);
      }
    }
  };

  if (e0 < e1) {
    // Unit state as scalars: walking-order entry, half, query head, first row.
    int ce = e0, chalf = 0, chi = 0;
    int cr0 = (((int)((unsigned)kt_ord[ce] & 0x7fffffffu)) - tr.qbase) * TQ;
    int cpart = (int)((unsigned)kt_ord[ce] >> 31);
    issue(cr0, 0, sQ0, sD0, sL0, sE0, sM0);
    wait_all_and_sync();
    bool have_cur = true;  // the P side has a unit this step
    int pb = 0;            // P buffer of the P side's unit (the dS side uses the other)
    bool first = true;
    // The work of one step, with every LDS buffer it touches as a distinct
    // __restrict__ parameter: the direct loads into the next unit's buffers
    // (n*) are then known not to write what the P side (c*), the dS side
    // (p*) and the P exchange (wP, rP) access, so no LDS access waits for
    // them.
    auto body = [&](auto cur_hi, auto prev_hi, const bool more, const int nr0, const int nhi,
                    unsigned short *__restrict__ nQ,
                    unsigned short *__restrict__ nD, float *__restrict__ nL,
                    float *__restrict__ nE, int *__restrict__ nM,
                    const unsigned short *__restrict__ cQ, const unsigned short *__restrict__ cD,
                    const float *__restrict__ cL, const int *__restrict__ cM,
                    const unsigned short *__restrict__ pQ, const unsigned short *__restrict__ pD,
                    const float *__restrict__ pE, unsigned short *__restrict__ wP,
                    const unsigned short *__restrict__ rP) __attribute__((always_inline)) {
      if (more) issue(nr0, nhi, nQ, nD, nL, nE, nM);
      if (side == 0) {
        if (have_cur) {
          const int vrows = min(64, tr.len - cr0);
          p_side(cur_hi, cr0, vrows, (cpart | (vrows < 64)) != 0, cQ, cD, cL, cM, wP);
        }
      } else if (!first) {
        ds_side(prev_hi, pQ, pD, pE, rP);
      }
    };
    // One step on Q/dO buffer B (the P side's unit; the dS side's is the
    // previous buffer, the next unit's loads go to the following one), with
    // the buffers as compile-time indices: the direct loads in flight then
    // provably write other LDS than the step reads.
    auto step = [&](auto bc) __attribute__((always_inline)) -> bool {
      constexpr int B = decltype(bc)::value, NBUF = (B + 1) % NB, PBUF = (B + NB - 1) % NB;
      // next unit: other half of this tile, else next head, else next entry
      int ne = ce, nhalf = 0, nhi = chi, nr0 = 0, npart = cpart;
      bool more = false;
      if (have_cur) {
        const bool second = chalf == 0 && cr0 + 64 < tr.len;
        const bool head = !second && chi + 1 < grp;
        const bool entry = !second && !head && ce + 1 < e1;
        more = second || head || entry;
        if (second) {
          nhalf = 1;
          nr0 = cr0 + 64;
        } else if (head) {
          nr0 = cr0 - chalf * 64;
          nhi = chi + 1;
        } else if (entry) {
          ne = ce + 1;
          const unsigned x = (unsigned)kt_ord[ne];
          nr0 = ((int)(x & 0x7fffffffu) - tr.qbase) * TQ;
          npart = (int)(x >> 31);
          nhi = 0;
        }
      }
      unsigned short *const Q[NB] = {sQ0, sQ1, sQ2}, *const Dd[NB] = {sD0, sD1, sD2};
      float *const Lr[NB] = {sL0, sL1, sL2}, *const Er[NB] = {sE0, sE1, sE2};
      int *const Mr[NB] = {sM0, sM1, sM2};
      body(std::integral_constant<bool, HIGH2 && B == HIBUF>{},
           std::integral_constant<bool, HIGH2 && PBUF == HIBUF>{},
           more, nr0, nhi, Q[NBUF], Dd[NBUF], Lr[NBUF], Er[NBUF], Mr[NBUF], Q[B], Dd[B], Lr[B],
           Mr[B], Q[PBUF], Dd[PBUF], Er[PBUF], sP[pb], sP[pb ^ 1]);
      __syncthreads();
      if (!have_cur) return false;
      have_cur = more;
      ce = ne;
      chalf = nhalf;
      chi = nhi;
      cr0 = nr0;
      cpart = npart;
      pb ^= 1;
      first = false;
      return true;
    };
    for (;;) {
      if (!step(std::integral_constant<int, 0>{})) break;
      if (!step(std::integral_constant<int, 1>{})) break;
      if (!step(std::integral_constant<int, 2>{})) break;
    }
  }

  // stage through LDS (RP key rows per pass) for coalesced stores;
  // accumulator D[i = key][j = d]
  wait_all_and_sync();
  TO *st = reinterpret_cast<TO *>(sQ0);
  constexpr int CH = 16 / sizeof(TO);   // elements per 16-byte chunk
  constexpr int RP = 128 / sizeof(TO);  // key rows per pass (16 KB)
  const float mul = side == 0 ? 1.f : scale;
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    TO *dst = which == 0 ? dv : dk;
#pragma unroll
    for (int pass = 0; pass < TQ / RP; ++pass) {
      if (side == which && kg * 32 >= pass * RP && kg * 32 < (pass + 1) * RP) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int kl = kg * 32 + 8 * (r >> 2) + 4 * hh + (r & 3) - pass * RP;
            const float val = acc[db][r] * mul;
            const int dd = db * 32 + col;
            if constexpr (sizeof(TO) == 2)
              st[kl * D + dd] = f2bf_bits(val);
            else
              st[kl * D + dd] = val;
          }
      }
      __syncthreads();
      for (int c = threadIdx.x; c < RP * D / CH; c += 512) {
        const int kl = c / (D / CH), ch = c % (D / CH);
        const int key = pass * RP + kl;
        if (key < tr.nrows) {
          const long row = tr.start + tr.row0 + key;
          *reinterpret_cast<u16x8 *>(dst + (row * hkv + hk) * D + ch * CH) =
              *reinterpret_cast<const u16x8 *>(st + kl * D + ch * CH);
        }
      }
      __syncthreads();
    }
  }
}

// dQ: one block = one q-tile x one query head, 4 waves of 32 query rows;
// units are 64-key halves of the listed k-tiles.  Recomputes S^T and dP^T per
// unit; dQ^T += K^T dS^T with K^T by transpose reads.  With FUSE (bf16
// inputs) the kernel also forms each of its rows' -Delta = -(dO . O) and
// log2-sum-exp from O and the natural-log LSE, uses them, and writes them for
// the dK/dV kernel that runs after it (no separate pre-pass); without FUSE it
// reads what the pre-pass wrote.
template <int D, class TO, bool FUSE>
__global__ void __launch_bounds__(256, 2) k_attn_bwd_dq(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const unsigned short *__restrict__ dout,
    const unsigned short *__restrict__ o, const float *__restrict__ lse,
    float *__restrict__ lse2, float *__restrict__ delta,
    const int32_t *__restrict__ seg_info, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ tok_meta, const int32_t *__restrict__ qt_ptr,
    const int32_t *__restrict__ qt_ord, const XcdRanges xr, int hq, int hkv, int W,
    float scale_log2, float scale, long P, TO *__restrict__ dq) {
  constexpr int KK = D / 16, DB = D / 32, T64 = 64 * D;
  __shared__ __attribute__((aligned(16))) unsigned short sK0[T64], sK1[T64], sV0[T64], sV1[T64];
  __shared__ __attribute__((aligned(16))) int sM0[64], sM1[64];

  int g, h;
  if (!xcd_block(xr, hq, hq / hkv, true, g, h)) return;
  const int hk = h / (hq / hkv);
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int qloc = wave * 32 + col;
  const bool qvalid = qloc < tr.nrows;
  const int qr = tr.row0 + (qvalid ? qloc : 0);
  const long qrow_abs = tr.start + qr;
  const int qstep = tok_meta[qrow_abs] >> 2;

  bf16x8 qf[KK], df[KK];
  {
    const unsigned short *qp = q + (qrow_abs * hq + h) * D;
    const unsigned short *dp = dout + (qrow_abs * hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = lds8(qp + kk * 16 + hh * 8);
      df[kk] = lds8(dp + kk * 16 + hh * 8);
    }
  }
  float l2, ndlt;  // log2-sum-exp and -Delta of the lane's query
  const long rv = (long)h * P + qrow_abs;
  if constexpr (FUSE) {
    // the lane holds half of the row's d (the other half in lane + 32):
    // bf16 products are exact in fp32, summed in a fixed order
    const unsigned short *op = o + (qrow_abs * hq + h) * D;
    float acc = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8 of = lds8(op + kk * 16 + hh * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{df[kk][2 * i], df[kk][2 * i + 1]},
                                              bf16x2{of[2 * i], of[2 * i + 1]}, acc, false);
    }
    acc += __shfl_xor(acc, 32, 64);
    ndlt = -acc;
    l2 = lse[rv] * LOG2E;
    if (qvalid && hh == 0) {
      delta[rv] = ndlt;
      lse2[rv] = l2;
    }
  } else {
    l2 = lse2[rv];
    ndlt = delta[rv];
  }
  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dqacc[db] = f32x16{};

  LaneOffsets<D> lo;
  lo.init(lane, 0);
  const long kv_stride = (long)hkv * D;
  const int row_bytes = (int)(kv_stride * 2);
  BufFill<D, 4> fp;
  fp.init(wave, lane, row_bytes);
  // the segment's rows of this kv head; rows past the segment read as zeros
  const __amdgpu_buffer_rsrc_t rK =
      make_rsrc(k + (long)hk * D + (long)tr.start * kv_stride, (unsigned)tr.len * row_bytes);
  const __amdgpu_buffer_rsrc_t rV =
      make_rsrc(v + (long)hk * D + (long)tr.start * kv_stride, (unsigned)tr.len * row_bytes);
  const __amdgpu_buffer_rsrc_t rM = make_rsrc(tok_meta + tr.start, (unsigned)tr.len * 4);

  // the wave index as a scalar: the direct loads' LDS addresses are then
  // formed in scalar registers (no readfirstlane per load)
  const int swave = __builtin_amdgcn_readfirstlane(wave);
  auto issue = [&](const Unit &u, unsigned short *__restrict__ nK, unsigned short *__restrict__ nV,
                   int *__restrict__ nM) __attribute__((always_inline)) {
    fp.issue(nK, rK, u.r0 * row_bytes, swave);
    fp.issue(nV, rV, u.r0 * row_bytes, swave);
    if (swave == 0) buf64_dw(nM, rM, lane, u.r0 * 4);
  };
  auto compute = [&](const Unit &u, const char *__restrict__ sK, const char *__restrict__ sV,
                     const int *__restrict__ sM) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb * 32 >= u.vrows) break;
      bf16x8 ak[KK], av[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        ak[kk] = frag_row<D>(sK, kb * 32, lo.row[kk]);
        av[kk] = frag_row<D>(sV, kb * 32, lo.row[kk]);
      }
      // dP^T - Delta: the chain starts from -Delta (one value per lane's query)
      f32x16 s = f32x16{}, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) dp[r] = ndlt;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        s = mfma32(ak[kk], qf[kk], s);
        dp = mfma32(av[kk], df[kk], dp);
      }
      // dS^T = P^T (dP^T - Delta); a masked pair gets exponent -inf (P = 0).
      // One uniform branch; inside, the predicate is bitwise (no branch per
      // element).
      if (__builtin_expect(u.partial, 0)) {
        // the lane's keys kc + 4 hh < lim are inside the unit and not after
        // its query
        const int lim = (qvalid ? min(u.vrows, qr - u.r0 + 1) : 0) - 4 * hh;
        const unsigned wfloor = window_floor(qstep, W);
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int kc0 = kb * 32 + 8 * rg;
          const i32x4 M4 = *reinterpret_cast<const i32x4 *>(sM + kc0 + 4 * hh);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int r = rg * 4 + j;
            const bool vis = (kc0 + j < lim) & (window_word(M4[j]) >= wfloor);
            const float x = vis ? fmaf(s[r], scale_log2, -l2) : -INFINITY;
            s[r] = __builtin_amdgcn_exp2f(x) * dp[r];
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -l2)) * dp[r];
      }
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        bf16x8 kt[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db)
          kt[db] = frag_tr<D>(sK, kb * 32 + c2 * 16, lo.tra[db], lo.trb[db]);
        const bf16x8 dsb = pack8(s, c2 * 8);
#pragma unroll
        for (int db = 0; db < DB; ++db) dqacc[db] = mfma32(kt[db], dsb, dqacc[db]);
      }
    }
  };
  auto step = [&](const Unit &u, const bool more, const Unit &nu,
                  const unsigned short *__restrict__ cK, const unsigned short *__restrict__ cV,
                  const int *__restrict__ cM, unsigned short *__restrict__ nK,
                  unsigned short *__restrict__ nV, int *__restrict__ nM)
                  __attribute__((always_inline)) {
    if (more) issue(nu, nK, nV, nM);
    compute(u, reinterpret_cast<const char *>(cK), reinterpret_cast<const char *>(cV), cM);
  };

  const int e0 = qt_ptr[g], e1 = qt_ptr[g + 1];
  auto next = [&](const Unit &u, Unit &n) __attribute__((always_inline)) -> bool {
    return next_unit(u, e1, qt_ord, tr.qbase, tr.len, n);
  };
  walk_units(make_unit(qt_ord, e0, 0, tr.qbase, tr.len), step, issue, next, sK0, sV0, sM0,
             sK1, sV1, sM1);

  if (qvalid) {
    TO *qrowp = dq + (qrow_abs * hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d0 = db * 32 + 8 * r4 + 4 * hh;
#pragma unroll
        for (int j = 0; j < 4; ++j) store_val(qrowp, d0 + j, dqacc[db][r4 * 4 + j] * scale);
      }
  }
}

// ------------------------------------------------------------- host side

struct AttnWs {
  size_t kn2, delta, lse2, qb, kb, vb, dob, total;
};

AttnWs attn_ws(const seg_sizes &sz, seg_dtype dt, int hq, int hkv, int d, int bwd) {
  AttnWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t P = (size_t)std::max<int64_t>(1, sz.packed_tokens);
  if (!bwd) w.kn2 = take((size_t)std::max(1, sz.num_segments) * hkv * sizeof(float));
  if (bwd) {
    w.delta = take(P * hq * sizeof(float));
    w.lse2 = take(P * hq * sizeof(float));
  }
  if (dt == SEG_F32) {
    w.qb = take(P * hq * d * 2);
    w.kb = take(P * hkv * d * 2);
    w.vb = take(P * hkv * d * 2);
    if (bwd) w.dob = take(P * hq * d * 2);
  }
  w.total = std::max<size_t>(off, 256);
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
  // the launch schedule: eight ranges covering every tile once
  for (const int32_t *b : {L->xcd_rows, L->xcd_cols}) {
    bool ok = b[0] == 0 && b[8] == sz->num_qtiles;
    for (int x = 0; x < 8; ++x) ok = ok && b[x] <= b[x + 1];
    SEG_CHECK(ok, SEG_ERR_ARG, "layout schedule ranges not set (build the layout first)");
  }
  SEG_CHECK((long)sz->packed_tokens * hq * d < (1L << 40), SEG_ERR_CAPACITY, "tensor too large");
  // tile loads address a segment's rows, and the per-row values of a head
  // group, with 32-bit byte offsets from one buffer resource
  SEG_CHECK((long)sz->max_seg_len * hq * d * 2 <= INT32_MAX, SEG_ERR_CAPACITY,
            "a segment of %d rows exceeds the 2 GiB addressable per tile stream", sz->max_seg_len);
  SEG_CHECK((long)sz->packed_tokens * hq * 4 <= INT32_MAX, SEG_ERR_CAPACITY,
            "%lld packed rows x %d heads of fp32 row values exceed 2 GiB",
            (long long)sz->packed_tokens, hq);
}

void to_bf16(const void *x, unsigned short *y, long n, hipStream_t st) {
  int grid = (int)std::min<long>(65536, (n + 255) / 256);
  ProfScope prof("attn_prep", st);
  k_f32_to_bf16<<<std::max(1, grid), 256, 0, st>>>(static_cast<const float *>(x), y, n);
  SEG_LAUNCH_CHECK();
}

template <int D, class TO>
void fwd_impl(const seg_layout *L, const seg_sizes *sz, int hq, int hkv, float scale,
              const unsigned short *q, const unsigned short *k, const unsigned short *v, void *o,
              float *lse, unsigned *kn2, hipStream_t st) {
  const int G = sz->num_qtiles;
  ProfScope prof("attn_fwd", st);
  fill32(kn2, (long)sz->num_segments * hkv, 0u, st);
  k_key_norm<D><<<dim3(G, hkv), 256, 0, st>>>(k, L->seg_info, L->tile_seg, hkv, kn2);
  SEG_LAUNCH_CHECK();
  const XcdRanges xr = xcd_ranges(L->xcd_rows);
  k_attn_fwd<D, TO><<<xcd_grid(xr, hq), 256, 0, st>>>(
      q, k, v, L->seg_info, L->tile_seg, L->tok_meta, L->qt_ptr, L->qt_ord,
      reinterpret_cast<const float *>(kn2), xr, hq, hkv, L->window, scale * LOG2E,
      sz->packed_tokens, static_cast<TO *>(o), lse);
  SEG_LAUNCH_CHECK();
}

template <int D, class TO, class TI>
void bwd_impl(const seg_layout *L, const seg_sizes *sz, int hq, int hkv, float scale,
              const unsigned short *q, const unsigned short *k, const unsigned short *v,
              const unsigned short *dout, const TI *o_raw, const TI *dout_raw,
              const float *lse, float *delta, float *lse2, void *dq, void *dk, void *dv,
              hipStream_t st) {
  const int G = sz->num_qtiles;
  const long P = sz->packed_tokens;
  // bf16 inputs: the dQ kernel forms -Delta and the log2-sum-exp of its rows
  // and runs first; fp32 inputs: the pre-pass forms them from the unrounded
  // O and dO
  constexpr bool FUSE = sizeof(TI) == 2;
  if constexpr (!FUSE) {
    const long threads = P * hq * (D / 8);
    ProfScope prof("attn_delta", st);
    k_delta<TI, D><<<(int)((threads + 255) / 256), 256, 0, st>>>(o_raw, dout_raw, lse, hq, P, delta,
                                                                 lse2);
    SEG_LAUNCH_CHECK();
  }
  {
    ProfScope prof("attn_bwd_dq", st);
    const XcdRanges xr = xcd_ranges(L->xcd_rows);
    k_attn_bwd_dq<D, TO, FUSE><<<xcd_grid(xr, hq), 256, 0, st>>>(
        q, k, v, dout, reinterpret_cast<const unsigned short *>(o_raw), lse, lse2, delta,
        L->seg_info, L->tile_seg, L->tok_meta, L->qt_ptr, L->qt_ord, xr, hq, hkv, L->window,
        scale * LOG2E, scale, P, static_cast<TO *>(dq));
    SEG_LAUNCH_CHECK();
  }
  {
    ProfScope prof("attn_bwd_dkdv", st);
    const XcdRanges xc = xcd_ranges(L->xcd_cols);
    k_attn_bwd_dkdv<D, TO><<<xcd_grid(xc, hkv), 512, 0, st>>>(
        q, k, v, dout, lse2, delta, L->seg_info, L->tile_seg, L->tok_meta, L->kt_ptr, L->kt_ord,
        xc, hq, hkv, L->window, scale * LOG2E, scale, P,
        static_cast<TO *>(dk), static_cast<TO *>(dv));
    SEG_LAUNCH_CHECK();
  }
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
    const long P = sz->packed_tokens;
    unsigned *kn2 = reinterpret_cast<unsigned *>(base + w.kn2);
    const unsigned short *qb, *kb, *vb;
    if (dt == SEG_F32) {
      unsigned short *q2 = reinterpret_cast<unsigned short *>(base + w.qb);
      unsigned short *k2 = reinterpret_cast<unsigned short *>(base + w.kb);
      unsigned short *v2 = reinterpret_cast<unsigned short *>(base + w.vb);
      to_bf16(q, q2, P * hq * d, stream);
      to_bf16(k, k2, P * hkv * d, stream);
      to_bf16(v, v2, P * hkv * d, stream);
      qb = q2;
      kb = k2;
      vb = v2;
    } else {
      qb = static_cast<const unsigned short *>(q);
      kb = static_cast<const unsigned short *>(k);
      vb = static_cast<const unsigned short *>(v);
    }
    if (d == 128) {
      if (dt == SEG_F32) fwd_impl<128, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, kn2, stream);
      else fwd_impl<128, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, kn2, stream);
    } else {
      if (dt == SEG_F32) fwd_impl<64, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, kn2, stream);
      else fwd_impl<64, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, kn2, stream);
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
    float *delta = reinterpret_cast<float *>(base + w.delta);
    float *lse2 = reinterpret_cast<float *>(base + w.lse2);
    if (dt == SEG_F32) {
      unsigned short *q2 = reinterpret_cast<unsigned short *>(base + w.qb);
      unsigned short *k2 = reinterpret_cast<unsigned short *>(base + w.kb);
      unsigned short *v2 = reinterpret_cast<unsigned short *>(base + w.vb);
      unsigned short *do2 = reinterpret_cast<unsigned short *>(base + w.dob);
      to_bf16(q, q2, P * hq * d, stream);
      to_bf16(k, k2, P * hkv * d, stream);
      to_bf16(v, v2, P * hkv * d, stream);
      to_bf16(d_o, do2, P * hq * d, stream);
      const float *o32 = static_cast<const float *>(o), *do32 = static_cast<const float *>(d_o);
      if (d == 128)
        bwd_impl<128, float, float>(L, sz, hq, hkv, softmax_scale, q2, k2, v2, do2, o32, do32,
                                    lse, delta, lse2, dq, dk, dv, stream);
      else
        bwd_impl<64, float, float>(L, sz, hq, hkv, softmax_scale, q2, k2, v2, do2, o32, do32, lse,
                                   delta, lse2, dq, dk, dv, stream);
    } else {
      const unsigned short *qb = static_cast<const unsigned short *>(q);
      const unsigned short *kb = static_cast<const unsigned short *>(k);
      const unsigned short *vb = static_cast<const unsigned short *>(v);
      const unsigned short *dob = static_cast<const unsigned short *>(d_o);
      const unsigned short *o16 = static_cast<const unsigned short *>(o);
      if (d == 128)
        bwd_impl<128, unsigned short, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb,
                                                      dob, o16, dob, lse, delta, lse2, dq, dk,
                                                      dv, stream);
      else
        bwd_impl<64, unsigned short, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb,
                                                     dob, o16, dob, lse, delta, lse2, dq, dk,
                                                     dv, stream);
    }
  });
}

// Workspace of seg_attn_bwd_noalloc: one copy of this array per GPU, held
// until the process ends.  Host code never uses the name itself (on the host
// it is a stand-in, not a device address): the device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[SEG_ATTN_BWD_SCRATCH_BYTES];

namespace seg {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device.
void *scratch_on_current_device() {
  int dev = -1;
  SEG_HIP(hipGetDevice(&dev));
  SEG_CHECK(dev >= 0 && dev < kMaxDevices, SEG_ERR_UNSUPPORTED, "device %d above %d", dev,
            kMaxDevices - 1);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    SEG_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    SEG_CHECK(ptr != nullptr, SEG_ERR_HIP, "no device address for the scratch array");
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace seg

extern "C" seg_status seg_attn_bwd_noalloc(const seg_layout *L, const seg_sizes *sz, seg_dtype dt,
                                           int32_t hq, int32_t hkv, int32_t d,
                                           float softmax_scale, const void *q, const void *k,
                                           const void *v, const void *o, const float *lse,
                                           const void *d_o, void *dq, void *dk, void *dv,
                                           hipStream_t stream) {
  void *ptr = nullptr;
  const seg_status st = guarded([&] {
    check_common(L, sz, dt, hq, hkv, d);
    const size_t need = attn_ws(*sz, dt, hq, hkv, d, 1).total;
    SEG_CHECK(need <= SEG_ATTN_BWD_SCRATCH_BYTES, SEG_ERR_WORKSPACE,
              "the backward needs %zu bytes of workspace, above the %zu-byte fixed scratch of "
              "seg_attn_bwd_noalloc (use seg_attn_bwd with a workspace)",
              need, (size_t)SEG_ATTN_BWD_SCRATCH_BYTES);
    if (sz->num_qtiles == 0) return;
    ptr = scratch_on_current_device();
  });
  if (st != SEG_OK) return st;
  return seg_attn_bwd(L, sz, dt, hq, hkv, d, softmax_scale, q, k, v, o, lse, d_o, dq, dk, dv, ptr,
                      SEG_ATTN_BWD_SCRATCH_BYTES, stream);
}
