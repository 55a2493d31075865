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
#include <type_traits>
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

// fp32 -> bf16 copy (row-major, any shape)
__global__ void k_f32_to_bf16(const float *__restrict__ x, unsigned short *__restrict__ y, long n) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    y[i] = f2bf_bits(x[i]);
}

// Delta[h][row] = sum_d dO[row][h][d] * O[row][h][d]  (D/8 lanes per (row, head)),
// and the row's log-sum-exp in log2 units for the backward kernels.
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
    delta[(long)h * P + row] = acc;
    lse2[(long)h * P + row] = lse[(long)h * P + row] * LOG2E;
  }
}

// ------------------------------------------------------------- pipelined kernels
//
// Tiles of 64 rows x d (row-major, bf16) are double-buffered in LDS: the
// loads of the next unit are in flight while the current one is computed.
// The forward and dQ kernels fill with direct 16-byte global->LDS loads; the
// dK/dV kernel, which has registers to spare, stages the next unit in
// registers (see the note on wait counts below).  Rows are stored with a
// 16-byte-chunk swizzle that keeps both 16-byte row reads (MFMA operands
// contracting over d; 16 lanes per LDS cycle) and 4x16 transpose reads
// (ds_read_b64_tr_b16: operands contracting over the rows; 32 lanes per
// cycle) free of bank conflicts on 64 four-byte banks, so no transposed copy
// of any tensor is needed.  Every lane's swizzled offsets are computed once;
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
template <int D>
__device__ __forceinline__ bf16x8 frag_tr(const char *tile, int R, int offa, int offb) {
  const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)(tile + R * D * 2 + offa));
  const v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)(tile + R * D * 2 + offb));
  const bf16x4 a4 = __builtin_bit_cast(bf16x4, a), b4 = __builtin_bit_cast(bf16x4, b);
  bf16x8 r;
  r[0] = a4[0]; r[1] = a4[1]; r[2] = a4[2]; r[3] = a4[3];
  r[4] = b4[0]; r[5] = b4[1]; r[6] = b4[2]; r[7] = b4[3];
  return r;
}

// Lane coordinates of a 64-row tile fill by NW waves (PW direct 16-byte
// global->LDS loads per lane; each wave instruction fills 1 KB of LDS,
// lane-contiguous).  The swizzle is applied by choosing which global chunk
// each lane loads.
template <int D, int NW>
struct FillPlan {
  static constexpr int CPR = D / 8, PW = 64 * CPR / (64 * NW);
  static_assert(PW >= 1, "tile too small for the wave count");
  int row[PW], chunk[PW];  // tile row and element offset of the lane's 16 bytes
  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int s = (wave * PW + i) * 64 + lane;
      row[i] = s / CPR;
      chunk[i] = ((s % CPR) ^ swz<D>(row[i])) * 8;
    }
  }
  // rows r0 + min(row, vrows - 1) of `base` (stride elements per row)
  __device__ __forceinline__ void issue(unsigned short *tile, const unsigned short *base, long stride,
                                        int r0, int vrows, int wave) const {
    // device pass only: the host pass of clang drops the launch stub of a
    // kernel that reaches this address-space cast
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const long r = r0 + min(row[i], vrows - 1);
      __builtin_amdgcn_global_load_lds(
          base + r * stride + chunk[i],
          (__attribute__((address_space(3))) void *)(tile + (wave * PW + i) * 64 * 8), 16, 0, 0);
    }
#endif
  }
};

// Register-staged fill of the same lane coordinates: `load` issues the global
// loads into registers, `store` writes them to LDS.
template <int D, int NW>
struct StagePlan {
  static constexpr int CPR = D / 8, PW = 64 * CPR / (64 * NW);
  int row[PW], chunk[PW];
  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int s = (wave * PW + i) * 64 + lane;
      row[i] = s / CPR;
      chunk[i] = ((s % CPR) ^ swz<D>(row[i])) * 8;
    }
  }
  __device__ __forceinline__ void load(u16x8 (&st)[PW], const unsigned short *base, long stride,
                                       int r0, int vrows) const {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const long r = r0 + min(row[i], vrows - 1);
      st[i] = *reinterpret_cast<const u16x8 *>(base + r * stride + chunk[i]);
    }
  }
  __device__ __forceinline__ void store(unsigned short *tile, const u16x8 (&st)[PW], int wave,
                                        int lane) const {
#pragma unroll
    for (int i = 0; i < PW; ++i)
      *reinterpret_cast<u16x8 *>(tile + ((wave * PW + i) * 64 + lane) * 8) = st[i];
  }
};

// one dword per lane into 64 consecutive dwords of LDS (direct load)
__device__ __forceinline__ void fill64_dw(void *dst, const void *src_lane) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(src_lane, (__attribute__((address_space(3))) void *)dst, 4, 0, 0);
#endif
}

// Software pipelining over units.  The loads of unit n+1 are issued, then
// unit n is computed from the other buffer, then a barrier ends the step.
// With direct loads, both happen inside one always-inline step whose LDS
// buffers are distinct __restrict__ parameters: a direct load's LDS write is
// counted with the global loads, and without the no-alias facts the compiler
// would wait for the loads in flight before the first LDS read of the
// compute.  Every LDS access of a step goes through those parameters.  While
// a direct load is in flight the compiler also gives up counted LDS waits
// (every wait becomes lgkmcnt(0)), which serialises read-ahead; the dK/dV
// kernel therefore stages its next unit in registers instead.

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
// contiguous tile range [x*C, (x+1)*C), C = ceil(ntiles / 8), and runs the nh
// heads of one tile back to back: heads of a tile read the same key/value
// tiles, and neighbouring tiles of a segment read mostly the same ones, so
// they meet in one L2.  Each range holds several whole segments, which keeps
// the XCDs balanced.  `reverse` walks the range from its end (the longest
// rows of each segment first).  The grid is 8*C*nh blocks; blocks past the
// last tile exit at once.
__device__ __forceinline__ bool xcd_block(int nh, int ntiles, bool reverse, int &tile, int &head) {
  const int b = blockIdx.x, x = b & 7, i = b >> 3;
  const int C = (ntiles + 7) >> 3;
  const int t = i / nh;
  head = i - t * nh;
  tile = x * C + (reverse ? C - 1 - t : t);
  return tile < ntiles;
}

__host__ __device__ inline int xcd_grid(int ntiles, int nh) { return (ntiles + 7) / 8 * 8 * nh; }

// A unit of work: 64 rows (half of a 128-row tile) of the tile listed at CSR
// entry e.
struct Unit {
  int e, half;
  int r0;       // segment-relative first row of the unit
  int vrows;    // valid rows (1..64)
  int partial;  // PARTIAL tile (an int: a struct without padding bytes is
                // copied field by field, never through private memory)
};

// Unit (e, half) read straight from the CSR arrays (the tile index is a
// uniform load through the scalar cache, which measured faster than staging
// the entries in LDS).
__device__ __forceinline__ Unit make_unit(const int32_t *col_idx, const uint8_t *cls, int e,
                                          int half, int qbase, int seg_len) {
  Unit u;
  u.e = e;
  u.half = half;
  const int t0 = (col_idx[e] - qbase) * TQ;
  u.r0 = t0 + half * 64;
  u.vrows = min(64, seg_len - u.r0);
  u.partial = cls[e] == SEG_TILE_PARTIAL;
  return u;
}

// next unit: the second half of the same tile when it has rows, else the next entry
__device__ __forceinline__ bool next_unit(const Unit &u, int e1, const int32_t *col_idx,
                                          const uint8_t *cls, int qbase, int seg_len, Unit &nu) {
  if (u.half == 0 && u.r0 + 64 < seg_len) {
    nu = make_unit(col_idx, cls, u.e, 1, qbase, seg_len);
    return true;
  }
  if (u.e + 1 < e1) {
    nu = make_unit(col_idx, cls, u.e + 1, 0, qbase, seg_len);
    return true;
  }
  return false;
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
    const int32_t *__restrict__ qt_ptr, const int32_t *__restrict__ qt_col,
    const uint8_t *__restrict__ qt_cls, const int32_t *__restrict__ work_order, int ntiles, int hq,
    int hkv, int W, float scale_log2, long P, TO *__restrict__ o, float *__restrict__ lse) {
  constexpr int KK = D / 16, DB = D / 32, T64 = 64 * D;
  __shared__ __attribute__((aligned(16))) unsigned short sK0[T64], sK1[T64], sV0[T64], sV1[T64];
  __shared__ __attribute__((aligned(16))) int sM0[64], sM1[64];

  int g, h;
  if (!xcd_block(hq, ntiles, true, g, h)) return;
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
  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  LaneOffsets<D> lo;
  lo.init(lane, 0);
  FillPlan<D, 4> fp;
  fp.init(wave, lane);
  const long kv_stride = (long)hkv * D;
  const unsigned short *kbase = k + (long)hk * D + (long)tr.start * kv_stride;
  const unsigned short *vbase = v + (long)hk * D + (long)tr.start * kv_stride;

  auto issue = [&](const Unit &u, unsigned short *__restrict__ nK, unsigned short *__restrict__ nV,
                   int *__restrict__ nM) __attribute__((always_inline)) {
    fp.issue(nK, kbase, kv_stride, u.r0, u.vrows, wave);
    fp.issue(nV, vbase, kv_stride, u.r0, u.vrows, wave);
    if (wave == 0) fill64_dw(nM, tok_meta + tr.start + u.r0 + min(lane, u.vrows - 1));
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
    // raw scores; masked entries -inf (scale > 0 keeps the order)
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
      const float m_new = grow ? mloc : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
      m_run = m_new;
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
    rsum += __shfl_xor(rsum, 32, 64);
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
    return next_unit(u, e1, qt_col, qt_cls, tr.qbase, tr.len, n);
  };
  Unit u = make_unit(qt_col, qt_cls, e0, 0, tr.qbase, tr.len), nu;
  issue(u, sK0, sV0, sM0);
  wait_all_and_sync();
  for (;;) {
    bool more = next(u, nu);
    step(u, more, nu, sK0, sV0, sM0, sK1, sV1, sM1);
    __syncthreads();
    if (!more) break;
    u = nu;
    more = next(u, nu);
    step(u, more, nu, sK1, sV1, sM1, sK0, sV0, sM0);
    __syncthreads();
    if (!more) break;
    u = nu;
  }

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

// dK/dV, one wave per SIMD: one block = one k-tile x one kv head, 4 waves of
// 32 keys each.  A wave holds the K and V fragments of its keys and the dK
// and dV accumulators over the whole head dimension (about 300 registers, so
// one wave per SIMD).  Per unit (64 rows of one query head) and 32-row block:
//   S = Q K^T, dP = dO V^T (queries on accumulator rows),
//   P = exp2(S * scale - lse), dS = P (dP - Delta),
//   dV += P^T dO, dK += dS^T Q (dO^T, Q^T by transpose reads).
// P and dS never leave the wave: the only barrier of a unit is the swap of
// the double buffer, whose next unit is staged in registers.  Units are 64-row halves of the listed q-tiles, for
// every query head of the group.  No atomics.
template <int D, class TO>
__global__ void __launch_bounds__(256, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) k_attn_bwd_dkdv(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const unsigned short *__restrict__ dout,
    const float *__restrict__ lse2, const float *__restrict__ delta,
    const int32_t *__restrict__ seg_info, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ tok_meta, const int32_t *__restrict__ kt_ptr,
    const int32_t *__restrict__ kt_row, const uint8_t *__restrict__ kt_cls, int ntiles, int hq,
    int hkv, int W, float scale_log2, float scale, long P, TO *__restrict__ dk,
    TO *__restrict__ dv) {
  constexpr int KK = D / 16, T64 = 64 * D, DB = D / 32;
  __shared__ __attribute__((aligned(16))) unsigned short sQ0[T64], sQ1[T64], sD0[T64], sD1[T64];
  __shared__ __attribute__((aligned(16))) float sL0[64], sL1[64], sE0[64], sE1[64];
  __shared__ __attribute__((aligned(16))) int sM0[64], sM1[64];

  // k-tiles in natural order: within a segment the earliest k-tiles have the
  // longest transposed-CSR columns, so they start first
  int g, hk;
  if (!xcd_block(hkv, ntiles, false, g, hk)) return;
  const int grp = hq / hkv;
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int kloc = wave * 32 + col;
  const bool kvalid = kloc < tr.nrows;
  const int kr = tr.row0 + (kvalid ? kloc : 0);
  const int kexp = key_expiry(tok_meta[tr.start + kr], W);

  bf16x8 kf[KK], vf[KK];
  {
    const long row = tr.start + kr;
    const unsigned short *ks = k + (row * hkv + hk) * D, *vs = v + (row * hkv + hk) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kf[kk] = lds8(ks + kk * 16 + hh * 8);
      vf[kk] = lds8(vs + kk * 16 + hh * 8);
    }
  }
  f32x16 dkacc[DB], dvacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dkacc[db] = f32x16{};
    dvacc[db] = f32x16{};
  }

  LaneOffsets<D> lo;
  lo.init(lane, 0);
  const long q_stride = (long)hq * D;
  const int e0 = kt_ptr[g], e1 = kt_ptr[g + 1];

  // register-staged prefetch of one unit: Q and dO rows, and one per-row
  // value by waves 0-2 (log2-sum-exp, Delta, turn)
  StagePlan<D, 4> sp;
  sp.init(wave, lane);
  u16x8 stq[StagePlan<D, 4>::PW], sto[StagePlan<D, 4>::PW];
  int stv = 0;
  auto load = [&](const Unit &u, int hi) __attribute__((always_inline)) {
    const int h = hk * grp + hi;
    sp.load(stq, q + (long)h * D + (long)tr.start * q_stride, q_stride, u.r0, u.vrows);
    sp.load(sto, dout + (long)h * D + (long)tr.start * q_stride, q_stride, u.r0, u.vrows);
    const long lrow = tr.start + u.r0 + min(lane, u.vrows - 1);
    if (wave == 0) stv = __builtin_bit_cast(int, lse2[(long)h * P + lrow]);
    else if (wave == 1) stv = __builtin_bit_cast(int, delta[(long)h * P + lrow]);
    else if (wave == 2) stv = tok_meta[lrow];
  };
  auto store = [&](unsigned short *__restrict__ nQ, unsigned short *__restrict__ nD,
                   float *__restrict__ nL, float *__restrict__ nE, int *__restrict__ nM)
                   __attribute__((always_inline)) {
    sp.store(nQ, stq, wave, lane);
    sp.store(nD, sto, wave, lane);
    if (wave == 0) nL[lane] = __builtin_bit_cast(float, stv);
    else if (wave == 1) nE[lane] = __builtin_bit_cast(float, stv);
    else if (wave == 2) nM[lane] = stv;
  };
  // S and dP of one 32-row block
  auto sdp = [&](const char *__restrict__ sQ, const char *__restrict__ sdO, const int qb,
                 f32x16 &s, f32x16 &dp) __attribute__((always_inline)) {
    bf16x8 aq[KK], ad[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      aq[kk] = frag_row<D>(sQ, qb * 32, lo.row[kk]);
      ad[kk] = frag_row<D>(sdO, qb * 32, lo.row[kk]);
    }
    s = f32x16{};
    dp = f32x16{};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      s = mfma32(aq[kk], kf[kk], s);
      dp = mfma32(ad[kk], vf[kk], dp);
    }
    // Scheduling groups (mask 0x100: LDS reads, 0x008: MFMA), in program
    // order for the whole unit: row reads run 4 ahead of the products.  The
    // compiler's own schedule issues each read right before its product.
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < 2 * KK - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };
  // P = exp2(S * scale - lse) (a masked pair gets exponent -inf, P = 0) and
  // dS = P (dP - Delta), packed to bf16
  auto pds = [&](const Unit &u, const bool masked, const float *__restrict__ sLse,
                 const float *__restrict__ sDel, const int *__restrict__ sMeta, const int qb,
                 f32x16 &s, f32x16 &dp, bf16x8 (&pa)[2], bf16x8 (&dsa)[2])
                 __attribute__((always_inline)) {
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      const int base = qb * 32 + 8 * rg + 4 * hh;
      const f32x4 L4 = *reinterpret_cast<const f32x4 *>(sLse + base);
      const f32x4 D4 = *reinterpret_cast<const f32x4 *>(sDel + base);
      i32x4 M4;
      if (masked) M4 = *reinterpret_cast<const i32x4 *>(sMeta + base);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = rg * 4 + j, ql = base + j;
        float x = fmaf(s[r], scale_log2, -L4[j]);
        if (masked) {
          const bool vis = kvalid & (ql < u.vrows) & (kr <= u.r0 + ql) & ((M4[j] >> 2) < kexp);
          x = vis ? x : -INFINITY;
        }
        s[r] = __builtin_amdgcn_exp2f(x);
        dp[r] = s[r] * (dp[r] - D4[j]);
      }
    }
    pa[0] = pack8(s, 0);
    pa[1] = pack8(s, 8);
    dsa[0] = pack8(dp, 0);
    dsa[1] = pack8(dp, 8);
    // this block's lse / Delta (/ turn) reads form their own group, so they
    // do not take the slots of the transpose reads below
    if (masked)
      __builtin_amdgcn_sched_group_barrier(0x100, 12, 0);
    else
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
  };
  // dV += P^T dO, dK += dS^T Q for one 32-row block
  auto dkv = [&](const char *__restrict__ sQ, const char *__restrict__ sdO, const int qb,
                 const bf16x8 (&pa)[2], const bf16x8 (&dsa)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      bf16x8 bo[DB], bq[DB];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        bo[db] = frag_tr<D>(sdO, qb * 32 + c2 * 16, lo.tra[db], lo.trb[db]);
        bq[db] = frag_tr<D>(sQ, qb * 32 + c2 * 16, lo.tra[db], lo.trb[db]);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        dvacc[db] = mfma32(pa[c2], bo[db], dvacc[db]);
        dkacc[db] = mfma32(dsa[c2], bq[db], dkacc[db]);
      }
    }
    // transpose reads run 4 fragments ahead of the products
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int i = 0; i < 4 * DB - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };
  // One unit over its two 32-row blocks, in the order S/dP(0), softmax(0),
  // S/dP(1), dV/dK(0), softmax(1), dV/dK(1) (measured best among the orders
  // tried; it also keeps the live state within the register budget).
  // FULL units with 64 query rows and every key of the tile valid need no
  // predicate (kvalid is false only in a segment's last k-tile, which is a
  // diagonal, PARTIAL tile); rows past vrows hold copies of the last row and
  // are masked.  `masked` is a constant in each inlined copy.
  auto compute = [&](const Unit &u, const bool masked, const char *__restrict__ sQ,
                     const char *__restrict__ sdO, const float *__restrict__ sLse,
                     const float *__restrict__ sDel, const int *__restrict__ sMeta)
                     __attribute__((always_inline)) {
    f32x16 s0, dp0, s1, dp1;
    bf16x8 pa0[2], ds0[2], pa1[2], ds1[2];
    sdp(sQ, sdO, 0, s0, dp0);
    pds(u, masked, sLse, sDel, sMeta, 0, s0, dp0, pa0, ds0);
    sdp(sQ, sdO, 1, s1, dp1);
    dkv(sQ, sdO, 0, pa0, ds0);
    pds(u, masked, sLse, sDel, sMeta, 1, s1, dp1, pa1, ds1);
    dkv(sQ, sdO, 1, pa1, ds1);
  };
  auto step = [&](const Unit &u, const bool more, const Unit &nu, int nhi,
                  const unsigned short *__restrict__ cQ, const unsigned short *__restrict__ cD,
                  const float *__restrict__ cL, const float *__restrict__ cE,
                  const int *__restrict__ cM, unsigned short *__restrict__ nQ,
                  unsigned short *__restrict__ nD, float *__restrict__ nL, float *__restrict__ nE,
                  int *__restrict__ nM) __attribute__((always_inline)) {
    if (more) load(nu, nhi);  // in flight during the products below
    const char *q8 = reinterpret_cast<const char *>(cQ), *d8 = reinterpret_cast<const char *>(cD);
    if (__builtin_expect(u.partial | (u.vrows < 64), 0))
      compute(u, true, q8, d8, cL, cE, cM);
    else
      compute(u, false, q8, d8, cL, cE, cM);
    if (more) store(nQ, nD, nL, nE, nM);
  };

  if (e0 < e1) {
    // Next unit: other half of this tile, else next head, else next entry.
    // Every field is computed from scalars: partial assignments of a
    // struct in different branches ended up in dynamically indexed private
    // memory, whose loads wait behind the prefetch loads.
    auto advance = [&](const Unit &cu, int chi, Unit &n, int &nh) __attribute__((always_inline)) -> bool {
      const bool second = cu.half == 0 && cu.r0 + 64 < tr.len;
      const bool head = !second && chi + 1 < grp;
      const bool entry = !second && !head && cu.e + 1 < e1;
      if (!(second || head || entry)) return false;
      int e = cu.e, half = 0, r0, partial = cu.partial;
      if (second) {
        half = 1;
        r0 = cu.r0 + 64;
        nh = chi;
      } else if (head) {
        r0 = cu.r0 - cu.half * 64;
        nh = chi + 1;
      } else {
        e = cu.e + 1;
        r0 = (kt_row[e] - tr.qbase) * TQ;
        partial = kt_cls[e] == SEG_TILE_PARTIAL;
        nh = 0;
      }
      n.e = e;
      n.half = half;
      n.r0 = r0;
      n.vrows = min(64, tr.len - r0);
      n.partial = partial;
      return true;
    };
    Unit cur = make_unit(kt_row, kt_cls, e0, 0, tr.qbase, tr.len), nx;
    int hcur = 0, hnx = 0;
    load(cur, hcur);
    store(sQ0, sD0, sL0, sE0, sM0);
    __syncthreads();
    for (;;) {
      bool more = advance(cur, hcur, nx, hnx);
      step(cur, more, nx, hnx, sQ0, sD0, sL0, sE0, sM0, sQ1, sD1, sL1, sE1, sM1);
      __syncthreads();
      if (!more) break;
      cur = nx;
      hcur = hnx;
      more = advance(cur, hcur, nx, hnx);
      step(cur, more, nx, hnx, sQ1, sD1, sL1, sE1, sM1, sQ0, sD0, sL0, sE0, sM0);
      __syncthreads();
      if (!more) break;
      cur = nx;
      hcur = hnx;
    }
  }

  // stage through LDS (RP key rows per pass) for coalesced stores;
  // accumulator D[i = key][j = d]
  wait_all_and_sync();
  TO *st = reinterpret_cast<TO *>(sQ0);
  constexpr int CH = 16 / sizeof(TO);   // elements per 16-byte chunk
  constexpr int RP = 128 / sizeof(TO);  // key rows per pass (16 KB)
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    TO *dst = which == 0 ? dk : dv;
#pragma unroll
    for (int pass = 0; pass < TQ / RP; ++pass) {
      if (wave * 32 >= pass * RP && wave * 32 < (pass + 1) * RP) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int kl = wave * 32 + 8 * (r >> 2) + 4 * hh + (r & 3) - pass * RP;
            const float val = which == 0 ? dkacc[db][r] * scale : dvacc[db][r];
            const int dd = db * 32 + col;
            if constexpr (sizeof(TO) == 2)
              st[kl * D + dd] = f2bf_bits(val);
            else
              st[kl * D + dd] = val;
          }
      }
      __syncthreads();
      for (int c = threadIdx.x; c < RP * D / CH; c += 256) {
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
// unit; dQ^T += K^T dS^T with K^T by transpose reads.
template <int D, class TO>
__global__ void __launch_bounds__(256, 2) k_attn_bwd_dq(
    const unsigned short *__restrict__ q, const unsigned short *__restrict__ k,
    const unsigned short *__restrict__ v, const unsigned short *__restrict__ dout,
    const float *__restrict__ lse2, const float *__restrict__ delta,
    const int32_t *__restrict__ seg_info, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ tok_meta, const int32_t *__restrict__ qt_ptr,
    const int32_t *__restrict__ qt_col, const uint8_t *__restrict__ qt_cls,
    const int32_t *__restrict__ work_order, int ntiles, int hq, int hkv, int W,
    float scale_log2, float scale, long P, TO *__restrict__ dq) {
  constexpr int KK = D / 16, DB = D / 32, T64 = 64 * D;
  __shared__ __attribute__((aligned(16))) unsigned short sK0[T64], sK1[T64], sV0[T64], sV1[T64];
  __shared__ __attribute__((aligned(16))) int sM0[64], sM1[64];

  int g, h;
  if (!xcd_block(hq, ntiles, true, g, h)) return;
  const int hk = h / (hq / hkv);
  const TileRows tr = tile_rows(seg_info, tile_seg, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, hh = lane >> 5;
  const int qloc = wave * 32 + col;
  const bool qvalid = qloc < tr.nrows;
  const int qr = tr.row0 + (qvalid ? qloc : 0);
  const long qrow_abs = tr.start + qr;
  const int qstep = tok_meta[qrow_abs] >> 2;
  const float l2 = lse2[(long)h * P + qrow_abs];
  const float dlt = delta[(long)h * P + qrow_abs];

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
  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dqacc[db] = f32x16{};

  LaneOffsets<D> lo;
  lo.init(lane, 0);
  FillPlan<D, 4> fp;
  fp.init(wave, lane);
  const long kv_stride = (long)hkv * D;
  const unsigned short *kbase = k + (long)hk * D + (long)tr.start * kv_stride;
  const unsigned short *vbase = v + (long)hk * D + (long)tr.start * kv_stride;

  auto issue = [&](const Unit &u, unsigned short *__restrict__ nK, unsigned short *__restrict__ nV,
                   int *__restrict__ nM) __attribute__((always_inline)) {
    fp.issue(nK, kbase, kv_stride, u.r0, u.vrows, wave);
    fp.issue(nV, vbase, kv_stride, u.r0, u.vrows, wave);
    if (wave == 0) fill64_dw(nM, tok_meta + tr.start + u.r0 + min(lane, u.vrows - 1));
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
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        s = mfma32(ak[kk], qf[kk], s);
        dp = mfma32(av[kk], df[kk], dp);
      }
      // dS^T = P^T (dP^T - Delta); a masked pair gets exponent -inf (P = 0).
      // One uniform branch; inside, the predicate is bitwise (no branch per
      // element).
      if (__builtin_expect(u.partial, 0)) {
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int kb0 = kb * 32 + 8 * rg + 4 * hh;
          const i32x4 M4 = *reinterpret_cast<const i32x4 *>(sM + kb0);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int r = rg * 4 + j, kl = kb0 + j;
            const bool vis = qvalid & (kl < u.vrows) & (u.r0 + kl <= qr) &
                             (qstep < key_expiry(M4[j], W));
            const float x = vis ? fmaf(s[r], scale_log2, -l2) : -INFINITY;
            s[r] = __builtin_amdgcn_exp2f(x) * (dp[r] - dlt);
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          s[r] = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -l2)) * (dp[r] - dlt);
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
    return next_unit(u, e1, qt_col, qt_cls, tr.qbase, tr.len, n);
  };
  Unit u = make_unit(qt_col, qt_cls, e0, 0, tr.qbase, tr.len), nu;
  issue(u, sK0, sV0, sM0);
  wait_all_and_sync();
  for (;;) {
    bool more = next(u, nu);
    step(u, more, nu, sK0, sV0, sM0, sK1, sV1, sM1);
    __syncthreads();
    if (!more) break;
    u = nu;
    more = next(u, nu);
    step(u, more, nu, sK1, sV1, sM1, sK0, sV0, sM0);
    __syncthreads();
    if (!more) break;
    u = nu;
  }

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
  size_t delta, lse2, qb, kb, vb, dob, total;
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
  SEG_CHECK((long)sz->packed_tokens * hq * d < (1L << 40), SEG_ERR_CAPACITY, "tensor too large");
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
              float *lse, hipStream_t st) {
  const int G = sz->num_qtiles;
  ProfScope prof("attn_fwd", st);
  k_attn_fwd<D, TO><<<xcd_grid(G, hq), 256, 0, st>>>(
      q, k, v, L->seg_info, L->tile_seg, L->tok_meta, L->qt_ptr, L->qt_col, L->qt_cls,
      L->work_order, G, hq, hkv, L->window, scale * LOG2E, sz->packed_tokens, static_cast<TO *>(o),
      lse);
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
  {
    const long threads = P * hq * (D / 8);
    ProfScope prof("attn_delta", st);
    k_delta<TI, D><<<(int)((threads + 255) / 256), 256, 0, st>>>(o_raw, dout_raw, lse, hq, P, delta,
                                                                 lse2);
    SEG_LAUNCH_CHECK();
  }
  {
    ProfScope prof("attn_bwd_dkdv", st);
    k_attn_bwd_dkdv<D, TO><<<xcd_grid(G, hkv), 256, 0, st>>>(
        q, k, v, dout, lse2, delta, L->seg_info, L->tile_seg, L->tok_meta, L->kt_ptr, L->kt_row,
        L->kt_cls, G, hq, hkv, L->window, scale * LOG2E, scale, P, static_cast<TO *>(dk),
        static_cast<TO *>(dv));
    SEG_LAUNCH_CHECK();
  }
  ProfScope prof("attn_bwd_dq", st);
  k_attn_bwd_dq<D, TO><<<xcd_grid(G, hq), 256, 0, st>>>(
      q, k, v, dout, lse2, delta, L->seg_info, L->tile_seg, L->tok_meta, L->qt_ptr, L->qt_col,
      L->qt_cls, L->work_order, G, hq, hkv, L->window, scale * LOG2E, scale, P,
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
    const long P = sz->packed_tokens;
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
      if (dt == SEG_F32) fwd_impl<128, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, stream);
      else fwd_impl<128, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, stream);
    } else {
      if (dt == SEG_F32) fwd_impl<64, float>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, stream);
      else fwd_impl<64, unsigned short>(L, sz, hq, hkv, softmax_scale, qb, kb, vb, o, lse, stream);
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
