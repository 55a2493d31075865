// Shared "NT" GEMMs of the libseg translation units (gfx950, bf16 MFMA):
//   C[m][n] = sum_k A[m][k] * B[n][k]     (both operands k-contiguous)
// Two block shapes with one epilogue interface (a functor called by every
// thread with its accumulators and a Tile that says where they sit):
//  - k_gemm_nt: 128x128 blocks, 4 waves of 64x64, K in steps of 32, the next
//    step staged in registers; two blocks per CU.  For grids too small to
//    fill the chip with 256-wide tiles.
//  - k_gemm_big: 256x256 blocks, 8 waves of 128x64 (two per SIMD), K in
//    steps of 64 fetched by direct buffer->LDS loads into two 64 KB stages;
//    XCD-aware grouped tile order.
//  - k_gemm_big_tn: the same block with transposed operands (both row-major
//    over K), fragments by transpose reads; up to three problems per launch.
#pragma once

#include "common.h"

namespace seg {
namespace gemm {

constexpr int BM = 128, BN = 128, BK = 32;

// Where a wave's accumulators sit: rows m0 + wr + bm*32 + 8*(r/4) + 4*hh + r%4,
// columns n0 + wc + bn*32 + col for register r of acc[bm][bn]; (wr, wc) is the
// wave tile's corner inside the block, brows the block's row count.
struct Tile {
  int m0, n0, M, N, wr, wc, col, hh, brows;
  __device__ __forceinline__ int row(int bm, int r) const {
    return m0 + wr + bm * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
  }
  __device__ __forceinline__ int column(int bn) const { return n0 + wc + bn * 32 + col; }
};

// Raw buffer resource over [base, base + bytes): loads at or past the end
// return zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t gemm_rsrc(const void *base, long bytes) {
  const long lim = bytes < 0x7fffffffL ? bytes : 0x7fffffffL;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)lim, 0x00020000);
}

// Calls f(m, n, v) for every accumulator of the wave inside [0, M) x [0, N)
// (plain global stores: with two waves per SIMD they measured faster than
// stores through a buffer resource).
template <int TM, int TN, class F>
__device__ __forceinline__ void tile_apply(const f32x16 (&acc)[TM][TN], const Tile &t, F &&f) {
#pragma unroll
  for (int bm = 0; bm < TM; ++bm)
#pragma unroll
    for (int bn = 0; bn < TN; ++bn) {
      const int n = t.column(bn);
      if (n >= t.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = t.row(bm, r);
        if (m < t.M) f(m, n, acc[bm][bn][r]);
      }
    }
}

// C = scale * A B^T stored as TO (leading dimension ldc)
template <class TO>
struct EpiStore {
  TO *c;
  long ldc;
  float scale;
  template <int TM, int TN>
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[TM][TN], const Tile &t) const {
    TO *cc = c;
    const long ld = ldc;
    const float s = scale;
    tile_apply(acc, t, [&](int m, int n, float v) { store_val(cc, (long)m * ld + n, v * s); });
  }
};

// C = R + scale * A B^T in bf16 (a residual connection); R may alias C
struct EpiResid {
  unsigned short *c;
  long ldc;
  const unsigned short *r;
  long ldr;
  float scale;
  template <int TM, int TN>
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[TM][TN], const Tile &t) const {
    unsigned short *cc = c;
    const unsigned short *rr = r;
    const long ld = ldc, lr = ldr;
    const float s = scale;
    tile_apply(acc, t, [&](int m, int n, float v) {
      cc[(long)m * ld + n] = f2bf_bits(bf_bits2f(rr[(long)m * lr + n]) + v * s);
    });
  }
};

// C += scale * A B^T in fp32 (gradients summed over row chunks, in chunk order)
struct EpiAccum {
  float *c;
  long ldc;
  float scale;
  template <int TM, int TN>
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[TM][TN], const Tile &t) const {
    float *cc = c;
    const long ld = ldc;
    const float s = scale;
    tile_apply(acc, t, [&](int m, int n, float v) { cc[(long)m * ld + n] += v * s; });
  }
};

// lda, ldb and K must be multiples of 8 (16-byte chunks); rows beyond M / N
// and chunks beyond K read as zero.  Grid: (ceil(N/BN), ceil(M/BM)).
template <class Epi>
__global__ void __launch_bounds__(256, 2) k_gemm_nt(const unsigned short *__restrict__ A, long lda,
                                                    const unsigned short *__restrict__ B, long ldb,
                                                    int M, int N, int K, Epi ep) {
  __shared__ unsigned short sA[2][BM * BK];
  __shared__ unsigned short sB[2][BN * BK];
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1, col = lane & 31, hh = lane >> 5;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  // each thread stages two 16-byte chunks of A and of B per K step
  u16x8 ra[2], rb[2];
  auto fetch = [&](int kt) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int c = tid + it * 256;
      const int row = c >> 2, ch = c & 3;
      const int gk = kt * BK + ch * 8;
      ra[it] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
      rb[it] = ra[it];
      if (m0 + row < M && gk < K) ra[it] = *reinterpret_cast<const u16x8 *>(A + (long)(m0 + row) * lda + gk);
      if (n0 + row < N && gk < K) rb[it] = *reinterpret_cast<const u16x8 *>(B + (long)(n0 + row) * ldb + gk);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int c = tid + it * 256;
      const int row = c >> 2, ch = c & 3;
      const int sw = (ch ^ ((row >> 2) & 3)) * 8;
      *reinterpret_cast<u16x8 *>(&sA[buf][row * BK + sw]) = ra[it];
      *reinterpret_cast<u16x8 *>(&sB[buf][row * BK + sw]) = rb[it];
    }
  };

  const int nk = (K + BK - 1) / BK;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) fetch(kt + 1);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int ch = kk * 2 + hh;
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int ra_ = wm * 64 + i * 32 + col;
        const int rb_ = wn * 64 + i * 32 + col;
        a[i] = *reinterpret_cast<const bf16x8 *>(&sA[buf][ra_ * BK + ((ch ^ ((ra_ >> 2) & 3)) * 8)]);
        b[i] = *reinterpret_cast<const bf16x8 *>(&sB[buf][rb_ * BK + ((ch ^ ((rb_ >> 2) & 3)) * 8)]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
    if (more) stash(buf ^ 1);
    __syncthreads();
  }
  ep(acc, Tile{m0, n0, M, N, wm * 64, wn * 64, col, hh, BM});
}

inline dim3 grid(int M, int N) { return dim3((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM)); }

// ---------------------------------------------------------------- 256x256

constexpr int BIG = 256, BKB = 64;
constexpr int BIG_STAGE = 2 * BIG * BKB;  // bf16 elements of one stage (A then B): 64 KB


// LDS layout of a 256 x 64 operand tile: row-major, 128 B per row, 16-byte
// chunk c of row r stored in slot c ^ ((r >> 1) & 7).  Sixteen consecutive
// rows then hit sixteen distinct 16-byte slots of the 64 banks (row parity
// picks the half of the 256-byte bank line), so a fragment read of 32 rows x
// 16 bytes is conflict-free.  A direct load writes 64 lanes x 16 bytes
// = 8 rows in slot order; each lane fetches the chunk that belongs there.
// The 8 waves of a block issue 4 such loads per operand and K step.
struct BigFill {
  int voff[4];   // byte offset of the lane's chunk in each of its 4 row groups
  int kchunk;    // the lane's logical k chunk (0..7)
  __device__ __forceinline__ void init(int wave, int lane, long ld) {
    const int rr = lane >> 3, slot = lane & 7;
    // row group j*8 + wave starts at a multiple of 8 rows; (row >> 1) & 7
    // depends only on the wave's parity and rr
    kchunk = slot ^ ((((wave & 1) * 8 + rr) >> 1) & 7);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = (j * 8 + wave) * 8 + rr;
      voff[j] = (int)(row * ld * 2) + kchunk * 16;
    }
  }
  // loads the 64-column K step starting at k0 (chunks at or past K read
  // zero; so does a whole step past the end); wave is wave-uniform
  __device__ __forceinline__ void issue(unsigned short *__restrict__ tile,
                                        __amdgpu_buffer_rsrc_t rs, int k0, int K, int wave) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const int add = k0 + kchunk * 8 < K ? k0 * 2 : 0x40000000;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void *)(tile + (j * 8 + wave) * 8 * BKB), 16,
          voff[j] + add, 0, 0, 0);
#endif
  }
};

// Tile order: a 1-D grid of 8 * ceil(T / 8) blocks for T tiles.  Block b runs
// on XCD b % 8; XCD x takes the contiguous tile range [x*C, (x+1)*C) so its
// concurrent blocks share an L2, and tiles are ordered in groups of 8 M-tiles
// (column by column inside a group) so those blocks reuse A and B rows.
__device__ __forceinline__ int big_index(int total) {
  const int per = (total + 7) / 8;
  return (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
}

__device__ __forceinline__ void big_tile_of(int idx, int nM, int nN, int &mt, int &nt) {
  const int G = 8;
  const int group = idx / (G * nN);
  const int first = group * G;
  const int gs = nM - first < G ? nM - first : G;
  const int in = idx - group * G * nN;
  mt = first + in % gs;
  nt = in / gs;
}

__device__ __forceinline__ bool big_tile(int nM, int nN, int &mt, int &nt) {
  const int idx = big_index(nM * nN);
  if (idx >= nM * nN) return false;
  big_tile_of(idx, nM, nN, mt, nt);
  return true;
}

inline unsigned big_blocks(int M, int N) {
  const long t = (long)((M + BIG - 1) / BIG) * ((N + BIG - 1) / BIG);
  return (unsigned)((t + 7) / 8 * 8);
}

// Both 256x256 kernels: a wave tile of 128 rows x 64 columns (8 waves, 2 x 4,
// two per SIMD): per slice 4 A and 2 B fragments feed 8 products.
struct NtFrags {
  bf16x8 a[4], b[2];
};

__device__ __forceinline__ void nt_load(NtFrags &f, const char *pa, const char *pb, int sw) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f.a[i] = *reinterpret_cast<const bf16x8 *>(pa + i * 32 * 128 + sw);
#pragma unroll
  for (int i = 0; i < 2; ++i) f.b[i] = *reinterpret_cast<const bf16x8 *>(pb + i * 32 * 128 + sw);
}

__device__ __forceinline__ void nt_mma(f32x16 (&acc)[4][2], const NtFrags &f) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(f.a[i], f.b[j], acc[i][j]);
}

// Scheduling of one slice: the six fragment reads of the next slice ride
// with the first six of its eight products, so their LDS latency hides under
// the MFMA pipe; the first slice of a step also carries the eight direct
// loads of the next step.
__device__ __forceinline__ void nt_interleave(bool with_loads) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (i < 6) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    if (with_loads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global load
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
  }
}

// First three slices of a K step: issue the next step's direct loads (past
// the end of K they read zeros into the idle buffer), then multiply slices
// 0-2 of the current stage while reading slices 1-3.  f0 holds slice 0 on
// entry; f1 holds slice 3 on exit.
__device__ __forceinline__ void nt_step(const unsigned short *__restrict__ rA,
                                        const unsigned short *__restrict__ rB,
                                        unsigned short *__restrict__ wA,
                                        unsigned short *__restrict__ wB, const BigFill &fa,
                                        const BigFill &fb, __amdgpu_buffer_rsrc_t ra,
                                        __amdgpu_buffer_rsrc_t rb, int k_next, int K, int wave,
                                        int offA, int offB, const int (&sw)[4], NtFrags &f0,
                                        NtFrags &f1, f32x16 (&acc)[4][2]) {
  fa.issue(wA, ra, k_next, K, wave);
  fb.issue(wB, rb, k_next, K, wave);
  const char *pa = reinterpret_cast<const char *>(rA) + offA;
  const char *pb = reinterpret_cast<const char *>(rB) + offB;
  nt_load(f1, pa, pb, sw[1]);
  nt_mma(acc, f0);
  nt_interleave(true);
  nt_load(f0, pa, pb, sw[2]);
  nt_mma(acc, f1);
  nt_interleave(false);
  nt_load(f1, pa, pb, sw[3]);
  nt_mma(acc, f0);
  nt_interleave(false);
}

// lda, ldb and K must be multiples of 8 and 256 * ld * 2 < 2^30; rows beyond
// M / N and chunks beyond K read as zero.  Grid: big_blocks(M, N) x BIG_THREADS.
constexpr int BIG_THREADS = 512;

template <class Epi>
__global__ void __launch_bounds__(BIG_THREADS, 1) k_gemm_big(const unsigned short *__restrict__ A,
                                                             long lda,
                                                             const unsigned short *__restrict__ B,
                                                             long ldb, int M, int N, int K, Epi ep) {
  __shared__ __attribute__((aligned(1024))) unsigned short lds[2 * BIG_STAGE];
  const int nM = (M + BIG - 1) / BIG, nN = (N + BIG - 1) / BIG;
  int mt, nt;
  if (!big_tile(nM, nN, mt, nt)) return;
  const int m0 = mt * BIG, n0 = nt * BIG;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3, col = lane & 31, hh = lane >> 5;

  // each resource covers only the block's own rows (< 2^30 bytes), so the
  // offset of a chunk past K (+2^30) is out of range and reads zero
  const __amdgpu_buffer_rsrc_t ra =
      gemm_rsrc(A + (long)m0 * lda, (long)(M - m0 < BIG ? M - m0 : BIG) * lda * 2);
  const __amdgpu_buffer_rsrc_t rb =
      gemm_rsrc(B + (long)n0 * ldb, (long)(N - n0 < BIG ? N - n0 : BIG) * ldb * 2);
  BigFill fa, fb;
  fa.init(wave, lane, lda);
  fb.init(wave, lane, ldb);

  // fragment reads: row (wave corner + i*32 + col), logical chunk 2*kk + hh
  const int sx = (col >> 1) & 7;
  int sw[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) sw[kk] = ((2 * kk + hh) ^ sx) * 16;
  const int offA = (wm * 128 + col) * 128, offB = (wn * 64 + col) * 128;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  unsigned short *s0 = lds, *s1 = lds + BIG_STAGE;
  const int nk = (K + BKB - 1) / BKB;
  fa.issue(s0, ra, 0, K, wave);
  fb.issue(s0 + BIG * BKB, rb, 0, K, wave);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  NtFrags f0, f1;
  nt_load(f0, reinterpret_cast<const char *>(s0) + offA,
          reinterpret_cast<const char *>(s0 + BIG * BKB) + offB, sw[0]);
  for (int kt = 0; kt < nk; ++kt) {
    unsigned short *cur = (kt & 1) ? s1 : s0;
    unsigned short *nxt = (kt & 1) ? s0 : s1;
    nt_step(cur, cur + BIG * BKB, nxt, nxt + BIG * BKB, fa, fb, ra, rb, (kt + 1) * BKB, K, wave,
            offA, offB, sw, f0, f1, acc);
    // every wave is done reading this stage and the next one has landed; the
    // last slice's products then cover the reads of the next stage's first
    // slice (after the last step they read the zero-filled idle buffer)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    nt_load(f0, reinterpret_cast<const char *>(nxt) + offA,
            reinterpret_cast<const char *>(nxt + BIG * BKB) + offB, sw[0]);
    nt_mma(acc, f1);
    nt_interleave(false);
  }
  ep(acc, Tile{m0, n0, M, N, wm * 128, wn * 64, col, hh, BIG});
}

// ------------------------------------------------- 256x256, transposed operands
// C[m][n] = sum_k At[k][m] * Bt[k][n] with At [K][lda], Bt [K][ldb] row-major
// (the weight gradients W^T-style: both operands run along the rows of a
// chunk); lda and ldb are multiples of 8 with lda >= M and ldb >= N.  Tiles hold 64 k-rows x 256 columns (512 B per row); 16-byte chunk
// c of row r sits in slot c ^ 4*(r & 3), so a 32-lane transpose read (4 rows x
// 64 bytes) hits 16 distinct slots of the 64 banks.  Fragments come from
// ds_read_b64_tr_b16 pairs: lane l gets column (l % 32) of rows
// {4h..4h+3, 8+4h..8+4h+3} (h = l / 32) of the slice; A and B use the same
// row order, so every product pairs equal k.

typedef short gemm_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) gemm_v4i16 gemm_lds_v4i16;

struct BigFillT {
  int voff[4];  // byte offset of the lane's chunk in each of its 4 row pairs
  __device__ __forceinline__ void init(int wave, int lane, long ld) {
    const int rr = lane >> 5, p = lane & 31;
    // op j of a wave covers rows 2*(8j + wave) + {0, 1}; row & 3 = (2*wave + rr) & 3
    const int c = p ^ (4 * ((2 * wave + rr) & 3));
#pragma unroll
    for (int j = 0; j < 4; ++j) voff[j] = (int)((2 * (j * 8 + wave) + rr) * ld * 2) + c * 16;
  }
  // rs covers the step's rows (from k0) of the block's columns
  __device__ __forceinline__ void issue(unsigned short *__restrict__ tile,
                                        __amdgpu_buffer_rsrc_t rs, int wave) const {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void *)(tile + (j * 8 + wave) * 2 * BIG), 16,
          voff[j], 0, 0, 0);
#endif
  }
};

// resource over rows [k0, min(K, k0 + 64)) of columns [c0, C) of a [K][ld]
// matrix (zero rows past K).  The last row stops at column C rounded up to
// a 16-byte chunk, so the range never ends inside a chunk or a dword whose
// first element is in range; ld is a multiple of 8 and every row holds ld
// elements, so the rounded end stays inside the matrix.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tn_rsrc(const unsigned short *X, long ld, int k0,
                                                         int K, int c0, int C) {
  const int rows = K - k0 < BKB ? K - k0 : BKB;
  const long bytes = rows > 0 ? ((long)(rows - 1) * ld + ((C - c0 + 7) & ~7)) * 2 : 0;
  return gemm_rsrc(X + (long)k0 * ld + c0, bytes);
}

__device__ __forceinline__ bf16x8 tr_frag(const char *p) {
  const gemm_v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((gemm_lds_v4i16 *)p);
  const gemm_v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((gemm_lds_v4i16 *)(p + 8 * 512));
  const bf16x4 a4 = __builtin_bit_cast(bf16x4, a), b4 = __builtin_bit_cast(bf16x4, b);
  bf16x8 r;
  r[0] = a4[0]; r[1] = a4[1]; r[2] = a4[2]; r[3] = a4[3];
  r[4] = b4[0]; r[5] = b4[1]; r[6] = b4[2]; r[7] = b4[3];
  return r;
}

// slice kk of the stage: rows 16*kk.. ; oa/ob: per-lane byte offsets of the
// four 32-column blocks (row part included)
__device__ __forceinline__ void big_load_tn(NtFrags &f, const char *pa, const char *pb,
                                            const int (&oa)[4], const int (&ob)[2], int kk) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f.a[i] = tr_frag(pa + kk * 16 * 512 + oa[i]);
#pragma unroll
  for (int i = 0; i < 2; ++i) f.b[i] = tr_frag(pb + kk * 16 * 512 + ob[i]);
}

// the twelve transpose reads of the next slice ride with its eight products
__device__ __forceinline__ void big_interleave_tn(bool with_loads) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (i < 4) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // two LDS reads
    else __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);       // one LDS read
    if (with_loads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global load
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // one MFMA
  }
}

__device__ __forceinline__ void big_step_tn(const unsigned short *__restrict__ rA,
                                            const unsigned short *__restrict__ rB,
                                            unsigned short *__restrict__ wA,
                                            unsigned short *__restrict__ wB, const BigFillT &fa,
                                            const BigFillT &fb, __amdgpu_buffer_rsrc_t ra,
                                            __amdgpu_buffer_rsrc_t rb, int wave, const int (&oa)[4],
                                            const int (&ob)[2], NtFrags &f0, NtFrags &f1,
                                            f32x16 (&acc)[4][2]) {
  fa.issue(wA, ra, wave);
  fb.issue(wB, rb, wave);
  const char *pa = reinterpret_cast<const char *>(rA);
  const char *pb = reinterpret_cast<const char *>(rB);
  big_load_tn(f1, pa, pb, oa, ob, 1);
  nt_mma(acc, f0);
  big_interleave_tn(true);
  big_load_tn(f0, pa, pb, oa, ob, 2);
  nt_mma(acc, f1);
  big_interleave_tn(false);
  big_load_tn(f1, pa, pb, oa, ob, 3);
  nt_mma(acc, f0);
  big_interleave_tn(false);
}

// Up to three transposed-operand problems over the same K rows, run by one
// launch (their tiles in sequence), so a short last wave of one problem is
// filled by the next.  Each: C_p[M_p][N_p] (+)= At_p^T Bt_p.
template <class Epi, int NP>
struct TnGroup {
  const unsigned short *At[NP], *Bt[NP];
  long lda[NP], ldb[NP];
  int M[NP], N[NP];
  Epi ep[NP];
  int start[NP + 1];  // first tile of each problem; start[NP] = all tiles
};

// lda, ldb multiples of 8, 64 * ld * 2 < 2^30; K >= 0 rows (rows past K read
// as zero); columns past M / N are computed from whatever the rows hold there
// and dropped by the epilogue.  Grid: 8 * ceil(tiles / 8) x 256.
template <class Epi, int NP>
__global__ void __launch_bounds__(512, 1) k_gemm_big_tn(const TnGroup<Epi, NP> g, int K) {
  __shared__ __attribute__((aligned(1024))) unsigned short lds[2 * BIG_STAGE];
  const int idx = big_index(g.start[NP]);
  if (idx >= g.start[NP]) return;
  // the problem's fields by unrolled selects (no dynamic indexing of the
  // kernel argument, which would copy it to scratch)
  const unsigned short *At = g.At[0], *Bt = g.Bt[0];
  long lda = g.lda[0], ldb = g.ldb[0];
  int M = g.M[0], N = g.N[0], first = 0;
  Epi ep = g.ep[0];
#pragma unroll
  for (int q = 1; q < NP; ++q)
    if (idx >= g.start[q]) {
      At = g.At[q];
      Bt = g.Bt[q];
      lda = g.lda[q];
      ldb = g.ldb[q];
      M = g.M[q];
      N = g.N[q];
      first = g.start[q];
      ep = g.ep[q];
    }
  int mt, nt;
  big_tile_of(idx - first, (M + BIG - 1) / BIG, (N + BIG - 1) / BIG, mt, nt);
  const int m0 = mt * BIG, n0 = nt * BIG;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2, wn = wave & 3, col = lane & 31, hh = lane >> 5;

  BigFillT fa, fb;
  fa.init(wave, lane, lda);
  fb.init(wave, lane, ldb);
  // transpose-read offsets: row 4*hh + (lane%16)/4 of the slice, column
  // (wave corner) + 32*i + 16*((lane/16)%2) + 4*(lane%4)
  const int l16 = lane & 15, r = 4 * hh + (l16 >> 2), sx = 4 * (r & 3);
  int oa[4], ob[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ca = wm * 128 + 32 * i + 16 * ((lane >> 4) & 1) + 4 * (l16 & 3);
    oa[i] = r * 512 + (((ca >> 3) ^ sx) << 4) + (ca & 7) * 2;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int cb = wn * 64 + 32 * i + 16 * ((lane >> 4) & 1) + 4 * (l16 & 3);
    ob[i] = r * 512 + (((cb >> 3) ^ sx) << 4) + (cb & 7) * 2;
  }

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  unsigned short *s0 = lds, *s1 = lds + BIG_STAGE;
  const int nk = (K + BKB - 1) / BKB;
  fa.issue(s0, tn_rsrc(At, lda, 0, K, m0, M), wave);
  fb.issue(s0 + BIG * BKB, tn_rsrc(Bt, ldb, 0, K, n0, N), wave);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  NtFrags f0, f1;
  big_load_tn(f0, reinterpret_cast<const char *>(s0), reinterpret_cast<const char *>(s0 + BIG * BKB),
              oa, ob, 0);
  for (int kt = 0; kt < nk; ++kt) {
    unsigned short *cur = (kt & 1) ? s1 : s0;
    unsigned short *nxt = (kt & 1) ? s0 : s1;
    const int k1 = (kt + 1) * BKB;
    big_step_tn(cur, cur + BIG * BKB, nxt, nxt + BIG * BKB, fa, fb, tn_rsrc(At, lda, k1, K, m0, M),
                tn_rsrc(Bt, ldb, k1, K, n0, N), wave, oa, ob, f0, f1, acc);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    big_load_tn(f0, reinterpret_cast<const char *>(nxt),
                reinterpret_cast<const char *>(nxt + BIG * BKB), oa, ob, 0);
    nt_mma(acc, f1);
    big_interleave_tn(false);
  }
  ep(acc, Tile{m0, n0, M, N, wm * 128, wn * 64, col, hh, BIG});
}

inline int big_tiles(int M, int N) {
  return M <= 0 || N <= 0 ? 0 : ((M + BIG - 1) / BIG) * ((N + BIG - 1) / BIG);
}

template <class Epi, int NP>
inline void gemm_launch_tn(TnGroup<Epi, NP> g, int K, hipStream_t st) {
  g.start[0] = 0;
  for (int q = 0; q < NP; ++q) g.start[q + 1] = g.start[q] + big_tiles(g.M[q], g.N[q]);
  if (g.start[NP] == 0) return;
  k_gemm_big_tn<Epi, NP><<<(unsigned)((g.start[NP] + 7) / 8 * 8), 512, 0, st>>>(g, K);
}

template <class Epi>
inline void gemm_launch_tn(const unsigned short *At, long lda, const unsigned short *Bt, long ldb,
                           int M, int N, int K, const Epi &ep, hipStream_t st) {
  TnGroup<Epi, 1> g{};
  g.At[0] = At;
  g.Bt[0] = Bt;
  g.lda[0] = lda;
  g.ldb[0] = ldb;
  g.M[0] = M;
  g.N[0] = N;
  g.ep[0] = ep;
  gemm_launch_tn(g, K, st);
}

// Block shape for a problem: the 256-wide tiles unless they would leave more
// than a quarter of the CUs idle in the first wave.
inline bool gemm_use_big(int M, int N) {
  return (long)((M + BIG - 1) / BIG) * ((N + BIG - 1) / BIG) >= 192;
}

template <class Epi>
inline void gemm_launch(const unsigned short *A, long lda, const unsigned short *B, long ldb, int M,
                        int N, int K, const Epi &ep, hipStream_t st) {
  if (M <= 0 || N <= 0) return;
  if (gemm_use_big(M, N))
    k_gemm_big<Epi><<<big_blocks(M, N), BIG_THREADS, 0, st>>>(A, lda, B, ldb, M, N, K, ep);
  else
    k_gemm_nt<Epi><<<grid(M, N), 256, 0, st>>>(A, lda, B, ldb, M, N, K, ep);
}

// y[c][r] = x[r][c] for a [rows][cols] matrix (ldx), output [cols][ldy]; x is
// bf16 bits or fp32 (rounded); optional row gather; zero for r >= rows up to
// pad_rows.
template <class TI>
__global__ void __launch_bounds__(256) k_transpose2d(const TI *__restrict__ x, long ldx,
                                                     const int32_t *__restrict__ rowmap, int rows,
                                                     int cols, int pad_rows,
                                                     unsigned short *__restrict__ y, long ldy) {
  __shared__ unsigned short t[64][66];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    unsigned short b = 0;
    if (r < rows && c < cols) {
      const long sr = rowmap ? rowmap[r] : r;
      b = load_bf(x, sr * ldx + c);
    }
    t[i][tx] = b;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < pad_rows) y[(long)c * ldy + r] = t[tx][i];
  }
}

inline dim3 grid64(long cols, long rows) {
  return dim3((unsigned)((cols + 63) / 64), (unsigned)((rows + 63) / 64));
}

}  // namespace gemm
}  // namespace seg
