// Shared "NT" GEMM of the libseg translation units (gfx950, bf16 MFMA):
//   C[m][n] = sum_k A[m][k] * B[n][k]     (both operands k-contiguous)
// 128x128 block tiles, 4 waves of 64x64, K in steps of 32.  The next K step
// is staged in registers (its global loads are in flight while the current
// step is multiplied) and written to the other LDS buffer afterwards.  The
// epilogue is a functor called by every thread with the accumulators.
#pragma once

#include "common.h"

namespace seg {
namespace gemm {

constexpr int BM = 128, BN = 128, BK = 32;

// Where a wave's accumulators sit: rows m0 + wm*64 + bm*32 + 8*(r/4) + 4*hh + r%4,
// columns n0 + wn*64 + bn*32 + col for register r of acc[bm][bn].
struct Tile {
  int m0, n0, M, N, wm, wn, col, hh;
  __device__ __forceinline__ int row(int bm, int r) const {
    return m0 + wm * 64 + bm * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
  }
  __device__ __forceinline__ int column(int bn) const { return n0 + wn * 64 + bn * 32 + col; }
};

// C = scale * A B^T stored as TO (leading dimension ldc)
template <class TO>
struct EpiStore {
  TO *c;
  long ldc;
  float scale;
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[2][2], const Tile &t) const {
#pragma unroll
    for (int bm = 0; bm < 2; ++bm)
#pragma unroll
      for (int bn = 0; bn < 2; ++bn) {
        const int n = t.column(bn);
        if (n >= t.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = t.row(bm, r);
          if (m < t.M) store_val(c, (long)m * ldc + n, acc[bm][bn][r] * scale);
        }
      }
  }
};

// C = R + scale * A B^T in bf16 (a residual connection); R may alias C
struct EpiResid {
  unsigned short *c;
  long ldc;
  const unsigned short *r;
  long ldr;
  float scale;
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[2][2], const Tile &t) const {
#pragma unroll
    for (int bm = 0; bm < 2; ++bm)
#pragma unroll
      for (int bn = 0; bn < 2; ++bn) {
        const int n = t.column(bn);
        if (n >= t.N) continue;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int m = t.row(bm, rr);
          if (m < t.M)
            c[(long)m * ldc + n] = f2bf_bits(bf_bits2f(r[(long)m * ldr + n]) + acc[bm][bn][rr] * scale);
        }
      }
  }
};

// C += scale * A B^T in fp32 (gradients summed over row chunks, in chunk order)
struct EpiAccum {
  float *c;
  long ldc;
  float scale;
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[2][2], const Tile &t) const {
#pragma unroll
    for (int bm = 0; bm < 2; ++bm)
#pragma unroll
      for (int bn = 0; bn < 2; ++bn) {
        const int n = t.column(bn);
        if (n >= t.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = t.row(bm, r);
          if (m < t.M) c[(long)m * ldc + n] += acc[bm][bn][r] * scale;
        }
      }
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
  ep(acc, Tile{m0, n0, M, N, wm, wn, col, hh});
}

inline dim3 grid(int M, int N) { return dim3((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM)); }

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
