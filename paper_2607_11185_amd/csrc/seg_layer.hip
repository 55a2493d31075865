// One decoder layer of the language model around the segmented attention
// (the policy-update model of Sec. 3.3 training items; the vision encoder is
// fixed during RL, App. E, so screenshot tokens enter as hidden states):
// pre-norm RMSNorm, q/k/v projections, rotary position embedding with the
// token's row inside its segment as position, the segmented attention of
// seg_attn.hip, output projection, RMSNorm and a SwiGLU MLP, with residual
// connections; forward and backward on gfx950.  Projections and the MLP run
// over row chunks with the shared GEMMs (gemm.h): data products with the NT
// kernel (weights transposed once per call), weight gradients with the
// transposed-operand kernel straight from the chunk's row-major activations.
// Weight gradients are summed chunk after chunk and the norm-weight gradients
// through fixed-order partial sums, so results are bitwise reproducible.
#include <cmath>

#include "common.h"
#include "gemm.h"

extern "C" seg_status seg_attn_fwd(const seg_layout *, const seg_sizes *, seg_dtype, int32_t,
                                   int32_t, int32_t, float, const void *, const void *,
                                   const void *, void *, float *, void *, size_t, hipStream_t);
extern "C" seg_status seg_attn_bwd(const seg_layout *, const seg_sizes *, seg_dtype, int32_t,
                                   int32_t, int32_t, float, const void *, const void *,
                                   const void *, const void *, const float *, const void *, void *,
                                   void *, void *, void *, size_t, hipStream_t);
extern "C" size_t seg_attn_workspace_bytes(const seg_sizes *, seg_dtype, int32_t, int32_t, int32_t,
                                           int32_t);

namespace seg {
namespace {

using gemm::EpiAccum;
using gemm::EpiResid;
using gemm::EpiStore;
using gemm::k_transpose2d;

constexpr int MAX_CH = 16;   // hidden <= 8 * 64 * MAX_CH
constexpr int RMS_ROWS = 32; // rows per block of the norm backward
constexpr int DEFAULT_CHUNK = 65536;     // rows per chunk when chunk_rows = 0
constexpr int MAX_CHUNK = 1 << 20;       // GEMM rows are addressed with 32-bit offsets

// ------------------------------------------------------------------ kernels

// pos[r] = row inside its segment, -1 for padding rows (segments sorted by start)
__global__ void k_positions(const int32_t *__restrict__ seg_info, int S, long P,
                            int32_t *__restrict__ pos) {
  for (long r = (long)blockIdx.x * blockDim.x + threadIdx.x; r < P; r += (long)gridDim.x * blockDim.x) {
    int lo = 0, hi = S - 1, s = -1;
    while (lo <= hi) {
      const int mid = (lo + hi) >> 1;
      if (seg_info[(long)mid * SEG_INFO_FIELDS + SEG_INFO_START] <= r) {
        s = mid;
        lo = mid + 1;
      } else {
        hi = mid - 1;
      }
    }
    int p = -1;
    if (s >= 0) {
      const long st = seg_info[(long)s * SEG_INFO_FIELDS + SEG_INFO_START];
      const long ln = seg_info[(long)s * SEG_INFO_FIELDS + SEG_INFO_LEN];
      if (r < st + ln) p = (int)(r - st);
    }
    pos[r] = p;
  }
}

// y = x / sqrt(mean(x^2) + eps) * g; one wave per row, fp32 arithmetic.
// Padding rows (pos < 0) give y = 0 and rstd = 0 whatever x holds there.
__global__ void __launch_bounds__(256) k_rms_fwd(const unsigned short *__restrict__ x, long ldx,
                                                 const unsigned short *__restrict__ g, float eps,
                                                 int rows, int H, const int32_t *__restrict__ pos,
                                                 unsigned short *__restrict__ y, long ldy,
                                                 float *__restrict__ rstd) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int nch = H / 8;
  if (pos[row] < 0) {
    if (lane == 0 && rstd) rstd[row] = 0.f;
    for (int c = lane; c < nch; c += 64)
      *reinterpret_cast<u16x8 *>(y + (long)row * ldy + c * 8) = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
    return;
  }
  const unsigned short *xr = x + (long)row * ldx;
  float ss = 0.f;
  for (int c = lane; c < nch; c += 64) {
    const u16x8 v = *reinterpret_cast<const u16x8 *>(xr + c * 8);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float f = bf_bits2f(v[j]);
      ss = fmaf(f, f, ss);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  const float r = 1.f / sqrtf(ss / (float)H + eps);
  if (lane == 0 && rstd) rstd[row] = r;
  unsigned short *yr = y + (long)row * ldy;
  for (int c = lane; c < nch; c += 64) {
    const u16x8 v = *reinterpret_cast<const u16x8 *>(xr + c * 8);
    const u16x8 gv = *reinterpret_cast<const u16x8 *>(g + c * 8);
    u16x8 o;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = f2bf_bits(bf_bits2f(v[j]) * r * bf_bits2f(gv[j]));
    *reinterpret_cast<u16x8 *>(yr + c * 8) = o;
  }
}

// Backward of y = x * r * g, r = (mean(x^2) + eps)^(-1/2), for dy (fp32):
//   out = resid + r g dy - r^3 x sum(g dy x) / H      (bf16; resid may alias out)
// and per-wave partial sums of dy x r for dg: part[(block*4 + wave)][H].
// Padding rows (pos < 0) pass resid through and add nothing to dg.
__global__ void __launch_bounds__(256) k_rms_bwd(const unsigned short *__restrict__ x, long ldx,
                                                 const unsigned short *__restrict__ g,
                                                 const float *__restrict__ rstd,
                                                 const float *__restrict__ dy, long lddy, int rows,
                                                 int H, const int32_t *__restrict__ pos,
                                                 const unsigned short *resid, long ldr,
                                                 unsigned short *out, long ldo,
                                                 float *__restrict__ part) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = H / 8;
  float dg[MAX_CH][8];
#pragma unroll
  for (int t = 0; t < MAX_CH; ++t)
#pragma unroll
    for (int j = 0; j < 8; ++j) dg[t][j] = 0.f;
  const int r_end = min(rows, (blockIdx.x + 1) * RMS_ROWS);
  for (int row = blockIdx.x * RMS_ROWS + wave; row < r_end; row += 4) {
    if (pos[row] < 0) {
      for (int c = lane; c < nch; c += 64)
        *reinterpret_cast<u16x8 *>(out + (long)row * ldo + c * 8) =
            *reinterpret_cast<const u16x8 *>(resid + (long)row * ldr + c * 8);
      continue;
    }
    const unsigned short *xr = x + (long)row * ldx;
    const float *dr = dy + (long)row * lddy;
    const float r = rstd[row];
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < MAX_CH; ++t) {
      const int c = lane + 64 * t;
      if (c < nch) {
        const u16x8 xv = *reinterpret_cast<const u16x8 *>(xr + c * 8);
        const u16x8 gv = *reinterpret_cast<const u16x8 *>(g + c * 8);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float xf = bf_bits2f(xv[j]), d = dr[c * 8 + j];
          s = fmaf(bf_bits2f(gv[j]) * d, xf, s);
          dg[t][j] = fmaf(d * xf, r, dg[t][j]);
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    const float k3 = r * r * r * s / (float)H;
    for (int c = lane; c < nch; c += 64) {
      const u16x8 xv = *reinterpret_cast<const u16x8 *>(xr + c * 8);
      const u16x8 gv = *reinterpret_cast<const u16x8 *>(g + c * 8);
      const u16x8 rv = *reinterpret_cast<const u16x8 *>(resid + (long)row * ldr + c * 8);
      u16x8 o;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = dr[c * 8 + j];
        const float dx = r * bf_bits2f(gv[j]) * d - k3 * bf_bits2f(xv[j]);
        o[j] = f2bf_bits(bf_bits2f(rv[j]) + dx);
      }
      *reinterpret_cast<u16x8 *>(out + (long)row * ldo + c * 8) = o;
    }
  }
  float *pr = part + ((long)blockIdx.x * 4 + wave) * H;
#pragma unroll
  for (int t = 0; t < MAX_CH; ++t) {
    const int c = lane + 64 * t;
    if (c < nch) {
#pragma unroll
      for (int j = 0; j < 8; ++j) pr[c * 8 + j] = dg[t][j];
    }
  }
}

// Column sums of part[nparts][H] in a fixed order, in two passes: block
// (x, y) sums parts [y*per, (y+1)*per) of 256 columns into part2[y][H], then
// out[h] += sum over y (in order) of part2[y][h].
constexpr int COLSUM_SPLIT = 16;

__global__ void __launch_bounds__(256) k_colsum_part(const float *__restrict__ part, int nparts,
                                                     int H, float *__restrict__ part2) {
  const int h = blockIdx.x * 256 + threadIdx.x;
  if (h >= H) return;
  const int per = (nparts + COLSUM_SPLIT - 1) / COLSUM_SPLIT;
  const int p0 = blockIdx.y * per, p1 = min(nparts, p0 + per);
  float s = 0.f;
#pragma unroll 8
  for (int p = p0; p < p1; ++p) s += part[(long)p * H + h];
  part2[(long)blockIdx.y * H + h] = s;
}

__global__ void k_colsum_add(const float *__restrict__ part2, int H, float *__restrict__ out) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= H) return;
  float s = 0.f;
#pragma unroll
  for (int y = 0; y < COLSUM_SPLIT; ++y) s += part2[(long)y * H + h];
  out[h] += s;
}

// Rotary embedding in place on x [P, heads, d] (row stride heads*d): the pair
// (x_i, x_{i+d/2}) turns by pos * base^(-2i/d) (by minus that angle with
// inverse, the transpose used by the backward).  The angle is formed and
// reduced modulo 2 pi in fp64; padding rows are left unchanged.
__global__ void __launch_bounds__(256) k_rope(unsigned short *__restrict__ x, long P, int heads,
                                              int d, const int32_t *__restrict__ pos,
                                              double log2_base, int inverse) {
  __shared__ double inv[64];
  const int half = d / 2;
  for (int i = threadIdx.x; i < half; i += blockDim.x) inv[i] = exp2(-2.0 * i / d * log2_base);
  __syncthreads();
  const long n = P * heads * half;
  const double two_pi = 6.283185307179586;
  for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
    const int i = (int)(e % half);
    const long rh = e / half;
    const long row = rh / heads;
    const int p = pos[row];
    if (p < 0) continue;
    double a = (double)p * inv[i];
    a -= two_pi * floor(a / two_pi);
    float s, c;
    sincosf((float)a, &s, &c);
    if (inverse) s = -s;
    unsigned short *xp = x + rh * d;
    const float x1 = bf_bits2f(xp[i]), x2 = bf_bits2f(xp[i + half]);
    xp[i] = f2bf_bits(x1 * c - x2 * s);
    xp[i + half] = f2bf_bits(x2 * c + x1 * s);
  }
}

__device__ __forceinline__ float sigmoidf_(float g) { return 1.f / (1.f + __expf(-g)); }

// Gate and up projections side by side: block j of 64 rows of wgu holds
// wg rows 32j..32j+31 then wu rows 32j..32j+31 (zero rows past I), so one
// GEMM against wgu gives, in each 64-column wave tile, the gate and up
// values of the same 32 features.  Grid-stride over 16-byte chunks.
constexpr int GU_BLOCK = 32;

__global__ void k_interleave_gu(const unsigned short *__restrict__ wg,
                                const unsigned short *__restrict__ wu, int I, int H, long rows2,
                                unsigned short *__restrict__ wgu) {
  const long h8 = H / 8, n = rows2 * h8;
  for (long c = (long)blockIdx.x * blockDim.x + threadIdx.x; c < n; c += (long)gridDim.x * blockDim.x) {
    const long R = c / h8, k = (c - R * h8) * 8;
    const long j = R / (2 * GU_BLOCK), w = R % (2 * GU_BLOCK);
    const long f = j * GU_BLOCK + (w % GU_BLOCK);
    u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
    if (f < I) v = *reinterpret_cast<const u16x8 *>((w < GU_BLOCK ? wg : wu) + f * H + k);
    *reinterpret_cast<u16x8 *>(wgu + R * H + k) = v;
  }
}

// Epilogue of the GEMM against wgu (the 256-wide NT kernel): m = silu(g) * u
// for the wave's 32 features, in fp32 from the accumulators (acc[.][0] holds
// the gate, acc[.][1] the up values of the same rows and features); with g
// and u set, also stores the gate and up values (the backward's recompute).
// Outputs are [rows][ld] bf16 at feature columns.
struct EpiSwiGLU {
  unsigned short *m, *g, *u;
  long ld;
  int I;
  template <int TM, int TN>
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[TM][TN],
                                             const gemm::Tile &t) const {
    static_assert(TN == 2, "SwiGLU epilogue expects 64-column wave tiles");
    const int f = (t.n0 + t.wc) / 2 + t.col;  // the lane's feature
    if (f >= I) return;
#pragma unroll
    for (int bm = 0; bm < TM; ++bm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = t.row(bm, r);
        if (row >= t.M) continue;
        const float gv = acc[bm][0][r], uv = acc[bm][1][r];
        const long off = (long)row * ld + f;
        m[off] = f2bf_bits(gv * sigmoidf_(gv) * uv);
        if (g) {
          g[off] = f2bf_bits(gv);
          u[off] = f2bf_bits(uv);
        }
      }
  }
};

// dg = dm * u * silu'(g), du = dm * silu(g), silu'(g) = s (1 + g (1 - s)),
// s = sigmoid(g) (8 elements per thread).  A streaming kernel: folded into the
// dm GEMM's epilogue its loads of g and u stall the one wave per SIMD.
__global__ void k_swiglu_bwd(const unsigned short *__restrict__ g, const unsigned short *__restrict__ u,
                             const unsigned short *__restrict__ dm, unsigned short *__restrict__ dg,
                             unsigned short *__restrict__ du, long n8) {
  for (long c = (long)blockIdx.x * blockDim.x + threadIdx.x; c < n8; c += (long)gridDim.x * blockDim.x) {
    const u16x8 gv = *reinterpret_cast<const u16x8 *>(g + c * 8);
    const u16x8 uv = *reinterpret_cast<const u16x8 *>(u + c * 8);
    const u16x8 mv = *reinterpret_cast<const u16x8 *>(dm + c * 8);
    u16x8 og, ou;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float gf = bf_bits2f(gv[j]), uf = bf_bits2f(uv[j]), d = bf_bits2f(mv[j]);
      const float s = sigmoidf_(gf);
      og[j] = f2bf_bits(d * uf * s * (1.f + gf * (1.f - s)));
      ou[j] = f2bf_bits(d * gf * s);
    }
    *reinterpret_cast<u16x8 *>(dg + c * 8) = og;
    *reinterpret_cast<u16x8 *>(du + c * 8) = ou;
  }
}

// dst[r] = pos[r] >= 0 ? src[r] : 0 for rows of W bf16 values (dst may be src)
__global__ void k_mask_rows(const unsigned short *src, const int32_t *__restrict__ pos, long P, int W,
                            unsigned short *dst) {
  const long n8 = P * (W / 8);
  for (long c = (long)blockIdx.x * blockDim.x + threadIdx.x; c < n8; c += (long)gridDim.x * blockDim.x) {
    const long row = c / (W / 8);
    u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
    if (pos[row] >= 0) v = *reinterpret_cast<const u16x8 *>(src + c * 8);
    *reinterpret_cast<u16x8 *>(dst + c * 8) = v;
  }
}

// ------------------------------------------------------------------ host side

int blocks_for(long n, int per = 256) { return (int)std::max<long>(1, std::min<long>(65536, (n + per - 1) / per)); }

struct Dims {
  long P;
  int H, I, hq, hkv, d, C, QD, KD;
};

Dims dims_of(const seg_sizes &sz, const seg_layer_cfg &c) {
  Dims m{};
  m.P = sz.packed_tokens;
  m.H = c.hidden;
  m.I = c.inter;
  m.hq = c.hq;
  m.hkv = c.hkv;
  m.d = c.d;
  m.QD = c.hq * c.d;
  m.KD = c.hkv * c.d;
  long C = c.chunk_rows > 0 ? c.chunk_rows : DEFAULT_CHUNK;
  C = std::max<long>(1, std::min<long>(C, std::max<long>(m.P, 1)));
  m.C = (int)C;
  return m;
}

struct LayerWs {
  size_t pos, a, m, wgu, attn;                                   // forward
  size_t wdT, wgT, wuT, woT, wqT, wkT, wvT, dy1, dO, dq, dk, dv;  // backward
  size_t g, u, dm, dg, du, dbf, part;
  size_t total;
};

LayerWs layer_ws(const seg_sizes &sz, const seg_layer_cfg &c, int bwd) {
  const Dims m = dims_of(sz, c);
  LayerWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 1));
    return o;
  };
  const size_t P = std::max<long>(m.P, 1), C = m.C, H = m.H, I = m.I;
  const size_t Ip = (I + GU_BLOCK - 1) / GU_BLOCK * GU_BLOCK;
  w.pos = take(P * 4);
  w.a = take(C * H * 2);
  w.m = take(C * I * 2);
  w.wgu = take(2 * Ip * H * 2);
  w.attn = take(seg_attn_workspace_bytes(&sz, SEG_BF16, c.hq, c.hkv, c.d, bwd));
  if (bwd) {
    w.wdT = take(I * H * 2);
    w.wgT = take(H * I * 2);
    w.wuT = take(H * I * 2);
    w.woT = take((size_t)m.QD * H * 2);
    w.wqT = take(H * m.QD * 2);
    w.wkT = take(H * m.KD * 2);
    w.wvT = take(H * m.KD * 2);
    w.dy1 = take(P * H * 2);
    w.dO = take(P * m.QD * 2);
    w.dq = take(P * m.QD * 2);
    w.dk = take(P * m.KD * 2);
    w.dv = take(P * m.KD * 2);
    w.g = take(C * I * 2);
    w.u = take(C * I * 2);
    w.dm = take(C * I * 2);
    w.dg = take(C * I * 2);
    w.du = take(C * I * 2);
    w.dbf = take(C * H * 4);
    w.part = take((((C + RMS_ROWS - 1) / RMS_ROWS) * 4 + COLSUM_SPLIT) * H * 4);
  }
  w.total = std::max<size_t>(off, 256);
  return w;
}

void check_layer(const seg_layout *L, const seg_sizes *sz, const seg_layer_cfg *c,
                 const seg_layer_weights *w) {
  SEG_CHECK(L && sz && c && w, SEG_ERR_ARG, "layout, sizes, cfg or weights is NULL");
  SEG_CHECK(c->hidden >= 8 && c->hidden % 8 == 0 && c->inter >= 8 && c->inter % 8 == 0,
            SEG_ERR_UNSUPPORTED, "hidden %d and inter %d must be positive multiples of 8",
            c->hidden, c->inter);
  SEG_CHECK(c->hidden <= 8 * 64 * MAX_CH, SEG_ERR_UNSUPPORTED, "hidden %d > %d", c->hidden,
            8 * 64 * MAX_CH);
  SEG_CHECK(c->hq >= 1 && c->hkv >= 1 && c->hq % c->hkv == 0 && (c->d == 64 || c->d == 128),
            SEG_ERR_UNSUPPORTED, "heads %d/%d, head_dim %d not supported", c->hq, c->hkv, c->d);
  SEG_CHECK(std::isfinite(c->rms_eps) && c->rms_eps > 0.f, SEG_ERR_ARG, "rms_eps must be > 0");
  SEG_CHECK(std::isfinite(c->rope_base) && c->rope_base > 1.f, SEG_ERR_ARG,
            "rope_base must be > 1");
  SEG_CHECK(c->chunk_rows >= 0, SEG_ERR_ARG, "chunk_rows must be >= 0");
  SEG_CHECK(c->chunk_rows <= MAX_CHUNK && c->inter <= MAX_CHUNK && (long)c->hq * c->d <= MAX_CHUNK,
            SEG_ERR_UNSUPPORTED, "chunk_rows %d, inter %d or hq*d above %d", c->chunk_rows,
            c->inter, MAX_CHUNK);
  SEG_CHECK(w->g1 && w->wq && w->wk && w->wv && w->wo && w->g2 && w->wg && w->wu && w->wd,
            SEG_ERR_ARG, "a weight pointer is NULL");
  SEG_CHECK((long)std::max<long>(sz->packed_tokens, 1) * std::max(c->hidden, c->inter) < (1L << 40),
            SEG_ERR_CAPACITY, "tensor too large");
}

#define US(p) reinterpret_cast<unsigned short *>(p)
#define CUS(p) reinterpret_cast<const unsigned short *>(p)

template <class Epi>
void gemm_nt(const unsigned short *A, long lda, const unsigned short *B, long ldb, int M, int N, int K,
             const Epi &ep, hipStream_t st) {
  gemm::gemm_launch(A, lda, B, ldb, M, N, K, ep, st);
  SEG_LAUNCH_CHECK();
}

void build_wgu(const seg_layer_weights &w, int I, int H, unsigned short *wgu, hipStream_t st) {
  const long rows2 = 2L * ((I + GU_BLOCK - 1) / GU_BLOCK * GU_BLOCK);
  k_interleave_gu<<<blocks_for(rows2 * (H / 8)), 256, 0, st>>>(CUS(w.wg), CUS(w.wu), I, H, rows2, wgu);
  SEG_LAUNCH_CHECK();
}

// rows x [gate | up] of a chunk against the interleaved weights, consumed by
// the SwiGLU epilogue (always the 256-wide tiles: it pairs the two 32-column
// halves of a 64-column wave tile)
void gate_up(const unsigned short *a, const unsigned short *wgu, int rows, int H, int I,
             const EpiSwiGLU &ep, hipStream_t st) {
  const int N = 2 * ((I + GU_BLOCK - 1) / GU_BLOCK * GU_BLOCK);
  if (rows <= 0) return;
  gemm::k_gemm_big<EpiSwiGLU><<<gemm::big_blocks(rows, N), gemm::BIG_THREADS, 0, st>>>(
      a, H, wgu, H, rows, N, H, ep);
  SEG_LAUNCH_CHECK();
}

// C[M][N] (+)= At^T Bt over K rows; At [K][lda], Bt [K][ldb]
template <class Epi>
void gemm_tn(const unsigned short *At, long lda, const unsigned short *Bt, long ldb, int M, int N,
             int K, const Epi &ep, hipStream_t st) {
  gemm::gemm_launch_tn(At, lda, Bt, ldb, M, N, K, ep, st);
  SEG_LAUNCH_CHECK();
}

void transpose(const unsigned short *x, long ldx, int rows, int cols, int pad_rows,
               unsigned short *y, hipStream_t st) {
  k_transpose2d<unsigned short><<<gemm::grid64(cols, pad_rows), 256, 0, st>>>(
      x, ldx, nullptr, rows, cols, pad_rows, y, pad_rows);
  SEG_LAUNCH_CHECK();
}

void rms_fwd(const unsigned short *x, long ldx, const void *g, float eps, int rows, int H,
             const int32_t *pos, unsigned short *y, float *rstd, hipStream_t st) {
  k_rms_fwd<<<(rows + 3) / 4, 256, 0, st>>>(x, ldx, CUS(g), eps, rows, H, pos, y, H, rstd);
  SEG_LAUNCH_CHECK();
}

void rms_bwd(const unsigned short *x, const void *g, const float *rstd, const float *dy, int rows,
             int H, const int32_t *pos, const unsigned short *resid, unsigned short *out,
             float *part, float *dgrad, hipStream_t st) {
  const int nb = (rows + RMS_ROWS - 1) / RMS_ROWS;
  k_rms_bwd<<<nb, 256, 0, st>>>(x, H, CUS(g), rstd, dy, H, rows, H, pos, resid, H, out, H, part);
  SEG_LAUNCH_CHECK();
  float *part2 = part + (long)nb * 4 * H;
  k_colsum_part<<<dim3((H + 255) / 256, COLSUM_SPLIT), 256, 0, st>>>(part, nb * 4, H, part2);
  SEG_LAUNCH_CHECK();
  k_colsum_add<<<(H + 255) / 256, 256, 0, st>>>(part2, H, dgrad);
  SEG_LAUNCH_CHECK();
}

void positions(const seg_layout *L, const seg_sizes *sz, long P, int32_t *pos, hipStream_t st) {
  k_positions<<<blocks_for(P), 256, 0, st>>>(L->seg_info, sz->num_segments, P, pos);
  SEG_LAUNCH_CHECK();
}

void rope(unsigned short *x, long P, int heads, int d, const int32_t *pos, float base, int inverse,
          hipStream_t st) {
  k_rope<<<blocks_for(P * heads * (d / 2)), 256, 0, st>>>(x, P, heads, d, pos,
                                                          std::log2((double)base), inverse);
  SEG_LAUNCH_CHECK();
}

void zero_grads(const seg_layer_grads &g, const seg_layer_cfg &c, hipStream_t st) {
  const long H = c.hidden, I = c.inter, QD = (long)c.hq * c.d, KD = (long)c.hkv * c.d;
  fill32(g.g1, H, 0u, st);
  fill32(g.g2, H, 0u, st);
  fill32(g.wq, QD * H, 0u, st);
  fill32(g.wk, KD * H, 0u, st);
  fill32(g.wv, KD * H, 0u, st);
  fill32(g.wo, H * QD, 0u, st);
  fill32(g.wg, I * H, 0u, st);
  fill32(g.wu, I * H, 0u, st);
  fill32(g.wd, H * I, 0u, st);
}

void check_status(seg_status s) {
  if (s != SEG_OK) throw Fail{s};
}

void layer_fwd_impl(const seg_layout *L, const seg_sizes *sz, const seg_layer_cfg &c,
                    const seg_layer_weights &w, const unsigned short *x, unsigned short *y,
                    const seg_layer_saved &sv, char *base, const LayerWs &W, size_t ws_bytes,
                    hipStream_t st) {
  const Dims m = dims_of(*sz, c);
  const long P = m.P;
  const int H = m.H, I = m.I;
  int32_t *pos = reinterpret_cast<int32_t *>(base + W.pos);
  unsigned short *a = US(base + W.a), *mb = US(base + W.m), *wgu = US(base + W.wgu);
  unsigned short *q = US(sv.q), *k = US(sv.k), *v = US(sv.v), *o = US(sv.o), *y1 = US(sv.y1);
  {
    ProfScope prof("ly_misc", st);
    positions(L, sz, P, pos, st);
    build_wgu(w, I, H, wgu, st);
  }
  for (long r0 = 0; r0 < P; r0 += m.C) {
    const int cr = (int)std::min<long>(m.C, P - r0);
    {
      ProfScope prof("ly_norm", st);
      rms_fwd(x + r0 * H, H, w.g1, c.rms_eps, cr, H, pos + r0, a, sv.rstd1 + r0, st);
    }
    ProfScope prof("ly_proj", st);
    gemm_nt(a, H, CUS(w.wq), H, cr, m.QD, H, EpiStore<unsigned short>{q + r0 * m.QD, m.QD, 1.f}, st);
    gemm_nt(a, H, CUS(w.wk), H, cr, m.KD, H, EpiStore<unsigned short>{k + r0 * m.KD, m.KD, 1.f}, st);
    gemm_nt(a, H, CUS(w.wv), H, cr, m.KD, H, EpiStore<unsigned short>{v + r0 * m.KD, m.KD, 1.f}, st);
  }
  {
    ProfScope prof("ly_rope", st);
    rope(q, P, m.hq, m.d, pos, c.rope_base, 0, st);
    rope(k, P, m.hkv, m.d, pos, c.rope_base, 0, st);
  }
  check_status(seg_attn_fwd(L, sz, SEG_BF16, m.hq, m.hkv, m.d, 1.f / std::sqrt((float)m.d), q, k, v,
                            o, sv.lse, base + W.attn, ws_bytes - W.attn, st));
  {
    ProfScope prof("ly_misc", st);
    k_mask_rows<<<blocks_for(P * (m.QD / 8)), 256, 0, st>>>(o, pos, P, m.QD, o);
    SEG_LAUNCH_CHECK();
  }
  for (long r0 = 0; r0 < P; r0 += m.C) {
    const int cr = (int)std::min<long>(m.C, P - r0);
    {
      ProfScope prof("ly_proj", st);
      gemm_nt(o + r0 * m.QD, m.QD, CUS(w.wo), m.QD, cr, H, m.QD,
              EpiResid{y1 + r0 * H, H, x + r0 * H, H, 1.f}, st);
    }
    {
      ProfScope prof("ly_norm", st);
      rms_fwd(y1 + r0 * H, H, w.g2, c.rms_eps, cr, H, pos + r0, a, sv.rstd2 + r0, st);
    }
    ProfScope prof("ly_mlp", st);
    gate_up(a, wgu, cr, H, I, EpiSwiGLU{mb, nullptr, nullptr, I, I}, st);
    gemm_nt(mb, I, CUS(w.wd), I, cr, H, I, EpiResid{y + r0 * H, H, y1 + r0 * H, H, 1.f}, st);
  }
}

void layer_bwd_impl(const seg_layout *L, const seg_sizes *sz, const seg_layer_cfg &c,
                    const seg_layer_weights &w, const unsigned short *x, const seg_layer_saved &sv,
                    const unsigned short *dy, unsigned short *dx, const seg_layer_grads &gr,
                    char *base, const LayerWs &W, size_t ws_bytes, hipStream_t st) {
  const Dims m = dims_of(*sz, c);
  const long P = m.P;
  const int H = m.H, I = m.I;
  int32_t *pos = reinterpret_cast<int32_t *>(base + W.pos);
  unsigned short *a = US(base + W.a), *gb = US(base + W.g), *ub = US(base + W.u), *mb = US(base + W.m),
                 *wgu = US(base + W.wgu);
  unsigned short *wdT = US(base + W.wdT), *wgT = US(base + W.wgT), *wuT = US(base + W.wuT);
  unsigned short *woT = US(base + W.woT), *wqT = US(base + W.wqT), *wkT = US(base + W.wkT),
                 *wvT = US(base + W.wvT);
  unsigned short *dy1 = US(base + W.dy1), *dO = US(base + W.dO), *dq = US(base + W.dq),
                 *dk = US(base + W.dk), *dv = US(base + W.dv);
  unsigned short *dm = US(base + W.dm), *dgb = US(base + W.dg), *dub = US(base + W.du);
  float *dbf = reinterpret_cast<float *>(base + W.dbf);
  float *part = reinterpret_cast<float *>(base + W.part);
  const unsigned short *q = CUS(sv.q), *k = CUS(sv.k), *v = CUS(sv.v), *o = CUS(sv.o),
                       *y1 = CUS(sv.y1);
  {
    ProfScope prof("ly_misc", st);
    zero_grads(gr, c, st);
    positions(L, sz, P, pos, st);
    build_wgu(w, I, H, wgu, st);
    // transposed weights (k-contiguous operands of the data-gradient GEMMs)
    transpose(CUS(w.wd), I, H, I, H, wdT, st);        // wd [H, I] -> [I, H]
    transpose(CUS(w.wg), H, I, H, I, wgT, st);        // wg [I, H] -> [H, I]
    transpose(CUS(w.wu), H, I, H, I, wuT, st);
    transpose(CUS(w.wo), m.QD, H, m.QD, H, woT, st);  // wo [H, QD] -> [QD, H]
    transpose(CUS(w.wq), H, m.QD, H, m.QD, wqT, st);  // wq [QD, H] -> [H, QD]
    transpose(CUS(w.wk), H, m.KD, H, m.KD, wkT, st);
    transpose(CUS(w.wv), H, m.KD, H, m.KD, wvT, st);
    // dy1 starts as dy with the padding rows zeroed
    k_mask_rows<<<blocks_for(P * (H / 8)), 256, 0, st>>>(dy, pos, P, H, dy1);
    SEG_LAUNCH_CHECK();
  }
  // MLP and output projection, chunk by chunk
  for (long r0 = 0; r0 < P; r0 += m.C) {
    const int cr = (int)std::min<long>(m.C, P - r0);
    unsigned short *dy1c = dy1 + r0 * H;
    {
      ProfScope prof("ly_norm", st);
      rms_fwd(y1 + r0 * H, H, w.g2, c.rms_eps, cr, H, pos + r0, a, nullptr, st);  // b
    }
    {
      ProfScope prof("ly_mlp", st);
      gate_up(a, wgu, cr, H, I, EpiSwiGLU{mb, gb, ub, I, I}, st);  // m, g, u
      gemm_nt(dy1c, H, wdT, H, cr, I, H, EpiStore<unsigned short>{dm, I, 1.f}, st);  // dm = dy wd
      const long n8 = (long)cr * I / 8;
      k_swiglu_bwd<<<blocks_for(n8), 256, 0, st>>>(gb, ub, dm, dgb, dub, n8);
      SEG_LAUNCH_CHECK();
      gemm_nt(dgb, I, wgT, I, cr, H, I, EpiStore<float>{dbf, H, 1.f}, st);  // db = dg wg + du wu
      gemm_nt(dub, I, wuT, I, cr, H, I, EpiAccum{dbf, H, 1.f}, st);
    }
    {
      // dWd += dy^T m, dWg += dg^T b, dWu += du^T b in one launch
      ProfScope prof("ly_wgrad", st);
      gemm::TnGroup<EpiAccum, 3> g{{dy1c, dgb, dub}, {mb, a, a}, {H, I, I}, {I, H, H}, {H, I, I},
                                   {I, H, H},
                                   {EpiAccum{gr.wd, I, 1.f}, EpiAccum{gr.wg, H, 1.f},
                                    EpiAccum{gr.wu, H, 1.f}}, {}};
      gemm::gemm_launch_tn(g, cr, st);
      SEG_LAUNCH_CHECK();
    }
    {
      ProfScope prof("ly_norm", st);
      rms_bwd(y1 + r0 * H, w.g2, sv.rstd2 + r0, dbf, cr, H, pos + r0, dy1c, dy1c, part, gr.g2, st);
    }
    ProfScope prof("ly_proj", st);
    gemm_tn(dy1c, H, o + r0 * m.QD, m.QD, H, m.QD, cr, EpiAccum{gr.wo, m.QD, 1.f}, st);  // dWo
    gemm_nt(dy1c, H, woT, H, cr, m.QD, H, EpiStore<unsigned short>{dO + r0 * m.QD, m.QD, 1.f}, st);
  }
  check_status(seg_attn_bwd(L, sz, SEG_BF16, m.hq, m.hkv, m.d, 1.f / std::sqrt((float)m.d), q, k, v,
                            o, sv.lse, dO, dq, dk, dv, base + W.attn, ws_bytes - W.attn, st));
  {
    ProfScope prof("ly_rope", st);
    k_mask_rows<<<blocks_for(P * (m.QD / 8)), 256, 0, st>>>(dq, pos, P, m.QD, dq);
    SEG_LAUNCH_CHECK();
    k_mask_rows<<<blocks_for(P * (m.KD / 8)), 256, 0, st>>>(dk, pos, P, m.KD, dk);
    SEG_LAUNCH_CHECK();
    k_mask_rows<<<blocks_for(P * (m.KD / 8)), 256, 0, st>>>(dv, pos, P, m.KD, dv);
    SEG_LAUNCH_CHECK();
    rope(dq, P, m.hq, m.d, pos, c.rope_base, 1, st);
    rope(dk, P, m.hkv, m.d, pos, c.rope_base, 1, st);
  }
  // q/k/v projections and the first norm, chunk by chunk
  for (long r0 = 0; r0 < P; r0 += m.C) {
    const int cr = (int)std::min<long>(m.C, P - r0);
    {
      ProfScope prof("ly_norm", st);
      rms_fwd(x + r0 * H, H, w.g1, c.rms_eps, cr, H, pos + r0, a, nullptr, st);  // a
    }
    {
      ProfScope prof("ly_proj", st);
      gemm_nt(dq + r0 * m.QD, m.QD, wqT, m.QD, cr, H, m.QD, EpiStore<float>{dbf, H, 1.f}, st);
      gemm_nt(dk + r0 * m.KD, m.KD, wkT, m.KD, cr, H, m.KD, EpiAccum{dbf, H, 1.f}, st);
      gemm_nt(dv + r0 * m.KD, m.KD, wvT, m.KD, cr, H, m.KD, EpiAccum{dbf, H, 1.f}, st);
    }
    {
      // dWq += dq^T a, dWk += dk^T a, dWv += dv^T a in one launch
      ProfScope prof("ly_wgrad", st);
      gemm::TnGroup<EpiAccum, 3> g{{dq + r0 * m.QD, dk + r0 * m.KD, dv + r0 * m.KD}, {a, a, a},
                                   {m.QD, m.KD, m.KD}, {H, H, H}, {m.QD, m.KD, m.KD}, {H, H, H},
                                   {EpiAccum{gr.wq, H, 1.f}, EpiAccum{gr.wk, H, 1.f},
                                    EpiAccum{gr.wv, H, 1.f}}, {}};
      gemm::gemm_launch_tn(g, cr, st);
      SEG_LAUNCH_CHECK();
    }
    ProfScope prof("ly_norm", st);
    rms_bwd(x + r0 * H, w.g1, sv.rstd1 + r0, dbf, cr, H, pos + r0, dy1 + r0 * H, dx + r0 * H, part,
            gr.g1, st);
  }
}

}  // namespace
}  // namespace seg

using namespace seg;

extern "C" size_t seg_layer_workspace_bytes(const seg_sizes *sz, const seg_layer_cfg *cfg,
                                            int32_t bwd) {
  if (!sz || !cfg || cfg->hidden < 1 || cfg->inter < 1 || cfg->hq < 1 || cfg->hkv < 1 ||
      cfg->d < 1)
    return 0;
  return layer_ws(*sz, *cfg, bwd ? 1 : 0).total;
}

extern "C" seg_status seg_layer_fwd(const seg_layout *L, const seg_sizes *sz,
                                    const seg_layer_cfg *cfg, const seg_layer_weights *w,
                                    const void *x, void *y, const seg_layer_saved *saved, void *ws,
                                    size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    check_layer(L, sz, cfg, w);
    const LayerWs W = layer_ws(*sz, *cfg, 0);
    SEG_CHECK(ws_bytes >= W.total, SEG_ERR_WORKSPACE, "workspace of %zu bytes < required %zu",
              ws_bytes, W.total);
    if (sz->packed_tokens == 0) return;
    SEG_CHECK(x && y && saved && ws, SEG_ERR_ARG, "x, y, saved or ws is NULL");
    SEG_CHECK(saved->q && saved->k && saved->v && saved->o && saved->lse && saved->y1 &&
                  saved->rstd1 && saved->rstd2,
              SEG_ERR_ARG, "a saved-buffer pointer is NULL");
    layer_fwd_impl(L, sz, *cfg, *w, CUS(x), US(y), *saved, static_cast<char *>(ws), W, ws_bytes,
                   stream);
  });
}

extern "C" seg_status seg_layer_bwd(const seg_layout *L, const seg_sizes *sz,
                                    const seg_layer_cfg *cfg, const seg_layer_weights *w,
                                    const void *x, const seg_layer_saved *saved, const void *dy,
                                    void *dx, const seg_layer_grads *g, void *ws, size_t ws_bytes,
                                    hipStream_t stream) {
  return guarded([&] {
    check_layer(L, sz, cfg, w);
    const LayerWs W = layer_ws(*sz, *cfg, 1);
    SEG_CHECK(ws_bytes >= W.total, SEG_ERR_WORKSPACE, "workspace of %zu bytes < required %zu",
              ws_bytes, W.total);
    SEG_CHECK(g && g->g1 && g->wq && g->wk && g->wv && g->wo && g->g2 && g->wg && g->wu && g->wd,
              SEG_ERR_ARG, "a gradient pointer is NULL");
    if (sz->packed_tokens == 0) {
      zero_grads(*g, *cfg, stream);
      return;
    }
    SEG_CHECK(x && saved && dy && dx && ws, SEG_ERR_ARG, "x, saved, dy, dx or ws is NULL");
    SEG_CHECK(saved->q && saved->k && saved->v && saved->o && saved->lse && saved->y1 &&
                  saved->rstd1 && saved->rstd2,
              SEG_ERR_ARG, "a saved-buffer pointer is NULL");
    layer_bwd_impl(L, sz, *cfg, *w, CUS(x), *saved, CUS(dy), US(dx), *g, static_cast<char *>(ws), W,
                   ws_bytes, stream);
  });
}
