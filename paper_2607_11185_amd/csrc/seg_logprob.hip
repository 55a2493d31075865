// Fused action-token log-prob and clipped policy-ratio loss with gradients
// (Eq. (loss) of App. E: min(rho A, clip(rho, 1 - eps_l, 1 + eps_h) A) over the
// trained action tokens, rho = pi_theta / pi_rollout), bf16 MFMA on gfx950.
//
// Only the R action rows are projected onto the vocabulary.  Pipeline:
//   1. zT[v][r] = s * W[v] . h[r] (MFMA, fp32 out) with a fused epilogue that
//      writes per-(row, 128-vocab tile) max / sum-exp partials and captures the
//      target logit;
//   2. per row: LSE from the partials (fixed order), logp, rho, loss, the
//      clipped flag and g = d loss_sum / d logp;
//   3. dz = g * (onehot(target) - softmax(z)) as bf16, written in both
//      orientations (one pass over zT);
//   4. dH = s * dz W and dW = s * dz^T h (MFMA).
// All GEMMs use the shared "NT" kernel of gemm.h: C[m][n] = sum_k A[m][k] B[n][k]
// with both operands k-contiguous.
#include <climits>
#include <cmath>

#include "common.h"
#include "gemm.h"

namespace seg {
namespace {

using gemm::EpiStore;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

// Epilogue of the logits GEMM (M = vocab, N = rows): writes zT, captures the
// target logit and the per-(row, vocab tile) max / sum-exp partials.
struct EpiLogits {
  float *zt;        // [M][ldz] fp32
  long ldz;
  float2 *stats;    // [ceil(M/128) slabs][N]: (max, sum exp(z - max)) in log2 units
  int nrows;        // N
  const int32_t *target;  // [N]
  float *ztgt;      // [N]
  float scale;
  // for the 256-wide NT kernel: a wave covers one 128-row slab of M; the two
  // lane halves of a column are combined by a shuffle
  template <int TM, int TN>
  __device__ __forceinline__ void operator()(const f32x16 (&acc)[TM][TN],
                                             const gemm::Tile &t) const {
    static_assert(TM == 4, "logits epilogue expects 128-row wave tiles");
    const int slab_row = t.m0 + t.wr;
#pragma unroll
    for (int bn = 0; bn < TN; ++bn) {
      const int n = t.column(bn);
      const bool nok = n < t.N;
      const int tgt = nok ? target[n] : -1;
      float mx = -INFINITY;
#pragma unroll
      for (int bm = 0; bm < TM; ++bm)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = t.row(bm, r);
          const float z = acc[bm][bn][r] * scale;
          if (nok && m < t.M) {
            zt[(long)m * ldz + n] = z;
            if (m == tgt) ztgt[n] = z;
            mx = fmaxf(mx, z * LOG2E);
          }
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      float sm = 0.f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int bm = 0; bm < TM; ++bm)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = t.row(bm, r);
            if (m < t.M) sm += exp2f(acc[bm][bn][r] * scale * LOG2E - mx);
          }
      }
      sm += __shfl_xor(sm, 32, 64);
      if (t.hh == 0 && nok && slab_row < t.M)
        stats[(long)(slab_row / 128) * nrows + n] = make_float2(mx, sm);
    }
  }
};

__global__ void __launch_bounds__(256) k_row_loss(
    const float2 *__restrict__ stats, int ntiles, int rows, const float *__restrict__ ztgt,
    const float *__restrict__ old_logp, const float *__restrict__ ref_logp,
    const float *__restrict__ adv, const int32_t *__restrict__ row_traj, int num_traj,
    seg_loss_cfg cfg, float *__restrict__ logp, float *__restrict__ loss_tok,
    uint8_t *__restrict__ clipped, float *__restrict__ kl_tok, float *__restrict__ lse_out,
    float *__restrict__ g_out) {
  __shared__ float2 red[256];
  const int r = blockIdx.x, t = threadIdx.x;
  float mx = -INFINITY, sm = 0.f;
  for (int i = t; i < ntiles; i += 256) {
    const float2 p = stats[(long)i * rows + r];
    if (p.x == -INFINITY) continue;
    if (p.x > mx) {
      sm = sm * exp2f(mx - p.x) + p.y;
      mx = p.x;
    } else {
      sm += p.y * exp2f(p.x - mx);
    }
  }
  red[t] = make_float2(mx, sm);
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) {
      const float2 a = red[t], b = red[t + o];
      const float m2 = fmaxf(a.x, b.x);
      float s2 = 0.f;
      if (m2 != -INFINITY) {
        if (a.x != -INFINITY) s2 += a.y * exp2f(a.x - m2);
        if (b.x != -INFINITY) s2 += b.y * exp2f(b.x - m2);
      }
      red[t] = make_float2(m2, s2);
    }
    __syncthreads();
  }
  if (t == 0) {
    const float lse = (red[0].x + log2f(red[0].y)) * LN2;
    const float lp = ztgt[r] - lse;
    // an out-of-range trajectory index yields NaN rather than a stray read
    const int tj = row_traj[r];
    const float A = (tj >= 0 && tj < num_traj) ? adv[tj] : __builtin_nanf("");
    const float rho = expf(lp - old_logp[r]);
    const float lo = 1.f - cfg.eps_low, hi = 1.f + cfg.eps_high;
    const float unc = rho * A;
    const float clp = fminf(fmaxf(rho, lo), hi) * A;
    float obj = fminf(unc, clp);
    bool cl = (A > 0.f && rho > hi) || (A < 0.f && rho < lo);
    if (cfg.dual_clip_c > 0.f && A < 0.f) {
      obj = fmaxf(obj, cfg.dual_clip_c * A);
      cl = cl || rho > cfg.dual_clip_c;
    }
    // KL(pi_theta || pi_ref) per token: e^x - x - 1 with x = ref - logp,
    // written expm1(x) - x (no cancellation for small x); its logp
    // derivative is 1 - e^x = -expm1(x)
    float kl = 0.f, dkl = 0.f;
    if (ref_logp) {
      const float x = ref_logp[r] - lp, em1 = expm1f(x);
      kl = em1 - x;
      dkl = -em1;
    }
    logp[r] = lp;
    loss_tok[r] = -obj + cfg.kl_coef * kl;
    clipped[r] = cl ? 1 : 0;
    if (kl_tok) kl_tok[r] = kl;
    lse_out[r] = lse;
    g_out[r] = (cl ? 0.f : -cfg.loss_scale * rho * A) + cfg.loss_scale * cfg.kl_coef * dkl;
  }
}

// loss_sum = loss_scale * sum(loss_tok), fixed-order reduction in one block.
__global__ void __launch_bounds__(256) k_loss_sum(const float *__restrict__ loss_tok, int rows,
                                                  float scale, float *__restrict__ out) {
  __shared__ double red[256];
  const int t = threadIdx.x;
  double s = 0.0;
  for (int i = t; i < rows; i += 256) s += (double)loss_tok[i];
  red[t] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  if (t == 0) *out = (float)(red[0] * (double)scale);
}

// dz = g[r] * (onehot(target[r]) - exp(z - lse[r])), from zT [V][ldz] to
// dz [Rp][Vp] and dzT [Vp][Rp] (bf16, zero in the padding).  64x64 tiles.
__global__ void __launch_bounds__(256) k_dz(const float *__restrict__ zt, long ldz, int V, int R,
                                            int Vp, int Rp, const float *__restrict__ lse,
                                            const float *__restrict__ g,
                                            const int32_t *__restrict__ target,
                                            unsigned short *__restrict__ dz,
                                            unsigned short *__restrict__ dzt) {
  __shared__ unsigned short t[64][66];
  const int v0 = blockIdx.y * 64, r0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int r = r0 + tx;
  const bool rok = r < R;
  const float lr = rok ? lse[r] : 0.f, gr = rok ? g[r] : 0.f;
  const int tg = rok ? target[r] : -1;
  for (int i = ty; i < 64; i += 4) {
    const int v = v0 + i;
    float val = 0.f;
    if (rok && v < V) {
      const float p = expf(zt[(long)v * ldz + r] - lr);
      val = gr * ((v == tg ? 1.f : 0.f) - p);
    }
    const unsigned short b = f2bf_bits(val);
    if (v < Vp && r < Rp) dzt[(long)v * Rp + r] = b;
    t[i][tx] = b;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int rr = r0 + i, v = v0 + tx;
    if (rr < Rp && v < Vp) dz[(long)rr * Vp + v] = t[tx][i];
  }
}

// y[r][:] = x[rowmap[r]][:] as bf16 (rows < rows_pad are zero beyond rows).
template <class TI>
__global__ void k_gather_rows(const TI *__restrict__ x, long ldx, const int32_t *__restrict__ rowmap,
                              int rows, int rows_pad, int cols, unsigned short *__restrict__ y) {
  const long n = (long)rows_pad * cols;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
    const int r = (int)(i / cols), c = (int)(i % cols);
    unsigned short b = 0;
    if (r < rows) b = load_bf(x, (long)(rowmap ? rowmap[r] : r) * ldx + c);
    y[i] = b;
  }
}

struct LpWs {
  size_t hb, wb, zt, stats, ztgt, lse, g, dz, dzt, total;
  int Rp, Vp, ntiles;
};

LpWs lp_ws(int rows, int hidden, int vocab, seg_dtype dt) {
  LpWs w{};
  w.Rp = (rows + 31) / 32 * 32;
  w.Vp = (vocab + 31) / 32 * 32;
  w.ntiles = (vocab + 127) / 128;  // 128-row slabs of the logits epilogue
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 1));
    return o;
  };
  const size_t Rp = w.Rp, Vp = w.Vp, H = hidden;
  w.hb = take(Rp * H * 2);
  w.wb = dt == SEG_F32 ? take((size_t)vocab * H * 2) : 0;
  w.zt = take((size_t)vocab * Rp * 4);
  w.stats = take((size_t)w.ntiles * std::max(rows, 1) * sizeof(float2));
  w.ztgt = take(Rp * 4);
  w.lse = take(Rp * 4);
  w.g = take(Rp * 4);
  w.dz = take(Rp * Vp * 2);
  w.dzt = take(Vp * Rp * 2);
  w.total = off;
  return w;
}

dim3 grid2(long cols, long rows, int t = 64) {
  return dim3((unsigned)((cols + t - 1) / t), (unsigned)((rows + t - 1) / t));
}

template <class TI, class TO>
void logprob_impl(int rows, int H, int V, const TI *h, const int32_t *row_index, const TI *w,
                  const int32_t *target, const float *old_logp, const float *ref_logp,
                  const float *adv, const int32_t *row_traj, int num_traj,
                  const seg_loss_cfg &cfg, float *logp, float *loss_tok, uint8_t *clipped,
                  float *kl_tok, float *loss_sum, void *dh, float *dw, char *base,
                  const LpWs &L, hipStream_t st) {
  const int Rp = L.Rp, Vp = L.Vp;
  unsigned short *hb = reinterpret_cast<unsigned short *>(base + L.hb);
  float *zt = reinterpret_cast<float *>(base + L.zt);
  float2 *stats = reinterpret_cast<float2 *>(base + L.stats);
  float *ztgt = reinterpret_cast<float *>(base + L.ztgt);
  float *lse = reinterpret_cast<float *>(base + L.lse);
  float *g = reinterpret_cast<float *>(base + L.g);
  unsigned short *dz = reinterpret_cast<unsigned short *>(base + L.dz);
  unsigned short *dzt = reinterpret_cast<unsigned short *>(base + L.dzt);

  // gathered action rows (bf16)
  {
    ProfScope prof("lp_prep", st);
    const long n = (long)Rp * H;
    k_gather_rows<TI><<<(int)std::min<long>(65536, (n + 255) / 256), 256, 0, st>>>(
        h, H, row_index, rows, Rp, H, hb);
    SEG_LAUNCH_CHECK();
  }
  const unsigned short *wb;
  if constexpr (sizeof(TI) == 4) {
    unsigned short *w2 = reinterpret_cast<unsigned short *>(base + L.wb);
    const long n = (long)V * H;
    ProfScope prof("lp_prep", st);
    k_gather_rows<TI><<<(int)std::min<long>(65536, (n + 255) / 256), 256, 0, st>>>(
        w, H, nullptr, V, V, H, w2);
    SEG_LAUNCH_CHECK();
    wb = w2;
  } else {
    wb = reinterpret_cast<const unsigned short *>(w);
  }
  // 1. logits zT = s * W h^T with partial softmax stats; the target logit
  //    stays NaN for a target outside [0, vocab)
  fill32(ztgt, Rp, 0xffffffffu, st);
  {
    EpiLogits e{zt, Rp, stats, rows, target, ztgt, cfg.logit_scale};
    ProfScope prof("logits", st);
    gemm::k_gemm_big<EpiLogits><<<gemm::big_blocks(V, rows), gemm::BIG_THREADS, 0, st>>>(
        wb, H, hb, H, V, rows, H, e);
    SEG_LAUNCH_CHECK();
  }
  // 2. per-row loss
  {
  ProfScope prof("row_loss", st);
  k_row_loss<<<rows, 256, 0, st>>>(stats, L.ntiles, rows, ztgt, old_logp, ref_logp, adv, row_traj,
                                   num_traj, cfg, logp, loss_tok, clipped, kl_tok, lse, g);
  SEG_LAUNCH_CHECK();
  k_loss_sum<<<1, 256, 0, st>>>(loss_tok, rows, cfg.loss_scale, loss_sum);
  SEG_LAUNCH_CHECK();
  }
  if (!cfg.want_grad) return;
  // 3. dz in both orientations
  {
  ProfScope prof("dz", st);
  k_dz<<<grid2(Rp, Vp), 256, 0, st>>>(zt, Rp, V, rows, Vp, Rp, lse, g, target, dz, dzt);
  SEG_LAUNCH_CHECK();
  }
  // 4. dH = s * dz W = s (dz^T)^T W: the transposed-operand GEMM over the
  //    vocabulary (At = dz^T [V][Rp], Bt = W [V][H]; M = rows, N = H, K = V)
  {
    EpiStore<TO> e{static_cast<TO *>(dh), H, cfg.logit_scale};
    ProfScope prof("dh", st);
    gemm::gemm_launch_tn(dzt, Rp, wb, H, rows, H, V, e, st);
    SEG_LAUNCH_CHECK();
  }
  //    dW = s * dz^T h over the rows (At = dz [Rp][Vp], Bt = h [Rp][H];
  //    M = V, N = H, K = rows)
  {
    EpiStore<float> e{dw, H, cfg.logit_scale};
    ProfScope prof("dw", st);
    gemm::gemm_launch_tn(dz, Vp, hb, H, V, H, rows, e, st);
    SEG_LAUNCH_CHECK();
  }
}

}  // namespace
}  // namespace seg

using namespace seg;

extern "C" size_t seg_logprob_workspace_bytes(int32_t rows, int32_t hidden, int32_t vocab,
                                              seg_dtype dt) {
  if (rows < 0 || hidden < 1 || vocab < 1) return 0;
  return lp_ws(rows, hidden, vocab, dt).total;
}

extern "C" seg_status seg_logprob_loss(int32_t rows, int32_t hidden, int32_t vocab, seg_dtype dt,
                                       const void *h, const int32_t *row_index, const void *w,
                                       const int32_t *target, const float *old_logp,
                                       const float *ref_logp, const float *adv,
                                       const int32_t *row_traj, int32_t num_traj,
                                       const seg_loss_cfg *cfg, float *logp, float *loss_tok,
                                       uint8_t *clipped, float *kl_tok, float *loss_sum,
                                       void *dh, float *dw, void *ws, size_t ws_bytes,
                                       hipStream_t stream) {
  return guarded([&] {
    SEG_CHECK(cfg != nullptr, SEG_ERR_ARG, "cfg is NULL");
    SEG_CHECK(dt == SEG_BF16 || dt == SEG_F32, SEG_ERR_ARG, "unknown dtype %d", (int)dt);
    SEG_CHECK(rows >= 0 && hidden >= 1 && vocab >= 1 && num_traj >= 0, SEG_ERR_ARG,
              "bad sizes rows=%d hidden=%d vocab=%d num_traj=%d", rows, hidden, vocab, num_traj);
    SEG_CHECK(hidden % 8 == 0, SEG_ERR_UNSUPPORTED, "hidden %d must be a multiple of 8", hidden);
    // GEMM operand rows (hidden, padded vocab, padded rows) are addressed with
    // 32-bit offsets inside a 256-row block
    SEG_CHECK(hidden <= (1 << 20) && vocab <= (1 << 20) - 256 && rows <= (1 << 20) - 256,
              SEG_ERR_CAPACITY, "rows %d, hidden %d or vocab %d above 2^20", rows, hidden, vocab);
    SEG_CHECK(std::isfinite(cfg->eps_low) && std::isfinite(cfg->eps_high) &&
                  std::isfinite(cfg->loss_scale) && std::isfinite(cfg->logit_scale) &&
                  std::isfinite(cfg->dual_clip_c) && std::isfinite(cfg->kl_coef),
              SEG_ERR_ARG, "non-finite loss setting");
    SEG_CHECK(cfg->eps_low >= 0.f && cfg->eps_high >= 0.f, SEG_ERR_ARG, "negative clip range");
    SEG_CHECK(cfg->kl_coef >= 0.f, SEG_ERR_ARG, "negative kl_coef");
    SEG_CHECK(cfg->kl_coef == 0.f || ref_logp != nullptr, SEG_ERR_ARG,
              "kl_coef > 0 needs ref_logp");
    const LpWs L = lp_ws(rows, hidden, vocab, dt);
    SEG_CHECK(ws_bytes >= L.total, SEG_ERR_WORKSPACE, "workspace of %zu bytes < required %zu",
              ws_bytes, L.total);
    SEG_CHECK(loss_sum != nullptr, SEG_ERR_ARG, "loss_sum is NULL");
    if (rows == 0) {
      fill32(loss_sum, 1, 0u, stream);
      if (cfg->want_grad && dw) fill32(dw, (long)vocab * hidden, 0u, stream);
      return;
    }
    SEG_CHECK(h && w && target && old_logp && adv && row_traj && logp && loss_tok && clipped && ws,
              SEG_ERR_ARG, "a tensor pointer is NULL");
    SEG_CHECK(num_traj >= 1, SEG_ERR_ARG, "num_traj must be >= 1 when rows > 0");
    if (cfg->want_grad) SEG_CHECK(dh && dw, SEG_ERR_ARG, "dh/dw is NULL with want_grad");
    char *base = static_cast<char *>(ws);
    if (dt == SEG_F32)
      logprob_impl<float, float>(rows, hidden, vocab, static_cast<const float *>(h), row_index,
                                 static_cast<const float *>(w), target, old_logp, ref_logp, adv,
                                 row_traj, num_traj, *cfg, logp, loss_tok, clipped, kl_tok,
                                 loss_sum, dh, dw, base, L, stream);
    else
      logprob_impl<unsigned short, unsigned short>(
          rows, hidden, vocab, static_cast<const unsigned short *>(h), row_index,
          static_cast<const unsigned short *>(w), target, old_logp, ref_logp, adv, row_traj,
          num_traj, *cfg, logp, loss_tok, clipped, kl_tok, loss_sum, dh, dw, base, L, stream);
  });
}
