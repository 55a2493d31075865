/*
 * seg.h - C ABI of libseg: the segmented training hot path of Visual Context
 * Segmentation (ScaleCUA, Sec. 3.3 "Visual Context Segmentation for
 * Long-Horizon Multimodal RL", App. D "Sliding-Window Details", Eq. (loss) of
 * App. E) on AMD Instinct MI355X (gfx950).
 *
 * A trajectory is a system prompt followed by T turns; turn j carries one
 * screenshot (an image-token block of img_len tokens) and one text block of
 * text_len tokens whose last action_len tokens are the trained action tokens.
 * Trajectories are cut into segments of at most L turns; inside a segment every
 * earlier text token stays visible while a screenshot is visible only to the
 * queries of the W turns starting at its own (the sliding window of W
 * screenshots, Sec. 3.3).  The library builds the packed layout and a 128x128
 * block-sparse tile map of it, runs masked GQA attention forward and backward
 * over the packed segments, and computes the action-token log-probs with the
 * clipped policy-ratio loss and its gradients.
 *
 * Conventions (all entry points):
 *  - "host" pointers are host memory; every other pointer is device memory on
 *    the current HIP device.  The caller owns all memory, including workspace;
 *    the library allocates no device memory.
 *  - Work is enqueued asynchronously on `stream`, except where a function says
 *    otherwise.  Arguments are validated on the host before any launch; on a
 *    non-OK status nothing has been enqueued unless the status is SEG_ERR_HIP.
 *  - No exception crosses the ABI.  A non-OK status leaves a thread-local
 *    message readable with seg_last_error().
 *  - Reductions run in a fixed order: repeated calls on the same inputs give
 *    bitwise-identical outputs.  Integer atomics are used only where their
 *    result does not depend on order.
 *  - Numeric kernels compute in bf16 with fp32 accumulation (MFMA).  SEG_F32
 *    inputs are rounded to bf16 (nearest-even) when loaded; outputs are written
 *    in the input dtype unless stated otherwise.
 */
#ifndef SEG_H
#define SEG_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SEG_OK = 0,
  SEG_ERR_ARG = 1,         /* invalid argument (null pointer, bad span, mismatched sizes) */
  SEG_ERR_CAPACITY = 2,    /* a turn does not fit max_seg_tokens / buffer_tokens, or int32 overflow */
  SEG_ERR_WORKSPACE = 3,   /* ws_bytes smaller than the required workspace */
  SEG_ERR_UNSUPPORTED = 4, /* shape the kernels do not support (head_dim, tile, head ratio) */
  SEG_ERR_HIP = 5          /* a HIP call failed; the message holds the HIP error string */
} seg_status;

typedef enum { SEG_BF16 = 0, SEG_F32 = 1 } seg_dtype;

/* Token kinds, stored in tok_meta = turn << 2 | kind (the prompt has turn 0). */
enum { SEG_KIND_PROMPT = 0, SEG_KIND_IMAGE = 1, SEG_KIND_TEXT = 2, SEG_KIND_PAD = 3 };
/* Tile classes stored in the CSR maps (skipped tiles are not stored). */
enum { SEG_TILE_PARTIAL = 1, SEG_TILE_FULL = 2 };
/* Fields of one seg_info record. */
enum {
  SEG_INFO_TRAJ = 0, SEG_INFO_FIRST_TURN = 1, SEG_INFO_END_TURN = 2, SEG_INFO_START = 3,
  SEG_INFO_LEN = 4, SEG_INFO_QTILE_BASE = 5, SEG_INFO_LOSS_BASE = 6, SEG_INFO_LOSS_COUNT = 7,
  SEG_INFO_FIELDS = 8
};

/*
 * A batch of trajectories (all arrays host memory, read during the call).
 * Turns of trajectory i are steps [step_offsets[i], step_offsets[i+1]), numbered
 * 1..T inside the trajectory.  prompt_len, img_len, text_len >= 0;
 * 0 <= action_len <= text_len.  A trajectory with no turns yields no segment.
 * A segment without tokens, or one whose first token is a trained token (no
 * row before it predicts it, Eq. (loss)), is an argument error.
 *
 * Segmentation (Sec. 3.3, App. D; the segment length L plays the removal
 * threshold Delta and W the kept-screenshot count K):
 *   - turns are cut into runs [a, b) of at most seg_steps turns, closed early
 *     when the next turn would push the segment past max_seg_tokens (0 = no cap);
 *   - segment [a, b) holds the prompt, then for every turn j < b its screenshot
 *     if j > a - W and its text (older screenshots are dropped, all text kept);
 *   - with buffer_tokens > 0 segments are packed in order into buffers of that
 *     many rows: a segment that does not fit the current buffer opens the next
 *     one, and the tail of a buffer is padding (tok_src = -1, kind PAD).
 * Visibility inside a segment: key k is visible to query q iff k is not after q
 * and k is not a screenshot token of a turn <= turn(q) - W.
 * tile: tile edge of the block-sparse map; 128 for the numeric kernels, any
 * value >= 1 for layout-only use.
 *
 * mode SEG_MODE_ANCHORED follows the App. D algorithm as printed, with
 * K = window screenshots kept and removal threshold Delta = seg_steps: the
 * screenshot count of the token stream is tracked turn by turn (observation
 * before response); when turn j's screenshot makes it exceed K + Delta the
 * stream is saved as a segment ending with turn j-1, the oldest Delta
 * screenshots are dropped and the re-tokenised history starts the next
 * segment at turn j.  So the first segment has K + Delta turns and later ones
 * Delta turns; segment [a, b) holds the screenshots of turns j >= a - K; every
 * token sees every earlier token of its segment (no window clause).
 * max_seg_tokens must be 0 in this mode.
 */
typedef enum { SEG_MODE_SLIDING = 0, SEG_MODE_ANCHORED = 1 } seg_mode;
#define SEG_WINDOW_ANCHORED (1 << 28)
typedef struct {
  int32_t num_traj;
  const int32_t *step_offsets; /* host [num_traj+1], step_offsets[0] = 0, non-decreasing */
  const int32_t *prompt_len;   /* host [num_traj] */
  const int32_t *img_len;      /* host [num_steps] screenshot tokens of each turn */
  const int32_t *text_len;     /* host [num_steps] non-image tokens of each turn */
  const int32_t *action_len;   /* host [num_steps] trained tokens = last action_len text tokens */
  int32_t window;              /* W >= 1: screenshots visible to a turn, its own included */
  int32_t seg_steps;           /* L >= 1: turns per segment (1 = step-wise decomposition) */
  int32_t max_seg_tokens;      /* 0 = no cap */
  int32_t buffer_tokens;       /* 0 = one contiguous packed buffer */
  int32_t tile;                /* >= 1 */
  int32_t mode;                /* seg_mode; 0 = sliding window (default) */
} seg_problem;

typedef struct {
  int32_t num_segments;
  int32_t num_buffers;
  int32_t loss_rows;      /* R: trained action tokens */
  int32_t num_qtiles;     /* tiles over all segments (q-tiles = k-tiles) */
  int32_t num_steps;
  int32_t max_seg_len;    /* rows of the longest segment */
  int64_t packed_tokens;  /* rows of the packed buffer, padding included */
  int64_t traj_tokens;    /* canonical tokens of the batch */
  int64_t tile_nnz_max;   /* lower-triangular tile count: bound on non-skipped tiles */
  size_t workspace_bytes; /* workspace needed by seg_build_layout */
} seg_sizes;

/*
 * Device arrays of a layout, sized from seg_sizes (S segments, P packed rows,
 * R loss rows, G q-tiles, Z = tile_nnz_max).  Filled by seg_build_layout, which
 * also sets the scalars `window` and `tile` and the launch schedule
 * (`xcd_rows`, `xcd_cols`) of the attention kernels.
 */
typedef struct {
  int32_t *seg_info;      /* [S*8] see SEG_INFO_*; turns are 1-based, segments in packed order */
  int32_t *tok_src;       /* [P] canonical token index (trajectory-major canonical order), -1 = pad */
  int32_t *tok_meta;      /* [P] turn << 2 | kind */
  int32_t *loss_pred_row; /* [R] packed row predicting the action token (its position - 1) */
  int32_t *loss_tgt_src;  /* [R] canonical index of the action token */
  int32_t *loss_traj;     /* [R] trajectory of the row (selects the advantage) */
  int32_t *tile_seg;      /* [G] segment of each tile */
  int32_t *qt_ptr;        /* [G+1] CSR over q-tiles: non-skipped k-tiles, ascending */
  int32_t *qt_col;        /* [Z] global tile index of the k-tile */
  uint8_t *qt_cls;        /* [Z] SEG_TILE_PARTIAL or SEG_TILE_FULL */
  int32_t *qt_ord;        /* [Z] the same entries per q-tile in the order the forward and dQ
                             kernels walk them: FULL k-tiles first, then PARTIAL ones (each
                             ascending); the global k-tile index, bit 31 set for PARTIAL */
  int32_t *kt_ptr;        /* [G+1] transposed CSR over k-tiles: non-skipped q-tiles, ascending */
  int32_t *kt_row;        /* [Z] */
  uint8_t *kt_cls;        /* [Z] */
  int32_t *kt_ord;        /* [Z] the same entries per k-tile in the order the dK/dV kernel walks
                             them: FULL q-tiles first, then PARTIAL ones (each descending); the
                             global q-tile index, bit 31 set for PARTIAL */
  int64_t *seg_pairs;     /* [S] exact visible (query, key) pairs of each segment */
  int64_t *tile_nnz;      /* [1] non-skipped tiles */
  int32_t window;         /* set by seg_build_layout: the visibility window the
                             attention kernels apply (W; SEG_WINDOW_ANCHORED,
                             larger than any turn index, in the anchored mode) */
  int32_t tile;           /* set by seg_build_layout */
  /* Set by seg_build_layout (host values): tile boundaries of the eight
   * ranges the attention kernels give to the chip's eight dies (XCDs, each
   * with its own L2), xcd_rows for the forward and dQ passes balanced by the
   * tiles' listed k-tiles, xcd_cols for the dK/dV pass balanced by their
   * listed q-tiles; [0] = 0, [8] = number of tiles, non-decreasing. */
  int32_t xcd_rows[9];
  int32_t xcd_cols[9];
} seg_layout;

/* Sizes of the layout of `p` (host only, no HIP call).  Errors: SEG_ERR_ARG for
 * invalid spans or parameters, SEG_ERR_CAPACITY when a single turn exceeds the
 * cap or the buffer, or a count overflows int32. */
seg_status seg_layout_query(const seg_problem *p, seg_sizes *out);

/* Build every array of `out` for `p` (Sec. 3.3 / App. D segmentation, the
 * sliding-window visibility and the tile map).  `sz` must be the result of
 * seg_layout_query(p); `ws` >= sz->workspace_bytes.  The segment table is
 * computed on the host and uploaded to `ws`; the call waits on `stream` once
 * after that small upload, then enqueues the token, loss-row and tile kernels. */
seg_status seg_build_layout(const seg_problem *p, const seg_sizes *sz, seg_layout *out,
                            void *ws, size_t ws_bytes, hipStream_t stream);

/* Workspace of seg_attn_fwd (bwd = 0: the largest key norm of each segment
 * and kv head, plus bf16 copies of fp32 inputs) or seg_attn_bwd (bwd = 1:
 * per-row -Delta and log2-sum-exp, plus bf16 copies of fp32 inputs). */
size_t seg_attn_workspace_bytes(const seg_sizes *sz, seg_dtype dt, int32_t hq, int32_t hkv,
                                int32_t d, int32_t bwd);

/*
 * Masked GQA attention forward over the packed segments (the attention of the
 * policy forward pass on VCS training items, Sec. 3.3).  Query head h reads
 * key/value head h / (hq / hkv).  Tiles classed as skipped are never touched;
 * partial tiles apply the visibility rule per element.
 *   q [P, hq, d], k/v [P, hkv, d] (dtype dt, row-major);
 *   o [P, hq, d] (dtype dt); lse [hq, P] fp32, natural-log sum of exp of the
 *   scaled scores of each row.  Padding rows of o and lse are not written.
 * Supported: d in {64, 128}, hq % hkv == 0, layout tile == 128.
 */
seg_status seg_attn_fwd(const seg_layout *L, const seg_sizes *sz, seg_dtype dt, int32_t hq,
                        int32_t hkv, int32_t d, float softmax_scale, const void *q,
                        const void *k, const void *v, void *o, float *lse, void *ws,
                        size_t ws_bytes, hipStream_t stream);

/*
 * Backward of seg_attn_fwd: given dO, the gradients of sum(O * dO) w.r.t. q, k
 * and v.  dk/dv of a kv head sum the contributions of all its query heads.
 * dq [P, hq, d], dk/dv [P, hkv, d] in dtype dt; padding rows are not written.
 * o and lse are the outputs of seg_attn_fwd on the same inputs.
 */
seg_status seg_attn_bwd(const seg_layout *L, const seg_sizes *sz, seg_dtype dt, int32_t hq,
                        int32_t hkv, int32_t d, float softmax_scale, const void *q,
                        const void *k, const void *v, const void *o, const float *lse,
                        const void *d_o, void *dq, void *dk, void *dv, void *ws,
                        size_t ws_bytes, hipStream_t stream);

/* Size of the fixed device scratch behind seg_attn_bwd_noalloc: 64 MiB. */
#define SEG_ATTN_BWD_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * seg_attn_bwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and kernels as
 * seg_attn_bwd; its workspace is a library-owned device array of
 * SEG_ATTN_BWD_SCRATCH_BYTES, one per GPU, held until the process ends
 * (its address on the current device is looked up once per device on the
 * first call there).  The call allocates nothing and needs
 * seg_attn_workspace_bytes(sz, dt, hq, hkv, d, 1) <= SEG_ATTN_BWD_SCRATCH_BYTES
 * (bf16: 8 * hq * packed_tokens bytes rounded up to 256, e.g. 28 heads x
 * 299,000 packed rows); a larger problem returns SEG_ERR_WORKSPACE before any
 * launch.  `stream` must belong to the current device.  Every call on a GPU
 * shares that GPU's scratch (nothing in it needs to start at zero: each call
 * writes what it reads), so calls that overlap on one GPU, on different
 * streams or from different threads, race and give wrong results: serialise
 * them.  Errors as seg_attn_bwd, plus SEG_ERR_HIP when the scratch address
 * cannot be obtained.
 */
seg_status seg_attn_bwd_noalloc(const seg_layout *L, const seg_sizes *sz, seg_dtype dt,
                                int32_t hq, int32_t hkv, int32_t d, float softmax_scale,
                                const void *q, const void *k, const void *v, const void *o,
                                const float *lse, const void *d_o, void *dq, void *dk, void *dv,
                                hipStream_t stream);

/*
 * Settings of the clipped policy-ratio objective with its KL penalty
 * (Eq. (loss), App. E): per row, rho = exp(logp - old_logp), A = adv[row_traj];
 * objective = min(rho A, clip(rho, 1 - eps_low, 1 + eps_high) A), and when
 * dual_clip_c > 0 and A < 0, objective = max(objective, dual_clip_c A);
 * kl = exp(ref_logp - logp) - (ref_logp - logp) - 1 (the per-token estimator
 * of KL(pi_theta || pi_ref) used by GRPO; the paper does not name one);
 * loss_tok = -objective + kl_coef * kl; loss_sum = loss_scale * sum(loss_tok).
 * Logits are logit_scale * h W^T.  Clipping uses strict inequalities.
 */
typedef struct {
  float eps_low;
  float eps_high;
  float dual_clip_c;  /* <= 0: off */
  float loss_scale;
  float logit_scale;
  int32_t want_grad;  /* 0: forward only (dh and dw untouched, may be NULL) */
  float kl_coef;      /* lambda >= 0 of the KL penalty; > 0 needs ref_logp */
} seg_loss_cfg;

size_t seg_logprob_workspace_bytes(int32_t rows, int32_t hidden, int32_t vocab, seg_dtype dt);

/*
 * Fused action-token log-prob, clipped-ratio loss with KL penalty, and
 * gradients (Eq. (loss), App. E).
 *   h [n_h, hidden] (dtype dt) hidden states; row_index [rows] selects the rows
 *   of h to use (e.g. loss_pred_row), or NULL to use rows 0..rows-1;
 *   w [vocab, hidden] (dtype dt) output projection; target [rows] token ids in
 *   [0, vocab); old_logp [rows] fp32 rollout log-probs; ref_logp [rows] fp32
 *   reference-policy log-probs, or NULL when cfg->kl_coef == 0 (else
 *   SEG_ERR_ARG); adv [num_traj] fp32; row_traj [rows] index into adv.
 * Outputs: logp, loss_tok [rows] fp32; clipped [rows] (1 where the clipped
 * branch of the ratio term is taken, so that term has no gradient); kl_tok
 * [rows] fp32 per-token KL estimate, or NULL; loss_sum [1] fp32;
 * with want_grad: dh [rows, hidden] (dtype dt) and dw [vocab, hidden] fp32
 * (overwritten), the gradients of loss_sum.  A forward-only call
 * (want_grad = 0) is the reference / old-policy log-prob pass.
 */
seg_status seg_logprob_loss(int32_t rows, int32_t hidden, int32_t vocab, seg_dtype dt,
                            const void *h, const int32_t *row_index, const void *w,
                            const int32_t *target, const float *old_logp,
                            const float *ref_logp, const float *adv, const int32_t *row_traj,
                            int32_t num_traj, const seg_loss_cfg *cfg, float *logp,
                            float *loss_tok, uint8_t *clipped, float *kl_tok, float *loss_sum,
                            void *dh, float *dw, void *ws, size_t ws_bytes,
                            hipStream_t stream);

/*
 * One decoder layer of the language model around the segmented attention
 * (the policy update trains the language model on VCS segments while the
 * vision encoder stays fixed, App. E RL stage, so the screenshot tokens enter
 * as given hidden states).  The paper does not spell the layer out; this is a
 * generic pre-norm Qwen-family layer (no projection biases, no per-head q/k
 * norm, one-dimensional positions), all matrices row-major, y = x W^T for a
 * weight W [out, in]:
 *   a = rms(x) * g1,  rms(x) = x / sqrt(mean(x^2) + rms_eps)
 *   q, k, v = a wq^T, a wk^T, a wv^T       ([P, hq, d], [P, hkv, d])
 *   q, k = rope(q), rope(k)                (rotate-half pairs (i, i + d/2) by
 *                                           pos * rope_base^(-2i/d); pos = the
 *                                           row inside its segment)
 *   o = seg_attn_fwd(q, k, v)              (scale 1/sqrt(d))
 *   y1 = x + o wo^T
 *   b = rms(y1) * g2
 *   y = y1 + (silu(b wg^T) * (b wu^T)) wd^T
 * bf16 storage, fp32 accumulation.  Padding rows: their outputs are
 * undefined and they contribute nothing to any gradient (dy there counts as
 * zero; dx there is 0).  Projections and the MLP run over chunks of
 * chunk_rows rows (0 = 65536; at most 2^20); weight gradients are summed over
 * the chunks in order, so results are bitwise reproducible.
 */
typedef struct {
  int32_t hidden;      /* H (multiple of 8) */
  int32_t inter;       /* I of the MLP (multiple of 8) */
  int32_t hq, hkv, d;  /* attention heads, as for seg_attn_fwd */
  float rms_eps;       /* > 0 */
  float rope_base;     /* > 1 */
  int32_t chunk_rows;  /* >= 0 */
} seg_layer_cfg;
typedef struct {       /* device, bf16: g1, g2 [H]; wq [hq*d, H]; wk, wv [hkv*d, H];
                          wo [H, hq*d]; wg, wu [I, H]; wd [H, I] */
  const void *g1, *wq, *wk, *wv, *wo, *g2, *wg, *wu, *wd;
} seg_layer_weights;
typedef struct {       /* device buffers written by seg_layer_fwd and read by seg_layer_bwd */
  void *q, *k, *v;     /* [P, hq, d], [P, hkv, d] bf16, after the rotary embedding */
  void *o;             /* [P, hq, d] bf16 (zero at padding rows) */
  float *lse;          /* [hq, P] */
  void *y1;            /* [P, H] bf16 */
  float *rstd1, *rstd2; /* [P] */
} seg_layer_saved;
typedef struct {       /* device fp32 gradients, same shapes as the weights; overwritten */
  float *g1, *wq, *wk, *wv, *wo, *g2, *wg, *wu, *wd;
} seg_layer_grads;

/* Workspace of seg_layer_fwd (bwd = 0) or seg_layer_bwd (bwd = 1). */
size_t seg_layer_workspace_bytes(const seg_sizes *sz, const seg_layer_cfg *cfg, int32_t bwd);

/* Layer forward: x [P, H] bf16 -> y [P, H] bf16 and the saved buffers.
 * Errors: SEG_ERR_ARG (null pointer, bad setting), SEG_ERR_UNSUPPORTED
 * (shape the attention or GEMM kernels do not take), SEG_ERR_WORKSPACE. */
seg_status seg_layer_fwd(const seg_layout *L, const seg_sizes *sz, const seg_layer_cfg *cfg,
                         const seg_layer_weights *w, const void *x, void *y,
                         const seg_layer_saved *saved, void *ws, size_t ws_bytes,
                         hipStream_t stream);

/* Layer backward: gradients of sum(y * dy) over the segment rows, given the
 * saved buffers of seg_layer_fwd on the same x and weights.  dx [P, H] bf16;
 * the weight gradients are written in fp32.  The MLP activations and the
 * normalised inputs are recomputed from x, y1 and the saved rstd values. */
seg_status seg_layer_bwd(const seg_layout *L, const seg_sizes *sz, const seg_layer_cfg *cfg,
                         const seg_layer_weights *w, const void *x, const seg_layer_saved *saved,
                         const void *dy, void *dx, const seg_layer_grads *g, void *ws,
                         size_t ws_bytes, hipStream_t stream);

/*
 * Kernel timing.  While enabled, every kernel the library launches is
 * bracketed by HIP events recorded on its launch stream.  seg_profile_read sums
 * the device time of all recorded launches of one kernel (names: "layout",
 * "attn_prep", "attn_fwd", "attn_delta" (fp32 inputs only: with bf16 inputs
 * the dQ kernel forms Delta itself), "attn_bwd_dkdv", "attn_bwd_dq", "logits", "row_loss", "dz", "lp_prep", "dh", "dw", and for the layer
 * "ly_norm", "ly_rope", "ly_proj", "ly_mlp", "ly_wgrad", "ly_misc"), waiting for them to
 * finish; seg_profile_reset forgets the records.  Timing adds two event
 * records per launch and is off by default.  These three calls are the one
 * place with process-wide state (an atomic enable flag and a mutex-guarded
 * record list shared by all threads and devices); with timing off a launch
 * only reads the flag.
 */
void seg_profile_enable(int32_t on);
void seg_profile_reset(void);
seg_status seg_profile_read(const char *name, double *total_ms, int64_t *launches);

/* Message of the last non-OK status on the calling thread ("" if none). */
const char *seg_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SEG_H */
