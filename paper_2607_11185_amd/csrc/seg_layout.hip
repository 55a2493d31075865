// Segmentation and packed layout of Visual Context Segmentation training items
// (Sec. 3.3; App. D, Alg. "Sliding-window trajectory processing with token-ID
// stream"), read with a sliding window of W screenshots and L-turn segments.
//
// Host part (seg_layout_query and the first half of seg_build_layout): cut each
// trajectory's turns into segments and pack them; this is O(turns) arithmetic on
// the span lists.  Device part: expand the per-segment span table into per-token
// descriptors, the loss rows, and the 128x128 block-sparse tile map with its
// transposed CSR and the exact visible-pair count of every segment.
#include <algorithm>
#include <climits>
#include <cstring>
#include <string>
#include <vector>

#include "common.h"

namespace seg {

static thread_local std::string g_err;
void set_error(const std::string &m) { g_err = m; }
void clear_error() { g_err.clear(); }

namespace {

// One contiguous run of tokens of a segment (a prompt, screenshot or text block).
struct Piece {
  int32_t off;    // segment-relative position of its first token
  int32_t canon;  // canonical index of its first token
  int32_t len;
  int32_t meta;   // turn << 2 | kind
};

// A run of trained action tokens (the tail of one turn's text block).
struct LossPiece {
  int32_t row_base;  // first loss row
  int32_t pos;       // packed row of the first action token
  int32_t canon;     // canonical index of the first action token
  int32_t traj;
};

// Per-segment record used by the kernels (device copy lives in the workspace).
struct DevSeg {
  int32_t start, len, qbase, nt;
  int32_t piece_base, piece_count, pad0, pad1;
  int64_t tri_base;  // offset of the segment's lower-triangular class matrix
};

struct Plan {
  seg_sizes sz{};
  std::vector<int32_t> seg_info;  // [S*8]
  std::vector<DevSeg> dsegs;
  std::vector<Piece> pieces;
  std::vector<LossPiece> lpieces;
  int32_t max_nt = 0;
  // launch schedule of the attention kernels (see seg_layout)
  std::vector<int32_t> row_work, col_work;  // [G] listed k-tiles / q-tiles of each tile
  int32_t xcd_rows[9] = {}, xcd_cols[9] = {};
};

// Listed partners of every tile of one segment, from its token runs.  Turns
// never decrease along a segment, so a q-tile's most permissive row is its
// first one; a k-tile's most permissive key is the one that expires last
// (text and prompt never do, a screenshot of turn s at turn s + Wv).  An
// off-diagonal pair (q-tile i > k-tile j) holds a visible pair iff the first
// row's turn of i is below the latest expiry in j, so k-tile j is listed by the
// contiguous q-tiles j .. r_j - 1 (the diagonal always).
void tile_work(const Piece *pc, int npc, int len, int tile, int Wv, int32_t *row_w,
               int32_t *col_w) {
  const int n = (len + tile - 1) / tile;
  std::vector<int64_t> first_turn(n), last_exp(n, INT64_MIN);
  int k = 0;
  for (int t = 0; t < n; ++t) {
    const int r0 = t * tile, r1 = std::min(len, r0 + tile);
    while (k + 1 < npc && pc[k + 1].off <= r0) ++k;
    first_turn[t] = pc[k].meta >> 2;
    for (int i = k; i < npc && pc[i].off < r1; ++i) {
      if (pc[i].len == 0 || pc[i].off + pc[i].len <= r0) continue;
      const int kind = pc[i].meta & 3;
      const int64_t e = kind == SEG_KIND_IMAGE ? (int64_t)(pc[i].meta >> 2) + Wv : INT64_MAX;
      last_exp[t] = std::max(last_exp[t], e);
    }
  }
  std::vector<int32_t> diff(n + 1, 0);
  for (int j = 0; j < n; ++j) {
    // first q-tile after j whose first row's turn has reached the expiry
    const int r = (int)(std::lower_bound(first_turn.begin() + j + 1, first_turn.end(), last_exp[j]) -
                        first_turn.begin());
    col_w[j] = r - j;
    diff[j + 1] += 1;
    diff[r] -= 1;
  }
  int run = 0;
  for (int i = 0; i < n; ++i) {
    run += diff[i];
    row_w[i] = 1 + run;
  }
}

// Boundaries of eight consecutive tile ranges with about equal total work.
void balance8(const std::vector<int32_t> &w, int32_t *b) {
  const int G = (int)w.size();
  std::vector<int64_t> pre(G + 1, 0);
  for (int g = 0; g < G; ++g) pre[g + 1] = pre[g] + w[g];
  b[0] = 0;
  for (int x = 1; x < 8; ++x) {
    const int64_t target = (pre[G] * x + 7) / 8;
    b[x] = (int32_t)(std::lower_bound(pre.begin(), pre.end(), target) - pre.begin());
    b[x] = std::max(b[x], b[x - 1]);
  }
  b[8] = G;
}

// Byte offsets of the build workspace regions.
struct BuildWs {
  size_t dseg, piece, lpiece, cls, qcnt, kcnt, total;
};

BuildWs build_ws_layout(const seg_sizes &sz, size_t npieces, size_t nlpieces) {
  BuildWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  w.dseg = take(sizeof(DevSeg) * std::max<int64_t>(1, sz.num_segments));
  w.piece = take(sizeof(Piece) * std::max<size_t>(1, npieces));
  w.lpiece = take(sizeof(LossPiece) * std::max<size_t>(1, nlpieces));
  w.cls = take(std::max<int64_t>(1, sz.tile_nnz_max));
  w.qcnt = take(sizeof(int32_t) * (size_t)std::max<int64_t>(1, sz.num_qtiles));
  w.kcnt = take(sizeof(int32_t) * (size_t)std::max<int64_t>(1, sz.num_qtiles));
  w.total = off;
  return w;
}

// Tokens of segment [a, b) of a trajectory: prompt + text of turns < b +
// screenshots of turns j with max(1, a - W + 1) <= j < b (turns 1-based).
int64_t seg_len(const int32_t *img, const int32_t *text, int64_t p, int W, int a, int b) {
  int64_t n = p;
  int lo = std::max(1, a - W + 1);
  for (int j = 1; j < b; ++j) {
    n += text[j - 1];
    if (j >= lo) n += img[j - 1];
  }
  return n;
}

void validate(const seg_problem *p) {
  SEG_CHECK(p != nullptr, SEG_ERR_ARG, "problem is NULL");
  SEG_CHECK(p->num_traj >= 0, SEG_ERR_ARG, "num_traj < 0");
  SEG_CHECK(p->window >= 1, SEG_ERR_ARG, "window must be >= 1 (got %d)", p->window);
  SEG_CHECK(p->seg_steps >= 1, SEG_ERR_ARG, "seg_steps must be >= 1 (got %d)", p->seg_steps);
  SEG_CHECK(p->max_seg_tokens >= 0, SEG_ERR_ARG, "max_seg_tokens < 0");
  SEG_CHECK(p->buffer_tokens >= 0, SEG_ERR_ARG, "buffer_tokens < 0");
  SEG_CHECK(p->tile >= 1, SEG_ERR_ARG, "tile must be >= 1 (got %d)", p->tile);
  SEG_CHECK(p->mode == SEG_MODE_SLIDING || p->mode == SEG_MODE_ANCHORED, SEG_ERR_ARG,
            "unknown mode %d", p->mode);
  SEG_CHECK(p->mode == SEG_MODE_SLIDING || p->max_seg_tokens == 0, SEG_ERR_UNSUPPORTED,
            "the anchored mode has no token cap (max_seg_tokens must be 0)");
  SEG_CHECK(p->mode == SEG_MODE_SLIDING || p->window < (SEG_WINDOW_ANCHORED >> 1), SEG_ERR_ARG,
            "window too large");
  if (p->num_traj == 0) return;
  SEG_CHECK(p->step_offsets && p->prompt_len, SEG_ERR_ARG, "step_offsets/prompt_len is NULL");
  SEG_CHECK(p->step_offsets[0] == 0, SEG_ERR_ARG, "step_offsets[0] must be 0");
  for (int t = 0; t < p->num_traj; ++t) {
    SEG_CHECK(p->step_offsets[t + 1] >= p->step_offsets[t], SEG_ERR_ARG,
              "step_offsets must be non-decreasing (trajectory %d)", t);
    SEG_CHECK(p->prompt_len[t] >= 0, SEG_ERR_ARG, "prompt_len[%d] < 0", t);
  }
  int32_t ns = p->step_offsets[p->num_traj];
  if (ns > 0)
    SEG_CHECK(p->img_len && p->text_len && p->action_len, SEG_ERR_ARG,
              "img_len/text_len/action_len is NULL");
  for (int s = 0; s < ns; ++s) {
    SEG_CHECK(p->img_len[s] >= 0, SEG_ERR_ARG, "img_len[%d] < 0", s);
    SEG_CHECK(p->text_len[s] >= 0, SEG_ERR_ARG, "text_len[%d] < 0", s);
    SEG_CHECK(p->action_len[s] >= 0 && p->action_len[s] <= p->text_len[s], SEG_ERR_ARG,
              "action_len[%d] must be in [0, text_len]", s);
  }
}

Plan make_plan(const seg_problem *p) {
  validate(p);
  Plan pl;
  seg_sizes &sz = pl.sz;
  // Anchored mode: a segment keeps the K = window screenshots before its
  // first turn (K + 1 with its own), the first segment runs K + Delta turns
  // and later ones Delta = seg_steps (the count of the algorithm's trigger).
  const bool anchored = p->mode == SEG_MODE_ANCHORED;
  const int W = anchored ? p->window + 1 : p->window, L = p->seg_steps, tile = p->tile;
  const int L0 = anchored ? p->window + p->seg_steps : L;  // turns of a trajectory's first segment
  const int64_t cap = p->max_seg_tokens, B = p->buffer_tokens;
  sz.num_steps = p->num_traj ? p->step_offsets[p->num_traj] : 0;

  struct S0 {
    int traj, a, b;
    int64_t len;
  };
  std::vector<S0> segs;
  std::vector<int64_t> canon0(p->num_traj + 1, 0);
  for (int t = 0; t < p->num_traj; ++t) {
    const int s0 = p->step_offsets[t], T = p->step_offsets[t + 1] - s0;
    const int32_t *img = p->img_len + s0, *text = p->text_len + s0;
    const int64_t pr = p->prompt_len[t];
    int64_t tot = pr;
    for (int j = 0; j < T; ++j) tot += (int64_t)img[j] + text[j];
    canon0[t + 1] = canon0[t] + tot;
    int a = 1;
    while (a <= T) {
      int64_t one = seg_len(img, text, pr, W, a, a + 1);
      SEG_CHECK(!cap || one <= cap, SEG_ERR_CAPACITY,
                "trajectory %d turn %d alone needs %lld tokens > max_seg_tokens %lld", t, a,
                (long long)one, (long long)cap);
      int b = a + 1;
      const int La = a == 1 ? L0 : L;
      while (b - a < La && b <= T && (!cap || seg_len(img, text, pr, W, a, b + 1) <= cap)) ++b;
      int64_t n = seg_len(img, text, pr, W, a, b);
      SEG_CHECK(n >= 1, SEG_ERR_ARG, "segment of trajectory %d, turns %d..%d holds no token", t, a,
                b - 1);
      SEG_CHECK(!B || n <= B, SEG_ERR_CAPACITY,
                "segment of %lld tokens (trajectory %d, turns %d..%d) exceeds buffer_tokens %lld",
                (long long)n, t, a, b - 1, (long long)B);
      segs.push_back({t, a, b, n});
      a = b;
    }
  }
  sz.traj_tokens = canon0[p->num_traj];
  SEG_CHECK(sz.traj_tokens <= INT32_MAX, SEG_ERR_CAPACITY, "more than 2^31-1 canonical tokens");
  SEG_CHECK(segs.size() <= (size_t)INT32_MAX / SEG_INFO_FIELDS, SEG_ERR_CAPACITY, "too many segments");

  // packing
  int64_t pos = 0, fill = 0;
  int nbuf = 0;
  std::vector<int64_t> starts(segs.size());
  for (size_t i = 0; i < segs.size(); ++i) {
    if (B) {
      if (nbuf == 0 || fill + segs[i].len > B) {
        pos = (int64_t)nbuf * B;
        ++nbuf;
        fill = 0;
      }
      fill += segs[i].len;
    }
    starts[i] = pos;
    pos += segs[i].len;
  }
  int64_t packed = B ? (int64_t)nbuf * B : pos;
  if (!B) nbuf = segs.empty() ? 0 : 1;
  SEG_CHECK(packed <= INT32_MAX, SEG_ERR_CAPACITY, "packed buffer exceeds 2^31-1 rows");
  sz.packed_tokens = packed;
  sz.num_buffers = nbuf;
  sz.num_segments = (int32_t)segs.size();
  sz.max_seg_len = 0;
  for (const S0 &sg : segs) sz.max_seg_len = std::max(sz.max_seg_len, (int32_t)sg.len);

  // per-segment tables
  int64_t qbase = 0, tri = 0, rows = 0;
  for (size_t i = 0; i < segs.size(); ++i) {
    const S0 &sg = segs[i];
    const int s0 = p->step_offsets[sg.traj];
    const int32_t *img = p->img_len + s0, *text = p->text_len + s0, *act = p->action_len + s0;
    const int64_t nt = (sg.len + tile - 1) / tile;
    DevSeg d{};
    d.start = (int32_t)starts[i];
    d.len = (int32_t)sg.len;
    d.qbase = (int32_t)qbase;
    d.nt = (int32_t)nt;
    d.piece_base = (int32_t)pl.pieces.size();
    d.tri_base = tri;
    // pieces: prompt, then per turn j < b: screenshot if j > a - W, text
    int32_t off = 0, c = (int32_t)canon0[sg.traj];
    int32_t pr = p->prompt_len[sg.traj];
    pl.pieces.push_back({off, c, pr, SEG_KIND_PROMPT});
    off += pr;
    c += pr;
    int64_t loss_base = rows;
    for (int j = 1; j < sg.b; ++j) {
      int32_t m = img[j - 1], x = text[j - 1];
      if (j > sg.a - W && m > 0) {
        pl.pieces.push_back({off, c, m, (j << 2) | SEG_KIND_IMAGE});
        off += m;
      }
      c += m;
      if (x > 0) {
        if (j >= sg.a && act[j - 1] > 0) {
          int32_t na = act[j - 1];
          // the ratio of a token uses the row before it (Eq. loss): a trained
          // token cannot open its segment
          SEG_CHECK(off + x - na > 0, SEG_ERR_ARG,
                    "trajectory %d turn %d: a trained token is the first token of its segment "
                    "(no row predicts it)", sg.traj, j);
          pl.lpieces.push_back({(int32_t)rows, d.start + off + x - na, c + x - na, sg.traj});
          rows += na;
        }
        pl.pieces.push_back({off, c, x, (j << 2) | SEG_KIND_TEXT});
        off += x;
      }
      c += x;
    }
    d.piece_count = (int32_t)pl.pieces.size() - d.piece_base;
    pl.dsegs.push_back(d);
    int32_t info[SEG_INFO_FIELDS] = {sg.traj, sg.a, sg.b, d.start, d.len, d.qbase,
                                     (int32_t)loss_base, (int32_t)(rows - loss_base)};
    pl.seg_info.insert(pl.seg_info.end(), info, info + SEG_INFO_FIELDS);
    pl.max_nt = std::max<int32_t>(pl.max_nt, (int32_t)nt);
    qbase += nt;
    tri += nt * (nt + 1) / 2;
    SEG_CHECK(qbase <= INT32_MAX && tri <= INT32_MAX && rows <= INT32_MAX, SEG_ERR_CAPACITY,
              "tile or loss-row count exceeds 2^31-1");
  }
  sz.num_qtiles = (int32_t)qbase;
  sz.tile_nnz_max = tri;
  // launch schedule: per-tile work and eight balanced tile ranges per pass
  {
    const int Wv = anchored ? SEG_WINDOW_ANCHORED : p->window;
    const int G = (int)qbase;
    pl.row_work.assign(G, 0);
    pl.col_work.assign(G, 0);
    for (const DevSeg &d : pl.dsegs)
      tile_work(pl.pieces.data() + d.piece_base, d.piece_count, d.len, tile, Wv,
                pl.row_work.data() + d.qbase, pl.col_work.data() + d.qbase);
    balance8(pl.row_work, pl.xcd_rows);
    balance8(pl.col_work, pl.xcd_cols);
  }
  sz.loss_rows = (int32_t)rows;
  sz.workspace_bytes = build_ws_layout(sz, pl.pieces.size(), pl.lpieces.size()).total;
  return pl;
}

// ------------------------------------------------------------------ kernels

// last index i in [0, n) with key(i) <= x (keys ascending); -1 if none
template <class F>
__device__ __forceinline__ int upper_index(int n, int x, F key) {
  int lo = 0, hi = n;  // answer in [lo-1, hi-1]
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (key(mid) <= x) lo = mid + 1;
    else hi = mid;
  }
  return lo - 1;
}

__global__ void k_tokens(const DevSeg *__restrict__ segs, int nseg, const Piece *__restrict__ pieces,
                         int32_t *__restrict__ tok_src, int32_t *__restrict__ tok_meta, int packed) {
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < packed; r += gridDim.x * blockDim.x) {
    int s = upper_index(nseg, r, [&](int i) { return segs[i].start; });
    int src = -1, meta = SEG_KIND_PAD;
    if (s >= 0 && r < segs[s].start + segs[s].len) {
      const DevSeg d = segs[s];
      int pos = r - d.start;
      const Piece *pc = pieces + d.piece_base;
      int i = upper_index(d.piece_count, pos, [&](int k) { return pc[k].off; });
      src = pc[i].canon + (pos - pc[i].off);
      meta = pc[i].meta;
    }
    tok_src[r] = src;
    tok_meta[r] = meta;
  }
}

__global__ void k_loss_rows(const LossPiece *__restrict__ lp, int nlp, int rows,
                            int32_t *__restrict__ pred, int32_t *__restrict__ tgt,
                            int32_t *__restrict__ traj) {
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < rows; r += gridDim.x * blockDim.x) {
    int i = upper_index(nlp, r, [&](int k) { return lp[k].row_base; });
    int o = r - lp[i].row_base;
    pred[r] = lp[i].pos + o - 1;
    tgt[r] = lp[i].canon + o;
    traj[r] = lp[i].traj;
  }
}

__global__ void k_tile_seg(const DevSeg *__restrict__ segs, int nseg, int ntiles,
                           int32_t *__restrict__ tile_seg) {
  for (int g = blockIdx.x * blockDim.x + threadIdx.x; g < ntiles; g += gridDim.x * blockDim.x)
    tile_seg[g] = upper_index(nseg, g, [&](int i) { return segs[i].qbase; });
}

__device__ __forceinline__ int wave_sum_int(int v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ long long wave_sum_ll(long long v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Classify every lower-triangular tile (i, j <= i) of q-tile g's segment.
// Visibility of key k to query q (segment-relative rows): k <= q and
// turn(q) < kexp(k), where kexp = turn(k) + W for screenshot tokens and
// "never expires" otherwise.  Turns never decrease along a segment, so for a
// key the most favourable query of a row range is the first one not before it.
__global__ void __launch_bounds__(256) k_classify(
    const DevSeg *__restrict__ segs, const int32_t *__restrict__ tile_seg,
    const int32_t *__restrict__ tok_meta, int W, int tile, uint8_t *__restrict__ cls,
    int32_t *__restrict__ qcnt, int32_t *__restrict__ kcnt, int64_t *__restrict__ seg_pairs) {
  const int g = blockIdx.x;
  const int s = tile_seg[g];
  const DevSeg d = segs[s];
  const int i = g - d.qbase;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t *meta = tok_meta + d.start;
  const int q_lo = i * tile, q_hi = min(d.len, (i + 1) * tile) - 1;
  const int step_qhi = meta[q_hi] >> 2;
  uint8_t *row_cls = cls + d.tri_base + (int64_t)i * (i + 1) / 2;
  long long pairs = 0;
  int nnz = 0;
  for (int j = wave; j <= i; j += 4) {
    const int k_lo = j * tile, k_hi = min(d.len, (j + 1) * tile) - 1;
    bool any = false, all = true;
    long long cnt = 0;
    for (int k = k_lo + lane; k <= k_hi; k += 64) {
      const int mk = meta[k];
      const int kexp = ((mk & 3) == SEG_KIND_IMAGE) ? (mk >> 2) + W : INT_MAX;
      const int qs = max(k, q_lo);
      if (qs <= q_hi && (meta[qs] >> 2) < kexp) {
        any = true;
        // last row in [qs, q_hi] whose turn is < kexp
        int lo = qs, hi = q_hi;
        if (kexp != INT_MAX && (step_qhi >= kexp)) {
          while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if ((meta[mid] >> 2) < kexp) lo = mid;
            else hi = mid - 1;
          }
        } else {
          lo = q_hi;
        }
        cnt += lo - qs + 1;
      }
      // every row of the tile sees key k: k <= q_lo (causal; a 1x1 diagonal
      // tile is full) and the last row's turn is before the key's expiry
      if (!(k <= q_lo && step_qhi < kexp)) all = false;
    }
    const bool t_any = __any(any);
    const bool t_all = __all(all) && (q_hi - q_lo + 1 == tile) && (k_hi - k_lo + 1 == tile);
    const long long t_cnt = wave_sum_ll(cnt);
    if (lane == 0) {
      uint8_t c = t_any ? (t_all ? SEG_TILE_FULL : SEG_TILE_PARTIAL) : 0;
      row_cls[j] = c;
      if (c) {
        atomicAdd(&kcnt[d.qbase + j], 1);
        ++nnz;
      }
      pairs += t_cnt;
    }
  }
  __shared__ long long sp[4];
  __shared__ int sn[4];
  if (lane == 0) {
    sp[wave] = pairs;
    sn[wave] = nnz;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    qcnt[g] = sn[0] + sn[1] + sn[2] + sn[3];
    long long t = sp[0] + sp[1] + sp[2] + sp[3];
    atomicAdd((unsigned long long *)&seg_pairs[s], (unsigned long long)t);
  }
}

// Exclusive scan of n counts into ptr[0..n] (one block of 1024 threads).
__global__ void __launch_bounds__(1024) k_scan(const int32_t *__restrict__ cnt, int n,
                                               int32_t *__restrict__ ptr,
                                               int64_t *__restrict__ total) {
  __shared__ int part[1024];
  const int t = threadIdx.x;
  const int per = (n + 1023) / 1024;
  const int b = min(n, t * per), e = min(n, b + per);
  int sum = 0;
  for (int i = b; i < e; ++i) sum += cnt[i];
  part[t] = sum;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    int v = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int run = part[t] - sum;
  for (int i = b; i < e; ++i) {
    ptr[i] = run;
    run += cnt[i];
  }
  if (t == 1023) {
    ptr[n] = part[1023];
    if (total) *total = part[1023];
  }
}

// CSR rows: one wave per q-tile, k-tiles ascending.
__global__ void __launch_bounds__(64) k_fill_rows(const DevSeg *__restrict__ segs,
                                                  const int32_t *__restrict__ tile_seg,
                                                  const uint8_t *__restrict__ cls,
                                                  const int32_t *__restrict__ ptr,
                                                  int32_t *__restrict__ col,
                                                  uint8_t *__restrict__ ccls,
                                                  int32_t *__restrict__ ord) {
  const int g = blockIdx.x, lane = threadIdx.x;
  const DevSeg d = segs[tile_seg[g]];
  const int i = g - d.qbase;
  const uint8_t *row = cls + d.tri_base + (int64_t)i * (i + 1) / 2;
  int out = ptr[g];
  for (int j0 = 0; j0 <= i; j0 += 64) {
    const int j = j0 + lane;
    const uint8_t c = j <= i ? row[j] : 0;
    const unsigned long long m = __ballot(c != 0);
    if (c) {
      const int r = __popcll(m & ((1ull << lane) - 1));
      col[out + r] = d.qbase + j;
      ccls[out + r] = c;
    }
    out += __popcll(m);
  }
  // The walking order of the q-tile-stationary kernels: the same entries,
  // FULL tiles first and PARTIAL ones after (each ascending), with bit 31
  // marking PARTIAL.
  out = ptr[g];
  for (int pass = 0; pass < 2; ++pass) {
    const uint8_t want = pass == 0 ? SEG_TILE_FULL : SEG_TILE_PARTIAL;
    for (int j0 = 0; j0 <= i; j0 += 64) {
      const int j = j0 + lane;
      const uint8_t c = j <= i ? row[j] : 0;
      const unsigned long long m = __ballot(c == want);
      if (c == want) {
        const int r = __popcll(m & ((1ull << lane) - 1));
        ord[out + r] = (int32_t)((unsigned)(d.qbase + j) | (pass ? 0x80000000u : 0u));
      }
      out += __popcll(m);
    }
  }
}

// Transposed CSR columns: one wave per k-tile, q-tiles ascending.
__global__ void __launch_bounds__(64) k_fill_cols(const DevSeg *__restrict__ segs,
                                                  const int32_t *__restrict__ tile_seg,
                                                  const uint8_t *__restrict__ cls,
                                                  const int32_t *__restrict__ ptr,
                                                  int32_t *__restrict__ rowi,
                                                  uint8_t *__restrict__ ccls,
                                                  int32_t *__restrict__ ord) {
  const int g = blockIdx.x, lane = threadIdx.x;
  const DevSeg d = segs[tile_seg[g]];
  const int j = g - d.qbase;
  const int e0 = ptr[g];
  int out = e0, nfull = 0;
  for (int i0 = j; i0 < d.nt; i0 += 64) {
    const int i = i0 + lane;
    const uint8_t c = i < d.nt ? cls[d.tri_base + (int64_t)i * (i + 1) / 2 + j] : 0;
    const unsigned long long m = __ballot(c != 0);
    if (c) {
      const int r = __popcll(m & ((1ull << lane) - 1));
      rowi[out + r] = d.qbase + i;
      ccls[out + r] = c;
    }
    out += __popcll(m);
    nfull += __popcll(__ballot(c == SEG_TILE_FULL));
  }
  // The walking order of the k-tile-stationary kernel: FULL q-tiles first,
  // then PARTIAL ones, each descending, with bit 31 marking PARTIAL.
  int rf = 0, rp = 0;  // ascending ranks so far within each class
  for (int i0 = j; i0 < d.nt; i0 += 64) {
    const int i = i0 + lane;
    const uint8_t c = i < d.nt ? cls[d.tri_base + (int64_t)i * (i + 1) / 2 + j] : 0;
    const unsigned long long mf = __ballot(c == SEG_TILE_FULL);
    const unsigned long long mp = __ballot(c == SEG_TILE_PARTIAL);
    const unsigned long long below = (1ull << lane) - 1;
    if (c == SEG_TILE_FULL) ord[e0 + nfull - 1 - (rf + __popcll(mf & below))] = d.qbase + i;
    if (c == SEG_TILE_PARTIAL)
      ord[out - 1 - (rp + __popcll(mp & below))] =
          (int32_t)((unsigned)(d.qbase + i) | 0x80000000u);
    rf += __popcll(mf);
    rp += __popcll(mp);
  }
}

int grid_for(int64_t n, int block = 256) {
  int64_t g = (n + block - 1) / block;
  return (int)std::max<int64_t>(1, std::min<int64_t>(g, 65536));
}

}  // namespace
}  // namespace seg

using namespace seg;

extern "C" const char *seg_last_error(void) { return g_err.c_str(); }

extern "C" seg_status seg_layout_query(const seg_problem *p, seg_sizes *out) {
  return guarded([&] {
    SEG_CHECK(out != nullptr, SEG_ERR_ARG, "sizes output is NULL");
    Plan pl = make_plan(p);
    *out = pl.sz;
  });
}

extern "C" seg_status seg_build_layout(const seg_problem *p, const seg_sizes *sz, seg_layout *out,
                                       void *ws, size_t ws_bytes, hipStream_t stream) {
  return guarded([&] {
    SEG_CHECK(sz != nullptr && out != nullptr, SEG_ERR_ARG, "sizes or layout is NULL");
    Plan pl = make_plan(p);
    SEG_CHECK(std::memcmp(&pl.sz, sz, sizeof(seg_sizes)) == 0, SEG_ERR_ARG,
              "sizes do not match seg_layout_query of this problem");
    SEG_CHECK(ws_bytes >= sz->workspace_bytes, SEG_ERR_WORKSPACE,
              "workspace of %zu bytes < required %zu", ws_bytes, sz->workspace_bytes);
    // visibility window of the kernels: none inside an anchored segment
    const int Wv = p->mode == SEG_MODE_ANCHORED ? SEG_WINDOW_ANCHORED : p->window;
    out->window = Wv;
    out->tile = p->tile;
    std::memcpy(out->xcd_rows, pl.xcd_rows, sizeof(pl.xcd_rows));
    std::memcpy(out->xcd_cols, pl.xcd_cols, sizeof(pl.xcd_cols));
    const int S = sz->num_segments, G = sz->num_qtiles, R = sz->loss_rows;
    const int P = (int)sz->packed_tokens;
    if (S > 0) {
      SEG_CHECK(ws && out->seg_info && out->tok_src && out->tok_meta && out->tile_seg &&
                    out->qt_ptr && out->qt_col && out->qt_cls && out->qt_ord && out->kt_ptr &&
                    out->kt_row && out->kt_ord &&
                    out->kt_cls && out->seg_pairs && out->tile_nnz,
                SEG_ERR_ARG, "a layout array is NULL");
      SEG_CHECK(R == 0 || (out->loss_pred_row && out->loss_tgt_src && out->loss_traj),
                SEG_ERR_ARG, "a loss-row array is NULL");
    }
    if (S == 0) {
      if (P > 0 || out->tile_nnz) {
        // nothing to compute; still define the scalar outputs
      }
      if (out->qt_ptr) SEG_HIP(hipMemsetAsync(out->qt_ptr, 0, sizeof(int32_t), stream));
      if (out->kt_ptr) SEG_HIP(hipMemsetAsync(out->kt_ptr, 0, sizeof(int32_t), stream));
      if (out->tile_nnz) SEG_HIP(hipMemsetAsync(out->tile_nnz, 0, sizeof(int64_t), stream));
      if (P > 0 && out->tok_src) {
        SEG_HIP(hipMemsetAsync(out->tok_src, 0xff, sizeof(int32_t) * P, stream));
      }
      return;
    }
    BuildWs w = build_ws_layout(*sz, pl.pieces.size(), pl.lpieces.size());
    char *base = static_cast<char *>(ws);
    DevSeg *d_segs = reinterpret_cast<DevSeg *>(base + w.dseg);
    Piece *d_pieces = reinterpret_cast<Piece *>(base + w.piece);
    LossPiece *d_lp = reinterpret_cast<LossPiece *>(base + w.lpiece);
    uint8_t *d_cls = reinterpret_cast<uint8_t *>(base + w.cls);
    int32_t *d_qcnt = reinterpret_cast<int32_t *>(base + w.qcnt);
    int32_t *d_kcnt = reinterpret_cast<int32_t *>(base + w.kcnt);

    SEG_HIP(hipMemcpyAsync(out->seg_info, pl.seg_info.data(), sizeof(int32_t) * pl.seg_info.size(),
                           hipMemcpyHostToDevice, stream));
    SEG_HIP(hipMemcpyAsync(d_segs, pl.dsegs.data(), sizeof(DevSeg) * pl.dsegs.size(),
                           hipMemcpyHostToDevice, stream));
    SEG_HIP(hipMemcpyAsync(d_pieces, pl.pieces.data(), sizeof(Piece) * pl.pieces.size(),
                           hipMemcpyHostToDevice, stream));
    if (!pl.lpieces.empty())
      SEG_HIP(hipMemcpyAsync(d_lp, pl.lpieces.data(), sizeof(LossPiece) * pl.lpieces.size(),
                             hipMemcpyHostToDevice, stream));
    // the host tables are locals of this call: wait until they have been read
    SEG_HIP(hipStreamSynchronize(stream));

    ProfScope prof("layout", stream);
    SEG_HIP(hipMemsetAsync(d_kcnt, 0, sizeof(int32_t) * G, stream));
    SEG_HIP(hipMemsetAsync(out->seg_pairs, 0, sizeof(int64_t) * S, stream));
    if (P > 0) {
      k_tokens<<<grid_for(P), 256, 0, stream>>>(d_segs, S, d_pieces, out->tok_src, out->tok_meta, P);
      SEG_LAUNCH_CHECK();
    }
    if (R > 0) {
      k_loss_rows<<<grid_for(R), 256, 0, stream>>>(d_lp, (int)pl.lpieces.size(), R,
                                                   out->loss_pred_row, out->loss_tgt_src,
                                                   out->loss_traj);
      SEG_LAUNCH_CHECK();
    }
    k_tile_seg<<<grid_for(G), 256, 0, stream>>>(d_segs, S, G, out->tile_seg);
    SEG_LAUNCH_CHECK();
    k_classify<<<G, 256, 0, stream>>>(d_segs, out->tile_seg, out->tok_meta, Wv, p->tile,
                                      d_cls, d_qcnt, d_kcnt, out->seg_pairs);
    SEG_LAUNCH_CHECK();
    k_scan<<<1, 1024, 0, stream>>>(d_qcnt, G, out->qt_ptr, out->tile_nnz);
    SEG_LAUNCH_CHECK();
    k_scan<<<1, 1024, 0, stream>>>(d_kcnt, G, out->kt_ptr, nullptr);
    SEG_LAUNCH_CHECK();
    k_fill_rows<<<G, 64, 0, stream>>>(d_segs, out->tile_seg, d_cls, out->qt_ptr, out->qt_col,
                                      out->qt_cls, out->qt_ord);
    SEG_LAUNCH_CHECK();
    k_fill_cols<<<G, 64, 0, stream>>>(d_segs, out->tile_seg, d_cls, out->kt_ptr, out->kt_row,
                                      out->kt_cls, out->kt_ord);
    SEG_LAUNCH_CHECK();
  });
}
