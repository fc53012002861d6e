// Host runtime of the draft-and-verify step: argument and state validation,
// workspace planning, slot state machine and kernel sequencing on one stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/osprey.h"
#include "internal.h"

#define OSPREY_API extern "C" __attribute__((visibility("default")))

namespace {

using namespace osp;

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return OSPREY_OK;
}

#define HIP_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess) return fail(OSPREY_E_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr int kMaxSplit = 64;
constexpr int kMaxSplitLen = 4096;
constexpr int kEvenSplitLen = 2048;   // longer splits unbalance ragged batches
constexpr int kVerifyChunk = 4096;
// A single sequence's pass of at most this many rows prepares its queries in the
// attention blocks (no separate row kernel).
constexpr int kOwnPrepRows = 8;

enum SlotState { S_EMPTY = 0, S_READY = 1, S_DRAFTED = 2, S_VERIFIED = 3 };

struct SlotHost {
  int state = S_EMPTY;
  long len_max = 0;   // upper bound of the device-side cached length (exact unless pending)
  int nblocks = 0;
  int drafted_k = 0;  // K of the last draft (bounds the next pending ingest)
};

// Device workspace carve-up.
struct Ws {
  int32_t* t2d;
  float* rope_cos;
  float* rope_sin;
  int32_t* slot_len;
  int32_t* pend_n;
  int32_t* pend_tok;
  int32_t* block_table;
  int32_t* slot_nblocks;
  uint32_t* err;
  int32_t *ing_seq, *ing_pos, *ing_tok, *ing_tap, *n_rows, *cu, *last_row, *committed, *bslot;
  int32_t *ar_pos, *ar_tok;
  int32_t *attn_items, *attn_n_items;   // attention work list of the current step
  float *x, *s, *gfb, *qkv, *o, *h;
  uint16_t *s_hi, *s_lo, *xa_hi, *xa_lo;   // matrix-core path inputs (bf16 hi / lo)
  float* attn_part;
  float* split;
  float* split_s;     // K-split partials of passes of at most kLmMaxRows rows
  float* split_s2;    // a second such buffer (the down projection reads gate/up partials)
  float* logits;
  float* lm_part;
  QStat* qstat;       // drafter row statistics of the last chain, [B][Km]
  int32_t* drafts;
  float* u_zero;
  float* v_part;
  double* v_res;
  double* v_sub;
  int32_t* vstate;
  double* vstat;
  int32_t* tree_removed;
  // draft-tree growth
  void* tree_kv;              // [B * kMaxTreeProc][n_layers][2][nkv][hd], cache dtype
  float* tree_cv;             // [B * kMaxTopk][kTkBlocks][kMaxTopk]
  int32_t* tree_cr;
  int32_t *c_tok, *c_par, *c_depth, *c_slot, *n_cand, *front;   // [B][kMaxCand] / [B] / [B][kMaxTopk]
  double* c_score;
  int32_t *r_tok, *r_pos, *r_attpos, *r_node, *r_anc;  // [B * kMaxTopk] (r_anc x kMaxTreeDepth)
  int32_t* r_cu;                                       // [B + 1]
  // block drafting: the block rows [B * Km] (the anchor's row + k) and temperatures
  int32_t* b_gather;
  float* b_temp;
  float* r_s;                 // [B * kMaxTopk][d]
  float* ones;                // [B * kMaxTopk] temperature 1 for the tree's LM-head records
  void* head_pk;              // bf16 drafters: the LM head in the matrix cores' order
};

struct Dims {
  int B, Km, Rmax, max_blocks, qkv_rows, nchunk_t, nchunk_d, lm_nblk_max;
};

Dims dims_of(const osprey_config& c) {
  Dims d;
  d.B = c.max_batch;
  d.Km = std::max(c.max_k, 1);
  d.Rmax = std::max(c.max_new_rows, c.max_batch * (c.max_k + 1));
  d.max_blocks = (c.max_seq_len + c.kv_block - 1) / c.kv_block;
  d.qkv_rows = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  d.nchunk_t = (c.vocab_target + kVerifyChunk - 1) / kVerifyChunk;
  d.nchunk_d = (c.vocab_draft + kVerifyChunk - 1) / kVerifyChunk;
  d.lm_nblk_max = kGemvMaxWaves;
  return d;
}

// Lays out the workspace; with base == nullptr only returns the size.
size_t plan(const osprey_config& c, char* base, Ws* w) {
  const Dims D = dims_of(c);
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    off = (off + 255) & ~size_t(255);
    char* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  };
  Ws t{};
  Ws& W = w ? *w : t;
  const long d = c.d_model, hd = c.head_dim, nq = c.n_q_heads;
  W.t2d = (int32_t*)take(4L * c.vocab_target);
  W.rope_cos = (float*)take(4L * c.max_seq_len * (hd / 2));
  W.rope_sin = (float*)take(4L * c.max_seq_len * (hd / 2));
  W.slot_len = (int32_t*)take(4L * D.B);
  W.pend_n = (int32_t*)take(4L * D.B);
  W.pend_tok = (int32_t*)take(4L * D.B * (c.max_k + 1));
  W.block_table = (int32_t*)take(4L * D.B * D.max_blocks);
  W.slot_nblocks = (int32_t*)take(4L * D.B);
  W.err = (uint32_t*)take(16);
  W.ing_seq = (int32_t*)take(4L * D.Rmax);
  W.ing_pos = (int32_t*)take(4L * D.Rmax);
  W.ing_tok = (int32_t*)take(4L * D.Rmax);
  W.ing_tap = (int32_t*)take(4L * D.Rmax);
  W.n_rows = (int32_t*)take(4);
  W.cu = (int32_t*)take(4L * (D.B + 1));
  W.last_row = (int32_t*)take(4L * D.B);
  W.committed = (int32_t*)take(4L * D.B);
  W.bslot = (int32_t*)take(4L * D.B);
  W.ar_pos = (int32_t*)take(4L * D.B);
  W.ar_tok = (int32_t*)take(4L * D.B);
  W.attn_items = (int32_t*)take(4L * D.B * kMaxSplit);
  W.attn_n_items = (int32_t*)take(4);
  W.x = (float*)take(4L * D.Rmax * d);
  W.s = (float*)take(4L * D.Rmax * d);
  W.gfb = (float*)take(4L * D.B * d);
  W.qkv = (float*)take(4L * D.Rmax * D.qkv_rows);
  W.o = (float*)take(4L * D.Rmax * nq * hd);
  W.h = (float*)take(4L * D.Rmax * c.d_ffn);
  {
    const long wa = std::max<long>(std::max<long>(d, nq * hd), c.d_ffn);
    W.s_hi = (uint16_t*)take(2L * D.Rmax * d);
    W.s_lo = (uint16_t*)take(2L * D.Rmax * d);
    W.xa_hi = (uint16_t*)take(2L * D.Rmax * wa);
    W.xa_lo = (uint16_t*)take(2L * D.Rmax * wa);
  }
  W.attn_part = (float*)take(4L * D.Rmax * nq * kMaxSplit * (hd + 2));
  {
    const long nmax = std::max<long>(std::max<long>(D.qkv_rows, 2L * c.d_ffn), d);
    W.split = (float*)take(4L * kMaxKSplit * D.Rmax * nmax);
    const long rs = kLmMaxRows;
    const long tap_w = (long)c.n_taps * c.target_hidden;
    long need = skinny_splits(rs, (int)tap_w) * d;
    need = std::max<long>(need, skinny_splits(rs, 2 * c.d_model) * (long)D.qkv_rows);
    need = std::max<long>(need, skinny_splits(rs, c.n_q_heads * c.head_dim) * d);
    need = std::max<long>(need, skinny_splits(rs, c.d_model) * 2L * c.d_ffn);
    need = std::max<long>(need, skinny_splits(rs, c.d_ffn) * d);
    W.split_s = (float*)take(4L * rs * need);
    W.split_s2 = (float*)take(4L * rs * need);
  }
  W.logits = (float*)take(4L * D.B * D.Km * c.vocab_draft);
  // (draft trees: B x k rows; blocks: B x K rows)
  W.lm_part = (float*)take(16L * D.B * std::max<long>(kMaxTopk, D.Km) * D.lm_nblk_max);
  W.qstat = (QStat*)take(sizeof(QStat) * D.B * D.Km);
  W.drafts = (int32_t*)take(4L * D.B * D.Km);
  W.u_zero = (float*)take(4L * D.B * D.Km);
  // chain rows ((Km + 1) target and Km drafter rows) or a draft tree's kMaxTreeNodes + 1 rows
  W.v_part = (float*)take(16L * D.B * std::max<long>((D.Km + 1) * D.nchunk_t + D.Km * D.nchunk_d,
                                                     (kMaxTreeNodes + 1L) * D.nchunk_t));
  W.tree_removed = (int32_t*)take(4L * D.B * kMaxTreeNodes);
  {
    const long el = c.dtype == OSPREY_BF16 ? 2 : 4;
    const long rows = (long)D.B * kMaxTopk;
    W.tree_kv = take(el * D.B * kMaxTreeProc * c.n_layers * 2 * c.n_kv_heads * c.head_dim);
    W.tree_cv = (float*)take(4L * rows * kTkBlocks * kMaxTopk);
    W.tree_cr = (int32_t*)take(4L * rows * kTkBlocks * kMaxTopk);
    W.c_tok = (int32_t*)take(4L * D.B * kMaxCand);
    W.c_par = (int32_t*)take(4L * D.B * kMaxCand);
    W.c_depth = (int32_t*)take(4L * D.B * kMaxCand);
    W.c_slot = (int32_t*)take(4L * D.B * kMaxCand);
    W.c_score = (double*)take(8L * D.B * kMaxCand);
    W.n_cand = (int32_t*)take(4L * D.B);
    W.front = (int32_t*)take(4L * D.B * kMaxTopk);
    W.r_tok = (int32_t*)take(4L * rows);
    W.r_pos = (int32_t*)take(4L * rows);
    W.r_attpos = (int32_t*)take(4L * rows);
    W.r_node = (int32_t*)take(4L * rows);
    W.r_cu = (int32_t*)take(4L * (D.B + 1));
    W.r_anc = (int32_t*)take(4L * rows * kMaxTreeDepth);
    W.r_s = (float*)take(4L * rows * d);
    W.ones = (float*)take(4L * rows);
  }
  {
    const long rows = (long)D.B * D.Km;
    W.b_gather = (int32_t*)take(4L * rows);
    W.b_temp = (float*)take(4L * rows);
  }
  W.head_pk = c.dtype == OSPREY_BF16 ? take(packed_head_bytes(c.vocab_draft, c.d_model)) : nullptr;
  W.v_res = (double*)take(16L * D.B * D.nchunk_t);
  W.v_sub = (double*)take(16L * kVSub * D.B * D.nchunk_t);
  W.vstate = (int32_t*)take(16L * D.B);
  W.vstat = (double*)take(32L * D.B);
  return (off + 255) & ~size_t(255);
}

int validate(const osprey_config* c) {
  if (!c) return fail(OSPREY_E_INVALID, "config is NULL");
  if (c->n_layers < 1 || c->n_layers > 64) return fail(OSPREY_E_INVALID, "n_layers %d not in [1, 64]", c->n_layers);
  if (c->d_model < 64 || c->d_model % 64) return fail(OSPREY_E_SHAPE, "d_model %d must be a positive multiple of 64", c->d_model);
  if (c->d_model > 4096) return fail(OSPREY_E_UNSUPPORTED, "d_model %d > 4096", c->d_model);
  // (the batch-1 LM head normalises its row in the kernel: checked here, before any call)
  if (!lm_head_norm_in_supported(1, c->d_model))
    return fail(OSPREY_E_UNSUPPORTED, "d_model %d: the batch-1 LM head cannot normalise its row", c->d_model);
  if (c->d_ffn < 64 || c->d_ffn % 64) return fail(OSPREY_E_SHAPE, "d_ffn %d must be a positive multiple of 64", c->d_ffn);
  if (c->n_q_heads < 1 || c->n_kv_heads < 1 || c->n_q_heads % c->n_kv_heads)
    return fail(OSPREY_E_SHAPE, "n_kv_heads %d must divide n_q_heads %d", c->n_kv_heads, c->n_q_heads);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(OSPREY_E_UNSUPPORTED, "head_dim %d (supported: 64, 128)", c->head_dim);
  if (c->vocab_draft < 1 || c->vocab_target < 1) return fail(OSPREY_E_SHAPE, "vocabularies must be non-empty");
  if (c->target_hidden < 8 || c->target_hidden % 8) return fail(OSPREY_E_SHAPE, "target_hidden %d must be a positive multiple of 8", c->target_hidden);
  if (c->n_taps < 1 || c->n_taps > 16) return fail(OSPREY_E_SHAPE, "n_taps %d not in [1, 16]", c->n_taps);
  // weight matrices are read through 32-bit byte offsets: each must stay under 1 GiB
  {
    const long qkv = (long)(c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim;
    const long mats[] = {(long)c->vocab_draft * c->d_model, (long)c->d_model * c->n_taps * c->target_hidden,
                         qkv * 2 * c->d_model, (long)c->d_model * c->n_q_heads * c->head_dim,
                         (long)c->d_ffn * c->d_model};
    for (long m : mats)
      if (m * 4 > 0x7fffffffL) return fail(OSPREY_E_UNSUPPORTED, "a weight matrix of %ld values is over 1 GiB in bf16", m);
  }
  if (c->dtype != OSPREY_F32 && c->dtype != OSPREY_BF16) return fail(OSPREY_E_INVALID, "dtype %d", c->dtype);
  if (c->qk_norm != 0 && c->qk_norm != 1) return fail(OSPREY_E_INVALID, "qk_norm must be 0 or 1");
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 1.f)) return fail(OSPREY_E_INVALID, "rms_eps must be > 0 and rope_theta > 1");
  if (c->max_batch < 1 || c->max_batch > kMaxBatch) return fail(OSPREY_E_INVALID, "max_batch %d not in [1, %d]", c->max_batch, kMaxBatch);
  if (c->max_k < 0 || c->max_k > 64) return fail(OSPREY_E_INVALID, "max_k %d not in [0, 64]", c->max_k);
  if (c->max_seq_len < 1) return fail(OSPREY_E_INVALID, "max_seq_len %d", c->max_seq_len);
  if (c->max_seq_len > kMaxSplit * kMaxSplitLen)
    return fail(OSPREY_E_UNSUPPORTED, "max_seq_len %d > %d", c->max_seq_len, kMaxSplit * kMaxSplitLen);
  if (c->kv_block != 16) return fail(OSPREY_E_UNSUPPORTED, "kv_block %d (supported: 16)", c->kv_block);
  if (c->kv_num_blocks < 1) return fail(OSPREY_E_INVALID, "kv_num_blocks %d", c->kv_num_blocks);
  if (c->max_new_rows < 1) return fail(OSPREY_E_INVALID, "max_new_rows %d", c->max_new_rows);
  const long tap_w = (long)c->n_taps * c->target_hidden;
  if (tap_w > (1 << 24)) return fail(OSPREY_E_SHAPE, "tap width too large");
  return ok();
}

}  // namespace

namespace osp {
int report_error(int code, const char* msg) {
  g_err = msg ? msg : "";
  return code;
}
}  // namespace osp

namespace {

struct TimerRec {
  int family;
  hipEvent_t a, b;
  int reps;   // launches between the two events
};

// A timed LM head is launched this many times back to back between its two events
// (it is idempotent: the same logits and records again), so that the events' own
// dispatch overhead is shared by as many launches.
constexpr int kTimedRepeats = 8;

}  // namespace

struct osprey_handle {
  osprey_config cfg;
  Dims D;
  int n_cu = 1;         // compute units of the device (grid of the LM head)
  osprey_weights w;
  std::vector<osprey_layer_weights> layers;
  void* kv;
  Ws W;
  hipStream_t stream;
  std::vector<SlotHost> slots;
  // the last draft_step, for the stateful verify
  int last_B = 0, last_K = 0;
  std::vector<int> last_slots;
  float* last_logits = nullptr;
  long last_ld_b = 0;
  // graph capture: attention splits are planned for contexts up to this bound (0: the
  // call's own contexts), so that replays of a captured iteration stay covered
  long ctx_plan = 0;
  // timing: bit f of `timing` enables event timing of family f
  int timing = 0;
  std::vector<TimerRec> timers;
  std::vector<hipEvent_t> free_events;

  hipEvent_t ev() {
    if (!free_events.empty()) {
      hipEvent_t e = free_events.back();
      free_events.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  int t_begin(int family) {
    if (!(timing >> family & 1)) return -1;
    TimerRec r{family, ev(), ev(), 1};
    if (!r.a || !r.b) return -1;
    hipEventRecord(r.a, stream);
    timers.push_back(r);
    return (int)timers.size() - 1;
  }
  void t_end(int i, int reps = 1) {
    if (i < 0) return;
    timers[i].reps = reps;
    hipEventRecord(timers[i].b, stream);
  }
};

namespace {

int check_handle(osprey_handle* h) {
  if (!h) return fail(OSPREY_E_INVALID, "handle is NULL");
  return OSPREY_OK;
}

int check_slot(osprey_handle* h, int slot) {
  if (slot < 0 || slot >= h->cfg.max_batch) return fail(OSPREY_E_INVALID, "slot %d not in [0, %d)", slot, h->cfg.max_batch);
  return OSPREY_OK;
}

int hip_last() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(OSPREY_E_DEVICE, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

// Context splits of the attention: fixed-length pieces (a multiple of one page).
// Every block pays a fixed start-up (query staging, page-table and first page
// latency) and end (wavefront merge, partial write), so splits are as long as
// possible while the grid still holds the target number of working blocks (below),
// but not beyond kEvenSplitLen tokens, so that sequences of very different
// lengths still split into blocks of about equal work; no sequence needs more than
// kMaxSplit of them, and a split is at most kMaxSplitLen tokens (64 pages per
// wavefront of the attention kernel).
constexpr long kKvStreamBytes = 160L << 20;   // pages of a pass over every layer
struct SplitPlan {
  int n_split, split_len;
  bool kv_stream;   // the context's pages over every layer outsize the last-level cache
};
SplitPlan plan_splits(const osprey_handle* h, long ctx_max, long ctx_total, int max_split = kMaxSplit,
                      int min_len = 64) {
  // as many blocks as can be resident (two per CU: the kernel's register and LDS
  // budget), the most pages in flight; splits of at most kEvenSplitLen keep the blocks
  // of ragged batches of about equal work
  const long target_blocks = 2L * h->n_cu;
  long len = (ctx_total * h->cfg.n_kv_heads + target_blocks - 1) / target_blocks;
  len = std::min<long>(std::max<long>(len, min_len), kEvenSplitLen);
  len = std::max<long>(len, (ctx_max + max_split - 1) / max_split);
  len = std::min<long>(len, kMaxSplitLen);
  len = (len + 15) / 16 * 16;
  SplitPlan p;
  p.split_len = (int)len;
  p.n_split = (int)std::max<long>(1, (ctx_max + len - 1) / len);
  // Pages that cannot stay in the 256 MB last-level cache from one pass to the next are
  // read non-temporally (faster, and the weights stay cached); a smaller context is
  // read again by every draft step and keeps plain loads.
  const long el = h->cfg.dtype == OSPREY_BF16 ? 2 : 4;
  p.kv_stream = ctx_total * h->cfg.n_layers * h->cfg.n_kv_heads * h->cfg.head_dim * 2 * el > kKvStreamBytes;
  return p;
}

// Attention over the cache and the merge of its context splits.  Timed (family 1),
// the pair runs kTimedRepeats times back to back between the events: it is idempotent
// (a new row's keys and values are written again with the same values, every output is
// overwritten), so the events' own overhead is shared by as many launches.
void run_attention(osprey_handle* h, const AttnArgs& a, bool merge = true) {
  const int t = h->t_begin(1);
  const int reps = t >= 0 ? kTimedRepeats : 1;
  for (int rep = 0; rep < reps; ++rep) {
    launch_attention(h->cfg.dtype, a, h->stream);
    if (merge) launch_attn_combine(a, h->stream);
  }
  h->t_end(t, reps);
}

// One forward pass of the body over `rows`; `s` holds the conditioning rows.  `pick`
// (a single sequence's draft step): layer 0 draws the step's token itself.
void run_body(osprey_handle* h, const RowMeta& rows, const int32_t* cu, int B, const float* s,
              bool from_embed, const SplitPlan& sp, int rows_per_seq, int slot0,
              const PickArgs* pick = nullptr) {
  const osprey_config& c = h->cfg;
  const Ws& W = h->W;
  const int d = c.d_model, hd = c.head_dim, nq = c.n_q_heads, nkv = c.n_kv_heads;
  const int qkv_w = h->D.qkv_rows;
  for (int l = 0; l < c.n_layers; ++l) {
    const osprey_layer_weights& L = h->layers[l];
    // expanded QKV over [s ; RMSNorm(x)] (Eq. 2-3)
    GemvArgs g{};
    g.max_rows = rows.max_rows;
    g.count = rows.count;
    g.xin = W.x;
    g.ldx = d;
    g.s = s;
    g.lds = d;
    if (l == 0 && from_embed) {
      g.embed = h->w.embed;
      g.tok = rows.tok;
      g.vocab_embed = c.vocab_target;
      g.x_out = W.x;
    }
    g.gamma = L.in_norm;
    g.eps = c.rms_eps;
    g.d_norm = d;
    g.Kd = 2 * d;
    g.w0 = L.w_qkv;
    g.N = qkv_w;
    g.y = W.qkv;
    g.ldy = qkv_w;
    g.split_buf = W.split;
    int t = h->t_begin(4);
    if (l == 0 && pick) {
      g.pick = *pick;
      launch_gemv_qkv_pick(g, h->stream);
    } else {
      launch_gemv(c.dtype, SRC_QKV, EPI_STORE, g, h->stream);
    }
    h->t_end(t);
    // QK-norm + RoPE + KV append, attention, split combine
    AttnArgs a{};
    a.rows = rows;
    a.cu = cu;
    a.bslot = W.bslot;
    a.slot0 = B == 1 ? slot0 : -1;
    a.B = B;
    a.rows_per_seq = rows_per_seq;
    a.qkv = W.qkv;
    a.qkv_w = qkv_w;
    a.q_norm = L.q_norm;
    a.k_norm = L.k_norm;
    a.qk_norm = c.qk_norm;
    a.eps = c.rms_eps;
    a.rope_cos = W.rope_cos;
    a.rope_sin = W.rope_sin;
    a.max_seq = c.max_seq_len;
    a.kv = h->kv;
    a.layer = l;
    a.n_layers = c.n_layers;
    a.block_table = W.block_table;
    a.slot_nblocks = W.slot_nblocks;
    a.max_blocks = h->D.max_blocks;
    a.kv_block = c.kv_block;
    a.nq = nq;
    a.nkv = nkv;
    a.hd = hd;
    a.scale = 1.0f / std::sqrt((float)hd);
    a.n_split = sp.n_split;
    a.split_len = sp.split_len;
    a.kv_stream = sp.kv_stream;
    // the longest-first work list only matters for several sequences
    a.items = B == 1 ? nullptr : W.attn_items;
    a.n_items = B == 1 ? nullptr : W.attn_n_items;
    a.part = W.attn_part;
    a.o = W.o;
    a.err = W.err;
    // A single row's O projection merges the context splits while it stages its input
    // (one launch fewer per layer); otherwise the merge kernel writes o.
    const bool merge_in_o = gemv_attn_supported(c.dtype, rows.max_rows, nq * hd, hd, sp.n_split);
    run_attention(h, a, !merge_in_o);
    // O projection + residual
    GemvArgs go{};
    go.max_rows = rows.max_rows;
    go.count = rows.count;
    go.xin = W.o;
    go.ldx = nq * hd;
    go.Kd = nq * hd;
    go.w0 = L.w_o;
    go.N = d;
    go.y = W.x;
    go.ldy = d;
    go.split_buf = W.split;
    if (merge_in_o) {
      go.attn_part = W.attn_part;
      go.attn_pos = rows.pos;
      go.attn_nsplit = sp.n_split;
      go.attn_split_len = sp.split_len;
      go.attn_hd = hd;
      launch_gemv_attn_resid(go, h->stream);
    } else {
      launch_gemv(c.dtype, SRC_PLAIN, EPI_RESID, go, h->stream);
    }
    // post-attention RMSNorm + gate/up + SwiGLU
    GemvArgs gu{};
    gu.max_rows = rows.max_rows;
    gu.count = rows.count;
    gu.xin = W.x;
    gu.ldx = d;
    gu.gamma = L.post_norm;
    gu.eps = c.rms_eps;
    gu.d_norm = d;
    gu.Kd = d;
    gu.w0 = L.w_gate;
    gu.w1 = L.w_up;
    gu.N = c.d_ffn;
    gu.y = W.h;
    gu.ldy = c.d_ffn;
    gu.split_buf = W.split;
    launch_gemv(c.dtype, SRC_NORM, EPI_SWIGLU, gu, h->stream);
    // down projection + residual
    GemvArgs gd{};
    gd.max_rows = rows.max_rows;
    gd.count = rows.count;
    gd.xin = W.h;
    gd.ldx = c.d_ffn;
    gd.Kd = c.d_ffn;
    gd.w0 = L.w_down;
    gd.N = d;
    gd.y = W.x;
    gd.ldy = d;
    gd.split_buf = W.split;
    launch_gemv(c.dtype, SRC_PLAIN, EPI_RESID, gd, h->stream);
  }
}

// The same pass on the matrix-core path (bf16 weights, two or more rows).  Row
// kernels close every product (split-K sums in fixed order, residual, norms,
// SwiGLU) and write the next product's input as bf16 hi / lo pairs; the last one
// leaves RMSNorm_final(x) for the LM head.  `s_src` holds the conditioning rows,
// or is null when they are the tap projection's `ks_taps` partial sums.
// A draft-tree pass: the rows are frontier nodes, one per (sequence, branch).
struct TreePass {
  const int32_t* node;      // [rows] tree-cache slot
  const int32_t* anc;       // [rows][kMaxTreeDepth] ancestors' slots, then the node's
  const int32_t* pos;       // [rows] the node's position (RoPE)
  const int32_t* bslot;     // [B] each sequence's cache slot (its committed context)
};

void run_body_mr(osprey_handle* h, const RowMeta& rows, const int32_t* cu, int B, const float* s_src,
                 int ks_taps, const SplitPlan& sp, int rows_per_seq, int slot0,
                 const TreePass* tree = nullptr, const PickArgs* pick = nullptr) {
  const osprey_config& c = h->cfg;
  const Ws& W = h->W;
  // passes of at most kLmMaxRows rows stream the weights once with the inputs
  // resident in LDS; larger passes take the tiled GEMM
  const bool skinny = rows.max_rows <= kLmMaxRows;
  float* part = skinny ? W.split_s : W.split;
  auto gemm = [&](SrcKind src, EpiKind epi, GemvArgs& g) -> int {
    g.split_buf = part;
    return skinny ? launch_skinny(src, g, h->stream) : launch_gemm(src, epi, g, h->stream);
  };
  const int d = c.d_model, hd = c.head_dim, nq = c.n_q_heads, nkv = c.n_kv_heads, F = c.d_ffn;
  const int qkv_w = h->D.qkv_rows;
  RowArgs ra{};
  ra.max_rows = rows.max_rows;
  ra.count = rows.count;
  ra.part = part;
  ra.x = W.x;
  ra.eps = c.rms_eps;
  ra.out_hi = W.xa_hi;
  ra.out_lo = W.xa_lo;
  {
    RowArgs p = ra;
    p.W = d;
    p.ks = ks_taps;
    p.ldp = d;
    p.gamma = h->layers[0].in_norm;
    p.s_src = s_src;
    p.s_hi = W.s_hi;
    p.s_lo = W.s_lo;
    p.embed = h->w.embed;
    p.tok = rows.tok;
    p.vocab_embed = c.vocab_target;
    if (pick) p.pick = *pick;   // each row draws its own token (autoregressive rows only)
    launch_rows_prep(p, h->stream);
  }
  GemvArgs gb{};
  gb.max_rows = rows.max_rows;
  gb.count = rows.count;
  gb.xa_hi = W.xa_hi;
  gb.xa_lo = W.xa_lo;
  for (int l = 0; l < c.n_layers; ++l) {
    const osprey_layer_weights& L = h->layers[l];
    // expanded QKV over [s ; RMSNorm(x)] (Eq. 2-3)
    GemvArgs g = gb;
    g.xs_hi = W.s_hi;
    g.xs_lo = W.s_lo;
    g.ld_xs = d;
    g.seg = d;
    g.ld_xa = d;
    g.Kd = 2 * d;
    g.w0 = L.w_qkv;
    g.N = qkv_w;
    int t = h->t_begin(4);
    const int ks_qkv = gemm(SRC_PREP, EPI_STORE, g);
    h->t_end(t);
    // QK-norm + RoPE + KV append, attention (sums the QKV splits), split combine
    AttnArgs a{};
    a.rows = rows;
    a.cu = cu;
    a.bslot = tree ? tree->bslot : W.bslot;
    a.slot0 = (B == 1 && !tree) ? slot0 : -1;
    a.B = B;
    a.rows_per_seq = rows_per_seq;
    a.qkv = part;
    a.qkv_w = qkv_w;
    a.qkv_ks = ks_qkv;
    a.qkv_split = (long)rows.max_rows * qkv_w;
    a.q_norm = L.q_norm;
    a.k_norm = L.k_norm;
    a.qk_norm = c.qk_norm;
    a.eps = c.rms_eps;
    a.rope_cos = W.rope_cos;
    a.rope_sin = W.rope_sin;
    a.max_seq = c.max_seq_len;
    a.kv = h->kv;
    a.layer = l;
    a.n_layers = c.n_layers;
    a.block_table = W.block_table;
    a.slot_nblocks = W.slot_nblocks;
    a.max_blocks = h->D.max_blocks;
    a.kv_block = c.kv_block;
    a.nq = nq;
    a.nkv = nkv;
    a.hd = hd;
    a.scale = 1.0f / std::sqrt((float)hd);
    a.n_split = sp.n_split;
    a.split_len = sp.split_len;
    a.kv_stream = sp.kv_stream;
    // the longest-first work list only matters for several sequences (it lists the
    // step's sequences, not a tree pass's branches)
    a.items = (B == 1 || tree) ? nullptr : W.attn_items;
    a.n_items = (B == 1 || tree) ? nullptr : W.attn_n_items;
    if (tree) {
      a.tree_node = tree->node;
      a.tree_anc = tree->anc;
      a.tree_pos = tree->pos;
      a.tree_kv = W.tree_kv;
      a.tree_slots = h->D.B * kMaxTreeProc;
    }
    a.part = W.attn_part;
    a.o = W.o;
    a.o_hi = W.xa_hi;
    a.o_lo = W.xa_lo;
    a.err = W.err;
    // Several rows per sequence: one row kernel prepares q (norm, RoPE, scale) and
    // appends k / v once, instead of every split block of the sequence doing it.  One
    // row per sequence (draft steps), or a few rows of a single sequence (the ingest at
    // batch 1): the attention blocks sum the QKV partials and prepare their own queries,
    // one launch fewer per layer.
    const bool own_prep = rows_per_seq == 1 || (B == 1 && rows_per_seq <= kOwnPrepRows);
    if (!own_prep || tree) {
      launch_rows_qkv(c.dtype, a, W.o, h->stream);
      a.q_prep = W.o;
    }
    // Passes that are not tree passes and have at most kAttnMergeMaxSplit splits merge
    // the context splits while the O projection stages its inputs (one launch fewer per
    // layer); otherwise the merge kernel writes o as the projection's input pairs.  (At
    // 32-64 rows each O block reads its inputs' bytes once per split: with 1024-position
    // splits c4 / c5 gained nothing, with 2048 (at most 3-5 splits) c5 3.168 -> 3.151 ms.)
    const bool merge_in_o = skinny && !tree && sp.n_split <= kAttnMergeMaxSplit;
    run_attention(h, a, !merge_in_o);
    // O projection; residual + post-attention RMSNorm
    GemvArgs go = gb;
    go.ld_xa = nq * hd;
    go.Kd = nq * hd;
    go.w0 = L.w_o;
    go.N = d;
    RowArgs rn = ra;
    rn.W = d;
    rn.ldp = d;
    if (merge_in_o) {
      go.attn_part = W.attn_part;
      go.attn_pos = rows.pos;
      go.attn_nsplit = sp.n_split;
      go.attn_split_len = sp.split_len;
      go.attn_hd = hd;
      rn.ks = gemm(SRC_ATTN, EPI_STORE, go);
    } else {
      rn.ks = gemm(SRC_PREP, EPI_STORE, go);
    }
    rn.gamma = L.post_norm;
    launch_rows_resid_norm(rn, h->stream);
    // gate/up, SwiGLU
    GemvArgs gu = gb;
    gu.ld_xa = d;
    gu.Kd = d;
    gu.w0 = L.w_gate;
    gu.w1 = L.w_up;
    gu.N = F;
    RowArgs rs = ra;
    rs.W = F;
    rs.ldp = 2 * F;
    rs.ks = gemm(SRC_PREP, EPI_SWIGLU, gu);
    // down projection; residual + the next layer's input norm (final norm after the last).
    // Passes of up to 16 rows form silu(gate) * up while staging the down projection's
    // inputs (each block re-reads the gate/up partials of its K range, which only stays
    // cheaper than a separate row kernel for few rows).
    GemvArgs gd = gb;
    gd.ld_xa = F;
    gd.Kd = F;
    gd.w0 = L.w_down;
    gd.N = d;
    RowArgs rd = ra;
    rd.W = d;
    rd.ldp = d;
    if (skinny && rows.max_rows <= 16) {
      gd.part_in = part;
      gd.ks_in = rs.ks;
      gd.part_in_split = (long)rows.max_rows * 2 * F;
      gd.ld_in = 2 * F;
      gd.split_buf = W.split_s2;
      rd.part = W.split_s2;
      rd.ks = launch_skinny(SRC_SWIGLU, gd, h->stream);
    } else {
      launch_rows_swiglu(rs, h->stream);
      rd.ks = gemm(SRC_PREP, EPI_STORE, gd);
      rd.part = part;
    }
    rd.gamma = l + 1 < c.n_layers ? h->layers[l + 1].in_norm : h->w.final_norm;
    launch_rows_resid_norm(rd, h->stream);
  }
}

// Final norm + LM head + block statistics, then the draft pick of step k.  `defer` (the
// next step draws the tokens where it consumes them: a single sequence's layer-0 QKV
// GEMV, gemv_pick_supported, or the matrix-core body's row preparation): no sampling
// kernel; *defer receives the pick, and a single normalised row is copied to the
// fed-back buffer by the head.
int run_head(osprey_handle* h, int B, int k, int K, const int32_t* gather, const float* temp,
             const float* u, float* logits, long ld_b, int32_t* drafts_out, PickArgs* defer = nullptr) {
  const osprey_config& c = h->cfg;
  const Ws& W = h->W;
  // bf16 heads run on the matrix cores at every batch size; the rows come prepared
  // by the matrix-core body, or are normalised in the head after the vector body
  const bool mr = c.dtype == OSPREY_BF16;
  const bool prepared = gemm_use_mfma(c.dtype, B);
  int tn, nblk;
  LmPlan lp{};
  if (mr) {
    lp = lm_head_plan(std::min(B, kLmMaxRows), c.vocab_draft, h->n_cu);
    tn = lp.blk_rows;
    nblk = lp.nblk;
  } else {
    const GemvShape sh = gemv_shape(c.dtype, EPI_LOGITS, B, c.vocab_draft, c.d_model);
    tn = sh.rows_per_wave;
    nblk = sh.waves;
  }
  GemvArgs g{};
  g.max_rows = B;
  g.xin = W.x;
  g.ldx = c.d_model;
  g.gather = gather;
  g.xa_hi = W.xa_hi;   // matrix-core path: RMSNorm_final(x) prepared by the body
  g.xa_lo = W.xa_lo;
  g.ld_xa = c.d_model;
  g.gamma = h->w.final_norm;
  g.eps = c.rms_eps;
  g.d_norm = c.d_model;
  g.Kd = c.d_model;
  g.w0 = mr ? W.head_pk : h->w.lm_head;
  g.N = c.vocab_draft;
  g.y = logits + (long)k * c.vocab_draft;
  g.ld_logits = ld_b * c.vocab_draft;
  g.d2t = h->w.d2t;
  g.temp = temp;
  g.part = W.lm_part;
  g.nblk = nblk;
  if (defer && !prepared) g.fb_out = W.gfb;
  int t = h->t_begin(0);
  const int reps = t >= 0 ? kTimedRepeats : 1;
  for (int rep = 0; rep < reps; ++rep) {
  if (mr) {
    // passes of at most kLmMaxRows rows, all with the same record layout
    for (int r0 = 0; r0 < B; r0 += kLmMaxRows) {
      GemvArgs p = g;
      p.max_rows = std::min(kLmMaxRows, B - r0);
      if (gather) {
        p.gather = gather + r0;
      } else {
        p.xa_hi = W.xa_hi + (long)r0 * c.d_model;
        p.xa_lo = W.xa_lo + (long)r0 * c.d_model;
        p.xin = W.x + (long)r0 * c.d_model;
      }
      p.y = g.y + (long)r0 * g.ld_logits;
      p.temp = temp + r0;
      p.part = W.lm_part + (long)r0 * nblk * 4;
      if (!launch_lm_head(p, lp, !prepared, h->stream))
        return fail(OSPREY_E_UNSUPPORTED, "LM head: %d rows of width %d cannot be normalised in the kernel",
                    p.max_rows, p.Kd);
    }
  } else {
    launch_gemv(c.dtype, SRC_NORM, EPI_LOGITS, g, h->stream);
  }
  }
  h->t_end(t, reps);
  if (defer) {
    PickArgs& p = *defer;
    p.part = W.lm_part;
    p.ld_part = (long)nblk * 4;
    p.nblk = nblk;
    p.blk_rows = tn;
    p.logits = logits + (long)k * c.vocab_draft;
    p.ld_logits = ld_b * c.vocab_draft;
    p.V = c.vocab_draft;
    p.d2t = h->w.d2t;
    p.temp = temp;
    p.u = u + k;
    p.ld_u = K;
    p.k = k;
    p.draft = W.drafts + k;
    p.ld_draft = h->D.Km;
    p.draft_out = drafts_out ? drafts_out + k : nullptr;
    p.ld_draft_out = K;
    p.ar_tok = W.ar_tok;
    p.ar_pos = W.ar_pos;
    p.committed = W.committed;
    p.qstat = W.qstat + k;
    p.ld_qstat = h->D.Km;
    return OSPREY_OK;
  }
  SampleArgs s{};
  s.B = B;
  s.k = k;
  s.K = K;
  s.logits = logits + (long)k * c.vocab_draft;
  s.ld_logits = ld_b * c.vocab_draft;
  s.V = c.vocab_draft;
  s.part = W.lm_part;
  s.nblk = nblk;
  s.blk_rows = tn;
  s.temp = temp;
  s.u = u;
  s.d2t = h->w.d2t;
  s.drafts = W.drafts;
  s.ld_drafts = h->D.Km;
  s.drafts_out = drafts_out;
  s.ar_tok = W.ar_tok;
  s.ar_pos = W.ar_pos;
  s.committed = W.committed;
  s.x = W.x;
  s.gather = gather;
  s.d = c.d_model;
  s.gfb = W.gfb;
  s.qstat = W.qstat;
  s.ld_qstat = h->D.Km;
  launch_sample(s, h->stream);
  return OSPREY_OK;
}

// LM head over `rows` rows (gathered through `gather`, else rows 0.. of the body's
// output), logits row r at y + r V, softmax records at the rows' temperatures `temp`
// (W.lm_part, nblk per row).  Draft trees: rows of a pass at temperature 1 into
// W.logits; blocks: a block's rows into the draft logits.  Returns the head's plan.
LmPlan run_head_rows(osprey_handle* h, int rows, const int32_t* gather, const float* temp, float* y,
                     int& rc) {
  const osprey_config& c = h->cfg;
  const Ws& W = h->W;
  const bool prepared = gemm_use_mfma(c.dtype, rows);
  const LmPlan lp = lm_head_plan(std::min(rows, kLmMaxRows), c.vocab_draft, h->n_cu);
  GemvArgs g{};
  g.xin = W.x;
  g.ldx = c.d_model;
  g.xa_hi = W.xa_hi;
  g.xa_lo = W.xa_lo;
  g.ld_xa = c.d_model;
  g.gamma = h->w.final_norm;
  g.eps = c.rms_eps;
  g.d_norm = c.d_model;
  g.Kd = c.d_model;
  g.w0 = W.head_pk;
  g.N = c.vocab_draft;
  g.ld_logits = c.vocab_draft;
  g.d2t = h->w.d2t;
  g.nblk = lp.nblk;
  const int t = h->t_begin(0);
  const int reps = t >= 0 ? kTimedRepeats : 1;
  for (int rep = 0; rep < reps; ++rep) {
    for (int r0 = 0; r0 < rows; r0 += kLmMaxRows) {
      GemvArgs p = g;
      p.max_rows = std::min(kLmMaxRows, rows - r0);
      if (gather) {
        p.gather = gather + r0;
      } else {
        p.xa_hi = W.xa_hi + (long)r0 * c.d_model;
        p.xa_lo = W.xa_lo + (long)r0 * c.d_model;
        p.xin = W.x + (long)r0 * c.d_model;
      }
      p.y = y + (long)r0 * c.vocab_draft;
      p.temp = temp + r0;
      p.part = W.lm_part + (long)r0 * lp.nblk * 4;
      if (!launch_lm_head(p, lp, !prepared, h->stream))
        rc = fail(OSPREY_E_UNSUPPORTED, "LM head: %d rows of width %d cannot be normalised in the kernel",
                  p.max_rows, p.Kd);
    }
  }
  h->t_end(t, reps);
  return lp;
}

LmPlan run_head_tree(osprey_handle* h, int rows, const int32_t* gather, int& rc) {
  return run_head_rows(h, rows, gather, h->W.ones, h->W.logits, rc);
}

void fill_verify_common(osprey_handle* h, VerifyArgs& v, int B, int K) {
  const osprey_config& c = h->cfg;
  v.B = B;
  v.K = K;
  v.d2t = h->w.d2t;
  v.t2d = h->W.t2d;
  v.V_T = c.vocab_target;
  v.V_d = c.vocab_draft;
  v.chunk = kVerifyChunk;
  v.nchunk_t = h->D.nchunk_t;
  v.nchunk_d = h->D.nchunk_d;
  v.part = h->W.v_part;
  v.res_part = h->W.v_res;
  v.res_sub = h->W.v_sub;
  v.vstate = h->W.vstate;
  v.vstat = h->W.vstat;
  v.err = h->W.err;
}

}  // namespace

// =====================================================================================
OSPREY_API int osprey_config_validate(const osprey_config* cfg) { return validate(cfg); }

OSPREY_API size_t osprey_kv_bytes(const osprey_config* c) {
  if (validate(c) != OSPREY_OK) return 0;
  const size_t el = c->dtype == OSPREY_BF16 ? 2 : 4;
  return (size_t)c->kv_num_blocks * kv_block_elems(c->n_layers, c->n_kv_heads, c->kv_block, c->head_dim) * el;
}

OSPREY_API size_t osprey_workspace_bytes(const osprey_config* c) {
  if (validate(c) != OSPREY_OK) return 0;
  return plan(*c, nullptr, nullptr);
}

OSPREY_API int osprey_draft_init(const osprey_config* cfg, const osprey_weights* w, void* kv_pool,
                                 size_t kv_bytes, void* workspace, size_t ws_bytes,
                                 void* hip_stream, osprey_handle** out) {
  int rc = validate(cfg);
  if (rc != OSPREY_OK) return rc;
  if (!w || !out) return fail(OSPREY_E_INVALID, "weights and out must be non-NULL");
  if (!w->embed || !w->w_c || !w->final_norm || !w->lm_head || !w->d2t || !w->layers)
    return fail(OSPREY_E_INVALID, "a top-level weight pointer is NULL");
  for (int l = 0; l < cfg->n_layers; ++l) {
    const osprey_layer_weights& L = w->layers[l];
    if (!L.in_norm || !L.w_qkv || !L.w_o || !L.post_norm || !L.w_gate || !L.w_up || !L.w_down ||
        (cfg->qk_norm && (!L.q_norm || !L.k_norm)))
      return fail(OSPREY_E_INVALID, "a weight pointer of layer %d is NULL", l);
  }
  if (!kv_pool || !workspace) return fail(OSPREY_E_INVALID, "kv_pool and workspace must be non-NULL");
  if (((uintptr_t)kv_pool & 255) || ((uintptr_t)workspace & 255))
    return fail(OSPREY_E_INVALID, "kv_pool and workspace must be 256-byte aligned");
  if (kv_bytes < osprey_kv_bytes(cfg)) return fail(OSPREY_E_CAPACITY, "kv_bytes %zu < %zu", kv_bytes, osprey_kv_bytes(cfg));
  const size_t need = plan(*cfg, nullptr, nullptr);
  if (ws_bytes < need) return fail(OSPREY_E_CAPACITY, "ws_bytes %zu < %zu", ws_bytes, need);
  int ndev = 0, dev = 0, n_cu = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return fail(OSPREY_E_DEVICE, "no HIP device");
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
    return fail(OSPREY_E_DEVICE, "querying the compute-unit count failed");

  osprey_handle* h = new osprey_handle();
  h->cfg = *cfg;
  h->D = dims_of(*cfg);
  h->n_cu = n_cu;
  h->w = *w;
  h->layers.assign(w->layers, w->layers + cfg->n_layers);
  h->w.layers = h->layers.data();
  h->kv = kv_pool;
  h->stream = (hipStream_t)hip_stream;
  h->slots.assign(cfg->max_batch, SlotHost{});
  plan(*cfg, (char*)workspace, &h->W);

  auto bail = [&](int code) { delete h; return code; };
  // vocabulary map: validate and invert on the host
  const int Vd = cfg->vocab_draft, Vt = cfg->vocab_target;
  std::vector<int32_t> d2t(Vd), t2d(Vt, -1);
  if (hipMemcpy(d2t.data(), w->d2t, 4L * Vd, hipMemcpyDeviceToHost) != hipSuccess)
    return bail(fail(OSPREY_E_DEVICE, "reading d2t failed"));
  int mapped = 0;
  for (int i = 0; i < Vd; ++i) {
    const int t = d2t[i];
    if (t == -1) continue;
    if (t < 0 || t >= Vt) return bail(fail(OSPREY_E_INVALID, "d2t[%d] = %d not in [-1, %d)", i, t, Vt));
    if (t2d[t] != -1) return bail(fail(OSPREY_E_INVALID, "d2t maps rows %d and %d to target id %d", t2d[t], i, t));
    t2d[t] = i;
    ++mapped;
  }
  if (!mapped) return bail(fail(OSPREY_E_INVALID, "d2t maps no row"));
  // RoPE table in float64, stored as float32
  const int half = cfg->head_dim / 2;
  std::vector<float> cs((size_t)cfg->max_seq_len * half), sn(cs.size());
  for (int p = 0; p < cfg->max_seq_len; ++p)
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow((double)cfg->rope_theta, -(2.0 * i) / cfg->head_dim);
      const double ang = (double)p * inv;
      cs[(size_t)p * half + i] = (float)std::cos(ang);
      sn[(size_t)p * half + i] = (float)std::sin(ang);
    }
  const Ws& W = h->W;
  if (hipMemcpy(W.t2d, t2d.data(), 4L * Vt, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(W.rope_cos, cs.data(), 4 * cs.size(), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(W.rope_sin, sn.data(), 4 * sn.size(), hipMemcpyHostToDevice) != hipSuccess)
    return bail(fail(OSPREY_E_DEVICE, "uploading tables failed"));
  const long B = h->D.B;
  // temperature 1 for the LM-head records of draft-tree passes
  launch_fill_i32(reinterpret_cast<int32_t*>(W.ones), 0x3f800000, B * kMaxTopk, h->stream);
  // bf16 heads are read from a packed copy (the matrix cores' order)
  if (W.head_pk) launch_pack_head(w->lm_head, Vd, cfg->d_model, W.head_pk, h->stream);
  if (hipMemset(W.slot_len, 0, 4 * B) != hipSuccess || hipMemset(W.pend_n, 0, 4 * B) != hipSuccess ||
      hipMemset(W.slot_nblocks, 0, 4 * B) != hipSuccess ||
      hipMemset(W.block_table, 0, 4L * B * h->D.max_blocks) != hipSuccess ||
      hipMemset(W.pend_tok, 0, 4L * B * (cfg->max_k + 1)) != hipSuccess ||
      hipMemset(W.err, 0, 16) != hipSuccess ||
      hipMemset(W.u_zero, 0, 4L * B * h->D.Km) != hipSuccess ||
      hipMemset(W.n_cand, 0, 4L * B) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
    return bail(fail(OSPREY_E_DEVICE, "clearing the workspace failed"));
  *out = h;
  return ok();
}

OSPREY_API int osprey_seq_reset(osprey_handle* h, int32_t slot, const int32_t* block_ids, int32_t n_blocks) {
  int rc = check_handle(h);
  if (rc) return rc;
  if ((rc = check_slot(h, slot))) return rc;
  if (n_blocks < 0 || n_blocks > h->D.max_blocks)
    return fail(OSPREY_E_CAPACITY, "n_blocks %d not in [0, %d]", n_blocks, h->D.max_blocks);
  if (n_blocks > 0 && !block_ids) return fail(OSPREY_E_INVALID, "block_ids is NULL");
  for (int i = 0; i < n_blocks; ++i)
    if (block_ids[i] < 0 || block_ids[i] >= h->cfg.kv_num_blocks)
      return fail(OSPREY_E_INVALID, "block_ids[%d] = %d not in [0, %d)", i, block_ids[i], h->cfg.kv_num_blocks);
  const Ws& W = h->W;
  HIP_TRY(hipStreamSynchronize(h->stream));
  if (n_blocks) HIP_TRY(hipMemcpy(W.block_table + (long)slot * h->D.max_blocks, block_ids, 4L * n_blocks, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(W.slot_nblocks + slot, &n_blocks, 4, hipMemcpyHostToDevice));
  launch_set_len(W.slot_len, W.pend_n, slot, 0, h->stream);
  HIP_TRY(hipStreamSynchronize(h->stream));
  SlotHost& s = h->slots[slot];
  s.state = S_READY;
  s.len_max = 0;
  s.nblocks = n_blocks;
  s.drafted_k = 0;
  return hip_last();
}

OSPREY_API int osprey_kv_append(osprey_handle* h, int32_t slot, int32_t n, const void* k, const void* v) {
  int rc = check_handle(h);
  if (rc) return rc;
  if ((rc = check_slot(h, slot))) return rc;
  SlotHost& s = h->slots[slot];
  if (s.state != S_READY) return fail(OSPREY_E_STATE, "slot %d is not READY", slot);
  if (n < 0) return fail(OSPREY_E_INVALID, "n %d < 0", n);
  if (n > 0 && (!k || !v)) return fail(OSPREY_E_INVALID, "k and v must be non-NULL");
  if (s.len_max + n > (long)s.nblocks * h->cfg.kv_block)
    return fail(OSPREY_E_CAPACITY, "slot %d: %ld + %d positions exceed its %d pages", slot, s.len_max, n, s.nblocks);
  if (n == 0) return ok();
  launch_kv_append(h->cfg.dtype, h->kv, k, v, h->cfg.n_layers, n, h->cfg.n_kv_heads, h->cfg.head_dim,
                   h->cfg.kv_block, h->W.block_table, slot, h->D.max_blocks, h->W.slot_len,
                   h->W.slot_len, h->stream);
  s.len_max += n;
  return hip_last();
}

OSPREY_API int osprey_seq_truncate(osprey_handle* h, int32_t slot, int32_t length) {
  int rc = check_handle(h);
  if (rc) return rc;
  if ((rc = check_slot(h, slot))) return rc;
  SlotHost& s = h->slots[slot];
  if (s.state != S_READY && s.state != S_VERIFIED) return fail(OSPREY_E_STATE, "slot %d is not READY or VERIFIED", slot);
  if (length < 0 || length > s.len_max) return fail(OSPREY_E_INVALID, "length %d not in [0, %ld]", length, s.len_max);
  launch_set_len(h->W.slot_len, h->W.pend_n, slot, length, h->stream);
  s.len_max = length;
  s.state = S_READY;
  return hip_last();
}

OSPREY_API int osprey_seq_length(osprey_handle* h, int32_t slot, int32_t* length) {
  int rc = check_handle(h);
  if (rc) return rc;
  if ((rc = check_slot(h, slot))) return rc;
  if (!length) return fail(OSPREY_E_INVALID, "length is NULL");
  HIP_TRY(hipStreamSynchronize(h->stream));
  HIP_TRY(hipMemcpy(length, h->W.slot_len + slot, 4, hipMemcpyDeviceToHost));
  SlotHost& s = h->slots[slot];
  if (s.state != S_DRAFTED) s.len_max = *length;
  return ok();
}

namespace {

// Validation, row layout and ingest of a draft call: the new rows of every sequence
// through the tap projection (Eq. 1) and the body.  K: the chain's drafts (the setup
// kernel's autoregressive positions); extra: positions past the ingest the call will
// use (chain: K - 1; tree: its depth).  block_mask >= 0 (block drafting): extra mask
// rows (token block_mask, the anchor's tap row) follow every sequence's new rows in
// the same pass.
int step_ingest(osprey_handle* h, const osprey_step_args* a, int K, int extra, SplitPlan& split,
                bool& pending, int& tt, int max_split = kMaxSplit, int block_mask = -1) {
  int rc;
  const osprey_config& c = h->cfg;
  const int B = a->batch;
  if (!a->slots || !a->taps || !a->temperature) return fail(OSPREY_E_INVALID, "slots, taps and temperature must be non-NULL");
  pending = a->n_new == nullptr;
  if (!pending && !a->new_tokens) return fail(OSPREY_E_INVALID, "new_tokens is NULL in explicit mode");
  if (a->taps_stride < 0) return fail(OSPREY_E_INVALID, "taps_stride < 0");
  if (pending && a->taps_stride == 0) return fail(OSPREY_E_INVALID, "pending mode needs taps_stride > 0");
  std::vector<char> seen(c.max_batch, 0);
  long rows = 0, ctx_max = 0, ctx_total = 0;
  int max_new = 0;
  for (int b = 0; b < B; ++b) {
    const int slot = a->slots[b];
    if ((rc = check_slot(h, slot))) return rc;
    if (seen[slot]) return fail(OSPREY_E_INVALID, "slot %d appears twice", slot);
    seen[slot] = 1;
    const SlotHost& s = h->slots[slot];
    int n;
    if (pending) {
      if (s.state != S_VERIFIED) return fail(OSPREY_E_STATE, "slot %d has no verified tokens pending", slot);
      n = s.drafted_k + 1;
      if (a->taps_stride < n) return fail(OSPREY_E_INVALID, "taps_stride %d < %d pending rows of slot %d", a->taps_stride, n, slot);
    } else {
      if (s.state != S_READY && s.state != S_VERIFIED) return fail(OSPREY_E_STATE, "slot %d is not READY or VERIFIED", slot);
      n = a->n_new[b];
      if (n < 1) return fail(OSPREY_E_INVALID, "n_new[%d] = %d < 1", b, n);
      if (a->taps_stride > 0 && n > a->taps_stride) return fail(OSPREY_E_INVALID, "n_new[%d] = %d > taps_stride", b, n);
    }
    const long need = s.len_max + n + extra;
    if (need > (long)s.nblocks * c.kv_block || need > c.max_seq_len)
      return fail(OSPREY_E_CAPACITY, "slot %d: up to %ld positions exceed its %d pages / max_seq_len", slot, need, s.nblocks);
    rows += n + (block_mask >= 0 ? extra : 0);
    max_new = std::max(max_new, n);
    ctx_max = std::max(ctx_max, need);
    ctx_total += need;
  }
  if (rows > h->D.Rmax) return fail(OSPREY_E_CAPACITY, "%ld new rows exceed the workspace's %d", rows, h->D.Rmax);
  if (!pending && rows > std::max(c.max_new_rows, c.max_batch * (c.max_k + 1)))
    return fail(OSPREY_E_CAPACITY, "%ld new rows exceed max_new_rows", rows);

  const Ws& W = h->W;
  if (h->ctx_plan > 0) {
    ctx_max = std::max(ctx_max, h->ctx_plan);
    ctx_total = std::max(ctx_total, h->ctx_plan * B);
  }
  // A single sequence's bf16 chain takes splits of at least 128 positions: its draft
  // steps attend faster over a 2K context in 17 splits than in 33, and their O
  // projection merges that few splits itself.  (Block passes and fp32 caches, whose
  // attention only loses by it, and trees keep 64.)
  const bool chain1 = B == 1 && c.dtype == OSPREY_BF16 && block_mask < 0 && K >= 2;
  split = plan_splits(h, ctx_max, ctx_total, max_split, chain1 ? 128 : 64);
  if (split.n_split > max_split)
    return fail(OSPREY_E_UNSUPPORTED, "a context of %ld positions needs %d splits (at most %d)", ctx_max,
                split.n_split, max_split);
  tt = h->t_begin(3);
  // ---- row layout of the ingest ---------------------------------------------------------
  SetupArgs sa{};
  sa.B = B;
  sa.explicit_rows = pending ? 0 : 1;
  for (int b = 0; b < B; ++b) {
    sa.slots[b] = a->slots[b];
    sa.n_new[b] = pending ? 0 : a->n_new[b];
  }
  sa.new_tokens = a->new_tokens;
  sa.taps_stride = a->taps_stride;
  sa.K = K;
  sa.max_new = pending ? c.max_k + 1 : std::max(max_new, 1);
  sa.V_T = c.vocab_target;
  sa.slot_len = W.slot_len;
  sa.pend_n = W.pend_n;
  sa.pend_tok = W.pend_tok;
  sa.pend_ld = c.max_k + 1;
  sa.slot_nblocks = W.slot_nblocks;
  sa.kv_block = c.kv_block;
  sa.ing_seq = W.ing_seq;
  sa.ing_pos = W.ing_pos;
  sa.ing_tok = W.ing_tok;
  sa.ing_tap = W.ing_tap;
  sa.n_rows = W.n_rows;
  sa.cu = W.cu;
  sa.last_row = W.last_row;
  sa.committed = W.committed;
  sa.bslot = W.bslot;
  sa.ar_pos = W.ar_pos;
  sa.err = W.err;
  sa.split_len = split.split_len;
  sa.attn_items = W.attn_items;
  sa.attn_n_items = W.attn_n_items;
  if (block_mask >= 0) {
    sa.extra = extra;
    sa.mask = block_mask;
    sa.temp = a->temperature;
    sa.blk_gather = W.b_gather;
    sa.blk_temp = W.b_temp;
  }
  launch_setup(sa, h->stream);

  // ---- ingest: tap projection (Eq. 1) then the body over every new row ------------------
  RowMeta ing{W.ing_seq, W.ing_pos, W.ing_tok, W.n_rows, (int)rows};
  GemvArgs gt{};
  gt.max_rows = (int)rows;
  gt.count = W.n_rows;
  gt.taps = a->taps;
  gt.tap_row = W.ing_tap;
  gt.ldt = (long)c.n_taps * c.target_hidden;
  gt.Kd = c.n_taps * c.target_hidden;
  gt.w0 = h->w.w_c;
  gt.N = c.d_model;
  gt.y = W.s;
  gt.ldy = c.d_model;
  gt.split_buf = W.split;
  if (gemm_use_mfma(c.dtype, (int)rows)) {
    int ks_taps;
    if (rows <= kLmMaxRows) {
      gt.split_buf = W.split_s;
      ks_taps = launch_skinny(SRC_TAPS, gt, h->stream);
    } else {
      ks_taps = launch_gemm(SRC_TAPS, EPI_STORE, gt, h->stream);
    }
    run_body_mr(h, ing, W.cu, B, nullptr, ks_taps, split, max_new + (block_mask >= 0 ? extra : 0), a->slots[0]);
  } else {
    launch_gemv(c.dtype, SRC_TAPS, EPI_STORE, gt, h->stream);
    run_body(h, ing, W.cu, B, W.s, true, split, max_new, a->slots[0]);
  }
  return OSPREY_OK;
}

// Slot bookkeeping after a draft call: the ingested rows are committed.
void step_commit(osprey_handle* h, const osprey_step_args* a, bool pending, int K) {
  for (int b = 0; b < a->batch; ++b) {
    SlotHost& s = h->slots[a->slots[b]];
    const int n = pending ? s.drafted_k + 1 : a->n_new[b];
    s.len_max += n;
    s.state = K >= 1 ? S_DRAFTED : S_READY;
    s.drafted_k = K;
  }
}

}  // namespace

OSPREY_API int osprey_draft_step(osprey_handle* h, const osprey_step_args* a) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!a) return fail(OSPREY_E_INVALID, "args is NULL");
  const osprey_config& c = h->cfg;
  const int B = a->batch, K = a->K;
  if (B < 1 || B > c.max_batch) return fail(OSPREY_E_INVALID, "batch %d not in [1, %d]", B, c.max_batch);
  if (K < 0 || K > c.max_k) return fail(OSPREY_E_INVALID, "K %d not in [0, %d]", K, c.max_k);
  SplitPlan split;
  bool pending;
  int tt;
  if ((rc = step_ingest(h, a, K, std::max(K - 1, 0), split, pending, tt))) return rc;
  const Ws& W = h->W;

  // ---- K autoregressive draft steps ---------------------------------------------------------
  float* logits = a->draft_logits ? a->draft_logits : W.logits;
  const long ld_b = a->draft_logits ? K : h->D.Km;
  const float* u = a->u_draft ? a->u_draft : W.u_zero;
  if (K >= 1) {
    RowMeta ar{nullptr, W.ar_pos, W.ar_tok, nullptr, B};
    const bool ar_mr = gemm_use_mfma(c.dtype, B);
    // Each draft but the last is drawn where the next step consumes it instead of by a
    // sampling kernel (one launch fewer per step): a single sequence on the vector body
    // draws in its layer-0 QKV GEMV (the head copies its gathered input row to the
    // fed-back buffer), the rows of the matrix-core body in their row preparation, whose
    // conditioning input is then the rows x themselves.  The latter needs row b of x to
    // be sequence b's, so the first draft, whose head reads the ingest's gathered last
    // rows (packed, several per sequence), keeps its sampling kernel there.
    const int lm_nblk = lm_head_plan(std::min(B, kLmMaxRows), c.vocab_draft, h->n_cu).nblk;
    const bool fuse = c.dtype == OSPREY_BF16 &&
                      (ar_mr ? lm_nblk <= kPickMaxRecords
                             : lm_head_norm_in_supported(B, c.d_model) && gemv_pick_supported(c.dtype, B, lm_nblk));
    auto deferred = [&](int k) { return fuse && k + 1 < K && (k >= 1 || !ar_mr); };
    PickArgs pick{};
    if ((rc = run_head(h, B, 0, K, W.last_row, a->temperature, u, logits, ld_b, a->draft_tokens,
                       deferred(0) ? &pick : nullptr)))
      return rc;
    for (int k = 1; k < K; ++k) {
      const bool drawn = deferred(k - 1);
      if (ar_mr) run_body_mr(h, ar, nullptr, B, drawn ? W.x : W.gfb, 1, split, 1, a->slots[0], nullptr, drawn ? &pick : nullptr);
      else run_body(h, ar, nullptr, B, W.gfb, true, split, 1, a->slots[0], drawn ? &pick : nullptr);
      if ((rc = run_head(h, B, k, K, nullptr, a->temperature, u, logits, ld_b, a->draft_tokens,
                         deferred(k) ? &pick : nullptr)))
        return rc;
    }
  }
  h->t_end(tt);
  if ((rc = hip_last())) return rc;
  step_commit(h, a, pending, K);
  h->last_B = B;
  h->last_K = K;
  h->last_slots.assign(a->slots, a->slots + B);
  h->last_logits = logits;
  h->last_ld_b = ld_b;
  return ok();
}

OSPREY_API int osprey_draft_block(osprey_handle* h, const osprey_step_args* a, int32_t mask_token) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!a) return fail(OSPREY_E_INVALID, "args is NULL");
  const osprey_config& c = h->cfg;
  const int B = a->batch, K = a->K;
  if (B < 1 || B > c.max_batch) return fail(OSPREY_E_INVALID, "batch %d not in [1, %d]", B, c.max_batch);
  if (K < 2 || K > c.max_k) return fail(OSPREY_E_INVALID, "K %d not in [2, %d] (one proposal is osprey_draft_step's first)", K, c.max_k);
  if (c.dtype != OSPREY_BF16) return fail(OSPREY_E_UNSUPPORTED, "block drafting needs bf16 weights (the matrix-core body)");
  if (mask_token < 0 || mask_token >= c.vocab_target)
    return fail(OSPREY_E_INVALID, "mask_token %d not in [0, %d)", mask_token, c.vocab_target);
  SplitPlan split;
  bool pending;
  int tt;
  // the ingest and the block in one pass: every sequence's new rows, then K - 1 mask rows
  if ((rc = step_ingest(h, a, K, K - 1, split, pending, tt, kMaxSplit, mask_token))) return rc;
  const Ws& W = h->W;
  const int rows = B * K;
  // ---- LM head over the block's rows, then one pick per (sequence, proposal) ------------
  float* logits = a->draft_logits ? a->draft_logits : W.logits;
  const LmPlan lp = run_head_rows(h, rows, W.b_gather, W.b_temp, logits, rc);
  if (rc) return rc;
  SampleArgs sm{};
  sm.block = 1;
  sm.B = B;
  sm.K = K;
  sm.logits = logits;
  sm.ld_logits = (long)K * c.vocab_draft;
  sm.V = c.vocab_draft;
  sm.part = W.lm_part;
  sm.nblk = lp.nblk;
  sm.blk_rows = lp.blk_rows;
  sm.temp = a->temperature;
  sm.u = a->u_draft ? a->u_draft : W.u_zero;
  sm.d2t = h->w.d2t;
  sm.drafts = W.drafts;
  sm.ld_drafts = h->D.Km;
  sm.drafts_out = a->draft_tokens;
  sm.committed = W.committed;
  sm.d = 0;
  sm.qstat = W.qstat;
  sm.ld_qstat = h->D.Km;
  launch_sample(sm, h->stream);
  h->t_end(tt);
  if ((rc = hip_last())) return rc;
  step_commit(h, a, pending, K);
  h->last_B = B;
  h->last_K = K;
  h->last_slots.assign(a->slots, a->slots + B);
  h->last_logits = logits;
  h->last_ld_b = K;
  return ok();
}

OSPREY_API int osprey_draft_tree(osprey_handle* h, const osprey_step_args* a, const osprey_tree_args* t) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!a || !t) return fail(OSPREY_E_INVALID, "args is NULL");
  const osprey_config& c = h->cfg;
  const int B = a->batch, k = t->topk, D = t->depth, N = t->n_nodes;
  if (B < 1 || B > c.max_batch) return fail(OSPREY_E_INVALID, "batch %d not in [1, %d]", B, c.max_batch);
  if (a->K != 0) return fail(OSPREY_E_INVALID, "a draft tree takes K = 0 in its step arguments (K %d)", a->K);
  if (c.dtype != OSPREY_BF16) return fail(OSPREY_E_UNSUPPORTED, "draft trees need bf16 weights (the matrix-core body)");
  const int kmax = std::min(kMaxTopk, std::max(c.max_k, 1));
  if (k < 2 || k > kmax) return fail(OSPREY_E_INVALID, "topk %d not in [2, %d] (top-k 1 is a chain: osprey_draft_step)", k, kmax);
  if (D < 1 || D > kMaxTreeDepth) return fail(OSPREY_E_INVALID, "depth %d not in [1, %d]", D, kMaxTreeDepth);
  const int n_cand = k + (D - 1) * k * k;
  if (N < 1 || N > std::min(kMaxTreeNodes, n_cand))
    return fail(OSPREY_E_INVALID, "n_nodes %d not in [1, %d]", N, std::min(kMaxTreeNodes, n_cand));
  if (!t->tokens || !t->parents) return fail(OSPREY_E_INVALID, "tree outputs are NULL");
  if (c.vocab_draft > kTkBlocks * 256 * 16 ||
      lm_head_plan(std::min(B * k, kLmMaxRows), c.vocab_draft, h->n_cu).nblk > kTkMaxRecords)
    return fail(OSPREY_E_UNSUPPORTED, "vocab_draft %d too large for trees", c.vocab_draft);
  SplitPlan split;
  bool pending;
  int tt;
  if ((rc = step_ingest(h, a, 0, D - 1, split, pending, tt, kMaxSplit - 1))) return rc;
  const Ws& W = h->W;
  TreeArgs ta{};
  ta.B = B;
  ta.k = k;
  ta.depth = D;
  ta.n_nodes = N;
  ta.V = c.vocab_draft;
  ta.d2t = h->w.d2t;
  ta.logits = W.logits;
  ta.ld_logits = c.vocab_draft;
  ta.cand_v = W.tree_cv;
  ta.cand_r = W.tree_cr;
  ta.rec = W.lm_part;
  ta.c_tok = W.c_tok;
  ta.c_par = W.c_par;
  ta.c_score = W.c_score;
  ta.c_depth = W.c_depth;
  ta.c_slot = W.c_slot;
  ta.n_cand = W.n_cand;
  ta.front = W.front;
  ta.r_tok = W.r_tok;
  ta.r_pos = W.r_pos;
  ta.r_attpos = W.r_attpos;
  ta.r_node = W.r_node;
  ta.r_anc = W.r_anc;
  ta.r_cu = W.r_cu;
  ta.r_s = W.r_s;
  ta.x = W.x;
  ta.d = c.d_model;
  ta.last_row = W.last_row;
  ta.committed = W.committed;
  ta.out_tok = t->tokens;
  ta.out_par = t->parents;
  ta.out_score = t->scores;
  // the root: the last ingest row of every sequence
  ta.pass = 0;
  // passes of many rows select their top-k from the LM-head records in the step kernel;
  // few rows spread each row over kTkBlocks blocks of a separate pass first
  auto select = [&](int rows, const LmPlan& lp) {
    ta.nblk = lp.nblk;
    ta.blk_rows = lp.blk_rows;
    ta.cand_v = rows >= kTkRecordRows ? nullptr : W.tree_cv;
    ta.cand_r = W.tree_cr;
    if (ta.cand_v) launch_tree_topk(ta, rows, h->stream);
  };
  select(B, run_head_tree(h, B, W.last_row, rc));
  if (rc) return rc;
  launch_tree_step(ta, h->stream);
  // every further depth: the frontier's B k rows through the body and the LM head
  const int rows = B * k;
  for (int p = 1; p < D; ++p) {
    RowMeta rm{nullptr, W.r_attpos, W.r_tok, nullptr, rows};
    TreePass tp{W.r_node, W.r_anc, W.r_pos, W.bslot};
    run_body_mr(h, rm, W.r_cu, B, W.r_s, 1, split, k, -1, &tp);
    ta.pass = p;
    select(rows, run_head_tree(h, rows, nullptr, rc));
    if (rc) return rc;
    launch_tree_step(ta, h->stream);
  }
  launch_tree_final(ta, h->stream);
  h->t_end(tt);
  if ((rc = hip_last())) return rc;
  step_commit(h, a, pending, 0);
  h->last_B = 0;
  return ok();
}

OSPREY_API int osprey_verify(osprey_handle* h, const osprey_verify_args* a) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!a) return fail(OSPREY_E_INVALID, "args is NULL");
  if (!a->slots || !a->target_logits || !a->temperature || !a->u_accept || !a->u_bonus ||
      !a->accept_len || !a->accept_mask || !a->out_tokens)
    return fail(OSPREY_E_INVALID, "a verify pointer is NULL");
  if (a->batch != h->last_B || a->K != h->last_K)
    return fail(OSPREY_E_STATE, "verify (batch %d, K %d) does not match the last draft_step (batch %d, K %d)",
                a->batch, a->K, h->last_B, h->last_K);
  if (a->K < 1) return fail(OSPREY_E_STATE, "the last draft_step proposed no drafts");
  for (int b = 0; b < a->batch; ++b) {
    if (a->slots[b] != h->last_slots[b]) return fail(OSPREY_E_STATE, "slots differ from the last draft_step");
    if (h->slots[a->slots[b]].state != S_DRAFTED) return fail(OSPREY_E_STATE, "slot %d is not DRAFTED", a->slots[b]);
  }
  VerifyArgs v{};
  fill_verify_common(h, v, a->batch, a->K);
  v.target = a->target_logits;
  v.draft = h->last_logits;
  v.ld_draft_b = h->last_ld_b;
  v.qstat = h->W.qstat;
  v.ld_qstat = h->D.Km;
  v.drafts = h->W.drafts;
  v.ld_drafts = h->D.Km;
  v.temp = a->temperature;
  v.temp_d = a->draft_temperature ? a->draft_temperature : a->temperature;
  v.u_acc = a->u_accept;
  v.u_bonus = a->u_bonus;
  v.accept_len = a->accept_len;
  v.accept_mask = a->accept_mask;
  v.out_tokens = a->out_tokens;
  v.bslot = h->W.bslot;
  v.pend_n = h->W.pend_n;
  v.pend_tok = h->W.pend_tok;
  v.pend_ld = h->cfg.max_k + 1;
  int t = h->t_begin(2);
  launch_verify(v, h->stream);
  h->t_end(t);
  if ((rc = hip_last())) return rc;
  for (int b = 0; b < a->batch; ++b) h->slots[a->slots[b]].state = S_VERIFIED;
  h->last_B = 0;
  return ok();
}

OSPREY_API int osprey_verify_rows(osprey_handle* h, const osprey_verify_rows_args* a) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!a) return fail(OSPREY_E_INVALID, "args is NULL");
  if (a->batch < 1 || a->batch > h->cfg.max_batch) return fail(OSPREY_E_INVALID, "batch %d not in [1, %d]", a->batch, h->cfg.max_batch);
  if (a->K < 0 || a->K > h->cfg.max_k) return fail(OSPREY_E_INVALID, "K %d not in [0, %d]", a->K, h->cfg.max_k);
  if (!a->target_logits || !a->temperature || !a->u_bonus || !a->accept_len || !a->accept_mask ||
      !a->out_tokens || (a->K > 0 && (!a->draft_logits || !a->draft_tokens || !a->u_accept)))
    return fail(OSPREY_E_INVALID, "a verify pointer is NULL");
  VerifyArgs v{};
  fill_verify_common(h, v, a->batch, a->K);
  v.target = a->target_logits;
  v.draft = a->draft_logits;
  v.ld_draft_b = a->K;
  v.drafts = a->draft_tokens;
  v.ld_drafts = a->K;
  v.temp = a->temperature;
  v.temp_d = a->draft_temperature ? a->draft_temperature : a->temperature;
  v.u_acc = a->u_accept;
  v.u_bonus = a->u_bonus;
  v.accept_len = a->accept_len;
  v.accept_mask = a->accept_mask;
  v.out_tokens = a->out_tokens;
  int t = h->t_begin(2);
  launch_verify(v, h->stream);
  h->t_end(t);
  return hip_last();
}

OSPREY_API int osprey_verify_tree(osprey_handle* h, const osprey_verify_tree_args* a) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!a) return fail(OSPREY_E_INVALID, "args is NULL");
  if (a->batch < 1 || a->batch > h->cfg.max_batch) return fail(OSPREY_E_INVALID, "batch %d not in [1, %d]", a->batch, h->cfg.max_batch);
  if (a->n_nodes < 0 || a->n_nodes > kMaxTreeNodes)
    return fail(OSPREY_E_INVALID, "n_nodes %d not in [0, %d]", a->n_nodes, kMaxTreeNodes);
  if (!a->target_logits || !a->temperature || !a->u_bonus || !a->accept_len || !a->out_tokens ||
      (a->n_nodes > 0 && (!a->tokens || !a->parents || !a->u_accept || !a->accept_path)))
    return fail(OSPREY_E_INVALID, "a verify_tree pointer is NULL");
  VerifyArgs v{};
  fill_verify_common(h, v, a->batch, a->n_nodes);
  v.target = a->target_logits;
  v.temp = a->temperature;
  v.temp_d = a->temperature;
  v.u_acc = a->u_accept;
  v.u_bonus = a->u_bonus;
  v.accept_len = a->accept_len;
  v.out_tokens = a->out_tokens;
  v.tree_tok = a->tokens;
  v.tree_par = a->parents;
  v.tree_path = a->accept_path;
  v.tree_removed = h->W.tree_removed;
  int t = h->t_begin(2);
  launch_verify_tree(v, h->stream);
  h->t_end(t);
  return hip_last();
}

// ---- one steady-state iteration as a HIP graph -------------------------------------------
struct osprey_graph {
  osprey_handle* h = nullptr;
  hipGraphExec_t exec = nullptr;
  int B = 0, K = 0, taps_stride = 0;
  long max_context = 0;
  std::vector<int> slots;
};

namespace {

// Positions a pending iteration of `g` may reach on `slot`: its committed length, the
// pending ingest and the K - 1 positions past it (chain steps or block mask rows).
long graph_need(const osprey_handle* h, const osprey_graph* g, int slot) {
  const SlotHost& s = h->slots[slot];
  return s.len_max + (s.drafted_k + 1) + (g->K - 1);
}

}  // namespace

OSPREY_API int osprey_graph_capture(osprey_handle* h, const osprey_step_args* step, int32_t mask_token,
                                    const osprey_verify_args* v, int32_t max_context, osprey_graph** out) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!step || !v || !out) return fail(OSPREY_E_INVALID, "arguments are NULL");
  if (!h->stream) return fail(OSPREY_E_INVALID, "capture needs a stream other than the null stream (osprey_set_stream)");
  if (h->timing) return fail(OSPREY_E_STATE, "kernel timing is on: disable it (osprey_kernel_timing(h, 0)) before capturing");
  if (step->n_new) return fail(OSPREY_E_INVALID, "a captured iteration ingests the pending tokens: n_new must be NULL");
  const int B = step->batch, K = step->K;
  if (B < 1 || B > h->cfg.max_batch || K < 1) return fail(OSPREY_E_INVALID, "batch %d / K %d", B, K);
  if (v->batch != B || v->K != K || !step->slots || !v->slots)
    return fail(OSPREY_E_INVALID, "draft and verify arguments must have the same batch, K and slots");
  for (int b = 0; b < B; ++b)
    if (step->slots[b] != v->slots[b]) return fail(OSPREY_E_INVALID, "draft and verify slots differ at %d", b);
  if (max_context < 1 || max_context > h->cfg.max_seq_len)
    return fail(OSPREY_E_INVALID, "max_context %d not in [1, %d]", max_context, h->cfg.max_seq_len);
  if (step->taps_stride < K + 1) return fail(OSPREY_E_INVALID, "taps_stride %d < K + 1", step->taps_stride);
  osprey_graph probe;
  probe.K = K;
  for (int b = 0; b < B; ++b) {
    if ((rc = check_slot(h, step->slots[b]))) return rc;
    if (graph_need(h, &probe, step->slots[b]) > max_context)
      return fail(OSPREY_E_CAPACITY, "slot %d already needs more than max_context %d positions", step->slots[b], max_context);
  }
  // the calls below validate everything else and update the host state as if they ran:
  // keep that state and put it back afterwards (launches advance it)
  const std::vector<SlotHost> saved = h->slots;
  const int sB = h->last_B, sK = h->last_K;
  const std::vector<int> sslots = h->last_slots;
  float* slog = h->last_logits;
  const long sld = h->last_ld_b;
  hipError_t e = hipStreamBeginCapture(h->stream, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) return fail(OSPREY_E_DEVICE, "hipStreamBeginCapture: %s", hipGetErrorString(e));
  h->ctx_plan = max_context;
  rc = mask_token < 0 ? osprey_draft_step(h, step) : osprey_draft_block(h, step, mask_token);
  if (rc == OSPREY_OK) rc = osprey_verify(h, v);
  h->ctx_plan = 0;
  const std::string msg = g_err;
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(h->stream, &graph);
  h->slots = saved;
  h->last_B = sB;
  h->last_K = sK;
  h->last_slots = sslots;
  h->last_logits = slog;
  h->last_ld_b = sld;
  if (rc != OSPREY_OK) {
    if (graph) hipGraphDestroy(graph);
    g_err = msg;
    return rc;
  }
  if (e != hipSuccess || !graph) return fail(OSPREY_E_DEVICE, "hipStreamEndCapture: %s", hipGetErrorString(e));
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (e != hipSuccess) return fail(OSPREY_E_DEVICE, "hipGraphInstantiate: %s", hipGetErrorString(e));
  osprey_graph* g = new osprey_graph();
  g->h = h;
  g->exec = exec;
  g->B = B;
  g->K = K;
  g->taps_stride = step->taps_stride;
  g->max_context = max_context;
  g->slots.assign(step->slots, step->slots + B);
  *out = g;
  return ok();
}

OSPREY_API int osprey_graph_launch(osprey_handle* h, osprey_graph* g) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!g || g->h != h) return fail(OSPREY_E_INVALID, "graph is NULL or was captured on another handle");
  for (int slot : g->slots) {
    const SlotHost& s = h->slots[slot];
    if (s.state != S_VERIFIED) return fail(OSPREY_E_STATE, "slot %d has no verified tokens pending", slot);
    if (s.drafted_k + 1 > g->taps_stride)
      return fail(OSPREY_E_INVALID, "slot %d: %d pending rows exceed the captured taps_stride %d", slot,
                  s.drafted_k + 1, g->taps_stride);
    const long need = graph_need(h, g, slot);
    if (need > g->max_context || need > (long)s.nblocks * h->cfg.kv_block)
      return fail(OSPREY_E_CAPACITY, "slot %d: up to %ld positions exceed the graph's max_context %ld or its pages",
                  slot, need, g->max_context);
  }
  HIP_TRY(hipGraphLaunch(g->exec, h->stream));
  for (int slot : g->slots) {
    SlotHost& s = h->slots[slot];
    s.len_max += s.drafted_k + 1;
    s.drafted_k = g->K;
    s.state = S_VERIFIED;
  }
  h->last_B = 0;
  return ok();
}

OSPREY_API int osprey_graph_destroy(osprey_graph* g) {
  if (!g) return ok();
  if (g->exec) hipGraphExecDestroy(g->exec);
  delete g;
  return ok();
}

OSPREY_API int osprey_device_errors(osprey_handle* h, uint32_t* flags) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!flags) return fail(OSPREY_E_INVALID, "flags is NULL");
  HIP_TRY(hipStreamSynchronize(h->stream));
  HIP_TRY(hipMemcpy(flags, h->W.err, 4, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemset(h->W.err, 0, 4));
  return ok();
}

OSPREY_API int osprey_kernel_timing(osprey_handle* h, int32_t families) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (families < 0 || families >= (1 << 5)) return fail(OSPREY_E_INVALID, "families mask %d", families);
  HIP_TRY(hipStreamSynchronize(h->stream));
  for (auto& r : h->timers) { h->free_events.push_back(r.a); h->free_events.push_back(r.b); }
  h->timers.clear();
  h->timing = families;
  return ok();
}

OSPREY_API int osprey_kernel_time(osprey_handle* h, int32_t family, double* total_ms, int64_t* launches) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!total_ms || !launches) return fail(OSPREY_E_INVALID, "outputs are NULL");
  HIP_TRY(hipStreamSynchronize(h->stream));
  double tot = 0;
  int64_t n = 0;
  for (auto& r : h->timers) {
    if (r.family != family) continue;
    float ms = 0;
    HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b));
    tot += ms;
    n += r.reps;
  }
  *total_ms = tot;
  *launches = n;
  return ok();
}

OSPREY_API int osprey_set_stream(osprey_handle* h, void* hip_stream) {
  int rc = check_handle(h);
  if (rc) return rc;
  h->stream = (hipStream_t)hip_stream;
  return ok();
}

OSPREY_API int osprey_draft_destroy(osprey_handle* h) {
  if (!h) return ok();
  hipStreamSynchronize(h->stream);
  for (auto& r : h->timers) { hipEventDestroy(r.a); hipEventDestroy(r.b); }
  for (auto e : h->free_events) hipEventDestroy(e);
  delete h;
  return ok();
}

OSPREY_API const char* osprey_last_error(void) { return g_err.c_str(); }
