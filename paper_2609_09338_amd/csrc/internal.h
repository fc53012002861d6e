// Internal interface between the host runtime (osprey.cpp) and the kernels.
// Not part of the public C-ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace osp {

// Rows processed by one forward pass of the drafter body.
struct RowMeta {
  const int32_t* seq;    // [rows] batch index of each row (nullptr: row r is sequence r)
  const int32_t* pos;    // [rows] absolute position of each row
  const int32_t* tok;    // [rows] target token id of each row
  const int32_t* count;  // device-side row count (nullptr: max_rows)
  int max_rows;          // host-side upper bound on the row count
};

// Input of a GEMV-family launch: how row r, column c of the virtual input X is formed.
enum SrcKind {
  SRC_PLAIN = 0,  // X[r][c] = xin[r*ldx + c] (fp32)
  SRC_NORM = 1,   // X[r][c] = rmsnorm(xin[row(r)])[c] * gamma[c] (row(r) = gather[r] or r)
  SRC_QKV = 2,    // c < d: s[srow(r)][c]; else rmsnorm(x or embed[tok])[c-d] * gamma
  SRC_TAPS = 3,   // X[r][c] = taps[tap_row[r]*ldt + c] (weight dtype)
  SRC_PREP = 4,   // matrix-core passes: X[r][c] prepared as bf16 hi + lo pairs,
                  // c < seg from (xs_hi, xs_lo) row r, else (xa_hi, xa_lo) row gather[r] or r
  SRC_SWIGLU = 5, // matrix-core passes of <= 64 rows: X[r][c] = silu(g) u with g, u the sums of
                  // the gate/up K-split partials part_in[k][r][c] and part_in[k][r][Kd + c]
  SRC_ATTN = 6,   // X[r][c] = the attention output of row r, head c / hd, merged from its
                  // context splits (attn_part) on staging: matrix-core passes of <= 64 rows,
                  // and the single-row vector O projection
  SRC_QKV_PICK = 7, // SRC_QKV of layer 0 for one sequence whose token the kernel draws itself
                    // from the previous LM head's records and logits (GemvArgs::pick)
};
constexpr int kAttnMergeMaxSplit = 8;   // SRC_ATTN: splits per row (bound; else a merge kernel)
enum EpiKind {
  EPI_STORE = 0,   // y[r][n] = acc
  EPI_RESID = 1,   // y[r][n] += acc
  EPI_SWIGLU = 2,  // y[r][n] = silu(acc_gate) * acc_up (two weight matrices)
  EPI_LOGITS = 3,  // logits with -inf for unmapped rows + per-block softmax statistics
};

// Statistics of one drafter logit row at the temperature its draft was drawn at:
// S = sum exp((l - M) / T_d) over mapped rows (T_d = 0: unused), M the max and am the
// lowest argmax row (-1: every row masked).
struct QStat {
  double S;
  float M;
  int am;
};

// The draft of step k of sequence r, drawn where the next step consumes it instead of
// by the sampling kernel (pick.h): in every block of the single sequence's layer-0 QKV
// GEMV (SRC_QKV_PICK, r = 0), or in row r's block of the matrix-core body's row
// preparation (RowArgs::pick).  Pointers are those of sequence 0 at step k; sequence
// r's are r strides on.  One block writes each draft out as the sampling kernel would.
struct PickArgs {
  const float* part;        // the LM head's records (nblk <= kPickMaxRecords per row)
  long ld_part;
  int nblk;
  int blk_rows;             // logits per record
  const float* logits;      // the rows' logits [V]
  long ld_logits;
  int V;
  const int32_t* d2t;
  const float* temp;        // [r] the sequence's temperature
  const float* u;           // the step's uniform
  int ld_u;
  int k;
  int32_t* draft;           // the step's draft slot (workspace)
  int ld_draft;
  int32_t* draft_out;       // the caller's copy of it (nullable)
  int ld_draft_out;
  int32_t* ar_tok;          // [r] next AR token / position (position = committed + k)
  int32_t* ar_pos;
  const int32_t* committed;
  QStat* qstat;             // the step's row statistics (nullable)
  int ld_qstat;
};
constexpr int kPickMaxRecords = 2048;   // 256 threads x 8 records

struct GemvArgs {
  int max_rows;
  const int32_t* count;     // device row count (nullable)
  // input
  const float* xin;         // fp32 rows (PLAIN, NORM, QKV token part)
  int ldx;
  const int32_t* gather;    // NORM/QKV: input row index per output row (nullable)
  const float* s;           // QKV: conditioning rows
  int lds;
  const int32_t* s_gather;  // QKV: conditioning row per output row (nullable)
  const void* embed;        // QKV layer 0: embedding table (weight dtype); x = embed[tok[r]]
  const int32_t* tok;
  int vocab_embed;
  float* x_out;             // QKV layer 0: where to materialise x = embed[tok] (by block 0)
  const void* gamma;        // norm gain (weight dtype)
  float eps;
  int d_norm;               // width of the normalised segment
  const void* taps;         // TAPS: [rows][ldt] weight dtype
  const int32_t* tap_row;
  long ldt;
  int Kd;                   // input width
  // weights [N][Kd] row-major
  const void* w0;
  const void* w1;           // SWIGLU: up matrix
  int N;
  // output
  float* y;
  int ldy;
  // logits epilogue
  const int32_t* d2t;       // [N]
  const float* temp;        // [B] temperature per sequence
  const int32_t* row_seq;   // batch index of output row r (nullable: r; the matrix-core LM head
                            // takes row r as sequence r)
  long ld_logits;           // stride between rows of y for logits
  float* part;              // [rows][nblk][4]: max, sumexp, argmax, unused
  int nblk;
  float* split_buf;         // matrix-core K-split partials [split][max_rows][N] (SwiGLU: 2 N)
  // SRC_PREP inputs (bf16 hi / lo pairs)
  const uint16_t* xs_hi;
  const uint16_t* xs_lo;
  int ld_xs;
  int seg;                  // columns [0, seg) come from xs, the rest from xa
  const uint16_t* xa_hi;
  const uint16_t* xa_lo;
  int ld_xa;
  // SRC_SWIGLU inputs: gate/up partial sums, split k row r at part_in + k * part_in_split + r * ld_in
  const float* part_in;
  int ks_in;
  long part_in_split;
  int ld_in;
  // SRC_ATTN inputs: attention partials [rows][Kd / attn_hd heads][attn_nsplit][attn_hd + 2]
  // (max, sum, unnormalised output per split); splits past pos[r] / attn_split_len hold
  // nothing for row r
  const float* attn_part;
  const int32_t* attn_pos;
  int attn_nsplit;
  int attn_split_len;
  int attn_hd;
  // SRC_QKV_PICK: the draft pick of the step; SK_NORM LM head: where block 0 also copies
  // its fp32 input row (the fed-back hidden state, so that no sampling kernel need copy it)
  PickArgs pick;
  float* fb_out;
  uint32_t* err;
};
constexpr int kMaxKSplit = 16;

void launch_gemv(int wdtype, SrcKind src, EpiKind epi, const GemvArgs& a, hipStream_t st);
// Single-row O projection + residual whose input row is the attention output merged from
// its context splits while the kernel stages it (attn_* fields; bf16 weights, one row,
// Kd = heads x hd <= 2048, at most 16 heads and 20 splits: gemv_attn_supported).
bool gemv_attn_supported(int wdtype, int rows, int Kd, int hd, int n_split);
void launch_gemv_attn_resid(const GemvArgs& a, hipStream_t st);
// Layer-0 expanded QKV of a single sequence that draws its own token (SRC_QKV_PICK; bf16
// weights, one row, a.pick.nblk <= kPickMaxRecords: gemv_pick_supported).
bool gemv_pick_supported(int wdtype, int rows, int nblk);
void launch_gemv_qkv_pick(const GemvArgs& a, hipStream_t st);

// Matrix-core GEMM for passes of several rows of bf16 weights: src SRC_TAPS or
// SRC_PREP; epi EPI_STORE or EPI_SWIGLU (K-split partial sums into split_buf, summed
// by the row kernels below) or EPI_LOGITS.  Returns the number of K splits written.
int launch_gemm(SrcKind src, EpiKind epi, const GemvArgs& a, hipStream_t st);
// True when a pass of `rows` rows takes the matrix-core path.
bool gemm_use_mfma(int wdtype, int rows);
int gemm_rows_per_block(EpiKind epi);

// LM head on the matrix cores for 1..64 rows per pass (inputs: RMSNorm_final(x),
// rows gathered through `gather`).  One softmax record
// per wavefront and row covers blk_rows consecutive logits; nblk records per row.
struct LmPlan {
  int mt;        // M tiles of 16 rows
  int grid;      // blocks
  int T;         // 16-row weight tiles per wavefront
  int nblk;      // records per row
  int blk_rows;  // logits per record (16 T)
};
constexpr int kLmMaxRows = 64;
LmPlan lm_head_plan(int rows, int N, int n_cu);
// The head's weights a.w0 are the packed copy that launch_pack_head writes, of the
// [N][Kd] bf16 matrix with N = a.N and Kd = a.Kd.
// norm_in: inputs are the fp32 rows xin (ldx, gathered), normalised with gamma / eps
// in the kernel (one row of at most 4096 columns: lm_head_norm_in_supported); else
// prepared pairs xa_hi / xa_lo.  Returns false, launching nothing, for an unsupported
// norm_in shape.
bool lm_head_norm_in_supported(int rows, int Kd);
bool launch_lm_head(const GemvArgs& a, const LmPlan& p, bool norm_in, hipStream_t st);
// Packed head: [ceil(N / 16) tiles][ceil(Kd / 256) units][8 k steps][64 lanes][8] bf16,
// lane (r, g) of step s of unit u in tile t holding row 16 t + r, columns
// 256 u + 8 g + 32 s .. + 8 (zero past N or Kd): the order in which the matrix cores
// take the weights.  packed_head_bytes: its size; launch_pack_head fills it from the
// row-major [N][Kd] matrix w (Kd a multiple of 8), on stream st.
long packed_head_bytes(int N, int Kd);
void launch_pack_head(const void* w, int N, int Kd, void* packed, hipStream_t st);

// Projections of passes of at most kLmMaxRows rows on the same streaming kernel:
// src SRC_PREP (pairs; [xs ; xa] when seg > 0), SRC_TAPS, or SRC_SWIGLU (the down
// projection forms silu(gate) * up from the gate/up partials itself); with w1 set, the up
// matrix supplies rows [N, 2N).  Writes K-split partial sums to
// split_buf[split][max_rows][N or 2N]; returns the number of splits.
int launch_skinny(SrcKind src, const GemvArgs& a, hipStream_t st);
int skinny_splits(int rows, int Kd);

// Row kernels of the matrix-core path: one block per row (SwiGLU: per column group).
struct RowArgs {
  int max_rows;
  const int32_t* count;     // device row count (nullable: max_rows)
  int W;                    // row width
  const float* part;        // partial sums: split k, row r at part + (k * max_rows + r) * ldp
  int ks;
  int ldp;
  float* x;                 // residual rows [max_rows][W]
  const void* gamma;        // RMSNorm gain (bf16)
  float eps;
  uint16_t* out_hi;         // next product's input, bf16 hi / lo [max_rows][W]
  uint16_t* out_lo;
  // prologue of a pass (conditioning segment + embedding)
  const float* s_src;       // conditioning rows (nullable: summed from part)
  uint16_t* s_hi;
  uint16_t* s_lo;
  const void* embed;
  const int32_t* tok;
  int vocab_embed;
  // (prep) pick.part non-null: row r's token is drawn here (PickArgs), not read from tok;
  // the conditioning rows s_src may then be the rows x that this kernel overwrites
  PickArgs pick;
};
// s = sum of partials or s_src -> (s_hi, s_lo); x = embed[tok]; out = rmsnorm(x) * gamma.
void launch_rows_prep(const RowArgs& a, hipStream_t st);
// x += sum of partials; out = rmsnorm(x) * gamma.
void launch_rows_resid_norm(const RowArgs& a, hipStream_t st);
// out = silu(sum of gate partials) * sum of up partials (columns [0, W) and [W, 2 W)).
void launch_rows_swiglu(const RowArgs& a, hipStream_t st);
// Partition of the N weight rows of a launch: each wavefront owns rows_per_wave
// consecutive rows; `waves` wavefronts carry rows (the logits epilogue writes
// one statistics record per wavefront).
struct GemvShape {
  int rows_per_wave;
  int waves;
};
constexpr int kGemvMaxWaves = 4096;
GemvShape gemv_shape(int wdtype, EpiKind epi, int rows, int N, int Kd);

// Attention.
struct AttnArgs {
  RowMeta rows;
  const int32_t* cu;        // [B+1] rows of sequence b are [cu[b], cu[b+1]) (nullable: [b, b+1))
  const int32_t* bslot;     // [B] slot of sequence b
  int slot0;                // the slot of sequence 0 when B == 1 (no load); -1: bslot
  int B;
  int rows_per_seq;         // host bound on the rows of one sequence in this pass
  const float* qkv;         // [rows][qkv_w] raw projections (split 0 of qkv_ks partials)
  int qkv_w;
  int qkv_ks;               // K-split partials to sum on load (1: plain rows)
  long qkv_split;           // elements between splits
  const void* q_norm;
  const void* k_norm;
  int qk_norm;
  float eps;
  const float* rope_cos;    // [max_seq][hd/2]
  const float* rope_sin;
  int max_seq;
  void* kv;                 // pool base
  int layer, n_layers;
  const int32_t* block_table;  // [S][max_blocks]
  const int32_t* slot_nblocks; // [S]
  int max_blocks;
  int kv_block;
  int nq, nkv, hd;
  float scale;
  int n_split;              // grid splits; split sp covers positions [sp * split_len, + split_len)
  int split_len;            // tokens per split (multiple of 64; 0: ceil(n_ctx / n_split) per sequence)
  int kv_stream;            // bf16 pages read with non-temporal loads (a context larger than
                            // the last-level cache, streamed once per pass)
  const int32_t* items;     // work list from k_setup (b | slot << 8 | split << 16), *n_items entries;
  const int32_t* n_items;   // nullable: block y = split * B + b
  const float* q_prep;      // [rows][nq][hd] queries already normalised, rotated and scaled, with
                            // the new keys/values already in the cache (nullable: done here)
  float* part;              // [rows][nq][n_split][hd + 2]
  float* o;                 // [rows][nq*hd]
  uint16_t* o_hi;           // matrix-core path: o as bf16 hi / lo pairs instead (nullable)
  uint16_t* o_lo;
  uint32_t* err;
  // draft-tree passes (nullable): the rows are frontier nodes, cu groups each
  // sequence's rows (they share its context pages); rows.pos holds the last committed
  // position (the split attention reads the committed context only), tree_pos the
  // node's own position (RoPE); its keys/values go to the tree cache at slot
  // tree_node[r] instead of the pages, and the combine adds the row's attention over
  // tree_anc[r] (its ancestors' slots, then its own; -1 padded) as one more split
  const int32_t* tree_node;
  const int32_t* tree_anc;  // [rows][kMaxTreeDepth]
  const int32_t* tree_pos;
  void* tree_kv;            // [slot][n_layers][2][nkv][hd], bf16
  int tree_slots;           // slots of tree_kv
};
void launch_attention(int kvdtype, const AttnArgs& a, hipStream_t st);
// Matrix-core path: per row, sum the QKV split partials, normalise and rotate q
// and k, write q * (1/sqrt(hd)) to q_out and the new k, v into the cache.
void launch_rows_qkv(int kvdtype, const AttnArgs& a, float* q_out, hipStream_t st);
void launch_attn_combine(const AttnArgs& a, hipStream_t st);

// Sampling from the LM-head block statistics.
struct SampleArgs {
  int B;
  int k;                    // draft step index
  int K;
  const float* logits;      // row b at logits + b*ld_logits
  long ld_logits;
  int V;                    // drafter vocab
  const float* part;        // [B][nblk][4]
  int nblk;
  int blk_rows;             // logits per block
  const float* temp;        // [B]
  const float* u;           // [B][K]
  const int32_t* d2t;
  int32_t* drafts;          // [B][Kmax] workspace
  int ld_drafts;
  int32_t* drafts_out;      // optional caller copy [B][K]
  int32_t* ar_tok;          // [B] next AR token
  int32_t* ar_pos;          // [B] next AR position
  const int32_t* committed; // [B]
  const float* x;           // rows holding g
  const int32_t* gather;    // row of g for sequence b (nullable: b)
  int d;
  float* gfb;               // [B][d] fed-back hidden state
  QStat* qstat;             // [B][ld_qstat]: row statistics of step k at column k (nullable)
  int ld_qstat;
  // block drafting: one block per (sequence b, proposal k), k = blockIdx.y < K; the
  // records and logits of row b K + k; no autoregressive bookkeeping (set d = 0)
  int block;
};
void launch_sample(const SampleArgs& a, hipStream_t st);


// Step setup.
constexpr int kMaxBatch = 256;
struct SetupArgs {
  int B;
  int explicit_rows;        // 1: n_new given here, tokens from new_tokens; 0: pending
  int32_t slots[kMaxBatch];
  int32_t n_new[kMaxBatch];
  const int32_t* new_tokens;
  int taps_stride;          // rows between sequences in taps (0: packed)
  int K;
  int max_new;              // per-sequence bound on new rows
  int V_T;
  int32_t* slot_len;
  int32_t* pend_n;
  const int32_t* pend_tok;
  int pend_ld;
  const int32_t* slot_nblocks;
  int kv_block;
  // outputs
  int32_t* ing_seq;
  int32_t* ing_pos;
  int32_t* ing_tok;
  int32_t* ing_tap;
  int32_t* n_rows;
  int32_t* cu;
  int32_t* last_row;
  int32_t* committed;
  int32_t* bslot;
  int32_t* ar_pos;
  // attention work list (longest first) for splits of split_len positions, sized
  // for the longest context of the step (ingest + K - 1 draft positions)
  int split_len;
  int32_t* attn_items;      // [B * n_split]: b | slot << 8 | split << 16 (b, slot < kMaxBatch = 256)
  int32_t* attn_n_items;
  uint32_t* err;
  // block drafting (extra > 0): every sequence's rows are its new tokens, then `extra`
  // mask rows at the following positions with the anchor's (last new row's) tap row;
  // blk_gather[b (extra + 1) + k] is the anchor's row + k, blk_temp its temperature
  int extra;
  int32_t mask;
  const float* temp;        // [B]
  int32_t* blk_gather;
  float* blk_temp;
};
void launch_setup(const SetupArgs& a, hipStream_t st);

// Sets the message osprey_last_error() returns on this thread ("" with OSPREY_OK) and
// returns `code`.
int report_error(int code, const char* msg);

// Verification.
struct VerifyArgs {
  int B;
  int K;
  const float* target;      // [B][K+1][V_T]
  const float* draft;       // row (b, k) at draft + (b*ld_draft_b + k)*V_d
  long ld_draft_b;          // rows per sequence in draft
  const int32_t* drafts;    // row b at drafts + b*ld_drafts
  int ld_drafts;
  const float* temp;        // [B] target temperature T
  const float* temp_d;      // [B] temperature the drafts were drawn at (0: greedy, q one-hot)
  const float* u_acc;       // [B][K]
  const float* u_bonus;     // [B]
  const int32_t* d2t;
  const int32_t* t2d;
  int V_T, V_d;
  int chunk;                // elements per partial block
  int nchunk_t, nchunk_d;
  float* part;              // [B][(K+1)*nchunk_t + (qstat ? 0 : K*nchunk_d)][4]
  // drafter row statistics kept by the draft step's sampling kernel ([B][ld_qstat],
  // column k); nullptr: computed here from the drafter rows
  const QStat* qstat;
  int ld_qstat;
  double* res_part;         // [B][nchunk_t][2]: residual and p sums per chunk
  double* res_sub;          // [B][nchunk_t][kVSub][2]: the same per 64 consecutive ids
  int32_t* vstate;          // [B][4]: a, argmax of p_a, one-hot drafter row of q_a (T_d = 0)
  double* vstat;            // [B][4]: M_a, S_a (target), m_a, s_a (draft)
  int32_t* accept_len;
  uint8_t* accept_mask;
  int32_t* out_tokens;
  // draft trees (nullable: chain verification).  K is then the number of nodes, the
  // target has K + 1 rows per sequence (root, then node i at row i + 1), and there are
  // no drafter rows.
  const int32_t* tree_tok;  // [B][K] node tokens (target ids)
  const int32_t* tree_par;  // [B][K] parents (-1: the root)
  int32_t* tree_path;       // [B][K] out: the accepted path's nodes, then -1
  int32_t* tree_removed;    // [B][kMaxTreeNodes] tokens rejected at the node the bonus is drawn at
  // state update (stateful verify); nullable
  const int32_t* bslot;
  int32_t* pend_n;
  int32_t* pend_tok;
  int pend_ld;
  uint32_t* err;
};
void launch_verify(const VerifyArgs& a, hipStream_t st);
constexpr int kMaxTreeNodes = 64;
constexpr int kVSub = 64;     // 64-id sub-ranges per 4096-id verification chunk
void launch_verify_tree(const VerifyArgs& a, hipStream_t st);

// Draft-tree growth (see tree.hip).
constexpr int kMaxTopk = 8;           // children per node
constexpr int kMaxTreeDepth = 8;      // depths
constexpr int kMaxTreeProc = 64;      // frontier nodes run through the drafter per sequence
constexpr int kTkRecordRows = 64;    // tree passes of at least this many rows select from the records
constexpr int kTkMaxRecords = 2048;   // LM-head records per row a draft tree takes (V_d <= 2048 x 128)
constexpr int kMaxCand = 512;         // candidates per sequence (>= 8 + 7 x 64)
constexpr int kTkBlocks = 64;         // blocks per LM-head row in the candidate pass
struct TreeArgs {
  int B, k, depth, pass, n_nodes;
  int V;                    // LM-head rows
  const int32_t* d2t;
  const float* logits;      // rows of this pass at logits + r * ld_logits
  long ld_logits;
  float* cand_v;            // [rows][kTkBlocks][kMaxTopk] best (logit, row) pairs per block
                            // (nullptr: the step kernel selects from the records)
  int32_t* cand_r;
  const float* rec;         // LM-head records [rows][nblk][4] at temperature 1
  int nblk;
  int blk_rows;              // logits per record
  // candidates per sequence [B][kMaxCand], generation order
  int32_t* c_tok;
  int32_t* c_par;
  double* c_score;
  int32_t* c_depth;
  int32_t* c_slot;          // tree-cache slot once run through the drafter (else -1)
  int32_t* n_cand;          // [B]
  int32_t* front;           // [B][kMaxTopk] the candidates of the current pass's rows
  // the next pass's rows b * k + j
  int32_t* r_tok;
  int32_t* r_pos;
  int32_t* r_attpos;
  int32_t* r_node;
  int32_t* r_anc;           // [rows][kMaxTreeDepth]
  int32_t* r_cu;            // [B + 1] the rows of sequence b: [b k, (b + 1) k)
  float* r_s;               // [rows][d] conditioning input: the parent's hidden state
  const float* x;           // this pass's body output rows (root pass: the ingest rows)
  int d;
  const int32_t* last_row;
  const int32_t* committed;
  int32_t* out_tok;         // [B][n_nodes]
  int32_t* out_par;
  double* out_score;        // [B][n_nodes] (nullable)
};
void launch_tree_topk(const TreeArgs& a, int rows, hipStream_t st);
void launch_tree_step(const TreeArgs& a, hipStream_t st);
void launch_tree_final(const TreeArgs& a, hipStream_t st);

// KV helpers.
void launch_kv_append(int kvdtype, void* kv, const void* k, const void* v, int n_layers, int n,
                      int nkv, int hd, int kv_block, const int32_t* block_table, int slot,
                      int max_blocks, const int32_t* slot_len, int32_t* slot_len_out,
                      hipStream_t st);
void launch_set_len(int32_t* slot_len, int32_t* pend_n, int slot, int len, hipStream_t st);
void launch_fill_i32(int32_t* p, int32_t v, long n, hipStream_t st);

// KV pool layout: [block][layer][2 (k, v)][nkv][page], where the key page is
// [kv_block][hd] (token-major) and the value page [hd][kv_block] (transposed, so
// that the matrix-core attention reads 4 consecutive tokens of one dimension).
__host__ __device__ inline long kv_block_elems(int n_layers, int nkv, int kv_block, int hd) {
  return (long)n_layers * 2 * nkv * kv_block * hd;
}
__host__ __device__ inline long kv_k_at(int tok, int e, int hd) { return (long)tok * hd + e; }
__host__ __device__ inline long kv_v_at(int tok, int e, int kv_block) { return (long)e * kv_block + tok; }

}  // namespace osp
