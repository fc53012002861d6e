/*
 * osprey.h -- C ABI of the Osprey speculative draft-and-verify step on AMD
 * MI355X (gfx950).
 *
 * The operation (arXiv 2609.09338, "Osprey: Target-agnostic Pre-training Makes
 * Stronger Drafters in Speculative Decoding"):
 *
 *   Section 3.1  Given a committed prefix, a drafter proposes K draft tokens
 *                that the target model checks in one forward pass with the
 *                standard speculative-decoding acceptance rule, unchanged.
 *   Section 3.2  The drafter is a shallow stack of the first N pretrained
 *                blocks of a source LM with its embedding, final norm and LM
 *                head.
 *   Section 3.3  Target hidden states of three layers are concatenated and
 *                projected, c_t = W_c [h_low; h_mid; h_high] (Eq. 1).  Every
 *                attention layer's QKV projection is widened with extra
 *                columns, W~_qkv = [W^c  W_qkv], applied to [c_{t-1}; z_t]
 *                (Eq. 2-3): the newest target state available when token t is
 *                drafted is that of position t-1.  The embedding and LM head
 *                are aligned to the target vocabulary (Eq. 4).
 *   Section 3.4  At draft steps the drafter's own hidden state takes the place
 *                of the target state in its autoregressive context.
 *
 * draft_step ingests the newly committed tokens (each with the projected
 * target taps of the preceding position), then runs K autoregressive steps
 * over the drafter's paged KV cache, sampling one draft per step.  verify
 * applies the acceptance rule against the target's logits: greedy prefix match
 * at temperature 0; otherwise draft k is accepted with probability
 * min(1, p_k(d_k) / q_k(d_k)), the first rejected position is resampled from
 * the normalised residual max(0, p - q), and a fully accepted chain gets a
 * bonus token from p_K.
 *
 * Beyond the paper's top-1 chains: osprey_draft_tree and osprey_verify_tree grow
 * and verify draft trees (top-k > 1, the dynamic draft trees the related work in
 * the appendix names), and osprey_draft_block proposes K drafts from one pass over
 * an anchor and mask rows (the EAGLE-style interface of the DFlash ablation in the
 * appendix), verified by osprey_verify.
 *
 * Conventions for every call:
 *  - Pointers are DEVICE pointers unless marked (host).
 *  - Every call is asynchronous on the handle's HIP stream, except
 *    osprey_draft_init, osprey_seq_reset, osprey_seq_length,
 *    osprey_device_errors and osprey_kernel_time, which synchronise it.
 *  - No call allocates device memory.  The caller owns every device buffer
 *    (weights, KV pool, workspace, inputs, outputs); each must stay valid
 *    until the stream has finished the call that uses it, and weights, KV pool
 *    and workspace until osprey_draft_destroy.
 *  - All argument, shape, capacity and state checks happen before anything is
 *    enqueued: a call that returns an error has changed no state.  The message
 *    is available from osprey_last_error() (per host thread).
 *  - Conditions only the device can see (a token id out of range, a pending
 *    ingest with no verification before it, a position beyond the slot's
 *    blocks) never cause an out-of-bounds access: the kernel clamps or skips
 *    and raises a flag that osprey_device_errors() reports.
 *  - One host thread per handle.
 */
#ifndef OSPREY_H
#define OSPREY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OSPREY_OK = 0,
  OSPREY_E_INVALID = -1,     /* bad argument value or null pointer */
  OSPREY_E_SHAPE = -2,       /* sizes inconsistent with the configuration */
  OSPREY_E_CAPACITY = -3,    /* a sequence would outgrow its KV blocks or the workspace */
  OSPREY_E_STATE = -4,       /* call not allowed in the slot's current state */
  OSPREY_E_DEVICE = -5,      /* no usable GPU, or a HIP runtime error */
  OSPREY_E_UNSUPPORTED = -6  /* valid but not implemented (e.g. head_dim other than 64/128) */
} osprey_status;

typedef enum { OSPREY_F32 = 0, OSPREY_BF16 = 1 } osprey_dtype;

/* Drafter and pool shape.  Weights, norm gains, taps and the KV cache share
 * `dtype`; activations and logits are fp32 throughout. */
typedef struct {
  int32_t n_layers;       /* N retained blocks (Section 3.2) */
  int32_t d_model;        /* drafter width d (multiple of 64, at most 4096) */
  int32_t n_q_heads;
  int32_t n_kv_heads;     /* divides n_q_heads; query head h reads kv head h*n_kv/n_q */
  int32_t head_dim;       /* 64 or 128 */
  int32_t d_ffn;          /* SwiGLU width (multiple of 64) */
  int32_t vocab_draft;    /* V_d: LM-head rows */
  int32_t vocab_target;   /* V_T: embedding rows (indexed by target id) and verify width */
  int32_t target_hidden;  /* H: width of one target hidden-state tap (multiple of 8) */
  int32_t n_taps;         /* number of concatenated taps (3 in the paper, Eq. 1) */
  int32_t dtype;          /* osprey_dtype */
  int32_t qk_norm;        /* 1: per-head RMSNorm on q and k before RoPE (Qwen3 body) */
  float rms_eps;
  float rope_theta;
  int32_t max_batch;      /* sequences per call and number of slots (<= 256) */
  int32_t max_k;          /* largest K (<= 64) */
  int32_t max_seq_len;    /* largest position + 1; at most 262144 */
  int32_t kv_block;       /* tokens per KV page; must be 16 */
  int32_t kv_num_blocks;  /* pages in the pool */
  int32_t max_new_rows;   /* largest explicit ingest (prompt prefill) summed over the batch */
} osprey_config;

/* Per-layer weights, row-major, `dtype`.  w_qkv is [(n_q + 2 n_kv) head_dim][2 d]:
 * columns [0, d) multiply the conditioning input c (the expansion of Eq. 2),
 * columns [d, 2 d) the normalised token stream z.  Rows: q heads, k heads, v heads. */
typedef struct {
  const void* in_norm;    /* [d] */
  const void* w_qkv;      /* [(n_q + 2 n_kv) hd][2 d] */
  const void* q_norm;     /* [hd] (ignored when qk_norm == 0) */
  const void* k_norm;     /* [hd] */
  const void* w_o;        /* [d][n_q hd] */
  const void* post_norm;  /* [d] */
  const void* w_gate;     /* [d_ffn][d] */
  const void* w_up;       /* [d_ffn][d] */
  const void* w_down;     /* [d][d_ffn] */
} osprey_layer_weights;

typedef struct {
  const void* embed;       /* [V_T][d], indexed by target id (Section 3.3, Eq. 4) */
  const void* w_c;         /* [d][n_taps H] (Eq. 1) */
  const void* final_norm;  /* [d] */
  const void* lm_head;     /* [V_d][d] */
  const int32_t* d2t;      /* [V_d] target id of each LM-head row, -1 = none; injective */
  const osprey_layer_weights* layers;  /* (host) array [n_layers] of device pointers */
} osprey_weights;

typedef struct osprey_handle osprey_handle;

/* Arguments of osprey_draft_step.
 *
 * New rows: sequence b ingests n_b newly committed tokens (target ids) at
 * positions len_b .. len_b + n_b - 1, where len_b is the slot's cached length.
 *  - explicit: n_new (host, [batch]) gives n_b >= 1 and new_tokens (device) the
 *    tokens packed in batch order ([sum n_b]).
 *  - pending: n_new == NULL.  Each slot ingests the a + 1 tokens the last
 *    osprey_verify committed for it (accepted drafts + the resampled or bonus
 *    token), read on the device: no host synchronisation is needed.
 * taps holds one row of n_taps * H values (dtype) per new token: the target
 * hidden states of the PRECEDING position (Eq. 2-3 use c_{t-1}).  Row j of
 * sequence b is at row index b * taps_stride + j, or, with taps_stride == 0
 * (explicit mode only), at the packed index sum_{b'<b} n_b' + j.  Pending mode
 * needs taps_stride >= the previous K + 1 (the target's verify pass yields
 * K + 1 rows per sequence; the first a + 1 are used).  The conditioning input
 * of the very first position of a sequence is zero: pass a zero tap row.
 *
 * Drafting (K >= 1): draft k is drawn from softmax(l_k / T_b) over drafter
 * rows by inverse CDF with u_draft[b][k] (ascending row order; T_b == 0:
 * argmax, lowest row on ties) and emitted as the target id d2t[row].  Step
 * k >= 1 feeds draft k-1 with the previous step's last-layer hidden state
 * (before the final norm) as its conditioning input (Section 3.4).  K == 0
 * only ingests (prompt prefill) and leaves the slots READY.
 */
typedef struct {
  int32_t batch;
  int32_t K;                   /* 0 .. max_k */
  const int32_t* slots;        /* (host) [batch] distinct slot ids */
  const int32_t* n_new;        /* (host) [batch] or NULL (pending) */
  const int32_t* new_tokens;   /* [sum n_new] target ids (explicit mode) */
  const void* taps;            /* tap rows, dtype */
  int32_t taps_stride;         /* rows per sequence in taps, or 0 = packed */
  const float* temperature;    /* [batch], >= 0 */
  const float* u_draft;        /* [batch][K] uniforms in [0, 1) (may be NULL if all T == 0) */
  int32_t* draft_tokens;       /* [batch][K] out, target ids (may be NULL) */
  float* draft_logits;         /* [batch][K][V_d] out (may be NULL: kept in the workspace).
                                  If given, verify reads the drafter's rows from here: leave
                                  them untouched until osprey_verify has run. */
} osprey_step_args;

/* Drafter temperature.  The rule checks each draft against the distribution it
 * was actually drawn from: q_k = softmax(l_k / T_d) carried to target ids, with T_d
 * the draft temperature of the request, while p_k = softmax(target row / T).
 * T_d = 0 is greedy drafting, the top-1 chain of the paper's serving setup
 * (Section 4, inference settings; serving configuration in the appendix on
 * adaptation): q_k is one-hot at the drafter's argmax row (lowest row on ties),
 * draft k is accepted iff u_k < p_k(d_k), and a rejected position is redrawn
 * from p_a with d_a removed (target-only acceptance).  Draft with
 * osprey_draft_step at temperature T_d (0 for greedy) and pass the same values
 * as draft_temperature here: osprey_verify takes each drafter row's max and
 * normaliser from the draft step (computed there at its temperature) and reads
 * the drafter's logits only at the drafted entries and in row a.  With T == 0 the rule is the
 * greedy prefix match whatever T_d is. */

/* Arguments of osprey_verify (stateful: the drafts and drafter rows of the last
 * draft_step on exactly these slots in this order with this K).  The target's
 * logits are for the K + 1 positions after the committed prefix followed by
 * d_0 .. d_{k-1} (row k scores draft k; row K scores the bonus).
 * Outputs: a_b in [0, K]; mask[b][k] = 1 for k < a_b; out_tokens[b] holds
 * d_0 .. d_{a-1}, then the resampled (a < K) or bonus (a == K) token at index a,
 * then -1.  Each slot's cached length returns to its post-ingest value (the
 * draft positions are discarded) and its a + 1 committed tokens become the
 * pending ingest of the next draft_step. */
typedef struct {
  int32_t batch;
  int32_t K;
  const int32_t* slots;         /* (host) [batch] */
  const float* target_logits;   /* [batch][K + 1][V_T] fp32 */
  const float* temperature;     /* [batch] the target's temperature T (>= 0) */
  const float* u_accept;        /* [batch][K] */
  const float* u_bonus;         /* [batch] */
  int32_t* accept_len;          /* [batch] out */
  uint8_t* accept_mask;         /* [batch][K] out */
  int32_t* out_tokens;          /* [batch][K + 1] out */
  const float* draft_temperature; /* [batch] temperature the drafts were drawn at (the
                                  draft_step's `temperature`), or NULL: the same as
                                  `temperature`.  See "Drafter temperature" below. */
} osprey_verify_args;

/* Arguments of osprey_verify_rows: the same rule on caller-supplied drafts and
 * drafter logits, with no slot state involved. */
typedef struct {
  int32_t batch;
  int32_t K;
  const float* target_logits;   /* [batch][K + 1][V_T] */
  const float* draft_logits;    /* [batch][K][V_d]; rows with d2t == -1 are ignored */
  const int32_t* draft_tokens;  /* [batch][K] target ids */
  const float* temperature;     /* [batch] */
  const float* u_accept;        /* [batch][K] */
  const float* u_bonus;         /* [batch] */
  int32_t* accept_len;
  uint8_t* accept_mask;
  int32_t* out_tokens;
  const float* draft_temperature;  /* [batch] or NULL (= temperature), as in osprey_verify_args */
} osprey_verify_rows_args;

/* Draft trees (top-k > 1).  The paper serves with a top-k parameter of 1 (chains;
 * Section 4, inference settings); with top-k > 1 each node of the draft carries
 * the drafter's k most likely tokens as children (dynamic draft trees, among the
 * related drafters the paper discusses), and the target scores every node in one
 * pass.  Children are deterministic candidates, not samples, so the lossless rule
 * is target-only acceptance (as for greedy chains, "Drafter temperature" below)
 * applied to the children in turn: at a node with target distribution p, child c
 * is accepted iff u_accept[c] < p'(token_c), with p' = p without the tokens of the
 * children already rejected there, renormalised; the walk continues from an
 * accepted child; when none is accepted the next token is drawn from p' by
 * inverse CDF with u_bonus.  T = 0: the walk follows the child whose token is the
 * target's argmax (lowest id on ties), and the bonus is that argmax.
 *
 * Nodes 0..n_nodes-1 are in topological order: parents[i] = -1 for a child of the
 * root, otherwise an index < i; a parent outside [-1, i) makes node i unreachable
 * (device error bit 5).  Children are tried in index order.  Row 0 of
 * target_logits is the root (the position after the committed prefix), row i + 1
 * node i.  Limits: 0 <= n_nodes <= 64. */
typedef struct {
  int32_t batch;
  int32_t n_nodes;
  const float* target_logits;   /* [batch][n_nodes + 1][V_T] fp32 */
  const int32_t* tokens;        /* [batch][n_nodes] target ids */
  const int32_t* parents;       /* [batch][n_nodes] */
  const float* temperature;     /* [batch] the target's temperature (>= 0) */
  const float* u_accept;        /* [batch][n_nodes] node i's uniform, used when it is tried */
  const float* u_bonus;         /* [batch] */
  int32_t* accept_len;          /* [batch] out: accepted nodes on the path */
  int32_t* accept_path;         /* [batch][n_nodes] out: the path's node indices, then -1 */
  int32_t* out_tokens;          /* [batch][n_nodes + 1] out: the path's tokens, the bonus, then -1 */
} osprey_verify_tree_args;

/* Arguments of osprey_draft_tree: growing a draft tree instead of a chain.  The root
 * is each sequence's last committed row; its topk most likely drafter rows are the
 * depth-1 candidates, scored by their log-probability at temperature 1 (the drafter's
 * confidence).  At every further depth the frontier (the topk best candidates of the
 * previous depth; depth 1: all of them) runs through the drafter, each node at
 * position committed + its depth - 1 with its parent's hidden state as the
 * conditioning input (Section 3.4), attending to the committed context and to its own
 * ancestors only; its topk most likely rows become candidates scored with the
 * parent's score plus their log-probability.  The n_nodes best candidates (higher
 * score, then generation order) form the tree, listed in generation order (parents
 * before children) for osprey_verify_tree.  Ties in the drafter's logits go to the
 * lower row.  Limits: 2 <= topk <= min(8, max_k), 1 <= depth <= 8,
 * n_nodes <= min(64, topk + (depth - 1) topk^2); bf16 weights. */
typedef struct {
  int32_t topk;
  int32_t depth;
  int32_t n_nodes;
  int32_t* tokens;              /* [batch][n_nodes] out: target ids */
  int32_t* parents;             /* [batch][n_nodes] out: -1 for the root's children, else an
                                   earlier node */
  double* scores;               /* [batch][n_nodes] out, optional (NULL: not written): each
                                   node's score, the sum of the log-probabilities on its path */
} osprey_tree_args;

/* Host-only check of a configuration.  Returns OSPREY_OK or the first problem. */
int osprey_config_validate(const osprey_config* cfg);

/* Bytes of the KV pool: kv_num_blocks pages of [n_layers][2][n_kv][kv_block * hd] (dtype);
 * within a page keys are token-major [kv_block][hd] and values dimension-major
 * [hd][kv_block].
 * Returns 0 for an invalid configuration. */
size_t osprey_kv_bytes(const osprey_config* cfg);

/* Bytes of device workspace the library needs (activations, statistics, slot state,
 * and for bf16 weights a copy of the LM head, [V_d][d] bf16 rounded up to 16 rows and
 * 256 columns).  Returns 0 for an invalid configuration. */
size_t osprey_workspace_bytes(const osprey_config* cfg);

/* Validate, carve the caller's KV pool and workspace (256-byte aligned), copy
 * the vocabulary map and build its inverse (d2t must be injective on mapped
 * rows and map at least one row), upload the RoPE table (computed in float64)
 * and reset every slot to EMPTY.  bf16 weights: the LM head is copied into the
 * workspace in the order the matrix cores take it, and later calls read that copy
 * (a change to w->lm_head after this call is not seen).  hip_stream is a hipStream_t (NULL: the null
 * stream).  Synchronises the stream.  *out receives the handle (host). */
int osprey_draft_init(const osprey_config* cfg, const osprey_weights* w, void* kv_pool,
                      size_t kv_bytes, void* workspace, size_t ws_bytes, void* hip_stream,
                      osprey_handle** out);

/* Give `slot` an empty sequence whose KV pages are block_ids (host, n_blocks
 * physical page ids < kv_num_blocks; capacity n_blocks * kv_block positions).
 * Pages must not be shared with another live slot.  Any state -> READY. */
int osprey_seq_reset(osprey_handle* h, int32_t slot, const int32_t* block_ids, int32_t n_blocks);

/* Append n positions of precomputed keys/values (post-RoPE, as the cache
 * stores them) to a READY slot, for every layer: k, v are [n_layers][n][n_kv][hd]
 * (dtype).  Fills a synthetic context without running the drafter. */
int osprey_kv_append(osprey_handle* h, int32_t slot, int32_t n, const void* k, const void* v);

/* Shorten a READY slot to `length` cached positions (<= its length) and drop
 * any pending ingest. */
int osprey_seq_truncate(osprey_handle* h, int32_t slot, int32_t length);

/* Synchronise and read the exact cached length of a slot (host out). */
int osprey_seq_length(osprey_handle* h, int32_t slot, int32_t* length);

/* Ingest the new rows and propose K drafts per sequence (see osprey_step_args).
 * State: READY (explicit) or VERIFIED (pending) -> DRAFTED (K >= 1) / READY (K == 0). */
int osprey_draft_step(osprey_handle* h, const osprey_step_args* a);

/* Ingest the new rows (as osprey_draft_step, with a->K = 0) and grow a draft tree
 * (see osprey_tree_args).  The tree's keys and values never enter the slot's pages:
 * the slot ends READY with the ingested rows committed, and the next call ingests the
 * tokens osprey_verify_tree accepted (explicit new_tokens).  State: READY or VERIFIED
 * -> READY. */
int osprey_draft_tree(osprey_handle* h, const osprey_step_args* a, const osprey_tree_args* t);

/* Block drafting (the EAGLE-style target interface of the DFlash ablation, appendix):
 * the new rows are ingested as osprey_draft_step does (the last new token of a
 * sequence is its block's anchor) and, in the same pass of the drafter, K - 1 mask
 * rows follow each sequence's new rows (token mask_token at positions committed ..
 * committed + K - 2), each with the anchor's conditioning input (the target feature
 * is taken once at the anchor and broadcast), attending causally to the cache; draft
 * k is drawn from block row k's logits (row 0: the anchor) at temperature[b] with
 * u_draft[b][k], independently of the other drafts.  The mask rows' cache entries lie
 * past the committed length and are rolled back like the chain's draft positions.
 * Arguments, outputs (draft_tokens, draft_logits [batch][K][V_d]), state transitions
 * and the following osprey_verify are those of osprey_draft_step with K drafts.
 * A pass holds sum_b (n_b + K - 1) rows: the workspace must hold them (the config's
 * max_new_rows >= batch x 2 max_k covers pending steps), else OSPREY_E_CAPACITY.
 * Limits: 2 <= K <= max_k; bf16 weights; 0 <= mask_token < vocab_target (else
 * OSPREY_E_INVALID, nothing enqueued). */
int osprey_draft_block(osprey_handle* h, const osprey_step_args* a, int32_t mask_token);

/* Verify the last drafts (see osprey_verify_args).  State: DRAFTED -> VERIFIED. */
int osprey_verify(osprey_handle* h, const osprey_verify_args* a);

/* Stateless verification of caller-supplied drafts (see osprey_verify_rows_args). */
int osprey_verify_rows(osprey_handle* h, const osprey_verify_rows_args* a);

/* osprey_verify_rows without a handle and without device memory of the caller's: for
 * callers that cannot allocate (code under HIP graph capture, serving loops and
 * harnesses that forbid allocation).  The same rule and kernels as
 * osprey_verify_rows on the same arguments; d2t [vocab_draft] (device) maps drafter
 * rows to target ids (-1 = none; injective, as osprey_draft_init requires: entries
 * outside [0, vocab_target) are treated as unmapped, and a target id several rows
 * map to takes the largest of them).  Every scratch buffer lives in a fixed device
 * array of the library (about 7.4 MB per GPU, held until the process ends), which
 * bounds a call: batch <= 64, K <= 16, both vocabularies <= 262144 (else
 * OSPREY_E_CAPACITY, nothing enqueued).  Enqueued on hip_stream (a hipStream_t; NULL:
 * the null stream).  Calls on one GPU share that array: calls that overlap on one
 * GPU (other streams, other host threads) race.  Make the first call on each device
 * outside graph capture (it looks the array's address up).  A draft id outside
 * [0, V_T) is rejected and not reported (there is no handle to report it to). */
int osprey_verify_rows_static(const osprey_verify_rows_args* a, const int32_t* d2t,
                              int32_t vocab_draft, int32_t vocab_target, void* hip_stream);

/* Stateless verification of a caller-supplied draft tree (see
 * osprey_verify_tree_args).  No slot state is involved. */
int osprey_verify_tree(osprey_handle* h, const osprey_verify_tree_args* a);

/* One steady-state iteration as a HIP graph.  At batch 1 an iteration is a chain of
 * about a hundred dependent kernels, each short enough that its launch is a large
 * part of its cost; the drafter's latency is what its shallow depth buys (Section
 * 3.2), so the iteration can be captured once and replayed with one launch.
 *
 * osprey_graph_capture records, without running it, a pending-mode draft call
 * (osprey_draft_step, or osprey_draft_block when mask_token >= 0) followed by
 * osprey_verify with these arguments, into a graph (osprey_graph, host handle).
 * The graph reads and writes exactly the buffers the arguments name, at these
 * addresses: write each iteration's inputs (taps, temperatures, uniforms, target
 * logits) there before launching it, stream-ordered.  Requirements: step->n_new ==
 * NULL (the ingest is the tokens the last verification committed), the same batch,
 * K and slots in both argument sets, taps_stride >= K + 1, kernel timing off, and a
 * stream other than the null stream (osprey_set_stream).  Attention is planned for
 * contexts up to max_context positions (<= max_seq_len): every launch must keep each
 * slot's committed length + pending tokens + K - 1 within it.  Capturing changes no
 * state and enqueues nothing; errors are those of the two calls.
 *
 * osprey_graph_launch enqueues one iteration on the handle's stream: the same
 * checks as the two calls (every slot VERIFIED, capacity within its pages and
 * max_context, else OSPREY_E_STATE / OSPREY_E_CAPACITY with nothing enqueued) and
 * the same state transitions (the slots end VERIFIED).  The graph stays valid
 * across launches; osprey_graph_destroy releases it (after the stream has finished
 * with it). */
typedef struct osprey_graph osprey_graph;
int osprey_graph_capture(osprey_handle* h, const osprey_step_args* step, int32_t mask_token,
                         const osprey_verify_args* verify, int32_t max_context,
                         osprey_graph** out /* (host) */);
int osprey_graph_launch(osprey_handle* h, osprey_graph* g);
int osprey_graph_destroy(osprey_graph* g);

/* Synchronise, read and clear the device error flags (host out):
 * bit 0 an ingest row count outside [1, max new rows] (pending without verify),
 * bit 1 a token id outside [0, V_T), bit 2 a sequence beyond its KV pages,
 * bit 3 a KV write beyond the slot's pages, bit 4 a draft id outside [0, V_T),
 * bit 5 a tree node whose parent is not an earlier node or the root. */
int osprey_device_errors(osprey_handle* h, uint32_t* flags);

/* Kernel timing for roofline reports.  `families` is a bit mask: bit f enables HIP
 * event timing of family f on the handle's stream (0 disables; every call clears
 * the records).  Families: 0 = LM head (final norm + vocabulary GEMV + softmax
 * statistics), 1 = attention (split pass + split merge), 2 = verify (all its
 * kernels), 3 = a whole draft_step, 4 = expanded-QKV GEMV.  Each event adds a few
 * microseconds of idle time to the stream, so time few families at once.  A timed
 * LM head, and a timed attention, runs 8 times back to back between its events
 * (the same outputs again), so its events' overhead is shared by 8 launches.
 * osprey_kernel_time synchronises and returns the summed duration (ms) and the
 * number of launches since the last osprey_kernel_timing call. */
int osprey_kernel_timing(osprey_handle* h, int32_t families);
int osprey_kernel_time(osprey_handle* h, int32_t family, double* total_ms, int64_t* launches);

/* Change the stream subsequent calls are enqueued on. */
int osprey_set_stream(osprey_handle* h, void* hip_stream);

/* Release the host handle (device buffers stay the caller's). */
int osprey_draft_destroy(osprey_handle* h);

/* Message of the last failed call on this host thread ("" if none). */
const char* osprey_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* OSPREY_H */
