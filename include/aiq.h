/*
 * aiq.h -- unified AI-query execution on one gfx950 GPU: C ABI.
 *
 * One call runs a hybrid SQL + LLM query as a single device-resident
 * pipeline on one HIP stream:
 *
 *   FROM      columnar table already in device memory            (Table 1, FROM)
 *   WHERE     conjunction of integer or fp32 column predicates -> stable
 *             selection (Table 1, WHERE)
 *   JOIN      optional inner PK-FK hash join with a filtered build table
 *             (the reviews-JOIN-movies workload of Section 4)
 *   AI_IF     gather + pack the selected rows' token lists into a variable-
 *             length batch, decoder-only transformer prefill, last-position
 *             label logits, strict "yes > no" or argmax decision
 *             (Table 1, AI_IF; Figure 2)
 *   aggregate COUNT, kept row ids, or GROUP BY key AVG(label)/COUNT(*)
 *             (Table 1, SELECT SUM as a masked reduction; Figure 2)
 *
 * Nothing is copied between host and device inside aiq_run: only the caller
 * reads the (small) outputs afterwards (Section 3.3, H2D boundary
 * consolidation).  Shapes stay data-dependent on the device: survivor counts,
 * token counts and sequence lengths are never read back, and the selection
 * skips non-matching rows before the model runs (Section 5, the dynamic-shape
 * and dynamic data-skipping roadmap items).
 *
 * Conventions
 *  - Every pointer documented as "device" is a device address owned by the
 *    caller; the library never allocates, frees or retains device memory.
 *  - Pointers documented as "host" are read during the call only, except
 *    that aiq_plan_create copies everything it needs into the plan.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Calls that take a
 *    stream only enqueue work; they never synchronise the device and never
 *    copy data to or from the host.
 *  - Host-detectable errors return a negative aiq_status and enqueue nothing.
 *    Errors that only the device can see (token id out of range, duplicate
 *    build key, capacity exceeded, ...) set bits of the device status word
 *    (aiq_out.scalars[AIQ_S_STATUS]); after such a bit is set the other
 *    outputs are unspecified.
 *  - No C++ exception crosses this interface.
 *  - A plan is immutable after creation and holds host metadata only; one
 *    plan may be used by concurrent calls provided each call has its own
 *    workspace and outputs.
 */
#ifndef AIQ_H
#define AIQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AIQ_ABI_VERSION 6

typedef enum aiq_status {
  AIQ_OK = 0,
  AIQ_EINVAL = -1,        /* null pointer, bad enum, inconsistent shapes      */
  AIQ_EUNSUPPORTED = -2,  /* valid request that this build does not implement */
  AIQ_ENOSPC = -3,        /* workspace or capacity too small                  */
  AIQ_EHIP = -4,          /* a HIP runtime call or kernel launch failed       */
  AIQ_ENOMEM = -5         /* host allocation of the plan failed               */
} aiq_status;

/* element types of columns and weights */
typedef enum aiq_dtype {
  AIQ_I8 = 1, AIQ_I16 = 2, AIQ_I32 = 3, AIQ_F32 = 4, AIQ_BF16 = 5, AIQ_F16 = 6
} aiq_dtype;

/* predicate operators: `col op k`, or `col IN (set)` */
typedef enum aiq_op {
  AIQ_LT = 0, AIQ_LE = 1, AIQ_GT = 2, AIQ_GE = 3, AIQ_EQ = 4, AIQ_NE = 5, AIQ_IN = 6
} aiq_op;

typedef enum aiq_act { AIQ_ACT_GELU_ERF = 1, AIQ_ACT_SWIGLU = 2 } aiq_act;
typedef enum aiq_decision { AIQ_DECIDE_BINARY_GT = 1, AIQ_DECIDE_ARGMAX = 2 } aiq_decision;
typedef enum aiq_agg {
  AIQ_AGG_COUNT = 1,             /* COUNT(*) of kept rows (+ their ids)                  */
  AIQ_AGG_AVG_LABEL_COUNT_BY = 2,/* GROUP BY probe column: COUNT(*), SUM/AVG(label)      */
  AIQ_AGG_COUNT_BY_PAYLOAD = 3,  /* GROUP BY joined build payload: COUNT(*) of kept rows */
  AIQ_AGG_SUM_F32 = 4            /* SUM of an fp32 probe column over the kept rows, in
                                    fp64 (+ COUNT and ids); Table 1 SUM row, Figure 2     */
} aiq_agg;
typedef enum aiq_logits_mode { AIQ_LOGITS_LABELS = 1, AIQ_LOGITS_FULL_VOCAB = 2 } aiq_logits_mode;

/* device status bits (aiq_out.scalars[AIQ_S_STATUS]) */
#define AIQ_DEV_TOKEN_RANGE 0x01  /* a token id outside [0, vocab): treated as 0   */
#define AIQ_DEV_DUP_KEY     0x02  /* duplicate key among the passing build rows     */
#define AIQ_DEV_HASH_FULL   0x04  /* hash table overflow, or an INT32_MIN build key  */
#define AIQ_DEV_IDS_CAP     0x08  /* more kept rows than aiq_out.ids_cap            */
#define AIQ_DEV_GROUP_RANGE 0x10  /* group key outside [0, n_group_keys): skipped   */
#define AIQ_DEV_LIST_LEN    0x20  /* a row's list longer than max_list_len          */
#define AIQ_DEV_GROUP_CAP   0x40  /* more groups than aiq_out.grp_cap               */
#define AIQ_DEV_PAIR_CAP    0x80  /* more candidate pairs than aiq_query.max_pairs:
                                     the pairs past it are dropped                  */
#define AIQ_DEV_SCAN_WAIT   0x100 /* a compaction block waited too long for an
                                     earlier block's totals: outputs invalid       */

/* indices into aiq_out.scalars (int64, device) */
#define AIQ_S_SELECTED 0   /* rows passing WHERE (and the join)                      */
#define AIQ_S_KEPT     1   /* rows kept after the AI decision (argmax: = selected)   */
#define AIQ_S_TOKENS   2   /* total prefill tokens (prefix + row tokens)             */
#define AIQ_S_STATUS   3   /* OR of AIQ_DEV_* bits                                   */
#define AIQ_S_GROUPS   4   /* number of non-empty groups written                     */
#define AIQ_S_PAIRS    5   /* pairs mode: candidate pairs classified (<= max_pairs)  */
#define AIQ_N_SCALARS  8

#define AIQ_MAX_PREDS 8
#define AIQ_MAX_IN_SET 32
#define AIQ_MAX_PREFIX 64
#define AIQ_MAX_LABELS 8
#define AIQ_MAX_GEN 512
#define AIQ_MAX_LIKE 16

/* One fixed-width column: `data` is a device array of n_rows elements,
 * 16-byte aligned (predicates read it in 16-byte vectors; a misaligned
 * column is rejected with AIQ_EINVAL at plan creation). */
typedef struct aiq_col {
  const void* data;
  int32_t dtype;          /* AIQ_I8, AIQ_I16 or AIQ_I32 */
} aiq_col;

/*
 * A columnar table in device memory.  The probe table also carries one list
 * column (the text of each row as token ids): row r owns
 * list_tokens[list_offsets[r] .. list_offsets[r+1]).
 */
typedef struct aiq_table {
  int64_t n_rows;
  int32_t n_cols;
  const aiq_col* cols;           /* host array of n_cols descriptors            */
  const int64_t* list_offsets;   /* device [n_rows + 1], non-decreasing, or NULL */
  const int32_t* list_tokens;    /* device                                      */
  int64_t n_list_tokens;         /* host: list_offsets[n_rows] - list_offsets[0] */
  int32_t max_list_len;          /* host: declared bound on any row's list length */
} aiq_table;

/*
 * One predicate atom: cols[col] op k, or cols[col] IN set[0..n_set).
 * Integer columns compare exactly with k; an AIQ_F32 column compares its
 * value, widened to fp64, with fk under IEEE rules (NaN fails every
 * comparison but NE); IN on an AIQ_F32 column is AIQ_EUNSUPPORTED.
 */
typedef struct aiq_pred {
  int32_t col;
  int32_t op;                    /* aiq_op */
  int64_t k;                     /* integer columns */
  int32_t n_set;
  int64_t set[AIQ_MAX_IN_SET];
  double fk;                     /* AIQ_F32 columns */
} aiq_pred;

/*
 * Decoder layer weights, device pointers.  Matrices are row-major [out, in]
 * in the model's weight dtype; norm gains are float32 [d_model].
 *   wq [n_heads*hd, d]   wk, wv [n_kv_heads*hd, d]   wo [d, n_heads*hd]
 *   SwiGLU:  w_gate, w_up [d_ff, d], w_down [d, d_ff]
 *   GELU:    w_gate = W1 [d_ff, d], w_up unused (NULL), w_down = W2 [d, d_ff]
 */
typedef struct aiq_layer {
  const float* attn_norm;
  const void* wq; const void* wk; const void* wv; const void* wo;
  const float* ffn_norm;
  const void* w_gate; const void* w_up; const void* w_down;
} aiq_layer;

typedef struct aiq_model {
  int32_t n_layers, d_model, n_heads, n_kv_heads, d_ff, vocab;
  int32_t act;                   /* aiq_act */
  int32_t wdtype;                /* AIQ_F32, AIQ_BF16 or AIQ_F16: storage type of the
                                    weights and the compute type of the projections
                                    (16-bit types run on MFMA with fp32 accumulation;
                                    activations fed to the projections use the same
                                    16-bit type, the residual stream stays fp32) */
  double rope_theta;             /* rotary base, e.g. 10000 */
  double norm_eps;               /* RMSNorm epsilon, e.g. 1e-5 */
  const void* emb;               /* device [vocab, d] */
  const aiq_layer* layers;       /* host array of n_layers */
  const float* final_norm;       /* device [d] */
  const void* lm_head;           /* device [vocab, d] */
} aiq_model;

typedef struct aiq_query {
  int32_t n_pred;
  aiq_pred preds[AIQ_MAX_PREDS];       /* conjunction over probe columns */
  /* optional inner join probe.cols[probe_key_col] = build.cols[build_key_col]
     with the build rows passing build_preds; the build key must be unique
     among passing rows and must not be INT32_MIN (the empty-slot value; such
     a build row sets AIQ_DEV_HASH_FULL, a probe key INT32_MIN matches
     nothing).  build_payload_col is carried to each joined row.  The passing
     build rows go into a hash table in device memory; when at most 1024 pass,
     the one-launch compaction probes a copy of it held in each workgroup's
     LDS (Section 4, reviews JOIN movies on the movie id). */
  int32_t join;                        /* 0 = no join, 1 = inner PK-FK join */
  int32_t probe_key_col, build_key_col, build_payload_col;
  int32_t n_build_pred;
  aiq_pred build_preds[AIQ_MAX_PREDS];
  int32_t n_prefix;                    /* prompt tokens placed before each row's list
                                          (shared between rows on 16-bit models, see
                                          AIQ_PLAN_UNSHARED_PREFIX) */
  int32_t prefix[AIQ_MAX_PREFIX];
  int32_t n_labels;                    /* 2..AIQ_MAX_LABELS */
  int32_t label_ids[AIQ_MAX_LABELS];
  int32_t decision;                    /* aiq_decision: BINARY_GT keeps a row iff
                                          logit[label_ids[0]] > logit[label_ids[1]] */
  int32_t agg;                         /* aiq_agg */
  int32_t group_col;                   /* AVG_LABEL_COUNT_BY: probe key column (integer);
                                          SUM_F32: the summed probe column (AIQ_F32) */
  int32_t n_group_keys;                /* > 0: group keys are codes in [0, n_group_keys),
                                          aggregated in dense bins (keys outside flag
                                          AIQ_DEV_GROUP_RANGE); 0: any int32 key
                                          (INT32_MIN included), aggregated in a hash
                                          table and emitted in ascending key order;
                                          out->grp_cap should then cover the distinct keys
                                          (at most the probe rows, or for COUNT_BY_PAYLOAD
                                          the build rows); with more, the grp_cap smallest
                                          keys are written and AIQ_DEV_GROUP_CAP is set */
  /* AI_TRANSFORM (Table 1; Section 4, Q3 and Q5).  gen_tokens > 0 replaces
     the label decision: every selected row's sequence is continued by up
     to gen_tokens tokens, each the argmax of the last position's logits over
     the whole vocabulary (ties to the lowest id); a row's generation stops
     after eos_id (kept as its last token) and its later slots hold pad_id.
     A row is kept iff its generated tokens (up to the end) contain
     like[0..n_like) contiguously (LIKE '%pattern%' on token ids); with
     n_like = 0 every selected row is kept.  n_labels / label_ids / decision
     are ignored; agg AVG_LABEL_COUNT_BY is refused.  16-bit models only
     (AIQ_EUNSUPPORTED otherwise, or when vocab % 256 != 0). */
  int32_t gen_tokens;                  /* 0 = AI_IF classification; 1..AIQ_MAX_GEN */
  int32_t eos_id;                      /* -1 = no end token */
  int32_t pad_id;
  int32_t n_like;                      /* 0..AIQ_MAX_LIKE */
  int32_t like[AIQ_MAX_LIKE];
  /* Pairs of rows (Section 4, Q4: a self-join on the movie id that classifies
     [A.text, B.text]).  pairs = 1: the candidates are every two selected rows
     A < B (row order) with equal values of probe column pair_key_col, whose
     values must lie in [0, n_group_keys) (n_group_keys <= 16384; others are
     flagged AIQ_DEV_GROUP_RANGE and left out); each pair's sequence is the
     prefix, A's tokens, then B's tokens, classified with the binary decision.
     Candidates are numbered ascending by (A, B); at most max_pairs are kept
     (AIQ_DEV_PAIR_CAP otherwise).  out->ids receives the numbers of the pairs
     the decision keeps, out->pair_a / pair_b their rows; sel_labels and
     sel_logits are per candidate pair.  Requires no join, no generation,
     agg COUNT and decision BINARY_GT. */
  int32_t pairs;
  int32_t pair_key_col;
  int64_t max_pairs;
} aiq_query;

typedef struct aiq_plan_opts {
  int64_t chunk_tokens;                /* prefill chunk size in tokens; 0 = default */
  int32_t n_layers_override;           /* diagnostics: 0 = every layer, n > 0 = the first n
                                          layers, negative = no layer (embedding -> head) */
  int32_t flags;                       /* AIQ_PLAN_* bits */
  int32_t reserved[4];
} aiq_plan_opts;

/*
 * AIQ_PLAN_RELATIONAL_ONLY: aiq_run executes only the relational part of the
 * query (Table 1: the FROM and WHERE clauses, and the join of Section 4): the
 * predicate (+ join), the stable compaction and each selected row's token
 * count (list length + prefix).  out->ids receives every selected row id
 * ascending; scalars SELECTED = KEPT = their count, TOKENS = their total
 * tokens.  No model, decision or aggregate runs (the model must still be a
 * valid one); the query's agg must be AIQ_AGG_COUNT (else AIQ_EINVAL at plan
 * creation); the probe table's token column is not read and may be NULL
 * (its offsets are required).
 */
#define AIQ_PLAN_RELATIONAL_ONLY 1

/*
 * Prompt prefix (the instruction of a prompted AI_IF, Table 1 and the join
 * query of Section 4).  Row i's sequence is always prefix || row i's tokens,
 * positions 0.. from the prefix start.  On 16-bit models with n_prefix > 0
 * and at least one layer, aiq_run prefills the prefix once, keeps its keys
 * and values for every layer, and runs each row's own tokens only, attending
 * to the kept prefix: the result is the same function of the inputs as the
 * per-row computation, with each row's own query positions meeting the same
 * key blocks in the same order.  A row with an empty token list is then
 * classified from the prefix's last token (per-row computation: the same).
 * AIQ_PLAN_UNSHARED_PREFIX: recompute the prefix inside every row's sequence
 * instead (fp32 models always do).  scalars[AIQ_S_TOKENS] counts the prefix
 * once per selected row in both modes.
 */
#define AIQ_PLAN_UNSHARED_PREFIX 2

/*
 * The WHERE (+ join) compaction and the selected rows' token offsets run as
 * one launch (decoupled look-back across blocks of rows) whenever a block's
 * token sum is bounded below 2^31 (8192 x (max_list_len + n_prefix)).
 * AIQ_PLAN_MULTIPASS_COMPACT: run them as separate mask, scan and scatter
 * launches instead.  Both give identical outputs.
 */
#define AIQ_PLAN_MULTIPASS_COMPACT 4

/*
 * The label head (Figure 2: the logits of the last position only) reads one
 * row per sequence, and in a causal decoder the last layer's rows after its
 * q|k|v projection feed no other position.  On 16-bit models (head dim 64 or
 * 128) aiq_run and aiq_prefill_packed therefore run the last layer's keys and
 * values for every position but its attention (one query per sequence, over
 * the sequence's keys), O projection, norm and FFN for the last position of
 * each sequence only.  The logits are the same function of the inputs; the
 * last layer's attention then sums in a different order than the full-layer
 * kernel, so they agree with the full computation to rounding, not bit for
 * bit.  AIQ_PLAN_FULL_LAST_LAYER: run the last layer on every position.
 */
#define AIQ_PLAN_FULL_LAST_LAYER 8

/*
 * Outputs, all device buffers owned by the caller.  Optional buffers may be
 * NULL.  Row ids are probe-table row indices.
 */
typedef struct aiq_out {
  int64_t* scalars;          /* [AIQ_N_SCALARS], see AIQ_S_* */
  int32_t* ids;              /* kept row ids, ascending; capacity ids_cap */
  int64_t ids_cap;
  int32_t* sel_ids;          /* optional: selected row ids (ascending), cap sel_cap */
  int32_t* sel_labels;       /* optional: label value per selected row (binary 1/0,
                                argmax: the winning label token id; AI_TRANSFORM:
                                1 if the row's generation matches the LIKE pattern) */
  float* sel_logits;         /* optional: [sel_cap, n_labels] label logits (not
                                written by AI_TRANSFORM queries) */
  int64_t sel_cap;
  int32_t* grp_key;          /* groups in ascending key order, capacity grp_cap */
  int64_t* grp_count;
  int64_t* grp_sum;          /* SUM(label) (0 for COUNT_BY_PAYLOAD) */
  double* grp_avg;           /* SUM/COUNT in fp64 (0 for COUNT_BY_PAYLOAD) */
  int64_t grp_cap;
  /* SUM_F32: the sum, accumulated in fp64 in an order fixed by the number of
     selected rows alone, so repeated runs give the same bits.  Its distance
     to the exactly rounded sum is at most 2^-52 * (n_kept + 64) * sum|v|. */
  double* sum_out;
  /* optional, AI_TRANSFORM: [sel_cap, gen_tokens] generated tokens of each
     selected row (same order as sel_ids), pad_id after a row's end */
  int32_t* sel_gen;
  /* optional, pairs mode: rows A and B of the kept pairs (capacity ids_cap)
     and of every candidate pair (capacity sel_cap), in pair order */
  int32_t* pair_a;
  int32_t* pair_b;
  int32_t* cand_a;
  int32_t* cand_b;
} aiq_out;

/*
 * Optional stage timing: the library records a pair of HIP events around
 * every kernel launch whose kind is selected in `kind_mask` (bit k = kind k,
 * see AIQ_K_*), writing tags[i] = kind for the pair events[2i], events[2i+1].
 * Recording starts at pair index `count` and advances it, so one trace can
 * span several calls (set count = 0 first); it stops silently once
 * `capacity` pairs are used.  events[] are hipEvent_t created by the caller
 * with timing enabled.
 */
typedef struct aiq_trace {
  void** events;
  int32_t* tags;
  int32_t capacity;
  int32_t count;
  uint32_t kind_mask;
} aiq_trace;

enum {
  AIQ_K_REL = 0,        /* predicate / join / compaction kernels */
  AIQ_K_PACK = 1,       /* sequence lengths, scans, token gather, chunking */
  AIQ_K_EMBED = 2,
  AIQ_K_NORM = 3,
  AIQ_K_GEMM_QKV = 4,
  AIQ_K_ATTN = 5,
  AIQ_K_GEMM_O = 6,
  AIQ_K_GEMM_UP = 7,    /* gate/up (SwiGLU) or W1 (GELU) */
  AIQ_K_GEMM_DOWN = 8,
  AIQ_K_HEAD = 9,
  AIQ_K_AGG = 10,
  AIQ_K_DECODE = 11,      /* AI_TRANSFORM generation steps: embedding, projections, norms */
  AIQ_K_DECODE_ATTN = 12, /* ... their attention over the kept keys and values */
  AIQ_K_DECODE_HEAD = 13, /* ... the full-vocabulary head and argmax; the LIKE match */
  AIQ_K_LAST = 14         /* the last layer after its q|k|v projection, last positions only */
};

typedef struct aiq_plan aiq_plan;

/*
 * Validates the model, tables and query and builds an immutable plan: the
 * host-side counterpart of the paper's compile step (Section 3.1, Figure 2:
 * the SQL clauses of Table 1 mapped to one program of tensor operations),
 * here a fixed sequence of device kernels whose data-dependent sizes stay on
 * the device.
 * probe may be NULL for a prefill-only plan (aiq_prefill_packed); build must
 * be non-NULL iff query->join.  query may be NULL for a prefill-only plan
 * that only uses AIQ_LOGITS_FULL_VOCAB.  opts may be NULL.
 * Errors: AIQ_EINVAL (bad pointer, dtype, op, column index, d_model % n_heads,
 * n_heads % n_kv_heads, head dim not in {32, 64, 128}), AIQ_EUNSUPPORTED,
 * AIQ_ENOMEM.  On error *out is set to NULL.
 */
aiq_status aiq_plan_create(const aiq_model* model, const aiq_table* probe, const aiq_table* build,
                           const aiq_query* query, const aiq_plan_opts* opts, aiq_plan** out);

/* Bytes of device workspace aiq_run needs (256-byte aligned base required):
 * the selection, the packed batch and one chunk's activations, sized from the
 * table and model alone so that nothing is allocated inside the run
 * (Section 3.3, everything resident on the device). */
aiq_status aiq_workspace_size(const aiq_plan* plan, size_t* bytes);

/*
 * Prefill passes aiq_run enqueues (Section 3.2: the scan over micro-batches
 * of the selected rows): the chunks of the packed batch, an upper
 * bound fixed at plan creation from the table's token total (chunks that
 * the selection leaves empty cost one launch per kernel and no work), plus
 * one pass for a shared prompt prefix.  Each pass launches the embedding,
 * per layer the four projections, attention and the norm row scales, and,
 * except the prefix pass, the label head.  For sizing trace buffers
 * (aiq_trace).  Errors: AIQ_EINVAL (NULL argument, prefill-only plan).
 */
aiq_status aiq_plan_passes(const aiq_plan* plan, int64_t* chunks, int32_t* prefix_pass);

/*
 * The chunk size of the plan's prefill passes (0 for a relational-only plan):
 * pass c covers the selected sequences i with cu[i] + i in
 * [c * chunk_tokens, (c + 1) * chunk_tokens), where cu[i] is the number of
 * packed tokens before sequence i; a sequence counts one unit besides its
 * tokens, so a pass never holds more than chunk_tokens sequences.  With
 * aiq_plan_passes this tells a caller which passes a given selection fills
 * (a trace's per-pass launches, Section 3.2's scan over micro-batches).
 * Errors: AIQ_EINVAL (NULL argument, prefill-only plan).
 */
aiq_status aiq_plan_chunk_tokens(const aiq_plan* plan, int64_t* chunk_tokens);

/*
 * *last_rows_only = 1 when the plan runs the last layer, after its q|k|v
 * projection, for the last position of each sequence only (Figure 2 reads
 * the logits of the last position alone; see
 * AIQ_PLAN_FULL_LAST_LAYER), else 0.  In that case every prefill pass (the
 * chunks and a shared prefix) launches the gate/up projection of every layer
 * but the last over all its positions, and the last layer's attention, O
 * projection, norm and FFN appear in traces as AIQ_K_LAST.
 * Errors: AIQ_EINVAL (NULL argument).
 */
aiq_status aiq_plan_last_layer_rows(const aiq_plan* plan, int32_t* last_rows_only);

/*
 * Enqueues the whole query on `stream` (Section 3.3: the relational part and
 * the semantic operator as one device program with no host round trip;
 * Figure 2's filter on the last-position label logits and masked
 * aggregate).  The workspace contents on entry do not matter.  Outputs are valid after the caller synchronises the stream.
 * Errors: AIQ_EINVAL (NULL plan/out/scalars/ids, prefill-only plan, a
 * group-by without grp_* buffers), AIQ_ENOSPC (ws_bytes too small),
 * AIQ_EHIP.  `trace` may be NULL.
 */
aiq_status aiq_run(const aiq_plan* plan, void* workspace, size_t ws_bytes, const aiq_out* out,
                   aiq_trace* trace, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * relational part of aiq_run for a relational-only plan
 * (AIQ_PLAN_RELATIONAL_ONLY, one-launch compaction), with no workspace
 * argument.  Its scratch (counters, the compaction's look-back words, the
 * join's hash table) lives in one fixed device array of 16 MiB inside the
 * library, which each GPU it runs on holds until the process ends; the call
 * allocates nothing.  Outputs as aiq_run with that plan: out->ids (and
 * out->sel_ids when sel_cap > 0) receive the selected row ids ascending,
 * scalars SELECTED = KEPT = their count, TOKENS = their token total.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (on different streams or threads) race and must not be issued.  Each call
 * clears what must start at zero itself.
 * Errors: AIQ_EINVAL (NULL plan/out/scalars, a plan that is not
 * relational-only), AIQ_EUNSUPPORTED (a plan using the multi-launch
 * compaction), AIQ_ENOSPC (the plan needs more than the 16 MiB scratch:
 * about 32 B per 4,096 probe rows plus 8 B per hash slot, i.e. 2 x the build
 * rows rounded up to a power of two; nothing is enqueued), AIQ_EHIP.
 */
aiq_status aiq_run_relational_static(const aiq_plan* plan, const aiq_out* out, void* stream);

/* Bytes of workspace aiq_prefill_packed needs for up to max_tokens tokens
 * (the split-execution baseline's model half, Section 3.3). */
aiq_status aiq_prefill_workspace_size(const aiq_plan* plan, int64_t max_tokens, size_t* bytes);

/*
 * Runs only the transformer on an already packed batch (device buffers):
 * sequence i is tok[cu_seqlens[i] .. cu_seqlens[i+1]), cu_seqlens int32
 * [n_seq+1] with cu_seqlens[0] = 0 and cu_seqlens[n_seq] = n_tok; positions
 * restart at 0 in every sequence.  Writes the last position's logits of each
 * sequence: AIQ_LOGITS_LABELS -> logits[n_seq, n_labels] for the plan's
 * query labels; AIQ_LOGITS_FULL_VOCAB -> logits[n_seq, vocab].  This is the
 * model half of the split-execution baseline (Section 3.3) and the kernel
 * parity entry point.  Errors: AIQ_EINVAL, AIQ_ENOSPC (workspace, or n_tok
 * above the workspace's token capacity), AIQ_EHIP.
 */
aiq_status aiq_prefill_packed(const aiq_plan* plan, const int32_t* tok, const int32_t* cu_seqlens,
                              int32_t n_seq, int64_t n_tok, int32_t logits_mode, float* logits,
                              void* workspace, size_t ws_bytes, void* stream);

/*
 * Converts n weight elements in device memory from src_dtype to dst_dtype on
 * `stream`: AIQ_BF16 -> AIQ_F16 only, each value widened exactly and rounded
 * to the nearest fp16 (ties to even; magnitudes below 2^-14 become fp16
 * subnormals, above 65504 infinities).  bf16-stored models run their 16-bit
 * projections on fp16 images of the weights (10 mantissa bits for the
 * activations instead of 7 at the same MFMA rate, the precision that keeps a
 * 16-layer model's label logits within the bf16 tolerance, Figure 2's
 * last-position comparison); aiq_model.wdtype = AIQ_F16 then points at the
 * converted arrays.  src and dst are 16-byte aligned, distinct, owned by the
 * caller.  Errors: AIQ_EINVAL (NULL pointer with n > 0, negative n,
 * misalignment), AIQ_EUNSUPPORTED (another pair of types), AIQ_EHIP.
 */
aiq_status aiq_convert_weights(const void* src, int32_t src_dtype, void* dst, int32_t dst_dtype, int64_t n,
                               void* stream);

/* Frees a plan (host memory only; NULL is ignored). */
void aiq_plan_destroy(aiq_plan* plan);

/* A static description of an aiq_status value. */
const char* aiq_status_str(int32_t status);
/* AIQ_ABI_VERSION of the library: bindings refuse another layout. */
int32_t aiq_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* AIQ_H */
