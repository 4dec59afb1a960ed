// Internal declarations shared by the HIP kernel files and the host orchestrator.
// Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/aiq.h"

namespace aiq {

// ---------------------------------------------------------------- device counters
// int64 slots in the workspace; cleared at the start of every run.
enum Ctr : int {
  C_SEL = 0,      // rows passing WHERE (+ join)
  C_KEPT = 1,     // rows kept after the decision
  C_TOK = 2,      // total prefill tokens
  C_STATUS = 3,   // OR of AIQ_DEV_* bits
  C_GROUPS = 4,   // non-empty groups
  C_SCRATCH = 5,  // scan totals land here before being copied
  C_NSEQ = 6,     // prefill-only: number of sequences
  C_PAIRS = 7,    // pairs mode: candidate pairs (the sequences)
  C_COUNT = 16
};

// chunk descriptor: int64 x 4 per chunk
enum Desc : int { D_TOK_BEGIN = 0, D_NTOK = 1, D_SEQ_BEGIN = 2, D_NSEQ = 3, D_STRIDE = 4 };

struct DPred {
  const void* data;
  int32_t dtype;
  int32_t op;
  int64_t k;          // integer columns
  double fk;          // AIQ_F32 columns
  int32_t n_set;
  int32_t set[AIQ_MAX_IN_SET];
};

struct DPredList {
  int32_t n;
  DPred p[AIQ_MAX_PREDS];
};

struct HashArgs {
  int32_t* keys;      // [cap], EMPTY = INT32_MIN
  int32_t* vals;      // [cap]
  int32_t cap_log2;
};

constexpr int32_t HASH_EMPTY = INT32_MIN;

// The join's build table rehashed for probing from LDS: 2^(*log2_out) slots
// (keys, vals) when that is at most JOIN_LDS_SLOTS, else *log2_out = 0 and
// the probes read the global table.
constexpr int JOIN_LDS_SLOTS = 2048;
struct StagedHash {
  int32_t* keys;      // [JOIN_LDS_SLOTS]
  int32_t* vals;      // [JOIN_LDS_SLOTS]
  int32_t* log2_out;  // device word
};

// GROUP BY over arbitrary int32 keys: an open-addressing table of 2^cap_log2
// slots in global memory (slot words: key bits | 1 << 32, 0 = empty; slot,
// cnt and sum are consecutive arrays of 2^cap_log2 entries each, cleared by
// the launcher), and the buffers of the sort of its occupied slots by key.
struct HashAggArgs {
  uint64_t* slot;
  int64_t* cnt;
  int64_t* sum;
  int32_t cap_log2;
  uint32_t* key0;     // [max_groups] x 4 ping-pong sort buffers
  uint32_t* val0;
  uint32_t* key1;
  uint32_t* val1;
  int64_t* hist;      // [256 * hash_group_sort_blocks(max_groups)]
  int64_t* n_groups;  // device word: occupied slots
};

// relational block geometry: 256 threads x 32 rows
constexpr int REL_THREADS = 256;
constexpr int REL_ROWS_PER_THREAD = 32;
constexpr int REL_ROWS_PER_BLOCK = REL_THREADS * REL_ROWS_PER_THREAD;   // 8192
constexpr int REL_WORDS_PER_BLOCK = REL_ROWS_PER_BLOCK / 64;             // 128
// the one-launch compaction's blocks hold at least this many rows (its look-back
// state is 4 int64 per block)
constexpr int LB_MIN_ROWS = 4096;

// ---------------------------------------------------------------- launchers
// Every launcher enqueues on `s` and returns hipGetLastError().

// relational
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
hipError_t launch_fill_i64(int64_t* p, int64_t n, int64_t v, hipStream_t s);
hipError_t launch_hash_build(const DPredList& preds, const void* key_col, int32_t key_dtype,
                             const void* pay_col, int32_t pay_dtype, int64_t n_rows, HashArgs h,
                             int64_t* ctr, hipStream_t s);
hipError_t launch_row_mask(const DPredList& preds, int64_t n_rows, const void* probe_key,
                           int32_t probe_key_dtype, HashArgs h, int join, uint64_t* mask,
                           int32_t* blk_cnt, hipStream_t s);
hipError_t launch_label_mask(const int32_t* label, const int64_t* n_ptr, int64_t n_ub,
                             uint64_t* mask, int32_t* blk_cnt, hipStream_t s);
// Exclusive scan of per-block values (one per REL_ROWS_PER_BLOCK rows of n):
// off[b] = sum of v[< b], off[nb] = *total_out = the sum of all.
hipError_t launch_scan_blocks(const int32_t* blk_cnt, const int64_t* n_ptr, int64_t n_ub,
                              int64_t* blk_off, int64_t* total_out, hipStream_t s);
hipError_t launch_scan_blocks64(const int64_t* blk_val, const int64_t* n_ptr, int64_t n_ub,
                                int64_t* blk_off, int64_t* total_out, hipStream_t s);
// Token counts of the selected rows, produced while compacting them: for
// output position i of row r, lens[i] = min(off[r+1] - off[r], max_len) +
// n_prefix (a list longer than max_len, or negative, flags AIQ_DEV_LIST_LEN),
// and blk_tok[b] = sum of lens over the rows of input block b.
struct ScatterLens {
  const int64_t* off;        // null: no lengths
  int32_t max_len, n_prefix;
  int32_t* lens;             // [n] by output position
  int64_t* blk_tok;          // [n_blocks]
};
// Stable compaction of the mask: out_ids[pos] = src_ids ? src_ids[r] : r for
// every set bit r, in row order (positions >= out_cap dropped and flagged);
// optionally a second copy (out_ids2, cap2), the join payload and lengths.
hipError_t launch_scatter_rows(const uint64_t* mask, const int64_t* blk_off, const int64_t* n_ptr,
                               int64_t n_ub, const int32_t* src_ids, int32_t* out_ids,
                               int64_t out_cap, const void* probe_key, int32_t probe_key_dtype,
                               HashArgs h, int join, int32_t* out_payload, int64_t* ctr,
                               hipStream_t s, int32_t* out_ids2 = nullptr, int64_t out_cap2 = 0,
                               ScatterLens lens = ScatterLens{});
// cu[0] = 0 and cu[i + 1] = cu[i] + lens[i] for the selected rows, from the
// per-block token offsets of the compaction (tok_off = scan of blk_tok).
hipError_t launch_cu_from_blocks(const int32_t* lens, const int64_t* blk_off, const int64_t* tok_off,
                                 int64_t n_ub, int64_t* cu, hipStream_t s);
// WHERE (+ join), stable compaction and token offsets in one launch (decoupled
// look-back over `lb`, 4 int64 per block of at least LB_MIN_ROWS rows,
// cleared here first): out_ids
// (and out_ids2) as launch_scatter_rows, ctr[C_SEL] = the count; with `off`
// also ctr[C_TOK] = the total token count (per row min(list length,
// max_len) + n_prefix) and, when cu is not NULL, cu[0..n_sel] (cu[i] =
// tokens of the selected rows before i).
// A block's token sum must stay below 2^31: REL_ROWS_PER_BLOCK *
// (max_len + n_prefix) < 2^31.
// With a join and st non-null, the probes read the LDS-staged table (st,
// written by launch_hash_stage) when it fits, else h.
hipError_t launch_select_lb(const DPredList& preds, int64_t n_rows, const void* probe_key, int32_t probe_key_dtype,
                            HashArgs h, int join, const StagedHash* st, int32_t* out_ids, int64_t out_cap,
                            int32_t* out_ids2, int64_t out_cap2, int32_t* out_payload, const int64_t* off,
                            int32_t max_len, int32_t n_prefix, int64_t* cu, int64_t* lb, int64_t* ctr,
                            hipStream_t s);
// ctr[C_KEPT] = ctr[C_SEL] (every selected row kept), flagged if above cap.
hipError_t launch_keep_selected(int64_t* ctr, int64_t cap, hipStream_t s);
hipError_t launch_group_accumulate(const int32_t* sel, const int32_t* label, const int32_t* payload,
                                   const uint8_t* keep_by_label, const int64_t* n_ptr, int64_t n_ub,
                                   const void* key_col, int32_t key_dtype, int mode,
                                   int32_t n_keys, int64_t* bins, int64_t* ctr, hipStream_t s);
// GROUP BY with a hash table (any int32 key; mode as launch_group_accumulate):
// groups in ascending key order written to key_out / cnt_out / sum_out /
// avg_out (at most cap, more flag AIQ_DEV_GROUP_CAP), ctr[C_GROUPS] = the
// number written.  max_groups bounds the distinct keys; 2^g.cap_log2 >=
// 2 * max_groups.
int64_t hash_group_sort_blocks(int64_t max_groups);
hipError_t launch_hash_group(const int32_t* sel, const int32_t* label, const int32_t* payload, const int64_t* n_ptr,
                             int64_t n_ub, const void* key_col, int32_t key_dtype, int mode, HashAggArgs g,
                             int64_t max_groups, int32_t* key_out, int64_t* cnt_out, int64_t* sum_out,
                             double* avg_out, int64_t cap, int64_t* ctr, hipStream_t s);
// Rehashes the built join table for LDS probing (see StagedHash).
hipError_t launch_hash_stage(HashArgs h, StagedHash st, hipStream_t s);
hipError_t launch_group_emit(const int64_t* bins, int32_t n_keys, int32_t* key_out,
                             int64_t* cnt_out, int64_t* sum_out, double* avg_out, int64_t cap,
                             int mode, int64_t* ctr, hipStream_t s);
hipError_t launch_copy_ids(const int32_t* src, const int64_t* n_ptr, int64_t n_ub, int32_t* dst,
                           int64_t cap, int64_t* ctr, int set_kept, hipStream_t s);
hipError_t launch_copy_f32(const float* src, const int64_t* n_ptr, int64_t n_ub, int32_t per_row,
                           float* dst, int64_t cap_rows, hipStream_t s);
// scalars[AIQ_S_TOKENS] adds tok_per_row tokens per sequence (ctr[seq_ctr])
// to ctr[C_TOK] (the shared prompt prefix, which is packed once, not per row).
hipError_t launch_finalize(const int64_t* ctr, int64_t* scalars, hipStream_t s, int32_t tok_per_row = 0,
                           int32_t seq_ctr = C_SEL);
// SUM_F32: fp64 sum of col[sel[i]] over the selected rows i < n_sel with
// label[i] == 1 (binary decision) or all of them (argmax), in a fixed order:
// SUM_BLOCKS fixed ranges of i, each reduced in a fixed tree, then the block
// partials in a fixed tree.  partial: [SUM_BLOCKS] scratch.
constexpr int SUM_BLOCKS = 1024;
hipError_t launch_sum_f32(const int32_t* sel, const int32_t* label, const int64_t* n_ptr, const float* col,
                          int binary, double* partial, double* out, hipStream_t s);

// packing / chunking
struct Prefix {
  int32_t n;
  int32_t tok[AIQ_MAX_PREFIX];
};
hipError_t launch_gather_tokens(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub,
                                const int64_t* offsets, const int32_t* tokens, const int64_t* cu,
                                const Prefix& prefix, int32_t vocab, int64_t t_ub, int32_t* packed,
                                int64_t* ctr, hipStream_t s);
// Chunk c: the sequences i with cu[i] + i in [c, c + 1) * chunk_tokens (at
// most chunk_tokens sequences per chunk, empty lists included); the last
// chunk runs to the last sequence.
hipError_t launch_chunk_desc(const int64_t* cu, const int64_t* n_ptr, int64_t chunk_tokens,
                             int64_t n_chunks, int64_t t_ub, int64_t* desc, hipStream_t s);
hipError_t launch_packed_desc(const int32_t* cu32, int32_t n_seq, int64_t n_tok, int64_t* cu64,
                              int64_t* desc, int64_t* ctr, hipStream_t s);
// The shared prompt prefix as a one-sequence batch: tok[0..n) = prefix,
// cu = {0, n}, desc = one chunk of n tokens.
hipError_t launch_prefix_batch(const Prefix& prefix, int32_t* tok, int64_t* cu, int64_t* desc, hipStream_t s);
// bf16 -> fp16 conversion of n elements (nearest, ties to even); src and dst
// 16-byte aligned.
hipError_t launch_bf16_to_f16(const void* src, void* dst, int64_t n, hipStream_t s);
hipError_t launch_copy_row_f32(const float* src, float* dst, int32_t n, hipStream_t s);

// per-chunk transformer
// cos/sin table [max_pos, hd/2] and the per-dim frequency in revolutions [hd/2]
hipError_t launch_rope_table(int32_t max_pos, int32_t half, double theta, int32_t hd, float* cos_t,
                             float* sin_t, float* rev, hipStream_t s);
hipError_t launch_embed(const int64_t* desc, const int64_t* cu, const int32_t* packed,
                        const void* emb, int32_t wdtype, int32_t d, int32_t vocab, float* x, int32_t* pos,
                        int64_t* ctr, int64_t t_cap, hipStream_t s);
// MFMA path: the embedding also writes the first projection's operand
// h = x * g (16-bit) and the row scale rs = 1 / sqrt(mean(x^2) + eps).
// pos_base is added to every position (the row tokens that follow a shared
// prefix start at the prefix length).  x may be null: the residual is then
// not written (the first layer's O projection reads the embedding rows).
hipError_t launch_embed_norm(const int64_t* desc, const int64_t* cu, const int32_t* packed, const void* emb,
                             int32_t wdtype, int32_t d, int32_t vocab, float* x, int32_t* pos, int64_t* ctr,
                             const float* g, float eps, void* h, int32_t h_act, float* rs, int64_t t_cap,
                             hipStream_t s, int32_t pos_base = 0);
// rs[t] = 1 / sqrt(sum_p ssp[t, p] / d + eps) for the chunk's tokens, the
// partial sums added in order p = 0, 1, ...
hipError_t launch_row_scale(const int64_t* desc, const float* ssp, int32_t n_part, int32_t d, float eps,
                            float* rs, int64_t t_cap, hipStream_t s);
// x += delta (when delta is non-null, written back), then out = RMSNorm(x) * g
// out_act: 0 fp32, 1 bf16, 2 fp16
hipError_t launch_rmsnorm(const int64_t* desc, float* x, const float* delta, const float* g, int32_t d,
                          float eps, void* out, int32_t out_act, int64_t t_cap, hipStream_t s);

// EPI_ARGMAX (MFMA path): no output matrix; C = int2 [M][N / 64] of
// (fp32 bits of the maximum, its column) over each 64-column slice of a row,
// the lowest column among equal maxima.
enum Epi : int {
  EPI_STORE_F32 = 0, EPI_QKV_ROPE = 1, EPI_SWIGLU = 3, EPI_GELU = 4, EPI_STORE_ACT = 5, EPI_RESID = 6, EPI_ARGMAX = 7,
  EPI_RESID_EMB = 8   // EPI_RESID reading the residual from the embedding table (x_emb)
};

struct GemmArgs {
  const void* A;             // [M, K] activations (bf16 or f32), row stride lda
  int64_t lda;
  const int64_t* m_ptr;      // device: number of rows M
  int64_t m_ub;              // host: upper bound on M (grid sizing)
  int32_t N, K;
  const void* B0;            // weight sources, row-major [rows, K]
  const void* B1;
  const void* B2;
  int32_t n_q, n_kv;         // QKV section widths (d_q, d_kv); SwiGLU: d_ff in n_q
  int32_t hd;
  void* C;                   // output
  int64_t ldc;
  const int32_t* pos;        // [M + 256] positions (EPI_QKV_ROPE; entries past M are ignored)
  const float* rope_cos;     // [max_pos, hd/2] (fp32 path)
  const float* rope_sin;
  const float* rope_rev;     // [hd/2] theta^(-2i/hd) / (2 pi) (MFMA path)
  int32_t f16;               // MFMA path: operands are fp16 (else bf16)
  // Residual stream with the RMSNorm folded into the projections (MFMA path):
  const float* rs;           // EPI_QKV_ROPE / EPI_SWIGLU: per-row scale 1/rms (rows padded by 256), or null
  float* x;                  // EPI_RESID: residual [M, ldc] fp32, x += A.W^T in place
  const float* gnext;        // EPI_RESID: gain of the RMSNorm that follows (null: only x is written)
  void* hout;                // EPI_RESID: [M, ldc] 16-bit, x * gnext (the next projection's operand)
  float* ssp;                // EPI_RESID: [M, n_part] sums of x^2 over each 64-column slice
  int32_t n_part;            // ldc / 64
  // EPI_RESID_EMB (first layer): the residual read is the embedding row of
  // the row's token (16-bit table [vocab, ldc]; token =
  // x_tok[x_tok_desc[D_TOK_BEGIN] + m], out of range read as 0), not x; x is
  // still written.
  const void* x_emb;
  const int32_t* x_tok;
  const int64_t* x_tok_desc;
  int32_t vocab;
};

hipError_t launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_f32(int epi, const GemmArgs& a, hipStream_t s);
hipError_t launch_rope_f32(const int64_t* desc, float* qkv, int64_t ld, int32_t n_q, int32_t n_kv,
                           int32_t hd, const int32_t* pos, const float* cos_t, const float* sin_t,
                           int64_t t_cap, hipStream_t s);

struct AttnArgs {
  const void* qkv;           // [T, ld] : q | k | v
  int64_t ld;
  void* out;                 // [T, ldo]
  int64_t ldo;
  const int64_t* desc;       // chunk descriptor (n_tok, n_seq, seq_begin)
  const int64_t* cu;         // global cu_seqlens (int64)
  int32_t n_heads, n_kv, hd;
  int64_t seq_ub;            // host upper bound on sequences per chunk
  int32_t out_act;           // MFMA path: output element type (1 bf16, 2 fp16)
  // Shared prompt prefix (MFMA path): every sequence is read as
  // pkv[0..npre) followed by its own rows, positions counted from the
  // prefix start; only the own rows are queries.  pkv: [npre, ld] q|k|v rows.
  const void* pkv;
  int32_t npre;
};
hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_f32(const AttnArgs& a, hipStream_t s);

struct HeadArgs {
  const int64_t* desc;
  const int64_t* cu;
  const float* x;            // residual [T, d]
  const float* delta;        // pending output of the last projection [T, d], or NULL
  const float* g;            // final norm gains
  float eps;
  int32_t d;
  const void* lm_head;       // [vocab, d]
  int32_t wdtype;
  int32_t n_labels;
  int32_t labels[AIQ_MAX_LABELS];
  int32_t decision;
  int32_t* label_out;        // [global seq]
  float* logits_out;         // [global seq, n_labels] or NULL
  void* hf_out;              // optional normalised rows [local seq, d] (full-vocab mode)
  int32_t hf_act;            // element type of hf_out (0 fp32, 1 bf16, 2 fp16)
  int64_t seq_ub;
  const float* x_pre;        // shared prefix: final residual of its last token, used by
                             // sequences with no own token (null: such sequences get 0 logits)
  int32_t x_compact;         // 1: x holds one row per sequence of desc (row i), not [T, d]
};
hipError_t launch_head(const HeadArgs& a, hipStream_t s);

// ---------------------------------------------------------------- pairs (Q4 self-join)
// Exclusive scan of v[0..n) (n = *n_ptr, or n_ub when n_ptr is null) into
// out[0..n] as int64, out[n] = *total_out = the sum.  blk: scratch of
// n_ub / 8192 + 2 int64 values for the block sums and their offsets (x2).
hipError_t launch_scan_i32_i64(const int32_t* v, const int64_t* n_ptr, int64_t n_ub, int64_t* out, int64_t* blk,
                               int64_t* total_out, hipStream_t s);
// kcount[k] += 1 for the key of every selected row (keys outside
// [0, n_keys) flagged AIQ_DEV_GROUP_RANGE and skipped)
hipError_t launch_pair_key_count(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub, const void* key_col,
                                 int32_t key_dt, int32_t n_keys, int32_t* kcount, int64_t* ctr, hipStream_t s);
// Stable counting sort of the selected rows by key: rank[i] = number of
// earlier selected rows with the same key, sorted[koff[key] + rank[i]] = i.
// One workgroup, 1024 rows per round; n_keys <= PAIR_MAX_KEYS.
constexpr int PAIR_MAX_KEYS = 16384;
hipError_t launch_pair_rank(const int32_t* sel, const int64_t* n_ptr, const void* key_col, int32_t key_dt,
                            int32_t n_keys, const int64_t* koff, int32_t* rank, int32_t* sorted, hipStream_t s);
// cnt[i] = later selected rows with the same key (0 for a key out of range)
hipError_t launch_pair_partners(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub, const void* key_col,
                                int32_t key_dt, int32_t n_keys, const int32_t* kcount, const int32_t* rank,
                                int32_t* cnt, hipStream_t s);
// ctr[C_PAIRS] = min(*total, cap), AIQ_DEV_PAIR_CAP when above
hipError_t launch_pair_total(const int64_t* total, int64_t cap, int64_t* ctr, hipStream_t s);
// pair numbers poff[i] .. poff[i] + cnt[i] - 1 below cap: (pa, pb) = (i, the
// later rows of i's key in order), as selected-row indices
hipError_t launch_pair_emit(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub, const void* key_col,
                            int32_t key_dt, int32_t n_keys, const int64_t* koff, const int32_t* rank,
                            const int32_t* sorted, const int32_t* cnt, const int64_t* poff, int64_t cap,
                            int32_t* pa, int32_t* pb, hipStream_t s);
// lens[q] = n_prefix + len(A) + len(B) of pair q < ctr[C_PAIRS] (a list
// longer than max_len flagged AIQ_DEV_LIST_LEN and cut to max_len)
hipError_t launch_pair_lens(const int32_t* pa, const int32_t* pb, const int32_t* sel, const int64_t* off,
                            int32_t max_len, int32_t n_prefix, int64_t cap, int32_t* lens, int64_t* ctr,
                            hipStream_t s);
// packed[cu[q] ..] = prefix, A's tokens, B's tokens (wave per pair)
hipError_t launch_pair_gather(const int32_t* pa, const int32_t* pb, const int32_t* sel, const int64_t* off,
                              const int32_t* tokens, const int64_t* cu, const Prefix& prefix, int32_t max_len,
                              int32_t vocab, int64_t t_ub, int64_t cap, int32_t* packed, int64_t* ctr,
                              hipStream_t s);
// rows of pairs: out_a[j] = sel[pa[q]], out_b[j] = sel[pb[q]] with q = ids[j]
// (ids null: q = j), j < min(*n_ptr, cap)
hipError_t launch_pair_rows(const int32_t* ids, const int64_t* n_ptr, int64_t n_ub, const int32_t* pa,
                            const int32_t* pb, const int32_t* sel, int32_t* out_a, int32_t* out_b, int64_t cap,
                            hipStream_t s);

// ---------------------------------------------------------------- AI_TRANSFORM generation
// A generation step works on one row per sequence of the chunk: its
// descriptor (D_TOK_BEGIN 0, D_NTOK = D_NSEQ = the chunk's sequences,
// D_SEQ_BEGIN = the chunk's first sequence) comes from the chunk's.  The
// full-vocabulary head runs in blocks of GEN_HEAD_ROWS rows; cnt[b] = rows
// of block b.
constexpr int GEN_HEAD_ROWS = 4096;
hipError_t launch_gen_desc(const int64_t* chunk_desc, int64_t* gen_desc, int64_t* cnt, int32_t n_blocks,
                           hipStream_t s);
// Embedding of each sequence's current token at position (its prompt
// length incl. a shared prefix of npre tokens) + step, with the first norm's
// operand h = x * g and row scale rs (as launch_embed_norm).
hipError_t launch_gen_embed(const int64_t* gen_desc, const int64_t* cu, const int32_t* tok, int32_t step,
                            int32_t npre, const void* emb, int32_t wdtype, int32_t d, int32_t vocab, float* x,
                            int32_t* pos, const float* g, float eps, void* h, int32_t h_act, float* rs,
                            int64_t seq_ub, hipStream_t s);
struct GenAttnArgs {
  const void* qkv;           // [n, ld] this step's q|k|v, one row per sequence
  const void* kvc;           // the chunk's prompt rows for this layer, [chunk tokens, ld] q|k|v
  const void* pkv;           // shared prefix rows for this layer [npre, ld], or null
  int32_t npre;
  void* gkv;                 // generated keys/values [seq_ub][gen][2 d_kv]; slot `step` is written
  int32_t step, gen;
  int64_t ld;
  const int64_t* gen_desc;
  const int64_t* chunk_desc; // for the chunk's first token
  const int64_t* cu;
  void* out;                 // [n, n_heads * hd]
  int32_t n_heads, n_kv, hd, out_act;
  int64_t seq_ub;
  // 1: the query of sequence i is its own last position and the keys are
  // the prefix and its own rows only (no generated tokens; gkv, step and gen
  // unused); sequences with no own row are skipped.  The query is row i of
  // qkv (stride ldq, q columns first) when qkv is set, else the last row in kvc.
  int32_t last_row;
  int64_t ldq;
};
hipError_t launch_attention_gen(const GenAttnArgs& a, hipStream_t s);
// Descriptors of the last positions of a chunk's sequences in blocks of R:
// block b (b < nb) covers local sequences [b R, min(n, (b + 1) R)):
// ldesc[b] = {chunk's first token, rows, chunk's first sequence + b R, rows}.
hipError_t launch_last_desc(const int64_t* chunk_desc, int64_t* ldesc, int32_t nb, int64_t R, hipStream_t s);
// The last position of sequence i (i < ldesc[D_NSEQ]): its 16-bit
// normalised row h (d values), row scale and position, into row i of hl, rsl
// and posl; sequences with no own row are left as they are.
hipError_t launch_last_h(const int64_t* ldesc, const int64_t* cu, const void* h, const float* rs, const int32_t* pos,
                         int32_t d, void* hl, float* rsl, int32_t* posl, int64_t R, hipStream_t s);
// xl[i] = x[last row of sequence i] (fp32 rows of d), i < ldesc[D_NSEQ];
// sequences with no own row are left as they are.
hipError_t launch_last_rows(const int64_t* ldesc, const int64_t* cu, const float* x, int32_t d, float* xl,
                            int64_t R, hipStream_t s);
// hf[i] = x[i] / rms * g in 16 bits, i < gen_desc[D_NSEQ]
hipError_t launch_norm_rows(const int64_t* gen_desc, const float* x, const float* g, int32_t d, float eps, void* hf,
                            int32_t act, int64_t seq_ub, hipStream_t s);
// Argmax over a block of full-vocabulary rows given as the head GEMM's
// EPI_ARGMAX partials (int2 [rows][vocab / 64]; ties to the lowest id):
// row r is sequence i = row0 + r; its token goes to gen[(seq_begin + i) * G +
// step] (pad_id once the sequence has ended), tok[i] and done[i].
hipError_t launch_gen_argmax(const void* part, int32_t vocab, const int64_t* cnt, int64_t row0,
                             const int64_t* gen_desc, int32_t step, int32_t G, int32_t eos, int32_t pad,
                             int32_t* tok, int32_t* done, int32_t* gen, hipStream_t s);
struct LikePattern {
  int32_t n;
  int32_t tok[AIQ_MAX_LIKE];
};
// label[i] = 1 iff the generated tokens of selected row i (up to its end
// token) contain the pattern contiguously (every row for an empty pattern).
hipError_t launch_gen_like(const int32_t* gen, const int64_t* n_ptr, int64_t n_ub, int32_t G, int32_t eos,
                           const LikePattern& pat, int32_t* label, hipStream_t s);
// dst[i * per_row ..] = src[i * per_row ..] for i < min(*n_ptr, cap_rows)
hipError_t launch_copy_rows_i32(const int32_t* src, const int64_t* n_ptr, int64_t n_ub, int32_t per_row,
                                int32_t* dst, int64_t cap_rows, hipStream_t s);

// Fixed device scratch of the entry point that allocates nothing
// (aiq_run_relational_static): STATIC_SCRATCH_BYTES of device memory per GPU,
// held until the process ends.  Returns its device address on the current
// device (looked up once per device) and its size.
constexpr size_t STATIC_SCRATCH_BYTES = size_t(16) << 20;
hipError_t static_scratch(void** ptr, size_t* bytes);

}  // namespace aiq
