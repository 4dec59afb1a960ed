// Host side of the C ABI: validation, plan construction, workspace carving and
// the single-stream enqueue of the whole AI query.
//
// The sequence of launches is fixed on the host; every data-dependent extent
// (selected rows, tokens, sequences per chunk) is produced and consumed on the
// device.  The host loops over an upper bound of chunks computed from sizes it
// knows (table rows and list tokens); kernels of a chunk with no work exit at
// once.  Nothing is copied between host and device and nothing synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "aiq_internal.h"

using namespace aiq;

struct aiq_plan {
  aiq_model model;
  std::vector<aiq_layer> layers;
  bool has_probe = false, has_build = false, has_query = false;
  bool rel_only = false;   // AIQ_PLAN_RELATIONAL_ONLY
  bool lb_compact = false; // single-launch compaction (not AIQ_PLAN_MULTIPASS_COMPACT)
  // the prompt prefix is prefilled once per run and its keys / values are
  // shared by every row (16-bit models, unless AIQ_PLAN_UNSHARED_PREFIX)
  bool share_prefix = false;
  // the last layer runs its rows after the q|k|v projection for the last
  // position of each sequence only (16-bit models, unless
  // AIQ_PLAN_FULL_LAST_LAYER)
  bool prune_last = false;
  // ... and its q|k|v projection computes keys and values for every position
  // but queries for the last positions only
  bool q_last_only = false;
  int32_t gen = 0;        // AI_TRANSFORM: tokens generated per selected row (0: AI_IF)
  bool pairs = false;     // Q4: the sequences are candidate pairs of selected rows
  int64_t n_seq_ub = 0;   // upper bound on sequences: selected rows, or max_pairs
  int32_t gen_blocks = 0; // row blocks of the full-vocabulary head
  aiq_table probe{}, build{};
  std::vector<aiq_col> probe_cols, build_cols;
  aiq_query q{};
  int n_layers = 0;
  // derived model shapes
  int hd = 0, d_q = 0, d_kv = 0, n_qkv = 0, n_up = 0;
  bool bf16 = false;   // 16-bit MFMA path (bf16 or fp16 operands)
  int act = 0;         // activation element type of that path (1 bf16, 2 fp16; 0 fp32 model)
  // derived run shapes
  int64_t n_rows = 0, t_ub = 0, chunk_tokens = 0, n_chunks = 0, t_cap = 0, seq_ub = 0;
  int32_t max_seq = 0;
  int hash_log2 = 0;
  // GROUP BY over arbitrary keys (n_group_keys == 0): table of 2^hgroup_log2
  // slots for at most hgroup_max distinct keys
  int hgroup_log2 = 0;
  int64_t hgroup_max = 0;
  DPredList probe_preds{}, build_preds{};
  Prefix prefix{};
};

namespace {

constexpr size_t ALIGN = 256;

struct Carver {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off += (bytes + ALIGN - 1) / ALIGN * ALIGN;
    return o;
  }
};

bool int_dtype(int dt) { return dt == AIQ_I8 || dt == AIQ_I16 || dt == AIQ_I32; }

int64_t dtype_min(int dt) { return dt == AIQ_I8 ? INT8_MIN : dt == AIQ_I16 ? INT16_MIN : INT32_MIN; }
int64_t dtype_max(int dt) { return dt == AIQ_I8 ? INT8_MAX : dt == AIQ_I16 ? INT16_MAX : INT32_MAX; }

aiq_status make_preds(const aiq_pred* src, int n, const std::vector<aiq_col>& cols, DPredList* out) {
  if (n < 0 || n > AIQ_MAX_PREDS) return AIQ_EINVAL;
  out->n = n;
  for (int i = 0; i < n; ++i) {
    const aiq_pred& p = src[i];
    if (p.col < 0 || p.col >= static_cast<int>(cols.size())) return AIQ_EINVAL;
    const aiq_col& c = cols[p.col];
    if (!int_dtype(c.dtype) && c.dtype != AIQ_F32) return AIQ_EUNSUPPORTED;
    if (p.op < AIQ_LT || p.op > AIQ_IN) return AIQ_EINVAL;
    if (c.dtype == AIQ_F32 && p.op == AIQ_IN) return AIQ_EUNSUPPORTED;
    DPred& d = out->p[i];
    d.data = c.data;
    d.dtype = c.dtype;
    d.op = p.op;
    d.k = p.k;
    d.fk = p.fk;
    d.n_set = 0;
    if (p.op == AIQ_IN) {
      if (p.n_set < 0 || p.n_set > AIQ_MAX_IN_SET) return AIQ_EINVAL;
      // values the column type cannot hold never match; drop them
      for (int j = 0; j < p.n_set; ++j)
        if (p.set[j] >= dtype_min(c.dtype) && p.set[j] <= dtype_max(c.dtype))
          d.set[d.n_set++] = static_cast<int32_t>(p.set[j]);
    }
  }
  return AIQ_OK;
}

// need_list: 0 no list column, 1 offsets (tokens optional), 2 offsets and tokens
aiq_status copy_table(const aiq_table* t, aiq_table* dst, std::vector<aiq_col>* cols, int need_list) {
  if (t->n_rows < 0 || t->n_rows > INT32_MAX) return AIQ_EINVAL;
  if (t->n_cols < 0 || (t->n_cols > 0 && !t->cols)) return AIQ_EINVAL;
  cols->assign(t->cols, t->cols + t->n_cols);
  for (const aiq_col& c : *cols) {
    if (!int_dtype(c.dtype) && c.dtype != AIQ_F32) return AIQ_EINVAL;
    if (!c.data && t->n_rows > 0) return AIQ_EINVAL;
    if (reinterpret_cast<uintptr_t>(c.data) % 16) return AIQ_EINVAL;   // columns are read in 16-byte vectors
  }
  if (need_list) {
    if (!t->list_offsets || (need_list == 2 && !t->list_tokens)) return AIQ_EINVAL;
    if (t->n_list_tokens < 0 || t->max_list_len < 1) return AIQ_EINVAL;
  }
  *dst = *t;
  dst->cols = cols->data();
  return AIQ_OK;
}

aiq_status validate_model(const aiq_model* m) {
  if (m->n_layers < 0 || m->d_model <= 0 || m->n_heads <= 0 || m->n_kv_heads <= 0 || m->d_ff <= 0 ||
      m->vocab <= 0)
    return AIQ_EINVAL;
  if (m->d_model % m->n_heads) return AIQ_EINVAL;
  if (m->n_heads % m->n_kv_heads) return AIQ_EINVAL;
  const int hd = m->d_model / m->n_heads;
  if (hd != 32 && hd != 64 && hd != 128) return AIQ_EINVAL;
  if (m->wdtype != AIQ_F32 && m->wdtype != AIQ_BF16 && m->wdtype != AIQ_F16) return AIQ_EINVAL;
  if (m->act != AIQ_ACT_GELU_ERF && m->act != AIQ_ACT_SWIGLU) return AIQ_EINVAL;
  if (!(m->norm_eps > 0.0) || !(m->rope_theta > 0.0)) return AIQ_EINVAL;
  if (!m->emb || !m->final_norm || !m->lm_head || (m->n_layers > 0 && !m->layers)) return AIQ_EINVAL;
  for (int l = 0; l < m->n_layers; ++l) {
    const aiq_layer& L = m->layers[l];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.ffn_norm || !L.w_gate || !L.w_down)
      return AIQ_EINVAL;
    if (m->act == AIQ_ACT_SWIGLU && !L.w_up) return AIQ_EINVAL;
  }
  const int d = m->d_model, d_q = m->n_heads * hd, d_kv = m->n_kv_heads * hd;
  if (m->wdtype == AIQ_BF16 || m->wdtype == AIQ_F16) {
    // MFMA path: 256-wide output tiles, 64-deep K steps, rotary pairs in registers
    if (m->act != AIQ_ACT_SWIGLU) return AIQ_EUNSUPPORTED;
    if (hd == 32) return AIQ_EUNSUPPORTED;
    if ((d_q + 2 * d_kv) % 256 || d % 256 || (2 * m->d_ff) % 256) return AIQ_EUNSUPPORTED;
    if (d % 64 || d_q % 64 || m->d_ff % 64) return AIQ_EUNSUPPORTED;
  } else {
    if (m->act != AIQ_ACT_GELU_ERF) return AIQ_EUNSUPPORTED;
    if (hd == 128) return AIQ_EUNSUPPORTED;
    if ((d_q + 2 * d_kv) % 64 || d % 64 || m->d_ff % 64 || d % 16 || d_q % 16 || m->d_ff % 16)
      return AIQ_EUNSUPPORTED;
  }
  return AIQ_OK;
}

struct Layout {
  size_t ctr, mask, blk_cnt, blk_off, sel, payload, lens, label, logits, cu, blk_tok, tok_off, packed, hkeys, hvals,
      bins, desc, rcos, rsin, rrev, x, delta, h, qkv, att, ffn, pos, hf, ssp, rs, pkv, ptok, pcu, pdesc, pxlast,
      kvc, gkv, glog, gtok, gdone, gen, gdesc, gcnt, kcount, koff, prank, psorted, pcnt, poff, pscan, pa, pb,
      lb, xl, ldesc, laux, jkeys, jvals, jlog2, gslot, gkey0, gval0, gkey1, gval1, ghist, gn, total;
};

size_t act_bytes(const aiq_plan* p) { return p->bf16 ? 2 : 4; }

// Per-token residual-stream bytes: x (fp32) plus, on the fp32 path, the
// pending projection output `delta`, or on the MFMA path the per-slice sums
// of squares (one float per 64 columns) and the row scale.
size_t resid_bytes(const aiq_plan* p) {
  const size_t d = static_cast<size_t>(p->model.d_model);
  return d * 4 + (p->bf16 ? d / 16 + 4 : d * 4);
}

// x, delta / ssp / rs and the 16-bit or fp32 activations of one chunk of T tokens
void take_resid(const aiq_plan* p, Carver& c, Layout& L, size_t T) {
  const size_t d = static_cast<size_t>(p->model.d_model);
  const size_t ab = act_bytes(p);
  L.x = c.take(T * d * 4);
  if (p->bf16) {
    L.ssp = c.take(T * (d / 64) * 4);
    L.rs = c.take((T + 256) * 4);   // GEMMs read row scales in 256-row tiles up to the tile edge
  } else {
    L.delta = c.take(T * d * 4);
  }
  L.h = c.take(T * d * ab);
  L.qkv = c.take(T * p->n_qkv * ab);
  L.att = c.take(T * p->d_q * ab);
  L.ffn = c.take(T * p->model.d_ff * ab);
  L.pos = c.take((T + 256) * 4);   // GEMM tiles read positions up to the tile edge
}

// Last positions of a chunk go through the pruned last layer in blocks of at
// most LAST_ROWS_MAX sequences (their fp32 residual rows: 3 GB at d 3072).
// Every block is launched for every chunk pass, also where the selection
// leaves it empty, so larger blocks mean fewer empty launches.
constexpr int64_t LAST_ROWS_MAX = 262144;

int64_t last_rows(int64_t seq) { return std::max<int64_t>(std::min<int64_t>(seq, LAST_ROWS_MAX), 1); }
int32_t last_blocks(int64_t seq) {
  const int64_t R = last_rows(seq);
  return static_cast<int32_t>(std::max<int64_t>((seq + R - 1) / R, 1));
}

// the pruned last layer's residual rows and block descriptors, for chunks of
// at most `seq` sequences
void take_last(const aiq_plan* p, Carver& c, Layout& L, int64_t seq) {
  if (!p->prune_last) return;
  L.xl = c.take(static_cast<size_t>(last_rows(seq)) * p->model.d_model * 4);
  L.ldesc = c.take(static_cast<size_t>(last_blocks(seq)) * D_STRIDE * 8);
  // row scales and positions of the last positions (GEMM tiles read 256 rows)
  if (p->q_last_only) L.laux = c.take(static_cast<size_t>(last_rows(seq) + 256) * 8);
}

Layout run_layout(const aiq_plan* p) {
  Layout L{};
  Carver c;
  const int64_t n = p->n_rows;
  const int64_t ns = std::max<int64_t>(n, p->n_seq_ub);   // rows, or candidate pairs, whichever is more
  const int64_t nb = (ns + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK + 1;
  const int d = p->model.d_model;
  const size_t ab = act_bytes(p);
  L.ctr = c.take(C_COUNT * 8);
  L.mask = c.take(static_cast<size_t>(nb) * REL_WORDS_PER_BLOCK * 8);
  L.blk_cnt = c.take(static_cast<size_t>(nb) * 4);
  L.blk_off = c.take(static_cast<size_t>(nb + 1) * 8);
  L.sel = c.take(static_cast<size_t>(n + 1) * 4);
  L.payload = c.take(static_cast<size_t>(n + 1) * 4);
  L.lens = c.take(static_cast<size_t>(ns + 24) * 4);   // read in 16-entry groups from an 8-aligned start
  L.label = c.take(static_cast<size_t>(ns + 1) * 4);
  L.logits = c.take(static_cast<size_t>(ns + 1) * p->q.n_labels * 4);
  L.cu = c.take(static_cast<size_t>(ns + 1) * 8);
  L.blk_tok = c.take(static_cast<size_t>(nb) * 8);
  L.tok_off = c.take(static_cast<size_t>(nb + 1) * 8);
  L.lb = c.take(static_cast<size_t>((ns + LB_MIN_ROWS - 1) / LB_MIN_ROWS + 1) * 4 * 8);
  const size_t hcap = p->hash_log2 ? (size_t(1) << p->hash_log2) : 1;
  L.hkeys = c.take(hcap * 4);
  L.hvals = c.take(hcap * 4);
  if (p->has_build) {   // the build table rehashed for LDS probes
    L.jkeys = c.take(JOIN_LDS_SLOTS * 4);
    L.jvals = c.take(JOIN_LDS_SLOTS * 4);
    L.jlog2 = c.take(4);
  }
  if (p->rel_only) {   // no packed batch, model activations or groups
    L.total = c.off;
    return L;
  }
  L.packed = c.take(static_cast<size_t>(p->t_ub + 1) * 4);
  L.bins = c.take(std::max<size_t>(static_cast<size_t>(std::max(p->q.n_group_keys, 1)) * 16,
                                   SUM_BLOCKS * sizeof(double)));   // group bins, or SUM partials
  if (p->hgroup_log2) {   // hash GROUP BY: slot | count | sum arrays, sort buffers, digit histograms
    const size_t hs = size_t(1) << p->hgroup_log2, mg = static_cast<size_t>(p->hgroup_max);
    L.gslot = c.take(hs * 24);
    L.gkey0 = c.take(mg * 4);
    L.gval0 = c.take(mg * 4);
    L.gkey1 = c.take(mg * 4);
    L.gval1 = c.take(mg * 4);
    L.ghist = c.take(static_cast<size_t>(256 * hash_group_sort_blocks(p->hgroup_max)) * 8);
    L.gn = c.take(8);
  }
  L.desc = c.take(static_cast<size_t>(p->n_chunks) * D_STRIDE * 8);
  L.rcos = c.take(static_cast<size_t>(p->max_seq) * (p->hd / 2) * 4);
  L.rsin = c.take(static_cast<size_t>(p->max_seq) * (p->hd / 2) * 4);
  L.rrev = c.take(static_cast<size_t>(p->hd / 2) * 4);
  take_resid(p, c, L, static_cast<size_t>(p->t_cap));
  take_last(p, c, L, p->seq_ub);
  L.hf = 0;
  if (p->share_prefix) {   // per-layer q|k|v rows of the prefix, its batch, its last token's final state
    const size_t np = static_cast<size_t>(p->prefix.n);
    L.pkv = c.take(static_cast<size_t>(p->n_layers) * np * p->n_qkv * ab);
    L.ptok = c.take(np * 4);
    L.pcu = c.take(2 * 8);
    L.pdesc = c.take(D_STRIDE * 8);
    L.pxlast = c.take(static_cast<size_t>(d) * 4);
  }
  if (p->pairs) {   // key histogram and offsets, ranks, the rows sorted by key, partner counts, pair lists
    const size_t nk = static_cast<size_t>(p->q.n_group_keys);
    L.kcount = c.take(nk * 4);
    L.koff = c.take((nk + 1) * 8);
    L.prank = c.take(static_cast<size_t>(n + 1) * 4);
    L.psorted = c.take(static_cast<size_t>(n + 1) * 4);
    L.pcnt = c.take(static_cast<size_t>(n + 1) * 4);
    L.poff = c.take(static_cast<size_t>(n + 1) * 8);
    L.pscan = c.take(static_cast<size_t>(2 * (std::max<int64_t>(ns, static_cast<int64_t>(nk)) / REL_ROWS_PER_BLOCK + 3)) * 8);
    L.pa = c.take(static_cast<size_t>(p->n_seq_ub) * 4);
    L.pb = c.take(static_cast<size_t>(p->n_seq_ub) * 4);
  }
  if (p->gen > 0) {   // AI_TRANSFORM: kept prompt keys / values, generated-token cache, head, tokens
    const size_t G = static_cast<size_t>(p->gen), su = static_cast<size_t>(p->seq_ub);
    L.kvc = c.take(static_cast<size_t>(p->n_layers) * p->t_cap * p->n_qkv * ab);
    L.gkv = c.take(static_cast<size_t>(p->n_layers) * su * G * 2 * p->d_kv * ab);
    L.hf = c.take(su * d * ab);
    L.glog = c.take(std::min<size_t>(su, GEN_HEAD_ROWS) * (p->model.vocab / 64) * 8);   // per-64-column maxima
    L.gtok = c.take(su * 4);
    L.gdone = c.take(su * 4);
    L.gen = c.take(static_cast<size_t>(n + 1) * G * 4);
    L.gdesc = c.take(D_STRIDE * 8);
    L.gcnt = c.take(static_cast<size_t>(p->gen_blocks) * 8);
  }
  L.total = c.off;
  return L;
}

// prefill-only layout for up to max_tokens tokens (and as many sequences)
Layout prefill_layout(const aiq_plan* p, int64_t max_tokens) {
  Layout L{};
  Carver c;
  const int d = p->model.d_model;
  const size_t ab = act_bytes(p);
  const size_t T = static_cast<size_t>(max_tokens);
  L.ctr = c.take(C_COUNT * 8);
  L.desc = c.take(D_STRIDE * 8);
  L.cu = c.take((T + 1) * 8);
  L.label = c.take((T + 1) * 4);
  L.rcos = c.take(T * (p->hd / 2) * 4);
  L.rsin = c.take(T * (p->hd / 2) * 4);
  L.rrev = c.take(static_cast<size_t>(p->hd / 2) * 4);
  take_resid(p, c, L, T);
  take_last(p, c, L, static_cast<int64_t>(T));   // sequences <= tokens
  L.hf = c.take(T * d * ab);
  L.total = c.off;
  return L;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

struct Tracer {
  aiq_trace* t;
  hipStream_t s;
  bool open = false;
  int kind = 0;
  void begin(int k) {
    open = false;
    if (!t || !t->events || !t->tags || t->count >= t->capacity || !((t->kind_mask >> k) & 1u)) return;
    if (hipEventRecord(static_cast<hipEvent_t>(t->events[2 * t->count]), s) != hipSuccess) return;
    open = true;
    kind = k;
  }
  void end() {
    if (!open) return;
    if (hipEventRecord(static_cast<hipEvent_t>(t->events[2 * t->count + 1]), s) == hipSuccess) {
      t->tags[t->count] = kind;
      t->count += 1;
    }
    open = false;
  }
};

#define HIP_TRY(expr)                         \
  do {                                        \
    if ((expr) != hipSuccess) return AIQ_EHIP; \
  } while (0)

#define TRACED(tr, kind, expr) \
  do {                         \
    (tr).begin(kind);          \
    HIP_TRY(expr);             \
    (tr).end();                \
  } while (0)

// Options of a chunk pass.  Shared prefix: the prefix's own pass stores each
// layer's q|k|v rows in qkv_layers (npre rows per layer) and runs no head;
// the row passes read them back (pkv_layers), number positions from npre and
// give rows without own tokens the prefix's final state (x_pre).
// AI_TRANSFORM: the row passes keep every layer's q|k|v rows in qkv_layers
// (qkv_rows rows per layer) for the generation steps.
struct PrefixUse {
  void* qkv_layers = nullptr;
  int64_t qkv_rows = 0;
  const void* pkv_layers = nullptr;
  int32_t npre = 0;
  const float* x_pre = nullptr;
  bool head = true;
};

// Enqueues embedding, the layer stack and the label head for one chunk.
aiq_status enqueue_chunk(const aiq_plan* p, void* ws, const Layout& L, const int64_t* desc, const int64_t* cu,
                         int64_t* ctr, const int32_t* packed, int64_t t_cap, int64_t seq_ub, int32_t* label_out,
                         float* logits_out, void* hf_out, Tracer& tr, hipStream_t s,
                         const PrefixUse& pu = PrefixUse{}) {
  const aiq_model& m = p->model;
  const int d = m.d_model;
  const int64_t* m_ptr = desc + D_NTOK;
  float* x = at<float>(ws, L.x);
  // fp32 path: output of the last O / down projection, added by the next norm
  float* delta = p->bf16 ? nullptr : at<float>(ws, L.delta);
  // MFMA path: per-slice sums of squares and row scales of the norm folded into the next projection
  float* ssp = p->bf16 ? at<float>(ws, L.ssp) : nullptr;
  float* rs = p->bf16 ? at<float>(ws, L.rs) : nullptr;
  void* h = at<void>(ws, L.h);
  void* qkv = at<void>(ws, L.qkv);
  void* att = at<void>(ws, L.att);
  void* ffn = at<void>(ws, L.ffn);
  int32_t* pos = at<int32_t>(ws, L.pos);
  const float* rcos = at<float>(ws, L.rcos);
  const float* rsin = at<float>(ws, L.rsin);
  const float* rrev = at<float>(ws, L.rrev);
  const float eps = static_cast<float>(m.norm_eps);
  auto gemm = [&](int epi, const void* A, int64_t lda, int N, int K, const void* B0, const void* B1, const void* B2,
                  void* C, int64_t ldc, const float* gnext = nullptr, const int64_t* rows_ptr = nullptr,
                  int64_t rows_ub = 0, float* xr = nullptr, bool x_table = false) {
    GemmArgs g{};
    g.A = A;
    g.lda = lda;
    g.m_ptr = rows_ptr ? rows_ptr : m_ptr;
    g.m_ub = rows_ptr ? rows_ub : t_cap;
    g.N = N;
    g.K = K;
    g.B0 = B0;
    g.B1 = B1;
    g.B2 = B2;
    g.n_q = p->d_q;
    g.n_kv = p->d_kv;
    g.hd = p->hd;
    g.C = C;
    g.ldc = ldc;
    g.pos = pos;
    g.rope_cos = rcos;
    g.rope_sin = rsin;
    g.rope_rev = rrev;
    g.f16 = p->act == 2;
    g.rs = rs;
    if (epi == EPI_RESID) {
      g.x = xr ? xr : x;
      g.gnext = gnext;
      g.hout = h;
      g.ssp = ssp;
      g.n_part = d / 64;
      if (x_table) {   // the residual before the first layer is the token's table row
        epi = EPI_RESID_EMB;
        g.x_emb = m.emb;
        g.x_tok = packed;
        g.x_tok_desc = desc;
        g.vocab = m.vocab;
      }
    }
    return p->bf16 ? launch_gemm_bf16(epi, g, s) : launch_gemm_f32(epi, g, s);
  };
  // a section of the q|k|v projection (rotary on q and k columns): n_q query
  // and n_kv key columns, then values, with its own rows, row scales and positions
  auto gemm_part = [&](const void* A, const int64_t* rows_ptr, int64_t rows_ub, int N, int n_q, int n_kv,
                       const void* B0, const void* B1, const void* B2, void* C, int64_t ldc, const float* rsr,
                       const int32_t* posr) {
    GemmArgs g{};
    g.A = A;
    g.lda = d;
    g.m_ptr = rows_ptr;
    g.m_ub = rows_ub;
    g.N = N;
    g.K = d;
    g.B0 = B0;
    g.B1 = B1;
    g.B2 = B2;
    g.n_q = n_q;
    g.n_kv = n_kv;
    g.hd = p->hd;
    g.C = C;
    g.ldc = ldc;
    g.pos = posr;
    g.rope_rev = rrev;
    g.f16 = p->act == 2;
    g.rs = rsr;
    return launch_gemm_bf16(EPI_QKV_ROPE, g, s);
  };
  HeadArgs ha{};
  ha.desc = desc;
  ha.cu = cu;
  ha.x = x;
  ha.delta = p->n_layers > 0 ? delta : nullptr;   // null on the MFMA path: x is complete
  ha.g = m.final_norm;
  ha.eps = eps;
  ha.d = d;
  ha.lm_head = m.lm_head;
  ha.wdtype = m.wdtype;
  ha.n_labels = (p->has_query && p->gen == 0) ? p->q.n_labels : 0;
  for (int k = 0; k < ha.n_labels; ++k) ha.labels[k] = p->q.label_ids[k];
  ha.decision = p->has_query ? p->q.decision : AIQ_DECIDE_BINARY_GT;
  ha.label_out = ha.n_labels >= 2 ? label_out : nullptr;
  ha.logits_out = ha.n_labels >= 2 ? logits_out : nullptr;
  ha.hf_out = hf_out;
  ha.hf_act = p->act;
  ha.seq_ub = seq_ub;
  ha.x_pre = pu.x_pre;
  // the last layer for the last positions only (the prefix pass, which has
  // no head, leaves its last position's final residual in row 0 of xl)
  const bool prune = p->prune_last;

  if (p->bf16) {
    // MFMA path: each RMSNorm is split between the producer of its input and
    // the projection that consumes it.  h = x * g (16-bit) and the row sums of
    // x^2 come from the embedding or from the residual projection's epilogue;
    // the consuming projection scales its rows by 1/rms, since
    // (x / rms * g) . W^T = ((x * g) . W^T) / rms.
    const float* g0 = p->n_layers > 0 ? p->layers[0].attn_norm : m.final_norm;
    const int32_t pos_base = pu.pkv_layers ? pu.npre : 0;
    // x after the embedding is the table row itself: the first layer's O
    // projection reads it from the table instead (unless that layer is the
    // pruned last one, which gathers x rows)
    const bool x_from_table = p->n_layers > 1 || (p->n_layers == 1 && !prune);
    TRACED(tr, AIQ_K_EMBED, launch_embed_norm(desc, cu, packed, m.emb, m.wdtype, d, m.vocab,
                                              x_from_table ? nullptr : x, pos, ctr, g0, eps,
                                              h, p->act, rs, t_cap, s, pos_base));
    const size_t pre_layer = static_cast<size_t>(pu.npre) * p->n_qkv * act_bytes(p);   // bytes per layer
    const size_t keep_layer = static_cast<size_t>(pu.qkv_rows) * p->n_qkv * act_bytes(p);
    for (int l = 0; l < p->n_layers; ++l) {
      const aiq_layer& W = p->layers[l];
      const bool last = l + 1 == p->n_layers;
      void* qkv_l = pu.qkv_layers ? static_cast<char*>(pu.qkv_layers) + l * keep_layer : qkv;
      if (last && prune && p->q_last_only) {
        // keys and values for every position (columns d_q.. of the q|k|v rows)
        TRACED(tr, AIQ_K_GEMM_QKV, gemm_part(h, m_ptr, t_cap, 2 * p->d_kv, 0, p->d_kv, W.wq, W.wk, W.wv,
                                             static_cast<char*>(qkv_l) + static_cast<size_t>(p->d_q) * act_bytes(p),
                                             p->n_qkv, rs, pos));
      } else {
        TRACED(tr, AIQ_K_GEMM_QKV, gemm(EPI_QKV_ROPE, h, d, p->n_qkv, d, W.wq, W.wk, W.wv, qkv_l, p->n_qkv));
      }
      AttnArgs aa{};
      aa.qkv = qkv_l;
      if (pu.pkv_layers) {
        aa.pkv = static_cast<const char*>(pu.pkv_layers) + l * pre_layer;
        aa.npre = pu.npre;
      }
      aa.ld = p->n_qkv;
      aa.out = att;
      aa.ldo = p->d_q;
      aa.desc = desc;
      aa.cu = cu;
      aa.n_heads = m.n_heads;
      aa.n_kv = m.n_kv_heads;
      aa.hd = p->hd;
      aa.seq_ub = seq_ub;
      aa.out_act = p->act;
      if (last && prune) {
        // blocks of R sequences: attention of each last position over its
        // sequence (decode form), then O, norm, FFN and the head on those rows
        const int64_t R = last_rows(seq_ub);
        const int32_t nb = last_blocks(seq_ub);
        int64_t* ldesc = at<int64_t>(ws, L.ldesc);
        float* xl = at<float>(ws, L.xl);
        const size_t hf_row = static_cast<size_t>(d) * (p->act ? 2 : 4);
        TRACED(tr, AIQ_K_LAST, launch_last_desc(desc, ldesc, nb, R, s));
        for (int32_t b = 0; b < nb; ++b) {
          const int64_t* bd = ldesc + static_cast<int64_t>(b) * D_STRIDE;
          GenAttnArgs ga{};
          if (p->q_last_only) {
            // queries of the last positions: their h rows, row scales and
            // positions gathered, then the q projection (rotary) into ffn
            float* rsl = at<float>(ws, L.laux);
            int32_t* posl = reinterpret_cast<int32_t*>(rsl + R + 256);
            TRACED(tr, AIQ_K_LAST, launch_last_h(bd, cu, h, rs, pos, d, att, rsl, posl, R, s));
            TRACED(tr, AIQ_K_LAST, gemm_part(att, bd + D_NTOK, R, p->d_q, p->d_q, 0, W.wq, W.wk, W.wv, ffn, p->d_q,
                                             rsl, posl));
            ga.qkv = ffn;
            ga.ldq = p->d_q;
          }
          ga.kvc = qkv_l;
          ga.pkv = aa.pkv;
          ga.npre = aa.npre;
          ga.ld = p->n_qkv;
          ga.gen_desc = bd;
          ga.chunk_desc = desc;
          ga.cu = cu;
          ga.out = att;
          ga.n_heads = m.n_heads;
          ga.n_kv = m.n_kv_heads;
          ga.hd = p->hd;
          ga.out_act = p->act;
          ga.seq_ub = R;
          ga.last_row = 1;
          TRACED(tr, AIQ_K_LAST, launch_attention_gen(ga, s));
          TRACED(tr, AIQ_K_LAST, launch_last_rows(bd, cu, x, d, xl, R, s));
          TRACED(tr, AIQ_K_LAST, gemm(EPI_RESID, att, p->d_q, d, p->d_q, W.wo, nullptr, nullptr, nullptr, d,
                                      W.ffn_norm, bd + D_NTOK, R, xl));
          TRACED(tr, AIQ_K_LAST, launch_row_scale(bd, ssp, d / 64, d, eps, rs, R, s));
          TRACED(tr, AIQ_K_LAST, gemm(EPI_SWIGLU, h, d, 2 * m.d_ff, d, W.w_gate, W.w_up, nullptr, ffn, m.d_ff,
                                      nullptr, bd + D_NTOK, R));
          TRACED(tr, AIQ_K_LAST, gemm(EPI_RESID, ffn, m.d_ff, d, m.d_ff, W.w_down, nullptr, nullptr, nullptr, d,
                                      nullptr, bd + D_NTOK, R, xl));
          if (!pu.head) continue;
          HeadArgs hb = ha;
          hb.desc = bd;
          hb.x = xl;
          hb.x_compact = 1;
          hb.seq_ub = R;
          hb.hf_out = hf_out ? static_cast<char*>(hf_out) + static_cast<size_t>(b) * R * hf_row : nullptr;
          TRACED(tr, AIQ_K_HEAD, launch_head(hb, s));
        }
        break;
      }
      TRACED(tr, AIQ_K_ATTN, launch_attention_bf16(aa, s));
      TRACED(tr, AIQ_K_GEMM_O, gemm(EPI_RESID, att, p->d_q, d, p->d_q, W.wo, nullptr, nullptr, nullptr, d,
                                    W.ffn_norm, nullptr, 0, nullptr, l == 0 && x_from_table));
      TRACED(tr, AIQ_K_NORM, launch_row_scale(desc, ssp, d / 64, d, eps, rs, t_cap, s));
      TRACED(tr, AIQ_K_GEMM_UP, gemm(EPI_SWIGLU, h, d, 2 * m.d_ff, d, W.w_gate, W.w_up, nullptr, ffn, m.d_ff));
      // the head normalises the last position itself: after the last layer only x is needed
      TRACED(tr, AIQ_K_GEMM_DOWN, gemm(EPI_RESID, ffn, m.d_ff, d, m.d_ff, W.w_down, nullptr, nullptr, nullptr, d,
                                       last ? nullptr : p->layers[l + 1].attn_norm));
      if (!last) TRACED(tr, AIQ_K_NORM, launch_row_scale(desc, ssp, d / 64, d, eps, rs, t_cap, s));
    }
  } else {
  TRACED(tr, AIQ_K_EMBED, launch_embed(desc, cu, packed, m.emb, m.wdtype, d, m.vocab, x, pos, ctr, t_cap, s));
  for (int l = 0; l < p->n_layers; ++l) {
    const aiq_layer& W = p->layers[l];
    TRACED(tr, AIQ_K_NORM, launch_rmsnorm(desc, x, l ? delta : nullptr, W.attn_norm, d, eps, h, p->act, t_cap, s));
    TRACED(tr, AIQ_K_GEMM_QKV, gemm(EPI_QKV_ROPE, h, d, p->n_qkv, d, W.wq, W.wk, W.wv, qkv, p->n_qkv));
    if (!p->bf16)
      TRACED(tr, AIQ_K_GEMM_QKV, launch_rope_f32(desc, static_cast<float*>(qkv), p->n_qkv, p->d_q, p->d_kv, p->hd,
                                                 pos, rcos, rsin, t_cap, s));
    AttnArgs aa{};
    aa.qkv = qkv;
    aa.ld = p->n_qkv;
    aa.out = att;
    aa.ldo = p->d_q;
    aa.desc = desc;
    aa.cu = cu;
    aa.n_heads = m.n_heads;
    aa.n_kv = m.n_kv_heads;
    aa.hd = p->hd;
    aa.seq_ub = seq_ub;
    aa.out_act = p->act;
    TRACED(tr, AIQ_K_ATTN, p->bf16 ? launch_attention_bf16(aa, s) : launch_attention_f32(aa, s));
    TRACED(tr, AIQ_K_GEMM_O, gemm(EPI_STORE_F32, att, p->d_q, d, p->d_q, W.wo, nullptr, nullptr, delta, d));
    TRACED(tr, AIQ_K_NORM, launch_rmsnorm(desc, x, delta, W.ffn_norm, d, eps, h, p->act, t_cap, s));
    if (p->bf16)
      TRACED(tr, AIQ_K_GEMM_UP, gemm(EPI_SWIGLU, h, d, 2 * m.d_ff, d, W.w_gate, W.w_up, nullptr, ffn, m.d_ff));
    else
      TRACED(tr, AIQ_K_GEMM_UP, gemm(EPI_GELU, h, d, m.d_ff, d, W.w_gate, nullptr, nullptr, ffn, m.d_ff));
    TRACED(tr, AIQ_K_GEMM_DOWN, gemm(EPI_STORE_F32, ffn, m.d_ff, d, m.d_ff, W.w_down, nullptr, nullptr, delta, d));
  }
  }
  if (!pu.head || prune) return AIQ_OK;   // pruned: the head ran per block of last positions
  TRACED(tr, AIQ_K_HEAD, launch_head(ha, s));
  return AIQ_OK;
}

// AI_TRANSFORM for the sequences of one chunk, after its prefill pass (which
// kept every layer's q|k|v rows and wrote each sequence's normalised last
// row to hf): the first token from hf, then gen - 1 steps of one row per
// sequence through the layer stack and the full-vocabulary head.
aiq_status enqueue_generation(const aiq_plan* p, void* ws, const Layout& L, const int64_t* cdesc, const int64_t* cu,
                              const PrefixUse& pu, Tracer& tr, hipStream_t s) {
  const aiq_model& m = p->model;
  const aiq_query& q = p->q;
  const int d = m.d_model, G = p->gen;
  const size_t ab = act_bytes(p);
  const int64_t su = p->seq_ub;
  int64_t* gd = at<int64_t>(ws, L.gdesc);
  int64_t* cnt = at<int64_t>(ws, L.gcnt);
  int32_t* tok = at<int32_t>(ws, L.gtok);
  int32_t* done = at<int32_t>(ws, L.gdone);
  int32_t* gen = at<int32_t>(ws, L.gen);
  float* logits = at<float>(ws, L.glog);
  void* hf = at<void>(ws, L.hf);
  float* x = at<float>(ws, L.x);
  float* ssp = at<float>(ws, L.ssp);
  float* rs = at<float>(ws, L.rs);
  void* h = at<void>(ws, L.h);
  void* qkv = at<void>(ws, L.qkv);
  void* att = at<void>(ws, L.att);
  void* ffn = at<void>(ws, L.ffn);
  int32_t* pos = at<int32_t>(ws, L.pos);
  const float eps = static_cast<float>(m.norm_eps);
  const int32_t npre = pu.pkv_layers ? pu.npre : 0;
  TRACED(tr, AIQ_K_DECODE, launch_gen_desc(cdesc, gd, cnt, p->gen_blocks, s));
  TRACED(tr, AIQ_K_DECODE, launch_fill_i32(done, su, 0, s));
  auto gemm = [&](int epi, const void* A, int64_t lda, const int64_t* m_ptr, int64_t m_ub, int N, int K,
                  const void* B0, const void* B1, const void* B2, void* C, int64_t ldc, const float* gnext,
                  bool resid) {
    GemmArgs g{};
    g.A = A;
    g.lda = lda;
    g.m_ptr = m_ptr;
    g.m_ub = m_ub;
    g.N = N;
    g.K = K;
    g.B0 = B0;
    g.B1 = B1;
    g.B2 = B2;
    g.n_q = p->d_q;
    g.n_kv = p->d_kv;
    g.hd = p->hd;
    g.C = C;
    g.ldc = ldc;
    g.pos = pos;
    g.rope_rev = at<float>(ws, L.rrev);
    g.f16 = p->act == 2;
    g.rs = rs;
    if (resid) {
      g.x = x;
      g.gnext = gnext;
      g.hout = h;
      g.ssp = ssp;
      g.n_part = d / 64;
    }
    return launch_gemm_bf16(epi, g, s);
  };
  // full-vocabulary head over hf in row blocks, argmax into generated slot `step`
  auto next_tokens = [&](int step) -> aiq_status {
    for (int b = 0; b < p->gen_blocks; ++b) {
      const int64_t row0 = static_cast<int64_t>(b) * GEN_HEAD_ROWS;
      TRACED(tr, AIQ_K_DECODE_HEAD, gemm(EPI_ARGMAX, static_cast<const char*>(hf) + row0 * d * ab, d, cnt + b,
                                         std::min<int64_t>(su - row0, GEN_HEAD_ROWS), m.vocab, d, m.lm_head,
                                         nullptr, nullptr, logits, m.vocab / 64, nullptr, false));
      TRACED(tr, AIQ_K_DECODE_HEAD, launch_gen_argmax(logits, m.vocab, cnt + b, row0, gd, step, G, q.eos_id, q.pad_id,
                                                 tok, done, gen, s));
    }
    return AIQ_OK;
  };
  aiq_status e = next_tokens(0);
  if (e != AIQ_OK) return e;
  const int64_t* n_rows = gd + D_NTOK;
  const size_t kv_layer = static_cast<size_t>(pu.qkv_rows) * p->n_qkv * ab;
  const size_t pre_layer = static_cast<size_t>(npre) * p->n_qkv * ab;
  const size_t gkv_layer = static_cast<size_t>(su) * G * 2 * p->d_kv * ab;
  const float* g0 = p->n_layers > 0 ? p->layers[0].attn_norm : m.final_norm;
  for (int k = 0; k + 1 < G; ++k) {
    TRACED(tr, AIQ_K_DECODE, launch_gen_embed(gd, cu, tok, k, npre, m.emb, m.wdtype, d, m.vocab, x, pos, g0, eps, h,
                                              p->act, rs, su, s));
    for (int l = 0; l < p->n_layers; ++l) {
      const aiq_layer& W = p->layers[l];
      const bool last = l + 1 == p->n_layers;
      TRACED(tr, AIQ_K_DECODE, gemm(EPI_QKV_ROPE, h, d, n_rows, su, p->n_qkv, d, W.wq, W.wk, W.wv, qkv, p->n_qkv,
                                    nullptr, false));
      GenAttnArgs ga{};
      ga.qkv = qkv;
      ga.kvc = static_cast<const char*>(pu.qkv_layers) + l * kv_layer;
      ga.pkv = npre ? static_cast<const char*>(pu.pkv_layers) + l * pre_layer : nullptr;
      ga.npre = npre;
      ga.gkv = at<char>(ws, L.gkv) + l * gkv_layer;
      ga.step = k;
      ga.gen = G;
      ga.ld = p->n_qkv;
      ga.gen_desc = gd;
      ga.chunk_desc = cdesc;
      ga.cu = cu;
      ga.out = att;
      ga.n_heads = m.n_heads;
      ga.n_kv = m.n_kv_heads;
      ga.hd = p->hd;
      ga.out_act = p->act;
      ga.seq_ub = su;
      TRACED(tr, AIQ_K_DECODE_ATTN, launch_attention_gen(ga, s));
      TRACED(tr, AIQ_K_DECODE, gemm(EPI_RESID, att, p->d_q, n_rows, su, d, p->d_q, W.wo, nullptr, nullptr, nullptr,
                                    d, W.ffn_norm, true));
      TRACED(tr, AIQ_K_DECODE, launch_row_scale(gd, ssp, d / 64, d, eps, rs, su, s));
      TRACED(tr, AIQ_K_DECODE, gemm(EPI_SWIGLU, h, d, n_rows, su, 2 * m.d_ff, d, W.w_gate, W.w_up, nullptr, ffn,
                                    m.d_ff, nullptr, false));
      TRACED(tr, AIQ_K_DECODE, gemm(EPI_RESID, ffn, m.d_ff, n_rows, su, d, m.d_ff, W.w_down, nullptr, nullptr,
                                    nullptr, d, last ? nullptr : p->layers[l + 1].attn_norm, true));
      if (!last) TRACED(tr, AIQ_K_DECODE, launch_row_scale(gd, ssp, d / 64, d, eps, rs, su, s));
    }
    TRACED(tr, AIQ_K_DECODE, launch_norm_rows(gd, x, m.final_norm, d, eps, hf, p->act, su, s));
    e = next_tokens(k + 1);
    if (e != AIQ_OK) return e;
  }
  return AIQ_OK;
}

}  // namespace

extern "C" {

int32_t aiq_abi_version(void) { return AIQ_ABI_VERSION; }

const char* aiq_status_str(int32_t st) {
  switch (st) {
    case AIQ_OK: return "ok";
    case AIQ_EINVAL: return "invalid argument";
    case AIQ_EUNSUPPORTED: return "unsupported";
    case AIQ_ENOSPC: return "workspace or capacity too small";
    case AIQ_EHIP: return "HIP runtime error";
    case AIQ_ENOMEM: return "host out of memory";
    default: return "unknown status";
  }
}

aiq_status aiq_plan_create(const aiq_model* model, const aiq_table* probe, const aiq_table* build,
                           const aiq_query* query, const aiq_plan_opts* opts, aiq_plan** out) {
  if (!out) return AIQ_EINVAL;
  *out = nullptr;
  if (!model) return AIQ_EINVAL;
  aiq_status st = validate_model(model);
  if (st != AIQ_OK) return st;
  aiq_plan* p = new (std::nothrow) aiq_plan();
  if (!p) return AIQ_ENOMEM;
  auto fail = [&](aiq_status e) {
    delete p;
    return e;
  };
  p->model = *model;
  p->layers.assign(model->layers, model->layers + model->n_layers);
  p->model.layers = p->layers.data();
  p->n_layers = model->n_layers;
  if (opts && opts->n_layers_override > 0) p->n_layers = std::min(opts->n_layers_override, model->n_layers);
  if (opts && opts->n_layers_override < 0) p->n_layers = 0;
  p->hd = model->d_model / model->n_heads;
  p->d_q = model->n_heads * p->hd;
  p->d_kv = model->n_kv_heads * p->hd;
  p->n_qkv = p->d_q + 2 * p->d_kv;
  p->bf16 = model->wdtype == AIQ_BF16 || model->wdtype == AIQ_F16;
  p->act = model->wdtype == AIQ_F16 ? 2 : model->wdtype == AIQ_BF16 ? 1 : 0;
  p->n_up = p->bf16 ? 2 * model->d_ff : model->d_ff;
  {
    const int rep = model->n_kv_heads > 0 ? model->n_heads / model->n_kv_heads : 0;
    p->prune_last = p->bf16 && p->n_layers > 0 && (p->hd == 64 || p->hd == 128) &&
                    (rep == 1 || rep == 2 || rep == 3 || rep == 4 || rep == 8) &&
                    !(opts && (opts->flags & AIQ_PLAN_FULL_LAST_LAYER));
    // separate key/value and query projections need 256-wide sections; the
    // queries of the last positions go through the FFN buffer
    p->q_last_only = p->prune_last && (2 * p->d_kv) % 256 == 0 && p->d_q % 256 == 0 && model->d_ff >= p->d_q;
  }

  if (query) {
    p->has_query = true;
    p->q = *query;
    const aiq_query& q = p->q;
    if (q.gen_tokens < 0 || q.gen_tokens > AIQ_MAX_GEN) return fail(AIQ_EINVAL);
    p->gen = q.gen_tokens;
    if (p->gen > 0) {   // AI_TRANSFORM: generation replaces the label decision
      if (!p->bf16 || model->vocab % 256 || model->n_heads / model->n_kv_heads > 8) return fail(AIQ_EUNSUPPORTED);
      if (q.eos_id < -1 || q.eos_id >= model->vocab) return fail(AIQ_EINVAL);
      if (q.n_like < 0 || q.n_like > AIQ_MAX_LIKE) return fail(AIQ_EINVAL);
      for (int k = 0; k < q.n_like; ++k)
        if (q.like[k] < 0 || q.like[k] >= model->vocab) return fail(AIQ_EINVAL);
    } else {
      if (q.n_labels < 2 || q.n_labels > AIQ_MAX_LABELS) return fail(AIQ_EINVAL);
      for (int k = 0; k < q.n_labels; ++k)
        if (q.label_ids[k] < 0 || q.label_ids[k] >= model->vocab) return fail(AIQ_EINVAL);
      if (q.decision != AIQ_DECIDE_BINARY_GT && q.decision != AIQ_DECIDE_ARGMAX) return fail(AIQ_EINVAL);
    }
    if (q.n_prefix < 0 || q.n_prefix > AIQ_MAX_PREFIX) return fail(AIQ_EINVAL);
    for (int k = 0; k < q.n_prefix; ++k)
      if (q.prefix[k] < 0 || q.prefix[k] >= model->vocab) return fail(AIQ_EINVAL);
  }
  if (probe) {
    if (!query) return fail(AIQ_EINVAL);
    p->has_probe = true;
    p->rel_only = opts && (opts->flags & AIQ_PLAN_RELATIONAL_ONLY);
    if (opts && (opts->flags & ~(AIQ_PLAN_RELATIONAL_ONLY | AIQ_PLAN_UNSHARED_PREFIX | AIQ_PLAN_MULTIPASS_COMPACT |
                                 AIQ_PLAN_FULL_LAST_LAYER)))
      return fail(AIQ_EINVAL);
    st = copy_table(probe, &p->probe, &p->probe_cols, p->rel_only ? 1 : 2);
    if (st != AIQ_OK) return fail(st);
    const aiq_query& q = p->q;
    st = make_preds(q.preds, q.n_pred, p->probe_cols, &p->probe_preds);
    if (st != AIQ_OK) return fail(st);
    if (q.join != 0 && q.join != 1) return fail(AIQ_EINVAL);
    if ((q.join == 1) != (build != nullptr)) return fail(AIQ_EINVAL);
    if (q.join) {
      p->has_build = true;
      st = copy_table(build, &p->build, &p->build_cols, 0);
      if (st != AIQ_OK) return fail(st);
      const int nc = static_cast<int>(p->build_cols.size());
      if (q.build_key_col < 0 || q.build_key_col >= nc || q.build_payload_col < 0 || q.build_payload_col >= nc)
        return fail(AIQ_EINVAL);
      if (q.probe_key_col < 0 || q.probe_key_col >= static_cast<int>(p->probe_cols.size())) return fail(AIQ_EINVAL);
      if (!int_dtype(p->build_cols[q.build_key_col].dtype) || !int_dtype(p->build_cols[q.build_payload_col].dtype) ||
          !int_dtype(p->probe_cols[q.probe_key_col].dtype))
        return fail(AIQ_EUNSUPPORTED);
      st = make_preds(q.build_preds, q.n_build_pred, p->build_cols, &p->build_preds);
      if (st != AIQ_OK) return fail(st);
      int lg = 6;
      while ((int64_t(1) << lg) < 2 * std::max<int64_t>(p->build.n_rows, 1)) ++lg;
      if (lg > 30) return fail(AIQ_EUNSUPPORTED);
      p->hash_log2 = lg;
    }
    if (p->rel_only && q.agg != AIQ_AGG_COUNT) return fail(AIQ_EINVAL);
    if (q.pairs != 0 && q.pairs != 1) return fail(AIQ_EINVAL);
    if (q.pairs) {   // Q4 pairs: binary AI_IF over every two selected rows of a key
      if (p->rel_only || q.join || p->gen > 0 || q.agg != AIQ_AGG_COUNT || q.decision != AIQ_DECIDE_BINARY_GT)
        return fail(AIQ_EINVAL);
      if (q.pair_key_col < 0 || q.pair_key_col >= static_cast<int>(p->probe_cols.size())) return fail(AIQ_EINVAL);
      if (!int_dtype(p->probe_cols[q.pair_key_col].dtype)) return fail(AIQ_EUNSUPPORTED);
      if (q.n_group_keys <= 0) return fail(AIQ_EINVAL);
      if (q.n_group_keys > PAIR_MAX_KEYS) return fail(AIQ_EUNSUPPORTED);
      if (q.max_pairs <= 0 || q.max_pairs > INT32_MAX) return fail(AIQ_EINVAL);
      p->pairs = true;
    }
    switch (q.agg) {
      case AIQ_AGG_COUNT: break;
      case AIQ_AGG_AVG_LABEL_COUNT_BY:
        if (p->gen > 0) return fail(AIQ_EINVAL);   // no label to average
        if (q.group_col < 0 || q.group_col >= static_cast<int>(p->probe_cols.size())) return fail(AIQ_EINVAL);
        if (!int_dtype(p->probe_cols[q.group_col].dtype)) return fail(AIQ_EUNSUPPORTED);
        if (q.n_group_keys < 0) return fail(AIQ_EINVAL);
        break;
      case AIQ_AGG_COUNT_BY_PAYLOAD:
        if (!q.join || q.n_group_keys < 0) return fail(AIQ_EINVAL);
        break;
      case AIQ_AGG_SUM_F32:
        if (q.group_col < 0 || q.group_col >= static_cast<int>(p->probe_cols.size())) return fail(AIQ_EINVAL);
        if (p->probe_cols[q.group_col].dtype != AIQ_F32) return fail(AIQ_EUNSUPPORTED);
        break;
      default: return fail(AIQ_EINVAL);
    }
    p->n_rows = p->probe.n_rows;
    p->share_prefix = p->bf16 && q.n_prefix > 0 && p->n_layers > 0 && !p->rel_only &&
                      !(opts && (opts->flags & AIQ_PLAN_UNSHARED_PREFIX));
    // packed tokens: the row lists (two per pair), plus the prefix per sequence
    // unless it is shared
    const int64_t npre_packed = p->share_prefix ? 0 : q.n_prefix;
    // one-launch compaction when a block's token sum fits 32 bits
    p->lb_compact = !(opts && (opts->flags & AIQ_PLAN_MULTIPASS_COMPACT)) &&
                    static_cast<int64_t>(REL_ROWS_PER_BLOCK) * (p->probe.max_list_len + npre_packed) < (int64_t(1) << 31);
    const int64_t max_own = (p->pairs ? 2 : 1) * static_cast<int64_t>(p->probe.max_list_len);
    p->n_seq_ub = p->pairs ? q.max_pairs : p->n_rows;
    p->t_ub = p->pairs ? q.max_pairs * (max_own + npre_packed)
                       : p->probe.n_list_tokens + p->n_rows * npre_packed;
    p->max_seq = static_cast<int32_t>(max_own + q.n_prefix);   // positions (rotary table rows)
    // longest packed sequence: a chunk must hold one whole
    const int64_t max_packed = p->share_prefix ? std::max<int64_t>(max_own, q.n_prefix) : p->max_seq;
    // default chunk: about 96 GB of per-token activations (a third of one
    // MI355X's 288 GB), at most 4M tokens.  The host loops over an upper bound
    // of chunks fixed by the table's tokens; the passes a selective query
    // leaves empty each cost one launch per kernel, so larger chunks also mean
    // fewer of them (+ every layer's kept q|k|v rows when the rows go on to
    // generate)
    const int64_t per_tok = static_cast<int64_t>(resid_bytes(p)) +
                            static_cast<int64_t>(model->d_model + p->n_qkv + p->d_q + model->d_ff) *
                                (p->bf16 ? 2 : 4) + 4 +
                            (p->gen > 0 ? static_cast<int64_t>(p->n_layers) * p->n_qkv * 2 : 0);
    const int64_t def_chunk = std::min<int64_t>((int64_t(96) << 30) / per_tok, int64_t(4) << 20);
    int64_t ct = (opts && opts->chunk_tokens > 0) ? opts->chunk_tokens : def_chunk;
    ct = std::max<int64_t>(ct, max_packed);
    ct = std::min<int64_t>(ct, std::max<int64_t>(p->t_ub + p->n_seq_ub, max_packed));   // one chunk when all fits
    p->chunk_tokens = ct;
    p->t_cap = ct + max_packed;
    // chunks are cut by cu[i] + i (a sequence counts one unit besides its
    // tokens): a chunk then holds at most ct sequences even where token lists
    // are empty, and the keys of all sequences stay below n_chunks * ct
    p->n_chunks = std::max<int64_t>((p->t_ub + p->n_seq_ub + ct - 1) / ct, 1);
    p->seq_ub = std::min<int64_t>(p->n_seq_ub, ct);
    p->gen_blocks = p->gen > 0 ? static_cast<int32_t>((p->seq_ub + GEN_HEAD_ROWS - 1) / GEN_HEAD_ROWS) : 0;
    p->prefix.n = q.n_prefix;
    for (int k = 0; k < q.n_prefix; ++k) p->prefix.tok[k] = q.prefix[k];
    // GROUP BY over any int32 key: at most one group per selected row (by
    // probe column) or per build row (by the joined payload)
    if ((q.agg == AIQ_AGG_AVG_LABEL_COUNT_BY || q.agg == AIQ_AGG_COUNT_BY_PAYLOAD) && q.n_group_keys == 0) {
      p->hgroup_max = std::max<int64_t>(q.agg == AIQ_AGG_COUNT_BY_PAYLOAD ? std::min(p->build.n_rows, p->n_rows)
                                                                           : p->n_rows, 1);
      int lg = 6;
      while ((int64_t(1) << lg) < 2 * p->hgroup_max) ++lg;
      if (lg > 31) return fail(AIQ_EUNSUPPORTED);
      p->hgroup_log2 = lg;
    }
  }
  *out = p;
  return AIQ_OK;
}

void aiq_plan_destroy(aiq_plan* plan) { delete plan; }

aiq_status aiq_workspace_size(const aiq_plan* plan, size_t* bytes) {
  if (!plan || !bytes) return AIQ_EINVAL;
  if (!plan->has_probe) return AIQ_EINVAL;
  *bytes = run_layout(plan).total;
  return AIQ_OK;
}

aiq_status aiq_plan_passes(const aiq_plan* plan, int64_t* chunks, int32_t* prefix_pass) {
  if (!plan || !chunks || !prefix_pass || !plan->has_probe) return AIQ_EINVAL;
  *chunks = plan->rel_only ? 0 : plan->n_chunks;
  *prefix_pass = plan->share_prefix ? 1 : 0;
  return AIQ_OK;
}

aiq_status aiq_plan_chunk_tokens(const aiq_plan* plan, int64_t* chunk_tokens) {
  if (!plan || !chunk_tokens || !plan->has_probe) return AIQ_EINVAL;
  *chunk_tokens = plan->rel_only ? 0 : plan->chunk_tokens;
  return AIQ_OK;
}

aiq_status aiq_plan_last_layer_rows(const aiq_plan* plan, int32_t* last_rows_only) {
  if (!plan || !last_rows_only) return AIQ_EINVAL;
  *last_rows_only = plan->prune_last ? 1 : 0;
  return AIQ_OK;
}

aiq_status aiq_prefill_workspace_size(const aiq_plan* plan, int64_t max_tokens, size_t* bytes) {
  if (!plan || !bytes || max_tokens <= 0) return AIQ_EINVAL;
  *bytes = prefill_layout(plan, max_tokens).total;
  return AIQ_OK;
}

aiq_status aiq_run(const aiq_plan* p, void* ws, size_t ws_bytes, const aiq_out* out, aiq_trace* trace,
                   void* stream) {
  if (!p || !out || !out->scalars || !ws) return AIQ_EINVAL;
  if (!p->has_probe) return AIQ_EINVAL;
  if (out->ids_cap < 0 || (out->ids_cap > 0 && !out->ids)) return AIQ_EINVAL;
  const aiq_query& q = p->q;
  const bool grouped = q.agg == AIQ_AGG_AVG_LABEL_COUNT_BY || q.agg == AIQ_AGG_COUNT_BY_PAYLOAD;
  if (grouped && (!out->grp_key || !out->grp_count || !out->grp_sum || !out->grp_avg || out->grp_cap <= 0))
    return AIQ_EINVAL;
  if (q.agg == AIQ_AGG_SUM_F32 && !out->sum_out) return AIQ_EINVAL;
  if (out->sel_cap < 0) return AIQ_EINVAL;
  const Layout L = run_layout(p);
  if (ws_bytes < L.total) return AIQ_ENOSPC;
  if (reinterpret_cast<uintptr_t>(ws) % ALIGN) return AIQ_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Tracer tr{trace, s};

  int64_t* ctr = at<int64_t>(ws, L.ctr);
  uint64_t* mask = at<uint64_t>(ws, L.mask);
  int32_t* blk_cnt = at<int32_t>(ws, L.blk_cnt);
  int64_t* blk_off = at<int64_t>(ws, L.blk_off);
  int32_t* sel = at<int32_t>(ws, L.sel);
  int32_t* payload = at<int32_t>(ws, L.payload);
  int32_t* lens = at<int32_t>(ws, L.lens);
  int32_t* label = at<int32_t>(ws, L.label);
  float* logits = at<float>(ws, L.logits);
  int64_t* cu = at<int64_t>(ws, L.cu);
  int64_t* blk_tok = at<int64_t>(ws, L.blk_tok);
  int64_t* tok_off = at<int64_t>(ws, L.tok_off);
  int32_t* packed = at<int32_t>(ws, L.packed);
  int64_t* desc = at<int64_t>(ws, L.desc);
  const int64_t n = p->n_rows;

  HashArgs h{};
  if (p->has_build) {
    h.keys = at<int32_t>(ws, L.hkeys);
    h.vals = at<int32_t>(ws, L.hvals);
    h.cap_log2 = p->hash_log2;
  }
  StagedHash staged{};
  if (p->has_build) {
    staged.keys = at<int32_t>(ws, L.jkeys);
    staged.vals = at<int32_t>(ws, L.jvals);
    staged.log2_out = at<int32_t>(ws, L.jlog2);
  }
  const void* pkey = p->has_build ? p->probe_cols[q.probe_key_col].data : nullptr;
  const int32_t pkey_dt = p->has_build ? p->probe_cols[q.probe_key_col].dtype : AIQ_I32;

  HIP_TRY(launch_fill_i64(ctr, C_COUNT, 0, s));
  // ---- relational: WHERE (+ join) -> ascending survivor ids
  tr.begin(AIQ_K_REL);
  if (p->has_build) {
    HIP_TRY(launch_fill_i32(h.keys, int64_t(1) << p->hash_log2, HASH_EMPTY, s));
    const aiq_col& kc = p->build_cols[q.build_key_col];
    const aiq_col& pc = p->build_cols[q.build_payload_col];
    HIP_TRY(launch_hash_build(p->build_preds, kc.data, kc.dtype, pc.data, pc.dtype, p->build.n_rows, h, ctr, s));
    if (p->lb_compact) HIP_TRY(launch_hash_stage(h, staged, s));
  }
  const int32_t npre_rows = p->share_prefix ? 0 : q.n_prefix;   // prefix tokens packed into each row
  // selected ids go straight into the caller's ids when nothing else follows
  int32_t* ids1 = p->rel_only ? out->ids : sel;
  const int64_t cap1 = p->rel_only ? out->ids_cap : n;
  int32_t* ids2 = p->rel_only && out->sel_cap > 0 ? out->sel_ids : nullptr;
  const int64_t cap2 = p->rel_only ? out->sel_cap : 0;
  if (p->lb_compact) {
    // masks, compaction, join payloads and token offsets in one launch
    HIP_TRY(launch_select_lb(p->probe_preds, n, pkey, pkey_dt, h, p->has_build, p->has_build ? &staged : nullptr,
                             ids1, cap1, ids2, cap2, payload,
                             p->pairs ? nullptr : p->probe.list_offsets, p->probe.max_list_len, npre_rows, cu,
                             at<int64_t>(ws, L.lb), ctr, s));
  } else {
    HIP_TRY(launch_row_mask(p->probe_preds, n, pkey, pkey_dt, h, p->has_build, mask, blk_cnt, s));
    HIP_TRY(launch_scan_blocks(blk_cnt, nullptr, n, blk_off, ctr + C_SEL, s));
    // compaction: selected ids, join payloads, token counts and per-block token sums
    ScatterLens sl{p->probe.list_offsets, p->probe.max_list_len, npre_rows, lens, blk_tok};
    HIP_TRY(launch_scatter_rows(mask, blk_off, nullptr, n, nullptr, ids1, cap1, pkey, pkey_dt, h, p->has_build,
                                payload, ctr, s, ids2, cap2, p->pairs ? ScatterLens{} : sl));
  }
  tr.end();
  // the sequences: the selected rows, or the candidate pairs
  const int64_t* n_seq = ctr + (p->pairs ? C_PAIRS : C_SEL);
  const int64_t ns_ub = p->n_seq_ub;
  int32_t* pa = p->pairs ? at<int32_t>(ws, L.pa) : nullptr;
  int32_t* pb = p->pairs ? at<int32_t>(ws, L.pb) : nullptr;
  Prefix row_prefix{};
  if (!p->share_prefix) row_prefix = p->prefix;
  tr.begin(AIQ_K_PACK);
  if (p->pairs) {
    // ---- candidate pairs: rows sorted stably by key, partners, numbering, packing
    const aiq_col& kc = p->probe_cols[q.pair_key_col];
    const int32_t nk = q.n_group_keys;
    int32_t* kcount = at<int32_t>(ws, L.kcount);
    int64_t* koff = at<int64_t>(ws, L.koff);
    int32_t* prank = at<int32_t>(ws, L.prank);
    int32_t* psorted = at<int32_t>(ws, L.psorted);
    int32_t* pcnt = at<int32_t>(ws, L.pcnt);
    int64_t* poff = at<int64_t>(ws, L.poff);
    int64_t* pscan = at<int64_t>(ws, L.pscan);
    HIP_TRY(launch_fill_i32(kcount, nk, 0, s));
    HIP_TRY(launch_pair_key_count(sel, ctr + C_SEL, n, kc.data, kc.dtype, nk, kcount, ctr, s));
    HIP_TRY(launch_scan_i32_i64(kcount, nullptr, nk, koff, pscan, ctr + C_SCRATCH, s));
    HIP_TRY(launch_pair_rank(sel, ctr + C_SEL, kc.data, kc.dtype, nk, koff, prank, psorted, s));
    HIP_TRY(launch_pair_partners(sel, ctr + C_SEL, n, kc.data, kc.dtype, nk, kcount, prank, pcnt, s));
    HIP_TRY(launch_scan_i32_i64(pcnt, ctr + C_SEL, n, poff, pscan, ctr + C_SCRATCH, s));
    HIP_TRY(launch_pair_total(ctr + C_SCRATCH, ns_ub, ctr, s));
    HIP_TRY(launch_pair_emit(sel, ctr + C_SEL, n, kc.data, kc.dtype, nk, koff, prank, psorted, pcnt, poff, ns_ub,
                             pa, pb, s));
    HIP_TRY(launch_pair_lens(pa, pb, sel, p->probe.list_offsets, p->probe.max_list_len, row_prefix.n, ns_ub, lens,
                             ctr, s));
    HIP_TRY(launch_scan_i32_i64(lens, n_seq, ns_ub, cu, pscan, ctr + C_TOK, s));
    HIP_TRY(launch_pair_gather(pa, pb, sel, p->probe.list_offsets, p->probe.list_tokens, cu, row_prefix,
                               p->probe.max_list_len, p->model.vocab, p->t_ub, ns_ub, packed, ctr, s));
  } else if (!p->lb_compact) {
    // ---- token offsets of the selected rows
    HIP_TRY(launch_scan_blocks64(blk_tok, nullptr, n, tok_off, ctr + C_TOK, s));
    HIP_TRY(launch_cu_from_blocks(lens, blk_off, tok_off, n, cu, s));
  }
  if (p->rel_only) {
    // relational part only: every selected id is kept
    tr.end();
    tr.begin(AIQ_K_AGG);
    HIP_TRY(launch_keep_selected(ctr, out->ids_cap, s));
    HIP_TRY(launch_finalize(ctr, out->scalars, s));
    tr.end();
    return AIQ_OK;
  }
  // ---- pack: tokens, chunk descriptors
  if (!p->pairs)
    HIP_TRY(launch_gather_tokens(sel, ctr + C_SEL, n, p->probe.list_offsets, p->probe.list_tokens, cu, row_prefix,
                                 p->model.vocab, p->t_ub, packed, ctr, s));
  HIP_TRY(launch_chunk_desc(cu, n_seq, p->chunk_tokens, p->n_chunks, p->t_ub, desc, s));
  HIP_TRY(launch_rope_table(p->max_seq, p->hd / 2, p->model.rope_theta, p->hd, at<float>(ws, L.rcos),
                            at<float>(ws, L.rsin), at<float>(ws, L.rrev), s));
  tr.end();
  // ---- shared prompt prefix: its own prefill pass keeps every layer's q|k|v rows
  PrefixUse rows_pu{};
  if (p->share_prefix) {
    const int32_t np = p->prefix.n;
    int32_t* ptok = at<int32_t>(ws, L.ptok);
    int64_t* pcu = at<int64_t>(ws, L.pcu);
    int64_t* pdesc = at<int64_t>(ws, L.pdesc);
    HIP_TRY(launch_prefix_batch(p->prefix, ptok, pcu, pdesc, s));
    PrefixUse pre_pu{};
    pre_pu.qkv_layers = at<void>(ws, L.pkv);
    pre_pu.qkv_rows = np;
    pre_pu.npre = np;
    pre_pu.head = false;
    const aiq_status e = enqueue_chunk(p, ws, L, pdesc, pcu, ctr, ptok, p->t_cap, 1, nullptr, nullptr, nullptr, tr,
                                       s, pre_pu);
    if (e != AIQ_OK) return e;
    float* pxl = at<float>(ws, L.pxlast);
    // the prefix's last position: row np - 1 of x, or row 0 of the pruned last layer's rows
    const float* xsrc = p->prune_last ? at<float>(ws, L.xl)
                                      : at<float>(ws, L.x) + static_cast<int64_t>(np - 1) * p->model.d_model;
    HIP_TRY(launch_copy_row_f32(xsrc, pxl, p->model.d_model, s));
    rows_pu.pkv_layers = at<void>(ws, L.pkv);
    rows_pu.npre = np;
    rows_pu.x_pre = pxl;
  }
  if (p->gen > 0) {   // the generation steps read every layer's prompt keys and values
    rows_pu.qkv_layers = at<void>(ws, L.kvc);
    rows_pu.qkv_rows = p->t_cap;
  }
  // ---- prefill + label head (or generation), chunk by chunk
  for (int64_t c = 0; c < p->n_chunks; ++c) {
    aiq_status e = enqueue_chunk(p, ws, L, desc + c * D_STRIDE, cu, ctr, packed, p->t_cap, p->seq_ub, label, logits,
                                 p->gen > 0 ? at<void>(ws, L.hf) : nullptr, tr, s, rows_pu);
    if (e != AIQ_OK) return e;
    if (p->gen > 0) {
      e = enqueue_generation(p, ws, L, desc + c * D_STRIDE, cu, rows_pu, tr, s);
      if (e != AIQ_OK) return e;
    }
  }
  int32_t* gen = p->gen > 0 ? at<int32_t>(ws, L.gen) : nullptr;
  if (p->gen > 0) {   // LIKE over each selected row's generation -> keep flags
    LikePattern pat{};
    pat.n = q.n_like;
    for (int k = 0; k < q.n_like; ++k) pat.tok[k] = q.like[k];
    TRACED(tr, AIQ_K_DECODE_HEAD, launch_gen_like(gen, ctr + C_SEL, n, p->gen, q.eos_id, pat, label, s));
  }
  // ---- decision -> kept ids, aggregates
  tr.begin(AIQ_K_AGG);
  const bool binary = q.decision == AIQ_DECIDE_BINARY_GT || p->gen > 0;   // label = keep flag
  if (binary) {   // kept rows (their ids), or kept pairs (their numbers)
    const int64_t ub = p->pairs ? ns_ub : n;
    HIP_TRY(launch_label_mask(label, n_seq, ub, mask, blk_cnt, s));
    HIP_TRY(launch_scan_blocks(blk_cnt, n_seq, ub, blk_off, ctr + C_KEPT, s));
    HIP_TRY(launch_scatter_rows(mask, blk_off, n_seq, ub, p->pairs ? nullptr : sel, out->ids, out->ids_cap, nullptr,
                                AIQ_I32, h, 0, nullptr, ctr, s));
    if (p->pairs && (out->pair_a || out->pair_b))
      HIP_TRY(launch_pair_rows(out->ids, ctr + C_KEPT, ub, pa, pb, sel, out->pair_a, out->pair_b, out->ids_cap, s));
  } else {
    HIP_TRY(launch_copy_ids(sel, ctr + C_SEL, n, out->ids, out->ids_cap, ctr, 1, s));
  }
  if (grouped) {
    const int mode = q.agg == AIQ_AGG_AVG_LABEL_COUNT_BY ? 1 : 2;
    const void* kcol = mode == 1 ? p->probe_cols[q.group_col].data : nullptr;
    const int32_t kdt = mode == 1 ? p->probe_cols[q.group_col].dtype : AIQ_I32;
    if (p->hgroup_log2) {   // any int32 key: hash table, then the groups sorted by key
      HashAggArgs g{};
      const size_t hs = size_t(1) << p->hgroup_log2;
      g.slot = at<uint64_t>(ws, L.gslot);
      g.cnt = at<int64_t>(ws, L.gslot + hs * 8);
      g.sum = at<int64_t>(ws, L.gslot + hs * 16);
      g.cap_log2 = p->hgroup_log2;
      g.key0 = at<uint32_t>(ws, L.gkey0);
      g.val0 = at<uint32_t>(ws, L.gval0);
      g.key1 = at<uint32_t>(ws, L.gkey1);
      g.val1 = at<uint32_t>(ws, L.gval1);
      g.hist = at<int64_t>(ws, L.ghist);
      g.n_groups = at<int64_t>(ws, L.gn);
      HIP_TRY(launch_hash_group(sel, label, payload, ctr + C_SEL, n, kcol, kdt, mode, g, p->hgroup_max,
                                out->grp_key, out->grp_count, out->grp_sum, out->grp_avg, out->grp_cap, ctr, s));
    } else {   // keys are codes in [0, n_group_keys): dense bins
      int64_t* bins = at<int64_t>(ws, L.bins);
      HIP_TRY(launch_fill_i64(bins, 2 * int64_t(q.n_group_keys), 0, s));
      HIP_TRY(launch_group_accumulate(sel, label, payload, nullptr, ctr + C_SEL, n, kcol, kdt, mode,
                                      q.n_group_keys, bins, ctr, s));
      HIP_TRY(launch_group_emit(bins, q.n_group_keys, out->grp_key, out->grp_count, out->grp_sum, out->grp_avg,
                                out->grp_cap, mode, ctr, s));
    }
  }
  if (q.agg == AIQ_AGG_SUM_F32)
    HIP_TRY(launch_sum_f32(sel, label, ctr + C_SEL, static_cast<const float*>(p->probe_cols[q.group_col].data),
                           binary, at<double>(ws, L.bins), out->sum_out, s));
  if (out->sel_cap > 0) {   // labels and logits are per sequence (row, or candidate pair)
    if (out->sel_ids) HIP_TRY(launch_copy_ids(sel, ctr + C_SEL, n, out->sel_ids, out->sel_cap, ctr, 0, s));
    if (out->sel_labels) HIP_TRY(launch_copy_ids(label, n_seq, ns_ub, out->sel_labels, out->sel_cap, ctr, 0, s));
    if (out->sel_logits && p->gen == 0)
      HIP_TRY(launch_copy_f32(logits, n_seq, ns_ub, q.n_labels, out->sel_logits, out->sel_cap, s));
    if (p->pairs && (out->cand_a || out->cand_b))
      HIP_TRY(launch_pair_rows(nullptr, n_seq, ns_ub, pa, pb, sel, out->cand_a, out->cand_b, out->sel_cap, s));
    if (out->sel_gen && p->gen > 0)
      HIP_TRY(launch_copy_rows_i32(gen, ctr + C_SEL, n, p->gen, out->sel_gen, out->sel_cap, s));
  }
  HIP_TRY(launch_finalize(ctr, out->scalars, s, p->share_prefix ? q.n_prefix : 0, p->pairs ? C_PAIRS : C_SEL));
  tr.end();
  return AIQ_OK;
}

// The relational part of aiq_run (a relational-only plan) with its scratch in
// the library's fixed device array instead of a caller workspace: counters,
// the compaction's look-back words and the join's hash table.  The same
// kernels as aiq_run's one-launch form; the per-row token offsets are not
// kept (only their total is an output here).
aiq_status aiq_run_relational_static(const aiq_plan* p, const aiq_out* out, void* stream) {
  if (!p || !out || !out->scalars) return AIQ_EINVAL;
  if (!p->has_probe || !p->rel_only) return AIQ_EINVAL;
  if (out->ids_cap < 0 || (out->ids_cap > 0 && !out->ids) || out->sel_cap < 0) return AIQ_EINVAL;
  if (!p->lb_compact) return AIQ_EUNSUPPORTED;
  Carver c;
  const size_t o_ctr = c.take(C_COUNT * 8);
  const int64_t nlb = (p->n_rows + LB_MIN_ROWS - 1) / LB_MIN_ROWS + 1;
  const size_t o_lb = c.take(static_cast<size_t>(nlb) * 4 * 8);
  const size_t hcap = p->has_build ? (size_t(1) << p->hash_log2) : 0;
  const size_t o_hk = c.take(hcap * 4);
  const size_t o_hv = c.take(hcap * 4);
  const size_t o_jk = c.take(p->has_build ? JOIN_LDS_SLOTS * 4 : 0);
  const size_t o_jv = c.take(p->has_build ? JOIN_LDS_SLOTS * 4 : 0);
  const size_t o_jl = c.take(p->has_build ? 4 : 0);
  if (c.off > STATIC_SCRATCH_BYTES) return AIQ_ENOSPC;   // before any HIP call: nothing enqueued
  void* base = nullptr;
  size_t cap = 0;
  HIP_TRY(static_scratch(&base, &cap));
  if (c.off > cap) return AIQ_ENOSPC;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const aiq_query& q = p->q;
  int64_t* ctr = at<int64_t>(base, o_ctr);
  int64_t* lb = at<int64_t>(base, o_lb);
  HashArgs h{};
  if (p->has_build) {
    h.keys = at<int32_t>(base, o_hk);
    h.vals = at<int32_t>(base, o_hv);
    h.cap_log2 = p->hash_log2;
  }
  StagedHash staged{at<int32_t>(base, o_jk), at<int32_t>(base, o_jv), at<int32_t>(base, o_jl)};
  const void* pkey = p->has_build ? p->probe_cols[q.probe_key_col].data : nullptr;
  const int32_t pkey_dt = p->has_build ? p->probe_cols[q.probe_key_col].dtype : AIQ_I32;
  HIP_TRY(launch_fill_i64(ctr, C_COUNT, 0, s));
  if (p->has_build) {
    HIP_TRY(launch_fill_i32(h.keys, static_cast<int64_t>(hcap), HASH_EMPTY, s));
    const aiq_col& kc = p->build_cols[q.build_key_col];
    const aiq_col& pc = p->build_cols[q.build_payload_col];
    HIP_TRY(launch_hash_build(p->build_preds, kc.data, kc.dtype, pc.data, pc.dtype, p->build.n_rows, h, ctr, s));
    HIP_TRY(launch_hash_stage(h, staged, s));
  }
  int32_t* ids2 = out->sel_cap > 0 ? out->sel_ids : nullptr;
  HIP_TRY(launch_select_lb(p->probe_preds, p->n_rows, pkey, pkey_dt, h, p->has_build,
                           p->has_build ? &staged : nullptr, out->ids, out->ids_cap, ids2, out->sel_cap, nullptr,
                           p->probe.list_offsets, p->probe.max_list_len, q.n_prefix, nullptr, lb, ctr, s));
  HIP_TRY(launch_keep_selected(ctr, out->ids_cap, s));
  HIP_TRY(launch_finalize(ctr, out->scalars, s));
  return AIQ_OK;
}

aiq_status aiq_convert_weights(const void* src, int32_t src_dtype, void* dst, int32_t dst_dtype, int64_t n,
                               void* stream) {
  if (n < 0 || (n > 0 && (!src || !dst))) return AIQ_EINVAL;
  if (src_dtype != AIQ_BF16 || dst_dtype != AIQ_F16) return AIQ_EUNSUPPORTED;
  if (reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(dst) % 16) return AIQ_EINVAL;
  HIP_TRY(launch_bf16_to_f16(src, dst, n, static_cast<hipStream_t>(stream)));
  return AIQ_OK;
}

aiq_status aiq_prefill_packed(const aiq_plan* p, const int32_t* tok, const int32_t* cu_seqlens, int32_t n_seq,
                              int64_t n_tok, int32_t logits_mode, float* logits, void* ws, size_t ws_bytes,
                              void* stream) {
  if (!p || !tok || !cu_seqlens || !logits || !ws) return AIQ_EINVAL;
  if (n_seq <= 0 || n_tok < n_seq) return AIQ_EINVAL;
  if (logits_mode != AIQ_LOGITS_LABELS && logits_mode != AIQ_LOGITS_FULL_VOCAB) return AIQ_EINVAL;
  if (logits_mode == AIQ_LOGITS_LABELS && !p->has_query) return AIQ_EINVAL;
  if (logits_mode == AIQ_LOGITS_FULL_VOCAB && p->model.vocab % (p->bf16 ? 256 : 64)) return AIQ_EUNSUPPORTED;
  if (reinterpret_cast<uintptr_t>(ws) % ALIGN) return AIQ_EINVAL;
  // the workspace must have been sized for at least n_tok tokens
  int64_t cap = n_tok;
  Layout L = prefill_layout(p, cap);
  if (ws_bytes < L.total) return AIQ_ENOSPC;
  // use the largest token capacity the workspace holds so layouts agree between calls
  {
    int64_t lo = n_tok, hi = n_tok;
    while (prefill_layout(p, hi * 2).total <= ws_bytes && hi < (int64_t(1) << 40)) hi *= 2;
    if (hi != n_tok) {
      lo = hi;
      hi = hi * 2;
      while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (prefill_layout(p, mid).total <= ws_bytes) lo = mid;
        else hi = mid;
      }
      cap = lo;
    }
    L = prefill_layout(p, cap);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  Tracer tr{nullptr, s};
  int64_t* ctr = at<int64_t>(ws, L.ctr);
  int64_t* desc = at<int64_t>(ws, L.desc);
  int64_t* cu = at<int64_t>(ws, L.cu);
  HIP_TRY(launch_fill_i64(ctr, C_COUNT, 0, s));
  HIP_TRY(launch_packed_desc(cu_seqlens, n_seq, n_tok, cu, desc, ctr, s));
  HIP_TRY(launch_rope_table(static_cast<int32_t>(std::min<int64_t>(cap, INT32_MAX)), p->hd / 2, p->model.rope_theta,
                            p->hd, at<float>(ws, L.rcos), at<float>(ws, L.rsin), at<float>(ws, L.rrev), s));
  const bool full = logits_mode == AIQ_LOGITS_FULL_VOCAB;
  void* hf = full ? at<void>(ws, L.hf) : nullptr;
  int32_t* label = at<int32_t>(ws, L.label);
  const aiq_status e = enqueue_chunk(p, ws, L, desc, cu, ctr, tok, n_tok, n_seq, full ? nullptr : label,
                                     full ? nullptr : logits, hf, tr, s);
  if (e != AIQ_OK) return e;
  if (full) {
    GemmArgs g{};
    g.A = hf;
    g.lda = p->model.d_model;
    g.m_ptr = ctr + C_NSEQ;
    g.m_ub = n_seq;
    g.N = p->model.vocab;
    g.K = p->model.d_model;
    g.B0 = p->model.lm_head;
    g.C = logits;
    g.ldc = p->model.vocab;
    g.f16 = p->act == 2;
    HIP_TRY(p->bf16 ? launch_gemm_bf16(EPI_STORE_F32, g, s) : launch_gemm_f32(EPI_STORE_F32, g, s));
  }
  return AIQ_OK;
}

}  // extern "C"
