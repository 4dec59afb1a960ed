"""Device-memory plumbing around the C ABI: uploads host arrays into torch
device tensors, fills the ABI structs with their addresses, allocates the
workspace and output buffers, and calls the library on torch's current
stream.  No arithmetic of the query happens here.

Inputs are plain host structures:
  tables = {"probe": {col: ndarray, "offsets": int64[n+1], "tokens": int32[nnz]},
            "build": {col: ndarray} or None, "prefix": int32[...]}
  model  = {"spec": <object with n_layers, d_model, ...>, "emb", "layers": [...],
            "final_norm", "lm_head"} with bf16 weights as uint16 bit patterns
  query  = <object with preds, labels, decision, agg, join, n_prefix, group_col,
            n_group_keys>
"""
from __future__ import annotations

import ctypes as C

import numpy as np
import torch

from . import binding as B

_NP_DTYPE = {np.dtype(np.int8): B.AIQ_I8, np.dtype(np.int16): B.AIQ_I16, np.dtype(np.int32): B.AIQ_I32,
             np.dtype(np.float32): B.AIQ_F32}
_DECISION = {"binary_gt": B.AIQ_DECIDE_BINARY_GT, "argmax": B.AIQ_DECIDE_ARGMAX}
_AGG = {"count": B.AIQ_AGG_COUNT, "avg_label_count_by": B.AIQ_AGG_AVG_LABEL_COUNT_BY,
        "count_by_payload": B.AIQ_AGG_COUNT_BY_PAYLOAD, "sum_f32": B.AIQ_AGG_SUM_F32}
_LIST_KEYS = ("offsets", "tokens")


def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:   # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


def _layers_opt(n_layers) -> int:
    # 0 asks for every layer; a request for zero layers is encoded as -1
    if n_layers is None:
        return 0
    return -1 if int(n_layers) == 0 else int(n_layers)


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


class DeviceModel:
    """Model weights resident in device memory plus the aiq_model struct.

    ``compute`` selects the projection type of a 16-bit model: "bf16" keeps the
    stored bf16 weights; "f16" uploads their fp16 images (exact except for
    |w| < 2**-14, which fp16 holds as subnormals) so that activations fed to
    the MFMA projections carry 10 mantissa bits instead of 7.  fp32 models
    are uploaded as they are."""

    def __init__(self, model: dict, device="cuda", compute: str | None = None):
        spec = model["spec"]
        self.spec = spec
        self.keep = []
        self.compute = "f32" if spec.dtype == "f32" else (compute or "f16")
        if self.compute not in ("f32", "bf16", "f16"):
            raise ValueError(compute)

        def up(a):
            t = _dev(a, device)
            if t.dtype == torch.bfloat16 and self.compute == "f16":   # fp16 images, converted by the library
                h = torch.empty(t.shape, dtype=torch.float16, device=t.device)
                B.aiq_convert_weights(t.data_ptr(), B.AIQ_BF16, h.data_ptr(), B.AIQ_F16, t.numel(),
                                      torch.cuda.current_stream(t.device).cuda_stream)
                t = h
            self.keep.append(t)
            return t

        self.emb = up(model["emb"])
        self.lm_head = up(model["lm_head"])
        self.final_norm = up(np.asarray(model["final_norm"], dtype=np.float32))
        L = len(model["layers"])
        self.layers = (B.aiq_layer * max(L, 1))()
        for i, lw in enumerate(model["layers"]):
            s = self.layers[i]
            s.attn_norm = _ptr(up(np.asarray(lw["attn_norm"], dtype=np.float32)))
            s.ffn_norm = _ptr(up(np.asarray(lw["ffn_norm"], dtype=np.float32)))
            for k in ("wq", "wk", "wv", "wo", "w_gate", "w_down"):
                setattr(s, k, _ptr(up(lw[k])))
            s.w_up = _ptr(up(lw["w_up"])) if "w_up" in lw else 0
        m = B.aiq_model()
        m.n_layers, m.d_model, m.n_heads = L, spec.d_model, spec.n_heads
        m.n_kv_heads, m.d_ff, m.vocab = spec.n_kv_heads, spec.d_ff, spec.vocab
        m.act = B.AIQ_ACT_SWIGLU if spec.act == "swiglu" else B.AIQ_ACT_GELU_ERF
        m.wdtype = {"f32": B.AIQ_F32, "bf16": B.AIQ_BF16, "f16": B.AIQ_F16}[self.compute]
        m.rope_theta, m.norm_eps = spec.rope_theta, spec.norm_eps
        m.emb, m.lm_head, m.final_norm = _ptr(self.emb), _ptr(self.lm_head), _ptr(self.final_norm)
        m.layers = C.cast(self.layers, C.POINTER(B.aiq_layer))
        self.struct = m


class DeviceTable:
    def __init__(self, cols: dict, device="cuda", with_list=True, max_list_len=None):
        self.names = [k for k in cols if k not in _LIST_KEYS]
        self.index = {k: i for i, k in enumerate(self.names)}
        self.tensors = {k: _dev(cols[k], device) for k in self.names}
        self.dtypes = {k: np.asarray(cols[k]).dtype for k in self.names}
        n = len(cols[self.names[0]]) if self.names else len(cols["offsets"]) - 1
        self.n_rows = n
        self.cols = (B.aiq_col * max(len(self.names), 1))()
        for i, k in enumerate(self.names):
            self.cols[i].data = _ptr(self.tensors[k])
            self.cols[i].dtype = _NP_DTYPE[self.dtypes[k]]
        t = B.aiq_table()
        t.n_rows, t.n_cols = n, len(self.names)
        t.cols = C.cast(self.cols, C.POINTER(B.aiq_col))
        if with_list:
            off = np.asarray(cols["offsets"], dtype=np.int64)
            self.offsets = _dev(off, device)
            t.list_offsets = _ptr(self.offsets)
            if "tokens" in cols:   # absent: offsets only (relational-only plans)
                tok = np.asarray(cols["tokens"], dtype=np.int32)
                self.tokens = _dev(tok if len(tok) else np.zeros(1, np.int32), device)
                t.list_tokens = _ptr(self.tokens)
            t.n_list_tokens = int(off[-1] - off[0])
            lens = np.diff(off)
            t.max_list_len = int(max_list_len if max_list_len is not None else max(1, lens.max(initial=1)))
        self.struct = t


def _pred(p, table: "DeviceTable") -> B.aiq_pred:
    s = B.aiq_pred()
    s.col = table.index[p.col]
    s.op = B.OPS[p.op]
    if table.dtypes[p.col].kind == "f":
        s.fk = float(p.k)
    else:
        s.k = int(p.k)
    vals = list(p.values)
    s.n_set = len(vals)
    for i, v in enumerate(vals):
        s.set[i] = int(v)
    return s


def make_query(query, probe: DeviceTable | None, build: DeviceTable | None, prefix) -> B.aiq_query:
    q = B.aiq_query()
    preds = list(getattr(query, "preds", ()))
    q.n_pred = len(preds)
    for i, p in enumerate(preds):
        q.preds[i] = _pred(p, probe)
    j = getattr(query, "join", None)
    if j is not None:
        q.join = 1
        q.probe_key_col = probe.index[j.probe_key]
        q.build_key_col = build.index[j.build_key]
        q.build_payload_col = build.index[j.payload]
        q.n_build_pred = len(j.build_preds)
        for i, p in enumerate(j.build_preds):
            q.build_preds[i] = _pred(p, build)
    n_prefix = int(getattr(query, "n_prefix", 0))
    q.n_prefix = n_prefix
    for i in range(n_prefix):
        q.prefix[i] = int(prefix[i])
    q.n_labels = len(query.labels)
    for i, l in enumerate(query.labels):
        q.label_ids[i] = int(l)
    q.decision = _DECISION[query.decision]
    q.agg = _AGG[query.agg]
    if getattr(query, "group_col", None):
        q.group_col = probe.index[query.group_col]
    q.n_group_keys = int(getattr(query, "n_group_keys", 0))
    q.gen_tokens = int(getattr(query, "gen_tokens", 0))
    q.eos_id = int(getattr(query, "eos_id", -1))
    q.pad_id = int(getattr(query, "pad_id", 0))
    like = tuple(getattr(query, "like", ()))
    q.n_like = len(like)
    for i, t in enumerate(like):
        q.like[i] = int(t)
    if getattr(query, "pair_key", None):
        q.pairs = 1
        q.pair_key_col = probe.index[query.pair_key]
        q.max_pairs = int(query.max_pairs)
    return q


class DeviceQuery:
    """A planned query over device-resident tables and weights."""

    def __init__(self, tables: dict, model, query, device="cuda", chunk_tokens: int = 0,
                 n_layers: int | None = None, dmodel: DeviceModel | None = None, relational_only: bool = False,
                 want_sel: bool = True, share_prefix: bool = True, multipass_compact: bool = False,
                 full_last_layer: bool = False):
        self.device = torch.device(device)
        self.query = query
        self.dm = dmodel if dmodel is not None else DeviceModel(model, device)
        self.probe = DeviceTable(tables["probe"], device)
        self.build = DeviceTable(tables["build"], device, with_list=False) if tables.get("build") is not None else None
        self.q = make_query(query, self.probe, self.build, tables.get("prefix", ()))
        opts = B.aiq_plan_opts()
        opts.chunk_tokens = int(chunk_tokens)
        opts.n_layers_override = _layers_opt(n_layers)
        opts.flags = (B.AIQ_PLAN_RELATIONAL_ONLY if relational_only else 0) | \
            (0 if share_prefix else B.AIQ_PLAN_UNSHARED_PREFIX) | \
            (B.AIQ_PLAN_MULTIPASS_COMPACT if multipass_compact else 0) | \
            (B.AIQ_PLAN_FULL_LAST_LAYER if full_last_layer else 0)
        self.plan = B.aiq_plan_create(self.dm.struct, self.probe.struct,
                                      self.build.struct if self.build else None, self.q, opts)
        self.ws_bytes = B.aiq_workspace_size(self.plan)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=self.device)
        base = self.ws.data_ptr()
        self.ws_ptr = (base + 255) // 256 * 256
        n = self.probe.n_rows
        K = len(query.labels)
        dev = self.device
        self.pairs = bool(getattr(query, "pair_key", None))
        n = max(n, int(query.max_pairs)) if self.pairs else n   # outputs per row, or per pair
        self.scalars = torch.zeros(B.AIQ_N_SCALARS, dtype=torch.int64, device=dev)
        self.ids = torch.zeros(max(n, 1), dtype=torch.int32, device=dev)
        self.sel_ids = torch.zeros(max(n, 1), dtype=torch.int32, device=dev)
        self.sel_labels = torch.zeros(max(n, 1), dtype=torch.int32, device=dev)
        self.sel_logits = torch.zeros(max(n, 1) * K, dtype=torch.float32, device=dev)
        # dense keys: one group per key code; any int32 key (n_group_keys 0):
        # at most one group per probe row
        G = int(getattr(query, "n_group_keys", 0)) or n
        G = max(G, 1)
        self.grp_key = torch.zeros(G, dtype=torch.int32, device=dev)
        self.grp_count = torch.zeros(G, dtype=torch.int64, device=dev)
        self.grp_sum = torch.zeros(G, dtype=torch.int64, device=dev)
        self.grp_avg = torch.zeros(G, dtype=torch.float64, device=dev)
        self.sum_out = torch.zeros(1, dtype=torch.float64, device=dev)
        self.gen = int(getattr(query, "gen_tokens", 0))
        self.sel_gen = torch.zeros(max(n, 1) * max(self.gen, 1), dtype=torch.int32, device=dev)
        o = B.aiq_out()
        o.scalars, o.ids, o.ids_cap = _ptr(self.scalars), _ptr(self.ids), n
        o.sel_ids, o.sel_labels, o.sel_logits, o.sel_cap = (_ptr(self.sel_ids), _ptr(self.sel_labels),
                                                            _ptr(self.sel_logits), n if want_sel else 0)
        o.grp_key, o.grp_count, o.grp_sum, o.grp_avg = (_ptr(self.grp_key), _ptr(self.grp_count),
                                                        _ptr(self.grp_sum), _ptr(self.grp_avg))
        o.grp_cap = G
        o.sum_out = _ptr(self.sum_out)
        o.sel_gen = _ptr(self.sel_gen) if self.gen else None
        if self.pairs:
            self.pair_a = torch.zeros(n, dtype=torch.int32, device=dev)
            self.pair_b = torch.zeros(n, dtype=torch.int32, device=dev)
            self.cand_a = torch.zeros(n, dtype=torch.int32, device=dev)
            self.cand_b = torch.zeros(n, dtype=torch.int32, device=dev)
            o.pair_a, o.pair_b, o.cand_a, o.cand_b = (_ptr(self.pair_a), _ptr(self.pair_b), _ptr(self.cand_a),
                                                      _ptr(self.cand_b))
        self.out = o

    def run(self, trace=None, stream=None) -> None:
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        B.aiq_run(self.plan, self.ws_ptr, self.ws_bytes, self.out, trace, s.cuda_stream)

    def run_static(self, stream=None) -> None:
        """The relational-only plan through the entry point that allocates
        nothing (its scratch is the library's fixed device array)."""
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        B.aiq_run_relational_static(self.plan, self.out, s.cuda_stream)

    def results(self) -> dict:
        """Copies the outputs to the host (after the stream has been synchronised)."""
        sc = self.scalars.cpu().numpy()
        n_sel, n_kept, n_groups = int(sc[B.AIQ_S_SELECTED]), int(sc[B.AIQ_S_KEPT]), int(sc[B.AIQ_S_GROUPS])
        K = len(self.query.labels)
        r = {"scalars": sc, "status": int(sc[B.AIQ_S_STATUS]), "n_selected": n_sel, "count": n_kept,
             "n_tokens": int(sc[B.AIQ_S_TOKENS]),
             "kept_ids": self.ids[:n_kept].cpu().numpy().astype(np.int64),
             "sel_ids": self.sel_ids[:n_sel].cpu().numpy().astype(np.int64),
             "labels": self.sel_labels[:n_sel].cpu().numpy().astype(np.int64),
             "logits": self.sel_logits[:n_sel * K].cpu().numpy().reshape(n_sel, K)}
        if self.query.agg == "sum_f32":
            r["sum"] = float(self.sum_out.cpu().item())
        if self.gen:
            r["gen"] = self.sel_gen[:n_sel * self.gen].cpu().numpy().astype(np.int64).reshape(n_sel, self.gen)
        if self.pairs:   # labels / logits are per candidate pair; ids are kept pair numbers
            P = int(sc[B.AIQ_S_PAIRS])
            r.update(n_pairs=P, kept_pairs=r["kept_ids"],
                     pair_a=self.pair_a[:n_kept].cpu().numpy().astype(np.int64),
                     pair_b=self.pair_b[:n_kept].cpu().numpy().astype(np.int64),
                     cand_a=self.cand_a[:P].cpu().numpy().astype(np.int64),
                     cand_b=self.cand_b[:P].cpu().numpy().astype(np.int64),
                     labels=self.sel_labels[:P].cpu().numpy().astype(np.int64),
                     logits=self.sel_logits[:P * K].cpu().numpy().reshape(P, K))
        if self.query.agg in ("avg_label_count_by", "count_by_payload"):
            r["groups"] = (self.grp_key[:n_groups].cpu().numpy().astype(np.int64),
                           self.grp_count[:n_groups].cpu().numpy(), self.grp_sum[:n_groups].cpu().numpy(),
                           self.grp_avg[:n_groups].cpu().numpy())
        return r

    def close(self) -> None:
        if self.plan:
            B.aiq_plan_destroy(self.plan)
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DevicePrefill:
    """Prefill-only plan: runs the transformer on caller-packed sequences."""

    def __init__(self, model, labels=(1, 2), max_tokens: int = 4096, device="cuda",
                 n_layers: int | None = None, dmodel: DeviceModel | None = None, full_last_layer: bool = False):
        self.device = torch.device(device)
        self.dm = dmodel if dmodel is not None else DeviceModel(model, device)
        q = B.aiq_query()
        q.n_labels = len(labels)
        for i, l in enumerate(labels):
            q.label_ids[i] = int(l)
        q.decision = B.AIQ_DECIDE_BINARY_GT if len(labels) == 2 else B.AIQ_DECIDE_ARGMAX
        q.agg = B.AIQ_AGG_COUNT
        self.q = q
        self.K = len(labels)
        opts = B.aiq_plan_opts()
        opts.n_layers_override = _layers_opt(n_layers)
        opts.flags = B.AIQ_PLAN_FULL_LAST_LAYER if full_last_layer else 0
        self.plan = B.aiq_plan_create(self.dm.struct, None, None, q, opts)
        self.max_tokens = int(max_tokens)
        self.ws_bytes = B.aiq_prefill_workspace_size(self.plan, self.max_tokens)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=self.device)
        self.ws_ptr = (self.ws.data_ptr() + 255) // 256 * 256

    def run(self, tok: torch.Tensor, cu: torch.Tensor, full_vocab: bool = False, stream=None) -> torch.Tensor:
        n_seq = cu.numel() - 1
        n_tok = tok.numel()
        width = self.dm.spec.vocab if full_vocab else self.K
        out = torch.empty(n_seq * width, dtype=torch.float32, device=self.device)
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        B.aiq_prefill_packed(self.plan, _ptr(tok), _ptr(cu), n_seq, n_tok,
                             B.AIQ_LOGITS_FULL_VOCAB if full_vocab else B.AIQ_LOGITS_LABELS,
                             _ptr(out), self.ws_ptr, self.ws_bytes, s.cuda_stream)
        return out.view(n_seq, width)

    def close(self) -> None:
        if self.plan:
            B.aiq_plan_destroy(self.plan)
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
