#!/usr/bin/env python3
"""Benchmark of the unified AI-query pipeline on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload sweep3b] [--query 0]

A step is one aiq_run of the whole query over device-resident inputs: WHERE
+ stable selection, varlen pack, decoder prefill, label head + decision,
kept ids + COUNT, on one HIP stream.  The default workload is the largest
configuration: the selectivity sweep's table (1,048,576 synthetic rows, seed
4) through the 28-layer d3072 3B-class decoder at its 1 % point (c < 10),
whose whole-table steps take about 15 s each.

Printed (one JSON line): rows/s (table rows / end-to-end step time) as the
value, tokens/s, a per-stage breakdown, the roofline of the dominant kernel
(the gate/up SwiGLU GEMM) measured with HIP events around its launches that
carry tokens, the CPU oracle timed on the same workload (its relational part
on the whole table, its transformer on a seeded sample of the selected rows,
projected to all of them by FLOPs), and a split-execution baseline (host
selection + pack, H2D copy of survivors in micro-batches of 128 rows, the
same device prefill with full-vocabulary logits copied back, host decision
and COUNT).
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "AI-query rows/s and prefill tokens/s on 1 MI355X; MFMA % peak, HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0

# HBM bytes of gate/up GEMM launches measured by rocprofv3 FETCH_SIZE and
# WRITE_SIZE runs of the default bench command, scaled by what the same
# counters read for a plain 1 GiB copy (x2.000 and x1.000), keyed by the
# launch's token count (profiles/ holds the summaries and commands).  Valid
# only for the GEMM source they were measured on: reported as null once
# gemm.hip, dev_util.h or the GemmArgs declaration change, or for launches
# not listed.  The hash is moved to a new source only when the gate/up
# kernel's device assembly is unchanged by the edit.
GATE_UP_TRAFFIC = {"workload": "sweep3b", "query": 0,
                   "bytes_by_tokens": {"638426": 151782014897, "1997610": 474910304578},
                   "source_sha256": "de785c6b76fdaabf4bb1f225b3b5f8d20ee4e129c66afd22f7aede5294a418c9"}


def gemm_source_sha256() -> str:
    """Hash of the projection GEMM's sources: gemm.hip, dev_util.h and the
    GemmArgs declaration in aiq_internal.h."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_10139_amd", "csrc")
    for f in ("gemm.hip", "dev_util.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(csrc, "aiq_internal.h")) as fh:
        text = fh.read()
    start = text.index("struct GemmArgs")
    h.update(text[start:text.index("};", start)].encode())
    return h.hexdigest()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ HIP events (raw handles for the C ABI)
class HipEvents:
    def __init__(self, n: int):
        self.hip = C.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.hip.hipEventDestroy.argtypes = [C.c_void_p]
        self.ev = (C.c_void_p * n)()
        for i in range(n):
            h = C.c_void_p()
            if self.hip.hipEventCreate(C.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.ev[i] = h
        self.n = n

    def elapsed_ms(self, i: int, j: int) -> float:
        ms = C.c_float()
        if self.hip.hipEventElapsedTime(C.byref(ms), self.ev[i], self.ev[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def close(self):
        for i in range(self.n):
            self.hip.hipEventDestroy(self.ev[i])


def make_trace(B, events: HipEvents, kind_mask: int):
    cap = events.n // 2
    tags = (C.c_int32 * cap)()
    t = B.aiq_trace()
    t.events = C.cast(events.ev, C.POINTER(C.c_void_p))
    t.tags = C.cast(tags, C.POINTER(C.c_int32))
    t.capacity, t.count, t.kind_mask = cap, 0, kind_mask
    t._tags = tags
    return t


def per_kind_ms(B, trace, events) -> dict:
    out = {}
    for i in range(trace.count):
        k = trace._tags[i]
        out.setdefault(k, []).append(events.elapsed_ms(2 * i, 2 * i + 1))
    return out


# ------------------------------------------------------------------ algorithmic work
def prefill_flops(spec, own: np.ndarray, n_labels: int, npre: int = 0, shared: bool = False,
                  last_rows_only: bool = False) -> dict:
    """Algorithmic FLOPs of the prefill (no padding): the four projections,
    causal attention (unmasked half: QK^T and PV), and the label head.
    own: each selected row's token count; npre: prompt prefix length, packed
    into every row, or with ``shared`` prefilled once and attended to by
    every row's own positions npre.. .  With ``last_rows_only`` the last
    layer needs keys and values at every position but its query, attention
    (one query over the sequence's keys), O projection and FFN at the last
    position of each sequence only ("last"; the shared prefix pass is one
    more sequence).  Keys qkv / o / up / down / attn cover the launches
    traced under those kinds."""
    own = np.asarray(own, dtype=np.float64)
    n = float(len(own))
    d, dq, dkv, f, L = spec.d_model, spec.d_q, spec.d_kv, spec.d_ff, spec.n_layers
    n_ffn = 3 if spec.act == "swiglu" else 2
    if shared and npre > 0:
        T_rows, T_pre = float(own.sum()), float(npre)
        attn_rows = float(np.sum(2.0 * dq * (2.0 * npre * own + own * (own + 1.0))))
        attn_pre = 2.0 * dq * npre * (npre + 1.0)
        keys = own + npre
    else:
        lens = own + npre
        T_rows, T_pre = float(lens.sum()), 0.0
        attn_rows, attn_pre = float(np.sum(2.0 * dq * lens * (lens + 1.0))), 0.0
        keys = lens
    Lf = L - 1 if last_rows_only else L   # layers run on every position
    T_full = (T_rows + T_pre) * Lf
    per = {
        "qkv": 2 * d * (dq + 2 * dkv) * T_full,
        "o": 2 * dq * d * T_full,
        "up": 2 * d * f * (n_ffn - 1) * T_full,
        "down": 2 * f * d * T_full,
        "attn": (attn_rows + attn_pre) * Lf,
        "last": 0.0,
        "head": 2.0 * n * n_labels * d,
    }
    if last_rows_only and L > 0:
        n_last = n + (1.0 if T_pre else 0.0)   # the prefix pass's own last position
        keys_all = float(np.sum(keys)) + T_pre
        # keys and values everywhere (traced with the q|k|v projections)
        per["qkv"] += 2 * d * 2 * dkv * (T_rows + T_pre)
        # the query projection, one query over each sequence's keys (QK^T and
        # PV), O and FFN at the last positions
        per["last"] = 4.0 * dq * keys_all + n_last * (2 * d * dq + 2 * dq * d + 2 * d * f * (n_ffn - 1) + 2 * f * d)
    per["total"] = sum(per.values())
    return per


def generation_report(spec, q, tables, sel, kinds, B, ms_step) -> dict:
    """AI_TRANSFORM: generated tokens/s over whole steps, per-step time, and
    the decode attention's algorithmic bytes (every kept key and value row
    read once per layer and step) against its traced time."""
    G = int(q.gen_tokens)
    n = len(sel)
    P = tables["probe"]["len"][sel].astype(np.float64) + q.n_prefix   # prompt positions per row
    d_kv = spec.n_kv_heads * spec.head_dim
    steps = G - 1                        # the first token comes from the prefill's last position
    # step k reads P + k earlier keys and values plus this token's, fp16
    keys = float(np.sum(P)) * steps + n * (steps * (steps + 1) / 2.0)
    attn_bytes = keys * 2 * d_kv * 2 * spec.n_layers
    t_attn = float(np.sum(kinds.get(B.AIQ_K_DECODE_ATTN, [0.0])))
    t_layers = float(np.sum(kinds.get(B.AIQ_K_DECODE, [0.0])))
    t_head = float(np.sum(kinds.get(B.AIQ_K_DECODE_HEAD, [0.0])))
    return {"tokens_per_row": G, "generated_tokens": n * G, "generated_tokens_per_s": round(n * G / (ms_step * 1e-3), 1),
            "ms": {"layers": round(t_layers, 3), "attention": round(t_attn, 3), "vocab_head_argmax": round(t_head, 3)},
            "ms_per_step": round((t_layers + t_attn + t_head) / max(G, 1), 4),
            "attention_bytes": attn_bytes,
            "attention_gbps": round(attn_bytes / (t_attn * 1e-3) / 1e9, 1) if t_attn > 0 else None}


def time_query(tables, model, dm, q, B, torch, steps, warmup, n_rows) -> dict:
    """Whole-query time of one more query of the workload (same tables, model)."""
    from paper_2608_10139_amd.device import DeviceQuery
    dq = DeviceQuery(tables, model, q, dmodel=dm)
    for _ in range(max(warmup, 1)):
        dq.run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dq.run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / steps * 1e3
    r = dq.results()
    dq.close()
    out = {"predicate": " and ".join(f"{p.col} {p.op} {p.k}" for p in q.preds) or "none",
           "selected": r["n_selected"], "kept": r["count"], "status": r["status"], "ms_per_step": round(ms, 3),
           "rows_per_s": round(n_rows / (ms * 1e-3), 1)}
    if getattr(q, "gen_tokens", 0):
        out["generated_tokens_per_s"] = round(r["n_selected"] * q.gen_tokens / (ms * 1e-3), 1)
    return out


def host_select(cols: dict, preds) -> np.ndarray:
    """Split baseline's host WHERE: numpy masks, then the ascending row ids."""
    n = len(cols["id"])
    m = np.ones(n, dtype=bool)
    ops = {"lt": np.less, "le": np.less_equal, "gt": np.greater, "ge": np.greater_equal,
           "eq": np.equal, "ne": np.not_equal}
    for p in preds:
        v = cols[p.col].astype(np.int64)
        m &= np.isin(v, np.asarray(p.values, dtype=np.int64)) if p.op == "in" else ops[p.op](v, p.k)
    return np.flatnonzero(m)


# ------------------------------------------------------------------ legs
def cpu_baseline_leg(tables, model, q, spec, budget_flop: float = 3.0e12, seed: int = 0) -> dict:
    """The CPU oracle (fp64, per sequence) on the same workload: its
    relational part (WHERE, join) on the whole table, then its transformer on
    a seeded sample of the selected rows of about ``budget_flop`` FLOPs,
    projected to every selected row: widening the weights to fp64 (timed on
    its own, done once per run) plus the sample's remaining time scaled by
    the FLOPs of all selected rows over the sample's."""
    import oracle
    from oracle.transformer import Weights64
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = 1
    cores = len(os.sched_getaffinity(0))
    probe = tables["probe"]
    n = len(probe["id"])
    t0 = time.perf_counter()
    rows, _ = oracle.relational(tables, q)
    t_rel = time.perf_counter() - t0
    own = probe["len"][rows].astype(np.float64)
    npre = q.n_prefix
    fl_all = prefill_flops(spec, own, len(q.labels), npre)["total"]
    rng = np.random.default_rng(seed)
    order = rng.permutation(len(rows))
    pick, fl_s = [], 0.0
    for i in order:
        if fl_s >= budget_flop:
            break
        pick.append(int(i))
        fl_s += prefill_flops(spec, own[[i]], len(q.labels), npre)["total"]
    pick = np.sort(np.asarray(pick, dtype=np.int64))
    t0 = time.perf_counter()
    W = Weights64(model)
    for l in range(spec.n_layers):
        W.layer(l)
    t_widen = time.perf_counter() - t0
    seqs = oracle.sequences(probe, rows[pick], tables["prefix"][:npre])
    t0 = time.perf_counter()
    oracle.label_logits(model, seqs, q.labels)
    t_sample = time.perf_counter() - t0
    t_compute = max(t_sample - t_widen, 1e-9)
    t_model = t_widen + t_compute * (fl_all / max(fl_s, 1.0)) if len(rows) else 0.0
    total = t_rel + t_model
    return {"value": round(n / total, 4), "unit": "rows/s", "cores": int(max(blas, 1)), "host_cores": cores,
            "kind": "oracle",
            "sample": f"relational part on all {n} table rows (measured {t_rel:.2f} s, {len(rows)} selected); "
                      f"transformer on {len(pick)} seeded selected rows ({fl_s:.3e} FLOP, measured "
                      f"{t_sample:.1f} s incl. {t_widen:.1f} s widening the weights to fp64), projected to all "
                      f"{len(rows)} selected rows ({fl_all:.3e} FLOP): {t_model:.0f} s",
            "seconds_measured": round(t_rel + t_sample + t_widen, 2), "seconds_projected": round(total, 1),
            "projected": True}


def split_baseline_leg(tables, model, q, dm, B, torch, micro=128) -> dict:
    """Host selection + pack, per micro-batch H2D, device prefill with the
    full-vocabulary last-position logits, D2H, host decision + COUNT."""
    from paper_2608_10139_amd.device import DevicePrefill
    probe = tables["probe"]
    lens_all = np.diff(probe["offsets"])
    max_tok = micro * (int(lens_all.max()) + q.n_prefix)
    pf = DevicePrefill(model, labels=q.labels, max_tokens=max_tok, dmodel=dm)
    V = dm.spec.vocab
    tok_pin = torch.empty(max_tok, dtype=torch.int32, pin_memory=True)
    cu_pin = torch.empty(micro + 1, dtype=torch.int32, pin_memory=True)
    out_pin = torch.empty(micro * V, dtype=torch.float32, pin_memory=True)
    tok_d = torch.empty(max_tok, dtype=torch.int32, device="cuda")
    cu_d = torch.empty(micro + 1, dtype=torch.int32, device="cuda")
    labels = list(q.labels)
    prefix = np.asarray(tables["prefix"][:q.n_prefix], dtype=np.int32)

    def one_pass(limit=None):
        rows = host_select(probe, q.preds)
        kept = 0
        end = len(rows) if limit is None else min(len(rows), limit)
        for b0 in range(0, end, micro):
            rb = rows[b0:b0 + micro]
            seqs = [np.concatenate([prefix, probe["tokens"][probe["offsets"][r]:probe["offsets"][r + 1]]])
                    for r in rb]
            cu = np.zeros(len(rb) + 1, dtype=np.int32)
            cu[1:] = np.cumsum([len(s) for s in seqs])
            n_tok = int(cu[-1])
            tok_pin[:n_tok].copy_(torch.from_numpy(np.concatenate(seqs).astype(np.int32)))
            cu_pin[:len(cu)].copy_(torch.from_numpy(cu))
            tok_d[:n_tok].copy_(tok_pin[:n_tok], non_blocking=True)
            cu_d[:len(cu)].copy_(cu_pin[:len(cu)], non_blocking=True)
            lg = pf.run(tok_d[:n_tok], cu_d[:len(cu)], full_vocab=True)
            out_pin[:lg.numel()].copy_(lg.reshape(-1), non_blocking=True)
            torch.cuda.synchronize()
            full = out_pin[:lg.numel()].numpy().reshape(len(rb), V)
            kept += int(np.sum(full[:, labels[0]] > full[:, labels[1]]))
        return len(rows), kept

    one_pass(micro)   # warm-up: one micro-batch
    t0 = time.perf_counter()
    n_sel, kept = one_pass()
    dt = time.perf_counter() - t0
    pf.close()
    n = len(probe["id"])
    return {"value": n / dt, "unit": "rows/s", "ms": dt * 1e3, "selected": n_sel, "kept": kept,
            "micro_batch": micro, "logits": f"fp32 [{micro}, {V}] per micro-batch, D2H"}


def relational_scale_leg(B, torch, sizes, thresholds, steps: int = 5, multipass: bool = False) -> list:
    """The relational part alone (WHERE c < k, stable compaction, per-row
    token counts) on the 1M-row sweep table's generator scaled to `sizes` rows
    (columns c and offsets; no token list), through a relational-only plan.
    Algorithmic bytes per run: 4 B of c per row, 4 B per selected id written,
    8 B per distinct offset entry read (off[r] and off[r + 1] of every
    selected row r: 16 B per row when the selected rows are isolated, 8 B
    when they are adjacent), 8 B per cu_seqlens entry written.  The counts
    are checked against numpy on the host."""
    import dataclasses
    from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
    from synth import WORKLOADS
    from synth.configs import Pred, Query
    from synth.gen import make_model, make_probe

    tiny = make_model(WORKLOADS["tiny"].model)
    dm = DeviceModel(tiny)
    out = []
    for n in sizes:
        log(f"[bench] relational scale: generating {n} rows (sweep-table generator, c and lengths)")
        spec = dataclasses.replace(WORKLOADS["sweep3b"].table, n_rows=n)
        probe = make_probe(spec, with_tokens=False)
        tables = {"probe": probe, "build": None, "prefix": np.zeros(0, np.int32)}
        for k in thresholds:
            q = Query(preds=(Pred("c", "lt", k),), labels=(1, 2), decision="binary_gt", agg="count")
            dq = DeviceQuery(tables, tiny, q, dmodel=dm, relational_only=True, want_sel=False,
                             multipass_compact=multipass)
            dq.run()
            torch.cuda.synchronize()
            res = dq.results()
            want = probe["c"] < k
            n_sel = int(np.count_nonzero(want))
            # offset entries read: r and r + 1 of every selected row r
            n_off = n_sel + int(np.count_nonzero(want & ~np.concatenate(([False], want[:-1]))))
            if res["status"] != 0 or res["n_selected"] != n_sel or res["n_tokens"] != int(probe["len"][want].sum()):
                raise RuntimeError(f"relational scale run disagrees with numpy at n={n}, c < {k}")
            ev = HipEvents(2 * 8 * steps)
            tr = make_trace(B, ev, (1 << B.AIQ_K_REL) | (1 << B.AIQ_K_PACK) | (1 << B.AIQ_K_AGG))
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                dq.run(trace=tr)
            torch.cuda.synchronize()
            wall = (time.perf_counter() - t0) / steps * 1e3
            kinds = per_kind_ms(B, tr, ev)
            ev.close()
            rel = float(np.sum(kinds.get(B.AIQ_K_REL, []))) / steps
            pack = float(np.sum(kinds.get(B.AIQ_K_PACK, []))) / steps
            agg = float(np.sum(kinds.get(B.AIQ_K_AGG, []))) / steps
            nbytes = 4 * n + 4 * n_sel + 8 * n_off + 8 * (n_sel + 1)
            gbps = nbytes / ((rel + pack) * 1e-3) / 1e9
            out.append({"rows": n, "predicate": f"c < {k}", "selected": n_sel, "tokens": res["n_tokens"],
                        "where_compact_ms": round(rel, 4), "token_counts_ms": round(pack, 4),
                        "ids_out_ms": round(agg, 4), "run_ms": round(wall, 4),
                        "algorithmic_bytes": nbytes, "gbps": round(gbps, 1),
                        "hbm_frac": round(gbps / PEAK_HBM_GBPS, 4)})
            log(f"[bench]   n={n} c<{k}: {out[-1]}")
            dq.close()
        del probe, tables
    return out


def pack_config_leg(B, torch, steps: int = 3) -> list:
    """The pack stage (token counts -> cu_seqlens, token gather of every
    selected row, chunk descriptors) at config size: the 1M-row sweep table
    with every row selected (c < 1000) and the 131k-row group-by table (no
    predicate).  Runs the whole query with no decoder layer (a 0-layer fp32
    model: embedding -> head) and reads the pack stage's HIP-event time.
    Algorithmic bytes: per selected row 4 B of its row id + 8 B of offsets
    (its list start) + 8 B of cu_seqlens read, per token 4 B read + 4 B
    written."""
    from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
    from synth import WORKLOADS
    from synth.configs import ModelSpec
    from synth.gen import make_model, make_tables

    # the tables' 32,000-token vocabulary; no layer runs (embedding -> head)
    tiny = make_model(ModelSpec(n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, d_ff=64, vocab=32000,
                                act="gelu", dtype="f32", weight_seed=7))
    dm = DeviceModel(tiny)
    out = []
    for name, qi in (("sweep3b", 3), ("groupby1b", 0)):
        w = WORKLOADS[name]
        log(f"[bench] pack at config size: generating {name}")
        tables = make_tables(w)
        q0 = w.queries[qi]
        # the tiny model's labels and vocabulary; the selection of the workload's query
        import dataclasses
        q = dataclasses.replace(q0, labels=(1, 2), decision="binary_gt", agg="count")
        probe = tables["probe"]
        dq = DeviceQuery(tables, tiny, q, dmodel=dm, n_layers=0, want_sel=False)
        dq.run()
        torch.cuda.synchronize()
        res = dq.results()
        ev = HipEvents(2 * 8 * steps)
        tr = make_trace(B, ev, 1 << B.AIQ_K_PACK)
        for _ in range(steps):
            dq.run(trace=tr)
        torch.cuda.synchronize()
        pack = float(np.sum(per_kind_ms(B, tr, ev).get(B.AIQ_K_PACK, []))) / steps
        ev.close()
        n_sel, n_tok = res["n_selected"], res["n_tokens"]
        nbytes = 20 * n_sel + 8 * n_tok
        gbps = nbytes / (pack * 1e-3) / 1e9
        out.append({"table": name, "rows": len(probe["id"]), "selected": n_sel, "tokens": n_tok,
                    "pack_ms": round(pack, 4), "algorithmic_bytes": nbytes, "gbps": round(gbps, 1),
                    "hbm_frac": round(gbps / PEAK_HBM_GBPS, 4), "status": res["status"]})
        log(f"[bench]   {out[-1]}")
        dq.close()
        del tables
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="sweep3b")
    ap.add_argument("--compute", default="f16", choices=["f16", "bf16"],
                    help="projection type for bf16-drawn weights (f16: exact fp16 images of the weights)")
    ap.add_argument("--cpu-flop", type=float, default=3.0e12,
                    help="FLOPs of the oracle's transformer sample in the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-split", action="store_true")
    ap.add_argument("--query", type=int, default=0, help="index of the workload's query to time")
    ap.add_argument("--all-queries", action="store_true",
                    help="also time every query of the workload (e.g. the Q3 selectivity sweep)")
    ap.add_argument("--unshared-prefix", action="store_true",
                    help="recompute the prompt prefix inside every row (default: prefilled once and shared)")
    ap.add_argument("--relational-scale", action="store_true",
                    help="only the relational part at 2^26 and 2^28 rows (relational-only plans); one JSON line")
    ap.add_argument("--multipass-compact", action="store_true",
                    help="with --relational-scale: separate mask / scan / scatter launches instead of one")
    ap.add_argument("--full-last-layer", action="store_true",
                    help="run the last layer on every position (default: its attention, O projection and FFN "
                         "for the last position of each sequence only)")
    ap.add_argument("--no-relational-scale", action="store_true",
                    help="skip the 2^26-row relational run of the default line")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (3 times): the reference "
                         "for scaling HBM traffic counters")
    a = ap.parse_args(argv)
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {a.gpus}); the pipeline is single-GPU "
              "and multi-GPU sharding is not implemented", file=sys.stderr)
        return 2

    import torch
    if a.calibrate_copy:
        n = a.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "repeats": 3}), flush=True)
        return 0
    from paper_2608_10139_amd import binding as B
    from paper_2608_10139_amd.device import DeviceModel, DeviceQuery
    if a.relational_scale:
        torch.cuda.set_device(0)
        runs = relational_scale_leg(B, torch, [1 << 26, 1 << 28], [10, 1000], steps=a.steps,
                                    multipass=a.multipass_compact)
        packs = pack_config_leg(B, torch)
        best = max(runs, key=lambda r: r["gbps"])
        print(json.dumps({"metric": "relational stages (WHERE + stable compaction + token counts) HBM GB/s",
                          "value": best["gbps"], "unit": "GB/s", "n_gpus": 1, "steps": a.steps, "warmup": 1,
                          "higher_is_better": True, "dtype": "int32", "data": "synthetic",
                          "config": {"workload": "sweep-table generator scaled to 2^26 and 2^28 rows, "
                                                 "c and offsets only, relational-only plans",
                                     "compaction": "multipass" if a.multipass_compact else "one launch"},
                          "roofline": {"bound": "hbm", "achieved": best["gbps"], "peak": PEAK_HBM_GBPS,
                                       "unit": "GB/s", "frac": best["hbm_frac"], "traffic": None},
                          "runs": runs, "pack_at_config_size": packs}), flush=True)
        return 0
    from synth import WORKLOADS
    from synth.gen import make_model, make_tables

    torch.cuda.set_device(0)
    w = WORKLOADS[a.workload]
    q = w.queries[a.query]
    gen = int(getattr(q, "gen_tokens", 0))
    pairs = bool(getattr(q, "pair_key", None))
    spec = w.model
    log(f"[bench] generating {a.workload}: {w.description}")
    tables = make_tables(w)
    model = make_model(spec)
    dm = DeviceModel(model, compute=a.compute)
    shared = q.n_prefix > 0 and dm.compute != "f32" and not a.unshared_prefix
    dq = DeviceQuery(tables, model, q, dmodel=dm, share_prefix=not a.unshared_prefix,
                     full_last_layer=a.full_last_layer)
    log(f"[bench] workspace {dq.ws_bytes / 2**30:.2f} GiB; warmup {a.warmup}")

    step_s = 0.0
    for i in range(a.warmup):
        t_w = time.perf_counter()
        dq.run()
        torch.cuda.synchronize()
        step_s = time.perf_counter() - t_w
        log(f"[bench] warm-up step {i + 1}/{a.warmup} done in {step_s:.3f} s")
    res = dq.results()
    if res["status"] != 0:
        raise RuntimeError(f"device status {res['status']:#x}")
    n_rows = len(tables["probe"]["id"])
    sel = res["sel_ids"]
    if pairs:   # the sequences are the candidate pairs: both rows' tokens
        ltab = tables["probe"]["len"]
        own = (ltab[res["cand_a"]] + ltab[res["cand_b"]]).astype(np.float64)
    else:
        own = tables["probe"]["len"][sel].astype(np.float64)
    lens = own + q.n_prefix
    T = int(lens.sum())
    assert T == res["n_tokens"]

    # ---- timed region: whole steps; HIP events around the dominant kernel's launches only
    # every prefill pass (the shared prefix, then each chunk) launches the
    # gate/up GEMM once per layer; with the last layer on the last positions
    # only, a pass's last gate/up runs on those rows and is traced as part of
    # that layer.  Passes the selection leaves empty launch and do no work.
    chunks, pre_pass = B.aiq_plan_passes(dq.plan)
    passes = chunks + pre_pass
    last_rows_only = B.aiq_plan_last_layer_rows(dq.plan)
    layers_full = spec.n_layers - (1 if last_rows_only else 0)
    launches_per_step = layers_full * passes
    # tokens of each pass, from the plan's chunking rule (cu[i] + i over chunk_tokens)
    ct = B.aiq_plan_chunk_tokens(dq.plan)
    packed = own + (0 if shared else q.n_prefix)
    cu = np.concatenate([[0.0], np.cumsum(packed)])
    cidx = np.minimum(((cu[:-1] + np.arange(len(packed))) // ct).astype(np.int64), chunks - 1)
    pass_tok = list(np.bincount(cidx, weights=packed, minlength=chunks).astype(np.int64))
    if pre_pass:
        pass_tok = [q.n_prefix] + pass_tok
    launch_tok = np.repeat(np.asarray(pass_tok, dtype=np.int64), layers_full)   # one step, in launch order
    ev = HipEvents(2 * a.steps * launches_per_step)
    trace = make_trace(B, ev, 1 << B.AIQ_K_GEMM_UP)
    log(f"[bench] timing {a.steps} steps ({chunks} chunk passes of {ct} units, "
        f"{int(np.count_nonzero(launch_tok))} of {len(launch_tok)} gate/up launches per step carry tokens)")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    long_steps = step_s > 30.0   # minutes-long queries: report each step as it ends
    for i in range(a.steps):
        dq.run(trace=trace)
        if long_steps:
            torch.cuda.synchronize()
            log(f"[bench] timed step {i + 1}/{a.steps} done at {time.perf_counter() - t0:.1f} s")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_step = dt / a.steps * 1e3
    if trace.count != a.steps * launches_per_step:
        raise RuntimeError(f"traced {trace.count} gate/up launches, expected {a.steps * launches_per_step}")
    up = np.asarray(per_kind_ms(B, trace, ev).get(B.AIQ_K_GEMM_UP, []), dtype=np.float64)
    ev.close()
    fl = prefill_flops(spec, own, len(q.labels), q.n_prefix, shared, last_rows_only)
    tok_all = np.tile(launch_tok, a.steps)
    real = tok_all > 0
    n_ffn = 3 if spec.act == "swiglu" else 2
    up_flops = 2.0 * tok_all[real] * (n_ffn - 1) * spec.d_ff * spec.d_model   # per launch that carries tokens
    up_ms = up[real]
    empty_ms = up[~real]
    up_flops_per_launch = float(np.mean(up_flops)) if len(up_flops) else 0.0
    up_avg_ms = float(np.mean(up_ms)) if len(up_ms) else float("nan")
    achieved = float(np.sum(up_flops)) / (float(np.sum(up_ms)) * 1e-3) / 1e12 if len(up_ms) else 0.0
    peak = PEAK_F32_TFLOPS if dm.compute == "f32" else PEAK_BF16_TFLOPS   # fp16 and bf16 MFMA peaks are equal

    # ---- one untimed traced step for the stage breakdown
    last_blocks = 8 * (n_rows // 65536 + 1)   # the last layer's row blocks (at most 65,536 sequences each)
    ev2 = HipEvents(2 * (passes * (gen + 1) * (8 * spec.n_layers + 16 + last_blocks) + 64))
    tr2 = make_trace(B, ev2, 0xFFFFFFFF)
    dq.run(trace=tr2)
    torch.cuda.synchronize()
    if tr2.count >= tr2.capacity:
        raise RuntimeError("stage trace buffer full")
    kinds = per_kind_ms(B, tr2, ev2)
    ev2.close()
    names = {B.AIQ_K_REL: "relational", B.AIQ_K_PACK: "pack", B.AIQ_K_EMBED: "embed", B.AIQ_K_NORM: "rmsnorm",
             B.AIQ_K_GEMM_QKV: "gemm_qkv_rope", B.AIQ_K_ATTN: "attention", B.AIQ_K_GEMM_O: "gemm_o_resid",
             B.AIQ_K_GEMM_UP: "gemm_gate_up_swiglu", B.AIQ_K_GEMM_DOWN: "gemm_down_resid", B.AIQ_K_HEAD: "head",
             B.AIQ_K_AGG: "decision_agg", B.AIQ_K_DECODE: "gen_layers", B.AIQ_K_DECODE_ATTN: "gen_attention",
             B.AIQ_K_DECODE_HEAD: "gen_vocab_head_argmax_like", B.AIQ_K_LAST: "last_layer_last_positions"}
    stages = {names[k]: round(float(np.sum(v)), 4) for k, v in sorted(kinds.items())}
    prefill_kinds = [B.AIQ_K_EMBED, B.AIQ_K_NORM, B.AIQ_K_GEMM_QKV, B.AIQ_K_ATTN, B.AIQ_K_GEMM_O,
                     B.AIQ_K_GEMM_UP, B.AIQ_K_GEMM_DOWN, B.AIQ_K_HEAD, B.AIQ_K_LAST]
    prefill_ms = sum(float(np.sum(kinds.get(k, []))) for k in prefill_kinds)
    gemm = {"gemm_qkv_rope": ("qkv", B.AIQ_K_GEMM_QKV), "gemm_o_resid": ("o", B.AIQ_K_GEMM_O),
            "gemm_gate_up_swiglu": ("up", B.AIQ_K_GEMM_UP), "gemm_down_resid": ("down", B.AIQ_K_GEMM_DOWN)}
    gemm_frac = {}
    for nm, (key, k) in gemm.items():
        t = float(np.sum(kinds.get(k, [0.0])))
        gemm_frac[nm] = round(fl[key] / (t * 1e-3) / 1e12 / peak, 4) if t > 0 else None
    # relational bytes: referenced columns per row + 4 B per selected id
    col_bytes = sum(np.asarray(tables["probe"][p.col]).dtype.itemsize for p in {p.col: p for p in q.preds}.values())
    rel_bytes = n_rows * col_bytes + 4 * len(sel)
    rel_ms = float(np.sum(kinds.get(B.AIQ_K_REL, [0.0])))

    traffic = None
    by_tok = GATE_UP_TRAFFIC["bytes_by_tokens"]
    real_tok = [int(t) for t in launch_tok if t > 0]
    if (a.workload == GATE_UP_TRAFFIC["workload"] and a.query == GATE_UP_TRAFFIC["query"] and real_tok
            and all(str(t) in by_tok for t in real_tok)
            and gemm_source_sha256() == GATE_UP_TRAFFIC["source_sha256"]):
        traffic = float(np.mean([by_tok[str(t)] for t in real_tok]))
    result = {
        "metric": METRIC, "value": round(n_rows / (ms_step * 1e-3), 2), "unit": "rows/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dm.compute,
        "data": "synthetic (seeded tables and random-init weights)",
        "config": {"workload": f"{a.workload}: {w.description}", "rows": n_rows, "selected": len(sel),
                   "kept": res["count"], "tokens": T, "model": f"{spec.n_layers}L d{spec.d_model} "
                   f"{spec.n_heads}q/{spec.n_kv_heads}kv ffn{spec.d_ff} {spec.act}, weights drawn in {spec.dtype}, "
                   f"projections in {dm.compute} with fp32 accumulation",
                   "parallelism": "single GPU"},
        "prompt_prefix": {"tokens": q.n_prefix, "shared": shared} if q.n_prefix else None,
        "last_layer": "last positions only" if last_rows_only else "every position",
        "prefill_flops": fl["total"],
        "tokens_per_s": round(T / (ms_step * 1e-3), 1),
        "prefill_tokens_per_s": round(T / (prefill_ms * 1e-3), 1) if prefill_ms > 0 else None,
        "prefill_mfma_frac": round(fl["total"] / (prefill_ms * 1e-3) / 1e12 / peak, 4) if prefill_ms > 0 else None,
        "gemm_mfma_frac": gemm_frac,
        "stages_ms": stages,
        "relational_gbps": round(rel_bytes / (rel_ms * 1e-3) / 1e9, 2) if rel_ms > 0 else None,
        "roofline": {"bound": "mfma", "kernel": "k_gemm_bf16<EPI_SWIGLU> (gate/up projection + SwiGLU)",
                     "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": traffic,
                     "traffic_source": ("rocprofv3 FETCH_SIZE x2.000 + WRITE_SIZE x1.000 per launch of this GEMM "
                                        "source, separate counter runs (profiles/sweep3b_hbm_traffic.md)")
                     if traffic is not None else None,
                     "launches": int(len(up_ms)), "avg_launch_ms": round(up_avg_ms, 5),
                     "flops_per_launch": up_flops_per_launch,
                     "tokens_per_launch": sorted(set(real_tok)),
                     "empty_launches": int(len(empty_ms)),
                     "empty_launch_avg_ms": round(float(np.mean(empty_ms)), 5) if len(empty_ms) else None},
    }
    if gen:
        result["generation"] = generation_report(spec, q, tables, sel, kinds, B, ms_step)
        if a.all_queries:
            result["queries"] = [time_query(tables, model, dm, qq, B, torch, a.steps, a.warmup, n_rows)
                                 for qq in w.queries]
        a.no_cpu_baseline = a.no_split = True   # the oracle and the split baseline classify; no generation
        result["cpu_baseline"] = None
    if pairs:
        result["pairs"] = {"candidates": res["n_pairs"], "kept": res["count"],
                           "pairs_per_s": round(res["n_pairs"] / (ms_step * 1e-3), 1)}
        a.no_cpu_baseline = a.no_split = True   # both classify single rows
        result["cpu_baseline"] = None
    if not a.no_relational_scale and not gen and not pairs:
        result["relational_scale"] = relational_scale_leg(B, torch, [1 << 26, 1 << 28], [10, 1000], steps=5)
    if not a.no_cpu_baseline:
        log("[bench] cpu baseline (oracle on a sample)")
        result["cpu_baseline"] = cpu_baseline_leg(tables, model, q, spec, a.cpu_flop)
    if not a.no_split:
        log("[bench] split-execution baseline")
        result["split_baseline"] = split_baseline_leg(tables, model, q, dm, B, torch)
    dq.close()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
