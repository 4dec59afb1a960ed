"""ctypes binding of libaiq.so (declared in include/aiq.h).

Argument marshalling only: the structs mirror the C declarations field by
field and the functions keep their C names.  Every step of the query runs in
the library's HIP kernels; this module never computes a result.  Loading
fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libaiq.so")

AIQ_ABI_VERSION = 6   # the struct layouts below
AIQ_OK, AIQ_EINVAL, AIQ_EUNSUPPORTED, AIQ_ENOSPC, AIQ_EHIP, AIQ_ENOMEM = 0, -1, -2, -3, -4, -5
AIQ_I8, AIQ_I16, AIQ_I32, AIQ_F32, AIQ_BF16, AIQ_F16 = 1, 2, 3, 4, 5, 6
AIQ_LT, AIQ_LE, AIQ_GT, AIQ_GE, AIQ_EQ, AIQ_NE, AIQ_IN = range(7)
AIQ_ACT_GELU_ERF, AIQ_ACT_SWIGLU = 1, 2
AIQ_DECIDE_BINARY_GT, AIQ_DECIDE_ARGMAX = 1, 2
AIQ_AGG_COUNT, AIQ_AGG_AVG_LABEL_COUNT_BY, AIQ_AGG_COUNT_BY_PAYLOAD, AIQ_AGG_SUM_F32 = 1, 2, 3, 4
AIQ_LOGITS_LABELS, AIQ_LOGITS_FULL_VOCAB = 1, 2
AIQ_PLAN_RELATIONAL_ONLY = 1
AIQ_PLAN_UNSHARED_PREFIX = 2
AIQ_PLAN_MULTIPASS_COMPACT = 4
AIQ_PLAN_FULL_LAST_LAYER = 8

AIQ_DEV_TOKEN_RANGE, AIQ_DEV_DUP_KEY, AIQ_DEV_HASH_FULL, AIQ_DEV_IDS_CAP = 0x01, 0x02, 0x04, 0x08
AIQ_DEV_GROUP_RANGE, AIQ_DEV_LIST_LEN, AIQ_DEV_GROUP_CAP, AIQ_DEV_PAIR_CAP = 0x10, 0x20, 0x40, 0x80
AIQ_DEV_SCAN_WAIT = 0x100
AIQ_S_SELECTED, AIQ_S_KEPT, AIQ_S_TOKENS, AIQ_S_STATUS, AIQ_S_GROUPS, AIQ_S_PAIRS = range(6)
AIQ_N_SCALARS = 8
AIQ_MAX_PREDS, AIQ_MAX_IN_SET, AIQ_MAX_PREFIX, AIQ_MAX_LABELS = 8, 32, 64, 8
AIQ_MAX_GEN, AIQ_MAX_LIKE = 512, 16

(AIQ_K_REL, AIQ_K_PACK, AIQ_K_EMBED, AIQ_K_NORM, AIQ_K_GEMM_QKV, AIQ_K_ATTN, AIQ_K_GEMM_O,
 AIQ_K_GEMM_UP, AIQ_K_GEMM_DOWN, AIQ_K_HEAD, AIQ_K_AGG, AIQ_K_DECODE, AIQ_K_DECODE_ATTN,
 AIQ_K_DECODE_HEAD, AIQ_K_LAST) = range(15)

OPS = {"lt": AIQ_LT, "le": AIQ_LE, "gt": AIQ_GT, "ge": AIQ_GE, "eq": AIQ_EQ, "ne": AIQ_NE, "in": AIQ_IN}


class aiq_col(C.Structure):
    _fields_ = [("data", C.c_void_p), ("dtype", C.c_int32)]


class aiq_table(C.Structure):
    _fields_ = [("n_rows", C.c_int64), ("n_cols", C.c_int32), ("cols", C.POINTER(aiq_col)),
                ("list_offsets", C.c_void_p), ("list_tokens", C.c_void_p),
                ("n_list_tokens", C.c_int64), ("max_list_len", C.c_int32)]


class aiq_pred(C.Structure):
    _fields_ = [("col", C.c_int32), ("op", C.c_int32), ("k", C.c_int64), ("n_set", C.c_int32),
                ("set", C.c_int64 * AIQ_MAX_IN_SET), ("fk", C.c_double)]


class aiq_layer(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm",
                                           "w_gate", "w_up", "w_down")]


class aiq_model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("d_ff", C.c_int32), ("vocab", C.c_int32),
                ("act", C.c_int32), ("wdtype", C.c_int32), ("rope_theta", C.c_double),
                ("norm_eps", C.c_double), ("emb", C.c_void_p), ("layers", C.POINTER(aiq_layer)),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)]


class aiq_query(C.Structure):
    _fields_ = [("n_pred", C.c_int32), ("preds", aiq_pred * AIQ_MAX_PREDS),
                ("join", C.c_int32), ("probe_key_col", C.c_int32), ("build_key_col", C.c_int32),
                ("build_payload_col", C.c_int32), ("n_build_pred", C.c_int32),
                ("build_preds", aiq_pred * AIQ_MAX_PREDS),
                ("n_prefix", C.c_int32), ("prefix", C.c_int32 * AIQ_MAX_PREFIX),
                ("n_labels", C.c_int32), ("label_ids", C.c_int32 * AIQ_MAX_LABELS),
                ("decision", C.c_int32), ("agg", C.c_int32), ("group_col", C.c_int32),
                ("n_group_keys", C.c_int32), ("gen_tokens", C.c_int32), ("eos_id", C.c_int32),
                ("pad_id", C.c_int32), ("n_like", C.c_int32), ("like", C.c_int32 * AIQ_MAX_LIKE),
                ("pairs", C.c_int32), ("pair_key_col", C.c_int32), ("max_pairs", C.c_int64)]


class aiq_plan_opts(C.Structure):
    _fields_ = [("chunk_tokens", C.c_int64), ("n_layers_override", C.c_int32), ("flags", C.c_int32),
                ("reserved", C.c_int32 * 4)]


class aiq_out(C.Structure):
    _fields_ = [("scalars", C.c_void_p), ("ids", C.c_void_p), ("ids_cap", C.c_int64),
                ("sel_ids", C.c_void_p), ("sel_labels", C.c_void_p), ("sel_logits", C.c_void_p),
                ("sel_cap", C.c_int64), ("grp_key", C.c_void_p), ("grp_count", C.c_void_p),
                ("grp_sum", C.c_void_p), ("grp_avg", C.c_void_p), ("grp_cap", C.c_int64),
                ("sum_out", C.c_void_p), ("sel_gen", C.c_void_p), ("pair_a", C.c_void_p),
                ("pair_b", C.c_void_p), ("cand_a", C.c_void_p), ("cand_b", C.c_void_p)]


class aiq_trace(C.Structure):
    _fields_ = [("events", C.POINTER(C.c_void_p)), ("tags", C.POINTER(C.c_int32)),
                ("capacity", C.c_int32), ("count", C.c_int32), ("kind_mask", C.c_uint32)]


EXPORTS = ("aiq_plan_create", "aiq_workspace_size", "aiq_plan_passes", "aiq_plan_chunk_tokens",
           "aiq_plan_last_layer_rows", "aiq_run", "aiq_run_relational_static", "aiq_convert_weights",
           "aiq_prefill_workspace_size",
           "aiq_prefill_packed", "aiq_plan_destroy", "aiq_status_str", "aiq_abi_version")


class AiqError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed: {msg} ({status})")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Loads libaiq.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_10139_amd.build`")
    lib = C.CDLL(path)
    P = C.c_void_p
    lib.aiq_plan_create.argtypes = [C.POINTER(aiq_model), C.POINTER(aiq_table), C.POINTER(aiq_table),
                                    C.POINTER(aiq_query), C.POINTER(aiq_plan_opts), C.POINTER(P)]
    lib.aiq_plan_create.restype = C.c_int
    lib.aiq_workspace_size.argtypes = [P, C.POINTER(C.c_size_t)]
    lib.aiq_workspace_size.restype = C.c_int
    lib.aiq_plan_passes.argtypes = [P, C.POINTER(C.c_int64), C.POINTER(C.c_int32)]
    lib.aiq_plan_passes.restype = C.c_int
    lib.aiq_plan_chunk_tokens.argtypes = [P, C.POINTER(C.c_int64)]
    lib.aiq_plan_chunk_tokens.restype = C.c_int
    lib.aiq_plan_last_layer_rows.argtypes = [P, C.POINTER(C.c_int32)]
    lib.aiq_plan_last_layer_rows.restype = C.c_int
    lib.aiq_run.argtypes = [P, P, C.c_size_t, C.POINTER(aiq_out), C.POINTER(aiq_trace), P]
    lib.aiq_run.restype = C.c_int
    lib.aiq_convert_weights.argtypes = [P, C.c_int32, P, C.c_int32, C.c_int64, P]
    lib.aiq_convert_weights.restype = C.c_int
    lib.aiq_run_relational_static.argtypes = [P, C.POINTER(aiq_out), P]
    lib.aiq_run_relational_static.restype = C.c_int
    lib.aiq_prefill_workspace_size.argtypes = [P, C.c_int64, C.POINTER(C.c_size_t)]
    lib.aiq_prefill_workspace_size.restype = C.c_int
    lib.aiq_prefill_packed.argtypes = [P, P, P, C.c_int32, C.c_int64, C.c_int32, P, P, C.c_size_t, P]
    lib.aiq_prefill_packed.restype = C.c_int
    lib.aiq_plan_destroy.argtypes = [P]
    lib.aiq_plan_destroy.restype = None
    lib.aiq_status_str.argtypes = [C.c_int32]
    lib.aiq_status_str.restype = C.c_char_p
    lib.aiq_abi_version.argtypes = []
    lib.aiq_abi_version.restype = C.c_int32
    if lib.aiq_abi_version() != AIQ_ABI_VERSION:
        raise RuntimeError(f"{path} has ABI version {lib.aiq_abi_version()}, this binding expects "
                           f"{AIQ_ABI_VERSION}: rebuild it")
    _lib = lib
    return lib


def check(fn: str, status: int) -> None:
    if status != AIQ_OK:
        raise AiqError(fn, status, load().aiq_status_str(status).decode())


# ---------------------------------------------------------------- same-name wrappers

def aiq_plan_create(model, probe, build, query, opts=None) -> C.c_void_p:
    plan = C.c_void_p()
    st = load().aiq_plan_create(C.byref(model), C.byref(probe) if probe is not None else None,
                                C.byref(build) if build is not None else None,
                                C.byref(query) if query is not None else None,
                                C.byref(opts) if opts is not None else None, C.byref(plan))
    check("aiq_plan_create", st)
    return plan


def aiq_plan_create_status(model, probe, build, query, opts=None) -> int:
    """Like aiq_plan_create but returns the status (for error-path tests)."""
    plan = C.c_void_p()
    st = load().aiq_plan_create(C.byref(model) if model is not None else None,
                                C.byref(probe) if probe is not None else None,
                                C.byref(build) if build is not None else None,
                                C.byref(query) if query is not None else None,
                                C.byref(opts) if opts is not None else None, C.byref(plan))
    if st == AIQ_OK:
        load().aiq_plan_destroy(plan)
    return st


def aiq_workspace_size(plan) -> int:
    n = C.c_size_t()
    check("aiq_workspace_size", load().aiq_workspace_size(plan, C.byref(n)))
    return n.value


def aiq_plan_passes(plan) -> tuple:
    """(chunk passes, 1 if a shared-prefix pass runs else 0) of aiq_run."""
    n = C.c_int64()
    pp = C.c_int32()
    check("aiq_plan_passes", load().aiq_plan_passes(plan, C.byref(n), C.byref(pp)))
    return n.value, pp.value


def aiq_plan_chunk_tokens(plan) -> int:
    """Units (tokens + sequences) per prefill pass of aiq_run."""
    v = C.c_int64()
    check("aiq_plan_chunk_tokens", load().aiq_plan_chunk_tokens(plan, C.byref(v)))
    return v.value


def aiq_plan_last_layer_rows(plan) -> bool:
    """True when the plan runs its last layer for the last positions only."""
    v = C.c_int32()
    check("aiq_plan_last_layer_rows", load().aiq_plan_last_layer_rows(plan, C.byref(v)))
    return bool(v.value)


def aiq_prefill_workspace_size(plan, max_tokens: int) -> int:
    n = C.c_size_t()
    check("aiq_prefill_workspace_size", load().aiq_prefill_workspace_size(plan, max_tokens, C.byref(n)))
    return n.value


def aiq_run(plan, ws_ptr: int, ws_bytes: int, out: aiq_out, trace=None, stream: int = 0) -> None:
    check("aiq_run", load().aiq_run(plan, ws_ptr, ws_bytes, C.byref(out),
                                    C.byref(trace) if trace is not None else None, stream))


def aiq_run_relational_static(plan, out: aiq_out, stream: int = 0) -> None:
    check("aiq_run_relational_static", load().aiq_run_relational_static(plan, C.byref(out), stream))


def aiq_run_relational_static_status(plan, out: aiq_out, stream: int = 0) -> int:
    """Like aiq_run_relational_static but returns the status (for error-path tests)."""
    return load().aiq_run_relational_static(plan, C.byref(out), stream)


def aiq_convert_weights(src_ptr: int, src_dtype: int, dst_ptr: int, dst_dtype: int, n: int, stream: int = 0) -> None:
    check("aiq_convert_weights", load().aiq_convert_weights(src_ptr, src_dtype, dst_ptr, dst_dtype, n, stream))


def aiq_prefill_packed(plan, tok_ptr: int, cu_ptr: int, n_seq: int, n_tok: int, mode: int,
                       logits_ptr: int, ws_ptr: int, ws_bytes: int, stream: int = 0) -> None:
    check("aiq_prefill_packed", load().aiq_prefill_packed(plan, tok_ptr, cu_ptr, n_seq, n_tok, mode,
                                                          logits_ptr, ws_ptr, ws_bytes, stream))


def aiq_plan_destroy(plan) -> None:
    load().aiq_plan_destroy(plan)


def aiq_abi_version() -> int:
    return load().aiq_abi_version()


def aiq_status_str(st: int) -> str:
    return load().aiq_status_str(st).decode()
