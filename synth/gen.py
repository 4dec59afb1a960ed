"""Seeded generators for tables, token lists and model weights.

Every column and every weight tensor has its own random stream,
``PCG64(SeedSequence([seed, stream, chunk]))``, so any one of them can be
regenerated on its own and large ones can be drawn in parallel chunks.  The
draw definitions (fixed here, used identically by every consumer):

* lognormal lengths: ``clip(rint(median * exp(sigma * z)), lo, hi)``, z ~ N(0,1) in fp64
  (numpy ``rint`` rounds half to even);
* bounded Zipf(s) over N items: P(k) proportional to k**-s for k = 1..N, drawn by
  inverse CDF (``searchsorted(cdf, u, 'right')`` on the fp64 CDF with its last
  entry set to 1); the value is the 0-based rank k - 1;
* weights: float32 standard normals times float32(std), rounded to nearest even
  into bf16 for bf16 models.  RMSNorm gains are ones.  No biases.

bf16 tensors are held as ``uint16`` bit patterns; ``as_f32`` widens them exactly.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .configs import WORKLOADS, ModelSpec, MoviesSpec, TableSpec, Workload

CHUNK = 1 << 22

# column stream ids
S_LEN, S_TOK, S_RATING, S_MOVIE, S_C, S_VALUES = 1, 2, 3, 4, 5, 6
S_MOVIES_ID, S_GENRE, S_YEAR = 10, 11, 12
S_PREFIX = 99
S_WEIGHT_BASE = 1000


def _rng(seed: int, stream: int, chunk: int | None = None) -> np.random.Generator:
    key = [seed, stream] if chunk is None else [seed, stream, chunk]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def zipf_cdf(s: float, n: int) -> np.ndarray:
    k = np.arange(1, n + 1, dtype=np.float64)
    p = k ** (-s)
    cdf = np.cumsum(p / p.sum())
    cdf[-1] = 1.0
    return cdf


def _zipf_draw(rng: np.random.Generator, cdf: np.ndarray, n: int) -> np.ndarray:
    u = rng.random(n)
    idx = np.searchsorted(cdf, u, side="right")
    np.minimum(idx, len(cdf) - 1, out=idx)
    return idx.astype(np.int32)


def _lengths(spec: TableSpec) -> np.ndarray:
    kind = spec.length[0]
    rng = _rng(spec.seed, S_LEN)
    if kind == "uniform":
        lo, hi = spec.length[1], spec.length[2]
        return rng.integers(lo, hi + 1, size=spec.n_rows).astype(np.int32)
    if kind == "lognormal":
        med, sigma, lo, hi = spec.length[1:]
        z = rng.standard_normal(spec.n_rows)
        return np.clip(np.rint(med * np.exp(sigma * z)), lo, hi).astype(np.int32)
    raise ValueError(kind)


def _tokens(spec: TableSpec, nnz: int) -> np.ndarray:
    out = np.empty(nnz, dtype=np.int32)
    kind = spec.tokens[0]
    cdf = zipf_cdf(spec.tokens[1], spec.tokens[2]) if kind == "zipf" else None

    def fill(c: int) -> None:
        lo, hi = c * CHUNK, min(nnz, (c + 1) * CHUNK)
        rng = _rng(spec.seed, S_TOK, c)
        if kind == "uniform":
            out[lo:hi] = rng.integers(0, spec.tokens[1], size=hi - lo, dtype=np.int32)
        else:
            out[lo:hi] = _zipf_draw(rng, cdf, hi - lo)

    n_chunks = (nnz + CHUNK - 1) // CHUNK
    if n_chunks <= 1:
        for c in range(n_chunks):
            fill(c)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(n_chunks)))
    return out


def make_probe(spec: TableSpec, movie_ids: np.ndarray | None = None, with_tokens: bool = True) -> dict:
    """Probe-table columns; with_tokens=False leaves out the token list (its
    offsets and lengths are still drawn, from the same streams)."""
    n = spec.n_rows
    lens = _lengths(spec)
    offsets = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    t = {"id": np.arange(n, dtype=np.int32), "len": lens, "offsets": offsets}
    if with_tokens:
        t["tokens"] = _tokens(spec, int(offsets[-1]))
    if spec.rating is not None:
        rng = _rng(spec.seed, S_RATING)
        if spec.rating[0] == "uniform":
            t["rating"] = rng.integers(spec.rating[1], spec.rating[2] + 1, size=n).astype(np.int8)
        else:
            p = np.asarray(spec.rating[1], dtype=np.float64)
            t["rating"] = (rng.choice(len(p), size=n, p=p) + 1).astype(np.int8)
    if spec.movie_id is not None:
        _, s, n_ids = spec.movie_id
        rank0 = _zipf_draw(_rng(spec.seed, S_MOVIE), zipf_cdf(s, n_ids), n)
        t["movie_id"] = rank0 if movie_ids is None else movie_ids[rank0].astype(np.int32)
    if spec.c_range is not None:
        lo, hi = spec.c_range
        t["c"] = _rng(spec.seed, S_C).integers(lo, hi + 1, size=n).astype(np.int32)
    if spec.values_a is not None:
        lo, hi = spec.values_a
        u = _rng(spec.seed, S_VALUES).random(n)
        t["values_a"] = np.minimum((lo + (hi - lo) * u).astype(np.float32), np.float32(hi))
    return t


def make_movies(spec: MoviesSpec) -> dict:
    n = spec.n_rows
    # distinct ids in [0, 2**31 - 2]; INT32_MIN stays free as an empty-slot value
    ids = _rng(spec.seed, S_MOVIES_ID).choice(2 ** 31 - 1, size=n, replace=False).astype(np.int32)
    genre = _rng(spec.seed, S_GENRE).integers(0, spec.n_genres, size=n).astype(np.int8)
    year = _rng(spec.seed, S_YEAR).integers(spec.year_lo, spec.year_hi + 1, size=n).astype(np.int16)
    return {"movie_id": ids, "genre": genre, "year": year}


def make_prefix(seed: int, n: int, vocab: int) -> np.ndarray:
    if n == 0:
        return np.zeros(0, dtype=np.int32)
    # uniform over [3, vocab): the label tokens 1 and 2 never appear in the prompt
    return _rng(seed, S_PREFIX).integers(3, vocab, size=n).astype(np.int32)


def make_tables(w: Workload) -> dict:
    """Returns {"probe": columns, "build": columns or None, "prefix": int32[n]}."""
    build = make_movies(w.movies) if w.movies is not None else None
    probe = make_probe(w.table, None if build is None else build["movie_id"])
    n_prefix = max(q.n_prefix for q in w.queries)
    return {"probe": probe, "build": build,
            "prefix": make_prefix(w.table.seed, n_prefix, w.model.vocab)}


# ---------------------------------------------------------------------------
# weights
# ---------------------------------------------------------------------------


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def as_f32(w: np.ndarray) -> np.ndarray:
    """Exact float32 view of a weight tensor (bf16 bit patterns are widened)."""
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << 16).view(np.float32)
    return w


def _draw_tensor(spec: ModelSpec, index: int, shape: tuple, pool: ThreadPoolExecutor | None) -> np.ndarray:
    n = int(np.prod(shape))
    dt = np.uint16 if spec.dtype == "bf16" else np.float32
    out = np.empty(n, dtype=dt)
    std = np.float32(spec.init_std)

    def fill(c: int) -> None:
        lo, hi = c * CHUNK, min(n, (c + 1) * CHUNK)
        x = _rng(spec.weight_seed, S_WEIGHT_BASE + index, c).standard_normal(hi - lo, dtype=np.float32)
        x *= std
        out[lo:hi] = bf16_round(x) if dt == np.uint16 else x

    chunks = range((n + CHUNK - 1) // CHUNK)
    if pool is None or len(chunks) == 1:
        for c in chunks:
            fill(c)
    else:
        list(pool.map(fill, chunks))
    return out.reshape(shape)


def make_model(spec: ModelSpec, n_layers: int | None = None) -> dict:
    """Weights of a random-init decoder.  All matrices are row-major [out, in].

    ``n_layers`` may truncate the stack (the tensors drawn are the same as the
    first layers of the full model)."""
    d, f, V = spec.d_model, spec.d_ff, spec.vocab
    L = spec.n_layers if n_layers is None else n_layers
    per = 9
    ones = np.ones(d, dtype=np.float32)
    with ThreadPoolExecutor(_threads()) as pool:
        m = {"spec": spec, "emb": _draw_tensor(spec, 0, (V, d), pool), "layers": []}
        for l in range(L):
            b = 1 + per * l
            layer = {
                "attn_norm": ones.copy(),
                "wq": _draw_tensor(spec, b + 1, (spec.d_q, d), pool),
                "wk": _draw_tensor(spec, b + 2, (spec.d_kv, d), pool),
                "wv": _draw_tensor(spec, b + 3, (spec.d_kv, d), pool),
                "wo": _draw_tensor(spec, b + 4, (d, spec.d_q), pool),
                "ffn_norm": ones.copy(),
                "w_gate": _draw_tensor(spec, b + 6, (f, d), pool),
                "w_down": _draw_tensor(spec, b + 8, (d, f), pool),
            }
            if spec.act == "swiglu":
                layer["w_up"] = _draw_tensor(spec, b + 7, (f, d), pool)
            m["layers"].append(layer)
        m["final_norm"] = ones.copy()
        m["lm_head"] = _draw_tensor(spec, 1 + per * spec.n_layers, (V, d), pool)
    return m


def make_workload(name: str, with_model: bool = True) -> dict:
    w = WORKLOADS[name]
    out = {"workload": w, **make_tables(w)}
    if with_model:
        out["model"] = make_model(w.model)
    return out
