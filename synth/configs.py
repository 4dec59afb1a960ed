"""The five synthetic AI-query workloads and their query specifications.

Each workload is a reviews-shaped table (a fixed-width numeric filter column,
a token-list "review text" column) optionally joined with a movies table, a
randomly initialised decoder-only language model, and one or more queries of
the form used in the paper's evaluation (Section 4, Table 2):

    SELECT <agg> FROM reviews [JOIN movies ON movie_id]
    WHERE <relational predicate> AND AI_IF(review, <prompt>) = 1

The semantic operator is the last-token label comparison of the Figure 2
program (Section 3.1); the relational predicate is the WHERE clause mapped to
a boolean mask (Table 1).  The SemBench Rotten-Tomatoes data and Gemma-2B used
in the paper are not available; these seeded tables and random-init models
stand in for them with the stated shapes and skew.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

# ---------------------------------------------------------------------------
# Model specifications
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class ModelSpec:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ff: int
    vocab: int
    act: str            # "gelu" (exact erf GELU, 2-matrix FFN) or "swiglu"
    dtype: str          # "f32" or "bf16": storage type of the weights
    weight_seed: int    # seed of the weight streams
    rope_theta: float = 10000.0
    norm_eps: float = 1e-5
    init_std: float = 0.02

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def d_q(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    def body_params(self) -> int:
        d, f = self.d_model, self.d_ff
        n_ffn = 3 if self.act == "swiglu" else 2
        per_layer = d * self.d_q + 2 * d * self.d_kv + self.d_q * d + n_ffn * d * f
        return self.n_layers * per_layer


TINY = ModelSpec(n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, d_ff=512, vocab=1024,
                 act="gelu", dtype="f32", weight_seed=0)
SMALL = ModelSpec(n_layers=4, d_model=512, n_heads=8, n_kv_heads=8, d_ff=2048, vocab=32000,
                  act="swiglu", dtype="bf16", weight_seed=1)
ONE_B = ModelSpec(n_layers=16, d_model=2048, n_heads=32, n_kv_heads=8, d_ff=8192, vocab=32000,
                  act="swiglu", dtype="bf16", weight_seed=2)
THREE_B = ModelSpec(n_layers=28, d_model=3072, n_heads=24, n_kv_heads=8, d_ff=8192, vocab=32000,
                    act="swiglu", dtype="bf16", weight_seed=4)

# ---------------------------------------------------------------------------
# Table specifications
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class TableSpec:
    """A reviews-shaped probe table.

    length: ("uniform", lo, hi) inclusive, or ("lognormal", median, sigma, lo, hi)
    tokens: ("uniform", vocab) or ("zipf", s, vocab)
    rating: None, ("uniform", 1, 5) or ("probs", (p1..p5))
    extra columns: movie_id ("zipf", s, n_keys) as a key rank, c uniform int range,
    values_a uniform in [lo, hi] rounded to fp32 (the float column the paper's SUM queries add up).
    """
    n_rows: int
    seed: int
    length: tuple
    tokens: tuple
    rating: Optional[tuple] = None
    movie_id: Optional[tuple] = None      # ("zipf", s, n_ids)
    c_range: Optional[Tuple[int, int]] = None   # uniform int32 in [lo, hi]
    values_a: Optional[Tuple[float, float]] = None   # uniform in [lo, hi], rounded to fp32


@dataclass(frozen=True)
class MoviesSpec:
    n_rows: int
    seed: int
    n_genres: int = 20
    year_lo: int = 1950
    year_hi: int = 2025


# ---------------------------------------------------------------------------
# Query specification (mirrors the C-ABI query struct)
# ---------------------------------------------------------------------------

OPS = ("lt", "le", "gt", "ge", "eq", "ne", "in")


@dataclass(frozen=True)
class Pred:
    col: str
    op: str
    k: float = 0   # int for integer columns; a float constant for fp32 columns
    values: Tuple[int, ...] = ()


@dataclass(frozen=True)
class Join:
    probe_key: str
    build_key: str
    payload: str
    build_preds: Tuple[Pred, ...]


@dataclass(frozen=True)
class Query:
    preds: Tuple[Pred, ...]
    labels: Tuple[int, ...]
    decision: str                     # "binary_gt" or "argmax"
    agg: str                          # "count", "avg_label_count_by", "count_by_payload"
    join: Optional[Join] = None
    n_prefix: int = 0                 # prefix tokens drawn by the generator (stream 99)
    group_col: Optional[str] = None   # probe column for avg_label_count_by
    n_group_keys: int = 0             # dense key domain [0, n_group_keys); 0: any int32 key (hash)
    gen_tokens: int = 0               # AI_TRANSFORM: tokens generated per selected row (0: AI_IF)
    eos_id: int = -1
    pad_id: int = 0
    like: Tuple[int, ...] = ()        # LIKE '%pattern%' over the generated token ids
    pair_key: Optional[str] = None    # Q4: classify pairs of selected rows with equal keys in this column
    max_pairs: int = 0                # Q4: capacity for candidate pairs


@dataclass(frozen=True)
class Workload:
    name: str
    table: TableSpec
    model: ModelSpec
    queries: Tuple[Query, ...]
    movies: Optional[MoviesSpec] = None
    description: str = ""
    extra: dict = field(default_factory=dict)


_BINARY = (1, 2)   # "yes" token 1, "no" token 2

_LOGN_120 = ("lognormal", 120.0, 0.6, 16, 512)
_ZIPF_TOK = ("zipf", 1.1, 32000)
_RATING_P = ("probs", (0.1, 0.1, 0.2, 0.3, 0.3))

_TINY_TABLE = TableSpec(n_rows=256, seed=0, length=("uniform", 8, 64), tokens=("uniform", 1024),
                        rating=("uniform", 1, 5), values_a=(0.0, 100.0))
_REVIEWS_TABLE = TableSpec(n_rows=16384, seed=1, length=_LOGN_120, tokens=_ZIPF_TOK, rating=_RATING_P,
                           values_a=(0.0, 100.0))

WORKLOADS = {
    "tiny": Workload(
        name="tiny", description="tiny select + semantic filter, 256 rows, 2-layer fp32 decoder",
        table=_TINY_TABLE,
        model=TINY,
        queries=(Query(preds=(Pred("rating", "ge", 3),), labels=_BINARY, decision="binary_gt",
                       agg="count"),),
    ),
    "reviews": Workload(
        name="reviews", description="reviews-shaped binary filter, 16,384 rows, 4-layer d512 bf16 decoder",
        table=_REVIEWS_TABLE,
        model=SMALL,
        queries=(Query(preds=(Pred("rating", "le", 2), Pred("len", "gt", 32)), labels=_BINARY,
                       decision="binary_gt", agg="count"),),
    ),
    # the paper's running query shape: SUM(values_a) WHERE values_a > 70 AND AI_IF(...)
    "reviews_sum": Workload(
        name="reviews_sum", description="SUM of a float column over rows passing a float filter and the "
                                        "semantic filter, 16,384 rows, 4-layer d512 bf16 decoder",
        table=_REVIEWS_TABLE,
        model=SMALL,
        queries=(Query(preds=(Pred("values_a", "gt", 70.0),), labels=_BINARY, decision="binary_gt",
                       agg="sum_f32", group_col="values_a"),),
    ),
    "tiny_sum": Workload(
        name="tiny_sum", description="tiny SUM of a float column under float and semantic filters, 256 rows",
        table=_TINY_TABLE,
        model=TINY,
        queries=(Query(preds=(Pred("values_a", "ge", 30.0), Pred("rating", "ne", 4)), labels=_BINARY,
                       decision="binary_gt", agg="sum_f32", group_col="values_a"),),
    ),
    # AI_TRANSFORM with a relational predicate (Q3): the selectivity sweep of
    # the paper's Table 4 (values_a < 10 .. 90), a short prompt, 32 new tokens
    "reviews_transform": Workload(
        name="reviews_transform", description="Q3: AI_TRANSFORM of rows passing values_a < t (t = 10 .. 90), "
                                              "32 generated tokens, 16,384 rows, 4-layer d512 bf16 decoder",
        table=_REVIEWS_TABLE,
        model=SMALL,
        queries=tuple(Query(preds=(Pred("values_a", "lt", float(t)),), labels=(), decision="binary_gt",
                            agg="count", n_prefix=8, gen_tokens=32) for t in (10, 30, 50, 70, 90)),
    ),
    # COUNT over long generations filtered by LIKE (Q5)
    "reviews_like": Workload(
        name="reviews_like", description="Q5: COUNT(*) WHERE AI_TRANSFORM(text) LIKE '%p%', 128 generated "
                                         "tokens per row, 16,384 rows, 4-layer d512 bf16 decoder",
        table=_REVIEWS_TABLE,
        model=SMALL,
        queries=(Query(preds=(), labels=(), decision="binary_gt", agg="count", n_prefix=12, gen_tokens=128,
                       eos_id=2, pad_id=0, like=(17, 17)),),
    ),
    # classification of pairs of reviews of the same movie (Q4): a self-join on
    # the movie id, AI_IF over both texts
    "reviews_pairs": Workload(
        name="reviews_pairs", description="Q4: AI_IF over pairs of reviews of the same movie among rows passing "
                                          "values_a < 40, 16,384 rows, 4-layer d512 bf16 decoder",
        table=TableSpec(n_rows=16384, seed=1, length=_LOGN_120, tokens=_ZIPF_TOK, rating=_RATING_P,
                        values_a=(0.0, 100.0), movie_id=("zipf", 0.5, 4096)),
        model=SMALL,
        queries=(Query(preds=(Pred("values_a", "lt", 40.0),), labels=_BINARY, decision="binary_gt", agg="count",
                       n_prefix=8, pair_key="movie_id", n_group_keys=4096, max_pairs=65536),),
    ),
    "groupby1b": Workload(
        name="groupby1b", description="1B-class 5-way classify + GROUP BY movie_id, 131,072 rows",
        table=TableSpec(n_rows=131072, seed=2, length=_LOGN_120, tokens=_ZIPF_TOK, rating=_RATING_P,
                        movie_id=("zipf", 1.2, 4096)),
        model=ONE_B,
        queries=(Query(preds=(), labels=(1, 2, 3, 4, 5), decision="argmax",
                       agg="avg_label_count_by", group_col="movie_id", n_group_keys=4096),),
    ),
    "join1b": Workload(
        name="join1b", description="reviews (262,144) JOIN movies (8,192) with shared 32-token prefix, 1B model",
        table=TableSpec(n_rows=262144, seed=3, length=_LOGN_120, tokens=_ZIPF_TOK,
                        movie_id=("zipf", 1.2, 8192)),
        movies=MoviesSpec(n_rows=8192, seed=3),
        model=ONE_B,
        queries=(Query(preds=(), labels=_BINARY, decision="binary_gt", agg="count_by_payload",
                       n_prefix=32, n_group_keys=20,
                       join=Join(probe_key="movie_id", build_key="movie_id", payload="genre",
                                 build_preds=(Pred("genre", "in", values=(2, 5, 11)),
                                              Pred("year", "gt", 2000)))),),
    ),
    "sweep3b": Workload(
        name="sweep3b", description="selectivity sweep, 1,048,576 rows, 3B-class decoder",
        table=TableSpec(n_rows=1048576, seed=4, length=("lognormal", 200.0, 0.7, 16, 1024),
                        tokens=_ZIPF_TOK, c_range=(0, 999)),
        model=THREE_B,
        queries=tuple(Query(preds=(Pred("c", "lt", t),), labels=_BINARY, decision="binary_gt",
                            agg="count") for t in (10, 100, 500, 1000)),
    ),
}

# the workload order used by the paper-shaped configuration list (seed = index)
ORDER = ("tiny", "reviews", "groupby1b", "join1b", "sweep3b")


def query_for(name: str, i: int = 0) -> Query:
    return WORKLOADS[name].queries[i]


def model_spec(name: str) -> ModelSpec:
    return WORKLOADS[name].model
