"""Seeded synthetic workloads shaped like the paper's five sparse-access tasks.

This module only draws random inputs: key ids, values, labels and initial
tables.  It holds none of the training arithmetic (no scores, gradients,
sorting or updates), so both the GPU path and the CPU oracle can take their
inputs from it without sharing any of the method.

Shapes follow the paper's task descriptions (Appendix C, "Task details", and
Table 3): matrix factorization of a Zipf-1.1 distributed 10m x 1m matrix,
ComplEx knowledge-graph embeddings trained with uniform negative sampling,
skip-gram word vectors with negative sampling and a window of 5, and a
click-through-rate model whose embedding tables are indexed by hashed
categorical features.  The real datasets (Wikidata5M, One Billion Word,
Criteo Kaggle) are replaced by synthetic streams with Zipf-distributed key
frequencies; nothing from those datasets is reproduced.

Every per-step batch is a pure function of (seed, step): batches are drawn
from a ``numpy.random.Generator`` keyed by ``SeedSequence([seed, tag, step])``
and the skip-gram token stream from a counter-based splitmix64 hash of the
stream position, so step ``s`` can be produced without generating steps
``0..s-1`` and the 1e9-entry streams are never materialized.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, field, replace

import numpy as np

# ---------------------------------------------------------------------------
# counter-based hashing (splitmix64, Steele, Lea & Flood, OOPSLA 2014)
# ---------------------------------------------------------------------------
_M64 = np.uint64(0xFFFFFFFFFFFFFFFF)


def splitmix64(x: np.ndarray) -> np.ndarray:
    """The splitmix64 finalizer applied elementwise to uint64 ``x + golden``."""
    with np.errstate(over="ignore"):
        z = np.asarray(x, dtype=np.uint64) + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def _hash_uniform(key: np.ndarray) -> np.ndarray:
    """Uniform doubles in [0, 1) from the top 53 bits of splitmix64(key)."""
    return (splitmix64(key) >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


def _rng(seed: int, tag: int, step: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, tag, step]))


# ---------------------------------------------------------------------------
# finite Zipf sampler: p(rank k) proportional to k^-s, k = 1..n, rank -> id
# through a seeded permutation so that hot ids are not contiguous
# ---------------------------------------------------------------------------
class Zipf:
    def __init__(self, n: int, s: float, seed: int, tag: int, permute: bool = True):
        self.n, self.s = int(n), float(s)
        w = np.arange(1, self.n + 1, dtype=np.float64) ** (-self.s)
        self.cdf = np.cumsum(w)
        self.total = float(self.cdf[-1])
        self.pmf = w / self.total
        if permute:
            self.perm = _rng(seed, tag, 0).permutation(self.n).astype(np.int64)
        else:
            self.perm = np.arange(self.n, dtype=np.int64)

    def ranks(self, u: np.ndarray) -> np.ndarray:
        r = np.searchsorted(self.cdf, np.asarray(u) * self.total, side="right")
        return np.minimum(r, self.n - 1)

    def ids_from_uniform(self, u: np.ndarray) -> np.ndarray:
        return self.perm[self.ranks(u)]

    def sample(self, rng: np.random.Generator, size) -> np.ndarray:
        return self.ids_from_uniform(rng.random(size))


# ---------------------------------------------------------------------------
# initial tables
# ---------------------------------------------------------------------------
def _fill_parallel(out: np.ndarray, seed: int, tag: int, fn, chunk_rows: int = 1 << 16):
    """Fill ``out`` (rows x d, float32) chunk by chunk; chunk i uses its own
    SeedSequence so the result does not depend on the number of threads."""
    rows = out.shape[0]
    nchunks = (rows + chunk_rows - 1) // chunk_rows

    def work(i):
        lo, hi = i * chunk_rows, min(rows, (i + 1) * chunk_rows)
        fn(_rng(seed, tag, 1_000_000 + i), out[lo:hi])

    threads = max(1, min(16, os.cpu_count() or 1))
    if nchunks <= 1 or threads == 1:
        for i in range(nchunks):
            work(i)
    else:
        with _cf.ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nchunks)))
    return out


def normal_table(rows: int, d: int, std: float, seed: int, tag: int) -> np.ndarray:
    out = np.empty((rows, d), dtype=np.float32)

    def fn(rng, blk):
        rng.standard_normal(blk.shape, dtype=np.float32, out=blk)
        blk *= np.float32(std)

    return _fill_parallel(out, seed, tag, fn)


def uniform_table(rows: int, d: int, lo: float, hi: float, seed: int, tag: int) -> np.ndarray:
    out = np.empty((rows, d), dtype=np.float32)

    def fn(rng, blk):
        blk[...] = rng.uniform(lo, hi, blk.shape).astype(np.float32)

    return _fill_parallel(out, seed, tag, fn)


# ---------------------------------------------------------------------------
# task configurations
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class AdaGradCfg:
    lr: float = 0.1
    eps: float = 1e-10


@dataclass(frozen=True)
class MFConfig:
    """Low-rank matrix factorization (Appendix C, "Matrix factorization";
    Table 3): squared loss with L2, rows uniform, columns Zipf."""
    name: str
    n_rows: int
    n_cols: int
    nnz: int
    rank: int
    batch: int
    zipf_s: float = 1.1
    lam: float = 1e-2
    init_std: float = 0.1
    opt: AdaGradCfg = field(default_factory=AdaGradCfg)
    seed: int = 0
    fixed_dataset: bool = False   # small case: one dataset, batches in order
    # "random": each batch draws its entries i.i.d.; "column": the paper's
    # visiting order, the entries of one column after another, columns in a
    # random order (Appendix C, "Matrix factorization")
    visit: str = "random"
    # rows uniform (None, the configurations above) or Zipf with this
    # exponent over a seeded permutation (users of very unequal activity)
    row_zipf_s: float | None = None

    @property
    def num_keys(self) -> int:
        return self.n_rows + self.n_cols

    @property
    def dim(self) -> int:
        return self.rank

    @property
    def steps_per_epoch(self) -> int:
        return (self.nnz + self.batch - 1) // self.batch

    def occurrences(self, b: int) -> int:
        return 2 * b


@dataclass(frozen=True)
class KGEConfig:
    """ComplEx knowledge-graph embeddings with uniform negative sampling
    (Appendix C, "Knowledge graph embeddings")."""
    name: str
    n_ent: int
    n_rel: int
    n_triples: int
    cdim: int            # complex dimension; a row holds [Re | Im] = 2*cdim floats
    n_neg: int
    n_head_neg: int
    batch: int
    zipf_s: float = 1.0
    init_std: float = 0.1
    opt: AdaGradCfg = field(default_factory=AdaGradCfg)
    seed: int = 0

    @property
    def num_keys(self) -> int:
        return self.n_ent + self.n_rel

    @property
    def dim(self) -> int:
        return 2 * self.cdim

    def occurrences(self, b: int) -> int:
        return b * (3 + self.n_neg)


@dataclass(frozen=True)
class SGNSConfig:
    """Skip-gram word vectors with negative sampling (Appendix C, "Word
    vectors"): input table keys [0, V), output table keys [V, 2V)."""
    name: str
    vocab: int
    n_tokens: int
    dim: int
    window: int
    n_neg: int
    batch: int
    zipf_s: float = 1.0
    neg_power: float = 0.75
    opt: AdaGradCfg = field(default_factory=AdaGradCfg)
    seed: int = 0
    subsample: float = 0.0        # word2vec's frequent-word threshold t (0: keep every token)
    dynamic_window: bool = False  # word2vec's per-centre window drawn uniformly from 1..window

    @property
    def num_keys(self) -> int:
        return 2 * self.vocab

    def occurrences(self, b: int) -> int:
        return b * (1 + 2 * self.window * (1 + self.n_neg))


@dataclass(frozen=True)
class CTRConfig:
    """Embedding part of a click-through-rate model (Appendix C,
    "Click-through-rate prediction"): categorical fields hashed into one
    table, pairwise dot-product interaction, logistic loss."""
    name: str
    n_fields: int
    table_rows: int
    dim: int
    batch: int
    vocab_min: int = 10
    vocab_max: int = 10_000_000
    zipf_s: float = 1.05
    p_click: float = 0.25
    init_std: float = 0.1
    opt: AdaGradCfg = field(default_factory=AdaGradCfg)
    seed: int = 0
    # Wide & Deep (empty deep: the embedding model with pairwise interaction):
    # rows hold [embedding (emb_dim) | wide weight | zero padding to dim],
    # the deep part is an MLP with these hidden widths over the F embeddings
    deep: tuple = ()
    emb_dim: int = 0

    @property
    def num_keys(self) -> int:
        return self.table_rows

    @property
    def dense_size(self) -> int:
        """Floats of the Wide & Deep dense buffer (hidden layers, output)."""
        n, fan = 0, self.n_fields * self.emb_dim
        for h in self.deep:
            n += fan * h + h
            fan = h
        return n + fan + 1

    def occurrences(self, b: int) -> int:
        return b * self.n_fields

    def vocab_sizes(self) -> list[int]:
        if self.n_fields == 1:
            return [self.vocab_max]
        f = np.arange(self.n_fields, dtype=np.float64)
        span = np.log10(self.vocab_max / self.vocab_min)
        return [int(round(self.vocab_min * 10 ** (span * x / (self.n_fields - 1)))) for x in f]


# The five workloads (tiny MF, MF at paper scale, ComplEx, skip-gram, CTR).
MF_TINY = MFConfig("mf_tiny_1000x500_r16", n_rows=1000, n_cols=500, nnz=20_000, rank=16,
                   batch=1024, fixed_dataset=True)
MF_10Mx1M = MFConfig("mf_10Mx1M_r100", n_rows=10_000_000, n_cols=1_000_000,
                     nnz=1_000_000_000, rank=100, batch=1_048_576)
KGE_COMPLEX = KGEConfig("kge_complex_4.6M_d128", n_ent=4_600_000, n_rel=822,
                        n_triples=20_000_000, cdim=128, n_neg=100, n_head_neg=50, batch=4096)
SGNS_1M = SGNSConfig("sgns_1M_d300", vocab=1_000_000, n_tokens=1_000_000_000, dim=300,
                     window=5, n_neg=25, batch=65_536)
CTR_33M = CTRConfig("ctr_26f_2^25_d64", n_fields=26, table_rows=1 << 25, dim=64, batch=8192)

# The paper's CTR model is Wide & Deep (Appendix C, "Click-through-rate
# prediction", learning rate 1e-4): embeddings of 64 plus a wide weight per
# key (rows of 68 floats with padding), three hidden layers of 1024.
CTR_33M_WD = replace(CTR_33M, name="ctr_26f_2^25_d64_widedeep", dim=68, emb_dim=64, deep=(1024, 1024, 1024),
                     opt=AdaGradCfg(lr=1e-4))

CONFIGS = [MF_TINY, MF_10Mx1M, KGE_COMPLEX, SGNS_1M, CTR_33M]

# The paper corrupts both the subject and the object n_neg = 100 times each
# (Appendix C, "Knowledge graph embeddings"): 100 head- then 100
# tail-corrupted negatives per triple.
KGE_COMPLEX_2x100 = replace(KGE_COMPLEX, name="kge_complex_4.6M_d128_2x100neg", n_neg=200, n_head_neg=100)

# word2vec's common parameters as the paper uses them (Appendix C, "Word
# vectors"): window 5 drawn per centre, frequent-word subsampling 0.01.
SGNS_1M_W2V = replace(SGNS_1M, name="sgns_1M_d300_w2v", subsample=0.01, dynamic_window=True)

# The paper's visiting order for MF: by column, columns in random order
# (Appendix C, "Matrix factorization").
MF_10Mx1M_COLORDER = replace(MF_10Mx1M, name="mf_10Mx1M_r100_colorder", visit="column")


def small_variant(cfg, scale: str = "small"):
    """Reduced sizes of the same workload for oracle-speed parity tests: the
    same distributions, fewer keys and a batch that spans several tiles and
    ends in a ragged tail."""
    if isinstance(cfg, MFConfig):
        return replace(cfg, name=cfg.name + "_" + scale, n_rows=20_000, n_cols=3_000,
                       nnz=10 * 5_003, rank=cfg.rank, batch=5_003, fixed_dataset=False)
    if isinstance(cfg, KGEConfig):
        return replace(cfg, name=cfg.name + "_" + scale, n_ent=5_000, n_rel=37,
                       n_triples=10 * 97, cdim=cfg.cdim, batch=97)
    if isinstance(cfg, SGNSConfig):
        return replace(cfg, name=cfg.name + "_" + scale, vocab=3_000, n_tokens=100_000,
                       batch=257)
    if isinstance(cfg, CTRConfig):
        return replace(cfg, name=cfg.name + "_" + scale, table_rows=1 << 16, vocab_max=100_000,
                       batch=301)
    raise TypeError(cfg)


# ---------------------------------------------------------------------------
# per-task batch generators
# ---------------------------------------------------------------------------
@dataclass
class MFBatch:
    row: np.ndarray   # int32 [B]
    col: np.ndarray   # int32 [B]
    val: np.ndarray   # float32 [B]


class MFWorkload:
    TAG = 101

    def __init__(self, cfg: MFConfig):
        self.cfg = cfg
        self.zipf = Zipf(cfg.n_cols, cfg.zipf_s, cfg.seed, self.TAG + 1)
        self.row_zipf = None if cfg.row_zipf_s is None else Zipf(cfg.n_rows, cfg.row_zipf_s, cfg.seed, self.TAG + 4)
        self._data = None
        if cfg.fixed_dataset:
            rng = _rng(cfg.seed, self.TAG, 0)
            self._data = self._draw(rng, cfg.nnz)
        if cfg.visit == "column":
            # each column holds its expected share of the nnz entries (largest
            # remainders round the shares to whole entries); columns are
            # visited in a seeded random order
            share = cfg.nnz * self.zipf.pmf
            cnt = np.floor(share).astype(np.int64)
            extra = cfg.nnz - int(cnt.sum())
            cnt[np.argsort(-(share - cnt), kind="stable")[:extra]] += 1
            counts = np.zeros(cfg.n_cols, np.int64)
            counts[self.zipf.perm] = cnt                 # by column id
            self.col_order = _rng(cfg.seed, self.TAG + 3, 0).permutation(cfg.n_cols).astype(np.int64)
            self.col_end = np.cumsum(counts[self.col_order])
        elif cfg.visit != "random":
            raise ValueError(f"unknown MF visiting order {cfg.visit!r}")

    def _draw(self, rng, b):
        if self.row_zipf is None:
            row = rng.integers(0, self.cfg.n_rows, b, dtype=np.int64).astype(np.int32)
        else:
            row = self.row_zipf.sample(rng, b).astype(np.int32)
        col = self.zipf.sample(rng, b).astype(np.int32)
        val = rng.standard_normal(b, dtype=np.float32)
        return MFBatch(row, col, val)

    def _column_batch(self, step: int) -> MFBatch:
        """Entries [lo, hi) of the column-ordered epoch: the columns that
        cover that span, each for its overlap; rows uniform, values N(0,1)."""
        cfg = self.cfg
        s = step % cfg.steps_per_epoch
        lo, hi = s * cfg.batch, min(cfg.nnz, (s + 1) * cfg.batch)
        i0 = int(np.searchsorted(self.col_end, lo, side="right"))
        i1 = int(np.searchsorted(self.col_end, hi - 1, side="right"))
        starts = np.concatenate([[0], self.col_end[:-1]])
        a = np.maximum(starts[i0:i1 + 1], lo)
        b = np.minimum(self.col_end[i0:i1 + 1], hi)
        col = np.repeat(self.col_order[i0:i1 + 1], b - a).astype(np.int32)
        rng = _rng(cfg.seed, self.TAG, step + 1)
        row = rng.integers(0, cfg.n_rows, hi - lo, dtype=np.int64).astype(np.int32)
        val = rng.standard_normal(hi - lo, dtype=np.float32)
        return MFBatch(row, col, val)

    def batch(self, step: int) -> MFBatch:
        cfg = self.cfg
        if cfg.visit == "column":
            return self._column_batch(step)
        if self._data is not None:
            lo = (step % cfg.steps_per_epoch) * cfg.batch
            hi = min(cfg.nnz, lo + cfg.batch)
            d = self._data
            return MFBatch(d.row[lo:hi].copy(), d.col[lo:hi].copy(), d.val[lo:hi].copy())
        return self._draw(_rng(cfg.seed, self.TAG, step + 1), cfg.batch)

    def init_table(self) -> np.ndarray:
        return normal_table(self.cfg.num_keys, self.cfg.dim, self.cfg.init_std, self.cfg.seed, self.TAG + 2)

    def hot_row_batch(self, counts, n_plain: int, step: int = 0) -> MFBatch:
        """A batch whose row keys include len(counts) distinct rows repeated
        counts[i] times each, mixed in random order with n_plain entries of
        the configuration's own distribution; columns and values as usual."""
        cfg = self.cfg
        rng = _rng(cfg.seed, self.TAG + 5, step)
        hot = rng.choice(cfg.n_rows, len(counts), replace=False)
        plain = self._draw(rng, n_plain)
        clash = np.isin(plain.row, hot)
        while clash.any():   # the hot rows keep exactly their counts
            plain.row[clash] = rng.integers(0, cfg.n_rows, int(clash.sum()), dtype=np.int64)
            clash = np.isin(plain.row, hot)
        n_hot = int(np.sum(counts))
        row = np.concatenate([np.repeat(hot, counts), plain.row]).astype(np.int32)
        col = np.concatenate([self.zipf.sample(rng, n_hot).astype(np.int32), plain.col])
        val = np.concatenate([rng.standard_normal(n_hot, dtype=np.float32), plain.val])
        order = rng.permutation(row.size)
        return MFBatch(row[order], col[order], val[order])


@dataclass
class KGEBatch:
    head: np.ndarray   # int32 [B]
    rel: np.ndarray    # int32 [B]
    tail: np.ndarray   # int32 [B]
    neg: np.ndarray    # int32 [B, n_neg]: first n_head_neg replace the head, the rest the tail


class KGEWorkload:
    TAG = 202

    def __init__(self, cfg: KGEConfig):
        self.cfg = cfg
        self.zipf = Zipf(cfg.n_ent, cfg.zipf_s, cfg.seed, self.TAG + 1)

    def batch(self, step: int) -> KGEBatch:
        cfg = self.cfg
        steps = (cfg.n_triples + cfg.batch - 1) // cfg.batch
        s = step % steps
        b = min(cfg.batch, cfg.n_triples - s * cfg.batch)
        rng = _rng(cfg.seed, self.TAG, step + 1)
        head = self.zipf.sample(rng, b).astype(np.int32)
        tail = self.zipf.sample(rng, b).astype(np.int32)
        rel = rng.integers(0, cfg.n_rel, b, dtype=np.int64).astype(np.int32)
        neg = rng.integers(0, cfg.n_ent, (b, cfg.n_neg), dtype=np.int64).astype(np.int32)
        return KGEBatch(head, rel, tail, neg)

    def init_table(self) -> np.ndarray:
        return normal_table(self.cfg.num_keys, self.cfg.dim, self.cfg.init_std, self.cfg.seed, self.TAG + 2)

    def hot_row_batch(self, counts, n_plain: int, step: int = 0) -> MFBatch:
        """A batch whose row keys include len(counts) distinct rows repeated
        counts[i] times each, mixed in random order with n_plain entries of
        the configuration's own distribution; columns and values as usual."""
        cfg = self.cfg
        rng = _rng(cfg.seed, self.TAG + 5, step)
        hot = rng.choice(cfg.n_rows, len(counts), replace=False)
        plain = self._draw(rng, n_plain)
        clash = np.isin(plain.row, hot)
        while clash.any():   # the hot rows keep exactly their counts
            plain.row[clash] = rng.integers(0, cfg.n_rows, int(clash.sum()), dtype=np.int64)
            clash = np.isin(plain.row, hot)
        n_hot = int(np.sum(counts))
        row = np.concatenate([np.repeat(hot, counts), plain.row]).astype(np.int32)
        col = np.concatenate([self.zipf.sample(rng, n_hot).astype(np.int32), plain.col])
        val = np.concatenate([rng.standard_normal(n_hot, dtype=np.float32), plain.val])
        order = rng.permutation(row.size)
        return MFBatch(row[order], col[order], val[order])


@dataclass
class SGNSBatch:
    centre: np.ndarray  # int32 [B]            word ids in [0, V)
    ctx: np.ndarray     # int32 [B, 2*window]  word ids, -1 where the window leaves the stream
    neg: np.ndarray     # int32 [B, 2*window, n_neg] word ids, -1 where ctx is -1


class SGNSWorkload:
    TAG = 303
    # counter ranges of the hash draws: tokens at the position itself, the
    # subsampling and window draws 2^40 and 2^41 positions further on
    _SUBSAMPLE_STREAM = np.uint64(1 << 40)
    _WINDOW_STREAM = np.uint64(1 << 41)

    def __init__(self, cfg: SGNSConfig):
        self.cfg = cfg
        self.zipf = Zipf(cfg.vocab, cfg.zipf_s, cfg.seed, self.TAG + 1)
        # negatives are drawn over the same word ids with frequency rank^-0.75
        self.noise = Zipf(cfg.vocab, cfg.zipf_s * cfg.neg_power, cfg.seed, self.TAG + 1)
        self.noise.perm = self.zipf.perm
        self._key = np.uint64((cfg.seed * 0x632BE59BD9B4E019 + self.TAG) & 0xFFFFFFFFFFFFFFFF)

    def tokens(self, pos: np.ndarray) -> np.ndarray:
        """Token id at each stream position (-1 outside [0, n_tokens))."""
        pos = np.asarray(pos, dtype=np.int64)
        ok = (pos >= 0) & (pos < self.cfg.n_tokens)
        u = _hash_uniform(pos.astype(np.uint64) ^ self._key)
        t = self.zipf.ids_from_uniform(u).astype(np.int32)
        return np.where(ok, t, -1).astype(np.int32)

    def offsets(self) -> np.ndarray:
        w = self.cfg.window
        return np.array([d for d in range(-w, w + 1) if d != 0], dtype=np.int64)

    def kept(self, pos: np.ndarray) -> np.ndarray:
        """Whether the token at each stream position survives subsampling:
        Mikolov et al.'s rule discards word w with probability
        1 - sqrt(t / f(w)), f(w) taken as w's probability in the stream."""
        pos = np.asarray(pos, dtype=np.int64)
        ok = (pos >= 0) & (pos < self.cfg.n_tokens)
        if self.cfg.subsample <= 0:
            return ok
        u = _hash_uniform(pos.astype(np.uint64) ^ self._key)
        f = self.zipf.pmf[self.zipf.ranks(u)]
        keep = np.minimum(1.0, np.sqrt(self.cfg.subsample / f))
        v = _hash_uniform((pos.astype(np.uint64) + self._SUBSAMPLE_STREAM) ^ self._key)
        return ok & (v < keep)

    def _w2v_batch(self, step: int) -> SGNSBatch:
        """The kept tokens of stream span [lo, lo + batch) as centres; each
        centre's context is the nearest kept tokens on either side, up to its
        window b (b uniform in 1..window when the window is dynamic)."""
        cfg = self.cfg
        w = cfg.window
        steps = (cfg.n_tokens + cfg.batch - 1) // cfg.batch
        lo = (step % steps) * cfg.batch
        hi = min(cfg.n_tokens, lo + cfg.batch)
        margin = 8 * w + 64
        while True:
            pos = np.arange(lo - margin, hi + margin, dtype=np.int64)
            kp = pos[self.kept(pos)]
            c0 = int(np.searchsorted(kp, lo))
            c1 = int(np.searchsorted(kp, hi))
            inside = (pos[0] < 0 or c0 >= w) and (pos[-1] >= cfg.n_tokens or len(kp) - c1 >= w)
            if inside:
                break
            margin *= 2
        B = c1 - c0
        centre_pos = kp[c0:c1]
        idx = np.arange(c0, c1)[:, None] + self.offsets()[None, :]
        valid = (idx >= 0) & (idx < len(kp))
        ctx_pos = np.where(valid, kp[np.clip(idx, 0, max(len(kp) - 1, 0))], -1)
        if cfg.dynamic_window:
            u = _hash_uniform((centre_pos.astype(np.uint64) + self._WINDOW_STREAM) ^ self._key)
            b = 1 + np.minimum((u * w).astype(np.int64), w - 1)
            valid &= np.abs(self.offsets())[None, :] <= b[:, None]
        centre = self.tokens(centre_pos)
        ctx = np.where(valid, self.tokens(np.where(valid, ctx_pos, -1)), -1).astype(np.int32)
        rng = _rng(cfg.seed, self.TAG, step + 1)
        neg = self.noise.sample(rng, (B, 2 * w, cfg.n_neg)).astype(np.int32)
        neg = np.where(ctx[:, :, None] < 0, -1, neg).astype(np.int32)
        return SGNSBatch(centre, ctx, neg)

    def batch(self, step: int) -> SGNSBatch:
        cfg = self.cfg
        if cfg.subsample > 0 or cfg.dynamic_window:
            return self._w2v_batch(step)
        steps = (cfg.n_tokens + cfg.batch - 1) // cfg.batch
        s = step % steps
        lo = s * cfg.batch
        b = min(cfg.batch, cfg.n_tokens - lo)
        pos = lo + np.arange(b, dtype=np.int64)
        centre = self.tokens(pos)
        ctx = self.tokens(pos[:, None] + self.offsets()[None, :])
        rng = _rng(cfg.seed, self.TAG, step + 1)
        neg = self.noise.sample(rng, (b, 2 * cfg.window, cfg.n_neg)).astype(np.int32)
        neg = np.where(ctx[:, :, None] < 0, -1, neg).astype(np.int32)
        return SGNSBatch(centre, ctx, neg)

    def init_table(self) -> np.ndarray:
        """word2vec's convention: input vectors U(-0.5/d, 0.5/d), output vectors 0."""
        cfg = self.cfg
        w = np.zeros((2 * cfg.vocab, cfg.dim), dtype=np.float32)
        w[: cfg.vocab] = uniform_table(cfg.vocab, cfg.dim, -0.5 / cfg.dim, 0.5 / cfg.dim,
                                       cfg.seed, self.TAG + 2)
        return w


@dataclass
class CTRBatch:
    keys: np.ndarray    # int64 [B, F] table rows
    label: np.ndarray   # float32 [B] in {0, 1}


class CTRWorkload:
    TAG = 404

    def __init__(self, cfg: CTRConfig):
        self.cfg = cfg
        self.fields = [Zipf(v, cfg.zipf_s, cfg.seed, self.TAG + 10 + f, permute=False)
                       for f, v in enumerate(cfg.vocab_sizes())]
        self._key = np.uint64((cfg.seed * 0x9E3779B97F4A7C15 + self.TAG) & 0xFFFFFFFFFFFFFFFF)

    def hash_key(self, f: int, rank: np.ndarray) -> np.ndarray:
        x = (np.uint64(f) << np.uint64(40)) | np.asarray(rank, dtype=np.uint64)
        return (splitmix64(x ^ self._key) % np.uint64(self.cfg.table_rows)).astype(np.int64)

    def batch(self, step: int) -> CTRBatch:
        cfg = self.cfg
        rng = _rng(cfg.seed, self.TAG, step + 1)
        keys = np.empty((cfg.batch, cfg.n_fields), dtype=np.int64)
        for f, z in enumerate(self.fields):
            keys[:, f] = self.hash_key(f, z.ranks(rng.random(cfg.batch)))
        label = (rng.random(cfg.batch) < cfg.p_click).astype(np.float32)
        return CTRBatch(keys, label)

    def init_table(self) -> np.ndarray:
        W = normal_table(self.cfg.num_keys, self.cfg.dim, self.cfg.init_std, self.cfg.seed, self.TAG + 2)
        if self.cfg.deep:
            W[:, self.cfg.emb_dim:] = 0.0      # wide weights start at zero; padding stays zero
        return W

    def init_dense(self) -> np.ndarray:
        """Wide & Deep dense buffer: each weight matrix (and the output
        vector) uniform in +-1/sqrt(fan_in), biases zero, in the layout
        [W_1, b_1, ..., W_L, b_L, w, c]."""
        cfg = self.cfg
        out = np.zeros(cfg.dense_size, np.float32)
        rng = _rng(cfg.seed, self.TAG + 5, 0)
        off, fan = 0, cfg.n_fields * cfg.emb_dim
        for h in cfg.deep:
            out[off:off + fan * h] = rng.uniform(-1, 1, fan * h) / np.sqrt(fan)
            off += fan * h + h
            fan = h
        out[off:off + fan] = rng.uniform(-1, 1, fan) / np.sqrt(fan)
        return out


def workload(cfg):
    if isinstance(cfg, MFConfig):
        return MFWorkload(cfg)
    if isinstance(cfg, KGEConfig):
        return KGEWorkload(cfg)
    if isinstance(cfg, SGNSConfig):
        return SGNSWorkload(cfg)
    if isinstance(cfg, CTRConfig):
        return CTRWorkload(cfg)
    raise TypeError(cfg)


def random_push(num_keys: int, n: int, dim: int, seed: int, zipf_s: float | None = None,
                grad_std: float = 1.0):
    """Keys (int64) and gradient rows (float32) for a bare push: keys uniform
    or Zipf over [0, num_keys)."""
    rng = _rng(seed, 505, n)
    if zipf_s is None:
        keys = rng.integers(0, num_keys, n, dtype=np.int64)
    else:
        keys = Zipf(num_keys, zipf_s, seed, 506).sample(rng, n).astype(np.int64)
    grads = (rng.standard_normal((n, dim), dtype=np.float32) * np.float32(grad_std))
    return keys, grads
