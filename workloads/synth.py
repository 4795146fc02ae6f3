"""Seeded synthetic inputs for the f-gram embedding path.

This module only draws inputs: token streams, f-gram sets with their ids, query
matrices and embedding-row tables.  It holds none of the lookup or gather
arithmetic, so both the GPU path and the CPU oracle can be fed from it without
sharing code with each other.

Stand-ins for the paper's data (its corpora, tokenizers and trained f-gram
tables are not available):

* tokens are bounded Zipf(1.1) over ranks 1..V, token id = rank - 1;
* an f-gram set is drawn with lengths uniform in [min_len, max_len] and Zipf
  tokens, duplicates rejected (first occurrence kept) until it holds N
  distinct f-grams, which get ids V, V+1, ... in draw order;
* a query row is filled left to right: with probability p a uniformly chosen
  f-gram is appended, otherwise one Zipf noise token; p is set so that the
  expected fraction of positions inside planted f-grams equals the requested
  coverage;
* the row table E has one row per id (token rows 0..V-1, then f-gram rows)
  and its elements are a counter-based function of (seed, element index), so
  any subset of rows can be regenerated bit-identically on any device.

Shapes follow the paper's inference study (Section 4.3: d = 2048, 16-bit,
10M f-grams, K = 5) and its GPT-2 scale d_model = 1024 (Appendix, WebText
model table).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

ZIPF_S = 1.1
TOKEN_BITS = 16  # tokens must fit 16 bits for the GPU key packing


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    V: int                 # token vocabulary size
    n_fgrams: int          # |V_fgram|
    min_len: int
    max_len: int           # K, the longest f-gram length in the set
    B: int                 # sequences
    T: int                 # tokens per sequence (decode: steps)
    coverage: float        # target fraction of positions inside planted f-grams
    max_n: int             # lookup window
    d: int                 # row width in elements
    dtype: str             # "f32" or "bf16"
    std: float             # row-element standard deviation
    placement: str         # "hbm" or "host"
    decode: bool = False   # one token per sequence per step
    seed: int = 0

    @property
    def n_rows(self) -> int:
        return self.V + self.n_fgrams

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def row_bytes(self) -> int:
        return self.d * self.elem_bytes

    @property
    def n_tok(self) -> int:
        return self.B * self.T

    def gather_bytes(self) -> int:
        """Algorithmic bytes of one gather: rows read + rows written + ids."""
        return self.n_tok * (2 * self.row_bytes + 4)


CONFIGS: Dict[str, Config] = {
    "tiny": Config("tiny", V=1000, n_fgrams=10_000, min_len=2, max_len=3, B=16,
                   T=512, coverage=0.5, max_n=3, d=64, dtype="f32", std=1.0,
                   placement="hbm", seed=1000),
    "c2_1m": Config("c2_1m", V=32768, n_fgrams=1_000_000, min_len=2, max_len=3,
                    B=64, T=2048, coverage=0.5, max_n=3, d=1024, dtype="bf16",
                    std=0.02, placement="hbm", seed=1001),
    "c3_10m_k5": Config("c3_10m_k5", V=32768, n_fgrams=10_000_000, min_len=2,
                        max_len=5, B=32, T=4096, coverage=0.6, max_n=5, d=2048,
                        dtype="bf16", std=0.02, placement="hbm", seed=1002),
    # Off-accelerator rows: 15M f-grams (61.6 GB of rows) is the largest round
    # size whose table fits within a 64 GiB limit on pinned host memory.
    "c4_host": Config("c4_host", V=32768, n_fgrams=15_000_000, min_len=2,
                      max_len=3, B=64, T=2048, coverage=0.5, max_n=3, d=2048,
                      dtype="bf16", std=0.02, placement="host", seed=1003),
    "c5_decode": Config("c5_decode", V=32768, n_fgrams=10_000_000, min_len=2,
                        max_len=3, B=256, T=1024, coverage=0.5, max_n=3,
                        d=2048, dtype="bf16", std=0.02, placement="hbm",
                        decode=True, seed=1004),
}


def scaled(cfg: Config, **kw) -> Config:
    """A copy of ``cfg`` with some fields replaced (smaller parity cases)."""
    return dataclasses.replace(cfg, **kw)


# ---------------------------------------------------------------- tokens ----

def zipf_cdf(V: int, s: float = ZIPF_S) -> np.ndarray:
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    c /= c[-1]
    return c


_GUIDE_BITS = 21
_guides: dict = {}


def _guide(cdf: np.ndarray) -> np.ndarray:
    """guide[b] = smallest rank k with cdf[k] > b / 2^21 (an index for the search)."""
    key = (len(cdf), float(cdf[0]))
    g = _guides.get(key)
    if g is None:
        M = 1 << _GUIDE_BITS
        g = np.searchsorted(cdf, np.arange(M, dtype=np.float64) / M, side="right")
        _guides[key] = g
    return g


def zipf_tokens(rng: np.random.Generator, cdf: np.ndarray, size) -> np.ndarray:
    """Inverse-CDF draw of bounded Zipf ranks, returned as token ids (rank-1).

    The result is the smallest k with cdf[k] > u, found from a guide table
    and a short forward scan (the same value as a binary search).
    """
    u = rng.random(size).reshape(-1)
    k = _guide(cdf)[(u * (1 << _GUIDE_BITS)).astype(np.int64)]
    last = len(cdf) - 1
    todo = np.nonzero(cdf[np.minimum(k, last)] <= u)[0]
    while todo.size:
        k[todo] += 1
        todo = todo[(k[todo] < last) & (cdf[np.minimum(k[todo], last)] <= u[todo])]
    return np.minimum(k, last).astype(np.int32).reshape(size)


# --------------------------------------------------------------- f-grams ----

def _fingerprint(rows: np.ndarray, lens: np.ndarray) -> np.ndarray:
    """64-bit fingerprint of (length, tokens) for duplicate rejection.

    Equal f-grams always share a fingerprint; two different f-grams share one
    with negligible probability, and then one of them is merely dropped, so
    the kept set is always a set of distinct f-grams.
    """
    with np.errstate(over="ignore"):
        h = lens.astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)
        for j in range(rows.shape[1]):
            h ^= (rows[:, j].astype(np.int64) + 1).astype(np.uint64)
            h *= np.uint64(0xFF51AFD7ED558CCD)
            h ^= h >> np.uint64(29)
        h *= np.uint64(0xC4CEB9FE1A85EC53)
        h ^= h >> np.uint64(32)
    return h


def make_fgrams(rng: np.random.Generator, cdf: np.ndarray, n: int,
                min_len: int, max_len: int):
    """Draw ``n`` distinct f-grams (first occurrence kept, draw order preserved).

    Returns (fgrams [n, max_len] int32 padded with -1, lengths [n] int32).
    """
    rows = np.empty((0, max_len), dtype=np.int32)
    lens = np.empty(0, dtype=np.int32)
    fps = np.empty(0, dtype=np.uint64)
    batch = max(1024, int(n * 1.1))
    rounds = 0
    while len(lens) < n:
        rounds += 1
        if rounds > 200:
            raise ValueError(f"cannot draw {n} distinct f-grams of length "
                             f"{min_len}..{max_len} from this vocabulary")
        bl = rng.integers(min_len, max_len + 1, size=batch).astype(np.int32)
        bt = zipf_tokens(rng, cdf, (batch, max_len))
        bt[np.arange(max_len)[None, :] >= bl[:, None]] = -1
        have = len(lens)
        allfp = np.concatenate([fps, _fingerprint(bt, bl)])
        _, first = np.unique(allfp, return_index=True)  # stable: earliest draw wins
        first.sort()
        new = first[first >= have] - have
        rows = np.concatenate([rows, bt[new]])
        lens = np.concatenate([lens, bl[new]])
        fps = np.concatenate([fps, allfp[have:][new]])
        deficit = n - len(lens)
        if deficit > 0:
            rate = max(len(new) / batch, 0.01)
            batch = max(1024, int(deficit / rate * 1.1))
    return np.ascontiguousarray(rows[:n]), np.ascontiguousarray(lens[:n])


# --------------------------------------------------------------- queries ----

def plant_probability(coverage: float, mean_len: float) -> float:
    """p such that p*L / (p*L + 1 - p) equals the coverage."""
    if coverage <= 0:
        return 0.0
    return coverage / (mean_len * (1.0 - coverage) + coverage)


def make_queries(rng: np.random.Generator, cdf: np.ndarray, fgrams: np.ndarray,
                 lengths: np.ndarray, B: int, T: int, coverage: float):
    """Query matrix [B, T] int32 and a planted mask [B, T] bool.

    Each row is filled left to right with planted f-grams (probability p) and
    single Zipf noise tokens; the last segment is cut at T.
    """
    X = np.empty((B, T), dtype=np.int32)
    planted = np.zeros((B, T), dtype=bool)
    ends_planted = np.zeros((B, T), dtype=np.int8)  # length of a planted f-gram ending here
    if B == 0 or T == 0:
        return X, planted, ends_planted
    n = len(lengths)
    mean_len = float(lengths.mean()) if n else 1.0
    p = plant_probability(coverage, mean_len) if n else 0.0
    for b in range(B):
        kind = rng.random(T) < p
        choice = rng.integers(0, max(n, 1), size=T)
        noise = zipf_tokens(rng, cdf, T)
        seglen = np.where(kind, lengths[choice] if n else 1, 1).astype(np.int64)
        ends = np.cumsum(seglen)
        nseg = int(np.searchsorted(ends, T, side="left")) + 1
        nseg = min(nseg, T)
        seglen, kind, choice, noise = seglen[:nseg], kind[:nseg], choice[:nseg], noise[:nseg]
        starts = np.concatenate([[0], np.cumsum(seglen)[:-1]])
        seg_of = np.repeat(np.arange(nseg), seglen)
        off = np.arange(len(seg_of)) - starts[seg_of]
        tok = np.where(kind[seg_of], fgrams[choice[seg_of], np.minimum(off, fgrams.shape[1] - 1)] if n else 0,
                       noise[seg_of])
        X[b] = tok[:T]
        planted[b] = kind[seg_of][:T]
        full = kind & (starts + seglen <= T)
        last = (starts + seglen - 1)[full]
        ends_planted[b, last] = seglen[full]
    return X, planted, ends_planted


@dataclasses.dataclass
class Workload:
    cfg: Config
    fgrams: np.ndarray      # [N, max_len] int32, padded with -1
    lengths: np.ndarray     # [N] int32
    ids: np.ndarray         # [N] int32
    tokens: np.ndarray      # [B, T] int32
    planted: np.ndarray     # [B, T] bool
    planted_end: np.ndarray  # [B, T] int8: length of a whole planted f-gram ending here


def make_workload(cfg: Config, seed: Optional[int] = None) -> Workload:
    seed = cfg.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    cdf = zipf_cdf(cfg.V)
    if cfg.n_fgrams:
        fg, ln = make_fgrams(rng, cdf, cfg.n_fgrams, cfg.min_len, cfg.max_len)
    else:
        fg = np.full((0, cfg.max_len), -1, dtype=np.int32)
        ln = np.zeros(0, dtype=np.int32)
    ids = (cfg.V + np.arange(len(ln))).astype(np.int32)
    X, planted, pend = make_queries(rng, cdf, fg, ln, cfg.B, cfg.T, cfg.coverage)
    return Workload(cfg, fg, ln, ids, X, planted, pend)


# ----------------------------------------------------------------- table ----
# Counter-based element generator.  Every element is a pure function of
# (seed, row * d + col) built from 32-bit integer mixing kept inside int64
# range, an Irwin-Hall sum of four 16-bit uniforms, one exact int->float
# conversion, one float32 multiply and (for bf16) one round-to-nearest-even
# conversion.  All of these are exact or correctly rounded, so the CPU and the
# GPU produce the same bits.

_M32 = 0xFFFFFFFF
_MIX = 0x45D9F3B          # 32-bit multiplicative mixing constant
_IH_STD = 65536.0 * math.sqrt(4.0 / 12.0)  # std of the sum of four U[0, 65536)


def _seed_words(seed: int):
    x = (seed * 0x9E3779B97F4A7C15 + 0x632BE59BD9B4E019) & ((1 << 64) - 1)
    out = []
    for _ in range(3):
        x = (x + 0x9E3779B97F4A7C15) & ((1 << 64) - 1)
        z = x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & ((1 << 64) - 1)
        out.append((z ^ (z >> 31)) & _M32)
    return out


def _mix32(x):
    x = (((x >> 16) ^ x) * _MIX) & _M32
    x = (((x >> 16) ^ x) * _MIX) & _M32
    return (x >> 16) ^ x


def table_values(seed: int, elem_index, std: float, dtype: str):
    """Elements for the given flat indices (an int64 torch tensor, any device)."""
    import torch
    s1, s2, s3 = _seed_words(seed)
    e = elem_index
    h2 = _mix32(_mix32((e & _M32) ^ s1) ^ (e >> 32) ^ s2)
    h3 = _mix32(h2 ^ s3)
    acc = (h2 & 0xFFFF) + (h2 >> 16) + (h3 & 0xFFFF) + (h3 >> 16) - 131070
    scale = torch.tensor(std / _IH_STD, dtype=torch.float32, device=e.device)
    v = acc.to(torch.float32) * scale
    if dtype == "bf16":
        return v.to(torch.bfloat16)
    return v


def table_rows(cfg: Config, rows, device="cpu", seed: Optional[int] = None):
    """Rows ``rows`` (int sequence or int64 tensor) of the table, [len, d]."""
    import torch
    seed = cfg.seed if seed is None else seed
    r = torch.as_tensor(rows, dtype=torch.int64, device=device).reshape(-1, 1)
    cols = torch.arange(cfg.d, dtype=torch.int64, device=device).reshape(1, -1)
    return table_values(seed, r * cfg.d + cols, cfg.std, cfg.dtype)


def fill_table(cfg: Config, out, seed: Optional[int] = None, chunk_elems: int = 1 << 27,
               row0: int = 0):
    """Fill a preallocated [n, d] tensor (any device) with rows row0 .. row0+n-1."""
    import torch
    seed = cfg.seed if seed is None else seed
    flat = out.view(-1)
    total = flat.numel()
    dev = out.device
    e0 = row0 * cfg.d
    for s in range(0, total, chunk_elems):
        e = torch.arange(e0 + s, e0 + min(total, s + chunk_elems), dtype=torch.int64, device=dev)
        flat[s:s + e.numel()].copy_(table_values(seed, e, cfg.std, cfg.dtype))
    return out


def torch_dtype(cfg: Config):
    import torch
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def match_stats(lens: np.ndarray, max_n: int) -> dict:
    """Histogram of matched lengths (1 = no f-gram) and the mean match length."""
    h = np.bincount(lens.reshape(-1).astype(np.int64), minlength=max(max_n, 1) + 1)
    tot = max(int(lens.size), 1)
    return {"hist": {int(k): int(v) for k, v in enumerate(h) if k >= 1 and v},
            "matched_frac": float((lens >= 2).sum()) / tot,
            "mean_len": float(lens.astype(np.float64).mean()) if lens.size else 0.0}


def query_batches(w: Workload, n: int):
    """``n`` query matrices of the workload's shape: the workload's own first,
    then fresh draws from the same f-gram set (rotating batches keep one
    step's rows from being served out of the caches filled by the last)."""
    out = [w.tokens]
    cdf = zipf_cdf(w.cfg.V)
    for k in range(1, n):
        rng = np.random.Generator(np.random.PCG64([w.cfg.seed, k]))
        X, _, _ = make_queries(rng, cdf, w.fgrams, w.lengths, w.cfg.B, w.cfg.T, w.cfg.coverage)
        out.append(X)
    return out
