"""Seeded synthetic inputs shaped like the paper's split LM-head workload.

The paper's setting (Section 7.3) is a 7B-class decoder with hidden size
D=4096 and a vocabulary of about 150 000 ids, a language subset keeping
30-40% of the vocabulary (100% in mixed mode), bf16 cloud weights, int8
payloads and speculative draft lengths N=2..8 (Section 7.3, Table 7).  Its
prompt workload is not available, so every input here is drawn from fixed
seeds:

* h    : standard normal fp32, rounded to bf16 (round-to-nearest-even).
* W    : standard normal / sqrt(d) fp32, rounded to bf16, stored vocab-major
         [V, d] and split into contiguous W_end [V, d_end] and
         W_cloud [V, d - d_end] (eq. 10: the endpoint owns the first d_end
         hidden dimensions).
* fp8  : the cloud slice re-encoded as OCP e4m3 codes with one fp32 scale per
         vocabulary row (row amax / 448), from the bf16 values.
* S    : sorted unique vocabulary ids (the language subset V_l, Section 5.4).
* drafts: per (session, draft position) a fair coin picks either a reference
         token for that row or a uniform id from S.

Config i draws its streams from ``numpy.random.SeedSequence(i).spawn(5)`` in
the order (h, W, subset, drafts, aux).
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = [
    "Config",
    "Workload",
    "CONFIGS",
    "make_workload",
    "with_subset",
    "make_drafts",
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "fp8_encode_rows",
    "scale_rows_bf16",
    "plant_masked_supertoken",
]

_W_CHUNK = 8192  # rows of W drawn per call; fixed so the stream is reproducible


@dataclass(frozen=True)
class Config:
    """Shape and mode of one split-head workload."""

    name: str
    seed_index: int
    d: int
    d_end: int
    vocab: int
    n_sub: int                     # |S|; equal to vocab for the full vocabulary
    subset_kind: str               # "perm" | "block+scatter" | "choice" | "full"
    sessions: int
    rows_per_session: int          # k + 1
    wtype: str = "bf16"            # "bf16" | "fp8"
    mode: str = "greedy"           # "greedy" | "sample"
    clip_c: float = 30.0
    temperature: float = 1.0
    top_p: float = 1.0
    philox_seed: int = 0
    block: int = 0                 # length of the contiguous block for "block+scatter"
    with_bias: bool = False

    @property
    def d_cloud(self) -> int:
        return self.d - self.d_end

    @property
    def M(self) -> int:
        return self.sessions * self.rows_per_session

    @property
    def k(self) -> int:
        return self.rows_per_session - 1

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five workloads of the split-head benchmark.  Shapes follow the paper's
# hidden sizes, vocabulary sizes, language-subset fractions and draft lengths.
CONFIGS = {
    "tiny": Config("tiny", 0, d=512, d_end=64, vocab=8192, n_sub=4096,
                   subset_kind="perm", sessions=1, rows_per_session=3),
    "decode": Config("decode", 1, d=4096, d_end=256, vocab=128256, n_sub=49152,
                     subset_kind="block+scatter", block=32768,
                     sessions=1, rows_per_session=5),
    "batched": Config("batched", 2, d=4096, d_end=512, vocab=152064, n_sub=60000,
                      subset_kind="choice", sessions=64, rows_per_session=5),
    "dense_full": Config("dense_full", 3, d=8192, d_end=512, vocab=128256, n_sub=128256,
                         subset_kind="full", sessions=256, rows_per_session=8),
    "dense_sub": Config("dense_sub", 3, d=8192, d_end=512, vocab=128256, n_sub=32768,
                        subset_kind="choice", sessions=256, rows_per_session=8),
    "sample_fp8": Config("sample_fp8", 4, d=5120, d_end=320, vocab=152064, n_sub=65536,
                         subset_kind="choice", sessions=128, rows_per_session=5,
                         wtype="fp8", mode="sample", temperature=0.7, top_p=0.9,
                         philox_seed=0x5EED_2607_1309_3ACE),
}


@dataclass
class Workload:
    cfg: Config
    h_bits: np.ndarray                       # uint16 [M, d]  (bf16 bit patterns)
    w_end_bits: np.ndarray                   # uint16 [V, d_end]
    w_cloud_bits: Optional[np.ndarray]       # uint16 [V, d_cloud] when wtype == "bf16"
    w_cloud_codes: Optional[np.ndarray]      # uint8  [V, d_cloud] when wtype == "fp8"
    w_cloud_scale: Optional[np.ndarray]      # fp32   [V]          when wtype == "fp8"
    bias: Optional[np.ndarray]               # fp32   [V] or None
    subset: np.ndarray                       # int32  [n_sub], strictly ascending
    full_vocab: bool
    rngs: dict = field(default_factory=dict)


# ---------------------------------------------------------------------------
# bit-level input encodings
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to bf16 (nearest, ties to even); return bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def fp8_encode_rows(w_bits: np.ndarray):
    """Re-encode bf16 rows as OCP e4m3 codes with one fp32 scale per row.

    scale_v = max_i |w[v, i]| / 448 so that the largest element lands on the
    format's largest finite value; codes = e4m3(w / scale_v) rounded to
    nearest even (torch's conversion).  Returns (codes uint8, scale fp32).
    """
    import torch

    codes = np.empty(w_bits.shape, dtype=np.uint8)
    scale = np.empty(w_bits.shape[0], dtype=np.float32)
    for r0 in range(0, w_bits.shape[0], _W_CHUNK):
        w = bf16_bits_to_f32(w_bits[r0:r0 + _W_CHUNK])
        amax = np.abs(w).max(axis=1)
        s = (amax / np.float32(448.0)).astype(np.float32)
        s[s == 0] = np.float32(1.0)
        x = torch.from_numpy(np.ascontiguousarray(w / s[:, None]))
        codes[r0:r0 + _W_CHUNK] = x.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        scale[r0:r0 + _W_CHUNK] = s
    return codes, scale


# ---------------------------------------------------------------------------
# workload generation
# ---------------------------------------------------------------------------

def _streams(seed_index: int):
    names = ("h", "w", "subset", "drafts", "aux")
    seqs = np.random.SeedSequence(seed_index).spawn(len(names))
    return {n: np.random.default_rng(s) for n, s in zip(names, seqs)}


def _draw_subset(cfg: Config, rng: np.random.Generator) -> np.ndarray:
    V, n = cfg.vocab, cfg.n_sub
    if cfg.subset_kind == "full":
        ids = np.arange(V, dtype=np.int64)
    elif cfg.subset_kind == "perm":
        ids = rng.permutation(V)[:n]
    elif cfg.subset_kind == "choice":
        ids = rng.choice(V, size=n, replace=False)
    elif cfg.subset_kind == "block+scatter":
        b = cfg.block
        b0 = int(rng.integers(0, V - b + 1))
        rest = np.concatenate([np.arange(0, b0), np.arange(b0 + b, V)])
        extra = rng.choice(rest, size=n - b, replace=False)
        ids = np.concatenate([np.arange(b0, b0 + b), extra])
    else:
        raise ValueError(f"unknown subset kind {cfg.subset_kind!r}")
    return np.sort(ids).astype(np.int32)


def make_workload(cfg: Config, h_rows: Optional[int] = None) -> Workload:
    """Draw every input of ``cfg`` from its fixed seed streams."""
    r = _streams(cfg.seed_index)
    M = cfg.M if h_rows is None else h_rows
    h = r["h"].standard_normal((M, cfg.d), dtype=np.float32)
    h_bits = f32_to_bf16_bits(h)

    V, d, de = cfg.vocab, cfg.d, cfg.d_end
    w_end = np.empty((V, de), dtype=np.uint16)
    w_cloud = np.empty((V, d - de), dtype=np.uint16)
    inv = np.float32(1.0 / np.sqrt(d))
    for r0 in range(0, V, _W_CHUNK):
        n = min(_W_CHUNK, V - r0)
        w = r["w"].standard_normal((n, d), dtype=np.float32) * inv
        wb = f32_to_bf16_bits(w)
        w_end[r0:r0 + n] = wb[:, :de]
        w_cloud[r0:r0 + n] = wb[:, de:]

    codes = scale = None
    if cfg.wtype == "fp8":
        codes, scale = fp8_encode_rows(w_cloud)
        w_cloud = None
    elif cfg.wtype != "bf16":
        raise ValueError(f"unknown weight type {cfg.wtype!r}")

    bias = None
    if cfg.with_bias:
        bias = r["aux"].standard_normal(V, dtype=np.float32)

    subset = _draw_subset(cfg, r["subset"])
    return Workload(cfg=cfg, h_bits=h_bits, w_end_bits=w_end, w_cloud_bits=w_cloud,
                    w_cloud_codes=codes, w_cloud_scale=scale, bias=bias,
                    subset=subset, full_vocab=(cfg.subset_kind == "full"), rngs=r)


def with_subset(wl: Workload, cfg: Config) -> Workload:
    """The workload of ``cfg`` built from the hidden states and weights already
    drawn for ``wl``: valid when both configurations draw them from the same
    seed streams with the same shapes (the same seed index, d, d_end,
    vocabulary, weight type, rows and bias) and differ only in the subset,
    which comes from its own stream.  Equal to ``make_workload(cfg)``."""
    a, b = wl.cfg, cfg
    same = (a.seed_index, a.d, a.d_end, a.vocab, a.wtype, a.M, a.with_bias) == \
           (b.seed_index, b.d, b.d_end, b.vocab, b.wtype, b.M, b.with_bias)
    if not same or wl.h_bits.shape[0] != cfg.M:
        raise ValueError("with_subset: the two configurations draw different inputs")
    r = _streams(cfg.seed_index)
    subset = _draw_subset(cfg, r["subset"])
    return Workload(cfg=cfg, h_bits=wl.h_bits, w_end_bits=wl.w_end_bits,
                    w_cloud_bits=wl.w_cloud_bits, w_cloud_codes=wl.w_cloud_codes,
                    w_cloud_scale=wl.w_cloud_scale, bias=wl.bias, subset=subset,
                    full_vocab=(cfg.subset_kind == "full"), rngs=r)


def make_drafts(cfg: Config, ref_tokens: np.ndarray, subset: np.ndarray,
                rng: Optional[np.random.Generator] = None) -> np.ndarray:
    """Drafted tokens, int32 [sessions, k].

    For each (session s, position r < k) a fair coin decides between the
    reference token of row s*(k+1)+r and a uniform id of the subset.
    """
    if rng is None:
        rng = _streams(cfg.seed_index)["drafts"]
    S, R, k = cfg.sessions, cfg.rows_per_session, cfg.k
    ref = np.asarray(ref_tokens, dtype=np.int64).reshape(S, R)[:, :k]
    coin = rng.random((S, k)) < 0.5
    rand = subset[rng.integers(0, len(subset), size=(S, k))]
    return np.where(coin, ref, rand).astype(np.int32)


def scale_rows_bf16(h_bits: np.ndarray, rows, factor: float) -> np.ndarray:
    """Copy of h with the given rows multiplied by ``factor`` (re-rounded to bf16)."""
    out = h_bits.copy()
    rows = np.atleast_1d(rows)
    out[rows] = f32_to_bf16_bits(bf16_bits_to_f32(h_bits[rows]) * np.float32(factor))
    return out


def plant_masked_supertoken(w_end_bits: np.ndarray, w_cloud_bits: np.ndarray,
                            h_bits: np.ndarray, row: int, subset: np.ndarray,
                            magnitude: float = 8.0) -> int:
    """Overwrite one vocabulary row outside the subset so that its full-head
    logit for ``row`` of h is far larger than any subset logit.

    The weights get sign(h[row]) * magnitude in every dimension, so the
    id's logit for that row is magnitude * sum|h[row]|.  Returns the id.
    """
    V = w_end_bits.shape[0]
    member = np.zeros(V, dtype=bool)
    member[subset] = True
    outside = np.flatnonzero(~member)
    if outside.size == 0:
        raise ValueError("subset covers the whole vocabulary")
    vid = int(outside[outside.size // 2])
    sign = np.sign(bf16_bits_to_f32(h_bits[row])).astype(np.float32)
    sign[sign == 0] = 1.0
    planted = f32_to_bf16_bits(sign * np.float32(magnitude))
    de = w_end_bits.shape[1]
    w_end_bits[vid] = planted[:de]
    w_cloud_bits[vid] = planted[de:]
    return vid
