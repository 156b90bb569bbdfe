"""Seeded synthetic inputs for the AMS image-embedding step.

This module draws every input of one training step -- behavior lists, image
IDs, the image-feature table, the embedding-model weights and the upstream
gradients -- and holds none of the method's arithmetic (no dedup, no MLP, no
pooling).  Both the HIP path and the float64 oracle consume what it returns.

Shapes follow the paper: each sample carries only image indices (behavior
images plus the ad image, section 4.2); each image is a 4096-D non-negative
feature (VGG16 FC6 after ReLU, section 5.1; "pre-processed to 4096-D float
feature", section 7.3); the trainable embedding model is a 4096-256-64-12
fully connected net (section 5.1); users carry tens to hundreds of behaviors
(sections 1 and 4).  The workloads below are the named batch shapes this
library is measured and tested on.

Feature-table values are a pure function of (seed, row, column) built from an
integer hash, so any subset of rows can be regenerated bit-identically on the
CPU or on the GPU (the 16 GB table of the long-behavior workload is only ever
materialised on the device; the oracle regenerates just the rows it touches).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

__all__ = [
    "Workload", "JointSpec", "WORKLOADS", "get", "make_batch", "make_weights",
    "table_rows", "table_full", "table_chunks", "occurrences",
    "ctr_dims", "make_joint", "joint_occurrences", "make_ctr_weights",
    "id_table_rows", "id_table_full",
]


@dataclasses.dataclass(frozen=True)
class JointSpec:
    """Worker side of a joint step (Algorithm 1, WORKERITERATION): sparse ID
    features embedded from key-value tables (section 4.1) next to the image
    embeddings, and the CTR model on top of them, trained with cross-entropy
    (section 3.1).

    id_rows:    rows of each ID table (one ID of each table per behavior and
                per ad), id_dim-wide float32 rows
    id_zipf:    Zipf exponent of the IDs of every table (ranks scattered by a
                seeded permutation per table)
    ctr_hidden: hidden widths of the CTR MLP; its input is the pooled user
                image vector, the ad image embedding and one bag per table
    n_classes:  softmax classes (2: click / no click)
    label_p:    probability of a click label
    lr, eps, acc0: sparse Adagrad on the touched ID rows
    query_table: -1, or the ID table whose ad row (the ad's category, say)
                is the query of a second attentive channel
                (MultiQueryAttentivePooling, section 5.2); its id_dim must be
                the image embedding's width, and the CTR input grows by one
                pooled vector
    """
    id_rows: tuple
    id_dim: int
    id_zipf: float
    ctr_hidden: tuple
    n_classes: int
    label_p: float
    lr: float = 0.01
    eps: float = 1e-8
    acc0: float = 0.0
    query_table: int = -1


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload.

    lengths: ("fixed", L) | ("uniform", lo, hi) inclusive | ("geometric", mean, cap)
    ids:     ("uniform",) | ("zipf", s) over the n_images pool
    dims:    layer widths of the embedding MLP, input first, e.g. (4096, 256, 64, 12)
    dtype:   "f32" or "bf16" storage of the feature table and MLP weights
    table:   "normal" (~N(0,1)) or "relu_normal" (max(N(0,1), 0), CNN-feature-like)
    pools:   aggregators exercised on this workload
    stream:  seed stream; workloads that differ only in storage dtype share it,
             so they see the same batch, the same table values and the same
             weights (rounded to bf16 where stored in bf16)
    joint:   the ID features and CTR model of a joint step, or None
    """
    name: str
    index: int
    batch: int
    lengths: tuple
    n_images: int
    ids: tuple
    dims: tuple
    dtype: str
    table: str
    pools: tuple
    stream: int = -1
    joint: JointSpec | None = None

    @property
    def seed_stream(self) -> int:
        return self.index if self.stream < 0 else self.stream

    @property
    def in_dim(self) -> int:
        return self.dims[0]

    @property
    def out_dim(self) -> int:
        return self.dims[-1]

    @property
    def n_layers(self) -> int:
        return len(self.dims) - 1


WORKLOADS = {
    # 64 samples x 8 behaviors + 1 ad, uniform over 512 images, 256-D N(0,1)
    # features, MLP 256-64-16, sum pooling.
    "tiny": Workload("tiny", 0, 64, ("fixed", 8), 512, ("uniform",),
                     (256, 64, 16), "f32", "normal", ("sum",)),
    # 1024 samples, U[10,100] behaviors, Zipf(1.1) over 200k images,
    # 200k x 4096 fp32 table, MLP 4096-256-64-12 fp32, ad-attentive pooling.
    "c1_f32": Workload("c1_f32", 1, 1024, ("uniform", 10, 100), 200_000,
                       ("zipf", 1.1), (4096, 256, 64, 12), "f32",
                       "relu_normal", ("att",)),
    # Same batch shape with the table and weights in bf16 (fp32 accumulate).
    "c2_bf16": Workload("c2_bf16", 2, 1024, ("uniform", 10, 100), 200_000,
                        ("zipf", 1.1), (4096, 256, 64, 12), "bf16",
                        "relu_normal", ("sum", "max", "att"), stream=1),
    # Long behaviors: 4096 samples, geometric(mean 200) capped at 500,
    # Zipf(1.05) over 2M images, 2M x 4096 bf16 table (16.4 GB).
    "c3_long": Workload("c3_long", 3, 4096, ("geometric", 200, 500), 2_000_000,
                        ("zipf", 1.05), (4096, 256, 64, 12), "bf16",
                        "relu_normal", ("att",)),
    # Joint step: the long-behavior image path (same stream: same batch, table
    # and weights) plus three ID tables (10M, 1M, 10k rows x 12 fp32), each
    # ID Zipf(1.05), bag-summed over the behaviors and the ad; CTR MLP
    # 60-200-80-2 fp32 with softmax cross-entropy; sparse Adagrad on the
    # touched ID rows.
    "c4_joint": Workload("c4_joint", 4, 4096, ("geometric", 200, 500), 2_000_000,
                         ("zipf", 1.05), (4096, 256, 64, 12), "bf16",
                         "relu_normal", ("att",), stream=3,
                         joint=JointSpec((10_000_000, 1_000_000, 10_000), 12, 1.05, (200, 80), 2, 0.05)),
    # Small joint step for tests: the tiny image path, small ID tables, a
    # narrow CTR MLP, clicks frequent enough that both classes occur.
    "tiny_joint": Workload("tiny_joint", 5, 64, ("fixed", 8), 512, ("uniform",),
                           (256, 64, 16), "f32", "normal", ("att",), stream=0,
                           joint=JointSpec((1000, 100, 10), 12, 1.05, (32, 16), 2, 0.3)),
    # MultiQueryAttentivePooling (section 5.2): the joint step with a second
    # attentive channel whose query is the ad's row of the 10k-row ID table
    # (a category-sized table); the two pooled vectors (24-D) feed the CTR
    # MLP, 72-200-80-2.  Same data as c4_joint.
    "c4_mqap": Workload("c4_mqap", 6, 4096, ("geometric", 200, 500), 2_000_000,
                        ("zipf", 1.05), (4096, 256, 64, 12), "bf16",
                        "relu_normal", ("att",), stream=3,
                        joint=JointSpec((10_000_000, 1_000_000, 10_000), 12, 1.05, (200, 80), 2, 0.05,
                                        query_table=2)),
    # Small MultiQueryAttentivePooling step for tests: the tiny batch with a
    # 12-wide embedding (the query's width), the 10-row table as the query.
    "tiny_mqap": Workload("tiny_mqap", 7, 64, ("fixed", 8), 512, ("uniform",),
                          (256, 64, 12), "f32", "normal", ("att",), stream=0,
                          joint=JointSpec((1000, 100, 10), 12, 1.05, (32, 16), 2, 0.3, query_table=2)),
}
_BY_INDEX = {w.index: w for w in WORKLOADS.values()}


def get(name_or_index) -> Workload:
    if isinstance(name_or_index, Workload):
        return name_or_index
    if isinstance(name_or_index, int):
        return _BY_INDEX[name_or_index]
    return WORKLOADS[name_or_index]


def _streams(w: Workload, k: int, seed: int):
    ss = np.random.SeedSequence([seed, w.seed_stream, k])
    kids = ss.spawn(4)
    return [np.random.default_rng(s) for s in kids]


def _lengths(w: Workload, rng) -> np.ndarray:
    kind = w.lengths[0]
    if kind == "fixed":
        return np.full(w.batch, w.lengths[1], dtype=np.int64)
    if kind == "uniform":
        lo, hi = w.lengths[1], w.lengths[2]
        return rng.integers(lo, hi + 1, size=w.batch, dtype=np.int64)
    if kind == "geometric":
        mean, cap = w.lengths[1], w.lengths[2]
        # support {1, 2, ...}, success probability 1/mean, then capped
        return np.minimum(rng.geometric(1.0 / mean, size=w.batch), cap).astype(np.int64)
    raise ValueError(kind)


_ZIPF_CACHE: dict = {}


def _zipf_ids(rng, n: int, N: int, s: float, perm: np.ndarray) -> np.ndarray:
    key = (N, s)
    cdf = _ZIPF_CACHE.get(key)
    if cdf is None:
        # finite Zipf: P(rank r) proportional to r^-s for r = 1..N
        pmf = np.arange(1, N + 1, dtype=np.float64) ** (-s)
        cdf = np.cumsum(pmf)
        cdf /= cdf[-1]
        _ZIPF_CACHE[key] = cdf
    u = rng.random(n)
    rank = np.minimum(np.searchsorted(cdf, u, side="right"), N - 1)
    # scatter hot ranks over the table with a seeded permutation
    return perm[rank].astype(np.int32)


def _draw_ids(w: Workload, rng, n: int, perm: np.ndarray | None) -> np.ndarray:
    if n == 0:
        return np.zeros(0, dtype=np.int32)
    if w.ids[0] == "uniform":
        return rng.integers(0, w.n_images, size=n, dtype=np.int64).astype(np.int32)
    return _zipf_ids(rng, n, w.n_images, float(w.ids[1]), perm)


def make_batch(w, k: int = 0, seed: int = 0, batch: int | None = None) -> dict:
    """One seeded batch: CSR behavior lists, ad IDs and upstream gradients.

    Returns numpy arrays: seg_off int32[B+1], beh_ids int32[n_beh],
    ad_ids int32[B], g_u float32[B, D], g_a float32[B, D].
    `batch` overrides the sample count (same distributions) for scaled tests.
    """
    w = get(w)
    if batch is not None:
        w = dataclasses.replace(w, batch=batch)
    r_len, r_beh, r_ad, r_grad = _streams(w, k, seed)
    lens = _lengths(w, r_len)
    seg_off = np.zeros(w.batch + 1, dtype=np.int64)
    np.cumsum(lens, out=seg_off[1:])
    if seg_off[-1] > np.iinfo(np.int32).max:
        raise ValueError("batch too large for int32 offsets")
    perm = None
    if w.ids[0] == "zipf":
        # the rank -> image permutation is a property of the image pool, fixed per seed
        perm = np.random.default_rng(np.random.SeedSequence([seed, w.seed_stream, 1 << 20])).permutation(w.n_images)
    beh = _draw_ids(w, r_beh, int(seg_off[-1]), perm)
    ad = _draw_ids(w, r_ad, w.batch, perm)
    D = w.out_dim
    g_u = r_grad.standard_normal((w.batch, D), dtype=np.float32)
    g_a = r_grad.standard_normal((w.batch, D), dtype=np.float32)
    return {
        "seg_off": seg_off.astype(np.int32),
        "beh_ids": beh,
        "ad_ids": ad,
        "g_u": g_u,
        "g_a": g_a,
    }


def occurrences(batch: dict) -> np.ndarray:
    """Behavior IDs followed by ad IDs: the ID list one step deduplicates."""
    return np.concatenate([batch["beh_ids"], batch["ad_ids"]]).astype(np.int32)


def make_weights(w, seed: int = 0, bias_scale: float = 0.1):
    """Glorot-uniform weights W_l [out, in] and biases U(-bias_scale, bias_scale).

    Returned as torch CPU tensors: weights in the workload's storage dtype
    (float32 or bfloat16, rounded to nearest even), biases float32.
    """
    w = get(w)
    rng = np.random.default_rng(np.random.SeedSequence([seed, w.seed_stream, 7]))
    Ws, bs = [], []
    for fi, fo in zip(w.dims[:-1], w.dims[1:]):
        lim = math.sqrt(6.0 / (fi + fo))
        W = rng.uniform(-lim, lim, size=(fo, fi)).astype(np.float32)
        b = rng.uniform(-bias_scale, bias_scale, size=(fo,)).astype(np.float32)
        Wt = torch.from_numpy(W)
        if w.dtype == "bf16":
            Wt = Wt.to(torch.bfloat16)
        Ws.append(Wt)
        bs.append(torch.from_numpy(b))
    return Ws, bs


# ---- feature table: counter-based, device independent -----------------------

_M32 = 0xFFFFFFFF


def _mix32(x: torch.Tensor) -> torch.Tensor:
    # 32-bit integer finaliser (xorshift-multiply, "lowbias32" constants from
    # C. Wellons' hash-prospector); x holds uint32 values in int64 lanes.
    x = x ^ (x >> 16)
    x = (x * 0x21F0AAAD) & _M32
    x = x ^ (x >> 15)
    x = (x * 0x735A2D97) & _M32
    x = x ^ (x >> 15)
    return x


def _table_values(w: Workload, rows: torch.Tensor, seed: int) -> torch.Tensor:
    """float32 [len(rows), F] for int64 row indices `rows` (any device)."""
    F = w.in_dim
    cols = torch.arange(F, device=rows.device, dtype=torch.int64)
    c = rows.to(torch.int64)[:, None] * F + cols[None, :]
    lo = c & _M32
    hi = c >> 32
    sa = (0x9E3779B9 * (2 * seed + 1) + 0x1234567 * w.seed_stream) & _M32
    sb = (0x85EBCA6B * (2 * seed + 1) + 0x7654321 * w.seed_stream) & _M32
    ha = _mix32(_mix32(lo ^ sa) ^ hi)
    hb = _mix32(_mix32(lo ^ sb) ^ hi)
    del lo, hi, c
    u1 = ha >> 11                                   # 21 bits
    u2 = hb >> 11                                   # 21 bits
    u3 = ((ha & 0x7FF) << 10) | (hb & 0x3FF)        # 21 bits
    # Irwin-Hall(3): zero mean, unit variance, support (-3, 3); integer-exact
    s = 2 * (u1 + u2 + u3) - 3 * ((1 << 21) - 1)
    z = s.to(torch.float32) * (1.0 / (1 << 21))
    if w.table == "relu_normal":
        z = torch.clamp_min(z, 0.0)
    return z


def _storage(w: Workload):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def table_rows(w, rows, device="cpu", seed: int = 0, chunk_rows: int = 8192) -> torch.Tensor:
    """Rows `rows` of the feature table, [len(rows), F] in the storage dtype."""
    w = get(w)
    rows = torch.as_tensor(np.asarray(rows), dtype=torch.int64).to(device)
    out = torch.empty((rows.numel(), w.in_dim), dtype=_storage(w), device=device)
    for s in range(0, rows.numel(), chunk_rows):
        e = min(rows.numel(), s + chunk_rows)
        out[s:e] = _table_values(w, rows[s:e], seed).to(out.dtype)
    return out


def table_chunks(w, device="cpu", seed: int = 0, chunk_rows: int = 16384):
    """Yield (start, tensor) chunks covering the whole table."""
    w = get(w)
    for s in range(0, w.n_images, chunk_rows):
        e = min(w.n_images, s + chunk_rows)
        r = torch.arange(s, e, device=device, dtype=torch.int64)
        yield s, _table_values(w, r, seed).to(_storage(w))


def table_full(w, device="cpu", seed: int = 0, chunk_rows: int = 16384) -> torch.Tensor:
    """The whole [n_images, F] table on `device` (16.4 GB for the 2M-image pool)."""
    w = get(w)
    out = torch.empty((w.n_images, w.in_dim), dtype=_storage(w), device=device)
    for s, vals in table_chunks(w, device, seed, chunk_rows):
        out[s:s + vals.shape[0]] = vals
    return out


# ---- joint step: ID features, labels, CTR weights ----------------------------

def ctr_dims(w) -> tuple:
    """Layer widths of the CTR MLP: [pooled user image vector (two with a
    query table), ad image embedding, one bag per ID table] -> hidden ->
    classes (60-200-80-2; 72-200-80-2 with the query channel)."""
    w = get(w)
    j = w.joint
    n_img = 3 if j.query_table >= 0 else 2
    return (n_img * w.out_dim + len(j.id_rows) * j.id_dim,) + tuple(j.ctr_hidden) + (j.n_classes,)


_PERM_CACHE: dict = {}


def _id_perm(w: Workload, t: int, seed: int) -> np.ndarray:
    key = (w.seed_stream, seed, t, w.joint.id_rows[t])
    p = _PERM_CACHE.get(key)
    if p is None:
        p = np.random.default_rng(np.random.SeedSequence([seed, w.seed_stream, 1 << 21, t])).permutation(
            w.joint.id_rows[t])
        _PERM_CACHE.clear()
        _PERM_CACHE[key] = p
    return p


def make_joint(w, batch: dict, k: int = 0, seed: int = 0) -> dict:
    """The ID features and click labels of batch `batch` (from make_batch):
    beh_ids[t] int32[n_beh] and ad_ids[t] int32[B] for every ID table t
    (behavior IDs in the same sample order as the image IDs), labels int32[B]
    in {0, 1} ~ Bernoulli(label_p).  Drawn from streams of their own, so the
    image part of the batch is that of the plain workload."""
    w = get(w)
    j = w.joint
    n_beh = int(batch["seg_off"][-1])
    B = batch["seg_off"].size - 1
    kids = np.random.SeedSequence([seed, w.seed_stream, k, 99]).spawn(2 * len(j.id_rows) + 1)
    rngs = [np.random.default_rng(x) for x in kids]
    beh, ad = [], []
    for t, N in enumerate(j.id_rows):
        perm = _id_perm(w, t, seed)
        beh.append(_zipf_ids(rngs[2 * t], n_beh, N, j.id_zipf, perm) if n_beh else np.zeros(0, np.int32))
        ad.append(_zipf_ids(rngs[2 * t + 1], B, N, j.id_zipf, perm))
    labels = (rngs[-1].random(B) < j.label_p).astype(np.int32)
    return {"beh_ids": beh, "ad_ids": ad, "labels": labels}


def joint_occurrences(jb: dict, t: int) -> np.ndarray:
    """Behavior IDs then ad IDs of ID table t: the list one step deduplicates."""
    return np.concatenate([jb["beh_ids"][t], jb["ad_ids"][t]]).astype(np.int32)


def make_ctr_weights(w, seed: int = 0, bias_scale: float = 0.1):
    """Glorot-uniform float32 weights [out, in] and U(-bias_scale, bias_scale)
    biases of the CTR MLP (torch CPU tensors)."""
    w = get(w)
    rng = np.random.default_rng(np.random.SeedSequence([seed, w.seed_stream, 8]))
    dims = ctr_dims(w)
    Ws, bs = [], []
    for fi, fo in zip(dims[:-1], dims[1:]):
        lim = math.sqrt(6.0 / (fi + fo))
        Ws.append(torch.from_numpy(rng.uniform(-lim, lim, size=(fo, fi)).astype(np.float32)))
        bs.append(torch.from_numpy(rng.uniform(-bias_scale, bias_scale, size=(fo,)).astype(np.float32)))
    return Ws, bs


def _id_values(w: Workload, t: int, rows: torch.Tensor, seed: int) -> torch.Tensor:
    """float32 [len(rows), id_dim] rows of ID table t: 0.1 x Irwin-Hall(3) from
    the same counter-based hash as the feature table, salted per table."""
    Dd = w.joint.id_dim
    cols = torch.arange(Dd, device=rows.device, dtype=torch.int64)
    c = rows.to(torch.int64)[:, None] * Dd + cols[None, :]
    lo = c & _M32
    hi = c >> 32
    sa = (0x27D4EB2F * (2 * seed + 1) + 0x165667B1 * (w.seed_stream + 16 * (t + 1))) & _M32
    sb = (0xC2B2AE3D * (2 * seed + 1) + 0x9E3779B9 * (w.seed_stream + 16 * (t + 1))) & _M32
    ha = _mix32(_mix32(lo ^ sa) ^ hi)
    hb = _mix32(_mix32(lo ^ sb) ^ hi)
    u1, u2 = ha >> 11, hb >> 11
    u3 = ((ha & 0x7FF) << 10) | (hb & 0x3FF)
    s = 2 * (u1 + u2 + u3) - 3 * ((1 << 21) - 1)
    return s.to(torch.float32) * (0.1 / (1 << 21))


def id_table_rows(w, t: int, rows, device="cpu", seed: int = 0, chunk_rows: int = 1 << 20) -> torch.Tensor:
    """Rows `rows` of ID table t, float32 [len(rows), id_dim]."""
    w = get(w)
    rows = torch.as_tensor(np.asarray(rows), dtype=torch.int64).to(device)
    out = torch.empty((rows.numel(), w.joint.id_dim), dtype=torch.float32, device=device)
    for s0 in range(0, rows.numel(), chunk_rows):
        e = min(rows.numel(), s0 + chunk_rows)
        out[s0:e] = _id_values(w, t, rows[s0:e], seed)
    return out


def id_table_full(w, t: int, device="cpu", seed: int = 0, chunk_rows: int = 1 << 20) -> torch.Tensor:
    """The whole ID table t, float32 [id_rows[t], id_dim] on `device`."""
    w = get(w)
    N = w.joint.id_rows[t]
    out = torch.empty((N, w.joint.id_dim), dtype=torch.float32, device=device)
    for s0 in range(0, N, chunk_rows):
        e = min(N, s0 + chunk_rows)
        out[s0:e] = _id_values(w, t, torch.arange(s0, e, device=device, dtype=torch.int64), seed)
    return out
