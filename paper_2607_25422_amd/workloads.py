"""Seeded synthetic workloads for the SKIP routing core.

This module only draws random inputs and lays them out; it performs none of
the routing method's arithmetic (no scoring, selection, graph construction or
attention).  Both the HIP path and the CPU checker consume what it returns.

The five named workloads mirror the shapes the paper's pipeline sees: a
24x24 patch grid per image tile (Sec. 5 setup: 576 visual tokens), question
token counts of a few tens, a handful of retrieved passages per question, and
an average bipartite degree of 4 (App. B.3, Def. B.3; degree-sweep table in
the hyper-parameter appendix).  The paper's datasets (OK-VQA, A-OKVQA,
InfoSeek, ...) and trained encoders are not available, so Gaussian tokens
stand in for encoder outputs; "planted" tokens correlated with the pooled
question stand in for question-relevant image regions.

Random streams: one ``numpy.random.Generator(PCG64(SeedSequence([seed,
workload_id, b])))`` per query ``b``, so ragged batches stay reproducible.
Seeds 2026, 42 and 137 are the ones the paper reports results over
(reproducibility statement, App. I).

Casting: values are drawn in float64 and rounded once, to float32 for the
fp32 workload and to bfloat16 (round-to-nearest-even, torch on the CPU) for
the others.  Everything downstream consumes the rounded tensors.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

SEEDS = (2026, 42, 137)


@dataclass(frozen=True)
class Workload:
    """Shape and distribution recipe of one synthetic batch."""

    name: str
    wid: int                      # stream id mixed into every SeedSequence
    dtype: str                    # "f32" or "bf16"
    B: int                        # questions in the batch
    N: int                        # visual tokens per question
    d: int                        # embedding width (= H * d_h)
    T: int                        # question tokens per question
    k_choices: Sequence[int]      # kept visual tokens per question (one value = fixed)
    P_choices: Sequence[int]      # retrieved passages per question
    L_p: int                      # tokens per passage
    H: int
    d_h: int
    visual: str                   # "unit" (N(0,1)) or "scaled" (N(0,1/d))
    planting: str                 # "random", "tiles", "heavy_tail" or "none"
    n_planted: int = 0
    tiles: int = 1                # 24x24 tiles making up the N tokens
    avg_degree: float = 4.0
    sm_scale: Optional[float] = None   # None -> 1/sqrt(d_h)

    @property
    def scale(self) -> float:
        return self.sm_scale if self.sm_scale is not None else 1.0 / math.sqrt(self.d_h)


# k = ceil(4 * sqrt(N)) for the fixed-budget workloads: 96, 192, 384.
WORKLOADS: Dict[str, Workload] = {
    "tiny_fp32": Workload(
        name="tiny_fp32", wid=1, dtype="f32", B=1, N=576, d=256, T=16,
        k_choices=(96,), P_choices=(4,), L_p=64, H=4, d_h=64,
        visual="unit", planting="random", n_planted=24),
    "llava_bf16": Workload(
        name="llava_bf16", wid=2, dtype="bf16", B=8, N=576, d=1024, T=32,
        k_choices=(96,), P_choices=(5,), L_p=128, H=16, d_h=64,
        visual="scaled", planting="random", n_planted=29,
        sm_scale=math.sqrt(1024) / math.sqrt(64)),
    "highres_bf16": Workload(
        name="highres_bf16", wid=3, dtype="bf16", B=16, N=2304, d=4096, T=32,
        k_choices=(192,), P_choices=(10,), L_p=256, H=32, d_h=128,
        visual="scaled", planting="tiles", n_planted=128, tiles=4,
        sm_scale=math.sqrt(4096) / math.sqrt(128)),
    "mixed_bf16": Workload(
        name="mixed_bf16", wid=4, dtype="bf16", B=64, N=2304, d=4096, T=32,
        k_choices=(48, 96, 192, 384), P_choices=(2, 5, 10, 20), L_p=256,
        H=32, d_h=128, visual="scaled", planting="tiles", n_planted=128,
        tiles=4, sm_scale=math.sqrt(4096) / math.sqrt(128)),
    "longctx_bf16": Workload(
        name="longctx_bf16", wid=5, dtype="bf16", B=4, N=9216, d=4096, T=64,
        k_choices=(384,), P_choices=(20,), L_p=512, H=32, d_h=128,
        visual="scaled", planting="heavy_tail", tiles=16,
        sm_scale=math.sqrt(4096) / math.sqrt(128)),
}

ORDER = ("tiny_fp32", "llava_bf16", "highres_bf16", "mixed_bf16", "longctx_bf16")


def keep_budget(N: int, c: float = 4.0) -> int:
    """Kept-token budget k = ceil(c * sqrt(N)).

    The paper's sparsity bound (Thm. 4.1) says the number of tokens that must
    be retained grows like sqrt(N), so the retained fraction falls like
    1/sqrt(N); with c = 4 this gives 96, 192 and 384 for N = 576, 2304, 9216.
    The library itself never computes k: it is an input (through offsets).
    """
    return int(math.ceil(c * math.sqrt(N) - 1e-9))


@dataclass
class Batch:
    """One synthetic batch, on the CPU, in the rounded element type."""

    wl: Workload
    seed: int
    V: torch.Tensor               # [B, N, d]
    Qtok: torch.Tensor            # [sum T_b, d]
    q_offsets: np.ndarray         # int32 [B+1]
    kept_offsets: np.ndarray      # int32 [B+1]
    Kh: torch.Tensor              # [sum M_b, H, d_h]
    Vh: torch.Tensor              # [sum M_b, H, d_h]
    passage_offsets: np.ndarray   # int32 [sum P_b + 1], token offsets
    query_passages: np.ndarray    # int32 [B+1], offsets into the passage table
    w_bias: Optional[torch.Tensor] = None   # [d] or None
    planted: List[np.ndarray] = field(default_factory=list)

    @property
    def B(self) -> int:
        return self.V.shape[0]

    @property
    def k(self) -> np.ndarray:
        return np.diff(self.kept_offsets)

    @property
    def P(self) -> np.ndarray:
        return np.diff(self.query_passages)

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.wl.dtype == "f32" else torch.bfloat16


def _round(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(torch.float32) if dtype == "f32" else t.to(torch.bfloat16)


def _stream(seed: int, wid: int, b: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wid, b])))


def _tile_block_positions(rng: np.random.Generator, tiles: int, n_blocks: int) -> np.ndarray:
    """Token indices of an 8x8 patch block in each of n_blocks random 24x24 tiles."""
    chosen = rng.choice(tiles, size=min(n_blocks, tiles), replace=False)
    idx = []
    for t in sorted(chosen):
        r0, c0 = rng.integers(0, 24 - 8 + 1, size=2)
        for r in range(r0, r0 + 8):
            for c in range(c0, c0 + 8):
                idx.append(int(t) * 576 + r * 24 + c)
    return np.array(sorted(idx), dtype=np.int64)


def _draw_query(wl: Workload, seed: int, b: int, N: int, d: int, T_choices,
                k_choices, P_choices, L_choices):
    rng = _stream(seed, wl.wid, b)
    k_b = int(rng.choice(np.asarray(k_choices)))
    P_b = int(rng.choice(np.asarray(P_choices)))
    T = int(rng.choice(np.asarray(T_choices)))
    sd = 1.0 if wl.visual == "unit" else 1.0 / math.sqrt(d)
    Q = rng.standard_normal((T, d)) * sd
    V = rng.standard_normal((N, d)) * sd
    planted = np.zeros(0, dtype=np.int64)
    if wl.planting != "none":
        # The question's own sample mean sets the planted direction.
        qm = Q.mean(axis=0)
        qdir = qm / max(np.linalg.norm(qm), 1e-30)
    if wl.planting == "random" and wl.n_planted > 0:
        planted = np.sort(rng.choice(N, size=min(wl.n_planted, N), replace=False))
        noise = rng.standard_normal((planted.size, d))
        if wl.visual == "unit":
            V[planted] = qm + 0.5 * noise
        else:
            V[planted] = 0.6 * qdir + 0.8 * sd * noise
    elif wl.planting == "tiles":
        planted = _tile_block_positions(rng, wl.tiles, 2)
        planted = planted[planted < N]
        noise = rng.standard_normal((planted.size, d))
        V[planted] = 0.6 * qdir + 0.8 * sd * noise
    elif wl.planting == "heavy_tail":
        t = rng.standard_t(3.0, size=N)
        V += 0.3 * t[:, None] * qdir[None, :]
    # Knowledge passages: per-passage mean direction plus unit noise for keys,
    # unit Gaussian values.
    Ls = [int(rng.choice(np.asarray(L_choices))) for _ in range(P_b)]
    Ks, Vs = [], []
    for j in range(P_b):
        mu = rng.standard_normal(d) * 0.5
        Ks.append(mu[None, :] + rng.standard_normal((Ls[j], d)))
        Vs.append(rng.standard_normal((Ls[j], d)))
    return k_b, P_b, Q, V, Ks, Vs, Ls, planted


def make_batch(wl: Workload | str, seed: int = 2026, *, B: Optional[int] = None,
               N: Optional[int] = None, d: Optional[int] = None,
               T: Optional[int] = None, H: Optional[int] = None,
               d_h: Optional[int] = None, k: Optional[Sequence[int]] = None,
               P: Optional[Sequence[int]] = None,
               L_p: Optional[Sequence[int] | int] = None,
               with_bias: bool = False, threads: int = 0) -> Batch:
    """Draw one batch.  Keyword overrides shrink or reshape a named workload
    (tests use them for small and ragged cases); ``k``, ``P`` and ``L_p``
    accept a set of choices drawn uniformly per question (per passage for
    ``L_p``)."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    if H is not None or d_h is not None:
        H = H if H is not None else wl.H
        d_h = d_h if d_h is not None else wl.d_h
        wl = replace(wl, H=H, d_h=d_h, d=H * d_h)
    if d is not None and d != wl.d:
        if d % wl.H:
            raise ValueError("d must be a multiple of H")
        wl = replace(wl, d=d, d_h=d // wl.H)
    B = wl.B if B is None else B
    N = wl.N if N is None else N
    if T is None:
        T_choices = (wl.T,)
    elif isinstance(T, int):
        T_choices = (T,)
    else:
        T_choices = tuple(T)
    if min(T_choices) < 1:
        raise ValueError("every question needs at least one token")
    k_choices = tuple(wl.k_choices if k is None else k)
    P_choices = tuple(wl.P_choices if P is None else P)
    if L_p is None:
        L_choices = (wl.L_p,)
    elif isinstance(L_p, int):
        L_choices = (L_p,)
    else:
        L_choices = tuple(L_p)
    if max(k_choices) > N:
        raise ValueError("a kept budget exceeds N")
    d = wl.d

    def one(b):
        return _draw_query(wl, seed, b, N, d, T_choices, k_choices, P_choices, L_choices)

    if threads and B > 1:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            parts = list(ex.map(one, range(B)))
    else:
        parts = [one(b) for b in range(B)]

    dt = wl.dtype
    V = torch.empty((B, N, d), dtype=torch.float32 if dt == "f32" else torch.bfloat16)
    for b, p in enumerate(parts):
        V[b] = _round(p[3], dt)
    Qtok = _round(np.concatenate([p[2] for p in parts], axis=0), dt)
    q_offsets = np.zeros(B + 1, dtype=np.int32)
    q_offsets[1:] = np.cumsum([p[2].shape[0] for p in parts])
    kept_offsets = np.zeros(B + 1, dtype=np.int32)
    kept_offsets[1:] = np.cumsum([p[0] for p in parts])
    query_passages = np.zeros(B + 1, dtype=np.int32)
    query_passages[1:] = np.cumsum([p[1] for p in parts])
    Ls = [L for p in parts for L in p[6]]
    passage_offsets = np.zeros(len(Ls) + 1, dtype=np.int32)
    passage_offsets[1:] = np.cumsum(Ls)
    M = int(passage_offsets[-1])
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    Kh = torch.empty((M, wl.H, wl.d_h), dtype=tdt)
    Vh = torch.empty((M, wl.H, wl.d_h), dtype=tdt)
    pos = 0
    for p in parts:
        for Kj, Vj in zip(p[4], p[5]):
            n = Kj.shape[0]
            Kh[pos:pos + n] = _round(Kj, dt).view(n, wl.H, wl.d_h)
            Vh[pos:pos + n] = _round(Vj, dt).view(n, wl.H, wl.d_h)
            pos += n
    w_bias = None
    if with_bias:
        rng = _stream(seed, wl.wid, 1 << 30)
        sd = 1.0 if wl.visual == "unit" else 1.0 / math.sqrt(d)
        w_bias = _round(rng.standard_normal(d) * sd / math.sqrt(d), dt)
    return Batch(wl=replace(wl, B=B, N=N, T=max(T_choices)), seed=seed, V=V, Qtok=Qtok,
                 q_offsets=q_offsets, kept_offsets=kept_offsets, Kh=Kh, Vh=Vh,
                 passage_offsets=passage_offsets, query_passages=query_passages,
                 w_bias=w_bias, planted=[p[7] for p in parts])


@dataclass
class ScorerWeights:
    """Synthetic weights of the main-text salience scorer, a two-layer
    perceptron on [v; q_bar; v * q_bar] (CPU tensors): W1 [h, 3d] bfloat16,
    b1 [h] and w2 [h] float32, b2 a float."""

    W1: torch.Tensor
    b1: torch.Tensor
    w2: torch.Tensor
    b2: float

    @property
    def hidden(self) -> int:
        return int(self.W1.shape[0])

    def as_dict(self) -> dict:
        return {"W1": self.W1, "b1": self.b1, "w2": self.w2, "b2": self.b2}


def make_scorer_weights(wl: Workload | str, hidden: int = 512, seed: int = 2026) -> ScorerWeights:
    """Gaussian weights scaled so that each of the three input blocks adds a
    term of order one to a hidden pre-activation for this workload's token
    distribution: the v block ~ N(0, 1/(d s_v^2)), the q_bar block ~ N(0, T/(d
    s_v^2)) (q_bar averages T tokens), the product block ~ N(0, T/(d s_v^4));
    s_v is the per-coordinate scale of a visual token (1 or 1/sqrt(d)).  b1 is
    a small Gaussian, so about half the hidden units are active; w2 ~ N(0,
    1/h).  No trained weights exist for the paper's scorer; the hidden width
    is not stated there (512 here)."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    d = wl.d
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wl.wid, 7919])))
    sv2 = 1.0 if wl.visual == "unit" else 1.0 / d
    Wa = rng.standard_normal((hidden, d)) * math.sqrt(1.0 / (d * sv2))
    Wb = rng.standard_normal((hidden, d)) * math.sqrt(wl.T / (d * sv2))
    Wc = rng.standard_normal((hidden, d)) * math.sqrt(wl.T / (d * sv2 * sv2))
    W1 = np.concatenate([Wa, Wb, Wc], axis=1)
    b1 = rng.standard_normal(hidden) * 0.1
    w2 = rng.standard_normal(hidden) / math.sqrt(hidden)
    return ScorerWeights(W1=_round(W1, "bf16"), b1=torch.from_numpy(b1.astype(np.float32)),
                         w2=torch.from_numpy(w2.astype(np.float32)),
                         b2=float(rng.standard_normal()))


@dataclass
class GateWeights:
    """Synthetic weights of the passage verification gate, a two-layer
    perceptron on [q_bar; v_bar; e; e * q_bar; |e - q_bar|] (CPU tensors):
    W [h, 5d] bfloat16, b1 [h] and w2 [h] float32, b2 a float."""

    W: torch.Tensor
    b1: torch.Tensor
    w2: torch.Tensor
    b2: float

    @property
    def hidden(self) -> int:
        return int(self.W.shape[0])


def make_gate_weights(wl: Workload | str, hidden: int = 512, seed: int = 2026) -> GateWeights:
    """Gaussian weights scaled so that each of the five input blocks adds a
    term of order one to a hidden pre-activation for this workload's
    distributions: with s_v the per-coordinate scale of a visual or question
    token (1 or 1/sqrt(d)) and 0.5 that of a passage key, the block standard
    deviations are sqrt(T)/(sqrt(d) s_v) for q_bar (a mean of T tokens),
    1/(sqrt(d) s_v) for v_bar, 2/sqrt(d) for e and |e - q_bar|, and
    2 sqrt(T)/(sqrt(d) s_v) for the product.  b1 is a small Gaussian, w2 ~
    N(0, 1/h) and b2 = 0, so a threshold of 1/2 on the gate probability
    passes about half of the passages.  No trained gate exists; the paper does
    not state its hidden width (512 here)."""
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    d = wl.d
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wl.wid, 104729])))
    sv = 1.0 if wl.visual == "unit" else 1.0 / math.sqrt(d)
    rd = 1.0 / math.sqrt(d)
    sds = (math.sqrt(wl.T) * rd / sv, rd / sv, 2.0 * rd, 2.0 * math.sqrt(wl.T) * rd / sv,
           2.0 * rd)
    W = np.concatenate([rng.standard_normal((hidden, d)) * s for s in sds], axis=1)
    b1 = rng.standard_normal(hidden) * 0.1
    w2 = rng.standard_normal(hidden) / math.sqrt(hidden)
    return GateWeights(W=_round(W, "bf16"), b1=torch.from_numpy(b1.astype(np.float32)),
                       w2=torch.from_numpy(w2.astype(np.float32)), b2=0.0)


def make_projection(d_out: int, d: int, seed: int = 2026) -> torch.Tensor:
    """A synthetic learned projection W [d_out, d] in bfloat16, N(0, 1/d)
    entries, so that W x keeps the scale of x.  No trained projections exist
    for this path."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, d_out, d, 31337])))
    return _round(rng.standard_normal((d_out, d)) / math.sqrt(d), "bf16")
