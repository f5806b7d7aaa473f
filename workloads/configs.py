"""The five synthetic sampling workloads and their seeded recipe.

The paper's evaluation feeds prompts from the Databricks-dolly-15k dataset through eight FP16 LLMs
(Evaluation, "Models" and "Workload" paragraphs) with every sampling feature enabled.  Neither the
dataset nor any weights are available here, so these generators stand in for the logits such models
produce: rows of Gaussian or Student-t noise with Zipf-ranked offsets, at the vocabulary widths of the
paper's model families (32000 for Llama-2, 128256 for Llama-3.1, 152064 for Qwen-2.5 / QwQ; 256000 is
a stress width), with token histories drawn Zipf-style over the same ranking.

Recipe (identical for every size, so reduced-size variants keep the structure):

* ``numpy.random.SeedSequence(20260000 + c + 1000 * variant).spawn(6)`` gives six independent
  generators, in order: noise, permutation, params, history, mask, uniforms.
* A permutation ``perm`` of ``[0, V)`` ranks the vocabulary; token ``perm[i]`` has rank ``i + 1``.
  "Zipf(s) offsets" add ``-s * ln(rank)`` to every logit of that token.
* bf16 logits are the float32 draw rounded to nearest even by ``torch`` on the CPU and kept as raw
  16-bit patterns.
* Uniforms are ``(u32 >> 8) * 2**-24`` as float32, so ``0 <= u < 1`` exactly.
* Token histories draw ranks ``r`` with probability proportional to ``r**-1.2`` on ``[1, V]`` and map
  them to ids with ``perm[r - 1]``.

Only random inputs are produced here; nothing in this module computes any part of the sampling method.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

__all__ = ["Workload", "CONFIGS", "generate", "uniforms_from_u32", "to_bf16_bits"]


@dataclasses.dataclass
class Workload:
    name: str
    B: int
    V: int
    dtype: str  # "bf16" or "f32"
    ld: int
    logits: np.ndarray  # [B, ld] uint16 (bf16 bit patterns) or float32
    uniforms: np.ndarray  # [B] float32 in [0, 1)
    temperature: Optional[np.ndarray] = None  # [B] float32
    top_k: Optional[np.ndarray] = None  # [B] int32
    top_p: Optional[np.ndarray] = None  # [B] float32
    min_p: Optional[np.ndarray] = None  # [B] float32
    repetition_penalty: Optional[np.ndarray] = None  # [B] float32
    frequency_penalty: Optional[np.ndarray] = None  # [B] float32
    presence_penalty: Optional[np.ndarray] = None  # [B] float32
    hist_offsets: Optional[np.ndarray] = None  # [B + 1] int64
    hist_ids: Optional[np.ndarray] = None  # [hist_offsets[B]] int32
    n_top: int = 0
    # a prompt history per row; when given, hist_* holds the output tokens only
    prompt_offsets: Optional[np.ndarray] = None  # [B + 1] int64
    prompt_ids: Optional[np.ndarray] = None  # [prompt_offsets[B]] int32

    def row_slice(self, lo: int, hi: int) -> "Workload":
        """Rows ``lo:hi`` as a workload of their own (histories re-based to start at 0)."""
        d = dataclasses.replace(self)
        d.B = hi - lo
        d.logits = self.logits[lo:hi]
        d.uniforms = self.uniforms[lo:hi]
        for f in ("temperature", "top_k", "top_p", "min_p", "repetition_penalty",
                  "frequency_penalty", "presence_penalty"):
            a = getattr(self, f)
            setattr(d, f, None if a is None else a[lo:hi])
        if self.hist_offsets is not None:
            o = self.hist_offsets[lo:hi + 1]
            d.hist_ids = self.hist_ids[o[0]:o[-1]]
            d.hist_offsets = (o - o[0]).astype(np.int64)
        if self.prompt_offsets is not None:
            o = self.prompt_offsets[lo:hi + 1]
            d.prompt_ids = self.prompt_ids[o[0]:o[-1]]
            d.prompt_offsets = (o - o[0]).astype(np.int64)
        return d

    @property
    def itemsize(self) -> int:
        return 2 if self.dtype == "bf16" else 4


def uniforms_from_u32(u32: np.ndarray) -> np.ndarray:
    """Map raw 32-bit integers to float32 uniforms in [0, 1) with 24 significant bits."""
    return ((u32.astype(np.uint64) >> 8).astype(np.float64) * 2.0 ** -24).astype(np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest-even, via torch on the CPU) and return the raw bit patterns."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _zipf_hist(rng: np.random.Generator, perm: np.ndarray, B: int, H: int, V: int, s: float = 1.2):
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    w /= w.sum()
    ranks = rng.choice(V, size=(B, H), p=w)  # rank - 1
    ids = perm[ranks].astype(np.int32).reshape(-1)
    offs = (np.arange(B + 1, dtype=np.int64) * H)
    return offs, ids


def _zipf_offsets(perm: np.ndarray, V: int, s: float) -> np.ndarray:
    rank = np.empty(V, dtype=np.float64)
    rank[perm] = np.arange(1, V + 1, dtype=np.float64)
    return (-s * np.log(rank)).astype(np.float32)


def _mixed_params(rng: np.random.Generator, B: int, with_min_p: bool):
    """Per-row mix: a quarter of the rows greedy, top_k from {1, 20, 100, off}, top_p ~ U(0.5, 1),
    temperature ~ U(0.3, 1.5); optionally min_p from {0, 0.01, 0.05, 0.1} on sampled rows."""
    temp = rng.uniform(0.3, 1.5, size=B).astype(np.float32)
    greedy = rng.permutation(B)[: B // 4]
    temp[greedy] = 0.0
    top_k = np.array([1, 20, 100, 0], dtype=np.int32)[rng.integers(0, 4, size=B)]
    top_p = rng.uniform(0.5, 1.0, size=B).astype(np.float32)
    min_p = None
    if with_min_p:
        min_p = np.array([0.0, 0.01, 0.05, 0.1], dtype=np.float32)[rng.integers(0, 4, size=B)]
        min_p[greedy] = 0.0
    return temp, top_k, top_p, min_p


def _full(B, v, dt):
    return np.full(B, v, dtype=dt)


CONFIGS = {
    1: dict(name="C1 B=4 V=32000 f32 N(0,2)+boost, T=0.8 k=50 p=0.9", B=4, V=32000, dtype="f32"),
    2: dict(name="C2 B=64 V=128256 bf16 N(0,3)+Zipf1.1, mixed params", B=64, V=128256, dtype="bf16"),
    3: dict(name="C3 B=256 V=152064 bf16 N(0,3)+Zipf1.1, penalties H=2048, T=0.7 k=40 p=0.95",
            B=256, V=152064, dtype="bf16"),
    4: dict(name="C4 B=512 V=152064 f32 2*t3, T=1 p=0.98 min_p=0.02", B=512, V=152064, dtype="f32"),
    5: dict(name="C5 B=1024 V=256000 bf16 N(0,2) 1% -inf, mixed params+min_p, penalties H=4096, top-20",
            B=1024, V=256000, dtype="bf16"),
}


def generate(cfg: int, B: Optional[int] = None, V: Optional[int] = None, variant: int = 0,
             ld: Optional[int] = None, H: Optional[int] = None) -> Workload:
    """Build workload ``cfg`` (1..5), optionally at a reduced batch ``B`` / vocabulary ``V`` /
    history length ``H`` with the same recipe.  ``ld`` >= V pads every row (pad entries are NaN bit
    patterns that a correct reader never touches)."""
    c = CONFIGS[cfg]
    B = c["B"] if B is None else B
    V = c["V"] if V is None else V
    ld = V if ld is None else ld
    ss = np.random.SeedSequence(20260000 + cfg + 1000 * variant).spawn(6)
    r_noise, r_perm, r_par, r_hist, r_mask, r_unif = (np.random.default_rng(s) for s in ss)
    perm = r_perm.permutation(V)
    kw = {}
    n_top = 0
    if cfg == 1:
        x = r_noise.normal(0.0, 2.0, size=(B, V)).astype(np.float32)
        for i in range(B):
            x[i, r_perm.choice(V, size=min(5, V), replace=False)] += np.float32(8.0)
        kw.update(temperature=_full(B, 0.8, np.float32), top_k=_full(B, 50, np.int32),
                  top_p=_full(B, 0.9, np.float32), min_p=_full(B, 0.0, np.float32))
    elif cfg == 2:
        x = r_noise.normal(0.0, 3.0, size=(B, V)).astype(np.float32) + _zipf_offsets(perm, V, 1.1)
        t, k, p, _ = _mixed_params(r_par, B, with_min_p=False)
        kw.update(temperature=t, top_k=k, top_p=p)
    elif cfg == 3:
        x = r_noise.normal(0.0, 3.0, size=(B, V)).astype(np.float32) + _zipf_offsets(perm, V, 1.1)
        kw.update(temperature=_full(B, 0.7, np.float32), top_k=_full(B, 40, np.int32),
                  top_p=_full(B, 0.95, np.float32), min_p=_full(B, 0.0, np.float32),
                  repetition_penalty=_full(B, 1.1, np.float32),
                  frequency_penalty=_full(B, 0.2, np.float32),
                  presence_penalty=_full(B, 0.1, np.float32))
        offs, ids = _zipf_hist(r_hist, perm, B, 2048 if H is None else H, V)
        kw.update(hist_offsets=offs, hist_ids=ids)
    elif cfg == 4:
        x = (2.0 * r_noise.standard_t(3.0, size=(B, V))).astype(np.float32)
        kw.update(temperature=_full(B, 1.0, np.float32), top_k=_full(B, 0, np.int32),
                  top_p=_full(B, 0.98, np.float32), min_p=_full(B, 0.02, np.float32))
    elif cfg == 5:
        x = r_noise.normal(0.0, 2.0, size=(B, V)).astype(np.float32)
        x[r_mask.random(size=(B, V)) < 0.01] = -np.inf
        t, k, p, mp = _mixed_params(r_par, B, with_min_p=True)
        kw.update(temperature=t, top_k=k, top_p=p, min_p=mp,
                  repetition_penalty=_full(B, 1.1, np.float32),
                  frequency_penalty=_full(B, 0.2, np.float32),
                  presence_penalty=_full(B, 0.1, np.float32))
        offs, ids = _zipf_hist(r_hist, perm, B, 4096 if H is None else H, V)
        kw.update(hist_offsets=offs, hist_ids=ids)
        n_top = 20
    else:
        raise ValueError(cfg)
    u = uniforms_from_u32(r_unif.integers(0, 2 ** 32, size=B, dtype=np.uint64).astype(np.uint32))
    dtype = c["dtype"]
    if dtype == "bf16":
        data = to_bf16_bits(x)
        pad_val = np.uint16(0x7FC1)
    else:
        data = x
        pad_val = np.float32(np.nan)
    if ld != V:
        full = np.empty((B, ld), dtype=data.dtype)
        full[:] = pad_val
        full[:, :V] = data
        data = full
    return Workload(name=c["name"], B=B, V=V, dtype=dtype, ld=ld, logits=data, uniforms=u, n_top=n_top, **kw)


def add_prompt(w: Workload, P: int, seed: int = 0, s: float = 1.2) -> Workload:
    """Give every row of ``w`` a prompt history of ``P`` ids, ranks drawn with probability proportional
    to ``r**-s`` over a seeded permutation of the vocabulary; ``w``'s own history becomes the output
    history (the split of the repetition penalty from the frequency and presence penalties)."""
    rng = np.random.default_rng(np.random.SeedSequence(20269000 + seed))
    perm = rng.permutation(w.V)
    offs, ids = _zipf_hist(rng, perm, w.B, P, w.V, s)
    w.prompt_offsets, w.prompt_ids = offs, ids
    return w

