"""Seeded synthetic workloads: document lengths and bf16 tensors.

This module holds no attention, planning or sharding arithmetic. It only
draws document lengths and normally distributed tensor values from fixed
seeds, so that the GPU path and the CPU oracle can be handed identical
inputs. Both sides receive its outputs as plain arrays; neither is imported
from here.

Length recipes (the paper's datasets are not available; these stand in for
their length distributions, FlashCP Sec. 4.1 "Datasets"):

* ``tiny``      2048 tokens, 3 documents cut at two distinct uniform points.
* ``llama8b``   65536 tokens, log-normal lengths (median 2048, sigma 1.0),
                clipped to [64, 65536].
* ``wholedoc``  65536 tokens, lengths uniform on [128, 4096].
* ``longdoc``   131072 tokens: one 98304-token document first, then
                log-normal lengths (median 2048, sigma 1.0, clip [64, 32768]).
* ``hybrid70b`` 262144 tokens, classic Pareto lengths (alpha 1.2, minimum
                256, clipped to 131072), drawn by inverse CDF.

Every recipe samples until the total reaches the context size and then
truncates the last document, as the paper does when packing (Sec. 4.1).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

BLOCK = 256  # tokens per independently seeded tensor block

TENSOR_IDS = {"q": 1, "k": 2, "v": 3, "do": 4}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int          # 1-based workload number, also the length seed
    context: int        # packed tokens C
    hq: int
    hkv: int
    d: int
    cp: int             # context-parallel degree N
    plan: str           # "per_doc" | "whole_lpt" | "hybrid"
    rank: str           # "0", "3", "last", "heaviest"
    two_pass: bool      # local and received KV as separate passes + merge


WORKLOADS = {
    "tiny": Workload("tiny", 1, 2048, 4, 4, 64, 2, "per_doc", "0", True),
    "llama8b": Workload("llama8b", 2, 65536, 32, 8, 128, 8, "per_doc", "3", True),
    "wholedoc": Workload("wholedoc", 3, 65536, 32, 8, 128, 8, "whole_lpt", "heaviest", True),
    "longdoc": Workload("longdoc", 4, 131072, 32, 8, 128, 16, "per_doc", "last", True),
    "hybrid70b": Workload("hybrid70b", 5, 262144, 64, 8, 128, 32, "hybrid", "heaviest", True),
}


def _fill(draw, total: int) -> list[int]:
    """Draw lengths until they reach ``total``; truncate the last one."""
    out: list[int] = []
    acc = 0
    while acc < total:
        x = int(draw())
        x = min(x, total - acc)
        out.append(x)
        acc += x
    return out


def _lognormal(rng, median, sigma, lo, hi):
    def draw():
        x = rng.lognormal(mean=math.log(median), sigma=sigma)
        return int(min(max(round(x), lo), hi))
    return draw


def doc_lengths(name: str, context: int | None = None, seed: int | None = None) -> np.ndarray:
    """Document lengths (int64) of workload ``name``.

    ``context`` overrides the packed size (for scaled-down test variants of
    the same recipe); ``seed`` overrides the default seed (the workload index).
    """
    w = WORKLOADS[name]
    C = w.context if context is None else int(context)
    rng = np.random.default_rng(w.index if seed is None else seed)
    if name == "tiny":
        cuts = np.sort(rng.choice(np.arange(1, C), size=2, replace=False))
        lens = [int(cuts[0]), int(cuts[1] - cuts[0]), int(C - cuts[1])]
    elif name == "llama8b":
        lens = _fill(_lognormal(rng, 2048, 1.0, 64, C), C)
    elif name == "wholedoc":
        lens = _fill(lambda: rng.integers(128, 4096, endpoint=True), C)
    elif name == "longdoc":
        first = (3 * C) // 4  # 98304 of 131072
        lens = [first] + _fill(_lognormal(rng, 2048, 1.0, 64, C - first), C - first)
    elif name == "hybrid70b":
        hi = C // 2

        def pareto():
            u = rng.random()
            return min(int(math.floor(256.0 * (1.0 - u) ** (-1.0 / 1.2))), hi)
        lens = _fill(pareto, C)
    else:
        raise KeyError(name)
    arr = np.asarray(lens, dtype=np.int64)
    assert arr.sum() == C and (arr > 0).all()
    return arr


def cu_seqlens(lengths) -> np.ndarray:
    """int32 prefix sums [0, d0, d0+d1, ...] (a plain running total)."""
    out = np.zeros(len(lengths) + 1, dtype=np.int64)
    np.cumsum(np.asarray(lengths, dtype=np.int64), out=out[1:])
    return out.astype(np.int32)


class TensorSource:
    """bf16 N(0,1) rows of the packed Q, K, V, dO tensors, seeded per block.

    Row ``g`` of tensor X lives in block ``g // BLOCK``; each block is drawn
    from its own PCG64 stream keyed by (workload seed, tensor, block), so any
    subset of rows is reproducible without materialising the whole tensor.
    """

    def __init__(self, seed: int, hq: int, hkv: int, d: int):
        self.seed = int(seed)
        self.heads = {"q": hq, "k": hkv, "v": hkv, "do": hq}
        self.d = int(d)

    def _block(self, name: str, b: int) -> np.ndarray:
        ss = np.random.SeedSequence([100 + self.seed, TENSOR_IDS[name], int(b)])
        rng = np.random.default_rng(ss)
        return rng.standard_normal((BLOCK, self.heads[name], self.d), dtype=np.float32)

    def rows(self, name: str, gpos) -> torch.Tensor:
        """bf16 tensor [len(gpos), H, d] holding rows ``gpos`` (any order)."""
        gpos = np.asarray(gpos, dtype=np.int64)
        H = self.heads[name]
        out = np.empty((gpos.size, H, self.d), dtype=np.float32)
        if gpos.size:
            blocks = gpos // BLOCK
            for b in np.unique(blocks):
                sel = np.nonzero(blocks == b)[0]
                out[sel] = self._block(name, int(b))[gpos[sel] - b * BLOCK]
        return torch.from_numpy(out).to(torch.bfloat16)
