"""Test cases for the GPU path: seeded workloads (full size or a scaled-down
context of the same recipe), the plan and rank they name, and inputs drawn
by the seeded generator. Shared by the GPU parity tests and the smoke check;
holds no attention arithmetic."""
from __future__ import annotations

import dataclasses

import numpy as np

from oracle import planner as OP
from oracle import view as OV
from paper_2606_08476_amd import synth


@dataclasses.dataclass
class Case:
    name: str
    cu: np.ndarray
    plan: np.ndarray
    cp: int
    rank: int
    hq: int
    hkv: int
    d: int
    seed: int
    oview: OV.RankView
    tiles: tuple | None = None


def make_case(name, workload, context=None, cp=None, rank=None, hq=None, hkv=None, d=None,
              seed=None, lens=None, plan=None, tiles=None) -> Case:
    w = synth.WORKLOADS[workload]
    cp = w.cp if cp is None else cp
    if lens is None:
        lens = synth.doc_lengths(workload, context=context, seed=seed)
    cu = synth.cu_seqlens(lens)
    kind = w.plan if plan is None else plan
    if kind == "per_seq":
        plan = OP.plan_per_seq(cu, cp)
    elif kind == "per_doc":
        plan = OP.plan_per_doc(cu, cp)
    elif kind == "whole_lpt":
        plan = OP.plan_whole_lpt(cu, cp)
    else:
        plan = OP.plan_hybrid(cu, cp)[0]
    if rank is None:
        if w.rank == "last":
            rank = cp - 1
        elif w.rank == "heaviest":
            work = OP.stats(cu, cp, plan, 1, 1)["work"]
            rank = int(np.argmax(work))
        else:
            rank = int(w.rank)
    return Case(name, cu, plan, cp, rank, hq or w.hq, hkv or w.hkv, d or w.d,
                w.index if seed is None else seed, OV.rank_view(cu, plan, rank), tiles)


def inputs(case: Case):
    """bf16 CPU tensors: q and dO at the rank's queries; k and v for local and
    received rows; the packed K/V the gather reads (rows the rank never
    needs are left zero)."""
    src = synth.TensorSource(case.seed, case.hq, case.hkv, case.d)
    qg, rg = case.oview.q_gpos, case.oview.recv_gpos
    T = int(case.cu[-1])
    q = src.rows("q", qg)
    do = src.rows("do", qg)
    k_loc, v_loc = src.rows("k", qg), src.rows("v", qg)
    k_recv, v_recv = src.rows("k", rg), src.rows("v", rg)
    import torch
    k_pk = torch.zeros((T, case.hkv, case.d), dtype=torch.bfloat16)
    v_pk = torch.zeros((T, case.hkv, case.d), dtype=torch.bfloat16)
    k_pk[qg], v_pk[qg] = k_loc, v_loc
    if rg.size:
        k_pk[rg], v_pk[rg] = k_recv, v_recv
    return dict(q=q, do=do, k_loc=k_loc, v_loc=v_loc, k_recv=k_recv, v_recv=v_recv,
                k_pk=k_pk, v_pk=v_pk)


SMALL = {
    "tiny": dict(workload="tiny"),
    "llama8b_8k": dict(workload="llama8b", context=8192),
    "wholedoc_16k": dict(workload="wholedoc", context=16384),
    "longdoc_16k": dict(workload="longdoc", context=16384),
    "hybrid70b_16k": dict(workload="hybrid70b", context=16384),
    # the Llama3 CP baseline plan (chunks of the whole sequence) through the
    # same kernels
    "llama8b_8k_per_seq": dict(workload="llama8b", context=8192, plan="per_seq"),
    # other grouped-query shapes through the same kernels
    "llama8b_8k_g2": dict(workload="llama8b", context=8192, hq=16, hkv=8),
    "llama8b_8k_g1": dict(workload="llama8b", context=8192, hq=8, hkv=8, rank=5),
    "tiny_d64_g8": dict(workload="tiny", hq=16, hkv=2),
    # many one-token and short documents
    "short_docs": dict(workload="llama8b", cp=2, rank=1,
                       lens=[1, 1, 3, 1, 70, 1, 2, 129, 1, 64, 5, 250, 1, 31]),
    # documents whose Per-Doc chunks are whole multiples of the 64-key and
    # 128-key tiles: no ragged tile anywhere, masks exactly on tile edges
    "aligned_docs": dict(workload="llama8b", cp=2, rank=0,
                         lens=[512, 1024, 256, 2048, 512]),
    # forward / dQ query tiles of 64 and 128 rows (2 and 1 heads per workgroup)
    "llama8b_8k_bm64": dict(workload="llama8b", context=8192, tiles=(64, 0, 0, 0)),
    "longdoc_16k_bm128": dict(workload="longdoc", context=16384, tiles=(128, 0, 0, 0)),
}


def small_case(key) -> Case:
    kw = dict(SMALL[key])
    return make_case(key, kw.pop("workload"), **kw)
