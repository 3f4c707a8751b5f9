"""Whole-method invariants of the oracle (fp64): sharding changes nothing but
where each token's result is computed (FlashCP Sec. 3: every plan computes
the same document-masked attention, only distributed differently)."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import planner as P
from oracle import view as V
from paper_2606_08476_amd import synth

TOL = 1e-10


def _per_seq_plan(cu, N):
    """Llama3-style sharding: the whole sequence cut into 2N equal pieces,
    worker i taking pieces i and 2N-1-i, expressed as per-document shards."""
    cu = np.asarray(cu)
    T = int(cu[-1])
    rows = []
    for i in range(2 * N):
        a, b = (i * T) // (2 * N), ((i + 1) * T) // (2 * N)
        r = i if i < N else 2 * N - 1 - i
        for k in range(len(cu) - 1):
            lo, hi = max(a, int(cu[k])), min(b, int(cu[k + 1]))
            if hi > lo:
                rows.append((k, r, lo - int(cu[k]), hi - lo))
    return P.canonical(rows)


def _setup(seed=0, lens=(70, 9, 130, 1, 46), hq=4, hkv=2, d=8):
    lens = list(lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    src = synth.TensorSource(seed, hq, hkv, d)
    T = int(cu[-1])
    g = np.arange(T)
    return cu, src.rows("q", g), src.rows("k", g), src.rows("v", g), src.rows("do", g)


def _rank_results(cu, plan, N, q, k, v, do, scale):
    """Per-rank forward (two partial passes + merge) and backward, scattered
    back to global positions."""
    T, hq, d = q.shape
    hkv = k.shape[1]
    O = torch.zeros(T, hq, d, dtype=torch.float64)
    L = torch.zeros(hq, T, dtype=torch.float64)
    dQ = torch.zeros(T, hq, d, dtype=torch.float64)
    dK = torch.zeros(T, hkv, d, dtype=torch.float64)
    dV = torch.zeros(T, hkv, d, dtype=torch.float64)
    for r in range(N):
        v_ = V.rank_view(cu, plan, r)
        qg, rg = v_.q_gpos, v_.recv_gpos
        if qg.size == 0:
            continue
        kv = np.concatenate([qg, rg])
        Oa, La = A.attention_fwd(cu, qg, q[qg], qg, k[qg], v[qg], scale)
        Ob, Lb = A.attention_fwd(cu, qg, q[qg], rg, k[rg], v[rg], scale)
        Om, Lm = A.lse_merge(Oa, La, Ob, Lb)
        Os, Ls = A.attention_fwd(cu, qg, q[qg], kv, k[kv], v[kv], scale)
        assert torch.allclose(Om, Os, atol=TOL) and torch.allclose(Lm, Ls, atol=TOL)
        O[qg], L[:, qg] = Om, Lm
        dq, dk, dv = A.attention_bwd(cu, qg, q[qg], kv, k[kv], v[kv], do[qg], scale)
        dQ[qg] = dq
        dK.index_add_(0, torch.from_numpy(kv), dk)
        dV.index_add_(0, torch.from_numpy(kv), dv)
    return O, L, dQ, dK, dV


@pytest.mark.parametrize("N", [2, 4])
def test_all_plans_equal_unsharded(N):
    cu, q, k, v, do = _setup()
    T = int(cu[-1])
    lens = np.diff(cu)
    if T % N:
        pytest.skip("hybrid needs N | C")
    scale = 0.35
    g = np.arange(T)
    O1, L1 = A.attention_fwd(cu, g, q, g, k, v, scale)
    dq1, dk1, dv1 = A.attention_bwd(cu, g, q, g, k, v, do, scale)
    plans = {
        "per_doc": P.plan_per_doc(cu, N),
        "whole_lpt": P.plan_whole_lpt(cu, N),
        "hybrid": P.plan_hybrid(cu, N)[0],
        "per_seq": _per_seq_plan(cu, N),
    }
    assert len(lens) == 5
    for name, plan in plans.items():
        P.validate(cu, N, plan)
        O, L, dQ, dK, dV = _rank_results(cu, plan, N, q, k, v, do, scale)
        for a, b in ((O, O1), (L, L1), (dQ, dq1), (dK, dk1), (dV, dv1)):
            assert (a - b).abs().max() <= TOL, name


def test_document_isolation():
    """Changing another document's Q/K/V/dO leaves a document's outputs
    bit-identical (the document mask of Sec. 2.1)."""
    cu, q, k, v, do = _setup(seed=3)
    T = int(cu[-1])
    plan = P.plan_per_doc(cu, 2)
    base = _rank_results(cu, plan, 2, q, k, v, do, 0.3)
    d0 = slice(int(cu[2]), int(cu[3]))        # perturb document 2
    q2, k2, v2, do2 = (x.clone() for x in (q, k, v, do))
    for x in (q2, k2, v2, do2):
        x[d0] = (x[d0].float() * -1.5 + 0.25).to(torch.bfloat16)
    pert = _rank_results(cu, plan, 2, q2, k2, v2, do2, 0.3)
    keep = np.r_[0:int(cu[2]), int(cu[3]):T]
    for a, b in zip(base, pert):
        if a.shape[0] == T:
            assert torch.equal(a[keep], b[keep])
        else:
            assert torch.equal(a[:, keep], b[:, keep])
    assert not torch.equal(base[0][d0], pert[0][d0])


def test_work_equals_sum_of_shard_workloads_on_workloads():
    """pairs_local + pairs_recv of a rank = sum of W_i over its shards (Eq. 3)
    on every workload's planned rank."""
    for name, w in synth.WORKLOADS.items():
        cu = synth.cu_seqlens(synth.doc_lengths(name))
        if w.plan == "per_doc":
            plan = P.plan_per_doc(cu, w.cp)
        elif w.plan == "whole_lpt":
            plan = P.plan_whole_lpt(cu, w.cp)
        else:
            plan = P.plan_hybrid(cu, w.cp)[0]
        st = P.stats(cu, w.cp, plan, w.hkv, w.d)
        for r in (0, w.cp - 1):
            v_ = V.rank_view(cu, plan, r)
            assert v_.pairs_loc + v_.pairs_recv == st["work"][r]
            assert len(v_.recv_gpos) == st["recv_tokens"][r]
