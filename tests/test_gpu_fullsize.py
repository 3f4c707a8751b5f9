"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (gather; both forward partial passes in one launch; LSE
merge; preprocess; dK/dV and dQ workgroups in one launch), against the fp64
oracle on outputs it can compute one by one:

* O, LSE and dQ on sampled query rows (every head), including the first and
  last rows of pieces;
* dK and dV on every key of a few whole documents (the oracle backward
  restricted to a document's queries is exact for that document's keys);
* the gathered K/V bit-exact; every output finite.

Tolerances as in test_gpu_parity.py.
"""
import sys

import numpy as np
import pytest
import torch

import _cases
from oracle import attention as A
from oracle import planner as OP
from paper_2606_08476_amd import flashcp as F
from paper_2606_08476_amd import synth

pytestmark = pytest.mark.gpu

TOL = 2e-2
LSE_TOL = 1e-3


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    F.lib()
    return torch.device("cuda:0")


def _sample_rows(view, rng, n=48):
    rows = set()
    for s, qs, qe, _, _ in view.pieces.tolist():
        rows.update((qs, qe - 1))
    rows = sorted(rows)
    rng.shuffle(rows)
    rows = rows[: n // 2]
    rows += rng.choice(len(view.q_gpos), size=n - len(rows), replace=False).tolist()
    return np.unique(np.asarray(rows, dtype=np.int64))


def _check_segments(view, nmax=3):
    """The cheapest document segments by oracle cost, a mid-sized one and the
    largest one (when the oracle can afford it: on the Whole-Doc workload its
    key tiles are the ones the backward splits across workgroups)."""
    qcu, rcu = view.q_cu_docseg, view.recv_cu
    cost = [(int(qcu[s + 1] - qcu[s]) * int(qcu[s + 1] - qcu[s] + rcu[s + 1] - rcu[s]), s)
            for s in range(len(view.seg_doc))]
    cost.sort()
    pick = [s for _, s in cost[:nmax - 1]]
    for c, s in (cost[len(cost) // 2], cost[-1]):   # a mid-sized and the largest document
        if s not in pick and c < 4e7:
            pick.append(s)
    return pick


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_full_size(name, dev):
    case = _cases.make_case(name, name)
    w = synth.WORKLOADS[name]
    # the product planner agrees with the oracle on the full workload
    plan_c = {"per_doc": F.fc_plan_per_doc, "whole_lpt": F.fc_plan_whole_lpt}.get(
        w.plan, lambda cu, n: F.fc_plan_hybrid(cu, n)[0])(case.cu, case.cp)
    assert np.array_equal(plan_c, case.plan)
    say(f"[gpu-full] {name}: rank {case.rank}, t_q {case.oview.q_gpos.size}, t_recv {case.oview.recv_gpos.size}")
    x = _cases.inputs(case)
    xd = {k: v.to(dev) for k, v in x.items()}
    v = F.View(case.cu, plan_c, case.cp, case.rank, case.hq, case.hkv, case.d).bind(dev)
    i = v.info
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], case.hq, case.hkv, case.d
    bf, f32 = torch.bfloat16, torch.float32
    e = lambda *s, dt=f32: torch.empty(*s, dtype=dt, device=dev)
    kl, vl, kr, vr = e(tq, hkv, d, dt=bf), e(tq, hkv, d, dt=bf), e(tr, hkv, d, dt=bf), e(tr, hkv, d, dt=bf)
    F.fc_kv_gather(v, xd["k_pk"], xd["v_pk"], kl, vl, kr, vr)
    oa, ob, la, lb = e(tq, hq, d), e(tq, hq, d), e(hq, tq), e(hq, tq)
    o, lse, delta = e(tq, hq, d, dt=bf), e(hq, tq), e(hq, tq)
    if tr:
        F.fc_attn_fwd_partials(v, xd["q"], kl, vl, kr, vr, 0.0, oa, la, ob, lb)
        F.fc_lse_merge(oa, la, ob, lb, o, None, lse)
    else:
        ws = torch.empty(1, dtype=torch.uint8, device=dev)
        F.fc_attn_fwd(v, xd["q"], kl, vl, kr, vr, 0.0, F.FC_TWO_PASS, o, None, lse, ws)
    F.fc_bwd_preprocess(v, o, xd["do"], delta)
    dq, dkl, dvl, dkr, dvr = e(tq, hq, d), e(tq, hkv, d), e(tq, hkv, d), e(tr, hkv, d), e(tr, hkv, d)
    ws = torch.empty(max(v.workspace_size()[2], 1), dtype=torch.uint8, device=dev)
    F.fc_attn_bwd_pass(v, xd["q"], kl, vl, kr, vr, lse, delta, xd["do"], 0.0, dq, dkl, dvl, dkr, dvr, ws)
    # the separate dK/dV and dQ kernels give the same bits
    dq2, dkl2, dvl2, dkr2, dvr2 = (torch.empty_like(t) for t in (dq, dkl, dvl, dkr, dvr))
    F.fc_attn_bwd_dkdv(v, xd["q"], kl, vl, kr, vr, lse, delta, xd["do"], 0.0, dkl2, dvl2, dkr2, dvr2, ws)
    F.fc_attn_bwd_dq(v, xd["q"], kl, vl, kr, vr, lse, delta, xd["do"], 0.0, dq2)
    torch.cuda.synchronize()
    say(f"[gpu-full] {name}: GPU done")
    for a, b in ((dq, dq2), (dkl, dkl2), (dvl, dvl2), (dkr, dkr2), (dvr, dvr2)):
        assert torch.equal(a, b)

    assert torch.equal(kl.cpu(), x["k_loc"]) and torch.equal(vl.cpu(), x["v_loc"])
    assert torch.equal(kr.cpu(), x["k_recv"]) and torch.equal(vr.cpu(), x["v_recv"])
    for t in (o, lse, dq, dkl, dvl, dkr, dvr):
        assert torch.isfinite(t).all()

    ov = case.oview
    kv = np.concatenate([ov.q_gpos, ov.recv_gpos])
    K = torch.cat([x["k_loc"], x["k_recv"]])
    V = torch.cat([x["v_loc"], x["v_recv"]])
    rng = np.random.default_rng(0)
    rows = _sample_rows(ov, rng)
    O_ref, L_ref = A.attention_fwd(case.cu, ov.q_gpos, x["q"], kv, K, V, rows=rows)
    dq_ref, _, _ = A.attention_bwd(case.cu, ov.q_gpos, x["q"], kv, K, V, x["do"], rows=rows)
    eo = float((o.cpu()[rows].double() - O_ref[rows]).abs().max())
    el = float(((lse.cpu()[:, rows].double() - L_ref[:, rows]).abs() / L_ref[:, rows].abs().clamp_min(1)).max())
    eq = float((dq.cpu()[rows].double() - dq_ref[rows]).abs().max())
    say(f"[gpu-full] {name}: {rows.size} rows: O {eo:.3e} LSE {el:.3e} dQ {eq:.3e}")
    assert eo <= TOL and el <= LSE_TOL and eq <= TOL

    for s in _check_segments(ov):
        q0, q1 = int(ov.q_cu_docseg[s]), int(ov.q_cu_docseg[s + 1])
        r0, r1 = int(ov.recv_cu[s]), int(ov.recv_cu[s + 1])
        seg_rows = np.arange(q0, q1)
        _, dk_ref, dv_ref = A.attention_bwd(case.cu, ov.q_gpos, x["q"], kv, K, V, x["do"], rows=seg_rows)
        ek = max(float((dkl.cpu()[q0:q1].double() - dk_ref[q0:q1]).abs().max()),
                 float((dkr.cpu()[r0:r1].double() - dk_ref[tq + r0:tq + r1]).abs().max()) if r1 > r0 else 0.0)
        ev = max(float((dvl.cpu()[q0:q1].double() - dv_ref[q0:q1]).abs().max()),
                 float((dvr.cpu()[r0:r1].double() - dv_ref[tq + r0:tq + r1]).abs().max()) if r1 > r0 else 0.0)
        say(f"[gpu-full] {name}: segment {s} ({q1 - q0} local, {r1 - r0} received keys): dK {ek:.3e} dV {ev:.3e}")
        assert ek <= TOL and ev <= TOL
    v.close()
