"""The launch tables the kernels read (fc_view_export_launch: copies of the
uploaded blob), checked on the CPU against the canonical tile maps and the
receive limits, by brute force rather than by the formulas that built them:

* each forward launch list is a permutation of its map-order list, largest
  first (key tiles of the item);
* every backward map item appears in the launch list either whole (slot -1)
  or as parts whose query ranges are consecutive runs of whole query tiles
  that cover the item's range exactly once; each part owns one partial slot,
  every slot is owned once, and each split item has one reduce entry naming
  exactly its parts' slots, in query order;
* bwd_qfirst of every launch item and 32-key wave equals the first query row
  of the part that sees the wave's first key, found by scanning the rows
  (local keys: the key's own row onward; received keys: rows whose receive
  limit exceeds the key);
* every index lies inside t_q, t_recv and the slot count.
"""
import numpy as np
import pytest

from oracle import planner as P
from oracle import view as V
from paper_2606_08476_amd import flashcp as F
from paper_2606_08476_amd import synth


def _cost_fwd(items, bn):
    return -(-(items[:, 3] - items[:, 2]) // bn) - (-(items[:, 5] - items[:, 4]) // bn)


def _rows(a):
    return sorted(map(tuple, a.tolist()))


def check_view(cu, plan, cp, rank, hq, hkv, d):
    v = F.View(cu, plan, cp, rank, hq, hkv, d)
    i = v.info
    e = v.export()
    L = v.export_launch()
    tq, tr = i["t_q"], i["t_recv"]
    lim = e["lim"].astype(np.int64)
    G = hq // hkv

    # forward launch lists
    for mode in ("local", "recv", "fused"):
        m, l = e["fwd_" + mode], L["fwd_" + mode]
        assert _rows(m) == _rows(l), mode
        c = _cost_fwd(l, i["bn_fwd"])
        assert (np.diff(c) <= 0).all(), mode
        if l.size:
            assert (l[:, 0] >= 0).all() and (l[:, 1] <= tq).all() and (l[:, 0] < l[:, 1]).all()
            assert (l[:, 2] >= 0).all() and (l[:, 3] <= tr).all() and (l[:, 2] <= l[:, 3]).all()
            assert (l[:, 4] >= 0).all() and (l[:, 5] <= tq).all() and (l[:, 4] <= l[:, 5]).all()

    # backward launch list against the map-order items
    bl, red, qf = L["bwd_launch"], L["bwd_reduce"], L["bwd_qfirst"]
    nslots = i["n_bwd_slots"]
    bm, bn = i["bm_bwd"], i["bn_bwd"]
    assert bl.shape[0] == i["n_bwd_launch"] and red.shape[0] == i["n_bwd_reduce"]
    owners = {}
    by_tile = {}
    for r in bl.tolist():
        k0, k1, q0, q1, qfull, src, seg, slot = r
        assert 0 <= k0 < k1 <= (tr if src else tq) and k1 - k0 <= bn
        assert 0 <= q0 < q1 <= tq
        by_tile.setdefault((src, k0), []).append(r)
        if slot >= 0:
            assert slot < nslots and slot not in owners
            owners[slot] = (src, k0, q0)
    assert sorted(owners) == list(range(nslots))
    reduce_of = {(s, k0): (k1, s0, ns) for s, k0, k1, s0, ns, _, _, _ in red.tolist()}
    assert len(reduce_of) == red.shape[0]
    for item in e["bwd"].tolist():
        k0, k1, q0, q1, qfull, src, seg, _ = item
        parts = sorted(by_tile.pop((src, k0)), key=lambda r: r[2])
        assert all(p[1] == k1 and p[4] == qfull and p[6] == seg for p in parts)
        if len(parts) == 1 and parts[0][7] == -1:
            assert parts[0][2:4] == [q0, q1] and (src, k0) not in reduce_of
            continue
        # split: consecutive whole query tiles covering [q0, q1) once
        assert parts[0][2] == q0 and parts[-1][3] == q1
        for a, b in zip(parts, parts[1:]):
            assert a[3] == b[2] and (a[3] - q0) % bm == 0
        k1r, s0, ns = reduce_of.pop((src, k0))
        assert k1r == k1 and [p[7] for p in parts] == list(range(s0, s0 + ns))
    assert not by_tile and not reduce_of

    # first query row that sees each wave's first key, by scanning rows
    assert qf.shape == (bl.shape[0], bn // 32)
    for r, row in zip(bl.tolist(), qf.tolist()):
        k0, k1, q0, q1, _, src, _, _ = r
        for w, got in enumerate(row):
            kw = k0 + 32 * w
            if not src:
                want = kw   # a local key is seen by its own row onward
            else:
                want = next((t for t in range(q0, q1) if lim[t] > kw), q1)
            assert got == want, (r, w)
    v.close()


def _random(ncase, seed):
    rng = np.random.default_rng(seed)
    for _ in range(ncase):
        n = int(rng.integers(1, 12))
        lens = rng.integers(1, 900, size=n)
        cp = int(rng.integers(1, 6))
        lens[-1] += (-lens.sum()) % cp
        yield np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), cp


def test_launch_tables_random():
    for cu, cp in _random(25, seed=31):
        for plan in (P.plan_per_doc(cu, cp), P.plan_hybrid(cu, cp)[0], P.plan_per_seq(cu, cp)):
            for r in range(cp):
                for hq, hkv in ((4, 4), (16, 2)):
                    check_view(cu, plan, cp, r, hq, hkv, 64)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_launch_tables_workloads(name):
    w = synth.WORKLOADS[name]
    cu = synth.cu_seqlens(synth.doc_lengths(name))
    plan = {"per_doc": P.plan_per_doc, "whole_lpt": P.plan_whole_lpt}.get(
        w.plan, lambda c, n: P.plan_hybrid(c, n)[0])(cu, w.cp)
    work = P.stats(cu, w.cp, plan, 1, 1)["work"]
    rank = {"last": w.cp - 1, "heaviest": int(np.argmax(work))}.get(w.rank, None)
    rank = int(w.rank) if rank is None else rank
    check_view(cu, plan, w.cp, rank, w.hq, w.hkv, w.d)
