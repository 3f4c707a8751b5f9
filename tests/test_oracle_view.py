"""Pins of the oracle rank view and tile maps against brute force over the
explicit document mask."""
import numpy as np
import pytest

from oracle import planner as P
from oracle import view as V
from paper_2606_08476_amd import synth


def _cu(lens):
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)


def _visible(cu, g, u):
    dg = np.searchsorted(cu, g, side="right") - 1
    du = np.searchsorted(cu, u, side="right") - 1
    return dg == du and u <= g


def _small_cases():
    rng = np.random.default_rng(2)
    cases = []
    for _ in range(6):
        N = int(rng.choice([2, 3, 4]))
        lens = [int(x) for x in rng.integers(1, 90, size=int(rng.integers(1, 6)))]
        lens[-1] += (-sum(lens)) % N
        cu = _cu(lens)
        for plan in (P.plan_per_doc(cu, N), P.plan_whole_lpt(cu, N), P.plan_hybrid(cu, N)[0]):
            cases.append((cu, N, plan))
    return cases


def test_view_against_definition_brute_force():
    for cu, N, plan in _small_cases():
        T = int(cu[-1])
        seen = np.zeros(T, dtype=int)
        for r in range(N):
            v = V.rank_view(cu, plan, r)
            seen[v.q_gpos] += 1
            Q = set(v.q_gpos.tolist())
            H = {u for g in Q for u in range(T) if _visible(cu, g, u)}
            assert set(v.recv_gpos.tolist()) == H - Q           # R_r = H_r \ Q_r
            assert list(v.recv_gpos) == sorted(v.recv_gpos)     # compacted ascending
            assert list(v.q_gpos) == sorted(v.q_gpos)
            pairs = sum(1 for g in Q for u in range(T) if _visible(cu, g, u))
            assert v.pairs_loc + v.pairs_recv == pairs
            assert pairs == P.stats(cu, N, plan, 1, 1)["work"][r]   # = sum of W_i (Eq. 3)
            assert len(v.recv_gpos) == P.stats(cu, N, plan, 1, 1)["recv_tokens"][r]
            # per-query received limit: exactly the received keys it sees
            for i, g in enumerate(v.q_gpos):
                vis_r = [j for j, u in enumerate(v.recv_gpos) if _visible(cu, g, u)]
                s = np.searchsorted(v.q_cu_docseg, i, side="right") - 1
                assert vis_r == list(range(int(v.recv_cu[s]), int(v.lim[i])))
        assert (seen == 1).all()                                # Eq. 1


def _expand_fwd(view, items, bn):
    """(query, source, key) triples covered by forward items, and the subset
    claimed to need no mask."""
    cover, nomask = [], []
    for q0, q1, r0, r1, l0, l1, ld, _ in items.tolist():
        for i in range(q0, q1):
            for r in range(r0, r1):
                cover.append((i, 1, r))
                nomask.append((i, 1, r))
            for k0 in range(l0, l1, bn):
                for j in range(k0, min(k0 + bn, l1)):
                    cover.append((i, 0, j))
                    if k0 < ld:
                        nomask.append((i, 0, j))
    return cover, nomask


def _vis_triple(view, cu, i, src, j):
    g = view.q_gpos[i]
    u = view.recv_gpos[j] if src else view.q_gpos[j]
    return _visible(cu, g, u)


@pytest.mark.parametrize("bm,bn", [(4, 8), (32, 64), (7, 5)])
def test_fwd_tiles_cover_mask_exactly(bm, bn):
    for cu, N, plan in _small_cases()[:9]:
        for r in range(N):
            view = V.rank_view(cu, plan, r)
            vis = {(i, s, j) for i in range(len(view.q_gpos))
                   for s, n in ((0, len(view.q_gpos)), (1, len(view.recv_gpos)))
                   for j in range(n) if _vis_triple(view, cu, i, s, j)}
            loc = {t for t in vis if t[1] == 0}
            rcv = {t for t in vis if t[1] == 1}
            for mode, want in (("local", loc), ("recv", rcv), ("fused", vis)):
                items = V.fwd_items(view, bm, bn, mode)
                cover, nomask = _expand_fwd(view, items, bn)
                # every visible pair appears exactly once among unmasked-or-visible entries
                visible_cover = [t for t in cover if _vis_triple(view, cu, *t)]
                assert sorted(visible_cover) == sorted(want)
                assert all(_vis_triple(view, cu, *t) for t in nomask)
                # each query row appears in exactly one item (its output row is written once)
                rows = [i for q0, q1, *_ in items.tolist() for i in range(q0, q1)]
                assert sorted(rows) == list(range(len(view.q_gpos)))


@pytest.mark.parametrize("bm,bn", [(4, 8), (32, 128), (5, 3)])
def test_bwd_tiles_cover_mask_exactly(bm, bn):
    for cu, N, plan in _small_cases()[:9]:
        for r in range(N):
            view = V.rank_view(cu, plan, r)
            items = V.bwd_items(view, bm, bn)
            got = []
            for k0, k1, q0, q1, qf, src, _, _ in items.tolist():
                for j in range(k0, k1):
                    for i in range(q0, q1):
                        if _vis_triple(view, cu, i, src, j):
                            got.append((i, src, j))
                        else:
                            assert i < qf        # an invisible pair only in masked tiles
                    # rows outside [q0, q1) see nothing of this key
                    for i in list(range(0, q0)) + list(range(q1, len(view.q_gpos))):
                        assert not _vis_triple(view, cu, i, src, j)
            want = [(i, s, j) for i in range(len(view.q_gpos))
                    for s, n in ((0, len(view.q_gpos)), (1, len(view.recv_gpos)))
                    for j in range(n) if _vis_triple(view, cu, i, s, j)]
            assert sorted(got) == sorted(want)
            # every key row of both sources belongs to exactly one item
            keys = sorted((src, j) for k0, k1, _, _, _, src, _, _ in items.tolist() for j in range(k0, k1))
            assert keys == [(0, j) for j in range(len(view.q_gpos))] + \
                [(1, j) for j in range(len(view.recv_gpos))]


def test_tiny_workload_rank0_structure():
    """Tiny workload: N = 2 Per-Doc, rank 0 holds chunks 0 and 3 of each doc;
    chunk 3 sees chunks 1-2 as received KV, chunk 0 sees none."""
    lens = synth.doc_lengths("tiny")
    cu = synth.cu_seqlens(lens)
    plan = P.plan_per_doc(cu, 2)
    v = V.rank_view(cu, plan, 0)
    assert len(v.pieces) == 6
    for (s, qs, qe, g0, n_p), k in zip(v.pieces.tolist(), np.repeat(range(3), 2)):
        L = int(lens[k])
        b = [(j * L) // 4 for j in range(5)]
        if qs == v.q_cu_docseg[s]:
            assert g0 == cu[k] + b[0] and n_p == 0 and qe - qs == b[1] - b[0]
        else:
            assert g0 == cu[k] + b[3] and n_p == b[3] - b[1] and qe - qs == b[4] - b[3]
