"""Oracle rank view and tile maps.

Test infrastructure only (see the package docstring).

Rank view (FlashCP Sec. 3.1 for shards and prefixes, Sec. 3.2 for the
sharding-aware receive set, Sec. 2.1 for the document mask):

* documents have lengths d_k and starts c_k; position g lies in doc(g);
* a query at g sees keys V(g) = {u : c_doc(g) <= u <= g} (intra-document
  causal mask, diagonal included: the count of such pairs over a shard is
  exactly W_i of Eq. 3);
* rank r's queries Q_r are its shards' positions in ascending order; this
  order is the rank's *local* order;
* the KV it must hold is H_r = union of V(g) over Q_r; the received set is
  R_r = H_r minus Q_r, compacted in ascending position (one contiguous
  buffer, no per-document padding, Sec. 3.2).

Derived structure used by the kernels (a consequence of the definitions):

* a *segment* is the run of local tokens of one document (contiguous in
  local order); inside it a query at local index i sees exactly the local
  keys j with seg_start <= j <= i;
* a *piece* is a maximal run of consecutive positions held by the rank
  inside one document; no received token lies inside a piece, so all its
  queries see the same first n_P received tokens of their document.

Tile maps are this build's own scheduling structure, not the paper's. Each
list is defined here from the visibility rule by corner checks on each
(query tile, key tile) block; tests expand them back into the mask.

Parity: pinned by brute force against the explicit mask (every visible pair
covered exactly once, no invisible pair in a block marked unmasked) and by
the integer identity pairs_local + pairs_recv = sum of W over the rank's
shards.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class RankView:
    q_gpos: np.ndarray      # int64 [T_q] global positions of local queries
    recv_gpos: np.ndarray   # int64 [T_r] global positions of received keys
    seg_doc: np.ndarray     # int64 [S]
    q_cu_docseg: np.ndarray  # int64 [S+1] local index bounds of segments
    recv_cu: np.ndarray     # int64 [S+1] received index bounds per segment
    pieces: np.ndarray      # int64 [P, 5]: seg, q_start, q_end, g_start, n_P
    lim: np.ndarray         # int64 [T_q] received-index end visible to each query
    pairs_loc: int
    pairs_recv: int


def doc_of(cu, g):
    return int(np.searchsorted(np.asarray(cu), g, side="right") - 1)


def rank_view(cu, plan, rank: int) -> RankView:
    cu = np.asarray(cu, dtype=np.int64)
    plan = np.asarray(plan, dtype=np.int64).reshape(-1, 4)
    mine = plan[plan[:, 1] == rank]
    pos = []
    for dd, _, o, l in mine:
        pos.extend(range(int(cu[dd] + o), int(cu[dd] + o + l)))
    q_gpos = np.asarray(sorted(pos), dtype=np.int64)
    held = set(q_gpos.tolist())
    # H_r = union over queries of [c_doc(g), g]
    need_hi = {}
    for g in q_gpos.tolist():
        k = doc_of(cu, g)
        need_hi[k] = max(need_hi.get(k, -1), g)
    docs = sorted(need_hi)
    recv = []
    recv_cu = [0]
    q_cu = [0]
    for k in docs:
        seg_recv = [u for u in range(int(cu[k]), need_hi[k] + 1) if u not in held]
        recv += seg_recv
        recv_cu.append(len(recv))
        q_cu.append(q_cu[-1] + int(sum(1 for g in q_gpos if cu[k] <= g < cu[k + 1])))
    recv_gpos = np.asarray(recv, dtype=np.int64)
    pieces = []
    lim = np.zeros(q_gpos.size, dtype=np.int64)
    for s, k in enumerate(docs):
        i = q_cu[s]
        while i < q_cu[s + 1]:
            j = i + 1
            while j < q_cu[s + 1] and q_gpos[j] == q_gpos[j - 1] + 1:
                j += 1
            g0 = int(q_gpos[i])
            seg_recv = recv_gpos[recv_cu[s]:recv_cu[s + 1]]
            n_p = int(np.count_nonzero(seg_recv < g0))
            pieces.append((s, i, j, g0, n_p))
            lim[i:j] = recv_cu[s] + n_p
            i = j
    seg_lens = np.diff(np.asarray(q_cu, dtype=np.int64))
    pairs_loc = int(sum(int(x) * (int(x) + 1) // 2 for x in seg_lens))
    pairs_recv = int(sum((p[2] - p[1]) * p[4] for p in pieces))
    return RankView(q_gpos, recv_gpos, np.asarray(docs, dtype=np.int64),
                    np.asarray(q_cu, dtype=np.int64), np.asarray(recv_cu, dtype=np.int64),
                    np.asarray(pieces, dtype=np.int64).reshape(-1, 5), lim,
                    pairs_loc, pairs_recv)


# ---------------------------------------------------------------- tile maps
#
# Visibility in local/received index space (equivalent to V(g) restricted to
# one source, by the derived structure above):
#   local  key j for local query i : same segment and j <= i
#   recv   key r for local query i : recv_cu[seg(i)] <= r < lim[i]


def seg_of_local(view: RankView) -> np.ndarray:
    """Segment index of every local query row."""
    if getattr(view, "_seg", None) is None:
        view._seg = np.repeat(np.arange(len(view.seg_doc)), np.diff(view.q_cu_docseg))
    return view._seg


def vis_local(view: RankView, rows: np.ndarray, j: int) -> np.ndarray:
    """Which local query rows see local key j."""
    seg = seg_of_local(view)
    return (seg[rows] == seg[j]) & (j <= rows)


def vis_recv(view: RankView, rows: np.ndarray, r: int) -> np.ndarray:
    """Which local query rows see received key r."""
    seg = seg_of_local(view)
    return (view.recv_cu[seg[rows]] <= r) & (r < view.lim[rows])


def fwd_items(view: RankView, bm: int, bn: int, mode: str) -> np.ndarray:
    """Forward work items, int32 [n, 8]: (q0, q1, r0, r1, l0, l1, ldiag, seg).

    Query rows [q0, q1) see received keys [r0, r1) with no mask, and local
    keys [l0, l1) where key tiles l0 + t*bn starting below ``ldiag`` are
    fully visible and those from ``ldiag`` on need the causal mask.

    mode "local": query tiles cut per segment, local keys only.
    mode "recv":  query tiles cut per piece, received keys only (pieces
                  with n_P = 0 give items with an empty key range).
    mode "fused": query tiles cut per piece, both sources.
    """
    out = []
    if mode == "local":
        for s in range(len(view.seg_doc)):
            s0, s1 = int(view.q_cu_docseg[s]), int(view.q_cu_docseg[s + 1])
            for t0 in range(s0, s1, bm):
                t1 = min(t0 + bm, s1)
                out.append((t0, t1, 0, 0) + _local_range(view, s0, t0, t1, bn) + (s,))
        return np.asarray(out, dtype=np.int32).reshape(-1, 8)
    for s, q_start, q_end, _, n_p in view.pieces.tolist():
        s0 = int(view.q_cu_docseg[s])
        r0 = int(view.recv_cu[s])
        for t0 in range(q_start, q_end, bm):
            t1 = min(t0 + bm, q_end)
            rows = np.arange(t0, t1)
            # every row of the tile sees exactly the received keys [r0, r0 + n_p)
            if n_p:
                assert vis_recv(view, rows, r0 + n_p - 1).all() and vis_recv(view, rows, r0).all()
            assert not vis_recv(view, rows, r0 + n_p).any() and not vis_recv(view, rows, r0 - 1).any()
            if mode == "recv":
                out.append((t0, t1, r0, r0 + n_p, 0, 0, 0, s))
            else:
                out.append((t0, t1, r0, r0 + n_p) + _local_range(view, s0, t0, t1, bn) + (s,))
    return np.asarray(out, dtype=np.int32).reshape(-1, 8)


def _local_range(view, s0, t0, t1, bn):
    """Key range [s0, t1) of query tile [t0, t1) and the first masked tile."""
    rows = np.arange(t0, t1)
    ldiag = None
    for k0 in range(s0, t1, bn):
        keys = range(k0, min(k0 + bn, t1))
        assert any(vis_local(view, rows, j).any() for j in keys)   # block not empty
        full = (k0 + bn <= t1) and all(vis_local(view, rows, j).all() for j in keys)
        if full:
            assert ldiag is None, "a fully visible tile after a masked one"
        elif ldiag is None:
            ldiag = k0
    assert not vis_local(view, rows, t1).any() if t1 < len(view.q_gpos) else True
    return (s0, t1, t1 if ldiag is None else ldiag)


def bwd_items(view: RankView, bm: int, bn: int) -> np.ndarray:
    """Backward work items (key-major), int32 [n, 8]:
    (k0, k1, q0, q1, qfull, src, seg, 0).

    Key rows [k0, k1) of source ``src`` (0 local, 1 received) are seen by
    query rows [q0, q1) and by no other row; query tiles q0 + t*bm starting
    at or after ``qfull`` see every key of the key tile, earlier ones need
    the mask.
    """
    out = []
    S = len(view.seg_doc)
    for src in (0, 1):
        for s in range(S):
            s0, s1 = int(view.q_cu_docseg[s]), int(view.q_cu_docseg[s + 1])
            if src == 0:
                lo, hi, vis = s0, s1, vis_local
            else:
                lo, hi, vis = int(view.recv_cu[s]), int(view.recv_cu[s + 1]), vis_recv
            # a key is only ever seen by queries of its own document
            allrows = np.arange(s0, s1)
            for k0 in range(lo, hi, bn):
                k1 = min(k0 + bn, hi)
                sees_any = np.zeros(allrows.size, dtype=bool)
                sees_all = np.ones(allrows.size, dtype=bool)
                for j in range(k0, k1):
                    v = vis(view, allrows, j)
                    sees_any |= v
                    sees_all &= v
                rows = s0 + np.nonzero(sees_any)[0]
                q0, q1 = int(rows[0]), int(rows[-1]) + 1
                assert rows.size == q1 - q0, "rows seeing a key tile are contiguous"
                qfull = q1
                for t0 in range(q0, q1, bm):
                    if sees_all[t0 - s0:min(t0 + bm, q1) - s0].all():
                        qfull = t0
                        break
                assert sees_all[qfull - s0:q1 - s0].all()
                out.append((k0, k1, q0, q1, qfull, src, s, 0))
    return np.asarray(out, dtype=np.int32).reshape(-1, 8)
