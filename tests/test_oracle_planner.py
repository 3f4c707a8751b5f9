"""Pins of the oracle planners: closed forms of W and Per-Doc, Eq. 1 and
Eq. 2, hand-worked examples, Graham's LPT bound against brute force, and the
termination rule of Algorithm 1."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import planner as P
from paper_2606_08476_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "planner_hand.json")))


def _cu(lens):
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)


def test_shard_work_counts_visible_pairs():
    """W(p, s) = number of (q, k) pairs with p <= q < p+s, 0 <= k <= q."""
    for p in range(0, 9):
        for s in range(0, 9):
            brute = sum(1 for q in range(p, p + s) for k in range(0, q + 1))
            assert P.shard_work(p, s) == brute


def test_per_doc_chunk_rule():
    """Worker i gets chunks i and 2N-1-i (0-indexed); N=2: rank 0 gets 0 and 3."""
    L, N = 1000, 2
    ch = P.per_doc_chunks(L, N)
    bounds = [0, 250, 500, 750, 1000]
    assert ch == [(0, 0, 250), (1, 250, 250), (1, 500, 250), (0, 750, 250)]
    assert [o for _, o, _ in ch] == bounds[:-1]
    for N in (3, 8, 16):
        ch = P.per_doc_chunks(16 * N * 5, N)
        for i, (r, o, l) in enumerate(ch):
            assert r == (i if i < N else 2 * N - 1 - i)


def test_per_doc_balanced_closed_form():
    """With 2N | L every worker's workload on a doc is c(2Nc+1), c = L/2N,
    so the imbalance is exactly 1."""
    N = 4
    lens = [8 * 3, 8 * 11, 8 * 1, 8 * 40]
    plan = P.plan_per_doc(_cu(lens), N)
    st = P.stats(_cu(lens), N, plan, 1, 1)
    expect = sum((L // 8) * (2 * N * (L // 8) + 1) for L in lens)
    assert st["work"] == [expect] * N
    assert st["imbalance"] == 1.0


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_plans_cover_every_token_once(name):
    w = synth.WORKLOADS[name]
    cu = synth.cu_seqlens(synth.doc_lengths(name))
    for plan in (P.plan_per_doc(cu, w.cp), P.plan_whole_lpt(cu, w.cp)):
        P.validate(cu, w.cp, plan)
    if cu[-1] % w.cp == 0:
        plan, isp = P.plan_hybrid(cu, w.cp)
        P.validate(cu, w.cp, plan, require_equal_tokens=True)   # Eq. 2
        st = P.stats(cu, w.cp, plan, w.hkv, w.d)
        assert st["imbalance"] <= 1.05 or isp.all()
        # whole-doc documents are never Per-Doc chunked
        assert isp.sum() < len(isp) or st["imbalance"] > 1.05


def test_validate_rejects_bad_plans():
    cu = _cu([5, 3])
    ok = np.array([[0, 0, 0, 5], [1, 1, 0, 3]])
    P.validate(cu, 2, ok)
    for bad in ([[0, 0, 0, 4], [1, 1, 0, 3]],             # gap
                [[0, 0, 0, 5], [0, 1, 4, 1], [1, 1, 0, 3]],  # overlap
                [[0, 0, 0, 6], [1, 1, 0, 3]],             # beyond doc
                [[0, 2, 0, 5], [1, 1, 0, 3]]):            # rank >= N
        with pytest.raises(ValueError):
            P.validate(cu, 2, np.array(bad))
    with pytest.raises(ValueError):
        P.validate(cu, 2, ok, require_equal_tokens=True)


def test_lpt_hand_example():
    g = GOLD["lpt"]
    cu = _cu(g["lengths"])
    plan = P.plan_whole_lpt(cu, g["cp"])
    assert plan.tolist() == g["plan"]
    st = P.stats(cu, g["cp"], plan, 1, 1)
    assert st["work"] == g["work"]
    assert st["imbalance"] == 70 * 2 / 133


def _brute_opt(lens, N):
    W = [L * (L + 1) // 2 for L in lens]
    best = None
    for assign in itertools.product(range(N), repeat=len(lens)):
        loads = [0] * N
        for w, a in zip(W, assign):
            loads[a] += w
        m = max(loads)
        best = m if best is None else min(best, m)
    return best


def test_lpt_within_graham_bound_of_brute_force():
    """LPT makespan <= (4/3 - 1/(3N)) * optimum over whole-doc placements
    (Graham 1969); the optimum is found by brute force (N = 2, <= 6 docs)."""
    rng = np.random.default_rng(11)
    for trial in range(60):
        n = int(rng.integers(2, 7))
        lens = [int(x) for x in rng.integers(1, 60, size=n)]
        N = 2
        plan = P.plan_whole_lpt(_cu(lens), N)
        lpt = max(P.stats(_cu(lens), N, plan, 1, 1)["work"])
        opt = _brute_opt(lens, N)
        assert opt <= lpt <= (4 / 3 - 1 / (3 * N)) * opt + 1e-9
    assert _brute_opt(GOLD["lpt"]["lengths"], 2) == GOLD["lpt"]["brute_force_optimum_max_work"]


@pytest.mark.parametrize("i", range(1 + len(GOLD["hybrid_more"])))
def test_hybrid_hand_example(i):
    """Algorithm 1 worked by hand: two passes on two workers (the first
    example), three passes on three workers, and one pass on three workers
    whose repair pops two pieces and splits a given piece over two
    receivers."""
    g = GOLD["hybrid"] if i == 0 else GOLD["hybrid_more"][i - 1]
    cu = _cu(g["lengths"])
    plan, isp = P.plan_hybrid(cu, g["cp"], g["target_r"])
    assert plan.tolist() == g["plan"]
    assert isp.tolist() == g["is_per_doc"]
    st = P.stats(cu, g["cp"], plan, 1, 1)
    assert st["work"] == g["work"]
    assert st["tokens"] == g["tokens"]
    assert st["recv_tokens"] == g["recv_tokens"]
    assert st["eq5"] == g["eq5_over_hkv_d"] and st["eq4"] == g["eq4_over_hkv_d"]


def test_hybrid_random_invariants():
    """Eq. 1, Eq. 2, termination (Cur_R <= R or all Per-Doc), conservation of
    total workload, and Per-Doc documents chunked by the Per-Doc rule."""
    rng = np.random.default_rng(5)
    for trial in range(40):
        N = int(rng.choice([2, 3, 4, 8]))
        n = int(rng.integers(1, 12))
        lens = [int(x) for x in rng.integers(1, 400, size=n)]
        C = sum(lens)
        lens[-1] += (-C) % N
        cu = _cu(lens)
        plan, isp = P.plan_hybrid(cu, N, 1.05)
        P.validate(cu, N, plan)
        st = P.stats(cu, N, plan, 1, 1)
        assert sum(st["work"]) == sum(P.shard_work(0, L) for L in lens)
        if not isp.all():
            # some rank holds a whole-doc piece; tokens equal unless stuck on Per-Doc rounding
            dev = max(abs(t - sum(lens) // N) for t in st["tokens"])
            assert dev <= int(isp.sum())
        assert st["imbalance"] <= 1.05 or isp.all()
        for k in np.nonzero(isp)[0]:
            rows = plan[plan[:, 0] == k]
            want = P.canonical([(k, r, o, l) for r, o, l in P.per_doc_chunks(lens[k], N)])
            assert rows.tolist() == want.tolist()
        if isp.any():
            # the Per-Doc documents are the longest ones
            assert min(lens[k] for k in np.nonzero(isp)[0]) >= max(
                [lens[k] for k in np.nonzero(isp == 0)[0]] or [0])


def test_two_equal_documents_need_no_communication():
    """Sec. 3.3, first example: two equal documents on two workers stay whole;
    nothing is exchanged and the workload is balanced."""
    cu = _cu([500, 500])
    for plan in (P.plan_whole_lpt(cu, 2), P.plan_hybrid(cu, 2)[0]):
        st = P.stats(cu, 2, plan, 8, 128)
        assert st["recv_tokens"] == [0, 0] and st["eq5"] == 0 and st["imbalance"] == 1.0


def test_eq4_eq5_and_receive_sets():
    """Eq. 4 is the full-KV volume; Eq. 5 counts only non-last shards; whole
    documents contribute nothing (Sec. 3.2)."""
    cu = synth.cu_seqlens(synth.doc_lengths("wholedoc"))
    plan = P.plan_whole_lpt(cu, 8)
    st = P.stats(cu, 8, plan, 8, 128)
    assert st["eq4"] == 4 * 65536 // 8 * 8 * 128 * 7
    assert st["eq5"] == 0 and st["recv_tokens"] == [0] * 8
    # Per-Doc: every chunk but the last of each doc is non-last
    lens = [16 * 7, 16 * 3]
    plan = P.plan_per_doc(_cu(lens), 8)
    st = P.stats(_cu(lens), 8, plan, 1, 1)
    # rank 0 holds chunk 0 (non-last) and chunk 15 (last); others hold two non-last chunks
    assert st["eq5"] == 4 * (2 * 7 + 2 * 3) * 7
    # receive set of rank j: prefix up to its last chunk minus what it holds
    c = [L // 16 for L in lens]
    for j in range(8):
        want = sum((16 - j) * ci - 2 * ci for ci in c)
        assert st["recv_tokens"][j] == want


def test_per_seq_hand_example():
    """Llama3 CP (Sec. 2.2) on documents [0,5), [5,12), [12,30), N = 2: the
    sequence is cut into [0,7), [7,15), [15,22), [22,30), going to workers
    0, 1, 1, 0. Document 1 is split at token 7 (offset 2); document 2's
    tokens 12..21 (chunks 1 and 2) stay together on worker 1 and 22..29 go to
    worker 0 (offset 10)."""
    plan = P.plan_per_seq(_cu([5, 7, 18]), 2)
    assert plan.tolist() == [[0, 0, 0, 5], [1, 0, 0, 2], [1, 1, 2, 5], [2, 1, 0, 10], [2, 0, 10, 8]]


def test_per_seq_of_one_document_is_per_doc():
    """With a single document the sequence cut and the document cut coincide."""
    for L in (1, 7, 64, 1000, 4099):
        for N in (1, 2, 3, 8):
            assert np.array_equal(P.plan_per_seq(_cu([L]), N), P.plan_per_doc(_cu([L]), N))


def test_per_seq_tokens_and_intervals():
    """Worker r holds exactly chunks r and 2N-1-r of the whole sequence: its
    token count is the closed form, and the oracle (token by token) equals
    an interval-intersection construction of the same rule."""
    rng = np.random.default_rng(7)
    for _ in range(40):
        N = int(rng.choice([1, 2, 3, 4, 8]))
        lens = [int(x) for x in rng.integers(1, 300, size=int(rng.integers(1, 9)))]
        cu = _cu(lens)
        T = int(cu[-1])
        plan = P.plan_per_seq(cu, N)
        P.validate(cu, N, plan)
        tok = [0] * N
        for _, r, _, l in plan:
            tok[r] += int(l)
        b = [(i * T) // (2 * N) for i in range(2 * N + 1)]
        assert tok == [(b[r + 1] - b[r]) + (b[2 * N - r] - b[2 * N - 1 - r]) for r in range(N)]
        rows = []
        for i in range(2 * N):
            r = i if i < N else 2 * N - 1 - i
            for k in range(len(lens)):
                lo, hi = max(b[i], int(cu[k])), min(b[i + 1], int(cu[k + 1]))
                if hi > lo:
                    rows.append((k, r, lo - int(cu[k]), hi - lo))
        assert np.array_equal(plan, P.canonical(rows))
