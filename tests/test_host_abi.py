"""Host side of the C ABI, no GPU: the library loads and exports every
function the header declares; planners, rank views and tile maps are
bit-exact with the oracle; invalid input is rejected with its error code
before anything is launched."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import planner as P
from oracle import view as V
from paper_2606_08476_amd import flashcp as F
from paper_2606_08476_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashcp.h")


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(F._LIB_PATH):
        from paper_2606_08476_amd import build
        build.build()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fc_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = _declared()
    assert len(names) >= 16
    lib = C.CDLL(F._LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(F.EXPORTS) == names


def _cu(lens):
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)


def _random_cases(n=25, seed=7):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        N = int(rng.choice([1, 2, 3, 4, 8]))
        k = int(rng.integers(1, 14))
        lens = [int(x) for x in rng.integers(1, 500, size=k)]
        lens[-1] += (-sum(lens)) % N
        yield _cu(lens), N


def test_planners_bit_exact_random():
    for cu, N in _random_cases():
        assert np.array_equal(F.fc_plan_per_doc(cu, N), P.plan_per_doc(cu, N))
        assert np.array_equal(F.fc_plan_per_seq(cu, N), P.plan_per_seq(cu, N))
        assert np.array_equal(F.fc_plan_whole_lpt(cu, N), P.plan_whole_lpt(cu, N))
        for R in (1.0, 1.05, 1.3):
            a, ia = F.fc_plan_hybrid(cu, N, R)
            b, ib = P.plan_hybrid(cu, N, R)
            assert np.array_equal(a, b) and np.array_equal(ia, ib)
            assert F.fc_plan_stats(cu, N, a, 2, 64) == P.stats(cu, N, b, 2, 64)


def test_planners_match_hand_worked_examples():
    """The library's LPT and hybrid planners and plan statistics on the
    examples of tests/golden worked by hand from Algorithm 1."""
    import json
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "planner_hand.json")))
    g = gold["lpt"]
    cu = np.concatenate([[0], np.cumsum(g["lengths"])])
    plan = F.fc_plan_whole_lpt(cu, g["cp"])
    assert plan.tolist() == g["plan"]
    assert F.fc_plan_stats(cu, g["cp"], plan, 1, 1)["work"] == g["work"]
    for g in [gold["hybrid"]] + gold["hybrid_more"]:
        cu = np.concatenate([[0], np.cumsum(g["lengths"])])
        plan, isp = F.fc_plan_hybrid(cu, g["cp"], g["target_r"])
        assert plan.tolist() == g["plan"] and isp.tolist() == g["is_per_doc"]
        st = F.fc_plan_stats(cu, g["cp"], plan, 1, 1)
        assert st["work"] == g["work"] and st["tokens"] == g["tokens"]
        assert st["recv_tokens"] == g["recv_tokens"]
        assert st["eq4"] == g["eq4_over_hkv_d"] and st["eq5"] == g["eq5_over_hkv_d"]


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_planners_bit_exact_workloads(name):
    w = synth.WORKLOADS[name]
    cu = synth.cu_seqlens(synth.doc_lengths(name))
    assert np.array_equal(F.fc_plan_per_doc(cu, w.cp), P.plan_per_doc(cu, w.cp))
    assert np.array_equal(F.fc_plan_per_seq(cu, w.cp), P.plan_per_seq(cu, w.cp))
    assert np.array_equal(F.fc_plan_whole_lpt(cu, w.cp), P.plan_whole_lpt(cu, w.cp))
    a, ia = F.fc_plan_hybrid(cu, w.cp)
    b, ib = P.plan_hybrid(cu, w.cp)
    assert np.array_equal(a, b) and np.array_equal(ia, ib)
    for plan in (a, F.fc_plan_per_doc(cu, w.cp), F.fc_plan_per_seq(cu, w.cp), F.fc_plan_whole_lpt(cu, w.cp)):
        assert F.fc_plan_stats(cu, w.cp, plan, w.hkv, w.d) == P.stats(cu, w.cp, plan, w.hkv, w.d)


def _compare_view(cu, plan, N, r, hq, hkv, d, tiles=None):
    v = F.View(cu, plan, N, r, hq, hkv, d, tiles=tiles)
    e = v.export()
    o = V.rank_view(cu, plan, r)
    i = v.info
    assert np.array_equal(e["q_gpos"], o.q_gpos)
    assert np.array_equal(e["recv_gpos"], o.recv_gpos)
    assert np.array_equal(e["seg_doc"], o.seg_doc)
    assert np.array_equal(e["q_cu_docseg"], o.q_cu_docseg)
    assert np.array_equal(e["recv_cu"], o.recv_cu)
    assert np.array_equal(e["pieces"], o.pieces)
    assert np.array_equal(e["lim"], o.lim)
    assert (i["pairs_loc"], i["pairs_recv"]) == (o.pairs_loc, o.pairs_recv)
    for mode in ("local", "recv", "fused"):
        assert np.array_equal(e["fwd_" + mode], V.fwd_items(o, i["bm_fwd"], i["bn_fwd"], mode)), mode
    assert np.array_equal(e["bwd"], V.bwd_items(o, i["bm_bwd"], i["bn_bwd"]))
    v.close()


def test_views_bit_exact_random():
    for cu, N in _random_cases(12, seed=9):
        for plan in (P.plan_per_doc(cu, N), P.plan_hybrid(cu, N)[0]):
            for r in range(N):
                for hq, hkv, d in ((4, 4, 64), (8, 2, 128), (16, 2, 128)):
                    _compare_view(cu, plan, N, r, hq, hkv, d)


def test_tile_shapes():
    """A view's forward query tile follows fc_tile_cfg.bm_fwd (32, 64 or 128
    rows: 4, 2 or 1 heads of a KV group per workgroup) and its tile maps
    equal the oracle's for that shape; shapes that are not compiled, or that
    put more heads in a workgroup than the group has, are rejected."""
    for cu, N in _random_cases(4, seed=21):
        plan = P.plan_per_doc(cu, N)
        for hq, hkv in ((16, 2), (8, 2), (4, 4)):
            G = hq // hkv
            for bm in (32, 64, 128):
                if G % (128 // bm):
                    with pytest.raises(F.FlashCPError) as ei:
                        F.View(cu, plan, N, 0, hq, hkv, 64, tiles=(bm, 0, 0, 0))
                    assert ei.value.code == -4
                    continue
                v = F.View(cu, plan, N, 0, hq, hkv, 64, tiles=(bm, 0, 0, 0))
                assert v.info["bm_fwd"] == bm
                v.close()
                for r in range(N):
                    _compare_view(cu, plan, N, r, hq, hkv, 64, tiles=(bm, 64, 32, 128))
    cu, N = next(iter(_random_cases(1, seed=22)))
    plan = P.plan_per_doc(cu, N)
    # defaults: as many heads per workgroup as the group allows, up to 4
    for hq, hkv, bm in ((32, 8, 32), (16, 8, 64), (8, 8, 128)):
        assert F.View(cu, plan, N, 0, hq, hkv, 128).info["bm_fwd"] == bm
    for bad in ((48, 0, 0, 0), (0, 128, 0, 0), (0, 0, 64, 0), (0, 0, 0, 64)):
        with pytest.raises(F.FlashCPError) as ei:
            F.View(cu, plan, N, 0, 32, 8, 128, tiles=bad)
        assert ei.value.code == -4


@pytest.mark.parametrize("name", ["tiny", "llama8b", "wholedoc"])
def test_views_bit_exact_workload_ranks(name):
    w = synth.WORKLOADS[name]
    cu = synth.cu_seqlens(synth.doc_lengths(name))
    plan = {"per_doc": P.plan_per_doc, "whole_lpt": P.plan_whole_lpt}[w.plan](cu, w.cp)
    ranks = [0, w.cp - 1] if name != "tiny" else [0, 1]
    for r in ranks:
        _compare_view(cu, plan, w.cp, r, w.hq, w.hkv, w.d)


def test_heaviest_rank_agrees():
    """The rank the workloads name as heaviest (argmax W, lowest on ties)
    is the same from the C ABI and the oracle."""
    for name in ("wholedoc", "hybrid70b"):
        w = synth.WORKLOADS[name]
        cu = synth.cu_seqlens(synth.doc_lengths(name))
        plan = F.fc_plan_whole_lpt(cu, w.cp) if w.plan == "whole_lpt" else F.fc_plan_hybrid(cu, w.cp)[0]
        a = F.fc_plan_stats(cu, w.cp, plan, w.hkv, w.d)["work"]
        b = P.stats(cu, w.cp, plan, w.hkv, w.d)["work"]
        assert a == b and int(np.argmax(a)) == int(np.argmax(b))


def _code(fn, *a):
    with pytest.raises(F.FlashCPError) as ei:
        fn(*a)
    return ei.value.code


def test_error_codes():
    cu = _cu([5, 3])
    ok = np.array([[0, 0, 0, 5], [1, 1, 0, 3]], dtype=np.int32)
    F.fc_plan_validate(cu, 2, ok)
    assert _code(F.fc_plan_validate, cu, 2, np.array([[0, 0, 0, 4], [1, 1, 0, 3]])) == -2   # gap
    assert _code(F.fc_plan_validate, cu, 2,
                 np.array([[0, 0, 0, 5], [0, 1, 4, 1], [1, 1, 0, 3]])) == -2               # overlap
    assert _code(F.fc_plan_validate, cu, 2, np.array([[0, 0, 0, 6], [1, 1, 0, 3]])) == -2   # beyond doc
    assert _code(F.fc_plan_validate, cu, 2, np.array([[0, 2, 0, 5], [1, 1, 0, 3]])) == -2   # rank >= N
    assert _code(F.fc_plan_validate, cu, 2, ok, True) == -2                                 # Eq. 2
    assert _code(F.fc_plan_per_doc, np.array([0, 4, 4], dtype=np.int32), 2) == -1           # empty doc
    assert _code(F.fc_plan_per_doc, cu, 0) == -1
    assert _code(F.fc_plan_hybrid, _cu([5, 2]), 2) == -1                                    # N does not divide C
    assert _code(F.View, cu, ok, 2, 0, 6, 4, 64) == -1                                       # hq % hkv
    assert _code(F.View, cu, ok, 2, 0, 4, 4, 96) == -4                                       # head dim
    assert _code(F.View, cu, ok, 2, 0, 12, 4, 64) == -4                                      # group of 3
    assert _code(F.View, cu, ok, 2, 2, 4, 4, 64) == -1                                       # rank
    assert _code(F.View, cu, np.array([[0, 0, 0, 4], [1, 1, 0, 3]]), 2, 0, 4, 4, 64) == -2  # bad plan
    # capacity: n_out reports the need
    lib = F.lib()
    n = C.c_int64(0)
    buf = (F.Shard * 1)()
    rc = lib.fc_plan_per_doc(cu.ctypes.data_as(F.I32P), 2, 2, buf, 1, C.byref(n))
    assert rc == -7 and n.value == len(P.plan_per_doc(cu, 2))
    assert lib.fc_plan_per_doc(None, 2, 2, buf, 1, C.byref(n)) == -1


def test_kernel_calls_rejected_before_launch():
    """Device entry points refuse an unbound view, bad modes and bad
    workspaces on the host: no GPU is touched."""
    lib = F.lib()
    cu = _cu([64, 64])
    plan = P.plan_per_doc(cu, 2)
    v = F.View(cu, plan, 2, 0, 4, 4, 64)
    h = v.handle
    a = 256   # a stand-in device address, aligned (nothing is dereferenced)
    assert lib.fc_kv_gather(h, a, a, 128, a, a, a, a, None) == -5
    assert lib.fc_attn_fwd(h, a, a, a, a, a, 0.0, 0, a, None, a, None, 0, None) == -5
    for det in (0, 1):
        assert lib.fc_attn_bwd(h, *([a] * 9), 0.0, det, *([a] * 5), None, 0, None) == -5
        assert lib.fc_attn_bwd_pass(h, *([a] * 8), 0.0, det, *([a] * 5), None, 0, None) == -5
        assert lib.fc_attn_bwd_noalloc(h, *([a] * 9), 0.0, det, *([a] * 5), None) == -5
    assert lib.fc_bwd_preprocess(h, a, None, a, a, None) == -5
    assert lib.fc_attn_bwd_dkdv(h, *([a] * 8), 0.0, *([a] * 4), None, 0, None) == -5
    assert lib.fc_attn_fwd_partial(h, 0, a, a, a, 0.0, a, a, None) == -5
    assert lib.fc_attn_fwd_partials(h, a, a, a, a, a, 0.0, a, a, a, a, None) == -5
    assert lib.fc_lse_merge(a, a, a, a, 4, 2, 96, a, None, a, None) == -4
    assert lib.fc_lse_merge(a, a, a, a, -1, 2, 64, a, None, a, None) == -1
    # misaligned pointers are refused first: row tensors and workspaces at 16
    # bytes, lse / delta at 4 (a + 8 and a + 2)
    m, s = a + 8, a + 2
    assert lib.fc_kv_gather(h, a, a, 128, a, m, a, a, None) == -1
    assert lib.fc_attn_fwd(h, m, a, a, a, a, 0.0, 0, a, None, a, None, 0, None) == -1
    assert lib.fc_attn_fwd(h, a, a, a, a, a, 0.0, 0, a, None, s, None, 0, None) == -1
    assert lib.fc_attn_fwd(h, a, a, a, a, a, 0.0, 0, a, None, a, m, 1 << 20, None) == -1
    assert lib.fc_attn_fwd_partial(h, 0, a, a, a, 0.0, m, a, None) == -1
    assert lib.fc_attn_fwd_partials(h, a, a, a, a, a, 0.0, a, a, a, s, None) == -1
    assert lib.fc_lse_merge(a, a, m, a, 4, 2, 64, a, None, a, None) == -1
    assert lib.fc_lse_merge(a, a, a, a, 4, 2, 64, a, None, s, None) == -1
    assert lib.fc_bwd_preprocess(h, a, m, a, a, None) == -1
    assert lib.fc_bwd_preprocess(h, a, None, a, s, None) == -1
    assert lib.fc_attn_bwd_dkdv(h, *([a] * 6), s, a, 0.0, *([a] * 4), None, 0, None) == -1
    assert lib.fc_attn_bwd_dq(h, *([a] * 8), 0.0, m, None) == -1
    for det in (0, 1):
        assert lib.fc_attn_bwd(h, *([a] * 9), 0.0, det, m, *([a] * 4), None, 0, None) == -1
        assert lib.fc_attn_bwd(h, *([a] * 9), 0.0, det, *([a] * 5), m, 1 << 20, None) == -1
        assert lib.fc_attn_bwd_pass(h, *([a] * 6), s, a, 0.0, det, *([a] * 5), None, 0, None) == -1
    f, b, k = v.workspace_size(F.FC_TWO_PASS)
    i = v.info
    # the two-pass forward keeps the received partial's fp32 O (merged in the
    # kernel): a slot of 32 rows x d per wave, 4 waves per workgroup of the
    # launch (fused items x KV heads x head chunks)
    wgs = i["n_fwd_fused"] * i["hkv"] * (i["hq"] // i["hkv"] // (128 // i["bm_fwd"]))
    assert f == (wgs * 4 * 32 * i["d"] * 4 + 255) // 256 * 256
    assert v.workspace_size(F.FC_FUSED)[0] == 0
    assert lib.fc_workspace_size(h, 7, None, None, None) == -1
    assert k == 0 and b == ((i["t_q"] * 4 * 4 + 255) // 256) * 256   # no split key tile here
    assert lib.fc_view_bind(h, None, 0, None) == -1
    assert lib.fc_view_bind(h, 256, 4, None) == -5       # too small, rejected before any copy
    assert lib.fc_view_bind(h, 257, 1 << 20, None) == -1  # misaligned
    v.close()


def test_empty_rank_view():
    """A rank with no shards has an empty view; its calls are no-ops."""
    cu = _cu([10])
    plan = np.array([[0, 0, 0, 10]], dtype=np.int32)
    v = F.View(cu, plan, 2, 1, 4, 4, 64)
    assert v.info["t_q"] == 0 and v.info["t_recv"] == 0 and v.info["n_bwd"] == 0
    v.close()


def test_backward_workspace_holds_the_partial_slots():
    """The dK/dV workspace is exactly the split key tiles' partial slots (two
    fp32 tiles of 128 keys x d per KV head each), and the Whole-Doc shard
    does split tiles. The split itself is checked against the tile map by
    brute force in test_launch_tables.py."""
    for name in ("wholedoc", "llama8b"):
        w = synth.WORKLOADS[name]
        cu = synth.cu_seqlens(synth.doc_lengths(name))
        plan = P.plan_whole_lpt(cu, w.cp) if w.plan == "whole_lpt" else P.plan_per_doc(cu, w.cp)
        rank = int(np.argmax(P.stats(cu, w.cp, plan, 1, 1)["work"]))
        v = F.View(cu, plan, w.cp, rank, w.hq, w.hkv, w.d)
        i = v.info
        slots = int((v.export_launch()["bwd_launch"][:, 7] >= 0).sum())
        assert slots == i["n_bwd_slots"]
        assert v.workspace_size()[2] == 2 * slots * w.hkv * 128 * w.d * 4
        if name == "wholedoc":
            assert slots > 0
        v.close()
