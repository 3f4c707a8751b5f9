"""Pins of the attention oracle against things other than itself: explicit
loops, torch's reference attention and autograd, finite differences, and
closed forms of special cases."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A


def _packed(lens, hq, hkv, d, seed):
    g = torch.Generator().manual_seed(seed)
    T = sum(lens)
    q = torch.randn(T, hq, d, generator=g).to(torch.bfloat16)
    k = torch.randn(T, hkv, d, generator=g).to(torch.bfloat16)
    v = torch.randn(T, hkv, d, generator=g).to(torch.bfloat16)
    do = torch.randn(T, hq, d, generator=g).to(torch.bfloat16)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return cu, q, k, v, do


def _dense_mask(cu, T):
    doc = np.searchsorted(cu, np.arange(T), side="right") - 1
    g = np.arange(T)
    return torch.from_numpy((doc[:, None] == doc[None, :]) & (g[None, :] <= g[:, None]))


@pytest.mark.parametrize("lens,hq,hkv", [([5, 1, 11, 7], 4, 2), ([16], 2, 2), ([3, 3, 3], 3, 1)])
def test_fwd_matches_brute_force(lens, hq, hkv):
    cu, q, k, v, _ = _packed(lens, hq, hkv, 8, 1)
    T = cu[-1]
    scale = 0.37
    O, L = A.attention_fwd(cu, np.arange(T), q, np.arange(T), k, v, scale)
    Ob, Lb = A.brute_fwd(cu, q, k, v, scale)
    assert torch.allclose(O, Ob, atol=1e-12, rtol=0)
    assert torch.allclose(L, Lb, atol=1e-12, rtol=0)


def _sdpa_ref(cu, q, k, v, scale):
    """torch's reference attention (math path, fp64) with an explicit mask;
    KV heads expanded for grouped queries."""
    T, hq, d = q.shape
    G = hq // k.shape[1]
    qh = q.double().permute(1, 0, 2)
    kh = k.double().repeat_interleave(G, dim=1).permute(1, 0, 2)
    vh = v.double().repeat_interleave(G, dim=1).permute(1, 0, 2)
    mask = _dense_mask(cu, T)
    o = torch.nn.functional.scaled_dot_product_attention(qh, kh, vh, attn_mask=mask, scale=scale)
    return o.permute(1, 0, 2)


def test_fwd_bwd_match_sdpa_autograd():
    lens = [37, 1, 90, 2, 50]
    cu, q, k, v, do = _packed(lens, 8, 2, 16, 2)
    T = cu[-1]
    scale = 1 / 4
    O, L = A.attention_fwd(cu, np.arange(T), q, np.arange(T), k, v, scale)
    qr, kr, vr = (x.double().requires_grad_() for x in (q, k, v))
    o_ref = _sdpa_ref(cu, qr, kr, vr, scale)
    assert torch.allclose(O, o_ref.detach(), atol=1e-12, rtol=0)
    o_ref.backward(do.double())
    dq, dk, dv = A.attention_bwd(cu, np.arange(T), q, np.arange(T), k, v, do, scale)
    assert torch.allclose(dq, qr.grad, atol=1e-11, rtol=0)
    assert torch.allclose(dk, kr.grad, atol=1e-11, rtol=0)
    assert torch.allclose(dv, vr.grad, atol=1e-11, rtol=0)


def test_lse_against_logsumexp():
    lens = [20, 12]
    cu, q, k, v, _ = _packed(lens, 2, 1, 8, 3)
    T = cu[-1]
    _, L = A.attention_fwd(cu, np.arange(T), q, np.arange(T), k, v, 0.5)
    s = 0.5 * torch.einsum("thd,ud->htu", q.double(), k.double()[:, 0])
    s = s.masked_fill(~_dense_mask(cu, T)[None], -math.inf)
    assert torch.allclose(L, torch.logsumexp(s, dim=2), atol=1e-12, rtol=0)


def test_bwd_finite_differences():
    lens = [6, 1, 9]
    cu, q, k, v, do = _packed(lens, 2, 1, 4, 4)
    T = cu[-1]
    scale = 0.8
    qd, kd, vd, dod = (x.double() for x in (q, k, v, do))

    def loss(qq, kk, vv):
        O, _ = A.attention_fwd(cu, np.arange(T), qq, np.arange(T), kk, vv, scale)
        return float((O * dod).sum())

    dq, dk, dv = A.attention_bwd(cu, np.arange(T), qd, np.arange(T), kd, vd, dod, scale)
    eps = 1e-6
    rng = np.random.default_rng(0)
    for name, x, grad in (("q", qd, dq), ("k", kd, dk), ("v", vd, dv)):
        for _ in range(12):
            idx = tuple(int(rng.integers(0, s)) for s in x.shape)
            xp, xm = x.clone(), x.clone()
            xp[idx] += eps
            xm[idx] -= eps
            args_p = [qd, kd, vd]
            args_m = [qd, kd, vd]
            pos = "qkv".index(name)
            args_p[pos], args_m[pos] = xp, xm
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - float(grad[idx])) < 1e-7, (name, idx, fd, float(grad[idx]))


def test_one_token_document():
    """A one-token document: O = v, LSE = s_gg; dQ = dK = 0 and dV = dO."""
    lens = [7, 1, 5]
    cu, q, k, v, do = _packed(lens, 2, 2, 8, 5)
    T = cu[-1]
    g = 7
    O, L = A.attention_fwd(cu, np.arange(T), q, np.arange(T), k, v, 0.3)
    dq, dk, dv = A.attention_bwd(cu, np.arange(T), q, np.arange(T), k, v, do, 0.3)
    for h in range(2):
        assert torch.equal(O[g, h], v[g, h].double())
        assert L[h, g] == pytest.approx(0.3 * float(torch.dot(q[g, h].double(), k[g, h].double())), abs=1e-13)
        assert torch.all(dq[g, h] == 0) and torch.all(dk[g, h] == 0)
        assert torch.allclose(dv[g, h], do[g, h].double(), atol=1e-15)


def test_identical_keys_give_mean_of_values():
    """All keys equal: O_g = mean of visible values, LSE = s + ln |V(g)|."""
    lens = [9, 14]
    cu, q, k, v, _ = _packed(lens, 2, 1, 8, 6)
    k = k[:1].expand_as(k).contiguous()
    T = cu[-1]
    O, L = A.attention_fwd(cu, np.arange(T), q, np.arange(T), k, v, 0.5)
    for g in range(T):
        doc = int(np.searchsorted(cu, g, side="right") - 1)
        vis = list(range(int(cu[doc]), g + 1))
        for h in range(2):
            assert torch.allclose(O[g, h], v[vis, 0].double().mean(dim=0), atol=1e-13)
            s = 0.5 * float(torch.dot(q[g, h].double(), k[0, 0].double()))
            assert float(L[h, g]) == pytest.approx(s + math.log(len(vis)), abs=1e-12)


def test_gqa_equals_mha_on_expanded_kv():
    """Hkv < Hq equals MHA on KV repeated per group; GQA dK/dV are the
    group sums of the MHA gradients."""
    lens = [13, 21]
    cu, q, k, v, do = _packed(lens, 6, 2, 8, 7)
    T = cu[-1]
    ar = np.arange(T)
    O, L = A.attention_fwd(cu, ar, q, ar, k, v, 0.4)
    ke, ve = k.repeat_interleave(3, dim=1), v.repeat_interleave(3, dim=1)
    Oe, Le = A.attention_fwd(cu, ar, q, ar, ke, ve, 0.4)
    assert torch.equal(O, Oe) and torch.equal(L, Le)
    dq, dk, dv = A.attention_bwd(cu, ar, q, ar, k, v, do, 0.4)
    dqe, dke, dve = A.attention_bwd(cu, ar, q, ar, ke, ve, do, 0.4)
    assert torch.allclose(dq, dqe, atol=1e-13)
    assert torch.allclose(dk, dke.reshape(T, 2, 3, 8).sum(2), atol=1e-13)
    assert torch.allclose(dv, dve.reshape(T, 2, 3, 8).sum(2), atol=1e-13)


def test_merge_of_arbitrary_split_equals_single_pass():
    lens = [30, 45]
    cu, q, k, v, _ = _packed(lens, 4, 2, 8, 8)
    T = cu[-1]
    ar = np.arange(T)
    rng = np.random.default_rng(3)
    side = rng.random(T) < 0.5
    a, b = np.nonzero(side)[0], np.nonzero(~side)[0]
    Oa, La = A.attention_fwd(cu, ar, q, a, k[a], v[a], 0.3)
    Ob, Lb = A.attention_fwd(cu, ar, q, b, k[b], v[b], 0.3)
    assert torch.isinf(La).any() or torch.isinf(Lb).any()  # some rows see one side only
    Om, Lm = A.lse_merge(Oa, La, Ob, Lb)
    O, L = A.attention_fwd(cu, ar, q, ar, k, v, 0.3)
    assert torch.allclose(Om, O, atol=1e-13) and torch.allclose(Lm, L, atol=1e-13)


def test_merge_of_two_empty_partials_is_empty():
    """Rows that see no key of either partial (three key sets: the merge of
    the first two is an empty partial for rows whose keys all lie in the
    third) merge to O = 0, LSE = -inf, and merging that result with the
    third partial gives the single pass."""
    lens = [6, 5]
    cu, q, k, v, _ = _packed(lens, 2, 1, 8, 12)
    T = cu[-1]
    ar = np.arange(T)
    a, b, c = np.array([1]), np.array([2]), np.setdiff1d(ar, [1, 2])
    Oa, La = A.attention_fwd(cu, ar, q, a, k[a], v[a], 0.3)
    Ob, Lb = A.attention_fwd(cu, ar, q, b, k[b], v[b], 0.3)
    Oab, Lab = A.lse_merge(Oa, La, Ob, Lb)
    empty = torch.isinf(La) & torch.isinf(Lb)
    assert empty.any() and (~empty).any()
    assert torch.equal(torch.isinf(Lab), empty) and (Lab[empty] < 0).all()
    assert torch.all(Oab.transpose(0, 1)[empty] == 0) and torch.isfinite(Oab).all()
    Oc, Lc = A.attention_fwd(cu, ar, q, c, k[c], v[c], 0.3)
    Om, Lm = A.lse_merge(Oab, Lab, Oc, Lc)
    O, L = A.attention_fwd(cu, ar, q, ar, k, v, 0.3)
    assert torch.allclose(Om, O, atol=1e-13) and torch.allclose(Lm, L, atol=1e-13)


def test_empty_partial_pass():
    lens = [4, 4]
    cu, q, k, v, _ = _packed(lens, 2, 1, 8, 9)
    O, L = A.attention_fwd(cu, np.arange(8), q, np.array([5]), k[5:6], v[5:6], 0.3)
    assert torch.isinf(L[:, :5]).all() and (L[:, :5] < 0).all()
    assert torch.all(O[:5] == 0)
    assert torch.isinf(L[:, 5:]).logical_not().all()


def test_row_restricted_backward_is_exact_for_its_documents():
    """Restricting the backward to the queries of some documents gives the
    full dQ on those rows and the full dK/dV on those documents' keys."""
    lens = [17, 30, 9]
    cu, q, k, v, do = _packed(lens, 4, 2, 8, 10)
    T = cu[-1]
    ar = np.arange(T)
    dq, dk, dv = A.attention_bwd(cu, ar, q, ar, k, v, do, 0.3)
    rows = np.arange(cu[1], cu[2])
    dq2, dk2, dv2 = A.attention_bwd(cu, ar, q, ar, k, v, do, 0.3, rows=rows)
    assert torch.allclose(dq2[rows], dq[rows], atol=1e-14)
    assert torch.allclose(dk2[rows], dk[rows], atol=1e-14)
    assert torch.allclose(dv2[rows], dv[rows], atol=1e-14)
    other = np.setdiff1d(ar, rows)
    assert torch.all(dq2[other] == 0) and torch.all(dk2[other] == 0)


def test_kv_head_restriction_equals_unrestricted():
    """Restricting the oracle to some KV heads computes exactly the values of
    the unrestricted call for those heads' query heads and KV rows (each head
    is computed on its own), and NaN elsewhere; with_fwd returns the
    forward's O and LSE alongside."""
    lens = [23, 40, 9]
    cu, q, k, v, do = _packed(lens, 8, 4, 8, 13)
    T = cu[-1]
    ar = np.arange(T)
    O, L = A.attention_fwd(cu, ar, q, ar, k, v, 0.3)
    dq, dk, dv = A.attention_bwd(cu, ar, q, ar, k, v, do, 0.3)
    for sel in ([1], [0, 3]):
        hs = [h for h in range(8) if h // 2 in sel]
        oth = [h for h in range(8) if h not in hs]
        kvo = [j for j in range(4) if j not in sel]
        O2, L2 = A.attention_fwd(cu, ar, q, ar, k, v, 0.3, kv_heads=sel)
        assert torch.equal(O2[:, hs], O[:, hs]) and torch.equal(L2[hs], L[hs])
        assert torch.isnan(O2[:, oth]).all() and torch.isnan(L2[oth]).all()
        dq2, dk2, dv2, O3, L3 = A.attention_bwd(cu, ar, q, ar, k, v, do, 0.3, kv_heads=sel,
                                                with_fwd=True)
        assert torch.equal(dq2[:, hs], dq[:, hs]) and torch.isnan(dq2[:, oth]).all()
        assert torch.equal(dk2[:, sel], dk[:, sel]) and torch.equal(dv2[:, sel], dv[:, sel])
        assert torch.isnan(dk2[:, kvo]).all() and torch.isnan(dv2[:, kvo]).all()
        assert torch.equal(O3[:, hs], O[:, hs]) and torch.equal(L3[hs], L[hs])
