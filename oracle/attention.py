"""Oracle document-masked causal attention: forward, backward, partial passes
and the log-sum-exp merge.

Test infrastructure only (see the package docstring).

Definitions (FlashCP Sec. 2.1 document mask; Sec. 3.1 workload W_i, whose
count fixes that the diagonal is visible):

* query at global position g sees the keys u with doc(u) == doc(g), u <= g;
* with query head h and KV head j = h // (Hq / Hkv) (grouped-query
  attention; the paper's H does not distinguish, reading stated in the
  design notes), s_gu = scale * <q_gh, k_uj>, LSE_gh = ln sum_u exp(s_gu),
  P_gu = exp(s_gu - LSE_gh), O_gh = sum_u P_gu v_uj;
* a *partial pass* uses only the visible keys inside a given key set; an
  empty visible set gives LSE = -inf and O = 0;
* the merge of two partials: LSE = ln(e^LSE_a + e^LSE_b), O = e^(LSE_a -
  LSE) O_a + e^(LSE_b - LSE) O_b (the partial-result aggregation that
  blockwise context-parallel attention needs, Sec. 2.3 and Sec. 4.2);
* backward, given dO: D_g = <dO_g, O_g>, dP_gu = <dO_g, v_u>,
  dS = P * (dP - D), dQ_g = scale sum_u dS_gu k_u,
  dK_u = scale sum_g dS_gu q_g, dV_u = sum_g P_gu dO_g, with dK and dV
  summed over the query heads of a KV head.

Everything is computed in the dtype requested (fp64 for parity, fp32 only
for the CPU-baseline timing) from bf16 inputs converted exactly. Scores are
materialised per block of at most ``ROW_BLOCK`` queries of one document; a
dense masked softmax follows, with no online rescaling.

Parity: pinned by a pure-Python brute force over explicit masks, by torch's
reference scaled-dot-product attention with autograd, by central finite
differences, and by special cases with closed forms (one-token documents,
identical keys, Hkv = Hq) in tests/test_oracle_attention.py.
"""
from __future__ import annotations

import math

import numpy as np
import torch

ROW_BLOCK = 512


def _docs(cu, gpos):
    cu = np.asarray(cu, dtype=np.int64)
    return np.searchsorted(cu, np.asarray(gpos, dtype=np.int64), side="right") - 1


def _blocks(cu, q_gpos, kv_gpos, rows):
    """Yield (query row indices, key indices, visible mask) per block of
    queries from one document."""
    qd = _docs(cu, q_gpos)
    kd = _docs(cu, kv_gpos)
    q_g = np.asarray(q_gpos, dtype=np.int64)
    k_g = np.asarray(kv_gpos, dtype=np.int64)
    rows = np.arange(q_g.size) if rows is None else np.asarray(rows, dtype=np.int64)
    for doc in np.unique(qd[rows]):
        rsel = rows[qd[rows] == doc]
        ksel = np.nonzero(kd == doc)[0]
        for b in range(0, rsel.size, ROW_BLOCK):
            r = rsel[b:b + ROW_BLOCK]
            mask = k_g[ksel][None, :] <= q_g[r][:, None]
            yield r, ksel, torch.from_numpy(mask)


def _heads(Hq, G, kv_heads):
    """Query heads to compute: all, or those of the given KV heads."""
    if kv_heads is None:
        return list(range(Hq))
    return [h for h in range(Hq) if h // G in set(int(j) for j in kv_heads)]


def attention_fwd(cu, q_gpos, q, kv_gpos, k, v, scale=None, rows=None, dtype=torch.float64,
                  kv_heads=None):
    """O [Tq, Hq, d] and LSE [Hq, Tq] of queries at ``q_gpos`` over the keys at
    ``kv_gpos`` (a partial pass whenever those keys are a subset of what the
    queries could see). ``rows`` restricts the computation to some queries;
    other rows are returned as NaN. ``kv_heads`` restricts it to the query
    heads of those KV heads (each head is computed on its own, so the values
    are those of the unrestricted call); other heads are NaN."""
    Tq, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    heads = _heads(Hq, G, kv_heads)
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else float(scale)
    q = q.to(dtype)
    k = k.to(dtype)
    v = v.to(dtype)
    O = torch.full((Tq, Hq, d), float("nan"), dtype=dtype)
    LSE = torch.full((Hq, Tq), float("nan"), dtype=dtype)
    rows_all = np.arange(Tq) if rows is None else np.asarray(rows, dtype=np.int64)
    ht = torch.as_tensor(heads, dtype=torch.long)
    O[rows_all[:, None], ht[None, :]] = 0
    LSE[ht[:, None], rows_all[None, :]] = -math.inf
    for r, ks, mask in _blocks(cu, q_gpos, kv_gpos, rows):
        if ks.size == 0:
            continue
        for h in heads:
            j = h // G
            s = scale * (q[r, h] @ k[ks, j].T)
            s = s.masked_fill(~mask, -math.inf)
            m = s.max(dim=1, keepdim=True).values
            has = torch.isfinite(m[:, 0])
            m = torch.where(torch.isfinite(m), m, torch.zeros_like(m))
            e = torch.exp(s - m)
            tot = e.sum(dim=1)
            lse = torch.where(has, m[:, 0] + torch.log(tot), torch.full_like(tot, -math.inf))
            p = torch.where(has[:, None], e / tot.clamp_min(1e-300)[:, None], torch.zeros_like(e))
            O[r, h] = p @ v[ks, j]
            LSE[h, r] = lse
    return O, LSE


def lse_merge(o_a, lse_a, o_b, lse_b):
    """Merge two partial results over disjoint key sets (O [T, H, d],
    LSE [H, T]); a -inf LSE carries weight 0, so a row that is empty in
    both partials stays empty (O = 0, LSE = -inf), as a pass over the union
    of the two key sets would leave it."""
    m = torch.maximum(lse_a, lse_b)
    m = torch.where(torch.isfinite(m), m, torch.zeros_like(m))
    wa = torch.exp(lse_a - m)
    wb = torch.exp(lse_b - m)
    tot = wa + wb
    lse = m + torch.log(tot)
    some = tot > 0
    safe = torch.where(some, tot, torch.ones_like(tot))
    ca = torch.where(some, wa / safe, torch.zeros_like(wa)).T[:, :, None]
    cb = torch.where(some, wb / safe, torch.zeros_like(wb)).T[:, :, None]
    return ca * o_a + cb * o_b, lse


def attention_bwd(cu, q_gpos, q, kv_gpos, k, v, do, scale=None, rows=None, dtype=torch.float64,
                  kv_heads=None, with_fwd=False):
    """dQ [Tq, Hq, d], dK and dV [Tk, Hkv, d] of the full (single-pass)
    attention of queries at ``q_gpos`` over keys at ``kv_gpos``. The key set
    must contain every key the queries see, so the softmax is complete.

    ``rows`` restricts the backward to some queries: dQ is then computed for
    those rows only (others are zero) and dK/dV hold only their
    contributions, which is the exact gradient for every key that no other
    query sees (e.g. all keys of a document whose queries are all in rows).
    ``kv_heads`` restricts it to those KV heads and their query heads (dQ of
    other heads, dK/dV of other KV heads are NaN). With ``with_fwd`` the
    forward's O and LSE are returned too, as (dQ, dK, dV, O, LSE)."""
    Tq, Hq, d = q.shape
    Tk, Hkv, _ = k.shape
    G = Hq // Hkv
    heads = _heads(Hq, G, kv_heads)
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else float(scale)
    O, LSE = attention_fwd(cu, q_gpos, q, kv_gpos, k, v, scale, rows=rows, dtype=dtype,
                           kv_heads=kv_heads)
    q = q.to(dtype)
    k = k.to(dtype)
    v = v.to(dtype)
    do = do.to(dtype)
    D = (do * torch.nan_to_num(O)).sum(dim=2).T  # [Hq, Tq]
    dq = torch.zeros((Tq, Hq, d), dtype=dtype)
    dk = torch.zeros((Tk, Hkv, d), dtype=dtype)
    dv = torch.zeros((Tk, Hkv, d), dtype=dtype)
    if kv_heads is not None:
        other = [h for h in range(Hq) if h not in heads]
        dq[:, other] = float("nan")
        okv = [j for j in range(Hkv) if j not in set(int(x) for x in kv_heads)]
        dk[:, okv] = float("nan")
        dv[:, okv] = float("nan")
    for r, ks, mask in _blocks(cu, q_gpos, kv_gpos, rows):
        if ks.size == 0:
            continue
        kt = torch.from_numpy(ks)
        for h in heads:
            j = h // G
            s = (scale * (q[r, h] @ k[ks, j].T)).masked_fill(~mask, -math.inf)
            p = torch.exp(s - LSE[h, r][:, None])
            dp = do[r, h] @ v[ks, j].T
            ds = p * (dp - D[h, r][:, None])
            dq[r, h] += scale * (ds @ k[ks, j])
            dk[:, j].index_add_(0, kt, scale * (ds.T @ q[r, h]))
            dv[:, j].index_add_(0, kt, p.T @ do[r, h])
    if with_fwd:
        return dq, dk, dv, O, LSE
    return dq, dk, dv


def brute_fwd(cu, q, k, v, scale):
    """Unsharded packed attention by explicit loops over (query, key) pairs.
    Only for tiny inputs (tests)."""
    T, Hq, d = q.shape
    G = Hq // k.shape[1]
    cu = [int(x) for x in cu]
    doc = [max(i for i in range(len(cu) - 1) if cu[i] <= g) for g in range(T)]
    q64, k64, v64 = q.double(), k.double(), v.double()
    O = torch.zeros((T, Hq, d), dtype=torch.float64)
    LSE = torch.zeros((Hq, T), dtype=torch.float64)
    for h in range(Hq):
        for g in range(T):
            vis = [u for u in range(T) if doc[u] == doc[g] and u <= g]
            s = [scale * float(torch.dot(q64[g, h], k64[u, h // G])) for u in vis]
            mx = max(s)
            z = sum(math.exp(x - mx) for x in s)
            LSE[h, g] = mx + math.log(z)
            for u, x in zip(vis, s):
                O[g, h] += math.exp(x - mx) / z * v64[u, h // G]
    return O, LSE
