"""fc_attn_bwd_noalloc (the backward with its workspace in the library's
static device scratch) against fc_attn_bwd with a caller workspace, through
the C ABI: bit-identical outputs on two calls in a row, the second on a
smaller view (the scratch keeps the first call's contents), and a view whose
workspace exceeds the scratch is rejected before any launch."""
import sys

import pytest
import torch

import _cases
from paper_2606_08476_amd import flashcp as F

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    F.lib()
    return torch.device("cuda:0")


def _forward(case, dev):
    x = {k: t.to(dev) for k, t in _cases.inputs(case).items()}
    v = F.View(case.cu, case.plan, case.cp, case.rank, case.hq, case.hkv, case.d).bind(dev)
    i = v.info
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    bf, f32 = torch.bfloat16, torch.float32
    kl, vl = torch.empty(tq, hkv, d, dtype=bf, device=dev), torch.empty(tq, hkv, d, dtype=bf, device=dev)
    kr, vr = torch.empty(tr, hkv, d, dtype=bf, device=dev), torch.empty(tr, hkv, d, dtype=bf, device=dev)
    F.fc_kv_gather(v, x["k_pk"], x["v_pk"], kl, vl, kr, vr)
    o = torch.empty(tq, hq, d, dtype=bf, device=dev)
    lse = torch.empty(hq, tq, dtype=f32, device=dev)
    fws = torch.empty(max(v.workspace_size(F.FC_TWO_PASS)[0], 1), dtype=torch.uint8, device=dev)
    F.fc_attn_fwd(v, x["q"], kl, vl, kr, vr, 0.0, F.FC_TWO_PASS, o, None, lse, fws)
    return v, (x["q"], kl, vl, kr, vr, o, lse, x["do"])


def _fwd_f32(v, a, dev):
    """The forward's fp32 O of the same inputs (delta is then taken from it)."""
    i = v.info
    o32 = torch.empty(i["t_q"], i["hq"], i["d"], dtype=torch.float32, device=dev)
    o = torch.empty_like(a[5])
    lse = torch.empty_like(a[6])
    fws = torch.empty(max(v.workspace_size(F.FC_TWO_PASS)[0], 1), dtype=torch.uint8, device=dev)
    F.fc_attn_fwd(v, a[0], a[1], a[2], a[3], a[4], 0.0, F.FC_TWO_PASS, o, o32, lse, fws)
    return o32


def _outputs(v, dev):
    i = v.info
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    e = lambda *s: torch.full(s, float("nan"), dtype=torch.float32, device=dev)
    return [e(tq, hq, d), e(tq, hkv, d), e(tq, hkv, d), e(tr, hkv, d), e(tr, hkv, d)]


def test_noalloc_equals_bwd_on_two_calls(dev):
    # the first view needs most of the scratch (60 split key tiles, one
    # partial slot each); the second is smaller and reuses what it left
    for key in ("llama8b_8k", "tiny"):
        case = _cases.small_case(key)
        v, a = _forward(case, dev)
        need = v.workspace_size()[1]
        assert 0 < need <= F.NOALLOC_SCRATCH_BYTES
        say(f"[gpu] noalloc case={key} workspace={need} slots={v.info['n_bwd_slots']}")
        ref = _outputs(v, dev)
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        F.fc_attn_bwd(v, *a, 0.0, *ref, ws)
        got = _outputs(v, dev)
        F.fc_attn_bwd_noalloc(v, *a, 0.0, *got)
        torch.cuda.synchronize()
        for name, r, g in zip(("dq", "dk_loc", "dv_loc", "dk_recv", "dv_recv"), ref, got):
            assert torch.isfinite(r).all(), name
            assert torch.equal(r, g), f"{key}: {name} differs"
        # the non-deterministic mode, delta from the fp32 O, through the same
        # scratch: dK/dV equal, dQ within fp32 reordering
        o32 = _fwd_f32(v, a, dev)
        ref_a, got_a = _outputs(v, dev), _outputs(v, dev)
        F.fc_attn_bwd(v, *a, 0.0, *ref_a, ws, deterministic=False, o_f32=o32)
        F.fc_attn_bwd_noalloc(v, *a, 0.0, *got_a, deterministic=False, o_f32=o32)
        torch.cuda.synchronize()
        for name, r, g in zip(("dk_loc", "dv_loc", "dk_recv", "dv_recv"), ref_a[1:], got_a[1:]):
            assert torch.equal(r, g), f"{key}: {name} differs (atomic mode)"
        assert float((ref_a[0] - got_a[0]).abs().max()) <= 1e-4
        v.close()


def test_noalloc_rejects_oversized_workspace(dev):
    case = _cases.small_case("wholedoc_16k")
    v, a = _forward(case, dev)
    assert v.workspace_size()[1] > F.NOALLOC_SCRATCH_BYTES
    outs = _outputs(v, dev)
    with pytest.raises(F.FlashCPError) as ei:
        F.fc_attn_bwd_noalloc(v, *a, 0.0, *outs)
    assert ei.value.code == -5 and "static scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert all(torch.isnan(t).all() for t in outs)   # nothing was launched
    v.close()
