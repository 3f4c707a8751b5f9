"""Python binding of the C ABI in ``include/flashcp.h``.

Argument marshalling only: every planner, view and kernel call goes to the
native library ``libflashcp.so`` built in this directory. Torch supplies
device memory and the current HIP stream; tensor shapes, dtypes and
devices are checked here so that no kernel is handed a buffer smaller than
the view implies. There is no fallback: if the library is missing, loading
fails with an error.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libflashcp.so")

FC_TWO_PASS = 0
FC_FUSED = 1

ERRORS = {
    -1: "FC_ERR_INVALID_ARG", -2: "FC_ERR_PLAN", -3: "FC_ERR_SHAPE", -4: "FC_ERR_UNSUPPORTED",
    -5: "FC_ERR_WORKSPACE", -6: "FC_ERR_HIP", -7: "FC_ERR_CAPACITY", -8: "FC_ERR_INTERNAL",
}

# every function the header declares
EXPORTS = [
    "fc_plan_per_doc", "fc_plan_per_seq", "fc_plan_whole_lpt", "fc_plan_hybrid", "fc_plan_validate",
    "fc_plan_stats", "fc_view_create", "fc_view_get_info", "fc_view_export", "fc_view_bind",
    "fc_view_destroy", "fc_view_export_launch", "fc_workspace_size", "fc_kv_gather", "fc_attn_fwd",
    "fc_attn_fwd_partial", "fc_attn_fwd_partials", "fc_lse_merge", "fc_attn_bwd", "fc_bwd_preprocess",
    "fc_attn_bwd_pass", "fc_attn_bwd_dkdv", "fc_attn_bwd_dq", "fc_attn_bwd_noalloc", "fc_last_error",
]

# bytes of the static device scratch behind fc_attn_bwd_noalloc (flashcp.h)
NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024


class FlashCPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class Shard(C.Structure):
    _fields_ = [("doc", C.c_int32), ("rank", C.c_int32), ("offset", C.c_int32), ("len", C.c_int32)]


class TileCfg(C.Structure):
    _fields_ = [("bm_fwd", C.c_int32), ("bn_fwd", C.c_int32), ("bm_bwd", C.c_int32),
                ("bn_bwd", C.c_int32)]


class ViewInfo(C.Structure):
    _fields_ = [
        ("t_q", C.c_int32), ("t_recv", C.c_int32), ("n_seg", C.c_int32), ("n_pieces", C.c_int32),
        ("hq", C.c_int32), ("hkv", C.c_int32), ("d", C.c_int32),
        ("bm_fwd", C.c_int32), ("bn_fwd", C.c_int32), ("bm_bwd", C.c_int32), ("bn_bwd", C.c_int32),
        ("pad_", C.c_int32),
        ("n_fwd_local", C.c_int64), ("n_fwd_recv", C.c_int64), ("n_fwd_fused", C.c_int64),
        ("n_bwd", C.c_int64), ("pairs_loc", C.c_int64), ("pairs_recv", C.c_int64),
        ("meta_bytes", C.c_int64), ("n_bwd_launch", C.c_int64), ("n_bwd_reduce", C.c_int64),
        ("n_bwd_slots", C.c_int64),
    ]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_ if k != "pad_"}


_lib = None
P = C.c_void_p
I32P = C.POINTER(C.c_int32)


def lib():
    """The loaded native library (loaded once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise FileNotFoundError(f"{_LIB_PATH} is not built; run python -m paper_2606_08476_amd.build")
        L = C.CDLL(_LIB_PATH)
        sig = {
            "fc_plan_per_doc": [I32P, C.c_int32, C.c_int32, C.POINTER(Shard), C.c_int64, C.POINTER(C.c_int64)],
            "fc_plan_per_seq": [I32P, C.c_int32, C.c_int32, C.POINTER(Shard), C.c_int64, C.POINTER(C.c_int64)],
            "fc_plan_whole_lpt": [I32P, C.c_int32, C.c_int32, C.POINTER(Shard), C.c_int64, C.POINTER(C.c_int64)],
            "fc_plan_hybrid": [I32P, C.c_int32, C.c_int32, C.c_double, C.POINTER(Shard), C.c_int64,
                               C.POINTER(C.c_int64), C.POINTER(C.c_uint8)],
            "fc_plan_validate": [I32P, C.c_int32, C.c_int32, C.POINTER(Shard), C.c_int64, C.c_int32],
            "fc_plan_stats": [I32P, C.c_int32, C.c_int32, C.POINTER(Shard), C.c_int64, C.c_int32, C.c_int32,
                              C.POINTER(C.c_int64), I32P, I32P, C.POINTER(C.c_int64), C.POINTER(C.c_int64),
                              C.POINTER(C.c_double)],
            "fc_view_create": [I32P, C.c_int32, C.POINTER(Shard), C.c_int64, C.c_int32, C.c_int32,
                               C.c_int32, C.c_int32, C.c_int32, C.POINTER(TileCfg), C.POINTER(P)],
            "fc_view_get_info": [P, C.POINTER(ViewInfo)],
            "fc_view_export": [P] + [I32P] * 11,
            "fc_view_bind": [P, P, C.c_size_t, P],
            "fc_view_export_launch": [P] + [I32P] * 6,
            "fc_workspace_size": [P, C.c_int32, C.POINTER(C.c_size_t), C.POINTER(C.c_size_t),
                                  C.POINTER(C.c_size_t)],
            "fc_kv_gather": [P, P, P, C.c_int64, P, P, P, P, P],
            "fc_attn_fwd": [P, P, P, P, P, P, C.c_float, C.c_int32, P, P, P, P, C.c_size_t, P],
            "fc_attn_fwd_partial": [P, C.c_int32, P, P, P, C.c_float, P, P, P],
            "fc_attn_fwd_partials": [P, P, P, P, P, P, C.c_float, P, P, P, P, P],
            "fc_lse_merge": [P, P, P, P, C.c_int32, C.c_int32, C.c_int32, P, P, P, P],
            "fc_attn_bwd": [P, P, P, P, P, P, P, P, P, P, C.c_float, C.c_int32, P, P, P, P, P, P,
                            C.c_size_t, P],
            "fc_bwd_preprocess": [P, P, P, P, P, P],
            "fc_attn_bwd_pass": [P, P, P, P, P, P, P, P, P, C.c_float, C.c_int32, P, P, P, P, P, P,
                                 C.c_size_t, P],
            "fc_attn_bwd_dkdv": [P, P, P, P, P, P, P, P, P, C.c_float, P, P, P, P, P, C.c_size_t, P],
            "fc_attn_bwd_dq": [P, P, P, P, P, P, P, P, P, C.c_float, P, P],
            "fc_attn_bwd_noalloc": [P, P, P, P, P, P, P, P, P, P, C.c_float, C.c_int32, P, P, P, P,
                                    P, P],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = C.c_int
        L.fc_view_destroy.argtypes = [P]
        L.fc_view_destroy.restype = None
        L.fc_last_error.argtypes = []
        L.fc_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _check(rc: int):
    if rc != 0:
        raise FlashCPError(rc, lib().fc_last_error().decode())


def _cu(cu):
    a = np.ascontiguousarray(np.asarray(cu, dtype=np.int32))
    return a, a.ctypes.data_as(I32P), int(a.size - 1)


def _shards(plan):
    plan = np.ascontiguousarray(np.asarray(plan, dtype=np.int32).reshape(-1, 4))
    arr = (Shard * max(1, len(plan)))()
    C.memmove(arr, plan.ctypes.data, plan.nbytes)
    return arr, len(plan)


def _plan_out(fn, *args):
    n = C.c_int64(0)
    cap = 1024
    while True:
        buf = (Shard * cap)()
        rc = fn(*args, buf, cap, C.byref(n))
        if rc == -7:
            cap = int(n.value)
            continue
        _check(rc)
        out = np.frombuffer(buf, dtype=np.int32, count=4 * n.value).reshape(-1, 4).copy()
        return out


# ------------------------------------------------------------------ planners

def fc_plan_per_doc(cu, cp: int) -> np.ndarray:
    a, p, n = _cu(cu)
    return _plan_out(lib().fc_plan_per_doc, p, n, cp)


def fc_plan_per_seq(cu, cp: int) -> np.ndarray:
    a, p, n = _cu(cu)
    return _plan_out(lib().fc_plan_per_seq, p, n, cp)


def fc_plan_whole_lpt(cu, cp: int) -> np.ndarray:
    a, p, n = _cu(cu)
    return _plan_out(lib().fc_plan_whole_lpt, p, n, cp)


def fc_plan_hybrid(cu, cp: int, target_r: float = 1.05):
    a, p, n = _cu(cu)
    isp = (C.c_uint8 * n)()
    cnt = C.c_int64(0)
    cap = 4 * n + 4 * cp + 16
    while True:
        buf = (Shard * cap)()
        rc = lib().fc_plan_hybrid(p, n, cp, float(target_r), buf, cap, C.byref(cnt), isp)
        if rc == -7:
            cap = int(cnt.value)
            continue
        _check(rc)
        plan = np.frombuffer(buf, dtype=np.int32, count=4 * cnt.value).reshape(-1, 4).copy()
        return plan, np.frombuffer(isp, dtype=np.uint8).copy()


def fc_plan_validate(cu, cp: int, plan, require_equal_tokens: bool = False) -> None:
    a, p, n = _cu(cu)
    s, m = _shards(plan)
    _check(lib().fc_plan_validate(p, n, cp, s, m, int(bool(require_equal_tokens))))


def fc_plan_stats(cu, cp: int, plan, hkv: int, d: int) -> dict:
    a, p, n = _cu(cu)
    s, m = _shards(plan)
    work = (C.c_int64 * cp)()
    tok = (C.c_int32 * cp)()
    rcv = (C.c_int32 * cp)()
    eq4, eq5, imb = C.c_int64(0), C.c_int64(0), C.c_double(0)
    _check(lib().fc_plan_stats(p, n, cp, s, m, hkv, d, work, tok, rcv, C.byref(eq4), C.byref(eq5),
                               C.byref(imb)))
    return dict(work=list(work), tokens=list(tok), recv_tokens=list(rcv), eq4=eq4.value,
                eq5=eq5.value, imbalance=imb.value)


# --------------------------------------------------------------------- views

class View:
    """An fc_view handle plus, once bound, the device buffer holding its
    tables. Destroyed with ``close()`` (or when garbage collected).
    ``tiles``: (bm_fwd, bn_fwd, bm_bwd, bn_bwd), 0 for a default; None for
    all defaults."""

    def __init__(self, cu, plan, cp: int, rank: int, hq: int, hkv: int, d: int, tiles=None):
        a, p, n = _cu(cu)
        s, m = _shards(plan)
        h = P()
        t = C.byref(TileCfg(*[int(x) for x in tiles])) if tiles is not None else None
        _check(lib().fc_view_create(p, n, s, m, cp, rank, hq, hkv, d, t, C.byref(h)))
        self._h = h
        self.meta = None
        info = ViewInfo()
        _check(lib().fc_view_get_info(self._h, C.byref(info)))
        self.info = info.as_dict()

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("view is closed")
        return self._h

    def export(self) -> dict:
        i = self.info
        sizes = dict(q_gpos=i["t_q"], recv_gpos=i["t_recv"], seg_doc=i["n_seg"],
                     q_cu_docseg=i["n_seg"] + 1, recv_cu=i["n_seg"] + 1, pieces=5 * i["n_pieces"],
                     lim=i["t_q"], fwd_local=8 * i["n_fwd_local"], fwd_recv=8 * i["n_fwd_recv"],
                     fwd_fused=8 * i["n_fwd_fused"], bwd=8 * i["n_bwd"])
        arrs = {k: np.zeros(max(1, v), dtype=np.int32) for k, v in sizes.items()}
        _check(lib().fc_view_export(self.handle, *[arrs[k].ctypes.data_as(I32P) for k in sizes]))
        out = {k: arrs[k][:sizes[k]] for k in sizes}
        out["pieces"] = out["pieces"].reshape(-1, 5)
        for k in ("fwd_local", "fwd_recv", "fwd_fused", "bwd"):
            out[k] = out[k].reshape(-1, 8)
        return out

    def export_launch(self) -> dict:
        """The launch tables exactly as uploaded (fc_view_export_launch)."""
        i = self.info
        nw = i["bn_bwd"] // 32
        sizes = dict(fwd_local=8 * i["n_fwd_local"], fwd_recv=8 * i["n_fwd_recv"],
                     fwd_fused=8 * i["n_fwd_fused"], bwd_launch=8 * i["n_bwd_launch"],
                     bwd_reduce=8 * i["n_bwd_reduce"], bwd_qfirst=nw * i["n_bwd_launch"])
        arrs = {k: np.zeros(max(1, v), dtype=np.int32) for k, v in sizes.items()}
        _check(lib().fc_view_export_launch(self.handle, *[arrs[k].ctypes.data_as(I32P) for k in sizes]))
        out = {k: arrs[k][:sizes[k]].reshape(-1, 8) for k in sizes if k != "bwd_qfirst"}
        out["bwd_qfirst"] = arrs["bwd_qfirst"][:sizes["bwd_qfirst"]].reshape(-1, nw)
        return out

    def bind(self, device="cuda", buf=None):
        """Upload the view's tables on the current stream into ``buf`` (a
        uint8 device tensor, allocated here if not given) and keep it."""
        import torch
        nbytes = int(self.info["meta_bytes"])
        if buf is None:
            buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-buf.data_ptr()) % 256
        if not buf.is_cuda or buf.numel() - off < nbytes:
            raise ValueError("metadata buffer too small or not on the device")
        self.meta = buf
        _check(lib().fc_view_bind(self.handle, buf.data_ptr() + off, nbytes, _stream()))
        return self

    def workspace_size(self, mode: int = FC_TWO_PASS):
        """(forward bytes, backward bytes, dK/dV-pass bytes)."""
        f, b, k = C.c_size_t(0), C.c_size_t(0), C.c_size_t(0)
        _check(lib().fc_workspace_size(self.handle, mode, C.byref(f), C.byref(b), C.byref(k)))
        return f.value, b.value, k.value

    def close(self):
        if getattr(self, "_h", None) is not None:
            lib().fc_view_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def _ptr(t, shape, dtype, name):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def fc_kv_gather(view: View, k_packed, v_packed, k_loc, v_loc, k_recv, v_recv):
    import torch
    i = view.info
    T = k_packed.shape[0]
    bf = torch.bfloat16
    args = [_ptr(k_packed, (T, i["hkv"], i["d"]), bf, "k_packed"),
            _ptr(v_packed, (T, i["hkv"], i["d"]), bf, "v_packed"), T,
            _ptr(k_loc, (i["t_q"], i["hkv"], i["d"]), bf, "k_loc"),
            _ptr(v_loc, (i["t_q"], i["hkv"], i["d"]), bf, "v_loc"),
            _ptr(k_recv, (i["t_recv"], i["hkv"], i["d"]), bf, "k_recv"),
            _ptr(v_recv, (i["t_recv"], i["hkv"], i["d"]), bf, "v_recv")]
    _check(lib().fc_kv_gather(view.handle, *args, _stream()))


def fc_attn_fwd(view: View, q, k_loc, v_loc, k_recv, v_recv, scale, mode, o, o_f32, lse, ws):
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    ws_ptr = ws.data_ptr() if ws is not None and ws.numel() else None
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().fc_attn_fwd(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), float(scale), int(mode),
        _ptr(o, (tq, hq, d), bf, "o"), _ptr(o_f32, (tq, hq, d), f32, "o_f32"),
        _ptr(lse, (hq, tq), f32, "lse"), ws_ptr, ws_bytes, _stream()))


def fc_attn_fwd_partial(view: View, src, q, k_src, v_src, scale, o_part, lse_part):
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, hq, hkv, d = i["t_q"], i["hq"], i["hkv"], i["d"]
    tk = tq if src == 0 else i["t_recv"]
    _check(lib().fc_attn_fwd_partial(
        view.handle, int(src), _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_src, (tk, hkv, d), bf, "k_src"),
        _ptr(v_src, (tk, hkv, d), bf, "v_src"), float(scale), _ptr(o_part, (tq, hq, d), f32, "o_part"),
        _ptr(lse_part, (hq, tq), f32, "lse_part"), _stream()))


def fc_attn_fwd_partials(view: View, q, k_loc, v_loc, k_recv, v_recv, scale, o_loc, lse_loc,
                         o_recv, lse_recv):
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    _check(lib().fc_attn_fwd_partials(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), float(scale),
        _ptr(o_loc, (tq, hq, d), f32, "o_loc"), _ptr(lse_loc, (hq, tq), f32, "lse_loc"),
        _ptr(o_recv, (tq, hq, d), f32, "o_recv"), _ptr(lse_recv, (hq, tq), f32, "lse_recv"),
        _stream()))


def fc_lse_merge(o_a, lse_a, o_b, lse_b, o_bf16, o_f32, lse_out):
    import torch
    t, h, d = o_a.shape
    f32, bf = torch.float32, torch.bfloat16
    _check(lib().fc_lse_merge(
        _ptr(o_a, (t, h, d), f32, "o_a"), _ptr(lse_a, (h, t), f32, "lse_a"),
        _ptr(o_b, (t, h, d), f32, "o_b"), _ptr(lse_b, (h, t), f32, "lse_b"), t, h, d,
        _ptr(o_bf16, (t, h, d), bf, "o_bf16"), _ptr(o_f32, (t, h, d), f32, "o_f32"),
        _ptr(lse_out, (h, t), f32, "lse_out"), _stream()))


def fc_attn_bwd(view: View, q, k_loc, v_loc, k_recv, v_recv, o, lse, dout, scale,
                dq, dk_loc, dv_loc, dk_recv, dv_recv, ws, deterministic: bool = True, o_f32=None):
    """o: the forward's bf16 output; o_f32 (optional): its fp32 output, from
    which delta is then computed (o may be None)."""
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    _check(lib().fc_attn_bwd(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), _ptr(o, (tq, hq, d), bf, "o"),
        _ptr(o_f32, (tq, hq, d), f32, "o_f32"), _ptr(lse, (hq, tq), f32, "lse"), _ptr(dout, (tq, hq, d), bf, "dout"), float(scale),
        int(bool(deterministic)),
        _ptr(dq, (tq, hq, d), f32, "dq"), _ptr(dk_loc, (tq, hkv, d), f32, "dk_loc"),
        _ptr(dv_loc, (tq, hkv, d), f32, "dv_loc"), _ptr(dk_recv, (tr, hkv, d), f32, "dk_recv"),
        _ptr(dv_recv, (tr, hkv, d), f32, "dv_recv"), ws.data_ptr(), ws.numel() * ws.element_size(),
        _stream()))


def fc_attn_bwd_noalloc(view: View, q, k_loc, v_loc, k_recv, v_recv, o, lse, dout, scale,
                        dq, dk_loc, dv_loc, dk_recv, dv_recv, deterministic: bool = True,
                        o_f32=None):
    """fc_attn_bwd with its workspace in the library's static device scratch
    (no device allocation)."""
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    _check(lib().fc_attn_bwd_noalloc(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), _ptr(o, (tq, hq, d), bf, "o"),
        _ptr(o_f32, (tq, hq, d), f32, "o_f32"), _ptr(lse, (hq, tq), f32, "lse"), _ptr(dout, (tq, hq, d), bf, "dout"), float(scale),
        int(bool(deterministic)),
        _ptr(dq, (tq, hq, d), f32, "dq"), _ptr(dk_loc, (tq, hkv, d), f32, "dk_loc"),
        _ptr(dv_loc, (tq, hkv, d), f32, "dv_loc"), _ptr(dk_recv, (tr, hkv, d), f32, "dk_recv"),
        _ptr(dv_recv, (tr, hkv, d), f32, "dv_recv"), _stream()))


def fc_bwd_preprocess(view: View, o, dout, delta, o_f32=None):
    """delta from the bf16 o, or from o_f32 when given (o may then be None)."""
    import torch
    i = view.info
    tq, hq, d = i["t_q"], i["hq"], i["d"]
    _check(lib().fc_bwd_preprocess(
        view.handle, _ptr(o, (tq, hq, d), torch.bfloat16, "o"),
        _ptr(o_f32, (tq, hq, d), torch.float32, "o_f32"),
        _ptr(dout, (tq, hq, d), torch.bfloat16, "dout"),
        _ptr(delta, (hq, tq), torch.float32, "delta"), _stream()))


def _ws(ws):
    if ws is None or ws.numel() == 0:
        return None, 0
    return ws.data_ptr(), ws.numel() * ws.element_size()


def fc_attn_bwd_pass(view: View, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale,
                     dq, dk_loc, dv_loc, dk_recv, dv_recv, ws=None, deterministic: bool = True):
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    _check(lib().fc_attn_bwd_pass(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), _ptr(lse, (hq, tq), f32, "lse"),
        _ptr(delta, (hq, tq), f32, "delta"), _ptr(dout, (tq, hq, d), bf, "dout"), float(scale),
        int(bool(deterministic)),
        _ptr(dq, (tq, hq, d), f32, "dq"), _ptr(dk_loc, (tq, hkv, d), f32, "dk_loc"),
        _ptr(dv_loc, (tq, hkv, d), f32, "dv_loc"), _ptr(dk_recv, (tr, hkv, d), f32, "dk_recv"),
        _ptr(dv_recv, (tr, hkv, d), f32, "dv_recv"), *_ws(ws), _stream()))


def fc_attn_bwd_dkdv(view: View, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale,
                     dk_loc, dv_loc, dk_recv, dv_recv, ws=None):
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    _check(lib().fc_attn_bwd_dkdv(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), _ptr(lse, (hq, tq), f32, "lse"),
        _ptr(delta, (hq, tq), f32, "delta"), _ptr(dout, (tq, hq, d), bf, "dout"), float(scale),
        _ptr(dk_loc, (tq, hkv, d), f32, "dk_loc"), _ptr(dv_loc, (tq, hkv, d), f32, "dv_loc"),
        _ptr(dk_recv, (tr, hkv, d), f32, "dk_recv"), _ptr(dv_recv, (tr, hkv, d), f32, "dv_recv"),
        *_ws(ws), _stream()))


def fc_attn_bwd_dq(view: View, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale, dq):
    import torch
    i = view.info
    bf, f32 = torch.bfloat16, torch.float32
    tq, tr, hq, hkv, d = i["t_q"], i["t_recv"], i["hq"], i["hkv"], i["d"]
    _check(lib().fc_attn_bwd_dq(
        view.handle, _ptr(q, (tq, hq, d), bf, "q"), _ptr(k_loc, (tq, hkv, d), bf, "k_loc"),
        _ptr(v_loc, (tq, hkv, d), bf, "v_loc"), _ptr(k_recv, (tr, hkv, d), bf, "k_recv"),
        _ptr(v_recv, (tr, hkv, d), bf, "v_recv"), _ptr(lse, (hq, tq), f32, "lse"),
        _ptr(delta, (hq, tq), f32, "delta"), _ptr(dout, (tq, hq, d), bf, "dout"), float(scale),
        _ptr(dq, (tq, hq, d), f32, "dq"), _stream()))
