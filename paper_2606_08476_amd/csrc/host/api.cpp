// C ABI entry points that launch device work. Everything is validated on the
// host before the first launch; launches are asynchronous on the caller's
// stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <initializer_list>

#include "../kernels/launch.hpp"
#include "internal.hpp"
#include "view.hpp"

using fc::fail;
using fc::View;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int check_view(fc_view view, View*& v) {
  if (!view) return fail(FC_ERR_INVALID_ARG, "view is null");
  v = reinterpret_cast<View*>(view);
  if (!v->dev_meta) return fail(FC_ERR_WORKSPACE, "view is not bound to device metadata");
  return FC_OK;
}

// The kernels move tensor rows with 16-byte vector accesses and read
// LSE/delta per element: row tensors and workspaces must be 16-byte aligned,
// LSE and delta 4-byte aligned (NULL pointers are checked elsewhere).
int check_aligned(std::initializer_list<const void*> rows,
                  std::initializer_list<const void*> scalars = {}) {
  for (const void* p : rows)
    if (reinterpret_cast<uintptr_t>(p) % 16)
      return fail(FC_ERR_INVALID_ARG, "tensor and workspace pointers must be 16-byte aligned");
  for (const void* p : scalars)
    if (reinterpret_cast<uintptr_t>(p) % 4)
      return fail(FC_ERR_INVALID_ARG, "lse and delta pointers must be 4-byte aligned");
  return FC_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return FC_OK;
  return fail(FC_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

float resolve_scale(float scale, int d) { return scale > 0.f ? scale : 1.f / std::sqrt(float(d)); }

struct FwdWs {
  size_t o_bytes, l_bytes, total;
};
// FC_TWO_PASS with received keys: the received partial's fp32 O (the
// kernel merges it with the local partial in its epilogue), one slot of 32
// rows x d per wave, four waves per workgroup of the launch
FwdWs fwd_ws(const View& v, int32_t mode) {
  FwdWs w{};
  if (mode == FC_TWO_PASS && v.t_recv() > 0) {
    const size_t wgs = (v.fwd_fused.size() / 8) * size_t(v.hkv) *
                       size_t(v.hq / v.hkv / v.heads_per_tile);
    w.o_bytes = align_up(wgs * 4 * 32 * size_t(v.d) * sizeof(float));
    w.total = w.o_bytes;
  }
  return w;
}
size_t delta_ws(const View& v) { return align_up(size_t(v.t_q()) * v.hq * sizeof(float)); }
size_t part_ws(const View& v) {
  return 2 * size_t(v.n_bwd_slots) * v.hkv * v.bn_bwd * v.d * sizeof(float);
}
size_t bwd_ws(const View& v) { return delta_ws(v) + part_ws(v); }

fck::FwdParams fwd_params(const View& v, const int32_t* items, int64_t n,
                          const void* q, const void* k_loc, const void* v_loc, const void* k_recv,
                          const void* v_recv, float scale) {
  fck::FwdParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k_loc = static_cast<const uint16_t*>(k_loc);
  p.v_loc = static_cast<const uint16_t*>(v_loc);
  p.k_recv = static_cast<const uint16_t*>(k_recv);
  p.v_recv = static_cast<const uint16_t*>(v_recv);
  p.items = items;
  p.n_items = int32_t(n);
  p.hq = v.hq;
  p.hkv = v.hkv;
  p.group = v.hq / v.hkv;
  p.head_chunks = p.group / v.heads_per_tile;
  p.scale_log2 = resolve_scale(scale, v.d) * 1.4426950408889634f;
  p.t_q = v.t_q();
  return p;
}

// Both partial passes of the two-pass forward in one launch over the fused
// items: each workgroup runs its query tile's received range, writes that
// partial (o_recv, lse_recv), then runs the local range (o_loc, lse_loc).
int launch_partials(const View& v, const void* q, const void* k_loc, const void* v_loc,
                    const void* k_recv, const void* v_recv, float scale, float* o_loc,
                    float* lse_loc, float* o_recv, float* lse_recv, hipStream_t s) {
  const int32_t* m = v.dev_meta;
  fck::FwdParams p = fwd_params(v, m + v.off.fwd_fused,
                                int64_t(v.fwd_fused.size() / 8), q, k_loc, v_loc, k_recv, v_recv,
                                scale);
  p.o_f32 = o_loc;
  p.lse = lse_loc;
  p.o_f32_recv = o_recv;
  p.lse_recv = lse_recv;
  return hip_status(fck::launch_fwd(p, v.d, v.heads_per_tile, false, s), "attn_fwd launch");
}

fck::BwdParams bwd_params(const View& v, const void* q, const void* k_loc, const void* v_loc,
                          const void* k_recv, const void* v_recv, const float* lse,
                          const float* delta, const void* dout, float scale, float* dk_loc,
                          float* dv_loc, float* dk_recv, float* dv_recv, void* ws, size_t part) {
  const int32_t* m = v.dev_meta;
  fck::BwdParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.dout = static_cast<const uint16_t*>(dout);
  p.lse = lse;
  p.delta = delta;
  p.k_loc = static_cast<const uint16_t*>(k_loc);
  p.v_loc = static_cast<const uint16_t*>(v_loc);
  p.k_recv = static_cast<const uint16_t*>(k_recv);
  p.v_recv = static_cast<const uint16_t*>(v_recv);
  p.items = m + v.off.bwd_launch;
  p.lim = m + v.off.lim;
  p.qfirst = m + v.off.bwd_qfirst;
  p.n_items = int32_t(v.bwd_launch.size() / 8);
  p.part_k = static_cast<float*>(ws);
  p.part_v = part ? reinterpret_cast<float*>(static_cast<char*>(ws) + part / 2) : nullptr;
  p.hq = v.hq;
  p.hkv = v.hkv;
  p.group = v.hq / v.hkv;
  p.scale = resolve_scale(scale, v.d);
  p.dk_loc = dk_loc;
  p.dv_loc = dv_loc;
  p.dk_recv = dk_recv;
  p.dv_recv = dv_recv;
  p.t_q = v.t_q();
  return p;
}

fck::DqParams dq_params(const View& v, const void* q, const void* k_loc, const void* v_loc,
                        const void* k_recv, const void* v_recv, const float* lse,
                        const float* delta, const void* dout, float scale, float* dq) {
  const int32_t* m = v.dev_meta;
  fck::DqParams d{};
  d.q = static_cast<const uint16_t*>(q);
  d.dout = static_cast<const uint16_t*>(dout);
  d.lse = lse;
  d.delta = delta;
  d.k_loc = static_cast<const uint16_t*>(k_loc);
  d.v_loc = static_cast<const uint16_t*>(v_loc);
  d.k_recv = static_cast<const uint16_t*>(k_recv);
  d.v_recv = static_cast<const uint16_t*>(v_recv);
  d.items = m + v.off.fwd_fused;
  d.n_items = int32_t(v.fwd_fused.size() / 8);
  d.hq = v.hq;
  d.hkv = v.hkv;
  d.group = v.hq / v.hkv;
  d.head_chunks = d.group / v.heads_per_tile;
  d.scale = resolve_scale(scale, v.d);
  d.dq = dq;
  d.t_q = v.t_q();
  return d;
}

int launch_reduce(const View& v, const fck::BwdParams& p, hipStream_t s) {
  return hip_status(fck::launch_bwd_reduce(v.dev_meta + v.off.bwd_reduce,
                                           int32_t(v.bwd_reduce.size() / 8), p.part_k, p.part_v,
                                           v.hkv, v.d, p.dk_loc, p.dv_loc, p.dk_recv, p.dv_recv, s),
                    "attn_bwd reduce launch");
}

// The backward pass once delta is known (arguments validated by the
// caller). Deterministic: dK/dV and dQ workgroups in one launch (dQ written
// once by the workgroup owning its rows). Otherwise key tiles only, each
// adding its share of dQ into `dq` with atomics; `dq` must be zero on
// entry. Either way the split key tiles' partial dK/dV are then reduced.
int run_pass(const View& v, const void* q, const void* k_loc, const void* v_loc,
             const void* k_recv, const void* v_recv, const float* lse, const float* delta,
             const void* dout, float scale, int32_t deterministic, float* dq, float* dk_loc,
             float* dv_loc, float* dk_recv, float* dv_recv, void* ws, size_t need,
             hipStream_t s) {
  fck::BwdParams p = bwd_params(v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale,
                                dk_loc, dv_loc, dk_recv, dv_recv, ws, need);
  if (deterministic) {
    const fck::DqParams d = dq_params(v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout,
                                      scale, dq);
    if (int rc = hip_status(fck::launch_bwd_grid(p, d, v.d, v.heads_per_tile, s),
                            "attn_bwd launch"))
      return rc;
  } else {
    p.dq = dq;
    if (int rc = hip_status(fck::launch_bwd_atomic(p, v.d, s), "attn_bwd (atomic dQ) launch"))
      return rc;
  }
  return launch_reduce(v, p, s);
}

}  // namespace

extern "C" {

int fc_workspace_size(fc_view view, int32_t mode, size_t* fwd_bytes, size_t* bwd_bytes,
                      size_t* dkdv_bytes) {
  fc::clear_error();
  if (!view) return fail(FC_ERR_INVALID_ARG, "view is null");
  if (mode != FC_TWO_PASS && mode != FC_FUSED) return fail(FC_ERR_INVALID_ARG, "bad mode");
  const View& v = *reinterpret_cast<View*>(view);
  if (fwd_bytes) *fwd_bytes = fwd_ws(v, mode).total;
  if (bwd_bytes) *bwd_bytes = bwd_ws(v);
  if (dkdv_bytes) *dkdv_bytes = part_ws(v);
  return FC_OK;
}

int fc_kv_gather(fc_view view, const void* k_packed, const void* v_packed, int64_t t_packed,
                 void* k_loc, void* v_loc, void* k_recv, void* v_recv, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({k_packed, v_packed, k_loc, v_loc, k_recv, v_recv})) return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() + v->t_recv() == 0) return FC_OK;
  // a part whose two outputs are both NULL is skipped
  const bool loc = k_loc || v_loc, rcv = k_recv || v_recv;
  if (!k_packed || !v_packed || (loc && (!k_loc || !v_loc)) || (rcv && (!k_recv || !v_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  if (!loc && !rcv) return fail(FC_ERR_INVALID_ARG, "nothing to gather: every output is null");
  const int64_t r0 = loc ? 0 : v->t_q(), r1 = rcv ? v->t_q() + v->t_recv() : v->t_q();
  // every gathered position must lie inside the packed tensors
  int64_t max_pos = -1;
  if (loc && v->t_q()) max_pos = std::max<int64_t>(max_pos, v->q_gpos.back());
  if (rcv && v->t_recv()) max_pos = std::max<int64_t>(max_pos, v->recv_gpos.back());
  if (max_pos >= t_packed)
    return fail(FC_ERR_SHAPE, "packed K/V have " + std::to_string(t_packed) +
                                  " rows, the view reads row " + std::to_string(max_pos));
  const int32_t* m = v->dev_meta;
  return hip_status(
      fck::launch_kv_gather(static_cast<const uint16_t*>(k_packed),
                            static_cast<const uint16_t*>(v_packed), m + v->off.q_gpos,
                            m + v->off.recv_gpos, v->t_q(), v->t_recv(), r0, r1, v->hkv * v->d,
                            static_cast<uint16_t*>(k_loc), static_cast<uint16_t*>(v_loc),
                            static_cast<uint16_t*>(k_recv), static_cast<uint16_t*>(v_recv),
                            reinterpret_cast<hipStream_t>(stream)),
      "kv_gather launch");
}

int fc_attn_fwd_partial(fc_view view, int32_t src, const void* q, const void* k_src,
                        const void* v_src, float scale, float* o_part, float* lse_part,
                        void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_src, v_src, o_part}, {lse_part})) return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (src != 0 && src != 1) return fail(FC_ERR_INVALID_ARG, "src must be 0 or 1");
  if (v->t_q() == 0) return FC_OK;
  const bool have_keys = src == 0 ? true : v->t_recv() > 0;
  if (!q || !o_part || !lse_part || (have_keys && (!k_src || !v_src)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  const int32_t* m = v->dev_meta;
  fck::FwdParams p =
      src == 0 ? fwd_params(*v, m + v->off.fwd_local,
                            int64_t(v->fwd_local.size() / 8), q, k_src, v_src, nullptr, nullptr,
                            scale)
               : fwd_params(*v, m + v->off.fwd_recv,
                            int64_t(v->fwd_recv.size() / 8), q, nullptr, nullptr, k_src, v_src,
                            scale);
  p.o_f32 = o_part;
  p.lse = lse_part;
  return hip_status(fck::launch_fwd(p, v->d, v->heads_per_tile, false,
                                    reinterpret_cast<hipStream_t>(stream)),
                    "attn_fwd launch");
}

int fc_attn_fwd_partials(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                         const void* k_recv, const void* v_recv, float scale, float* o_loc,
                         float* lse_loc, float* o_recv, float* lse_recv, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_loc, v_loc, k_recv, v_recv, o_loc, o_recv},
                              {lse_loc, lse_recv}))
    return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() == 0) return FC_OK;
  if (!q || !k_loc || !v_loc || !o_loc || !lse_loc || !o_recv || !lse_recv ||
      (v->t_recv() && (!k_recv || !v_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  return launch_partials(*v, q, k_loc, v_loc, k_recv, v_recv, scale, o_loc, lse_loc, o_recv,
                         lse_recv, reinterpret_cast<hipStream_t>(stream));
}

int fc_attn_fwd(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                const void* k_recv, const void* v_recv, float scale, int32_t mode, void* o,
                float* o_f32, float* lse, void* ws, size_t ws_bytes, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_loc, v_loc, k_recv, v_recv, o, o_f32, ws}, {lse})) return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (mode != FC_TWO_PASS && mode != FC_FUSED) return fail(FC_ERR_INVALID_ARG, "bad mode");
  if (v->t_q() == 0) return FC_OK;
  if (!q || !k_loc || !v_loc || !o || !lse || (v->t_recv() && (!k_recv || !v_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  const FwdWs w = fwd_ws(*v, mode);
  if (ws_bytes < w.total || (w.total && !ws))
    return fail(FC_ERR_WORKSPACE, "forward workspace of " + std::to_string(ws_bytes) +
                                      " bytes, need " + std::to_string(w.total));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int32_t* m = v->dev_meta;
  if (mode == FC_FUSED || v->t_recv() == 0) {
    // one pass: both sources (fused items), or the local source alone
    const bool fused = mode == FC_FUSED && v->t_recv() > 0;
    fck::FwdParams p =
        fused ? fwd_params(*v, m + v->off.fwd_fused,
                           int64_t(v->fwd_fused.size() / 8), q, k_loc, v_loc, k_recv, v_recv, scale)
              : fwd_params(*v, m + v->off.fwd_local,
                           int64_t(v->fwd_local.size() / 8), q, k_loc, v_loc, nullptr, nullptr,
                           scale);
    p.o_bf16 = static_cast<uint16_t*>(o);
    p.o_f32 = o_f32;
    p.lse = lse;
    return hip_status(fck::launch_fwd(p, v->d, v->heads_per_tile, true, s), "attn_fwd launch");
  }
  // both partial passes and their log-sum-exp merge in one launch: each
  // workgroup runs its query tile's received range (partial O to the
  // workspace), then its local range, and merges the two in its epilogue
  fck::FwdParams p = fwd_params(*v, m + v->off.fwd_fused,
                                int64_t(v->fwd_fused.size() / 8), q, k_loc, v_loc, k_recv,
                                v_recv, scale);
  p.o_f32_recv = static_cast<float*>(ws);
  p.o_bf16 = static_cast<uint16_t*>(o);
  p.o_f32 = o_f32;
  p.lse = lse;
  return hip_status(fck::launch_fwd(p, v->d, v->heads_per_tile, true, s), "attn_fwd launch");
}

int fc_lse_merge(const float* o_a, const float* lse_a, const float* o_b, const float* lse_b,
                 int32_t t, int32_t h, int32_t d, void* o_bf16, float* o_f32, float* lse_out,
                 void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({o_a, o_b, o_bf16, o_f32}, {lse_a, lse_b, lse_out})) return rc;
  if (t < 0 || h < 0) return fail(FC_ERR_INVALID_ARG, "negative size");
  if (d != 64 && d != 128) return fail(FC_ERR_UNSUPPORTED, "head dim must be 64 or 128");
  if (int64_t(t) * h == 0) return FC_OK;
  if (!o_a || !lse_a || !o_b || !lse_b || !o_bf16 || !lse_out)
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  return hip_status(fck::launch_lse_merge(o_a, lse_a, o_b, lse_b, t, h, d,
                                          static_cast<uint16_t*>(o_bf16), o_f32, lse_out,
                                          reinterpret_cast<hipStream_t>(stream)),
                    "lse_merge launch");
}

int fc_bwd_preprocess(fc_view view, const void* o, const float* o_f32, const void* dout,
                      float* delta, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({o, o_f32, dout}, {delta})) return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() == 0) return FC_OK;
  if ((!o && !o_f32) || !dout || !delta) return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  return hip_status(fck::launch_bwd_preprocess(static_cast<const uint16_t*>(o), o_f32,
                                               static_cast<const uint16_t*>(dout), delta,
                                               v->t_q(), v->hq, v->d, nullptr,
                                               reinterpret_cast<hipStream_t>(stream)),
                    "bwd preprocess launch");
}

int fc_attn_bwd_dkdv(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                     const void* k_recv, const void* v_recv, const float* lse, const float* delta,
                     const void* dout, float scale, float* dk_loc, float* dv_loc, float* dk_recv,
                     float* dv_recv, void* ws, size_t ws_bytes, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_loc, v_loc, k_recv, v_recv, dout, dk_loc, dv_loc, dk_recv,
                               dv_recv, ws},
                              {lse, delta}))
    return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() == 0) return FC_OK;
  if (!q || !k_loc || !v_loc || !lse || !delta || !dout || !dk_loc || !dv_loc ||
      (v->t_recv() && (!k_recv || !v_recv || !dk_recv || !dv_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  const size_t need = part_ws(*v);
  if (need && (!ws || ws_bytes < need))
    return fail(FC_ERR_WORKSPACE, "dK/dV workspace of " + std::to_string(ws_bytes) +
                                      " bytes, need " + std::to_string(need));
  fck::BwdParams p = bwd_params(*v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale,
                                dk_loc, dv_loc, dk_recv, dv_recv, ws, need);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (int rc = hip_status(fck::launch_bwd(p, v->d, s), "attn_bwd dK/dV launch")) return rc;
  return launch_reduce(*v, p, s);
}

int fc_attn_bwd_dq(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                   const void* k_recv, const void* v_recv, const float* lse, const float* delta,
                   const void* dout, float scale, float* dq, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_loc, v_loc, k_recv, v_recv, dout, dq}, {lse, delta})) return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() == 0) return FC_OK;
  if (!q || !k_loc || !v_loc || !lse || !delta || !dout || !dq ||
      (v->t_recv() && (!k_recv || !v_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  fck::DqParams d = dq_params(*v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale, dq);
  return hip_status(fck::launch_bwd_dq(d, v->d, v->heads_per_tile,
                                       reinterpret_cast<hipStream_t>(stream)),
                    "attn_bwd dQ launch");
}

int fc_attn_bwd_pass(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                     const void* k_recv, const void* v_recv, const float* lse, const float* delta,
                     const void* dout, float scale, int32_t deterministic, float* dq,
                     float* dk_loc, float* dv_loc, float* dk_recv, float* dv_recv, void* ws,
                     size_t ws_bytes, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_loc, v_loc, k_recv, v_recv, dout, dq, dk_loc, dv_loc, dk_recv,
                               dv_recv, ws},
                              {lse, delta}))
    return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() == 0) return FC_OK;
  if (!q || !k_loc || !v_loc || !lse || !delta || !dout || !dq || !dk_loc || !dv_loc ||
      (v->t_recv() && (!k_recv || !v_recv || !dk_recv || !dv_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  const size_t need = part_ws(*v);
  if (need && (!ws || ws_bytes < need))
    return fail(FC_ERR_WORKSPACE, "dK/dV workspace of " + std::to_string(ws_bytes) +
                                      " bytes, need " + std::to_string(need));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (!deterministic &&
      hip_status(fck::launch_fill_zero(dq, int64_t(v->t_q()) * v->hq * v->d, s), "dq zero fill"))
    return FC_ERR_HIP;
  return run_pass(*v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale, deterministic,
                  dq, dk_loc, dv_loc, dk_recv, dv_recv, ws, need, s);
}

int fc_attn_bwd(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                const void* k_recv, const void* v_recv, const void* o, const float* o_f32,
                const float* lse, const void* dout, float scale, int32_t deterministic, float* dq,
                float* dk_loc, float* dv_loc, float* dk_recv, float* dv_recv, void* ws,
                size_t ws_bytes, void* stream) {
  fc::clear_error();
  if (int rc = check_aligned({q, k_loc, v_loc, k_recv, v_recv, o, o_f32, dout, dq, dk_loc, dv_loc,
                               dk_recv, dv_recv, ws},
                              {lse}))
    return rc;
  View* v;
  if (int rc = check_view(view, v)) return rc;
  if (v->t_q() == 0) return FC_OK;
  const size_t need = bwd_ws(*v);
  if (!ws || ws_bytes < need)
    return fail(FC_ERR_WORKSPACE, "backward workspace of " + std::to_string(ws_bytes) +
                                      " bytes, need " + std::to_string(need));
  if ((!o && !o_f32) || !q || !k_loc || !v_loc || !lse || !dout || !dq || !dk_loc || !dv_loc ||
      (v->t_recv() && (!k_recv || !v_recv || !dk_recv || !dv_recv)))
    return fail(FC_ERR_INVALID_ARG, "null tensor pointer");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  float* delta = static_cast<float*>(ws);
  // the preprocess also zeroes dq for the atomic pass
  if (int rc = hip_status(fck::launch_bwd_preprocess(static_cast<const uint16_t*>(o), o_f32,
                                                     static_cast<const uint16_t*>(dout), delta,
                                                     v->t_q(), v->hq, v->d,
                                                     deterministic ? nullptr : dq, s),
                          "bwd preprocess launch"))
    return rc;
  const size_t dbytes = delta_ws(*v);
  return run_pass(*v, q, k_loc, v_loc, k_recv, v_recv, lse, delta, dout, scale, deterministic,
                  dq, dk_loc, dv_loc, dk_recv, dv_recv, static_cast<char*>(ws) + dbytes,
                  part_ws(*v), s);
}

}  // extern "C"
