// Kernel parameter blocks and host-side launchers (implemented in the .hip
// files). Only the C ABI layer calls these, after validating everything.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fck {

struct FwdParams {
  const uint16_t* q;        // [t_q, hq, d] bf16
  const uint16_t* k_recv;   // [t_r, hkv, d]
  const uint16_t* v_recv;
  const uint16_t* k_loc;    // [t_q, hkv, d]
  const uint16_t* v_loc;
  const int32_t* items;     // 8 int32 per item, in launch order: q0 q1 r0 r1 l0 l1 ldiag seg
  int32_t n_items;
  int32_t hq, hkv, group, head_chunks;
  float scale_log2;         // softmax scale * log2(e)
  // outputs; final: o_bf16 (+ o_f32 if non-null) + lse; partial: o_f32 + lse
  uint16_t* o_bf16;
  float* o_f32;
  float* lse;               // [hq, t_q]
  int32_t t_q;
  // both partials at once (non-null o_f32_recv): items carry a received and
  // a local range; the received partial goes to o_f32_recv/lse_recv, the
  // local one to o_f32/lse; with final output, the two are merged in the
  // kernel (o_f32_recv is then a workspace, lse_recv unused) and the final
  // O/LSE written as for the one-pass final output
  float* o_f32_recv;
  float* lse_recv;
};

struct BwdParams {
  const uint16_t* q;        // [t_q, hq, d]
  const uint16_t* dout;     // [t_q, hq, d]
  const float* lse;         // [hq, t_q] natural log
  const float* delta;       // [hq, t_q] rowsum(dO * O)
  const uint16_t* k_loc;
  const uint16_t* v_loc;
  const uint16_t* k_recv;
  const uint16_t* v_recv;
  const int32_t* items;     // 8 int32 per item, in launch order: k0 k1 q0 q1 qfull src seg slot
  const int32_t* lim;       // [t_q] receive index end per query
  const int32_t* qfirst;    // per item, per 32-key wave: first query row that sees it
  float* part_k;            // [slots, hkv, 128, d] partial dK/dV of split key tiles
  float* part_v;
  int32_t n_items;
  int32_t hq, hkv, group;
  float scale;
  float* dk_loc;            // [t_q, hkv, d] fp32
  float* dv_loc;
  float* dk_recv;           // [t_r, hkv, d] fp32
  float* dv_recv;
  int32_t t_q;
  float* dq;                // [t_q, hq, d] fp32, added into (atomic pass only)
};

struct DqParams {
  const uint16_t* q;        // [t_q, hq, d]
  const uint16_t* dout;     // [t_q, hq, d]
  const float* lse;         // [hq, t_q] natural log
  const float* delta;       // [hq, t_q]
  const uint16_t* k_recv;
  const uint16_t* v_recv;
  const uint16_t* k_loc;
  const uint16_t* v_loc;
  const int32_t* items;     // fused forward items, in launch order: q0 q1 r0 r1 l0 l1 ldiag seg
  int32_t n_items;
  int32_t hq, hkv, group, head_chunks;
  float scale;
  float* dq;                // [t_q, hq, d] fp32, written
  int32_t t_q;
};

hipError_t launch_fwd(const FwdParams& p, int d, int heads_per_tile, bool final_out,
                      hipStream_t s);
hipError_t launch_bwd_dq(const DqParams& p, int d, int heads_per_tile, hipStream_t s);
hipError_t launch_bwd(const BwdParams& p, int d, hipStream_t s);
// dK/dV with dQ added into p.dq by atomics (p.dq zeroed beforehand)
hipError_t launch_bwd_atomic(const BwdParams& p, int d, hipStream_t s);
// dK/dV and dQ in one launch (dK/dV workgroups first)
hipError_t launch_bwd_grid(const BwdParams& bp, const DqParams& dp, int d, int heads_per_tile,
                           hipStream_t s);
hipError_t launch_bwd_reduce(const int32_t* entries, int32_t n, const float* part_k,
                             const float* part_v, int32_t hkv, int32_t d, float* dk_loc,
                             float* dv_loc, float* dk_recv, float* dv_recv, hipStream_t s);
// delta = rowsum(dout * o), o the fp32 o_f32 when non-null, else the bf16
// o; with a non-null dq_zero, also zeroes that [t, h, d] fp32 tensor (the
// atomic backward's dQ) in the same pass
hipError_t launch_bwd_preprocess(const uint16_t* o, const float* o_f32, const uint16_t* dout,
                                 float* delta, int32_t t, int32_t h, int32_t d, float* dq_zero,
                                 hipStream_t s);
hipError_t launch_fill_zero(float* x, int64_t n, hipStream_t s);
hipError_t launch_lse_merge(const float* o_a, const float* lse_a, const float* o_b,
                            const float* lse_b, int32_t t, int32_t h, int32_t d, uint16_t* o_bf16,
                            float* o_f32, float* lse_out, hipStream_t s);
// rows r0 .. r1-1 of the concatenation (local rows 0 .. t_q-1, then the
// receive set)
hipError_t launch_kv_gather(const uint16_t* k, const uint16_t* v, const int32_t* q_gpos,
                            const int32_t* recv_gpos, int32_t t_q, int32_t t_r, int64_t r0,
                            int64_t r1, int32_t row_elems,
                            uint16_t* k_loc, uint16_t* v_loc, uint16_t* k_recv, uint16_t* v_recv,
                            hipStream_t s);

}  // namespace fck
