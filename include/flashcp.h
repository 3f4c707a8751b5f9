/*
 * flashcp.h -- C ABI of the MI355X rank-shard attention library.
 *
 * The library computes one context-parallel rank's share of
 * document-masked causal attention, forward and backward, for a packed
 * multi-document sequence sharded by a FlashCP plan (FlashCP, "Load-Balanced
 * Communication-Efficient Context Parallelism for LLM Training").
 *
 *   - Problem statement (documents D, CP degree N, shards s_i with prefix
 *     p_i, assignment x_ij, equal-token constraint): Sec. 3.1, Eq. 1-3.
 *   - Sharding-aware receive set (only the KV prefix a rank's queries need,
 *     compacted into one buffer): Sec. 3.2, Eq. 5.
 *   - Per-Doc sharding (worker i takes chunks i and 2N-1-i): Sec. 2.3.
 *   - Whole-Doc and hybrid sharding (Algorithm 1): Sec. 3.3-3.4.
 *   - Document mask (a query sees earlier-or-same tokens of its own
 *     document): Sec. 2.1.
 *   - Partial results over separate KV sets merged by log-sum-exp (the
 *     aggregation blockwise CP attention needs): Sec. 2.3, Sec. 4.2.
 *
 * Conventions
 *   - Every call returns an fc_status: FC_OK (0) or a negative FC_ERR_*.
 *     On error fc_last_error() returns a message (thread-local), and
 *     nothing has been launched: all validation is done on the host first.
 *   - Device calls are asynchronous on the caller's stream (`stream` is a
 *     hipStream_t; NULL means the default stream).
 *   - The caller owns every buffer it passes. Device pointers must point to
 *     device memory of at least the size stated; the library cannot check
 *     their extent. Host pointers are read or written before return.
 *   - Alignment: tensors of d-element rows (q, k, v, o, dout, dq, dk, dv,
 *     fp32 outputs and partials) and workspaces 16 bytes, lse and delta 4
 *     bytes; a misaligned pointer is rejected with FC_ERR_INVALID_ARG.
 *   - The library owns fc_view objects (host memory only). A view is bound
 *     to a caller-owned device buffer by fc_view_bind; that buffer must stay
 *     alive and unmodified while work launched with the view is in flight.
 *   - Tensor layouts are row-major ("THD"):
 *       q, o, dout, dq            [T_q, Hq, d]
 *       k_loc, v_loc, dk_loc, dv_loc   [T_q, Hkv, d]   (the rank's own tokens,
 *                                                       in local order)
 *       k_recv, v_recv, dk_recv, dv_recv [T_r, Hkv, d]  (received tokens,
 *                                                       ascending position)
 *       lse                       [Hq, T_q] fp32, natural logarithm
 *     bf16 for q/k/v/o/dout, fp32 for lse/dq/dk/dv. d is 64 or 128,
 *     Hq % Hkv == 0, and Hq / Hkv is 1, 2, 4 or 8. Query head h uses KV head
 *     h / (Hq / Hkv). scale <= 0 selects 1/sqrt(d).
 *   - Local order: a rank's query tokens sorted by global position.
 */
#ifndef FLASHCP_H
#define FLASHCP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  FC_OK = 0,
  FC_ERR_INVALID_ARG = -1, /* null pointer, negative size, bad enum value */
  FC_ERR_PLAN = -2,        /* plan violates Eq. 1 (or Eq. 2 when required) */
  FC_ERR_SHAPE = -3,       /* sizes inconsistent with the view */
  FC_ERR_UNSUPPORTED = -4, /* head dim or group size not compiled in */
  FC_ERR_WORKSPACE = -5,   /* workspace too small, or view not bound */
  FC_ERR_HIP = -6,         /* a HIP runtime call failed */
  FC_ERR_CAPACITY = -7,    /* output array too small; *n_out holds the need */
  FC_ERR_INTERNAL = -8     /* a table the library built failed its own bounds
                              check before upload (a library bug) */
};

/* fwd pass modes */
enum {
  FC_TWO_PASS = 0, /* local pass + received pass, then the LSE merge */
  FC_FUSED = 1     /* one pass over received then local keys, no merge */
};

/* One document shard (Sec. 3.1): `len` tokens of document `doc` starting
 * `offset` tokens into it (its prefix length p_i), assigned to worker
 * `rank` (x_ij = 1). */
typedef struct {
  int32_t doc, rank, offset, len;
} fc_shard;

/* ------------------------------------------------------------------ plans
 * Inputs common to the planners: cu_seqlens[n_docs+1] (host, int32,
 * cu_seqlens[0] = 0, non-decreasing, every document length >= 1), the CP
 * degree cp >= 1. Outputs are canonical: sorted by (doc, offset), adjacent
 * shards of one document on one rank joined. `out` (host, capacity `cap`
 * shards) receives the plan and *n_out its length; if cap is too small,
 * FC_ERR_CAPACITY is returned with *n_out set to the needed count. */

/* Per-Doc sharding (Sec. 2.3): document k of length L is cut at
 * floor(j*L/(2cp)), j = 0..2cp; chunk i goes to worker min(i, 2cp-1-i);
 * empty chunks are dropped. */
int fc_plan_per_doc(const int32_t* cu_seqlens, int32_t n_docs, int32_t cp,
                    fc_shard* out, int64_t cap, int64_t* n_out);

/* Per-sequence sharding, the Llama3 CP baseline (Sec. 2.2): the packed
 * sequence of C = cu_seqlens[n_docs] tokens, not each document, is cut at
 * floor(j*C/(2cp)), j = 0..2cp; chunk i goes to worker min(i, 2cp-1-i); a
 * chunk that spans documents gives one shard per document it meets. */
int fc_plan_per_seq(const int32_t* cu_seqlens, int32_t n_docs, int32_t cp,
                    fc_shard* out, int64_t cap, int64_t* n_out);

/* Whole documents only, longest first onto the least-loaded worker by
 * workload W (Algorithm 1, the Min_Worker_Add loop); ties go to the lower
 * document index and the lower worker index. Eq. 2 is not enforced. */
int fc_plan_whole_lpt(const int32_t* cu_seqlens, int32_t n_docs, int32_t cp,
                      fc_shard* out, int64_t cap, int64_t* n_out);

/* The hybrid heuristic (Algorithm 1): whole-doc LPT, an equal-token repair
 * that moves only document prefixes (Whole_Doc_Shard_and_Add, Sec. 3.3),
 * and the longest remaining document moved to Per-Doc while the imbalance
 * max W / mean W exceeds target_r (> 0; 1.05 is the usual value).
 * Requires cp | C. is_per_doc (host, n_docs bytes, may be NULL) receives 1
 * for documents sharded Per-Doc. */
int fc_plan_hybrid(const int32_t* cu_seqlens, int32_t n_docs, int32_t cp,
                   double target_r, fc_shard* out, int64_t cap, int64_t* n_out,
                   uint8_t* is_per_doc);

/* FC_OK if every token is assigned to exactly one worker (Eq. 1) and, when
 * require_equal_tokens != 0, every worker holds C/cp tokens (Eq. 2);
 * FC_ERR_PLAN otherwise. Shards need not be in canonical order. */
int fc_plan_validate(const int32_t* cu_seqlens, int32_t n_docs, int32_t cp,
                     const fc_shard* shards, int64_t n_shards,
                     int32_t require_equal_tokens);

/* Plan statistics (host outputs, each array of cp entries):
 *   work[j]        sum over j's shards of W_i = (2p_i + s_i + 1) s_i / 2
 *                  (Sec. 3.1), the pairs its queries see;
 *   tokens[j]      tokens held;
 *   recv_tokens[j] size of j's sharding-aware receive set (Sec. 3.2);
 *   *eq4           4 * (C/cp) * hkv * d * (cp-1) elements (Eq. 4, full KV);
 *   *eq5           4 * max_j (tokens of j's non-last shards) * hkv * d *
 *                  (cp-1) elements (Eq. 5);
 *   *imbalance     max_j work / mean_j work (Sec. 3.4).
 * Any output pointer may be NULL. The plan must pass fc_plan_validate. */
int fc_plan_stats(const int32_t* cu_seqlens, int32_t n_docs, int32_t cp,
                  const fc_shard* shards, int64_t n_shards, int32_t hkv, int32_t d,
                  int64_t* work, int32_t* tokens, int32_t* recv_tokens,
                  int64_t* eq4, int64_t* eq5, double* imbalance);

/* ------------------------------------------------------------------ views
 * A rank view: the rank's query tokens (local order), its receive set R_r
 * (all earlier tokens of its documents that it does not hold, ascending,
 * compacted), and the tile maps the kernels execute, for one head
 * configuration. Built on the host only. */
typedef struct fc_view_s* fc_view;

typedef struct {
  int32_t t_q, t_recv;          /* local query tokens, received tokens */
  int32_t n_seg, n_pieces;      /* documents present, contiguous pieces */
  int32_t hq, hkv, d;
  int32_t bm_fwd, bn_fwd;       /* forward tile: query tokens, keys */
  int32_t bm_bwd, bn_bwd;       /* backward tile: query tokens, keys */
  int32_t pad_;
  int64_t n_fwd_local, n_fwd_recv, n_fwd_fused, n_bwd; /* work items */
  int64_t pairs_loc, pairs_recv; /* visible (query, key) pairs per head */
  int64_t meta_bytes;           /* device bytes fc_view_bind needs */
  int64_t n_bwd_launch;         /* backward launch items after splitting long */
  int64_t n_bwd_reduce;         /*   key tiles; key tiles split; partial slots */
  int64_t n_bwd_slots;
} fc_view_info;

/* Tile shapes of a view; 0 in a field selects its default.
 *   bm_fwd  query rows per workgroup of the forward and of the dQ pass: 32,
 *           64 or 128, i.e. 4, 2 or 1 query heads of a KV-head group per
 *           workgroup (each wave takes a quarter of the rows of every one of
 *           those heads, a (row, head) per lane); 128/bm_fwd must divide
 *           Hq/Hkv. Default: as many heads per workgroup as the group
 *           allows, min(Hq/Hkv, 4) (bm_fwd = 32 when Hq/Hkv >= 4).
 *   bn_fwd  keys per forward / dQ tile: 64 (the compiled shape).
 *   bm_bwd  (query row, head) pairs per dK/dV iteration: 32 (compiled;
 *           8 rows of 4 heads, 16 of 2 or 32 of 1, as the group allows).
 *   bn_bwd  keys per dK/dV workgroup: 128 (compiled).
 * Other values give FC_ERR_UNSUPPORTED. */
typedef struct {
  int32_t bm_fwd, bn_fwd, bm_bwd, bn_bwd;
} fc_tile_cfg;

/* Build rank `rank`'s view of a validated plan (FC_ERR_PLAN otherwise) for
 * hq query heads, hkv KV heads and head dim d, with the tile shapes of
 * `tiles` (NULL: all defaults). *out receives the view. */
int fc_view_create(const int32_t* cu_seqlens, int32_t n_docs, const fc_shard* shards,
                   int64_t n_shards, int32_t cp, int32_t rank, int32_t hq, int32_t hkv,
                   int32_t d, const fc_tile_cfg* tiles, fc_view* out);

int fc_view_get_info(fc_view view, fc_view_info* out);

/* Copy the view's tables to host arrays (any pointer may be NULL):
 *   q_gpos[t_q], recv_gpos[t_recv]   global positions;
 *   seg_doc[n_seg]                   document of each segment;
 *   q_cu_docseg[n_seg+1]             local index bounds of each segment;
 *   recv_cu[n_seg+1]                 receive-buffer bounds of each segment;
 *   pieces[n_pieces*5]               (seg, q_start, q_end, g_start, n_P):
 *                                    a maximal run of held positions and
 *                                    the count of received tokens before it;
 *   lim[t_q]                         receive index end each query sees;
 *   fwd_local/fwd_recv/fwd_fused[n*8] (q0, q1, r0, r1, l0, l1, ldiag, seg);
 *   bwd[n_bwd*8]                     (k0, k1, q0, q1, qfull, src, seg, 0). */
int fc_view_export(fc_view view, int32_t* q_gpos, int32_t* recv_gpos, int32_t* seg_doc,
                   int32_t* q_cu_docseg, int32_t* recv_cu, int32_t* pieces, int32_t* lim,
                   int32_t* fwd_local, int32_t* fwd_recv, int32_t* fwd_fused, int32_t* bwd);

/* The launch tables a view's kernels read, copied from exactly the blob
 * fc_view_bind uploads (for checks; any pointer may be NULL):
 *   fwd_local/fwd_recv/fwd_fused[n*8]  the forward items of fc_view_export,
 *                                      in launch order (largest first);
 *   bwd_launch[n_bwd_launch*8]         (k0, k1, q0, q1, qfull, src, seg, slot):
 *                                      the backward items, key tiles seen by
 *                                      many query tiles split into parts over
 *                                      consecutive query tiles, each part
 *                                      writing partial slot `slot` (-1: no
 *                                      split), largest first;
 *   bwd_reduce[n_bwd_reduce*8]         (src, k0, k1, first slot, slot count,
 *                                      0, 0, 0) per split key tile;
 *   bwd_qfirst[n_bwd_launch*(bn_bwd/32)] per launch item and 32-key wave
 *                                      (keys k0 + 32w ...): the first query
 *                                      row in [q0, q1) that sees key k0 + 32w
 *                                      (q1 if none). */
int fc_view_export_launch(fc_view view, int32_t* fwd_local, int32_t* fwd_recv,
                          int32_t* fwd_fused, int32_t* bwd_launch, int32_t* bwd_reduce,
                          int32_t* bwd_qfirst);

/* Upload the view's tables into `dev_meta` (device, >= meta_bytes, 256-byte
 * aligned) on `stream` and remember that buffer for later kernel calls. */
int fc_view_bind(fc_view view, void* dev_meta, size_t bytes, void* stream);

void fc_view_destroy(fc_view view);

/* Workspace bytes fc_attn_fwd (for `mode`), fc_attn_bwd and, alone,
 * fc_attn_bwd_dkdv / fc_attn_bwd_pass need (any pointer may be NULL). */
int fc_workspace_size(fc_view view, int32_t mode, size_t* fwd_bytes, size_t* bwd_bytes,
                      size_t* dkdv_bytes);

/* ---------------------------------------------------------------- kernels */

/* The simulated receive (Sec. 3.2; the "data copy" cost of Sec. 4.3): from
 * packed k,v [t_packed, Hkv, d] (bf16, device) gather the rank's own rows
 * into k_loc/v_loc and its receive set, compacted, into k_recv/v_recv.
 * Either part may be skipped by passing NULL for both of its outputs (the
 * two parts can then run on different streams, the receive overlapping the
 * local pass as in Sec. 3.2); at least one part must be given. */
int fc_kv_gather(fc_view view, const void* k_packed, const void* v_packed, int64_t t_packed,
                 void* k_loc, void* v_loc, void* k_recv, void* v_recv, void* stream);

/* Forward. Writes o (bf16 [T_q,Hq,d]), optionally o_f32 (fp32, same shape;
 * NULL to skip) and lse (fp32 [Hq,T_q]). FC_TWO_PASS runs the local and the
 * received pass (Sec. 3.2) and their log-sum-exp merge in one launch: each
 * query tile's received partial O goes to the workspace and is merged with
 * its local partial in the kernel; o and lse are exactly what
 * fc_attn_fwd_partials followed by fc_lse_merge write. FC_FUSED computes
 * both sources in one online softmax. ws: device, >= fc_workspace_size. */
int fc_attn_fwd(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                const void* k_recv, const void* v_recv, float scale, int32_t mode,
                void* o, float* o_f32, float* lse, void* ws, size_t ws_bytes, void* stream);

/* One partial pass over one key source (src 0 local, 1 received): fp32
 * o_part [T_q,Hq,d] and lse_part [Hq,T_q]; rows that see no key of the
 * source get O = 0 and LSE = -inf. */
int fc_attn_fwd_partial(fc_view view, int32_t src, const void* q, const void* k_src,
                        const void* v_src, float scale, float* o_part, float* lse_part,
                        void* stream);

/* Both partial passes in one launch (the two-pass forward's first step,
 * for a caller that merges later): local keys into o_loc/lse_loc,
 * received keys into o_recv/lse_recv, with the shapes and the empty-row
 * rule of fc_attn_fwd_partial; results are identical to the two separate
 * calls. k_recv/v_recv may be NULL when the view receives no keys (the
 * received partial is then O = 0, LSE = -inf everywhere). */
int fc_attn_fwd_partials(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                         const void* k_recv, const void* v_recv, float scale, float* o_loc,
                         float* lse_loc, float* o_recv, float* lse_recv, void* stream);

/* LSE merge of two partial results over disjoint key sets, t rows of h
 * heads of dim d (d % 4 == 0): lse_out = ln(e^lse_a + e^lse_b), o =
 * e^(lse_a-lse_out) o_a + e^(lse_b-lse_out) o_b; a -inf partial has weight
 * 0. o_a, o_b fp32 [t,h,d]; lse_* fp32 [h,t]; o_bf16 [t,h,d] bf16 and
 * o_f32 (nullable) fp32. Device pointers. */
int fc_lse_merge(const float* o_a, const float* lse_a, const float* o_b, const float* lse_b,
                 int32_t t, int32_t h, int32_t d, void* o_bf16, float* o_f32, float* lse_out,
                 void* stream);

/* Backward of the rank's attention (the gradient of the merged two-pass
 * result is the softmax gradient with the merged LSE, Sec. 2.3), given the
 * forward's output and final lse, and dout. The output is o (bf16) or, when
 * o_f32 (fp32 [T_q,Hq,d], 16-byte aligned, nullable) is given, o_f32 (o is
 * then not read and may be NULL): delta = rowsum(dout * O) from the fp32 O
 * is exact to fp32 rounding, from the bf16 O it carries O's rounding into
 * every dS of the row. Writes dq (fp32 [T_q,Hq,d],
 * 16-byte aligned), dk_loc/dv_loc (fp32 [T_q,Hkv,d]) and dk_recv/dv_recv
 * (fp32 [T_r,Hkv,d]); dK/dV are summed over the query heads of each KV
 * head. ws: device, >= bwd bytes of fc_workspace_size.
 * deterministic != 0: no atomics anywhere, results bitwise reproducible for
 * fixed inputs (a query-major pass recomputes S and dP for dQ).
 * deterministic == 0: the key-major pass also adds dQ with fp32 atomics (no
 * recompute); dK/dV are still reproducible, dQ's last bits vary from run to
 * run with the order of the additions. */
int fc_attn_bwd(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                const void* k_recv, const void* v_recv, const void* o, const float* o_f32,
                const float* lse, const void* dout, float scale, int32_t deterministic,
                float* dq, float* dk_loc, float* dv_loc, float* dk_recv, float* dv_recv,
                void* ws, size_t ws_bytes, void* stream);

/* The backward in its two steps (fc_attn_bwd runs both):
 * fc_bwd_preprocess writes delta[h, t] = sum_i dout[t,h,i] * O[t,h,i] (fp32
 * [Hq,T_q], device), O being o_f32 when non-null, else the bf16 o;
 * fc_attn_bwd_pass then computes dk_*, dv_* (key-major
 * kernel) and dq from lse and delta: by a query-major kernel when
 * deterministic != 0, else by atomics from the key-major kernel (dq is
 * zeroed first, on the stream). */
int fc_bwd_preprocess(fc_view view, const void* o, const float* o_f32, const void* dout,
                      float* delta, void* stream);
/* The two kernels of fc_attn_bwd_pass, callable alone: the key-major
 * dK/dV pass (writes dk_*, dv_*) and the query-major dQ pass (writes dq).
 * Key tiles seen by very many query tiles are split across workgroups that
 * write fp32 partials into ws, then summed in a fixed order, so dK/dV stay
 * reproducible. ws: device, >= the dkdv_bytes of fc_workspace_size; may be
 * NULL when that is 0 (no split key tile). */
int fc_attn_bwd_dkdv(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                     const void* k_recv, const void* v_recv, const float* lse, const float* delta,
                     const void* dout, float scale, float* dk_loc, float* dv_loc, float* dk_recv,
                     float* dv_recv, void* ws, size_t ws_bytes, void* stream);
int fc_attn_bwd_dq(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                   const void* k_recv, const void* v_recv, const float* lse, const float* delta,
                   const void* dout, float scale, float* dq, void* stream);
int fc_attn_bwd_pass(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                     const void* k_recv, const void* v_recv, const float* lse, const float* delta,
                     const void* dout, float scale, int32_t deterministic, float* dq,
                     float* dk_loc, float* dv_loc, float* dk_recv, float* dv_recv, void* ws,
                     size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fc_attn_bwd with the same arguments except the workspace, which comes
 * from a library-owned static device array of FC_NOALLOC_SCRATCH_BYTES per
 * GPU (held from module load until the process ends). Makes no device
 * allocation. FC_ERR_WORKSPACE, before any launch, when the view's
 * backward workspace (fc_workspace_size) exceeds that size; FC_ERR_INVALID_ARG
 * when `stream` belongs to another device than the current one. Results
 * are those of fc_attn_bwd. Every call on one GPU shares that GPU's array:
 * calls whose work overlaps on the same GPU (other streams, other threads)
 * race and must be serialised by the caller. */
#define FC_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)
int fc_attn_bwd_noalloc(fc_view view, const void* q, const void* k_loc, const void* v_loc,
                        const void* k_recv, const void* v_recv, const void* o,
                        const float* o_f32, const float* lse, const void* dout, float scale,
                        int32_t deterministic, float* dq,
                        float* dk_loc, float* dv_loc, float* dk_recv, float* dv_recv,
                        void* stream);

const char* fc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLASHCP_H */
