// Rank view and tile maps (host side).
//
// A rank's queries are its shards' tokens in ascending global position
// ("local order"). Under the document mask (Sec. 2.1) a query sees the
// earlier tokens of its own document, so the KV a rank must hold is, per
// document, the prefix up to its last held token; the part it does not hold
// is its sharding-aware receive set (Sec. 3.2), stored compacted in
// ascending position.
//
// Two consequences shape the kernels' work lists:
//   * the rank's tokens of one document ("segment") are contiguous in local
//     order, and a query at local index i sees exactly the local keys
//     seg_start..i: the local pass is ordinary variable-length causal
//     attention over the segments;
//   * inside a maximal run of held positions ("piece") no received token
//     occurs, so every query of the piece sees the same first n_P received
//     tokens of its document: the received pass is mask-free per piece.
// Tiles that no query of a block can see are never listed.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <numeric>

#include "internal.hpp"
#include "view.hpp"

namespace fc {

namespace {

int32_t ceil_div(int64_t a, int64_t b) { return int32_t((a + b - 1) / b); }

// First tile start q0 + t*bm at or after `from`, or q1 if there is none.
int32_t first_tile_at_or_after(int32_t q0, int32_t q1, int32_t bm, int64_t from) {
  if (from <= q0) return q0;
  const int64_t t = q0 + int64_t(bm) * ceil_div(from - q0, bm);
  return t >= q1 ? q1 : int32_t(t);
}

std::vector<int32_t> lpt_order(const std::vector<int64_t>& cost) {
  std::vector<int32_t> idx(cost.size());
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(),
                   [&](int32_t a, int32_t b) { return cost[a] > cost[b]; });
  return idx;
}

}  // namespace

void View::build_tiles() {
  const int32_t S = int32_t(seg_doc.size());
  auto ldiag_of = [&](int32_t s0, int32_t t0) {
    // key tiles s0 + j*bn with s0 + j*bn + bn - 1 <= t0 are seen whole by
    // every row of a query tile starting at t0
    return s0 + ((t0 - s0 + 1) / bn_fwd) * bn_fwd;
  };
  auto push8 = [](std::vector<int32_t>& v, std::initializer_list<int32_t> x) {
    v.insert(v.end(), x.begin(), x.end());
  };
  // forward, local pass: query tiles per segment
  for (int32_t s = 0; s < S; ++s) {
    const int32_t s0 = q_cu[s], s1 = q_cu[s + 1];
    for (int32_t t0 = s0; t0 < s1; t0 += bm_fwd) {
      const int32_t t1 = std::min(t0 + bm_fwd, s1);
      push8(fwd_local, {t0, t1, 0, 0, s0, t1, ldiag_of(s0, t0), s});
    }
  }
  // forward, received and fused passes: query tiles per piece
  for (size_t p = 0; p < pieces.size() / 5; ++p) {
    const int32_t s = pieces[5 * p], qs = pieces[5 * p + 1], qe = pieces[5 * p + 2];
    const int32_t np = pieces[5 * p + 4];
    const int32_t r0 = recv_cu[s], s0 = q_cu[s];
    for (int32_t t0 = qs; t0 < qe; t0 += bm_fwd) {
      const int32_t t1 = std::min(t0 + bm_fwd, qe);
      push8(fwd_recv, {t0, t1, r0, r0 + np, 0, 0, 0, s});
      push8(fwd_fused, {t0, t1, r0, r0 + np, s0, t1, ldiag_of(s0, t0), s});
    }
  }
  // backward, key-major: local key tiles then received key tiles
  for (int32_t s = 0; s < S; ++s) {
    const int32_t s0 = q_cu[s], s1 = q_cu[s + 1];
    for (int32_t k0 = s0; k0 < s1; k0 += bn_bwd) {
      const int32_t k1 = std::min(k0 + bn_bwd, s1);
      // rows i >= k0 see key k0; rows i >= k1-1 see the whole tile
      push8(bwd, {k0, k1, k0, s1, first_tile_at_or_after(k0, s1, bm_bwd, k1 - 1), 0, s, 0});
    }
  }
  for (int32_t s = 0; s < S; ++s) {
    const int32_t s1 = q_cu[s + 1];
    const int32_t rl = recv_cu[s], rh = recv_cu[s + 1];
    // the segment's pieces in local order have non-decreasing n_P
    const int32_t pa = seg_piece[s], pb = seg_piece[s + 1];
    for (int32_t k0 = rl; k0 < rh; k0 += bn_bwd) {
      const int32_t k1 = std::min(k0 + bn_bwd, rh);
      int32_t q0 = s1, qa = s1;
      for (int32_t p = pa; p < pb; ++p) {
        const int32_t lim_p = rl + pieces[5 * p + 4];
        if (q0 == s1 && lim_p > k0) q0 = pieces[5 * p + 1];
        if (lim_p >= k1) {
          qa = pieces[5 * p + 1];
          break;
        }
      }
      push8(bwd, {k0, k1, q0, s1, first_tile_at_or_after(q0, s1, bm_bwd, qa), 1, s, 0});
    }
  }
  // largest-first launch orders (the lists themselves stay in map order)
  auto fwd_cost = [&](const std::vector<int32_t>& items) {
    std::vector<int64_t> c(items.size() / 8);
    for (size_t i = 0; i < c.size(); ++i) {
      const int32_t* it = &items[8 * i];
      c[i] = ceil_div(it[3] - it[2], bn_fwd) + ceil_div(it[5] - it[4], bn_fwd);
    }
    return c;
  };
  perm_fwd_local = lpt_order(fwd_cost(fwd_local));
  perm_fwd_recv = lpt_order(fwd_cost(fwd_recv));
  perm_fwd_fused = lpt_order(fwd_cost(fwd_fused));
  std::vector<int64_t> bc(bwd.size() / 8);
  for (size_t i = 0; i < bc.size(); ++i) bc[i] = ceil_div(bwd[8 * i + 3] - bwd[8 * i + 2], bm_bwd);
  perm_bwd = lpt_order(bc);
  build_bwd_launch();
}

// Split key tiles whose query range is much longer than a fair share of the
// backward's work: with about 512 workgroups resident at a time (256 CUs, two
// per CU), an item longer than total/512 iterations would finish after
// everything else. Its query tiles are cut into equal parts; each part
// writes fp32 partial dK/dV to its own slot and a reduce pass sums the parts
// in slot order (deterministic).
void View::build_bwd_launch() {
  constexpr int64_t kSlotsResident = 512;
  const int64_t G = hq / hkv;
  const size_t n = bwd.size() / 8;
  int64_t total = 0;
  for (size_t i = 0; i < n; ++i) total += ceil_div(bwd[8 * i + 3] - bwd[8 * i + 2], bm_bwd) * G;
  const int64_t cap = std::max<int64_t>(16, (total * hkv + kSlotsResident - 1) / kSlotsResident);
  bwd_launch.clear();
  bwd_reduce.clear();
  n_bwd_slots = 0;
  std::vector<int64_t> cost;
  for (size_t i = 0; i < n; ++i) {
    const int32_t* it = &bwd[8 * i];
    const int32_t ntile = ceil_div(it[3] - it[2], bm_bwd);
    const int32_t parts = int32_t(std::max<int64_t>(1, (int64_t(ntile) * G + cap - 1) / cap));
    if (parts == 1) {
      bwd_launch.insert(bwd_launch.end(), {it[0], it[1], it[2], it[3], it[4], it[5], it[6], -1});
      cost.push_back(int64_t(ntile) * G);
      continue;
    }
    const int32_t per = ceil_div(ntile, parts);
    bwd_reduce.insert(bwd_reduce.end(), {it[5], it[0], it[1], n_bwd_slots, 0, 0, 0, 0});
    int32_t made = 0;
    for (int32_t t = 0; t < ntile; t += per) {
      const int32_t a = it[2] + t * bm_bwd;
      const int32_t b = std::min(it[3], it[2] + (t + per) * bm_bwd);
      bwd_launch.insert(bwd_launch.end(), {it[0], it[1], a, b, it[4], it[5], it[6], n_bwd_slots});
      cost.push_back(int64_t(std::min(per, ntile - t)) * G);
      ++n_bwd_slots;
      ++made;
    }
    bwd_reduce[bwd_reduce.size() - 4] = made;
  }
  // the launch list itself goes in largest-first order: workgroup b takes
  // item b / hkv, with no order table to read first
  {
    const std::vector<int32_t> order = lpt_order(cost);
    std::vector<int32_t> sorted;
    sorted.reserve(bwd_launch.size());
    for (int32_t i : order) sorted.insert(sorted.end(), &bwd_launch[8 * i], &bwd_launch[8 * i + 8]);
    bwd_launch.swap(sorted);
  }
  // per launch item and wave (32 keys from k0 + 32w): the first query row
  // that sees the wave's first key -- for local keys the key's own index,
  // for received keys the first row whose receive limit exceeds it (limits
  // do not decrease along a segment)
  bwd_qfirst.clear();
  for (size_t i = 0; i < bwd_launch.size() / 8; ++i) {
    const int32_t* it = &bwd_launch[8 * i];
    for (int32_t w = 0; w < bn_bwd / 32; ++w) {
      const int32_t kw = it[0] + 32 * w;
      int32_t qf = kw;
      if (it[5]) {
        const int32_t* b = lim.data() + it[2];
        const int32_t* e = lim.data() + it[3];
        qf = it[2] + int32_t(std::upper_bound(b, e, kw) - b);
      }
      bwd_qfirst.push_back(qf);
    }
  }
}

// Every index the kernels will take from the tables, checked against the
// extents they index (t_q, t_recv, the slot count) before anything is
// uploaded: a table out of range is a library bug, reported as such rather
// than handed to a kernel.
int View::check_tables() const {
  const int32_t tq = t_q(), tr = t_recv();
  auto bad = [](const char* what, size_t i) {
    return fail(FC_ERR_INTERNAL, std::string("internal: ") + what + " entry " + std::to_string(i) +
                                     " out of range");
  };
  for (const auto* list : {&fwd_local, &fwd_recv, &fwd_fused}) {
    for (size_t i = 0; i < list->size() / 8; ++i) {
      const int32_t* it = &(*list)[8 * i];
      if (!(0 <= it[0] && it[0] < it[1] && it[1] <= tq && it[1] - it[0] <= bm_fwd))
        return bad("forward item (queries)", i);
      if (!(0 <= it[2] && it[2] <= it[3] && it[3] <= tr)) return bad("forward item (received)", i);
      if (!(0 <= it[4] && it[4] <= it[5] && it[5] <= tq)) return bad("forward item (local)", i);
    }
  }
  for (size_t i = 0; i < bwd_launch.size() / 8; ++i) {
    const int32_t* it = &bwd_launch[8 * i];
    const int32_t hi = it[5] ? tr : tq;
    if (!((it[5] == 0 || it[5] == 1) && 0 <= it[0] && it[0] < it[1] && it[1] <= hi &&
          it[1] - it[0] <= bn_bwd && 0 <= it[2] && it[2] < it[3] && it[3] <= tq &&
          -1 <= it[7] && it[7] < n_bwd_slots))
      return bad("backward launch item", i);
  }
  for (size_t i = 0; i < bwd_reduce.size() / 8; ++i) {
    const int32_t* e = &bwd_reduce[8 * i];
    const int32_t hi = e[0] ? tr : tq;
    if (!((e[0] == 0 || e[0] == 1) && 0 <= e[1] && e[1] < e[2] && e[2] <= hi && 0 <= e[3] &&
          0 < e[4] && e[3] + e[4] <= n_bwd_slots))
      return bad("backward reduce entry", i);
  }
  if (bwd_qfirst.size() != bwd_launch.size() / 8 * size_t(bn_bwd / 32)) return bad("qfirst", 0);
  for (size_t i = 0; i < lim.size(); ++i)
    if (!(0 <= lim[i] && lim[i] <= tr)) return bad("receive limit", i);
  return FC_OK;
}

void View::build_meta() {
  meta.clear();
  auto put = [&](const std::vector<int32_t>& v) {
    const int64_t off = int64_t(meta.size());
    meta.insert(meta.end(), v.begin(), v.end());
    meta.resize((meta.size() + 63) / 64 * 64, 0);  // 256-byte aligned sections
    return off;
  };
  // forward item lists in their launch (largest-first) order: workgroup b
  // reads its item directly, with no order table to read first
  auto in_order = [](const std::vector<int32_t>& items, const std::vector<int32_t>& order) {
    std::vector<int32_t> r;
    r.reserve(items.size());
    for (int32_t i : order) r.insert(r.end(), &items[8 * i], &items[8 * i + 8]);
    return r;
  };
  off.fwd_local = put(in_order(fwd_local, perm_fwd_local));
  off.fwd_recv = put(in_order(fwd_recv, perm_fwd_recv));
  off.fwd_fused = put(in_order(fwd_fused, perm_fwd_fused));
  off.q_gpos = put(q_gpos);
  off.recv_gpos = put(recv_gpos);
  off.lim = put(lim);
  off.bwd_launch = put(bwd_launch);
  off.bwd_reduce = put(bwd_reduce);
  off.bwd_qfirst = put(bwd_qfirst);
  if (meta.empty()) meta.resize(64, 0);
}

int build_view(const int32_t* cu, int32_t n_docs, const fc_shard* shards, int64_t n_shards,
               int32_t cp, int32_t rank, int32_t hq, int32_t hkv, int32_t d,
               const fc_tile_cfg* tiles, View& v) {
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  if (int rc = validate_plan(lens, cp, shards, n_shards, false)) return rc;
  if (rank < 0 || rank >= cp) return fail(FC_ERR_INVALID_ARG, "rank out of range");
  if (d != 64 && d != 128) return fail(FC_ERR_UNSUPPORTED, "head dim must be 64 or 128");
  if (hq < 1 || hkv < 1 || hq % hkv)
    return fail(FC_ERR_INVALID_ARG, "need hq, hkv >= 1 and hq % hkv == 0");
  const int32_t G = hq / hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(FC_ERR_UNSUPPORTED, "hq/hkv must be 1, 2, 4 or 8");
  if (int64_t(cu[n_docs]) > (int64_t(1) << 30))
    return fail(FC_ERR_UNSUPPORTED, "context longer than 2^30 tokens");
  v.hq = hq;
  v.hkv = hkv;
  v.d = d;
  // tile shapes: the forward / dQ query tile is 128 / (heads per workgroup)
  // rows, each of the 4 waves taking a quarter of them for every head; the
  // other shapes are compiled
  const fc_tile_cfg t = tiles ? *tiles : fc_tile_cfg{0, 0, 0, 0};
  if (t.bm_fwd == 0) {
    v.heads_per_tile = std::min(G, 4);
  } else {
    if (t.bm_fwd != 32 && t.bm_fwd != 64 && t.bm_fwd != 128)
      return fail(FC_ERR_UNSUPPORTED, "bm_fwd must be 32, 64 or 128");
    v.heads_per_tile = 128 / t.bm_fwd;
    if (G % v.heads_per_tile)
      return fail(FC_ERR_UNSUPPORTED, "bm_fwd " + std::to_string(t.bm_fwd) + " puts " +
                                          std::to_string(v.heads_per_tile) +
                                          " query heads in a workgroup; hq/hkv is " +
                                          std::to_string(G));
  }
  if ((t.bn_fwd && t.bn_fwd != 64) || (t.bm_bwd && t.bm_bwd != 32) || (t.bn_bwd && t.bn_bwd != 128))
    return fail(FC_ERR_UNSUPPORTED, "compiled tile shapes: bn_fwd 64, bm_bwd 32, bn_bwd 128");
  v.bm_fwd = 32 * (4 / v.heads_per_tile);
  v.bn_fwd = 64;
  v.bm_bwd = 32;
  v.bn_bwd = 128;

  std::vector<fc_shard> mine;
  for (int64_t i = 0; i < n_shards; ++i)
    if (shards[i].rank == rank) mine.push_back(shards[i]);
  std::sort(mine.begin(), mine.end(), [](const fc_shard& a, const fc_shard& b) {
    return a.doc != b.doc ? a.doc < b.doc : a.offset < b.offset;
  });
  v.q_cu.assign(1, 0);
  v.recv_cu.assign(1, 0);
  v.seg_piece.assign(1, 0);
  for (size_t i = 0; i < mine.size();) {
    const int32_t doc = mine[i].doc, c0 = cu[doc];
    const int32_t seg = int32_t(v.seg_doc.size());
    v.seg_doc.push_back(doc);
    int32_t held_end = 0;  // offset just past the previous piece
    int32_t gap_total = 0; // received tokens of this document so far
    while (i < mine.size() && mine[i].doc == doc) {
      // one piece: a maximal run of consecutive held offsets
      const int32_t a = mine[i].offset;
      int32_t b = a + mine[i].len;
      ++i;
      while (i < mine.size() && mine[i].doc == doc && mine[i].offset == b) b += mine[i++].len;
      for (int32_t u = held_end; u < a; ++u) v.recv_gpos.push_back(c0 + u);
      gap_total += a - held_end;
      const int32_t qs = int32_t(v.q_gpos.size());
      for (int32_t u = a; u < b; ++u) v.q_gpos.push_back(c0 + u);
      const int32_t qe = int32_t(v.q_gpos.size());
      v.pieces.insert(v.pieces.end(), {seg, qs, qe, c0 + a, gap_total});
      v.lim.insert(v.lim.end(), size_t(qe - qs), v.recv_cu[seg] + gap_total);
      v.pairs_recv += int64_t(qe - qs) * gap_total;
      held_end = b;
    }
    v.q_cu.push_back(int32_t(v.q_gpos.size()));
    v.recv_cu.push_back(int32_t(v.recv_gpos.size()));
    v.seg_piece.push_back(int32_t(v.pieces.size() / 5));
    const int64_t seg_len = v.q_cu[seg + 1] - v.q_cu[seg];
    v.pairs_loc += seg_len * (seg_len + 1) / 2;
  }
  v.build_tiles();
  if (int rc = v.check_tables()) return rc;
  v.build_meta();
  return FC_OK;
}

}  // namespace fc

using namespace fc;

extern "C" {

int fc_view_create(const int32_t* cu, int32_t n_docs, const fc_shard* shards, int64_t n_shards,
                   int32_t cp, int32_t rank, int32_t hq, int32_t hkv, int32_t d,
                   const fc_tile_cfg* tiles, fc_view* out) {
  clear_error();
  if (!out) return fail(FC_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  View* v = new View();
  if (int rc = build_view(cu, n_docs, shards, n_shards, cp, rank, hq, hkv, d, tiles, *v)) {
    delete v;
    return rc;
  }
  *out = reinterpret_cast<fc_view>(v);
  return FC_OK;
}

int fc_view_get_info(fc_view view, fc_view_info* out) {
  clear_error();
  if (!view || !out) return fail(FC_ERR_INVALID_ARG, "null argument");
  const View& v = *reinterpret_cast<View*>(view);
  *out = fc_view_info{};
  out->t_q = int32_t(v.q_gpos.size());
  out->t_recv = int32_t(v.recv_gpos.size());
  out->n_seg = int32_t(v.seg_doc.size());
  out->n_pieces = int32_t(v.pieces.size() / 5);
  out->hq = v.hq;
  out->hkv = v.hkv;
  out->d = v.d;
  out->bm_fwd = v.bm_fwd;
  out->bn_fwd = v.bn_fwd;
  out->bm_bwd = v.bm_bwd;
  out->bn_bwd = v.bn_bwd;
  out->n_fwd_local = int64_t(v.fwd_local.size() / 8);
  out->n_fwd_recv = int64_t(v.fwd_recv.size() / 8);
  out->n_fwd_fused = int64_t(v.fwd_fused.size() / 8);
  out->n_bwd = int64_t(v.bwd.size() / 8);
  out->pairs_loc = v.pairs_loc;
  out->pairs_recv = v.pairs_recv;
  out->meta_bytes = int64_t(v.meta.size() * sizeof(int32_t));
  out->n_bwd_launch = int64_t(v.bwd_launch.size() / 8);
  out->n_bwd_reduce = int64_t(v.bwd_reduce.size() / 8);
  out->n_bwd_slots = v.n_bwd_slots;
  return FC_OK;
}

int fc_view_export(fc_view view, int32_t* q_gpos, int32_t* recv_gpos, int32_t* seg_doc,
                   int32_t* q_cu_docseg, int32_t* recv_cu, int32_t* pieces, int32_t* lim,
                   int32_t* fwd_local, int32_t* fwd_recv, int32_t* fwd_fused, int32_t* bwd) {
  clear_error();
  if (!view) return fail(FC_ERR_INVALID_ARG, "view is null");
  const View& v = *reinterpret_cast<View*>(view);
  auto cp = [](int32_t* dst, const std::vector<int32_t>& src) {
    if (dst) std::copy(src.begin(), src.end(), dst);
  };
  cp(q_gpos, v.q_gpos);
  cp(recv_gpos, v.recv_gpos);
  cp(seg_doc, v.seg_doc);
  cp(q_cu_docseg, v.q_cu);
  cp(recv_cu, v.recv_cu);
  cp(pieces, v.pieces);
  cp(lim, v.lim);
  cp(fwd_local, v.fwd_local);
  cp(fwd_recv, v.fwd_recv);
  cp(fwd_fused, v.fwd_fused);
  cp(bwd, v.bwd);
  return FC_OK;
}

int fc_view_export_launch(fc_view view, int32_t* fwd_local, int32_t* fwd_recv,
                          int32_t* fwd_fused, int32_t* bwd_launch, int32_t* bwd_reduce,
                          int32_t* bwd_qfirst) {
  clear_error();
  if (!view) return fail(FC_ERR_INVALID_ARG, "view is null");
  const View& v = *reinterpret_cast<View*>(view);
  auto cp = [&](int32_t* dst, int64_t off, size_t n) {
    if (dst) std::copy(v.meta.begin() + off, v.meta.begin() + off + int64_t(n), dst);
  };
  cp(fwd_local, v.off.fwd_local, v.fwd_local.size());
  cp(fwd_recv, v.off.fwd_recv, v.fwd_recv.size());
  cp(fwd_fused, v.off.fwd_fused, v.fwd_fused.size());
  cp(bwd_launch, v.off.bwd_launch, v.bwd_launch.size());
  cp(bwd_reduce, v.off.bwd_reduce, v.bwd_reduce.size());
  cp(bwd_qfirst, v.off.bwd_qfirst, v.bwd_qfirst.size());
  return FC_OK;
}

int fc_view_bind(fc_view view, void* dev_meta, size_t bytes, void* stream) {
  clear_error();
  if (!view || !dev_meta) return fail(FC_ERR_INVALID_ARG, "null argument");
  View& v = *reinterpret_cast<View*>(view);
  const size_t need = v.meta.size() * sizeof(int32_t);
  if (bytes < need)
    return fail(FC_ERR_WORKSPACE, "metadata buffer of " + std::to_string(bytes) +
                                      " bytes, need " + std::to_string(need));
  if (reinterpret_cast<uintptr_t>(dev_meta) % 256)
    return fail(FC_ERR_INVALID_ARG, "metadata buffer must be 256-byte aligned");
  hipError_t e = hipMemcpyAsync(dev_meta, v.meta.data(), need, hipMemcpyHostToDevice,
                                reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FC_ERR_HIP, std::string("hipMemcpyAsync: ") + hipGetErrorString(e));
  v.dev_meta = reinterpret_cast<const int32_t*>(dev_meta);
  return FC_OK;
}

void fc_view_destroy(fc_view view) { delete reinterpret_cast<View*>(view); }

}  // extern "C"
