// Host representation of a rank view (the opaque fc_view).
#pragma once

#include <cstdint>
#include <vector>

#include "flashcp.h"

namespace fc {

struct View {
  int32_t hq = 0, hkv = 0, d = 0, heads_per_tile = 1;
  int32_t bm_fwd = 0, bn_fwd = 0, bm_bwd = 0, bn_bwd = 0;

  std::vector<int32_t> q_gpos, recv_gpos;   // global positions, local / receive order
  std::vector<int32_t> seg_doc, q_cu, recv_cu, seg_piece;
  std::vector<int32_t> pieces;              // 5 per piece: seg, q_start, q_end, g_start, n_P
  std::vector<int32_t> lim;                 // receive index end seen by each query
  int64_t pairs_loc = 0, pairs_recv = 0;

  // work lists, 8 int32 per item (layout documented in flashcp.h), in map
  // order, and their largest-first launch orders
  std::vector<int32_t> fwd_local, fwd_recv, fwd_fused, bwd;
  std::vector<int32_t> perm_fwd_local, perm_fwd_recv, perm_fwd_fused, perm_bwd;
  // backward launch list, largest first: the key-major items with long query
  // ranges split into parts that write partial dK/dV (last field: partial
  // slot, -1 for a direct write), and one reduce entry per split key tile
  // (src, k0, k1, first slot, slot count, 0, 0, 0)
  std::vector<int32_t> bwd_launch, bwd_reduce;
  int32_t n_bwd_slots = 0;
  // per launch item, per 32-key wave: first query row that sees its first key
  std::vector<int32_t> bwd_qfirst;

  // device blob: every table above that a kernel reads (the forward lists in
  // launch order), int32, sections aligned to 256 bytes; `off` holds section
  // offsets in int32 elements
  std::vector<int32_t> meta;
  struct {
    int64_t fwd_local, fwd_recv, fwd_fused;
    int64_t q_gpos, recv_gpos, lim;
    int64_t bwd_launch, bwd_reduce, bwd_qfirst;
  } off{};
  const int32_t* dev_meta = nullptr;        // set by fc_view_bind

  int32_t t_q() const { return int32_t(q_gpos.size()); }
  int32_t t_recv() const { return int32_t(recv_gpos.size()); }
  void build_tiles();
  void build_bwd_launch();
  void build_meta();
  int check_tables() const;
};

int build_view(const int32_t* cu, int32_t n_docs, const fc_shard* shards, int64_t n_shards,
               int32_t cp, int32_t rank, int32_t hq, int32_t hkv, int32_t d,
               const fc_tile_cfg* tiles, View& v);

}  // namespace fc
