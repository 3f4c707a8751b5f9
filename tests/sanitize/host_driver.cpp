// Host driver of the library's C ABI for the sanitizer build: the host
// sources (planners, rank views and tile maps, the device entry points'
// validation and parameter building) compiled with g++ under
// AddressSanitizer and UndefinedBehaviorSanitizer, no HIP runtime linked.
//
// hipMemcpyAsync and hipGetErrorString are stubs (the "device" blob a view is
// bound to is host memory here), and so are the kernel launchers: they launch
// nothing, but check that every table pointer they are handed lies inside the
// bound blob together with the whole extent the kernel would read, and that
// the sizes they carry agree with the view. Every failure aborts with a
// message; the sanitizers abort on any memory or undefined-behaviour error.
//
// Usage: host_driver [workload-file]; each line of the file holds
// "name cp plan rank_rule n_docs hq hkv d cu_0 ... cu_n" (plan: per_doc,
// whole_lpt or hybrid; rank_rule: a rank number, "last" or "heaviest").
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <random>
#include <sstream>
#include <string>
#include <vector>

#include "../../paper_2606_08476_amd/csrc/kernels/launch.hpp"
#include "flashcp.h"

#define CHECK(c)                                                               \
  do {                                                                         \
    if (!(c)) {                                                                \
      std::fprintf(stderr, "check failed at %s:%d: %s (%s)\n", __FILE__,      \
                   __LINE__, #c, fc_last_error());                             \
      std::abort();                                                            \
    }                                                                          \
  } while (0)

// ------------------------------------------------------------ stubs

namespace {
const char* g_blob = nullptr;   // the bound "device" blob
size_t g_blob_bytes = 0;
int64_t g_launches = 0;

void in_blob(const void* p, int64_t n_int32, const char* what) {
  if (n_int32 == 0) return;
  const char* c = static_cast<const char*>(p);
  if (!(c >= g_blob && c + 4 * n_int32 <= g_blob + g_blob_bytes)) {
    std::fprintf(stderr, "%s: %lld int32 at %p outside the bound blob\n", what,
                 (long long)n_int32, p);
    std::abort();
  }
}
}  // namespace

extern "C" hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind,
                                     hipStream_t) {
  std::memcpy(dst, src, bytes);
  return hipSuccess;
}
extern "C" const char* hipGetErrorString(hipError_t) { return "stub"; }

namespace fck {
hipError_t launch_fwd(const FwdParams& p, int d, int hpt, bool, hipStream_t) {
  CHECK((d == 64 || d == 128) && (hpt == 1 || hpt == 2 || hpt == 4) && p.n_items >= 0);
  CHECK(p.group % hpt == 0 && p.head_chunks * hpt == p.group && p.hq == p.group * p.hkv);
  in_blob(p.items, 8 * int64_t(p.n_items), "forward items");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_bwd_dq(const DqParams& p, int d, int hpt, hipStream_t) {
  CHECK((d == 64 || d == 128) && (hpt == 1 || hpt == 2 || hpt == 4));
  in_blob(p.items, 8 * int64_t(p.n_items), "dQ items");
  ++g_launches;
  return hipSuccess;
}
static void check_bwd(const BwdParams& p) {
  in_blob(p.items, 8 * int64_t(p.n_items), "backward launch items");
  in_blob(p.qfirst, 4 * int64_t(p.n_items), "backward qfirst");
  in_blob(p.lim, p.t_q, "receive limits");
  CHECK(p.dk_loc && p.dv_loc && p.lse && p.delta);
}
hipError_t launch_bwd(const BwdParams& p, int, hipStream_t) {
  check_bwd(p);
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_bwd_atomic(const BwdParams& p, int, hipStream_t) {
  check_bwd(p);
  CHECK(p.dq);
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_bwd_grid(const BwdParams& bp, const DqParams& dp, int, int, hipStream_t) {
  check_bwd(bp);
  in_blob(dp.items, 8 * int64_t(dp.n_items), "dQ items");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_bwd_reduce(const int32_t* e, int32_t n, const float*, const float*, int32_t,
                             int32_t, float*, float*, float*, float*, hipStream_t) {
  in_blob(e, 8 * int64_t(n), "reduce entries");
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_bwd_preprocess(const uint16_t* o, const float* of, const uint16_t* dout,
                                 float* delta, int32_t t, int32_t h, int32_t d, float*,
                                 hipStream_t) {
  CHECK((o || of) && dout && delta && t >= 0 && h > 0 && (d == 64 || d == 128));
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_fill_zero(float* x, int64_t n, hipStream_t) {
  CHECK(x && n >= 0 && n % 4 == 0);
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_lse_merge(const float*, const float*, const float*, const float*, int32_t t,
                            int32_t h, int32_t d, uint16_t*, float*, float*, hipStream_t) {
  CHECK(t >= 0 && h >= 0 && (d == 64 || d == 128));
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_kv_gather(const uint16_t*, const uint16_t*, const int32_t* qg,
                            const int32_t* rg, int32_t tq, int32_t tr, int64_t r0, int64_t r1,
                            int32_t row_elems, uint16_t*, uint16_t*, uint16_t*, uint16_t*,
                            hipStream_t) {
  CHECK(0 <= r0 && r0 <= r1 && r1 <= int64_t(tq) + tr && row_elems > 0);
  in_blob(qg, tq, "local positions");
  in_blob(rg, tr, "received positions");
  ++g_launches;
  return hipSuccess;
}
}  // namespace fck

// ------------------------------------------------------------ driver

namespace {

// a 256-byte aligned "device" pointer for data arguments (never read)
alignas(256) char g_dummy[256];
void* const D = g_dummy;
float* const Df = reinterpret_cast<float*>(g_dummy);

std::vector<fc_shard> plan_of(const std::vector<int32_t>& cu, int cp, const std::string& kind) {
  const int32_t n = int32_t(cu.size()) - 1;
  int64_t need = 0;
  int rc;
  // capacity probe first: FC_ERR_CAPACITY with the needed count
  std::vector<uint8_t> isp(std::max<int32_t>(n, 1));
  if (kind == "per_doc") rc = fc_plan_per_doc(cu.data(), n, cp, nullptr, 0, &need);
  else if (kind == "per_seq") rc = fc_plan_per_seq(cu.data(), n, cp, nullptr, 0, &need);
  else if (kind == "whole_lpt") rc = fc_plan_whole_lpt(cu.data(), n, cp, nullptr, 0, &need);
  else rc = fc_plan_hybrid(cu.data(), n, cp, 1.05, nullptr, 0, &need, isp.data());
  CHECK(rc == FC_OK || rc == FC_ERR_CAPACITY);
  std::vector<fc_shard> out(size_t(std::max<int64_t>(need, 1)));
  int64_t got = 0;
  if (kind == "per_doc") rc = fc_plan_per_doc(cu.data(), n, cp, out.data(), need, &got);
  else if (kind == "per_seq") rc = fc_plan_per_seq(cu.data(), n, cp, out.data(), need, &got);
  else if (kind == "whole_lpt") rc = fc_plan_whole_lpt(cu.data(), n, cp, out.data(), need, &got);
  else rc = fc_plan_hybrid(cu.data(), n, cp, 1.05, out.data(), need, &got, isp.data());
  CHECK(rc == FC_OK && got == need);
  out.resize(size_t(got));
  CHECK(fc_plan_validate(cu.data(), n, cp, out.data(), got, 0) == FC_OK);
  return out;
}

// Build a view, export everything at exactly the sizes fc_view_get_info
// reports, bind it to host "device" memory and call every device entry
// point (valid calls and host-rejected ones).
void exercise_view(const std::vector<int32_t>& cu, const std::vector<fc_shard>& plan, int cp,
                   int rank, int hq, int hkv, int d, const fc_tile_cfg* tiles) {
  const int32_t n = int32_t(cu.size()) - 1;
  fc_view v = nullptr;
  const int rc = fc_view_create(cu.data(), n, plan.data(), int64_t(plan.size()), cp, rank, hq,
                                hkv, d, tiles, &v);
  if (rc == FC_ERR_UNSUPPORTED) return;  // a tile shape the group does not allow
  CHECK(rc == FC_OK && v);
  fc_view_info i{};
  CHECK(fc_view_get_info(v, &i) == FC_OK);
  auto buf = [](int64_t k) { return std::vector<int32_t>(size_t(std::max<int64_t>(k, 1))); };
  auto qg = buf(i.t_q), rg = buf(i.t_recv), sd = buf(i.n_seg), qcu = buf(i.n_seg + 1),
       rcu = buf(i.n_seg + 1), pc = buf(5 * int64_t(i.n_pieces)), lim = buf(i.t_q),
       fl = buf(8 * i.n_fwd_local), fr = buf(8 * i.n_fwd_recv), ff = buf(8 * i.n_fwd_fused),
       bw = buf(8 * i.n_bwd);
  CHECK(fc_view_export(v, qg.data(), rg.data(), sd.data(), qcu.data(), rcu.data(), pc.data(),
                       lim.data(), fl.data(), fr.data(), ff.data(), bw.data()) == FC_OK);
  auto ll = buf(8 * i.n_fwd_local), lr = buf(8 * i.n_fwd_recv), lf = buf(8 * i.n_fwd_fused),
       bl = buf(8 * i.n_bwd_launch), br = buf(8 * i.n_bwd_reduce),
       qf = buf(int64_t(i.bn_bwd / 32) * i.n_bwd_launch);
  CHECK(fc_view_export_launch(v, ll.data(), lr.data(), lf.data(), bl.data(), br.data(),
                              qf.data()) == FC_OK);
  CHECK(qcu[size_t(i.n_seg)] == i.t_q && rcu[size_t(i.n_seg)] == i.t_recv);

  size_t fws = 0, bws = 0, dws = 0;
  CHECK(fc_workspace_size(v, FC_TWO_PASS, &fws, &bws, &dws) == FC_OK);
  // every device call on an unbound view is refused before any launch
  const int64_t before = g_launches;
  CHECK(fc_kv_gather(v, D, D, cu.back(), D, D, D, D, nullptr) == FC_ERR_WORKSPACE);
  CHECK(fc_attn_bwd(v, D, D, D, D, D, D, nullptr, Df, D, 0.f, 1, Df, Df, Df, Df, Df, D, bws,
                    nullptr) == FC_ERR_WORKSPACE || i.t_q == 0);
  CHECK(g_launches == before);

  // bind to host memory standing in for the device
  std::vector<char> blob(size_t(i.meta_bytes) + 256);
  char* base = blob.data() + ((256 - reinterpret_cast<uintptr_t>(blob.data()) % 256) % 256);
  CHECK(fc_view_bind(v, base, size_t(i.meta_bytes), nullptr) == FC_OK);
  g_blob = base;
  g_blob_bytes = size_t(i.meta_bytes);

  CHECK(fc_kv_gather(v, D, D, cu.back(), D, D, D, D, nullptr) == FC_OK);
  CHECK(fc_kv_gather(v, D, D, cu.back(), nullptr, nullptr, D, D, nullptr) == FC_OK);
  CHECK(fc_kv_gather(v, D, D, cu.back(), D, D, nullptr, nullptr, nullptr) == FC_OK);
  if (i.t_q + i.t_recv > 0)
    CHECK(fc_kv_gather(v, D, D, 0, D, D, D, D, nullptr) == FC_ERR_SHAPE);
  for (int32_t mode : {FC_TWO_PASS, FC_FUSED}) {
    size_t need = 0;
    CHECK(fc_workspace_size(v, mode, &need, nullptr, nullptr) == FC_OK);
    CHECK(fc_attn_fwd(v, D, D, D, D, D, 0.f, mode, D, Df, Df, D, need, nullptr) == FC_OK);
    if (need && i.t_q)
      CHECK(fc_attn_fwd(v, D, D, D, D, D, 0.f, mode, D, Df, Df, D, need - 1, nullptr) ==
            FC_ERR_WORKSPACE);
  }
  CHECK(fc_attn_fwd(v, D, D, D, D, D, 0.f, 7, D, Df, Df, D, fws, nullptr) == FC_ERR_INVALID_ARG);
  CHECK(fc_attn_fwd_partial(v, 0, D, D, D, 0.f, Df, Df, nullptr) == FC_OK);
  CHECK(fc_attn_fwd_partial(v, 1, D, D, D, 0.f, Df, Df, nullptr) == FC_OK);
  CHECK(fc_attn_fwd_partials(v, D, D, D, D, D, 0.f, Df, Df, Df, Df, nullptr) == FC_OK);
  CHECK(fc_bwd_preprocess(v, D, nullptr, D, Df, nullptr) == FC_OK);
  CHECK(fc_bwd_preprocess(v, nullptr, Df, D, Df, nullptr) == FC_OK);
  for (int32_t det : {0, 1}) {
    CHECK(fc_attn_bwd(v, D, D, D, D, D, D, Df, Df, D, 0.f, det, Df, Df, Df, Df, Df, D, bws,
                      nullptr) == FC_OK);
    CHECK(fc_attn_bwd_pass(v, D, D, D, D, D, Df, Df, D, 0.f, det, Df, Df, Df, Df, Df, D, dws,
                           nullptr) == FC_OK);
    if (i.t_q)
      CHECK(fc_attn_bwd(v, D, D, D, D, D, D, Df, Df, D, 0.f, det, Df, Df, Df, Df, Df, D, bws - 1,
                        nullptr) == FC_ERR_WORKSPACE);
  }
  CHECK(fc_attn_bwd_dkdv(v, D, D, D, D, D, Df, Df, D, 0.f, Df, Df, Df, Df, D, dws, nullptr) ==
        FC_OK);
  CHECK(fc_attn_bwd_dq(v, D, D, D, D, D, Df, Df, D, 0.f, Df, nullptr) == FC_OK);
  if (i.t_q) {
    CHECK(fc_attn_bwd(v, nullptr, D, D, D, D, D, Df, Df, D, 0.f, 1, Df, Df, Df, Df, Df, D, bws,
                      nullptr) == FC_ERR_INVALID_ARG);
    CHECK(fc_attn_fwd(v, nullptr, D, D, D, D, 0.f, FC_TWO_PASS, D, Df, Df, D, fws, nullptr) ==
          FC_ERR_INVALID_ARG);
  }
  CHECK(fc_lse_merge(Df, Df, Df, Df, 5, 3, 128, D, Df, Df, nullptr) == FC_OK);
  CHECK(fc_lse_merge(Df, Df, Df, Df, 5, 3, 96, D, Df, Df, nullptr) == FC_ERR_UNSUPPORTED);
  g_blob = nullptr;
  g_blob_bytes = 0;
  fc_view_destroy(v);
}

void exercise_plan_stats(const std::vector<int32_t>& cu, const std::vector<fc_shard>& plan,
                         int cp) {
  const int32_t n = int32_t(cu.size()) - 1;
  std::vector<int64_t> work(static_cast<size_t>(cp));
  std::vector<int32_t> tok(static_cast<size_t>(cp)), rcv(static_cast<size_t>(cp));
  int64_t e4 = 0, e5 = 0;
  double imb = 0;
  CHECK(fc_plan_stats(cu.data(), n, cp, plan.data(), int64_t(plan.size()), 8, 128, work.data(),
                      tok.data(), rcv.data(), &e4, &e5, &imb) == FC_OK);
  CHECK(fc_plan_stats(cu.data(), n, cp, plan.data(), int64_t(plan.size()), 8, 128, nullptr,
                      nullptr, nullptr, nullptr, nullptr, nullptr) == FC_OK);
  int64_t total = 0;
  for (int32_t t : tok) total += t;
  CHECK(total == cu.back());
}

void error_paths() {
  const std::vector<int32_t> cu = {0, 10, 30};
  int64_t k = 0;
  fc_shard out[16];
  CHECK(fc_plan_per_doc(nullptr, 2, 2, out, 16, &k) == FC_ERR_INVALID_ARG);
  CHECK(fc_plan_per_doc(cu.data(), 2, 0, out, 16, &k) != FC_OK);
  const std::vector<int32_t> bad = {0, 10, 5};
  CHECK(fc_plan_per_doc(bad.data(), 2, 2, out, 16, &k) != FC_OK);
  CHECK(fc_plan_hybrid(cu.data(), 2, 4, 1.05, out, 16, &k, nullptr) != FC_OK);  // 4 does not divide 30
  const fc_shard overlap[2] = {{0, 0, 0, 10}, {0, 1, 5, 5}};
  CHECK(fc_plan_validate(cu.data(), 2, 2, overlap, 2, 0) == FC_ERR_PLAN);
  fc_view v = nullptr;
  CHECK(fc_view_create(cu.data(), 2, overlap, 2, 2, 0, 4, 4, 64, nullptr, &v) == FC_ERR_PLAN);
  const fc_shard ok[2] = {{0, 0, 0, 10}, {1, 1, 0, 20}};
  CHECK(fc_view_create(cu.data(), 2, ok, 2, 2, 5, 4, 4, 64, nullptr, &v) == FC_ERR_INVALID_ARG);
  CHECK(fc_view_create(cu.data(), 2, ok, 2, 2, 0, 4, 4, 96, nullptr, &v) == FC_ERR_UNSUPPORTED);
  CHECK(fc_view_create(cu.data(), 2, ok, 2, 2, 0, 6, 4, 64, nullptr, &v) == FC_ERR_INVALID_ARG);
  const fc_tile_cfg t48{48, 0, 0, 0};
  CHECK(fc_view_create(cu.data(), 2, ok, 2, 2, 0, 4, 4, 64, &t48, &v) == FC_ERR_UNSUPPORTED);
  CHECK(fc_view_create(cu.data(), 2, ok, 2, 2, 0, 4, 4, 64, nullptr, nullptr) ==
        FC_ERR_INVALID_ARG);
  CHECK(fc_view_get_info(nullptr, nullptr) == FC_ERR_INVALID_ARG);
  fc_view_destroy(nullptr);
}

}  // namespace

int main(int argc, char** argv) {
  error_paths();
  // random contexts: document counts, lengths (one-token documents
  // included), CP degrees, plans, every rank, several head shapes and tiles
  std::mt19937 rng(12345);
  const fc_tile_cfg tile_cfgs[3] = {{0, 0, 0, 0}, {64, 64, 32, 128}, {128, 0, 0, 0}};
  int views = 0;
  for (int c = 0; c < 60; ++c) {
    const int n = 1 + int(rng() % 14);
    const int cp = 1 + int(rng() % 6);
    std::vector<int32_t> cu = {0};
    for (int j = 0; j < n; ++j)
      cu.push_back(cu.back() + (rng() % 5 == 0 ? 1 : 1 + int(rng() % 1500)));
    cu.back() += (cp - cu.back() % cp) % cp;  // cp | C for the hybrid planner
    for (const char* kind : {"per_doc", "per_seq", "whole_lpt", "hybrid"}) {
      const auto plan = plan_of(cu, cp, kind);
      exercise_plan_stats(cu, plan, cp);
      for (int r = 0; r < cp; ++r)
        for (int s = 0; s < 3; ++s) {
          const int shapes[3][3] = {{4, 4, 64}, {16, 2, 128}, {32, 8, 128}};
          exercise_view(cu, plan, cp, r, shapes[s][0], shapes[s][1], shapes[s][2],
                        &tile_cfgs[(c + r + s) % 3]);
          ++views;
        }
    }
  }
  // the workloads at full size
  if (argc > 1) {
    std::ifstream f(argv[1]);
    CHECK(f.good());
    std::string line;
    while (std::getline(f, line)) {
      std::istringstream in(line);
      std::string name, kind, rule;
      int cp, nd, hq, hkv, d;
      in >> name >> cp >> kind >> rule >> nd >> hq >> hkv >> d;
      std::vector<int32_t> cu(size_t(nd) + 1);
      for (auto& x : cu) in >> x;
      CHECK(!in.fail());
      const auto plan = plan_of(cu, cp, kind);
      exercise_plan_stats(cu, plan, cp);
      std::vector<int64_t> work(static_cast<size_t>(cp));
      CHECK(fc_plan_stats(cu.data(), nd, cp, plan.data(), int64_t(plan.size()), hkv, d,
                          work.data(), nullptr, nullptr, nullptr, nullptr, nullptr) == FC_OK);
      const int rank = rule == "last" ? cp - 1
                       : rule == "heaviest"
                           ? int(std::max_element(work.begin(), work.end()) - work.begin())
                           : std::atoi(rule.c_str());
      for (const auto& t : tile_cfgs) {
        exercise_view(cu, plan, cp, rank, hq, hkv, d, &t);
        ++views;
      }
      std::printf("workload %s: rank %d checked\n", name.c_str(), rank);
    }
  }
  std::printf("host driver: %d views, %lld stub launches, all checks passed\n", views,
              (long long)g_launches);
  return 0;
}
