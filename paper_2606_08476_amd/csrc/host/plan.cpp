// Shard planners and plan statistics (FlashCP Sec. 2.3, 3.1-3.4, Algorithm 1).
//
// Readings of what the paper leaves open are stated once, in the header's
// comments on each entry point; the repair loop of Algorithm 1 follows this
// reading of Max_Token_Worker_Pop / Whole_Doc_Shard_and_Add:
//   the worker with the largest token excess e (lowest index on ties) pops its
//   whole-document pieces last-in-first-out until they cover e, keeps the
//   tail of the last popped piece so that it ends at exactly C/N tokens, and
//   hands every earlier popped piece and then the head of that piece, in the
//   order they were popped and each from its first token on, to the
//   under-full workers with the least workload (lowest index on ties), each
//   taking what it has room for. Only document prefixes move, so
//   the extra receive volume stays proportional to the moved length (Sec. 3.3).
#include <algorithm>
#include <cstring>
#include <numeric>

#include "internal.hpp"

namespace fc {

namespace {

thread_local std::string g_err;

struct Piece {
  int32_t doc;
  int64_t off, len;
};

// Cut of document length L into 2cp Per-Doc chunks: chunk i spans
// [floor(i*L/2cp), floor((i+1)*L/2cp)) and belongs to worker min(i, 2cp-1-i).
template <class F>
void for_each_per_doc_chunk(int64_t L, int32_t cp, F&& f) {
  const int64_t parts = 2 * int64_t(cp);
  for (int64_t i = 0; i < parts; ++i) {
    const int64_t a = i * L / parts, b = (i + 1) * L / parts;
    if (b > a) f(int32_t(i < cp ? i : parts - 1 - i), a, b - a);
  }
}

std::vector<int32_t> longest_first(const std::vector<int64_t>& lens) {
  std::vector<int32_t> idx(lens.size());
  std::iota(idx.begin(), idx.end(), 0);
  std::stable_sort(idx.begin(), idx.end(),
                   [&](int32_t a, int32_t b) { return lens[a] > lens[b]; });
  return idx;
}

// Least workload among eligible workers, lowest index on ties; -1 if none.
int32_t least_loaded(const std::vector<int64_t>& work, const std::vector<int64_t>* tokens,
                     int64_t cap) {
  int32_t best = -1;
  for (int32_t j = 0; j < int32_t(work.size()); ++j) {
    if (tokens && (*tokens)[j] >= cap) continue;
    if (best < 0 || work[j] < work[best]) best = j;
  }
  return best;
}

double imbalance_of(const std::vector<int64_t>& work) {
  int64_t mx = 0, sum = 0;
  for (int64_t w : work) {
    mx = std::max(mx, w);
    sum += w;
  }
  return double(mx) * double(work.size()) / double(sum);
}

int emit(const std::vector<fc_shard>& rows, fc_shard* out, int64_t cap, int64_t* n_out) {
  if (!n_out) return fail(FC_ERR_INVALID_ARG, "n_out is null");
  *n_out = int64_t(rows.size());
  if (int64_t(rows.size()) > cap)
    return fail(FC_ERR_CAPACITY, "output capacity " + std::to_string(cap) + " < " +
                                     std::to_string(rows.size()) + " shards");
  if (!rows.empty() && !out) return fail(FC_ERR_INVALID_ARG, "out is null");
  if (!rows.empty()) std::memcpy(out, rows.data(), rows.size() * sizeof(fc_shard));
  return FC_OK;
}

}  // namespace

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}
void clear_error() { g_err.clear(); }
const char* last_error() { return g_err.c_str(); }

int doc_lengths(const int32_t* cu, int32_t n_docs, std::vector<int64_t>& lens) {
  if (!cu) return fail(FC_ERR_INVALID_ARG, "cu_seqlens is null");
  if (n_docs < 1) return fail(FC_ERR_INVALID_ARG, "n_docs must be >= 1");
  if (cu[0] != 0) return fail(FC_ERR_INVALID_ARG, "cu_seqlens[0] must be 0");
  lens.resize(n_docs);
  for (int32_t k = 0; k < n_docs; ++k) {
    lens[k] = int64_t(cu[k + 1]) - int64_t(cu[k]);
    if (lens[k] < 1)
      return fail(FC_ERR_INVALID_ARG, "document " + std::to_string(k) + " has length < 1");
  }
  return FC_OK;
}

std::vector<fc_shard> canonicalize(std::vector<fc_shard> v) {
  v.erase(std::remove_if(v.begin(), v.end(), [](const fc_shard& s) { return s.len <= 0; }),
          v.end());
  std::sort(v.begin(), v.end(), [](const fc_shard& a, const fc_shard& b) {
    return a.doc != b.doc ? a.doc < b.doc : a.offset < b.offset;
  });
  std::vector<fc_shard> out;
  for (const fc_shard& s : v) {
    if (!out.empty() && out.back().doc == s.doc && out.back().rank == s.rank &&
        out.back().offset + out.back().len == s.offset)
      out.back().len += s.len;
    else
      out.push_back(s);
  }
  return out;
}

int validate_plan(const std::vector<int64_t>& lens, int32_t cp, const fc_shard* s, int64_t n,
                  bool equal_tokens) {
  if (cp < 1) return fail(FC_ERR_INVALID_ARG, "cp must be >= 1");
  if (n < 0 || (n > 0 && !s)) return fail(FC_ERR_INVALID_ARG, "bad shard array");
  std::vector<fc_shard> v(s, s + n);
  std::vector<int64_t> tokens(cp, 0);
  for (const fc_shard& x : v) {
    if (x.doc < 0 || x.doc >= int32_t(lens.size()) || x.rank < 0 || x.rank >= cp ||
        x.len < 1 || x.offset < 0 || int64_t(x.offset) + x.len > lens[x.doc])
      return fail(FC_ERR_PLAN, "shard (doc " + std::to_string(x.doc) + ", rank " +
                                   std::to_string(x.rank) + ", offset " +
                                   std::to_string(x.offset) + ", len " +
                                   std::to_string(x.len) + ") out of range");
    tokens[x.rank] += x.len;
  }
  std::sort(v.begin(), v.end(), [](const fc_shard& a, const fc_shard& b) {
    return a.doc != b.doc ? a.doc < b.doc : a.offset < b.offset;
  });
  // Eq. 1: the shards of each document tile it exactly.
  size_t i = 0;
  for (int32_t k = 0; k < int32_t(lens.size()); ++k) {
    int64_t at = 0;
    while (i < v.size() && v[i].doc == k) {
      if (v[i].offset != at)
        return fail(FC_ERR_PLAN, "document " + std::to_string(k) +
                                     " is not covered exactly once at offset " +
                                     std::to_string(at));
      at += v[i].len;
      ++i;
    }
    if (at != lens[k])
      return fail(FC_ERR_PLAN, "document " + std::to_string(k) + " not fully covered");
  }
  if (equal_tokens) {
    const int64_t C = std::accumulate(lens.begin(), lens.end(), int64_t(0));
    if (C % cp) return fail(FC_ERR_PLAN, "C not divisible by cp (Eq. 2)");
    for (int32_t j = 0; j < cp; ++j)
      if (tokens[j] != C / cp)
        return fail(FC_ERR_PLAN, "rank " + std::to_string(j) + " holds " +
                                     std::to_string(tokens[j]) + " tokens, not C/N (Eq. 2)");
  }
  return FC_OK;
}

// Algorithm 1 state for one pass: Per-Doc chunks are fixed, whole-document
// pieces form a stack per worker.
struct HybridPass {
  int32_t cp;
  int64_t T;
  std::vector<std::vector<Piece>> fixed, stack;
  std::vector<int64_t> tokens, work;

  explicit HybridPass(int32_t n, int64_t t)
      : cp(n), T(t), fixed(n), stack(n), tokens(n, 0), work(n, 0) {}

  void add(std::vector<Piece>& list, int32_t j, Piece p) {
    list.push_back(p);
    tokens[j] += p.len;
    work[j] += shard_work(p.off, p.len);
  }

  void refresh(int32_t j) {
    tokens[j] = 0;
    work[j] = 0;
    for (const auto* lst : {&fixed[j], &stack[j]})
      for (const Piece& p : *lst) {
        tokens[j] += p.len;
        work[j] += shard_work(p.off, p.len);
      }
  }

  // Equal-token repair; returns when every worker holds T tokens or the
  // fullest worker has no whole-document piece left.
  void repair() {
    for (;;) {
      int32_t top = 0;
      bool equal = true;
      for (int32_t j = 0; j < cp; ++j) {
        if (tokens[j] != T) equal = false;
        if (tokens[j] > tokens[top]) top = j;
      }
      if (equal || stack[top].empty()) return;
      const int64_t excess = tokens[top] - T;
      std::vector<Piece> given;
      int64_t got = 0;
      while (got < excess && !stack[top].empty()) {
        given.push_back(stack[top].back());
        stack[top].pop_back();
        got += given.back().len;
      }
      if (got > excess) {  // keep the tail of the last popped piece
        Piece& last = given.back();
        const int64_t head = excess - (got - last.len);
        stack[top].push_back({last.doc, last.off + head, last.len - head});
        last.len = head;
      }
      refresh(top);
      for (const Piece& p : given) {
        int64_t pos = p.off, left = p.len;
        while (left > 0) {
          const int32_t r = least_loaded(work, &tokens, T);
          const int64_t take = std::min(left, T - tokens[r]);
          add(stack[r], r, {p.doc, pos, take});
          pos += take;
          left -= take;
        }
      }
    }
  }
};

}  // namespace fc

using namespace fc;

extern "C" {

const char* fc_last_error(void) { return fc::last_error(); }

int fc_plan_per_doc(const int32_t* cu, int32_t n_docs, int32_t cp, fc_shard* out, int64_t cap,
                    int64_t* n_out) {
  clear_error();
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  if (cp < 1) return fail(FC_ERR_INVALID_ARG, "cp must be >= 1");
  std::vector<fc_shard> rows;
  for (int32_t k = 0; k < n_docs; ++k)
    for_each_per_doc_chunk(lens[k], cp, [&](int32_t r, int64_t o, int64_t l) {
      rows.push_back({k, r, int32_t(o), int32_t(l)});
    });
  return emit(canonicalize(rows), out, cap, n_out);
}

int fc_plan_per_seq(const int32_t* cu, int32_t n_docs, int32_t cp, fc_shard* out, int64_t cap,
                    int64_t* n_out) {
  clear_error();
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  if (cp < 1) return fail(FC_ERR_INVALID_ARG, "cp must be >= 1");
  // chunk i of the whole packed sequence, intersected with every document it
  // meets (documents and chunks are both sorted, so one merge walk)
  const int64_t total = cu[n_docs], parts = 2 * int64_t(cp);
  std::vector<fc_shard> rows;
  int32_t k = 0;
  for (int64_t i = 0; i < parts; ++i) {
    const int64_t a = i * total / parts, b = (i + 1) * total / parts;
    const int32_t r = int32_t(i < cp ? i : parts - 1 - i);
    while (k < n_docs && cu[k + 1] <= a) ++k;
    for (int32_t d = k; d < n_docs && cu[d] < b; ++d) {
      const int64_t lo = std::max<int64_t>(a, cu[d]), hi = std::min<int64_t>(b, cu[d + 1]);
      if (hi > lo) rows.push_back({d, r, int32_t(lo - cu[d]), int32_t(hi - lo)});
    }
  }
  return emit(canonicalize(rows), out, cap, n_out);
}

int fc_plan_whole_lpt(const int32_t* cu, int32_t n_docs, int32_t cp, fc_shard* out, int64_t cap,
                      int64_t* n_out) {
  clear_error();
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  if (cp < 1) return fail(FC_ERR_INVALID_ARG, "cp must be >= 1");
  std::vector<int64_t> work(cp, 0);
  std::vector<fc_shard> rows;
  for (int32_t k : longest_first(lens)) {
    const int32_t j = least_loaded(work, nullptr, 0);
    rows.push_back({k, j, 0, int32_t(lens[k])});
    work[j] += shard_work(0, lens[k]);
  }
  return emit(canonicalize(rows), out, cap, n_out);
}

int fc_plan_hybrid(const int32_t* cu, int32_t n_docs, int32_t cp, double target_r, fc_shard* out,
                   int64_t cap, int64_t* n_out, uint8_t* is_per_doc) {
  clear_error();
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  if (cp < 1) return fail(FC_ERR_INVALID_ARG, "cp must be >= 1");
  if (!(target_r > 0)) return fail(FC_ERR_INVALID_ARG, "target_r must be > 0");
  const int64_t C = std::accumulate(lens.begin(), lens.end(), int64_t(0));
  if (C % cp) return fail(FC_ERR_INVALID_ARG, "context length not divisible by cp");
  const std::vector<int32_t> order = longest_first(lens);
  size_t n_per = 0;
  for (;;) {
    HybridPass st(cp, C / cp);
    for (size_t a = 0; a < n_per; ++a) {
      const int32_t k = order[a];
      for_each_per_doc_chunk(lens[k], cp, [&](int32_t r, int64_t o, int64_t l) {
        st.add(st.fixed[r], r, {k, o, l});
      });
    }
    for (size_t a = n_per; a < order.size(); ++a) {
      const int32_t k = order[a];
      const int32_t j = least_loaded(st.work, nullptr, 0);
      st.add(st.stack[j], j, {k, 0, lens[k]});
    }
    st.repair();
    const bool all_per_doc = n_per == order.size();
    if (imbalance_of(st.work) <= target_r || all_per_doc) {
      std::vector<fc_shard> rows;
      for (int32_t j = 0; j < cp; ++j)
        for (const auto* lst : {&st.fixed[j], &st.stack[j]})
          for (const Piece& p : *lst) rows.push_back({p.doc, j, int32_t(p.off), int32_t(p.len)});
      if (is_per_doc) {
        std::memset(is_per_doc, 0, size_t(n_docs));
        for (size_t a = 0; a < n_per; ++a) is_per_doc[order[a]] = 1;
      }
      return emit(canonicalize(rows), out, cap, n_out);
    }
    ++n_per;
  }
}

int fc_plan_validate(const int32_t* cu, int32_t n_docs, int32_t cp, const fc_shard* shards,
                     int64_t n_shards, int32_t require_equal_tokens) {
  clear_error();
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  return validate_plan(lens, cp, shards, n_shards, require_equal_tokens != 0);
}

int fc_plan_stats(const int32_t* cu, int32_t n_docs, int32_t cp, const fc_shard* shards,
                  int64_t n_shards, int32_t hkv, int32_t d, int64_t* work, int32_t* tokens,
                  int32_t* recv_tokens, int64_t* eq4, int64_t* eq5, double* imbalance) {
  clear_error();
  std::vector<int64_t> lens;
  if (int rc = doc_lengths(cu, n_docs, lens)) return rc;
  if (int rc = validate_plan(lens, cp, shards, n_shards, false)) return rc;
  if (hkv < 1 || d < 1) return fail(FC_ERR_INVALID_ARG, "hkv and d must be >= 1");
  std::vector<int64_t> w(cp, 0), tok(cp, 0), nonlast(cp, 0);
  std::vector<int32_t> last_off(n_docs, -1);
  for (int64_t i = 0; i < n_shards; ++i)
    last_off[shards[i].doc] = std::max(last_off[shards[i].doc], shards[i].offset);
  // held[(rank, doc)] -> (tokens held, end of the furthest held shard)
  std::vector<std::pair<int64_t, int64_t>> held(size_t(cp) * n_docs, {0, 0});
  for (int64_t i = 0; i < n_shards; ++i) {
    const fc_shard& s = shards[i];
    w[s.rank] += shard_work(s.offset, s.len);
    tok[s.rank] += s.len;
    auto& h = held[size_t(s.rank) * n_docs + s.doc];
    h.first += s.len;
    h.second = std::max<int64_t>(h.second, int64_t(s.offset) + s.len);
    if (s.offset != last_off[s.doc]) nonlast[s.rank] += s.len;
  }
  const int64_t C = std::accumulate(lens.begin(), lens.end(), int64_t(0));
  for (int32_t j = 0; j < cp; ++j) {
    if (work) work[j] = w[j];
    if (tokens) tokens[j] = int32_t(tok[j]);
    if (recv_tokens) {
      int64_t r = 0;
      for (int32_t k = 0; k < n_docs; ++k) {
        const auto& h = held[size_t(j) * n_docs + k];
        r += h.second - h.first;  // needed prefix minus what is held
      }
      recv_tokens[j] = int32_t(r);
    }
  }
  if (eq4) *eq4 = 4 * C * hkv * d * (cp - 1) / cp;
  if (eq5) *eq5 = 4 * *std::max_element(nonlast.begin(), nonlast.end()) * hkv * d * (cp - 1);
  if (imbalance) *imbalance = imbalance_of(w);
  return FC_OK;
}

}  // extern "C"
