// Internal declarations shared by the host side of the library.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "flashcp.h"

namespace fc {

// Record a message for fc_last_error() and return `code`.
int fail(int code, const std::string& msg);
void clear_error();

// Workload of a shard with prefix p and length s: the (query, key) pairs its
// queries see under the document mask, diagonal included (Sec. 3.1, Eq. 3).
inline int64_t shard_work(int64_t p, int64_t s) { return (2 * p + s + 1) * s / 2; }

// Checks cu_seqlens and returns the document lengths.
int doc_lengths(const int32_t* cu, int32_t n_docs, std::vector<int64_t>& lens);

// Sorts by (doc, offset), drops empty shards and joins adjacent shards of one
// document held by one rank.
std::vector<fc_shard> canonicalize(std::vector<fc_shard> v);

// Eq. 1 (and Eq. 2 when `equal_tokens`) check; message in fc_last_error().
int validate_plan(const std::vector<int64_t>& lens, int32_t cp, const fc_shard* s,
                  int64_t n, bool equal_tokens);

}  // namespace fc
