// Internal interface between the cluster index (index.hip) and the lookup
// (lookup.hip): the query-side plan of an indexed lookup.
#pragma once

#include "lc_common.hpp"

namespace lc {

constexpr int64_t kItemRows = 8192;  // cluster rows per work item at most

struct IndexPlanWs {
  uint32_t* mask;                  // [B][ceil(K / 32)] candidate clusters per query
  uint32_t* keys[2];               // primary-cluster sort
  uint32_t* vals[2];
  uint32_t* hist;
  uint32_t* dsum;
  uint32_t* dbase;
  int64_t* qmap;                   // [B] internal query order -> original query
  float* zq_sorted;                // [B][d] queries in internal order
  int64_t* items;                  // [capacity][3]
  int64_t capacity;
  unsigned long long* counters;    // [0] items, [1] pairs, [2] overflow
};

size_t index_plan_layout(int64_t B, int d, int K, int64_t n_indexed, int qblock, IndexPlanWs* w, char* base);

// Candidate clusters of every query (||q - mu_c|| < R_c, tested with a
// rigorous float32 slack), queries sorted by their nearest cluster, and the
// work list: for every block of `qblock` sorted queries, the rows of each
// cluster any of its queries needs (split into items of <= kItemRows rows).
// Reads back the item and pair counts (sync).
lipcache_status index_query_plan(const lipcache_index* idx, const float* zq, int64_t B, int d, int qblock,
                                 const IndexPlanWs& w, int64_t& n_items, int64_t& pairs, hipStream_t s);

}  // namespace lc
