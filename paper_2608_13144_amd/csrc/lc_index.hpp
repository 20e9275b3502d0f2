// Internal interface between the cluster index (index.hip) and the lookup
// (lookup.hip): the query-side plan of an indexed lookup.
#pragma once

#include "lc_common.hpp"

namespace lc {

constexpr int64_t kItemRows = 1024;     // cluster rows per work item at most (short lists)
constexpr int64_t kItemRowsMax = 2048;  // the same for long lists
constexpr int kMaxCand = 256;        // a query with more candidate clusters scans every indexed row

struct IndexPlanWs {
  uint32_t* mask;                  // [B][ceil(K / 32)] candidate clusters per query
  uint32_t* ccount;                // [K + 1] queries per cluster list (list K: queries scanned densely)
  uint32_t* cfill;                 // [K + 1] fill cursors
  int64_t* coff;                   // [K + 2] list offsets into qlist
  int32_t* qlist;                  // [qcap] the lists, concatenated
  int64_t qcap;
  int64_t* items;                  // [capacity][4]: query positions [0], [1); rows [2], [3)
  int64_t capacity;
  uint32_t* icount;                // [K + 1] work items per list
  int64_t* ioff;                   // [K + 2] first item of each list
  unsigned long long* counters;    // [0] items, [1] pairs, [2] overflow, [3] long shape
  double* qnorm;                   // [B] ||q||^2 (written by the lookup's query pass)
  double* cterm;                   // [K] centre term of the candidate test (Y_c)
  uint16_t* c16;                   // [K][d] float16 copy of the centres
};

size_t index_plan_layout(int64_t B, int d, int K, int64_t n_indexed, int qblock, IndexPlanWs* w, char* base);

// Candidate clusters of every query (every c with ||q - mu_c|| < R_c, tested
// on the float16 matrix cores with a rigorous slack), the list of queries of
// every cluster, and the work list: for every cluster, its queries in blocks
// against its rows in row chunks.  Short lists (under 512 queries on average
// over the K + 1 lists) are cut in query blocks of qb_short and chunks of at
// most kItemRows rows; long lists in blocks of qb_long and chunks of at most
// kItemRowsMax (long_items).  A query with more than kMaxCand candidates
// joins list K, which is scanned against all indexed rows.  Needs w.qnorm
// (||q||^2 in float64) and zq16 (the float16 copy of the queries) filled.
// Reads back the item and pair counts and the shape (sync).
lipcache_status index_query_plan(const lipcache_index* idx, const uint16_t* zq16, int64_t B, int d, int qb_short,
                                 int qb_long, const IndexPlanWs& w, int64_t& n_items, int64_t& pairs, bool& long_items,
                                 hipStream_t s);

}  // namespace lc
