// Exercises the host side of the C ABI (schedule construction and argument
// checks) on many generated graphs; built with g++ and AddressSanitizer /
// UBSan by tests/test_host_sanitizers.py.  Prints "ok <cases>" on success and
// exits non-zero on the first violated property.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "featgraph_hip.h"

namespace {

uint64_t g_state = 0x9e3779b97f4a7c15ull;
uint64_t next_u64() {  // splitmix64
  uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
int64_t below(int64_t n) { return n <= 0 ? 0 : (int64_t)(next_u64() % (uint64_t)n); }

int g_fail = 0;
#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "check failed line %d: %s\n", __LINE__, #cond);   \
      std::exit(1);                                                          \
    }                                                                        \
  } while (0)

struct Graph {
  int64_t rows = 0, cols = 1;
  std::vector<int32_t> indptr, indices;
};

// Row degrees: mostly small, some empty, a few hubs; sources sorted per row
// unless `unsorted`.
// Rows in blocks of 40 that draw their sources from one block of 64 ids
// (neighbouring ids share sources), with degrees 20-60.
Graph make_blocked_graph(int64_t rows, int64_t cols) {
  Graph g;
  g.rows = rows;
  g.cols = cols;
  g.indptr.assign((size_t)rows + 1, 0);
  for (int64_t r = 0; r < rows; ++r) g.indptr[(size_t)r + 1] = g.indptr[(size_t)r] + 20 + (int32_t)below(41);
  g.indices.resize((size_t)g.indptr[(size_t)rows]);
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t base = ((r / 40) * 64) % std::max<int64_t>(cols - 64, 1);
    auto b = g.indices.begin() + g.indptr[(size_t)r], e = g.indices.begin() + g.indptr[(size_t)r + 1];
    for (auto it = b; it != e; ++it) *it = (int32_t)std::min<int64_t>(base + below(64), cols - 1);
    std::sort(b, e);
  }
  return g;
}

Graph make_graph(int64_t rows, int64_t cols, int64_t hub_deg, bool unsorted) {
  Graph g;
  g.rows = rows;
  g.cols = cols;
  g.indptr.assign((size_t)rows + 1, 0);
  for (int64_t r = 0; r < rows; ++r) {
    int64_t d = below(4) == 0 ? 0 : below(40);
    if (hub_deg > 0 && below(50) == 0) d = 1 + below(hub_deg);
    g.indptr[(size_t)r + 1] = g.indptr[(size_t)r] + (int32_t)d;
  }
  g.indices.resize((size_t)g.indptr[(size_t)rows]);
  for (int64_t r = 0; r < rows; ++r) {
    auto b = g.indices.begin() + g.indptr[(size_t)r], e = g.indices.begin() + g.indptr[(size_t)r + 1];
    for (auto it = b; it != e; ++it) *it = (int32_t)below(cols);
    if (!unsorted) std::sort(b, e);
  }
  return g;
}

void check_schedule(const Graph& g, const fg_plan_options& opt, int64_t width, int which,
                    bool with_indices) {
  const int32_t* ix = with_indices && !g.indices.empty() ? g.indices.data() : nullptr;
  int64_t nseg = -1, nsplit = -1, nslot = -1;
  fg_status st = fg_schedule_host(g.indptr.data(), ix, g.rows, g.cols, width, &opt, which,
                                  nullptr, 0, &nseg, &nsplit, &nslot);
  CHECK(st == FG_OK);
  CHECK(nseg >= g.rows && nsplit >= 0 && nslot >= 0);
  std::vector<fg_segment> segs((size_t)nseg + 1);
  segs[(size_t)nseg].row = 12345;  // sentinel past the requested capacity
  int64_t n2 = 0, s2 = 0, t2 = 0;
  st = fg_schedule_host(g.indptr.data(), ix, g.rows, g.cols, width, &opt, which, segs.data(), nseg,
                        &n2, &s2, &t2);
  CHECK(st == FG_OK && n2 == nseg && s2 == nsplit && t2 == nslot);
  CHECK(segs[(size_t)nseg].row == 12345);
  // every edge of every row covered exactly once; slots consecutive per row
  std::vector<int64_t> covered((size_t)g.rows, 0), pieces((size_t)g.rows, 0);
  std::vector<char> slot_seen((size_t)nslot, 0);
  int64_t slots = 0;
  for (int64_t i = 0; i < nseg; ++i) {
    const fg_segment& s = segs[(size_t)i];
    if (s.row < 0) {
      CHECK(s.row == -1 && s.begin == 0 && s.end == 0 && s.slot == -1);
      continue;
    }
    CHECK(s.row < g.rows);
    CHECK(s.begin >= g.indptr[(size_t)s.row] && s.end <= g.indptr[(size_t)s.row + 1]);
    CHECK(s.begin <= s.end);
    covered[(size_t)s.row] += s.end - s.begin;
    ++pieces[(size_t)s.row];
    if (s.slot >= 0) {
      CHECK(s.slot < nslot && !slot_seen[(size_t)s.slot]);
      slot_seen[(size_t)s.slot] = 1;
      ++slots;
    }
  }
  CHECK(slots == nslot);
  int64_t split_rows = 0;
  for (int64_t r = 0; r < g.rows; ++r) {
    CHECK(covered[(size_t)r] == g.indptr[(size_t)r + 1] - g.indptr[(size_t)r]);
    CHECK(pieces[(size_t)r] >= 1);
    if (pieces[(size_t)r] >= 2) ++split_rows;
  }
  // (the SDDMM's own schedule, which = 2, cuts rows without slots)
  CHECK((which == 2 && nslot == 0) || split_rows == nsplit);
  // pieces of one row never overlap: total covered equals nnz and each piece
  // lies in its row, so overlap would exceed the row's length (checked above)
  // a short capacity writes a prefix and leaves the rest untouched
  if (nseg > 1) {
    std::vector<fg_segment> part((size_t)nseg, fg_segment{7, 7, 7, 7});
    st = fg_schedule_host(g.indptr.data(), ix, g.rows, g.cols, width, &opt, which, part.data(),
                          nseg / 2, nullptr, nullptr, nullptr);
    CHECK(st == FG_OK);
    for (int64_t i = 0; i < nseg / 2; ++i)
      CHECK(part[(size_t)i].row == segs[(size_t)i].row && part[(size_t)i].begin == segs[(size_t)i].begin);
    CHECK(part[(size_t)(nseg / 2)].row == 7);
  }
}

void invalid_arguments() {
  const int32_t ip_ok[3] = {0, 2, 3}, ip_bad[3] = {0, 3, 2}, ix[3] = {0, 1, 4};
  fg_plan_options o{};
  int64_t n = 0;
  CHECK(fg_schedule_host(nullptr, nullptr, 2, 5, 8, &o, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  CHECK(fg_schedule_host(ip_bad, nullptr, 2, 5, 8, &o, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  CHECK(fg_schedule_host(ip_ok, ix, 2, 4, 8, &o, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);  // source id 4 with 4 columns
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 0, &o, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, FG_MAX_WIDTH + 1, &o, 0, nullptr, 0, &n, nullptr,
                         nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &o, -1, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  CHECK(fg_schedule_host(ip_ok, ix, -1, 5, 8, &o, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &o, 3, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  fg_plan_options bad = o;
  bad.segment_edges = -1;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  bad = o;
  bad.max_row_segments = 1;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  bad = o;
  bad.partition_min_degree = -3;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  bad = o;
  bad.item_order = 4;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  bad = o;
  bad.reserved[0] = 1;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  bad = o;
  bad.band_row_edges = -2;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  bad = o;
  bad.max_backward = 2;
  CHECK(fg_schedule_host(ip_ok, ix, 2, 5, 8, &bad, 0, nullptr, 0, &n, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  // entry points reject bad arguments before any device work
  fg_graph g{};
  g.num_rows = 2;
  g.num_cols = 5;
  g.nnz = 3;
  g.indptr = ip_ok;
  g.indices = ix;
  float buf[64];
  int32_t ibuf[64];
  CHECK(fg_gspmm(nullptr, FG_MSG_COPY_SRC, FG_REDUCE_SUM, 1, 4, buf, nullptr, buf + 32, nullptr,
                 nullptr, nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_gspmm(&g, (fg_msg_op)7, FG_REDUCE_SUM, 1, 4, buf, nullptr, buf + 32, nullptr, nullptr,
                 nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_gspmm(&g, FG_MSG_COPY_SRC, FG_REDUCE_MAX, 1, 4, buf, nullptr, buf + 32, nullptr,
                 nullptr, nullptr) == FG_ERR_INVALID_ARG);  // max needs arg_eid
  CHECK(fg_gspmm(&g, FG_MSG_COPY_SRC, FG_REDUCE_SUM, 0, 4, buf, nullptr, buf + 32, nullptr,
                 nullptr, nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_gspmm(&g, FG_MSG_COPY_SRC, FG_REDUCE_SUM, 1, 4, buf, nullptr, buf + 2, nullptr,
                 nullptr, nullptr) == FG_ERR_INVALID_ARG);  // out overlaps x
  CHECK(fg_gsddmm(&g, (fg_edge_op)3, 1, 4, buf, buf, buf + 40, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  CHECK(fg_edge_softmax(&g, 0, buf, 1, 0.2f, buf + 32, nullptr, nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_gspmm_max_backward(&g, FG_MSG_COPY_SRC, 1, 4, buf, nullptr, ibuf, buf + 8, buf + 32,
                              buf + 48, nullptr, nullptr) == FG_ERR_INVALID_ARG);  // no edge grad
  CHECK(fg_dense_matmul(-1, 2, 2, buf, buf, buf, nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_mlp_aggregate(&g, 0, 4, buf, buf, buf, buf, ibuf, buf, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  fg_graph bad_g = g;
  bad_g.nnz = -1;
  CHECK(fg_gsddmm(&bad_g, FG_EDGE_DOT, 1, 4, buf, buf, buf + 40, nullptr, nullptr) ==
        FG_ERR_INVALID_ARG);
  fg_plan* p = nullptr;
  CHECK(fg_plan_create(&g, ip_ok, ix, 0, nullptr, &p, nullptr) == FG_ERR_INVALID_ARG && !p);
  CHECK(fg_plan_create(&g, ip_bad, ix, 8, nullptr, &p, nullptr) == FG_ERR_INVALID_ARG && !p);
  CHECK(fg_plan_destroy(nullptr) == FG_ERR_INVALID_ARG);
  fg_plan_info info;
  CHECK(fg_plan_get_info(nullptr, &info) == FG_ERR_INVALID_ARG);
  uint64_t h1 = 0, h2 = 0;
  CHECK(fg_indptr_checksum(ip_ok, 2, &h1) == FG_OK);
  CHECK(fg_indptr_checksum(ip_bad, 2, &h2) == FG_OK && h1 != h2);
  CHECK(fg_indptr_checksum(nullptr, 2, &h1) == FG_ERR_INVALID_ARG);
  CHECK(fg_plan_validate(nullptr, &g, ip_ok, nullptr) == FG_ERR_INVALID_ARG);
  CHECK(fg_gspmm_noalloc(&g, FG_MSG_COPY_SRC, FG_REDUCE_MAX, 1, 4, buf, nullptr, buf + 32,
                         nullptr, nullptr, nullptr) == FG_ERR_INVALID_ARG);  // max needs arg_eid
  for (int s = -5; s <= 1; ++s) CHECK(fg_status_string((fg_status)s) != nullptr);
  CHECK(fg_abi_version() == FG_ABI_VERSION);
}

}  // namespace

int main() {
  invalid_arguments();
  int cases = 0;
  const int32_t seg_opts[] = {0, 1, 7, 64, 4096};
  const int32_t cap_opts[] = {0, 2, 5, 128};
  const int32_t slab_opts[] = {0, -1, 1, 64, 1000};
  const int32_t min_opts[] = {0, 1, 10, 1000};
  const int64_t widths[] = {1, 32, 128, 1024};
  const int32_t band_opts[] = {0, -1, 1, 9};
  for (int rep = 0; rep < 30; ++rep) {
    const int64_t rows = rep < 3 ? rep : below(3000);
    const int64_t cols = 1 + below(rep % 2 ? 50000 : 300);
    const Graph g = rep % 5 == 4 ? make_blocked_graph(rows, cols + 64)
                                 : make_graph(rows, cols, rep % 3 ? 20000 : 0, rep % 7 == 5);
    for (int t = 0; t < 6; ++t) {
      fg_plan_options o{};
      o.segment_edges = seg_opts[below(5)];
      o.max_row_segments = cap_opts[below(4)];
      o.source_slab_rows = slab_opts[below(5)];
      o.partition_min_degree = min_opts[below(4)];
      o.item_order = (int32_t)below(4);
      o.band_row_edges = band_opts[below(4)];
      const int64_t w = widths[below(4)];
      for (int which = 0; which < 3; ++which)
        for (int ind = 0; ind < 2; ++ind) {
          check_schedule(g, o, w, which, ind != 0);
          ++cases;
        }
    }
  }
  std::printf("ok %d\n", cases);
  return g_fail;
}
