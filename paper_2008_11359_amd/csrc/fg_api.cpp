// fg_api.cpp -- C ABI of the library: host-side argument checks, the
// degree-aware schedule (plan), and dispatch to the gfx950 kernels.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstring>
#include <new>
#include <utility>
#include <vector>

#include "featgraph_hip.h"
#include "fg_internal.h"

// A plan holds two schedules over one workspace: the "gather" schedule used
// by the operators that gather source feature rows (gSpMM, gSDDMM, the fused
// attention kernel) and the plain length-ordered schedule used by edge
// softmax, which gathers nothing.
struct fg_plan {
  int64_t num_rows = 0, nnz = 0, max_width = 0;
  const int32_t* indptr = nullptr;  // device pointer the plan was built for
  int32_t segment_edges = 0, max_row_segments = 0, slab_rows = 0, partition_min_degree = 0;
  int64_t num_partitioned_rows = 0;
  int32_t item_order = 0;  // 1: longest first, 2: length classes, rows in id order
  int device = 0;
  fg::PlanView gather, plain;
  fg::PlanView edge;  // the SDDMM's own schedule on spread graphs (num_segments 0: none)
  // graphs with explicit edge ids: edge id -> storage position (the max
  // gradient needs the source of an edge given its id)
  const int32_t* edge_ids = nullptr;
  int64_t nnz_total = 0;
  int32_t* eid_pos = nullptr;
  fg::BinWorkspace bin;  // binned max backward (plan option), else empty
  std::vector<void*> mem;
  int64_t workspace_bytes = 0;
  uint64_t indptr_sum = 0;  // checksum of the indptr the schedules were built from
};

static_assert(fg::kNoAllocScratchBytes == FG_NOALLOC_SCRATCH_BYTES,
              "the fixed scratch size is part of the ABI");

namespace {

// The gather schedule cuts rows into pieces of at most 1,536 edges by
// default: the pieces of the long rows are what spreads them over the dies
// (die-banded order), and at this length a piece's partial result is still
// small next to the features it gathers (a sweep of 1,024-2,048 with the
// band threshold below put the power-law graph's step 2% faster here than at
// 2,048 with 512).
constexpr int32_t kDefaultSegmentEdges = 1536;
// The plain schedule (edge softmax) cuts only rows longer than this by
// default: a whole row of up to 16,384 scores is streamed by one wavefront
// (read twice, the second time mostly from the L2), while a cut row passes
// its statistics to a second kernel that reads it again from memory.
constexpr int32_t kDefaultPlainSegmentEdges = 16384;
constexpr int32_t kMaxSegmentEdges = 1 << 24;
constexpr int32_t kDefaultMaxRowSegments = 128;
// In the die-banded order, rows of more than this many edges are cut into at
// least one piece per die, so that each die gathers from one eighth of their
// sorted sources too (on the power-law graph, 4% off every gather kernel).
constexpr int32_t kDefaultBandRowEdges = 256;
constexpr int32_t kMaxRowSegmentsLimit = 1 << 20;

fg_status check_graph(const fg_graph* g) {
  if (!g) return FG_ERR_INVALID_ARG;
  if (g->num_rows < 0 || g->num_cols < 0 || g->nnz < 0) return FG_ERR_INVALID_ARG;
  if (g->num_rows >= INT32_MAX || g->num_cols > INT32_MAX || g->nnz > INT32_MAX)
    return FG_ERR_INVALID_ARG;
  if (g->nnz_total < 0 || g->nnz_total > INT32_MAX) return FG_ERR_INVALID_ARG;
  if (!g->edge_ids && g->nnz_total != 0 && g->nnz_total < g->nnz) return FG_ERR_INVALID_ARG;
  if (!g->indptr) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && !g->indices) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && g->num_cols == 0) return FG_ERR_INVALID_ARG;
  return FG_OK;
}

int64_t nnz_total_of(const fg_graph* g) { return g->nnz_total ? g->nnz_total : g->nnz; }

fg_status check_width(int64_t H, int64_t dh) {
  if (H < 1 || dh < 1 || H > FG_MAX_WIDTH || dh > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  if (H * dh > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  return FG_OK;
}

// true if [a, a+na) and [b, b+nb) (bytes) intersect; null or empty never do
bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
  if (!a || !b || na <= 0 || nb <= 0) return false;
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + (uintptr_t)nb && pb < pa + (uintptr_t)na;
}

fg_status check_plan(const fg_plan* p, const fg_graph* g, int64_t width) {
  if (!p) return FG_OK;
  if (p->num_rows != g->num_rows || p->nnz != g->nnz || p->indptr != g->indptr)
    return FG_ERR_INVALID_ARG;
  if (width > p->max_width) return FG_ERR_INVALID_ARG;
  return FG_OK;
}

fg::GraphView view_of(const fg_graph* g) {
  fg::GraphView v;
  v.num_rows = g->num_rows;
  v.num_cols = g->num_cols;
  v.nnz = g->nnz;
  v.nnz_total = nnz_total_of(g);
  v.indptr = g->indptr;
  v.indices = g->indices;
  v.edge_ids = g->edge_ids;
  return v;
}

fg_status from_hip(hipError_t e) { return e == hipSuccess ? FG_OK : FG_ERR_HIP; }

// 64-bit FNV-1a over the bytes of the int32 entries (little endian).
uint64_t checksum_of(const int32_t* ip, int64_t n) {
  uint64_t h = 14695981039346656037ull;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t v = (uint32_t)ip[i];
    for (int b = 0; b < 4; ++b) {
      h ^= (v >> (8 * b)) & 0xFFu;
      h *= 1099511628211ull;
    }
  }
  return h;
}

bool indptr_valid(const int32_t* ip, int64_t num_rows, int64_t nnz) {
  if (ip[0] != 0 || ip[num_rows] != nnz) return false;
  for (int64_t r = 0; r < num_rows; ++r)
    if (ip[r + 1] < ip[r]) return false;
  return true;
}

constexpr int kXcds = 8;            // MI355X: 8 accelerator dies, workgroups dealt round-robin
constexpr int kWavesPerGroup = 4;   // work items per workgroup (kernels launch 4 wavefronts)
// automatic slab width: the larger of 8 MiB of features and 1/16 of the
// source feature matrix (measured best on graphs without gather locality)
constexpr int64_t kAutoSlabBytes = 8 << 20;
constexpr int64_t kAutoSlabsPerMatrix = 16;
// automatic mode leaves feature matrices that the eight dies' L2s (4 MB
// each) hold together unpartitioned: there the pieces cost more than they save
constexpr int64_t kAutoMinMatrixBytes = int64_t(kXcds) * (4 << 20);
// by default (source_slab_rows == 0) automatic slabs are used once the source
// features exceed half the 256 MB Infinity Cache; below that the caches serve
// graphs with hubs or communities better than the pieces would
constexpr int64_t kDefaultPartitionBytes = int64_t(128) << 20;
constexpr int32_t kSlabsAuto = -1;  // source_slab_rows: automatic above 32 MiB
constexpr int32_t kSlabsOff = -2;   // source_slab_rows: never partition
// unless given, the smallest partitioned row has max(64, 8 * id slabs) edges:
// its pieces average at least 8 edges
constexpr int64_t kMinPartitionDegree = 64;
constexpr int64_t kMinPieceEdges = 8;

constexpr int32_t kOrderAuto = 0, kOrderByLength = 1, kOrderById = 2, kOrderDieBanded = 3;
constexpr int64_t kOrderWindows = 64, kOrderWindowRows = 32, kOrderWindowEdges = 1 << 16;

// Windows of up to kOrderWindowRows consecutive rows (at most
// kOrderWindowEdges edges each) spread evenly over the rows: [r0, r1).
std::vector<std::pair<int64_t, int64_t>> order_windows(const int32_t* ip, int64_t num_rows) {
  std::vector<std::pair<int64_t, int64_t>> w;
  if (num_rows < 2 * kOrderWindowRows) return w;
  const int64_t nw = std::min<int64_t>(kOrderWindows, num_rows / kOrderWindowRows);
  for (int64_t k = 0; k < nw; ++k) {
    const int64_t r0 = k * (num_rows - kOrderWindowRows) / std::max<int64_t>(nw - 1, 1);
    int64_t r1 = r0;
    while (r1 < r0 + kOrderWindowRows && (int64_t)ip[r1 + 1] - ip[r0] <= kOrderWindowEdges) ++r1;
    if (r1 - r0 >= 2) w.push_back({r0, r1});
  }
  return w;
}

// |a n b| / min(|a|, |b|) of two sorted lists (as multisets).
double overlap(const std::vector<int32_t>& a, const std::vector<int32_t>& b) {
  if (a.empty() || b.empty()) return 0.0;
  size_t i = 0, j = 0, c = 0;
  while (i < a.size() && j < b.size()) {
    if (a[i] < b[j]) ++i;
    else if (b[j] < a[i]) ++j;
    else { ++c; ++i; ++j; }
  }
  return (double)c / (double)std::min(a.size(), b.size());
}

// Whether rows with neighbouring ids draw on the same sources, as in graphs
// whose communities occupy id ranges.  win_ix[w] holds the indices of the
// rows of window w.  Rows of at least 4 edges: the mean source overlap of
// adjacent rows must be at least 2% and eight times that of rows from
// windows half the graph apart.
bool ids_share_sources(const int32_t* ip, const std::vector<std::pair<int64_t, int64_t>>& wins,
                       const std::vector<std::vector<int32_t>>& win_ix) {
  const size_t nw = wins.size();
  if (nw < 2) return false;
  auto row = [&](size_t w, int64_t r) {
    const int64_t base = ip[wins[w].first];
    std::vector<int32_t> v(win_ix[w].begin() + (ip[r] - base), win_ix[w].begin() + (ip[r + 1] - base));
    std::sort(v.begin(), v.end());
    return v;
  };
  double adj = 0.0, far = 0.0;
  int64_t na = 0, nf = 0;
  for (size_t w = 0; w < nw; ++w) {
    const int64_t r0 = wins[w].first, r1 = wins[w].second;
    const size_t w2 = (w + nw / 2) % nw;
    for (int64_t r = r0; r + 1 < r1; ++r) {
      if (ip[r + 1] - ip[r] < 4) continue;
      const std::vector<int32_t> a = row(w, r);
      if (ip[r + 2] - ip[r + 1] >= 4) {
        adj += overlap(a, row(w, r + 1));
        ++na;
      }
      const int64_t q = wins[w2].first + (r - r0);
      if (q < wins[w2].second && ip[q + 1] - ip[q] >= 4) {
        far += overlap(a, row(w2, q));
        ++nf;
      }
    }
  }
  if (na < 16 || nf < 16) return false;
  adj /= (double)na;
  far /= (double)nf;
  return adj >= 0.02 && adj >= 8.0 * far;
}

// ids_share_sources() on host indices.
bool ids_share_sources_host(const int32_t* ip, const int32_t* ix, int64_t num_rows) {
  const auto wins = order_windows(ip, num_rows);
  std::vector<std::vector<int32_t>> win_ix;
  for (const auto& w : wins) win_ix.emplace_back(ix + ip[w.first], ix + ip[w.second]);
  return ids_share_sources(ip, wins, win_ix);
}

// Share of the edges whose source is among the `rows` most used sources: the
// hit rate an L2 holding that many feature rows could at best reach.
double hot_source_share(const int32_t* ix, int64_t nnz, int64_t num_cols, int64_t rows) {
  if (nnz <= 0) return 1.0;
  std::vector<int32_t> cnt((size_t)num_cols, 0);
  for (int64_t q = 0; q < nnz; ++q) ++cnt[(size_t)ix[q]];
  if (rows < num_cols) {
    std::nth_element(cnt.begin(), cnt.begin() + rows, cnt.end(), std::greater<int32_t>());
    cnt.resize((size_t)rows);
  }
  int64_t top = 0;
  for (int32_t c : cnt) top += c;
  return (double)top / (double)nnz;
}

// Below the default threshold, features of more than kAutoMinMatrixBytes get
// slabs if the gathers are spread: the hottest 4 MB of source rows (one die's
// L2) take less than this share of the edges, and rows with neighbouring ids
// do not share sources.  (The power-law graph at d = 128: 66%, kept whole;
// rand-100K and uniform graphs at d = 128: 35% and 10%, cut.)
constexpr double kSpreadShare = 0.45;
constexpr int64_t kDieL2Bytes = 4 << 20;
// Spread graphs with source slabs at widths of this many floats or more, and
// features that the Infinity Cache holds, get a schedule of their own for
// the SDDMM: every row cut where its sources change slab (kEdgeSlabs slabs of
// about equal edge shares), with no merge to pay since the SDDMM writes
// per-edge results.  (The uniform graph's SDDMM: 1.36 -> 0.89 ms at d = 256,
// 2.76 -> 2.43 ms at d = 512; rand-100K's 5.62 -> 4.55 ms at d = 512.  At
// d = 128 the cut costs more than it gains, 0.40 -> 0.56 ms, and so it does
// on the 1M-vertex R-MAT graph's 1 GiB of features, 2.39 -> 2.90 ms.)
constexpr int64_t kEdgeScheduleMinWidth = 256;
constexpr int64_t kEdgeSlabs = 16;
constexpr int64_t kInfinityCacheBytes = int64_t(256) << 20;

struct Options {
  int32_t S, cap, slab, min_deg;  // slab 0: no source partitioning
  int32_t S_plain;                // segment length of the plain (edge softmax) schedule
  int32_t order;                  // item order: 0 automatic, 1 by length, 2 by class + id,
                                  // 3 die-banded gather schedule
  bool band_auto;                 // automatic order settled on 1: band the gather schedule
                                  // if some row has kXcds or more pieces
  bool slab_if_spread;            // keep the slabs only if the gathers are spread
  bool max_backward;              // reserve the binned max-backward workspace
  int32_t band_rows;              // die-banded: rows of more edges get >= kXcds pieces (-1: off)
  bool spread = false;            // slabs on spread gathers at a wide max_width whose features
                                  // the Infinity Cache holds: the SDDMM gets its own schedule
};

// Settles the automatic choices that depend on the graph: the item order and
// conditional slabs.  ix: host indices (all of them) or null; id_local: the
// result of ids_share_sources() if already known (-1: not known).
void settle_options(Options& o, const int32_t* ip, const int32_t* ix, int64_t num_rows,
                    int64_t num_cols, int64_t max_width, int id_local) {
  if (id_local < 0 && ix && (o.order == kOrderAuto || o.slab_if_spread))
    id_local = ids_share_sources_host(ip, ix, num_rows) ? 1 : 0;
  if (o.order == kOrderAuto) {
    o.order = id_local == 1 ? kOrderById : kOrderByLength;
    o.band_auto = o.order == kOrderByLength;
  }
  const int64_t rows = kDieL2Bytes / (4 * std::max<int64_t>(max_width, 1));
  double share = -1.0;  // hot_source_share, computed once if needed
  if (o.slab_if_spread) {
    if (!ix || id_local != 0 || (share = hot_source_share(ix, ip[num_rows], num_cols, rows)) >= kSpreadShare)
      o.slab = 0;
    o.slab_if_spread = false;
  }
  o.spread = false;
  if (ix && o.slab > 0 && max_width >= kEdgeScheduleMinWidth &&
      num_cols * max_width * 4 <= kInfinityCacheBytes) {
    if (id_local < 0) id_local = ids_share_sources_host(ip, ix, num_rows) ? 1 : 0;
    if (id_local == 0) {
      if (share < 0.0) share = hot_source_share(ix, ip[num_rows], num_cols, rows);
      o.spread = share < kSpreadShare;
    }
  }
}

struct Schedule {
  bool banded = false;  // die-banded order (band_by_die)
  std::vector<fg::Seg> segs;
  std::vector<fg::Fix> fix;
  std::vector<int32_t> slot_fix;  // slot -> index into fix
  std::vector<int32_t> slot_seg;  // slot -> index into segs
  int64_t partitioned_rows = 0;
};

// Pieces of a row cut into k (nearly) equal parts.
void cut_even(int32_t r, int64_t b, int64_t e, int64_t k, int32_t part,
              std::vector<std::pair<fg::Seg, int32_t>>& out) {
  const int64_t len = e - b;
  for (int64_t i = 0; i < k; ++i)
    out.push_back({fg::Seg{r, (int32_t)(b + len * i / k), (int32_t)(b + len * (i + 1) / k), -1},
                   part});
}

// Numbers the slots of rows with two or more pieces (consecutive per row, in
// row order), fills the split-row table, and returns the pieces.
void number_slots(std::vector<std::pair<fg::Seg, int32_t>>& pieces, Schedule& sc) {
  // pieces arrive grouped by row, in edge order within a row
  size_t i = 0;
  int32_t slot = 0;
  while (i < pieces.size()) {
    size_t j = i;
    while (j < pieces.size() && pieces[j].first.row == pieces[i].first.row) ++j;
    if (j - i >= 2) {
      fg::Fix fx;
      fx.row = pieces[i].first.row;
      fx.slot_begin = slot;
      for (size_t t = i; t < j; ++t) {
        pieces[t].first.slot = slot++;
        sc.slot_fix.push_back((int32_t)sc.fix.size());
      }
      fx.slot_end = slot;
      fx.pad = 0;
      sc.fix.push_back(fx);
    }
    i = j;
  }
  sc.slot_seg.assign(sc.slot_fix.size(), -1);
}

// Longest first (ties by row, then position).
bool longer(const fg::Seg& a, const fg::Seg& b) {
  const int64_t la = (int64_t)a.end - a.begin, lb = (int64_t)b.end - b.begin;
  if (la != lb) return la > lb;
  if (a.row != b.row) return a.row < b.row;
  return a.begin < b.begin;
}

// Length class of an item: -1 without edges, else ceil(log2(len)); rows of
// at most kShortRowEdges = 64 edges are classes <= 6, longer ones >= 7.
int len_class(int64_t len) {
  if (len <= 0) return -1;
  int c = 0;
  while ((int64_t(1) << c) < len) ++c;
  return c;
}

// Longest class first, then by row and position: the longest-processing-time
// order to within a factor of two in length, with the rows of one class in id
// order, which keeps the locality of graphs whose neighbouring ids share
// sources (communities).  Exact length order scatters such rows when their
// degrees differ slightly (the transposed clustered graph ran 1.7x slower);
// on graphs without such locality exact length order is faster (the
// power-law graph: 15%), so ids_share_sources() picks between the two.
bool longer_class(const fg::Seg& a, const fg::Seg& b) {
  const int ca = len_class((int64_t)a.end - a.begin), cb = len_class((int64_t)b.end - b.begin);
  if (ca != cb) return ca > cb;
  if (a.row != b.row) return a.row < b.row;
  return a.begin < b.begin;
}

// Plain schedule: rows with more than S edges are cut into
// k = min(ceil(deg / S), cap) equal pieces, and with band_rows >= 0 rows of
// more than band_rows edges into at least min(kXcds, cap, deg); items ordered
// longest first (longest-processing-time-first list scheduling), or by
// length class with rows in id order within a class (o.order ==
// kOrderById); rows without edges last.
void build_plain(const int32_t* ip, int64_t num_rows, const Options& o, Schedule& sc,
                 int64_t band_rows = -1) {
  std::vector<std::pair<fg::Seg, int32_t>> pieces;
  const int64_t kmin = std::min<int64_t>(kXcds, o.cap);
  for (int64_t r = 0; r < num_rows; ++r) {
    const int64_t deg = (int64_t)ip[r + 1] - ip[r];
    int64_t k = deg > o.S ? (deg + o.S - 1) / o.S : 1;
    if (k > o.cap) k = o.cap;
    if (band_rows >= 0 && deg > band_rows && k < kmin) k = std::min(kmin, deg);
    cut_even((int32_t)r, ip[r], ip[r + 1], k, -1, pieces);
  }
  number_slots(pieces, sc);
  sc.segs.reserve(pieces.size());
  for (auto& pc : pieces) sc.segs.push_back(pc.first);
  if (o.order == kOrderById) std::stable_sort(sc.segs.begin(), sc.segs.end(), longer_class);
  else std::stable_sort(sc.segs.begin(), sc.segs.end(), longer);
  for (size_t i = 0; i < sc.segs.size(); ++i)
    if (sc.segs[i].slot >= 0) sc.slot_seg[sc.segs[i].slot] = (int32_t)i;
}

// Deals per-die item streams into one item list: workgroup i (four items)
// runs on die i mod 8, so round r holds four items of die 0, then four of die
// 1, and so on; exhausted streams are padded with empty items (row = -1)
// that the kernels skip.  Fills slot -> item.
void interleave_streams(const std::vector<std::vector<fg::Seg>>& stream, Schedule& sc) {
  size_t longest = 0;
  for (auto& st : stream) longest = std::max(longest, st.size());
  const size_t rounds = (longest + kWavesPerGroup - 1) / kWavesPerGroup;
  sc.segs.reserve(rounds * kXcds * kWavesPerGroup);
  const fg::Seg none{-1, 0, 0, -1};
  for (size_t rd = 0; rd < rounds; ++rd)
    for (int x = 0; x < kXcds; ++x)
      for (int w = 0; w < kWavesPerGroup; ++w) {
        const size_t i = rd * kWavesPerGroup + w;
        sc.segs.push_back(i < stream[x].size() ? stream[x][i] : none);
      }
  for (size_t i = 0; i < sc.segs.size(); ++i)
    if (sc.segs[i].slot >= 0) sc.slot_seg[sc.segs[i].slot] = (int32_t)i;
}

// Gather schedule with source partitioning (the paper's 1D graph partitioning
// of source vertices, Sec. III-C, sized for one die's L2 instead of a CPU's
// LLC).  A row with at least o.min_deg edges whose sources are sorted is
// partitioned.  Source ids are cut
// into consecutive slabs of at most o.slab vertices that also hold about equal
// shares of the partitioned rows' edges (so that labellings which put the
// busy sources together still spread over the dies); partitioned rows are cut
// where their sources change slab, then into pieces of at most S edges.  Each
// slab goes, in slab order, to the die with the fewest partitioned edges so
// far, and its pieces join that die's stream: each die works through its
// slabs one at a time and finds their feature rows in its L2.  The remaining
// rows are cut as in the plain schedule and dealt to the streams, longest
// first, to even out the edges per die.  The streams are interleaved four
// items (one workgroup) at a time, following the round-robin order in which
// workgroups reach the dies; exhausted streams are padded with empty items
// (row = -1) that the kernels skip.
bool build_partitioned(const int32_t* ip, const int32_t* ix, int64_t num_rows, int64_t num_cols,
                       const Options& o, Schedule& sc) {
  if (o.slab <= 0) return false;
  const int64_t id_slabs = (num_cols + o.slab - 1) / o.slab;
  if (id_slabs < 2) return false;
  const int64_t min_deg = o.min_deg;
  // partitioned rows and the edges each source contributes to them
  std::vector<char> part_row((size_t)num_rows, 0);
  std::vector<int64_t> work((size_t)num_cols, 0);
  int64_t total = 0;
  for (int64_t r = 0; r < num_rows; ++r) {
    const int64_t b = ip[r], e = ip[r + 1];
    bool part = e - b >= min_deg;
    for (int64_t q = b + 1; part && q < e; ++q)
      if (ix[q] < ix[q - 1]) part = false;  // unsorted row: no contiguous slab ranges
    if (!part) continue;
    part_row[(size_t)r] = 1;
    for (int64_t q = b; q < e; ++q) ++work[(size_t)ix[q]];
    total += e - b;
  }
  if (total == 0) return false;
  // slab boundaries: at most o.slab ids and about total / max(id_slabs, dies) edges
  const int64_t target = (total + std::max<int64_t>(id_slabs, kXcds) - 1) /
                         std::max<int64_t>(id_slabs, kXcds);
  std::vector<int32_t> slab_of((size_t)num_cols);
  std::vector<int64_t> slab_work;
  int64_t start = 0, acc = 0;
  for (int64_t u = 0; u < num_cols; ++u) {
    if (u > start && (u - start == o.slab || acc >= target)) {
      slab_work.push_back(acc);
      start = u;
      acc = 0;
    }
    slab_of[(size_t)u] = (int32_t)slab_work.size();
    acc += work[(size_t)u];
  }
  slab_work.push_back(acc);
  const int64_t slabs = (int64_t)slab_work.size();

  std::vector<std::pair<fg::Seg, int32_t>> pieces;
  for (int64_t r = 0; r < num_rows; ++r) {
    const int64_t b = ip[r], e = ip[r + 1], deg = e - b;
    if (!part_row[(size_t)r]) {
      int64_t k = deg > o.S ? (deg + o.S - 1) / o.S : 1;
      if (k > o.cap) k = o.cap;
      cut_even((int32_t)r, b, e, k, -1, pieces);
      continue;
    }
    ++sc.partitioned_rows;
    int64_t q = b;
    while (q < e) {
      const int32_t slab = slab_of[(size_t)ix[q]];
      int64_t t = q;
      while (t < e && slab_of[(size_t)ix[t]] == slab) ++t;
      cut_even((int32_t)r, q, t, (t - q + o.S - 1) / o.S, slab, pieces);
      q = t;
    }
  }
  if (sc.partitioned_rows == 0) return false;
  number_slots(pieces, sc);

  // streams: partitioned pieces by (slab, row, position); then the rest
  std::vector<std::vector<fg::Seg>> stream(kXcds);
  std::vector<int64_t> load(kXcds, 0);
  std::vector<std::vector<fg::Seg>> by_slab((size_t)slabs);
  std::vector<fg::Seg> rest;
  for (auto& pc : pieces) {
    if (pc.second >= 0) by_slab[(size_t)pc.second].push_back(pc.first);
    else rest.push_back(pc.first);
  }
  for (int64_t sl = 0; sl < slabs; ++sl) {
    int x = 0;
    for (int y = 1; y < kXcds; ++y)
      if (load[y] < load[x]) x = y;
    for (auto& sg : by_slab[(size_t)sl]) {
      stream[x].push_back(sg);
      load[x] += (int64_t)sg.end - sg.begin;
    }
  }
  std::stable_sort(rest.begin(), rest.end(), longer);
  for (auto& sg : rest) {
    int x = 0;
    for (int y = 1; y < kXcds; ++y) {
      const int64_t len = (int64_t)sg.end - sg.begin;
      if (len > 0 ? load[y] < load[x] : stream[y].size() < stream[x].size()) x = y;
    }
    stream[x].push_back(sg);
    load[x] += (int64_t)sg.end - sg.begin;
  }
  interleave_streams(stream, sc);
  return true;
}

// Die-banded order of a plain schedule (item_order 3, gather schedule only).
// Piece k of a row cut into K pieces covers the fraction [k/K, (k+1)/K) of
// the row.  With K >= 8 it goes to die floor(8 (k + 1/2) / K), the eighth of
// the row its midpoint falls in; with fewer pieces it spans the dies
// [floor(8k/K), ceil(8(k+1)/K)), and the pieces of all rows that share one
// span take its dies in turn.  A row's sources are sorted, so the pieces
// that one die runs draw on about one eighth of their rows' source id range,
// instead of every die gathering from the whole feature matrix at once.  The
// pieces and their slots are unchanged (so are the results).  Whole rows go,
// longest first, to the die with the fewest edges so far; each die runs its
// items longest first.
void band_by_die(Schedule& sc) {
  std::vector<std::vector<fg::Seg>> stream(kXcds);
  std::vector<int64_t> load(kXcds, 0);
  std::vector<fg::Seg> rest;
  int64_t turn[kXcds][kXcds + 1] = {};
  for (const fg::Seg& sg : sc.segs) {
    if (sg.slot < 0) {
      rest.push_back(sg);
      continue;
    }
    const fg::Fix& fx = sc.fix[(size_t)sc.slot_fix[(size_t)sg.slot]];
    const int64_t k = sg.slot - fx.slot_begin, K = (int64_t)fx.slot_end - fx.slot_begin;
    int x;
    if (K >= kXcds) {
      x = (int)((2 * kXcds * k + kXcds) / (2 * K));  // die of the piece's midpoint
    } else {
      // fewer pieces than dies: the piece spans dies [lo, hi) of the row;
      // successive pieces of that span take them in turn
      const int lo = (int)(kXcds * k / K), hi = (int)((kXcds * (k + 1) + K - 1) / K);
      x = lo + (int)(turn[lo][hi]++ % (hi - lo));
    }
    stream[x].push_back(sg);
    load[x] += (int64_t)sg.end - sg.begin;
  }
  std::stable_sort(rest.begin(), rest.end(), longer);
  for (auto& sg : rest) {
    int x = 0;
    for (int y = 1; y < kXcds; ++y) {
      const int64_t len = (int64_t)sg.end - sg.begin;
      if (len > 0 ? load[y] < load[x] : stream[y].size() < stream[x].size()) x = y;
    }
    stream[x].push_back(sg);
    load[x] += (int64_t)sg.end - sg.begin;
  }
  for (auto& st : stream) std::stable_sort(st.begin(), st.end(), longer);
  sc.segs.clear();
  interleave_streams(stream, sc);
  sc.banded = true;
}

fg_status read_options(const fg_plan_options* opt, int64_t num_cols, int64_t max_width,
                       Options* o) {
  o->S = kDefaultSegmentEdges;
  o->S_plain = kDefaultPlainSegmentEdges;
  o->cap = kDefaultMaxRowSegments;
  o->slab = 0;
  o->min_deg = 0;
  int32_t slab_opt = 0, min_opt = 0;
  o->order = kOrderAuto;
  o->band_auto = false;
  o->band_rows = kDefaultBandRowEdges;
  o->slab_if_spread = false;
  o->max_backward = false;
  if (opt) {
    for (int32_t r : opt->reserved)
      if (r != 0) return FG_ERR_INVALID_ARG;
    if (opt->max_backward < 0 || opt->max_backward > 1) return FG_ERR_INVALID_ARG;
    o->max_backward = opt->max_backward == 1;
    if (opt->item_order < kOrderAuto || opt->item_order > kOrderDieBanded)
      return FG_ERR_INVALID_ARG;
    o->order = opt->item_order;
    if (opt->segment_edges < 0 || opt->segment_edges > kMaxSegmentEdges) return FG_ERR_INVALID_ARG;
    if (opt->max_row_segments < 0 || opt->max_row_segments > kMaxRowSegmentsLimit)
      return FG_ERR_INVALID_ARG;
    if (opt->partition_min_degree < 0) return FG_ERR_INVALID_ARG;
    if (opt->source_slab_rows < kSlabsOff) return FG_ERR_INVALID_ARG;
    if (opt->segment_edges) o->S = o->S_plain = opt->segment_edges;
    if (opt->softmax_segment_edges < 0 || opt->softmax_segment_edges > kMaxSegmentEdges)
      return FG_ERR_INVALID_ARG;
    if (opt->softmax_segment_edges) o->S_plain = opt->softmax_segment_edges;
    if (opt->band_row_edges < -1 || opt->band_row_edges > kMaxSegmentEdges)
      return FG_ERR_INVALID_ARG;
    if (opt->band_row_edges) o->band_rows = opt->band_row_edges;
    if (opt->max_row_segments) o->cap = opt->max_row_segments;
    slab_opt = opt->source_slab_rows;
    min_opt = opt->partition_min_degree;
  }
  if (o->cap < 2) return FG_ERR_INVALID_ARG;
  const int64_t feature_bytes = num_cols * 4 * std::max<int64_t>(max_width, 1);
  if (slab_opt > 0) {
    o->slab = slab_opt;
  } else if ((slab_opt == 0 && feature_bytes > kAutoMinMatrixBytes) ||
             (slab_opt == kSlabsAuto && feature_bytes > kAutoMinMatrixBytes)) {
    o->slab_if_spread = slab_opt == 0 && feature_bytes <= kDefaultPartitionBytes;
    const int64_t rows = std::max<int64_t>(kAutoSlabBytes / (4 * std::max<int64_t>(max_width, 1)),
                                           (num_cols + kAutoSlabsPerMatrix - 1) / kAutoSlabsPerMatrix);
    o->slab = (int32_t)std::min<int64_t>(std::max<int64_t>(64, rows), INT32_MAX);
  }
  if (o->slab > 0) {
    const int64_t id_slabs = (std::max<int64_t>(num_cols, 1) + o->slab - 1) / o->slab;
    o->min_deg = min_opt ? min_opt
                         : (int32_t)std::min<int64_t>(
                               std::max(kMinPartitionDegree, kMinPieceEdges * id_slabs), INT32_MAX);
  }
  return FG_OK;
}

// Both schedules of a graph.  indices may be null: no source partitioning.
fg_status make_schedules(const int32_t* ip, const int32_t* ix, int64_t num_rows, int64_t num_cols,
                         const Options& o, Schedule& gather, Schedule& plain,
                         Schedule* edge = nullptr) {
  try {
    Options op = o;
    op.S = o.S_plain;
    build_plain(ip, num_rows, op, plain);
    if (!ix || !build_partitioned(ip, ix, num_rows, num_cols, o, gather)) {
      bool band = o.order == kOrderDieBanded;
      if (o.band_auto) {  // some row cut into kXcds or more pieces by length
        int64_t max_deg = 0;
        for (int64_t r = 0; r < num_rows; ++r) max_deg = std::max<int64_t>(max_deg, ip[r + 1] - ip[r]);
        band = std::min<int64_t>((max_deg + o.S - 1) / o.S, o.cap) >= kXcds;
      }
      const int64_t band_rows = band ? o.band_rows : -1;
      if (o.S_plain == o.S && band_rows < 0) {
        gather = plain;
      } else {
        gather = Schedule();
        build_plain(ip, num_rows, o, gather, band_rows);
      }
      gather.partitioned_rows = 0;
      if (band) band_by_die(gather);
    }
    if (edge) {
      // the SDDMM's schedule on spread graphs: every row cut at slab
      // boundaries; its per-edge results need no slots
      *edge = Schedule();
      Options oe = o;
      oe.slab = (int32_t)std::max<int64_t>(1, (num_cols + kEdgeSlabs - 1) / kEdgeSlabs);
      oe.min_deg = 1;
      if (ix && o.spread && build_partitioned(ip, ix, num_rows, num_cols, oe, *edge)) {
        for (fg::Seg& sg : edge->segs) sg.slot = -1;
        edge->fix.clear();
        edge->slot_fix.clear();
        edge->slot_seg.clear();
      } else {
        *edge = Schedule();
      }
    }
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  return FG_OK;
}

bool indices_valid(const int32_t* ix, int64_t nnz, int64_t num_cols) {
  for (int64_t q = 0; q < nnz; ++q)
    if (ix[q] < 0 || ix[q] >= num_cols) return false;
  return true;
}

}  // namespace

extern "C" {

const char* fg_status_string(fg_status s) {
  switch (s) {
    case FG_OK: return "ok";
    case FG_ERR_INVALID_ARG: return "invalid argument";
    case FG_ERR_UNSUPPORTED: return "unsupported combination";
    case FG_ERR_HIP: return "HIP runtime error";
    case FG_ERR_NO_MEMORY: return "out of memory";
    case FG_ERR_SCRATCH_LIMIT:
      return "the split-row partials exceed the fixed scratch of the allocation-free entry point";
  }
  return "unknown status";
}

int32_t fg_abi_version(void) { return FG_ABI_VERSION; }

fg_status fg_schedule_host(const int32_t* indptr_host, const int32_t* indices_host,
                           int64_t num_rows, int64_t num_cols, int64_t max_width,
                           const fg_plan_options* opt, int32_t which, fg_segment* segs,
                           int64_t capacity, int64_t* num_segments, int64_t* num_split_rows,
                           int64_t* num_slots) {
  if (!indptr_host || num_rows < 0 || num_rows >= INT32_MAX || num_cols < 0 ||
      num_cols > INT32_MAX || capacity < 0 || which < 0 || which > 2)
    return FG_ERR_INVALID_ARG;
  if (max_width < 1 || max_width > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  Options o;
  fg_status st = read_options(opt, num_cols, max_width, &o);
  if (st != FG_OK) return st;
  const int64_t nnz = indptr_host[num_rows];
  if (!indptr_valid(indptr_host, num_rows, nnz)) return FG_ERR_INVALID_ARG;
  if (indices_host && !indices_valid(indices_host, nnz, num_cols)) return FG_ERR_INVALID_ARG;
  try {
    settle_options(o, indptr_host, indices_host, num_rows, num_cols, max_width, -1);
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  Schedule gather, plain, edge;
  if ((st = make_schedules(indptr_host, indices_host, num_rows, num_cols, o, gather, plain,
                           &edge)) != FG_OK)
    return st;
  // which 2: the SDDMM's schedule (the gather schedule where it has none)
  const Schedule& sc = which == 1 ? plain : (which == 2 && !edge.segs.empty() ? edge : gather);
  if (num_segments) *num_segments = (int64_t)sc.segs.size();
  if (num_split_rows) *num_split_rows = (int64_t)sc.fix.size();
  if (num_slots) *num_slots = (int64_t)sc.slot_fix.size();
  if (segs) {
    const int64_t n = std::min<int64_t>(capacity, (int64_t)sc.segs.size());
    for (int64_t i = 0; i < n; ++i) {
      segs[i].row = sc.segs[i].row;
      segs[i].begin = sc.segs[i].begin;
      segs[i].end = sc.segs[i].end;
      segs[i].slot = sc.segs[i].slot;
    }
  }
  return FG_OK;
}

fg_status fg_plan_destroy(fg_plan* plan) {
  if (!plan) return FG_ERR_INVALID_ARG;
  int cur = 0;
  const bool have_dev = hipGetDevice(&cur) == hipSuccess;
  if (have_dev && cur != plan->device) (void)hipSetDevice(plan->device);
  fg_status st = FG_OK;
  for (void*& m : plan->mem) {
    if (m && hipFree(m) != hipSuccess) st = FG_ERR_HIP;
    m = nullptr;
  }
  if (have_dev && cur != plan->device) (void)hipSetDevice(cur);
  delete plan;
  return st;
}

namespace {

// Device copy of one schedule; the plan owns the allocations.
fg_status upload(fg_plan* p, const Schedule& sc, fg::PlanView& v, hipStream_t hs) {
  auto put = [&](const void* src, size_t bytes, void** dst) -> fg_status {
    void* d = nullptr;
    if (hipMalloc(&d, std::max<size_t>(bytes, 16)) != hipSuccess) return FG_ERR_NO_MEMORY;
    p->mem.push_back(d);
    if (bytes && hipMemcpyAsync(d, src, bytes, hipMemcpyHostToDevice, hs) != hipSuccess)
      return FG_ERR_HIP;
    *dst = d;
    return FG_OK;
  };
  void *a, *b, *c, *d;
  fg_status st;
  if ((st = put(sc.segs.data(), sizeof(fg::Seg) * sc.segs.size(), &a)) != FG_OK) return st;
  if ((st = put(sc.fix.data(), sizeof(fg::Fix) * sc.fix.size(), &b)) != FG_OK) return st;
  if ((st = put(sc.slot_fix.data(), sizeof(int32_t) * sc.slot_fix.size(), &c)) != FG_OK) return st;
  if ((st = put(sc.slot_seg.data(), sizeof(int32_t) * sc.slot_seg.size(), &d)) != FG_OK) return st;
  v.segs = static_cast<const fg::Seg*>(a);
  v.fix = static_cast<const fg::Fix*>(b);
  v.slot_fix = static_cast<const int32_t*>(c);
  v.slot_seg = static_cast<const int32_t*>(d);
  v.num_segments = (int64_t)sc.segs.size();
  // leading long items, then short non-empty rows, then empty rows (the
  // plain schedule's order by length class); any other order keeps every item
  // in the first group
  int64_t nl = 0, nn = 0, nm = 0;
  bool ordered = true, short_whole = true, medium_whole = true;
  int prev = INT32_MAX;
  for (const fg::Seg& sg : sc.segs) {
    const int64_t len = (int64_t)sg.end - sg.begin;
    const int cls = len_class(len);
    if (sg.row < 0 || cls > prev) ordered = false;
    prev = cls;
    if (len > fg::kMediumRowEdges) ++nm;
    else if (len > fg::kShortRowEdges && sg.slot >= 0) medium_whole = false;
    if (len > fg::kShortRowEdges) ++nl;
    else if (len > 0 && sg.slot >= 0) short_whole = false;  // a piece of a split row
    if (len > 0) ++nn;
  }
  // (kMediumRowEdges and kShortRowEdges are powers of two, so the length
  // classes that order the items separate the three groups)
  v.num_nonempty = ordered ? nn : v.num_segments;
  v.num_long = (ordered && short_whole) ? nl : v.num_nonempty;
  v.num_medium = (ordered && short_whole && medium_whole) ? nm : v.num_long;
  v.num_split_rows = (int64_t)sc.fix.size();
  v.num_slots = (int64_t)sc.slot_fix.size();
  return FG_OK;
}

}  // namespace

fg_status fg_plan_create(const fg_graph* g, const int32_t* indptr_host,
                         const int32_t* indices_host, int64_t max_width,
                         const fg_plan_options* opt, fg_plan** out, void* stream) {
  if (!out) return FG_ERR_INVALID_ARG;
  *out = nullptr;
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if (max_width < 1 || max_width > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  Options o;
  if ((st = read_options(opt, g->num_cols, max_width, &o)) != FG_OK) return st;
  // binned max-backward records are addressed with int32 offsets
  if (o.max_backward && g->num_rows * max_width > INT32_MAX) return FG_ERR_UNSUPPORTED;
  hipStream_t hs = static_cast<hipStream_t>(stream);

  std::vector<int32_t> ip_copy, ix_copy;
  const int32_t* ip = indptr_host;
  const int32_t* ix = indices_host;
  try {
    if (!ip) {
      ip_copy.resize((size_t)g->num_rows + 1);
      if (hipMemcpyAsync(ip_copy.data(), g->indptr, sizeof(int32_t) * ip_copy.size(),
                         hipMemcpyDeviceToHost, hs) != hipSuccess ||
          hipStreamSynchronize(hs) != hipSuccess)
        return FG_ERR_HIP;
      ip = ip_copy.data();
    }
    if (!indptr_valid(ip, g->num_rows, g->nnz)) return FG_ERR_INVALID_ARG;
    if (!ix && o.slab > 0 && g->nnz > 0) {
      ix_copy.resize((size_t)g->nnz);
      if (hipMemcpyAsync(ix_copy.data(), g->indices, sizeof(int32_t) * ix_copy.size(),
                         hipMemcpyDeviceToHost, hs) != hipSuccess ||
          hipStreamSynchronize(hs) != hipSuccess)
        return FG_ERR_HIP;
      ix = ix_copy.data();
    }
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  if (ix && !indices_valid(ix, g->nnz, g->num_cols)) return FG_ERR_INVALID_ARG;
  try {
    if (ix) {
      settle_options(o, ip, ix, g->num_rows, g->num_cols, max_width, -1);
    } else if (o.order == kOrderAuto) {  // sample windows of the device indices
      const auto wins = order_windows(ip, g->num_rows);
      std::vector<std::vector<int32_t>> win_ix;
      for (const auto& w : wins) {
        win_ix.emplace_back((size_t)(ip[w.second] - ip[w.first]));
        if (!win_ix.back().empty() &&
            hipMemcpyAsync(win_ix.back().data(), g->indices + ip[w.first],
                           sizeof(int32_t) * win_ix.back().size(), hipMemcpyDeviceToHost,
                           hs) != hipSuccess)
          return FG_ERR_HIP;
      }
      if (!wins.empty() && hipStreamSynchronize(hs) != hipSuccess) return FG_ERR_HIP;
      o.order = ids_share_sources(ip, wins, win_ix) ? kOrderById : kOrderByLength;
      o.band_auto = o.order == kOrderByLength;
    }
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  if (o.slab_if_spread) o.slab = 0;  // (conditional slabs always come with host indices)
  if (o.slab <= 0) ix = nullptr;

  Schedule gather, plain, edge;
  if ((st = make_schedules(ip, ix, g->num_rows, g->num_cols, o, gather, plain, &edge)) != FG_OK)
    return st;
  fg_plan* p = nullptr;
  try {
    p = new fg_plan();
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  p->num_rows = g->num_rows;
  p->nnz = g->nnz;
  p->max_width = max_width;
  p->indptr = g->indptr;
  p->indptr_sum = checksum_of(ip, g->num_rows + 1);
  p->segment_edges = o.S;
  p->max_row_segments = o.cap;
  p->slab_rows = ix ? o.slab : 0;
  p->partition_min_degree = ix ? o.min_deg : 0;
  p->num_partitioned_rows = gather.partitioned_rows;
  p->item_order = gather.banded ? kOrderDieBanded : o.order;
  if (hipGetDevice(&p->device) != hipSuccess) {
    delete p;
    return FG_ERR_HIP;
  }
  if ((st = upload(p, gather, p->gather, hs)) != FG_OK ||
      (st = upload(p, plain, p->plain, hs)) != FG_OK ||
      (!edge.segs.empty() && (st = upload(p, edge, p->edge, hs)) != FG_OK)) {
    (void)hipStreamSynchronize(hs);
    fg_plan_destroy(p);
    return st;
  }
  // shared workspace: per slot F partial values (or 2H softmax pairs, or the
  // fused kernel's F + 2H) and F argmax ids; per split row 2H merged pairs
  const int64_t nslots = std::max(p->gather.num_slots, p->plain.num_slots);
  const int64_t nsplit = std::max(p->gather.num_split_rows, p->plain.num_split_rows);
  const int64_t ws_width = 2 * max_width;
  const size_t wb[3] = {sizeof(float) * (size_t)std::max<int64_t>(nslots * ws_width, 4),
                        sizeof(int32_t) * (size_t)std::max<int64_t>(nslots * max_width, 4),
                        sizeof(float) * (size_t)std::max<int64_t>(nsplit * ws_width, 4)};
  void* w[3] = {nullptr, nullptr, nullptr};
  for (int i = 0; i < 3; ++i) {
    if (hipMalloc(&w[i], wb[i]) != hipSuccess) {
      (void)hipStreamSynchronize(hs);
      fg_plan_destroy(p);
      return FG_ERR_NO_MEMORY;
    }
    p->mem.push_back(w[i]);
  }
  for (fg::PlanView* v : {&p->gather, &p->plain}) {
    v->ws_f = static_cast<float*>(w[0]);
    v->ws_i = static_cast<int32_t*>(w[1]);
    v->ws_row = static_cast<float*>(w[2]);
    v->ws_width = ws_width;
  }
  p->workspace_bytes = (int64_t)(wb[0] + wb[1] + wb[2]);
  if (g->edge_ids) {
    p->edge_ids = g->edge_ids;
    p->nnz_total = nnz_total_of(g);
    void* m = nullptr;
    const size_t mb = sizeof(int32_t) * (size_t)std::max<int64_t>(p->nnz_total, 1);
    if (hipMalloc(&m, mb) != hipSuccess) {
      (void)hipStreamSynchronize(hs);
      fg_plan_destroy(p);
      return FG_ERR_NO_MEMORY;
    }
    p->mem.push_back(m);
    p->eid_pos = static_cast<int32_t*>(m);
    p->workspace_bytes += (int64_t)mb;
    if (fg::launch_build_eid_pos(g->edge_ids, g->nnz, p->nnz_total, p->eid_pos, hs) !=
        hipSuccess) {
      (void)hipStreamSynchronize(hs);
      fg_plan_destroy(p);
      return FG_ERR_HIP;
    }
  }
  if (o.max_backward) {
    // one 8-byte record per gradient element; bin tables; per-group runs
    // for the most tiles any width up to max_width needs (narrower rows put
    // more sources in a tile)
    const int64_t cap = std::max<int64_t>(g->num_rows * max_width, 1);
    const int64_t bins = std::max<int64_t>(
        1, std::min<int64_t>(fg::kMaxBins,
                             fg::bin_tiles(g->num_cols, std::min<int64_t>(max_width,
                                                                          fg::kBinTileFloats))));
    const size_t sz[3] = {8 * (size_t)cap, sizeof(int32_t) * 4 * (size_t)(fg::kMaxBins + 1),
                          sizeof(int32_t) * (size_t)fg::kBinGroups * (size_t)bins};
    void* m[3] = {nullptr, nullptr, nullptr};
    for (int i = 0; i < 3; ++i) {
      if (hipMalloc(&m[i], sz[i]) != hipSuccess) {
        (void)hipStreamSynchronize(hs);
        fg_plan_destroy(p);
        return FG_ERR_NO_MEMORY;
      }
      p->mem.push_back(m[i]);
      p->workspace_bytes += (int64_t)sz[i];
    }
    p->bin.rec = m[0];
    p->bin.rec_capacity = cap;
    p->bin.tables = static_cast<int32_t*>(m[1]);
    p->bin.runs = static_cast<int32_t*>(m[2]);
    p->bin.max_bins = bins;
  }
  if (hipStreamSynchronize(hs) != hipSuccess) {  // host schedules die on return
    fg_plan_destroy(p);
    return FG_ERR_HIP;
  }
  *out = p;
  return FG_OK;
}

fg_status fg_plan_get_info(const fg_plan* plan, fg_plan_info* info) {
  if (!plan || !info) return FG_ERR_INVALID_ARG;
  std::memset(info, 0, sizeof(*info));
  info->num_rows = plan->num_rows;
  info->nnz = plan->nnz;
  info->num_segments = plan->gather.num_segments;
  info->num_split_rows = plan->gather.num_split_rows;
  info->num_slots = plan->gather.num_slots;
  info->num_partitioned_rows = plan->num_partitioned_rows;
  info->plain_segments = plan->plain.num_segments;
  info->plain_split_rows = plan->plain.num_split_rows;
  info->plain_slots = plan->plain.num_slots;
  info->max_width = plan->max_width;
  info->workspace_bytes = plan->workspace_bytes;
  info->segment_edges = plan->segment_edges;
  info->max_row_segments = plan->max_row_segments;
  info->source_slab_rows = plan->slab_rows;
  info->partition_min_degree = plan->partition_min_degree;
  info->item_order = plan->item_order;
  info->max_backward = plan->bin.rec ? 1 : 0;
  info->indptr_checksum = plan->indptr_sum;
  info->sddmm_segments = plan->edge.num_segments;
  return FG_OK;
}

fg_status fg_indptr_checksum(const int32_t* indptr_host, int64_t num_rows, uint64_t* out) {
  if (!indptr_host || !out || num_rows < 0 || num_rows >= INT32_MAX) return FG_ERR_INVALID_ARG;
  *out = checksum_of(indptr_host, num_rows + 1);
  return FG_OK;
}

fg_status fg_plan_validate(const fg_plan* plan, const fg_graph* g, const int32_t* indptr_host,
                           void* stream) {
  if (!plan) return FG_ERR_INVALID_ARG;
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_plan(plan, g, 1)) != FG_OK) return st;
  std::vector<int32_t> copy;
  const int32_t* ip = indptr_host;
  if (!ip) {
    try {
      copy.resize((size_t)g->num_rows + 1);
    } catch (const std::bad_alloc&) {
      return FG_ERR_NO_MEMORY;
    }
    hipStream_t hs = static_cast<hipStream_t>(stream);
    if (hipMemcpyAsync(copy.data(), g->indptr, sizeof(int32_t) * copy.size(),
                       hipMemcpyDeviceToHost, hs) != hipSuccess ||
        hipStreamSynchronize(hs) != hipSuccess)
      return FG_ERR_HIP;
    ip = copy.data();
  }
  return checksum_of(ip, g->num_rows + 1) == plan->indptr_sum ? FG_OK : FG_ERR_INVALID_ARG;
}

}  // extern "C"

namespace {

// Host-side checks shared by fg_gspmm and fg_gspmm_noalloc.
fg_status check_gspmm(const fg_graph* g, fg_msg_op msg, fg_reduce_op red, int32_t num_heads,
                      int64_t head_dim, const float* x_src, const float* edge_val,
                      const float* out, const int32_t* arg_eid, const fg_plan* plan) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_width(num_heads, head_dim)) != FG_OK) return st;
  if (msg != FG_MSG_COPY_SRC && msg != FG_MSG_SRC_MUL_EDGE) return FG_ERR_INVALID_ARG;
  if (red != FG_REDUCE_SUM && red != FG_REDUCE_MAX) return FG_ERR_INVALID_ARG;
  const int64_t F = (int64_t)num_heads * head_dim;
  const bool mul = msg == FG_MSG_SRC_MUL_EDGE, mx = red == FG_REDUCE_MAX;
  if (mul != (edge_val != nullptr)) return FG_ERR_INVALID_ARG;
  if (mx != (arg_eid != nullptr)) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && !x_src) return FG_ERR_INVALID_ARG;
  if (g->num_rows > 0 && !out) return FG_ERR_INVALID_ARG;
  if ((st = check_plan(plan, g, F)) != FG_OK) return st;
  const int64_t out_b = g->num_rows * F * 4;
  const int64_t x_b = g->num_cols * F * 4;
  const int64_t ev_b = nnz_total_of(g) * num_heads * 4;
  if (overlaps(out, out_b, x_src, x_b) || overlaps(out, out_b, edge_val, ev_b) ||
      overlaps(arg_eid, out_b, x_src, x_b) || overlaps(arg_eid, out_b, edge_val, ev_b) ||
      overlaps(out, out_b, arg_eid, out_b))
    return FG_ERR_INVALID_ARG;
  return FG_OK;
}

}  // namespace

extern "C" {

fg_status fg_gspmm(const fg_graph* g, fg_msg_op msg, fg_reduce_op red, int32_t num_heads,
                   int64_t head_dim, const float* x_src, const float* edge_val, float* out,
                   int32_t* arg_eid, fg_plan* plan, void* stream) {
  const fg_status st =
      check_gspmm(g, msg, red, num_heads, head_dim, x_src, edge_val, out, arg_eid, plan);
  if (st != FG_OK) return st;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_gspmm(gv, plan ? &plan->gather : nullptr, (int)msg, (int)red,
                                   num_heads, head_dim, x_src, edge_val, out, arg_eid,
                                   static_cast<hipStream_t>(stream)));
}

fg_status fg_gspmm_noalloc(const fg_graph* g, fg_msg_op msg, fg_reduce_op red, int32_t num_heads,
                           int64_t head_dim, const float* x_src, const float* edge_val,
                           float* out, int32_t* arg_eid, fg_plan* plan, void* stream) {
  fg_status st =
      check_gspmm(g, msg, red, num_heads, head_dim, x_src, edge_val, out, arg_eid, plan);
  if (st != FG_OK) return st;
  void* base = nullptr;  // this device's copy of the fixed scratch
  if (fg::noalloc_scratch(&base) != hipSuccess) return FG_ERR_HIP;
  const int64_t F = (int64_t)num_heads * head_dim;
  const bool mx = red == FG_REDUCE_MAX;
  const fg::GraphView gv = view_of(g);
  if (!plan || plan->gather.num_split_rows == 0)  // no partial results to keep
    return from_hip(fg::launch_gspmm(gv, plan ? &plan->gather : nullptr, (int)msg, (int)red,
                                     num_heads, head_dim, x_src, edge_val, out, arg_eid,
                                     static_cast<hipStream_t>(stream)));
  const int64_t slots = plan->gather.num_slots;
  if (fg::noalloc_bytes(slots, F, mx) > fg::kNoAllocScratchBytes) return FG_ERR_SCRATCH_LIMIT;
  // the plan's schedule with the fixed scratch in place of its workspace;
  // every slot is written before the merge reads it, so nothing is cleared
  fg::PlanView v = plan->gather;
  v.ws_f = static_cast<float*>(base);
  v.ws_i = mx ? reinterpret_cast<int32_t*>(static_cast<char*>(base) +
                                           fg::noalloc_ids_offset(slots, F))
              : nullptr;
  v.ws_row = nullptr;
  v.ws_width = F;
  return from_hip(fg::launch_gspmm(gv, &v, (int)msg, (int)red, num_heads, head_dim, x_src,
                                   edge_val, out, arg_eid, static_cast<hipStream_t>(stream)));
}

fg_status fg_gsddmm(const fg_graph* g, fg_edge_op op, int32_t num_heads, int64_t head_dim,
                    const float* x_src, const float* x_dst, float* out, fg_plan* plan,
                    void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_width(num_heads, head_dim)) != FG_OK) return st;
  if (op != FG_EDGE_DOT) return FG_ERR_INVALID_ARG;
  const int64_t F = (int64_t)num_heads * head_dim;
  if (g->nnz > 0 && (!x_src || !x_dst || !out)) return FG_ERR_INVALID_ARG;
  if ((st = check_plan(plan, g, F)) != FG_OK) return st;
  const int64_t out_b = nnz_total_of(g) * num_heads * 4;
  if (overlaps(out, out_b, x_src, g->num_cols * F * 4) ||
      overlaps(out, out_b, x_dst, g->num_rows * F * 4))
    return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  // wide rows of a spread graph: the plan's SDDMM schedule, if it has one
  const fg::PlanView* v = nullptr;
  if (plan)
    v = (plan->edge.num_segments > 0 && F >= kEdgeScheduleMinWidth) ? &plan->edge : &plan->gather;
  return from_hip(fg::launch_gsddmm(gv, v, num_heads, head_dim, x_src, x_dst, out,
                                    static_cast<hipStream_t>(stream)));
}

fg_status fg_edge_softmax(const fg_graph* g, int32_t num_heads, const float* scores,
                          int32_t apply_leaky_relu, float negative_slope, float* out,
                          fg_plan* plan, void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if (num_heads < 1 || num_heads > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && (!scores || !out)) return FG_ERR_INVALID_ARG;
  // the plan's softmax workspace holds 2*H floats per slot
  if ((st = check_plan(plan, g, num_heads)) != FG_OK) return st;
  const int64_t b = nnz_total_of(g) * num_heads * 4;
  if (out != scores && overlaps(out, b, scores, b)) return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_edge_softmax(gv, plan ? &plan->plain : nullptr, num_heads, scores,
                                          apply_leaky_relu != 0, negative_slope, out,
                                          static_cast<hipStream_t>(stream)));
}

fg_status fg_gat_aggregate(const fg_graph* g, int32_t num_heads, int64_t head_dim,
                           const float* x_src, const float* x_dst, int32_t apply_leaky_relu,
                           float negative_slope, float* out, fg_plan* plan, void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_width(num_heads, head_dim)) != FG_OK) return st;
  const int64_t F = (int64_t)num_heads * head_dim;
  if (g->num_rows > 0 && !out) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && (!x_src || !x_dst)) return FG_ERR_INVALID_ARG;
  if ((st = check_plan(plan, g, F)) != FG_OK) return st;
  const int64_t out_b = g->num_rows * F * 4;
  if (overlaps(out, out_b, x_src, g->num_cols * F * 4) ||
      overlaps(out, out_b, x_dst, g->num_rows * F * 4))
    return FG_ERR_INVALID_ARG;
  const uintptr_t al = reinterpret_cast<uintptr_t>(x_src) | reinterpret_cast<uintptr_t>(x_dst) |
                       reinterpret_cast<uintptr_t>(out);
  if (!fg::gat_fused_supported(num_heads, head_dim) || (al & 15u) != 0) return FG_ERR_UNSUPPORTED;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_gat_fused(gv, plan ? &plan->gather : nullptr, num_heads, head_dim,
                                       x_src, x_dst, apply_leaky_relu != 0, negative_slope, out,
                                       static_cast<hipStream_t>(stream)));
}

fg_status fg_gsddmm_edge_softmax(const fg_graph* g, int32_t num_heads, int64_t head_dim,
                                 const float* x_src, const float* x_dst, int32_t apply_leaky_relu,
                                 float negative_slope, float* scores, float* out, fg_plan* plan,
                                 void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_width(num_heads, head_dim)) != FG_OK) return st;
  const int64_t F = (int64_t)num_heads * head_dim;
  if (g->nnz > 0 && (!x_src || !x_dst || !scores || !out)) return FG_ERR_INVALID_ARG;
  // the plan holds F partial values per slot (SDDMM) and 2H per slot (softmax)
  if ((st = check_plan(plan, g, std::max<int64_t>(F, num_heads))) != FG_OK) return st;
  const int64_t eb = nnz_total_of(g) * num_heads * 4;
  const int64_t xs_b = g->num_cols * F * 4, xd_b = g->num_rows * F * 4;
  if (overlaps(scores, eb, out, eb) || overlaps(scores, eb, x_src, xs_b) ||
      overlaps(scores, eb, x_dst, xd_b) || overlaps(out, eb, x_src, xs_b) ||
      overlaps(out, eb, x_dst, xd_b))
    return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  hipStream_t hs = static_cast<hipStream_t>(stream);
  // The fused kernel gathers like the SDDMM, so it takes the gather schedule
  // (die-banded on power-law graphs: 3.26 -> 3.06 ms against the plain one).
  // On plans of long items the SDDMM's wide batches and the streaming
  // softmax are faster than its one-value-per-lane passes (2.82 against
  // 3.06 ms on the power-law graph), so those run the two kernels.
  const bool long_items =
      plan && g->nnz >= fg::kWideItemEdges * std::max<int64_t>(plan->gather.num_segments, 1);
  if (!long_items && fg::gsddmm_softmax_fused(num_heads, head_dim, x_src, x_dst))
    return from_hip(fg::launch_gsddmm_softmax(gv, plan ? &plan->gather : nullptr, F, x_src, x_dst,
                                              apply_leaky_relu != 0, negative_slope, scores, out,
                                              hs));
  // long items and other shapes: the two operators one after the other
  hipError_t e = fg::launch_gsddmm(gv, plan ? &plan->gather : nullptr, num_heads, head_dim, x_src,
                                   x_dst, scores, hs);
  if (e != hipSuccess) return FG_ERR_HIP;
  return from_hip(fg::launch_edge_softmax(gv, plan ? &plan->plain : nullptr, num_heads, scores,
                                          apply_leaky_relu != 0, negative_slope, out, hs));
}

fg_status fg_gspmm_max_backward(const fg_graph* g, fg_msg_op msg, int32_t num_heads,
                                int64_t head_dim, const float* x_src, const float* edge_val,
                                const int32_t* arg_eid, const float* grad_out, float* grad_src,
                                float* grad_edge, fg_plan* plan, void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_width(num_heads, head_dim)) != FG_OK) return st;
  if (msg != FG_MSG_COPY_SRC && msg != FG_MSG_SRC_MUL_EDGE) return FG_ERR_INVALID_ARG;
  const bool mul = msg == FG_MSG_SRC_MUL_EDGE;
  if (mul != (edge_val != nullptr)) return FG_ERR_INVALID_ARG;
  if (!mul && grad_edge) return FG_ERR_INVALID_ARG;  // copy_src has no edge values
  if (grad_edge && g->nnz > 0 && !x_src) return FG_ERR_INVALID_ARG;
  if (g->num_rows > 0 && g->nnz > 0 && (grad_src || grad_edge) && (!arg_eid || !grad_out))
    return FG_ERR_INVALID_ARG;
  if ((st = check_plan(plan, g, 1)) != FG_OK) return st;
  if (g->edge_ids && g->nnz > 0 &&
      (!plan || plan->edge_ids != g->edge_ids || plan->nnz_total != nnz_total_of(g)))
    return FG_ERR_INVALID_ARG;  // the plan of this graph holds the id -> position map
  const int64_t F = (int64_t)num_heads * head_dim;
  const int64_t src_b = g->num_cols * F * 4, edge_b = nnz_total_of(g) * num_heads * 4;
  const int64_t row_b = g->num_rows * F * 4;
  for (const auto& o : {std::make_pair((const void*)grad_src, src_b),
                        std::make_pair((const void*)grad_edge, edge_b)}) {
    if (overlaps(o.first, o.second, x_src, src_b) || overlaps(o.first, o.second, edge_val, edge_b) ||
        overlaps(o.first, o.second, arg_eid, row_b) || overlaps(o.first, o.second, grad_out, row_b))
      return FG_ERR_INVALID_ARG;
  }
  if (overlaps(grad_src, src_b, grad_edge, edge_b)) return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_gspmm_max_backward(gv, plan ? plan->eid_pos : nullptr, (int)msg,
                                                num_heads, head_dim, x_src, edge_val, arg_eid,
                                                grad_out, grad_src, grad_edge,
                                                plan ? &plan->bin : nullptr,
                                                static_cast<hipStream_t>(stream)));
}

fg_status fg_edge_softmax_backward(const fg_graph* g, int32_t num_heads, const float* out,
                                   const float* grad_out, const float* scores,
                                   int32_t apply_leaky_relu, float negative_slope,
                                   float* grad_scores, fg_plan* plan, void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if (num_heads < 1 || num_heads > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && (!out || !grad_out || !grad_scores)) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && apply_leaky_relu && !scores) return FG_ERR_INVALID_ARG;
  // the plan's workspace holds H floats per slot
  if ((st = check_plan(plan, g, num_heads)) != FG_OK) return st;
  const int64_t b = nnz_total_of(g) * num_heads * 4;
  if (overlaps(grad_scores, b, out, b) || overlaps(grad_scores, b, apply_leaky_relu ? scores : nullptr, b))
    return FG_ERR_INVALID_ARG;
  if (grad_scores != grad_out && overlaps(grad_scores, b, grad_out, b)) return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_edge_softmax_backward(
      gv, plan ? &plan->plain : nullptr, num_heads, out, grad_out,
      apply_leaky_relu ? scores : nullptr, apply_leaky_relu != 0, negative_slope, grad_scores,
      static_cast<hipStream_t>(stream)));
}

fg_status fg_gsddmm_edge_softmax_backward(const fg_graph* g, int32_t num_heads, int64_t head_dim,
                                          const float* x_src, const float* x_dst,
                                          const float* out, const float* scores,
                                          int32_t apply_leaky_relu, float negative_slope,
                                          float* grad_scores, fg_plan* plan, void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if ((st = check_width(num_heads, head_dim)) != FG_OK) return st;
  const int64_t F = (int64_t)num_heads * head_dim;
  if (g->nnz > 0 && (!x_src || !x_dst || !out || !grad_scores)) return FG_ERR_INVALID_ARG;
  if (g->nnz > 0 && apply_leaky_relu && !scores) return FG_ERR_INVALID_ARG;
  // the SDDMM may run on the gather schedule (F wide) and the softmax
  // backward keeps H floats per slot
  if ((st = check_plan(plan, g, F)) != FG_OK) return st;
  const int64_t b = nnz_total_of(g) * num_heads * 4;
  if (overlaps(grad_scores, b, x_src, g->num_cols * F * 4) ||
      overlaps(grad_scores, b, x_dst, g->num_rows * F * 4) || overlaps(grad_scores, b, out, b) ||
      overlaps(grad_scores, b, apply_leaky_relu ? scores : nullptr, b))
    return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_gsddmm_softmax_backward(
      gv, plan ? &plan->gather : nullptr, plan ? &plan->plain : nullptr, num_heads, head_dim,
      x_src, x_dst, out, apply_leaky_relu ? scores : nullptr, apply_leaky_relu != 0,
      negative_slope, grad_scores, static_cast<hipStream_t>(stream)));
}

fg_status fg_dense_matmul(int64_t n, int64_t d_in, int64_t d_out, const float* x, const float* w,
                          float* y, void* stream) {
  if (n < 0 || n > INT32_MAX || d_in < 1 || d_out < 1 || d_in > FG_MAX_WIDTH ||
      d_out > FG_MAX_WIDTH)
    return FG_ERR_INVALID_ARG;
  if (n > 0 && (!x || !w || !y)) return FG_ERR_INVALID_ARG;
  const int64_t yb = n * d_out * 4;
  if (overlaps(y, yb, x, n * d_in * 4) || overlaps(y, yb, w, d_in * d_out * 4))
    return FG_ERR_INVALID_ARG;
  return from_hip(
      fg::launch_dense_matmul(n, d_in, d_out, x, w, y, static_cast<hipStream_t>(stream)));
}

fg_status fg_mlp_aggregate(const fg_graph* g, int64_t d_in, int64_t d_out, const float* x_src,
                           const float* x_dst, const float* weight, float* out, int32_t* arg_eid,
                           float* workspace, fg_plan* plan, void* stream) {
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if (d_in < 1 || d_out < 1 || d_in > FG_MAX_WIDTH || d_out > FG_MAX_WIDTH)
    return FG_ERR_INVALID_ARG;
  if (g->num_rows > 0 && (!out || !arg_eid)) return FG_ERR_INVALID_ARG;
  if ((g->num_rows > 0 || g->num_cols > 0) && (!x_src || !x_dst || !weight || !workspace))
    return FG_ERR_INVALID_ARG;
  if (x_dst == x_src && g->num_rows != g->num_cols) return FG_ERR_INVALID_ARG;
  if ((st = check_plan(plan, g, d_out)) != FG_OK) return st;
  const int64_t out_b = g->num_rows * d_out * 4;
  const int64_t xs_b = g->num_cols * d_in * 4, xd_b = g->num_rows * d_in * 4;
  const int64_t w_b = d_in * d_out * 4, ws_b = (g->num_cols + g->num_rows) * d_out * 4;
  for (const auto& o : {std::make_pair((const void*)out, out_b),
                        std::make_pair((const void*)arg_eid, out_b),
                        std::make_pair((const void*)workspace, ws_b)}) {
    if (overlaps(o.first, o.second, x_src, xs_b) || overlaps(o.first, o.second, x_dst, xd_b) ||
        overlaps(o.first, o.second, weight, w_b))
      return FG_ERR_INVALID_ARG;
  }
  if (overlaps(out, out_b, arg_eid, out_b) || overlaps(out, out_b, workspace, ws_b) ||
      overlaps(arg_eid, out_b, workspace, ws_b))
    return FG_ERR_INVALID_ARG;
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_mlp_aggregate(gv, plan ? &plan->gather : nullptr, d_in, d_out, x_src,
                                           x_dst, weight, out, arg_eid, workspace,
                                           static_cast<hipStream_t>(stream)));
}

}  // extern "C"
