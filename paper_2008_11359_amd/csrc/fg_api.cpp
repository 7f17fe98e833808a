// fg_api.cpp -- C ABI of the library: host-side argument checks, the
// degree-aware schedule (plan), and dispatch to the gfx950 kernels.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "featgraph_hip.h"
#include "fg_internal.h"

struct fg_plan {
  int64_t num_rows = 0, nnz = 0, max_width = 0;
  const int32_t* indptr = nullptr;  // device pointer the plan was built for
  int32_t segment_edges = 0, max_row_segments = 0;
  int device = 0;
  fg::PlanView view;
  void* mem[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  int64_t workspace_bytes = 0;
};

namespace {

constexpr int32_t kDefaultSegmentEdges = 4096;
constexpr int32_t kMaxSegmentEdges = 1 << 24;
constexpr int32_t kDefaultMaxRowSegments = 128;
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

bool indptr_valid(const int32_t* ip, int64_t num_rows, int64_t nnz) {
  if (ip[0] != 0 || ip[num_rows] != nnz) return false;
  for (int64_t r = 0; r < num_rows; ++r)
    if (ip[r + 1] < ip[r]) return false;
  return true;
}

// Segment length and count of one row: k = ceil(deg / S) pieces, at most
// `cap`; a row is split when k >= 2.
struct Cut {
  int64_t k;
};

Cut cut_row(int64_t deg, int32_t S, int32_t cap) {
  int64_t k = deg > S ? (deg + S - 1) / S : 1;
  if (k > cap) k = cap;
  return Cut{k};
}

// The schedule.  Order: segments of split rows first, rows with the longest
// segments first (ties by row id), slots numbered in that order so slot ==
// position; then whole rows by decreasing degree (ties by row id); rows
// without edges last.  Long work items start first, which keeps the tail of a
// launch short (longest-processing-time-first list scheduling).
void build_schedule(const int32_t* ip, int64_t num_rows, int32_t S, int32_t cap,
                    std::vector<fg::Seg>& segs, std::vector<fg::Fix>& fix,
                    std::vector<int32_t>& slot_fix) {
  segs.clear();
  fix.clear();
  slot_fix.clear();
  std::vector<int32_t> split, whole, empty;
  for (int64_t r = 0; r < num_rows; ++r) {
    const int64_t deg = (int64_t)ip[r + 1] - ip[r];
    if (deg == 0) empty.push_back((int32_t)r);
    else if (cut_row(deg, S, cap).k >= 2) split.push_back((int32_t)r);
    else whole.push_back((int32_t)r);
  }
  auto deg_of = [ip](int32_t r) { return (int64_t)ip[r + 1] - ip[r]; };
  std::stable_sort(split.begin(), split.end(), [&](int32_t a, int32_t b) {
    const int64_t da = deg_of(a), db = deg_of(b);
    const int64_t ka = cut_row(da, S, cap).k, kb = cut_row(db, S, cap).k;
    return da * kb > db * ka;  // da/ka > db/kb: longer segments first
  });
  std::stable_sort(whole.begin(), whole.end(),
                   [&](int32_t a, int32_t b) { return deg_of(a) > deg_of(b); });
  for (int32_t r : split) {
    const int64_t deg = deg_of(r);
    const int64_t k = cut_row(deg, S, cap).k;
    fg::Fix fx;
    fx.row = r;
    fx.slot_begin = (int32_t)segs.size();
    for (int64_t i = 0; i < k; ++i) {
      fg::Seg s;
      s.row = r;
      s.begin = (int32_t)(ip[r] + deg * i / k);
      s.end = (int32_t)(ip[r] + deg * (i + 1) / k);
      s.slot = (int32_t)segs.size();
      slot_fix.push_back((int32_t)fix.size());
      segs.push_back(s);
    }
    fx.slot_end = (int32_t)segs.size();
    fx.pad = 0;
    fix.push_back(fx);
  }
  segs.reserve(segs.size() + whole.size() + empty.size());
  for (int32_t r : whole) segs.push_back(fg::Seg{r, ip[r], ip[r + 1], -1});
  for (int32_t r : empty) segs.push_back(fg::Seg{r, ip[r], ip[r], -1});
}

fg_status read_options(const fg_plan_options* opt, int32_t* S, int32_t* cap) {
  *S = kDefaultSegmentEdges;
  *cap = kDefaultMaxRowSegments;
  if (!opt) return FG_OK;
  for (int32_t r : opt->reserved)
    if (r != 0) return FG_ERR_INVALID_ARG;
  if (opt->segment_edges < 0 || opt->segment_edges > kMaxSegmentEdges) return FG_ERR_INVALID_ARG;
  if (opt->max_row_segments < 0 || opt->max_row_segments > kMaxRowSegmentsLimit)
    return FG_ERR_INVALID_ARG;
  if (opt->segment_edges) *S = opt->segment_edges;
  if (opt->max_row_segments) *cap = opt->max_row_segments;
  if (*cap < 2) return FG_ERR_INVALID_ARG;
  return FG_OK;
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
  }
  return "unknown status";
}

int32_t fg_abi_version(void) { return FG_ABI_VERSION; }

fg_status fg_schedule_host(const int32_t* indptr_host, int64_t num_rows,
                           const fg_plan_options* opt, fg_segment* segs, int64_t capacity,
                           int64_t* num_segments, int64_t* num_split_rows, int64_t* num_slots) {
  if (!indptr_host || num_rows < 0 || num_rows >= INT32_MAX || capacity < 0)
    return FG_ERR_INVALID_ARG;
  int32_t S, cap;
  fg_status st = read_options(opt, &S, &cap);
  if (st != FG_OK) return st;
  if (!indptr_valid(indptr_host, num_rows, indptr_host[num_rows])) return FG_ERR_INVALID_ARG;
  std::vector<fg::Seg> s;
  std::vector<fg::Fix> fx;
  std::vector<int32_t> sf;
  try {
    build_schedule(indptr_host, num_rows, S, cap, s, fx, sf);
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  if (num_segments) *num_segments = (int64_t)s.size();
  if (num_split_rows) *num_split_rows = (int64_t)fx.size();
  if (num_slots) *num_slots = (int64_t)sf.size();
  if (segs) {
    const int64_t n = std::min<int64_t>(capacity, (int64_t)s.size());
    for (int64_t i = 0; i < n; ++i) {
      segs[i].row = s[i].row;
      segs[i].begin = s[i].begin;
      segs[i].end = s[i].end;
      segs[i].slot = s[i].slot;
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

fg_status fg_plan_create(const fg_graph* g, const int32_t* indptr_host, int64_t max_width,
                         const fg_plan_options* opt, fg_plan** out, void* stream) {
  if (!out) return FG_ERR_INVALID_ARG;
  *out = nullptr;
  fg_status st = check_graph(g);
  if (st != FG_OK) return st;
  if (max_width < 1 || max_width > FG_MAX_WIDTH) return FG_ERR_INVALID_ARG;
  int32_t S, cap;
  if ((st = read_options(opt, &S, &cap)) != FG_OK) return st;
  hipStream_t hs = static_cast<hipStream_t>(stream);

  std::vector<int32_t> ip_copy;
  const int32_t* ip = indptr_host;
  try {
    if (!ip) {
      ip_copy.resize((size_t)g->num_rows + 1);
      if (hipMemcpyAsync(ip_copy.data(), g->indptr, sizeof(int32_t) * ip_copy.size(),
                         hipMemcpyDeviceToHost, hs) != hipSuccess)
        return FG_ERR_HIP;
      if (hipStreamSynchronize(hs) != hipSuccess) return FG_ERR_HIP;
      ip = ip_copy.data();
    }
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  if (!indptr_valid(ip, g->num_rows, g->nnz)) return FG_ERR_INVALID_ARG;

  std::vector<fg::Seg> segs;
  std::vector<fg::Fix> fix;
  std::vector<int32_t> slot_fix;
  fg_plan* p = nullptr;
  try {
    build_schedule(ip, g->num_rows, S, cap, segs, fix, slot_fix);
    p = new fg_plan();
  } catch (const std::bad_alloc&) {
    return FG_ERR_NO_MEMORY;
  }
  p->num_rows = g->num_rows;
  p->nnz = g->nnz;
  p->max_width = max_width;
  p->indptr = g->indptr;
  p->segment_edges = S;
  p->max_row_segments = cap;
  if (hipGetDevice(&p->device) != hipSuccess) {
    delete p;
    return FG_ERR_HIP;
  }
  const int64_t nslots = (int64_t)slot_fix.size();
  // workspace per slot: F partial values (sum / max) or 2*H softmax pairs
  const int64_t ws_width = 2 * max_width;
  const int64_t nsplit = (int64_t)fix.size();
  const size_t bytes[6] = {
      sizeof(fg::Seg) * std::max<size_t>(segs.size(), 1),
      sizeof(fg::Fix) * std::max<size_t>(fix.size(), 1),
      sizeof(int32_t) * std::max<size_t>(slot_fix.size(), 1),
      sizeof(float) * (size_t)std::max<int64_t>(nslots * ws_width, 1),
      sizeof(int32_t) * (size_t)std::max<int64_t>(nslots * max_width, 1),
      sizeof(float) * (size_t)std::max<int64_t>(nsplit * ws_width, 1),
  };
  for (int i = 0; i < 6; ++i) {
    if (hipMalloc(&p->mem[i], bytes[i]) != hipSuccess) {
      p->mem[i] = nullptr;
      fg_plan_destroy(p);
      return FG_ERR_NO_MEMORY;
    }
  }
  hipError_t e = hipSuccess;
  if (!segs.empty())
    e = hipMemcpyAsync(p->mem[0], segs.data(), sizeof(fg::Seg) * segs.size(),
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && !fix.empty())
    e = hipMemcpyAsync(p->mem[1], fix.data(), sizeof(fg::Fix) * fix.size(),
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && !slot_fix.empty())
    e = hipMemcpyAsync(p->mem[2], slot_fix.data(), sizeof(int32_t) * slot_fix.size(),
                       hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);  // host vectors die on return
  if (e != hipSuccess) {
    fg_plan_destroy(p);
    return FG_ERR_HIP;
  }
  p->view.segs = static_cast<const fg::Seg*>(p->mem[0]);
  p->view.fix = static_cast<const fg::Fix*>(p->mem[1]);
  p->view.slot_fix = static_cast<const int32_t*>(p->mem[2]);
  p->view.ws_f = static_cast<float*>(p->mem[3]);
  p->view.ws_i = static_cast<int32_t*>(p->mem[4]);
  p->view.ws_row = static_cast<float*>(p->mem[5]);
  p->view.num_segments = (int64_t)segs.size();
  p->view.num_split_rows = (int64_t)fix.size();
  p->view.num_slots = nslots;
  p->view.ws_width = ws_width;
  p->workspace_bytes = (int64_t)(bytes[3] + bytes[4] + bytes[5]);
  *out = p;
  return FG_OK;
}

fg_status fg_plan_get_info(const fg_plan* plan, fg_plan_info* info) {
  if (!plan || !info) return FG_ERR_INVALID_ARG;
  std::memset(info, 0, sizeof(*info));
  info->num_rows = plan->num_rows;
  info->nnz = plan->nnz;
  info->num_segments = plan->view.num_segments;
  info->num_split_rows = plan->view.num_split_rows;
  info->num_slots = plan->view.num_slots;
  info->max_width = plan->max_width;
  info->workspace_bytes = plan->workspace_bytes;
  info->segment_edges = plan->segment_edges;
  info->max_row_segments = plan->max_row_segments;
  return FG_OK;
}

fg_status fg_gspmm(const fg_graph* g, fg_msg_op msg, fg_reduce_op red, int32_t num_heads,
                   int64_t head_dim, const float* x_src, const float* edge_val, float* out,
                   int32_t* arg_eid, fg_plan* plan, void* stream) {
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
  const fg::GraphView gv = view_of(g);
  return from_hip(fg::launch_gspmm(gv, plan ? &plan->view : nullptr, (int)msg, (int)red,
                                   num_heads, head_dim, x_src, edge_val, out, arg_eid,
                                   static_cast<hipStream_t>(stream)));
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
  return from_hip(fg::launch_gsddmm(gv, plan ? &plan->view : nullptr, num_heads, head_dim, x_src,
                                    x_dst, out, static_cast<hipStream_t>(stream)));
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
  return from_hip(fg::launch_edge_softmax(gv, plan ? &plan->view : nullptr, num_heads, scores,
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
  return from_hip(fg::launch_gat_fused(gv, plan ? &plan->view : nullptr, num_heads, head_dim,
                                       x_src, x_dst, apply_leaky_relu != 0, negative_slope, out,
                                       static_cast<hipStream_t>(stream)));
}

}  // extern "C"
