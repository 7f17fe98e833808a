// Internal interface between the C-ABI layer (fg_api.cpp) and the gfx950
// kernels (fg_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace fg {

// One wavefront work item.  Same layout as fg_segment in the public header.
struct Seg {
  int32_t row, begin, end, slot;
};

// One split row: its partial-result slots are [slot_begin, slot_end).
struct Fix {
  int32_t row, slot_begin, slot_end, pad;
};

// Device view of a plan (all pointers are device memory).
struct PlanView {
  const Seg* segs = nullptr;      // [num_segments]; row == -1 marks an empty (padding) item
  const Fix* fix = nullptr;       // [num_split_rows]
  const int32_t* slot_fix = nullptr;  // [num_slots] -> index into fix
  const int32_t* slot_seg = nullptr;  // [num_slots] -> index into segs
  float* ws_f = nullptr;          // [num_slots * ws_width] partial values
  int32_t* ws_i = nullptr;        // [num_slots * ws_width] partial argmax edge ids
  float* ws_row = nullptr;        // [num_split_rows * ws_width] merged per-row values
  int64_t num_segments = 0, num_split_rows = 0, num_slots = 0;
  int64_t ws_width = 0;           // floats per slot
  // items are ordered longest first with empty rows last: [0, num_long) have
  // more than kShortRowEdges edges, [num_long, num_nonempty) at most that
  // many (whole rows), the rest none (a partitioned schedule sets both to
  // num_segments); [num_medium, num_long) are whole rows of more than
  // kShortRowEdges and at most kMediumRowEdges edges (num_medium == num_long
  // when the order does not guarantee it)
  int64_t num_long = 0, num_nonempty = 0, num_medium = 0;
};

// Rows of at most this many edges are short: the edge softmax packs four of
// them into one wavefront.
constexpr int kShortRowEdges = 64;
// Plans whose items average at least this many edges take the gather
// kernels' wide (256-edge) batches with two lane groups (rows of 65-128
// floats), and the SDDMM + softmax call runs as two kernels there.
constexpr int64_t kWideItemEdges = 128;
// The same for four or more lane groups (rows of at most 64 floats).
constexpr int64_t kWideItemEdgesMany = 64;

// Rows of at most this many edges (and more than kShortRowEdges) also go
// several to a wavefront: four, with float4 lanes.
constexpr int kMediumRowEdges = 256;

struct GraphView {
  int64_t num_rows, num_cols, nnz, nnz_total;
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* edge_ids;
};

enum MsgOp { kCopySrc = 0, kSrcMulEdge = 1 };
enum RedOp { kSum = 0, kMax = 1 };

// Each launcher enqueues its kernels on `stream` and returns the result of
// hipGetLastError() after the last launch.  `plan` may be null (one wavefront
// per row).  Arguments are assumed validated by the caller.
hipError_t launch_gspmm(const GraphView& g, const PlanView* plan, int msg, int red, int64_t H,
                        int64_t dh, const float* x, const float* ev, float* out, int32_t* arg,
                        hipStream_t stream);
hipError_t launch_gsddmm(const GraphView& g, const PlanView* plan, int64_t H, int64_t dh,
                         const float* xs, const float* xd, float* out, hipStream_t stream);
hipError_t launch_edge_softmax(const GraphView& g, const PlanView* plan, int64_t H,
                               const float* scores, bool leaky, float slope, float* out,
                               hipStream_t stream);

// SDDMM dot with one head and the edge softmax of its scores in one pass
// (writes both); covers F % 4 == 0, F <= 1024, 16-byte aligned features.
bool gsddmm_softmax_fused(int64_t H, int64_t dh, const float* xs, const float* xd);
hipError_t launch_gsddmm_softmax(const GraphView& g, const PlanView* plan, int64_t F,
                                 const float* xs, const float* xd, bool leaky, float slope,
                                 float* scores, float* att, hipStream_t stream);

// Binned gSpMM-max backward: a source tile holds 2^logR source rows of F
// floats, at most kBinTileFloats (64 KiB of LDS); at most kMaxBins tiles;
// kBinGroups row groups in the counting and scatter kernels.
constexpr int kBinTileFloats = 16384;
constexpr int kMaxBins = 8192;
constexpr int kBinGroups = 256;

// log2 of the source rows per tile at width F (1 <= F <= kBinTileFloats).
inline int bin_log_rows(int64_t F) {
  int l = 0;
  while (((int64_t)2 << l) * F <= kBinTileFloats) ++l;
  return l;
}

// Tiles needed for num_cols sources at width F.
inline int64_t bin_tiles(int64_t num_cols, int64_t F) {
  const int l = bin_log_rows(F);
  return (num_cols + ((int64_t)1 << l) - 1) >> l;
}

// Its workspace, owned by a plan: 8-byte records (one per gradient element),
// four tables of kMaxBins + 1 int32 (bin sizes, first records, first
// pieces, cursors) and kBinGroups x max_bins int32 (per-group counts).
struct BinWorkspace {
  void* rec = nullptr;
  int64_t rec_capacity = 0;  // records
  int32_t* tables = nullptr;
  int32_t* runs = nullptr;
  int64_t max_bins = 0;
};

// Backward of gSpMM-max: sends each upstream gradient element to the source
// of the edge the forward picked; gsrc / gedge (either may be null) are fully
// overwritten.  With a workspace whose capacity covers rows x F records (and
// widths and source counts its tables fit), grad_src is built by binning the
// elements per source tile and summing each tile in LDS; otherwise, and for
// gedge always, with fp32 atomics into zero-filled arrays.  eid_pos maps
// edge id -> storage position and is used only when g.edge_ids is set.
hipError_t launch_gspmm_max_backward(const GraphView& g, const int32_t* eid_pos, int msg,
                                     int64_t H, int64_t dh, const float* x, const float* ev,
                                     const int32_t* arg, const float* go, float* gsrc,
                                     float* gedge, const BinWorkspace* ws, hipStream_t stream);
// Score gradient of an attention layer: SDDMM x_src . x_dst per head, then
// the edge-softmax backward of its results, written to ds.  One fused kernel
// on the plain schedule when it cuts no row (2 <= H <= 16, dh in {16, 32,
// 64}, H * dh <= 256, aligned features); otherwise the two operators (the
// SDDMM on the gather schedule into ds, then the softmax backward in place).
hipError_t launch_gsddmm_softmax_backward(const GraphView& g, const PlanView* gather,
                                          const PlanView* plain, int64_t H, int64_t dh,
                                          const float* xs, const float* xd, const float* a,
                                          const float* scores, bool leaky, float slope, float* ds,
                                          hipStream_t stream);
// Backward of edge softmax (leaky ReLU optional) on the plain schedule.
hipError_t launch_edge_softmax_backward(const GraphView& g, const PlanView* plan, int64_t H,
                                        const float* a, const float* go, const float* scores,
                                        bool leaky, float slope, float* ds, hipStream_t stream);
// pos[edge_ids[q]] = q for the nnz stored edges, -1 for ids not stored.
hipError_t launch_build_eid_pos(const int32_t* eids, int64_t nnz, int64_t nnz_total, int32_t* pos,
                                hipStream_t stream);

// Y[n, M] = X[n, K] W[K, M] (fp32, matrix cores).
hipError_t launch_dense_matmul(int64_t n, int64_t K, int64_t M, const float* x, const float* w,
                               float* y, hipStream_t stream);
// MLP aggregation: P = X W for sources (and destinations) into ws, then a
// gSpMM with message relu(P_src[u] + P_dst[v]) and max/argmax.
hipError_t launch_mlp_aggregate(const GraphView& g, const PlanView* plan, int64_t d_in,
                                int64_t d_out, const float* xs, const float* xd, const float* w,
                                float* out, int32_t* arg, float* ws, hipStream_t stream);

// Fixed device scratch of the allocation-free gSpMM (fg_gspmm_noalloc): a
// file-scope device array of this many bytes in fg_kernels.hip.  It holds
// the split-row partial values and, for max, their edge ids.
constexpr int64_t kNoAllocScratchBytes = int64_t(32) << 20;

// Byte offset of the edge-id partials in the scratch (after the values,
// rounded up to 256 bytes) and the bytes a schedule with `slots` partial
// slots of F floats needs.
inline int64_t noalloc_ids_offset(int64_t slots, int64_t F) {
  return (slots * F * 4 + 255) / 256 * 256;
}
inline int64_t noalloc_bytes(int64_t slots, int64_t F, bool with_ids) {
  return with_ids ? noalloc_ids_offset(slots, F) + slots * F * 4 : slots * F * 4;
}

// Device address of that array on the current device.  The first call on a
// device looks it up with hipGetSymbolAddress (once per device, under a
// lock); later calls return the kept address.
hipError_t noalloc_scratch(void** ptr);

// Fused SDDMM -> leaky ReLU -> edge softmax -> weighted gSpMM.  Supported
// shapes: dh % 4 == 0, dh / 4 a power of two, H * dh <= 256; aligned inputs.
bool gat_fused_supported(int64_t H, int64_t dh);
hipError_t launch_gat_fused(const GraphView& g, const PlanView* plan, int64_t H, int64_t dh,
                            const float* xs, const float* xd, bool leaky, float slope, float* out,
                            hipStream_t stream);

}  // namespace fg
