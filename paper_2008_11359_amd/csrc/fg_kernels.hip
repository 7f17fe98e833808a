// fg_kernels.hip -- gfx950 kernels for FeatGraph's generalized SpMM,
// generalized SDDMM and edge softmax.
//
// Work decomposition (all kernels): one 64-lane wavefront per work item, four
// wavefronts per workgroup.  A work item is either a whole CSR row (no plan)
// or a segment of a row taken from the plan's degree-aware schedule.  The
// feature dimension is spread across lanes (the paper binds it to threads,
// Sec. III-B GPU FDS and Sec. III-C vertex parallelization) with float4
// accesses: G lanes cover one feature row (G*4 floats per pass), so one row of
// 128 floats is one 512-byte request of 32 lanes and a wavefront works on
// 64/G edges at once.  Neighbour indices (and edge values) of up to 64 edges
// are fetched with one coalesced load per lane and handed to the lane groups
// with scalar readlanes (one or two groups) or cross-lane permutes.  SDDMM dot
// products reduce across the lanes of a feature row with DPP row operations
// (the paper's tree reduction, Fig. 4 FDS), never through memory.  No atomics:
// split rows write partial results that a second kernel merges in a fixed
// order, so every result is deterministic for a given plan.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "fg_internal.h"

namespace fg {
namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;

// Work item of the calling wavefront, as a wave-uniform (scalar) value.
__device__ __forceinline__ int64_t wave_item() {
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  return (int64_t)blockIdx.x * kWavesPerBlock + w;
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Compile-time flag passed to generic lambdas (decltype(tag)::value).
template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};

// Offset of source row `src` in a [rows, F] array.  Both factors are
// non-negative and below 2^32 (src < 2^31, F <= 65536), so one unsigned
// 32 x 32 -> 64-bit multiply replaces the signed 64-bit product, which costs
// two 32-bit multiplies, a 64-bit multiply-add and a sign extension (the
// gather kernels are partly bound by vector instruction issue).
__device__ __forceinline__ uint64_t row_off(int32_t src, int64_t F) {
  return (uint64_t)(uint32_t)src * (uint32_t)F;
}

// The same for a lane's element pointer xl (the array plus the lane's
// element offset) and the row size in bytes (F * 4 <= 2^18): one unsigned
// 32 x 32 + 64-bit multiply-add per gather, where p + row_off(src, F) + f
// takes a multiply, a shift and a 64-bit add.
__device__ __forceinline__ const float* row_at(const char* xl, int32_t src, uint32_t rb) {
  return reinterpret_cast<const float*>(xl + (uint64_t)(uint32_t)src * rb);
}

template <int VEC>
__device__ __forceinline__ void load_vec(const float* p, float (&r)[VEC]) {
  if constexpr (VEC == 4) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    r[0] = t.x; r[1] = t.y; r[2] = t.z; r[3] = t.w;
  } else {
    r[0] = *p;
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float* p, const float (&r)[VEC]) {
  if constexpr (VEC == 4) {
    *reinterpret_cast<float4*>(p) = make_float4(r[0], r[1], r[2], r[3]);
  } else {
    *p = r[0];
  }
}

// Non-temporal forms for results no later step of the kernel reads: they
// should not displace the gathered rows from the L2.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

template <int VEC>
__device__ __forceinline__ void store_vec_nt(float* p, const float (&r)[VEC]) {
  if constexpr (VEC == 4) {
    __builtin_nontemporal_store(f32x4{r[0], r[1], r[2], r[3]}, reinterpret_cast<f32x4*>(p));
  } else {
    __builtin_nontemporal_store(r[0], p);
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec_i_nt(int32_t* p, const int32_t (&r)[VEC]) {
  if constexpr (VEC == 4) {
    __builtin_nontemporal_store(i32x4{r[0], r[1], r[2], r[3]}, reinterpret_cast<i32x4*>(p));
  } else {
    __builtin_nontemporal_store(r[0], p);
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec_i(int32_t* p, const int32_t (&r)[VEC]) {
  if constexpr (VEC == 4) {
    *reinterpret_cast<int4*>(p) = make_int4(r[0], r[1], r[2], r[3]);
  } else {
    *p = r[0];
  }
}

// (value, edge id) order of the max reducer: larger value wins, equal values
// (IEEE ==, so -0 == +0) go to the smaller edge id.
__device__ __forceinline__ bool takes_over(float m, int32_t e, float best, int32_t best_e) {
  return m > best || (m == best && e < best_e);
}

// A NaN message competes as -inf: it never beats a number, and a row whose
// messages are all NaN or -inf reports -inf with its smallest edge id.  (The
// positional-id comparison "strictly greater replaces" behaves so by itself.)
__device__ __forceinline__ float max_key(float m) { return m != m ? -INFINITY : m; }

// ---- cross-lane primitives --------------------------------------------------

// DPP controls (GFX9 encoding, valid on gfx950).
constexpr int kDppQuadXor1 = 0xB1;      // quad_perm:[1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;      // quad_perm:[2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowBcast15 = 0x142;   // lane 15 of each row -> next row
constexpr int kDppRowBcast31 = 0x143;   // lane 31 -> rows 2 and 3

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false));
}

// Sum over aligned groups of W lanes (W a power of two <= 64).  The total is
// valid in lane W-1 of every group; for W <= 16 in every lane of the group.
// Every lane of the wavefront must execute this.
template <int W>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (W >= 2) v += dpp_f<kDppQuadXor1>(v);
  if constexpr (W >= 4) v += dpp_f<kDppQuadXor2>(v);
  if constexpr (W >= 8) v += dpp_f<kDppRowHalfMirror>(v);
  if constexpr (W >= 16) v += dpp_f<kDppRowMirror>(v);
  if constexpr (W >= 32) v += dpp_f<kDppRowBcast15, 0xA>(v);
  if constexpr (W >= 64) v += dpp_f<kDppRowBcast31, 0x8>(v);
  return v;
}

// Value of lane (jb + gid) where jb is wave-uniform and gid < NG is the lane
// group of the caller.  One or two groups use scalar readlanes.
template <int NG>
__device__ __forceinline__ int bcast_lane(int v, int jb, int gid) {
  if constexpr (NG == 1) {
    return __builtin_amdgcn_readlane(v, jb);
  } else if constexpr (NG == 2) {
    const int a = __builtin_amdgcn_readlane(v, jb);
    const int b = __builtin_amdgcn_readlane(v, jb + 1);
    return gid ? b : a;
  } else {
    return __shfl(v, jb + gid);
  }
}

template <int NG>
__device__ __forceinline__ float bcast_lane_f(float v, int jb, int gid) {
  return __builtin_bit_cast(float, bcast_lane<NG>(__builtin_bit_cast(int, v), jb, gid));
}

// Wide batches of Q * 64 edges (gather kernels on long items): lane l holds
// edges Q*l .. Q*l + Q - 1 of the batch (Q = 4 when a step covers whole
// lanes, else 1), so the ids of 256 edges arrive in one 16-byte load per lane
// (and the SDDMM's results leave in one 16-byte store): the address unit that
// bounds the gather kernels spends one instruction on each instead of four,
// and an item of up to 256 edges waits for one id load instead of several.
template <int NG, int U>
constexpr int ids_per_lane() { return (NG * U) % 4 == 0 && (NG == 1 || U % 4 == 0) ? 4 : 1; }

// Average item length from which wide batches pay: two lane groups (rows of
// 65-128 floats) gain from the quarter of the id loads on long items only;
// four or more groups (narrower rows, where a step of U edges per group
// spans 64 or more edges) also gain from waiting for one id load per item.
template <int NG>
constexpr int64_t wide_item_edges() { return NG >= 4 ? kWideItemEdgesMany : kWideItemEdges; }


template <int Q, typename T>
__device__ __forceinline__ T pick(const T (&v)[Q], int c) {
  if constexpr (Q == 1) {
    return v[0];
  } else {
    return c == 0 ? v[0] : c == 1 ? v[1] : c == 2 ? v[2] : v[3];
  }
}

typedef int32_t int4_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef float float4_a4 __attribute__((ext_vector_type(4), aligned(4)));


// Edges base + Q*lane + q (q < Q) of a batch of `cnt` edges from a streamed
// int32 array of `len` elements (non-temporal); 0 past cnt.  A lane with
// edges in the batch takes its Q with one 16-byte load (4-byte aligned:
// gfx950 loads it unaligned) when they lie inside the array, else (only at
// its very end) one by one, so nothing past the array is read.
template <int Q>
__device__ __forceinline__ void load_ids(const int32_t* ptr, int64_t len, int64_t base, int lane,
                                         int cnt, int32_t (&out)[Q]) {
  const int k0 = lane * Q;
#pragma unroll
  for (int q = 0; q < Q; ++q) out[q] = 0;
  if (k0 >= cnt) return;
  if constexpr (Q == 1) {
    out[0] = __builtin_nontemporal_load(ptr + base + k0);
  } else if (base + k0 + Q <= len) {
    const int4_a4 v = __builtin_nontemporal_load(reinterpret_cast<const int4_a4*>(ptr + base + k0));
    out[0] = v.x;
    out[1] = k0 + 1 < cnt ? v.y : 0;
    out[2] = k0 + 2 < cnt ? v.z : 0;
    out[3] = k0 + 3 < cnt ? v.w : 0;
  } else {
#pragma unroll
    for (int q = 0; q < Q; ++q)
      if (k0 + q < cnt) out[q] = __builtin_nontemporal_load(ptr + base + k0 + q);
  }
}

// Value of edge (jb + gid) of the batch (jb wave-uniform, gid < NG the
// caller's lane group) when each lane holds Q consecutive edges; jb % Q is
// c0, known after unrolling.  One group reads its id into a scalar
// register; two groups take theirs through one cross-lane permute (the
// vector unit, which partly bounds the gather kernels, then only forms the
// lane index).  Several groups with four ids per lane use the LDS table below.
template <int NG, int Q>
__device__ __forceinline__ int bcast_q(const int32_t (&v)[Q], int jb, int c0, int gid) {
  if constexpr (NG == 1) {
    return __builtin_amdgcn_readlane(pick<Q>(v, c0), jb / Q);
  } else {
    static_assert(Q == 1, "four ids per lane: one group, or the LDS table for two");
    if constexpr (NG == 2) return __shfl(v[0], jb + gid);
    else return bcast_lane<NG>(v[0], jb, gid);
  }
}

// Wide batches of NG >= 2 lane groups keep their 256 ids (or weights) in a
// per-wavefront LDS table, group by group: edge k of the batch at
// (k % NG) * wide_half<NG>() + k / NG, so that group g's edges of a step
// (j0 + NG u + g, u < U) are U consecutive entries, read with U / 4 16-byte
// LDS reads instead of one cross-lane permute (and a select) per edge.  The
// 4-entry pad after each group's 256 / NG entries puts the groups' reads of
// one step in different banks.
template <int NG>
constexpr int wide_half() { return 4 * kWave / NG + 4; }
template <int NG>
constexpr int wide_tab() { return NG * wide_half<NG>(); }

// Lane l holds edges 4l .. 4l + 3 of the batch.  Two groups: 4l and 4l + 2
// go to group 0's entries 2l and 2l + 1, 4l + 1 and 4l + 3 to group 1's.
// NG = 4m groups: edge 4l + q goes to group 4 (l % m) + q, entry l / m.
template <int NG, typename T>
__device__ __forceinline__ void wide_put(T* tab, int lane, const int32_t (&q)[4]) {
  static_assert(sizeof(T) == 4, "4-byte entries");
  static_assert(NG == 2 || NG % 4 == 0, "two lane groups or a multiple of four");
  int32_t* t = reinterpret_cast<int32_t*>(tab);
  constexpr int H = wide_half<NG>();
  if constexpr (NG == 2) {
    *reinterpret_cast<int2*>(t + 2 * lane) = make_int2(q[0], q[2]);
    *reinterpret_cast<int2*>(t + H + 2 * lane) = make_int2(q[1], q[3]);
  } else {
    constexpr int M = NG / 4;
    const int g0 = 4 * (lane % M), pos = lane / M;
#pragma unroll
    for (int c = 0; c < 4; ++c) t[(g0 + c) * H + pos] = q[c];
  }
}

// Group gid's U entries of the step that starts at batch edge j0 (a multiple
// of NG U, so the reads are 16-byte aligned).
template <int NG, int U, typename T>
__device__ __forceinline__ void wide_get(const T* tab, int gid, int j0, T (&out)[U]) {
  static_assert(U % 4 == 0, "whole 16-byte reads");
  const T* t = tab + gid * wide_half<NG>() + j0 / NG;
#pragma unroll
  for (int k = 0; k < U; k += 4) {
    typedef T T4 __attribute__((ext_vector_type(4)));
    const T4 v = *reinterpret_cast<const T4*>(t + k);
    out[k] = v.x;
    out[k + 1] = v.y;
    out[k + 2] = v.z;
    out[k + 3] = v.w;
  }
}

// ----------------------------------------------------------------------------
// generalized SpMM
// ----------------------------------------------------------------------------

struct SpmmParams {
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* eids;
  const float* x;
  const float* ev;
  const float* xd;  // destination features of the u_add_v message (ADD kernels only)
  float* out;
  int32_t* arg;
  const Seg* segs;
  float* ws_f;
  int32_t* ws_i;
  int64_t n_items;
  int64_t nnz;      // length of indices (and of ev with one head and positional ids)
  int64_t F;
  int32_t H;
  int32_t dh;
  int32_t logG;     // runtime group width (generic kernel only)
  int32_t ev_vec4;  // edge-value rows are 16-byte aligned float4s (H % 4 == 0)
};

// Largest head count whose per-batch edge values a wavefront stages in LDS.
constexpr int kTabHeads = 16;

// Orders one wavefront's LDS accesses around a cross-lane hand-off (the
// hardware executes a wavefront's LDS operations in order; the fences keep
// the compiler from moving accesses across).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct Item {
  int64_t row, b, e;
  int32_t slot;
};

template <bool SEG>
__device__ __forceinline__ Item load_item(const Seg* segs, const int32_t* indptr, int64_t item) {
  Item it;
  if constexpr (SEG) {
    const Seg s = segs[item];
    it.row = s.row; it.b = s.begin; it.e = s.end; it.slot = s.slot;
  } else {
    it.row = item; it.b = indptr[item]; it.e = indptr[item + 1]; it.slot = -1;
  }
  return it;
}

// Epilogues of the u_add_v max (MLP aggregation).  Its edges are compared by
// their transformed source value P_src[u] (raw: before adding P_dst[v]); fp32
// rounding of a sum is monotone in each operand, so the edge with the largest
// raw value also has the largest rounded message relu(P_src[u] + P_dst[v]),
// and the row's output is relu(acc + xd[v]).  When that is not positive every
// message is 0 and the row's smallest edge id is reported.
//  kEpiFirst  (positional edge ids): acc / am are the max and smallest argmax
//             of the raw values; the smallest id of the row is its first
//             position.
//  kEpiMasked (any edge ids): edges whose rounded sum is not positive compete
//             as -inf, so am already is the smallest id of the row when
//             nothing is positive.
constexpr int kEpiNone = 0, kEpiFirst = 1, kEpiMasked = 2;

// Writes one lane's accumulated vector: to the plan workspace for a split
// row's segment, else to the output (max: empty -> 0 / -1; EPI: see above).
template <int VEC, bool MAX, bool SEG, int EPI = kEpiNone>
__device__ __forceinline__ void spmm_store(const SpmmParams& p, const Item& it, int64_t f,
                                           const float (&acc)[VEC], const int32_t (&am)[VEC]) {
  if (SEG && it.slot >= 0) {
    store_vec_nt<VEC>(p.ws_f + (int64_t)it.slot * p.F + f, acc);
    if constexpr (MAX) store_vec_i_nt<VEC>(p.ws_i + (int64_t)it.slot * p.F + f, am);
  } else if constexpr (MAX) {
    float o[VEC];
    int32_t a[VEC];
    float pdv[VEC];
    if constexpr (EPI != kEpiNone) load_vec<VEC>(p.xd + it.row * p.F + f, pdv);
#pragma unroll
    for (int c = 0; c < VEC; ++c) {
      const bool none = am[c] == INT_MAX;
      if constexpr (EPI != kEpiNone) {
        const float t = acc[c] + pdv[c];
        const bool pos = t > 0.0f;
        o[c] = (none || !pos) ? 0.0f : t;
        a[c] = none ? -1 : ((pos || EPI == kEpiMasked) ? am[c] : (int32_t)it.b);
      } else {
        o[c] = none ? 0.0f : acc[c];
        a[c] = none ? -1 : am[c];
      }
    }
    store_vec_nt<VEC>(p.out + it.row * p.F + f, o);
    store_vec_i_nt<VEC>(p.arg + it.row * p.F + f, a);
  } else {
    store_vec_nt<VEC>(p.out + it.row * p.F + f, acc);
  }
}

// Fast path: float4 lanes, G (compile time) lanes per feature row, NV float4
// per lane per edge (feature chunk G*4*NV = blockIdx.y), U edges in flight per
// lane group, MUL: src_mul_edge, MAX: max/argmax, EIDS: the graph carries an
// edge-id array (else edge id = position), SEG: items from a plan.
//
// Max with positional edge ids: a lane group visits its edges in increasing
// position, hence increasing edge id, so "strictly greater replaces" keeps the
// smallest edge id among equal maxima; a group whose messages were all -inf
// never replaces and takes its first edge afterwards.  Groups, segments and
// slots are then merged with the full (value, edge id) order.
// ADD: the message is relu(x[u] + xd[v]) (MLP aggregation with the dense
// transform applied to the vertices beforehand); requires MAX and !MUL.  Edges
// compete by their raw x[u] (see the epilogues above spmm_store).  With
// positional edge ids the add and relu move to the store (kEpiFirst); with
// explicit edge ids each edge's sum is formed in the loop to mask the edges
// whose message is 0 (kEpiMasked).
// TAB (per-head edge values, 2 <= H <= kTabHeads): each batch of 64 edges
// stages its edge values in an LDS table, a few loads per lane, and every step
// reads its weights from there; loading them per step would add one more
// vector-memory instruction per gather, and the address unit is what bounds
// these kernels.
//
// WIDE (two or more lane groups, positional ids, one head): 256-edge batches
// whose ids (and weights) arrive four per lane in one 16-byte load (a quarter
// of the id loads for the address unit) and go to the group-major LDS table.
// Without weights they are held to 7 wavefronts per SIMD (72 registers): the
// max kernel otherwise takes 85 (5 wavefronts), with no spill either way.
template <int G, int NV, int U, bool MUL, bool MAX, bool EIDS, bool SEG, bool ADD = false,
          bool TAB = false, bool WIDE = false>
__global__ __launch_bounds__(kBlock, (WIDE && !MUL) ? 7 : 1) void spmm_fast_kernel(SpmmParams p) {
  constexpr int NG = kWave / G;
  constexpr bool POS = MAX && !EIDS;
  static_assert(NG * U <= kWave, "one batch of 64 edges must cover whole steps");
  static_assert(!WIDE || (NG >= 2 && U % 4 == 0 && !EIDS && !TAB),
                "wide batches serve several lane groups with positional ids");
  constexpr int BATCH = WIDE ? 4 * kWave : kWave;
  constexpr int WT = WIDE ? wide_tab<NG>() : 1;
  __shared__ __align__(16) int32_t wid_all[WIDE ? kWavesPerBlock * WT : 1];
  __shared__ __align__(16) float wwt_all[WIDE && MUL ? kWavesPerBlock * WT : 1];
  int32_t* wid = wid_all + (WIDE ? (threadIdx.x >> 6) * WT : 0);
  float* wwt = wwt_all + (WIDE && MUL ? (threadIdx.x >> 6) * WT : 0);
  static_assert(!ADD || (MAX && !MUL), "u_add_v messages are max-reduced copies");
  static_assert(!TAB || MUL, "the table holds edge values");
  constexpr bool EPI = ADD && POS;
  constexpr bool ELEM = ADD && !POS;
  constexpr int EPK = EPI ? kEpiFirst : (ELEM ? kEpiMasked : kEpiNone);
  __shared__ __align__(16) float tab_all[TAB ? kWavesPerBlock * kWave * kTabHeads : 1];
  float* tab = tab_all + (TAB ? (threadIdx.x >> 6) * kWave * kTabHeads : 0);
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  const int lane = lane_id();
  const int gid = lane / G;
  const int li = lane % G;
  const int64_t F = p.F;
  const int64_t c0 = (int64_t)blockIdx.y * (G * 4 * NV);

  int64_t f[NV];
  bool act[NV];
  int hv[NV];
  const char* xl[NV];  // this lane's elements of source row 0
  const uint32_t rb = (uint32_t)F * 4u;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = c0 + (int64_t)(v * G + li) * 4;
    act[v] = f[v] < F;
    hv[v] = (MUL && act[v]) ? (int)(f[v] / p.dh) : 0;
    xl[v] = reinterpret_cast<const char*>(p.x) + f[v] * 4;
  }
  float acc[NV][4];
  int32_t am[NV][4];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      acc[v][c] = MAX ? -INFINITY : 0.0f;
      am[v][c] = INT_MAX;
    }
  float pd[NV][4];  // this row's destination features (per-element messages)
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    if (ELEM && act[v]) {
      load_vec<4>(p.xd + it.row * F + f[v], pd[v]);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) pd[v][c] = 0.0f;
    }
  }

  // TAB with edge ids: the edge values of batch k+1 are fetched into
  // registers while batch k computes (ids two batches ahead)
  constexpr bool PIPE = TAB && EIDS;
  float qn[PIPE ? kTabHeads : 1];
  int eid_n1 = 0, eid_n2 = 0;  // edge ids of the next batch and the one after
  // The table's loads: with 4, 8 or 16 heads (16-byte aligned rows) lpe =
  // H / 4 lanes share an edge, one float4 each, so that an instruction reads
  // 64 / lpe whole edge rows (one 64-byte cache tag each for 8 heads) rather
  // than one float4 of 64 different edges; load i of a lane holds part
  // lane % lpe of edge i * 64 / lpe + lane / lpe.
  const int lpe = (TAB && p.ev_vec4 && (p.H == 4 || p.H == 8 || p.H == 16)) ? p.H >> 2 : 0;
  const int lpe_part = lpe ? lane % lpe : 0;
  const int lpe_sub = lpe ? lane / lpe : 0;
  auto fetch_ids = [&](int64_t b0, int& e) {
    e = 0;
    const int c = (int)min((int64_t)kWave, it.e - b0);
    if (b0 < it.e && lane < c) e = __builtin_nontemporal_load(p.eids + b0 + lane);
  };
  auto fetch_vals = [&](int64_t b0, int e) {
    const int c = (int)min((int64_t)kWave, it.e - b0);
    if (lpe) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < lpe) {
          const int k = i * (kWave / lpe) + lpe_sub;
          const int ek = __shfl(e, k);
          if (b0 < it.e && k < c) {
            float q4[4];
            load_vec<4>(p.ev + (int64_t)ek * p.H + lpe_part * 4, q4);
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4) qn[4 * i + c4] = q4[c4];
          }
        }
      return;
    }
    if (b0 < it.e && lane < c) {
      const float* er = p.ev + (int64_t)e * p.H;
#pragma unroll
      for (int h = 0; h < kTabHeads; h += 4)
        if (h < p.H) {
          if (p.ev_vec4) {
            float q4[4];
            load_vec<4>(er + h, q4);
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4) qn[h + c4] = q4[c4];
          } else {
#pragma unroll
            for (int c4 = 0; c4 < 4; ++c4)
              if (h + c4 < p.H) qn[h + c4] = er[h + c4];
          }
        }
    }
  };
  if constexpr (PIPE) {
    fetch_ids(it.b, eid_n1);
    fetch_vals(it.b, eid_n1);
    fetch_ids(it.b + kWave, eid_n2);
  }
  for (int64_t base = it.b; base < it.e; base += BATCH) {
    const int cnt = (int)min((int64_t)BATCH, it.e - base);
    int my_src = 0, my_eid = 0;
    float my_w = 0.0f;
    if constexpr (WIDE) {
      int32_t qs[4], qw[4];
      load_ids<4>(p.indices, p.nnz, base, lane, cnt, qs);
      if constexpr (MUL)  // the weights' bits (0.0f past the batch)
        load_ids<4>(reinterpret_cast<const int32_t*>(p.ev), p.nnz, base, lane, cnt, qw);
      wave_lds_sync();  // the previous batch's table reads are done
      wide_put<NG>(wid, lane, qs);
      if constexpr (MUL) wide_put<NG>(wwt, lane, qw);
      wave_lds_sync();
    } else if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
      if constexpr (PIPE) my_eid = eid_n1;
      else if constexpr (EIDS) my_eid = __builtin_nontemporal_load(p.eids + base + lane);
      else my_eid = (int)(base + lane);
      if constexpr (MUL) {
        if (p.H == 1) my_w = p.ev[my_eid];
      }
    }
    if constexpr (PIPE) {
      wave_lds_sync();
      if (lpe) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (i < lpe) {
            const int k = i * (kWave / lpe) + lpe_sub;
            if (k < cnt) {
              const float q4[4] = {qn[4 * i], qn[4 * i + 1], qn[4 * i + 2], qn[4 * i + 3]};
              store_vec<4>(tab + k * p.H + lpe_part * 4, q4);
            }
          }
      } else if (lane < cnt) {
        float* tr = tab + lane * p.H;
#pragma unroll
        for (int h = 0; h < kTabHeads; ++h)
          if (h < p.H) tr[h] = qn[h];
      }
      wave_lds_sync();
      eid_n1 = eid_n2;
      fetch_vals(base + kWave, eid_n1);       // next batch's values, in flight during this one
      fetch_ids(base + 2 * kWave, eid_n2);
    } else if constexpr (TAB) {
      wave_lds_sync();  // the previous batch's table reads are done
      if (lpe) {  // positional edge ids (explicit ones take the PIPE path)
        float q4[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = i * (kWave / lpe) + lpe_sub;
          if (i < lpe && k < cnt) load_vec<4>(p.ev + (base + k) * p.H + lpe_part * 4, q4[i]);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = i * (kWave / lpe) + lpe_sub;
          if (i < lpe && k < cnt) store_vec<4>(tab + k * p.H + lpe_part * 4, q4[i]);
        }
      } else if (lane < cnt) {
        const float* er = p.ev + (int64_t)my_eid * p.H;
        float* tr = tab + lane * p.H;
        if (p.ev_vec4) {
          for (int h = 0; h < p.H; h += 4) {
            float q[4];
            load_vec<4>(er + h, q);
            store_vec<4>(tr + h, q);
          }
        } else {
          for (int h = 0; h < p.H; ++h) tr[h] = er[h];
        }
      }
      wave_lds_sync();
    }
    // one step of U edges per lane group; FULL: every edge of the step is in
    // the batch and every feature chunk in the row (no per-edge masking)
    // H1: one head (weights broadcast from the batch; else loaded per edge)
    auto step = [&](int j0, auto full_tag, auto h1_tag) {
      constexpr bool FULL = decltype(full_tag)::value;
      constexpr bool H1 = decltype(h1_tag)::value;
      float val[U][NV][4];
      float wv[U][NV];
      int32_t eu[U];
      bool ok[U];
      // wide batches: this group's U ids (and weights) of the step
      int32_t tsrc[WIDE ? U : 1];
      float tw[WIDE && MUL ? U : 1];
      if constexpr (WIDE) {
        wide_get<NG, U>(wid, gid, j0, tsrc);
        if constexpr (MUL) wide_get<NG, U>(wwt, gid, j0, tw);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jb = j0 + u * NG;
        ok[u] = FULL || jb + gid < cnt;
        int src;
        if constexpr (WIDE) src = tsrc[u];
        else src = __shfl(my_src, jb + gid);
        if constexpr (EIDS) eu[u] = bcast_lane<NG>(my_eid, jb, gid);
        else eu[u] = (int)(base + jb + gid);
        // the weight via the LDS crossbar (one permute) rather than two
        // readlanes and a select on the vector unit
        float w1 = 1.0f;
        if constexpr (MUL && H1) {
          if constexpr (WIDE) w1 = tw[u];
          else w1 = __shfl(my_w, jb + gid);
        }
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if (FULL || (ok[u] && act[v])) {
            load_vec<4>(row_at(xl[v], src, rb), val[u][v]);
            if constexpr (ELEM) {
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                const float t = val[u][v][c] + pd[v][c];
                val[u][v][c] = t > 0.0f ? val[u][v][c] : -INFINITY;
              }
            }
            if constexpr (TAB)
              wv[u][v] = tab[(jb + gid) * p.H + hv[v]];
            else
              wv[u][v] = (MUL && !H1) ? p.ev[(int64_t)eu[u] * p.H + hv[v]] : w1;
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) val[u][v][c] = MAX ? -INFINITY : 0.0f;
            wv[u][v] = 1.0f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            if constexpr (POS) {
              // invalid slots hold -inf with weight 1: never strictly greater
              const float m = MUL ? wv[u][v] * val[u][v][c] : val[u][v][c];
              if (m > acc[v][c]) {
                acc[v][c] = m;
                am[v][c] = eu[u];
              }
            } else if constexpr (MAX) {
              const float m = max_key(MUL ? wv[u][v] * val[u][v][c] : val[u][v][c]);
              if ((FULL || ok[u]) && takes_over(m, eu[u], acc[v][c], am[v][c])) {
                acc[v][c] = m;
                am[v][c] = eu[u];
              }
            } else if constexpr (MUL) {
              acc[v][c] += wv[u][v] * val[u][v][c];
            } else {
              acc[v][c] += val[u][v][c];
            }
          }
    };
    // full steps (wave-uniform test) take the unmasked body
    const bool all_feat = c0 + (int64_t)G * 4 * NV <= F;
    auto steps = [&](auto h1_tag) {
      int j0 = 0;
      if (all_feat)
        for (; j0 + NG * U <= cnt; j0 += NG * U) step(j0, BoolTag<true>{}, h1_tag);
      for (; j0 < cnt; j0 += NG * U) step(j0, BoolTag<false>{}, h1_tag);
    };
    // (without weights, or with a table, the head count plays no part; wide
    // batches are launched for one head only)
    if (!MUL || TAB || WIDE || p.H == 1) steps(BoolTag<true>{});
    else steps(BoolTag<false>{});
  }
  if constexpr (POS) {
    const int64_t first = it.b + gid;  // this group's first edge
    if (first < it.e) {
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (am[v][c] == INT_MAX) am[v][c] = (int32_t)first;
    }
  }

  // merge the lane groups (each holds a strided subset of the edges)
#pragma unroll
  for (int s = G; s < kWave; s <<= 1) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if constexpr (MAX) {
          const float ob = __shfl_xor(acc[v][c], s);
          const int32_t oa = __shfl_xor(am[v][c], s);
          if (takes_over(ob, oa, acc[v][c], am[v][c])) {
            acc[v][c] = ob;
            am[v][c] = oa;
          }
        } else {
          acc[v][c] += __shfl_xor(acc[v][c], s);
        }
      }
  }
  if (gid != 0) return;
#pragma unroll
  for (int v = 0; v < NV; ++v)
    if (act[v]) spmm_store<4, MAX, SEG, EPK>(p, it, f[v], acc[v], am[v]);
}

// Generic path: any width (scalar lanes), runtime group width G = 2^logG.
template <int NV, int U, bool MUL, bool MAX, bool SEG, bool ADD = false>
__global__ __launch_bounds__(kBlock) void spmm_generic_kernel(SpmmParams p) {
  static_assert(!ADD || (MAX && !MUL), "u_add_v messages are max-reduced copies");
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  const int lane = lane_id();
  const int G = 1 << p.logG;
  const int ngroups = kWave >> p.logG;
  const int gid = lane >> p.logG;
  const int li = lane & (G - 1);
  const int64_t F = p.F;
  const int64_t c0 = (int64_t)blockIdx.y * G * NV;

  int64_t f[NV];
  bool act[NV];
  int hv[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = c0 + (int64_t)(v * G + li);
    act[v] = f[v] < F;
    hv[v] = (MUL && act[v]) ? (int)(f[v] / p.dh) : 0;
  }
  float acc[NV][1];
  int32_t am[NV][1];
  float pd[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    acc[v][0] = MAX ? -INFINITY : 0.0f;
    am[v][0] = INT_MAX;
    pd[v] = (ADD && act[v]) ? p.xd[it.row * F + f[v]] : 0.0f;
  }

  for (int64_t base = it.b; base < it.e; base += kWave) {
    const int cnt = (int)min((int64_t)kWave, it.e - base);
    int my_src = 0, my_eid = 0;
    float my_w = 0.0f;
    if (lane < cnt) {
      my_src = p.indices[base + lane];
      if constexpr (MAX || MUL) my_eid = p.eids ? p.eids[base + lane] : (int)(base + lane);
      if constexpr (MUL) {
        if (p.H == 1) my_w = p.ev[my_eid];
      }
    }
    for (int j0 = 0; j0 < cnt; j0 += ngroups * U) {
      float val[U][NV];
      float wv[U][NV];
      int32_t eu[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * ngroups + gid;
        ok[u] = j < cnt;
        const int jl = j & (kWave - 1);
        const int src = __shfl(my_src, jl);
        eu[u] = (MAX || MUL) ? __shfl(my_eid, jl) : 0;
        const float w1 = MUL ? __shfl(my_w, jl) : 1.0f;
        const float* xr = p.x + (int64_t)src * F;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if (ok[u] && act[v]) {
            val[u][v] = xr[f[v]];
            if constexpr (ADD) {  // raw value; edges with a zero message compete as -inf
              const float t = val[u][v] + pd[v];
              val[u][v] = t > 0.0f ? val[u][v] : -INFINITY;
            }
            wv[u][v] = (MUL && p.H != 1) ? p.ev[(int64_t)eu[u] * p.H + hv[v]] : w1;
          } else {
            val[u][v] = MAX ? -INFINITY : 0.0f;
            wv[u][v] = 1.0f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if constexpr (MAX) {
            const float m = max_key(MUL ? wv[u][v] * val[u][v] : val[u][v]);
            if (ok[u] && takes_over(m, eu[u], acc[v][0], am[v][0])) {
              acc[v][0] = m;
              am[v][0] = eu[u];
            }
          } else if constexpr (MUL) {
            acc[v][0] += wv[u][v] * val[u][v];
          } else {
            acc[v][0] += val[u][v];
          }
        }
    }
  }
  for (int s = G; s < kWave; s <<= 1) {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      if constexpr (MAX) {
        const float ob = __shfl_xor(acc[v][0], s);
        const int32_t oa = __shfl_xor(am[v][0], s);
        if (takes_over(ob, oa, acc[v][0], am[v][0])) {
          acc[v][0] = ob;
          am[v][0] = oa;
        }
      } else {
        acc[v][0] += __shfl_xor(acc[v][0], s);
      }
    }
  }
  if (gid != 0) return;
#pragma unroll
  for (int v = 0; v < NV; ++v)
    if (act[v]) spmm_store<1, MAX, SEG, ADD ? kEpiMasked : kEpiNone>(p, it, f[v], acc[v], am[v]);
}

// Merges the partial results of each split row.  Block = 4 wavefronts over a
// tile of 64 feature columns (blockIdx.y); wavefront w takes slots
// sb+w, sb+w+4, ... in increasing order (4 loads in flight), then the four
// wavefront results are combined in order w = 0..3.
// EPI: the partials are raw max / argmax of the source values of a u_add_v
// max (see spmm_store); the merged result gets the same relu epilogue.
template <bool MAX, int EPI = kEpiNone>
__global__ __launch_bounds__(kBlock) void spmm_fixup_kernel(const Fix* fix, const float* ws_f,
                                                            const int32_t* ws_i, int64_t F,
                                                            float* out, int32_t* arg,
                                                            const float* xd,
                                                            const int32_t* indptr) {
  __shared__ float red_v[kWavesPerBlock][kWave];
  __shared__ int32_t red_a[kWavesPerBlock][kWave];
  const int w = threadIdx.x >> 6;
  const int lane = lane_id();
  const int64_t col = (int64_t)blockIdx.y * kWave + lane;
  const bool valid = col < F;
  const Fix fx = fix[blockIdx.x];
  constexpr int kStride = kWavesPerBlock;
  float acc = MAX ? -INFINITY : 0.0f;
  int32_t am = INT_MAX;
  if (valid) {
    for (int s0 = fx.slot_begin + w; s0 < fx.slot_end; s0 += 4 * kStride) {
      float v[4];
      int32_t a[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int s = s0 + k * kStride;
        v[k] = MAX ? -INFINITY : 0.0f;
        a[k] = INT_MAX;
        if (s < fx.slot_end) {
          v[k] = ws_f[(int64_t)s * F + col];
          if constexpr (MAX) a[k] = ws_i[(int64_t)s * F + col];
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (MAX) {
          if (takes_over(v[k], a[k], acc, am)) {
            acc = v[k];
            am = a[k];
          }
        } else {
          acc += v[k];
        }
      }
    }
  }
  red_v[w][lane] = acc;
  red_a[w][lane] = am;
  __syncthreads();
  if (w != 0 || !valid) return;
  acc = red_v[0][lane];
  am = red_a[0][lane];
#pragma unroll
  for (int k = 1; k < kWavesPerBlock; ++k) {
    if constexpr (MAX) {
      if (takes_over(red_v[k][lane], red_a[k][lane], acc, am)) {
        acc = red_v[k][lane];
        am = red_a[k][lane];
      }
    } else {
      acc += red_v[k][lane];
    }
  }
  const int64_t o = (int64_t)fx.row * F + col;
  if constexpr (EPI != kEpiNone) {
    const bool none = am == INT_MAX;
    const float t = acc + xd[o];
    const bool pos = t > 0.0f;
    out[o] = (none || !pos) ? 0.0f : t;
    arg[o] = none ? -1 : ((pos || EPI == kEpiMasked) ? am : indptr[fx.row]);
  } else if constexpr (MAX) {
    const bool none = am == INT_MAX;
    out[o] = none ? 0.0f : acc;
    arg[o] = none ? -1 : am;
  } else {
    out[o] = acc;
  }
}

// The same merge with float4 lanes (F % 4 == 0, 16-byte aligned out / arg):
// a wavefront covers 256 columns, so each slot costs one 1 KiB load per
// wavefront instead of four.  Same slot order and combination order.
template <bool MAX, int EPI = kEpiNone>
__global__ __launch_bounds__(kBlock) void spmm_fixup4_kernel(const Fix* fix, const float* ws_f,
                                                             const int32_t* ws_i, int64_t F,
                                                             float* out, int32_t* arg,
                                                             const float* xd,
                                                             const int32_t* indptr) {
  __shared__ float red_v[kWavesPerBlock][kWave][4];
  __shared__ int32_t red_a[kWavesPerBlock][kWave][4];
  const int w = threadIdx.x >> 6;
  const int lane = lane_id();
  const int64_t col = ((int64_t)blockIdx.y * kWave + lane) * 4;
  const bool valid = col < F;
  const Fix fx = fix[blockIdx.x];
  constexpr int kStride = kWavesPerBlock;
  float acc[4];
  int32_t am[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    acc[c] = MAX ? -INFINITY : 0.0f;
    am[c] = INT_MAX;
  }
  if (valid) {
    for (int s0 = fx.slot_begin + w; s0 < fx.slot_end; s0 += 4 * kStride) {
      float v[4][4];
      int32_t a[4][4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int s = s0 + k * kStride;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          v[k][c] = MAX ? -INFINITY : 0.0f;
          a[k][c] = INT_MAX;
        }
        if (s < fx.slot_end) {
          load_vec<4>(ws_f + (int64_t)s * F + col, v[k]);
          if constexpr (MAX) {
            const int4 t = *reinterpret_cast<const int4*>(ws_i + (int64_t)s * F + col);
            a[k][0] = t.x; a[k][1] = t.y; a[k][2] = t.z; a[k][3] = t.w;
          }
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          if constexpr (MAX) {
            if (takes_over(v[k][c], a[k][c], acc[c], am[c])) {
              acc[c] = v[k][c];
              am[c] = a[k][c];
            }
          } else {
            acc[c] += v[k][c];
          }
        }
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    red_v[w][lane][c] = acc[c];
    red_a[w][lane][c] = am[c];
  }
  __syncthreads();
  if (w != 0 || !valid) return;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    acc[c] = red_v[0][lane][c];
    am[c] = red_a[0][lane][c];
  }
#pragma unroll
  for (int k = 1; k < kWavesPerBlock; ++k)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if constexpr (MAX) {
        if (takes_over(red_v[k][lane][c], red_a[k][lane][c], acc[c], am[c])) {
          acc[c] = red_v[k][lane][c];
          am[c] = red_a[k][lane][c];
        }
      } else {
        acc[c] += red_v[k][lane][c];
      }
    }
  const int64_t o = (int64_t)fx.row * F + col;
  if constexpr (EPI != kEpiNone || MAX) {
    float ov[4];
    int32_t oa[4];
    float xv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (EPI != kEpiNone) load_vec<4>(xd + o, xv);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bool none = am[c] == INT_MAX;
      if constexpr (EPI != kEpiNone) {
        const float t = acc[c] + xv[c];
        const bool pos = t > 0.0f;
        ov[c] = (none || !pos) ? 0.0f : t;
        oa[c] = none ? -1 : ((pos || EPI == kEpiMasked) ? am[c] : indptr[fx.row]);
      } else {
        ov[c] = none ? 0.0f : acc[c];
        oa[c] = none ? -1 : am[c];
      }
    }
    store_vec<4>(out + o, ov);
    store_vec_i<4>(arg + o, oa);
  } else {
    store_vec<4>(out + o, acc);
  }
}

// ----------------------------------------------------------------------------
// generalized SDDMM (dot, per head)
// ----------------------------------------------------------------------------

struct SddmmParams {
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* eids;
  const float* xs;
  const float* xd;
  float* out;
  const Seg* segs;
  int64_t n_items;
  int64_t nnz;  // stored edges: elements of indices and eids
  int64_t F;
  int32_t H;
  int32_t dh;
  int32_t logG;  // lanes per feature row (runtime kernels)
  int32_t logS;  // lanes per head (runtime headed kernel)
  int32_t out_vec4;  // output rows of H values are 16-byte aligned float4s
};

// Single head, float4 lanes, G lanes per feature row, NV float4 per lane.  The
// destination row stays in registers for the whole item; each edge gathers
// its source row, multiplies, and reduces across its G lanes with DPP.
template <int G, int NV, int U, bool SEG, bool WIDE = false>
__global__ __launch_bounds__(kBlock) void sddmm_fast_kernel(SddmmParams p) {
  constexpr int NG = kWave / G;
  static_assert(NG * U <= kWave, "one batch of 64 edges must cover whole steps");
  constexpr int QB = WIDE ? ids_per_lane<NG, U>() : 1;
  // one or two groups, and wide batches, hand each edge's dot product over
  // through this per-wavefront table (the group's last lane writes it; each
  // lane reads its QB results after the batch) instead of readlanes and
  // selects, or a cross-lane permute per step
  constexpr bool RTAB = NG <= 2 || WIDE;
  __shared__ __align__(16) float res_all[RTAB ? kWavesPerBlock * kWave * QB : 1];
  float* res_tab = res_all + (RTAB ? (threadIdx.x >> 6) * kWave * QB : 0);
  // wide batches of several groups take their ids from the group-major table
  constexpr bool IDTAB = WIDE && NG >= 2;
  constexpr int WT = IDTAB ? wide_tab<NG>() : 1;
  __shared__ __align__(16) int32_t sid_all[IDTAB ? kWavesPerBlock * WT : 1];
  int32_t* sid = sid_all + (IDTAB ? (threadIdx.x >> 6) * WT : 0);
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  if (it.b >= it.e) return;
  const int lane = lane_id();
  const int gid = lane / G;
  const int li = lane % G;
  const int64_t F = p.F;

  int64_t f[NV];
  bool act[NV];
  float xd[NV][4];
  const char* xl[NV];  // this lane's elements of source row 0
  const uint32_t rb = (uint32_t)F * 4u;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = (int64_t)(v * G + li) * 4;
    act[v] = f[v] < F;
    xl[v] = reinterpret_cast<const char*>(p.xs) + f[v] * 4;
    if (act[v]) {
      load_vec<4>(p.xd + it.row * F + f[v], xd[v]);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) xd[v][c] = 0.0f;
    }
  }

  const bool all_feat = (int64_t)G * 4 * NV <= F;
  constexpr int Q = WIDE ? ids_per_lane<NG, U>() : 1;
  static_assert((NG * U) % Q == 0, "every step starts on a lane's first edge");
  for (int64_t base = it.b; base < it.e; base += Q * kWave) {
    const int cnt = (int)min((int64_t)(Q * kWave), it.e - base);
    int32_t my_src[Q], my_eid[Q];
    load_ids<Q>(p.indices, p.nnz, base, lane, cnt, my_src);
    if constexpr (IDTAB) {
      wave_lds_sync();  // the previous batch's table reads are done
      wide_put<NG>(sid, lane, my_src);
      wave_lds_sync();
    }
    if (p.eids) {
      load_ids<Q>(p.eids, p.nnz, base, lane, cnt, my_eid);
    } else {
#pragma unroll
      for (int q = 0; q < Q; ++q) my_eid[q] = (int)(base + lane * Q + q);
    }
    // lane j collects the dot products of edges base + Q*j + q, so the batch's
    // results leave in one store instead of one store per step with one lane
    // per group active, which would cost the address unit as much as a
    // gather: one or two groups, and wide batches, hand their sums over
    // through the LDS table, more groups with one cross-lane permute per step
    float res[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) res[q] = 0.0f;
    // one step of U edges per lane group; FULL: every edge of the step is in
    // the batch and every feature chunk in the row (no per-edge masking)
    auto step = [&](int j0, auto full_tag) {
      constexpr bool FULL = decltype(full_tag)::value;
      float val[U][NV][4];
      bool ok[U];
      int32_t tsrc[IDTAB ? U : 1];
      if constexpr (IDTAB) wide_get<NG, U>(sid, gid, j0, tsrc);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jb = j0 + u * NG;
        ok[u] = FULL || jb + gid < cnt;
        int src;
        if constexpr (IDTAB) src = tsrc[u];
        else src = bcast_q<NG, Q>(my_src, jb, (u * NG) % Q, gid);
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if (FULL || (ok[u] && act[v])) {
            load_vec<4>(row_at(xl[v], src, rb), val[u][v]);
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) val[u][v][c] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float part = 0.0f;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int c = 0; c < 4; ++c) part += val[u][v][c] * xd[v][c];
        part = group_sum<G>(part);
        const int jb = j0 + u * NG;
        // the last lane of group g holds the sum of edge jb + g
        if constexpr (RTAB) {
          if (li == G - 1 && (FULL || jb + gid < cnt)) res_tab[jb + gid] = part;
        } else {
          const int rel = lane - jb;
          const bool mine = rel >= 0 && rel < NG && lane < cnt;
          const float got = __shfl(part, mine ? rel * G + (G - 1) : lane);
          if (mine) res[0] = got;  // Q == 1 without the table
        }
      }
    };
    // full steps (wave-uniform test) take the unmasked body
    int j0 = 0;
    if (all_feat)
      for (; j0 + NG * U <= cnt; j0 += NG * U) step(j0, BoolTag<true>{});
    for (; j0 < cnt; j0 += NG * U) step(j0, BoolTag<false>{});
    if constexpr (RTAB) {
      wave_lds_sync();  // the table holds the batch's results
      if constexpr (Q == 4) {
        const float4 t = *reinterpret_cast<const float4*>(res_tab + lane * Q);
        res[0] = t.x;
        res[1] = t.y;
        res[2] = t.z;
        res[3] = t.w;
      } else {
        res[0] = res_tab[lane];
      }
      wave_lds_sync();  // read before the next batch writes
    }
    bool stored = false;
    if constexpr (Q == 4) {
      if (!p.eids && lane * Q + Q <= cnt) {  // four positional results: one 16-byte store
        __builtin_nontemporal_store(float4_a4{res[0], res[1], res[2], res[3]},
                                    reinterpret_cast<float4_a4*>(p.out + base + lane * Q));
        stored = true;
      }
    }
    if (!stored) {
#pragma unroll
      for (int q = 0; q < Q; ++q)
        if (lane * Q + q < cnt) __builtin_nontemporal_store(res[q], p.out + my_eid[q]);
    }
  }
}

// Several heads, float4 lanes, S lanes per head (compile time), G lanes per
// feature row (runtime, <= 64, one float4 per lane).
// Results of a batch are staged per edge in an LDS table (one row of H
// values per edge) and leave in one pass of per-lane stores per batch, when
// H <= kTabHeads; otherwise each step stores its heads directly.
template <int S, bool SEG>
__global__ __launch_bounds__(kBlock) void sddmm_headed_kernel(SddmmParams p) {
  constexpr int U = 4;
  __shared__ __align__(16) float tab_all[kWavesPerBlock * kWave * kTabHeads];
  float* tab = tab_all + (threadIdx.x >> 6) * kWave * kTabHeads;
  const bool staged = p.H <= kTabHeads;
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  if (it.b >= it.e) return;
  const int lane = lane_id();
  const int lpe = (p.out_vec4 && (p.H == 4 || p.H == 8 || p.H == 16)) ? p.H >> 2 : 0;
  const int lpe_part = lpe ? lane % lpe : 0;
  const int lpe_sub = lpe ? lane / lpe : 0;
  const int G = 1 << p.logG;
  const int ngroups = kWave >> p.logG;
  const int gid = lane >> p.logG;
  const int li = lane & (G - 1);
  const int64_t F = p.F;
  const int64_t f = (int64_t)li * 4;
  const bool act = f < F;
  const int64_t h = act ? f / p.dh : 0;
  float xd[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (act) load_vec<4>(p.xd + it.row * F + f, xd);
  const char* xl = reinterpret_cast<const char*>(p.xs) + f * 4;  // lane's elements of row 0
  const uint32_t rb = (uint32_t)F * 4u;

  for (int64_t base = it.b; base < it.e; base += kWave) {
    const int cnt = (int)min((int64_t)kWave, it.e - base);
    int my_src = 0, my_eid = 0;
    if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
      my_eid = p.eids ? __builtin_nontemporal_load(p.eids + base + lane) : (int)(base + lane);
    }
    for (int j0 = 0; j0 < cnt; j0 += ngroups * U) {
      float val[U][4];
      int32_t eu[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * ngroups + gid;
        ok[u] = j < cnt;
        const int jl = j & (kWave - 1);
        const int src = __shfl(my_src, jl);
        eu[u] = __shfl(my_eid, jl);
        if (ok[u] && act) {
          load_vec<4>(row_at(xl, src, rb), val[u]);
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) val[u][c] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float part = 0.0f;
#pragma unroll
        for (int c = 0; c < 4; ++c) part += val[u][c] * xd[c];
        part = group_sum<S>(part);
        if (ok[u] && act && (li % S) == S - 1) {
          if (staged)
            tab[(j0 + u * ngroups + gid) * p.H + h] = part;
          else
            p.out[(int64_t)eu[u] * p.H + h] = part;
        }
      }
    }
    if (staged) {
      wave_lds_sync();
      if (lpe) {
        // lpe = H / 4 lanes share an edge (one float4 each), so that a store
        // instruction writes 64 / lpe whole edge rows
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (i < lpe) {
            const int k = i * (kWave / lpe) + lpe_sub;
            const int ek = __shfl(my_eid, k);
            if (k < cnt) {
              float q[4];
              load_vec<4>(tab + k * p.H + lpe_part * 4, q);
              store_vec<4>(p.out + (int64_t)ek * p.H + lpe_part * 4, q);
            }
          }
      } else if (lane < cnt) {
        const float* tr = tab + lane * p.H;
        float* orow = p.out + (int64_t)my_eid * p.H;
        if (p.out_vec4) {
          for (int hh = 0; hh < p.H; hh += 4) {
            float q[4];
            load_vec<4>(tr + hh, q);
            store_vec<4>(orow + hh, q);
          }
        } else {
          for (int hh = 0; hh < p.H; ++hh) orow[hh] = tr[hh];
        }
      }
      wave_lds_sync();  // the table is rewritten by the next batch
    }
  }
}

// Scalar lanes, runtime widths: G = 2^logG lanes per feature row, NV values
// per lane; when HEADED, 2^logS lanes per head.  Reductions use xor permutes.
template <int NV, int U, bool HEADED, bool SEG>
__global__ __launch_bounds__(kBlock) void sddmm_scalar_kernel(SddmmParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  if (it.b >= it.e) return;
  const int lane = lane_id();
  const int G = 1 << p.logG;
  const int ngroups = kWave >> p.logG;
  const int gid = lane >> p.logG;
  const int li = lane & (G - 1);
  const int S = HEADED ? (1 << p.logS) : G;
  const int64_t F = p.F;

  int64_t f[NV];
  bool act[NV];
  float xd[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = (int64_t)(v * G + li);
    act[v] = f[v] < F;
    xd[v] = act[v] ? p.xd[it.row * F + f[v]] : 0.0f;
  }

  for (int64_t base = it.b; base < it.e; base += kWave) {
    const int cnt = (int)min((int64_t)kWave, it.e - base);
    int my_src = 0, my_eid = 0;
    if (lane < cnt) {
      my_src = p.indices[base + lane];
      my_eid = p.eids ? p.eids[base + lane] : (int)(base + lane);
    }
    for (int j0 = 0; j0 < cnt; j0 += ngroups * U) {
      float val[U][NV];
      int32_t eu[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * ngroups + gid;
        ok[u] = j < cnt;
        const int jl = j & (kWave - 1);
        const int src = __shfl(my_src, jl);
        eu[u] = __shfl(my_eid, jl);
#pragma unroll
        for (int v = 0; v < NV; ++v)
          val[u][v] = (ok[u] && act[v]) ? p.xs[row_off(src, F) + f[v]] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if constexpr (!HEADED) {
          float part = 0.0f;
#pragma unroll
          for (int v = 0; v < NV; ++v) part += val[u][v] * xd[v];
          for (int s = 1; s < G; s <<= 1) part += __shfl_xor(part, s);
          if (ok[u] && li == 0) p.out[eu[u]] = part;
        } else {
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            float part = val[u][v] * xd[v];
            for (int s = 1; s < S; s <<= 1) part += __shfl_xor(part, s);
            if (ok[u] && act[v] && (li & (S - 1)) == 0)
              p.out[(int64_t)eu[u] * p.H + f[v] / p.dh] = part;
          }
        }
      }
    }
  }
}

// Fallback for shapes the lane mappings above do not cover (head sizes that
// are not a power of two lanes, very wide rows): one lane per (edge, head)
// pair, sequential dot product.
template <bool SEG>
__global__ __launch_bounds__(kBlock) void sddmm_generic_kernel(SddmmParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  const int lane = lane_id();
  const int64_t H = p.H, dh = p.dh, F = p.F;
  const int64_t total = (it.e - it.b) * H;
  for (int64_t t = lane; t < total; t += kWave) {
    const int64_t q = it.b + t / H;
    const int64_t h = t % H;
    const int64_t src = p.indices[q];
    const int64_t eid = p.eids ? p.eids[q] : q;
    const float* a = p.xs + src * F + h * dh;
    const float* d = p.xd + it.row * F + h * dh;
    float acc = 0.0f;
    for (int64_t k = 0; k < dh; ++k) acc += a[k] * d[k];
    p.out[eid * H + h] = acc;
  }
}

// ----------------------------------------------------------------------------
// edge softmax (leaky ReLU optional), per destination row and head
// ----------------------------------------------------------------------------

struct SoftmaxParams {
  const int32_t* indptr;
  const int32_t* eids;
  const float* scores;
  float* out;
  const Seg* segs;
  const Fix* fix;
  const int32_t* slot_fix;
  const int32_t* slot_seg;
  float* ws;      // [slot][H][2]  per-segment (max, scaled sum)
  float* ws_row;  // [split row][H][2] merged per row
  int64_t n_items;
  int32_t H;
  int32_t leaky;
  float slope;
  int32_t contig;  // edge id == position, H a power of two <= 64, 16-byte aligned arrays
  int32_t self_merge;  // contig and H == 1: the split kernel merges its row's (m, z) itself
};

__device__ __forceinline__ float leaky_relu(float s, int on, float slope) {
  return (on && !(s > 0.0f)) ? slope * s : s;
}

// e^x for x <= 0 through the hardware 2^x instruction: the rounding of
// x * log2(e) gives a relative error of about |x| * 2^-23 (2e-6 at x = -20,
// below which a term weighs less than 2e-9 of the row's largest), in two
// instructions instead of the ten or so of the correctly rounded expf.  Used
// for the running (max, sum) statistics, the fused attention weights and the
// edge softmax outputs (the softmax is partly bound by vector instruction
// issue; the relative error stays within the 1e-5 * sqrt(degree) tolerance).
__device__ __forceinline__ float exp_nonpos(float x) {
  return __builtin_amdgcn_exp2f(x * 1.44269504088896341f);
}

// (m, z) stands for sum_i exp(x_i - m) = z.  Merging two such pairs.
__device__ __forceinline__ void lse_merge(float& m, float& z, float om, float oz) {
  if (om == -INFINITY) return;
  if (m == -INFINITY) {
    m = om;
    z = oz;
    return;
  }
  const float nm = fmaxf(m, om);
  z = z * exp_nonpos(m - nm) + oz * exp_nonpos(om - nm);
  m = nm;
}

__device__ __forceinline__ void lse_push(float& m, float& z, float s) {
  if (s > m) {
    z = z * exp_nonpos(m - s) + 1.0f;
    m = s;
  } else {
    z += exp_nonpos(s - m);
  }
}

constexpr int kSoftmaxU = 4;  // scores in flight per lane

// Whole row held in registers (H a power of two <= 64, at most 4 values per
// lane): one read of the scores, max and sum by xor butterflies over the lanes
// of a head, one write.
__device__ __forceinline__ void softmax_row_in_registers(const SoftmaxParams& p, const Item& it) {
  const int lane = lane_id();
  const int H = p.H;
  const int epw = kWave / H;
  const int eo = lane / H;
  const int h = lane % H;
  float sv[kSoftmaxU];
  int64_t ev[kSoftmaxU];
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < kSoftmaxU; ++k) {
    const int64_t q = it.b + eo + (int64_t)k * epw;
    ev[k] = -1;
    sv[k] = -INFINITY;
    if (q < it.e) {
      ev[k] = p.eids ? p.eids[q] : q;
      sv[k] = leaky_relu(p.scores[ev[k] * H + h], p.leaky, p.slope);
    }
  }
#pragma unroll
  for (int k = 0; k < kSoftmaxU; ++k) mx = fmaxf(mx, sv[k]);
  for (int off = H; off < kWave; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  float z = 0.0f;
#pragma unroll
  for (int k = 0; k < kSoftmaxU; ++k) {
    sv[k] = ev[k] >= 0 ? exp_nonpos(sv[k] - mx) : 0.0f;
    z += sv[k];
  }
  for (int off = H; off < kWave; off <<= 1) z += __shfl_xor(z, off);
  const float inv = 1.0f / z;
#pragma unroll
  for (int k = 0; k < kSoftmaxU; ++k)
    if (ev[k] >= 0) p.out[ev[k] * H + h] = sv[k] * inv;
}

// ---- contiguous rows: edge id == position, so a row's scores are the flat
// range [b*H, e*H) of the [E, H] array.  Lane l reads float4 number
// k = l + 64 i of the range starting at T0 = (b*H) rounded down to 4; since H
// divides 256, element c of every float4 a lane reads has the same head
// (T0 + 4l + c) mod H.  Partial float4s at the ends (H < 4) use scalar access.

constexpr int kContigRegs = 12;  // float4 per lane held in registers (3072 values)
constexpr int kStreamDepth = 8;  // float4 loads in flight per lane when streaming a row

struct ContigRange {
  int64_t lo, hi, T0, K;  // valid flat range, aligned start, number of float4
};

__device__ __forceinline__ ContigRange contig_range(int64_t b, int64_t e, int H) {
  ContigRange r;
  r.lo = b * H;
  r.hi = e * H;
  r.T0 = r.lo & ~int64_t(3);
  r.K = (r.hi - r.T0 + 3) >> 2;
  return r;
}

// Loads float4 k of the range as stored (a 16-byte load when it lies inside
// the range, else element loads); elements outside the range get -inf.  The
// leaky ReLU is applied apart (contig_leaky), after every load of a batch is
// issued: applied inside the load's branch, it made the compiler wait for
// each load before issuing the next, one load in flight per wavefront.
__device__ __forceinline__ void contig_load(const SoftmaxParams& p, const ContigRange& r,
                                            int64_t k, float (&v)[4]) {
  const int64_t t0 = r.T0 + 4 * k;
  if (t0 >= r.lo && t0 + 4 <= r.hi) {
    load_vec<4>(p.scores + t0, v);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t t = t0 + c;
      v[c] = (t >= r.lo && t < r.hi) ? p.scores[t] : -INFINITY;
    }
  }
}

// Leaky ReLU of the elements of float4 k that lie inside the range.
__device__ __forceinline__ void contig_leaky(const SoftmaxParams& p, const ContigRange& r,
                                             int64_t k, float (&v)[4]) {
  if (!p.leaky) return;
  const int64_t t0 = r.T0 + 4 * k;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int64_t t = t0 + c;
    if (t >= r.lo && t < r.hi) v[c] = leaky_relu(v[c], 1, p.slope);
  }
}

__device__ __forceinline__ void contig_store(const SoftmaxParams& p, const ContigRange& r,
                                             int64_t k, const float (&v)[4]) {
  const int64_t t0 = r.T0 + 4 * k;
  if (t0 >= r.lo && t0 + 4 <= r.hi) {
    store_vec<4>(p.out + t0, v);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t t = t0 + c;
      if (t >= r.lo && t < r.hi) p.out[t] = v[c];
    }
  }
}

// Combines the 4 slots of a lane that hold the same head (H < 4), then the
// lanes that hold the same heads (xor over lane bits >= log2(max(H/4, 1))).
__device__ __forceinline__ void contig_allmax(float (&m)[4], int H) {
  if (H == 1) {
    float t = fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3]));
    for (int off = 1; off < kWave; off <<= 1) t = fmaxf(t, __shfl_xor(t, off));
    m[0] = m[1] = m[2] = m[3] = t;
  } else if (H == 2) {
    float a = fmaxf(m[0], m[2]), b = fmaxf(m[1], m[3]);
    for (int off = 1; off < kWave; off <<= 1) {
      a = fmaxf(a, __shfl_xor(a, off));
      b = fmaxf(b, __shfl_xor(b, off));
    }
    m[0] = m[2] = a;
    m[1] = m[3] = b;
  } else {
    for (int off = H / 4; off < kWave; off <<= 1)
#pragma unroll
      for (int c = 0; c < 4; ++c) m[c] = fmaxf(m[c], __shfl_xor(m[c], off));
  }
}

__device__ __forceinline__ void contig_allsum(float (&z)[4], int H) {
  if (H == 1) {
    float t = (z[0] + z[1]) + (z[2] + z[3]);
    for (int off = 1; off < kWave; off <<= 1) t += __shfl_xor(t, off);
    z[0] = z[1] = z[2] = z[3] = t;
  } else if (H == 2) {
    float a = z[0] + z[2], b = z[1] + z[3];
    for (int off = 1; off < kWave; off <<= 1) {
      a += __shfl_xor(a, off);
      b += __shfl_xor(b, off);
    }
    z[0] = z[2] = a;
    z[1] = z[3] = b;
  } else {
    for (int off = H / 4; off < kWave; off <<= 1)
#pragma unroll
      for (int c = 0; c < 4; ++c) z[c] += __shfl_xor(z[c], off);
  }
}

__device__ __forceinline__ void contig_alllse(float (&m)[4], float (&z)[4], int H) {
  if (H == 1) {
    for (int c = 1; c < 4; ++c) lse_merge(m[0], z[0], m[c], z[c]);
    m[1] = m[2] = m[3] = m[0];
    z[1] = z[2] = z[3] = z[0];
  } else if (H == 2) {
    lse_merge(m[0], z[0], m[2], z[2]);
    lse_merge(m[1], z[1], m[3], z[3]);
    m[2] = m[0]; z[2] = z[0];
    m[3] = m[1]; z[3] = z[1];
  }
  for (int off = H >= 4 ? H / 4 : 1; off < kWave; off <<= 1)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float om = __shfl_xor(m[c], off), oz = __shfl_xor(z[c], off);
      lse_merge(m[c], z[c], om, oz);
    }
}

// Head of slot c of this lane, and whether this lane publishes that head's
// per-segment statistics (one lane per head).
__device__ __forceinline__ int contig_head(const ContigRange& r, int lane, int c, int H) {
  return (int)((r.T0 + 4 * lane + c) % H);
}

// Whole row in registers: exact max, one exp per value, one read, one write.
__device__ __forceinline__ void softmax_contig_regs(const SoftmaxParams& p, const Item& it) {
  const int lane = lane_id();
  const int H = p.H;
  const ContigRange r = contig_range(it.b, it.e, H);
  const int rounds = (int)((r.K + kWave - 1) / kWave);  // wave-uniform, <= kContigRegs
  float v[kContigRegs][4];
  float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
  for (int i = 0; i < kContigRegs; ++i) {  // every load first, then their use
    const int64_t k = lane + (int64_t)kWave * i;
#pragma unroll
    for (int c = 0; c < 4; ++c) v[i][c] = -INFINITY;
    if (i < rounds && k < r.K) contig_load(p, r, k, v[i]);
  }
#pragma unroll
  for (int i = 0; i < kContigRegs; ++i) {
    const int64_t k = lane + (int64_t)kWave * i;
    if (i < rounds) {
      if (k < r.K) contig_leaky(p, r, k, v[i]);
#pragma unroll
      for (int c = 0; c < 4; ++c) m[c] = fmaxf(m[c], v[i][c]);
    }
  }
  contig_allmax(m, H);
  float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int i = 0; i < kContigRegs; ++i) {
    if (i < rounds) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        v[i][c] = v[i][c] == -INFINITY ? 0.0f : exp_nonpos(v[i][c] - m[c]);
        z[c] += v[i][c];
      }
    }
  }
  contig_allsum(z, H);
  float inv[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) inv[c] = 1.0f / z[c];
#pragma unroll
  for (int i = 0; i < kContigRegs; ++i) {
    const int64_t k = lane + (int64_t)kWave * i;
    if (i < rounds && k < r.K) {
      float o[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) o[c] = v[i][c] * inv[c];
      contig_store(p, r, k, o);
    }
  }
}

// Longer rows and segments of split rows: running (max, sum) per slot over the
// float4s, kStreamDepth in flight; then either publish per-segment
// statistics or re-read and normalise.  Each batch first takes its maximum,
// rescales the running sum once to it and adds its exponentials: one
// exponential per value and no divergent branch (a value-by-value running
// update would take a data-dependent branch per value).
__device__ __forceinline__ void softmax_contig_stream(const SoftmaxParams& p, const Item& it) {
  const int lane = lane_id();
  const int H = p.H;
  const ContigRange r = contig_range(it.b, it.e, H);
  float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t k0 = lane; k0 < r.K; k0 += kStreamDepth * kWave) {
    float v[kStreamDepth][4];
#pragma unroll
    for (int i = 0; i < kStreamDepth; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) {
        contig_load(p, r, k, v[i]);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) v[i][c] = -INFINITY;
      }
    }
#pragma unroll
    for (int i = 0; i < kStreamDepth; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) contig_leaky(p, r, k, v[i]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float bm = v[0][c];
#pragma unroll
      for (int i = 1; i < kStreamDepth; ++i) bm = fmaxf(bm, v[i][c]);
      const float nm = fmaxf(m[c], bm);
      if (nm == -INFINITY) continue;  // nothing but padding so far
      // exp(-inf) = 0 covers an empty running sum and padded values
      float acc = z[c] * exp_nonpos(m[c] - nm);
#pragma unroll
      for (int i = 0; i < kStreamDepth; ++i) acc += exp_nonpos(v[i][c] - nm);
      z[c] = acc;
      m[c] = nm;
    }
  }
  contig_alllse(m, z, H);
  if (it.slot >= 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int h = contig_head(r, lane, c, H);
      // one publishing lane per head: the lowest lane/slot holding it
      const bool pub = H >= 4 ? lane < H / 4 : (lane == 0 && c < H);
      if (pub) {
        p.ws[((int64_t)it.slot * H + h) * 2 + 0] = m[c];
        p.ws[((int64_t)it.slot * H + h) * 2 + 1] = z[c];
      }
    }
    return;
  }
  float inv[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) inv[c] = 1.0f / z[c];
  for (int64_t k0 = lane; k0 < r.K; k0 += kStreamDepth * kWave) {
    float v[kStreamDepth][4];
#pragma unroll
    for (int i = 0; i < kStreamDepth; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) contig_load(p, r, k, v[i]);
    }
#pragma unroll
    for (int i = 0; i < kStreamDepth; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) {
        contig_leaky(p, r, k, v[i]);
        float o[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) o[c] = exp_nonpos(v[i][c] - m[c]) * inv[c];
        contig_store(p, r, k, o);
      }
    }
  }
}

// Lanes map to (edge offset, head) pairs: hc = heads per pass, epw = 64/hc
// edges per pass.  Pass 1 keeps a running (max, sum) per lane; lanes of one
// head then merge in a fixed tree; pass 2 writes exp(s' - m) / z.  Segments
// of split rows stop after pass 1 and leave (m, z) in the workspace.
template <bool SEG>
__global__ __launch_bounds__(kBlock) void softmax_kernel(SoftmaxParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  if (it.b >= it.e) return;
  const int lane = lane_id();
  const int H = p.H;
  // float4 lanes once a row fills the wavefront or has >= 4 heads; short rows
  // with one or two heads use one value per lane instead
  if (p.contig && (H >= 4 || (it.e - it.b) * H > (int64_t)kWave * kSoftmaxU)) {
    const int64_t nvec = contig_range(it.b, it.e, H).K;
    if (!(SEG && it.slot >= 0) && nvec <= (int64_t)kWave * kContigRegs)
      softmax_contig_regs(p, it);
    else
      softmax_contig_stream(p, it);
    return;
  }
  if (!(SEG && it.slot >= 0) && H <= kWave && (H & (H - 1)) == 0 &&
      (it.e - it.b) * H <= (int64_t)kWave * kSoftmaxU) {
    softmax_row_in_registers(p, it);
    return;
  }
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int h = h0 + lane % hc;
    const bool active = eo < epw;
    float m = -INFINITY, z = 0.0f;
    if (active) {
      for (int64_t q0 = it.b + eo; q0 < it.e; q0 += (int64_t)kSoftmaxU * epw) {
        float sv[kSoftmaxU];
#pragma unroll
        for (int k = 0; k < kSoftmaxU; ++k) {
          const int64_t q = q0 + (int64_t)k * epw;
          sv[k] = -INFINITY;
          if (q < it.e) {
            const int64_t eid = p.eids ? p.eids[q] : q;
            sv[k] = leaky_relu(p.scores[eid * H + h], p.leaky, p.slope);
          }
        }
#pragma unroll
        for (int k = 0; k < kSoftmaxU; ++k)
          if (q0 + (int64_t)k * epw < it.e) lse_push(m, z, sv[k]);
      }
    }
    // tree over edge offsets: offset eo merges eo + k for k = 1, 2, 4, ...
    for (int k = 1; k < epw; k <<= 1) {
      const int partner = (lane + k * hc) & (kWave - 1);
      const float om = __shfl(m, partner);
      const float oz = __shfl(z, partner);
      if (active && (eo % (2 * k)) == 0 && eo + k < epw) lse_merge(m, z, om, oz);
    }
    m = __shfl(m, lane % hc);
    z = __shfl(z, lane % hc);
    if (SEG && it.slot >= 0) {
      if (active && eo == 0) {
        p.ws[((int64_t)it.slot * H + h) * 2 + 0] = m;
        p.ws[((int64_t)it.slot * H + h) * 2 + 1] = z;
      }
      continue;
    }
    if (active) {
      const float inv = 1.0f / z;
      for (int64_t q0 = it.b + eo; q0 < it.e; q0 += (int64_t)kSoftmaxU * epw) {
        float sv[kSoftmaxU];
        int64_t ev[kSoftmaxU];
#pragma unroll
        for (int k = 0; k < kSoftmaxU; ++k) {
          const int64_t q = q0 + (int64_t)k * epw;
          ev[k] = -1;
          if (q < it.e) {
            ev[k] = p.eids ? p.eids[q] : q;
            sv[k] = leaky_relu(p.scores[ev[k] * H + h], p.leaky, p.slope);
          }
        }
#pragma unroll
        for (int k = 0; k < kSoftmaxU; ++k)
          if (ev[k] >= 0) p.out[ev[k] * H + h] = exp_nonpos(sv[k] - m) * inv;
      }
    }
  }
}

// Merges the per-segment (m, z) of each split row into one pair per head.
// Block = 4 wavefronts; lane (eo, head) of wavefront w takes slots
// t = w*epw + eo, t + 4*epw, ... in order; the 4*epw partial pairs are then
// merged in order of t by the first lane of each head.
__global__ __launch_bounds__(kBlock) void softmax_rowstats_kernel(SoftmaxParams p) {
  __shared__ float red_m[kBlock];
  __shared__ float red_z[kBlock];
  const Fix fx = p.fix[blockIdx.x];
  const int w = threadIdx.x >> 6;
  const int lane = lane_id();
  const int H = p.H;
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int hh = lane % hc;
    const int h = h0 + hh;
    const int lanes = kWavesPerBlock * epw;
    const int t = w * epw + eo;
    float m = -INFINITY, z = 0.0f;
    if (eo < epw) {
      for (int s = fx.slot_begin + t; s < fx.slot_end; s += lanes)
        lse_merge(m, z, p.ws[((int64_t)s * H + h) * 2 + 0], p.ws[((int64_t)s * H + h) * 2 + 1]);
    }
    red_m[threadIdx.x] = m;
    red_z[threadIdx.x] = z;
    __syncthreads();
    if (t == 0 && eo < epw) {
      // thread index of slot-lane tt for head hh: (tt / epw) * 64 + (tt % epw) * hc + hh;
      // slot-lanes at or beyond the row's slot count hold nothing
      const int used = min(lanes, fx.slot_end - fx.slot_begin);
      for (int tt = 1; tt < used; ++tt) {
        const int idx = (tt / epw) * kWave + (tt % epw) * hc + hh;
        lse_merge(m, z, red_m[idx], red_z[idx]);
      }
      p.ws_row[((int64_t)blockIdx.x * H + h) * 2 + 0] = m;
      p.ws_row[((int64_t)blockIdx.x * H + h) * 2 + 1] = z;
    }
    __syncthreads();
  }
}

// Second pass for segments of split rows: normalise this segment's edges with
// its row's merged (m, z).  Item = slot.
__global__ __launch_bounds__(kBlock) void softmax_split_kernel(SoftmaxParams p, int64_t n_slots) {
  const int64_t slot = wave_item();
  if (slot >= n_slots) return;
  const Seg s = p.segs[p.slot_seg[slot]];
  const int64_t fi = p.slot_fix[slot];
  const int lane = lane_id();
  const int H = p.H;
  if (p.contig) {
    const ContigRange r = contig_range(s.begin, s.end, H);
    float m[4], inv[4];
    if (p.self_merge) {
      // one head: every wavefront of the row merges the row's segment
      // statistics itself (lane l takes slots l, l + 64, ... in order, then a
      // fixed butterfly; lse_merge is symmetric, so all lanes agree bitwise)
      const Fix fx = p.fix[fi];
      float mm = -INFINITY, zz = 0.0f;
      for (int t = fx.slot_begin + lane; t < fx.slot_end; t += kWave)
        lse_merge(mm, zz, p.ws[(int64_t)t * 2 + 0], p.ws[(int64_t)t * 2 + 1]);
      for (int off = 1; off < kWave; off <<= 1) {
        const float om = __shfl_xor(mm, off);
        const float oz = __shfl_xor(zz, off);
        lse_merge(mm, zz, om, oz);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        m[c] = mm;
        inv[c] = 1.0f / zz;
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int h = contig_head(r, lane, c, H);
        m[c] = p.ws_row[(fi * H + h) * 2 + 0];
        inv[c] = 1.0f / p.ws_row[(fi * H + h) * 2 + 1];
      }
    }
    for (int64_t k0 = lane; k0 < r.K; k0 += kStreamDepth * kWave) {
      float v[kStreamDepth][4];
#pragma unroll
      for (int i = 0; i < kStreamDepth; ++i) {
        const int64_t k = k0 + (int64_t)kWave * i;
        if (k < r.K) contig_load(p, r, k, v[i]);
      }
#pragma unroll
      for (int i = 0; i < kStreamDepth; ++i) {
        const int64_t k = k0 + (int64_t)kWave * i;
        if (k < r.K) {
          contig_leaky(p, r, k, v[i]);
          float o[4];
#pragma unroll
          for (int c = 0; c < 4; ++c) o[c] = exp_nonpos(v[i][c] - m[c]) * inv[c];
          contig_store(p, r, k, o);
        }
      }
    }
    return;
  }
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int h = h0 + lane % hc;
    if (eo >= epw) continue;
    const float m = p.ws_row[(fi * H + h) * 2 + 0];
    const float inv = 1.0f / p.ws_row[(fi * H + h) * 2 + 1];
    for (int64_t q0 = s.begin + eo; q0 < s.end; q0 += (int64_t)kSoftmaxU * epw) {
      float sv[kSoftmaxU];
      int64_t ev[kSoftmaxU];
#pragma unroll
      for (int k = 0; k < kSoftmaxU; ++k) {
        const int64_t q = q0 + (int64_t)k * epw;
        ev[k] = -1;
        if (q < s.end) {
          ev[k] = p.eids ? p.eids[q] : q;
          sv[k] = leaky_relu(p.scores[ev[k] * H + h], p.leaky, p.slope);
        }
      }
#pragma unroll
      for (int k = 0; k < kSoftmaxU; ++k)
        if (ev[k] >= 0) p.out[ev[k] * H + h] = exp_nonpos(sv[k] - m) * inv;
    }
  }
}

// ----------------------------------------------------------------------------
// SDDMM dot (one head) with the edge softmax of its scores fused in
// ----------------------------------------------------------------------------

// Scores are produced as in sddmm_fast_kernel (lane j collects the score of
// edge j of each 64-edge batch) and written out; each lane also keeps a
// running (max, sum) of the leaky scores it collected.  A wavefront merges
// them in a fixed butterfly.  A whole row is then normalised: from registers
// when it is a single batch, else by re-reading the scores this wavefront
// just wrote (same lane, same address: program order).  A segment of a split
// row publishes its (max, sum) for softmax_rowstats_kernel and
// softmax_split_kernel.  The normalisation runs where the scores are made,
// without a second launch re-reading them from memory.
template <int G, int NV, int U, bool SEG>
__global__ __launch_bounds__(kBlock) void sddmm_softmax_kernel(SddmmParams p, float* att,
                                                               float* ws, int32_t leaky,
                                                               float slope) {
  constexpr int NG = kWave / G;
  static_assert(NG * U <= kWave, "one batch of 64 edges must cover whole steps");
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;
  if (it.b >= it.e) return;
  const int lane = lane_id();
  const int gid = lane / G;
  const int li = lane % G;
  const int64_t F = p.F;

  int64_t f[NV];
  bool act[NV];
  float xd[NV][4];
  const char* xl[NV];  // this lane's elements of source row 0
  const uint32_t rb = (uint32_t)F * 4u;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = (int64_t)(v * G + li) * 4;
    act[v] = f[v] < F;
    xl[v] = reinterpret_cast<const char*>(p.xs) + f[v] * 4;
    if (act[v]) {
      load_vec<4>(p.xd + it.row * F + f[v], xd[v]);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) xd[v][c] = 0.0f;
    }
  }

  float m = -INFINITY, z = 0.0f;  // this lane's leaky scores so far
  float res = 0.0f;
  int cnt = 0, my_eid = 0;
  for (int64_t base = it.b; base < it.e; base += kWave) {
    cnt = (int)min((int64_t)kWave, it.e - base);
    int my_src = 0;
    my_eid = 0;
    if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
      my_eid = p.eids ? __builtin_nontemporal_load(p.eids + base + lane) : (int)(base + lane);
    }
    res = 0.0f;
    for (int j0 = 0; j0 < cnt; j0 += NG * U) {
      float val[U][NV][4];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jb = j0 + u * NG;
        ok[u] = jb + gid < cnt;
        const int src = bcast_lane<NG>(my_src, jb, gid);
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if (ok[u] && act[v]) {
            load_vec<4>(row_at(xl[v], src, rb), val[u][v]);
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) val[u][v][c] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float part = 0.0f;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int c = 0; c < 4; ++c) part += val[u][v][c] * xd[v][c];
        part = group_sum<G>(part);
        const int jb = j0 + u * NG;
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          if (jb + g < cnt) {
            const int sum =
                __builtin_amdgcn_readlane(__builtin_bit_cast(int, part), (g + 1) * G - 1);
            if (lane == jb + g) res = __builtin_bit_cast(float, sum);
          }
        }
      }
    }
    if (lane < cnt) {
      p.out[my_eid] = res;
      lse_push(m, z, leaky_relu(res, leaky, slope));
    }
  }
  for (int off = 1; off < kWave; off <<= 1) {
    const float om = __shfl_xor(m, off), oz = __shfl_xor(z, off);
    lse_merge(m, z, om, oz);
  }
  if (SEG && it.slot >= 0) {
    if (lane == 0) {
      ws[(int64_t)it.slot * 2 + 0] = m;
      ws[(int64_t)it.slot * 2 + 1] = z;
    }
    return;
  }
  const float inv = 1.0f / z;
  if (it.e - it.b <= kWave) {
    if (lane < cnt) att[my_eid] = expf(leaky_relu(res, leaky, slope) - m) * inv;
    return;
  }
  for (int64_t q = it.b + lane; q < it.e; q += kWave) {
    const int64_t e = p.eids ? (int64_t)p.eids[q] : q;
    att[e] = expf(leaky_relu(p.out[e], leaky, slope) - m) * inv;
  }
}

// ----------------------------------------------------------------------------
// backward of gSpMM-max and of edge softmax
// ----------------------------------------------------------------------------

// Zero fill (a kernel, not a memset, so that a caller may capture it in a
// graph).  VEC4: the array is 16-byte aligned and n is a multiple of 4.
template <bool VEC4>
__global__ __launch_bounds__(kBlock) void zero_kernel(float* p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if constexpr (VEC4) {
    float4* q = reinterpret_cast<float4*>(p);
    for (int64_t i = t; i < n / 4; i += stride) q[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  } else {
    for (int64_t i = t; i < n; i += stride) p[i] = 0.0f;
  }
}

__global__ __launch_bounds__(kBlock) void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) p[i] = v;
}

// pos[edge_ids[q]] = q for every stored edge q (ids outside [0, nnz_total)
// are skipped; with distinct ids every write has its own address).
__global__ __launch_bounds__(kBlock) void eid_pos_kernel(const int32_t* eids, int64_t nnz,
                                                         int64_t nnz_total, int32_t* pos) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < nnz; q += stride) {
    const int32_t e = eids[q];
    if (e >= 0 && e < nnz_total) pos[e] = (int32_t)q;
  }
}

struct MaxBwdParams {
  const int32_t* indices;
  const int32_t* eid_pos;  // edge id -> storage position; null: edge id == position
  const int32_t* arg;      // [rows, F] edge id chosen by the forward, -1 for none
  const float* go;         // [rows, F] upstream gradient
  const float* x;          // [cols, F] source features (edge gradient only)
  const float* ev;         // [nnz_total, H] edge values (src_mul_edge only)
  float* gsrc;             // [cols, F] or null, zero-filled beforehand
  float* gedge;            // [nnz_total, H] or null, zero-filled beforehand
  int64_t num_rows, F, id_limit;  // ids >= id_limit are ignored
  int32_t H, dh, mul;
};

// One wavefront per destination row, lanes over its F output elements (two
// coalesced loads per element).  Each element's upstream gradient goes to the
// source of the edge its forward value came from, by a hardware fp32 atomic
// add in L2: about rows x F atomics in all, instead of re-reading every edge's
// argmax through the transposed graph (rows x F << E x F).  The order of the
// adds into one address is not fixed, so sums of several contributions may
// differ in the last bits between runs.
__global__ __launch_bounds__(kBlock) void spmm_max_bwd_kernel(MaxBwdParams p) {
  const int64_t v = wave_item();
  if (v >= p.num_rows) return;
  const int lane = lane_id();
  const int64_t base = v * p.F;
  for (int64_t f = lane; f < p.F; f += kWave) {
    const int32_t e = p.arg[base + f];
    if (e < 0 || e >= p.id_limit) continue;
    const int64_t q = p.eid_pos ? (int64_t)p.eid_pos[e] : (int64_t)e;
    if (q < 0) continue;
    const int64_t u = p.indices[q];
    const float g = p.go[base + f];
    const int64_t he = (int64_t)e * p.H + (p.H == 1 ? 0 : (int32_t)f / p.dh);
    if (p.gsrc) unsafeAtomicAdd(&p.gsrc[u * p.F + f], p.mul ? p.ev[he] * g : g);
    if (p.gedge) unsafeAtomicAdd(&p.gedge[he], p.x[u * p.F + f] * g);
  }
}

// ---- binned gSpMM-max backward
//
// The same sums as spmm_max_bwd_kernel without global atomics: a counting
// sort moves every gradient element, as an 8-byte (slot, value) record, into
// the bin of its source tile (2^logR consecutive source rows, at most
// kBinTileFloats values), and then one workgroup per piece of a bin adds its
// records in LDS and writes the tile's rows with coalesced stores.  Device
// fp32 atomics at scattered addresses run at about 2e10 per second on MI355X
// whatever their contention (measured with the real target addresses and
// with random ones), so the atomic kernel is bound by their rate; the binned
// form streams arg, grad_out and the records instead.  Bins with more than
// kBinPiece records are split over several workgroups, which add their
// partial tiles with atomics into rows zeroed beforehand.
//
// Kernels, in stream order: counts per (group, bin) and per bin; prefix sums
// over bins; the scatter of the records (each group reserves one run per bin
// with an atomic add on the bin's cursor); the per-tile sums.  A group of the
// counting and scatter kernels owns a range of whole rows, the same in both.

constexpr int kBinPiece = 16384;       // records per accumulating workgroup
constexpr int kBinBlock = 512;         // threads of an accumulating workgroup
constexpr int kBinThreads = 1024;      // threads of a counting / scatter group
constexpr int kBinUnroll = 4;          // elements in flight per thread

struct BinParams {
  const int32_t* indices;
  const int32_t* eid_pos;  // edge id -> storage position; null: edge id == position
  const int32_t* arg;      // [rows, F]
  const float* go;         // [rows, F]
  const float* ev;         // [nnz_total, H] edge values (src_mul_edge only)
  float* gsrc;             // [cols, F]
  int32_t* total;          // [nb] records per bin (zeroed beforehand)
  int32_t* start;          // [nb + 1] first record of each bin
  int32_t* piece;          // [nb + 1] first accumulating workgroup of each bin
  int32_t* cursor;         // [nb] next free record of each bin
  int32_t* runs;           // [groups, nb] records per group and bin
  int2* rec;               // records (slot in the tile, value bits)
  int64_t num_rows, num_cols, id_limit;
  int32_t F, H, dh, mul, logR, nb, rows_per_group;
};

// Source of the element whose forward took edge id e; -1 if e is not an edge
// of this graph.
__device__ __forceinline__ int32_t bin_source(const BinParams& p, int32_t e) {
  if (e < 0 || e >= p.id_limit) return -1;
  const int32_t q = p.eid_pos ? p.eid_pos[e] : e;
  return q < 0 ? -1 : p.indices[q];
}

__device__ __forceinline__ int32_t bin_pieces(int32_t records) {
  return records <= kBinPiece ? 1 : (records + kBinPiece - 1) / kBinPiece;
}

// Elements [first, first + n) of the flat [rows, F] arrays that this group
// of the counting and scatter kernels owns (whole rows).
__device__ __forceinline__ void bin_range(const BinParams& p, int64_t& first, int32_t& n) {
  const int64_t r0 = (int64_t)blockIdx.x * p.rows_per_group;
  const int64_t r1 = min(p.num_rows, r0 + p.rows_per_group);
  first = r0 * p.F;
  n = r1 > r0 ? (int32_t)((r1 - r0) * p.F) : 0;
}

// Records per (group, bin), counted in LDS; per bin also one global add.
__global__ __launch_bounds__(kBinThreads) void bin_count_kernel(BinParams p) {
  extern __shared__ int32_t bin_lds[];
  int32_t* cnt = bin_lds;  // [nb]
  for (int b = threadIdx.x; b < p.nb; b += kBinThreads) cnt[b] = 0;
  __syncthreads();
  int64_t first;
  int32_t n;
  bin_range(p, first, n);
  for (int32_t t0 = threadIdx.x; t0 < n; t0 += kBinThreads * kBinUnroll) {
    int32_t e[kBinUnroll];
#pragma unroll
    for (int k = 0; k < kBinUnroll; ++k) {
      const int32_t t = t0 + k * kBinThreads;
      e[k] = t < n ? p.arg[first + t] : -1;
    }
    int32_t u[kBinUnroll];
#pragma unroll
    for (int k = 0; k < kBinUnroll; ++k) u[k] = bin_source(p, e[k]);
#pragma unroll
    for (int k = 0; k < kBinUnroll; ++k)
      if (u[k] >= 0) atomicAdd(&cnt[u[k] >> p.logR], 1);
  }
  __syncthreads();
  int32_t* mine = p.runs + (int64_t)blockIdx.x * p.nb;
  for (int b = threadIdx.x; b < p.nb; b += kBinThreads) {
    const int32_t c = cnt[b];
    mine[b] = c;
    if (c) atomicAdd(&p.total[b], c);
  }
}

// Exclusive prefix sums of the bin sizes (record offsets) and of their piece
// counts (accumulating workgroups); one workgroup of 1024 threads.
constexpr int kBinScanThreads = 1024;
__global__ __launch_bounds__(kBinScanThreads) void bin_scan_kernel(BinParams p) {
  __shared__ int32_t s_rec[kBinScanThreads];
  __shared__ int32_t s_pc[kBinScanThreads];
  const int t = threadIdx.x;
  const int per = (p.nb + kBinScanThreads - 1) / kBinScanThreads;
  const int b0 = min(p.nb, t * per), b1 = min(p.nb, b0 + per);
  int32_t rec = 0, pc = 0;
  for (int b = b0; b < b1; ++b) {
    rec += p.total[b];
    pc += bin_pieces(p.total[b]);
  }
  s_rec[t] = rec;
  s_pc[t] = pc;
  __syncthreads();
  for (int off = 1; off < kBinScanThreads; off <<= 1) {
    const int32_t a = t >= off ? s_rec[t - off] : 0;
    const int32_t c = t >= off ? s_pc[t - off] : 0;
    __syncthreads();
    s_rec[t] += a;
    s_pc[t] += c;
    __syncthreads();
  }
  rec = s_rec[t] - rec;
  pc = s_pc[t] - pc;
  for (int b = b0; b < b1; ++b) {
    p.start[b] = rec;
    p.cursor[b] = rec;
    p.piece[b] = pc;
    rec += p.total[b];
    pc += bin_pieces(p.total[b]);
  }
  if (t == kBinScanThreads - 1) {
    p.start[p.nb] = s_rec[t];
    p.piece[p.nb] = s_pc[t];
  }
}

// Zeroes the rows of every split bin (their pieces add with atomics), then
// reserves this group's run in each bin it feeds and writes each element's
// record into it, ranked inside the run through LDS.
__global__ __launch_bounds__(kBinThreads) void bin_scatter_kernel(BinParams p) {
  extern __shared__ int32_t bin_lds[];
  int32_t* cnt = bin_lds;          // [nb]
  int32_t* run = bin_lds + p.nb;   // [nb]
  const int64_t tile = ((int64_t)1 << p.logR) * p.F;
  for (int b = blockIdx.x; b < p.nb; b += gridDim.x) {
    if (p.piece[b + 1] - p.piece[b] == 1) continue;
    const int64_t lo = (int64_t)b * tile;
    const int64_t hi = min(p.num_cols * p.F, lo + tile);
    for (int64_t t = lo + threadIdx.x; t < hi; t += kBinThreads) p.gsrc[t] = 0.0f;
  }
  const int32_t* mine = p.runs + (int64_t)blockIdx.x * p.nb;
  for (int b = threadIdx.x; b < p.nb; b += kBinThreads) {
    const int32_t c = mine[b];
    cnt[b] = 0;
    run[b] = c ? atomicAdd(&p.cursor[b], c) : 0;
  }
  __syncthreads();
  int64_t first;
  int32_t n;
  bin_range(p, first, n);
  for (int32_t t0 = threadIdx.x; t0 < n; t0 += kBinThreads * kBinUnroll) {
    int32_t e[kBinUnroll];
    float g[kBinUnroll];
#pragma unroll
    for (int k = 0; k < kBinUnroll; ++k) {
      const int32_t t = t0 + k * kBinThreads;
      e[k] = -1;
      g[k] = 0.0f;
      if (t < n) {
        e[k] = p.arg[first + t];
        g[k] = p.go[first + t];
      }
    }
    int32_t u[kBinUnroll];
#pragma unroll
    for (int k = 0; k < kBinUnroll; ++k) u[k] = bin_source(p, e[k]);
#pragma unroll
    for (int k = 0; k < kBinUnroll; ++k) {
      if (u[k] < 0) continue;
      const int32_t t = t0 + k * kBinThreads;
      const int32_t b = u[k] >> p.logR;
      const int32_t r = atomicAdd(&cnt[b], 1);
      const int32_t f = t % p.F;
      float v = g[k];
      if (p.mul) v = p.ev[(int64_t)e[k] * p.H + (p.H == 1 ? 0 : f / p.dh)] * v;
      const int32_t slot = (u[k] - (b << p.logR)) * p.F + f;
      p.rec[run[b] + r] = make_int2(slot, __float_as_int(v));
    }
  }
}

// One piece of one bin: adds its records into an LDS tile and writes the
// tile's rows (plain stores for a whole bin, atomics for a split one).
__global__ __launch_bounds__(kBinBlock) void bin_accumulate_kernel(BinParams p) {
  __shared__ float tile[kBinTileFloats];
  const int32_t i = (int32_t)blockIdx.x;
  if (i >= p.piece[p.nb]) return;
  int lo = 0, hi = p.nb - 1;  // the last bin whose first piece is <= i
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.piece[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  const int b = lo;
  const int32_t k = i - p.piece[b];
  const bool whole = p.piece[b + 1] - p.piece[b] == 1;
  const int64_t r0 = (int64_t)p.start[b] + (int64_t)k * kBinPiece;
  const int64_t r1 = min((int64_t)p.start[b + 1], r0 + kBinPiece);
  const int64_t row0 = (int64_t)b << p.logR;
  const int32_t n_el = (int32_t)(min((int64_t)1 << p.logR, p.num_cols - row0) * p.F);
  for (int32_t t = threadIdx.x; t < n_el; t += kBinBlock) tile[t] = 0.0f;
  __syncthreads();
  for (int64_t j0 = r0 + threadIdx.x; j0 < r1; j0 += kBinBlock * kBinUnroll) {
    int2 q[kBinUnroll];
#pragma unroll
    for (int k2 = 0; k2 < kBinUnroll; ++k2) {
      const int64_t j = j0 + k2 * kBinBlock;
      q[k2] = j < r1 ? p.rec[j] : make_int2(-1, 0);
    }
#pragma unroll
    for (int k2 = 0; k2 < kBinUnroll; ++k2)
      if (q[k2].x >= 0) atomicAdd(&tile[q[k2].x], __int_as_float(q[k2].y));
  }
  __syncthreads();
  float* dst = p.gsrc + row0 * p.F;
  if (whole) {
    for (int32_t t = threadIdx.x; t < n_el; t += kBinBlock) dst[t] = tile[t];
  } else {
    for (int32_t t = threadIdx.x; t < n_el; t += kBinBlock) {
      const float v = tile[t];
      if (v != 0.0f) unsafeAtomicAdd(&dst[t], v);
    }
  }
}

// float4 k of a contiguous row's flat range of an [E, H] array; elements
// outside the range read as `fill` / are not written.
__device__ __forceinline__ void flat_load4(const float* base, const ContigRange& r, int64_t k,
                                           float (&v)[4], float fill) {
  const int64_t t0 = r.T0 + 4 * k;
  if (t0 >= r.lo && t0 + 4 <= r.hi) {
    load_vec<4>(base + t0, v);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t t = t0 + c;
      v[c] = (t >= r.lo && t < r.hi) ? base[t] : fill;
    }
  }
}

__device__ __forceinline__ void flat_store4(float* base, const ContigRange& r, int64_t k,
                                            const float (&v)[4]) {
  const int64_t t0 = r.T0 + 4 * k;
  if (t0 >= r.lo && t0 + 4 <= r.hi) {
    store_vec<4>(base + t0, v);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t t = t0 + c;
      if (t >= r.lo && t < r.hi) base[t] = v[c];
    }
  }
}

struct SoftmaxBwdParams {
  const int32_t* indptr;
  const int32_t* eids;
  const float* a;   // forward output (attention weights)
  const float* go;  // upstream gradient w.r.t. a
  const float* s;   // forward input scores (leaky ReLU only)
  float* ds;        // gradient w.r.t. the scores
  const Seg* segs;
  const Fix* fix;
  const int32_t* slot_fix;
  const int32_t* slot_seg;
  float* ws;  // [slot][H] partial sums of a * go
  int64_t n_items;
  int32_t H;
  int32_t leaky;
  float slope;
  int32_t contig;  // edge id == position, H a power of two <= 64, 16-byte aligned arrays
};

// ---- contiguous rows (same lane layout as the forward's float4 path: slot c
// of every float4 a lane touches holds one fixed head)

// Pass 2 over a range: ds = a * (go - c) * leaky factor, c per slot.
__device__ __forceinline__ void softmax_bwd_contig_apply(const SoftmaxBwdParams& p,
                                                         const ContigRange& r,
                                                         const float (&c)[4]) {
  const int lane = lane_id();
  for (int64_t k0 = lane; k0 < r.K; k0 += 4 * kWave) {
    float a[4][4], g[4][4], sv[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) {
        flat_load4(p.a, r, k, a[i], 0.0f);
        flat_load4(p.go, r, k, g[i], 0.0f);
        if (p.leaky) flat_load4(p.s, r, k, sv[i], 1.0f);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) {
        float o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          o[q] = a[i][q] * (g[i][q] - c[q]);
          if (p.leaky && !(sv[i][q] > 0.0f)) o[q] *= p.slope;
        }
        flat_store4(p.ds, r, k, o);
      }
    }
  }
}

// Pass 1 (sum of a * go per head, four float4 pairs in flight per lane), then
// pass 2 for a whole row, or the partial sums published for a split row.
__device__ __forceinline__ void softmax_bwd_contig(const SoftmaxBwdParams& p, const Item& it) {
  const int lane = lane_id();
  const int H = p.H;
  const ContigRange r = contig_range(it.b, it.e, H);
  float c[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t k0 = lane; k0 < r.K; k0 += 4 * kWave) {
    float a[4][4], g[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t k = k0 + (int64_t)kWave * i;
      if (k < r.K) {
        flat_load4(p.a, r, k, a[i], 0.0f);
        flat_load4(p.go, r, k, g[i], 0.0f);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) a[i][q] = g[i][q] = 0.0f;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) c[q] = fmaf(a[i][q], g[i][q], c[q]);
  }
  contig_allsum(c, H);
  if (it.slot >= 0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool pub = H >= 4 ? lane < H / 4 : (lane == 0 && q < H);
      if (pub) p.ws[(int64_t)it.slot * H + contig_head(r, lane, q, H)] = c[q];
    }
    return;
  }
  softmax_bwd_contig_apply(p, r, c);
}

// Multi-head SDDMM with the edge-softmax backward of its results fused in: the
// score gradient of an attention layer.  Per row v and head h, with a the
// forward's attention weights and s its scores:
//   g_e = <x_src[u_e, h, :], x_dst[v, h, :]>      (the SDDMM: dL/da)
//   c   = sum_e a_e g_e,   ds_e = a_e (g_e - c) * (leaky && !(s_e > 0) ? slope : 1)
// Pass 1 computes g as sddmm_headed_kernel does (staged per 64-edge batch in
// LDS), writes it to ds and accumulates c; pass 2 re-reads g (just written by
// this wavefront, so mostly from L2), a and s and writes ds.  This replaces
// the softmax backward's separate pass over the [E, H] arrays.
// FLAT (edge id = position, H in {4, 8, 16}, aligned [E, H] arrays): a batch's
// [cnt, H] block of a / g is a flat range handled as float4s, lane l always on
// the heads (4l + q) mod H, exactly as softmax_bwd_contig lays out a row, so
// pass 2 is softmax_bwd_contig_apply with g in place of the upstream
// gradient; the batch's a loads are issued before its gathers.  Otherwise
// lane j takes edge j of a batch and loops over its heads.  Whole rows only:
// the launcher uses this kernel when no row is split (H <= kTabHeads).
template <int S, bool SEG, bool FLAT>
__global__ __launch_bounds__(kBlock) void sddmm_softmax_bwd_kernel(SddmmParams p, const float* a,
                                                                   const float* sc, int leaky,
                                                                   float slope) {
  constexpr int U = 4;
  constexpr int NC = FLAT ? 4 : kTabHeads;
  __shared__ __align__(16) float tab_all[kWavesPerBlock * kWave * kTabHeads];
  float* tab = tab_all + (threadIdx.x >> 6) * kWave * kTabHeads;
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  if (it.b >= it.e) return;
  const int lane = lane_id();
  const int H = p.H;
  const int G = 1 << p.logG;
  const int ngroups = kWave >> p.logG;
  const int gid = lane >> p.logG;
  const int li = lane & (G - 1);
  const int64_t F = p.F;
  const int64_t f = (int64_t)li * 4;
  const bool act = f < F;
  const int64_t h = act ? f / p.dh : 0;
  float xd[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (act) load_vec<4>(p.xd + it.row * F + f, xd);
  const char* xl = reinterpret_cast<const char*>(p.xs) + f * 4;  // lane's elements of row 0
  const uint32_t rb = (uint32_t)F * 4u;
  float c[NC];  // FLAT: per float4 slot (fixed head); else per head
#pragma unroll
  for (int k = 0; k < NC; ++k) c[k] = 0.0f;

  for (int64_t base = it.b; base < it.e; base += kWave) {
    const int cnt = (int)min((int64_t)kWave, it.e - base);
    int my_src = 0, my_eid = 0;
    if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
      my_eid = p.eids ? __builtin_nontemporal_load(p.eids + base + lane) : (int)(base + lane);
    }
    const int n4 = cnt * H / 4;  // FLAT: float4s of the batch's [cnt, H] block
    float a4[4][4];
    if constexpr (FLAT) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = lane + kWave * i;
        if (k < n4) {
          load_vec<4>(a + base * H + 4 * k, a4[i]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) a4[i][q] = 0.0f;
        }
      }
    }
    for (int j0 = 0; j0 < cnt; j0 += ngroups * U) {
      float val[U][4];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * ngroups + gid;
        ok[u] = j < cnt;
        const int src = __shfl(my_src, j & (kWave - 1));
        if (ok[u] && act) {
          load_vec<4>(row_at(xl, src, rb), val[u]);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k) val[u][k] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float part = 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k) part += val[u][k] * xd[k];
        part = group_sum<S>(part);
        if (ok[u] && act && (li % S) == S - 1) tab[(j0 + u * ngroups + gid) * H + h] = part;
      }
    }
    wave_lds_sync();
    if constexpr (FLAT) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = lane + kWave * i;
        if (k < n4) {
          float g4[4];
          load_vec<4>(tab + 4 * k, g4);
          store_vec<4>(p.out + base * H + 4 * k, g4);
#pragma unroll
          for (int q = 0; q < 4; ++q) c[q] = fmaf(a4[i][q], g4[q], c[q]);
        }
      }
    } else if (lane < cnt) {  // lane j: edge base + j, its H values of g
      const float* tr = tab + lane * H;
      float* orow = p.out + (int64_t)my_eid * H;
      const float* arow = a + (int64_t)my_eid * H;
#pragma unroll
      for (int hh = 0; hh < kTabHeads; ++hh)
        if (hh < H) {
          const float q = tr[hh];
          orow[hh] = q;
          c[hh] = fmaf(arow[hh], q, c[hh]);
        }
    }
    wave_lds_sync();  // the table is rewritten by the next batch
  }

  if constexpr (FLAT) {
    contig_allsum(c, H);
    SoftmaxBwdParams q;
    q.a = a;
    q.go = p.out;
    q.s = sc;
    q.ds = p.out;
    q.H = H;
    q.leaky = leaky;
    q.slope = slope;
    softmax_bwd_contig_apply(q, contig_range(it.b, it.e, H), c);
    return;
  } else {
    // c per head over the row: the lanes' shares, in a fixed butterfly
#pragma unroll
    for (int hh = 0; hh < kTabHeads; ++hh)
      if (hh < H)
        for (int off = 1; off < kWave; off <<= 1) c[hh] += __shfl_xor(c[hh], off);
    for (int64_t base = it.b; base < it.e; base += kWave) {
      const int cnt = (int)min((int64_t)kWave, it.e - base);
      if (lane >= cnt) continue;
      const int64_t e = p.eids ? (int64_t)p.eids[base + lane] : base + lane;
      float* orow = p.out + e * H;
      const float* arow = a + e * H;
#pragma unroll
      for (int hh = 0; hh < kTabHeads; ++hh)
        if (hh < H) {
          float o = arow[hh] * (orow[hh] - c[hh]);
          if (leaky && !(sc[e * H + hh] > 0.0f)) o *= slope;
          orow[hh] = o;
        }
    }
  }
}

// ds_e = a_e * (go_e - c) * (leaky && s_e <= 0 ? slope : 1), c = sum_row a go.
__device__ __forceinline__ void softmax_bwd_write(const SoftmaxBwdParams& p, int64_t b,
                                                  int64_t e, int eo, int epw, int h, float c) {
  const int H = p.H;
  for (int64_t q0 = b + eo; q0 < e; q0 += (int64_t)kSoftmaxU * epw) {
    float av[kSoftmaxU], gv[kSoftmaxU], lf[kSoftmaxU];
    int64_t ix[kSoftmaxU];
#pragma unroll
    for (int k = 0; k < kSoftmaxU; ++k) {
      const int64_t q = q0 + (int64_t)k * epw;
      ix[k] = -1;
      if (q < e) {
        ix[k] = (p.eids ? (int64_t)p.eids[q] : q) * H + h;
        av[k] = p.a[ix[k]];
        gv[k] = p.go[ix[k]];
        lf[k] = (p.leaky && !(p.s[ix[k]] > 0.0f)) ? p.slope : 1.0f;
      }
    }
#pragma unroll
    for (int k = 0; k < kSoftmaxU; ++k)
      if (ix[k] >= 0) p.ds[ix[k]] = av[k] * (gv[k] - c) * lf[k];
  }
}

// One wavefront per item, lanes on (edge offset, head) pairs as in the
// forward.  Pass 1 sums a * go per lane, lanes of one head combine in a fixed
// tree; a whole row then writes its gradients (pass 2), a segment of a split
// row leaves its partial sum in the workspace instead.
template <bool SEG>
__global__ __launch_bounds__(kBlock) void softmax_bwd_kernel(SoftmaxBwdParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0 || it.b >= it.e) return;
  const int lane = lane_id();
  const int H = p.H;
  // float4 lanes once a row fills the wavefront or has >= 4 heads
  if (p.contig && (H >= 4 || (it.e - it.b) * H > (int64_t)kWave * kSoftmaxU)) {
    softmax_bwd_contig(p, it);
    return;
  }
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int h = h0 + lane % hc;
    const bool active = eo < epw;
    float c = 0.0f;
    if (active) {
      for (int64_t q0 = it.b + eo; q0 < it.e; q0 += (int64_t)kSoftmaxU * epw) {
        float av[kSoftmaxU], gv[kSoftmaxU];
#pragma unroll
        for (int k = 0; k < kSoftmaxU; ++k) {
          const int64_t q = q0 + (int64_t)k * epw;
          av[k] = 0.0f;
          gv[k] = 0.0f;
          if (q < it.e) {
            const int64_t ix = (p.eids ? (int64_t)p.eids[q] : q) * H + h;
            av[k] = p.a[ix];
            gv[k] = p.go[ix];
          }
        }
#pragma unroll
        for (int k = 0; k < kSoftmaxU; ++k) c = fmaf(av[k], gv[k], c);
      }
    }
    for (int k = 1; k < epw; k <<= 1) {
      const int partner = (lane + k * hc) & (kWave - 1);
      const float oc = __shfl(c, partner);
      if (active && (eo % (2 * k)) == 0 && eo + k < epw) c += oc;
    }
    c = __shfl(c, lane % hc);
    if (SEG && it.slot >= 0) {
      if (active && eo == 0) p.ws[(int64_t)it.slot * H + h] = c;
      continue;
    }
    if (active) softmax_bwd_write(p, it.b, it.e, eo, epw, h, c);
  }
}

// Segments of split rows: add the row's partial sums in slot order (every
// segment of the row forms the same total), then write this segment's
// gradients.  Item = slot.
__global__ __launch_bounds__(kBlock) void softmax_bwd_split_kernel(SoftmaxBwdParams p,
                                                                   int64_t n_slots) {
  const int64_t slot = wave_item();
  if (slot >= n_slots) return;
  const Seg sg = p.segs[p.slot_seg[slot]];
  const Fix fx = p.fix[p.slot_fix[slot]];
  const int lane = lane_id();
  const int H = p.H;
  if (p.contig) {
    const ContigRange r = contig_range(sg.begin, sg.end, H);
    float c[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int h = contig_head(r, lane, q, H);
      c[q] = 0.0f;
      for (int t = fx.slot_begin; t < fx.slot_end; ++t) c[q] += p.ws[(int64_t)t * H + h];
    }
    softmax_bwd_contig_apply(p, r, c);
    return;
  }
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int h = h0 + lane % hc;
    if (eo >= epw) continue;
    float c = 0.0f;
    for (int t = fx.slot_begin; t < fx.slot_end; ++t) c += p.ws[(int64_t)t * H + h];
    softmax_bwd_write(p, sg.begin, sg.end, eo, epw, h, c);
  }
}

// Short single-head rows (at most kShortRowEdges edges, whole rows): four
// per wavefront, a 16-lane quarter per row holding up to 4 scores per lane;
// max and sum reduce within the quarter.  Items [first, last) of the plan.
constexpr int kPackLanes = 16;
static_assert(kShortRowEdges <= kPackLanes * 4, "a short row must fit one quarter");

__global__ __launch_bounds__(kBlock) void softmax_pack_kernel(SoftmaxParams p, int64_t first,
                                                              int64_t last) {
  const int64_t w = wave_item();
  const int64_t item0 = first + w * (kWave / kPackLanes);
  if (item0 >= last) return;
  const int lane = lane_id();
  const int64_t item = item0 + lane / kPackLanes;
  const int j = lane % kPackLanes;
  int64_t b = 0, e = 0;
  if (item < last) {
    const Seg sg = p.segs[item];
    b = sg.begin;
    e = sg.end;
  }
  float v[4];
  int64_t ev[4];
  float m = -INFINITY;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t q = b + j + (int64_t)k * kPackLanes;
    ev[k] = -1;
    v[k] = -INFINITY;
    if (q < e) {
      ev[k] = p.eids ? p.eids[q] : q;
      v[k] = leaky_relu(p.scores[ev[k]], p.leaky, p.slope);
    }
    m = fmaxf(m, v[k]);
  }
  for (int off = 1; off < kPackLanes; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
  float z = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[k] = ev[k] >= 0 ? exp_nonpos(v[k] - m) : 0.0f;
    z += v[k];
  }
  for (int off = 1; off < kPackLanes; off <<= 1) z += __shfl_xor(z, off);
  const float inv = 1.0f / z;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (ev[k] >= 0) p.out[ev[k]] = v[k] * inv;
}

// Whole rows of kShortRowEdges + 1 .. kMediumRowEdges edges, one head, scores
// contiguous (edge id = position): four rows per wavefront, kPackLanes lanes
// each; lane j of a row's group holds float4 j, j + 16, ... of the row's
// range aligned down to 16 bytes (at most 66 float4 for 256 edges, so
// kPack4Vec = 5 per lane covers it).  Exact maximum, one expf per value, one
// read and one write, like the register path of one row per wavefront.
constexpr int kPack4Vec = 5;
static_assert(kMediumRowEdges + 6 <= kPackLanes * kPack4Vec * 4,
              "a medium row's aligned float4 range must fit one quarter");

__global__ __launch_bounds__(kBlock) void softmax_pack4_kernel(SoftmaxParams p, int64_t first,
                                                               int64_t last) {
  const int64_t w = wave_item();
  const int64_t item0 = first + w * (kWave / kPackLanes);
  if (item0 >= last) return;
  const int lane = lane_id();
  const int64_t item = item0 + lane / kPackLanes;
  const int j = lane % kPackLanes;
  int64_t b = 0, e = 0;
  if (item < last) {
    const Seg sg = p.segs[item];
    b = sg.begin;
    e = sg.end;
  }
  const ContigRange r = contig_range(b, e, 1);
  float v[kPack4Vec][4];
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kPack4Vec; ++i) {
    const int64_t k = j + (int64_t)kPackLanes * i;
    if (k < r.K) {
      contig_load(p, r, k, v[i]);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) v[i][c] = -INFINITY;
    }
  }
#pragma unroll
  for (int i = 0; i < kPack4Vec; ++i) {
    const int64_t k = j + (int64_t)kPackLanes * i;
    if (k < r.K) contig_leaky(p, r, k, v[i]);
#pragma unroll
    for (int c = 0; c < 4; ++c) m = fmaxf(m, v[i][c]);
  }
  for (int off = 1; off < kPackLanes; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
  float z = 0.0f;
#pragma unroll
  for (int i = 0; i < kPack4Vec; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      v[i][c] = v[i][c] == -INFINITY ? 0.0f : exp_nonpos(v[i][c] - m);
      z += v[i][c];
    }
  for (int off = 1; off < kPackLanes; off <<= 1) z += __shfl_xor(z, off);
  const float inv = 1.0f / z;
#pragma unroll
  for (int i = 0; i < kPack4Vec; ++i) {
    const int64_t k = j + (int64_t)kPackLanes * i;
    if (k < r.K) {
      float o[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) o[c] = v[i][c] * inv;
      contig_store(p, r, k, o);
    }
  }
}

// ----------------------------------------------------------------------------
// fused attention aggregation: SDDMM -> leaky ReLU -> edge softmax -> gSpMM
// ----------------------------------------------------------------------------

// Floats per plan slot of the fused attention kernel: F partial sums, then H
// maxima and H exp-sums, padded so every slot starts 16-byte aligned.
__host__ __device__ __forceinline__ int64_t gat_ws_stride(int64_t F, int64_t H) {
  return F + ((2 * H + 3) & ~int64_t(3));
}

struct GatParams {
  const int32_t* indptr;
  const int32_t* indices;
  const float* xs;
  const float* xd;
  float* out;
  const Seg* segs;
  float* ws;  // per slot: [F] scaled partial sum, [H] running max, [H] scaled exp-sum
  int64_t n_items;
  int64_t nnz;  // length of indices
  int64_t F;
  int32_t H;
  int32_t dh;
  int32_t SH;  // lanes per head = dh / 4
  int32_t leaky;
  float slope;
};

// Sum over aligned groups of W lanes, returned in every lane of the group.
// For W = 32 a lane takes the total of its own half of the wavefront (a
// feature row of 64 lanes holds two such heads).
template <int W>
__device__ __forceinline__ float group_allsum(float v) {
  v = group_sum<W>(v);
  if constexpr (W == 32) {
    const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 31));
    const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
    v = (lane_id() & 32) ? b : a;
  } else if constexpr (W == 64) {
    v = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
  }
  return v;
}

// Merges a running-softmax state (m, z, acc) with another one.
__device__ __forceinline__ void attn_merge(float& m, float& z, float (&acc)[4], float om, float oz,
                                           const float (&oacc)[4]) {
  if (om == -INFINITY) return;
  if (m == -INFINITY) {
    m = om;
    z = oz;
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = oacc[c];
    return;
  }
  const float nm = fmaxf(m, om);
  const float a = expf(m - nm), b = expf(om - nm);
  z = z * a + oz * b;
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = acc[c] * a + oacc[c] * b;
  m = nm;
}

// One wavefront per row or segment; G lanes (float4 each) per feature row,
// SH lanes per head.  Per edge: dot of the gathered source row with the
// destination row held in registers, DPP reduction over the head's lanes,
// leaky ReLU, then an online-softmax update of (max, exp-sum, weighted sum of
// the same gathered source row).  The source row is read once per edge and no
// per-edge score is written.
// SH: lanes per head (dh / 4), a compile-time constant so the per-edge head
// reduction has no branches.  The running (max, sum, weighted sum) of a head
// is rescaled only when a score exceeds the current maximum (a branch the
// whole wavefront skips when no lane needs it); otherwise an edge costs one
// exponential and a multiply-add per feature.
// WIDE (two lane groups): 256-edge batches, ids four per lane in one load
// and through the group-major LDS table.
template <int G, int SH, bool SEG, bool WIDE = false>
__global__ __launch_bounds__(kBlock) void gat_fused_kernel(GatParams p) {
  constexpr int NG = kWave / G;
  constexpr int U = NG * 4 <= kWave ? 4 : 1;
  static_assert(SH <= G, "a head's lanes lie inside one lane group");
  static_assert(!WIDE || (NG == 2 && U % 4 == 0), "wide batches serve two lane groups");
  constexpr int BATCH = WIDE ? 4 * kWave : kWave;
  constexpr int WT = WIDE ? wide_tab<NG>() : 1;
  __shared__ __align__(16) int32_t wid_all[WIDE ? kWavesPerBlock * WT : 1];
  int32_t* wid = wid_all + (WIDE ? (threadIdx.x >> 6) * WT : 0);
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  const Item it = load_item<SEG>(p.segs, p.indptr, item);
  if (it.row < 0) return;  // padding item of a partitioned schedule
  const int lane = lane_id();
  const int gid = lane / G;
  const int li = lane % G;
  const int64_t F = p.F;
  const int64_t f = (int64_t)li * 4;
  const bool act = f < F;
  const int h = act ? (int)(f / p.dh) : 0;
  float xd[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (act) load_vec<4>(p.xd + it.row * F + f, xd);
  const char* xl = reinterpret_cast<const char*>(p.xs) + f * 4;  // lane's elements of row 0
  const uint32_t rb = (uint32_t)F * 4u;
  const bool all_act = (int64_t)G * 4 <= F;  // every lane holds a feature chunk
  float m = -INFINITY, z = 0.0f;
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};

  for (int64_t base = it.b; base < it.e; base += BATCH) {
    const int cnt = (int)min((int64_t)BATCH, it.e - base);
    int my_src = 0;
    if constexpr (WIDE) {
      int32_t q[4];
      load_ids<4>(p.indices, p.nnz, base, lane, cnt, q);
      wave_lds_sync();  // the previous batch's table reads are done
      wide_put<NG>(wid, lane, q);
      wave_lds_sync();
    } else if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
    }
    // one step of U edges per lane group; FULL: all of them in the batch and
    // every lane active (no masking)
    auto step = [&](int j0, auto full_tag) {
      constexpr bool FULL = decltype(full_tag)::value;
      float val[U][4];
      bool ok[U];
      int32_t tsrc[WIDE ? U : 1];
      if constexpr (WIDE) wide_get<NG, U>(wid, gid, j0, tsrc);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jb = j0 + u * NG;
        ok[u] = FULL || jb + gid < cnt;
        // (two or fewer groups: one cross-lane permute, off the vector ALU)
        int src;
        if constexpr (WIDE) src = tsrc[u];
        else src = NG <= 2 ? __shfl(my_src, jb + gid) : bcast_lane<NG>(my_src, jb, gid);
        if (FULL || (ok[u] && act)) {
          load_vec<4>(row_at(xl, src, rb), val[u]);
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) val[u][c] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float part = val[u][0] * xd[0] + val[u][1] * xd[1] + val[u][2] * xd[2] + val[u][3] * xd[3];
        float sc = SH == 1 ? part : group_allsum<SH>(part);
        sc = leaky_relu(sc, p.leaky, p.slope);
        if (FULL || ok[u]) {
          if (sc > m) {  // new maximum: move the state to it (m = -inf: a = 0)
            const float a = exp_nonpos(m - sc);
            z *= a;
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[c] *= a;
            m = sc;
          }
          const float b = exp_nonpos(sc - m);
          z += b;
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[c] = fmaf(b, val[u][c], acc[c]);
        }
      }
    };
    int j0 = 0;
    if (all_act)
      for (; j0 + NG * U <= cnt; j0 += NG * U) step(j0, BoolTag<true>{});
    for (; j0 < cnt; j0 += NG * U) step(j0, BoolTag<false>{});
  }
  // merge the lane groups
  for (int s = G; s < kWave; s <<= 1) {
    const float om = __shfl_xor(m, s), oz = __shfl_xor(z, s);
    float oacc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) oacc[c] = __shfl_xor(acc[c], s);
    attn_merge(m, z, acc, om, oz, oacc);
  }
  if (gid != 0 || !act) return;
  if (SEG && it.slot >= 0) {
    float* w = p.ws + (int64_t)it.slot * gat_ws_stride(F, p.H);
    store_vec<4>(w + f, acc);
    if (li % p.SH == 0) {
      w[F + h] = m;
      w[F + p.H + h] = z;
    }
    return;
  }
  float o[4];
  const float inv = z > 0.0f ? 1.0f / z : 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c) o[c] = acc[c] * inv;
  store_vec<4>(p.out + it.row * F + f, o);
}

// Merges the per-segment states of each split row and writes acc / z.
__global__ __launch_bounds__(kBlock) void gat_fixup_kernel(GatParams p, const Fix* fix) {
  const Fix fx = fix[blockIdx.x];
  const int64_t F = p.F;
  const int64_t stride = gat_ws_stride(F, p.H);
  for (int64_t f = threadIdx.x; f < F; f += kBlock) {
    const int64_t h = f / p.dh;
    float m = -INFINITY;
    for (int s = fx.slot_begin; s < fx.slot_end; ++s) m = fmaxf(m, p.ws[s * stride + F + h]);
    float z = 0.0f, acc = 0.0f;
    for (int s = fx.slot_begin; s < fx.slot_end; ++s) {
      const float ms = p.ws[s * stride + F + h];
      if (ms == -INFINITY) continue;
      const float a = expf(ms - m);
      z += p.ws[s * stride + F + p.H + h] * a;
      acc += p.ws[s * stride + f] * a;
    }
    p.out[(int64_t)fx.row * F + f] = z > 0.0f ? acc / z : 0.0f;
  }
}

// ----------------------------------------------------------------------------
// host-side dispatch
// ----------------------------------------------------------------------------

int ilog2_ceil(int64_t q) {
  int l = 0;
  while ((int64_t(1) << l) < q) ++l;
  return l;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

dim3 grid_for(int64_t items, int64_t chunks) {
  return dim3((unsigned)((items + kWavesPerBlock - 1) / kWavesPerBlock), (unsigned)chunks, 1);
}

#define FG_LAUNCH(kernel, grid, stream, ...) \
  hipLaunchKernelGGL((kernel), (grid), dim3(kBlock), 0, (stream), __VA_ARGS__)

// avg: the items' average edge count (256-edge batches where the lane layout
// allows them and the items are long enough, wide_item_edges)
template <int G, int NV, int U, bool MUL, bool MAX, bool EIDS, bool ADD, bool TAB>
void spmm_fast_seg2(const SpmmParams& prm, bool seg, int64_t avg, dim3 grid, hipStream_t st) {
  if constexpr (kWave / G >= 2 && U % 4 == 0 && !EIDS && !TAB) {
    if (avg >= wide_item_edges<kWave / G>() && (!MUL || prm.H == 1)) {
      if (seg)
        FG_LAUNCH((spmm_fast_kernel<G, NV, U, MUL, MAX, EIDS, true, ADD, TAB, true>), grid, st,
                  prm);
      else
        FG_LAUNCH((spmm_fast_kernel<G, NV, U, MUL, MAX, EIDS, false, ADD, TAB, true>), grid, st,
                  prm);
      return;
    }
  }
  if (seg) FG_LAUNCH((spmm_fast_kernel<G, NV, U, MUL, MAX, EIDS, true, ADD, TAB>), grid, st, prm);
  else FG_LAUNCH((spmm_fast_kernel<G, NV, U, MUL, MAX, EIDS, false, ADD, TAB>), grid, st, prm);
}

template <int G, int NV, int U, bool MUL, bool MAX, bool EIDS, bool ADD = false>
void spmm_fast_seg(const SpmmParams& prm, bool seg, int64_t avg, dim3 grid, hipStream_t st) {
  // per-head edge values come from a per-batch LDS table
  if constexpr (MUL) {
    if (prm.H >= 2 && prm.H <= kTabHeads) {
      spmm_fast_seg2<G, NV, U, MUL, MAX, EIDS, ADD, true>(prm, seg, avg, grid, st);
      return;
    }
  }
  spmm_fast_seg2<G, NV, U, MUL, MAX, EIDS, ADD, false>(prm, seg, avg, grid, st);
}

template <int G, int NV, int U, bool MUL, bool MAX, bool ADD = false>
void spmm_fast_eids(const SpmmParams& prm, bool seg, int64_t avg, dim3 grid, hipStream_t st) {
  // copy + sum never looks at edge ids
  if (prm.eids && (MUL || MAX))
    spmm_fast_seg<G, NV, U, MUL, MAX, true, ADD>(prm, seg, avg, grid, st);
  else
    spmm_fast_seg<G, NV, U, MUL, MAX, false, ADD>(prm, seg, avg, grid, st);
}

template <int G, int NV, int U>
void spmm_fast_ops(const SpmmParams& prm, bool mul, bool mx, bool seg, int64_t avg, dim3 grid,
                   hipStream_t st) {
  if (prm.xd) {
    spmm_fast_eids<G, NV, U, false, true, true>(prm, seg, avg, grid, st);
  } else if (mul) {
    if (mx) spmm_fast_eids<G, NV, U, true, true>(prm, seg, avg, grid, st);
    else spmm_fast_eids<G, NV, U, true, false>(prm, seg, avg, grid, st);
  } else {
    if (mx) spmm_fast_eids<G, NV, U, false, true>(prm, seg, avg, grid, st);
    else spmm_fast_eids<G, NV, U, false, false>(prm, seg, avg, grid, st);
  }
}

template <int NV, int U, bool MUL, bool MAX, bool ADD = false>
void spmm_generic_seg(const SpmmParams& prm, bool seg, dim3 grid, hipStream_t st) {
  if (seg) FG_LAUNCH((spmm_generic_kernel<NV, U, MUL, MAX, true, ADD>), grid, st, prm);
  else FG_LAUNCH((spmm_generic_kernel<NV, U, MUL, MAX, false, ADD>), grid, st, prm);
}

template <int NV, int U>
void spmm_generic_ops(const SpmmParams& prm, bool mul, bool mx, bool seg, dim3 grid,
                      hipStream_t st) {
  if (prm.xd) {
    spmm_generic_seg<NV, U, false, true, true>(prm, seg, grid, st);
  } else if (mul) {
    if (mx) spmm_generic_seg<NV, U, true, true>(prm, seg, grid, st);
    else spmm_generic_seg<NV, U, true, false>(prm, seg, grid, st);
  } else {
    if (mx) spmm_generic_seg<NV, U, false, true>(prm, seg, grid, st);
    else spmm_generic_seg<NV, U, false, false>(prm, seg, grid, st);
  }
}

// avg: the items' average edge count (batches of four ids per lane where the
// lane layout allows it and the items are long enough, wide_item_edges)
template <int G, int NV, int U>
void sddmm_fast_go(const SddmmParams& prm, bool seg, int64_t avg, dim3 grid, hipStream_t st) {
  if constexpr (ids_per_lane<kWave / G, U>() > 1) {
    if (avg >= wide_item_edges<kWave / G>()) {
      if (seg) FG_LAUNCH((sddmm_fast_kernel<G, NV, U, true, true>), grid, st, prm);
      else FG_LAUNCH((sddmm_fast_kernel<G, NV, U, false, true>), grid, st, prm);
      return;
    }
  }
  if (seg) FG_LAUNCH((sddmm_fast_kernel<G, NV, U, true>), grid, st, prm);
  else FG_LAUNCH((sddmm_fast_kernel<G, NV, U, false>), grid, st, prm);
}

template <int S>
void sddmm_headed_go(const SddmmParams& prm, bool seg, dim3 grid, hipStream_t st) {
  if (seg) FG_LAUNCH((sddmm_headed_kernel<S, true>), grid, st, prm);
  else FG_LAUNCH((sddmm_headed_kernel<S, false>), grid, st, prm);
}

template <int NV, int U, bool HEADED>
void sddmm_scalar_go(const SddmmParams& prm, bool seg, dim3 grid, hipStream_t st) {
  if (seg) FG_LAUNCH((sddmm_scalar_kernel<NV, U, HEADED, true>), grid, st, prm);
  else FG_LAUNCH((sddmm_scalar_kernel<NV, U, HEADED, false>), grid, st, prm);
}

}  // namespace

namespace {

// gSpMM launch; xd != null selects the u_add_v + relu message (max only).
hipError_t launch_spmm_core(const GraphView& g, const PlanView* plan, int msg, int red, int64_t H,
                            int64_t dh, const float* x, const float* ev, const float* xd,
                            float* out, int32_t* arg, hipStream_t stream) {
  if (g.num_rows == 0) return hipSuccess;
  const int64_t F = H * dh;
  const bool mul = msg == kSrcMulEdge;
  const bool mx = red == kMax;
  const bool seg = plan != nullptr;
  const bool vec4 = (F % 4 == 0) && (H == 1 || dh % 4 == 0) && aligned16(x) && aligned16(out) &&
                    (!mx || aligned16(arg)) && (!xd || aligned16(xd));
  SpmmParams prm;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.eids = g.edge_ids;
  prm.x = x;
  prm.ev = ev;
  prm.xd = xd;
  prm.out = out;
  prm.arg = arg;
  prm.segs = seg ? plan->segs : nullptr;
  prm.ws_f = seg ? plan->ws_f : nullptr;
  prm.ws_i = seg ? plan->ws_i : nullptr;
  prm.n_items = seg ? plan->num_segments : g.num_rows;
  prm.nnz = g.nnz;
  prm.F = F;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.logG = 6;
  prm.ev_vec4 = (ev && H % 4 == 0 && aligned16(ev)) ? 1 : 0;
  if (vec4) {
    const int64_t Q = F / 4;  // float4 per row
    const int64_t avg = g.nnz / std::max<int64_t>(prm.n_items, 1);
    const dim3 grid1 = grid_for(prm.n_items, 1);
    if (Q <= 4) spmm_fast_ops<4, 1, 4>(prm, mul, mx, seg, avg, grid1, stream);
    else if (Q <= 8) spmm_fast_ops<8, 1, 8>(prm, mul, mx, seg, avg, grid1, stream);
    else if (Q <= 16) spmm_fast_ops<16, 1, 8>(prm, mul, mx, seg, avg, grid1, stream);
    else if (Q <= 32) spmm_fast_ops<32, 1, 8>(prm, mul, mx, seg, avg, grid1, stream);
    else if (Q <= 64) spmm_fast_ops<64, 1, 8>(prm, mul, mx, seg, avg, grid1, stream);
    else if (Q <= 128) spmm_fast_ops<64, 2, 4>(prm, mul, mx, seg, avg, grid1, stream);
    else
      spmm_fast_ops<64, 4, 2>(prm, mul, mx, seg, avg, grid_for(prm.n_items, (Q + 255) / 256),
                              stream);
  } else {
    // scalar lanes: G = 2^ceil(log2 F) up to 64, then NV values per lane
    int nv = 1;
    int64_t chunks = 1;
    if (F <= kWave) {
      prm.logG = ilog2_ceil(F);
    } else {
      nv = F <= 2 * kWave ? 2 : 4;
      chunks = (F + (int64_t)kWave * nv - 1) / ((int64_t)kWave * nv);
    }
    const dim3 grid = grid_for(prm.n_items, chunks);
    if (nv == 1) spmm_generic_ops<1, 4>(prm, mul, mx, seg, grid, stream);
    else if (nv == 2) spmm_generic_ops<2, 2>(prm, mul, mx, seg, grid, stream);
    else spmm_generic_ops<4, 1>(prm, mul, mx, seg, grid, stream);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (seg && plan->num_split_rows > 0) {
    // u_add_v partials are raw values: the merge applies the epilogue (the
    // float4 kernel with positional edge ids keeps them unmasked)
    const int epi = !xd ? kEpiNone : ((vec4 && !g.edge_ids) ? kEpiFirst : kEpiMasked);
    // float4 merge: vec4 already checked F % 4, out (and arg, xd) alignment
    if (vec4) {
      const dim3 fgrid((unsigned)plan->num_split_rows, (unsigned)((F + 4 * kWave - 1) / (4 * kWave)),
                       1);
      if (epi == kEpiFirst)
        FG_LAUNCH((spmm_fixup4_kernel<true, kEpiFirst>), fgrid, stream, plan->fix, plan->ws_f,
                  plan->ws_i, F, out, arg, xd, g.indptr);
      else if (epi == kEpiMasked)
        FG_LAUNCH((spmm_fixup4_kernel<true, kEpiMasked>), fgrid, stream, plan->fix, plan->ws_f,
                  plan->ws_i, F, out, arg, xd, g.indptr);
      else if (mx)
        FG_LAUNCH((spmm_fixup4_kernel<true>), fgrid, stream, plan->fix, plan->ws_f, plan->ws_i,
                  F, out, arg, nullptr, nullptr);
      else
        FG_LAUNCH((spmm_fixup4_kernel<false>), fgrid, stream, plan->fix, plan->ws_f, plan->ws_i,
                  F, out, arg, nullptr, nullptr);
      return hipGetLastError();
    }
    const dim3 fgrid((unsigned)plan->num_split_rows, (unsigned)((F + kWave - 1) / kWave), 1);
    if (epi == kEpiFirst)
      FG_LAUNCH((spmm_fixup_kernel<true, kEpiFirst>), fgrid, stream, plan->fix, plan->ws_f,
                plan->ws_i, F, out, arg, xd, g.indptr);
    else if (epi == kEpiMasked)
      FG_LAUNCH((spmm_fixup_kernel<true, kEpiMasked>), fgrid, stream, plan->fix, plan->ws_f,
                plan->ws_i, F, out, arg, xd, g.indptr);
    else if (mx)
      FG_LAUNCH((spmm_fixup_kernel<true>), fgrid, stream, plan->fix, plan->ws_f, plan->ws_i, F,
                out, arg, nullptr, nullptr);
    else
      FG_LAUNCH((spmm_fixup_kernel<false>), fgrid, stream, plan->fix, plan->ws_f, plan->ws_i, F,
                out, arg, nullptr, nullptr);
    err = hipGetLastError();
  }
  return err;
}

// Y[n, M] = X[n, K] W[K, M] on the matrix cores (v_mfma_f32_16x16x4_f32,
// fp32 in and out).  One wavefront per 16-row x 64-column tile of Y, four
// 16x16 accumulators, K in steps of 4 (zero-padded).  Operand layout of the
// instruction: lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] and
// receives D[4 (l / 16) + r][l % 16], r = 0..3.
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kMmTileCols = 64;

__global__ __launch_bounds__(kBlock) void dense_matmul_kernel(const float* x, const float* w,
                                                              float* y, int64_t n, int32_t K,
                                                              int32_t M, int64_t n_tiles) {
  const int64_t t = wave_item();
  if (t >= n_tiles) return;
  const int64_t col_tiles = (M + kMmTileCols - 1) / kMmTileCols;
  const int64_t rt = t / col_tiles, ct = t % col_tiles;
  const int lane = lane_id();
  const int i = lane & 15, q = lane >> 4;
  const int64_t arow = rt * 16 + i;
  f32x4 acc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) acc[b] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  for (int k0 = 0; k0 < K; k0 += 4) {
    const int k = k0 + q;
    const float a = (arow < n && k < K) ? x[arow * K + k] : 0.0f;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int64_t col = ct * kMmTileCols + b * 16 + i;
      const float bv = (k < K && col < M) ? w[(int64_t)k * M + col] : 0.0f;
      acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv, acc[b], 0, 0, 0);
    }
  }
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int64_t col = ct * kMmTileCols + b * 16 + i;
    if (col >= M) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t orow = rt * 16 + q * 4 + r;
      if (orow < n) y[orow * M + col] = acc[b][r];
    }
  }
}

}  // namespace

hipError_t launch_gspmm(const GraphView& g, const PlanView* plan, int msg, int red, int64_t H,
                        int64_t dh, const float* x, const float* ev, float* out, int32_t* arg,
                        hipStream_t stream) {
  return launch_spmm_core(g, plan, msg, red, H, dh, x, ev, nullptr, out, arg, stream);
}

hipError_t launch_dense_matmul(int64_t n, int64_t K, int64_t M, const float* x, const float* w,
                               float* y, hipStream_t stream) {
  if (n == 0 || M == 0) return hipSuccess;
  const int64_t tiles = ((n + 15) / 16) * ((M + kMmTileCols - 1) / kMmTileCols);
  FG_LAUNCH(dense_matmul_kernel, grid_for(tiles, 1), stream, x, w, y, n, (int32_t)K, (int32_t)M,
            tiles);
  return hipGetLastError();
}

hipError_t launch_mlp_aggregate(const GraphView& g, const PlanView* plan, int64_t d_in,
                                int64_t d_out, const float* xs, const float* xd, const float* w,
                                float* out, int32_t* arg, float* ws, hipStream_t stream) {
  // (x_u + x_v) W = x_u W + x_v W: transform the vertices once, then each
  // edge's message is relu(P_src[u] + P_dst[v])
  float* ps = ws;
  float* pd = ws;
  hipError_t err = launch_dense_matmul(g.num_cols, d_in, d_out, xs, w, ps, stream);
  if (err != hipSuccess) return err;
  if (!(xd == xs && g.num_rows == g.num_cols)) {
    pd = ws + g.num_cols * d_out;
    if ((err = launch_dense_matmul(g.num_rows, d_in, d_out, xd, w, pd, stream)) != hipSuccess)
      return err;
  }
  return launch_spmm_core(g, plan, kCopySrc, kMax, 1, d_out, ps, nullptr, pd, out, arg, stream);
}

hipError_t launch_gsddmm(const GraphView& g, const PlanView* plan, int64_t H, int64_t dh,
                         const float* xs, const float* xd, float* out, hipStream_t stream) {
  if (g.num_rows == 0 || g.nnz == 0) return hipSuccess;
  const int64_t F = H * dh;
  const bool seg = plan != nullptr;
  SddmmParams prm;
  prm.nnz = g.nnz;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.eids = g.edge_ids;
  prm.xs = xs;
  prm.xd = xd;
  prm.out = out;
  prm.segs = seg ? plan->segs : nullptr;
  prm.n_items = seg ? plan->num_nonempty : g.num_rows;  // empty rows (last) write nothing
  prm.F = F;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.logG = 6;
  prm.logS = 0;
  prm.out_vec4 = (H % 4 == 0 && aligned16(out)) ? 1 : 0;
  const dim3 grid = grid_for(prm.n_items, 1);
  const bool vec4 = (F % 4 == 0) && (H == 1 || dh % 4 == 0) && aligned16(xs) && aligned16(xd);
  if (vec4 && H == 1 && F <= 4 * 4 * kWave) {
    const int64_t Q = F / 4;
    // items long enough on average (wide_item_edges) take the 256-edge
    // batches; short items (source-slab pieces) keep 64-edge batches
    const int64_t items = seg ? plan->num_segments : g.num_rows;
    const int64_t avg = g.nnz / std::max<int64_t>(items, 1);
    if (Q <= 4) sddmm_fast_go<4, 1, 4>(prm, seg, avg, grid, stream);
    else if (Q <= 8) sddmm_fast_go<8, 1, 8>(prm, seg, avg, grid, stream);
    else if (Q <= 16) sddmm_fast_go<16, 1, 8>(prm, seg, avg, grid, stream);
    else if (Q <= 32) sddmm_fast_go<32, 1, 8>(prm, seg, avg, grid, stream);
    else if (Q <= 64) sddmm_fast_go<64, 1, 8>(prm, seg, avg, grid, stream);
    else if (Q <= 128) sddmm_fast_go<64, 2, 4>(prm, seg, avg, grid, stream);
    else sddmm_fast_go<64, 4, 2>(prm, seg, avg, grid, stream);
    return hipGetLastError();
  }
  if (vec4 && H > 1 && F <= 4 * kWave && (dh == 16 || dh == 32 || dh == 64)) {
    prm.logG = ilog2_ceil(F / 4);
    if (dh == 16) sddmm_headed_go<4>(prm, seg, grid, stream);
    else if (dh == 32) sddmm_headed_go<8>(prm, seg, grid, stream);
    else sddmm_headed_go<16>(prm, seg, grid, stream);
    return hipGetLastError();
  }
  // scalar lanes: one value per lane, G = 2^ceil(log2 F) <= 64, NV <= 4
  const bool headed = H > 1;
  bool generic = F > 4 * kWave;
  if (headed) {
    prm.logS = ilog2_ceil(dh);
    if ((int64_t(1) << prm.logS) != dh || dh > kWave) generic = true;
  }
  if (generic) {
    if (seg) FG_LAUNCH((sddmm_generic_kernel<true>), grid, stream, prm);
    else FG_LAUNCH((sddmm_generic_kernel<false>), grid, stream, prm);
    return hipGetLastError();
  }
  int nv = 1;
  if (F <= kWave) prm.logG = ilog2_ceil(F);
  else nv = F <= 2 * kWave ? 2 : 4;
  if (headed) {
    if (nv == 1) sddmm_scalar_go<1, 4, true>(prm, seg, grid, stream);
    else if (nv == 2) sddmm_scalar_go<2, 2, true>(prm, seg, grid, stream);
    else sddmm_scalar_go<4, 1, true>(prm, seg, grid, stream);
  } else {
    if (nv == 1) sddmm_scalar_go<1, 4, false>(prm, seg, grid, stream);
    else if (nv == 2) sddmm_scalar_go<2, 2, false>(prm, seg, grid, stream);
    else sddmm_scalar_go<4, 1, false>(prm, seg, grid, stream);
  }
  return hipGetLastError();
}

hipError_t launch_gsddmm_softmax_backward(const GraphView& g, const PlanView* gather,
                                          const PlanView* plain, int64_t H, int64_t dh,
                                          const float* xs, const float* xd, const float* a,
                                          const float* scores, bool leaky, float slope, float* ds,
                                          hipStream_t stream) {
  if (g.num_rows == 0 || g.nnz == 0) return hipSuccess;
  const int64_t F = H * dh;
  const bool fused = H >= 2 && H <= kTabHeads && (dh == 16 || dh == 32 || dh == 64) &&
                     F <= 4 * kWave && aligned16(xs) && aligned16(xd) &&
                     (!plain || plain->num_slots == 0);
  if (!fused) {  // the two operators, the second in place
    hipError_t err = launch_gsddmm(g, gather, H, dh, xs, xd, ds, stream);
    if (err != hipSuccess) return err;
    return launch_edge_softmax_backward(g, plain, H, a, ds, scores, leaky, slope, ds, stream);
  }
  const bool seg = plain != nullptr;
  SddmmParams prm;
  prm.nnz = g.nnz;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.eids = g.edge_ids;
  prm.xs = xs;
  prm.xd = xd;
  prm.out = ds;
  prm.segs = seg ? plain->segs : nullptr;
  prm.n_items = seg ? plain->num_nonempty : g.num_rows;
  prm.F = F;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.logG = ilog2_ceil(F / 4);
  prm.logS = 0;
  prm.out_vec4 = 0;
  const bool flat = g.edge_ids == nullptr && H % 4 == 0 && aligned16(ds) && aligned16(a) &&
                    (!leaky || aligned16(scores));
  const dim3 grid = grid_for(prm.n_items, 1);
  const int lk = leaky ? 1 : 0;
#define FG_SSB3(SS, SG, FL) \
  FG_LAUNCH((sddmm_softmax_bwd_kernel<SS, SG, FL>), grid, stream, prm, a, scores, lk, slope)
#define FG_SSB(SS)                 \
  if (seg && flat)                 \
    FG_SSB3(SS, true, true);       \
  else if (seg)                    \
    FG_SSB3(SS, true, false);      \
  else if (flat)                   \
    FG_SSB3(SS, false, true);      \
  else                             \
    FG_SSB3(SS, false, false);
  if (dh == 16) {
    FG_SSB(4)
  } else if (dh == 32) {
    FG_SSB(8)
  } else {
    FG_SSB(16)
  }
#undef FG_SSB3
#undef FG_SSB
  return hipGetLastError();
}

bool gsddmm_softmax_fused(int64_t H, int64_t dh, const float* xs, const float* xd) {
  const int64_t F = H * dh;
  return H == 1 && F % 4 == 0 && F <= 4 * 4 * kWave && aligned16(xs) && aligned16(xd);
}

hipError_t launch_gsddmm_softmax(const GraphView& g, const PlanView* plan, int64_t F,
                                 const float* xs, const float* xd, bool leaky, float slope,
                                 float* scores, float* att, hipStream_t stream) {
  if (g.num_rows == 0 || g.nnz == 0) return hipSuccess;
  const bool seg = plan != nullptr;
  SddmmParams prm;
  prm.nnz = g.nnz;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.eids = g.edge_ids;
  prm.xs = xs;
  prm.xd = xd;
  prm.out = scores;
  prm.segs = seg ? plan->segs : nullptr;
  prm.n_items = seg ? plan->num_nonempty : g.num_rows;  // empty rows write nothing
  prm.F = F;
  prm.H = 1;
  prm.dh = (int32_t)F;
  prm.logG = 6;
  prm.logS = 0;
  prm.out_vec4 = 0;
  float* ws = seg ? plan->ws_f : nullptr;
  const int32_t lk = leaky ? 1 : 0;
  const dim3 grid = grid_for(prm.n_items, 1);
  const int64_t Q = F / 4;
#define FG_SDS(GG, NVV, UU)                                                                 \
  if (seg) FG_LAUNCH((sddmm_softmax_kernel<GG, NVV, UU, true>), grid, stream, prm, att, ws, lk, \
                     slope);                                                                \
  else FG_LAUNCH((sddmm_softmax_kernel<GG, NVV, UU, false>), grid, stream, prm, att, ws, lk, slope);
  if (Q <= 4) { FG_SDS(4, 1, 4) }
  else if (Q <= 8) { FG_SDS(8, 1, 8) }
  else if (Q <= 16) { FG_SDS(16, 1, 8) }
  else if (Q <= 32) { FG_SDS(32, 1, 8) }
  else if (Q <= 64) { FG_SDS(64, 1, 8) }
  else if (Q <= 128) { FG_SDS(64, 2, 4) }
  else { FG_SDS(64, 4, 2) }
#undef FG_SDS
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !seg || plan->num_slots == 0) return err;
  // split rows: merge the segments' (max, sum), then normalise their edges
  SoftmaxParams sp;
  sp.indptr = g.indptr;
  sp.eids = g.edge_ids;
  sp.scores = scores;
  sp.out = att;
  sp.segs = plan->segs;
  sp.fix = plan->fix;
  sp.slot_fix = plan->slot_fix;
  sp.slot_seg = plan->slot_seg;
  sp.ws = plan->ws_f;
  sp.ws_row = plan->ws_row;
  sp.n_items = plan->num_segments;
  sp.H = 1;
  sp.leaky = lk;
  sp.slope = slope;
  sp.contig = (g.edge_ids == nullptr && aligned16(scores) && aligned16(att)) ? 1 : 0;
  sp.self_merge = sp.contig;
  if (!sp.self_merge) {
    FG_LAUNCH(softmax_rowstats_kernel, dim3((unsigned)plan->num_split_rows, 1, 1), stream, sp);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  FG_LAUNCH(softmax_split_kernel, grid_for(plan->num_slots, 1), stream, sp, plan->num_slots);
  return hipGetLastError();
}

hipError_t launch_edge_softmax(const GraphView& g, const PlanView* plan, int64_t H,
                               const float* scores, bool leaky, float slope, float* out,
                               hipStream_t stream) {
  if (g.num_rows == 0 || g.nnz == 0) return hipSuccess;
  SoftmaxParams prm;
  prm.indptr = g.indptr;
  prm.eids = g.edge_ids;
  prm.scores = scores;
  prm.out = out;
  prm.segs = plan ? plan->segs : nullptr;
  prm.fix = plan ? plan->fix : nullptr;
  prm.slot_fix = plan ? plan->slot_fix : nullptr;
  prm.slot_seg = plan ? plan->slot_seg : nullptr;
  prm.ws = plan ? plan->ws_f : nullptr;
  prm.ws_row = plan ? plan->ws_row : nullptr;
  prm.n_items = plan ? plan->num_segments : g.num_rows;
  prm.H = (int32_t)H;
  prm.leaky = leaky ? 1 : 0;
  prm.slope = slope;
  prm.contig = (g.edge_ids == nullptr && H <= kWave && (H & (H - 1)) == 0 && aligned16(scores) &&
                aligned16(out)) ? 1 : 0;
  prm.self_merge = (prm.contig && H == 1) ? 1 : 0;
  // with a plan: empty rows (last) need no work; short single-head rows go
  // four to a wavefront, and so do medium rows with contiguous scores
  const bool pack = plan && H == 1 && plan->num_long < plan->num_nonempty;
  const bool pack4 = plan && H == 1 && prm.contig && plan->num_medium < plan->num_long;
  if (plan)
    prm.n_items = pack4 ? plan->num_medium : (pack ? plan->num_long : plan->num_nonempty);
  hipError_t err = hipSuccess;
  if (prm.n_items > 0) {
    const dim3 grid = grid_for(prm.n_items, 1);
    if (plan) FG_LAUNCH((softmax_kernel<true>), grid, stream, prm);
    else FG_LAUNCH((softmax_kernel<false>), grid, stream, prm);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (pack4) {
    const int64_t rows = plan->num_long - plan->num_medium;
    const int64_t per = kWave / kPackLanes;
    FG_LAUNCH(softmax_pack4_kernel, grid_for((rows + per - 1) / per, 1), stream, prm,
              plan->num_medium, plan->num_long);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (pack) {
    const int64_t rows = plan->num_nonempty - plan->num_long;
    const int64_t per = kWave / kPackLanes;
    FG_LAUNCH(softmax_pack_kernel, grid_for((rows + per - 1) / per, 1), stream, prm,
              plan->num_long, plan->num_nonempty);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (!plan || plan->num_slots == 0) return err;
  if (!prm.self_merge) {
    FG_LAUNCH(softmax_rowstats_kernel, dim3((unsigned)plan->num_split_rows, 1, 1), stream, prm);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  FG_LAUNCH(softmax_split_kernel, grid_for(plan->num_slots, 1), stream, prm, plan->num_slots);
  return hipGetLastError();
}

bool gat_fused_supported(int64_t H, int64_t dh) {
  const int64_t F = H * dh;
  if (dh % 4 != 0 || F > 4 * kWave) return false;
  const int64_t sh = dh / 4;
  return (sh & (sh - 1)) == 0;
}

hipError_t launch_gat_fused(const GraphView& g, const PlanView* plan, int64_t H, int64_t dh,
                            const float* xs, const float* xd, bool leaky, float slope, float* out,
                            hipStream_t stream) {
  if (g.num_rows == 0) return hipSuccess;
  const bool seg = plan != nullptr;
  GatParams prm;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.xs = xs;
  prm.xd = xd;
  prm.out = out;
  prm.segs = seg ? plan->segs : nullptr;
  prm.ws = seg ? plan->ws_f : nullptr;
  prm.n_items = seg ? plan->num_segments : g.num_rows;
  prm.nnz = g.nnz;
  prm.F = H * dh;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.SH = (int32_t)(dh / 4);
  prm.leaky = leaky ? 1 : 0;
  prm.slope = slope;
  const dim3 grid = grid_for(prm.n_items, 1);
  const int64_t Q = prm.F / 4;
  const int G = Q <= 4 ? 4 : Q <= 8 ? 8 : Q <= 16 ? 16 : Q <= 32 ? 32 : 64;
  // lanes of a head must not straddle the group (SH <= G always holds: dh <= F);
  // two lane groups on items of kWideItemEdges edges or more on average take
  // 256-edge batches
  const bool wide = g.nnz >= kWideItemEdges * std::max<int64_t>(prm.n_items, 1);
#define FG_GAT2(GG, SS)                                                              \
  if (GG == 32 && wide) {                                                            \
    if (seg) FG_LAUNCH((gat_fused_kernel<GG, SS, true, GG == 32>), grid, stream, prm); \
    else FG_LAUNCH((gat_fused_kernel<GG, SS, false, GG == 32>), grid, stream, prm);    \
  } else if (seg) {                                                                  \
    FG_LAUNCH((gat_fused_kernel<GG, SS, true>), grid, stream, prm);                  \
  } else {                                                                           \
    FG_LAUNCH((gat_fused_kernel<GG, SS, false>), grid, stream, prm);                 \
  }
#define FG_GAT(GG)                                                             \
  switch (prm.SH) {                                                            \
    case 1: { FG_GAT2(GG, 1) } break;                                          \
    case 2: { FG_GAT2(GG, (GG >= 2 ? 2 : 1)) } break;                          \
    case 4: { FG_GAT2(GG, (GG >= 4 ? 4 : 1)) } break;                          \
    case 8: { FG_GAT2(GG, (GG >= 8 ? 8 : 1)) } break;                          \
    case 16: { FG_GAT2(GG, (GG >= 16 ? 16 : 1)) } break;                       \
    case 32: { FG_GAT2(GG, (GG >= 32 ? 32 : 1)) } break;                       \
    default: { FG_GAT2(GG, (GG >= 64 ? 64 : 1)) } break;                       \
  }
  switch (G) {
    case 4: FG_GAT(4) break;
    case 8: FG_GAT(8) break;
    case 16: FG_GAT(16) break;
    case 32: FG_GAT(32) break;
    default: FG_GAT(64) break;
  }
#undef FG_GAT
#undef FG_GAT2
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !seg || plan->num_split_rows == 0) return err;
  FG_LAUNCH(gat_fixup_kernel, dim3((unsigned)plan->num_split_rows, 1, 1), stream, prm, plan->fix);
  return hipGetLastError();
}

namespace {

dim3 stride_grid(int64_t n) {
  const int64_t b = (n + kBlock - 1) / kBlock;
  return dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>(b, 8192)), 1, 1);
}

hipError_t zero_fill(float* p, int64_t n, hipStream_t stream) {
  if (!p || n <= 0) return hipSuccess;
  if (aligned16(p) && n % 4 == 0)
    FG_LAUNCH((zero_kernel<true>), stride_grid(n / 4), stream, p, n);
  else
    FG_LAUNCH((zero_kernel<false>), stride_grid(n), stream, p, n);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_build_eid_pos(const int32_t* eids, int64_t nnz, int64_t nnz_total, int32_t* pos,
                                hipStream_t stream) {
  if (nnz_total > 0) FG_LAUNCH(fill_i32_kernel, stride_grid(nnz_total), stream, pos, nnz_total, -1);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || nnz == 0) return err;
  FG_LAUNCH(eid_pos_kernel, stride_grid(nnz), stream, eids, nnz, nnz_total, pos);
  return hipGetLastError();
}

// Tile rows (log2) and bin count of the binned max backward for width F;
// false if the shape does not fit the workspace, its LDS tables or int32
// record offsets.
static bool bin_shape(const GraphView& g, int64_t F, const BinWorkspace* ws, int& logR, int& nb) {
  if (!ws || !ws->rec || F < 1 || F > kBinTileFloats) return false;
  if (g.num_rows * F > INT32_MAX || g.num_rows * F > ws->rec_capacity) return false;
  const int64_t bins = bin_tiles(g.num_cols, F);
  if (bins < 1 || bins > kMaxBins || bins > ws->max_bins) return false;
  logR = bin_log_rows(F);
  nb = (int)bins;
  return true;
}

hipError_t launch_gspmm_max_backward(const GraphView& g, const int32_t* eid_pos, int msg,
                                     int64_t H, int64_t dh, const float* x, const float* ev,
                                     const int32_t* arg, const float* go, float* gsrc,
                                     float* gedge, const BinWorkspace* ws, hipStream_t stream) {
  const int64_t F = H * dh;
  int logR = 0, nb = 0;
  if (gsrc && g.num_rows > 0 && g.nnz > 0 && bin_shape(g, F, ws, logR, nb)) {
    // the edge gradient (if asked) still goes through the atomic kernel
    hipError_t err = hipSuccess;
    if (gedge) {
      err = launch_gspmm_max_backward(g, eid_pos, msg, H, dh, x, ev, arg, go, nullptr, gedge,
                                      nullptr, stream);
      if (err != hipSuccess) return err;
    }
    BinParams bp;
    bp.indices = g.indices;
    bp.eid_pos = g.edge_ids ? eid_pos : nullptr;
    bp.arg = arg;
    bp.go = go;
    bp.ev = ev;
    bp.gsrc = gsrc;
    bp.total = ws->tables;
    bp.start = ws->tables + (kMaxBins + 1);
    bp.piece = ws->tables + 2 * (kMaxBins + 1);
    bp.cursor = ws->tables + 3 * (kMaxBins + 1);
    bp.runs = ws->runs;
    bp.rec = static_cast<int2*>(ws->rec);
    bp.num_rows = g.num_rows;
    bp.num_cols = g.num_cols;
    bp.id_limit = g.edge_ids ? g.nnz_total : g.nnz;
    bp.F = (int32_t)F;
    bp.H = (int32_t)H;
    bp.dh = (int32_t)dh;
    bp.mul = msg == kSrcMulEdge ? 1 : 0;
    bp.logR = logR;
    bp.nb = nb;
    bp.rows_per_group = (int32_t)((g.num_rows + kBinGroups - 1) / kBinGroups);
    const int32_t groups = (int32_t)((g.num_rows + bp.rows_per_group - 1) / bp.rows_per_group);
    FG_LAUNCH(fill_i32_kernel, stride_grid(nb), stream, bp.total, (int64_t)nb, 0);
    hipLaunchKernelGGL(bin_count_kernel, dim3((unsigned)groups), dim3(kBinThreads),
                       (size_t)nb * 4, stream, bp);
    hipLaunchKernelGGL(bin_scan_kernel, dim3(1), dim3(kBinScanThreads), 0, stream, bp);
    hipLaunchKernelGGL(bin_scatter_kernel, dim3((unsigned)groups), dim3(kBinThreads),
                       (size_t)nb * 8, stream, bp);
    const int64_t pieces = nb + (g.num_rows * F + kBinPiece - 1) / kBinPiece;
    hipLaunchKernelGGL(bin_accumulate_kernel, dim3((unsigned)pieces), dim3(kBinBlock), 0, stream,
                       bp);
    return hipGetLastError();
  }
  hipError_t err = zero_fill(gsrc, g.num_cols * F, stream);
  if (err != hipSuccess) return err;
  if ((err = zero_fill(gedge, g.nnz_total * H, stream)) != hipSuccess) return err;
  if (g.num_rows == 0 || g.nnz == 0 || (!gsrc && !gedge)) return hipSuccess;
  MaxBwdParams prm;
  prm.indices = g.indices;
  prm.eid_pos = g.edge_ids ? eid_pos : nullptr;
  prm.arg = arg;
  prm.go = go;
  prm.x = x;
  prm.ev = ev;
  prm.gsrc = gsrc;
  prm.gedge = gedge;
  prm.num_rows = g.num_rows;
  prm.F = F;
  prm.id_limit = g.edge_ids ? g.nnz_total : g.nnz;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.mul = msg == kSrcMulEdge ? 1 : 0;
  FG_LAUNCH(spmm_max_bwd_kernel, grid_for(g.num_rows, 1), stream, prm);
  return hipGetLastError();
}

hipError_t launch_edge_softmax_backward(const GraphView& g, const PlanView* plan, int64_t H,
                                        const float* a, const float* go, const float* scores,
                                        bool leaky, float slope, float* ds, hipStream_t stream) {
  if (g.num_rows == 0 || g.nnz == 0) return hipSuccess;
  SoftmaxBwdParams prm;
  prm.indptr = g.indptr;
  prm.eids = g.edge_ids;
  prm.a = a;
  prm.go = go;
  prm.s = scores;
  prm.ds = ds;
  prm.segs = plan ? plan->segs : nullptr;
  prm.fix = plan ? plan->fix : nullptr;
  prm.slot_fix = plan ? plan->slot_fix : nullptr;
  prm.slot_seg = plan ? plan->slot_seg : nullptr;
  prm.ws = plan ? plan->ws_f : nullptr;
  prm.n_items = plan ? plan->num_nonempty : g.num_rows;  // empty rows (last) need no work
  prm.H = (int32_t)H;
  prm.leaky = leaky ? 1 : 0;
  prm.slope = slope;
  prm.contig = (g.edge_ids == nullptr && H <= kWave && (H & (H - 1)) == 0 && aligned16(a) &&
                aligned16(go) && aligned16(ds) && (!leaky || aligned16(scores))) ? 1 : 0;
  const dim3 grid = grid_for(prm.n_items, 1);
  if (plan) FG_LAUNCH((softmax_bwd_kernel<true>), grid, stream, prm);
  else FG_LAUNCH((softmax_bwd_kernel<false>), grid, stream, prm);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !plan || plan->num_slots == 0) return err;
  FG_LAUNCH(softmax_bwd_split_kernel, grid_for(plan->num_slots, 1), stream, prm, plan->num_slots);
  return hipGetLastError();
}

}  // namespace fg

// Scratch of fg_gspmm_noalloc, for callers that cannot allocate device
// memory: the split-row partial values (and argmax edge ids) of one call.
// Every device holds its own copy from the library's load until the process
// ends; calls on one device share it, so calls that overlap in time on one
// device race.  Host code never passes this name to a kernel: on the host it
// is a stand-in, and the device address comes from noalloc_scratch().
static __device__ __align__(256) unsigned char scratch[fg::kNoAllocScratchBytes];

namespace fg {
namespace {
constexpr int kScratchDevices = 256;
std::mutex scratch_mu;
void* scratch_addr[kScratchDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    scratch_addr[dev] = p;
  }
  *ptr = scratch_addr[dev];
  return hipSuccess;
}

}  // namespace fg
