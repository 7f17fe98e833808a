// fg_kernels.hip -- gfx950 kernels for FeatGraph's generalized SpMM,
// generalized SDDMM and edge softmax.
//
// Work decomposition (all kernels): one 64-lane wavefront per work item, four
// wavefronts per workgroup.  A work item is either a whole CSR row (no plan)
// or a segment of a row taken from the plan's degree-aware schedule.  The
// feature dimension is spread across lanes (the paper binds it to threads,
// Sec. III-B GPU FDS and Sec. III-C vertex parallelization) with float4
// accesses, so one X row of 128 floats is one 512-byte request of 32 lanes and
// a wavefront works on 64/G edges at once, G = lanes per feature row.
// Neighbour indices (and edge values) of up to 64 edges are fetched with one
// coalesced load per lane and broadcast to the lanes that need them with
// cross-lane permutes.  SDDMM dot products reduce across the lanes of a
// feature row with xor butterflies (the paper's tree reduction, Fig. 4 FDS).
// No atomics: split rows write partial results that a second kernel merges in
// a fixed order, so every result is deterministic for a given plan.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

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

// ----------------------------------------------------------------------------
// generalized SpMM
// ----------------------------------------------------------------------------

struct SpmmParams {
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* eids;
  const float* x;
  const float* ev;
  float* out;
  int32_t* arg;
  const Seg* segs;
  float* ws_f;
  int32_t* ws_i;
  int64_t n_items;
  int64_t F;
  int32_t H;
  int32_t dh;
  int32_t logG;
};

// VEC: floats per lane access (4 or 1); NV: accesses per lane per edge (the
// feature chunk is G*VEC*NV floats, chunk index = blockIdx.y); U: edges in
// flight per lane group; MUL: src_mul_edge message; MAX: max/argmax reducer;
// SEG: items come from a plan.
template <int VEC, int NV, int U, bool MUL, bool MAX, bool SEG>
__global__ __launch_bounds__(kBlock) void spmm_kernel(SpmmParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  int64_t row, b, e;
  int32_t slot = -1;
  if constexpr (SEG) {
    const Seg s = p.segs[item];
    row = s.row; b = s.begin; e = s.end; slot = s.slot;
  } else {
    row = item; b = p.indptr[item]; e = p.indptr[item + 1];
  }
  const int lane = lane_id();
  const int G = 1 << p.logG;
  const int ngroups = kWave >> p.logG;
  const int gid = lane >> p.logG;
  const int li = lane & (G - 1);
  const int64_t F = p.F;
  const int64_t c0 = (int64_t)blockIdx.y * G * VEC * NV;

  int64_t f[NV];
  bool act[NV];
  int hv[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = c0 + (int64_t)(v * G + li) * VEC;
    act[v] = f[v] < F;
    hv[v] = (MUL && act[v]) ? (int)(f[v] / p.dh) : 0;
  }

  float acc[NV][VEC];
  int32_t am[NV][VEC];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int c = 0; c < VEC; ++c) {
      acc[v][c] = MAX ? -INFINITY : 0.0f;
      am[v][c] = INT_MAX;
    }

  for (int64_t base = b; base < e; base += kWave) {
    const int cnt = (int)min((int64_t)kWave, e - base);
    int my_src = 0, my_eid = 0;
    float my_w = 0.0f;
    if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
      if constexpr (MAX || MUL)
        my_eid = p.eids ? __builtin_nontemporal_load(p.eids + base + lane) : (int)(base + lane);
      if constexpr (MUL) {
        if (p.H == 1) my_w = p.ev[my_eid];
      }
    }
    for (int j0 = 0; j0 < cnt; j0 += ngroups * U) {
      float val[U][NV][VEC];
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
            load_vec<VEC>(xr + f[v], val[u][v]);
            wv[u][v] = (MUL && p.H != 1) ? p.ev[(int64_t)eu[u] * p.H + hv[v]] : w1;
          } else {
#pragma unroll
            for (int c = 0; c < VEC; ++c) val[u][v][c] = MAX ? -INFINITY : 0.0f;
            wv[u][v] = 1.0f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
#pragma unroll
          for (int c = 0; c < VEC; ++c) {
            if constexpr (MAX) {
              const float m = MUL ? wv[u][v] * val[u][v][c] : val[u][v][c];
              if (ok[u] && takes_over(m, eu[u], acc[v][c], am[v][c])) {
                acc[v][c] = m;
                am[v][c] = eu[u];
              }
            } else {
              if (MUL) acc[v][c] += wv[u][v] * val[u][v][c];
              else acc[v][c] += val[u][v][c];
            }
          }
        }
      }
    }
  }

  // merge the lane groups (each holds a strided subset of the edges)
  for (int s = G; s < kWave; s <<= 1) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int c = 0; c < VEC; ++c) {
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
  for (int v = 0; v < NV; ++v) {
    if (!act[v]) continue;
    if (SEG && slot >= 0) {
      store_vec<VEC>(p.ws_f + (int64_t)slot * F + f[v], acc[v]);
      if constexpr (MAX) store_vec_i<VEC>(p.ws_i + (int64_t)slot * F + f[v], am[v]);
    } else if constexpr (MAX) {
      float o[VEC];
      int32_t a[VEC];
#pragma unroll
      for (int c = 0; c < VEC; ++c) {
        const bool none = am[v][c] == INT_MAX;
        o[c] = none ? 0.0f : acc[v][c];
        a[c] = none ? -1 : am[v][c];
      }
      store_vec<VEC>(p.out + row * F + f[v], o);
      store_vec_i<VEC>(p.arg + row * F + f[v], a);
    } else {
      store_vec<VEC>(p.out + row * F + f[v], acc[v]);
    }
  }
}

// Merges the partial results of each split row, slot by slot in order.
template <bool MAX>
__global__ __launch_bounds__(256) void spmm_fixup_kernel(const Fix* fix, const float* ws_f,
                                                         const int32_t* ws_i, int64_t F,
                                                         float* out, int32_t* arg) {
  const int64_t f = (int64_t)blockIdx.y * 256 + threadIdx.x;
  if (f >= F) return;
  const Fix fx = fix[blockIdx.x];
  if constexpr (MAX) {
    float best = -INFINITY;
    int32_t be = INT_MAX;
    for (int s = fx.slot_begin; s < fx.slot_end; ++s) {
      const float m = ws_f[(int64_t)s * F + f];
      const int32_t a = ws_i[(int64_t)s * F + f];
      if (takes_over(m, a, best, be)) {
        best = m;
        be = a;
      }
    }
    const bool none = be == INT_MAX;
    out[(int64_t)fx.row * F + f] = none ? 0.0f : best;
    arg[(int64_t)fx.row * F + f] = none ? -1 : be;
  } else {
    float acc = 0.0f;
    for (int s = fx.slot_begin; s < fx.slot_end; ++s) acc += ws_f[(int64_t)s * F + f];
    out[(int64_t)fx.row * F + f] = acc;
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
  int64_t F;
  int32_t H;
  int32_t dh;
  int32_t logG;  // lanes per feature row
  int32_t logS;  // lanes per head (HEADED only)
};

// The destination row's features stay in registers for the whole item; each
// edge gathers its source row, multiplies, and reduces across the lanes of one
// head with xor butterflies.  Requires the whole row in one chunk
// (F <= G*VEC*NV) and, when HEADED, dh/VEC = 2^logS lanes per head.
template <int VEC, int NV, int U, bool HEADED, bool SEG>
__global__ __launch_bounds__(kBlock) void sddmm_kernel(SddmmParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  int64_t row, b, e;
  if constexpr (SEG) {
    const Seg s = p.segs[item];
    row = s.row; b = s.begin; e = s.end;
  } else {
    row = item; b = p.indptr[item]; e = p.indptr[item + 1];
  }
  if (b >= e) return;
  const int lane = lane_id();
  const int G = 1 << p.logG;
  const int ngroups = kWave >> p.logG;
  const int gid = lane >> p.logG;
  const int li = lane & (G - 1);
  const int S = HEADED ? (1 << p.logS) : G;
  const int64_t F = p.F;

  int64_t f[NV];
  bool act[NV];
  float xd[NV][VEC];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    f[v] = (int64_t)(v * G + li) * VEC;
    act[v] = f[v] < F;
    if (act[v]) {
      load_vec<VEC>(p.xd + row * F + f[v], xd[v]);
    } else {
#pragma unroll
      for (int c = 0; c < VEC; ++c) xd[v][c] = 0.0f;
    }
  }

  for (int64_t base = b; base < e; base += kWave) {
    const int cnt = (int)min((int64_t)kWave, e - base);
    int my_src = 0, my_eid = 0;
    if (lane < cnt) {
      my_src = __builtin_nontemporal_load(p.indices + base + lane);
      my_eid = p.eids ? __builtin_nontemporal_load(p.eids + base + lane) : (int)(base + lane);
    }
    for (int j0 = 0; j0 < cnt; j0 += ngroups * U) {
      float val[U][NV][VEC];
      int32_t eu[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * ngroups + gid;
        ok[u] = j < cnt;
        const int jl = j & (kWave - 1);
        const int src = __shfl(my_src, jl);
        eu[u] = __shfl(my_eid, jl);
        const float* xr = p.xs + (int64_t)src * F;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if (ok[u] && act[v]) {
            load_vec<VEC>(xr + f[v], val[u][v]);
          } else {
#pragma unroll
            for (int c = 0; c < VEC; ++c) val[u][v][c] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if constexpr (!HEADED) {
          float part = 0.0f;
#pragma unroll
          for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int c = 0; c < VEC; ++c) part += val[u][v][c] * xd[v][c];
          for (int s = 1; s < G; s <<= 1) part += __shfl_xor(part, s);
          if (ok[u] && li == 0) p.out[eu[u]] = part;
        } else {
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            float part = 0.0f;
#pragma unroll
            for (int c = 0; c < VEC; ++c) part += val[u][v][c] * xd[v][c];
            for (int s = 1; s < S; s <<= 1) part += __shfl_xor(part, s);
            if (ok[u] && act[v] && (li & (S - 1)) == 0)
              p.out[(int64_t)eu[u] * p.H + f[v] / p.dh] = part;
          }
        }
      }
    }
  }
}

// Fallback for shapes the lane mapping above does not cover (odd head sizes,
// very wide rows): one lane per (edge, head) pair, sequential dot product.
template <bool SEG>
__global__ __launch_bounds__(kBlock) void sddmm_generic_kernel(SddmmParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  int64_t row, b, e;
  if constexpr (SEG) {
    const Seg s = p.segs[item];
    row = s.row; b = s.begin; e = s.end;
  } else {
    row = item; b = p.indptr[item]; e = p.indptr[item + 1];
  }
  const int lane = lane_id();
  const int64_t H = p.H, dh = p.dh, F = p.F;
  const int64_t total = (e - b) * H;
  for (int64_t t = lane; t < total; t += kWave) {
    const int64_t q = b + t / H;
    const int64_t h = t % H;
    const int64_t src = p.indices[q];
    const int64_t eid = p.eids ? p.eids[q] : q;
    const float* a = p.xs + src * F + h * dh;
    const float* d = p.xd + row * F + h * dh;
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
  float* ws;  // [slot][H][2] = (running max, scaled sum)
  int64_t n_items;
  int32_t H;
  int32_t leaky;
  float slope;
};

__device__ __forceinline__ float leaky_relu(float s, int on, float slope) {
  return (on && !(s > 0.0f)) ? slope * s : s;
}

// (m, z) represents sum_i exp(x_i - m) = z.  Combining two such pairs.
__device__ __forceinline__ void lse_merge(float& m, float& z, float om, float oz) {
  if (om == -INFINITY) return;
  if (m == -INFINITY) {
    m = om;
    z = oz;
    return;
  }
  const float nm = fmaxf(m, om);
  z = z * expf(m - nm) + oz * expf(om - nm);
  m = nm;
}

// Lanes map to (edge offset, head) pairs: hc = heads per pass, epw = 64/hc
// edges per pass.  Pass 1 keeps a running (max, sum); lanes of one head then
// merge in a fixed tree; pass 2 writes exp(s' - m) / z.  Segments of split
// rows stop after pass 1 and leave (m, z) in the workspace.
template <bool SEG>
__global__ __launch_bounds__(kBlock) void softmax_kernel(SoftmaxParams p) {
  const int64_t item = wave_item();
  if (item >= p.n_items) return;
  int64_t row, b, e;
  int32_t slot = -1;
  if constexpr (SEG) {
    const Seg s = p.segs[item];
    row = s.row; b = s.begin; e = s.end; slot = s.slot;
  } else {
    row = item; b = p.indptr[item]; e = p.indptr[item + 1];
  }
  (void)row;
  if (b >= e) return;
  const int lane = lane_id();
  const int H = p.H;
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int h = h0 + lane % hc;
    const bool active = eo < epw;
    float m = -INFINITY, z = 0.0f;
    if (active) {
      for (int64_t q = b + eo; q < e; q += epw) {
        const int64_t eid = p.eids ? p.eids[q] : q;
        const float s = leaky_relu(p.scores[eid * H + h], p.leaky, p.slope);
        if (s > m) {
          z = z * expf(m - s) + 1.0f;
          m = s;
        } else {
          z += expf(s - m);
        }
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
    if (SEG && slot >= 0) {
      if (active && eo == 0) {
        p.ws[((int64_t)slot * H + h) * 2 + 0] = m;
        p.ws[((int64_t)slot * H + h) * 2 + 1] = z;
      }
      continue;
    }
    if (active) {
      const float inv = 1.0f / z;
      for (int64_t q = b + eo; q < e; q += epw) {
        const int64_t eid = p.eids ? p.eids[q] : q;
        const float s = leaky_relu(p.scores[eid * H + h], p.leaky, p.slope);
        p.out[eid * H + h] = expf(s - m) * inv;
      }
    }
  }
}

// Second pass for segments of split rows: merge the row's (m, z) partials in
// slot order, then normalise this segment's edges.  Item = slot.
__global__ __launch_bounds__(kBlock) void softmax_split_kernel(SoftmaxParams p, int64_t n_slots) {
  const int64_t slot = wave_item();
  if (slot >= n_slots) return;
  const Seg s = p.segs[slot];
  const Fix fx = p.fix[p.slot_fix[slot]];
  const int lane = lane_id();
  const int H = p.H;
  for (int h0 = 0; h0 < H; h0 += kWave) {
    const int hc = min(H - h0, kWave);
    const int epw = kWave / hc;
    const int eo = lane / hc;
    const int h = h0 + lane % hc;
    if (eo >= epw) continue;
    float m = -INFINITY, z = 0.0f;
    for (int t = fx.slot_begin; t < fx.slot_end; ++t)
      lse_merge(m, z, p.ws[((int64_t)t * H + h) * 2 + 0], p.ws[((int64_t)t * H + h) * 2 + 1]);
    const float inv = 1.0f / z;
    for (int64_t q = s.begin + eo; q < s.end; q += epw) {
      const int64_t eid = p.eids ? p.eids[q] : q;
      const float sc = leaky_relu(p.scores[eid * H + h], p.leaky, p.slope);
      p.out[eid * H + h] = expf(sc - m) * inv;
    }
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

template <int VEC, int NV, int U, bool MUL, bool MAX>
void spmm_go(const SpmmParams& prm, bool seg, dim3 grid, hipStream_t st) {
  if (seg)
    hipLaunchKernelGGL((spmm_kernel<VEC, NV, U, MUL, MAX, true>), grid, dim3(kBlock), 0, st, prm);
  else
    hipLaunchKernelGGL((spmm_kernel<VEC, NV, U, MUL, MAX, false>), grid, dim3(kBlock), 0, st, prm);
}

template <int VEC, int NV, int U>
void spmm_ops(const SpmmParams& prm, bool mul, bool mx, bool seg, dim3 grid, hipStream_t st) {
  if (mul) {
    if (mx) spmm_go<VEC, NV, U, true, true>(prm, seg, grid, st);
    else spmm_go<VEC, NV, U, true, false>(prm, seg, grid, st);
  } else {
    if (mx) spmm_go<VEC, NV, U, false, true>(prm, seg, grid, st);
    else spmm_go<VEC, NV, U, false, false>(prm, seg, grid, st);
  }
}

template <int VEC>
void spmm_nv(const SpmmParams& prm, int nv, bool mul, bool mx, bool seg, dim3 grid,
             hipStream_t st) {
  if (nv == 1) spmm_ops<VEC, 1, 4>(prm, mul, mx, seg, grid, st);
  else if (nv == 2) spmm_ops<VEC, 2, 2>(prm, mul, mx, seg, grid, st);
  else spmm_ops<VEC, 4, 1>(prm, mul, mx, seg, grid, st);
}

template <int VEC, int NV, int U, bool HEADED>
void sddmm_go(const SddmmParams& prm, bool seg, dim3 grid, hipStream_t st) {
  if (seg)
    hipLaunchKernelGGL((sddmm_kernel<VEC, NV, U, HEADED, true>), grid, dim3(kBlock), 0, st, prm);
  else
    hipLaunchKernelGGL((sddmm_kernel<VEC, NV, U, HEADED, false>), grid, dim3(kBlock), 0, st, prm);
}

template <int VEC>
void sddmm_nv(const SddmmParams& prm, int nv, bool headed, bool seg, dim3 grid, hipStream_t st) {
  if (headed) {
    if (nv == 1) sddmm_go<VEC, 1, 4, true>(prm, seg, grid, st);
    else if (nv == 2) sddmm_go<VEC, 2, 2, true>(prm, seg, grid, st);
    else sddmm_go<VEC, 4, 1, true>(prm, seg, grid, st);
  } else {
    if (nv == 1) sddmm_go<VEC, 1, 4, false>(prm, seg, grid, st);
    else if (nv == 2) sddmm_go<VEC, 2, 2, false>(prm, seg, grid, st);
    else sddmm_go<VEC, 4, 1, false>(prm, seg, grid, st);
  }
}

}  // namespace

hipError_t launch_gspmm(const GraphView& g, const PlanView* plan, int msg, int red, int64_t H,
                        int64_t dh, const float* x, const float* ev, float* out, int32_t* arg,
                        hipStream_t stream) {
  if (g.num_rows == 0) return hipSuccess;
  const int64_t F = H * dh;
  const bool mul = msg == kSrcMulEdge;
  const bool mx = red == kMax;
  const bool vec4 = (F % 4 == 0) && (H == 1 || dh % 4 == 0) && aligned16(x) && aligned16(out) &&
                    (!mx || aligned16(arg));
  const int VEC = vec4 ? 4 : 1;
  const int64_t Q = F / VEC;
  int logG, nv;
  int64_t chunks = 1;
  if (Q <= kWave) {
    logG = ilog2_ceil(Q);
    nv = 1;
  } else {
    logG = 6;
    nv = Q <= 2 * kWave ? 2 : 4;
    chunks = (Q + (int64_t)kWave * nv - 1) / ((int64_t)kWave * nv);
  }
  SpmmParams prm;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.eids = g.edge_ids;
  prm.x = x;
  prm.ev = ev;
  prm.out = out;
  prm.arg = arg;
  prm.segs = plan ? plan->segs : nullptr;
  prm.ws_f = plan ? plan->ws_f : nullptr;
  prm.ws_i = plan ? plan->ws_i : nullptr;
  prm.n_items = plan ? plan->num_segments : g.num_rows;
  prm.F = F;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.logG = logG;
  const bool seg = plan != nullptr;
  const dim3 grid = grid_for(prm.n_items, chunks);
  if (vec4) spmm_nv<4>(prm, nv, mul, mx, seg, grid, stream);
  else spmm_nv<1>(prm, nv, mul, mx, seg, grid, stream);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (plan && plan->num_split_rows > 0) {
    const dim3 fgrid((unsigned)plan->num_split_rows, (unsigned)((F + 255) / 256), 1);
    if (mx)
      hipLaunchKernelGGL((spmm_fixup_kernel<true>), fgrid, dim3(256), 0, stream, plan->fix,
                         plan->ws_f, plan->ws_i, F, out, arg);
    else
      hipLaunchKernelGGL((spmm_fixup_kernel<false>), fgrid, dim3(256), 0, stream, plan->fix,
                         plan->ws_f, plan->ws_i, F, out, arg);
    err = hipGetLastError();
  }
  return err;
}

hipError_t launch_gsddmm(const GraphView& g, const PlanView* plan, int64_t H, int64_t dh,
                         const float* xs, const float* xd, float* out, hipStream_t stream) {
  if (g.num_rows == 0 || g.nnz == 0) return hipSuccess;
  const int64_t F = H * dh;
  const bool vec4 = (F % 4 == 0) && (H == 1 || dh % 4 == 0) && aligned16(xs) && aligned16(xd);
  const int VEC = vec4 ? 4 : 1;
  const int64_t Q = F / VEC;
  const bool headed = H > 1;
  int logS = 0;
  bool generic = Q > 4 * kWave;
  if (headed) {
    const int64_t S = dh / VEC;
    logS = ilog2_ceil(S);
    if ((int64_t(1) << logS) != S || S > kWave) generic = true;
  }
  int logG = 6, nv = 1;
  if (Q <= kWave) {
    logG = ilog2_ceil(Q);
  } else {
    nv = Q <= 2 * kWave ? 2 : 4;
  }
  SddmmParams prm;
  prm.indptr = g.indptr;
  prm.indices = g.indices;
  prm.eids = g.edge_ids;
  prm.xs = xs;
  prm.xd = xd;
  prm.out = out;
  prm.segs = plan ? plan->segs : nullptr;
  prm.n_items = plan ? plan->num_segments : g.num_rows;
  prm.F = F;
  prm.H = (int32_t)H;
  prm.dh = (int32_t)dh;
  prm.logG = logG;
  prm.logS = logS;
  const bool seg = plan != nullptr;
  const dim3 grid = grid_for(prm.n_items, 1);
  if (generic) {
    if (seg) hipLaunchKernelGGL((sddmm_generic_kernel<true>), grid, dim3(kBlock), 0, stream, prm);
    else hipLaunchKernelGGL((sddmm_generic_kernel<false>), grid, dim3(kBlock), 0, stream, prm);
  } else if (vec4) {
    sddmm_nv<4>(prm, nv, headed, seg, grid, stream);
  } else {
    sddmm_nv<1>(prm, nv, headed, seg, grid, stream);
  }
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
  prm.ws = plan ? plan->ws_f : nullptr;
  prm.n_items = plan ? plan->num_segments : g.num_rows;
  prm.H = (int32_t)H;
  prm.leaky = leaky ? 1 : 0;
  prm.slope = slope;
  const dim3 grid = grid_for(prm.n_items, 1);
  if (plan) hipLaunchKernelGGL((softmax_kernel<true>), grid, dim3(kBlock), 0, stream, prm);
  else hipLaunchKernelGGL((softmax_kernel<false>), grid, dim3(kBlock), 0, stream, prm);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !plan || plan->num_slots == 0) return err;
  hipLaunchKernelGGL(softmax_split_kernel, grid_for(plan->num_slots, 1), dim3(kBlock), 0, stream,
                     prm, plan->num_slots);
  return hipGetLastError();
}

}  // namespace fg
