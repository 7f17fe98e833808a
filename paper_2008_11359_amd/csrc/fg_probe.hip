// fg_probe.hip -- measurement probe, not part of the library's ABI: the
// per-compute-unit cost of one vector-memory gather instruction when the data
// is cache-resident, i.e. the floor that the gather path (texture addresser
// and data return) sets under the sparse kernels whatever the memory
// hierarchy behind it delivers.  Built into its own shared library
// (_build/libfg_probe.so) and run by `bench.py --gather-floor`, which also
// times a read-only stream over a buffer four times the Infinity Cache.
//
// Each wavefront issues `iters` float4 loads in batches of 8 independent
// loads; lane l of a wavefront reads float4 (l % 32) of a 512-byte row, so one
// instruction fetches two rows (1 KiB), the lane layout of the gSpMM / gSDDMM
// kernels at 128 features.  Rows come from a register hash (no dependent index
// loads) over a table of `rows` rows that the caches hold.  Only the first
// `active` lanes load (the rest are masked off), which shows whether the cost
// is per instruction or per lane.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;
constexpr int kBatch = 8;

__global__ __launch_bounds__(kBlock) void gather_floor_kernel(const float4* __restrict__ x,
                                                              uint32_t row_mask,
                                                              float4* __restrict__ out,
                                                              int iters, int active,
                                                              unsigned long long* clocks) {
  const int lane = threadIdx.x & 63;
  const uint32_t wave = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  uint64_t t0 = 0, r0 = 0;
  const bool timer = blockIdx.x == 0 && threadIdx.x == 0;
  if (timer) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int it = 0; it < iters; it += kBatch) {
    float4 v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const uint32_t h = (uint32_t)(it + j) * 2654435761u ^ (wave * 2246822519u) ^
                         ((uint32_t)(lane >> 5) * 3266489917u);
      const uint32_t row = (h ^ (h >> 15)) & row_mask;
      v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (lane < active) v[j] = x[(size_t)row * 32 + (lane & 31)];
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      acc.x += v[j].x;
      acc.y += v[j].y;
      acc.z += v[j].z;
      acc.w += v[j].w;
    }
  }
  out[(size_t)blockIdx.x * kBlock + threadIdx.x] = acc;
  if (timer) {
    clocks[0] = __builtin_amdgcn_s_memtime() - t0;
    clocks[1] = __builtin_amdgcn_s_memrealtime() - r0;
  }
}

// Read-only stream: every thread sums its float4s of a large buffer
// (grid-stride, 8 loads in flight); the attainable rate of reads alone.
__global__ __launch_bounds__(kBlock) void read_stream_kernel(const float4* __restrict__ x,
                                                             size_t n, float4* __restrict__ out) {
  const size_t stride = (size_t)gridDim.x * kBlock;
  size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (; i + (kBatch - 1) * stride < n; i += kBatch * stride) {
    float4 v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) v[j] = x[i + j * stride];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      acc.x += v[j].x;
      acc.y += v[j].y;
      acc.z += v[j].z;
      acc.w += v[j].w;
    }
  }
  for (; i < n; i += stride) {
    const float4 v = x[i];
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  out[(size_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

// Chunked read: wavefront w reads float4s [w * chunk, (w + 1) * chunk) of the
// buffer, 8 per lane in flight, then exits (the access pattern of a kernel
// that gives each wavefront one contiguous range).
__global__ __launch_bounds__(kBlock) void read_chunks_kernel(const float4* __restrict__ x,
                                                             size_t n, size_t chunk,
                                                             float4* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const size_t wave = (size_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const size_t b = wave * chunk;
  const size_t e = b + chunk < n ? b + chunk : n;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (size_t k0 = b + lane; k0 < e; k0 += kBatch * 64) {
    float4 v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const size_t k = k0 + (size_t)j * 64;
      v[j] = k < e ? x[k] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      acc.x += v[j].x;
      acc.y += v[j].y;
      acc.z += v[j].z;
      acc.w += v[j].w;
    }
  }
  out[(size_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

// Scattered 8-byte record writes, the pattern of a counting-sort scatter:
// `groups` workgroups of 1024 threads each own `per_group` consecutive
// elements; element i goes to bin hash(i) % bins, at the next position of its
// group's run in that bin (ranked by an LDS atomic).  Runs have a fixed
// capacity `cap` (records beyond it are dropped), laid out bin-major, so the
// runs of one bin are adjacent as in the real sort.
__global__ __launch_bounds__(1024) void scatter_runs_kernel(int2* __restrict__ rec, int per_group,
                                                            int bins, int cap) {
  extern __shared__ int32_t cnt[];
  for (int b = threadIdx.x; b < bins; b += 1024) cnt[b] = 0;
  __syncthreads();
  const int64_t first = (int64_t)blockIdx.x * per_group;
  for (int t = threadIdx.x; t < per_group; t += 1024) {
    const uint32_t i = (uint32_t)(first + t);
    uint32_t h = i * 2654435761u;
    h ^= h >> 16;
    h *= 2246822519u;
    h ^= h >> 13;
    const int b = (int)(h % (uint32_t)bins);
    const int r = atomicAdd(&cnt[b], 1);
    if (r < cap)
      rec[((int64_t)b * gridDim.x + blockIdx.x) * cap + r] = make_int2((int)i, (int)h);
  }
}

}  // namespace

extern "C" {

// Times scatter_runs_kernel (`reps` launches after one warm-up); the record
// array holds groups * bins * cap records.  Allocates and frees its buffers.
int fgp_scatter_runs(int groups, int per_group, int bins, int cap, int reps, float* ms_out) {
  if (groups < 1 || per_group < 1 || bins < 1 || bins > 16384 || cap < 1 || reps < 1 || !ms_out)
    return -1;
  int2* rec = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = -2;
  const size_t n = (size_t)groups * bins * cap;
  if (hipMalloc(&rec, n * sizeof(int2)) != hipSuccess || hipEventCreate(&e0) != hipSuccess ||
      hipEventCreate(&e1) != hipSuccess)
    goto done;
  scatter_runs_kernel<<<groups, 1024, (size_t)bins * 4>>>(rec, per_group, bins, cap);
  if (hipEventRecord(e0) != hipSuccess) goto done;
  for (int r = 0; r < reps; ++r)
    scatter_runs_kernel<<<groups, 1024, (size_t)bins * 4>>>(rec, per_group, bins, cap);
  if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) goto done;
  {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) goto done;
    *ms_out = ms / (float)reps;
    rc = hipGetLastError() == hipSuccess ? 0 : -3;
  }
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (rec) (void)hipFree(rec);
  return rc;
}

// Reads a buffer of `bytes` in contiguous chunks of `chunk_bytes` (both
// multiples of 16), one per wavefront, `reps` times after a warm-up; writes
// the mean time per pass (ms).  Allocates and frees its own buffers.
int fgp_read_chunks(size_t bytes, size_t chunk_bytes, int reps, float* ms_out) {
  if (bytes < 16 || bytes % 16 != 0 || chunk_bytes < 16 || chunk_bytes % 16 != 0 || reps < 1 ||
      !ms_out)
    return -1;
  const size_t n = bytes / 16, chunk = chunk_bytes / 16;
  const size_t waves = (n + chunk - 1) / chunk;
  const size_t blocks = (waves + 3) / 4;
  if (blocks > (size_t)INT32_MAX) return -1;
  float4 *x = nullptr, *out = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = -2;
  if (hipMalloc(&x, bytes) != hipSuccess ||
      hipMalloc(&out, blocks * kBlock * sizeof(float4)) != hipSuccess ||
      hipMemset(x, 0, bytes) != hipSuccess || hipEventCreate(&e0) != hipSuccess ||
      hipEventCreate(&e1) != hipSuccess)
    goto done;
  read_chunks_kernel<<<(unsigned)blocks, kBlock>>>(x, n, chunk, out);
  if (hipEventRecord(e0) != hipSuccess) goto done;
  for (int r = 0; r < reps; ++r) read_chunks_kernel<<<(unsigned)blocks, kBlock>>>(x, n, chunk, out);
  if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) goto done;
  {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) goto done;
    *ms_out = ms / (float)reps;
    rc = hipGetLastError() == hipSuccess ? 0 : -3;
  }
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (out) (void)hipFree(out);
  if (x) (void)hipFree(x);
  return rc;
}

// Reads a buffer of `bytes` (a multiple of 16) `reps` times after one
// warm-up pass with `blocks` workgroups; writes the mean time per pass (ms).
// Allocates and frees its own buffers.  0 on success.
int fgp_read_stream(size_t bytes, int blocks, int reps, float* ms_out) {
  if (bytes < 16 || bytes % 16 != 0 || blocks < 1 || reps < 1 || !ms_out) return -1;
  float4 *x = nullptr, *out = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = -2;
  const size_t n = bytes / 16;
  if (hipMalloc(&x, bytes) != hipSuccess ||
      hipMalloc(&out, (size_t)blocks * kBlock * sizeof(float4)) != hipSuccess ||
      hipMemset(x, 0, bytes) != hipSuccess || hipEventCreate(&e0) != hipSuccess ||
      hipEventCreate(&e1) != hipSuccess)
    goto done;
  read_stream_kernel<<<blocks, kBlock>>>(x, n, out);
  if (hipEventRecord(e0) != hipSuccess) goto done;
  for (int r = 0; r < reps; ++r) read_stream_kernel<<<blocks, kBlock>>>(x, n, out);
  if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) goto done;
  {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) goto done;
    *ms_out = ms / (float)reps;
    rc = hipGetLastError() == hipSuccess ? 0 : -3;
  }
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (out) (void)hipFree(out);
  if (x) (void)hipFree(x);
  return rc;
}

// Runs the probe `reps` times after one warm-up launch: `blocks` workgroups
// of 4 wavefronts, `iters` loads per wavefront (a multiple of 8), a table of
// `rows` (a power of two) 512-byte rows.  Writes the mean launch time (ms)
// and the shader-clock and 100 MHz real-time ticks that wavefront 0 counted
// during its last launch.  Allocates and frees its own buffers.  0 on success.
int fgp_gather_floor(int rows, int blocks, int iters, int active, int reps, float* ms_out,
                     unsigned long long* clock_ticks, unsigned long long* real_ticks) {
  if (rows < 1 || (rows & (rows - 1)) != 0 || blocks < 1 || iters < kBatch ||
      iters % kBatch != 0 || active < 1 || active > 64 || reps < 1 || !ms_out)
    return -1;
  float4 *x = nullptr, *out = nullptr;
  unsigned long long* clocks = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = -2;
  if (hipMalloc(&x, (size_t)rows * 512) != hipSuccess ||
      hipMalloc(&out, (size_t)blocks * kBlock * sizeof(float4)) != hipSuccess ||
      hipMalloc(&clocks, 2 * sizeof(unsigned long long)) != hipSuccess ||
      hipMemset(x, 0, (size_t)rows * 512) != hipSuccess ||
      hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess)
    goto done;
  gather_floor_kernel<<<blocks, kBlock>>>(x, (uint32_t)(rows - 1), out, iters, active, clocks);
  if (hipEventRecord(e0) != hipSuccess) goto done;
  for (int r = 0; r < reps; ++r)
    gather_floor_kernel<<<blocks, kBlock>>>(x, (uint32_t)(rows - 1), out, iters, active, clocks);
  if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) goto done;
  {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) goto done;
    *ms_out = ms / (float)reps;
    unsigned long long h[2] = {0, 0};
    if (hipMemcpy(h, clocks, sizeof(h), hipMemcpyDeviceToHost) != hipSuccess) goto done;
    if (clock_ticks) *clock_ticks = h[0];
    if (real_ticks) *real_ticks = h[1];
    rc = hipGetLastError() == hipSuccess ? 0 : -3;
  }
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (clocks) (void)hipFree(clocks);
  if (out) (void)hipFree(out);
  if (x) (void)hipFree(x);
  return rc;
}

}  // extern "C"
