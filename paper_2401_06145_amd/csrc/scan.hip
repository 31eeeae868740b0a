// Device-wide exclusive prefix sum of uint32 values.  Up to 16384 values run in
// one workgroup (1024 threads x 16 values); larger inputs use tile sums -> scan
// of the sums -> tile scan with a base.  Used for the radix-sort digit offsets,
// the unique-coordinate compaction of Eq. 1, and the work-item and match
// offsets of the double-traversed binary search (Section 5.1.2).
#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 1024;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;
constexpr int kWaves = kThreads / kWave;

// Exclusive scan of one value per thread across the workgroup; *total gets the sum.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_wave, uint32_t* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, kWave);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) s_wave[wave] = x;
  __syncthreads();
  if (wave == 0) {
    uint32_t s = (lane < kWaves) ? s_wave[lane] : 0u;
    uint32_t incl = s;
#pragma unroll
    for (int d = 1; d < kWaves; d <<= 1) {
      const uint32_t y = __shfl_up(incl, d, kWave);
      if (lane >= d) incl += y;
    }
    if (lane < kWaves) s_wave[kWaves + lane] = incl - s;  // exclusive wave prefix
    if (lane == kWaves - 1) s_wave[2 * kWaves] = incl;
  }
  __syncthreads();
  const uint32_t before = s_wave[kWaves + wave];
  *total = s_wave[2 * kWaves];
  __syncthreads();  // s_wave is reused by the caller's next scan
  return before + x - v;
}

// Loads kItems consecutive values of the tile for this thread (zeros past n).
__device__ __forceinline__ void load_items(const uint32_t* in, int64_t n, int64_t first, uint32_t v[kItems]) {
  if (first + kItems <= n && ((reinterpret_cast<uintptr_t>(in + first) & 15) == 0)) {
    const uint4* p = reinterpret_cast<const uint4*>(in + first);
#pragma unroll
    for (int q = 0; q < kItems / 4; ++q) {
      const uint4 u = p[q];
      v[4 * q] = u.x;
      v[4 * q + 1] = u.y;
      v[4 * q + 2] = u.z;
      v[4 * q + 3] = u.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kItems; ++i) v[i] = (first + i < n) ? in[first + i] : 0u;
  }
}

__global__ __launch_bounds__(kThreads) void k_tile_reduce(const uint32_t* in, int64_t n, uint32_t* sums) {
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  uint32_t v[kItems];
  load_items(in, n, (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems, v);
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) acc += v[i];
  uint32_t total;
  block_excl_scan(acc, s_wave, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// out may alias in (each value is read, then written, by the same thread).
__global__ __launch_bounds__(kThreads) void k_tile_scan(const uint32_t* in, uint32_t* out, int64_t n,
                                                        const uint32_t* tile_base, uint32_t* d_total) {
  __shared__ uint32_t s_wave[2 * kWaves + 1];
  const int64_t first = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
  uint32_t v[kItems];
  load_items(in, n, first, v);
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) acc += v[i];
  uint32_t total;
  uint32_t run = block_excl_scan(acc, s_wave, &total) + (tile_base ? tile_base[blockIdx.x] : 0u);
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const uint32_t t = v[i];
    v[i] = run;
    run += t;
  }
  if (first + kItems <= n && ((reinterpret_cast<uintptr_t>(out + first) & 15) == 0)) {
    uint4* p = reinterpret_cast<uint4*>(out + first);
#pragma unroll
    for (int q = 0; q < kItems / 4; ++q) p[q] = make_uint4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  } else {
#pragma unroll
    for (int i = 0; i < kItems; ++i)
      if (first + i < n) out[first + i] = v[i];
  }
  if (d_total && blockIdx.x == gridDim.x - 1 && threadIdx.x == kThreads - 1) *d_total = run;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

size_t scan_temp_bytes(int64_t n) {
  if (n <= kTile) return 0;
  const int64_t nt = (n + kTile - 1) / kTile;
  return align256((size_t)nt * sizeof(uint32_t)) + scan_temp_bytes(nt);
}

namespace {
hipError_t scan_impl(const uint32_t* d_in, uint32_t* d_out, int64_t n, uint32_t* d_total, void* d_temp,
                     hipStream_t s) {
  if (n <= kTile) {
    hipLaunchKernelGGL(k_tile_scan, dim3(1), dim3(kThreads), 0, s, d_in, d_out, n, nullptr, d_total);
    return hipGetLastError();
  }
  const int64_t nt = (n + kTile - 1) / kTile;
  uint32_t* sums = static_cast<uint32_t*>(d_temp);
  void* rest = static_cast<char*>(d_temp) + align256((size_t)nt * sizeof(uint32_t));
  hipLaunchKernelGGL(k_tile_reduce, dim3((unsigned)nt), dim3(kThreads), 0, s, d_in, n, sums);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = scan_impl(sums, sums, nt, nullptr, rest, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_tile_scan, dim3((unsigned)nt), dim3(kThreads), 0, s, d_in, d_out, n, sums, d_total);
  return hipGetLastError();
}
}  // namespace

hipError_t scan_exclusive_u32(const uint32_t* d_in, uint32_t* d_out, int64_t n, uint32_t* d_total,
                              void* d_temp, hipStream_t s) {
  if (n <= 0) {
    if (d_total) return launch_fill_u32(d_total, 0u, 1, s);
    return hipSuccess;
  }
  ProfScope ps(KN_SCAN, s);
  return scan_impl(d_in, d_out, n, d_total, d_temp, s);
}

}  // namespace spc
