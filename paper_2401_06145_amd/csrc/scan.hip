// Device-wide exclusive prefix sum of uint32 values (tile reduce -> scan of tile
// sums -> tile scan with base).  Used for radix-sort digit offsets, for the
// unique-coordinate compaction of Eq. 1, and for the query-block balancing step
// of Section 5.1.2.
#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 256;
constexpr int kRounds = 16;
constexpr int kTile = kThreads * kRounds;  // 4096 values per workgroup

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
  uint32_t before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < kThreads / kWave; ++w) {
    const uint32_t s = s_wave[w];
    before += (w < wave) ? s : 0u;
    sum += s;
  }
  __syncthreads();  // s_wave is reused by the next call
  *total = sum;
  return before + x - v;
}

__global__ __launch_bounds__(kThreads) void k_tile_reduce(const uint32_t* in, int64_t n, uint32_t* sums) {
  __shared__ uint32_t s_wave[kThreads / kWave];
  const int64_t base = (int64_t)blockIdx.x * kTile;
  uint32_t acc = 0;
#pragma unroll 4
  for (int r = 0; r < kRounds; ++r) {
    const int64_t i = base + r * kThreads + threadIdx.x;
    acc += (i < n) ? in[i] : 0u;
  }
  uint32_t total;
  block_excl_scan(acc, s_wave, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// out may alias in (each element is read and written by the same thread).
__global__ __launch_bounds__(kThreads) void k_tile_scan(const uint32_t* in, uint32_t* out, int64_t n,
                                                        const uint32_t* tile_base, uint32_t* d_total) {
  __shared__ uint32_t s_wave[kThreads / kWave];
  const int64_t base = (int64_t)blockIdx.x * kTile;
  uint32_t carry = tile_base ? tile_base[blockIdx.x] : 0u;
  for (int r = 0; r < kRounds; ++r) {
    const int64_t i = base + r * kThreads + threadIdx.x;
    const uint32_t v = (i < n) ? in[i] : 0u;
    uint32_t round_total;
    const uint32_t ex = block_excl_scan(v, s_wave, &round_total);
    if (i < n) out[i] = carry + ex;
    carry += round_total;
  }
  if (d_total && threadIdx.x == 0 && blockIdx.x == gridDim.x - 1) *d_total = carry;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

size_t scan_temp_bytes(int64_t n) {
  if (n <= kTile) return 0;
  const int64_t nt = (n + kTile - 1) / kTile;
  return align256((size_t)nt * sizeof(uint32_t)) + scan_temp_bytes(nt);
}

hipError_t scan_exclusive_u32(const uint32_t* d_in, uint32_t* d_out, int64_t n, uint32_t* d_total,
                              void* d_temp, hipStream_t s) {
  if (n <= 0) {
    if (d_total) return launch_fill_u32(d_total, 0u, 1, s);
    return hipSuccess;
  }
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
  e = scan_exclusive_u32(sums, sums, nt, nullptr, rest, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_tile_scan, dim3((unsigned)nt), dim3(kThreads), 0, s, d_in, d_out, n, sums, d_total);
  return hipGetLastError();
}

}  // namespace spc
