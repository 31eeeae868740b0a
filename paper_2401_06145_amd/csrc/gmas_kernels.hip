// Gather / Scatter of the GMaS step (Section 2.2, Step 2; Section 5.2.1).
//
// Metadata tables (Section 2.2): IMT[j][k] is the input-buffer row that input j
// is copied to for offset k, OMT[i][k] the output-buffer row holding output i's
// partial result for offset k; -1 where (j, k) / (i, k) has no pair.  For a
// fixed point and offset there is at most one partner (q = p - delta), so each
// table is a dense [rows][K^3] array, padded to a multiple of 4 entries per row.
//
// Gather follows Algorithm 1: one thread per (channel tile, input point) reads
// its tile once and writes it to every buffer row listed in the point's IMT
// row.  Scatter is its mirror image: one thread per (channel tile, output point)
// sums the partials listed in the point's OMT row in float32 (offsets in
// ascending order) and writes the tile once.  The tile size T (channels per
// thread) is the paper's autotuned parameter.
#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void k_mt_pairs(const int32_t* pin, const int32_t* pout, int64_t m_total,
                                                       OffsetTable t, int32_t* imt, int32_t* omt, int stride) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= m_total) return;
  // offset k of pair m: last k with pair_start[k] <= m
  int lo = 0, hi = t.K3 - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (t.pair_start[mid] <= m) lo = mid;
    else hi = mid - 1;
  }
  const int k = lo;
  const int32_t row = (int32_t)(t.row_base[k] + (m - t.pair_start[k]));
  imt[(int64_t)pin[m] * stride + k] = row;
  omt[(int64_t)pout[m] * stride + k] = row;
}

// V = 16-byte vectors per thread (tile T = V * 16 / element bytes channels).
template <int V>
__global__ __launch_bounds__(kThreads) void k_gather(const uint4* __restrict__ x, int64_t n_in, int row_vec,
                                                     const int32_t* __restrict__ imt, int stride, int K3,
                                                     uint4* __restrict__ buf) {
  const int tiles = row_vec / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t j = gid / tiles;
  const int t = (int)(gid - j * tiles);
  if (j >= n_in) return;
  uint4 v[V];
  const uint4* src = x + j * row_vec + (int64_t)t * V;
#pragma unroll
  for (int u = 0; u < V; ++u) v[u] = src[u];
  const int4* mt = reinterpret_cast<const int4*>(imt + j * stride);
  for (int k4 = 0; k4 < stride / 4; ++k4) {
    const int4 r4 = mt[k4];
    const int32_t r[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (r[e] >= 0 && k4 * 4 + e < K3) {
        uint4* dst = buf + (int64_t)r[e] * row_vec + (int64_t)t * V;
#pragma unroll
        for (int u = 0; u < V; ++u) dst[u] = v[u];
      }
    }
  }
}

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<__half>(__half v) { return __half2float(v); }
template <>
__device__ __forceinline__ float to_f32<__hip_bfloat16>(__hip_bfloat16 v) { return __bfloat162float(v); }

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ __half from_f32<__half>(float v) { return __float2half_rn(v); }
template <>
__device__ __forceinline__ __hip_bfloat16 from_f32<__hip_bfloat16>(float v) { return __float2bfloat16(v); }

// TILE channels per thread; partials of type TP, output of type TO.  Optional
// epilogue fused into the single write: y = relu?(sum + residual).  `residual`
// may alias y (each thread reads its tile before writing it).
template <int TILE, typename TP, typename TO>
__global__ __launch_bounds__(kThreads) void k_scatter(const TP* __restrict__ buf, int64_t n_out, int c_out,
                                                      const int32_t* __restrict__ omt, int stride, int K3,
                                                      TO* y, const TO* residual, int relu) {
  static_assert((TILE * sizeof(TP)) % 16 == 0, "partial tile must be whole 16-byte vectors");
  constexpr int VP = TILE * sizeof(TP) / 16;
  const int tiles = c_out / TILE;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t i = gid / tiles;
  const int t = (int)(gid - i * tiles);
  if (i >= n_out) return;
  float acc[TILE];
#pragma unroll
  for (int c = 0; c < TILE; ++c) acc[c] = 0.f;
  const int4* mt = reinterpret_cast<const int4*>(omt + i * stride);
  for (int k4 = 0; k4 < stride / 4; ++k4) {
    const int4 r4 = mt[k4];
    const int32_t r[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (r[e] >= 0 && k4 * 4 + e < K3) {
        const uint4* src = reinterpret_cast<const uint4*>(buf + (int64_t)r[e] * c_out + (int64_t)t * TILE);
#pragma unroll
        for (int u = 0; u < VP; ++u) {
          const uint4 v = src[u];
          const TP* p = reinterpret_cast<const TP*>(&v);
#pragma unroll
          for (int c = 0; c < 16 / (int)sizeof(TP); ++c) acc[u * (16 / sizeof(TP)) + c] += to_f32<TP>(p[c]);
        }
      }
    }
  }
  if (residual) {
    const TO* rsd = residual + i * (int64_t)c_out + (int64_t)t * TILE;
#pragma unroll
    for (int c = 0; c < TILE; ++c) acc[c] += to_f32<TO>(rsd[c]);
  }
  if (relu) {
#pragma unroll
    for (int c = 0; c < TILE; ++c) acc[c] = fmaxf(acc[c], 0.f);
  }
  TO out[TILE];
#pragma unroll
  for (int c = 0; c < TILE; ++c) out[c] = from_f32<TO>(acc[c]);
  TO* dst = y + i * (int64_t)c_out + (int64_t)t * TILE;
  constexpr int BYTES = TILE * sizeof(TO);
  if constexpr (BYTES % 16 == 0) {
#pragma unroll
    for (int u = 0; u < BYTES / 16; ++u) reinterpret_cast<uint4*>(dst)[u] = reinterpret_cast<const uint4*>(out)[u];
  } else if constexpr (BYTES % 8 == 0) {
#pragma unroll
    for (int u = 0; u < BYTES / 8; ++u) reinterpret_cast<uint2*>(dst)[u] = reinterpret_cast<const uint2*>(out)[u];
  } else {
#pragma unroll
    for (int c = 0; c < TILE; ++c) dst[c] = out[c];
  }
}

unsigned blocks_for(int64_t threads) { return (unsigned)((threads + kThreads - 1) / kThreads); }

template <typename TP, typename TO>
hipError_t scatter_t(const void* buf, int64_t n_out, int c_out, const int32_t* omt, int stride, int K3, void* y,
                     int tile, const void* residual, int relu, hipStream_t s) {
  ProfScope ps(KN_SCATTER, s);
  const int64_t threads = n_out * (c_out / tile);
  const dim3 g(blocks_for(threads)), b(kThreads);
  const TP* p = static_cast<const TP*>(buf);
  TO* o = static_cast<TO*>(y);
  const TO* r = static_cast<const TO*>(residual);
  switch (tile) {
#define SPC_SC(T)                                                                                    \
  case T:                                                                                            \
    if constexpr ((T * sizeof(TP)) % 16 == 0) {                                                      \
      hipLaunchKernelGGL((k_scatter<T, TP, TO>), g, b, 0, s, p, n_out, c_out, omt, stride, K3, o, r, relu); \
      return hipGetLastError();                                                                      \
    }                                                                                                \
    return hipErrorInvalidValue;
    SPC_SC(4)
    SPC_SC(8)
    SPC_SC(16)
    SPC_SC(32)
    SPC_SC(64)
#undef SPC_SC
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_mt_fill(int32_t* imt, int64_t n_in, int32_t* omt, int64_t n_out, int stride, hipStream_t s) {
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(imt), 0xFFFFFFFFu, n_in * stride, s);
  if (e != hipSuccess) return e;
  return launch_fill_u32(reinterpret_cast<uint32_t*>(omt), 0xFFFFFFFFu, n_out * stride, s);
}

hipError_t launch_mt_pairs(const int32_t* pin, const int32_t* pout, int64_t m_total, const OffsetTable& t,
                           int32_t* imt, int32_t* omt, int stride, hipStream_t s) {
  if (m_total <= 0) return hipSuccess;
  ProfScope ps(KN_MT_PAIRS, s);
  hipLaunchKernelGGL(k_mt_pairs, dim3(blocks_for(m_total)), dim3(kThreads), 0, s, pin, pout, m_total, t, imt, omt,
                     stride);
  return hipGetLastError();
}

hipError_t launch_gather(const void* x, int64_t n_in, int c_in, int elem, const int32_t* imt, int mt_stride, int K3,
                         void* buf_in, int tile, hipStream_t s) {
  if (n_in <= 0) return hipSuccess;
  const int row_vec = c_in * elem / 16;
  const int v = tile * elem / 16;
  if (v <= 0 || row_vec % v != 0) return hipErrorInvalidValue;
  ProfScope ps(KN_GATHER, s);
  const int64_t threads = n_in * (row_vec / v);
  const dim3 g(blocks_for(threads)), b(kThreads);
  const uint4* xp = static_cast<const uint4*>(x);
  uint4* bp = static_cast<uint4*>(buf_in);
  switch (v) {
    case 1: hipLaunchKernelGGL(k_gather<1>, g, b, 0, s, xp, n_in, row_vec, imt, mt_stride, K3, bp); break;
    case 2: hipLaunchKernelGGL(k_gather<2>, g, b, 0, s, xp, n_in, row_vec, imt, mt_stride, K3, bp); break;
    case 4: hipLaunchKernelGGL(k_gather<4>, g, b, 0, s, xp, n_in, row_vec, imt, mt_stride, K3, bp); break;
    case 8: hipLaunchKernelGGL(k_gather<8>, g, b, 0, s, xp, n_in, row_vec, imt, mt_stride, K3, bp); break;
    case 16: hipLaunchKernelGGL(k_gather<16>, g, b, 0, s, xp, n_in, row_vec, imt, mt_stride, K3, bp); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_scatter(const void* buf_out, int part_dtype, int64_t n_out, int c_out, const int32_t* omt,
                          int mt_stride, int K3, void* y, int dtype, int tile, const void* residual, int relu,
                          hipStream_t s) {
  if (n_out <= 0) return hipSuccess;
  if (tile <= 0 || c_out % tile != 0) return hipErrorInvalidValue;
  // part_dtype / dtype: 0 = f32, 1 = f16, 2 = bf16
  if (part_dtype == 0) {
    if (dtype == 0) return scatter_t<float, float>(buf_out, n_out, c_out, omt, mt_stride, K3, y, tile, residual, relu, s);
    if (dtype == 1)
      return scatter_t<float, __half>(buf_out, n_out, c_out, omt, mt_stride, K3, y, tile, residual, relu, s);
    if (dtype == 2)
      return scatter_t<float, __hip_bfloat16>(buf_out, n_out, c_out, omt, mt_stride, K3, y, tile, residual, relu, s);
  } else if (part_dtype == 1 && dtype == 1) {
    return scatter_t<__half, __half>(buf_out, n_out, c_out, omt, mt_stride, K3, y, tile, residual, relu, s);
  } else if (part_dtype == 2 && dtype == 2) {
    return scatter_t<__hip_bfloat16, __hip_bfloat16>(buf_out, n_out, c_out, omt, mt_stride, K3, y, tile, residual,
                                                     relu, s);
  }
  return hipErrorInvalidValue;
}

namespace {
// out[i] = [a[i] (ca channels) | b[i] (cb channels)]; one thread per 16-byte vector of out.
__global__ __launch_bounds__(kThreads) void k_concat(const uint4* a, int va, const uint4* b, int vb, uint4* out,
                                                     int64_t n) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int vo = va + vb;
  const int64_t i = gid / vo;
  const int v = (int)(gid - i * vo);
  if (i >= n) return;
  out[gid] = (v < va) ? a[i * va + v] : b[i * vb + (v - va)];
}
}  // namespace

hipError_t launch_concat(const void* a, int ca, const void* b, int cb, void* out, int64_t n, int elem, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int va = ca * elem / 16, vb = cb * elem / 16;
  const int64_t threads = n * (va + vb);
  hipLaunchKernelGGL(k_concat, dim3(blocks_for(threads)), dim3(kThreads), 0, s, static_cast<const uint4*>(a), va,
                     static_cast<const uint4*>(b), vb, static_cast<uint4*>(out), n);
  return hipGetLastError();
}

}  // namespace spc
