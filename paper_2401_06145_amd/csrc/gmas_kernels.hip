// Gather / Scatter of the GMaS step (Section 2.2, Step 2; Section 5.2.1).
//
// Metadata tables (Section 2.2): the input table gives, for input point j and
// offset k, the input-buffer row that j is copied to; the output table, for
// output point i and offset k, the output-buffer row holding i's partial
// result; -1 where (j, k) / (i, k) has no pair.  For a fixed point and offset
// there is at most one partner (q = p - delta), so each table is dense.  The
// Map step writes both while it ranks the pairs: they are stored offset-major
// and indexed by the points' sorted positions, entry [k * stride + p], so the
// map writes and the threads here read them with unit stride across points; a
// permutation turns sorted positions back into caller rows.
//
// Gather follows Algorithm 1: one thread per (channel tile, input point) reads
// its tile once and writes it to every buffer row listed for the point.
// Scatter is its mirror image: one thread per (channel tile, output point)
// sums the partials listed for the point in float32 (offsets in ascending
// order) and writes the tile once.  The tile size T (channels per thread) is
// the paper's autotuned parameter.
#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 256;
// metadata entries loaded ahead per gather thread (independent loads in flight)
constexpr int kMtBatch = 8;

// V = 16-byte vectors per thread (tile T = V * 16 / element bytes channels).
template <int V>
__global__ __launch_bounds__(kThreads) void k_gather(const uint4* __restrict__ x, int64_t n_in, int row_vec,
                                                     const int32_t* __restrict__ imt, int64_t stride,
                                                     const uint32_t* __restrict__ perm, int K3,
                                                     uint4* __restrict__ buf) {
  const int tiles = row_vec / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t p = gid / tiles;
  const int t = (int)(gid - p * tiles);
  if (p >= n_in) return;
  const int64_t j = perm ? (int64_t)perm[p] : p;
  uint4 v[V];
  const uint4* src = x + j * row_vec + (int64_t)t * V;
#pragma unroll
  for (int u = 0; u < V; ++u) v[u] = src[u];
  for (int k0 = 0; k0 < K3; k0 += kMtBatch) {
    int32_t r[kMtBatch];
#pragma unroll
    for (int e = 0; e < kMtBatch; ++e) r[e] = (k0 + e < K3) ? imt[(int64_t)(k0 + e) * stride + p] : -1;
#pragma unroll
    for (int e = 0; e < kMtBatch; ++e) {
      if (r[e] >= 0) {
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
// may alias y (each thread reads its tile before writing it).  The output
// stores are plain: a store instruction leaves each line partly written (the
// lanes' tiles are TILE channels apart) and the next ones complete it, which
// L2 merges; as non-temporal stores the wide tiles ran at half speed (C = 256,
// 300k outputs: T = 32 from 162 to 283 us).
template <int TILE, typename TP, typename TO>
__global__ __launch_bounds__(kThreads) void k_scatter(const TP* __restrict__ buf, int64_t n_out, int c_out,
                                                      const int32_t* __restrict__ omt, int64_t stride,
                                                      const uint32_t* __restrict__ perm, int K3, TO* y,
                                                      const TO* residual, int relu) {
  static_assert((TILE * sizeof(TP)) % 16 == 0, "partial tile must be whole 16-byte vectors");
  constexpr int VP = TILE * sizeof(TP) / 16;
  const int tiles = c_out / TILE;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t p = gid / tiles;
  const int t = (int)(gid - p * tiles);
  if (p >= n_out) return;
  const int64_t i = perm ? (int64_t)perm[p] : p;
  float acc[TILE];
#pragma unroll
  for (int c = 0; c < TILE; ++c) acc[c] = 0.f;
  for (int k0 = 0; k0 < K3; k0 += kMtBatch) {
    int32_t r[kMtBatch];
#pragma unroll
    for (int e = 0; e < kMtBatch; ++e) r[e] = (k0 + e < K3) ? omt[(int64_t)(k0 + e) * stride + p] : -1;
#pragma unroll
    for (int e = 0; e < kMtBatch; ++e) {
      if (r[e] >= 0) {
        const uint4* src = reinterpret_cast<const uint4*>(buf + (int64_t)r[e] * c_out + (int64_t)t * TILE);
#pragma unroll
        for (int u = 0; u < VP; ++u) {
          const uint4 v = src[u];
          const TP* pv = reinterpret_cast<const TP*>(&v);
#pragma unroll
          for (int c = 0; c < 16 / (int)sizeof(TP); ++c) acc[u * (16 / sizeof(TP)) + c] += to_f32<TP>(pv[c]);
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
    for (int u = 0; u < BYTES / 16; ++u) {
      reinterpret_cast<uint4*>(dst)[u] = reinterpret_cast<const uint4*>(out)[u];
    }
  } else if constexpr (BYTES % 8 == 0) {
#pragma unroll
    for (int u = 0; u < BYTES / 8; ++u) {
      reinterpret_cast<uint2*>(dst)[u] = reinterpret_cast<const uint2*>(out)[u];
    }
  } else {
#pragma unroll
    for (int c = 0; c < TILE; ++c) dst[c] = out[c];
  }
}

// Row-group scatter (the default tile: one 16-byte partial vector per thread).  A
// group of LP = c_out / W lanes of one wave owns an output row, lane `sub` holding
// channels [sub W, sub W + W) for W = 16 / sizeof(TP) (CH such vectors per lane when
// the row is wider than a wave).  So:
//  * the output's table entries are read once per output, not once per tile: lane
//    sub reads offsets sub, sub + LP, ...; a wave ballot then ranks the listed ones
//    in offset order, and their rows go to a per-group list in LDS;
//  * every partial row is read by the group as whole contiguous 16-byte vectors, and
//    the output row is written the same way;
//  * the rows of a batch of listed entries are all requested before the first is
//    added.
// Offsets are summed in ascending order, as in the tiled scatter, so both give the
// same result bit for bit.
constexpr int kRowList = 32;       // table entries per group and batch (at least LP)
constexpr int kRowListWave = 1024;  // list entries per wave

template <typename TP, typename TO, int CH>
__global__ __launch_bounds__(kThreads) void k_scatter_rows(const TP* __restrict__ buf, int64_t n_out, int c_out,
                                                           const int32_t* __restrict__ omt, int64_t stride,
                                                           const uint32_t* __restrict__ perm, int K3, TO* y,
                                                           const TO* residual, int relu, int LP, int stream) {
  constexpr int W = 16 / (int)sizeof(TP);  // channels per 16-byte partial vector
  constexpr int WPB = kThreads / kWave;
  __shared__ int32_t s_list[WPB][kRowListWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int gpw = kWave / LP;  // groups per wave (lanes past gpw * LP idle)
  const int group = lane / LP;
  const int sub = lane - group * LP;
  const int64_t p = ((int64_t)blockIdx.x * WPB + wave) * gpw + group;
  const bool active = group < gpw && p < n_out;
  const int64_t i = active ? (perm ? (int64_t)perm[p] : p) : 0;
  // the group's slice of the wave's 64 lanes
  const uint64_t gmask = (LP >= kWave ? ~0ull : ((1ull << LP) - 1ull)) << (group < gpw ? group * LP : 0);
  const int per_batch = max(1, kRowList / LP);  // table entries per lane and batch
  // the group's list holds one batch: per_batch * LP entries (gpw of them fit a wave's
  // kRowListWave: at most 32 groups of 32 entries)
  int32_t* list = &s_list[wave][(group < gpw ? group : 0) * per_batch * LP];
  float acc[CH][W];
#pragma unroll
  for (int c = 0; c < CH; ++c)
#pragma unroll
    for (int e = 0; e < W; ++e) acc[c][e] = 0.f;
  float rsd[CH][W];
  if (residual && active) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const TO* rp = residual + i * (int64_t)c_out + (int64_t)(c * LP + sub) * W;
#pragma unroll
      for (int e = 0; e < W; ++e) rsd[c][e] = to_f32<TO>(rp[e]);
    }
  }
  for (int kb = 0; kb < K3; kb += per_batch * LP) {
    // this batch's offsets kb + sub + LP m, m < per_batch
    int nv = 0;
    for (int m = 0; m < per_batch; ++m) {
      const int k = kb + sub + LP * m;
      const int32_t r = (active && k < K3) ? omt[(int64_t)k * stride + p] : -1;
      const uint64_t bal = __ballot(r >= 0) & gmask;
      if (r >= 0) list[nv + popc64(bal & lanemask_lt())] = r;
      nv += popc64(bal);
    }
    // listed rows, in offset order (the list is the group's own: no barrier)
    for (int j0 = 0; j0 < nv; j0 += 4) {
      int32_t row[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) row[j] = (j0 + j < nv) ? list[j0 + j] : -1;
      uint4 v[4][CH];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int c = 0; c < CH; ++c)
          v[j][c] = (row[j] >= 0) ? *reinterpret_cast<const uint4*>(buf + (int64_t)row[j] * c_out +
                                                                     (int64_t)(c * LP + sub) * W)
                                  : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (row[j] >= 0) {
#pragma unroll
          for (int c = 0; c < CH; ++c) {
            const TP* pv = reinterpret_cast<const TP*>(&v[j][c]);
#pragma unroll
            for (int e = 0; e < W; ++e) acc[c][e] += to_f32<TP>(pv[e]);
          }
        }
      }
    }
  }
  if (!active) return;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    TO out[W];
#pragma unroll
    for (int e = 0; e < W; ++e) {
      float a = acc[c][e];
      if (residual) a += rsd[c][e];
      if (relu) a = fmaxf(a, 0.f);
      out[e] = from_f32<TO>(a);
    }
    TO* dst = y + i * (int64_t)c_out + (int64_t)(c * LP + sub) * W;
    constexpr int BYTES = W * sizeof(TO);
    if constexpr (BYTES == 16) {
      const uint4 v = *reinterpret_cast<const uint4*>(out);
      if (stream)
        store_stream(dst, v);
      else
        *reinterpret_cast<uint4*>(dst) = v;
    } else if constexpr (BYTES == 8) {
      const uint2 v = *reinterpret_cast<const uint2*>(out);
      if (stream)
        store_stream(dst, v);
      else
        *reinterpret_cast<uint2*>(dst) = v;
    } else {
#pragma unroll
      for (int e = 0; e < W; ++e) dst[e] = out[e];
    }
  }
}

unsigned blocks_for(int64_t threads) { return (unsigned)((threads + kThreads - 1) / kThreads); }

// Lanes per output row of the row-group scatter, or 0 where it does not apply: it
// serves the tile of one 16-byte partial vector per thread when a row is at most a
// wave of such vectors, or 2 or 4 per lane of a full wave.
int scatter_row_lanes(int c_out, int pelem, int tile) {
  if (tile * pelem != 16 || (c_out * pelem) % 16 != 0) return 0;
  const int vec = c_out * pelem / 16;
  if (vec <= kWave) return vec;
  if (vec == 2 * kWave || vec == 4 * kWave) return kWave;
  return 0;
}

template <typename TP, typename TO>
hipError_t scatter_t(const void* buf, int64_t n_out, int c_out, const int32_t* omt, int64_t stride,
                     const uint32_t* perm, int K3, void* y, int tile, const void* residual, int relu, bool stream,
                     hipStream_t s) {
  ProfScope ps(KN_SCATTER, s);
  const int st = stream ? 1 : 0;
  const TP* p = static_cast<const TP*>(buf);
  TO* o = static_cast<TO*>(y);
  const TO* r = static_cast<const TO*>(residual);
  const int lp = scatter_row_lanes(c_out, (int)sizeof(TP), tile);
  if (lp > 0) {
    // row-group scatter: one 16-byte partial vector per lane and row slice
    const int vec = c_out * (int)sizeof(TP) / 16;
    const int ch = vec / lp;
    const int64_t per_block = (int64_t)(kThreads / kWave) * (kWave / lp);
    const dim3 g((unsigned)((n_out + per_block - 1) / per_block)), b(kThreads);
    switch (ch) {
      case 1: hipLaunchKernelGGL((k_scatter_rows<TP, TO, 1>), g, b, 0, s, p, n_out, c_out, omt, stride, perm, K3, o, r, relu, lp, st); break;
      case 2: hipLaunchKernelGGL((k_scatter_rows<TP, TO, 2>), g, b, 0, s, p, n_out, c_out, omt, stride, perm, K3, o, r, relu, lp, st); break;
      case 4: hipLaunchKernelGGL((k_scatter_rows<TP, TO, 4>), g, b, 0, s, p, n_out, c_out, omt, stride, perm, K3, o, r, relu, lp, st); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int64_t threads = n_out * (c_out / tile);
  const dim3 g(blocks_for(threads)), b(kThreads);
  switch (tile) {
#define SPC_SC(T)                                                                                    \
  case T:                                                                                            \
    if constexpr ((T * sizeof(TP)) % 16 == 0) {                                                      \
      hipLaunchKernelGGL((k_scatter<T, TP, TO>), g, b, 0, s, p, n_out, c_out, omt, stride, perm, K3, o, r, relu);     \
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

hipError_t launch_gather(const void* x, int64_t n_in, int c_in, int elem, const int32_t* imt, int64_t mt_stride,
                         const uint32_t* perm, int K3, void* buf_in, int tile, hipStream_t s) {
  if (n_in <= 0 || K3 <= 0) return hipSuccess;
  const int row_vec = c_in * elem / 16;
  const int v = tile * elem / 16;
  if (v <= 0 || row_vec % v != 0) return hipErrorInvalidValue;
  ProfScope ps(KN_GATHER, s);
  const int64_t threads = n_in * (row_vec / v);
  const dim3 g(blocks_for(threads)), b(kThreads);
  const uint4* xp = static_cast<const uint4*>(x);
  uint4* bp = static_cast<uint4*>(buf_in);
  switch (v) {
#define SPC_G(V)                                                                                         \
  case V:                                                                                                \
    hipLaunchKernelGGL(k_gather<V>, g, b, 0, s, xp, n_in, row_vec, imt, mt_stride, perm, K3, bp); \
    break;
    SPC_G(1)
    SPC_G(2)
    SPC_G(4)
    SPC_G(8)
    SPC_G(16)
#undef SPC_G
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_scatter(const void* buf_out, int part_dtype, int64_t n_out, int c_out, const int32_t* omt,
                          int64_t mt_stride, const uint32_t* perm, int K3, void* y, int dtype, int tile,
                          const void* residual, int relu, bool stream, hipStream_t s) {
  if (n_out <= 0) return hipSuccess;
  if (tile <= 0 || c_out % tile != 0) return hipErrorInvalidValue;
  // part_dtype / dtype: 0 = f32, 1 = f16, 2 = bf16
#define SPC_S(TP, TO) scatter_t<TP, TO>(buf_out, n_out, c_out, omt, mt_stride, perm, K3, y, tile, residual, relu, stream, s)
  if (part_dtype == 0) {
    if (dtype == 0) return SPC_S(float, float);
    if (dtype == 1) return SPC_S(float, __half);
    if (dtype == 2) return SPC_S(float, __hip_bfloat16);
  } else if (part_dtype == 1 && dtype == 1) {
    return SPC_S(__half, __half);
  } else if (part_dtype == 2 && dtype == 2) {
    return SPC_S(__hip_bfloat16, __hip_bfloat16);
  }
#undef SPC_S
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
