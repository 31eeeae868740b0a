// Grouped per-offset GEMMs of the GMaS step on MFMA (Section 2.2, Step 2;
// Section 5.2.2).  For every offset k of a group: buf_out[rows of k] =
// buf_in[rows of k] * W_k, with W_k a c_in x c_out matrix.
//
// A workgroup owns a run of rows of one offset and one slice of BN = 16*NT
// output columns.  It stages W_k's slice transposed in LDS once, then its four
// waves stream 16-row blocks of buf_in straight from HBM into MFMA operands:
//   D[n][m] = sum_c W_k[c][n] * A[m][c]  (the transposed product), so each lane
// ends up owning 4 consecutive output channels of one row and stores them with
// one vector store.  f16 / bf16 use v_mfma_f32_16x16x32_{f16,bf16}; f32 uses
// v_mfma_f32_16x16x4_f32.  Accumulation is float32.
//
// Operand layouts of these instructions (checked on gfx950), lane l:
//   A operand: row l%16, k = KSUB*(l/16) .. +KSUB-1;  B operand: column l%16, same k;
//   result:    row 4*(l/16)+i, column l%16, i = 0..3.
// Group padding rows (segment height > rows) are fed as zeros: they cost MFMA
// cycles, like the zero-padded batched GEMMs of the paper, but no memory traffic.
//
// Two kernels.  k_gemm_wide (f16 / bf16, c_in <= 256) gives a workgroup the full
// output width whenever W_k^T fits the 160 KiB of LDS, so every buf_in row is
// read from HBM once; it stages W_k^T from a transposed copy of the weights
// with 16-byte copies, and each wave loads the next 16-row block of buf_in while
// it multiplies the current one.  k_gemm is the general fallback (any c_in,
// float32) with a narrower column slice per workgroup.
#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxSegPerLaunch = 64;

struct GemmLaunchArgs {
  int n_seg;
  int tile_start[kMaxSegPerLaunch + 1];  // prefix of tiles per segment
  int k[kMaxSegPerLaunch];
  int rows[kMaxSegPerLaunch];
  int height[kMaxSegPerLaunch];
  int64_t row0[kMaxSegPerLaunch];
};

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <typename T>
struct Mfma;

template <>
struct Mfma<__half> {
  static constexpr int KS = 32;   // k per instruction
  static constexpr int KSUB = 8;  // k values per lane
  using frag = f16x8;
  __device__ static frag load(const __half* p) { return *reinterpret_cast<const frag*>(p); }
  __device__ static frag zero() { return frag{0, 0, 0, 0, 0, 0, 0, 0}; }
  __device__ static f32x4 mma(frag a, frag b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0); }
};

template <>
struct Mfma<__hip_bfloat16> {
  static constexpr int KS = 32;
  static constexpr int KSUB = 8;
  using frag = bf16x8;
  __device__ static frag load(const __hip_bfloat16* p) { return *reinterpret_cast<const frag*>(p); }
  __device__ static frag zero() {
    frag z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
    return z;
  }
  __device__ static f32x4 mma(frag a, frag b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0); }
};

template <>
struct Mfma<float> {
  static constexpr int KS = 4;
  static constexpr int KSUB = 1;
  using frag = float;
  __device__ static frag load(const float* p) { return *p; }
  __device__ static frag zero() { return 0.f; }
  __device__ static f32x4 mma(frag a, frag b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }
};

template <typename T>
__device__ __forceinline__ T zero_elem() { return T(0.0f); }

__device__ __forceinline__ void store4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
__device__ __forceinline__ void store4(__half* p, f32x4 v) {
  __half h[4] = {__float2half_rn(v[0]), __float2half_rn(v[1]), __float2half_rn(v[2]), __float2half_rn(v[3])};
  *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(h);
}
__device__ __forceinline__ void store4(__hip_bfloat16* p, f32x4 v) {
  __hip_bfloat16 h[4] = {__float2bfloat16(v[0]), __float2bfloat16(v[1]), __float2bfloat16(v[2]), __float2bfloat16(v[3])};
  *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(h);
}

// T: operand type; TO: partial (output buffer) type; NT: 16-column tiles per workgroup.
template <typename T, typename TO, int NT>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmLaunchArgs g, const T* __restrict__ A, const T* __restrict__ W,
                                                   TO* __restrict__ C, int c_in, int c_out, int kp, int ldk,
                                                   int rows_per_tile) {
  using M = Mfma<T>;
  extern __shared__ __align__(16) unsigned char smem[];
  T* lw = reinterpret_cast<T*>(smem);  // [BN][ldk], W_k^T slice
  constexpr int BN = 16 * NT;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;

  int s = 0;
  while (s + 1 < g.n_seg && g.tile_start[s + 1] <= (int)blockIdx.x) ++s;
  const int k = g.k[s];
  const int64_t row0 = g.row0[s];
  const int rows = g.rows[s];
  const int height = g.height[s];
  const int tile = (int)blockIdx.x - g.tile_start[s];
  const int n0 = blockIdx.y * BN;

  const T* wk = W + (int64_t)k * c_in * c_out;
  for (int idx = tid; idx < BN * kp; idx += kThreads) {
    const int c = idx / BN;
    const int n = idx - c * BN;
    lw[n * ldk + c] = (c < c_in) ? wk[(int64_t)c * c_out + n0 + n] : zero_elem<T>();
  }
  __syncthreads();

  const int r_begin = tile * rows_per_tile;
  const int r_end = min(r_begin + rows_per_tile, height);
  const int sub = lane >> 4;  // which k-slice of the fragment this lane carries
  const int col = lane & 15;
  for (int m0 = r_begin + wave * 16; m0 < r_end; m0 += 64) {
    const int row = m0 + col;
    const bool real = row < rows;
    const T* arow = A + (row0 + row) * (int64_t)c_in;
    f32x4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < kp; ks += M::KS) {
      const int kk = ks + M::KSUB * sub;
      const typename M::frag b = (real && kk < c_in) ? M::load(arow + kk) : M::zero();
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const typename M::frag a = M::load(lw + (16 * t + col) * ldk + kk);
        acc[t] = M::mma(a, b, acc[t]);
      }
    }
    if (real) {
      TO* crow = C + (row0 + row) * (int64_t)c_out + n0 + 4 * sub;
#pragma unroll
      for (int t = 0; t < NT; ++t) store4(crow + 16 * t, acc[t]);
    }
  }
}

constexpr int kWideThreads = 512;
constexpr int kWideWaves = kWideThreads / kWave;
constexpr size_t kLdsMax = 160 * 1024;

// NT = 16-column tiles per workgroup; ksteps = padded c_in / 32 <= kMaxKsteps.
// wt is W^T, [K^3][c_out][c_in] row-major.
constexpr int kMaxKsteps = 8;
template <typename T, typename TO, int NT>
__global__ __launch_bounds__(kWideThreads) void k_gemm_wide(GemmLaunchArgs g, const T* __restrict__ A,
                                                            const T* __restrict__ wt, TO* __restrict__ C, int c_in,
                                                            int c_out, int ksteps, int ldk, int rows_per_tile) {
  using M = Mfma<T>;
  static_assert(M::KS == 32, "16-bit operands only");
  extern __shared__ __align__(16) unsigned char smem[];
  T* lw = reinterpret_cast<T*>(smem);  // [BN][ldk], W_k^T slice
  constexpr int BN = 16 * NT;
  const int KP = 32 * ksteps;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;

  int s = 0;
  while (s + 1 < g.n_seg && g.tile_start[s + 1] <= (int)blockIdx.x) ++s;
  const int k = g.k[s];
  const int64_t row0 = g.row0[s];
  const int rows = g.rows[s];
  const int height = g.height[s];
  const int tile = (int)blockIdx.x - g.tile_start[s];
  const int n0 = blockIdx.y * BN;

  // W_k^T rows n0 .. n0 + BN, 8 elements (16 bytes) per copy; columns past c_in are zero
  const T* wk = wt + ((int64_t)k * c_out + n0) * c_in;
  const int CH = KP / 8;  // 16-byte chunks per LDS row
  for (int idx = tid; idx < BN * CH; idx += kWideThreads) {
    const int n = idx / CH;
    const int c = (idx - n * CH) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (c < c_in) v = *reinterpret_cast<const uint4*>(wk + (int64_t)n * c_in + c);
    *reinterpret_cast<uint4*>(lw + n * ldk + c) = v;
  }
  __syncthreads();

  const int r_begin = tile * rows_per_tile;
  const int r_end = min(r_begin + rows_per_tile, height);
  const int sub = lane >> 4;
  const int col = lane & 15;
  typename M::frag cur[kMaxKsteps], nxt[kMaxKsteps];
  auto load_block = [&](int m0, typename M::frag* f) {
    const int row = m0 + col;
    const bool real = row < rows;
    const T* arow = A + (row0 + row) * (int64_t)c_in;
#pragma unroll
    for (int q = 0; q < kMaxKsteps; ++q) {
      const int kk = 32 * q + 8 * sub;
      f[q] = (q < ksteps && real && kk < c_in) ? M::load(arow + kk) : M::zero();
    }
  };
  int m0 = r_begin + wave * 16;
  if (m0 < r_end) load_block(m0, cur);
  for (; m0 < r_end; m0 += 16 * kWideWaves) {
    const int m1 = m0 + 16 * kWideWaves;
    if (m1 < r_end) load_block(m1, nxt);
    f32x4 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < kMaxKsteps; ++q) {
      if (q >= ksteps) break;
      const int kk = 32 * q + 8 * sub;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const typename M::frag a = M::load(lw + (16 * t + col) * ldk + kk);
        acc[t] = M::mma(a, cur[q], acc[t]);
      }
    }
    const int row = m0 + col;
    if (row < rows) {
      TO* crow = C + (row0 + row) * (int64_t)c_out + n0 + 4 * sub;
#pragma unroll
      for (int t = 0; t < NT; ++t) store4(crow + 16 * t, acc[t]);
    }
#pragma unroll
    for (int q = 0; q < kMaxKsteps; ++q) cur[q] = nxt[q];
  }
}

// Column tiles per workgroup for the wide kernel: the widest instantiated divisor
// of c_out / 16 whose W^T slice fits the LDS; 0 if the wide kernel does not apply.
int wide_nt(int c_in, int c_out, int elem) {
  if (elem != 2 || c_in > 32 * kMaxKsteps || c_in % 8 != 0 || c_out % 16 != 0) return 0;
  const int kp = (c_in + 31) / 32 * 32;
  const int ldk = kp + 8;
  const int nt_all = c_out / 16;
  for (int nt : {16, 12, 8, 6, 4, 3, 2, 1})
    if (nt_all % nt == 0 && (size_t)16 * nt * ldk * 2 <= kLdsMax) return nt;
  return 0;
}

template <typename T, typename TO>
hipError_t gemm_wide_t(const GemmLaunchArgs& g, int total_tiles, const void* A, const void* WT, void* C, int c_in,
                       int c_out, int rows_per_tile, hipStream_t s) {
  const int nt = wide_nt(c_in, c_out, 2);
  const int ksteps = (c_in + 31) / 32;
  const int ldk = 32 * ksteps + 8;
  const size_t lds = (size_t)16 * nt * ldk * sizeof(T);
  ProfScope ps(KN_GEMM, s);
  const dim3 grid((unsigned)total_tiles, (unsigned)(c_out / 16 / nt));
  const T* a = static_cast<const T*>(A);
  const T* w = static_cast<const T*>(WT);
  TO* c = static_cast<TO*>(C);
  switch (nt) {
#define SPC_W(N)                                                                                                \
  case N:                                                                                                       \
    hipLaunchKernelGGL((k_gemm_wide<T, TO, N>), grid, dim3(kWideThreads), lds, s, g, a, w, c, c_in, c_out,      \
                       ksteps, ldk, rows_per_tile);                                                             \
    return hipGetLastError();
    SPC_W(1)
    SPC_W(2)
    SPC_W(3)
    SPC_W(4)
    SPC_W(6)
    SPC_W(8)
    SPC_W(12)
    SPC_W(16)
#undef SPC_W
    default:
      return hipErrorInvalidValue;
  }
}

// wt[k][n][c] = w[k][c][n] through a 32 x 32 LDS tile (16-bit elements).
__global__ __launch_bounds__(256) void k_transpose_w(const uint16_t* __restrict__ w, uint16_t* __restrict__ wt,
                                                     int c_in, int c_out) {
  __shared__ uint16_t t[32][33];
  const int k = blockIdx.z;
  const int c0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
  const uint16_t* src = w + (int64_t)k * c_in * c_out;
  uint16_t* dst = wt + (int64_t)k * c_in * c_out;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int r = ty; r < 32; r += 8) {
    const int c = c0 + r, n = n0 + tx;
    t[r][tx] = (c < c_in && n < c_out) ? src[(int64_t)c * c_out + n] : 0;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int n = n0 + r, c = c0 + tx;
    if (n < c_out && c < c_in) dst[(int64_t)n * c_in + c] = t[tx][r];
  }
}

template <typename T, typename TO>
hipError_t gemm_t(const GemmLaunchArgs& g, int total_tiles, const void* A, const void* W, void* C, int c_in,
                  int c_out, int rows_per_tile, hipStream_t s) {
  const int KS = Mfma<T>::KS;
  const int kp = (c_in + KS - 1) / KS * KS;
  const int ldk = kp + 16 / (int)sizeof(T);
  // widest column slice whose W^T tile fits 64 KiB of LDS
  const int nt_all = c_out / 16;
  int nt = 0;
  const int cand[] = {8, 6, 4, 3, 2, 1};
  for (int c : cand)
    if (nt_all % c == 0 && (size_t)16 * c * ldk * sizeof(T) <= 65536) {
      nt = c;
      break;
    }
  if (nt == 0) return hipErrorInvalidValue;
  ProfScope ps(KN_GEMM, s);
  const size_t lds = (size_t)16 * nt * ldk * sizeof(T);
  const dim3 grid((unsigned)total_tiles, (unsigned)(nt_all / nt));
  const T* a = static_cast<const T*>(A);
  const T* w = static_cast<const T*>(W);
  TO* c = static_cast<TO*>(C);
  switch (nt) {
#define SPC_G(N)                                                                                     \
  case N:                                                                                            \
    hipLaunchKernelGGL((k_gemm<T, TO, N>), grid, dim3(kThreads), lds, s, g, a, w, c, c_in, c_out, kp, ldk, \
                       rows_per_tile);                                                               \
    break;
    SPC_G(1)
    SPC_G(2)
    SPC_G(3)
    SPC_G(4)
    SPC_G(6)
    SPC_G(8)
#undef SPC_G
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool gemm_wide(int c_in, int c_out, int dtype, int part_dtype) {
  // built for 16-bit operands with partials of the same type, and f16 with f32 partials
  const bool pair = part_dtype == dtype || (dtype == 1 && part_dtype == 0);
  return dtype != 0 && pair && wide_nt(c_in, c_out, 2) > 0;
}

hipError_t launch_transpose_w(const void* w, void* wt, int K3, int c_in, int c_out, hipStream_t s) {
  const dim3 grid((unsigned)((c_out + 31) / 32), (unsigned)((c_in + 31) / 32), (unsigned)K3);
  hipLaunchKernelGGL(k_transpose_w, grid, dim3(256), 0, s, static_cast<const uint16_t*>(w),
                     static_cast<uint16_t*>(wt), c_in, c_out);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmSeg* segs, int n_seg, const void* buf_in, const void* w, const void* wt,
                       void* buf_out, int c_in, int c_out, int dtype, int part_dtype, hipStream_t s) {
  if (c_out % 16 != 0) return hipErrorInvalidValue;
  const bool wide = wt && gemm_wide(c_in, c_out, dtype, part_dtype);
  int64_t rows_all = 0;
  for (int i = 0; i < n_seg; ++i) rows_all += segs[i].height;
  // enough workgroups to fill 256 CUs several times; tiles are whole rounds of the
  // workgroup's 16-row waves
  int rows_per_tile = wide ? 16 * kWideWaves : 64;
  while (rows_per_tile < 2048 && rows_all / (rows_per_tile * 2) >= 1024) rows_per_tile *= 2;
  for (int base = 0; base < n_seg; base += kMaxSegPerLaunch) {
    GemmLaunchArgs g{};
    g.n_seg = 0;
    int tiles = 0;
    for (int i = base; i < n_seg && g.n_seg < kMaxSegPerLaunch; ++i) {
      const GemmSeg& sg = segs[i];
      if (sg.height <= 0) continue;
      const int j = g.n_seg++;
      g.k[j] = sg.k;
      g.row0[j] = sg.row0;
      g.rows[j] = (int)sg.rows;
      g.height[j] = (int)sg.height;
      g.tile_start[j] = tiles;
      tiles += (int)((sg.height + rows_per_tile - 1) / rows_per_tile);
    }
    g.tile_start[g.n_seg] = tiles;
    if (tiles == 0) continue;
    hipError_t e = hipErrorInvalidValue;
    if (wide) {
      if (dtype == 1 && part_dtype == 0)
        e = gemm_wide_t<__half, float>(g, tiles, buf_in, wt, buf_out, c_in, c_out, rows_per_tile, s);
      else if (dtype == 1 && part_dtype == 1)
        e = gemm_wide_t<__half, __half>(g, tiles, buf_in, wt, buf_out, c_in, c_out, rows_per_tile, s);
      else if (dtype == 2 && part_dtype == 2)
        e = gemm_wide_t<__hip_bfloat16, __hip_bfloat16>(g, tiles, buf_in, wt, buf_out, c_in, c_out, rows_per_tile,
                                                        s);
    } else if (dtype == 0 && part_dtype == 0)
      e = gemm_t<float, float>(g, tiles, buf_in, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 1 && part_dtype == 0)
      e = gemm_t<__half, float>(g, tiles, buf_in, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 1 && part_dtype == 1)
      e = gemm_t<__half, __half>(g, tiles, buf_in, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 2 && part_dtype == 0)
      e = gemm_t<__hip_bfloat16, float>(g, tiles, buf_in, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 2 && part_dtype == 2)
      e = gemm_t<__hip_bfloat16, __hip_bfloat16>(g, tiles, buf_in, w, buf_out, c_in, c_out, rows_per_tile, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace spc
