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
// The A operand is either the gathered buffer (row r of the launch is buffer row
// r, Algorithm 1's layout) or, with the gather fused into the operand loads, the
// layer's input features themselves: row r is then input row a_rows[r], the input
// index of pair r.  The fused form never writes or reads the gathered buffer.
//
// Two kernels.  k_gemm_wide (f16 / bf16, c_in <= 512) gives a workgroup the full
// output width whenever W_k^T fits the 160 KiB of LDS, so every buf_in row is
// read from HBM once; it stages W_k^T from a transposed copy of the weights
// with 16-byte copies, and each wave loads the next 16-row block of buf_in while
// it multiplies the current one.  k_gemm is the general fallback (any c_in,
// float32) with a narrower column slice per workgroup.
#include <algorithm>
#include <mutex>
#include <type_traits>
#include <vector>

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
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
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
__global__ __launch_bounds__(kThreads) void k_gemm(GemmLaunchArgs g, const T* __restrict__ A,
                                                   const int32_t* __restrict__ arows, const T* __restrict__ W,
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
    const int64_t src = !real ? 0 : (arows ? (int64_t)arows[row0 + row] : row0 + row);
    const T* arow = A + src * (int64_t)c_in;
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
// Per-wave LDS stage of the partial stores: 16 rows of one segment of at most 128
// bytes, each row padded by 16 bytes.
constexpr int kStageRow = 128 + 16;
constexpr size_t kStageBytes = (size_t)kWideWaves * 16 * kStageRow;
// LDS of one full-width workgroup: the W_k^T slice plus the store stages.
constexpr size_t wide_lds(int nt, int ldk) { return (size_t)16 * nt * ldk * 2 + kStageBytes; }

// Register blocking of the full-width kernel.  A wave computes MB 16-row blocks
// times NTW 16-column tiles, so every W^T fragment it reads from LDS feeds MB
// MFMAs (the W fragment reads, 1 KiB per wave per MFMA at MB = 1, otherwise
// bound the kernel from 128 columns up); CG waves split the workgroup's NT =
// CG * NTW column tiles, the others take further rows.  Two row blocks per wave
// while their operands (and the next blocks' in flight) take at most 128
// registers and the layer is wide enough for the LDS reads to matter: 65 to 128
// input channels (from 160 channels the two blocks and their successors in
// flight need 160 registers and the kernel spills).  The columns of a two-block
// wave are produced in NCH chunks of at most 8 tiles, so that operands,
// accumulators and fragments stay within the 256 registers a wave has at two
// waves per SIMD (and at 385 to 512 input channels in chunks of two tiles, as the
// operands alone take 128 registers there).  Measured on gfx950: C = 128 GEMM 0.142 -> 0.132 ms; at C = 64
// one block per wave is faster (26.5 vs 28.5 us on the 120k LiDAR layer), at
// C = 32 the two are equal; one block per wave stays faster in one chunk; CG > 1
// cost more occupancy than it saved.
constexpr int wide_cg(int) { return 1; }
constexpr int wide_mb(int, int ksteps) { return (ksteps == 3 || ksteps == 4) ? 2 : 1; }
constexpr int wide_nch(int ntw, int mb, int ksteps) {
  int nch = 1;
  while ((mb > 1 || ksteps >= 16) && ntw / nch > (mb > 1 ? 8 : 2) && ntw % (2 * nch) == 0) nch *= 2;
  return nch;
}

// NT = 16-column tiles per workgroup; KSTEPS >= c_in / 32 k-steps of 32 (k past
// c_in is zero).  w is W, [K^3][c_in][c_out]; wt is NULL or W^T, [K^3][c_out][c_in]
// (then W_k^T is staged from it with 16-byte copies); dump is one spare
// row of c_out partials that absorbs the stores of rows without data.  Loads
// never branch: lanes without data (rows past the segment, k past c_in) read a
// valid dummy address; k past c_in is then zeroed, rows past the segment compute
// values that only reach the dump row.  So the compiler keeps the next blocks'
// loads in flight across the current blocks' MFMAs.
template <typename T, typename TO, int NT, int KSTEPS, bool GATHER>
__global__ __launch_bounds__(kWideThreads) void k_gemm_wide(GemmLaunchArgs g, const T* __restrict__ A,
                                                            const int32_t* __restrict__ arows,
                                                            const T* __restrict__ w, const T* __restrict__ wt,
                                                            TO* __restrict__ C,
                                                            TO* __restrict__ dump, int c_in, int c_out, int ldk,
                                                            int rows_per_tile, int nsl, int stream) {
  using M = Mfma<T>;
  using F = typename M::frag;
  static_assert(M::KS == 32, "16-bit operands only");
  constexpr int CG = wide_cg(NT);
  constexpr int NTW = NT / CG;
  constexpr int MB = wide_mb(NTW, KSTEPS);
  constexpr int NCH = wide_nch(NTW, MB, KSTEPS);
  constexpr int NTC = NTW / NCH;  // column tiles per chunk
  static_assert(NTW % NCH == 0, "chunks must split the tiles");
  constexpr int RG = kWideWaves / CG;   // row groups
  constexpr int STEP = RG * MB * 16;    // rows per round of the workgroup
  static_assert(NT % CG == 0, "column groups must split the tiles");
  extern __shared__ __align__(16) unsigned char smem[];
  T* lw = reinterpret_cast<T*>(smem);  // [BN][ldk], W_k^T slice
  constexpr int BN = 16 * NT;
  constexpr int KP = 32 * KSTEPS;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int cg = wave % CG, rg = wave / CG;

  // With nsl > 1 column slices per tile, the grid is one-dimensional and the
  // slices of a tile take workgroup ids 8 apart: workgroups go to the eight dies
  // in turn, so the slices of a tile run on one die at about the same time and
  // share its L2 for the tile's input rows (slice-major, every input row would be
  // read from memory once per slice).
  int bx = (int)blockIdx.x, by = (int)blockIdx.y;
  if (nsl > 1) {
    const int grp = bx / (8 * nsl), r = bx - grp * (8 * nsl);
    by = r / 8;
    bx = grp * 8 + (r - by * 8);
    if (bx >= g.tile_start[g.n_seg]) return;  // the last group's missing tiles (workgroup-uniform)
  }
  int s = 0;
  while (s + 1 < g.n_seg && g.tile_start[s + 1] <= bx) ++s;
  const int k = g.k[s];
  const int64_t row0 = g.row0[s];
  const int rows = g.rows[s];
  const int height = g.height[s];
  const int tile = bx - g.tile_start[s];
  const int n0 = by * BN;

  const int r_begin = tile * rows_per_tile;
  const int r_end = min(r_begin + rows_per_tile, height);
  const int sub = lane >> 4;
  const int col = lane & 15;
  const int nw = 16 * NTW * cg;  // this wave's first column within the slice
  const T* lwp = lw + (nw + col) * ldk + 8 * sub;
  // store stage: GC tiles per segment (128 bytes, or fewer tiles when the chunk's
  // tile count is not a multiple), SLANES lanes of 16 bytes per row, SROWS rows
  // per read, SREADS reads for the 16 rows
  unsigned char* stg = smem + (size_t)BN * ldk * sizeof(T) + (size_t)wave * 16 * kStageRow;
  constexpr int GC0 = 128 / (16 * (int)sizeof(TO));
  constexpr int GC = (NTC % GC0 == 0) ? GC0 : ((NTC % 2 == 0 && GC0 >= 2) ? 2 : 1);
  constexpr int SLANES = GC * 16 * (int)sizeof(TO) / 16;
  constexpr int SROWS = kWave / SLANES;
  constexpr int SREADS = (16 + SROWS - 1) / SROWS;
  const int row_lim = min(rows, r_end);  // rows of this tile that hold data
  // raw: the next blocks as loaded (dummy data where masked); cur: the blocks in use
  F raw[MB][KSTEPS], cur[MB][KSTEPS];
  // GATHER: source rows of the blocks issued next, fetched one round ahead so the
  // operand loads never wait for their index (masked lanes read the segment's first)
  int32_t src[MB];
  auto fetch_rows = [&](int mb) {
    if constexpr (GATHER) {
#pragma unroll
      for (int b = 0; b < MB; ++b) {
        const int row = mb + 16 * b + col;
        src[b] = arows[row0 + (row < row_lim ? row : 0)];
      }
    }
  };
  auto issue = [&](int mb) {
#pragma unroll
    for (int b = 0; b < MB; ++b) {
      const int row = mb + 16 * b + col;
      const int64_t r = GATHER ? (int64_t)src[b] : row0 + row;
      const T* arow = A + r * (int64_t)c_in;
#pragma unroll
      for (int q = 0; q < KSTEPS; ++q) {
        const int kk = 32 * q + 8 * sub;
        raw[b][q] = M::load((row < row_lim && kk < c_in) ? arow + kk : A);
      }
    }
  };

  // Prologue, ordered so that its round trips overlap: the first blocks' source
  // rows, then the first kWStage 16-byte chunks of the W_k^T slice per thread, then
  // the first blocks' operands (they wait only for their rows), then the chunks go
  // to LDS.  A chunk is 8 consecutive k of one column n when read from the
  // transposed copy, or 8 consecutive n of one k when read from W itself (and
  // transposed on the way into LDS).  k past c_in is zero.
  const int m_first = r_begin + rg * MB * 16;
  fetch_rows(m_first);
  constexpr int CH_T = KP / 8;  // chunks per W^T row (transposed copy)
  constexpr int CH_N = BN / 8;  // chunks per W row slice (plain copy)
  constexpr int NCHUNK = BN * KP / 8;
  const T* wk_t = wt ? wt + ((int64_t)k * c_out + n0) * c_in : nullptr;
  const T* wk_p = w + (int64_t)k * c_in * c_out + n0;
  auto chunk_nc = [&](int idx, int* n, int* c) {
    if (wt) {
      *n = idx / CH_T;
      *c = (idx - *n * CH_T) * 8;
    } else {
      *c = idx / CH_N;
      *n = (idx - *c * CH_N) * 8;
    }
  };
  auto load_chunk = [&](int idx) -> uint4 {
    int n, c;
    chunk_nc(idx, &n, &c);
    if (idx >= NCHUNK || c >= c_in) return make_uint4(0, 0, 0, 0);
    return wt ? *reinterpret_cast<const uint4*>(wk_t + (int64_t)n * c_in + c)
              : *reinterpret_cast<const uint4*>(wk_p + (int64_t)c * c_out + n);
  };
  auto store_chunk = [&](int idx, const uint4& v) {
    if (idx >= NCHUNK) return;
    int n, c;
    chunk_nc(idx, &n, &c);
    if (wt) {
      *reinterpret_cast<uint4*>(lw + n * ldk + c) = v;
    } else {
      const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
      for (int j = 0; j < 8; ++j) lw[(n + j) * ldk + c] = e[j];
    }
  };
  constexpr int kWStage = 8;  // chunks per thread in flight at a time
  uint4 wv[kWStage];
#pragma unroll
  for (int u = 0; u < kWStage; ++u) wv[u] = load_chunk(u * kWideThreads + tid);
  issue(m_first);
#pragma unroll
  for (int u = 0; u < kWStage; ++u) store_chunk(u * kWideThreads + tid, wv[u]);
  for (int cb = kWStage * kWideThreads; cb < NCHUNK; cb += kWStage * kWideThreads) {
#pragma unroll
    for (int u = 0; u < kWStage; ++u) wv[u] = load_chunk(cb + u * kWideThreads + tid);
#pragma unroll
    for (int u = 0; u < kWStage; ++u) store_chunk(cb + u * kWideThreads + tid, wv[u]);
  }
  __syncthreads();

  // Lanes past c_in must feed zeros (a non-finite dummy value times the zero
  // weights would still poison the sums); rows past the tile may feed anything,
  // their results go to the dump row.  The zeroing is an AND with a per-k-step mask
  // the compiler cannot see through: a select on the loaded value lets it sink the
  // loads into the select's branch, after the MFMAs, and the prefetch is lost.
  uint32_t kmask[KSTEPS];
#pragma unroll
  for (int q = 0; q < KSTEPS; ++q) {
    uint32_t m = (32 * q + 8 * sub < c_in) ? 0xFFFFFFFFu : 0u;
    asm("" : "+v"(m));
    kmask[q] = m;
  }
  auto take = [&](int) {
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
      for (int q = 0; q < KSTEPS; ++q)
        cur[b][q] = __builtin_bit_cast(F, __builtin_bit_cast(u32x4, raw[b][q]) & kmask[q]);
  };
  // The next round's source rows must be in registers wherever a round starts.
  // Waited for here and at the end of each round (they were requested before that
  // round's stores), so the loop head needs no wait: on this chip loads and stores
  // share one counter, and a wait there would also drain the previous round's
  // stores before the next operands are requested.
  auto rows_ready = [&]() {
    if constexpr (GATHER) {
#pragma unroll
      for (int b = 0; b < MB; ++b) asm volatile("" ::"v"(src[b]));
    }
  };
  int m0 = m_first;
  fetch_rows(m0 + STEP);
  take(m0);
  rows_ready();
  for (; m0 < r_end; m0 += STEP) {
    const int m1 = m0 + STEP;
    issue(m1);  // masked to the dummy address past the tile; lands during the MFMAs below
    fetch_rows(m1 + STEP);
    // keeps the W^T fragment reads inside the loop: hoisted, they would need
    // 4 * NTW * KSTEPS registers and spill
    asm volatile("" ::: "memory");
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      f32x4 acc[MB][NTC];
#pragma unroll
      for (int b = 0; b < MB; ++b)
#pragma unroll
        for (int t = 0; t < NTC; ++t) acc[b][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < KSTEPS; ++q) {
        // with two row blocks, one k-step's fragments at a time (the scheduler
        // would otherwise fetch a whole chunk's ahead and spill)
        if constexpr (MB > 1) asm volatile("" ::: "memory");
        F wf[NTC];
#pragma unroll
        for (int t = 0; t < NTC; ++t) wf[t] = M::load(lwp + 16 * (ch * NTC + t) * ldk + 32 * q);
#pragma unroll
        for (int t = 0; t < NTC; ++t)
#pragma unroll
          for (int b = 0; b < MB; ++b) acc[b][t] = M::mma(wf[t], cur[b][q], acc[b][t]);
      }
      // The partials leave through this wave's LDS stage: a lane holds 4 channels
      // of one row per tile (16 rows x 8 or 16 bytes per tile and store), and
      // stored straight the 16 rows would take 16 partial-line writes per store.
      // Staged, each store writes whole row segments of GC tiles (up to 128 bytes).
      // Lanes without a row store into the dump row instead of branching, so the
      // store count is fixed and the wait for the next blocks below skips the stores.
#pragma unroll
      for (int b = 0; b < MB; ++b) {
#pragma unroll
        for (int t0 = 0; t0 < NTC; t0 += GC) {
#pragma unroll
          for (int u = 0; u < GC; ++u)
            store4(reinterpret_cast<TO*>(stg + col * kStageRow) + 16 * u + 4 * sub, acc[b][t0 + u]);
          // the stage is written and read through different types: keep the compiler
          // from moving the reads above these writes, or the next segment's writes
          // above these reads (the LDS itself serves one wave's accesses in order)
          asm volatile("" ::: "memory");
#pragma unroll
          for (int h = 0; h < SREADS; ++h) {
            const int rr = lane / SLANES + SROWS * h;
            const int row = m0 + 16 * b + rr;
            // (with two lanes per row, rows 16..31 of the read repeat row 15 and are not stored)
            const uint4 v = *reinterpret_cast<const uint4*>(stg + (rr < 16 ? rr : 15) * kStageRow + (lane % SLANES) * 16);
            TO* dst = (row < row_lim ? C + (row0 + row) * (int64_t)c_out : dump) + n0 + nw +
                      16 * (ch * NTC + t0) + (lane % SLANES) * (16 / (int)sizeof(TO));
            if (rr < 16) {
              if (stream)
                store_stream(dst, v);
              else
                *reinterpret_cast<uint4*>(dst) = v;
            }
          }
          asm volatile("" ::: "memory");
        }
      }
    }
    take(m1);
    // the masked operands are complete here, not at the top of the next round:
    // there the compiler's wait would also cover the stores just issued
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
      for (int q = 0; q < KSTEPS; ++q) asm volatile("" ::"v"(cur[b][q]));
    rows_ready();
  }
}

// ---------------------------------------------------------------------------
// The submanifold centre offset inside the scatter (Section 2.2, Steps 2 and 3).
// For odd K the centre offset pairs every output with the input at the same sorted
// position, so its GEMM partial row would be written once and read back once.  Here
// the scatter computes it: the outputs go in blocks of 16 consecutive sorted
// positions, and CS waves share a block, each owning 16 * NTW of its output
// channels.  A wave multiplies the block's input rows by its slice of W_c on MFMA
// (W_c^T held in LDS for the workgroup's whole run: the grid is one round of
// workgroups that loop over the blocks), adds the other offsets' partial rows in
// ascending offset order and writes its slice of each output row once, with the
// optional residual + ReLU.  The grouped GEMM skips the centre offset.  A wave
// fetches the next block's table entries and row indices while it works on the
// current block, so a block costs one round trip for its operand and first partial
// rows (a partial row more per lane and NTW / 2 16-byte vectors in flight).
//
// Accumulator layout.  In the transposed product a lane owns 4 consecutive MFMA
// columns of one row per 16-column tile.  The columns of W_c^T in LDS are permuted
// so that tiles 2u and 2u + 1 of lane (row, sub) are the 8 consecutive channels
// 32u + 8 sub .. +7 of the wave's slice: each partial, residual and output access
// of a lane is one 16-byte vector (two for float32 partials), and a wave's access
// covers 64 contiguous bytes of each of its 16 rows.
constexpr int kCentreThreads = 768;  // 12 waves: three per SIMD, 168 registers each
constexpr int kCentreWaves = kCentreThreads / kWave;
constexpr int kCentreList = 28;  // table entries per row and batch (4 lanes x 7)
// (at 256 x 256 channels: 135,168 bytes of W_c^T plus 12 waves x 1,792 bytes of
// lists, 153 KiB of the 160 KiB of a CU)
constexpr size_t centre_lds(int nt, int ldk) {
  return (size_t)16 * nt * ldk * 2 + (size_t)kCentreWaves * 16 * kCentreList * 4;
}
// column tiles per wave: the most, up to 8 (128 channels), that split the row
// into a number of slices dividing the workgroup's waves
constexpr int centre_ntw(int nt) {
  for (int w = 8; w >= 2; w -= 2)
    if (nt % w == 0 && kCentreWaves % (nt / w) == 0) return w;
  return nt;
}
// physical channel of MFMA column n (tile t = n / 16, lane group s, element i)
__host__ __device__ constexpr int centre_phys(int n) {
  return 32 * ((n >> 4) >> 1) + 8 * ((n >> 2) & 3) + 4 * ((n >> 4) & 1) + (n & 3);
}
// and back
__host__ __device__ constexpr int centre_logical(int c) {
  return 16 * (2 * (c >> 5) + ((c >> 2) & 1)) + 4 * ((c >> 3) & 3) + (c & 3);
}

template <typename TP>
__device__ __forceinline__ void add8(f32x4& lo, f32x4& hi, const TP* p);
// f16: acc + h * 1.0 as one fused multiply-add per element, which the compiler can
// issue as a single mixed-precision FMA reading h from either half of a dword (the
// same single rounding as converting h exactly and adding)
// (the 1.0 is hidden from the compiler, which would otherwise fold the FMA into a
// conversion and an add)
template <>
__device__ __forceinline__ void add8<__half>(f32x4& lo, f32x4& hi, const __half* p) {
  const f16x8 v = *reinterpret_cast<const f16x8*>(p);
  float one = 1.0f;
  asm("" : "+v"(one));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    lo[i] = __builtin_fmaf((float)v[i], one, lo[i]);
    hi[i] = __builtin_fmaf((float)v[4 + i], one, hi[i]);
  }
}
template <>
__device__ __forceinline__ void add8<__hip_bfloat16>(f32x4& lo, f32x4& hi, const __hip_bfloat16* p) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    lo[2 * i] += __uint_as_float(v[i] << 16);
    lo[2 * i + 1] += __uint_as_float(v[i] & 0xFFFF0000u);
    hi[2 * i] += __uint_as_float(v[2 + i] << 16);
    hi[2 * i + 1] += __uint_as_float(v[2 + i] & 0xFFFF0000u);
  }
}
template <>
__device__ __forceinline__ void add8<float>(f32x4& lo, f32x4& hi, const float* p) {
  lo += *reinterpret_cast<const f32x4*>(p);
  hi += *reinterpret_cast<const f32x4*>(p + 4);
}

// 16 bytes of partial type TP at p, or zeros (mask 0); the AND keeps the load
// unconditional, so every load of a batch is requested before the first add.
template <typename TP>
struct PartVec {
  static constexpr int N = (int)sizeof(TP) / 2;  // 16-byte vectors per 8 channels
  u32x4 v[N];
  __device__ void load(const TP* p) {
#pragma unroll
    for (int j = 0; j < N; ++j) v[j] = reinterpret_cast<const u32x4*>(p)[j];
  }
  __device__ void add_to(f32x4& lo, f32x4& hi, uint32_t mask) const {
    u32x4 m[N];
#pragma unroll
    for (int j = 0; j < N; ++j) m[j] = v[j] & mask;
    add8<TP>(lo, hi, reinterpret_cast<const TP*>(m));
  }
};

// 8 float32 sums rounded to the layer type, as one 16-byte vector
__device__ __forceinline__ u32x4 pack8(__half*, const f32x4& lo, const f32x4& hi) {
  f16x8 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = (_Float16)lo[i];
    v[4 + i] = (_Float16)hi[i];
  }
  return __builtin_bit_cast(u32x4, v);
}
__device__ __forceinline__ u32x4 pack8(__hip_bfloat16*, const f32x4& lo, const f32x4& hi) {
  __hip_bfloat16 h[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = __float2bfloat16(lo[i]);
    h[4 + i] = __float2bfloat16(hi[i]);
  }
  return *reinterpret_cast<const u32x4*>(h);
}
// the value of lane i xor 8 (within each row of 16 lanes: a DPP row rotation by 8)
__device__ __forceinline__ uint32_t swap8(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false);
}

// T: layer type (operands and output); TP: partial type; NT = c_out / 16 (even);
// KSTEPS >= c_in / 32.  perm: caller row of each sorted position (NULL: identity),
// the same for inputs and outputs of a submanifold map.  wt: W^T ([K^3][c_out][c_in])
// or NULL (W_c is then transposed while staging).  residual may alias y.
template <typename T, typename TP, int NT, int KSTEPS>
__global__ __launch_bounds__(kCentreThreads) void k_scatter_centre(
    const T* __restrict__ x, const uint32_t* __restrict__ perm, const T* __restrict__ w, const T* __restrict__ wt,
    int kc, const TP* __restrict__ buf, const int32_t* __restrict__ omt, int64_t stride, int K3, T* y,
    const T* residual, int relu, int n_out, int c_in, int c_out, int ldk, int stream) {
  using M = Mfma<T>;
  using F = typename M::frag;
  static_assert(M::KS == 32, "16-bit operands only");
  static_assert(NT % 2 == 0, "channel pairs of tiles");
  constexpr int BN = 16 * NT;
  constexpr int KP = 32 * KSTEPS;
  constexpr int NTW = centre_ntw(NT);  // tiles per wave
  constexpr int CS = NT / NTW;         // waves per block
  constexpr int BPR = kCentreWaves / CS;  // blocks per workgroup round
  static_assert(kCentreWaves % CS == 0, "waves must split into whole blocks");
  constexpr int NU = NTW / 2;  // 16-byte output vectors per lane
  // partial rows requested together: their vectors take NTW * sizeof(TP) registers each
  // partial rows requested together: ENT in the round with the centre product (its
  // operands hold registers then), ENT2 in later rounds; an entry's vectors take
  // NTW * sizeof(TP) registers
  constexpr int ENT = (NTW * (int)sizeof(TP) <= 8) ? 4 : ((NTW * (int)sizeof(TP) <= 16) ? 2 : 1);
  constexpr int ENT2 = ENT;
  constexpr int NM = kCentreList / 4;  // table entries per lane and batch
  extern __shared__ __align__(16) unsigned char smem[];
  T* lw = reinterpret_cast<T*>(smem);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int sub = lane >> 4;
  const int col = lane & 15;
  const int cs = wave % CS;  // this wave's channel slice
  int32_t* list = reinterpret_cast<int32_t*>(smem + (size_t)BN * ldk * sizeof(T)) +
                  (wave * 16 + col) * kCentreList;

  // stage W_c^T, columns permuted: LDS row n holds channel centre_phys(n); a
  // thread's 16-byte chunks are requested in batches of kStage before they are
  // written (one at a time they would cost a round trip each)
  {
    const T* wc_t = wt ? wt + (int64_t)kc * c_out * c_in : nullptr;
    const T* wc = w + (int64_t)kc * c_in * c_out;
    constexpr int CH_T = KP / 8, CH_N = BN / 8;
    constexpr int NCHUNK = BN * KP / 8;
    constexpr int kStage = 8;
    for (int i0 = 0; i0 < NCHUNK; i0 += kStage * kCentreThreads) {
      uint4 v[kStage];
#pragma unroll
      for (int u = 0; u < kStage; ++u) {
        const int idx = i0 + u * kCentreThreads + tid;
        v[u] = make_uint4(0, 0, 0, 0);
        if (idx < NCHUNK) {
          if (wt) {
            const int n = idx / CH_T, c = (idx - n * CH_T) * 8;
            if (c < c_in) v[u] = *reinterpret_cast<const uint4*>(wc_t + (int64_t)centre_phys(n) * c_in + c);
          } else {
            const int c = idx / CH_N, n8 = (idx - c * CH_N) * 8;  // 8 physical channels of row c
            if (c < c_in) v[u] = *reinterpret_cast<const uint4*>(wc + (int64_t)c * c_out + n8);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kStage; ++u) {
        const int idx = i0 + u * kCentreThreads + tid;
        if (idx >= NCHUNK) continue;
        if (wt) {
          const int n = idx / CH_T, c = (idx - n * CH_T) * 8;
          *reinterpret_cast<uint4*>(lw + n * ldk + c) = v[u];
        } else {
          const int c = idx / CH_N, n8 = (idx - c * CH_N) * 8;
          const T* e = reinterpret_cast<const T*>(&v[u]);
#pragma unroll
          for (int j = 0; j < 8; ++j) lw[centre_logical(n8 + j) * ldk + c] = e[j];
        }
      }
    }
  }
  __syncthreads();

  const int klim = c_in - 8 * sub;  // k-steps q with 32 q >= klim are zeroed in this lane
  // the wave's slice: MFMA columns 16 NTW cs .. (LDS rows), channels 32 NU cs ..
  const T* lwp = lw + (16 * NTW * cs + col) * ldk + 8 * sub;
  const int ch0 = 32 * NU * cs + 8 * sub;
  const uint64_t rowmask = 0x0001000100010001ull << col;
  const int blocks = (n_out + 15) / 16;
  const int bstride = gridDim.x * BPR;
  // One batch of table entries: lane sub reads offsets kb + sub + 4 m.  The loads
  // are unconditional (index 0 where there is no entry, then OR-ed to -1 with a mask
  // the compiler cannot see through), so a batch is requested at once.  Table
  // indices fit 32 bits (K^3 * rows < 2^31).
  auto table = [&](int kb, int p, bool valid, int32_t* r) {
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      const int k = kb + sub + 4 * m;
      const bool has = valid && k < K3 && k != kc;
      uint32_t none = has ? 0u : 0xFFFFFFFFu;
      asm("" : "+v"(none));
      r[m] = omt[has ? k * (int)stride + p : 0] | (int32_t)none;
    }
  };
  // row index and first table batch of a block, fetched a block ahead
  auto fetch = [&](int blk, uint32_t* row, int32_t* r) {
    const int p = blk * 16 + col;
    const bool valid = blk < blocks && p < n_out;
    const int pc = valid ? p : 0;
    *row = perm ? perm[pc] : (uint32_t)pc;
    table(0, pc, valid, r);
  };
  // this row's listed table entries of one batch, in offset order, ranked with a
  // ballot over the row's four lanes; returns the row's count and the wave's largest
  auto build_list = [&](const int32_t* r, int* mx) {
    int cnt = 0;
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      const uint64_t bal = __ballot(r[m] >= 0) & rowmask;
      if (r[m] >= 0) list[cnt + popc64(bal & lanemask_lt())] = r[m];
      cnt += popc64(bal);
    }
    int x_ = cnt;
#pragma unroll
    for (int d = 1; d < 16; d <<= 1) x_ = max(x_, __shfl_xor(x_, d));
    *mx = x_;
    return cnt;
  };
  f32x4 acc[NTW];
  using First = std::integral_constant<bool, true>;
  using Later = std::integral_constant<bool, false>;

  int blk = blockIdx.x * BPR + wave / CS;
  uint32_t row_n;
  int32_t r_n[NM];
  fetch(blk, &row_n, r_n);
  // the centre operand of a block: its outputs' own input rows, requested one block
  // ahead (right after the previous block's MFMAs, into the same registers)
  F a[KSTEPS];
  auto load_a = [&](int64_t row) {
    const T* arow = x + row * c_in;
#pragma unroll
    for (int q = 0; q < KSTEPS; ++q) {
      const int kk = 32 * q + 8 * sub;
      a[q] = M::load(kk < c_in ? arow + kk : x);
    }
  };
  load_a(row_n);
  for (; blk < blocks; blk += bstride) {
    const int p = blk * 16 + col;
    const bool valid = p < n_out;
    const int64_t row = row_n;
    int mx;
    int cnt = build_list(r_n, &mx);
    fetch(blk + bstride, &row_n, r_n);
#pragma unroll
    for (int t = 0; t < NTW; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the centre's product comes first in every output's sum, then the other offsets
    // in ascending order; k past c_in is zeroed
    auto centre = [&]() {
#pragma unroll
      for (int q = 0; q < KSTEPS; ++q) {
        // one k-step's W fragments at a time (fetched all ahead they would spill)
        asm volatile("" ::: "memory");
        uint32_t km = (32 * q < klim) ? 0xFFFFFFFFu : 0u;
        asm("" : "+v"(km));
        const F b = __builtin_bit_cast(F, __builtin_bit_cast(u32x4, a[q]) & km);
#pragma unroll
        for (int t = 0; t < NTW; ++t) acc[t] = M::mma(M::load(lwp + 16 * t * ldk + 32 * q), b, acc[t]);
      }
    };
    // ENT listed partial rows from entry j0 on, requested together, then added; in
    // the first round the centre product runs while they are in flight
    auto partial_round = [&](int j0, int cnt, auto first) {
      constexpr int NE = decltype(first)::value ? ENT : ENT2;
      PartVec<TP> v[NE][NU];
      uint32_t msk[NE];
#pragma unroll
      for (int e = 0; e < NE; ++e) {
        const bool has = j0 + e < cnt;
        const int32_t rr = has ? list[j0 + e] : 0;
        msk[e] = has ? 0xFFFFFFFFu : 0u;
        asm("" : "+v"(msk[e]));
        const TP* src = buf + (int64_t)rr * c_out + ch0;
#pragma unroll
        for (int u = 0; u < NU; ++u) v[e][u].load(src + 32 * u);
      }
      if constexpr (decltype(first)::value) {
        asm volatile("" ::: "memory");
        centre();
        load_a(row_n);  // the next block's
      }
#pragma unroll
      for (int e = 0; e < NE; ++e)
#pragma unroll
        for (int u = 0; u < NU; ++u) v[e][u].add_to(acc[2 * u], acc[2 * u + 1], msk[e]);
    };
    partial_round(0, cnt, First{});
    for (int j0 = ENT; j0 < mx; j0 += ENT2) partial_round(j0, cnt, Later{});
    asm volatile("" ::: "memory");
    for (int kb = kCentreList; kb < K3; kb += kCentreList) {
      int32_t r[NM];
      table(kb, valid ? p : 0, valid, r);
      cnt = build_list(r, &mx);
      for (int j0 = 0; j0 < mx; j0 += ENT2) partial_round(j0, cnt, Later{});
      asm volatile("" ::: "memory");
    }
    if (residual && valid) {
      const T* rs = residual + row * (int64_t)c_out + ch0;
#pragma unroll
      for (int u = 0; u < NU; ++u) add8<T>(acc[2 * u], acc[2 * u + 1], rs + 32 * u);
    }
    if (relu) {
#pragma unroll
      for (int t = 0; t < NTW; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[t][i] = fmaxf(acc[t][i], 0.f);
    }
    if constexpr (NU % 2 == 0) {
      // Whole 128-byte lines: a lane holds, per 64-channel line L of its row, the
      // chunks 2L and 2L + 1 of its lane group.  Lanes of rows r and r + 8 (lanes
      // i and i xor 8) swap one chunk, so that one store writes line L of rows 0..7
      // (rows r < 8 their own chunk 2L, lanes of rows r + 8 the received chunk 2L + 1
      // of row r) and the next line L of rows 8..15.  Stores of 16 rows x 64 bytes
      // measured 30% slower than stores of whole lines.
      const bool lower = col < 8;
      const uint32_t row_o = swap8((uint32_t)row);
      const int64_t row_x = lower ? row : (int64_t)row_o, row_y = lower ? (int64_t)row_o : row;
      const bool valid_x = blk * 16 + (col & 7) < n_out, valid_y = blk * 16 + 8 + (col & 7) < n_out;
#pragma unroll
      for (int L = 0; L < NU / 2; ++L) {
        const u32x4 oa = pack8((T*)nullptr, acc[4 * L], acc[4 * L + 1]);
        const u32x4 ob = pack8((T*)nullptr, acc[4 * L + 2], acc[4 * L + 3]);
        const u32x4 send = lower ? ob : oa;
        u32x4 recv;
#pragma unroll
        for (int d = 0; d < 4; ++d) recv[d] = swap8(send[d]);
        const int ch = ch0 + 32 * (2 * L + (lower ? 0 : 1));
        const u32x4 dx = lower ? oa : recv, dy = lower ? recv : ob;
        T* px = y + row_x * (int64_t)c_out + ch;
        T* py = y + row_y * (int64_t)c_out + ch;
        if (stream) {
          if (valid_x) store_stream(px, make_uint4(dx[0], dx[1], dx[2], dx[3]));
          if (valid_y) store_stream(py, make_uint4(dy[0], dy[1], dy[2], dy[3]));
        } else {
          if (valid_x) *reinterpret_cast<u32x4*>(px) = dx;
          if (valid_y) *reinterpret_cast<u32x4*>(py) = dy;
        }
      }
    } else {
      if (valid) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          const u32x4 o = pack8((T*)nullptr, acc[2 * u], acc[2 * u + 1]);
          T* po = y + row * (int64_t)c_out + ch0 + 32 * u;
          if (stream)
            store_stream(po, make_uint4(o[0], o[1], o[2], o[3]));
          else
            *reinterpret_cast<u32x4*>(po) = o;
        }
      }
    }
  }
}


int centre_ksteps(int c_in) {
  const int ks = (c_in + 31) / 32;
  for (int c : {1, 2, 4, 8})
    if (ks <= c) return c;
  return 0;
}

template <typename T, typename TP>
const void* centre_kernel(int nt, int ks) {
#define SPC_C(N, KS_)                                                                                     \
  if constexpr (centre_lds(N, 32 * KS_ + 8) <= kLdsMax) {                                                 \
    if (nt == N && ks == KS_) return reinterpret_cast<const void*>(&k_scatter_centre<T, TP, N, KS_>);     \
  }
#define SPC_CK(N) SPC_C(N, 1) SPC_C(N, 2) SPC_C(N, 4) SPC_C(N, 8)
  SPC_CK(2) SPC_CK(4) SPC_CK(6) SPC_CK(8) SPC_CK(12) SPC_CK(16)
#undef SPC_CK
#undef SPC_C
  return nullptr;
}

const void* centre_kernel_for(int dtype, int part_dtype, int nt, int ks) {
  if (dtype == 1 && part_dtype == 1) return centre_kernel<__half, __half>(nt, ks);
  if (dtype == 1 && part_dtype == 0) return centre_kernel<__half, float>(nt, ks);
  if (dtype == 2 && part_dtype == 2) return centre_kernel<__hip_bfloat16, __hip_bfloat16>(nt, ks);
  if (dtype == 2 && part_dtype == 0) return centre_kernel<__hip_bfloat16, float>(nt, ks);
  return nullptr;
}

// k-steps instantiated for the wide kernel (c_in up to 512); others round up
int wide_ksteps(int c_in) {
  const int ks = (c_in + 31) / 32;
  for (int c : {1, 2, 3, 4, 6, 8, 12, 16})
    if (ks <= c) return c;
  return 0;
}

// Instantiated (NT, KSTEPS) pairs: the W^T slice fits the LDS.
constexpr bool wide_fits(int nt, int ks) { return wide_lds(nt, 32 * ks + 8) <= kLdsMax; }

// Column tiles per workgroup for the wide kernel: the widest instantiated divisor
// of c_out / 16 whose W^T slice fits the LDS; 0 if the wide kernel does not apply.
int wide_nt(int c_in, int c_out, int elem) {
  if (elem != 2 || c_in % 8 != 0 || c_out % 16 != 0) return 0;
  const int ks = wide_ksteps(c_in);
  if (ks == 0) return 0;
  const int ldk = 32 * ks + 8;
  const int nt_all = c_out / 16;
  for (int nt : {16, 12, 8, 6, 4, 3, 2, 1})
    if (nt_all % nt == 0 && wide_lds(nt, ldk) <= kLdsMax) return nt;
  return 0;
}

// Rows of one round of the workgroup (tiles are whole rounds).
int wide_round_rows(int nt, int ks) {
  const int cg = wide_cg(nt);
  return kWideWaves / cg * wide_mb(nt / cg, ks) * 16;
}

template <typename T, typename TO, bool GATHER>
const void* wide_kernel(int nt, int ks) {
#define SPC_W(N, KS_)                                                                                     \
  if constexpr (wide_fits(N, KS_)) {                                                                       \
    if (nt == N && ks == KS_) return reinterpret_cast<const void*>(&k_gemm_wide<T, TO, N, KS_, GATHER>); \
  }
#define SPC_WK(N) \
  SPC_W(N, 1) SPC_W(N, 2) SPC_W(N, 3) SPC_W(N, 4) SPC_W(N, 6) SPC_W(N, 8) SPC_W(N, 12) SPC_W(N, 16)
  SPC_WK(1) SPC_WK(2) SPC_WK(3) SPC_WK(4) SPC_WK(6) SPC_WK(8) SPC_WK(12) SPC_WK(16)
#undef SPC_WK
#undef SPC_W
  return nullptr;
}

const void* wide_kernel_for(int dtype, int part_dtype, bool gather, int nt, int ks) {
  if (dtype == 1 && part_dtype == 0)
    return gather ? wide_kernel<__half, float, true>(nt, ks) : wide_kernel<__half, float, false>(nt, ks);
  if (dtype == 1 && part_dtype == 1)
    return gather ? wide_kernel<__half, __half, true>(nt, ks) : wide_kernel<__half, __half, false>(nt, ks);
  if (dtype == 2 && part_dtype == 2)
    return gather ? wide_kernel<__hip_bfloat16, __hip_bfloat16, true>(nt, ks)
                  : wide_kernel<__hip_bfloat16, __hip_bfloat16, false>(nt, ks);
  if (dtype == 2 && part_dtype == 0)
    return gather ? wide_kernel<__hip_bfloat16, float, true>(nt, ks) : wide_kernel<__hip_bfloat16, float, false>(nt, ks);
  return nullptr;
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

// The same for c_in and c_out multiples of 64: 64 x 64 tiles, 16-byte loads and
// stores (each lane moves two 8-element row pieces each way) and a quarter of the
// workgroups (same-box A/B of the 300k-voxel layer: C = 256 0.4434 -> 0.4409 ms,
// C = 128 0.2759 -> 0.2744 ms).
__global__ __launch_bounds__(256) void k_transpose_w64(const uint16_t* __restrict__ w, uint16_t* __restrict__ wt,
                                                       int c_in, int c_out) {
  __shared__ uint16_t t[64][64 + 8];
  const int k = blockIdx.z;
  const int c0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const uint16_t* src = w + (int64_t)k * c_in * c_out;
  uint16_t* dst = wt + (int64_t)k * c_in * c_out;
  const int piece = threadIdx.x & 7, row = threadIdx.x >> 3;  // 8 pieces of 8 elements per row
  uint4 v[2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
    v[i] = *reinterpret_cast<const uint4*>(src + (int64_t)(c0 + row + 32 * i) * c_out + n0 + piece * 8);
#pragma unroll
  for (int i = 0; i < 2; ++i) *reinterpret_cast<uint4*>(&t[row + 32 * i][piece * 8]) = v[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int n = row + 32 * i;
    uint16_t e[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = t[piece * 8 + j][n];
    *reinterpret_cast<uint4*>(dst + (int64_t)(n0 + n) * c_in + c0 + piece * 8) = *reinterpret_cast<const uint4*>(e);
  }
}

template <typename T, typename TO>
hipError_t gemm_t(const GemmLaunchArgs& g, int total_tiles, const void* A, const int32_t* arows, const void* W,
                  void* C, int c_in, int c_out, int rows_per_tile, hipStream_t s) {
  const int KS = Mfma<T>::KS;
  const int kp = (c_in + KS - 1) / KS * KS;
  const int ldk = kp + 16 / (int)sizeof(T);
  // widest column slice whose W^T tile fits 64 KiB of LDS (a single 16-column tile
  // may take up to the 160 KiB of the CU: f32 at 1024 input channels needs 65.8 KB)
  const int nt_all = c_out / 16;
  int nt = 0;
  const int cand[] = {8, 6, 4, 3, 2, 1};
  for (int c : cand)
    if (nt_all % c == 0 && (size_t)16 * c * ldk * sizeof(T) <= (c == 1 ? kLdsMax : 65536)) {
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
    hipLaunchKernelGGL((k_gemm<T, TO, N>), grid, dim3(kThreads), lds, s, g, a, arows, w, c, c_in, c_out, kp, \
                       ldk, rows_per_tile);                                                          \
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

bool gemm_wide_transposed(int c_in, int c_out) { return c_in * c_out >= 128 * 128; }

bool gemm_wide(int c_in, int c_out, int dtype, int part_dtype) {
  // built for 16-bit operands with partials of the same type or of float32
  const bool pair = part_dtype == dtype || part_dtype == 0;
  return dtype != 0 && pair && wide_nt(c_in, c_out, 2) > 0;
}

hipError_t launch_transpose_w(const void* w, void* wt, int K3, int c_in, int c_out, hipStream_t s) {
  if (c_in % 64 == 0 && c_out % 64 == 0) {
    hipLaunchKernelGGL(k_transpose_w64, dim3((unsigned)(c_out / 64), (unsigned)(c_in / 64), (unsigned)K3), dim3(256), 0,
                       s, static_cast<const uint16_t*>(w), static_cast<uint16_t*>(wt), c_in, c_out);
    return hipGetLastError();
  }
  const dim3 grid((unsigned)((c_out + 31) / 32), (unsigned)((c_in + 31) / 32), (unsigned)K3);
  hipLaunchKernelGGL(k_transpose_w, grid, dim3(256), 0, s, static_cast<const uint16_t*>(w),
                     static_cast<uint16_t*>(wt), c_in, c_out);
  return hipGetLastError();
}

// Workgroups per CU of a wide-GEMM instance and the device's CU count, queried once
// per (device, kernel, LDS size) and kept (the queries cost the host microseconds
// on every forward otherwise).
hipError_t wide_occupancy(const void* fn, size_t lds, int* per_cu, int* cus, int threads = kWideThreads) {
  struct Entry {
    int dev;
    const void* fn;
    size_t lds;
    int per_cu, cus;
  };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  {
    std::lock_guard<std::mutex> lk(mu);
    for (const Entry& x : cache)
      if (x.dev == dev && x.fn == fn && x.lds == lds) {
        *per_cu = x.per_cu;
        *cus = x.cus;
        return hipSuccess;
      }
  }
  Entry x{dev, fn, lds, 0, 0};
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&x.per_cu, fn, threads, lds)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&x.cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  cache.push_back(x);
  *per_cu = x.per_cu;
  *cus = x.cus;
  return hipSuccess;
}

hipError_t launch_gemm(const GemmSeg* segs, int n_seg, const void* buf_in, const int32_t* a_rows, const void* w,
                       const void* wt, void* buf_out, void* dump_row, int c_in, int c_out, int dtype, int part_dtype,
                       int tile_rows, bool stream, hipStream_t s) {
  if (c_out % 16 != 0) return hipErrorInvalidValue;
  const bool wide = dump_row && gemm_wide(c_in, c_out, dtype, part_dtype);
  int64_t rows_all = 0;
  for (int i = 0; i < n_seg; ++i) rows_all += segs[i].height;
  int rows_per_tile = 64;
  const void* wfn = nullptr;
  int nt = 0, ks = 0, ldk = 0;
  size_t lds = 0;
  if (wide) {
    // about two tiles per workgroup slot: larger tiles amortise the W^T staging, and
    // two rounds of them keep the last round's idle CUs few; at least 512 rows (smaller
    // tiles measured slower: C = 256 GEMM 155 -> 150 us, 120k LiDAR layer 16.4 -> 15.5 us)
    nt = wide_nt(c_in, c_out, 2);
    ks = wide_ksteps(c_in);
    ldk = 32 * ks + 8;
    lds = wide_lds(nt, ldk);
    wfn = wide_kernel_for(dtype, part_dtype, a_rows != nullptr, nt, ks);
    if (!wfn) return hipErrorInvalidValue;
    int per_cu = 0, cus = 0;
    hipError_t e = wide_occupancy(wfn, lds, &per_cu, &cus);
    if (e != hipSuccess) return e;
    const int64_t slots = (int64_t)std::max(per_cu, 1) * std::max(cus, 1);
    const int round = wide_round_rows(nt, ks);
    const int64_t want = tile_rows > 0 ? tile_rows : std::max<int64_t>(512, (rows_all + 2 * slots - 1) / (2 * slots));
    const int64_t cap = tile_rows > 0 ? (int64_t)1 << 20 : 16 * round;
    rows_per_tile = (int)std::min<int64_t>(std::max<int64_t>((want + round - 1) / round, 1) * round, cap);
  } else if (tile_rows > 0) {
    rows_per_tile = (tile_rows + 15) / 16 * 16;
  } else {
    // enough workgroups to fill 256 CUs several times, at most 1024 rows each
    while (rows_per_tile < 1024 && rows_all / (rows_per_tile * 2) >= 2048) rows_per_tile *= 2;
  }
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
      ProfScope ps(KN_GEMM, s);
      int nsl = c_out / 16 / nt;  // column slices per tile
      const dim3 grid = nsl > 1 ? dim3((unsigned)((tiles + 7) / 8 * 8 * nsl)) : dim3((unsigned)tiles);
      const void* a = buf_in;
      const void* wtp = wt;
      void* c = buf_out;
      void* d = dump_row;
      const void* wp = w;
      const int32_t* ar = a_rows;
      int st = stream ? 1 : 0;
      void* args[] = {&g, &a, &ar, &wp, &wtp, &c, &d, &c_in, &c_out, &ldk, &rows_per_tile, &nsl, &st};
      e = hipLaunchKernel(wfn, grid, dim3(kWideThreads), args, lds, s);
    } else if (dtype == 0 && part_dtype == 0)
      e = gemm_t<float, float>(g, tiles, buf_in, a_rows, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 1 && part_dtype == 0)
      e = gemm_t<__half, float>(g, tiles, buf_in, a_rows, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 1 && part_dtype == 1)
      e = gemm_t<__half, __half>(g, tiles, buf_in, a_rows, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 2 && part_dtype == 0)
      e = gemm_t<__hip_bfloat16, float>(g, tiles, buf_in, a_rows, w, buf_out, c_in, c_out, rows_per_tile, s);
    else if (dtype == 2 && part_dtype == 2)
      e = gemm_t<__hip_bfloat16, __hip_bfloat16>(g, tiles, buf_in, a_rows, w, buf_out, c_in, c_out, rows_per_tile, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}


bool centre_fusable(int c_in, int c_out, int dtype, int part_dtype) {
  if ((dtype != 1 && dtype != 2) || c_in % 8 != 0 || c_out % 32 != 0) return false;
  const int ks = centre_ksteps(c_in);
  return ks > 0 && centre_kernel_for(dtype, part_dtype, c_out / 16, ks) != nullptr;
}

hipError_t launch_scatter_centre(const void* x, const uint32_t* perm, const void* w, const void* wt, int kc,
                                 const void* buf_out, const int32_t* omt, int64_t mt_stride, int K3, void* y,
                                 const void* residual, int relu, int64_t n_out, int c_in, int c_out, int dtype,
                                 int part_dtype, bool stream, hipStream_t s) {
  if (n_out <= 0) return hipSuccess;
  const int nt = c_out / 16, ks = centre_ksteps(c_in);
  const void* fn = (c_out % 32 == 0 && ks > 0) ? centre_kernel_for(dtype, part_dtype, nt, ks) : nullptr;
  if (!fn || n_out >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  int ldk = 32 * ks + 8;
  const size_t lds = centre_lds(nt, ldk);
  int per_cu = 0, cus = 0;
  hipError_t e = wide_occupancy(fn, lds, &per_cu, &cus, kCentreThreads);
  if (e != hipSuccess) return e;
  // one round of workgroups; each wave walks 16-output blocks strided by the grid
  const int64_t blocks = (n_out + 15) / 16;
  const int64_t bpr = kCentreWaves / (nt / centre_ntw(nt));  // blocks per workgroup round
  const int64_t need = (blocks + bpr - 1) / bpr;
  const unsigned grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>(need, (int64_t)std::max(per_cu, 1) * std::max(cus, 1)));
  ProfScope ps(KN_SCATTER_CENTRE, s);
  int n = (int)n_out;
  int st = stream ? 1 : 0;
  void* args[] = {&x, &perm, &w, &wt, &kc, &buf_out, &omt, &mt_stride, &K3, &y, &residual, &relu, &n, &c_in, &c_out, &ldk, &st};
  e = hipLaunchKernel(fn, dim3(grid), dim3(kCentreThreads), args, lds, s);
  return e;
}

}  // namespace spc
