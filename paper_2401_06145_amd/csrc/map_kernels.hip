// Map step kernels (Section 5.1): coordinate keys, radix sort, output
// coordinates (Eq. 1), and the segmented-query double-traversed binary search
// (Section 5.1.2) with in-order compaction of matches into per-offset pair lists.
#include <climits>

#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 256;

__global__ void k_fill_u32(uint32_t* p, uint32_t v, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

unsigned grid_for(int64_t n, int per_block = kThreads, int64_t cap = 1 << 20) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

// ----------------------------------------------------------------------------
// Coordinate bounds (for the key layout)
// ----------------------------------------------------------------------------
__global__ void k_minmax_init(ControlBlock* cb) {
  const int t = threadIdx.x;
  if (t < 4) {
    cb->minmax[t] = INT_MAX;
    cb->minmax[4 + t] = INT_MIN;
  }
  if (t == 0) {
    cb->err = 0;
    cb->n_q = 0;
    cb->n_items = 0;
    cb->ticket = 0;
  }
}

__global__ __launch_bounds__(kThreads) void k_minmax(const int4* c, int64_t n, ControlBlock* cb) {
  int32_t mn[4] = {INT_MAX, INT_MAX, INT_MAX, INT_MAX};
  int32_t mx[4] = {INT_MIN, INT_MIN, INT_MIN, INT_MIN};
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int4 v = c[i];
    const int32_t a[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      mn[f] = min(mn[f], a[f]);
      mx[f] = max(mx[f], a[f]);
    }
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      mn[f] = min(mn[f], __shfl_xor(mn[f], off, kWave));
      mx[f] = max(mx[f], __shfl_xor(mx[f], off, kWave));
    }
  }
  if ((threadIdx.x & (kWave - 1)) == 0) {
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      atomicMin(&cb->minmax[f], mn[f]);
      atomicMax(&cb->minmax[4 + f], mx[f]);
    }
  }
}

// ----------------------------------------------------------------------------
// Key packing
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_pack(const int4* c, int64_t n, KeyLayout L, uint64_t* keys,
                                                   uint32_t* vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int4 v = c[i];
  const int32_t a[4] = {v.x, v.y, v.z, v.w};
  keys[i] = pack_key(L, a);
  vals[i] = (uint32_t)i;
}

__global__ __launch_bounds__(kThreads) void k_unpack(const uint64_t* keys, int64_t n, KeyLayout L, int4* c) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t k = keys[i];
  c[i] = make_int4(key_field(L, k, 0), key_field(L, k, 1), key_field(L, k, 2), key_field(L, k, 3));
}

__global__ __launch_bounds__(kThreads) void k_check_dup(const uint64_t* keys, int64_t n, ControlBlock* cb) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x + 1;
  if (i < n && keys[i] == keys[i - 1]) atomicOr(&cb->err, kErrDup);
}

// ----------------------------------------------------------------------------
// LSD radix sort of (u64 key, u32 value), 8-bit digits, stable.
// Per pass: per-tile digit histograms -> exclusive scan (digit-major) -> stable
// scatter.  Ranks inside a tile come from wave64 ballots that match equal digits.
// ----------------------------------------------------------------------------
constexpr int kRsItems = 8;
constexpr int kRsTile = kThreads * kRsItems;

// Lanes of the wave whose digit equals this lane's digit (among active lanes).
__device__ __forceinline__ uint64_t match_digit(uint32_t d) {
  uint64_t m = __ballot(1);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (d >> b) & 1u;
    const uint64_t bal = __ballot(bit);
    m &= bit ? bal : ~bal;
  }
  return m;
}

__global__ __launch_bounds__(kThreads) void k_radix_hist(const uint64_t* keys, int64_t n, int shift,
                                                         uint32_t* hist, int64_t ntiles) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kRsTile;
#pragma unroll
  for (int r = 0; r < kRsItems; ++r) {
    const int64_t i = base + r * kThreads + threadIdx.x;
    if (i < n) {
      const uint32_t d = (uint32_t)(keys[i] >> shift) & 255u;
      const uint64_t peers = match_digit(d);
      if ((peers & lanemask_lt()) == 0) atomicAdd(&h[d], (uint32_t)popc64(peers));
    }
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(kThreads) void k_radix_scatter(const uint64_t* kin, const uint32_t* vin,
                                                            uint64_t* kout, uint32_t* vout, int64_t n,
                                                            int shift, const uint32_t* offs,
                                                            int64_t ntiles) {
  __shared__ uint32_t run[256];
  __shared__ uint32_t wcnt[kThreads / kWave][256];
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  run[tid] = offs[(int64_t)tid * ntiles + blockIdx.x];
#pragma unroll
  for (int w = 0; w < kThreads / kWave; ++w) wcnt[w][tid] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kRsTile;
  for (int r = 0; r < kRsItems; ++r) {
    const int64_t i = base + r * kThreads + tid;
    const bool valid = i < n;
    uint64_t key = 0;
    uint32_t val = 0, d = 0, rank = 0;
    if (valid) {
      key = kin[i];
      val = vin[i];
      d = (uint32_t)(key >> shift) & 255u;
      const uint64_t peers = match_digit(d);
      rank = (uint32_t)popc64(peers & lanemask_lt());
      if (rank == 0) wcnt[wave][d] = (uint32_t)popc64(peers);
    }
    __syncthreads();
    if (valid) {
      uint32_t pos = run[d] + rank;
      for (int w = 0; w < wave; ++w) pos += wcnt[w][d];
      kout[pos] = key;
      vout[pos] = val;
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int w = 0; w < kThreads / kWave; ++w) {
      add += wcnt[w][tid];
      wcnt[w][tid] = 0;
    }
    run[tid] += add;
    __syncthreads();
  }
}

// ----------------------------------------------------------------------------
// Output coordinates of a downsampling layer (Eq. 1): floor each spatial field
// to a multiple of the cell t*s; b is kept.
// ----------------------------------------------------------------------------
__device__ __forceinline__ int64_t floor_to_cell(int64_t v, int64_t cell) {
  int64_t q = v / cell;
  if (v % cell != 0 && v < 0) q -= 1;
  return q * cell;
}

__global__ __launch_bounds__(kThreads) void k_down_keys(const uint64_t* skeys, int64_t n, KeyLayout L,
                                                        int64_t cell, uint64_t* dkeys, uint32_t* vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t k = skeys[i];
  int32_t c[4];
  c[0] = key_field(L, k, 0);
#pragma unroll
  for (int f = 1; f < 4; ++f) c[f] = (int32_t)floor_to_cell(key_field(L, k, f), cell);
  dkeys[i] = pack_key(L, c);
  vals[i] = (uint32_t)i;
}

__global__ __launch_bounds__(kThreads) void k_unique_flags(const uint64_t* keys, int64_t n, uint32_t* flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  flags[i] = (i == 0 || keys[i] != keys[i - 1]) ? 1u : 0u;
}

__global__ __launch_bounds__(kThreads) void k_unique_write(const uint64_t* keys, int64_t n, KeyLayout L,
                                                           const uint32_t* flags, const uint32_t* pos,
                                                           uint64_t* qkeys, uint32_t* qrow, int4* coords) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n || flags[i] == 0) return;
  const uint32_t p = pos[i];
  const uint64_t k = keys[i];
  qkeys[p] = k;
  qrow[p] = p;
  coords[p] = make_int4(key_field(L, k, 0), key_field(L, k, 1), key_field(L, k, 2), key_field(L, k, 3));
}

// ----------------------------------------------------------------------------
// Backward binary search (Section 5.1.2): for source block b and offset k, the
// query block is the run of sorted queries q with key(q) + dk in
// (pivot_{b-1}, pivot_b], pivot_b being the block's last key.  bounds[k][b] is
// the number of queries with key(q) + dk <= pivot_b (an upper bound), found by
// one wave with a 64-way ballot search: each round every lane tests one probe.
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_backward(SearchArgs a, int64_t nb, uint32_t* bounds) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wid = (int64_t)blockIdx.x * (kThreads / kWave) + threadIdx.x / kWave;
  if (wid >= (int64_t)a.K3 * nb) return;  // wave-uniform
  const int k = (int)(wid / nb);
  const int64_t b = wid - (int64_t)k * nb;
  const int64_t nq = a.n_q_dev ? (int64_t)*a.n_q_dev : a.n_q;
  const int64_t last = min((b + 1) * (int64_t)a.B, a.n_src) - 1;
  // key(q) + dk <= pivot  <=>  key(q) <= pivot - dk, evaluated in signed 64 bits
  const int64_t thr = (int64_t)a.skeys[last] - a.dk[k];
  int64_t lo = 0, hi = nq;  // answer in [lo, hi]
  while (hi - lo > kWave) {
    const int64_t step = (hi - lo + kWave - 1) / kWave;
    const int64_t pos = lo + (int64_t)(lane + 1) * step - 1;
    const bool pred = pos < hi && (int64_t)a.qkeys[pos] <= thr;
    const int c = popc64(__ballot(pred));
    const int64_t nlo = lo + (int64_t)c * step;
    const int64_t nhi = min(lo + (int64_t)(c + 1) * step - 1, hi);
    lo = nlo;
    hi = nhi;
  }
  const int64_t pos = lo + lane;
  const bool pred = pos < hi && (int64_t)a.qkeys[pos] <= thr;
  const int64_t ub = lo + popc64(__ballot(pred));
  if (lane == 0) bounds[wid] = (uint32_t)ub;
}

// Balance (Section 5.1.2): query blocks larger than Cq are split into chunks.
__global__ __launch_bounds__(kThreads) void k_chunks(const uint32_t* bounds, int64_t nkb, int64_t nb, int Cq,
                                                     uint32_t* chunks) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nkb) return;
  const int64_t b = i % nb;
  const uint32_t lo = (b == 0) ? 0u : bounds[i - 1];
  const uint32_t hi = bounds[i];
  chunks[i] = (hi - lo + (uint32_t)Cq - 1u) / (uint32_t)Cq;
}

__global__ __launch_bounds__(kThreads) void k_emit(const uint32_t* chunks, const uint32_t* start, int64_t nkb,
                                                   int2* items, uint64_t* status, int64_t max_items,
                                                   ControlBlock* cb) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) cb->ticket = 0;
  if (i >= nkb) return;
  const uint32_t c = chunks[i];
  const uint32_t s = start[i];
  for (uint32_t j = 0; j < c; ++j) {
    const int64_t w = (int64_t)s + j;
    if (w >= max_items) {
      atomicOr(&cb->err, kErrOverflow);
      return;
    }
    items[w] = make_int2((int)i, (int)j);
    status[w] = 0ull;
  }
}

// ----------------------------------------------------------------------------
// Forward binary search (Section 5.1.2) + compaction.  One workgroup per
// load-balanced query block: the source block goes to LDS, each lane binary-
// searches its queries there.  Matches are ranked with wave ballots and the
// workgroup's base position comes from a decoupled look-back over work items,
// so the pair lists are written in (offset, sorted query) order in one pass.
// ----------------------------------------------------------------------------
constexpr uint64_t kFlagAgg = 1ull << 62;
constexpr uint64_t kFlagIncl = 2ull << 62;
constexpr uint64_t kValMask = (1ull << 62) - 1ull;
constexpr uint32_t kSpinLimit = 1u << 22;

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

template <int ROUNDS>
__global__ __launch_bounds__(kThreads) void k_forward(SearchArgs a, const uint32_t* bounds, int64_t nb,
                                                      const int2* items, uint64_t* status, int32_t* pin,
                                                      int32_t* pout, uint32_t* counts, ControlBlock* cb,
                                                      int log2B) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ uint32_t s_ticket;
  __shared__ uint32_t s_cnt[ROUNDS][kThreads / kWave];
  __shared__ uint64_t s_base;
  uint64_t* lkey = reinterpret_cast<uint64_t*>(smem);
  uint32_t* lidx = reinterpret_cast<uint32_t*>(smem + sizeof(uint64_t) * a.B);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;

  if (tid == 0) s_ticket = atomicAdd(&cb->ticket, 1u);
  __syncthreads();
  const uint32_t w = s_ticket;
  if (w >= cb->n_items) return;  // workgroup-uniform; later tickets are idle too

  const int2 it = items[w];
  const int64_t kb = it.x;
  const int k = (int)(kb / nb);
  const int64_t b = kb - (int64_t)k * nb;
  const int64_t blo = (b == 0) ? 0 : (int64_t)bounds[kb - 1];
  const int64_t bhi = bounds[kb];
  const int64_t q0 = blo + (int64_t)it.y * a.Cq;
  const int64_t q1 = min(q0 + (int64_t)a.Cq, bhi);

  const int64_t s0 = b * (int64_t)a.B;
  const int nB = (int)min((int64_t)a.B, a.n_src - s0);
  for (int e = tid; e < nB; e += kThreads) {
    lkey[e] = a.skeys[s0 + e];
    lidx[e] = a.sidx[s0 + e];
  }
  __syncthreads();

  const int64_t dk = a.dk[k];
  int32_t r_in[ROUNDS], r_out[ROUNDS];
  uint64_t bal[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int64_t qp = q0 + (int64_t)r * kThreads + tid;
    bool hit = false;
    r_in[r] = 0;
    r_out[r] = 0;
    if (qp < q1) {
      const uint64_t key = a.qkeys[qp] + (uint64_t)dk;
      // number of LDS keys < key, by binary lifting over a power-of-two range
      int pos = 0;
      for (int step = 1 << (log2B - 1); step > 0; step >>= 1)
        if (pos + step <= nB && lkey[pos + step - 1] < key) pos += step;
      if (pos < nB && lkey[pos] < key) ++pos;
      if (pos < nB && lkey[pos] == key) {
        hit = true;
        const int32_t src = (int32_t)lidx[pos];
        const int32_t qry = (int32_t)a.qrow[qp];
        r_in[r] = a.swap_roles ? qry : src;
        r_out[r] = a.swap_roles ? src : qry;
      }
    }
    bal[r] = __ballot(hit);
    if (lane == 0) s_cnt[r][wave] = (uint32_t)popc64(bal[r]);
  }
  __syncthreads();

  // block-local exclusive offsets in (round, wave) order
  uint32_t total = 0;
  uint32_t before[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
#pragma unroll
    for (int v = 0; v < kThreads / kWave; ++v) {
      if (v == wave) before[r] = total;
      total += s_cnt[r][v];
    }
  }

  if (wave == 0) {
    uint64_t excl = 0;
    if (w == 0) {
      if (lane == 0) st_release_agent(&status[0], kFlagIncl | (uint64_t)total);
    } else {
      if (lane == 0) st_release_agent(&status[w], kFlagAgg | (uint64_t)total);
      int64_t p = (int64_t)w - 1;
      uint32_t spins = 0;
      while (true) {
        const int64_t idx = p - lane;
        const uint64_t sv = (idx >= 0) ? ld_acquire_agent(&status[idx]) : kFlagIncl;
        const uint32_t flag = (uint32_t)(sv >> 62);
        if (__ballot(flag == 0) != 0) {
          if (++spins > kSpinLimit) {
            if (lane == 0) atomicOr(&cb->err, kErrSpin);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
          continue;
        }
        const uint64_t incl = __ballot(flag == 2);
        const uint64_t val = sv & kValMask;
        if (incl != 0) {
          const int first = __ffsll((unsigned long long)incl) - 1;
          excl += wave_sum_u64(lane <= first ? val : 0ull);
          break;
        }
        excl += wave_sum_u64(val);
        p -= kWave;
      }
      if (lane == 0) st_release_agent(&status[w], kFlagIncl | (excl + (uint64_t)total));
    }
    if (lane == 0) s_base = excl;
  }
  __syncthreads();
  const uint64_t base = s_base;
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    if ((bal[r] >> lane) & 1ull) {
      const uint64_t o = base + before[r] + (uint64_t)popc64(bal[r] & lanemask_lt());
      pin[o] = r_in[r];
      pout[o] = r_out[r];
    }
  }
  if (tid == 0 && total != 0) atomicAdd(&counts[k], total);
}

}  // namespace

// ----------------------------------------------------------------------------
// Launchers
// ----------------------------------------------------------------------------
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(n, kThreads, 4096)), dim3(kThreads), 0, s, p, v, n);
  return hipGetLastError();
}

hipError_t launch_minmax_init(ControlBlock* cb, hipStream_t s) {
  hipLaunchKernelGGL(k_minmax_init, dim3(1), dim3(64), 0, s, cb);
  return hipGetLastError();
}

hipError_t launch_minmax(const int32_t* coords, int64_t n, ControlBlock* cb, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_minmax, dim3(grid_for(n, kThreads, 1024)), dim3(kThreads), 0, s,
                     reinterpret_cast<const int4*>(coords), n, cb);
  return hipGetLastError();
}

hipError_t launch_pack(const int32_t* coords, int64_t n, KeyLayout L, uint64_t* keys, uint32_t* vals,
                       hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_pack, dim3(grid_for(n)), dim3(kThreads), 0, s, reinterpret_cast<const int4*>(coords),
                     n, L, keys, vals);
  return hipGetLastError();
}

hipError_t launch_unpack(const uint64_t* keys, int64_t n, KeyLayout L, int32_t* coords, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_unpack, dim3(grid_for(n)), dim3(kThreads), 0, s, keys, n, L,
                     reinterpret_cast<int4*>(coords));
  return hipGetLastError();
}

hipError_t launch_check_dup(const uint64_t* keys, int64_t n, ControlBlock* cb, hipStream_t s) {
  if (n <= 1) return hipSuccess;
  hipLaunchKernelGGL(k_check_dup, dim3(grid_for(n - 1)), dim3(kThreads), 0, s, keys, n, cb);
  return hipGetLastError();
}

size_t radix_temp_bytes(int64_t n) {
  const int64_t ntiles = (n + kRsTile - 1) / kRsTile;
  const int64_t nh = 256 * (ntiles < 1 ? 1 : ntiles);
  return (((size_t)nh * sizeof(uint32_t) + 255) & ~(size_t)255) + scan_temp_bytes(nh);
}

hipError_t radix_sort_kv(uint64_t* keys, uint32_t* vals, uint64_t* keys_alt, uint32_t* vals_alt, int64_t n,
                         int bits, void* d_temp, hipStream_t s) {
  if (n <= 1 || bits <= 0) return hipSuccess;
  const int64_t ntiles = (n + kRsTile - 1) / kRsTile;
  uint32_t* hist = static_cast<uint32_t*>(d_temp);
  void* scan_tmp = static_cast<char*>(d_temp) + (((size_t)256 * ntiles * sizeof(uint32_t) + 255) & ~(size_t)255);
  uint64_t* ka = keys;
  uint32_t* va = vals;
  uint64_t* kb = keys_alt;
  uint32_t* vb = vals_alt;
  const int passes = (bits + 7) / 8;
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    hipLaunchKernelGGL(k_radix_hist, dim3((unsigned)ntiles), dim3(kThreads), 0, s, ka, n, shift, hist, ntiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = scan_exclusive_u32(hist, hist, 256 * ntiles, nullptr, scan_tmp, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_radix_scatter, dim3((unsigned)ntiles), dim3(kThreads), 0, s, ka, va, kb, vb, n, shift,
                       hist, ntiles);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    uint64_t* tk = ka;
    ka = kb;
    kb = tk;
    uint32_t* tv = va;
    va = vb;
    vb = tv;
  }
  if (ka != keys) {
    hipError_t e = hipMemcpyAsync(keys, ka, (size_t)n * sizeof(uint64_t), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
    e = hipMemcpyAsync(vals, va, (size_t)n * sizeof(uint32_t), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_down_keys(const uint64_t* skeys, int64_t n, KeyLayout L, int64_t cell, uint64_t* dkeys,
                            uint32_t* vals, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_down_keys, dim3(grid_for(n)), dim3(kThreads), 0, s, skeys, n, L, cell, dkeys, vals);
  return hipGetLastError();
}

hipError_t unique_keys(const uint64_t* keys, int64_t n, KeyLayout L, uint32_t* flags, uint32_t* pos,
                       void* d_temp, uint64_t* qkeys, uint32_t* qrow, int32_t* out_coords, ControlBlock* cb,
                       hipStream_t s) {
  if (n <= 0) return launch_fill_u32(&cb->n_q, 0u, 1, s);
  hipLaunchKernelGGL(k_unique_flags, dim3(grid_for(n)), dim3(kThreads), 0, s, keys, n, flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = scan_exclusive_u32(flags, pos, n, &cb->n_q, d_temp, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_unique_write, dim3(grid_for(n)), dim3(kThreads), 0, s, keys, n, L, flags, pos, qkeys,
                     qrow, reinterpret_cast<int4*>(out_coords));
  return hipGetLastError();
}

hipError_t launch_backward(const SearchArgs& a, int64_t nb, uint32_t* bounds, hipStream_t s) {
  const int64_t waves = (int64_t)a.K3 * nb;
  if (waves <= 0) return hipSuccess;
  const int64_t blocks = (waves + (kThreads / kWave) - 1) / (kThreads / kWave);
  hipLaunchKernelGGL(k_backward, dim3((unsigned)blocks), dim3(kThreads), 0, s, a, nb, bounds);
  return hipGetLastError();
}

hipError_t balance(const SearchArgs& a, int64_t nb, const uint32_t* bounds, uint32_t* chunks, uint32_t* item_start,
                   void* d_temp, int32_t* items, uint64_t* status, int64_t max_items, ControlBlock* cb,
                   hipStream_t s) {
  const int64_t nkb = (int64_t)a.K3 * nb;
  if (nkb <= 0) return launch_fill_u32(&cb->n_items, 0u, 1, s);
  hipLaunchKernelGGL(k_chunks, dim3(grid_for(nkb)), dim3(kThreads), 0, s, bounds, nkb, nb, a.Cq, chunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = scan_exclusive_u32(chunks, item_start, nkb, &cb->n_items, d_temp, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_emit, dim3(grid_for(nkb)), dim3(kThreads), 0, s, chunks, item_start, nkb,
                     reinterpret_cast<int2*>(items), status, max_items, cb);
  return hipGetLastError();
}

hipError_t launch_forward(const SearchArgs& a, const uint32_t* bounds, int64_t nb, const int32_t* items,
                          uint64_t* status, int64_t max_items, int32_t* pin, int32_t* pout, uint32_t* counts,
                          ControlBlock* cb, hipStream_t s) {
  if (max_items <= 0 || nb <= 0) return hipSuccess;
  int log2B = 0;
  while ((1 << log2B) < a.B) ++log2B;
  const size_t lds = (size_t)a.B * (sizeof(uint64_t) + sizeof(uint32_t));
  const int rounds = a.Cq / kThreads;
  const int2* it = reinterpret_cast<const int2*>(items);
  switch (rounds) {
    case 1:
      hipLaunchKernelGGL(k_forward<1>, dim3((unsigned)max_items), dim3(kThreads), lds, s, a, bounds, nb, it,
                         status, pin, pout, counts, cb, log2B);
      break;
    case 2:
      hipLaunchKernelGGL(k_forward<2>, dim3((unsigned)max_items), dim3(kThreads), lds, s, a, bounds, nb, it,
                         status, pin, pout, counts, cb, log2B);
      break;
    case 4:
      hipLaunchKernelGGL(k_forward<4>, dim3((unsigned)max_items), dim3(kThreads), lds, s, a, bounds, nb, it,
                         status, pin, pout, counts, cb, log2B);
      break;
    case 8:
      hipLaunchKernelGGL(k_forward<8>, dim3((unsigned)max_items), dim3(kThreads), lds, s, a, bounds, nb, it,
                         status, pin, pout, counts, cb, log2B);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace spc
