// Map step kernels (Section 5.1): coordinate keys, radix sort, output
// coordinates (Eq. 1), and the segmented-query double-traversed binary search
// (Section 5.1.2) with in-order compaction of matches into per-offset pair lists.
//
// MI355X notes: atomics on one address from many workgroups serialise across the
// eight XCDs, so no kernel here has such a hot spot: reductions go through
// per-block partials, and the match compaction is count -> scan -> write (the
// count pass leaves each query's search result in the query-side table, which
// the write pass reads back) instead of a single pass with a look-back.
#include <algorithm>
#include <climits>

#include "common.h"

namespace spc {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

__global__ void k_fill_u32(uint32_t* p, uint32_t v, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

unsigned grid_for(int64_t n, int per_block = kThreads, int64_t cap = 1 << 20) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (unsigned)g;
}

// ----------------------------------------------------------------------------
// Coordinate bounds: per-block partial min / max, then one block reduces them.
// ----------------------------------------------------------------------------
constexpr int kMinmaxBlocks = 256;
constexpr int kMinmaxBatch = 8;  // rows in flight per thread
constexpr int kMaxPartials = kMinmaxBlocks;  // bounds partials reduced by the layout kernel

// Per-block bounds of the coordinates; the device reduces the partials and lays
// out the keys (inside the first sort histogram, or k_layout), so the host does
// not wait for them.  Block 0 also resets the control block's counters for the
// map build.
__global__ __launch_bounds__(kThreads) void k_minmax_partial(const int4* a, int64_t na, const int4* b, int64_t nb,
                                                             int32_t* partial, ControlBlock* cb) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    cb->err = 0;
    cb->n_q = 0;
    cb->n_pairs = 0;
  }
  int32_t mn[4] = {INT_MAX, INT_MAX, INT_MAX, INT_MAX};
  int32_t mx[4] = {INT_MIN, INT_MIN, INT_MIN, INT_MIN};
  const int64_t n = na + nb;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // batches of kMinmaxBatch rows per thread, all requested before the first is used
  // (rows past n re-read row n - 1, which leaves the bounds unchanged)
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += kMinmaxBatch * stride) {
    int4 v[kMinmaxBatch];
#pragma unroll
    for (int u = 0; u < kMinmaxBatch; ++u) {
      const int64_t i = min(i0 + u * stride, n - 1);
      v[u] = *((i < na) ? a + i : b + (i - na));
    }
#pragma unroll
    for (int u = 0; u < kMinmaxBatch; ++u) {
      const int32_t c[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        mn[f] = min(mn[f], c[f]);
        mx[f] = max(mx[f], c[f]);
      }
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
  __shared__ int32_t s[kWavesPerBlock][8];
  const int wave = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      s[wave][f] = mn[f];
      s[wave][4 + f] = mx[f];
    }
  }
  __syncthreads();
  if (threadIdx.x < 8) {
    const int f = threadIdx.x;
    int32_t r = s[0][f];
    for (int w = 1; w < kWavesPerBlock; ++w) r = (f < 4) ? min(r, s[w][f]) : max(r, s[w][f]);
    partial[blockIdx.x * 8 + f] = r;
  }
}


// Key layout on the device, from the bounds partials: one workgroup reduces them,
// biases each field by its minimum minus the kernel reach and the Eq. 1 cell (b is
// never offset), gives it the bit width of its extent, packs the fields b, x, y, z
// from the most significant end, and writes the layout and the packed key delta
// of every offset into the control block.  Flags: kErrRange if the key needs more
// than 62 bits, kErrWide if it needs more than the 8 * passes bits the host
// planned its sort for.  Nothing waits for the host, so the map build needs no
// read-back before the sort.
__device__ __forceinline__ int bit_length_u64(uint64_t v) { return v ? 64 - __clzll((long long)v) : 0; }

// One workgroup of kThreads threads computes the layout into *sL (LDS) from the
// partials; with publish it also stores the layout, the offset deltas and the
// flags in the control block.  Every thread of the workgroup must call it.
__device__ void layout_from_partials(const LayoutArgs& la, bool publish, KeyLayout* sL) {
  __shared__ int32_t red[kThreads];
  __shared__ int32_t mm[8];
  const int tid = threadIdx.x;
  // thread tid reduces field f = tid % 8 over partials tid / 8, tid / 8 + 32, ...
  // (all of its loads in flight together), then 32 values per field in LDS
  {
    const int f = tid & 7;
    const bool is_min = f < 4;
    int32_t r = is_min ? INT_MAX : INT_MIN;
    int32_t v[kMaxPartials / 32];
#pragma unroll
    for (int u = 0; u < kMaxPartials / 32; ++u) {
      const int i = tid / 8 + 32 * u;
      v[u] = (i < la.np) ? la.partial[i * 8 + f] : r;
    }
#pragma unroll
    for (int u = 0; u < kMaxPartials / 32; ++u) r = is_min ? min(r, v[u]) : max(r, v[u]);
    red[tid] = r;
  }
  __syncthreads();
  if (tid < 8) {
    int32_t r = red[tid];
    for (int i = 1; i < 32; ++i) r = (tid < 4) ? min(r, red[i * 8 + tid]) : max(r, red[i * 8 + tid]);
    mm[tid] = r;
  }
  __syncthreads();
  if (tid == 0) {
    const int64_t pad = (int64_t)la.t * (la.K - 1) + (int64_t)la.t * la.stride;
    KeyLayout L;
    int w[4];
    for (int f = 0; f < 4; ++f) {
      const int64_t p = (f == 0) ? 0 : pad;
      L.lo[f] = (int64_t)mm[f] - p;
      w[f] = bit_length_u64((uint64_t)((int64_t)mm[4 + f] + p - L.lo[f]));
      L.width[f] = w[f];
    }
    L.total_bits = w[0] + w[1] + w[2] + w[3];
    // shifts stay below 64 even when the extent does not fit (the build then fails)
    L.shift[3] = 0;
    L.shift[2] = min(w[3], 63);
    L.shift[1] = min(w[3] + w[2], 63);
    L.shift[0] = min(w[3] + w[2] + w[1], 63);
    *sL = L;
    if (publish) {
      uint32_t err = 0;
      if (L.total_bits > 62) err |= kErrRange;
      if (L.total_bits > 8 * la.passes) err |= kErrWide;
      la.cb->layout = L;
      if (err) atomicOr(&la.cb->err, err);
    }
  }
  __syncthreads();
  if (publish) {
    // Delta(K, t): offset k = ix K^2 + iy K + iz is t (ix - c, iy - c, iz - c)
    const int K = la.K;
    const int c = (K % 2 == 1) ? (K - 1) / 2 : 0;
    for (int k = tid; k < la.K3; k += kThreads) {
      const int ix = k / (K * K), iy = (k / K) % K, iz = k % K;
      const int64_t dx = (int64_t)la.t * (ix - c), dy = (int64_t)la.t * (iy - c), dz = (int64_t)la.t * (iz - c);
      la.cb->dk[k] = (int64_t)((uint64_t)dx << sL->shift[1]) + (int64_t)((uint64_t)dy << sL->shift[2]) +
                     (int64_t)((uint64_t)dz << sL->shift[3]);
    }
  }
}

__global__ __launch_bounds__(kThreads) void k_layout(LayoutArgs la) {
  __shared__ KeyLayout sL;
  layout_from_partials(la, true, &sL);
}

// ----------------------------------------------------------------------------
// Key packing helpers
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_pack(const int4* c, int64_t n, const KeyLayout* __restrict__ Lp, uint64_t* keys,
                                                   uint32_t* vals) {
  const KeyLayout L = *Lp;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int4 v = c[i];
  const int32_t a[4] = {v.x, v.y, v.z, v.w};
  keys[i] = pack_key(L, a);
  vals[i] = (uint32_t)i;
}

// ----------------------------------------------------------------------------
// LSD radix sort of (u64 key, u32 value), 8-bit digits, stable.  Large inputs
// run one kernel per pass: an up-front kernel counts the digits of every pass
// in one read (per-block partials, reduced by a second small kernel, no global
// atomics); each pass kernel then takes a tile ticket, ranks its keys within
// each wave (per-wave LDS masks of the lanes holding each digit), publishes its
// per-digit counts, and
// adds up the counts of all earlier tiles by looking back over their published
// words.  Tiles are numbered in start order, so every tile a workgroup waits
// for is already running; waits are bounded and report an error flag instead
// of hanging.  The first pass may read int32 coordinates and pack the keys
// itself.  Every scatter goes through LDS: the tile is first ordered by digit
// there, so that consecutive threads write consecutive addresses of a digit's
// run.
// ----------------------------------------------------------------------------
constexpr int kRsItems = 8;                   // keys per thread of the tiled sort's larger tiles
// keys per thread of a one-kernel pass: long runs per digit and tile for the stores
// (16M keys: pass 193 -> 166 us against 8 keys per thread)
constexpr int kRsItemsLarge = 16;
constexpr int kRsTile = kThreads * kRsItems;
constexpr int kRsTileLarge = kThreads * kRsItemsLarge;
constexpr int kRsItemsSmall = 4;              // keys per thread of the small sorts' passes
constexpr int kRsTileSmall = kThreads * kRsItemsSmall;
constexpr int kRsUpBlocks = 512;
constexpr int kRsMaxPasses = 8;
constexpr uint32_t kStAgg = 1u << 30;   // word holds this tile's count of the digit
constexpr uint32_t kStIncl = 2u << 30;  // word holds the count over tiles 0..this one
constexpr uint32_t kStVal = (1u << 30) - 1u;
constexpr uint32_t kSpinLimit = 1u << 20;
constexpr int kLookWindow = 16;

// Device-coherent (agent-scope) loads and stores of look-back words.  A word carries
// its own payload (flag + count) and no other data is published with it, so relaxed
// ordering suffices, which keeps a window of loads in flight together.
__device__ __forceinline__ uint32_t ld_coherent(uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Lanes of the wave whose digit equals this lane's digit, among the active lanes
// that pass `valid`.
template <bool FROM_COORDS>
__device__ __forceinline__ uint64_t load_key(const uint64_t* keys, const int4* coords, const KeyLayout& L, int64_t i) {
  if constexpr (FROM_COORDS) {
    const int4 v = coords[i];
    const int32_t a[4] = {v.x, v.y, v.z, v.w};
    return pack_key(L, a);
  } else {
    return keys[i];
  }
}

// Exclusive scan of one value per thread over the 256-thread block (4 waves).
__device__ __forceinline__ uint32_t block_excl256(uint32_t v, uint32_t* s_wave) {
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
  uint32_t e = x - v;
  for (int w = 0; w < wave; ++w) e += s_wave[w];
  __syncthreads();  // s_wave may be reused
  return e;
}

// LDS of one tile scatter of ITEMS keys per thread.
template <int ITEMS>
struct TileLds {
  uint64_t key[kThreads * ITEMS];
  uint32_t val[kThreads * ITEMS];
  uint32_t ldig[256];   // tile-local first position of each digit
  uint32_t gbase[256];  // global position of the tile's first key of each digit
  uint32_t cnt[256];    // the tile's count of each digit
  uint32_t wc[kWavesPerBlock][256];  // per-wave digit counts, then each wave's first position
  uint64_t pm[kWavesPerBlock][256];  // per-wave lanes holding each digit (zero between uses)
  uint32_t s_wave[kWavesPerBlock];
};

// Tile layout: wave w holds keys base + w * 64 ITEMS + r * 64 + lane, r < ITEMS, so
// each wave owns a contiguous run of the tile and can rank it on its own.
template <int ITEMS>
__device__ __forceinline__ int64_t tile_index(int64_t base, int r) {
  return base + (int64_t)(threadIdx.x / kWave) * (kWave * ITEMS) + (int64_t)r * kWave + (threadIdx.x & (kWave - 1));
}

template <bool FROM_COORDS, int ITEMS>
__device__ __forceinline__ void tile_load(const uint64_t* kin, const uint32_t* vin, const int4* coords,
                                          const KeyLayout& L, int64_t base, int64_t n, uint64_t key[ITEMS],
                                          uint32_t val[ITEMS]) {
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const int64_t i = tile_index<ITEMS>(base, r);
    key[r] = 0;
    val[r] = 0;
    if (i < n) {
      key[r] = load_key<FROM_COORDS>(kin, coords, L, i);
      val[r] = FROM_COORDS ? (uint32_t)i : vin[i];
    }
  }
}

// The same tile in two steps, so that the loads need not wait for the key
// layout (device memory written by an earlier kernel): tile_fetch requests the
// keys, or the coordinates, and the values (lanes past n re-read the last
// element; later steps mask them out); tile_pack packs fetched coordinates.
template <bool FROM_COORDS, int ITEMS>
__device__ __forceinline__ void tile_fetch(const uint64_t* kin, const uint32_t* vin, const int4* coords, int64_t base,
                                           int64_t n, uint64_t key[ITEMS], int4 crd[ITEMS], uint32_t val[ITEMS]) {
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const int64_t i = tile_index<ITEMS>(base, r);
    const int64_t ic = min(i, n - 1);
    if constexpr (FROM_COORDS) {
      crd[r] = coords[ic];
      val[r] = (uint32_t)i;
    } else {
      key[r] = kin[ic];
      val[r] = vin[ic];
    }
  }
}

template <bool FROM_COORDS, int ITEMS>
__device__ __forceinline__ void tile_pack(const KeyLayout& L, const int4 crd[ITEMS], uint64_t key[ITEMS]) {
  if constexpr (FROM_COORDS) {
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
      const int32_t a[4] = {crd[r].x, crd[r].y, crd[r].z, crd[r].w};
      key[r] = pack_key(L, a);
    }
  }
}

// Stable ranks within the wave's run: rank[r] = number of earlier keys of the
// wave with the same digit.  Leaves the wave's digit counts in t.wc[wave] (which
// must be zero).  Each lane ORs its bit into the wave's mask word of its digit
// and reads the word back: the lanes holding the same digit.  The lowest of them
// bumps the counter and clears the word (t.pm must be zero and is left so).  No
// workgroup barrier: a wave's LDS accesses complete in order, so every lane reads
// a word before its digit's leader rewrites it.
template <int ITEMS>
__device__ __forceinline__ void tile_rank(TileLds<ITEMS>& t, const uint64_t key[ITEMS], int64_t base, int64_t n,
                                          int shift, uint32_t rank[ITEMS]) {
  const int wave = threadIdx.x / kWave;
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const bool valid = tile_index<ITEMS>(base, r) < n;
    const uint32_t d = (uint32_t)(key[r] >> shift) & 255u;
    rank[r] = 0;
    if (valid) {
      __hip_atomic_fetch_or(&t.pm[wave][d], 1ull << (threadIdx.x & (kWave - 1)), __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_WORKGROUP);
      const uint64_t peers = __hip_atomic_load(&t.pm[wave][d], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      const uint32_t before = (uint32_t)popc64(peers & lanemask_lt());
      rank[r] = t.wc[wave][d] + before;
      if (before == 0) {
        t.wc[wave][d] += (uint32_t)popc64(peers);
        t.pm[wave][d] = 0ull;
      }
    }
  }
}

// Places a ranked tile.  Needs t.wc (per-wave counts) and t.gbase, a barrier
// since, and for STAGED t.cnt.  STAGED: each key goes to its digit-ordered tile
// position in LDS, then the tile is written out so that consecutive threads
// store consecutive positions of a digit's run (pays off once the sort is
// bandwidth-bound).  Otherwise each key is stored at its global position
// straight away (fewer steps, for small latency-bound sorts).
template <bool STAGED, int ITEMS>
__device__ __forceinline__ void tile_place(TileLds<ITEMS>& t, const uint64_t key[ITEMS], const uint32_t val[ITEMS],
                                           const uint32_t rank[ITEMS], int64_t base, int64_t n, int shift,
                                           uint64_t* kout, uint32_t* vout) {
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  uint32_t start;  // first position of digit tid in this tile: tile-local (STAGED) or global
  if (STAGED) {
    start = block_excl256(t.cnt[tid], t.s_wave);
    t.ldig[tid] = start;
  } else {
    start = t.gbase[tid];
  }
  // each wave's first position of digit tid
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) {
    const uint32_t c = t.wc[w][tid];
    t.wc[w][tid] = start;
    start += c;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    if (tile_index<ITEMS>(base, r) < n) {
      const uint32_t d = (uint32_t)(key[r] >> shift) & 255u;
      const uint32_t pos = t.wc[wave][d] + rank[r];
      if (STAGED) {
        t.key[pos] = key[r];
        t.val[pos] = val[r];
      } else {
        kout[pos] = key[r];
        vout[pos] = val[r];
      }
    }
  }
  if (!STAGED) return;
  __syncthreads();
  const int tile_n = (int)min((int64_t)(kThreads * ITEMS), n - base);
  for (int i = tid; i < tile_n; i += kThreads) {
    const uint64_t k = t.key[i];
    const uint32_t d = (uint32_t)(k >> shift) & 255u;
    const uint32_t g = t.gbase[d] + (uint32_t)i - t.ldig[d];
    kout[g] = k;
    vout[g] = t.val[i];
  }
}

template <bool FROM_COORDS>
__global__ __launch_bounds__(kThreads) void k_radix_upsweep(const uint64_t* keys, const int4* coords, const KeyLayout* __restrict__ Lp,
                                                            int64_t n, int passes, uint32_t* gpart, uint32_t* status,
                                                            int64_t status_words, uint32_t* tickets) {
  const KeyLayout L = *Lp;
  __shared__ uint32_t h[kRsMaxPasses][256];
  for (int p = 0; p < passes; ++p) h[p][threadIdx.x] = 0;
  __syncthreads();
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
    const uint64_t key = load_key<FROM_COORDS>(keys, coords, L, i);
    for (int p = 0; p < passes; ++p) {
      const uint32_t d = (uint32_t)(key >> (8 * p)) & 255u;
      atomicAdd(&h[p][d], 1u);
    }
  }
  __syncthreads();
  for (int p = 0; p < passes; ++p) gpart[((int64_t)blockIdx.x * passes + p) * 256 + threadIdx.x] = h[p][threadIdx.x];
  // clear the pass kernels' look-back words and tickets
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < status_words; i += (int64_t)gridDim.x * kThreads)
    status[i] = 0u;
  if (blockIdx.x == 0 && (int)threadIdx.x < passes) tickets[threadIdx.x] = 0u;
}

// One workgroup per pass: sums the up-front partials of its pass over the
// gblocks blocks (4 partial sums per digit) and writes the exclusive scan over
// digits, i.e. the first sorted position of each digit: gofs[pass][d].
__global__ __launch_bounds__(1024) void k_radix_totals(const uint32_t* gpart, int gblocks, int passes,
                                                        uint32_t* gofs) {
  __shared__ uint32_t part[4][256];
  __shared__ uint32_t s_wave[16];
  const int p = blockIdx.x;
  const int d = threadIdx.x & 255, q = threadIdx.x >> 8;
  uint32_t s = 0;
#pragma unroll 8
  for (int g = q; g < gblocks; g += 4) s += gpart[((int64_t)g * passes + p) * 256 + d];
  part[q][d] = s;
  __syncthreads();
  // every thread takes part in the scan (threads past the first 256 carry zeros),
  // so every barrier is reached by the whole workgroup
  const uint32_t tot = (q == 0) ? part[0][d] + part[1][d] + part[2][d] + part[3][d] : 0u;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t x = tot;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) s_wave[wave] = x;
  __syncthreads();
  if (q == 0) {
    uint32_t e = x - tot;
    for (int w = 0; w < wave; ++w) e += s_wave[w];
    gofs[p * 256 + d] = e;
  }
}

template <bool FROM_COORDS, int ITEMS>
__global__ __launch_bounds__(kThreads) void k_radix_pass(const uint64_t* kin, const uint32_t* vin, const int4* coords,
                                                         const KeyLayout* __restrict__ Lp, uint64_t* kout, uint32_t* vout, int64_t n,
                                                         int pass, const uint32_t* gofs, uint32_t* status,
                                                         uint32_t* tickets, uint32_t* err) {
  const KeyLayout L = *Lp;
  __shared__ TileLds<ITEMS> t;
  __shared__ uint32_t s_tile;
  const int tid = threadIdx.x;
  const int shift = 8 * pass;
  if (tid == 0) s_tile = atomicAdd(&tickets[pass], 1u);
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) {
    t.wc[w][tid] = 0;
    t.pm[w][tid] = 0ull;
  }
  __syncthreads();
  const int64_t tile = s_tile;
  const int64_t base = tile * (kThreads * ITEMS);

  uint64_t key[ITEMS];
  uint32_t val[ITEMS];
  uint32_t rank[ITEMS];
  tile_load<FROM_COORDS, ITEMS>(kin, vin, coords, L, base, n, key, val);
  tile_rank<ITEMS>(t, key, base, n, shift, rank);
  __syncthreads();

  // publish this tile's count of digit `tid` and look back over earlier tiles
  uint32_t c = 0;
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) c += t.wc[w][tid];
  t.cnt[tid] = c;
  uint32_t* st = status + (int64_t)pass * gridDim.x * 256;
  uint32_t excl = 0;
  if (tile == 0) {
    st_coherent(&st[tid], kStIncl | c);
  } else {
    st_coherent(&st[tile * 256 + tid], kStAgg | c);
    // Windows of kLookWindow predecessor words are fetched together (independent
    // loads in flight, each a device-coherent round trip), then consumed in order
    // until an inclusive word ends the walk.
    int64_t j = tile - 1;
    uint32_t spins = 0;
    bool done = false;
    while (!done && j >= 0) {
      uint32_t v[kLookWindow];
#pragma unroll
      for (int q = 0; q < kLookWindow; ++q) v[q] = (j - q >= 0) ? ld_coherent(&st[(j - q) * 256 + tid]) : kStIncl;
      int q = 0;
      for (; q < kLookWindow; ++q) {
        const uint32_t f = v[q] & ~kStVal;
        if (f == 0) break;  // not published yet: fetch again from here
        excl += v[q] & kStVal;
        if (f == kStIncl) {
          done = true;
          break;
        }
      }
      if (done) break;
      j -= q;
      if (q < kLookWindow) {
        if (++spins > kSpinLimit) {
          atomicOr(err, kErrSpin);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    st_coherent(&st[tile * 256 + tid], kStIncl | (excl + c));
  }
  t.gbase[tid] = gofs[pass * 256 + tid] + excl;
  __syncthreads();
  tile_place<true, ITEMS>(t, key, val, rank, base, n, shift, kout, vout);
}

// Small inputs (few tiles): per-tile digit histograms, then a stable scatter.
// With few tiles every workgroup of a one-kernel pass would start at once and
// find no inclusive prefix to stop its look-back, so this variant is faster
// there.  With up to kFusedScanTiles tiles the histograms are stored
// tile-major and every scatter workgroup adds up the counts it needs itself
// (two launches per pass); with more, a device scan over the digit-major
// histograms gives the offsets (three launches).  Up to kSmallTiles tiles of
// 1024 keys the tiles take 1024 keys, else 2048.  (512 summed tiles of 2048 keys
// against the scan: LiDAR sorts 0.131 -> 0.097 ms at 0.60M keys, 0.139 -> 0.109
// ms at 0.84M; 1024 of them lost from 1.5M keys on.)
constexpr int64_t kFusedScanTiles = 512;
constexpr int64_t kSmallTiles = 256;

// Bit position of the key's top 8-bit digit (0 for keys of at most 8 bits).
__device__ __forceinline__ int top_digit_shift(const KeyLayout& L) { return max(L.total_bits - 8, 0); }

// la.partial non-null (coordinates only): the key layout is not computed yet;
// every workgroup computes it from the bounds partials and workgroup 0 publishes
// it (saving the layout kernel's launch).
template <bool FROM_COORDS, bool TILE_MAJOR, int ITEMS>
__global__ __launch_bounds__(kThreads) void k_radix_tile_hist(const uint64_t* keys, const int4* coords, const KeyLayout* __restrict__ Lp,
                                                         int64_t n, int shift, uint32_t* hist, int64_t ntiles,
                                                         LayoutArgs la) {
  __shared__ uint32_t h[256];
  __shared__ KeyLayout sL;
  const int64_t base = (int64_t)blockIdx.x * (kThreads * ITEMS);
  // all of the thread's keys (or coordinates) are requested first, before the key
  // layout is read (lanes past n re-read the last key and are masked out of the
  // counts)
  uint64_t key[ITEMS];
  int4 crd[FROM_COORDS ? ITEMS : 1];
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const int64_t i = min(base + r * kThreads + threadIdx.x, n - 1);
    if constexpr (FROM_COORDS)
      crd[r] = coords[i];
    else
      key[r] = keys[i];
  }
  h[threadIdx.x] = 0;
  KeyLayout L;
  if (FROM_COORDS && la.partial) {  // kernel-argument uniform
    layout_from_partials(la, blockIdx.x == 0, &sL);
    L = sL;
  } else {
    L = *Lp;
  }
  // a digit above the key's bits is zero for every key: the scatter copies the
  // tile and needs no histogram (the tile is counted as empty rather than left by
  // an early return, which would let the compiler move the key loads after the
  // layout read)
  const bool active = FROM_COORDS || shift < L.total_bits;
  // shift < 0: the key's top digit (the bucket pass of the small sorts)
  const int sh = (shift >= 0) ? shift : top_digit_shift(L);
  __syncthreads();
  if constexpr (FROM_COORDS) {
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
      const int32_t a[4] = {crd[r].x, crd[r].y, crd[r].z, crd[r].w};
      key[r] = pack_key(L, a);
    }
  }
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const bool valid = active && base + r * kThreads + threadIdx.x < n;
    const uint32_t d = (uint32_t)(key[r] >> sh) & 255u;
    if (valid) atomicAdd(&h[d], 1u);
  }
  __syncthreads();
  if (TILE_MAJOR)  // 16-bit counts (a tile holds at most kThreads * ITEMS <= 2048 keys)
    reinterpret_cast<uint16_t*>(hist)[(int64_t)blockIdx.x * 256 + threadIdx.x] = (uint16_t)h[threadIdx.x];
  else
    hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

// FUSED: `offs` holds tile-major histograms of 16-bit counts; the first position
// of digit d in this tile is (keys of smaller digits) + (keys of digit d in
// earlier tiles).  Every workgroup reads all of them, so their size, not their
// latency, sets this step's time (measured: 4 of the pass's 8.6 us at 118 tiles
// of 32-bit counts).  Otherwise `offs` is the scanned digit-major histogram.
// shift < 0 sorts by the key's top digit; then (FUSED) workgroup 0 also stores
// the first position of every digit in bucket_start[0..256] (bucket_start[256] = n).
template <bool FROM_COORDS, bool FUSED, int ITEMS>
__global__ __launch_bounds__(kThreads) void k_radix_tile_scatter(const uint64_t* kin, const uint32_t* vin,
                                                            const int4* coords, const KeyLayout* __restrict__ Lp, uint64_t* kout,
                                                            uint32_t* vout, int64_t n, int shift,
                                                            const uint32_t* offs, int64_t ntiles,
                                                            uint32_t* bucket_start) {
  __shared__ TileLds<ITEMS> t;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int64_t base = (int64_t)blockIdx.x * (kThreads * ITEMS);
  // The tile's keys and the offset sums' loads go out first; the key layout
  // (needed to pack coordinates, and to tell an identity pass) is read while they
  // are in flight.
  uint64_t key[ITEMS];
  uint32_t val[ITEMS];
  uint32_t rank[ITEMS];
  int4 crd[FROM_COORDS ? ITEMS : 1];
  tile_fetch<FROM_COORDS, ITEMS>(kin, vin, coords, base, n, key, crd, val);
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) {
    t.wc[w][tid] = 0;
    t.pm[w][tid] = 0ull;
  }
  if (FUSED) {
    // A 16-byte load holds 8 counts, so a wave's load covers two tiles: lane l
    // reads digits 8 (l % 32) .. + 7 of tile 2 p + l / 32 for tile pairs
    // p = wave, wave + 4, ...; all of a wave's loads are independent and in flight
    // together.
    const int lane = tid & (kWave - 1);
    const int64_t tile = blockIdx.x;
    const int half = lane >> 5;
    const uint4* h4 = reinterpret_cast<const uint4*>(offs);
    uint32_t tot8[8], bef8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) tot8[e] = bef8[e] = 0;
    const int64_t npairs = (ntiles + 1) / 2;
    for (int64_t p0 = wave; p0 < npairs; p0 += 16 * kWavesPerBlock) {
      uint4 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int64_t tt = 2 * (p0 + (int64_t)u * kWavesPerBlock) + half;
        v[u] = (tt < ntiles) ? h4[tt * 32 + (lane & 31)] : make_uint4(0, 0, 0, 0);
      }
      // the batch is summed on the packed pairs: a 16-bit half gathers at most 16
      // tiles of at most 2048 keys, so no carry crosses into its neighbour
      uint32_t tp[4] = {0, 0, 0, 0}, bp[4] = {0, 0, 0, 0};
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int64_t tt = 2 * (p0 + (int64_t)u * kWavesPerBlock) + half;
        const bool early = tt < tile;
        tp[0] += v[u].x; tp[1] += v[u].y; tp[2] += v[u].z; tp[3] += v[u].w;
        bp[0] += early ? v[u].x : 0u; bp[1] += early ? v[u].y : 0u;
        bp[2] += early ? v[u].z : 0u; bp[3] += early ? v[u].w : 0u;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        tot8[e] += (tp[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
        bef8[e] += (bp[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
      }
    }
    // per-(wave, half) partial sums -> per-digit sums (thread d); the key stage
    // serves as scratch (this kernel writes keys straight to their global
    // positions): 8 rows of 256 counts
    uint32_t* s_part = reinterpret_cast<uint32_t*>(t.key);
    static_assert(sizeof(t.key) >= 2 * kWavesPerBlock * 256 * sizeof(uint32_t), "scratch rows fit the key stage");
    uint32_t* row = s_part + (2 * wave + half) * 256 + 8 * (lane & 31);
#pragma unroll
    for (int e = 0; e < 8; ++e) row[e] = tot8[e];
    __syncthreads();
    uint32_t tot = 0;
#pragma unroll
    for (int w = 0; w < 2 * kWavesPerBlock; ++w) tot += s_part[w * 256 + tid];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 8; ++e) row[e] = bef8[e];
    __syncthreads();
    uint32_t before = 0;
#pragma unroll
    for (int w = 0; w < 2 * kWavesPerBlock; ++w) before += s_part[w * 256 + tid];
    t.gbase[tid] = block_excl256(tot, t.s_wave) + before;
    if (bucket_start && blockIdx.x == 0) {  // workgroup 0: before = 0
      bucket_start[tid] = t.gbase[tid];
      if (tid == 0) bucket_start[256] = (uint32_t)n;
    }
  } else {
    t.gbase[tid] = offs[(int64_t)tid * ntiles + blockIdx.x];
  }
  const KeyLayout L = *Lp;
  if (!FROM_COORDS && shift >= L.total_bits) {
    // identity pass (the planned pass count exceeds the key's bits): stable copy
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
      const int64_t i = tile_index<ITEMS>(base, r);
      if (i < n) {
        kout[i] = key[r];
        vout[i] = val[r];
      }
    }
    return;
  }
  tile_pack<FROM_COORDS, ITEMS>(L, crd, key);
  const int sh = (shift >= 0) ? shift : top_digit_shift(L);
  __syncthreads();  // wc cleared
  tile_rank<ITEMS>(t, key, base, n, sh, rank);
  __syncthreads();
  tile_place<false, ITEMS>(t, key, val, rank, base, n, sh, kout, vout);
}

// ----------------------------------------------------------------------------
// Small sorts by bucket: one stable pass on the key's top digit puts every key
// in its bucket (k_radix_tile_hist / k_radix_tile_scatter with shift < 0), then
// one workgroup per bucket sorts the bucket by the remaining low bits in LDS,
// 8-bit digit by digit: three launches instead of two per digit.  A bucket
// larger than kBucketCap keys raises kErrBucket and is left unsorted (the map
// build is then redone with the digit-by-digit sort).
// ----------------------------------------------------------------------------
constexpr int kBucketThreads = 1024;
constexpr int kBucketWaves = kBucketThreads / kWave;
constexpr int kBucketItems = 8;
constexpr int kBucketCap = kBucketThreads * kBucketItems;
// keys, per-wave peer masks (u64 per digit), values, per-wave digit counters, wave totals
constexpr size_t kBucketLds = (size_t)kBucketCap * (sizeof(uint64_t) + sizeof(uint32_t)) +
                              (size_t)kBucketWaves * 256 * (sizeof(uint64_t) + sizeof(uint32_t)) + 64 * sizeof(uint32_t);

// Inclusive prefix sum over the 64 lanes: shifts within each 16-lane row (DPP
// row_shr; a lane with no source lane adds 0), then the totals of the rows below.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x, int lane) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = lane >> 4;
  return x + (row > 0 ? r0 : 0u) + (row > 1 ? r1 : 0u) + (row > 2 ? r2 : 0u);
}

// Bucket b = [bucket_start[b], bucket_start[b + 1]) of (kin, vin), sorted into the
// same positions of (kout, vout) (which may be kin, vin: each workgroup reads its
// whole bucket before it writes).  A bucket of m keys takes ipt = ceil(m / 1024)
// items per lane, spread over all waves: slot s is item r of lane l of wave w for
// s = w 64 ipt + r 64 + l, so each wave ranks a contiguous run of slots (stable)
// in ipt rounds; LDS holds the permuted bucket between digits.
//
// Ranking an item: the lane ORs its bit into its wave's mask word for its digit
// and reads the word back, which gives the lanes of the wave holding the same
// digit (two LDS operations in place of a match by eight wave ballots); the lowest such lane
// adds their count to the wave's digit counter and clears the word again.  The
// counters are then turned into first positions by one scan over (digit, wave)
// in digit-major order: each thread sums four waves of one digit, the waves scan
// those sums, and the sixteen wave totals are added in.
__global__ __launch_bounds__(kBucketThreads) void k_bucket_sort(const uint64_t* kin, const uint32_t* vin,
                                                                uint64_t* kout, uint32_t* vout,
                                                                const uint32_t* __restrict__ bucket_start,
                                                                const KeyLayout* __restrict__ Lp, uint32_t* err) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* skey = reinterpret_cast<uint64_t*>(smem);
  uint64_t(*pm)[256] = reinterpret_cast<uint64_t(*)[256]>(skey + kBucketCap);
  uint32_t* sval = reinterpret_cast<uint32_t*>(&pm[kBucketWaves][0]);
  uint32_t(*wc)[256] = reinterpret_cast<uint32_t(*)[256]>(sval + kBucketCap);
  uint32_t* s_part = &wc[kBucketWaves][0];  // wave totals of the scan
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int bits = max(Lp->total_bits - 8, 0);  // the bucket pass sorted the bits above
  const uint32_t b0 = bucket_start[blockIdx.x];
  const uint32_t b1 = bucket_start[blockIdx.x + 1];
  const int m = (b1 > b0) ? (int)min(b1 - b0, (uint32_t)(kBucketCap + 1)) : 0;
  if (m > kBucketCap) {  // workgroup-uniform
    if (tid == 0) atomicOr(err, kErrBucket);
    return;
  }
  if (m <= 1) {
    if (m == 1 && tid == 0 && kout != kin) {  // a lone key still moves to the output
      kout[b0] = kin[b0];
      vout[b0] = vin[b0];
    }
    return;
  }
  // Items per lane: the ranking rounds run serially, so a bucket is spread over
  // all waves (a typical bucket then takes one round).  Only the first nwv waves
  // hold slots; the others skip every step but the barriers and the scan, and
  // item r of a wave is skipped as a whole past ipt or once its slots start past
  // the bucket (both wave-uniform).
  const int ipt = (m + kBucketThreads - 1) / kBucketThreads;
  auto slot = [&](int r) { return wave * (kWave * ipt) + r * kWave + lane; };
  auto item_live = [&](int r) { return r < ipt && wave * (kWave * ipt) + r * kWave < m; };
  uint64_t key[kBucketItems];
  uint32_t val[kBucketItems];
#pragma unroll
  for (int r = 0; r < kBucketItems; ++r) {
    const int64_t i = (int64_t)b0 + min(slot(r), m - 1);
    key[r] = item_live(r) ? kin[i] : 0ull;
    val[r] = item_live(r) ? vin[i] : 0u;
  }
  // counters (all 16 rows: 4 words per thread) and peer masks start at zero;
  // every use of a mask word leaves it zero again
  uint4* wc4 = reinterpret_cast<uint4*>(&wc[0][0]);
  wc4[tid] = make_uint4(0, 0, 0, 0);
  for (int i = tid; i < kBucketWaves * 256; i += kBucketThreads) (&pm[0][0])[i] = 0ull;
  const uint64_t mybit = 1ull << lane;
  const int sd = tid >> 2;        // scan: this thread's digit ...
  const int sw = (tid & 3) * 4;   // ... and its first of four waves
  __syncthreads();
  for (int sh = 0; sh < bits; sh += 8) {
    uint32_t rank[kBucketItems];
#pragma unroll
    for (int r = 0; r < kBucketItems; ++r) {
      rank[r] = 0;
      if (!item_live(r)) continue;
      if (slot(r) < m) {
        const uint32_t d = (uint32_t)(key[r] >> sh) & 255u;
        __hip_atomic_fetch_or(&pm[wave][d], mybit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        const uint64_t peers = __hip_atomic_load(&pm[wave][d], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        const uint32_t before = (uint32_t)popc64(peers & lanemask_lt());
        rank[r] = wc[wave][d] + before;
        if (before == 0) {
          wc[wave][d] += (uint32_t)popc64(peers);
          pm[wave][d] = 0ull;
        }
      }
    }
    __syncthreads();
    const uint32_t c0 = wc[sw][sd], c1 = wc[sw + 1][sd], c2 = wc[sw + 2][sd], c3 = wc[sw + 3][sd];
    const uint32_t tsum = c0 + c1 + c2 + c3;
    const uint32_t incl = wave_incl_scan(tsum, lane);
    if (lane == kWave - 1) s_part[wave] = incl;
    __syncthreads();
    uint32_t start = incl - tsum;
#pragma unroll
    for (int q = 0; q < kBucketWaves / 4; ++q) {
      const uint4 v = reinterpret_cast<const uint4*>(s_part)[q];
      start += (4 * q < wave ? v.x : 0u) + (4 * q + 1 < wave ? v.y : 0u) + (4 * q + 2 < wave ? v.z : 0u) +
               (4 * q + 3 < wave ? v.w : 0u);
    }
    wc[sw][sd] = start;
    wc[sw + 1][sd] = start + c0;
    wc[sw + 2][sd] = start + c0 + c1;
    wc[sw + 3][sd] = start + c0 + c1 + c2;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kBucketItems; ++r) {
      if (r < ipt && slot(r) < m) {
        const uint32_t d = (uint32_t)(key[r] >> sh) & 255u;
        const uint32_t pos = wc[wave][d] + rank[r];
        skey[pos] = key[r];
        sval[pos] = val[r];
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kBucketItems; ++r) {
      if (!item_live(r)) continue;
      const int sl = min(slot(r), m - 1);
      key[r] = skey[sl];
      val[r] = sval[sl];
    }
    wc4[tid] = make_uint4(0, 0, 0, 0);  // the next digit's counters
    __syncthreads();                    // ... and its stage
  }
#pragma unroll
  for (int r = 0; r < kBucketItems; ++r) {
    if (r < ipt && slot(r) < m) {
      kout[(int64_t)b0 + slot(r)] = key[r];
      vout[(int64_t)b0 + slot(r)] = val[r];
    }
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

__global__ __launch_bounds__(kThreads) void k_down_keys(const uint64_t* skeys, int64_t n, const KeyLayout* __restrict__ Lp, int64_t cell,
                                                        uint64_t* dkeys, uint32_t* vals) {
  const KeyLayout L = *Lp;
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

// Unique keys of a sorted array in two launches, for up to kUniqueTiles tiles of
// kUniqueTile keys: per-tile counts of first occurrences, then every tile adds up
// the counts of the tiles before it, ranks its own first occurrences with a
// workgroup scan and writes them.  Thread t of a tile holds its keys
// 8 t .. 8 t + 7.  Larger arrays go through a device scan of per-key flags.
constexpr int kUniqueItems = 8;
constexpr int kUniqueTile = kThreads * kUniqueItems;
constexpr int64_t kUniqueTiles = 1024;

// this thread's first occurrences among its keys (f), their keys (k) and count
__device__ __forceinline__ uint32_t unique_items(const uint64_t* keys, int64_t n, uint64_t (&k)[kUniqueItems],
                                                 bool (&f)[kUniqueItems]) {
  const int64_t i0 = (int64_t)blockIdx.x * kUniqueTile + (int64_t)threadIdx.x * kUniqueItems;
  uint64_t prev = (i0 > 0 && i0 - 1 < n) ? keys[i0 - 1] : 0;
  uint32_t c = 0;
#pragma unroll
  for (int r = 0; r < kUniqueItems; ++r) {
    const int64_t i = i0 + r;
    k[r] = (i < n) ? keys[i] : 0;
    f[r] = i < n && (i == 0 || k[r] != prev);
    prev = k[r];
    c += f[r] ? 1u : 0u;
  }
  return c;
}

// sum of one value per thread over the 256-thread block, in every thread
__device__ __forceinline__ uint32_t block_sum256(uint32_t v, uint32_t* s_wave) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) v += __shfl_xor(v, d, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0) s_wave[threadIdx.x / kWave] = v;
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int w = 0; w < kWavesPerBlock; ++w) t += s_wave[w];
  __syncthreads();  // s_wave may be reused
  return t;
}

__global__ __launch_bounds__(kThreads) void k_unique_tile_count(const uint64_t* keys, int64_t n, uint32_t* cnt) {
  __shared__ uint32_t s_wave[kWavesPerBlock];
  uint64_t k[kUniqueItems];
  bool f[kUniqueItems];
  const uint32_t t = block_sum256(unique_items(keys, n, k, f), s_wave);
  if (threadIdx.x == 0) cnt[blockIdx.x] = t;
}

__global__ __launch_bounds__(kThreads) void k_unique_tile_write(const uint64_t* keys, int64_t n,
                                                                const KeyLayout* __restrict__ Lp, const uint32_t* cnt,
                                                                uint64_t* qkeys, uint32_t* qrow, int4* coords,
                                                                uint32_t* n_unique) {
  __shared__ uint32_t s_wave[kWavesPerBlock];
  const KeyLayout L = *Lp;
  uint64_t k[kUniqueItems];
  bool f[kUniqueItems];
  const uint32_t c = unique_items(keys, n, k, f);
  uint32_t part = 0;
  for (int j = threadIdx.x; j < (int)blockIdx.x; j += kThreads) part += cnt[j];
  const uint32_t base = block_sum256(part, s_wave);
  uint32_t p = base + block_excl256(c, s_wave);
#pragma unroll
  for (int r = 0; r < kUniqueItems; ++r) {
    if (!f[r]) continue;
    qkeys[p] = k[r];
    qrow[p] = p;
    coords[p] = make_int4(key_field(L, k[r], 0), key_field(L, k[r], 1), key_field(L, k[r], 2), key_field(L, k[r], 3));
    ++p;
  }
  // the last thread of the last tile ends at the total
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == kThreads - 1) *n_unique = p;
}

__global__ __launch_bounds__(kThreads) void k_unique_flags(const uint64_t* keys, int64_t n, uint32_t* flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  flags[i] = (i == 0 || keys[i] != keys[i - 1]) ? 1u : 0u;
}

__global__ __launch_bounds__(kThreads) void k_unique_write(const uint64_t* keys, int64_t n, const KeyLayout* __restrict__ Lp,
                                                           const uint32_t* flags, const uint32_t* pos,
                                                           uint64_t* qkeys, uint32_t* qrow, int4* coords) {
  const KeyLayout L = *Lp;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n || flags[i] == 0) return;
  const uint32_t p = pos[i];
  const uint64_t k = keys[i];
  qkeys[p] = k;
  qrow[p] = p;
  coords[p] = make_int4(key_field(L, k, 0), key_field(L, k, 1), key_field(L, k, 2), key_field(L, k, 3));
}

// ----------------------------------------------------------------------------
// 64-way wave search: number of entries of sorted a[0..n) that are <= thr
// (each round every lane tests one probe; ~log64(n) dependent loads).
// ----------------------------------------------------------------------------
template <typename T, typename V>
__device__ __forceinline__ int64_t wave_upper_bound(const T* a, int64_t n, V thr) {
  const int lane = threadIdx.x & (kWave - 1);
  int64_t lo = 0, hi = n;  // answer in [lo, hi]
  while (hi - lo > kWave) {
    const int64_t step = (hi - lo + kWave - 1) / kWave;
    const int64_t pos = lo + (int64_t)(lane + 1) * step - 1;
    const bool pred = pos < hi && (V)a[pos] <= thr;
    const int c = popc64(__ballot(pred));
    const int64_t nlo = lo + (int64_t)c * step;
    const int64_t nhi = min(lo + (int64_t)(c + 1) * step - 1, hi);
    lo = nlo;
    hi = nhi;
  }
  const int64_t pos = lo + lane;
  const bool pred = pos < hi && (V)a[pos] <= thr;
  return lo + popc64(__ballot(pred));
}

// ----------------------------------------------------------------------------
// Backward binary search (Section 5.1.2).  For source block b and offset k the
// query block is the run of sorted queries q with key(q) + dk in (pivot_{b-1},
// pivot_b], pivot_b being the block's last key.  One wave per (k, b) finds
// bounds[k][b] = #{q : key(q) + dk <= pivot_b}; the block's queries are then
// [bounds[k][b - 1], bounds[k][b]), which the forward passes split into chunks
// of at most Cq (the balancing step).  The last block also takes the queries beyond its
// pivot (they all miss), so that every (offset, query) pair is searched once and
// the per-query tables come out complete.  For transposed maps the k = 0 waves
// also check the sorted query keys for repeats (a point cloud is a set); the
// count pass checks the source keys in LDS.
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_backward(SearchArgs a, int64_t nb, uint32_t* bounds, ControlBlock* cb) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wid = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  if (wid >= (int64_t)a.K3 * nb) return;  // wave-uniform
  const int k = (int)(wid / nb);
  const int64_t b = wid - (int64_t)k * nb;
  const int64_t nq = a.n_q_dev ? (int64_t)*a.n_q_dev : a.n_q;
  const int64_t dk = a.dk[k];
  // key(q) + dk <= pivot  <=>  key(q) <= pivot - dk, evaluated in signed 64 bits
  const int64_t last = min((b + 1) * (int64_t)a.B, a.n_src) - 1;
  // hi: the last block also takes every query past its pivot; lo: none before block 0
  // (a bound without a neighbouring pivot uses a threshold that every key, or no
  // key, passes)
  const int64_t thr_hi = (b == nb - 1) ? INT64_MAX : (int64_t)a.skeys[last] - dk;
  const int64_t hi = wave_upper_bound<uint64_t, int64_t>(a.qkeys, nq, thr_hi);
  // keys that are not in order (a build whose sort was planned too short, or rows
  // wrongly declared presorted; both are reported) can invert a block's bounds:
  // the passes then give the block no queries, so none reads past the query keys
  if (lane == 0) bounds[wid] = (uint32_t)hi;
  if (k == 0 && a.check_q) {
    // the query keys of a transposed map (the coarse inputs) must be strictly
    // increasing too; the count pass checks the source keys
    bool dup = false, unsorted = false;
    const int64_t per = (nq + nb - 1) / nb;
    for (int64_t e = b * per + lane; e < min((b + 1) * per, nq); e += kWave)
      if (e > 0) {
        dup |= a.qkeys[e] == a.qkeys[e - 1];
        unsorted |= a.qkeys[e] < a.qkeys[e - 1];
      }
    if (__ballot(dup) != 0 && lane == 0) atomicOr(&cb->err, kErrDup);
    if (__ballot(unsorted) != 0 && lane == 0) atomicOr(&cb->err, kErrUnsorted);
  }
}

// ----------------------------------------------------------------------------
// Forward binary search (Section 5.1.2) over the work items, one per (offset,
// source block) pair, whose query block is run in chunks of at most Cq queries
// (the load balancing): the source block is staged in LDS and each lane
// binary-searches its queries there, recording the match (or -1) in T_q.  Count
// pass: matches per work item.  Write pass: matches ranked with wave ballots; pair e of the item goes
// to index o = item_off + e, so every offset's pairs come out in sorted-query
// order, and o, the pair's GEMM buffer row, is also stored in both metadata
// tables (T_q in place of the source position, T_s at the source position).
// ----------------------------------------------------------------------------
// a value that every lane of the wave holds alike (say, read from LDS), in a
// scalar register, so that loops and branches on it stay scalar
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Sorted position of ROUNDS independent keys at once in the LDS block, by binary
// lifting: the block holds 2^LOG2B + 1 keys, padded past its nB real keys with
// the largest key (never smaller than a query), so no step needs a bounds check.
// Positions are kept as byte offsets and every step's distance is a constant, so
// a step is one LDS read, one 64-bit compare and one select per key, and the
// ROUNDS reads of a step are issued together.  pos = number of keys < key (at
// most 2^LOG2B - 1; then the final probe tells a hit from a key past the block),
// hit = whether the key is present.
template <int ROUNDS, int LOG2B>
__device__ __forceinline__ void lds_search(const uint64_t* lkey, const uint64_t (&key)[ROUNDS], int (&pos)[ROUNDS],
                                           bool (&hit)[ROUNDS]) {
  const char* base = reinterpret_cast<const char*>(lkey);
  uint32_t off[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) off[r] = 0;
#pragma unroll
  for (int step = 1 << (LOG2B - 1); step > 0; step >>= 1) {
    uint64_t v[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) v[r] = *reinterpret_cast<const uint64_t*>(base + off[r] + 8 * (step - 1));
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) off[r] += (v[r] < key[r]) ? 8u * step : 0u;
  }
  uint64_t v[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) v[r] = *reinterpret_cast<const uint64_t*>(base + off[r]);
  // every chain ends here, in every lane: a caller's use of a result under a lane
  // mask must not move that chain into the masked branch, after the others
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) asm volatile("" ::"v"(v[r]), "v"(off[r]));
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    hit[r] = v[r] == key[r];
    pos[r] = (int)(off[r] >> 3);
  }
}

// Forward search, write pass: one workgroup per work item (k, b), the query
// block [bounds[k][b - 1], bounds[k][b]) in chunks of at most Cq queries.  The
// count pass left each query's result in T_q (matching sorted source position,
// or -1); matches are ranked with wave ballots from the item's scanned match
// offset onward, chunk after chunk, so every offset's pairs come out in
// sorted-query order, and pair index o (the pair's GEMM buffer row) replaces the
// source position in T_q and is stored in T_s.  The loads of all rounds of a
// chunk are issued together: results first, then the rows of the matches, and
// the next chunk's results before the chunk's barrier.
template <int ROUNDS, int TH>
__global__ __launch_bounds__(TH) void k_forward_write(SearchArgs a, const uint32_t* bounds, int64_t nb,
                                                            const uint32_t* item_off, int32_t* pin, int32_t* pout,
                                                            ControlBlock* cb) {
  __shared__ uint32_t s_cnt[2][ROUNDS][(TH / kWave)];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int64_t w = blockIdx.x;  // k nb + b
  const int k = (int)(w / nb);
  const int64_t b = w - (int64_t)k * nb;
  const int64_t q_hi = bounds[w];
  // min(): keys out of order can invert the bounds (the block then has no queries)
  const int64_t q_lo = (b == 0) ? 0 : min((int64_t)bounds[w - 1], q_hi);
  const uint64_t base0 = item_off[w];

  if (w == 0 && wave == 0) {
    // per-offset pair starts: offset k's items are k nb .. k nb + nb - 1
    for (int kk = lane; kk <= a.K3; kk += kWave) {
      const uint32_t off = (kk < a.K3) ? item_off[(int64_t)kk * nb] : cb->n_pairs;
      cb->seg_pair_start[kk] = off;
      if (a.pub)
        __hip_atomic_store(&a.pub[offsetof(ControlBlock, seg_pair_start) / 4 + kk], off, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_SYSTEM);
    }
    if (a.pub) {
      // The rest of the head: every flag that the map can raise is final here but
      // kErrOverflow of this pass, which only follows keys out of order (flagged
      // by the count pass).  One wave publishes, so its fence orders all the
      // stores before the flag.
      constexpr int kSeg0 = offsetof(ControlBlock, seg_pair_start) / 4;
      constexpr int kSeg1 = kSeg0 + kMaxOffsets + 3;
      const uint32_t* head = reinterpret_cast<const uint32_t*>(cb);
      for (int i = lane; i < (int)(kControlHeadBytes / 4); i += kWave)
        if (i < kSeg0 || i >= kSeg1) __hip_atomic_store(&a.pub[i], head[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __threadfence_system();
      if (lane == 0)
        __hip_atomic_store(&a.pub[kPubFlagOffset / 4], a.pub_seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }

  int32_t* res = a.res + (int64_t)k * a.res_stride;
  int32_t* ts = a.ts + (int64_t)k * a.ts_stride;
  uint64_t base = base0;
  // a chunk's count pass results; the next chunk's are requested while this one's
  // rows are in flight
  int32_t sp[ROUNDS];
  auto load_res = [&](int64_t q0, int32_t* v) {
    const int64_t q1 = min(q0 + (int64_t)a.Cq, q_hi);
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
      const int64_t qp = q0 + (int64_t)r * TH + tid;
      v[r] = (qp < q1) ? res[qp] : -1;
    }
  };
  if (q_lo < q_hi) load_res(q_lo, sp);
  int par = 0;  // s_cnt buffer of this chunk: two, so one barrier per chunk suffices
  for (int64_t q0 = q_lo; q0 < q_hi; q0 += a.Cq) {  // workgroup-uniform
    int32_t r_in[ROUNDS], r_out[ROUNDS];
    uint64_t bal[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
      // rows of the match (a valid dummy address for lanes without one)
      const int64_t qp = q0 + (int64_t)r * TH + tid;
      const bool hit = sp[r] >= 0;
      const int32_t src = (int32_t)a.sidx[hit ? sp[r] : 0];
      const int32_t qry = (int32_t)a.qrow[hit ? qp : 0];
      r_in[r] = a.swap_roles ? qry : src;
      r_out[r] = a.swap_roles ? src : qry;
      bal[r] = __ballot(hit);
      if (lane == 0) s_cnt[par][r][wave] = (uint32_t)popc64(bal[r]);
    }
    int32_t sp_next[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) sp_next[r] = -1;
    if (q0 + a.Cq < q_hi) load_res(q0 + a.Cq, sp_next);
    __syncthreads();
    uint32_t total = 0;
    uint32_t before[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
#pragma unroll
      for (int v = 0; v < (TH / kWave); ++v) {
        if (v == wave) before[r] = total;
        total += s_cnt[par][r][v];
      }
    }
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
      if ((bal[r] >> lane) & 1ull) {
        const uint64_t o = base + before[r] + (uint64_t)popc64(bal[r] & lanemask_lt());
        const int64_t qp = q0 + (int64_t)r * TH + tid;
        if (o >= (uint64_t)a.pair_cap) {  // only when keys were out of order (reported)
          atomicOr(&cb->err, kErrOverflow);
          continue;
        }
        pin[o] = r_in[r];
        pout[o] = r_out[r];
        res[qp] = (int32_t)o;
        if (a.write_ts) ts[sp[r]] = (int32_t)o;
      }
    }
    base += total;
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) sp[r] = sp_next[r];
    // a wave reuses this chunk's s_cnt buffer two chunks on, past the next chunk's
    // barrier, which every wave reaches only after reading it
    par ^= 1;
  }
}

// Forward search, count pass, with source-block reuse: one workgroup per
// (source block b, group of at most 64 offsets) stages block b in LDS once and
// then searches the query block of (k, b) for every offset k of its group, in
// chunks of at most Cq queries (the balancing step).  Each query's result goes to
// T_q, and each (k, b) work item's match count to item_cnt[k nb + b].
// With few source blocks the groups are small, so that the grid still fills the
// GPU; with many, one workgroup takes several offsets of its block and reads the
// block from HBM once instead of once per offset.  The query blocks of offsets
// that differ only in y or z nearly coincide (their key deltas are below one
// x-slab), so consecutive offsets whose blocks together span little more than
// the largest of them form a run: each chunk of the run's span is read once and
// searched for every offset of the run, each lane keeping only the queries inside
// that offset's own block (read per offset, these keys missed L2 once the cloud
// outgrew it).  Match counts are kept per wave (lane j counts the group's offset
// j), so the chunks need no workgroup barrier.  The block's keys, the group's
// query bounds and, for a lone offset, the keys of its first chunk are all
// requested before the first wait; each chunk's ROUNDS searches run as
// independent chains.
template <int ROUNDS, int LOG2B, int TH>
__global__ __launch_bounds__(TH) void k_forward_count(SearchArgs a, const uint32_t* bounds, int64_t nb,
                                                            uint32_t* item_cnt, int G, ControlBlock* cb) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int32_t s_lo[kWave], s_hi[kWave];   // query block of the group's offset j
  __shared__ uint32_t s_tot[TH / kWave][kWave];  // matches of offset j found by each wave
  uint64_t* lkey = reinterpret_cast<uint64_t*>(smem);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  // (nb < 2^31: 32-bit division, not the 64-bit software sequence)
  const int64_t b = (int)blockIdx.x % (int)nb;
  const int g = (int)blockIdx.x / (int)nb;

  const int64_t s0 = b * (int64_t)a.B;
  const int nB = (int)min((int64_t)a.B, a.n_src - s0);
  const int k_first = g * G;
  const int nk = min(a.K3 - k_first, G);  // 1 .. 64 (the host caps G)
  auto block_of = [&](int j, int64_t* lo, int64_t* hi) {
    const int64_t kb = (int64_t)(k_first + j) * nb + b;
    *hi = bounds[kb];
    // min(): keys out of order can invert the bounds (the block then has no queries)
    *lo = (b == 0) ? 0 : min((int64_t)bounds[kb - 1], *hi);
  };
  uint64_t sv[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) sv[u] = a.skeys[s0 + min(u * TH + tid, nB - 1)];
  const uint64_t key_before = a.skeys[s0 > 0 ? s0 - 1 : 0];
  int64_t my_lo = 0, my_hi = 0;
  if (tid < nk) block_of(tid, &my_lo, &my_hi);
  uint64_t qk[ROUNDS];  // the current chunk's query keys (lanes past its end re-read its first key)
  auto load_keys = [&](int64_t q0, int64_t q1) {
    const uint64_t* qb = a.qkeys + q0;
    const int n = (int)(q1 - q0);
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) qk[r] = qb[r * TH + tid < n ? r * TH + tid : 0];
  };
  int64_t pre_lo = -1;  // first query of the chunk already in qk, if any
  if (nk == 1) {
    int64_t lo, hi;
    block_of(0, &lo, &hi);
    if (lo < hi) {
      load_keys(lo, min(lo + (int64_t)a.Cq, hi));
      pre_lo = lo;
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
    if (u * TH + tid < nB) lkey[u * TH + tid] = sv[u];
  for (int e = 4 * TH + tid; e < nB; e += TH) lkey[e] = a.skeys[s0 + e];  // B > 4 * TH
  for (int e = nB + tid; e <= (1 << LOG2B); e += TH) lkey[e] = ~0ull;   // padding
  if (tid < nk) {  // (query positions fit 31 bits: the bounds are 32-bit)
    s_lo[tid] = (int32_t)my_lo;
    s_hi[tid] = (int32_t)my_hi;
  }
  __syncthreads();
  if (g == 0) {
    // the sorted source keys must be strictly increasing: equal neighbours are
    // repeated coordinates, decreasing ones an unsorted input declared sorted
    bool dup = false, unsorted = false;
    for (int e = tid; e < nB; e += TH) {
      const uint64_t prev = (e > 0) ? lkey[e - 1] : key_before;
      if (e > 0 || s0 > 0) {
        dup |= lkey[e] == prev;
        unsorted |= lkey[e] < prev;
      }
    }
    if (__ballot(dup) != 0 && lane == 0) atomicOr(&cb->err, kErrDup);
    if (__ballot(unsorted) != 0 && lane == 0) atomicOr(&cb->err, kErrUnsorted);
  }

  uint32_t tot = 0;  // lane j: this wave's matches of offset k_first + j
  for (int j = 0; j < nk;) {  // workgroup-uniform
    // the run j .. je - 1: its blocks span [u_lo, u_hi), at most 1/8 (+ 64 queries)
    // more than the largest of them; empty blocks join any run
    int u_lo = uniform(s_lo[j]), u_hi = uniform(s_hi[j]), mx = u_hi - u_lo;
    int je = j + 1;
    for (; je < nk; ++je) {
      const int lo = uniform(s_lo[je]), hi = uniform(s_hi[je]);
      if (lo >= hi) continue;
      if (u_lo >= u_hi) {
        u_lo = lo;
        u_hi = hi;
        mx = hi - lo;
        continue;
      }
      const int nlo = min(u_lo, lo), nhi = max(u_hi, hi), nmx = max(mx, hi - lo);
      if (nhi - nlo > nmx + nmx / 8 + 64) break;
      u_lo = nlo;
      u_hi = nhi;
      mx = nmx;
    }
    for (int64_t q0w = u_lo; q0w < u_hi; q0w += a.Cq) {  // (64-bit: q0 + Cq may pass 2^31)
      const int q0 = (int)q0w, q1 = (int)min(q0w + a.Cq, (int64_t)u_hi);
      if (q0 != pre_lo) load_keys(q0, q1);
      pre_lo = -1;
      for (int jj = j; jj < je; ++jj) {
        const int lo = uniform(s_lo[jj]), hi = uniform(s_hi[jj]);
        if (q1 <= lo || q0 >= hi) continue;  // the chunk misses this offset's block
        // the chunk's part of the block, relative to q0
        const int r_lo = max(lo, q0) - q0, r_hi = min(hi, q1) - q0;
        int32_t* res = a.res + (int64_t)(k_first + jj) * a.res_stride + q0;
        const uint64_t dk = (uint64_t)a.dk[k_first + jj];
        // the shifted keys take the raw keys' registers and give them back after
        // the search (modular arithmetic: exact)
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) qk[r] += dk;
        int pos[ROUNDS];
        bool hit[ROUNDS];
        lds_search<ROUNDS, LOG2B>(lkey, qk, pos, hit);
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) qk[r] -= dk;
        uint32_t nh = 0;
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) {
          const int e = r * TH + tid;
          const bool valid = e >= r_lo && e < r_hi;
          if (valid) {
            const int32_t v = hit[r] ? (int32_t)(s0 + pos[r]) : -1;
            if (a.stream_tq)
              __builtin_nontemporal_store(v, res + e);
            else
              res[e] = v;
          }
          nh += (uint32_t)popc64(__ballot(valid && hit[r]));
        }
        if (lane == jj) tot += nh;
      }
    }
    j = je;
  }
  s_tot[wave][lane] = tot;
  __syncthreads();
  if (tid < nk) {
    uint32_t sum = 0;
#pragma unroll
    for (int v = 0; v < TH / kWave; ++v) sum += s_tot[v][tid];
    item_cnt[(int64_t)(k_first + tid) * nb + b] = sum;
  }
}

template <int ROUNDS, int TH>
hipError_t forward_count_t(unsigned grid, hipStream_t s, const SearchArgs& a, const uint32_t* bounds, int64_t nb,
                           uint32_t* item_cnt, int G, ControlBlock* cb, int log2B) {
  // the block plus its padding: 2^log2B + 1 keys
  const size_t lds = (((size_t)1 << log2B) + 1) * sizeof(uint64_t);
  switch (log2B) {
#define SPC_FC(L2)                                                                                              \
  case L2:                                                                                                      \
    hipLaunchKernelGGL((k_forward_count<ROUNDS, L2, TH>), dim3(grid), dim3(TH), lds, s, a, bounds, nb, item_cnt, \
                       G, cb);                                                                                  \
    break;
    SPC_FC(6) SPC_FC(7) SPC_FC(8) SPC_FC(9) SPC_FC(10) SPC_FC(11) SPC_FC(12)
#undef SPC_FC
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int ROUNDS, int TH>
hipError_t forward_write_t(unsigned grid, hipStream_t s, const SearchArgs& a, const uint32_t* bounds, int64_t nb,
                           const uint32_t* item_off, int32_t* pin, int32_t* pout, ControlBlock* cb) {
  hipLaunchKernelGGL((k_forward_write<ROUNDS, TH>), dim3(grid), dim3(TH), 0, s, a, bounds, nb, item_off, pin, pout, cb);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Hash-table search (the prior-art Map of Section 2.2, Step 1), kept as an
// ablation of the sorted-array search.  Inputs are inserted in caller order into
// an open-addressing table (linear probing, load <= 1/2); every (offset, output)
// pair then probes it once.  Probe and insert walks are bounded by the table
// size, so no wave loops forever.
// ----------------------------------------------------------------------------
__device__ __forceinline__ uint64_t hash_slot(uint64_t key, int log2cap) {
  return (key * 0x9E3779B97F4A7C15ull) >> (64 - log2cap);
}

__global__ __launch_bounds__(kThreads) void k_hash_insert(const int4* c, int64_t n, const KeyLayout* __restrict__ Lp, uint64_t* hkeys,
                                                          uint32_t* hvals, int log2cap, uint64_t* keys, uint32_t* idx,
                                                          uint32_t* err) {
  const KeyLayout L = *Lp;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int4 v = c[i];
  const int32_t a[4] = {v.x, v.y, v.z, v.w};
  const uint64_t key = pack_key(L, a);
  keys[i] = key;
  idx[i] = (uint32_t)i;
  const uint64_t mask = (1ull << log2cap) - 1ull;
  uint64_t slot = hash_slot(key, log2cap);
  for (uint64_t step = 0; step <= mask; ++step) {
    const unsigned long long prev =
        atomicCAS(reinterpret_cast<unsigned long long*>(&hkeys[slot]), (unsigned long long)kHashEmpty,
                  (unsigned long long)key);
    if (prev == kHashEmpty) {
      hvals[slot] = (uint32_t)i;
      return;
    }
    if (prev == key) {  // a point cloud is a set
      atomicOr(err, kErrDup);
      return;
    }
    slot = (slot + 1) & mask;
  }
  atomicOr(err, kErrOverflow);  // table full: cannot happen at load 1/2
}

// The hash-table search's work items: block b of offset k is queries
// [b Cq, (b + 1) Cq), recorded as the upper bounds the write pass reads.
__global__ void k_hash_items(int K3, int64_t n_q, int Cq, int64_t nb, uint32_t* bounds) {
  const int64_t nkb = (int64_t)K3 * nb;
  for (int64_t kb = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; kb < nkb; kb += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = kb % nb;
    bounds[kb] = (uint32_t)min((b + 1) * (int64_t)Cq, n_q);
  }
}

// One workgroup per work item (offset k, block b of Cq queries).
template <int ROUNDS>
__global__ __launch_bounds__(kThreads) void k_hash_count(SearchArgs a, const uint64_t* __restrict__ hkeys,
                                                         const uint32_t* __restrict__ hvals, int log2cap, int64_t nb,
                                                         uint32_t* item_cnt) {
  __shared__ uint32_t s_cnt[ROUNDS][kWavesPerBlock];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int64_t w = blockIdx.x;  // k nb + b
  const int k = (int)(w / nb);
  const int64_t q0 = (w - (int64_t)k * nb) * a.Cq;
  const int64_t q1 = min(q0 + (int64_t)a.Cq, a.n_q);
  const uint64_t dk = (uint64_t)a.dk[k];
  const uint64_t mask = (1ull << log2cap) - 1ull;
  int32_t* res = a.res + (int64_t)k * a.res_stride;
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int64_t qp = q0 + (int64_t)r * kThreads + tid;
    bool hit = false;
    if (qp < q1) {
      const uint64_t key = a.qkeys[qp] + dk;
      uint64_t slot = hash_slot(key, log2cap);
      int32_t found = -1;
      for (uint64_t step = 0; step <= mask; ++step) {
        const uint64_t kk = hkeys[slot];
        if (kk == key) {
          found = (int32_t)hvals[slot];
          break;
        }
        if (kk == kHashEmpty) break;
        slot = (slot + 1) & mask;
      }
      hit = found >= 0;
      res[qp] = found;
    }
    const uint64_t bal = __ballot(hit);
    if (lane == 0) s_cnt[r][wave] = (uint32_t)popc64(bal);
  }
  __syncthreads();
  if (tid == 0) {
    uint32_t total = 0;
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r)
#pragma unroll
      for (int v = 0; v < kWavesPerBlock; ++v) total += s_cnt[r][v];
    item_cnt[w] = total;
  }
}

}  // namespace

// ----------------------------------------------------------------------------
// Launchers
// ----------------------------------------------------------------------------
// ----------------------------------------------------------------------------
// Source-side table from the pair lists (Section 2.2's metadata table of the
// inputs): entry (k, p) = buffer row of sorted source p's pair at offset k.
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_inverse_perm(const uint32_t* __restrict__ perm, int64_t n,
                                                           uint32_t* __restrict__ inv) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) inv[perm[i]] = (uint32_t)i;
}

__global__ __launch_bounds__(kThreads) void k_ts_from_pairs(const int32_t* __restrict__ pin,
                                                            const uint32_t* __restrict__ seg, int K3,
                                                            int64_t n_pairs, const uint32_t* __restrict__ inv,
                                                            int32_t* __restrict__ ts, int64_t stride) {
  __shared__ uint32_t s_seg[kMaxOffsets + 1];
  for (int i = threadIdx.x; i <= K3; i += kThreads) s_seg[i] = seg[i];
  __syncthreads();
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= n_pairs) return;
  // the pair's offset: seg[lo] <= e < seg[hi] throughout (seg[0] = 0, seg[K3] = n_pairs)
  int lo = 0, hi = K3;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)s_seg[mid] <= e) lo = mid; else hi = mid;
  }
  const int32_t row = pin[e];
  const int64_t p = inv ? (int64_t)inv[row] : (int64_t)row;
  ts[(int64_t)lo * stride + p] = (int32_t)e;
}

hipError_t launch_ts_from_pairs(const int32_t* pin, const uint32_t* seg, int K3, int64_t n_pairs,
                                const uint32_t* perm, int64_t n_src, uint32_t* inv, int32_t* ts,
                                int64_t stride, hipStream_t s) {
  if (K3 < 1 || K3 > kMaxOffsets || n_src > stride) return hipErrorInvalidValue;
  if (n_pairs <= 0) return hipSuccess;
  if (perm) {
    hipLaunchKernelGGL(k_inverse_perm, dim3((unsigned)((n_src + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                       perm, n_src, inv);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_ts_from_pairs, dim3((unsigned)((n_pairs + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                     pin, seg, K3, n_pairs, perm ? inv : nullptr, ts, stride);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfScope ps(KN_FILL, s);
  hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(n, kThreads, 4096)), dim3(kThreads), 0, s, p, v, n);
  return hipGetLastError();
}

size_t minmax_temp_bytes() { return (size_t)kMinmaxBlocks * 8 * sizeof(int32_t); }

hipError_t launch_minmax(const int32_t* a, int64_t na, const int32_t* b, int64_t nb, int32_t* partial,
                         ControlBlock* cb, int* n_partial, hipStream_t s) {
  ProfScope ps(KN_MINMAX, s);
  const unsigned g = grid_for(na + nb, kThreads * 8, kMinmaxBlocks);
  *n_partial = (int)g;
  hipLaunchKernelGGL(k_minmax_partial, dim3(g), dim3(kThreads), 0, s, reinterpret_cast<const int4*>(a), na,
                     reinterpret_cast<const int4*>(b), nb, partial, cb);
  return hipGetLastError();
}

hipError_t launch_layout(const LayoutArgs& la, hipStream_t s) {
  ProfScope ps(KN_MINMAX, s);
  hipLaunchKernelGGL(k_layout, dim3(1), dim3(kThreads), 0, s, la);
  return hipGetLastError();
}

hipError_t launch_pack(const int32_t* coords, int64_t n, const KeyLayout* L, uint64_t* keys, uint32_t* vals, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfScope ps(KN_PACK, s);
  hipLaunchKernelGGL(k_pack, dim3(grid_for(n)), dim3(kThreads), 0, s, reinterpret_cast<const int4*>(coords), n, L,
                     keys, vals);
  return hipGetLastError();
}

// One-kernel passes need many more tiles than workgroups that run at once, so
// that most look-backs stop at a finished predecessor: they serve from this many
// tiles of kRsTileLarge keys (4.2M keys) on.  Below, the tiled sort with its
// scanned offsets was faster (LiDAR keys: 0.257 -> 0.231 ms at 2.5M, 0.342 ->
// 0.313 ms at 4.07M, against one-kernel passes of 2048-key tiles); above, the
// one-kernel passes win (0.386 against 0.417 ms at 6M keys).
constexpr int64_t kOnesweepMinTiles = 1024;

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t radix_temp_bytes(int64_t n) {
  const int64_t ntiles = std::max<int64_t>(1, (n + kRsTile - 1) / kRsTile);
  const size_t gpart = (size_t)kRsUpBlocks * kRsMaxPasses * 256 * sizeof(uint32_t);
  const size_t gofs = (size_t)kRsMaxPasses * 256 * sizeof(uint32_t);
  const size_t status = (size_t)kRsMaxPasses * ntiles * 256 * sizeof(uint32_t);
  const size_t onesweep = align256(gpart) + align256(gofs) + align256(status) + 256;
  // the small sorts use tiles of kRsTileSmall keys when that keeps their offsets fused
  const int64_t tiles_small = std::max<int64_t>(1, (n + kRsTileSmall - 1) / kRsTileSmall);
  const int64_t tiles_tiled = std::max(ntiles, tiles_small);
  const size_t tiled = align256((size_t)256 * tiles_tiled * sizeof(uint32_t)) + scan_temp_bytes(256 * tiles_tiled);
  // by-bucket sorts: 16-bit tile histograms, then the 257 bucket starts
  const size_t bucket = align256((size_t)tiles_small * 256 * sizeof(uint16_t)) + 257 * sizeof(uint32_t);
  return std::max(std::max(onesweep, tiled), bucket);
}

namespace {
// Small inputs: tile histograms, then the scatter (with a device scan between
// them once there are too many tiles to sum in each workgroup).  ITEMS keys per
// thread: smaller tiles shorten each workgroup's chain while the launch is
// latency-bound.
template <int ITEMS>
hipError_t radix_sort_tiled_t(const int32_t* coords, const KeyLayout* L, uint64_t* keys, uint32_t* vals, uint64_t* keys_alt,
                              uint32_t* vals_alt, int64_t n, int passes, void* d_temp, const LayoutArgs& lay,
                              hipStream_t s) {
  const int64_t ntiles = (n + kThreads * ITEMS - 1) / (kThreads * ITEMS);
  uint32_t* hist = static_cast<uint32_t*>(d_temp);
  void* scan_tmp = static_cast<char*>(d_temp) + align256((size_t)256 * ntiles * sizeof(uint32_t));
  const int4* c4 = reinterpret_cast<const int4*>(coords);
  uint64_t* kb[2] = {keys, keys_alt};
  uint32_t* vb[2] = {vals, vals_alt};
  int cur = (passes % 2 == 0) ? 0 : 1;
  if (!coords && passes % 2 == 1) {
    ProfScope ps(KN_COPY, s);
    hipError_t e = hipMemcpyAsync(keys_alt, keys, (size_t)n * 8, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(vals_alt, vals, (size_t)n * 4, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  const bool fused = ntiles <= kFusedScanTiles;
  const unsigned g = (unsigned)ntiles;
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    const bool first = (p == 0) && coords;
    const int src = cur, dst = (first ? ((passes % 2 == 1) ? 0 : 1) : cur ^ 1);
    hipError_t e;
    {
      ProfScope ps(KN_RADIX_HIST, s);
#define SPC_H(FC, TM)                                                                                           \
  hipLaunchKernelGGL((k_radix_tile_hist<FC, TM, ITEMS>), dim3(g), dim3(kThreads), 0, s, FC ? nullptr : kb[src],      \
                     FC ? c4 : nullptr, L, n, shift, hist, ntiles, FC ? lay : LayoutArgs{})
      if (first) {
        if (fused) SPC_H(true, true); else SPC_H(true, false);
      } else {
        if (fused) SPC_H(false, true); else SPC_H(false, false);
      }
#undef SPC_H
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    if (!fused) {
      e = scan_exclusive_u32(hist, hist, 256 * ntiles, nullptr, scan_tmp, s);
      if (e != hipSuccess) return e;
    }
    {
      ProfScope ps(KN_RADIX_SCATTER, s);
#define SPC_S(FC, FU)                                                                                           \
  hipLaunchKernelGGL((k_radix_tile_scatter<FC, FU, ITEMS>), dim3(g), dim3(kThreads), 0, s, FC ? nullptr : kb[src],   \
                     FC ? nullptr : vb[src], FC ? c4 : nullptr, L, kb[dst], vb[dst], n, shift, hist, ntiles, nullptr)
      if (first) {
        if (fused) SPC_S(true, true); else SPC_S(true, false);
      } else {
        if (fused) SPC_S(false, true); else SPC_S(false, false);
      }
#undef SPC_S
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    cur = dst;
  }
  return hipSuccess;
}

hipError_t radix_sort_tiled(const int32_t* coords, const KeyLayout* L, uint64_t* keys, uint32_t* vals, uint64_t* keys_alt,
                            uint32_t* vals_alt, int64_t n, int passes, void* d_temp, const LayoutArgs& lay,
                            hipStream_t s) {
  if ((n + kRsTileSmall - 1) / kRsTileSmall <= kSmallTiles)
    return radix_sort_tiled_t<kRsItemsSmall>(coords, L, keys, vals, keys_alt, vals_alt, n, passes, d_temp, lay, s);
  return radix_sort_tiled_t<kRsItems>(coords, L, keys, vals, keys_alt, vals_alt, n, passes, d_temp, lay, s);
}

// By-bucket sort (three launches; see radix_bucket_applies for its sizes): tile histograms
// of the top digit (1024-key tiles, so the scatter sums them itself), the stable
// bucket pass (into (keys, vals) from coordinates, else into the alternates), and
// one workgroup per bucket sorting it into (keys, vals).
hipError_t radix_sort_bucket(const int32_t* coords, const KeyLayout* L, uint64_t* keys, uint32_t* vals,
                             uint64_t* keys_alt, uint32_t* vals_alt, int64_t n, void* d_temp, uint32_t* err,
                             const LayoutArgs& lay, hipStream_t s) {
  constexpr int ITEMS = kRsItemsSmall;
  const int64_t ntiles = (n + kThreads * ITEMS - 1) / (kThreads * ITEMS);
  uint32_t* hist = static_cast<uint32_t*>(d_temp);
  uint32_t* bstart =
      reinterpret_cast<uint32_t*>(static_cast<char*>(d_temp) + align256((size_t)ntiles * 256 * sizeof(uint16_t)));
  const int4* c4 = reinterpret_cast<const int4*>(coords);
  uint64_t* mk = coords ? keys : keys_alt;
  uint32_t* mv = coords ? vals : vals_alt;
  const unsigned g = (unsigned)ntiles;
  {
    ProfScope ps(KN_RADIX_HIST, s);
    if (coords)
      hipLaunchKernelGGL((k_radix_tile_hist<true, true, ITEMS>), dim3(g), dim3(kThreads), 0, s, nullptr, c4, L, n, -1,
                         hist, ntiles, lay);
    else
      hipLaunchKernelGGL((k_radix_tile_hist<false, true, ITEMS>), dim3(g), dim3(kThreads), 0, s, keys, nullptr, L, n,
                         -1, hist, ntiles, LayoutArgs{});
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  {
    ProfScope ps(KN_RADIX_SCATTER, s);
    if (coords)
      hipLaunchKernelGGL((k_radix_tile_scatter<true, true, ITEMS>), dim3(g), dim3(kThreads), 0, s, nullptr, nullptr,
                         c4, L, mk, mv, n, -1, hist, ntiles, bstart);
    else
      hipLaunchKernelGGL((k_radix_tile_scatter<false, true, ITEMS>), dim3(g), dim3(kThreads), 0, s, keys, vals,
                         nullptr, L, mk, mv, n, -1, hist, ntiles, bstart);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  ProfScope ps(KN_RADIX_LOCAL, s);
  hipLaunchKernelGGL(k_bucket_sort, dim3(256), dim3(kBucketThreads), kBucketLds, s, mk, mv, keys, vals, bstart, L, err);
  return hipGetLastError();
}

}  // namespace

// The by-bucket sort serves the sizes of the 1024-key tiles (at most kSmallTiles
// of them), whose histograms the bucket pass sums itself.
bool radix_bucket_applies(int64_t n) { return n > 1 && (n + kRsTileSmall - 1) / kRsTileSmall <= kSmallTiles; }

// Whether radix_sort_kv of n coordinates starts with a tile histogram (by bucket,
// or digit by digit below the one-kernel passes), which can compute the layout.
bool radix_fuses_layout(int64_t n, int passes, bool by_bucket) {
  if (by_bucket && radix_bucket_applies(n)) return true;
  return n > 1 && passes > 0 && passes <= kRsMaxPasses && n < ((int64_t)1 << 30) &&
         (n + kRsTileLarge - 1) / kRsTileLarge < kOnesweepMinTiles;
}

hipError_t radix_sort_kv(const int32_t* coords, const KeyLayout* L, uint64_t* keys, uint32_t* vals, uint64_t* keys_alt,
                         uint32_t* vals_alt, int64_t n, int passes, bool by_bucket, void* d_temp, uint32_t* err,
                         const LayoutArgs* lay, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const bool fuse = lay && coords && radix_fuses_layout(n, passes, by_bucket);
  if (lay && !fuse) {
    hipError_t e = launch_layout(*lay, s);
    if (e != hipSuccess) return e;
  }
  const LayoutArgs none{};
  const LayoutArgs& la = fuse ? *lay : none;
  if (by_bucket && radix_bucket_applies(n))
    return radix_sort_bucket(coords, L, keys, vals, keys_alt, vals_alt, n, d_temp, err, la, s);
  if (coords && (passes == 0 || n == 1)) return launch_pack(coords, n, L, keys, vals, s);
  if (n <= 1 || passes == 0) return hipSuccess;
  if (passes > kRsMaxPasses || n >= ((int64_t)1 << 30)) return hipErrorInvalidValue;
  if ((n + kRsTileLarge - 1) / kRsTileLarge < kOnesweepMinTiles)
    return radix_sort_tiled(coords, L, keys, vals, keys_alt, vals_alt, n, passes, d_temp, la, s);
  // one kernel per pass (the status words are sized for tiles of kRsTile keys, of
  // which there are more)
  const int64_t ntiles = (n + kRsTileLarge - 1) / kRsTileLarge;
  const size_t gpart_bytes = (size_t)kRsUpBlocks * kRsMaxPasses * 256 * sizeof(uint32_t);
  uint32_t* gpart = static_cast<uint32_t*>(d_temp);
  uint32_t* gofs = reinterpret_cast<uint32_t*>(static_cast<char*>(d_temp) + align256(gpart_bytes));
  uint32_t* status = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(gofs) +
                                                 align256((size_t)kRsMaxPasses * 256 * sizeof(uint32_t)));
  const int64_t status_words = (int64_t)passes * ntiles * 256;
  uint32_t* tickets = reinterpret_cast<uint32_t*>(
      reinterpret_cast<char*>(status) +
      (((size_t)kRsMaxPasses * ntiles * 256 * sizeof(uint32_t) + 255) & ~(size_t)255));
  const int gblocks = (int)std::min<int64_t>(kRsUpBlocks, ntiles);
  const int4* c4 = reinterpret_cast<const int4*>(coords);
  hipError_t e;
  {
    ProfScope ps(KN_RADIX_HIST, s);
    if (coords)
      hipLaunchKernelGGL(k_radix_upsweep<true>, dim3(gblocks), dim3(kThreads), 0, s, nullptr, c4, L, n, passes, gpart,
                         status, status_words, tickets);
    else
      hipLaunchKernelGGL(k_radix_upsweep<false>, dim3(gblocks), dim3(kThreads), 0, s, keys, nullptr, L, n, passes,
                         gpart, status, status_words, tickets);
    e = hipGetLastError();
    if (e == hipSuccess) {
      hipLaunchKernelGGL(k_radix_totals, dim3(passes), dim3(1024), 0, s, gpart, gblocks, passes, gofs);
      e = hipGetLastError();
    }
  }
  if (e != hipSuccess) return e;
  // ping-pong so that the last pass lands in (keys, vals)
  uint64_t* kb[2] = {keys, keys_alt};
  uint32_t* vb[2] = {vals, vals_alt};
  int cur = (passes % 2 == 0) ? 0 : 1;  // buffer holding the input of the next pass
  if (!coords && passes % 2 == 1) {
    // input is in (keys, vals); an odd pass count needs one copy into the other buffer
    ProfScope ps(KN_COPY, s);
    e = hipMemcpyAsync(keys_alt, keys, (size_t)n * 8, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(vals_alt, vals, (size_t)n * 4, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  for (int p = 0; p < passes; ++p) {
    const bool first = (p == 0) && coords;
    // the first pass from coordinates writes into buffer (passes odd ? 0 : 1) directly
    const int src = cur, dst = (first ? ((passes % 2 == 1) ? 0 : 1) : cur ^ 1);
    {
      ProfScope ps(KN_RADIX_SCATTER, s);
      if (first)
        hipLaunchKernelGGL((k_radix_pass<true, kRsItemsLarge>), dim3((unsigned)ntiles), dim3(kThreads), 0, s, nullptr,
                           nullptr, c4, L, kb[dst], vb[dst], n, p, gofs, status, tickets, err);
      else
        hipLaunchKernelGGL((k_radix_pass<false, kRsItemsLarge>), dim3((unsigned)ntiles), dim3(kThreads), 0, s,
                           kb[src], vb[src], nullptr, L, kb[dst], vb[dst], n, p, gofs, status, tickets, err);
      e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    cur = dst;
  }
  return hipSuccess;
}

hipError_t launch_down_keys(const uint64_t* skeys, int64_t n, const KeyLayout* L, int64_t cell, uint64_t* dkeys,
                            uint32_t* vals, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfScope ps(KN_DOWN_KEYS, s);
  hipLaunchKernelGGL(k_down_keys, dim3(grid_for(n)), dim3(kThreads), 0, s, skeys, n, L, cell, dkeys, vals);
  return hipGetLastError();
}

hipError_t unique_keys(const uint64_t* keys, int64_t n, const KeyLayout* L, uint32_t* flags, uint32_t* pos, void* d_temp,
                       uint64_t* qkeys, uint32_t* qrow, int32_t* out_coords, ControlBlock* cb, hipStream_t s) {
  if (n <= 0) return launch_fill_u32(&cb->n_q, 0u, 1, s);
  ProfScope ps(KN_UNIQUE, s);
  const int64_t ntiles = (n + kUniqueTile - 1) / kUniqueTile;
  if (ntiles <= kUniqueTiles) {
    // (the per-key flags' buffer holds the tile counts: n >= ntiles)
    hipLaunchKernelGGL(k_unique_tile_count, dim3((unsigned)ntiles), dim3(kThreads), 0, s, keys, n, flags);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_unique_tile_write, dim3((unsigned)ntiles), dim3(kThreads), 0, s, keys, n, L, flags, qkeys,
                       qrow, reinterpret_cast<int4*>(out_coords), &cb->n_q);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_unique_flags, dim3(grid_for(n)), dim3(kThreads), 0, s, keys, n, flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = scan_exclusive_u32(flags, pos, n, &cb->n_q, d_temp, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_unique_write, dim3(grid_for(n)), dim3(kThreads), 0, s, keys, n, L, flags, pos, qkeys, qrow,
                     reinterpret_cast<int4*>(out_coords));
  return hipGetLastError();
}

hipError_t launch_backward(const SearchArgs& a, int64_t nb, uint32_t* bounds, ControlBlock* cb, hipStream_t s) {
  const int64_t nkb = (int64_t)a.K3 * nb;
  if (nkb <= 0) return hipSuccess;
  const int64_t blocks = (nkb + kWavesPerBlock - 1) / kWavesPerBlock;
  ProfScope ps(KN_BACKWARD, s);
  hipLaunchKernelGGL(k_backward, dim3((unsigned)blocks), dim3(kThreads), 0, s, a, nb, bounds, cb);
  return hipGetLastError();
}

// Workgroups the count pass aims for when choosing its offset groups.
constexpr int64_t kCountTargetGroups = 4096;

hipError_t launch_forward(const SearchArgs& a, bool write, const uint32_t* bounds, int64_t nb, uint32_t* item_cnt,
                          const uint32_t* item_off, int32_t* pin, int32_t* pout, ControlBlock* cb, hipStream_t s) {
  if (nb <= 0) return hipSuccess;
  int log2B = 0;
  while ((1 << log2B) < a.B) ++log2B;
  const int th = a.wg > 0 ? a.wg : kThreads;
  const int rounds = a.Cq / th;
  // (threads, rounds) pairs: each chunk of Cq queries is rounds x threads
#define SPC_TR(TH_, R_, CALL) \
  if (th == TH_ && rounds == R_) return CALL;
#define SPC_TR_ALL(F, ...)                                                                                      \
  SPC_TR(128, 2, (F<2, 128>(__VA_ARGS__))) SPC_TR(128, 4, (F<4, 128>(__VA_ARGS__)))                            \
  SPC_TR(128, 8, (F<8, 128>(__VA_ARGS__))) SPC_TR(256, 1, (F<1, 256>(__VA_ARGS__)))                            \
  SPC_TR(256, 2, (F<2, 256>(__VA_ARGS__))) SPC_TR(256, 4, (F<4, 256>(__VA_ARGS__)))                            \
  SPC_TR(256, 8, (F<8, 256>(__VA_ARGS__))) SPC_TR(512, 1, (F<1, 512>(__VA_ARGS__)))                            \
  SPC_TR(512, 2, (F<2, 512>(__VA_ARGS__))) SPC_TR(512, 4, (F<4, 512>(__VA_ARGS__)))
  if (write) {
    const unsigned grid = (unsigned)((int64_t)a.K3 * nb);
    ProfScope ps(KN_FORWARD_WRITE, s);
    SPC_TR_ALL(forward_write_t, grid, s, a, bounds, nb, item_off, pin, pout, cb)
    return hipErrorInvalidValue;
  }
  const int64_t ngroups0 = std::min<int64_t>(a.K3, std::max<int64_t>(1, (kCountTargetGroups + nb - 1) / nb));
  // (at most 64 offsets per group: the kernel counts an offset's matches in one lane)
  const int G = std::min<int>(std::min(kWave, a.K3),
                              a.count_group > 0 ? a.count_group : (int)((a.K3 + ngroups0 - 1) / ngroups0));
  const int64_t ngroups = (a.K3 + G - 1) / G;
  const unsigned grid = (unsigned)(nb * ngroups);
  ProfScope ps(KN_FORWARD_COUNT, s);
  SPC_TR_ALL(forward_count_t, grid, s, a, bounds, nb, item_cnt, G, cb, log2B)
#undef SPC_TR_ALL
#undef SPC_TR
  return hipErrorInvalidValue;
}

hipError_t launch_hash_build(const int32_t* coords, int64_t n, const KeyLayout* L, uint64_t* hkeys, uint32_t* hvals,
                             int log2cap, uint64_t* keys, uint32_t* idx, uint32_t* err, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(hkeys), 0xFFFFFFFFu, (int64_t)2 << log2cap, s);
  if (e != hipSuccess) return e;
  ProfScope ps(KN_HASH_INSERT, s);
  hipLaunchKernelGGL(k_hash_insert, dim3(grid_for(n)), dim3(kThreads), 0, s, reinterpret_cast<const int4*>(coords), n,
                     L, hkeys, hvals, log2cap, keys, idx, err);
  return hipGetLastError();
}

hipError_t launch_hash_items(int K3, int64_t n_q, int Cq, int64_t nb, uint32_t* bounds, hipStream_t s) {
  const int64_t nkb = (int64_t)K3 * nb;
  if (nkb <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_hash_items, dim3(grid_for(nkb)), dim3(kThreads), 0, s, K3, n_q, Cq, nb, bounds);
  return hipGetLastError();
}

hipError_t launch_hash_count(const SearchArgs& a, const uint64_t* hkeys, const uint32_t* hvals, int log2cap,
                             int64_t nb, uint32_t* item_cnt, hipStream_t s) {
  const int64_t nkb = (int64_t)a.K3 * nb;
  if (nkb <= 0) return hipSuccess;
  ProfScope ps(KN_HASH_PROBE, s);
  const unsigned grid = (unsigned)nkb;
  switch (a.Cq / kThreads) {
#define SPC_H(R)                                                                                                   \
  case R:                                                                                                          \
    hipLaunchKernelGGL((k_hash_count<R>), dim3(grid), dim3(kThreads), 0, s, a, hkeys, hvals, log2cap, nb,         \
                       item_cnt);                                                                                  \
    break;
    SPC_H(1)
    SPC_H(2)
    SPC_H(4)
    SPC_H(8)
#undef SPC_H
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace spc
