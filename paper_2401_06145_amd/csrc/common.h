// Internal declarations shared by the library's HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>

#include <cstddef>
#include <cstdint>

namespace spc {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Coordinate keys.  (b, x, y, z) is packed into one unsigned 64-bit key whose
// unsigned order is the lexicographic order of the signed tuple: each field is
// biased by its low bound and given a fixed bit width, b in the top bits.  The
// bias leaves room for the kernel's reach, so for any offset delta the key of
// q + delta is key(q) + dkey(delta) with no carry between fields; a query
// segment of sorted outputs (Section 5.1.1) is then sorted in key order too.
// ---------------------------------------------------------------------------
struct KeyLayout {
  int64_t lo[4];   // value subtracted from field f before packing
  int shift[4];    // bit position of field f
  int width[4];    // bits of field f
  int total_bits;  // sum of widths (<= 62)
};

__device__ __forceinline__ uint64_t pack_key(const KeyLayout& L, const int32_t* c) {
  uint64_t k = 0;
#pragma unroll
  for (int f = 0; f < 4; ++f) k |= (uint64_t)((int64_t)c[f] - L.lo[f]) << L.shift[f];
  return k;
}

__device__ __forceinline__ int32_t key_field(const KeyLayout& L, uint64_t k, int f) {
  const uint64_t mask = (L.width[f] >= 64) ? ~0ull : ((1ull << L.width[f]) - 1ull);
  return (int32_t)((int64_t)((k >> L.shift[f]) & mask) + L.lo[f]);
}

// Wave helpers (wave64).
__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (kWave - 1);
  return (lane == 0) ? 0ull : (~0ull >> (64 - lane));
}

__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }

// Stores of rows that no kernel reads again soon (GEMM partial rows, layer outputs):
// non-temporal, so they stream to memory instead of leaving dirty lines in the
// caches that later kernels' traffic would have to write back.
__device__ __forceinline__ void store_stream(void* p, uint4 v) {
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(v4u{v.x, v.y, v.z, v.w}, reinterpret_cast<v4u*>(p));
}
__device__ __forceinline__ void store_stream(void* p, uint2 v) {
  typedef uint32_t v2u __attribute__((ext_vector_type(2)));
  __builtin_nontemporal_store(v2u{v.x, v.y}, reinterpret_cast<v2u*>(p));
}

// ---------------------------------------------------------------------------
// Device error flags, OR-ed into ControlBlock::err by kernels.
// ---------------------------------------------------------------------------
enum : uint32_t {
  kErrDup = 1u,          // two equal keys among the sorted inputs
  kErrSpin = 2u,         // a look-back wait exceeded its bound
  kErrOverflow = 4u,     // more work items than the launch was sized for
  kErrUnsorted = 8u,     // rows declared sorted are not in (b, x, y, z) order
  kErrRange = 16u,       // the coordinate extent plus kernel reach needs more than 62 key bits
  kErrWide = 32u,        // the key needs more bits than the sort passes planned by the host
  kErrBucket = 64u,      // a bucket of the by-bucket small sort exceeds what one workgroup sorts
};

// Small control block in device memory, read back once at the end of a map build.
constexpr int kMaxOffsets = 125;  // K <= 5
struct ControlBlock {
  uint32_t err;           // kErr* flags
  uint32_t n_q;           // number of distinct output coordinates (DOWN)
  uint32_t n_pairs;       // total matches
  uint32_t seg_pair_start[kMaxOffsets + 3];  // first pair of offset k; [K3] = n_pairs
  KeyLayout layout;       // key layout, computed on the device from the coordinate bounds
  int64_t dk[kMaxOffsets];  // packed key delta of each offset under that layout
};
// The part of the control block the host reads back after a build (counts, flags,
// the layout's width); the offset deltas stay on the device.
constexpr size_t kControlHeadBytes = offsetof(ControlBlock, dk);

// Inputs of the device-side key layout: the bounds partials of launch_minmax and
// the layer's geometry (kernel size, stride, tensor stride, K^3); passes = the
// digit passes the host planned its sort for (kErrWide above that).
struct LayoutArgs {
  const int32_t* partial;
  int np, K, stride, t, K3, passes;
  ControlBlock* cb;
};

// ---------------------------------------------------------------------------
// Measurement: HIP events around phases and around individual kernel launches,
// recorded only for the ids enabled in the profiling mask (api.hip).
// ---------------------------------------------------------------------------
enum ProfId : int {
  // phases (host-visible steps, including the read-back synchronisations)
  PH_BOUNDS = 0, PH_SORT, PH_OUTCOORDS, PH_BACKWARD, PH_BALANCE, PH_FORWARD, PH_READBACK,
  PH_METADATA, PH_GATHER, PH_GEMM, PH_SCATTER, PH_HASH,
  // kernels
  KN_MINMAX = 16, KN_RADIX_HIST, KN_RADIX_SCATTER, KN_SCAN, KN_COPY, KN_DOWN_KEYS, KN_UNIQUE,
  KN_BACKWARD, KN_FORWARD_COUNT, KN_FORWARD_WRITE, KN_FILL, KN_RADIX_LOCAL, KN_GATHER, KN_GEMM, KN_SCATTER,
  KN_PACK, KN_HASH_INSERT, KN_HASH_PROBE, KN_SCATTER_CENTRE,
  PROF_IDS = 40
};
struct ProfScope {
  void* rec = nullptr;
  ProfScope(int id, hipStream_t s);
  ~ProfScope();
};

// ---------------------------------------------------------------------------
// Launchers (host functions, defined next to their kernels).
// ---------------------------------------------------------------------------

// scan.hip: exclusive prefix sum of n uint32 values; *d_total (optional) gets the sum.
size_t scan_temp_bytes(int64_t n);
hipError_t scan_exclusive_u32(const uint32_t* d_in, uint32_t* d_out, int64_t n, uint32_t* d_total,
                              void* d_temp, hipStream_t s);

// map_kernels.hip
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s);
// T_s from the pair lists: ts[k stride + sorted source position of pin[e]] = e
// for every pair e of offset k (seg: the device's K3 + 1 pair starts).  perm:
// caller row of each sorted source position, or NULL (identity); inv: n_src
// words of scratch for its inverse.  The table must be filled with -1 first.
hipError_t launch_ts_from_pairs(const int32_t* pin, const uint32_t* seg, int K3, int64_t n_pairs,
                                const uint32_t* perm, int64_t n_src, uint32_t* inv, int32_t* ts,
                                int64_t stride, hipStream_t s);
size_t minmax_temp_bytes();
// Per-block coordinate bounds of a[0..na) and b[0..nb): *n_partial rows of 8
// int32 (min b,x,y,z then max b,x,y,z) in `partial`; also resets cb's counters.
hipError_t launch_minmax(const int32_t* a, int64_t na, const int32_t* b, int64_t nb, int32_t* partial,
                         ControlBlock* cb, int* n_partial, hipStream_t s);
hipError_t launch_pack(const int32_t* coords, int64_t n, const KeyLayout* L, uint64_t* keys, uint32_t* vals,
                       hipStream_t s);
size_t radix_temp_bytes(int64_t n);
// Device-side key layout from the bounds partials, into cb->layout and cb->dk (see
// k_layout); flags kErrRange / kErrWide (more than 8 * passes key bits).
hipError_t launch_layout(const LayoutArgs& la, hipStream_t s);
// Sorts by the low 8 * passes key bits (passes whose digit lies above the layout's
// key bits are plain copies); the result ends in (keys, vals).  If `coords` is
// non-null the input is those coordinates (keys packed with the device layout *L,
// values = row index).  Look-back waits that exceed their bound set kErrSpin in *err
// (nothing hangs).  by_bucket: where radix_bucket_applies(n), sort by the key's top
// digit and then each bucket in one workgroup instead (all key bits, whatever
// `passes`); a bucket too large for that sets kErrBucket and stays unsorted.
// lay: the layout is not computed yet; a sort of coordinates whose first kernel is a
// tile histogram (radix_fuses_layout) computes it there, in every workgroup, from
// these arguments (workgroup 0 publishes it), and any other sort launches the
// layout kernel first.  NULL: *L is ready.
bool radix_bucket_applies(int64_t n);
bool radix_fuses_layout(int64_t n, int passes, bool by_bucket);
hipError_t radix_sort_kv(const int32_t* coords, const KeyLayout* L, uint64_t* keys, uint32_t* vals,
                         uint64_t* keys_alt, uint32_t* vals_alt, int64_t n, int passes, bool by_bucket,
                         void* d_temp, uint32_t* err, const LayoutArgs* lay, hipStream_t s);
hipError_t launch_down_keys(const uint64_t* skeys, int64_t n, const KeyLayout* L, int64_t cell,
                            uint64_t* dkeys, uint32_t* vals, hipStream_t s);
// Distinct consecutive keys of sorted `keys` -> qkeys, qrow = position, coords; n_q into cb.
hipError_t unique_keys(const uint64_t* keys, int64_t n, const KeyLayout* L, uint32_t* flags,
                       uint32_t* pos, void* d_temp, uint64_t* qkeys, uint32_t* qrow,
                       int32_t* out_coords, ControlBlock* cb, hipStream_t s);

struct SearchArgs {
  const uint64_t* skeys;  // sorted source keys [n_src]
  const uint32_t* sidx;   // their caller rows
  int64_t n_src;
  const uint64_t* qkeys;  // sorted query base keys [n_q] (n_q read from n_q_dev if non-null)
  const uint32_t* qrow;   // their caller rows
  int64_t n_q;
  const uint32_t* n_q_dev;
  int K3;
  const int64_t* dk;      // key delta of each offset (device, from the layout kernel)
  int B;                  // source block size
  int Cq;                 // query block limit
  int swap_roles;         // UP: pairs are (query row, source row)
  int check_q;            // also check the query keys for repeats
  // Per-(offset, query) table T_q [K3][res_stride], indexed by sorted query
  // position: the count pass stores the matching sorted source position or -1,
  // the write pass replaces each match by its pair index (= GEMM buffer row).
  int32_t* res;
  int64_t res_stride;
  // Per-(offset, source) table T_s [K3][ts_stride], indexed by sorted source
  // position: pair index or -1.  The write pass stores the matches; the -1
  // entries come from a fill before it.
  int32_t* ts;
  int64_t ts_stride;
  int64_t pair_cap;       // capacity of the pair lists (K3 * queries)
  int wg;                 // threads per workgroup of the count and write passes (0: 256)
  int count_group;        // offsets per count-pass workgroup, at most 64 (0: size rule)
  int stream_tq;          // the count pass stores T_q with non-temporal stores
  // Submanifold map with odd K (offset k and K^3 - 1 - k are mirror images).
  int sym;
  // 0: the write pass leaves T_s alone (a symmetric map's T_s is filled from the
  // pair lists when a table-driven gather first needs it); else it stores T_s's
  // matches after a -1 fill.
  int write_ts;
  // Mapped, coherent host buffer (or NULL).  The write pass's first workgroup
  // copies the control block's head (kControlHeadBytes) into it, then stores
  // pub_seq at byte kPubFlagOffset: the host reads the counts while the rest of
  // the pass still runs, instead of waiting for the stream.
  uint32_t* pub;
  uint32_t pub_seq;
};
constexpr size_t kPubFlagOffset = 1024;
constexpr size_t kPubBytes = 4096;
static_assert(kControlHeadBytes % 4 == 0 && kControlHeadBytes <= kPubFlagOffset, "head fits before the flag");
// Section 5.1.2, backward search: bounds[k nb + b] = the end of the query block of
// offset k and source block b (its start is the previous block's end, 0 for b = 0);
// also the repeat check of transposed maps' query keys.
hipError_t launch_backward(const SearchArgs& a, int64_t nb, uint32_t* bounds, ControlBlock* cb, hipStream_t s);
// Forward search over the work items (k, b), each query block in chunks of at most
// Cq queries: count pass (write = false) fills T_q and item_cnt[k nb + b]; write
// pass places pairs from item_off[k nb + b] on and fills cb->seg_pair_start.
hipError_t launch_forward(const SearchArgs& a, bool write, const uint32_t* bounds, int64_t nb, uint32_t* item_cnt,
                          const uint32_t* item_off, int32_t* pin, int32_t* pout, ControlBlock* cb, hipStream_t s);

// Hash-table search (the prior-art Map, kept as an ablation): open addressing
// with linear probing over 64-bit keys, 2^log2cap slots (load <= 1/2).
constexpr uint64_t kHashEmpty = ~0ull;
// Clears the table, packs every input row (caller order) into keys[i] with
// idx[i] = i, and inserts (key, i); repeated keys set kErrDup in *err.
hipError_t launch_hash_build(const int32_t* coords, int64_t n, const KeyLayout* L, uint64_t* hkeys, uint32_t* hvals,
                             int log2cap, uint64_t* keys, uint32_t* idx, uint32_t* err, hipStream_t s);
// Work items of the probe: nb = ceil(n_q / Cq) blocks of Cq queries per offset,
// recorded as bounds[k nb + b] = min((b + 1) Cq, n_q) for the write pass.
hipError_t launch_hash_items(int K3, int64_t n_q, int Cq, int64_t nb, uint32_t* bounds, hipStream_t s);
// Probe pass: res[k][q] = matching input row or -1, item_cnt = matches per item.
hipError_t launch_hash_count(const SearchArgs& a, const uint64_t* hkeys, const uint32_t* hvals, int log2cap,
                             int64_t nb, uint32_t* item_cnt, hipStream_t s);

// gmas_kernels.hip.  Metadata tables are offset-major over sorted positions:
// entry [k * stride + p] is the buffer row of point p's pair at offset k, or -1;
// perm[p] is the caller row of sorted position p (NULL: the identity).
// Algorithm 1 gather with tile T channels per thread; elem = element bytes.
hipError_t launch_gather(const void* x, int64_t n_in, int c_in, int elem, const int32_t* imt,
                         int64_t mt_stride, const uint32_t* perm, int K3, void* buf_in, int tile,
                         hipStream_t s);
// Scatter: y[perm[p]] = sum_k buf_out[omt[k][p]] (float32 sum, k ascending), tile T
// channels per thread.  Optional epilogue: y = relu?(sum + residual) (residual NULL: none).
// stream: the row-group kernel's output rows go out with non-temporal stores
// (store_stream); the one-thread-per-tile kernel always stores plainly.
hipError_t launch_scatter(const void* buf_out, int part_dtype, int64_t n_out, int c_out,
                          const int32_t* omt, int64_t mt_stride, const uint32_t* perm, int K3, void* y,
                          int dtype, int tile, const void* residual, int relu, bool stream, hipStream_t s);
// out[i] = [a[i] | b[i]] for row-major a [n][ca], b [n][cb] (16-byte multiples).
hipError_t launch_concat(const void* a, int ca, const void* b, int cb, void* out, int64_t n, int elem,
                         hipStream_t s);

// gemm_mfma.hip: grouped per-offset GEMMs, buf_out[rows of k] = buf_in[rows of k] W_k.
// A segment is one offset's run of buffer rows; `height` >= `rows` is the padded
// height the group computes (padding rows are zeros: computed, never loaded or stored).
struct GemmSeg {
  int k;
  int64_t row0;
  int64_t rows;
  int64_t height;
};
// Whether the full-width kernel applies, and whether it wants the weights
// transposed beforehand (large W_k; small ones are transposed while staging).
bool gemm_wide(int c_in, int c_out, int dtype, int part_dtype);
bool gemm_wide_transposed(int c_in, int c_out);
// wt[k][n][c] = w[k][c][n] for 16-bit weights.
hipError_t launch_transpose_w(const void* w, void* wt, int K3, int c_in, int c_out, hipStream_t s);
// Launches the segments (any number; split into launches of at most 64 segments).
// a_rows NULL: buffer row r of the A operand is buf_in row r (the gathered buffer).
// a_rows set: the gather is fused into the operand loads, row r is buf_in row
// a_rows[r] (buf_in is then the layer's input features, a_rows the pairs' input rows).
// wt: transposed weights (launch_transpose_w) or NULL;
// dump_row: one spare row of c_out partials the full-width kernel may overwrite.
// tile_rows: output rows per workgroup tile (0: about two tiles per workgroup slot)
// stream: the full-width kernel writes the partial rows with non-temporal stores.
hipError_t launch_gemm(const GemmSeg* segs, int n_seg, const void* buf_in, const int32_t* a_rows, const void* w,
                       const void* wt, void* buf_out, void* dump_row, int c_in, int c_out, int dtype, int part_dtype,
                       int tile_rows, bool stream, hipStream_t s);
// The submanifold centre offset computed inside the scatter (odd K): y[perm[p]] =
// relu?(x[perm[p]] W_kc + sum over k != kc of buf_out[omt[k][p]] + residual), the
// centre first, then k ascending, in float32.  Whether an instance exists for the
// layer (16-bit layers, c_in % 8 == 0 up to 256, c_out % 32 == 0 up to 256), and
// its launcher.  wt: transposed weights or NULL.
bool centre_fusable(int c_in, int c_out, int dtype, int part_dtype);
hipError_t launch_scatter_centre(const void* x, const uint32_t* perm, const void* w, const void* wt, int kc,
                                 const void* buf_out, const int32_t* omt, int64_t mt_stride, int K3, void* y,
                                 const void* residual, int relu, int64_t n_out, int c_in, int c_out, int dtype,
                                 int part_dtype, bool stream, hipStream_t s);

}  // namespace spc
