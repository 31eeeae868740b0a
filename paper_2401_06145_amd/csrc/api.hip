// Host side of the C-ABI (include/spconv.h): argument checks, workspace plans,
// the Map-step orchestration (Section 5.1) and the GMaS plan (Section 5.2).
#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "common.h"
#include "spconv.h"

using namespace spc;

struct spconv_map {
  int mode = 0, K = 0, K3 = 0, stride = 1, tstride = 1;
  int64_t n_in = 0, n_out = 0;
  const int32_t* out_coords = nullptr;
  const int32_t* pin = nullptr;   // concatenated pair lists, offset-major
  const int32_t* pout = nullptr;
  std::vector<int64_t> counts;    // |M_k|
  std::vector<int64_t> ptr;       // prefix of counts, K3 + 1 entries
  // metadata tables, offset-major over sorted positions (entry k * stride + p:
  // buffer row of point p's pair at offset k, or -1), and the caller row of each
  // sorted position (NULL: identity); NULL tables for a map without pairs
  const int32_t* imt = nullptr;
  const int32_t* omt = nullptr;
  int64_t imt_stride = 0, omt_stride = 0;
  const uint32_t* in_perm = nullptr;
  const uint32_t* out_perm = nullptr;
  bool transposed = false;
  // A symmetric submanifold map leaves its source-side table (imt) to be filled
  // from the pair lists by the first forward call that gathers through it; the
  // fused gather reads the pair lists and never needs it.
  mutable bool imt_pending = false;
  const uint32_t* seg_dev = nullptr;  // device pair starts, K3 + 1 entries
  uint32_t* inv_scratch = nullptr;    // n_in words of the build's scratch
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(SPCONV_EHIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define SPC_TRY(expr, where)              \
  do {                                    \
    hipError_t _e = (expr);               \
    if (_e != hipSuccess) return hip_fail(_e, where); \
  } while (0)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Bump allocator over a workspace; with base == nullptr it only measures.
struct Bump {
  char* base;
  size_t off = 0;
  explicit Bump(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(int64_t n) {
    off = align_up(off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += (size_t)(n > 0 ? n : 0) * sizeof(T);
    return p;
  }
  void* take_bytes(size_t n) {
    off = align_up(off, 256);
    void* p = base ? base + off : nullptr;
    off += n;
    return p;
  }
};

// ---------------------------------------------------------------------------
// Phase timing (measurement API): HIP events around each phase on the stream.
// ---------------------------------------------------------------------------
const char* prof_name(int id) {
  static const char* kNames[PROF_IDS] = {
      "bounds", "sort", "outcoords", "backward", "balance", "forward", "readback", "metadata", "gather", "gemm",
      "scatter", "hash", "", "", "", "",
      "k_minmax", "k_radix_hist", "k_radix_scatter", "k_scan", "k_copy", "k_down_keys", "k_unique", "k_backward",
      "k_forward_count", "k_forward_write", "k_fill", "k_radix_local", "k_gather", "k_gemm", "k_scatter", "k_pack",
      "k_hash_insert", "k_hash_probe", "k_scatter_centre", "", "", "", "", ""};
  return (id >= 0 && id < PROF_IDS) ? kNames[id] : "";
}
struct PhaseRec {
  int phase;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
uint64_t g_prof_mask = 0;
std::vector<PhaseRec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t ev_get() {
  hipEvent_t e = nullptr;
  if (!g_pool.empty()) {
    e = g_pool.back();
    g_pool.pop_back();
  } else if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
    // timing events only: no system-scope release needed around the timed kernels
    e = nullptr;
  }
  return e;
}

struct OpenRec {
  int id;
  hipStream_t s;
  hipEvent_t a;
};

}  // namespace

namespace spc {
ProfScope::ProfScope(int id, hipStream_t s) {
  if (!((g_prof_mask >> id) & 1ull)) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t a = ev_get();
  if (!a) return;
  (void)hipEventRecord(a, s);
  rec = new (std::nothrow) OpenRec{id, s, a};
}
ProfScope::~ProfScope() {
  if (!rec) return;
  OpenRec* r = static_cast<OpenRec*>(rec);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t b = ev_get();
  if (b) {
    (void)hipEventRecord(b, r->s);
    g_recs.push_back({r->id, r->a, b});
  }
  delete r;
}
}  // namespace spc

namespace {
using PhaseScope = spc::ProfScope;

// Mapped, coherent host buffer into which a map build's write pass publishes the
// control block's head (one per thread: a build returns only once it has read
// it).  Allocated on a thread's first build and kept; the device address of
// mapped memory is the same on every device.
struct PubBuffer {
  uint32_t* host = nullptr;
  uint32_t* dev = nullptr;
  uint32_t seq = 0;
};
thread_local PubBuffer g_pub;

PubBuffer* pub_buffer() {
  if (!g_pub.host) {
    void* p = nullptr;
    if (hipHostMalloc(&p, kPubBytes, hipHostMallocMapped | hipHostMallocPortable | hipHostMallocCoherent) != hipSuccess)
      return nullptr;
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, p, 0) != hipSuccess) {
      (void)hipHostFree(p);
      return nullptr;
    }
    std::memset(p, 0, kPubBytes);
    g_pub.host = static_cast<uint32_t*>(p);
    g_pub.dev = static_cast<uint32_t*>(d);
  }
  return &g_pub;
}

// Waits until the write pass has published sequence number `seq`: spins on the
// flag for up to 2 ms (the head is published at the start of the pass), then
// blocks on the stream, after which the flag must be set.
hipError_t pub_wait(const PubBuffer* pb, uint32_t seq, hipStream_t s, bool* ok) {
  const uint32_t* flag = pb->host + kPubFlagOffset / 4;
  const auto t0 = std::chrono::steady_clock::now();
  for (uint32_t spin = 0;; ++spin) {
    if (__atomic_load_n(flag, __ATOMIC_ACQUIRE) == seq) {
      *ok = true;
      return hipSuccess;
    }
    if ((spin & 1023u) == 1023u && std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(2)) break;
    __builtin_ia32_pause();
  }
  const hipError_t e = hipStreamSynchronize(s);
  *ok = __atomic_load_n(flag, __ATOMIC_ACQUIRE) == seq;
  return e;
}

// ---------------------------------------------------------------------------
// Map workspace plan
// ---------------------------------------------------------------------------
struct MapBufs {
  uint64_t* skeys;
  uint32_t* sidx;
  uint64_t* qkeys;
  uint32_t* qrow;
  int32_t* qcoords;
  int32_t* pin;
  int32_t* pout;
  uint32_t* counts;
  ControlBlock* cb;
  uint64_t* kalt;
  uint32_t* valt;
  uint64_t* dkeys;
  uint32_t* dvals;
  uint32_t* flags;
  uint32_t* pos;
  void* sort_tmp;
  uint32_t* bounds;  // per work item (offset, block): end of its query block
  int32_t* res;   // T_q, kept as the map's query-side metadata table
  int32_t* ts;    // T_s, the source-side table
  // Row strides of the two tables: the point counts rounded up to 32 entries, so
  // that every row starts on a 128-byte line.  The scatter (and the gather) read
  // 32 consecutive positions of a row per workgroup; with unpadded rows those
  // straddled two lines, each shared with a neighbouring workgroup that usually
  // runs on another die and fetched it again.
  int64_t res_stride;
  int64_t ts_stride;
  uint32_t* item_cnt;
  uint32_t* item_off;
  uint64_t* hkeys;  // hash-table search only
  uint32_t* hvals;
  int log2cap;
  int32_t* mm_partial;
  void* scan_tmp;
  int64_t max_items;  // work items: K3 * nb_items
  int64_t nb;         // source blocks of B keys
  int64_t nb_items;   // blocks per offset of the work items: nb, or for the hash-table
                      // search blocks of Cq queries
};

struct Tunables {
  int B = 1024;
  int Cq = 1024;
  int wg = 256;
  int count_group = 0;  // offsets per count-pass workgroup (0: size rule)
  bool presorted = false;
  bool hash = false;  // hash-table search instead of the sorted-array search
};

// Search hyperparameters (Section 5.1.4) left at 0 follow the source-set size:
// B = 1024, Cq = 1024 and 256-thread workgroups below 2^18 points, B = 4096,
// Cq = 2048 and 512 threads from there on (measured on gfx950: the 300k-point indoor
// room's search 90.7 -> 75.2 us, 4M-16M uniform and LiDAR clouds 2-13% faster;
// below 2^18 points the smaller blocks win: LiDAR 120k 31.1 vs 34.6 us, the 200k
// downsampling map 23.1 vs 27.7 us).  The rule applies only when none of the three
// is given.
void apply_size_rule(const spconv_options* opt, int64_t n_src, Tunables* t) {
  if (opt && (opt->B || opt->Cq || opt->wg)) return;
  if (n_src >= ((int64_t)1 << 18)) {
    t->B = 4096;
    t->Cq = 2048;
    t->wg = 512;
  }
}

int read_tunables(const spconv_options* opt, Tunables* t) {
  if (!opt) return SPCONV_OK;
  if (opt->B) {
    if (opt->B < 64 || opt->B > 4096 || (opt->B & (opt->B - 1)))
      return fail(SPCONV_EINVAL, "B must be a power of two in [64, 4096]");
    t->B = opt->B;
  }
  if (opt->Cq) {
    const int r = opt->Cq / 256;
    if (opt->Cq % 256 != 0 || !(r == 1 || r == 2 || r == 4 || r == 8))
      return fail(SPCONV_EINVAL, "Cq must be 256, 512, 1024 or 2048");
    t->Cq = opt->Cq;
  }
  if (opt->wg) {
    if (opt->wg != 128 && opt->wg != 256 && opt->wg != 512) return fail(SPCONV_EINVAL, "wg must be 128, 256 or 512");
    t->wg = opt->wg;
  }
  {
    const int r = t->Cq / t->wg;
    if (t->Cq % t->wg != 0 || !(r == 1 || r == 2 || r == 4 || r == 8))
      return fail(SPCONV_EINVAL, "Cq / wg must be 1, 2, 4 or 8");
  }
  if (opt->count_group < 0 || opt->count_group > 64) return fail(SPCONV_EINVAL, "count_group must be in [0, 64]");
  t->count_group = opt->count_group;
  t->presorted = opt->presorted != 0;
  if (opt->search < 0 || opt->search > 1) return fail(SPCONV_EINVAL, "search must be 0 or 1");
  t->hash = opt->search == 1;
  return SPCONV_OK;
}

size_t plan_map(void* base, int64_t n_src, int64_t nq_max, int K3, const Tunables& tu, int mode, MapBufs* b) {
  Bump m(base);
  const int64_t nmax = std::max(n_src, nq_max);
  b->nb = (n_src + tu.B - 1) / tu.B;
  b->nb_items = tu.hash ? (nq_max + tu.Cq - 1) / tu.Cq : b->nb;
  b->max_items = (int64_t)K3 * b->nb_items;
  b->skeys = m.take<uint64_t>(n_src);
  b->sidx = m.take<uint32_t>(n_src);
  b->qkeys = (mode == SPCONV_SUBM) ? nullptr : m.take<uint64_t>(nq_max);
  b->qrow = (mode == SPCONV_SUBM) ? nullptr : m.take<uint32_t>(nq_max);
  b->qcoords = (mode == SPCONV_DOWN) ? m.take<int32_t>(4 * nq_max) : nullptr;
  b->pin = m.take<int32_t>((int64_t)K3 * nq_max);
  b->pout = m.take<int32_t>((int64_t)K3 * nq_max);
  b->counts = m.take<uint32_t>(K3);
  b->cb = m.take<ControlBlock>(1);
  // build-time scratch
  b->kalt = m.take<uint64_t>(nmax);
  b->valt = m.take<uint32_t>(nmax);
  b->dkeys = (mode == SPCONV_DOWN) ? m.take<uint64_t>(n_src) : nullptr;
  b->dvals = (mode == SPCONV_DOWN) ? m.take<uint32_t>(n_src) : nullptr;
  b->flags = (mode == SPCONV_DOWN) ? m.take<uint32_t>(n_src) : nullptr;
  b->pos = (mode == SPCONV_DOWN) ? m.take<uint32_t>(n_src) : nullptr;
  b->sort_tmp = m.take_bytes(radix_temp_bytes(nmax));
  b->bounds = m.take<uint32_t>(b->max_items);
  b->res_stride = (int64_t)align_up((size_t)nq_max, 32);
  b->ts_stride = (int64_t)align_up((size_t)n_src, 32);
  b->res = m.take<int32_t>((int64_t)K3 * b->res_stride);
  b->ts = m.take<int32_t>((int64_t)K3 * b->ts_stride);
  b->item_cnt = m.take<uint32_t>(b->max_items);
  b->item_off = m.take<uint32_t>(b->max_items);
  b->mm_partial = static_cast<int32_t*>(m.take_bytes(minmax_temp_bytes()));
  b->scan_tmp = m.take_bytes(scan_temp_bytes(std::max(n_src, b->max_items)));
  b->log2cap = 0;
  b->hkeys = nullptr;
  b->hvals = nullptr;
  if (tu.hash) {
    // 2^log2cap >= 2 n slots: load at most 1/2
    int lg = 2;
    while (((int64_t)1 << lg) < 2 * std::max<int64_t>(n_src, 1)) ++lg;
    b->log2cap = lg;
    b->hkeys = m.take<uint64_t>((int64_t)1 << lg);
    b->hvals = m.take<uint32_t>((int64_t)1 << lg);
  }
  return align_up(m.off, 256);
}

int check_map_args(int64_t n_in, int64_t n_out, int K, int stride, int t, int mode) {
  if (K < 1 || K > 5) return fail(SPCONV_EUNSUPPORTED, "K must be in [1, 5]");
  if (t < 1) return fail(SPCONV_EINVAL, "tensor_stride must be >= 1");
  if (mode != SPCONV_SUBM && mode != SPCONV_DOWN && mode != SPCONV_UP) return fail(SPCONV_EINVAL, "bad mode");
  if (mode == SPCONV_SUBM && stride != 1) return fail(SPCONV_EINVAL, "SPCONV_SUBM requires stride 1");
  if (stride < 1) return fail(SPCONV_EINVAL, "stride must be >= 1");
  if (n_in < 0 || n_out < 0) return fail(SPCONV_EINVAL, "negative size");
  if (n_in >= (int64_t)1 << 31 || n_out >= (int64_t)1 << 31) return fail(SPCONV_EUNSUPPORTED, "more than 2^31 rows");
  // pair indices (and GEMM buffer rows) are int32: K^3 * max(n_in, n_out) bounds their count
  if ((int64_t)K * K * K * std::max(n_in, n_out) >= (int64_t)1 << 31)
    return fail(SPCONV_EUNSUPPORTED, "K^3 * rows must stay below 2^31");
  return SPCONV_OK;
}

// ---------------------------------------------------------------------------
// GMaS plan: GEMM grouping (Section 5.2.2) and tiles (Algorithm 1)
// ---------------------------------------------------------------------------
struct GmasPlan {
  int dtype = 0, elem = 4, pelem = 4, part_dtype = 0;
  int t_gather = 0, t_scatter = 0;
  int grouping = SPCONV_GROUP_RAGGED;
  int gather = 2;  // 1: Algorithm 1 into a buffer; 2: fused into the GEMM's operand loads
  int gemm_tile_rows = 0;  // 0: the occupancy rule
  // odd-K submanifold maps: the centre offset's product is computed inside the
  // scatter (k_scatter_centre) and the GEMMs skip that offset; -1: not fused
  int centre_k = -1;
  int64_t rows_pairs = 0;                 // all pairs of the map (partial buffer rows)
  int64_t rows_real = 0, rows_padded = 0;  // the GEMMs' rows, without and with padding
  int n_launches = 0;
  std::vector<std::vector<GemmSeg>> launches;  // one entry per GEMM launch (group)
};

int elem_bytes(int dtype) { return dtype == SPCONV_F32 ? 4 : 2; }

// Groups consecutive entries of `order` (offset ids) minimising
// sum_g (launch_cost + members_g * max_count_g); returns group boundaries.
std::vector<int> dp_groups(const std::vector<int>& order, const std::vector<int64_t>& cnt, int64_t launch_cost) {
  const int n = (int)order.size();
  std::vector<int64_t> best(n + 1, INT64_MAX);
  std::vector<int> from(n + 1, 0);
  best[0] = 0;
  for (int j = 1; j <= n; ++j) {
    int64_t mx = 0;
    for (int i = j - 1; i >= 0; --i) {
      mx = std::max(mx, cnt[order[i]]);
      const int64_t c = best[i] + launch_cost + (int64_t)(j - i) * mx;
      if (c < best[j]) {
        best[j] = c;
        from[j] = i;
      }
    }
  }
  std::vector<int> cuts;
  for (int j = n; j > 0; j = from[j]) cuts.push_back(j);
  cuts.push_back(0);
  std::reverse(cuts.begin(), cuts.end());
  return cuts;
}

// Large regions that the forward writes once and a later kernel reads once (the
// GEMM partial rows, the layer's output rows) go out with non-temporal stores.
// Otherwise their dirty lines stay in the caches, and the next kernels' traffic has to
// write them back.
constexpr int64_t kStreamPartialBytes = (int64_t)128 << 20;
constexpr int64_t kStreamOutputBytes = (int64_t)64 << 20;

int make_plan(const spconv_map* m, int c_in, int c_out, int dtype, const spconv_options* opt, GmasPlan* p) {
  if (!m) return fail(SPCONV_EINVAL, "map is NULL");
  if (dtype != SPCONV_F32 && dtype != SPCONV_F16 && dtype != SPCONV_BF16) return fail(SPCONV_EUNSUPPORTED, "dtype");
  p->dtype = dtype;
  p->elem = elem_bytes(dtype);
  if (c_in < 1 || c_out < 1 || c_in > 1024 || c_out > 1024) return fail(SPCONV_EUNSUPPORTED, "channels must be in [1, 1024]");
  if ((c_in * p->elem) % 16 != 0) return fail(SPCONV_EUNSUPPORTED, "c_in rows must be whole 16-byte vectors");
  if (c_out % 16 != 0) return fail(SPCONV_EUNSUPPORTED, "c_out must be a multiple of 16");
  // GEMM partials: 1 = float32, 2 = the layer dtype; default the layer dtype (the
  // scatter sums them in float32 either way)
  const int pd = opt ? opt->partial_dtype : 0;
  if (pd < 0 || pd > 2) return fail(SPCONV_EINVAL, "partial_dtype must be 0, 1 or 2");
  p->part_dtype = (pd == 1) ? SPCONV_F32 : dtype;
  p->pelem = elem_bytes(p->part_dtype);
  // tiles: default one 16-byte vector per thread for gather and for the partial reads of scatter
  p->t_gather = (opt && opt->t_gather) ? opt->t_gather : 16 / p->elem;
  // scatter: one 16-byte partial vector per thread (the row-group scatter, which reads
  // each output's table entries once)
  p->t_scatter = (opt && opt->t_scatter) ? opt->t_scatter : 16 / p->pelem;
  if (p->t_gather <= 0 || c_in % p->t_gather != 0 || (p->t_gather * p->elem) % 16 != 0 ||
      (p->t_gather * p->elem / 16) > 16 || ((p->t_gather * p->elem / 16) & (p->t_gather * p->elem / 16 - 1)))
    return fail(SPCONV_EINVAL, "t_gather must divide c_in and span 1, 2, 4, 8 or 16 16-byte vectors");
  const int ts = p->t_scatter;
  if (!(ts == 4 || ts == 8 || ts == 16 || ts == 32 || ts == 64) || c_out % ts != 0 || (ts * p->pelem) % 16 != 0)
    return fail(SPCONV_EINVAL, "t_scatter must be 4..64 (power of two), divide c_out and span whole 16-byte partial vectors");
  p->grouping = (opt && opt->grouping) ? opt->grouping - 1 : SPCONV_GROUP_RAGGED;
  if (p->grouping < 0 || p->grouping > 2) return fail(SPCONV_EINVAL, "grouping");
  p->gather = (opt && opt->gather) ? opt->gather : SPCONV_GATHER_FUSED;
  p->gemm_tile_rows = opt ? opt->gemm_tile_rows : 0;
  if (p->gemm_tile_rows < 0 || p->gemm_tile_rows > (1 << 20)) return fail(SPCONV_EINVAL, "gemm_tile_rows must be in [0, 2^20]");
  if (p->gather != SPCONV_GATHER_BUFFER && p->gather != SPCONV_GATHER_FUSED)
    return fail(SPCONV_EINVAL, "gather must be 0, SPCONV_GATHER_BUFFER or SPCONV_GATHER_FUSED");

  const int K3 = m->K3;
  p->rows_pairs = m->ptr[K3];
  p->rows_padded = 0;
  p->launches.clear();
  const int centre = opt ? opt->centre : 0;
  if (centre < 0 || centre > 2) return fail(SPCONV_EINVAL, "centre must be 0, 1 or 2");
  p->centre_k = -1;
  if (centre != 1) {
    const int kc = (K3 - 1) / 2;
    const bool applies = m->mode == SPCONV_SUBM && m->K % 2 == 1 && m->omt && m->n_out > 0 &&
                         m->counts[kc] == m->n_out && p->gather == SPCONV_GATHER_FUSED &&
                         c_in <= 256 && c_out <= 256 && centre_fusable(c_in, c_out, dtype, p->part_dtype);
    if (applies) p->centre_k = kc;
    else if (centre == 2)
      return fail(SPCONV_EUNSUPPORTED, "centre = 2: the centre offset cannot be fused into the scatter here (needs "
                                       "an odd-K submanifold map, the fused gather, a 16-bit layer, c_in % 8 == 0 "
                                       "and c_out % 32 == 0, both at most 256)");
  }
  auto in_gemm = [&](int k) { return m->counts[k] > 0 && k != p->centre_k; };
  p->rows_real = p->rows_pairs - (p->centre_k >= 0 ? m->counts[p->centre_k] : 0);
  // Buffer rows follow the concatenated pair lists (row of pair e of offset k =
  // ptr[k] + e); grouping decides launches and padded heights only.
  if (p->grouping == SPCONV_GROUP_RAGGED) {
    std::vector<int> order;
    for (int k = 0; k < K3; ++k)
      if (in_gemm(k)) order.push_back(k);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return m->counts[a] > m->counts[b]; });
    std::vector<GemmSeg> segs;
    for (int k : order) segs.push_back(GemmSeg{k, m->ptr[k], m->counts[k], m->counts[k]});
    p->rows_padded = p->rows_real;
    if (!segs.empty()) p->launches.push_back(segs);
  } else {
    std::vector<int> order(K3);
    for (int k = 0; k < K3; ++k) order[k] = k;
    if (p->grouping == SPCONV_GROUP_SORTED)  // non-decreasing pair count
      std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return m->counts[a] < m->counts[b]; });
    std::vector<int> nz;
    for (int k : order)
      if (in_gemm(k)) nz.push_back(k);
    const int64_t L = (opt && opt->launch_cost_rows > 0) ? opt->launch_cost_rows : 32768;
    const std::vector<int> cuts = dp_groups(nz, m->counts, L);
    for (size_t g = 0; g + 1 < cuts.size(); ++g) {
      int64_t h = 0;
      for (int i = cuts[g]; i < cuts[g + 1]; ++i) h = std::max(h, m->counts[nz[i]]);
      std::vector<GemmSeg> segs;
      for (int i = cuts[g]; i < cuts[g + 1]; ++i) {
        const int k = nz[i];
        segs.push_back(GemmSeg{k, m->ptr[k], m->counts[k], h});
        p->rows_padded += h;
      }
      p->launches.push_back(segs);
    }
  }
  p->n_launches = (int)p->launches.size();
  return SPCONV_OK;
}

struct FwdBufs {
  void* wt;  // transposed weights for the full-width GEMM, or NULL
  void* buf_in;
  void* buf_out;
};

size_t plan_forward_ws(void* base, const spconv_map* m, int c_in, int c_out, const GmasPlan& p, FwdBufs* b) {
  Bump a(base);
  b->wt = (gemm_wide(c_in, c_out, p.dtype, p.part_dtype) && gemm_wide_transposed(c_in, c_out))
              ? a.take_bytes((size_t)m->K3 * c_in * c_out * p.elem)
              : nullptr;
  // the fused gather reads the input rows directly: no gathered buffer
  b->buf_in = (p.gather == SPCONV_GATHER_BUFFER) ? a.take_bytes((size_t)p.rows_pairs * c_in * p.elem) : nullptr;
  // one spare row past the partials: the full-width GEMM's stores of rows without data
  // (rows are pair indices: with the centre fused its rows stay unused)
  b->buf_out = a.take_bytes((size_t)(p.rows_pairs + 1) * c_out * p.pelem);
  return align_up(a.off, 256);
}

}  // namespace

// ===========================================================================
// C-ABI
// ===========================================================================
extern "C" {

const char* spconv_last_error(void) { return g_err.c_str(); }

size_t spconv_map_workspace_bytes(int64_t n_in, int64_t n_out, int K, int mode, const spconv_options* opt) {
  if (check_map_args(n_in, n_out, K, mode == SPCONV_SUBM ? 1 : 2, 1, mode) != SPCONV_OK) return 0;
  Tunables tu;
  if (read_tunables(opt, &tu) != SPCONV_OK) return 0;
  const int64_t n_src = (mode == SPCONV_UP) ? n_out : n_in;
  apply_size_rule(opt, n_src, &tu);
  const int64_t nq_max = n_in;
  MapBufs b;
  return plan_map(nullptr, n_src, nq_max, K * K * K, tu, mode, &b);
}

}  // extern "C"

namespace {

// Sort passes to plan for a build before its key layout is known (the layout is
// computed on the device, so the host never waits for the bounds): the count the
// same inputs needed last time, else the last count needed on this thread (start:
// 4 passes, a 32-bit key).  A build whose key turns out wider is redone with the
// passes it needs.  Inputs are told apart by address, sizes and layer arguments
// only, so a new cloud at a reused address inherits a plan; a wrong plan costs at
// most that redo (or, planned too long, digit passes that copy).
// Sort plan of a map build, kept per input from the previous build of it: the
// digit passes of the digit-by-digit sort, and whether the small sorts may go by
// bucket (no bucket of the previous build was too large for one workgroup).
struct SortPlan {
  int passes = 4;
  bool by_bucket = true;
};
struct PassHint {
  std::unordered_map<std::string, SortPlan> by_input;
  int last = 4;
};
thread_local PassHint g_pass_hint;

std::string pass_key(const int32_t* a, int64_t na, const int32_t* b, int64_t nb, int K, int stride, int t, int mode) {
  char buf[160];
  snprintf(buf, sizeof(buf), "%p/%lld/%p/%lld/%d/%d/%d/%d", (const void*)a, (long long)na, (const void*)b,
           (long long)nb, K, stride, t, mode);
  return buf;
}

int build_map_impl(const int32_t* d_in_coords, int64_t n_in, const int32_t* d_out_coords, int64_t n_out, int K,
                   int stride, int tensor_stride, int mode, const spconv_options* opt, void* d_workspace,
                   size_t ws_bytes, void* stream, spconv_map** out_map, int passes, bool by_bucket,
                   int* passes_needed, bool* bucket_failed) {
  *passes_needed = 0;
  *bucket_failed = false;
  if (!out_map) return fail(SPCONV_EINVAL, "out_map is NULL");
  *out_map = nullptr;
  int st = check_map_args(n_in, mode == SPCONV_UP ? n_out : 0, K, stride, tensor_stride, mode);
  if (st != SPCONV_OK) return st;
  if (n_in > 0 && !d_in_coords) return fail(SPCONV_EINVAL, "d_in_coords is NULL");
  if (mode == SPCONV_UP && n_out > 0 && !d_out_coords) return fail(SPCONV_EINVAL, "d_out_coords is NULL");
  if (mode != SPCONV_UP) n_out = 0;
  Tunables tu;
  if ((st = read_tunables(opt, &tu)) != SPCONV_OK) return st;
  if (tu.hash && mode != SPCONV_SUBM) return fail(SPCONV_EUNSUPPORTED, "the hash-table search covers SPCONV_SUBM only");
  const int K3 = K * K * K;
  const int64_t n_src = (mode == SPCONV_UP) ? n_out : n_in;
  apply_size_rule(opt, n_src, &tu);
  const int64_t nq_max = n_in;
  MapBufs b;
  const size_t need = plan_map(nullptr, n_src, nq_max, K3, tu, mode, &b);
  if (!d_workspace || ws_bytes < need) return fail(SPCONV_ENOSPC, "map workspace too small");
  if (reinterpret_cast<uintptr_t>(d_workspace) % 256 != 0) return fail(SPCONV_EINVAL, "workspace must be 256-byte aligned");
  plan_map(d_workspace, n_src, nq_max, K3, tu, mode, &b);
  hipStream_t s = static_cast<hipStream_t>(stream);

  spconv_map* m = new (std::nothrow) spconv_map();
  if (!m) return fail(SPCONV_EINVAL, "out of host memory");
  m->mode = mode;
  m->K = K;
  m->K3 = K3;
  m->stride = stride;
  m->tstride = tensor_stride;
  m->n_in = n_in;
  m->n_out = (mode == SPCONV_SUBM) ? n_in : (mode == SPCONV_UP ? n_out : 0);
  m->out_coords = (mode == SPCONV_SUBM) ? d_in_coords : (mode == SPCONV_UP ? d_out_coords : b.qcoords);
  m->pin = b.pin;
  m->pout = b.pout;
  m->counts.assign(K3, 0);
  m->ptr.assign(K3 + 1, 0);
  auto done_empty = [&]() {
    *out_map = m;
    return SPCONV_OK;
  };
  if (n_in == 0 || n_src == 0) return done_empty();

  const int32_t* src_coords = (mode == SPCONV_UP) ? d_out_coords : d_in_coords;
  auto bail = [&](int code) {
    delete m;
    return code;
  };
  // key layout on the device (no host wait): bounds partials, then the layout,
  // computed by the source sort's first kernel when that is a tile histogram of the
  // coordinates, else by one workgroup of its own
  const KeyLayout* L = &b.cb->layout;
  LayoutArgs la{};
  const bool sort_first = !tu.hash && !tu.presorted;
  {
    PhaseScope ph(PH_BOUNDS, s);
    int np = 0;
    hipError_t e = launch_minmax(d_in_coords, n_in, d_out_coords, mode == SPCONV_UP ? n_out : 0, b.mm_partial,
                                 b.cb, &np, s);
    // builds that do not sort the keys digit by digit take any key width (up to 62
    // bits): no sort, or every sort by bucket
    const bool all_bucket = by_bucket && radix_bucket_applies(n_src) && (mode != SPCONV_UP || radix_bucket_applies(n_in));
    const int plan = (tu.hash || (tu.presorted && mode != SPCONV_DOWN) || all_bucket) ? 8 : passes;
    la = LayoutArgs{b.mm_partial, np, K, stride, tensor_stride, K3, plan, b.cb};
    if (e == hipSuccess && !sort_first) e = launch_layout(la, s);
    if (e != hipSuccess) return bail(hip_fail(e, "coordinate bounds"));
  }
  if (tu.hash) {
    PhaseScope ph(PH_HASH, s);
    hipError_t e = launch_hash_build(d_in_coords, n_in, L, b.hkeys, b.hvals, b.log2cap, b.skeys, b.sidx, &b.cb->err, s);
    if (e != hipSuccess) return bail(hip_fail(e, "hash build"));
  } else {
    PhaseScope ph(PH_SORT, s);
    // sorted inputs (a previous layer's outputs) only need their keys packed (Section 5.1.1)
    hipError_t e = tu.presorted ? launch_pack(src_coords, n_src, L, b.skeys, b.sidx, s)
                                : radix_sort_kv(src_coords, L, b.skeys, b.sidx, b.kalt, b.valt, n_src, passes, by_bucket,
                                                b.sort_tmp, &b.cb->err, &la, s);
    if (e == hipSuccess && mode == SPCONV_UP)
      e = tu.presorted ? launch_pack(d_in_coords, n_in, L, b.qkeys, b.qrow, s)
                       : radix_sort_kv(d_in_coords, L, b.qkeys, b.qrow, b.kalt, b.valt, n_in, passes, by_bucket,
                                       b.sort_tmp, &b.cb->err, nullptr, s);
    if (e != hipSuccess) return bail(hip_fail(e, "sort"));
  }
  if (mode == SPCONV_DOWN) {
    PhaseScope ph(PH_OUTCOORDS, s);
    const int64_t cell = (int64_t)tensor_stride * stride;
    hipError_t e = launch_down_keys(b.skeys, n_src, L, cell, b.dkeys, b.dvals, s);
    if (e == hipSuccess)
      e = radix_sort_kv(nullptr, L, b.dkeys, b.dvals, b.kalt, b.valt, n_src, passes, by_bucket, b.sort_tmp,
                        &b.cb->err, nullptr, s);
    if (e == hipSuccess)
      e = unique_keys(b.dkeys, n_src, L, b.flags, b.pos, b.scan_tmp, b.qkeys, b.qrow, b.qcoords, b.cb, s);
    if (e != hipSuccess) return bail(hip_fail(e, "output coordinates"));
  }

  SearchArgs a;
  std::memset(&a, 0, sizeof(a));
  a.skeys = b.skeys;
  a.sidx = b.sidx;
  a.n_src = n_src;
  a.qkeys = (mode == SPCONV_SUBM) ? b.skeys : b.qkeys;
  a.qrow = (mode == SPCONV_SUBM) ? b.sidx : b.qrow;
  a.n_q = nq_max;
  a.n_q_dev = (mode == SPCONV_DOWN) ? &b.cb->n_q : nullptr;
  a.K3 = K3;
  a.dk = b.cb->dk;
  a.B = tu.B;
  a.Cq = tu.Cq;
  a.wg = tu.wg;
  a.count_group = tu.count_group;
  // A table T_q far larger than the caches streams to memory: the write pass reads
  // it back from there either way, and left dirty in the caches it slowed the
  // write pass (LiDAR Map 2.75 -> 2.68 ms at 15.9M voxels, 0.790 -> 0.768 ms at
  // 4.07M; at 1.08M voxels, 117 MB of table, streaming lost 6 us).
  a.stream_tq = (int64_t)K3 * b.res_stride * (int64_t)sizeof(int32_t) >= ((int64_t)256 << 20) ? 1 : 0;
  a.swap_roles = (mode == SPCONV_UP) ? 1 : 0;
  a.check_q = (mode == SPCONV_UP) ? 1 : 0;
  a.res = b.res;
  a.res_stride = b.res_stride;
  a.ts = b.ts;
  a.ts_stride = b.ts_stride;
  a.sym = (mode == SPCONV_SUBM && K % 2 == 1) ? 1 : 0;
  a.write_ts = a.sym ? 0 : 1;
  a.pair_cap = (int64_t)K3 * nq_max;
  PubBuffer* pb = pub_buffer();
  if (!pb) return bail(fail(SPCONV_EHIP, "mapped host buffer allocation failed"));
  if (++pb->seq == 0) pb->seq = 1;
  a.pub = pb->dev;
  a.pub_seq = pb->seq;
  // work items (k, b): the sorted search's source blocks, or the hash-table
  // search's blocks of Cq queries; the passes split a query block into chunks of
  // at most Cq themselves, so the balancing step needs no scan of its own
  const int64_t nb = b.nb_items;
  {
    PhaseScope ph(PH_BACKWARD, s);
    hipError_t e = tu.hash ? launch_hash_items(K3, nq_max, tu.Cq, nb, b.bounds, s)
                           : launch_backward(a, nb, b.bounds, b.cb, s);
    if (e != hipSuccess) return bail(hip_fail(e, "backward search"));
  }
  if (!a.sym) {
    // sources without a partner at some offset: no query visits their entry
    PhaseScope ph(PH_METADATA, s);
    hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(b.ts), 0xFFFFFFFFu, (int64_t)K3 * b.ts_stride, s);
    if (e != hipSuccess) return bail(hip_fail(e, "metadata fill"));
  }
  {
    PhaseScope ph(PH_FORWARD, s);
    hipError_t e = tu.hash ? launch_hash_count(a, b.hkeys, b.hvals, b.log2cap, nb, b.item_cnt, s)
                           : launch_forward(a, false, b.bounds, nb, b.item_cnt, nullptr, b.pin, b.pout, b.cb, s);
    if (e == hipSuccess) e = scan_exclusive_u32(b.item_cnt, b.item_off, b.max_items, &b.cb->n_pairs, b.scan_tmp, s);
    if (e == hipSuccess)
      e = launch_forward(a, true, b.bounds, nb, b.item_cnt, b.item_off, b.pin, b.pout, b.cb, s);
    if (e != hipSuccess) return bail(hip_fail(e, "forward search"));
  }
  {
    // the head as the write pass published it (the pass may still be running)
    PhaseScope ph(PH_READBACK, s);
    bool ok = false;
    hipError_t e = pub_wait(pb, a.pub_seq, s, &ok);
    if (e != hipSuccess) return bail(hip_fail(e, "count read-back"));
    if (!ok) return bail(fail(SPCONV_EHIP, "the write pass did not publish its counts"));
    ControlBlock head;
    std::memcpy(&head, pb->host, kControlHeadBytes);
    const ControlBlock* hc = &head;
    if (hc->err & kErrRange)
      return bail(fail(SPCONV_ERANGE, "coordinate extent (plus kernel reach) needs more than 62 key bits"));
    if (hc->err & kErrBucket) {
      // a bucket too large for one workgroup: the caller redoes the build digit by digit
      *passes_needed = (hc->layout.total_bits + 7) / 8;
      *bucket_failed = true;
      return bail(SPCONV_OK);
    }
    if (hc->err & kErrWide) {
      // the key is wider than the sort planned for: the caller redoes the build
      *passes_needed = (hc->layout.total_bits + 7) / 8;
      return bail(SPCONV_OK);
    }
    *passes_needed = (hc->layout.total_bits + 7) / 8;
    if (hc->err & kErrDup) return bail(fail(SPCONV_EDUP, "duplicate coordinates"));
    if (hc->err & kErrOverflow) return bail(fail(SPCONV_EHIP, "overflow of the work items or of the hash table"));
    if (hc->err & kErrSpin) return bail(fail(SPCONV_EHIP, "a look-back exceeded its wait bound"));
    if (hc->err & kErrUnsorted)
      return bail(fail(SPCONV_EINVAL, "rows declared presorted are not in ascending (b, x, y, z) order"));
    if (mode == SPCONV_DOWN) m->n_out = hc->n_q;
    for (int k = 0; k < K3; ++k) {
      m->counts[k] = (int64_t)hc->seg_pair_start[k + 1] - hc->seg_pair_start[k];
      m->ptr[k + 1] = hc->seg_pair_start[k + 1];
    }
    if (m->ptr[K3] != hc->n_pairs) return bail(fail(SPCONV_EHIP, "pair count mismatch"));
  }
  // T_q is indexed by sorted query position, T_s by sorted source position.
  // Inputs are the sources except for a direct UP map, whose inputs are the
  // queries; presorted rows are their own sorted positions.
  // (hash-table maps index the inputs in caller order: no permutation)
  const uint32_t* src_perm = (tu.presorted || tu.hash) ? nullptr : b.sidx;
  const uint32_t* q_perm = (mode == SPCONV_SUBM) ? src_perm
                           : (mode == SPCONV_DOWN ? nullptr : (tu.presorted ? nullptr : b.qrow));
  if (mode == SPCONV_UP) {
    m->imt = b.res;
    m->imt_stride = b.res_stride;
    m->in_perm = q_perm;
    m->omt = b.ts;
    m->omt_stride = b.ts_stride;
    m->out_perm = src_perm;
  } else {
    m->imt = b.ts;
    m->imt_stride = b.ts_stride;
    m->in_perm = src_perm;
    m->omt = b.res;
    m->omt_stride = b.res_stride;
    m->out_perm = q_perm;
  }
  if (!a.write_ts) {
    m->imt_pending = true;
    m->seg_dev = b.cb->seg_pair_start;
    m->inv_scratch = b.valt;
  }
  *out_map = m;
  return SPCONV_OK;
}

}  // namespace

extern "C" {

int spconv_build_map(const int32_t* d_in_coords, int64_t n_in, const int32_t* d_out_coords, int64_t n_out, int K,
                     int stride, int tensor_stride, int mode, const spconv_options* opt, void* d_workspace,
                     size_t ws_bytes, void* stream, spconv_map** out_map) {
  PassHint& hint = g_pass_hint;
  const std::string key = pass_key(d_in_coords, n_in, d_out_coords, n_out, K, stride, tensor_stride, mode);
  const auto it = hint.by_input.find(key);
  SortPlan plan;
  if (it != hint.by_input.end())
    plan = it->second;
  else
    plan.passes = hint.last;
  int needed = 0, st = SPCONV_OK;
  // at most one redo for a too large bucket and one for a key wider than planned
  for (int attempt = 0; attempt < 3; ++attempt) {
    bool bucket_failed = false;
    st = build_map_impl(d_in_coords, n_in, d_out_coords, n_out, K, stride, tensor_stride, mode, opt, d_workspace,
                        ws_bytes, stream, out_map, plan.passes, plan.by_bucket, &needed, &bucket_failed);
    if (st != SPCONV_OK || *out_map) break;
    if (bucket_failed && plan.by_bucket) {
      plan.by_bucket = false;
      if (needed > plan.passes) plan.passes = needed;
    } else if (needed > plan.passes) {
      plan.passes = needed;
    } else {
      return fail(SPCONV_EHIP, "key layout changed between two builds");
    }
  }
  if (st == SPCONV_OK && !*out_map) return fail(SPCONV_EHIP, "map build did not settle on a sort plan");
  if (needed > 0) {
    if (hint.by_input.size() >= 256) hint.by_input.clear();
    plan.passes = needed;
    hint.by_input[key] = plan;
    hint.last = needed;
  }
  return st;
}

int spconv_map_transpose(const spconv_map* down, spconv_map** out_map) {
  if (!down || !out_map) return fail(SPCONV_EINVAL, "NULL argument");
  *out_map = nullptr;
  if (down->mode != SPCONV_DOWN) return fail(SPCONV_EINVAL, "only SPCONV_DOWN maps can be transposed");
  spconv_map* m = new (std::nothrow) spconv_map(*down);
  if (!m) return fail(SPCONV_EINVAL, "out of host memory");
  m->mode = SPCONV_UP;
  m->transposed = true;
  m->n_in = down->n_out;
  m->n_out = down->n_in;
  m->pin = down->pout;
  m->pout = down->pin;
  std::swap(m->imt, m->omt);
  std::swap(m->imt_stride, m->omt_stride);
  std::swap(m->in_perm, m->out_perm);
  m->out_coords = nullptr;  // the fine coordinates are the DOWN map's inputs (caller-owned)
  *out_map = m;
  return SPCONV_OK;
}

int64_t spconv_map_n_in(const spconv_map* m) { return m ? m->n_in : -1; }
int64_t spconv_map_n_out(const spconv_map* m) { return m ? m->n_out : -1; }
int spconv_map_kvol(const spconv_map* m) { return m ? m->K3 : -1; }
const int32_t* spconv_map_out_coords(const spconv_map* m) { return m ? m->out_coords : nullptr; }

int spconv_map_counts(const spconv_map* m, int64_t* h_counts) {
  if (!m || !h_counts) return fail(SPCONV_EINVAL, "NULL argument");
  for (int k = 0; k < m->K3; ++k) h_counts[k] = m->counts[k];
  return SPCONV_OK;
}

int spconv_map_pairs(const spconv_map* m, int k, const int32_t** d_in_idx, const int32_t** d_out_idx, int64_t* count) {
  if (!m || !d_in_idx || !d_out_idx || !count) return fail(SPCONV_EINVAL, "NULL argument");
  if (k < 0 || k >= m->K3) return fail(SPCONV_EINVAL, "offset index out of range");
  *d_in_idx = m->pin + m->ptr[k];
  *d_out_idx = m->pout + m->ptr[k];
  *count = m->counts[k];
  return SPCONV_OK;
}

int spconv_map_copy_pairs(const spconv_map* m, int32_t* d_in_idx, int32_t* d_out_idx, void* stream) {
  if (!m) return fail(SPCONV_EINVAL, "map is NULL");
  const int64_t n = m->ptr[m->K3];
  if (n == 0) return SPCONV_OK;
  if (!d_in_idx || !d_out_idx) return fail(SPCONV_EINVAL, "NULL destination");
  hipStream_t s = static_cast<hipStream_t>(stream);
  SPC_TRY(hipMemcpyAsync(d_in_idx, m->pin, (size_t)n * 4, hipMemcpyDeviceToDevice, s), "copy pairs");
  SPC_TRY(hipMemcpyAsync(d_out_idx, m->pout, (size_t)n * 4, hipMemcpyDeviceToDevice, s), "copy pairs");
  return SPCONV_OK;
}

int spconv_map_copy_out_coords(const spconv_map* m, int32_t* d_coords, void* stream) {
  if (!m) return fail(SPCONV_EINVAL, "map is NULL");
  if (m->n_out == 0) return SPCONV_OK;
  if (!d_coords) return fail(SPCONV_EINVAL, "NULL destination");
  if (!m->out_coords) return fail(SPCONV_EINVAL, "this map does not hold its output coordinates");
  SPC_TRY(hipMemcpyAsync(d_coords, m->out_coords, (size_t)m->n_out * 16, hipMemcpyDeviceToDevice,
                         static_cast<hipStream_t>(stream)),
          "copy coordinates");
  return SPCONV_OK;
}

void spconv_free_map(spconv_map* m) { delete m; }

size_t spconv_forward_workspace_bytes(const spconv_map* m, int c_in, int c_out, int dtype, const spconv_options* opt) {
  GmasPlan p;
  if (make_plan(m, c_in, c_out, dtype, opt, &p) != SPCONV_OK) return 0;
  FwdBufs b;
  return plan_forward_ws(nullptr, m, c_in, c_out, p, &b);
}

int spconv_forward_plan(const spconv_map* m, int c_in, int c_out, int dtype, const spconv_options* opt,
                        spconv_plan_info* info) {
  if (!info) return fail(SPCONV_EINVAL, "info is NULL");
  GmasPlan p;
  const int st = make_plan(m, c_in, c_out, dtype, opt, &p);
  if (st != SPCONV_OK) return st;
  info->rows_real = p.rows_real;
  info->rows_padded = p.rows_padded;
  info->n_gemm_launches = p.n_launches;
  info->t_gather = p.t_gather;
  info->t_scatter = p.t_scatter;
  info->grouping = p.grouping;
  info->gather = p.gather;
  info->centre = p.centre_k >= 0 ? 1 : 0;
  return SPCONV_OK;
}

int spconv_forward(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in, int c_out, int dtype,
                   const spconv_options* opt, void* d_workspace, size_t ws_bytes, void* stream) {
  return spconv_forward_ex(m, d_x, d_w, d_y, c_in, c_out, dtype, nullptr, 0, opt, d_workspace, ws_bytes, stream);
}

int spconv_concat_rows(const void* d_a, int c_a, const void* d_b, int c_b, void* d_out, int64_t n, int dtype,
                       void* stream) {
  if (dtype != SPCONV_F32 && dtype != SPCONV_F16 && dtype != SPCONV_BF16) return fail(SPCONV_EUNSUPPORTED, "dtype");
  const int e = elem_bytes(dtype);
  if (n < 0 || c_a < 0 || c_b < 0 || (c_a * e) % 16 != 0 || (c_b * e) % 16 != 0)
    return fail(SPCONV_EUNSUPPORTED, "concat needs 16-byte channel blocks");
  if (n == 0 || c_a + c_b == 0) return SPCONV_OK;
  if (!d_out || (c_a && !d_a) || (c_b && !d_b)) return fail(SPCONV_EINVAL, "NULL pointer");
  SPC_TRY(launch_concat(d_a, c_a, d_b, c_b, d_out, n, e, static_cast<hipStream_t>(stream)), "concat");
  return SPCONV_OK;
}

}  // extern "C"

namespace {

int forward_impl(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in, int c_out, int dtype,
                 const void* d_residual, int relu, const spconv_options* opt, void* d_workspace, size_t ws_bytes,
                 void* stream) {
  GmasPlan p;
  int st = make_plan(m, c_in, c_out, dtype, opt, &p);
  if (st != SPCONV_OK) return st;
  if (m->n_out > 0 && !d_y) return fail(SPCONV_EINVAL, "d_y is NULL");
  if (p.rows_pairs > 0 && (!d_x || !d_w)) return fail(SPCONV_EINVAL, "d_x / d_w is NULL");
  auto misaligned = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) != 0; };
  if (misaligned(d_x) || misaligned(d_w) || misaligned(d_y) || misaligned(d_residual))
    return fail(SPCONV_EINVAL, "d_x, d_w, d_y and d_residual must be 16-byte aligned");
  FwdBufs b;
  const size_t need = plan_forward_ws(nullptr, m, c_in, c_out, p, &b);
  if (need > 0 && (!d_workspace || ws_bytes < need)) return fail(SPCONV_ENOSPC, "forward workspace too small");
  if (reinterpret_cast<uintptr_t>(d_workspace) % 256 != 0) return fail(SPCONV_EINVAL, "workspace must be 256-byte aligned");
  plan_forward_ws(d_workspace, m, c_in, c_out, p, &b);
  if (m->n_out == 0) return SPCONV_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // a map without tables has no pairs: the scatter then writes zeros (plus the epilogue)
  const int K3 = m->omt ? m->K3 : 0;
  if (p.rows_pairs > 0) {
    const bool fused = p.gather == SPCONV_GATHER_FUSED;
    if (!fused && m->imt_pending) {
      PhaseScope ph(PH_METADATA, s);
      int32_t* ts = const_cast<int32_t*>(m->imt);
      SPC_TRY(launch_fill_u32(reinterpret_cast<uint32_t*>(ts), 0xFFFFFFFFu, (int64_t)m->K3 * m->imt_stride, s),
              "source-side table fill");
      SPC_TRY(launch_ts_from_pairs(m->pin, m->seg_dev, m->K3, m->ptr[m->K3], m->in_perm, m->n_in, m->inv_scratch, ts,
                                   m->imt_stride, s),
              "source-side table from the pairs");
      m->imt_pending = false;
    }
    if (!fused) {
      PhaseScope ph(PH_GATHER, s);
      SPC_TRY(launch_gather(d_x, m->n_in, c_in, p.elem, m->imt, m->imt_stride, m->in_perm, K3, b.buf_in, p.t_gather,
                            s),
              "gather");
    }
    {
      PhaseScope ph(PH_GEMM, s);
      if (b.wt) SPC_TRY(launch_transpose_w(d_w, b.wt, m->K3, c_in, c_out, s), "weight transpose");
      // fused: the A rows are the input rows of the pairs (pair r reads x[pin[r]])
      const void* a_src = fused ? d_x : b.buf_in;
      const int32_t* a_rows = fused ? m->pin : nullptr;
      const bool stream = (int64_t)p.rows_pairs * c_out * p.pelem >= kStreamPartialBytes;
      for (const auto& segs : p.launches)
        SPC_TRY(launch_gemm(segs.data(), (int)segs.size(), a_src, a_rows, d_w, b.wt, b.buf_out,
                            static_cast<char*>(b.buf_out) + (size_t)p.rows_pairs * c_out * p.pelem, c_in, c_out,
                            dtype, p.part_dtype, p.gemm_tile_rows, stream, s),
                "grouped GEMM");
    }
  }
  {
    PhaseScope ph(PH_SCATTER, s);
    const bool stream = m->n_out * c_out * p.elem >= kStreamOutputBytes;
    if (p.centre_k >= 0)
      SPC_TRY(launch_scatter_centre(d_x, m->out_perm, d_w, b.wt, p.centre_k, b.buf_out, m->omt, m->omt_stride, K3,
                                    d_y, d_residual, relu, m->n_out, c_in, c_out, dtype, p.part_dtype, stream, s),
              "scatter with the centre offset");
    else
      SPC_TRY(launch_scatter(b.buf_out, p.part_dtype, m->n_out, c_out, m->omt, m->omt_stride, m->out_perm, K3, d_y,
                             dtype, p.t_scatter, d_residual, relu, stream, s),
              "scatter");
  }
  return SPCONV_OK;
}

// Scratch of the allocation-free forward: device memory the library holds itself,
// one copy per GPU for the whole process.  In host code `scratch` names a host-side
// stand-in, so host code only ever uses the device address that hipGetSymbolAddress
// returns for the current device, kept per device below.
static __device__ __align__(256) unsigned char scratch[SPCONV_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
std::vector<void*> g_scratch_addr;  // by device ordinal; NULL until looked up

// The current device's address of `scratch`, looked up on the first call on that
// device (with it current) and kept.
int scratch_address(void** out) {
  int dev = 0;
  SPC_TRY(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (dev < 0) return fail(SPCONV_EHIP, "negative device ordinal");
  if ((size_t)dev >= g_scratch_addr.size()) g_scratch_addr.resize((size_t)dev + 1, nullptr);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    SPC_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "scratch address");
    if (!p) return fail(SPCONV_EHIP, "scratch address is NULL");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return SPCONV_OK;
}

}  // namespace

extern "C" {

int spconv_forward_ex(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in, int c_out,
                      int dtype, const void* d_residual, int relu, const spconv_options* opt, void* d_workspace,
                      size_t ws_bytes, void* stream) {
  return forward_impl(m, d_x, d_w, d_y, c_in, c_out, dtype, d_residual, relu, opt, d_workspace, ws_bytes, stream);
}

int spconv_forward_noalloc(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in, int c_out,
                           int dtype, const void* d_residual, int relu, const spconv_options* opt, void* stream) {
  GmasPlan p;
  int st = make_plan(m, c_in, c_out, dtype, opt, &p);
  if (st != SPCONV_OK) return st;
  FwdBufs b;
  const size_t need = plan_forward_ws(nullptr, m, c_in, c_out, p, &b);
  if (need > (size_t)SPCONV_NOALLOC_SCRATCH_BYTES)
    return fail(SPCONV_ENOSPC, "layer needs " + std::to_string(need) + " bytes of forward workspace; the "
                "allocation-free forward holds " + std::to_string((size_t)SPCONV_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  if ((st = scratch_address(&ws)) != SPCONV_OK) return st;
  return forward_impl(m, d_x, d_w, d_y, c_in, c_out, dtype, d_residual, relu, opt, ws,
                      (size_t)SPCONV_NOALLOC_SCRATCH_BYTES, stream);
}

// --------------------------------------------------------------- measurement
int spconv_profile_enable(uint64_t mask) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_mask = mask;
  return SPCONV_OK;
}

int spconv_profile_phase_count(void) { return PROF_IDS; }
const char* spconv_profile_phase_name(int i) { return prof_name(i); }

int spconv_profile_read(double* ms, int64_t* launches, int n, int reset) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!ms || !launches || n < PROF_IDS) return fail(SPCONV_EINVAL, "need spconv_profile_phase_count() entries");
  for (int i = 0; i < PROF_IDS; ++i) {
    ms[i] = 0.0;
    launches[i] = 0;
  }
  for (auto& r : g_recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess) return fail(SPCONV_EHIP, "event sync");
    if (hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) return fail(SPCONV_EHIP, "event elapsed");
    ms[r.phase] += t;
    launches[r.phase] += 1;
  }
  if (reset) {
    for (auto& r : g_recs) {
      g_pool.push_back(r.a);
      g_pool.push_back(r.b);
    }
    g_recs.clear();
  }
  return SPCONV_OK;
}

}  // extern "C"
