// CPU ORACLE for the sparse-convolution layer -- TEST INFRASTRUCTURE ONLY.
//
// Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
// load or call this library.  The product (the HIP library) never does, and the
// two share no code: no headers, helpers, tables or key layouts.
//
// What it computes is the plain definition of a sparse convolution, written out
// directly (Section 2.1, Eq. 1 and Eq. 2; Section 2.2, Eq. 3):
//   * weight offsets  Delta(K, t)                     -- Section 2.1, text after Eq. 2
//   * output coordinates Q = unique(floor(p/(t s)) (t s)) -- Eq. 1
//   * kernel map M = {(j, i, k) : p_j = q_i + delta_k}  -- Eq. 3, built with a
//     hash table over the input coordinates exactly as the prior-art Map step of
//     Section 2.2 (Step 1) describes
//   * features  y_i = sum_k sum_{(j,i) in M_k} x_j W_k  -- Eq. 2, in float64, summed
//     in the fixed order k ascending, then input channel ascending.
//
// Readings where the paper is silent (they are listed with the design notes):
//   * the offset scale is the input coordinate spacing t ("tensor stride"); for
//     odd K offsets are centred, for even K they run 0..K-1 (times t);
//   * offsets are enumerated x-major: k = ix K^2 + iy K + iz, so the first offset
//     of Delta(5,2) is (-4,-4,-4) as the paper states;
//   * the batch index b is never offset;
//   * transposed (upsampling) maps: pair (j coarse, i fine) in M_k iff
//     fine_i = coarse_j + delta_k (the downsampling map with roles swapped);
//   * input coordinates form a set: duplicates are rejected.
//
// Parity pins for every function live in the CPU test suite (dense conv3d on
// tiny grids, brute-force all-pairs maps, kernel-map invariants, hand examples,
// the paper's own worked examples).  Nothing here is unpinned.
#include <algorithm>
#include <array>
#include <cstdint>
#include <cstring>
#include <unordered_map>
#include <vector>
#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_EDUP = -3, ORC_ENOSPC = -4 };
enum { MODE_SUBM = 0, MODE_DOWN = 1, MODE_UP = 2 };

struct Coord {
  int64_t b, x, y, z;
  bool operator==(const Coord& o) const { return b == o.b && x == o.x && y == o.y && z == o.z; }
};

struct CoordHash {
  size_t operator()(const Coord& c) const {
    // Any deterministic mixing works; this one is splitmix64 applied field by field.
    uint64_t h = 0x9E3779B97F4A7C15ull;
    const int64_t f[4] = {c.b, c.x, c.y, c.z};
    for (int i = 0; i < 4; ++i) {
      uint64_t v = (uint64_t)f[i] + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
      v ^= v >> 30; v *= 0xBF58476D1CE4E5B9ull;
      v ^= v >> 27; v *= 0x94D049BB133111EBull;
      v ^= v >> 31;
      h ^= v;
    }
    return (size_t)h;
  }
};

Coord coord_at(const int32_t* c, int64_t row) {
  return Coord{c[4 * row + 0], c[4 * row + 1], c[4 * row + 2], c[4 * row + 3]};
}

// Mathematical floor of a / g for g > 0 (also for negative a).
int64_t floor_div(int64_t a, int64_t g) {
  int64_t q = a / g;
  if (a % g != 0 && a < 0) q -= 1;
  return q;
}

// Delta(K, t) in the canonical order k = ix K^2 + iy K + iz.
std::vector<std::array<int64_t, 3>> make_offsets(int K, int t) {
  const int c = (K % 2 == 1) ? (K - 1) / 2 : 0;
  std::vector<std::array<int64_t, 3>> d;
  for (int ix = 0; ix < K; ++ix)
    for (int iy = 0; iy < K; ++iy)
      for (int iz = 0; iz < K; ++iz)
        d.push_back({(int64_t)t * (ix - c), (int64_t)t * (iy - c), (int64_t)t * (iz - c)});
  return d;
}

}  // namespace

extern "C" {

// Weight offsets Delta(K, t), written as int32 [K^3][3] (dx, dy, dz).  Returns K^3.
int orc_offsets(int K, int t, int32_t* out) {
  if (K <= 0 || t <= 0 || out == nullptr) return ORC_EINVAL;
  std::vector<std::array<int64_t, 3>> d = make_offsets(K, t);
  for (size_t k = 0; k < d.size(); ++k)
    for (int a = 0; a < 3; ++a) out[3 * k + a] = (int32_t)d[k][a];
  return (int)d.size();
}

// Eq. 1: Q = { (b, floor(x/g) g, floor(y/g) g, floor(z/g) g) : p in P } with g = t s,
// duplicates removed, sorted lexicographically by signed (b, x, y, z).
// `out` must hold n rows.  Returns |Q| or a negative status.
int64_t orc_out_coords(const int32_t* in, int64_t n, int s, int t, int32_t* out) {
  if (n < 0 || s <= 0 || t <= 0 || (n > 0 && (in == nullptr || out == nullptr))) return ORC_EINVAL;
  const int64_t g = (int64_t)t * s;
  std::vector<std::array<int64_t, 4>> q((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    Coord p = coord_at(in, i);
    q[i] = {p.b, floor_div(p.x, g) * g, floor_div(p.y, g) * g, floor_div(p.z, g) * g};
  }
  std::sort(q.begin(), q.end());
  q.erase(std::unique(q.begin(), q.end()), q.end());
  for (size_t i = 0; i < q.size(); ++i)
    for (int a = 0; a < 4; ++a) out[4 * i + a] = (int32_t)q[i][a];
  return (int64_t)q.size();
}

// Eq. 3 kernel map, built with a hash table over the input coordinates.
//   SUBM: outputs are the inputs (out_c ignored, n_out must equal n_in);
//   DOWN: outputs are out_c (normally orc_out_coords' result);
//   UP:   inputs are the coarse coordinates, outputs the fine out_c; pair (j, i)
//         in M_k iff fine_i - delta_k = coarse_j.
// Pairs are written grouped by offset k (ascending), and inside one offset by
// ascending output row.  counts[k] = |M_k|.  Returns the total number of pairs,
// or a negative status (EDUP for repeated input / output coordinates, ENOSPC if
// more than `cap` pairs exist).
int64_t orc_kernel_map(const int32_t* in_c, int64_t n_in, const int32_t* out_c, int64_t n_out,
                       int K, int t, int mode, int64_t* counts, int32_t* pin, int32_t* pout,
                       int64_t cap) {
  if (K <= 0 || t <= 0 || n_in < 0 || n_out < 0 || counts == nullptr) return ORC_EINVAL;
  if (mode != MODE_SUBM && mode != MODE_DOWN && mode != MODE_UP) return ORC_EINVAL;
  if (mode == MODE_SUBM) {
    out_c = in_c;
    if (n_out != n_in) return ORC_EINVAL;
  }
  if ((n_in > 0 && in_c == nullptr) || (n_out > 0 && out_c == nullptr)) return ORC_EINVAL;
  const std::vector<std::array<int64_t, 3>> d = make_offsets(K, t);
  const int K3 = (int)d.size();

  // Hash table: input coordinate -> input row (Section 2.2, Step 1).
  std::unordered_map<Coord, int64_t, CoordHash> H;
  H.reserve((size_t)n_in * 2 + 1);
  for (int64_t j = 0; j < n_in; ++j)
    if (!H.emplace(coord_at(in_c, j), j).second) return ORC_EDUP;
  if (mode != MODE_SUBM) {
    std::unordered_map<Coord, int64_t, CoordHash> seen;
    seen.reserve((size_t)n_out * 2 + 1);
    for (int64_t i = 0; i < n_out; ++i)
      if (!seen.emplace(coord_at(out_c, i), i).second) return ORC_EDUP;
  }

  int64_t total = 0;
  for (int k = 0; k < K3; ++k) {
    int64_t cnt = 0;
    for (int64_t i = 0; i < n_out; ++i) {
      Coord q = coord_at(out_c, i);
      Coord p;
      if (mode == MODE_UP)  // the coarse input that fine output q receives through delta_k
        p = Coord{q.b, q.x - d[k][0], q.y - d[k][1], q.z - d[k][2]};
      else                  // the candidate input q + delta_k (Section 2.2, the query)
        p = Coord{q.b, q.x + d[k][0], q.y + d[k][1], q.z + d[k][2]};
      auto it = H.find(p);
      if (it == H.end()) continue;
      if (total < cap) {
        pin[total] = (int32_t)it->second;
        pout[total] = (int32_t)i;
      }
      ++total;
      ++cnt;
    }
    counts[k] = cnt;
  }
  if (total > cap) return ORC_ENOSPC;
  return total;
}

// Eq. 2 in float64: y[r] = sum_k sum_{(j, rows[r]) in M_k} x_j W_k for each
// requested output row (rows == NULL means all rows 0..n_out-1, n_rows = n_out).
// x: [n_in][cin], w: [K3][cin][cout] (W_k maps a row vector of cin to cout),
// y: [n_rows][cout].  For every output element the sum runs over k ascending,
// then input channel ascending.  OpenMP splits work by output row only, so the
// result does not depend on the thread count.
int orc_features(const double* x, int64_t n_in, int cin, const double* w, int cout, int K3,
                 const int64_t* counts, const int32_t* pin, const int32_t* pout,
                 int64_t n_out, const int64_t* rows, int64_t n_rows, double* y, int nthreads) {
  if (cin <= 0 || cout <= 0 || K3 <= 0 || n_in < 0 || n_out < 0 || n_rows < 0) return ORC_EINVAL;
  // Per output row and offset, the single input row that meets it (or -1).
  std::vector<int64_t> nbr((size_t)n_out * K3, -1);
  int64_t m = 0;
  for (int k = 0; k < K3; ++k) {
    for (int64_t e = 0; e < counts[k]; ++e, ++m) {
      const int64_t j = pin[m], i = pout[m];
      if (j < 0 || j >= n_in || i < 0 || i >= n_out) return ORC_EINVAL;
      if (nbr[(size_t)i * K3 + k] != -1) return ORC_EDUP;  // at most one input per (q_i, delta_k)
      nbr[(size_t)i * K3 + k] = j;
    }
  }
  for (int64_t r = 0; r < n_rows; ++r)
    if (rows && (rows[r] < 0 || rows[r] >= n_out)) return ORC_EINVAL;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 64)
#endif
  for (int64_t r = 0; r < n_rows; ++r) {
    const int64_t i = rows ? rows[r] : r;
    double* yr = y + (size_t)r * cout;
    for (int co = 0; co < cout; ++co) yr[co] = 0.0;
    for (int k = 0; k < K3; ++k) {
      const int64_t j = nbr[(size_t)i * K3 + k];
      if (j < 0) continue;
      const double* xj = x + (size_t)j * cin;
      const double* wk = w + (size_t)k * cin * cout;
      for (int ci = 0; ci < cin; ++ci) {
        const double xv = xj[ci];
        const double* wrow = wk + (size_t)ci * cout;
        for (int co = 0; co < cout; ++co) yr[co] += xv * wrow[co];
      }
    }
  }
  return ORC_OK;
}

int orc_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

}  // extern "C"
