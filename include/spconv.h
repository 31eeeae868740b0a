/*
 * spconv.h -- C-ABI of the MI355X (gfx950) sparse-convolution layer library.
 *
 * A sparse convolution (Section 2.1, Eq. 1 and Eq. 2) runs in two steps
 * (Section 2.2): the Map step builds the kernel map (Eq. 3) and the
 * Gather-GEMM-Scatter (GMaS) step applies it to the features.
 *
 *   spconv_build_map   Map step: sorted coordinates, output coordinates (Eq. 1),
 *                      segmented query sorting (Section 5.1.1), the
 *                      double-traversed binary search (Section 5.1.2), and the
 *                      GMaS metadata tables (Section 2.2), written as the
 *                      search ranks its matches.
 *   spconv_forward     GMaS step: autotunable-tile Gather (Algorithm 1),
 *                      reordered and grouped per-offset GEMMs on MFMA
 *                      (Section 5.2.2) and Scatter (Section 2.2, Step 2).
 *   spconv_free_map    releases a map's host object.
 *
 * Conventions shared by every entry point:
 *   - Pointers named d_* are DEVICE pointers, h_* HOST pointers.  The caller owns
 *     and allocates every buffer, including both workspaces; the library never
 *     allocates device memory (the one device array it holds, the workspace of
 *     spconv_forward_noalloc, is set aside when the library is loaded).  `stream`
 *     is a hipStream_t (NULL = default stream).
 *   - Coordinates are int32 [n][4] rows (b, x, y, z); b is the batch index and is
 *     never offset.  Input coordinates must be unique (the paper's point cloud is
 *     a set, Section 2.1).
 *   - Weight offsets follow Delta(K, t) of Section 2.1: offset k = ix K^2 + iy K + iz
 *     (ix, iy, iz in [0, K)) is t * (ix - c, iy - c, iz - c) with c = (K-1)/2 for odd
 *     K and c = 0 for even K; t is the input coordinate spacing ("tensor stride").
 *   - Functions return SPCONV_OK (0) or a negative spconv_status; the message of
 *     the last failure on the calling thread is spconv_last_error().  Nothing
 *     aborts and no C++ exception crosses the ABI.
 */
#ifndef SPCONV_H
#define SPCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPCONV_OK = 0,
  SPCONV_EINVAL = -1,      /* bad argument (K <= 0, stride, mode, NULL pointer, ...) */
  SPCONV_ERANGE = -2,      /* coordinates (plus kernel reach) do not fit a 62-bit key */
  SPCONV_EDUP = -3,        /* repeated input (or, for SPCONV_UP, output) coordinate */
  SPCONV_ENOSPC = -4,      /* workspace smaller than the *_workspace_bytes() figure */
  SPCONV_EHIP = -5,        /* a HIP runtime call failed, or a device-side check did */
  SPCONV_EUNSUPPORTED = -6 /* dtype / channel count / kernel size not supported */
} spconv_status;

typedef enum {
  SPCONV_SUBM = 0, /* stride 1, outputs are the inputs, same rows (Section 2.1: s = 1 gives Q = P) */
  SPCONV_DOWN = 1, /* outputs Q = unique(floor(p / (t s)) (t s)) (Eq. 1), sorted by (b, x, y, z) */
  SPCONV_UP = 2    /* transposed (upsampling) conv: the DOWN map of the given fine outputs with
                      input and output roles swapped */
} spconv_mode;

typedef enum { SPCONV_F32 = 0, SPCONV_F16 = 1, SPCONV_BF16 = 2 } spconv_dtype;

typedef enum {
  SPCONV_GROUP_RAGGED = 0, /* one grouped launch over all offsets, no padding rows */
  SPCONV_GROUP_SORTED = 1, /* Section 5.2.2: offsets sorted by pair count, adjacent
                              ones grouped, each group padded to its largest member */
  SPCONV_GROUP_MAPORDER = 2 /* prior-art grouping in Map (offset) order, for comparison */
} spconv_grouping;

/* How the GEMMs get their A rows (Section 2.2, Step 2). */
typedef enum {
  SPCONV_GATHER_BUFFER = 1, /* Algorithm 1: a gather kernel copies each input row to the
                               per-pair buffer rows listed in the input metadata table */
  SPCONV_GATHER_FUSED = 2   /* the GEMM kernels load pair r's input row straight from the
                               features (its row index is the pair list's input index) */
} spconv_gather;

/* Tunables; any field left 0 takes its default.  The Map-step fields are the
 * hyperparameters of Section 5.1.4 (B = source-block size, C = query-block
 * limit); the GMaS fields are the Gather / Scatter tile sizes of Algorithm 1
 * (channels per thread) and the GEMM grouping of Section 5.2.2. */
typedef struct {
  int B;             /* source block size, power of two in [64, 4096] */
  int Cq;            /* query block limit (the paper's C): 256, 512, 1024 or 2048.  B, Cq and wg
                        all 0: 1024, 1024 and 256 below 2^18 source points, 4096, 2048 and 512
                        from there on; any of them given: the others default to 1024 / 1024 / 256 */
  int t_gather;      /* gather tile T in channels; must divide c_in; default: tuned rule */
  int t_scatter;     /* scatter tile T in channels; must divide c_out; default: tuned rule */
  int grouping;      /* spconv_grouping + 1 (0 = default SPCONV_GROUP_RAGGED) */
  int partial_dtype; /* GEMM partial (output buffer) precision: 1 = float32, 2 = layer dtype;
                        0 = default (layer dtype; sums are float32 either way) */
  int launch_cost_rows; /* grouping policy: one launch costs this many padded rows; default 32768 */
  int presorted;     /* spconv_build_map: 1 = the input rows are already unique and in ascending
                        (b, x, y, z) order (e.g. a DOWN map's outputs), so the sort is skipped
                        (Section 5.1.1); checked on the device (SPCONV_EINVAL if not sorted) */
  int search;        /* spconv_build_map, SPCONV_SUBM only: 0 = sorted arrays and the double-
                        traversed binary search (Section 5.1, default); 1 = a GPU hash table over
                        the input coordinates probed once per (output, offset), the prior-art
                        Map of Section 2.2 Step 1, kept as an ablation.  Same pairs (as sets),
                        listed in caller-row order within each offset */
  int gather;        /* spconv_forward: SPCONV_GATHER_BUFFER = Algorithm 1, input rows copied into a
                        per-pair buffer that the GEMMs read; SPCONV_GATHER_FUSED = the GEMMs load
                        each pair's input row directly (no buffer); 0 = default (fused).  Results
                        are bit-identical */
  int wg;            /* spconv_build_map: threads per workgroup of the forward search's count and
                        write passes (Section 5.1.4's thread-block size): 128, 256 or 512, and
                        Cq / wg must be 1, 2, 4 or 8 */
  int gemm_tile_rows; /* spconv_forward: output rows per GEMM workgroup tile, rounded up to the
                        kernel's rows per round (16 to 256); default 0 = about two tiles per
                        workgroup slot of the GPU, at least 512 rows */
  int centre;        /* spconv_forward, odd-K SPCONV_SUBM maps: 0 = default, the centre offset (which
                        pairs every output with its own input row) is multiplied inside the scatter
                        and the GEMMs skip it, where the layer allows (fused gather, 16-bit layer,
                        c_in % 8 == 0 and c_out % 32 == 0, both at most 256); 1 = off, the centre goes
                        through the GEMM and its partial buffer like every offset; 2 = on, and
                        SPCONV_EUNSUPPORTED where it does not apply.  The sums differ from the
                        unfused path only in rounding (the centre's product is not rounded to the
                        partial type) */
  int count_group;   /* spconv_build_map, sorted search (Section 5.1.2): offsets per workgroup
                        of the forward search's count pass, which stages a source block once for
                        all of them; 1 to 64 (more than K^3 acts as K^3, SPCONV_EINVAL outside
                        [0, 64]); 0 = default, sized so that the pass has about 4k workgroups.
                        Changes only the launch shape: the same map */
  int reserved[2];
} spconv_options;

typedef struct spconv_map spconv_map; /* opaque host-side object */

/* ---------------------------------------------------------------- Map step --
 * Device workspace needed by spconv_build_map for n_in input and (SPCONV_UP)
 * n_out fine output coordinates; for SPCONV_DOWN pass n_out = 0 (|Q| <= n_in).
 * The workspace holds the map's device arrays and must stay allocated, and not
 * be reused, until spconv_free_map() of this map (and of maps transposed from it).
 * Returns 0 for invalid arguments. */
size_t spconv_map_workspace_bytes(int64_t n_in, int64_t n_out, int K, int mode,
                                  const spconv_options* opt);

/* Builds the kernel map M = {(j, i, k)} of Eq. 3 (Section 2.2, Step 1) with
 * segmented query sorting and the double-traversed binary search (Section 5.1).
 *   d_in_coords  [n_in][4] int32 input coordinates, any row order, unique.
 *   d_out_coords SPCONV_UP only: [n_out][4] fine output coordinates; else NULL / 0.
 *   K            kernel size (1..5); K^3 offsets.
 *   stride       s of Eq. 1 (SPCONV_SUBM requires 1; SPCONV_DOWN / SPCONV_UP: >= 1).
 *   tensor_stride t: spacing of the input coordinates (SPCONV_UP: of the fine ones).
 *   opt          NULL or tunables (B, Cq).
 *   d_workspace  at least spconv_map_workspace_bytes(...) bytes, 256-byte aligned.
 * Pair indices are rows of the caller's arrays: input rows in the caller's order;
 * output rows in the caller's order for SUBM / UP and in sorted (b,x,y,z) order for
 * DOWN.  The map also holds the metadata tables of the GMaS step.  K^3 * max(n_in,
 * n_out) must stay below 2^31 (int32 pair indices; SPCONV_EUNSUPPORTED otherwise).
 * The key layout is computed on the device, so the host waits once, at the end
 * of the build, for the per-offset counts and error flags: the search's last
 * kernel publishes them into mapped host memory as it starts, and the build
 * returns while that kernel still writes the pair lists and tables.  Work on
 * `stream` (or after synchronising it) sees the complete map; other streams must
 * wait for `stream` first.  Up to 262,144 points the sort goes by bucket (the
 * key's top digit, then each bucket in one workgroup); a bucket of more than 8192
 * points is detected and the build redone digit by digit.  The host plans the
 * digit-by-digit sort's passes before the layout is known (from the previous build
 * of the same inputs); a key wider than planned is detected and the build redone.
 * Both choices are kept per input, so only a first build can cost two passes
 * over the Map.  An input is recognised by its device address, sizes and layer
 * arguments (the host never reads the coordinates): a different cloud later
 * placed at the same address (a caching allocator reuses addresses) inherits the
 * plan; a plan too short for it is detected and costs one redo, a longer one
 * runs its extra digit passes as copies.  While it waits for the counts the
 * calling thread spins for at most 2 ms, then blocks on the stream.
 * On success *out_map owns a host object to release with spconv_free_map(). */
int spconv_build_map(const int32_t* d_in_coords, int64_t n_in, const int32_t* d_out_coords,
                     int64_t n_out, int K, int stride, int tensor_stride, int mode,
                     const spconv_options* opt, void* d_workspace, size_t ws_bytes,
                     void* stream, spconv_map** out_map);

/* The transposed map of a SPCONV_DOWN map: pairs (j, i, k) become (i, j, k); no
 * device work.  The result borrows `down`'s device arrays: free it before `down`. */
int spconv_map_transpose(const spconv_map* down, spconv_map** out_map);

/* Sizes of the map: |P| input and |Q| output points (Section 2.1), and the number
 * of offsets of the stencil Delta(K, t), K^3 (Section 2.1). */
int64_t spconv_map_n_in(const spconv_map* m);
int64_t spconv_map_n_out(const spconv_map* m);
int spconv_map_kvol(const spconv_map* m); /* K^3 */
/* Device pointer to the [n_out][4] output coordinates Q: SPCONV_DOWN's sorted Q of
 * Eq. 1, SPCONV_SUBM's inputs (Q = P), SPCONV_UP's given fine coordinates. */
const int32_t* spconv_map_out_coords(const spconv_map* m);
/* h_counts[k] = |M_k| for k in [0, K^3): the size of offset k's part of the kernel
 * map M of Eq. 3 (Section 2.2, Step 1), from the host copy (no device work). */
int spconv_map_counts(const spconv_map* m, int64_t* h_counts);
/* Device pointers to offset k's pairs, M_k of Eq. 3 (Section 2.2, Step 1):
 * (*d_in_idx)[e] meets (*d_out_idx)[e] through W_k, e in [0, *count).  Order inside
 * one offset: ascending sorted query position (caller-row order for maps built with
 * the hash-table search).  The pointers stay valid until the map is freed. */
int spconv_map_pairs(const spconv_map* m, int k, const int32_t** d_in_idx,
                     const int32_t** d_out_idx, int64_t* count);
/* Stream-ordered copies into caller buffers: all pairs, offset-major (offset k's
 * list starts at sum_{k' < k} |M_k'|), into d_in_idx / d_out_idx of M entries;
 * and the [n_out][4] output coordinates into d_coords. */
int spconv_map_copy_pairs(const spconv_map* m, int32_t* d_in_idx, int32_t* d_out_idx, void* stream);
int spconv_map_copy_out_coords(const spconv_map* m, int32_t* d_coords, void* stream);
/* Releases the host object (the caller frees the device workspace). */
void spconv_free_map(spconv_map* m);

/* --------------------------------------------------------------- GMaS step --
 * Device workspace for spconv_forward with this map and these channel counts. */
size_t spconv_forward_workspace_bytes(const spconv_map* m, int c_in, int c_out, int dtype,
                                      const spconv_options* opt);

/* Gather-GEMM-Scatter (Section 2.2, Step 2; Section 5.2):
 *   y_i = sum_k sum_{(j,i) in M_k} x_j W_k       (Eq. 2)
 *   d_x [n_in][c_in], d_w [K^3][c_in][c_out] (W_k maps a c_in row vector to c_out),
 *   d_y [n_out][c_out], all row-major in `dtype`; d_y is fully overwritten (rows
 *   without pairs get zeros).  Products accumulate in float32.
 * Requirements: c_in, c_out in [1, 1024]; 16-byte rows (c * element size % 16 == 0)
 * and c_out % 16 == 0; d_x, d_w, d_y (and d_residual) 16-byte aligned, else
 * SPCONV_EINVAL.  Asynchronous on `stream`; no host synchronisation.
 * A SPCONV_SUBM map with odd K builds the input-side metadata table of Algorithm
 * 1's gather lazily: the first call that gathers through the table (gather =
 * SPCONV_GATHER_BUFFER) fills it from the pair lists on its `stream`, so calls on
 * other streams must be ordered after that one, and calls with the same map must
 * not run concurrently from several host threads.  The fused gather (the default)
 * reads the pair lists and never needs the table. */
int spconv_forward(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in,
                   int c_out, int dtype, const spconv_options* opt, void* d_workspace,
                   size_t ws_bytes, void* stream);

/* spconv_forward with an elementwise epilogue fused into the scatter's single
 * write: y = act(sum + residual).  d_residual: NULL or [n_out][c_out] in `dtype`
 * (may equal d_y); relu != 0 applies max(0, .) after the add.  For networks of
 * sparse-conv layers (residual blocks, ReLU after each conv). */
int spconv_forward_ex(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in,
                      int c_out, int dtype, const void* d_residual, int relu,
                      const spconv_options* opt, void* d_workspace, size_t ws_bytes, void* stream);

/* Maximum forward workspace of spconv_forward_noalloc (64 MiB). */
#define SPCONV_NOALLOC_SCRATCH_BYTES (64u << 20)

/* spconv_forward_ex for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the forward
 * workspace is a device array the library holds itself, one per GPU, of
 * SPCONV_NOALLOC_SCRATCH_BYTES, set aside when the library is loaded and kept until
 * the process ends.  The caller still owns d_x, d_w, d_y and d_residual (same
 * meaning, layout and alignment rules as spconv_forward_ex).  A layer whose
 * spconv_forward_workspace_bytes() exceeds the limit gets SPCONV_ENOSPC before any
 * device work.  The call allocates nothing and does not synchronise; the first call
 * on a device looks up that device's array address (a HIP symbol query).  Every
 * call on one GPU shares that GPU's array and nothing in it needs clearing between
 * calls, but calls whose work overlaps on one GPU (different streams, or several
 * host threads without ordering) race on it: order them on one stream. */
int spconv_forward_noalloc(const spconv_map* m, const void* d_x, const void* d_w, void* d_y, int c_in,
                           int c_out, int dtype, const void* d_residual, int relu, const spconv_options* opt,
                           void* stream);

/* Row-wise channel concatenation d_out[i] = [d_a[i] | d_b[i]] of [n][c_a] and
 * [n][c_b] in `dtype` (c * element size a multiple of 16 bytes); for the skip
 * connections of encoder-decoder networks.  Asynchronous on `stream`. */
int spconv_concat_rows(const void* d_a, int c_a, const void* d_b, int c_b, void* d_out, int64_t n,
                       int dtype, void* stream);

/* What spconv_forward will launch for this map (host-only): padded and real
 * buffer rows (padding overhead = (padded - real) / real, Section 3 figure on
 * GEMM reordering), number of GEMM launches, the tiles used and the gather form. */
typedef struct {
  int64_t rows_real;
  int64_t rows_padded;
  int n_gemm_launches;
  int t_gather;
  int t_scatter;
  int grouping;
  int gather; /* spconv_gather */
  int centre; /* 1: the centre offset is computed in the scatter (rows_* then leave out its rows) */
} spconv_plan_info;
int spconv_forward_plan(const spconv_map* m, int c_in, int c_out, int dtype,
                        const spconv_options* opt, spconv_plan_info* info);

/* ------------------------------------------------------------ measurement --
 * Event timing: for every id whose bit is set in `mask`, the library records HIP
 * events on the caller's stream around that phase of spconv_build_map /
 * spconv_forward (ids 0..10: bounds, sort, outcoords, backward, balance, forward,
 * readback, metadata (the table fill of maps other than odd-K submanifold ones),
 * gather, gemm, scatter) or around each launch of that kernel
 * (ids 16..39; spconv_profile_phase_name() gives the names, "" for unused ids).
 * mask = 0 turns timing off.  spconv_profile_read() waits for the recorded events
 * and writes the summed milliseconds and the number of timed intervals per id
 * into host arrays of at least spconv_profile_phase_count() entries; reset != 0
 * clears the record. */
int spconv_profile_enable(uint64_t mask);
int spconv_profile_phase_count(void);
const char* spconv_profile_phase_name(int i);
int spconv_profile_read(double* h_ms, int64_t* h_intervals, int n, int reset);

/* Thread-local message describing the last non-OK status. */
const char* spconv_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPCONV_H */
