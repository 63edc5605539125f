/*
 * fathom.h -- C ABI of libfathom, an MI355X (gfx950) implementation of the
 * per-query variable-depth key scan of "Fathom: Per-Query Read Depth for Sparse
 * Decoding over Offloaded KV Caches" (arXiv 2609.17652).
 *
 * Terms (Sec. 3.1 cost model, Sec. 3.2 store, Sec. 3.3 read depth):
 *   unit u   one (sequence, layer, KV head); U units per call, independent.
 *   n[u]     tokens cached for unit u.  nb_cap >= ceil(max_u n[u] / 64) is the
 *            common block stride of the store; blocks are 64 tokens.
 *   D        head dimension (channels).  This version supports D == 128.
 *   G        query heads per KV head (grouped-query attention), 1..8.  Query
 *            head h of unit u is row h of that unit's [G][D] query block.
 *
 * Conventions shared by every entry point:
 *   - All pointers to array data are DEVICE pointers unless stated otherwise.
 *     The caller allocates and owns every buffer; the library never allocates
 *     device memory and keeps no state between calls (the one exception is
 *     the device array behind fathom_scan_topk_noalloc, which holds nothing
 *     from one call to the next that a later call reads).
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream) and never synchronises the host.
 *   - Argument errors detectable on the host return an error status before
 *     anything is launched.  FATHOM_ERR_HIP reports a launch/runtime error.
 *   - Conditions found on the device are OR-ed into *dev_status (a device
 *     word; may be NULL).  The caller zeroes it and reads it after its own
 *     synchronisation.  Outputs whose inputs raised a device condition are
 *     defined as documented per bit below, not checked further.
 *   - Integer and index results (planes, scales, depths, top-k indices) are
 *     deterministic; floating-point results are computed in the fixed order
 *     stated per entry point, so repeated calls are bit-identical.
 */
#ifndef FATHOM_H
#define FATHOM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FATHOM_OK = 0,
  FATHOM_ERR_INVALID = -1,     /* null pointer, negative size, bad stride or alignment */
  FATHOM_ERR_UNSUPPORTED = -2, /* D != 128, G outside 1..8, k above FATHOM_MAX_K, unknown dtype */
  FATHOM_ERR_RANGE = -3,       /* budget outside [0, 4D] or r outside [0, D] */
  FATHOM_ERR_HIP = -4,         /* HIP launch or runtime error */
  FATHOM_ERR_WORKSPACE = -5    /* workspace missing or smaller than the *_workspace_size() */
} fathom_status;

typedef enum { FATHOM_F32 = 0, FATHOM_F16 = 1 } fathom_dtype;

typedef enum {
  FATHOM_WATERFILL = 0,   /* Sec. 3.3 Eq. (wf): graded depths under a bit budget B */
  FATHOM_UNIFORM_TOPR = 1 /* Sec. 2 (SparQ grouped rule): r channels at all 4 planes */
} fathom_mode;

#define FATHOM_MAX_K 8192 /* largest k accepted by the top-k entry points */

/* device status bits */
#define FATHOM_DEV_SCALE_OVERFLOW 1u /* a block absmax rounds to fp16 infinity; that block's codes are 8 */
#define FATHOM_DEV_NONFINITE 2u      /* NaN/Inf in K, q, var, g or scores (NaN keys take code 8; NaN scores rank last) */
#define FATHOM_DEV_TOPK_FALLBACK 4u  /* the fused filter under-collected and the exact unfiltered path ran */
#define FATHOM_DEV_TOPK_SHORT 8u     /* fewer than k eligible keys: trailing slots hold index -1, value NaN */
#define FATHOM_DEV_BAD_N 16u         /* n[u] < 0 or > 64 * nb_cap: that unit is treated as empty */

/*
 * fathom_pack -- Sec. 3.2, Eq. (2): per-channel 4-bit quantisation with one
 * fp16 scale per 64-token block, stored channel-major as bit planes.
 *
 * For unit u, block b (tokens 64b .. 64b+63 below n[u]) and channel j:
 *   a16 = fp16_rne(max |K| over the block's valid tokens), s = a16 / 8,
 *   c   = clip(floor(k / s), -8, 7) + 8 in [0, 16)  (exact real floor; c = 8
 *         when a16 == 0 or the key is NaN),
 *   planes[u][j][p][b] bit i = bit (3 - p) of c of token 64b + i  (p = 0 is
 *         the sign/most significant plane; bit i is token 64b + i),
 *   scales[u][j][b] = bit pattern of a16.
 * Pad bits (tokens >= n[u]) and blocks b >= ceil(n[u]/64) are written as 0,
 * so the first t planes of a channel are its exact t-bit quantiser.
 *
 *   K        [U][n][D] keys, element (u, i, c) at K[u*ld_unit + i*ld_tok + c];
 *            kdt FATHOM_F32 or FATHOM_F16 (converted to fp32 exactly).
 *            16-byte aligned; ld_tok >= D; ld_tok and ld_unit multiples of 16 bytes.
 *   n        [U] int64 (device): valid tokens per unit.
 *   planes   [U][D][4][nb_cap] uint64 (device, written).
 *   scales   [U][D][nb_cap] uint16 fp16 bits (device, written).
 * Device status: SCALE_OVERFLOW, NONFINITE, BAD_N.
 */
fathom_status fathom_pack(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                          const int64_t* n, int U, int D, int64_t nb_cap, uint64_t* planes,
                          uint16_t* scales, uint32_t* dev_status, void* stream);

/*
 * fathom_pack_append -- decode-time growth of a store built by fathom_pack
 * (Sec. 3.2, Eq. (2) applied to a growing cache).  Every unit grows from
 * n_old[u] to n[u] tokens.  A block's fp16 scale depends on all of its tokens,
 * so blocks floor(n_old/64) .. ceil(n/64)-1 are re-packed from K (the last
 * partial block together with the new tokens; only those rows are read).
 * Afterwards the store equals fathom_pack of the first n[u] tokens, bit for
 * bit, provided it held fathom_pack of the first n_old[u] (or earlier appends
 * reaching n_old[u]).  Blocks past ceil(n/64) are not written.
 *
 *   K, ld_tok, ld_unit, kdt, nb_cap, planes, scales: as fathom_pack; rows
 *            [64 floor(n_old/64), n) of each unit must hold its keys.
 *   n_old    [U] int64 (device): tokens already in the store.
 *   n        [U] int64 (device): tokens after the append.
 *   max_new  host bound on n[u] - n_old[u] over all units; sizes the launch.
 * Device status: BAD_N (n outside [0, 64 nb_cap], n_old outside [0, n], or
 * more new blocks than max_new allows: that unit is left unchanged),
 * SCALE_OVERFLOW, NONFINITE.
 */
fathom_status fathom_pack_append(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                 const int64_t* n_old, const int64_t* n, int64_t max_new, int U, int D,
                                 int64_t nb_cap, uint64_t* planes, uint16_t* scales, uint32_t* dev_status,
                                 void* stream);

/*
 * fathom_gather_store -- Sec. 3.6 (host-resident store): per decode step only
 * the bytes the depths read cross the host link.  For every unit u and channel
 * j with t = min(depths[u][j], 4) > 0, copies planes[u][j][0..t-1][*] (one
 * contiguous run) and scales[u][j][*] from the host store to the device store
 * of the same shape; other rows of the device store are not written.  A scan
 * over the device store then reads exactly what it would read from the full
 * store, so fathom_scan / fathom_scan_topk results are unchanged.
 *
 *   host_planes  [U][D][4][nb_cap] uint64, host_scales [U][D][nb_cap] uint16:
 *                pinned host memory (hipHostMalloc; torch pin_memory), the
 *                bases 16-byte aligned.  Other host memory: FATHOM_ERR_INVALID.
 *   depths       [U][D] uint8 (device).
 *   planes, scales  the device store (device, 16-byte aligned, written).
 * Device status: none.
 */
fathom_status fathom_gather_store(const uint64_t* host_planes, const uint16_t* host_scales,
                                  const uint8_t* depths, int U, int D, int64_t nb_cap,
                                  uint64_t* planes, uint16_t* scales, void* stream);

/*
 * fathom_alloc_depths -- Sec. 3.3, Eq. (g) and Eq. (wf): the per-query read
 * depth of every channel, shared by the G query heads of a unit.
 *
 * FATHOM_WATERFILL, budget B in [0, 4D] code bits per key:
 *   g_j = fl32(fl32(sum_h fl32(q_hj^2)) * var_j)   (heads ascending, no FMA)
 *   candidates c_{j,m} = g_j * 2^-(2m-1), m = 1..4, exact in fp64;
 *   theta* = the (B+1)-th largest candidate (0 when B >= 4D);
 *   depths[u][j] = #{m : c_{j,m} > theta*}.
 *   This is Eq. (wf) with round-half-up, clip to [0, 4], evaluated at any
 *   water line in (theta*, next candidate]: the smallest water line at which
 *   sum_j t_j <= B.  theta[u] = fp32(theta*).
 * FATHOM_UNIFORM_TOPR, r in [0, D]:
 *   w_j = fl32(sum_h |q_hj|) (heads ascending); the r channels first in
 *   (w desc, j asc) order get depth 4, all others 0; theta[u] = w of the r-th.
 *
 *   q        [U][G][D] queries, qdt FATHOM_F32 or FATHOM_F16, contiguous.
 *   var      [U][D] fp32 channel variances (calibration statistic), >= 0.
 *   depths   [U][D] uint8 (written).   theta  [U] fp32 (written) or NULL.
 * Device status: NONFINITE (non-finite or negative g / w).
 */
fathom_status fathom_alloc_depths(const void* q, fathom_dtype qdt, int U, int G, int D,
                                  const float* var, fathom_mode mode, int budget_or_r,
                                  uint8_t* depths, float* theta, uint32_t* dev_status,
                                  void* stream);

/*
 * fathom_scan -- Sec. 3.2-3.3: approximate scores from the first t_j planes
 * of every active channel (t_j = depths[u][j] > 0), for all G heads:
 *   s_h(i) = sum_{j: t_j > 0} q_hj * khat_ij,
 *   khat_ij = (c^(t) + 1/2 - 2^(t-1)) * a16 * 2^(1-t),  c^(t) = first t bits of c.
 * Raw q.khat, no 1/sqrt(D) (App. A).  Floating-point order, per (h, i),
 * channels ascending: khat is exact in fp32 (<= 16 significant bits) and
 * acc = fmaf(q_hj, khat, acc) from acc = +0 (q_hj converted to fp32 exactly).
 *
 *   planes, scales  the store written by fathom_pack.
 *   q        [U][G][D] (qdt), depths [U][D] (values above 4 are read as 4).
 *   scores   [U][G][ld_s] fp32 (written for i < min(n[u], ld_s) only).
 * Device status: BAD_N.
 */
fathom_status fathom_scan(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U,
                          int D, int64_t nb_cap, const void* q, fathom_dtype qdt, int G,
                          const uint8_t* depths, float* scores, int64_t ld_s,
                          uint32_t* dev_status, void* stream);

/*
 * fathom_topk -- Sec. 2 (top-k decoding): per query head, the k indices with
 * the largest scores among the eligible positions [lo, n[u] - tail), ordered
 * by (score desc, index asc); -0.0 ranks equal to +0.0 and NaN below every
 * number.  The paper's protocol keeps the first 4 and last 32 tokens
 * unconditionally (lo = 4, tail = 32) and selects the remaining k - 36.
 *
 *   scores   [U][G][ld_s] fp32.     idx [U][G][k] int32 (written).
 *   val      [U][G][k] fp32 (written: the selected scores) or NULL.
 *   ws       device workspace of at least fathom_topk_workspace_size(U, G, max_n, k) bytes.
 * Device status: NONFINITE, TOPK_SHORT, BAD_N.
 */
fathom_status fathom_topk(const float* scores, int64_t ld_s, const int64_t* n, int U, int G,
                          int k, int64_t lo, int64_t tail, int32_t* idx, float* val, void* ws,
                          size_t ws_bytes, uint32_t* dev_status, void* stream);
size_t fathom_topk_workspace_size(int U, int G, int64_t max_n, int k);

/*
 * fathom_scan_topk -- fathom_scan followed by fathom_topk in one call, with
 * the same outputs bit for bit (same scores, same order rules), without the
 * score array as an output.  This is the decode-step scan.
 *   ws       device workspace of at least
 *            fathom_scan_topk_workspace_size(U, G, max_n, k) bytes (any
 *            contents: every call sets the state it reads).
 * The filter that spares most keys their exact score serves units of at most
 * 4 query heads per KV head; with G > 4 every row takes the exact path (the
 * same outputs; TOPK_FALLBACK is raised).
 * Device status: NONFINITE, TOPK_SHORT, TOPK_FALLBACK, BAD_N.
 */
fathom_status fathom_scan_topk(const uint64_t* planes, const uint16_t* scales, const int64_t* n,
                               int U, int D, int64_t nb_cap, const void* q, fathom_dtype qdt,
                               int G, const uint8_t* depths, int k, int64_t lo, int64_t tail,
                               int32_t* idx, float* val, void* ws, size_t ws_bytes,
                               uint32_t* dev_status, void* stream);
size_t fathom_scan_topk_workspace_size(int U, int G, int64_t max_n, int k);

/*
 * fathom_scan_topk_ex -- fathom_scan_topk with a caller's bound on the depth
 * bits of every unit, max_unit_bits >= sum_j min(depths[u][j], 4) for all u
 * (0: no bound).  The outputs are those of fathom_scan_topk for any bound;
 * the bound only selects work: with max_unit_bits <= 80 the filter pass for
 * units of more bits is not launched, so a unit that exceeds a wrong bound is
 * recomputed by the exact path (TOPK_FALLBACK); with 64 < max_unit_bits <= 80
 * the filter is instantiated for units of up to 80 bits, which otherwise take
 * the wider filter pass.
 * Water-filling at budget B (Sec. 3.3) gives every unit at most B bits.
 * Errors: as fathom_scan_topk; max_unit_bits < 0 is FATHOM_ERR_INVALID.
 */
fathom_status fathom_scan_topk_ex(const uint64_t* planes, const uint16_t* scales, const int64_t* n,
                                  int U, int D, int64_t nb_cap, const void* q, fathom_dtype qdt,
                                  int G, const uint8_t* depths, int k, int64_t lo, int64_t tail,
                                  int max_unit_bits, int32_t* idx, float* val, void* ws,
                                  size_t ws_bytes, uint32_t* dev_status, void* stream);

/*
 * fathom_scan_topk_noalloc -- fathom_scan_topk_ex for callers that cannot
 * allocate or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  Same arguments and outputs as
 * fathom_scan_topk_ex (bit for bit) minus ws / ws_bytes: the workspace is a
 * device array inside the library, fathom_scan_topk_noalloc_capacity() bytes
 * per device, loaded with the library and held until the process ends.  The
 * call itself allocates nothing.
 *   - A shape whose fathom_scan_topk_workspace_size(U, G, 64 * nb_cap, k)
 *     exceeds the capacity returns FATHOM_ERR_WORKSPACE before any launch.
 *   - Every call on one device uses that device's one array, and each call's
 *     kernels clear what they need from it.  Calls that overlap on one device
 *     (different streams or threads without ordering between them) race on
 *     it and give undefined results; calls ordered on one stream are safe.
 * Errors: as fathom_scan_topk_ex, plus FATHOM_ERR_HIP if the array's device
 * address cannot be obtained.
 */
fathom_status fathom_scan_topk_noalloc(const uint64_t* planes, const uint16_t* scales, const int64_t* n,
                                       int U, int D, int64_t nb_cap, const void* q, fathom_dtype qdt,
                                       int G, const uint8_t* depths, int k, int64_t lo, int64_t tail,
                                       int max_unit_bits, int32_t* idx, float* val,
                                       uint32_t* dev_status, void* stream);
size_t fathom_scan_topk_noalloc_capacity(void);

/*
 * fathom_sparse_attn -- Sec. 2 (top-k decoding) and Sec. 4 (fidelity metric):
 * exact attention of each query head over its selected set
 *   S_h = sink [0, ns) U local [l0, n) U {idx[u][h][r] in [ns, l0)},
 *   ns = min(n_sink, n[u]),  l0 = max(ns, n[u] - n_local);
 * index entries outside [ns, l0) (including -1) are skipped, so S_h has no
 * duplicates when idx does not.
 *   out_h = sum_{i in S_h} softmax_i(sm_scale * q_h . K_i) V_i,  fp32 arithmetic
 *   (the set is processed in chunks whose softmax partials are combined).
 *
 *   q        [U][G][D] (qdt).
 *   Krows, Vrows  [U][n][D] fp16 rows, element (u, i, c) at [u*ld_unit + i*ld_tok + c];
 *            4-byte aligned; ld_tok >= D; ld_tok, ld_unit even.
 *   idx      [U][G][k] int32 (k may be 0; idx may then be NULL).
 *   out      [U][G][D] fp32 (written; 0 for an empty set).
 *   ws       device workspace of at least
 *            fathom_sparse_attn_workspace_size(U, G, k, n_sink, n_local) bytes, 256-byte aligned.
 * Device status: BAD_N (nb_cap is not known here: only n[u] < 0 is flagged).
 */
fathom_status fathom_sparse_attn(const void* q, fathom_dtype qdt, const uint16_t* Krows,
                                 const uint16_t* Vrows, int64_t ld_tok, int64_t ld_unit,
                                 const int64_t* n, int U, int G, int D, const int32_t* idx, int k,
                                 int n_sink, int n_local, float sm_scale, float* out, void* ws,
                                 size_t ws_bytes, uint32_t* dev_status, void* stream);
size_t fathom_sparse_attn_workspace_size(int U, int G, int k, int n_sink, int n_local);

/*
 * KLT-rotated store -- Sec. 3.5 (basis rule).  The rotated variant of the
 * method stores the planes of (k - mu) V instead of k, with mu the mean and V
 * the orthonormal eigenbasis of the covariance of a unit's calibration keys,
 * and allocates depths with g_j = sum_h ((q_h V)_j)^2 lambda_j, lambda_j the
 * eigenvalue of column j.  Nothing else changes: pack the rotated keys with
 * fathom_pack (fp32), pass the rotated queries and var = lambda to
 * fathom_alloc_depths, and the rotated queries to the scan.  Scores are then
 * q . (k - mu): per head they differ from q . k by the constant q . mu, so the
 * top-k order is that of q . k (up to the quantisation).
 *
 * fathom_klt_calibrate -- per unit: mu = mean of its n[u] keys, covariance
 * C = (1/n) sum (k - mu)(k - mu)^T (fp64 sums), and its eigen-decomposition
 * (fp32 cyclic Jacobi, 12 sweeps).  Columns are ordered by eigenvalue,
 * largest first (the paper orders by calibration score variance, the same
 * order for isotropic queries); each column's largest-magnitude entry is
 * positive.  A unit with n[u] = 0 gets mu = 0, V = I, lambda = 0.
 *   K        [U][n][D] keys (kdt), element (u, i, c) at K[u*ld_unit + i*ld_tok + c];
 *            ld_tok >= D, ld_unit >= 0; element-aligned.
 *   n        [U] int64 (device), 0 <= n[u] <= n_cap, else BAD_N and the unit is empty.
 *   mu       [U][D] fp32, V [U][D][D] fp32 (V[u][j][c]: entry j of eigenvector c),
 *   lam      [U][D] fp32 -- written.
 *   ws       device workspace of fathom_klt_calibrate_workspace_size(U) bytes,
 *            256-byte aligned (chunk partial sums; contents on entry unused).
 * One-time per store (prefill); about 4 MiB of workspace per unit.
 */
fathom_status fathom_klt_calibrate(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                   const int64_t* n, int64_t n_cap, int U, int D, float* mu, float* V,
                                   float* lam, void* ws, size_t ws_bytes, uint32_t* dev_status, void* stream);
size_t fathom_klt_calibrate_workspace_size(int U);

/*
 * fathom_klt_rotate_keys -- the stored coordinates (k - mu) V of every key,
 * fp32, in a fixed order: d_j = fl(k_j - mu_j); for j = 0 .. D-1,
 * acc_c = fl(acc_c + fl(d_j * V[j][c])) from acc_c = +0 (no fused multiply-add).
 *   K, ld_tok, ld_unit, n, n_cap   as fathom_klt_calibrate.
 *   mu [U][D], V [U][D][D] fp32    (from fathom_klt_calibrate or the caller).
 *   out      [U] blocks of ld_out_unit floats (ld_out_unit >= n_cap * D): row i of
 *            unit u at out[u*ld_out_unit + i*D]; rows i < n[u] are written, the
 *            rest left as they were.  Pack it with fathom_pack (FATHOM_F32,
 *            ld_tok = D, ld_unit = ld_out_unit).
 * Device status: BAD_N.
 */
fathom_status fathom_klt_rotate_keys(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                     const int64_t* n, int64_t n_cap, int U, int D, const float* mu,
                                     const float* V, float* out, int64_t ld_out_unit, uint32_t* dev_status,
                                     void* stream);

/*
 * fathom_klt_rotate_q -- q_h V per (unit, head), fp32 [U][G][D], in the order of
 * fathom_klt_rotate_keys (no mean).  q [U][G][D] (qdt), V [U][D][D] fp32,
 * 16-byte aligned.  Runs once per decode step, before fathom_alloc_depths.
 */
fathom_status fathom_klt_rotate_q(const void* q, fathom_dtype qdt, int U, int G, int D, const float* V,
                                  float* out, void* stream);

/* Human-readable name of a status code (static storage). */
const char* fathom_status_string(fathom_status s);

/* Library version string, e.g. "fathom-mi355x 0.1 gfx950" (static storage). */
const char* fathom_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FATHOM_H */
