// C ABI of libfathom: host-side argument checks, then asynchronous launches.
// Declarations and the meaning of every argument are in include/fathom.h.
#include "common.hpp"

namespace fathom {
fathom_status launch_gather(const uint64_t*, const uint16_t*, const uint8_t*, int, int64_t, uint64_t*, uint16_t*,
                            hipStream_t);
fathom_status launch_pack(const void*, fathom_dtype, int64_t, int64_t, const int64_t*, const int64_t*, int64_t, int,
                          int64_t, uint64_t*, uint16_t*, uint32_t*, hipStream_t);
fathom_status launch_alloc(const void*, fathom_dtype, int, int, const float*, fathom_mode, int, uint8_t*, float*,
                           uint32_t*, hipStream_t);
fathom_status launch_scan(const uint64_t*, const uint16_t*, const int64_t*, int, int64_t, const void*,
                          fathom_dtype, int, const uint8_t*, float*, int64_t, uint32_t*, hipStream_t);
fathom_status launch_topk(const float*, int64_t, const int64_t*, int, int, int, int64_t, int64_t, int32_t*, float*,
                          void*, uint32_t*, hipStream_t);
fathom_status launch_sparse_attn(const void*, fathom_dtype, const uint16_t*, const uint16_t*, int64_t, int64_t,
                                 const int64_t*, int, int, const int32_t*, int, int, int, float, float*, void*,
                                 uint32_t*, hipStream_t);
size_t attn_ws_bytes(int U, int G, int k, int n_sink, int n_local);
size_t topk_ws_bytes(int R, int64_t max_n, int k);
size_t fused_ws_bytes(int R, int U, int64_t nb_cap, int k);
fathom_status launch_scan_topk_fused(const uint64_t*, const uint16_t*, const int64_t*, int, int64_t, const void*,
                                     fathom_dtype, int, const uint8_t*, int, int64_t, int64_t, int, int32_t*, float*,
                                     void*, uint32_t*, hipStream_t);
int attn_max_sink_local();
size_t scratch_capacity();
fathom_status scratch_address(void** out);
size_t klt_ws_bytes(int U);
fathom_status launch_klt_calibrate(const void*, fathom_dtype, int64_t, int64_t, const int64_t*, int64_t, int, float*,
                                   float*, float*, void*, uint32_t*, hipStream_t);
fathom_status launch_klt_rotate_keys(const void*, fathom_dtype, int64_t, int64_t, const int64_t*, int64_t, int,
                                     const float*, const float*, float*, int64_t, uint32_t*, hipStream_t);
fathom_status launch_klt_rotate_q(const void*, fathom_dtype, int, int, const float*, float*, hipStream_t);
}  // namespace fathom

using namespace fathom;

namespace {

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
inline bool dtype_ok(fathom_dtype t) { return t == FATHOM_F32 || t == FATHOM_F16; }
inline size_t dtype_size(fathom_dtype t) { return t == FATHOM_F32 ? 4 : 2; }
inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }

// common shape checks for the store-reading calls
fathom_status check_store(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int D,
                          int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths) {
  if (U < 0 || nb_cap < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (G < 1 || G > kMaxG || !dtype_ok(qdt)) return FATHOM_ERR_UNSUPPORTED;
  if (nb_cap > ((int64_t)1 << 25)) return FATHOM_ERR_UNSUPPORTED;  // 2^31 tokens per unit
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  if (!planes || !scales || !n || !q || !depths) return FATHOM_ERR_INVALID;
  if (!aligned(planes, 8) || !aligned(scales, 2) || !aligned(n, 8) || !aligned(q, dtype_size(qdt)))
    return FATHOM_ERR_INVALID;
  return FATHOM_OK;
}

size_t scan_topk_ws(int U, int G, int64_t max_n, int k) {
  const int64_t nb = (max_n + 63) / 64;
  return fused_ws_bytes(U * G, U, nb > 0 ? nb : 1, k);
}

}  // namespace

extern "C" {

// KLT-rotated store (Sec. 3.5): keys as in fathom_pack, read element by element.
static fathom_status check_klt_keys(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                    const int64_t* n, int64_t n_cap, int U, int D) {
  if (U < 0 || n_cap < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (!dtype_ok(kdt)) return FATHOM_ERR_UNSUPPORTED;
  if (n_cap > ((int64_t)1 << 31)) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0) return FATHOM_OK;
  if (!n || !aligned(n, 8)) return FATHOM_ERR_INVALID;
  if (n_cap > 0) {
    if (!K || !aligned(K, dtype_size(kdt))) return FATHOM_ERR_INVALID;
    if (ld_tok < D || ld_unit < 0) return FATHOM_ERR_INVALID;
  }
  return FATHOM_OK;
}

size_t fathom_klt_calibrate_workspace_size(int U) { return U > 0 ? klt_ws_bytes(U) : 0; }

fathom_status fathom_klt_calibrate(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                   const int64_t* n, int64_t n_cap, int U, int D, float* mu, float* V, float* lam,
                                   void* ws, size_t ws_bytes, uint32_t* dev_status, void* stream) {
  const fathom_status e = check_klt_keys(K, kdt, ld_tok, ld_unit, n, n_cap, U, D);
  if (e != FATHOM_OK || U == 0) return e;
  if (!mu || !V || !lam || !ws) return FATHOM_ERR_INVALID;
  if (!aligned(mu, 4) || !aligned(V, 4) || !aligned(lam, 4) || !aligned(ws, 256)) return FATHOM_ERR_INVALID;
  if (ws_bytes < klt_ws_bytes(U)) return FATHOM_ERR_WORKSPACE;
  return launch_klt_calibrate(K, kdt, ld_tok, ld_unit, n, n_cap, U, mu, V, lam, ws, dev_status, as_stream(stream));
}

fathom_status fathom_klt_rotate_keys(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                     const int64_t* n, int64_t n_cap, int U, int D, const float* mu,
                                     const float* V, float* out, int64_t ld_out_unit, uint32_t* dev_status,
                                     void* stream) {
  const fathom_status e = check_klt_keys(K, kdt, ld_tok, ld_unit, n, n_cap, U, D);
  if (e != FATHOM_OK || U == 0 || n_cap == 0) return e;
  if (!mu || !V || !out) return FATHOM_ERR_INVALID;
  if (!aligned(mu, 4) || !aligned(V, 4) || !aligned(out, 4)) return FATHOM_ERR_INVALID;
  if (ld_out_unit < n_cap * D) return FATHOM_ERR_INVALID;
  return launch_klt_rotate_keys(K, kdt, ld_tok, ld_unit, n, n_cap, U, mu, V, out, ld_out_unit, dev_status,
                                as_stream(stream));
}

fathom_status fathom_klt_rotate_q(const void* q, fathom_dtype qdt, int U, int G, int D, const float* V, float* out,
                                  void* stream) {
  if (U < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (G < 1 || G > kMaxG || !dtype_ok(qdt)) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0) return FATHOM_OK;
  if (!q || !V || !out) return FATHOM_ERR_INVALID;
  if (!aligned(q, dtype_size(qdt)) || !aligned(V, 16) || !aligned(out, 4)) return FATHOM_ERR_INVALID;
  return launch_klt_rotate_q(q, qdt, U, G, V, out, as_stream(stream));
}

const char* fathom_status_string(fathom_status s) {
  switch (s) {
    case FATHOM_OK: return "FATHOM_OK";
    case FATHOM_ERR_INVALID: return "FATHOM_ERR_INVALID";
    case FATHOM_ERR_UNSUPPORTED: return "FATHOM_ERR_UNSUPPORTED";
    case FATHOM_ERR_RANGE: return "FATHOM_ERR_RANGE";
    case FATHOM_ERR_HIP: return "FATHOM_ERR_HIP";
    case FATHOM_ERR_WORKSPACE: return "FATHOM_ERR_WORKSPACE";
  }
  return "FATHOM_ERR_UNKNOWN";
}

const char* fathom_version(void) { return "fathom-mi355x 0.1 gfx950"; }

fathom_status fathom_pack(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit, const int64_t* n,
                          int U, int D, int64_t nb_cap, uint64_t* planes, uint16_t* scales, uint32_t* dev_status,
                          void* stream) {
  if (U < 0 || nb_cap < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (!dtype_ok(kdt)) return FATHOM_ERR_UNSUPPORTED;
  if (nb_cap > ((int64_t)1 << 25)) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  if (!K || !n || !planes || !scales) return FATHOM_ERR_INVALID;
  const int64_t vec = 16 / (int64_t)dtype_size(kdt);  // elements per 16-byte load
  if (ld_tok < D || ld_tok % vec || ld_unit < 0 || ld_unit % vec) return FATHOM_ERR_INVALID;
  if (!aligned(K, 16) || !aligned(planes, 8) || !aligned(scales, 2) || !aligned(n, 8)) return FATHOM_ERR_INVALID;
  return launch_pack(K, kdt, ld_tok, ld_unit, n, nullptr, 0, U, nb_cap, planes, scales, dev_status,
                     as_stream(stream));
}

fathom_status fathom_pack_append(const void* K, fathom_dtype kdt, int64_t ld_tok, int64_t ld_unit,
                                 const int64_t* n_old, const int64_t* n, int64_t max_new, int U, int D,
                                 int64_t nb_cap, uint64_t* planes, uint16_t* scales, uint32_t* dev_status,
                                 void* stream) {
  if (U < 0 || nb_cap < 0 || max_new < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (!dtype_ok(kdt)) return FATHOM_ERR_UNSUPPORTED;
  if (nb_cap > ((int64_t)1 << 25)) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  if (!K || !n || !n_old || !planes || !scales) return FATHOM_ERR_INVALID;
  const int64_t vec = 16 / (int64_t)dtype_size(kdt);
  if (ld_tok < D || ld_tok % vec || ld_unit < 0 || ld_unit % vec) return FATHOM_ERR_INVALID;
  if (!aligned(K, 16) || !aligned(planes, 8) || !aligned(scales, 2) || !aligned(n, 8) || !aligned(n_old, 8))
    return FATHOM_ERR_INVALID;
  return launch_pack(K, kdt, ld_tok, ld_unit, n, n_old, max_new, U, nb_cap, planes, scales, dev_status,
                     as_stream(stream));
}

fathom_status fathom_gather_store(const uint64_t* host_planes, const uint16_t* host_scales, const uint8_t* depths,
                                 int U, int D, int64_t nb_cap, uint64_t* planes, uint16_t* scales, void* stream) {
  if (U < 0 || nb_cap < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (nb_cap > ((int64_t)1 << 25)) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  if (!host_planes || !host_scales || !depths || !planes || !scales) return FATHOM_ERR_INVALID;
  if (!aligned(host_planes, 16) || !aligned(planes, 16) || !aligned(host_scales, 16) || !aligned(scales, 16))
    return FATHOM_ERR_INVALID;
  return launch_gather(host_planes, host_scales, depths, U, nb_cap, planes, scales, as_stream(stream));
}

fathom_status fathom_alloc_depths(const void* q, fathom_dtype qdt, int U, int G, int D, const float* var,
                                  fathom_mode mode, int budget_or_r, uint8_t* depths, float* theta,
                                  uint32_t* dev_status, void* stream) {
  if (U < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (G < 1 || G > kMaxG || !dtype_ok(qdt)) return FATHOM_ERR_UNSUPPORTED;
  if (mode != FATHOM_WATERFILL && mode != FATHOM_UNIFORM_TOPR) return FATHOM_ERR_UNSUPPORTED;
  if (mode == FATHOM_WATERFILL && (budget_or_r < 0 || budget_or_r > 4 * D)) return FATHOM_ERR_RANGE;
  if (mode == FATHOM_UNIFORM_TOPR && (budget_or_r < 0 || budget_or_r > D)) return FATHOM_ERR_RANGE;
  if (U == 0) return FATHOM_OK;
  if (!q || !depths || (mode == FATHOM_WATERFILL && !var)) return FATHOM_ERR_INVALID;
  if (!aligned(q, dtype_size(qdt)) || (var && !aligned(var, 4)) || (theta && !aligned(theta, 4)))
    return FATHOM_ERR_INVALID;
  return launch_alloc(q, qdt, U, G, var, mode, budget_or_r, depths, theta, dev_status, as_stream(stream));
}

fathom_status fathom_scan(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int D,
                          int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths,
                          float* scores, int64_t ld_s, uint32_t* dev_status, void* stream) {
  fathom_status e = check_store(planes, scales, n, U, D, nb_cap, q, qdt, G, depths);
  if (e != FATHOM_OK) return e;
  if (ld_s < 1) return FATHOM_ERR_INVALID;
  if (U == 0 || nb_cap == 0) return FATHOM_OK;
  if (!scores || !aligned(scores, 4)) return FATHOM_ERR_INVALID;
  return launch_scan(planes, scales, n, U, nb_cap, q, qdt, G, depths, scores, ld_s, dev_status, as_stream(stream));
}

size_t fathom_topk_workspace_size(int U, int G, int64_t max_n, int k) {
  if (U <= 0 || G <= 0 || k <= 0 || max_n < 0) return 0;
  return topk_ws_bytes(U * G, max_n, k);
}

fathom_status fathom_topk(const float* scores, int64_t ld_s, const int64_t* n, int U, int G, int k, int64_t lo,
                          int64_t tail, int32_t* idx, float* val, void* ws, size_t ws_bytes, uint32_t* dev_status,
                          void* stream) {
  if (U < 0 || ld_s < 1 || lo < 0 || tail < 0 || k < 1) return FATHOM_ERR_INVALID;
  if (G < 1 || G > kMaxG) return FATHOM_ERR_UNSUPPORTED;
  if (k > FATHOM_MAX_K) return FATHOM_ERR_UNSUPPORTED;
  if (ld_s > ((int64_t)1 << 31) - 1) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0) return FATHOM_OK;
  if (!scores || !n || !idx || !ws) return FATHOM_ERR_INVALID;
  if (!aligned(scores, 4) || !aligned(n, 8) || !aligned(idx, 4) || (val && !aligned(val, 4)) || !aligned(ws, 256))
    return FATHOM_ERR_INVALID;
  if (ws_bytes < topk_ws_bytes(U * G, ld_s, k)) return FATHOM_ERR_WORKSPACE;
  return launch_topk(scores, ld_s, n, U, G, k, lo, tail, idx, val, ws, dev_status, as_stream(stream));
}

size_t fathom_scan_topk_workspace_size(int U, int G, int64_t max_n, int k) {
  if (U <= 0 || G <= 0 || k <= 0 || max_n < 0) return 0;
  return scan_topk_ws(U, G, max_n, k);
}

fathom_status fathom_scan_topk_ex(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int D,
                                  int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths, int k,
                                  int64_t lo, int64_t tail, int max_unit_bits, int32_t* idx, float* val, void* ws,
                                  size_t ws_bytes, uint32_t* dev_status, void* stream) {
  fathom_status e = check_store(planes, scales, n, U, D, nb_cap, q, qdt, G, depths);
  if (e != FATHOM_OK) return e;
  if (lo < 0 || tail < 0 || k < 1 || max_unit_bits < 0) return FATHOM_ERR_INVALID;
  if (k > FATHOM_MAX_K) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0) return FATHOM_OK;
  if (!idx || !ws || !aligned(idx, 4) || (val && !aligned(val, 4)) || !aligned(ws, 256)) return FATHOM_ERR_INVALID;
  if (ws_bytes < scan_topk_ws(U, G, nb_cap * 64, k)) return FATHOM_ERR_WORKSPACE;
  return launch_scan_topk_fused(planes, scales, n, U, nb_cap, q, qdt, G, depths, k, lo, tail, max_unit_bits, idx, val,
                                ws, dev_status, as_stream(stream));
}

size_t fathom_scan_topk_noalloc_capacity(void) { return scratch_capacity(); }

fathom_status fathom_scan_topk_noalloc(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int D,
                                       int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths,
                                       int k, int64_t lo, int64_t tail, int max_unit_bits, int32_t* idx, float* val,
                                       uint32_t* dev_status, void* stream) {
  fathom_status e = check_store(planes, scales, n, U, D, nb_cap, q, qdt, G, depths);
  if (e != FATHOM_OK) return e;
  if (lo < 0 || tail < 0 || k < 1 || max_unit_bits < 0) return FATHOM_ERR_INVALID;
  if (k > FATHOM_MAX_K) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0) return FATHOM_OK;
  if (!idx || !aligned(idx, 4) || (val && !aligned(val, 4))) return FATHOM_ERR_INVALID;
  if (scan_topk_ws(U, G, nb_cap * 64, k) > scratch_capacity()) return FATHOM_ERR_WORKSPACE;
  void* ws = nullptr;
  e = scratch_address(&ws);
  if (e != FATHOM_OK) return e;
  return launch_scan_topk_fused(planes, scales, n, U, nb_cap, q, qdt, G, depths, k, lo, tail, max_unit_bits, idx, val,
                                ws, dev_status, as_stream(stream));
}

fathom_status fathom_scan_topk(const uint64_t* planes, const uint16_t* scales, const int64_t* n, int U, int D,
                               int64_t nb_cap, const void* q, fathom_dtype qdt, int G, const uint8_t* depths, int k,
                               int64_t lo, int64_t tail, int32_t* idx, float* val, void* ws, size_t ws_bytes,
                               uint32_t* dev_status, void* stream) {
  return fathom_scan_topk_ex(planes, scales, n, U, D, nb_cap, q, qdt, G, depths, k, lo, tail, 0, idx, val, ws,
                             ws_bytes, dev_status, stream);
}

size_t fathom_sparse_attn_workspace_size(int U, int G, int k, int n_sink, int n_local) {
  if (U <= 0 || G <= 0 || k < 0 || n_sink < 0 || n_local < 0) return 0;
  return attn_ws_bytes(U, G, k, n_sink, n_local);
}

fathom_status fathom_sparse_attn(const void* q, fathom_dtype qdt, const uint16_t* Krows, const uint16_t* Vrows,
                                 int64_t ld_tok, int64_t ld_unit, const int64_t* n, int U, int G, int D,
                                 const int32_t* idx, int k, int n_sink, int n_local, float sm_scale, float* out,
                                 void* ws, size_t ws_bytes, uint32_t* dev_status, void* stream) {
  if (U < 0 || k < 0 || n_sink < 0 || n_local < 0) return FATHOM_ERR_INVALID;
  if (D != kD) return FATHOM_ERR_UNSUPPORTED;
  if (G < 1 || G > kMaxG || !dtype_ok(qdt)) return FATHOM_ERR_UNSUPPORTED;
  if (k > FATHOM_MAX_K || n_sink + n_local > attn_max_sink_local()) return FATHOM_ERR_UNSUPPORTED;
  if (U == 0) return FATHOM_OK;
  if (!q || !Krows || !Vrows || !n || !out || (k > 0 && !idx)) return FATHOM_ERR_INVALID;
  if (ld_tok < D || ld_tok % 2 || ld_unit < 0 || ld_unit % 2) return FATHOM_ERR_INVALID;
  if (!aligned(Krows, 4) || !aligned(Vrows, 4) || !aligned(q, dtype_size(qdt)) || !aligned(out, 4) ||
      !aligned(n, 8) || (idx && !aligned(idx, 4)))
    return FATHOM_ERR_INVALID;
  if (!ws || !aligned(ws, 256)) return FATHOM_ERR_INVALID;
  if (ws_bytes < attn_ws_bytes(U, G, k, n_sink, n_local)) return FATHOM_ERR_WORKSPACE;
  return launch_sparse_attn(q, qdt, Krows, Vrows, ld_tok, ld_unit, n, U, G, idx, k, n_sink, n_local, sm_scale, out,
                            ws, dev_status, as_stream(stream));
}

}  // extern "C"
