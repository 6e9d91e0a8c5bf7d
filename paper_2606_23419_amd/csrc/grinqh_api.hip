// libgrinqh C ABI: host-side validation and dispatch.  Every check happens
// before anything is enqueued, so a failing call writes nothing.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "grinqh_internal.h"

namespace grinqh {

static thread_local char g_err[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return status;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRINQH_EHIP, "%s: %s", what, hipGetErrorString(e));
  return GRINQH_OK;
}

static void clear_error() { g_err[0] = '\0'; }

static Options g_opt = {};

int option(int Options::*field) { return __atomic_load_n(&(g_opt.*field), __ATOMIC_RELAXED); }

// Validate a descriptor and fill a Layer.
static int resolve(const grinqh_layer_desc* d, Layer* L, grinqh_layer_desc* out) {
  if (!d) return fail(GRINQH_EINVAL, "desc is NULL");
  if (d->K <= 0 || d->N <= 0) return fail(GRINQH_EINVAL, "K=%d and N=%d must be positive", d->K, d->N);
  if (d->group != kGroup)
    return fail(GRINQH_EUNSUPPORTED, "group=%d: only groups of %d channels are implemented", d->group, kGroup);
  if (d->K % kGroup) return fail(GRINQH_EINVAL, "K=%d is not a multiple of the group %d", d->K, kGroup);
  if (d->K > (1 << 20)) return fail(GRINQH_EUNSUPPORTED, "K=%d exceeds 2^20", d->K);
  if (d->N > (1 << 20)) return fail(GRINQH_EUNSUPPORTED, "N=%d exceeds 2^20", d->N);
  const int nl = d->n_levels;
  if (nl < 2 || nl > kMaxLevels) return fail(GRINQH_EINVAL, "n_levels=%d outside 2..%d", nl, kMaxLevels);
  if (d->level_bits[0] != 0) return fail(GRINQH_EINVAL, "level_bits[0] must be 0 (the skip level)");
  const int bmax = d->level_bits[nl - 1];
  if (bmax != 4 && bmax != 6 && bmax != 8)
    return fail(GRINQH_EUNSUPPORTED, "the top level is the stored width b_max and must be 4, 6 or 8 (got %d)", bmax);
  bool all_even = true;
  for (int i = 1; i < nl; ++i) {
    if (d->level_bits[i] <= d->level_bits[i - 1])
      return fail(GRINQH_EINVAL, "level_bits must be strictly increasing (index %d)", i);
    if (d->level_bits[i] & 1) all_even = false;
  }
  int u = d->plane_bits;
  if (u == 0) u = all_even ? 2 : 1;
  if (u != 1 && u != 2) return fail(GRINQH_EUNSUPPORTED, "plane_bits=%d: only 1 and 2 are implemented", d->plane_bits);
  for (int i = 1; i < nl; ++i)
    if (d->level_bits[i] % u)
      return fail(GRINQH_EINVAL, "level %d has %d bits, not a multiple of plane_bits=%d", i, d->level_bits[i], u);
  int T = d->tile_n;
  if (T == 0) {
    // Auto: the widest tile (fewer, longer rows per workgroup) that still
    // leaves at least 256 (tile, group) work units for 256 CUs; if none does,
    // the tile giving the most units.  1-bit planes take 512 first: their
    // 64-byte plane rows pair up in 128-byte lines, and every Qwen3-8B layer
    // measured faster at 512 than at 1024.
    const long groups = d->K / kGroup;
    const int cand2[] = {1024, 512, 256}, cand1[] = {512, 1024, 256};
    for (int c : (u == 1 ? cand1 : cand2)) {
      if (c * u >= 512 && d->N % c == 0 && (long)(d->N / c) * groups >= 256) { T = c; break; }
    }
    if (T == 0) {
      for (int c : {256, 512, 1024, 2048}) {
        if (c * u >= 512 && d->N % c == 0) { T = c; break; }
      }
    }
    if (T == 0) return fail(GRINQH_EUNSUPPORTED, "N=%d has no supported tile width for plane_bits=%d", d->N, u);
  } else {
    if (T != 256 && T != 512 && T != 1024 && T != 2048)
      return fail(GRINQH_EUNSUPPORTED, "tile_n=%d: use 256, 512, 1024 or 2048", T);
    if (T * u < 512) return fail(GRINQH_EUNSUPPORTED, "tile_n=%d with plane_bits=%d gives planes under 64 bytes", T, u);
    if (d->N % T) return fail(GRINQH_EINVAL, "N=%d is not a multiple of tile_n=%d", d->N, T);
  }
  if (L) {
    L->K = d->K; L->N = d->N; L->n_levels = nl; L->u = u; L->bmax = bmax; L->P = bmax / u; L->T = T;
    L->RB = T * bmax / 8;
    L->sfac = ldexpf(1.0f, bmax - 8);
    L->tiles = d->N / T; L->groups = d->K / kGroup;
    L->planes_packed = 0;
    for (int i = 0; i < kMaxLevels; ++i) {
      L->bits[i] = i < nl ? d->level_bits[i] : 0;
      L->planes[i] = i < nl ? d->level_bits[i] / u : 0;
      L->planes_packed |= (uint64_t)L->planes[i] << (4 * i);
    }
  }
  if (out) {
    *out = *d;
    out->plane_bits = u;
    out->tile_n = T;
  }
  return GRINQH_OK;
}

static int check_thresholds(const Layer& L, const float* th, Thresholds* out) {
  if (!th) return fail(GRINQH_EINVAL, "thresholds is NULL");
  const int n = L.n_levels - 1;
  for (int j = 0; j < n; ++j) {
    if (std::isnan(th[j])) return fail(GRINQH_EINVAL, "threshold %d is NaN", j + 1);
    if (j && th[j] < th[j - 1]) return fail(GRINQH_EINVAL, "thresholds must be non-decreasing (index %d)", j + 1);
  }
  out->n = n;
  for (int j = 0; j < kMaxLevels - 1; ++j) out->theta[j] = j < n ? th[j] : INFINITY;
  return GRINQH_OK;
}

}  // namespace grinqh

using namespace grinqh;

extern "C" {

int grinqh_resolve_desc(const grinqh_layer_desc* in, grinqh_layer_desc* out) {
  clear_error();
  if (!out) return fail(GRINQH_EINVAL, "out is NULL");
  return resolve(in, nullptr, out);
}

int grinqh_packed_bytes(const grinqh_layer_desc* desc, size_t* codes_bytes, size_t* scales_bytes) {
  clear_error();
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (!codes_bytes || !scales_bytes) return fail(GRINQH_EINVAL, "output pointers are NULL");
  *codes_bytes = (size_t)L.K * (size_t)L.N * (size_t)L.bmax / 8;
  *scales_bytes = (size_t)L.groups * (size_t)L.N * 2;
  return GRINQH_OK;
}

int grinqh_pack(const grinqh_layer_desc* desc, int src_kind, const void* src, const void* src_scales,
                void* packed_codes, void* packed_scales, void* stream) {
  clear_error();
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (src_kind != GRINQH_SRC_FP16_RTN && src_kind != GRINQH_SRC_CODES_U8)
    return fail(GRINQH_EINVAL, "src_kind=%d is not a known source kind", src_kind);
  if (!src || !packed_codes) return fail(GRINQH_EINVAL, "src and packed_codes must not be NULL");
  if (src_kind == GRINQH_SRC_FP16_RTN && src_scales) return fail(GRINQH_EINVAL, "src_scales must be NULL for an fp16 source");
  if (src_kind == GRINQH_SRC_FP16_RTN && !packed_scales) return fail(GRINQH_EINVAL, "packed_scales is NULL for an fp16 source");
  if (src_kind == GRINQH_SRC_CODES_U8 && (!src_scales) != (!packed_scales))
    return fail(GRINQH_EINVAL, "a codes source takes src_scales and packed_scales together, or neither");
  return launch_pack(L, src_kind, src, src_scales, packed_codes, packed_scales, (hipStream_t)stream);
}

int grinqh_topk_counts(int32_t K, int32_t n_levels, const int32_t* p_bp, int32_t* counts_out) {
  clear_error();
  if (K <= 0) return fail(GRINQH_EINVAL, "K=%d must be positive", K);
  if (n_levels < 2 || n_levels > kMaxLevels) return fail(GRINQH_EINVAL, "n_levels=%d outside 2..%d", n_levels, kMaxLevels);
  if (!p_bp || !counts_out) return fail(GRINQH_EINVAL, "p_bp and counts_out must not be NULL");
  long long total = 0;
  for (int j = 0; j < n_levels; ++j) {
    if (p_bp[j] < 0) return fail(GRINQH_EINVAL, "p_bp[%d]=%d is negative", j, p_bp[j]);
    total += p_bp[j];
  }
  if (total != 10000) return fail(GRINQH_EINVAL, "p_bp sums to %lld, not 10000", total);
  long long C[kMaxLevels + 1];
  for (int j = 0; j < n_levels; ++j) {
    long long U = 0;
    for (int i = j; i < n_levels; ++i) U += p_bp[i];
    C[j] = (U * (long long)K + 5000) / 10000;
  }
  C[n_levels] = 0;
  for (int j = 0; j < n_levels; ++j) counts_out[j] = (int32_t)(C[j] - C[j + 1]);
  return GRINQH_OK;
}

int grinqh_workspace_bytes(const grinqh_layer_desc* desc, int32_t B, size_t* bytes) {
  clear_error();
  int st = resolve(desc, nullptr, nullptr);
  if (st) return st;
  if (B < 1) return fail(GRINQH_EINVAL, "B=%d must be positive", B);
  if (!bytes) return fail(GRINQH_EINVAL, "bytes is NULL");
  *bytes = 0;
  return GRINQH_OK;
}

// Validation shared by both calibration entry points, and the quantile
// positions h = (K-1) U_k / 10000 taken exactly: lo = floor(h), frac its
// fraction.
static int calibrate_checks(const grinqh_layer_desc* desc, const void* x, int32_t S,
                            const int32_t* p_bp, float* theta, Layer* L, QuantilePos* qp) {
  int st = resolve(desc, L, nullptr);
  if (st) return st;
  if (!x || !p_bp || !theta) return fail(GRINQH_EINVAL, "x, p_bp and theta must not be NULL");
  if (S < 1 || S > 65535) return fail(GRINQH_EINVAL, "S=%d outside 1..65535", S);
  if (L->K > 16384) return fail(GRINQH_EUNSUPPORTED, "calibration needs K <= 16384 (K=%d)", L->K);
  if ((uintptr_t)x & 3u) return fail(GRINQH_EINVAL, "x must be 4-byte aligned");
  if ((uintptr_t)theta & 3u) return fail(GRINQH_EINVAL, "theta must be 4-byte aligned");
  long long total = 0;
  for (int j = 0; j < L->n_levels; ++j) {
    if (p_bp[j] < 0) return fail(GRINQH_EINVAL, "p_bp[%d]=%d is negative", j, p_bp[j]);
    total += p_bp[j];
  }
  if (total != 10000) return fail(GRINQH_EINVAL, "p_bp sums to %lld, not 10000", total);
  *qp = QuantilePos{};
  qp->n = L->n_levels - 1;
  long long U = 0;
  for (int k = 0; k < qp->n; ++k) {
    U += p_bp[k];
    const long long num = (long long)(L->K - 1) * U;
    qp->lo[k] = (int)(num / 10000);
    qp->hi[k] = qp->lo[k] + 1 < L->K ? qp->lo[k] + 1 : L->K - 1;
    qp->frac[k] = (double)(num % 10000) / 10000.0;
  }
  return GRINQH_OK;
}

int grinqh_calibrate(const grinqh_layer_desc* desc, const void* x, int32_t S, const int32_t* p_bp,
                     double* per_sample, float* theta, void* stream) {
  clear_error();
  if (!per_sample) return fail(GRINQH_EINVAL, "per_sample must not be NULL");
  if ((uintptr_t)per_sample & 7u) return fail(GRINQH_EINVAL, "per_sample must be 8-byte aligned");
  Layer L;
  QuantilePos qp;
  int st = calibrate_checks(desc, x, S, p_bp, theta, &L, &qp);
  if (st) return st;
  return launch_calibrate(L, x, S, qp, per_sample, theta, (hipStream_t)stream);
}

int grinqh_calibrate_noalloc(const grinqh_layer_desc* desc, const void* x, int32_t S,
                             const int32_t* p_bp, float* theta, void* stream) {
  clear_error();
  Layer L;
  QuantilePos qp;
  int st = calibrate_checks(desc, x, S, p_bp, theta, &L, &qp);
  if (st) return st;
  return launch_calibrate_noalloc(L, x, S, qp, theta, (hipStream_t)stream);
}

// Per-level channel counts -> cumulative cuts C_j (channels at level >= j + 1).
static int topk_cuts(const Layer& L, const int32_t* counts, TopkCuts* cuts) {
  if (!counts) return fail(GRINQH_EINVAL, "counts is NULL");
  if (L.K > 16384) return fail(GRINQH_EUNSUPPORTED, "top-k assignment needs K <= 16384 (K=%d)", L.K);
  long long total = 0;
  for (int j = 0; j < L.n_levels; ++j) {
    if (counts[j] < 0) return fail(GRINQH_EINVAL, "counts[%d]=%d is negative", j, counts[j]);
    total += counts[j];
  }
  if (total != L.K) return fail(GRINQH_EINVAL, "counts sum to %lld, not K=%d", total, L.K);
  cuts->n = L.n_levels - 1;
  for (int j = 0; j < kMaxLevels; ++j) {
    long long c = 0;
    if (j < cuts->n)
      for (int i = j + 1; i < L.n_levels; ++i) c += counts[i];
    cuts->cum[j] = (int)c;
  }
  return GRINQH_OK;
}

int grinqh_assign(const grinqh_layer_desc* desc, int mode, const void* x, int32_t B,
                  const float* thresholds, const int32_t* counts, uint8_t* level_map,
                  void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  (void)workspace; (void)ws_bytes;
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (B < 1 || B > 65535) return fail(GRINQH_EINVAL, "B=%d outside 1..65535", B);
  if (!x || !level_map) return fail(GRINQH_EINVAL, "x and level_map must not be NULL");
  if (mode == GRINQH_ASSIGN_THRESHOLD) {
    if (counts) return fail(GRINQH_EINVAL, "counts must be NULL in threshold mode");
    Thresholds th;
    st = check_thresholds(L, thresholds, &th);
    if (st) return st;
    return launch_assign_threshold(L, x, B, th, level_map, (hipStream_t)stream);
  }
  if (mode == GRINQH_ASSIGN_TOPK) {
    if (thresholds) return fail(GRINQH_EINVAL, "thresholds must be NULL in top-k mode");
    TopkCuts cuts;
    st = topk_cuts(L, counts, &cuts);
    if (st) return st;
    return launch_assign_topk(L, x, B, cuts, level_map, (hipStream_t)stream);
  }
  return fail(GRINQH_EINVAL, "mode=%d is not a known assignment mode", mode);
}

static int vmm_common_checks(const Layer& L, const void* codes, const void* scales, const void* x,
                             int32_t B, float* y, int32_t flags) {
  if (!codes || !scales || !x || !y) return fail(GRINQH_EINVAL, "codes, scales, x and y must not be NULL");
  if (B < 1 || B > kMaxB) return fail(GRINQH_EUNSUPPORTED, "B=%d outside 1..%d", B, kMaxB);
  if (flags & ~GRINQH_VMM_ACCUMULATE) return fail(GRINQH_EINVAL, "unknown flags 0x%x", flags);
  if (((uintptr_t)codes | (uintptr_t)scales) & 15u)
    return fail(GRINQH_EINVAL, "packed codes and scales must be 16-byte aligned");
  if (((uintptr_t)x | (uintptr_t)y) & 3u) return fail(GRINQH_EINVAL, "x and y must be 4-byte aligned");
  (void)L;
  return GRINQH_OK;
}

int grinqh_vmm(const grinqh_layer_desc* desc, const void* packed_codes, const void* packed_scales,
               const void* x, const uint8_t* level_map, int32_t B, float* y, int32_t flags,
               void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  (void)workspace; (void)ws_bytes;
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  st = vmm_common_checks(L, packed_codes, packed_scales, x, B, y, flags);
  if (st) return st;
  if (!level_map) return fail(GRINQH_EINVAL, "level_map is NULL");
  if ((uintptr_t)level_map & 1u) return fail(GRINQH_EINVAL, "level_map must be 2-byte aligned");
  return launch_vmm(L, packed_codes, packed_scales, x, level_map, nullptr, nullptr, B, y,
                    flags & GRINQH_VMM_ACCUMULATE, (hipStream_t)stream);
}

int grinqh_vmm_threshold(const grinqh_layer_desc* desc, const void* packed_codes,
                         const void* packed_scales, const void* x, int32_t B,
                         const float* thresholds, uint8_t* level_map_out, float* y,
                         int32_t flags, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  (void)workspace; (void)ws_bytes;
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  st = vmm_common_checks(L, packed_codes, packed_scales, x, B, y, flags);
  if (st) return st;
  Thresholds th;
  st = check_thresholds(L, thresholds, &th);
  if (st) return st;
  return launch_vmm(L, packed_codes, packed_scales, x, nullptr, &th, level_map_out, B, y,
                    flags & GRINQH_VMM_ACCUMULATE, (hipStream_t)stream);
}

int grinqh_vmm_topk(const grinqh_layer_desc* desc, const void* packed_codes,
                    const void* packed_scales, const void* x, int32_t B, const int32_t* counts,
                    uint8_t* level_map_out, float* y, int32_t flags, void* workspace,
                    size_t ws_bytes, void* stream) {
  clear_error();
  (void)workspace; (void)ws_bytes;
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  st = vmm_common_checks(L, packed_codes, packed_scales, x, B, y, flags);
  if (st) return st;
  TopkCuts cuts;
  st = topk_cuts(L, counts, &cuts);
  if (st) return st;
  if (B != 1 || !vmm_pp_supported(L, 1) || option(&Options::vmm_kernel))
    return fail(GRINQH_EUNSUPPORTED,
                "the fused top-k VMM runs at B = 1 on 2-bit planes with T in {256, 512, 1024}; "
                "use grinqh_assign (top-k) and grinqh_vmm");
  if (((uintptr_t)x & 15u)) return fail(GRINQH_EINVAL, "x must be 16-byte aligned in top-k mode");
  return launch_vmm_topk(L, packed_codes, packed_scales, x, cuts, level_map_out, y,
                         flags & GRINQH_VMM_ACCUMULATE, (hipStream_t)stream);
}

int grinqh_prefill(const grinqh_layer_desc* desc, const void* packed_codes,
                   const void* packed_scales, const void* x, int32_t M, float* y, int32_t flags,
                   void* stream) {
  clear_error();
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (!packed_codes || !packed_scales || !x || !y)
    return fail(GRINQH_EINVAL, "codes, scales, x and y must not be NULL");
  if (M < 1 || M > (1 << 24)) return fail(GRINQH_EINVAL, "M=%d outside 1..2^24", M);
  if (flags & ~GRINQH_VMM_ACCUMULATE) return fail(GRINQH_EINVAL, "unknown flags 0x%x", flags);
  if (((uintptr_t)packed_codes | (uintptr_t)packed_scales | (uintptr_t)x) & 15u)
    return fail(GRINQH_EINVAL, "packed codes, scales and x must be 16-byte aligned");
  if ((uintptr_t)y & 3u) return fail(GRINQH_EINVAL, "y must be 4-byte aligned");
  return launch_prefill(L, packed_codes, packed_scales, x, M, y, flags & GRINQH_VMM_ACCUMULATE,
                        (hipStream_t)stream);
}

int grinqh_lut_entries(const grinqh_layer_desc* desc, size_t* entries) {
  clear_error();
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (!entries) return fail(GRINQH_EINVAL, "entries is NULL");
  LutDesc D;
  lut_desc(L, &D);
  *entries = (size_t)L.N * (size_t)D.entries;
  return GRINQH_OK;
}

int grinqh_vmm_lut(const grinqh_layer_desc* desc, const void* packed_codes, const void* luts,
                   const void* x, const uint8_t* level_map, int32_t B, float* y, int32_t flags,
                   void* stream) {
  clear_error();
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (!packed_codes || !luts || !x || !level_map || !y)
    return fail(GRINQH_EINVAL, "codes, luts, x, level_map and y must not be NULL");
  if (B < 1 || B > 65535) return fail(GRINQH_EINVAL, "B=%d outside 1..65535", B);
  if (flags & ~GRINQH_VMM_ACCUMULATE) return fail(GRINQH_EINVAL, "unknown flags 0x%x", flags);
  if (((uintptr_t)packed_codes | (uintptr_t)luts) & 15u)
    return fail(GRINQH_EINVAL, "packed codes and luts must be 16-byte aligned");
  if (((uintptr_t)x | (uintptr_t)y) & 3u) return fail(GRINQH_EINVAL, "x and y must be 4-byte aligned");
  return launch_vmm_lut(L, packed_codes, luts, x, level_map, nullptr, nullptr, B, y,
                        flags & GRINQH_VMM_ACCUMULATE, (hipStream_t)stream);
}

int grinqh_vmm_lut_threshold(const grinqh_layer_desc* desc, const void* packed_codes, const void* luts,
                             const void* x, int32_t B, const float* thresholds, uint8_t* level_map_out,
                             float* y, int32_t flags, void* stream) {
  clear_error();
  Layer L;
  int st = resolve(desc, &L, nullptr);
  if (st) return st;
  if (!packed_codes || !luts || !x || !y) return fail(GRINQH_EINVAL, "codes, luts, x and y must not be NULL");
  if (B < 1 || B > 65535) return fail(GRINQH_EINVAL, "B=%d outside 1..65535", B);
  if (flags & ~GRINQH_VMM_ACCUMULATE) return fail(GRINQH_EINVAL, "unknown flags 0x%x", flags);
  if (((uintptr_t)packed_codes | (uintptr_t)luts) & 15u)
    return fail(GRINQH_EINVAL, "packed codes and luts must be 16-byte aligned");
  if (((uintptr_t)x | (uintptr_t)y) & 3u) return fail(GRINQH_EINVAL, "x and y must be 4-byte aligned");
  Thresholds th;
  st = check_thresholds(L, thresholds, &th);
  if (st) return st;
  return launch_vmm_lut(L, packed_codes, luts, x, nullptr, &th, level_map_out, B, y,
                        flags & GRINQH_VMM_ACCUMULATE, (hipStream_t)stream);
}

int grinqh_set_option(int opt, int value) {
  clear_error();
  int Options::*field = nullptr;
  int lo = 0, hi = 0;
  switch (opt) {
    case GRINQH_OPT_VMM_KERNEL: field = &Options::vmm_kernel; hi = GRINQH_KERNEL_GENERAL; break;
    case GRINQH_OPT_GROUPS_PER_WG: field = &Options::groups_per_wg; hi = 4; break;
    case GRINQH_OPT_PREFILL_TILE: field = &Options::prefill_tile; hi = 3; break;
    case GRINQH_OPT_LUT_GROUPS: field = &Options::lut_groups; hi = 16; break;
    case GRINQH_OPT_PREFILL_CUS: field = &Options::prefill_cus; hi = 4096; break;
    default: return fail(GRINQH_EINVAL, "option=%d is not a known option", opt);
  }
  if (value < lo || value > hi) return fail(GRINQH_EINVAL, "option %d: value %d outside %d..%d", opt, value, lo, hi);
  __atomic_store_n(&(g_opt.*field), value, __ATOMIC_RELAXED);
  return GRINQH_OK;
}

int grinqh_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  clear_error();
  if (!src || !sink) return fail(GRINQH_EINVAL, "src and sink must not be NULL");
  if (((uintptr_t)src & 15u) || ((uintptr_t)sink & 3u)) return fail(GRINQH_EINVAL, "src must be 16-byte and sink 4-byte aligned");
  if (bytes == 0 || bytes % (2u << 20) || bytes / 512 > 0xFFFFFFFFull)
    return fail(GRINQH_EINVAL, "bytes=%zu must be a positive multiple of 2 MiB below 2 TiB", bytes);
  return launch_stream_read(src, bytes, sink, (hipStream_t)stream);
}

const char* grinqh_last_error(void) { return g_err; }

}  // extern "C"
