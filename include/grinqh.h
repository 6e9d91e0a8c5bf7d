/*
 * grinqh.h -- C ABI of libgrinqh, the nested-precision decode VMM of GRINQH
 * (Graded Input-based Quantization Hierarchy, arXiv 2606.23419) for AMD
 * Instinct MI355X (gfx950).
 *
 * The path (Sec. 3 of the paper):
 *   offline   W (fp16) --RTN, 8 bits, group 128--> codes + scales
 *             codes --nest + pack--> bit planes, most significant first
 *   per token x --magnitude grading--> a level per input channel
 *             y = W_hat(levels) x, each weight row read only to the depth its
 *             channel's level asks for (Sec. 3.3 "Storage Layout and Weight
 *             Loading"; App. C.1 "Sparse bit-loading").
 *
 * Conventions for every entry point
 *   - Device pointers are plain HIP device addresses owned by the caller; the
 *     library never allocates, frees or synchronises.  Host pointers are read
 *     during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All work is enqueued on it; nothing waits for it.
 *   - Every argument is validated on the host before anything is enqueued; a
 *     failing call returns a negative status, writes nothing and leaves a
 *     message for grinqh_last_error().  A failing launch returns GRINQH_EHIP.
 *     Faults inside kernels surface at the caller's next synchronisation.
 *   - Calls are thread-safe; the error message is per thread.
 *
 * Packed layout (the contract between grinqh_pack and grinqh_vmm)
 *   b_max (the top level's bits) in {4, 6, 8}: codes q are b_max-bit offset
 *   binary, w_hat = s*(q - 2^(b_max-1)) at full depth (Sec. 3.3 stores b_max
 *   = 4, 6 or 8).  u (plane_bits) in {1, 2}; P = b_max/u planes; T (tile_n)
 *   outputs per tile; R = T*b_max/8 bytes per stored row.
 *   codes buffer: (N/T) tiles x K rows x R bytes = K*N*b_max/8 bytes.
 *   Row (tile t, channel k) starts at byte (t*K + k)*R.  Plane j (1-based,
 *   j = 1 most significant) starts at byte (j-1)*T*u/8 of the row and holds,
 *   for local output o = n - t*T, the field (q >> (b_max - j*u)) & (2^u - 1)
 *   at bit o*u of the plane (byte floor(o*u/8), bit (o*u) % 8, little-endian).
 *   Reading b bits of a channel therefore reads the first b*T/8 bytes of its
 *   row in every tile: a contiguous prefix, a multiple of 64 bytes.
 *   scales buffer: fp16 [K/128][N], the scale of group g for output n at
 *   index g*N + n.
 */
#ifndef GRINQH_H
#define GRINQH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define GRINQH_API __attribute__((visibility("default")))
#else
#define GRINQH_API
#endif

typedef enum {
  GRINQH_OK = 0,
  GRINQH_EINVAL = -1,       /* invalid argument: null pointer, bad shape, bad ordering */
  GRINQH_EUNSUPPORTED = -2, /* well-formed but outside what these kernels implement */
  GRINQH_ESIZE = -3,        /* workspace too small, or a size overflows */
  GRINQH_EHIP = -4          /* the HIP runtime reported an error at launch */
} grinqh_status;

#define GRINQH_MAX_LEVELS 9

/* Layer descriptor: 36 bytes, natural alignment, no implicit padding. */
typedef struct {
  int32_t K;          /* input channels (d_in); a multiple of `group` */
  int32_t N;          /* outputs (d_out); a multiple of the tile width */
  int32_t group;      /* quantisation group along K; must be 128 */
  int32_t n_levels;   /* number of levels n+1 including level 0; 2..9 */
  uint8_t level_bits[GRINQH_MAX_LEVELS];
                      /* b_0 = 0 < b_1 < ... < b_n = b_max (Sec. 3.1: the set
                         B); b_max in {4, 6, 8} is the stored code width;
                         every b_i a multiple of plane_bits */
  uint8_t reserved_[3];
  int32_t plane_bits; /* u: 0 = auto (2 if every b_i is even, else 1); or 1, 2 */
  int32_t tile_n;     /* T: 0 = auto; else 256, 512, 1024 or 2048 with T*u >= 512 */
} grinqh_layer_desc;

enum { GRINQH_SRC_FP16_RTN = 0, GRINQH_SRC_CODES_U8 = 1 };
enum { GRINQH_ASSIGN_THRESHOLD = 0, GRINQH_ASSIGN_TOPK = 1 };
enum { GRINQH_VMM_ACCUMULATE = 1 };
/* Options of grinqh_set_option, and the kernels GRINQH_OPT_VMM_KERNEL names. */
enum { GRINQH_OPT_VMM_KERNEL = 1, GRINQH_OPT_GROUPS_PER_WG = 2, GRINQH_OPT_PREFILL_TILE = 3,
       GRINQH_OPT_LUT_GROUPS = 4, GRINQH_OPT_PREFILL_CUS = 5 };
enum { GRINQH_KERNEL_AUTO = 0, GRINQH_KERNEL_PER_PLANE = 1, GRINQH_KERNEL_GENERAL = 2 };

/* Infrastructure, not an operation of the paper.  Fill the auto fields
 * (plane_bits, tile_n) of *in into *out after validating it.  Host only.
 * Every other entry point resolves the same way. */
GRINQH_API int grinqh_resolve_desc(const grinqh_layer_desc* in, grinqh_layer_desc* out);

/* Infrastructure, not an operation of the paper: sizes of the packed buffers
 * of a layer (host only), codes K*N*b_max/8 bytes, scales 2*(K/128)*N bytes. */
GRINQH_API int grinqh_packed_bytes(const grinqh_layer_desc* desc, size_t* codes_bytes,
                        size_t* scales_bytes);

/* Offline quantise + nest + pack (Sec. 3.3, App. C.1).
 *   src_kind GRINQH_SRC_FP16_RTN: src = fp16 W[N][K] (torch Linear.weight
 *     layout), src_scales = NULL.  Symmetric RTN at b_max bits per (output,
 *     group of 128 channels), with h = 2^(b_max-1): s = fp16_rne(fp32(max|w|)
 *     / (h - 1)), q = clamp(rne(w/s), -h, h - 1) + h; a group with s == 0
 *     gets q = h.  W must be finite.
 *   src_kind GRINQH_SRC_CODES_U8: src = uint8 codes q[N][K] (q < 2^b_max;
 *     higher bits are ignored) from any base quantiser with the same
 *     offset-binary convention, src_scales = fp16 s[N][K/128] (the method is
 *     quantisation-agnostic, Sec. 3.3).  Codes of the look-up-table format
 *     (grinqh_vmm_lut) have no scales: pass src_scales = packed_scales = NULL.
 *   Outputs: packed_codes (K*N*b_max/8 bytes, layout above), packed_scales
 *   (fp16 [K/128][N]).  Inputs and outputs must not overlap. */
GRINQH_API int grinqh_pack(const grinqh_layer_desc* desc, int src_kind, const void* src,
                const void* src_scales, void* packed_codes, void* packed_scales,
                void* stream);

/* Integer channel counts for a precision distribution P given in basis
 * points (p_0..p_n, each >= 0, summing to 10000; App. A.1).  With
 * U_j = sum_{i>=j} p_i, C_j = floor((U_j*K + 5000)/10000) channels get level
 * >= j; counts_out[j] = C_j - C_{j+1} (n+1 values summing to K).  Host only. */
GRINQH_API int grinqh_topk_counts(int32_t K, int32_t n_levels, const int32_t* p_bp,
                       int32_t* counts_out);
/* (p_bp and counts_out each hold exactly n_levels entries.) */

/* Infrastructure, not an operation of the paper: device workspace needed by
 * grinqh_assign / grinqh_vmm for B tokens.  The present kernels need none and
 * report 0; callers may pass NULL/0. */
GRINQH_API int grinqh_workspace_bytes(const grinqh_layer_desc* desc, int32_t B, size_t* bytes);

/* Offline threshold calibration (Sec. 3.2 calibration of the thresholds;
 * App. A.1).  x: fp16 [S][K] (device) calibration activations, one sample per
 * row, finite; p_bp: host int32 p_0..p_n in basis points (each >= 0, summing
 * to 10000; exactly n_levels entries are read).  For each sample and each
 * k = 1..n (n = n_levels-1) the sample threshold is the type-7 sample
 * quantile of |x| at q_k = U_k / 10000, U_k = p_0 + .. + p_(k-1): with the K
 * magnitudes sorted ascending a_0 <= .. <= a_(K-1), h = (K-1) U_k / 10000 is
 * split exactly into lo = floor(h) and frac = (h - lo) as a float64 quotient
 * of integers, and the threshold is a_lo + frac * (a_(lo+1) - a_lo) in
 * float64 (a_(lo+1) = a_lo at lo = K-1).  theta_k is the float64 mean of the
 * sample thresholds, summed in sample order, rounded to fp32.
 *   per_sample: device float64 [S][n] scratch, written (8-byte aligned).
 *   theta: device fp32 [n] out.  Requires 1 <= S <= 65535, K <= 16384. */
GRINQH_API int grinqh_calibrate(const grinqh_layer_desc* desc, const void* x, int32_t S,
                                const int32_t* p_bp, double* per_sample, float* theta,
                                void* stream);

/* grinqh_calibrate for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the per-sample scratch lives in a static device array of the library
 * (1 MiB, float64, each GPU holds its own until the process ends), so the
 * caller passes no workspace.  Arguments and result as grinqh_calibrate;
 * S * (n_levels - 1) must not exceed 131072 (GRINQH_ESIZE otherwise).  No
 * entry point here allocates; calls that overlap on one GPU share the
 * scratch and race, so keep them in one stream (or serialise them). */
GRINQH_API int grinqh_calibrate_noalloc(const grinqh_layer_desc* desc, const void* x, int32_t S,
                                        const int32_t* p_bp, float* theta, void* stream);

/* Per-token precision assignment (Sec. 3.1; App. A.1).
 *   x: fp16 [B][K] (device), finite.
 *   mode GRINQH_ASSIGN_THRESHOLD: thresholds = host fp32 theta_1..theta_n
 *     (exactly n = n_levels-1 entries are read), non-decreasing, not NaN
 *     (+inf allowed); channel k gets the level l with |x_k| in
 *     [theta_l, theta_{l+1}), theta_0 = 0, theta_{n+1} = +inf, |x| compared
 *     in fp32.  counts = NULL.
 *   mode GRINQH_ASSIGN_TOPK: counts = host int32 c_0..c_n (exactly n_levels
 *     entries are read) summing to K (e.g. from grinqh_topk_counts).
 *     Channels are ordered by |x| descending, ties by lower index; the first
 *     c_n get level n, the next c_{n-1} level n-1, and so on.
 *     thresholds = NULL.  Requires K <= 16384.
 *   level_map: uint8 [B][K] (device), the level index per channel. */
GRINQH_API int grinqh_assign(const grinqh_layer_desc* desc, int mode, const void* x, int32_t B,
                  const float* thresholds, const int32_t* counts, uint8_t* level_map,
                  void* workspace, size_t ws_bytes, void* stream);

/* Nested-precision decode VMM (Sec. 3.3 reconstruction; App. C.1).
 *   y[t][n] = sum_k x[t][k] * w_hat(k, n), with w_hat = s*(q_b*2^(b_max-b)
 *   + phi - 2^(b_max-1)) for the b = level_bits[level_map[t][k]] most
 *   significant bits q_b of the code, phi = 2^(b_max-b-1) for 0 < b < b_max,
 *   phi = 0 at b = b_max, and channels at level 0 skipped.  Only the first b*T/8 bytes of each of a channel's
 *   rows are read; for B > 1 the deepest level over the B tokens is read once
 *   and each token uses its own prefix of it.
 *   x: fp16 [B][K]; level_map: uint8 [B][K], values < n_levels (a larger
 *   value is read as the top level); y: fp32 [B][N]; 1 <= B <= 4.
 *   flags: 0 -> y is overwritten (cleared by one extra launch before the
 *   VMM, whose workgroups add their partial sums into y); GRINQH_VMM_ACCUMULATE
 *   -> y += result (the caller initialised y, e.g. once for many VMMs into
 *   one buffer).  Accumulation order across K is not fixed, so y is
 *   reproducible to rounding, not bit for bit.  Any other flag bit is
 *   GRINQH_EINVAL. */
GRINQH_API int grinqh_vmm(const grinqh_layer_desc* desc, const void* packed_codes,
               const void* packed_scales, const void* x, const uint8_t* level_map,
               int32_t B, float* y, int32_t flags, void* workspace, size_t ws_bytes,
               void* stream);

/* The VMM with the threshold assignment of Sec. 3.1 fused into it: each
 * channel's level is graded inside the kernel from |x| and `thresholds`
 * (host fp32 theta_1..theta_n, rules as in grinqh_assign), so no level map
 * is read; if level_map_out is not NULL the levels are also written there
 * (uint8 [B][K]).  Other arguments as grinqh_vmm. */
GRINQH_API int grinqh_vmm_threshold(const grinqh_layer_desc* desc, const void* packed_codes,
                         const void* packed_scales, const void* x, int32_t B,
                         const float* thresholds, uint8_t* level_map_out, float* y,
                         int32_t flags, void* workspace, size_t ws_bytes, void* stream);

/* The batch-1 VMM with the exact top-k assignment of App. A.1 fused into
 * it: every workgroup selects the token's per-level cuts from the whole x
 * (the counts[j] channels of largest |x| at level j from the top, ties to the
 * lower channel index, exactly as grinqh_assign in top-k mode) and grades its
 * own channels against them, so no level map is read and no assignment
 * launch is needed.  counts: int32 [n_levels] (host), summing to K.
 * Requires B = 1, K <= 16384, 2-bit planes with tile_n in {256, 512, 1024}
 * (GRINQH_EUNSUPPORTED otherwise: grinqh_assign + grinqh_vmm serve the
 * other cases) and x 16-byte aligned.  level_map_out, if not NULL, receives
 * the levels (uint8 [K]).  Other arguments as grinqh_vmm.
 * Every workgroup repeats the selection, so on Llama3-8B-sized layers this
 * is slower than grinqh_assign (top-k) followed by grinqh_vmm; it serves
 * callers that cannot keep a level map or launch the assignment apart. */
GRINQH_API int grinqh_vmm_topk(const grinqh_layer_desc* desc, const void* packed_codes,
                               const void* packed_scales, const void* x, int32_t B,
                               const int32_t* counts, uint8_t* level_map_out, float* y,
                               int32_t flags, void* workspace, size_t ws_bytes, void* stream);

/* Prefill, the stage-decoupled dense path (Sec. 3: prefill reads the weights
 * at the fixed top precision; Sec. 4 "Prefill vs. Decoding Evaluation"): for
 * M tokens at once, every channel at all b_max bits,
 *   Y[m][n] = sum_k X[m][k] * w_hat[n][k],  w_hat = s[k/128][n] * (q[n][k] - 2^(b_max-1)),
 * with each w_hat rounded once to fp16 (the dequantised weight of a dense
 * fp16 GEMM), fp16 x fp16 products and fp32 accumulation: per element
 * |Y - exact| <= (2^-11 + K 2^-24) sum_k |X[m][k]| |w_hat[n][k]|.  Reads the
 * same packed buffers as grinqh_vmm (any plane_bits and tile_n).
 *   x: fp16 [M][K] (device, 16-byte aligned), finite; y: fp32 [M][N]
 *   (device, 4-byte aligned); 1 <= M <= 2^24.
 *   flags: 0 -> y is overwritten; GRINQH_VMM_ACCUMULATE -> y += result.
 * The summation order is fixed, so a result is reproducible bit for bit. */
GRINQH_API int grinqh_prefill(const grinqh_layer_desc* desc, const void* packed_codes,
                              const void* packed_scales, const void* x, int32_t M, float* y,
                              int32_t flags, void* stream);

/* Infrastructure, not an operation of the paper: number of fp16 table
 * entries of a layer's look-up tables (host only), N * sum over levels
 * l >= 1 of 2^b_l. */
GRINQH_API int grinqh_lut_entries(const grinqh_layer_desc* desc, size_t* entries);

/* Decode VMM over non-uniform nested weights read through look-up tables
 * (Sec. 3.3: any quantiser with the nested property, e.g. nested k-means
 * weights, whose levels are centred so no midpoint bias applies; appendix
 * on nested weight formats).  Codes are packed as for grinqh_vmm (codes
 * source, no scales).
 *   luts: fp16, for each level l = 1..n (b = b_l bits) a table [N][2^b],
 *   the tables consecutive in level order: level l's table starts at
 *   element N * sum_{1 <= i < l} 2^b_i (16-byte aligned base).
 *   y[t][n] = sum_k x[t][k] * luts_l[n][q_b], l = level_map[t][k] (a value
 *   >= n_levels is read as the top level), q_b = the b leading bits of the
 *   b_max-bit code; level 0 skipped.
 *   x: fp16 [B][K]; level_map: uint8 [B][K]; y: fp32 [B][N]; 1 <= B <= 65535.
 *   flags: 0 -> y is overwritten; GRINQH_VMM_ACCUMULATE -> y += result.
 *   Partial sums meet in atomics: reproducible to rounding, not bit for bit. */
GRINQH_API int grinqh_vmm_lut(const grinqh_layer_desc* desc, const void* packed_codes,
                              const void* luts, const void* x, const uint8_t* level_map,
                              int32_t B, float* y, int32_t flags, void* stream);

/* The LUT VMM with the threshold assignment of Sec. 3.1 fused into it: each
 * channel's level is graded inside the kernel from |x| and `thresholds`
 * (host fp32 theta_1..theta_n, rules as in grinqh_assign), so no level map
 * is read; if level_map_out is not NULL the levels are also written there
 * (uint8 [B][K], device).  Other arguments as grinqh_vmm_lut. */
GRINQH_API int grinqh_vmm_lut_threshold(const grinqh_layer_desc* desc, const void* packed_codes,
                                        const void* luts, const void* x, int32_t B,
                                        const float* thresholds, uint8_t* level_map_out, float* y,
                                        int32_t flags, void* stream);

/* Infrastructure for tests and measurements, not an operation of the paper:
 * process-wide overrides of launch choices that never change results beyond
 * rounding order.  Value 0 restores each launcher's own choice.
 *   GRINQH_OPT_VMM_KERNEL: GRINQH_KERNEL_PER_PLANE or GRINQH_KERNEL_GENERAL
 *     runs that kernel for B = 1 too (the batch kernels otherwise).
 *   GRINQH_OPT_GROUPS_PER_WG: 1..4 groups of 128 channels per workgroup
 *     (kernels that take fewer use their maximum).
 *   GRINQH_OPT_PREFILL_TILE: 1, 2, 3 = 256x256, 256x128, 128x128 prefill tiles.
 *   GRINQH_OPT_LUT_GROUPS: 1..16 groups per workgroup of the LUT VMM.
 *   GRINQH_OPT_PREFILL_CUS: 1..4096, the CU count the prefill balances its
 *     rounds of 256x256 tiles for (0: the device's).
 * Returns GRINQH_EINVAL for an unknown option or a value out of range.  The
 * setting is read when a call enqueues its kernels; set it between calls. */
GRINQH_API int grinqh_set_option(int option, int value);

/* Measurement infrastructure, not an operation of the paper: read `bytes` of
 * device memory at src (16-byte aligned; a positive multiple of 2 MiB) with
 * non-temporal 16-byte loads, eight in flight per lane, as fast as the chip
 * streams them, and XOR a fold of the data into *sink (device uint32).  It
 * gives the measured streaming-read ceiling the VMM's bandwidth is compared
 * with. */
GRINQH_API int grinqh_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream);

/* Infrastructure, not an operation of the paper: the message of the last
 * failing call on this thread ("" if none), valid until that thread's next
 * call. */
GRINQH_API const char* grinqh_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GRINQH_H */
