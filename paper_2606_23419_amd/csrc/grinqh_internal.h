// Internal definitions shared by the libgrinqh translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/grinqh.h"

namespace grinqh {

constexpr int kGroup = 128;       // quantisation group along K
constexpr int kMaxLevels = GRINQH_MAX_LEVELS;
constexpr int kMaxB = 4;          // tokens per VMM call

// A validated, resolved layer descriptor, passed to kernels by value.
struct Layer {
  int K, N, n_levels;
  int u;            // plane width in bits (1 or 2)
  int bmax;         // stored code width b_max (the top level's bits): 4, 6 or 8
  int P;            // number of stored planes, bmax/u
  int T;            // outputs per tile
  int RB;           // bytes of one stored row, T * bmax / 8
  float sfac;       // 2^(bmax - 8): kernels work in 8-bit code units
  int tiles;        // N / T
  int groups;       // K / 128
  int bits[kMaxLevels];    // b_l
  int planes[kMaxLevels];  // b_l / u: planes read at level l
  // planes[l] in bits 4l..4l+3.  Kernels index levels per lane; a by-value
  // array indexed that way is read from kernel-argument memory one lane at a
  // time, while this word is one scalar register pair.
  uint64_t planes_packed;
};

__host__ __device__ __forceinline__ int level_planes(uint64_t packed, int level) {
  return (int)((packed >> (4 * level)) & 0xFu);
}

struct Thresholds {
  float theta[kMaxLevels - 1];   // theta_1 .. theta_n, then +inf (kernels compare all)
  int n;
};

// Quantile positions for threshold calibration: ascending ranks lo/hi and
// the interpolation fraction, per threshold.
struct QuantilePos {
  int lo[kMaxLevels - 1], hi[kMaxLevels - 1];
  double frac[kMaxLevels - 1];
  int n;
};

// Per-output look-up tables of the LUT VMM: level l's table [N][2^b_l]
// starts at element offset[l] of the table array; cum[l] = sum of 2^b_i over
// 1 <= i < l (the level's position within one output's entries).
struct LutDesc {
  long offset[kMaxLevels];
  int cum[kMaxLevels];
  int entries;      // sum over levels >= 1 of 2^b_l
  int quad_pad;     // LDS padding (entries) after each 16-output quad of a level's tables: 16 or 0
};

struct TopkCuts {
  int cum[kMaxLevels];           // cum[j] = C_{j+1}: channels at level >= j+1
  int n;
};

// fp16 <-> fp32 helpers on raw bits.
__device__ __forceinline__ float h2f(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}
__device__ __forceinline__ uint16_t f2h_rn(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// Launch overrides set through grinqh_set_option (tests and measurements);
// 0 everywhere means each launcher's own choice.  Read with relaxed loads.
struct Options {
  int vmm_kernel;       // GRINQH_KERNEL_*: the batch-1 kernel
  int groups_per_wg;    // groups of 128 channels per workgroup, where a kernel allows it
  int prefill_tile;     // 1..3: 256x256, 256x128, 128x128
  int lut_groups;       // groups per workgroup of the LUT VMM
  int prefill_cus;      // CUs the prefill counts its rounds in (0: the device's)
};
int option(int Options::*field);

// Error reporting (per thread), defined in grinqh_api.hip.
int fail(int status, const char* fmt, ...);
int check_launch(const char* what);

// Kernel launchers (defined next to their kernels).
int launch_pack(const Layer& L, int src_kind, const void* src, const void* src_scales,
                void* packed_codes, void* packed_scales, hipStream_t s);
int launch_assign_threshold(const Layer& L, const void* x, int B, const Thresholds& th,
                            uint8_t* level_map, hipStream_t s);
int launch_assign_topk(const Layer& L, const void* x, int B, const TopkCuts& cuts,
                       uint8_t* level_map, hipStream_t s);
int launch_calibrate(const Layer& L, const void* x, int S, const QuantilePos& qp,
                     double* per_sample, float* theta, hipStream_t s);
// float64 entries of the static per-sample scratch of grinqh_calibrate_noalloc
constexpr int kCalibScratch = 1 << 17;   // 1 MiB
int launch_calibrate_noalloc(const Layer& L, const void* x, int S, const QuantilePos& qp,
                             float* theta, hipStream_t s);
bool vmm_pp_supported(const Layer& L, int B);
// levels from the level map, or graded in the kernel from thresholds (th) or
// the exact top-k cuts of x (tk), then optionally written to level_map_out
int launch_vmm_pp(const Layer& L, const void* codes, const void* scales, const void* x,
                  const uint8_t* level_map, const Thresholds* th, const TopkCuts* tk,
                  uint8_t* level_map_out, float* y, hipStream_t s);
// the batch-1 VMM with exact top-k assignment in its prologue (B = 1)
int launch_vmm_topk(const Layer& L, const void* codes, const void* scales, const void* x,
                    const TopkCuts& cuts, uint8_t* level_map_out, float* y, int accumulate,
                    hipStream_t s);
bool vmm_dot2_supported(const Layer& L);
int launch_vmm_dot2(const Layer& L, const void* codes, const void* scales, const void* x,
                    const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out,
                    int B, float* y, hipStream_t s);
int launch_vmm(const Layer& L, const void* codes, const void* scales, const void* x,
               const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out,
               int B, float* y, int accumulate, hipStream_t s);
int launch_prefill(const Layer& L, const void* codes, const void* scales, const void* x, int M,
                   float* y, int accumulate, hipStream_t s);
int lut_desc(const Layer& L, LutDesc* D);
int launch_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t s);
// level_map == nullptr with th != nullptr: levels graded from x in the kernel,
// written to level_map_out if that is not null
int launch_vmm_lut(const Layer& L, const void* codes, const void* luts, const void* x,
                   const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out, int B,
                   float* y, int accumulate, hipStream_t s);

}  // namespace grinqh
