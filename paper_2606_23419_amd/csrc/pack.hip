// Offline quantise + nest + pack (Sec. 3.3 "Storage Layout and Weight
// Loading"; App. C.1 "Sparse bit-loading", "Bit-packing").
//
// Two kernels: one wave per (output, group) computes the RTN scale; then one
// thread per (tile, 32-output chunk, channel) quantises its 32 codes and
// scatters their fields into the u-bit planes of the channel's row.
#include "grinqh_internal.h"

namespace grinqh {

// s = fp16_rne(fp32(max|w|) / qmax) per (output n, group g), written [g][n];
// qmax = 2^(b_max-1) - 1 (127 at 8 bits).
__global__ __launch_bounds__(256) void k_rtn_scales(const uint16_t* __restrict__ W,
                                                    uint16_t* __restrict__ scales, int N, int K,
                                                    float qmax) {
  const int G = K / kGroup;
  const long wave = ((long)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wave >= (long)N * G) return;
  const int n = (int)(wave / G), g = (int)(wave % G);
  const uint16_t* p = W + (size_t)n * K + (size_t)g * kGroup;
  float a = fmaxf(fabsf(h2f(p[lane])), fabsf(h2f(p[lane + 64])));
  for (int off = 32; off > 0; off >>= 1) a = fmaxf(a, __shfl_xor(a, off));
  if (lane == 0) scales[(size_t)g * N + n] = f2h_rn(__fdiv_rn(a, qmax));
}

// Externally quantised codes: scales arrive [n][g] and are stored [g][n].
__global__ __launch_bounds__(256) void k_transpose_scales(const uint16_t* __restrict__ src,
                                                          uint16_t* __restrict__ dst, int N, int G) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)N * G) return;
  const int g = (int)(i / N), n = (int)(i % N);
  dst[i] = src[(size_t)n * G + g];
}

// b_max-bit codes (b_max = L.bmax), L.P = b_max/U planes per row of L.RB bytes.
template <int U>
__global__ __launch_bounds__(256) void k_pack(const void* __restrict__ src, int from_fp16,
                                              const uint16_t* __restrict__ scales,
                                              uint8_t* __restrict__ out, Layer L) {
  constexpr int P = 8 / U;              // planes of the widest (8-bit) code
  constexpr int WORDS = U;              // 32 outputs * U bits = U dwords per plane
  constexpr uint32_t MASK = (1u << U) - 1u;
  const int chunks = L.T / 32;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long total = (long)L.tiles * chunks * L.K;
  if (idx >= total) return;
  const int k = (int)(idx % L.K);
  const long r = idx / L.K;
  const int c = (int)(r % chunks);
  const int t = (int)(r / chunks);
  const int g = k / kGroup;

  uint32_t plane[P][WORDS];
#pragma unroll
  for (int j = 0; j < P; ++j)
#pragma unroll
    for (int w = 0; w < WORDS; ++w) plane[j][w] = 0u;

  const int half = 1 << (L.bmax - 1);
  const float lo = (float)-half, hi = (float)(half - 1);
#pragma unroll 4
  for (int e = 0; e < 32; ++e) {
    const int n = t * L.T + c * 32 + e;
    uint32_t q;
    if (from_fp16) {
      const float s = h2f(scales[(size_t)g * L.N + n]);
      const float w = h2f(((const uint16_t*)src)[(size_t)n * L.K + k]);
      if (s == 0.0f) {
        q = (uint32_t)half;
      } else {
        float rq = rintf(__fdiv_rn(w, s));
        rq = fminf(fmaxf(rq, lo), hi);
        q = (uint32_t)((int)rq + half);
      }
    } else {
      q = ((const uint8_t*)src)[(size_t)n * L.K + k];
    }
    // left-align the b_max-bit code in 8 bits: plane j's field is then the
    // same bit slice for every b_max (bits above b_max of a given code drop out)
    q = (q << (8 - L.bmax)) & 0xFFu;
    const int bit = e * U;
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const uint32_t field = (q >> (8 - (j + 1) * U)) & MASK;
      plane[j][bit >> 5] |= field << (bit & 31);
    }
  }
  uint8_t* row = out + ((size_t)t * L.K + k) * L.RB;
  const int plane_bytes = L.T * U / 8;
#pragma unroll
  for (int j = 0; j < P; ++j) {
    if (j >= L.P) break;
    uint32_t* dst = (uint32_t*)(row + (size_t)j * plane_bytes + (size_t)c * 32 * U / 8);
#pragma unroll
    for (int w = 0; w < WORDS; ++w) dst[w] = plane[j][w];
  }
}

int launch_pack(const Layer& L, int src_kind, const void* src, const void* src_scales,
                void* packed_codes, void* packed_scales, hipStream_t s) {
  const bool from_fp16 = src_kind == GRINQH_SRC_FP16_RTN;
  if (from_fp16) {
    const long waves = (long)L.N * L.groups;
    const long blocks = (waves * 64 + 255) / 256;
    hipLaunchKernelGGL(k_rtn_scales, dim3((unsigned)blocks), dim3(256), 0, s,
                       (const uint16_t*)src, (uint16_t*)packed_scales, L.N, L.K,
                       (float)((1 << (L.bmax - 1)) - 1));
  } else if (src_scales) {   // codes without scales: the look-up-table format
    const long n = (long)L.N * L.groups;
    hipLaunchKernelGGL(k_transpose_scales, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint16_t*)src_scales, (uint16_t*)packed_scales, L.N, L.groups);
  }
  int st = check_launch("pack scales");
  if (st) return st;
  const long total = (long)L.tiles * (L.T / 32) * L.K;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (L.u == 2)
    hipLaunchKernelGGL(k_pack<2>, grid, dim3(256), 0, s, src, (int)from_fp16,
                       (const uint16_t*)packed_scales, (uint8_t*)packed_codes, L);
  else
    hipLaunchKernelGGL(k_pack<1>, grid, dim3(256), 0, s, src, (int)from_fp16,
                       (const uint16_t*)packed_scales, (uint8_t*)packed_codes, L);
  return check_launch("pack codes");
}

}  // namespace grinqh
