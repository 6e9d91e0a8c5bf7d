// Nested-precision decode VMM (Sec. 3.3 reconstruction with the midpoint
// bias; App. C.1 sparse bit-loading), first version: correctness first.
//
// Grid: (tiles x K-splits, tokens).  A workgroup owns one tile of T outputs
// and a range of whole groups.  Its 256 threads form lane groups of T/16
// lanes; each lane holds 16 consecutive outputs of the tile.  Lane group lg
// takes the rows lg, lg + nlg, ... of every group, reads the first
// planes[level] planes of each row (a contiguous prefix), rebuilds the
// truncated code t = q_b << (8 - b) and accumulates x_k * t.  Per group,
//   y_n += s_{g,n} * (sum_k x_k t_{k,n} + beta_g),
//   beta_g = sum_{k in g, level > 0} x_k (phi_b - 128),
// which is sum_k x_k * s * (t + phi - 128) with the scale factored out.
// Lane groups are reduced through LDS and added into y with atomics.
#include "grinqh_internal.h"

namespace grinqh {

constexpr int kVmmThreads = 256;

__device__ __forceinline__ float midpoint_minus_offset(int b, int bmax) {
  // phi_b - 128 in 8-bit code units: phi_b = 2^(7-b) for 0 < b < b_max and
  // 0 at b = b_max (a b_max-bit code is the top b_max bits of an 8-bit one)
  return (b < bmax ? (float)(1 << (7 - b)) : 0.0f) - 128.0f;
}

__global__ __launch_bounds__(256) void k_zero(float* __restrict__ y, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = 0.0f;
}

template <int U>
__global__ __launch_bounds__(kVmmThreads) void k_vmm_v0(
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ lm, float* __restrict__ y,
    Layer L, int groups_per_split, int fused, Thresholds th, uint8_t* __restrict__ lm_out) {
  constexpr uint32_t MASK = (1u << U) - 1u;
  __shared__ float red[kVmmThreads * 16];

  const int t = blockIdx.x % L.tiles;
  const int split = blockIdx.x / L.tiles;
  const int tok = blockIdx.y;
  const int lanes = L.T / 16;
  const int nlg = kVmmThreads / lanes;
  const int lg = threadIdx.x / lanes, li = threadIdx.x % lanes;
  const int g0 = split * groups_per_split;
  const int g1 = min(g0 + groups_per_split, L.groups);
  const uint16_t* xt = x + (size_t)tok * L.K;
  const int plane_bytes = L.T * U / 8;

  float yacc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) yacc[e] = 0.0f;

  for (int g = g0; g < g1; ++g) {
    float acc[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
    float beta = 0.0f;
    for (int r = lg; r < kGroup; r += nlg) {
      const int k = g * kGroup + r;
      const float xv = h2f(xt[k]);
      int lvl;
      if (fused) {
        const float a = fabsf(xv);
        lvl = 0;
        for (int j = 0; j < th.n; ++j) lvl += a >= th.theta[j] ? 1 : 0;
        if (lm_out && t == 0 && li == 0) lm_out[(size_t)tok * L.K + k] = (uint8_t)lvl;
      } else {
        lvl = min((int)lm[(size_t)tok * L.K + k], L.n_levels - 1);
      }
      if (lvl == 0) continue;
      const int d = level_planes(L.planes_packed, lvl);
      const int b = d * U;
      const uint8_t* row = codes + ((size_t)t * L.K + k) * L.RB;
      uint32_t code[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) code[e] = 0u;
      for (int j = 0; j < d; ++j) {
        uint32_t word;
        if (U == 2) word = *(const uint32_t*)(row + (size_t)j * plane_bytes + li * 4);
        else word = *(const uint16_t*)(row + (size_t)j * plane_bytes + li * 2);
#pragma unroll
        for (int e = 0; e < 16; ++e) code[e] = (code[e] << U) | ((word >> (e * U)) & MASK);
      }
      const int sh = 8 - b;
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e] = fmaf(xv, (float)(code[e] << sh), acc[e]);
      beta = fmaf(xv, midpoint_minus_offset(b, L.bmax), beta);
    }
    const uint16_t* sg = scales + (size_t)g * L.N + (size_t)t * L.T + li * 16;
#pragma unroll
    for (int e = 0; e < 16; ++e) yacc[e] = fmaf(h2f(sg[e]), acc[e] + beta, yacc[e]);
  }

#pragma unroll
  for (int e = 0; e < 16; ++e) red[lg * L.T + li * 16 + e] = yacc[e];
  __syncthreads();
  float* yt = y + (size_t)tok * L.N + (size_t)t * L.T;
  for (int o = threadIdx.x; o < L.T; o += kVmmThreads) {
    float s = 0.0f;
    for (int q = 0; q < nlg; ++q) s += red[q * L.T + o];
    atomicAdd(&yt[o], s * L.sfac);   // 8-bit code units -> b_max units
  }
}

// Streaming read for the measured read ceiling (measurement infrastructure):
// workgroup b reads bytes [b*chunk, (b+1)*chunk) in 16-byte pieces per lane,
// eight loads in flight, and folds them with XOR; each wave leaves its fold
// in sink with one atomic XOR so the loads cannot be dropped.
constexpr int kStreamThreads = 256, kStreamRing = 8;

__global__ __launch_bounds__(kStreamThreads) void k_stream_read(const uint8_t* __restrict__ src,
                                                               uint32_t chunk, int n_it,
                                                               uint32_t* __restrict__ sink) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr int STEP = kStreamThreads * 16;
  const uint8_t* p = src + (size_t)blockIdx.x * chunk + threadIdx.x * 16;
  u32x4 r[kStreamRing];
  uint32_t acc = 0u;
#pragma unroll
  for (int i = 0; i < kStreamRing - 1; ++i)
    r[i] = __builtin_nontemporal_load((const u32x4*)(p + (size_t)min(i, n_it - 1) * STEP));
  for (int it = 0; it < n_it; it += kStreamRing) {
#pragma unroll
    for (int i = 0; i < kStreamRing; ++i) {
      const int j = min(it + i + kStreamRing - 1, n_it - 1);
      r[(i + kStreamRing - 1) % kStreamRing] = __builtin_nontemporal_load((const u32x4*)(p + (size_t)j * STEP));
      if (it + i < n_it) acc ^= r[i].x ^ r[i].y ^ r[i].z ^ r[i].w;
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  for (int o = 32; o > 0; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
  if ((threadIdx.x & 63) == 0) atomicXor(sink, acc);
}

int launch_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t s) {
  // 512 workgroups, each a contiguous chunk of bytes / 512 (a multiple of
  // 4 KiB below 4 GiB: the caller passes a multiple of 2 MiB below 2 TiB)
  constexpr size_t kStep = (size_t)kStreamThreads * 16;
  constexpr int nwg = 512;
  const size_t chunk = bytes / nwg;
  hipLaunchKernelGGL(k_stream_read, dim3((unsigned)nwg), dim3(kStreamThreads), 0, s,
                     (const uint8_t*)src, (uint32_t)chunk, (int)(chunk / kStep), sink);
  return check_launch("stream read");
}

int launch_vmm(const Layer& L, const void* codes, const void* scales, const void* x,
               const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out,
               int B, float* y, int accumulate, hipStream_t s) {
  if (!accumulate) {
    const long n = (long)B * L.N;
    hipLaunchKernelGGL(k_zero, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, y, n);
    int st = check_launch("vmm zero-fill");
    if (st) return st;
  }
  const int force = option(&Options::vmm_kernel);   // tests and measurements
  const bool want_dot2 = force == GRINQH_KERNEL_PER_PLANE, want_v0 = force == GRINQH_KERNEL_GENERAL;
  if (!want_dot2 && !want_v0 && vmm_pp_supported(L, B))
    return launch_vmm_pp(L, codes, scales, x, level_map, th, nullptr, level_map_out, y, s);
  if (!want_v0 && vmm_dot2_supported(L))
    return launch_vmm_dot2(L, codes, scales, x, level_map, th, level_map_out, B, y, s);
  // about 512 workgroups per token over the whole chip
  int ksplit = (512 + L.tiles - 1) / L.tiles;
  if (ksplit > L.groups) ksplit = L.groups;
  const int gps = (L.groups + ksplit - 1) / ksplit;
  ksplit = (L.groups + gps - 1) / gps;
  const dim3 grid((unsigned)(L.tiles * ksplit), (unsigned)B);
  Thresholds none{};
  const int fused = th != nullptr;
  if (L.u == 2)
    hipLaunchKernelGGL(k_vmm_v0<2>, grid, dim3(kVmmThreads), 0, s, (const uint8_t*)codes,
                       (const uint16_t*)scales, (const uint16_t*)x, level_map, y, L, gps, fused,
                       fused ? *th : none, level_map_out);
  else
    hipLaunchKernelGGL(k_vmm_v0<1>, grid, dim3(kVmmThreads), 0, s, (const uint8_t*)codes,
                       (const uint16_t*)scales, (const uint16_t*)x, level_map, y, L, gps, fused,
                       fused ? *th : none, level_map_out);
  return check_launch("vmm");
}

int launch_vmm_topk(const Layer& L, const void* codes, const void* scales, const void* x,
                    const TopkCuts& cuts, uint8_t* level_map_out, float* y, int accumulate,
                    hipStream_t s) {
  if (!accumulate) {
    hipLaunchKernelGGL(k_zero, dim3((unsigned)((L.N + 255) / 256)), dim3(256), 0, s, y, (long)L.N);
    int st = check_launch("vmm zero-fill");
    if (st) return st;
  }
  return launch_vmm_pp(L, codes, scales, x, nullptr, nullptr, &cuts, level_map_out, y, s);
}

}  // namespace grinqh
