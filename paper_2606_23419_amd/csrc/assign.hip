// Per-token precision assignment (Sec. 3.1 threshold grading; App. A.1 top-p
// partition of |x| into the fractions P).
#include "grinqh_internal.h"

namespace grinqh {

// |x| of an fp16 value as an integer key: same order as |x| for finite x.
__device__ __forceinline__ uint32_t mag_key(uint16_t b) { return b & 0x7FFFu; }

// Level = number of interior thresholds theta_j <= |x| (fp32 compare).  With
// non-decreasing thresholds this is the l with |x| in [theta_l, theta_{l+1}).
__global__ __launch_bounds__(256) void k_assign_threshold(const uint16_t* __restrict__ x,
                                                          uint8_t* __restrict__ lm, long total,
                                                          Thresholds th) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const float a = fabsf(h2f(x[i]));
  int l = 0;
#pragma unroll
  for (int j = 0; j < kMaxLevels - 1; ++j) l += (j < th.n && a >= th.theta[j]) ? 1 : 0;
  lm[i] = (uint8_t)l;
}

// Top-k: one workgroup of 1024 threads per token.  For every level j the cut
// is the C_j-th largest key (C_j = channels at level >= j), found by a
// two-digit radix select (8 high bits, then 7 low bits) with LDS histograms
// for all levels at once.  Channels strictly above the cut key are in; of
// the channels equal to it, the lowest indices are in, counted in index order
// with a ballot + mbcnt prefix inside each wave and a scan over waves.
constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;

__global__ __launch_bounds__(kTopkThreads) void k_assign_topk(const uint16_t* __restrict__ x,
                                                              uint8_t* __restrict__ lm, int K,
                                                              TopkCuts cuts) {
  __shared__ uint32_t hist1[256];
  __shared__ uint32_t hist2[kMaxLevels - 1][128];
  __shared__ int cut_bin[kMaxLevels - 1], need_bin[kMaxLevels - 1];
  __shared__ uint32_t cut_key[kMaxLevels - 1];
  __shared__ int need_eq[kMaxLevels - 1];
  __shared__ uint32_t wave_eq[kTopkWaves][kMaxLevels - 1];
  __shared__ uint32_t running[kMaxLevels - 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = cuts.n;
  const uint16_t* xt = x + (size_t)blockIdx.x * K;
  uint8_t* out = lm + (size_t)blockIdx.x * K;

  for (int i = tid; i < 256; i += kTopkThreads) hist1[i] = 0;
  for (int i = tid; i < (kMaxLevels - 1) * 128; i += kTopkThreads) (&hist2[0][0])[i] = 0;
  if (tid < kMaxLevels - 1) running[tid] = 0;
  __syncthreads();

  for (int k = tid; k < K; k += kTopkThreads) atomicAdd(&hist1[mag_key(xt[k]) >> 7], 1u);
  __syncthreads();

  if (tid < n) {
    const int C = cuts.cum[tid];
    int bin = 256, need = 0;
    if (C > 0) {
      int acc = 0;
      for (int b = 255; b >= 0; --b) {
        const int h = (int)hist1[b];
        if (acc + h >= C) { bin = b; need = C - acc; break; }
        acc += h;
      }
    }
    cut_bin[tid] = bin;
    need_bin[tid] = need;
  }
  __syncthreads();

  for (int k = tid; k < K; k += kTopkThreads) {
    const uint32_t key = mag_key(xt[k]);
    const int bin = (int)(key >> 7);
    for (int j = 0; j < n; ++j)
      if (bin == cut_bin[j]) atomicAdd(&hist2[j][key & 127u], 1u);
  }
  __syncthreads();

  if (tid < n) {
    uint32_t ck = 0x8000u;   // above every key: nobody is in
    int need = 0;
    if (cut_bin[tid] < 256) {
      int acc = 0;
      for (int s = 127; s >= 0; --s) {
        const int h = (int)hist2[tid][s];
        if (acc + h >= need_bin[tid]) { ck = ((uint32_t)cut_bin[tid] << 7) | (uint32_t)s; need = need_bin[tid] - acc; break; }
        acc += h;
      }
    }
    cut_key[tid] = ck;
    need_eq[tid] = need;
  }
  __syncthreads();

  for (int base = 0; base < K; base += kTopkThreads) {
    const int k = base + tid;
    const bool valid = k < K;
    const uint32_t key = valid ? mag_key(xt[k]) : 0u;
    uint32_t pre[kMaxLevels - 1];
    bool eq[kMaxLevels - 1];
#pragma unroll
    for (int j = 0; j < kMaxLevels - 1; ++j) {
      eq[j] = valid && j < n && key == cut_key[j];
      const uint64_t bal = __ballot(eq[j]);
      pre[j] = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                         __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
      if (lane == 0) wave_eq[wave][j] = (uint32_t)__popcll(bal);
    }
    __syncthreads();
    int lvl = 0;
#pragma unroll
    for (int j = 0; j < kMaxLevels - 1; ++j) {
      if (j >= n) break;
      uint32_t before = running[j];
      for (int w = 0; w < wave; ++w) before += wave_eq[w][j];
      const bool in = valid && (key > cut_key[j] || (eq[j] && (int)(before + pre[j]) < need_eq[j]));
      lvl += in ? 1 : 0;
    }
    __syncthreads();
    if (tid < n) {
      uint32_t tot = 0;
      for (int w = 0; w < kTopkWaves; ++w) tot += wave_eq[w][tid];
      running[tid] += tot;
    }
    if (valid) out[k] = (uint8_t)lvl;
    __syncthreads();
  }
}

int launch_assign_threshold(const Layer& L, const void* x, int B, const Thresholds& th,
                            uint8_t* level_map, hipStream_t s) {
  const long total = (long)B * L.K;
  hipLaunchKernelGGL(k_assign_threshold, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     (const uint16_t*)x, level_map, total, th);
  return check_launch("assign (threshold)");
}

int launch_assign_topk(const Layer& L, const void* x, int B, const TopkCuts& cuts,
                       uint8_t* level_map, hipStream_t s) {
  hipLaunchKernelGGL(k_assign_topk, dim3((unsigned)B), dim3(kTopkThreads), 0, s,
                     (const uint16_t*)x, level_map, L.K, cuts);
  return check_launch("assign (top-k)");
}

}  // namespace grinqh
