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

// Top-k: one workgroup of 1024 threads per token, every key in registers
// (K <= 16384).  For every level j the cut is the C_j-th largest key (C_j =
// channels at level >= j).  A two-digit radix select finds all cuts at once:
// per-wave LDS histograms of the high 8 bits, a parallel suffix scan to find
// the bin holding each cut, then 128-bin histograms of the low 7 bits inside
// those bins.  Channels strictly above the cut key are in.  Of the channels
// equal to it, the first ones in index order are in: per-(chunk, wave) ballots
// of key == cut are stored, and one wave per level walks them in index order
// to find the channel index where the count reaches the number still needed.
constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kTopkPer = 16;                     // keys per thread
constexpr int kTopkMaxK = kTopkThreads * kTopkPer;
constexpr int kCuts = kMaxLevels - 1;

__device__ __forceinline__ uint32_t incl_scan64(uint32_t v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(v, off);
    if (lane >= off) v += o;
  }
  return v;
}

// Position (0..63) of the r-th set bit (r >= 1) of m.
__device__ __forceinline__ int nth_set_bit(uint64_t m, int r) {
  int pos = 0;
#pragma unroll
  for (int w = 32; w > 0; w >>= 1) {
    const uint64_t low = m & ((w == 64 ? ~0ull : (1ull << w) - 1ull));
    const int c = __popcll(low);
    if (r > c) {
      r -= c;
      m >>= w;
      pos += w;
    } else {
      m = low;
    }
  }
  return pos;
}

__global__ __launch_bounds__(kTopkThreads) void k_assign_topk(const uint16_t* __restrict__ x,
                                                              uint8_t* __restrict__ lm, int K,
                                                              TopkCuts cuts) {
  __shared__ uint32_t s_h1[kTopkWaves][256];
  __shared__ uint32_t s_h2[kCuts][128];
  __shared__ uint32_t s_wsum[kTopkWaves];
  __shared__ int s_cut_bin[kCuts], s_need[kCuts], s_need_eq[kCuts], s_idx_lim[kCuts];
  __shared__ uint32_t s_cut_key[kCuts];
  __shared__ uint64_t s_bal[kTopkPer][kTopkWaves][kCuts];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = cuts.n;
  const int M = (K + kTopkThreads - 1) / kTopkThreads;
  const uint16_t* xt = x + (size_t)blockIdx.x * K;
  uint8_t* out = lm + (size_t)blockIdx.x * K;

  uint32_t key[kTopkPer];
#pragma unroll
  for (int m = 0; m < kTopkPer; ++m) {
    const int k = m * kTopkThreads + tid;
    key[m] = (m < M && k < K) ? mag_key(xt[k]) : 0xFFFFu;   // 0xFFFF: no channel
  }
  for (int i = tid; i < kTopkWaves * 256; i += kTopkThreads) (&s_h1[0][0])[i] = 0u;
  for (int i = tid; i < kCuts * 128; i += kTopkThreads) (&s_h2[0][0])[i] = 0u;
  if (tid < kCuts) {
    s_cut_bin[tid] = 256;
    s_need[tid] = 0;
    s_cut_key[tid] = 0x8000u;   // above every key: nobody is in
    s_need_eq[tid] = 0;
    s_idx_lim[tid] = 0;
  }
  __syncthreads();

  // high-digit histograms, one per wave
#pragma unroll
  for (int m = 0; m < kTopkPer; ++m)
    if (key[m] != 0xFFFFu) atomicAdd(&s_h1[wave][key[m] >> 7], 1u);
  __syncthreads();

  // suffix counts over bins: thread i < 256 takes bin 255 - i
  uint32_t tot = 0, incl = 0;
  if (tid < 256) {
    const int b = 255 - tid;
    for (int w = 0; w < kTopkWaves; ++w) tot += s_h1[w][b];
    incl = incl_scan64(tot, lane);
    if (lane == 63) s_wsum[wave] = incl;
  }
  __syncthreads();
  if (tid < 256) {
    for (int w = 0; w < wave; ++w) incl += s_wsum[w];
    const uint32_t above = incl - tot;   // keys in higher bins
    for (int j = 0; j < n; ++j) {
      const uint32_t C = (uint32_t)cuts.cum[j];
      if (C > above && C <= incl) {
        s_cut_bin[j] = 255 - tid;
        s_need[j] = (int)(C - above);
      }
    }
  }
  __syncthreads();

  // low-digit histograms inside each cut bin
#pragma unroll
  for (int m = 0; m < kTopkPer; ++m) {
    if (key[m] == 0xFFFFu) continue;
    const int hi = (int)(key[m] >> 7);
    for (int j = 0; j < n; ++j)
      if (hi == s_cut_bin[j]) atomicAdd(&s_h2[j][key[m] & 127u], 1u);
  }
  __syncthreads();

  // per level j (threads 128 j .. 128 j + 127), suffix over sub-bins
  {
    const int j = tid >> 7, i = tid & 127, sb = 127 - i;
    const uint32_t h = j < n ? s_h2[j][sb] : 0u;
    uint32_t inc2 = incl_scan64(h, lane);
    if (lane == 63) s_wsum[wave] = inc2;
    __syncthreads();
    if (wave & 1) inc2 += s_wsum[wave - 1];
    if (j < n && s_cut_bin[j] < 256) {
      const uint32_t need = (uint32_t)s_need[j];
      const uint32_t above = inc2 - h;
      if (need > above && need <= inc2) {
        s_cut_key[j] = ((uint32_t)s_cut_bin[j] << 7) | (uint32_t)sb;
        s_need_eq[j] = (int)(need - above);
      }
    }
  }
  __syncthreads();

  // ballots of key == cut key, per (chunk, wave, level)
#pragma unroll
  for (int m = 0; m < kTopkPer; ++m) {
    if (m >= M) break;
    for (int j = 0; j < n; ++j) {
      const uint64_t bal = __ballot(key[m] == s_cut_key[j]);
      if (lane == 0) s_bal[m][wave][j] = bal;
    }
  }
  __syncthreads();

  // wave j finds the index of the need_eq-th channel equal to cut key j
  if (wave < n) {
    const int j = wave;
    const int need = s_need_eq[j];
    const int E = M * kTopkWaves;
    int carry = 0;
    for (int base = 0; base < E && need > 0; base += 64) {
      const int e = base + lane;
      const uint64_t bal = e < E ? s_bal[e / kTopkWaves][e % kTopkWaves][j] : 0ull;
      const uint32_t c = (uint32_t)__popcll(bal);
      const uint32_t inc = incl_scan64(c, lane) + (uint32_t)carry;
      const uint32_t before = inc - c;
      if ((uint32_t)need > before && (uint32_t)need <= inc) {
        const int bit = nth_set_bit(bal, need - (int)before);
        // entry e covers channels (e / 16) * 1024 + (e % 16) * 64 + bit
        s_idx_lim[j] = (e / kTopkWaves) * kTopkThreads + (e % kTopkWaves) * 64 + bit + 1;
      }
      carry = (int)__shfl(inc, 63);
      if (carry >= need) break;
    }
  }
  __syncthreads();

#pragma unroll
  for (int m = 0; m < kTopkPer; ++m) {
    if (m >= M) break;
    const int k = m * kTopkThreads + tid;
    if (k >= K) continue;
    int lvl = 0;
    for (int j = 0; j < n; ++j) {
      const uint32_t ck = s_cut_key[j];
      lvl += (key[m] > ck || (key[m] == ck && k < s_idx_lim[j])) ? 1 : 0;
    }
    out[k] = (uint8_t)lvl;
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
