// Exact top-k cuts of one token's |x| (App. A.1 top-p partition), computed
// by the 256 threads of a VMM workgroup in its prologue, so that the top-k
// mode needs no separate assignment launch.  Every workgroup of a launch
// computes the same cuts from the whole x.
//
// Cut j (0 <= j < n) is the set of the C_j = cum[j] channels of largest |x|,
// ties going to the lower channel index (the order of the standalone top-k
// kernel).  It is returned as a composite: channel k with 15-bit magnitude
// key q_k is in cut j iff (q_k << 16) + 65535 - k >= cut[j], and a channel's
// level is the number of cuts it is in.  C_j = 0 gives 0xFFFFFFFF (nobody).
//
//   1. Each thread owns a contiguous run of KP keys (KP = ceil(K / 256)
//      rounded up to 8), so thread order is channel order; each pass below
//      re-reads the run from x (L2-resident after the first pass), which
//      measured faster than holding the run in registers.
//   2. A 256-bin histogram of q >> 7 (LDS atomics); wave w scans it from the
//      top for cuts w, w + 4: the coarse bin holding the C_j-th largest key.
//   3. A 128-bin histogram of q & 127 over the keys of each cut's coarse bin
//      gives the exact key ck_j, the keys above it and those equal to it;
//      need_j = C_j - above of the keys equal to ck_j are in.
//   4. For each cut where need_j is less than all of them, a block scan of
//      each thread's count of keys equal to ck_j (in channel order) finds
//      the channel of the need_j-th one; the cut's index limit is the
//      channel after it.
#pragma once

#include "grinqh_internal.h"

namespace grinqh {
namespace topksel {

constexpr int kCutsMax = kMaxLevels - 1;
constexpr int kThreads = 256;
constexpr int kMaxK = 16384;   // channel indices fit the low 16 bits of a composite
static_assert(kMaxK <= 65536, "a composite holds 65535 - k in 16 bits");

struct Scratch {
  uint32_t hist1[256];
  uint32_t hist2[kCutsMax][128];
  uint32_t binmask[256];               // bit j: coarse bin of cut j
  uint32_t bin[kCutsMax], above[kCutsMax], ck[kCutsMax], need[kCutsMax];
  uint32_t tie;                        // bit j: cut j needs the channel-order scan
  uint32_t wtot[kCutsMax][4];          // per-wave totals of the tie counts, a row per cut
  uint32_t cut[kCutsMax];
};

// Inclusive prefix sum over the 64 lanes (DPP row shifts, then row broadcasts).
__device__ __forceinline__ uint32_t incl_scan(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);   // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);   // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);   // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);   // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);   // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);   // row_bcast:31
  return v;
}

__device__ __forceinline__ int first_lane(bool pred) {
  const uint64_t m = __ballot(pred);
  return m ? (int)__builtin_ctzll(m) : 0;
}

// Lane l's value; called where every lane of the wave is active.
__device__ __forceinline__ uint32_t rdlane(uint32_t v, int l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

// Eight consecutive 15-bit magnitude keys of this thread's run, two per
// dword; a word at or past K reads 0xFFFF keys, above every real one.
__device__ __forceinline__ uint4 key_word(const uint16_t* __restrict__ x, int K, int k0) {
  if (k0 >= K) return make_uint4(0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu);
  uint4 v = *(const uint4*)(x + k0);
  v.x &= 0x7FFF7FFFu; v.y &= 0x7FFF7FFFu; v.z &= 0x7FFF7FFFu; v.w &= 0x7FFF7FFFu;
  return v;
}

__device__ __forceinline__ uint32_t key_at(const uint4& v, int i) {
  const uint32_t w = (i >> 1) == 0 ? v.x : (i >> 1) == 1 ? v.y : (i >> 1) == 2 ? v.z : v.w;
  return (w >> (16 * (i & 1))) & 0xFFFFu;
}

// Leaves the cuts in S.cut; ends with a workgroup barrier.  x: the token's
// fp16 x [K], K a multiple of 128 and at most kMaxK, 16-byte aligned.
__device__ __forceinline__ void select_cuts(const uint16_t* __restrict__ x, int K, const TopkCuts& tk,
                                            Scratch& S) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = tk.n;
  const int KP = (((K + kThreads - 1) / kThreads) + 7) & ~7;   // keys per thread
  const int kb = tid * KP;                                       // this thread's first channel
  const int words = KP >> 3;

  S.hist1[tid] = 0u;
  S.binmask[tid] = 0u;
  for (int i = tid; i < kCutsMax * 128; i += kThreads) (&S.hist2[0][0])[i] = 0u;
  if (tid == 0) S.tie = 0u;
  __syncthreads();
  for (int w = 0; w < words; ++w) {
    const uint4 v = key_word(x, K, kb + 8 * w);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t q = key_at(v, i);
      if (q < 0x8000u) atomicAdd(&S.hist1[q >> 7], 1u);
    }
  }
  __syncthreads();

  // coarse bins, from the top: lane l holds bins 255 - 4l .. 252 - 4l
  for (int j = wave; j < n; j += 4) {
    const uint32_t C = (uint32_t)tk.cum[j];
    if (!C) continue;
    const uint4 h4 = *(const uint4*)&S.hist1[252 - 4 * lane];   // bins 252-4l .. 255-4l
    const uint32_t h[4] = {h4.w, h4.z, h4.y, h4.x};               // descending bin order
    const uint32_t s = h[0] + h[1] + h[2] + h[3];
    const uint32_t pre = incl_scan(s);
    const uint32_t above_l = pre - s;
    uint32_t b = 0u, ab = 0u, acc = above_l;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (acc < C && C <= acc + h[i]) {
        b = (uint32_t)(255 - 4 * lane - i);
        ab = acc;
      }
      acc += h[i];
    }
    const int L = first_lane(above_l < C && C <= pre);
    // cross-lane reads stay outside the lane-0 branch: lane L must be active
    const uint32_t bin = rdlane(b, L), above = rdlane(ab, L);
    if (lane == 0) {
      atomicOr(&S.binmask[bin], 1u << j);
      S.bin[j] = bin;
      S.above[j] = above;
    }
  }
  __syncthreads();

  // fine bins inside each cut's coarse bin
  for (int w = 0; w < words; ++w) {
    const uint4 v = key_word(x, K, kb + 8 * w);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t q = key_at(v, i);
      if (q < 0x8000u) {
        uint32_t m = S.binmask[q >> 7];
        while (m) {
          const int j = __builtin_ctz(m);
          atomicAdd(&S.hist2[j][q & 127u], 1u);
          m &= m - 1u;
        }
      }
    }
  }
  __syncthreads();

  // exact keys: lane l holds fine bins 127 - 2l and 126 - 2l
  for (int j = wave; j < n; j += 4) {
    const uint32_t C = (uint32_t)tk.cum[j];
    if (!C) {
      if (lane == 0) S.cut[j] = 0xFFFFFFFFu;
      continue;
    }
    const uint2 h2 = *(const uint2*)&S.hist2[j][126 - 2 * lane];   // bins 126-2l, 127-2l
    const uint32_t h[2] = {h2.y, h2.x};
    const uint32_t s = h[0] + h[1];
    const uint32_t pre = incl_scan(s) + S.above[j];
    const uint32_t above_l = pre - s;
    uint32_t f = 0u, ab = 0u, acc = above_l;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (acc < C && C <= acc + h[i]) {
        f = (uint32_t)(127 - 2 * lane - i);
        ab = acc;
      }
      acc += h[i];
    }
    const int L = first_lane(above_l < C && C <= pre);
    const uint32_t fine = rdlane(f, L), above = rdlane(ab, L);
    const uint32_t ck = (S.bin[j] << 7) | fine;
    const uint32_t equal = S.hist2[j][fine];
    const uint32_t need = C - above;   // 1 <= need <= equal
    if (lane == 0) {
      S.ck[j] = ck;
      S.need[j] = need;
      if (need == equal) S.cut[j] = (ck << 16) + 65536u - (uint32_t)K;   // every equal key is in
      else atomicOr(&S.tie, 1u << j);
    }
  }
  __syncthreads();

  // ties: the need-th key equal to ck in channel order, one cut at a time
  for (uint32_t tie = S.tie; tie; tie &= tie - 1u) {
    const int j = __builtin_ctz(tie);
    const uint32_t ck = S.ck[j], need = S.need[j];
    uint32_t e = 0u;
    for (int w = 0; w < words; ++w) {
      const uint4 v = key_word(x, K, kb + 8 * w);
#pragma unroll
      for (int i = 0; i < 8; ++i) e += key_at(v, i) == ck ? 1u : 0u;
    }
    const uint32_t pre = incl_scan(e);
    if (lane == 63) S.wtot[j][wave] = pre;
    __syncthreads();
    uint32_t off = 0u;
    for (int w = 0; w < wave; ++w) off += S.wtot[j][w];
    const uint32_t incl = pre + off, excl = incl - e;
    if (excl < need && need <= incl) {   // exactly one thread
      uint32_t seen = excl;
      int lim = kb;
      for (int w = 0; w < words; ++w) {
        const uint4 v = key_word(x, K, kb + 8 * w);
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (key_at(v, i) == ck && ++seen == need) lim = kb + 8 * w + i + 1;
      }
      S.cut[j] = (ck << 16) + 65536u - (uint32_t)lim;
    }
    __syncthreads();
  }
}

// The level of channel k with fp16 bits xb: the number of cuts it is in.
__device__ __forceinline__ int level_of(uint32_t xb, int k, int n, const Scratch& S) {
  const uint32_t comp = ((xb & 0x7FFFu) << 16) + (uint32_t)(65535 - k);
  int l = 0;
#pragma unroll
  for (int j = 0; j < kCutsMax; ++j) l += (j < n && comp >= S.cut[j]) ? 1 : 0;
  return l;
}

}  // namespace topksel
}  // namespace grinqh
