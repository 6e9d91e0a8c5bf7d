// Per-token precision assignment (Sec. 3.1 threshold grading; App. A.1 top-p
// partition of |x| into the fractions P).
#include <mutex>

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

// Top-k: one workgroup of 512 threads per token, K <= 16384, every key in
// registers.  For every level j the cut is the C_j-th largest key (C_j =
// channels at level >= j); channels strictly above it are in, and of those
// equal to it the first ones in channel order.
//   1. A histogram of all 2^15 key values (two 16-bit counts per LDS word) and
//      per-thread totals of 64 consecutive values.
//   2. Wave j finds cut j: a wave scan over the totals picks the thread range,
//      a second one the key value; then it counts the channels equal to the cut
//      key in channel order (each lane a contiguous span of the keys kept in
//      LDS), picks the lane and the 8-key chunk where the count reaches the
//      number still needed, and from it the channel-index limit.
//   3. Every thread grades its channels against the cuts.
constexpr int kTkThreads = 512;
constexpr int kTkChunk = kTkThreads * 8;   // channels per load round, 8 per thread
constexpr int kTkMaxK = 16384;
constexpr int kTkBins = 1 << 15;           // every 15-bit key value
constexpr int kCuts = kMaxLevels - 1;

// Inclusive prefix sum over the 64 lanes: shifts within rows of 16 lanes, then
// the row broadcasts of lanes 15 and 31.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);   // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);   // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);   // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);   // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);   // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);   // row_bcast:31
  return v;
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int first_lane(bool pred) {
  const uint64_t m = __ballot(pred);
  return m ? (int)__builtin_ctzll(m) : 0;
}

__device__ __forceinline__ uint32_t readlane(uint32_t v, int l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

__device__ __forceinline__ int count_eq8(const uint4& w, uint32_t key) {
  const uint32_t a[4] = {w.x, w.y, w.z, w.w};
  int c = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) c += ((a[i] & 0xFFFFu) == key) + ((a[i] >> 16) == key);
  return c;
}

// Round r of thread tid holds channels r*kTkChunk + 8*tid .. +7 as eight
// 15-bit |x| keys packed in pairs (K is a multiple of 128).  The address is
// clamped so that every thread loads; rounds past K are not used.
template <int R>
__device__ __forceinline__ void load_keys(const uint16_t* xt, int K, int tid, uint32_t (&kw)[R][4]) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int k0 = min(r * kTkChunk + 8 * tid, K - 8);
    uint32_t v[4];
    __builtin_memcpy(v, xt + k0, 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) kw[r][i] = v[i] & 0x7FFF7FFFu;
  }
}

// Histogram of every key value, two 16-bit counts per word (s_hist zeroed and
// a barrier passed before), then per-thread totals of 64 consecutive values:
// thread t covers key values 64t .. 64t+63.  Ends with a barrier.
template <int R>
__device__ __forceinline__ void key_histogram(const uint32_t (&kw)[R][4], int K, int tid,
                                              uint32_t* s_hist, uint32_t* s_tot) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r * kTkChunk + 8 * tid >= K) continue;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t key = (kw[r][i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
      atomicAdd(&s_hist[key >> 1], 1u << (16 * (key & 1u)));
    }
  }
  __syncthreads();
  {   // 16-bit lanes cannot overflow (K < 2^16)
    u16x2 acc = {0, 0};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      // rotated so that the lanes of a wave hit different LDS banks
      const uint4 w = reinterpret_cast<const uint4*>(s_hist)[8 * tid + ((i + tid) & 7)];
      acc += __builtin_bit_cast(u16x2, w.x) + __builtin_bit_cast(u16x2, w.y) +
             __builtin_bit_cast(u16x2, w.z) + __builtin_bit_cast(u16x2, w.w);
    }
    s_tot[tid] = (uint32_t)acc[0] + (uint32_t)acc[1];
  }
  __syncthreads();
}

// One wave: the C-th largest key (1 <= C <= number of keys), found from the
// per-thread totals and then the owning thread's 64 counts.  Returns the key;
// *above = keys strictly greater, *equal = keys equal to it.
__device__ __forceinline__ uint32_t select_key(uint32_t C, const uint32_t* s_hist,
                                               const uint32_t* s_tot, int lane, uint32_t* above,
                                               uint32_t* equal) {
  // lane l: threads 8l .. 8l+7, i.e. key values 512 l .. 512 l + 511
  const uint4 a = reinterpret_cast<const uint4*>(s_tot)[2 * lane];
  const uint4 b = reinterpret_cast<const uint4*>(s_tot)[2 * lane + 1];
  const uint32_t sl = a.x + a.y + a.z + a.w + b.x + b.y + b.z + b.w;
  const uint32_t pre = wave_incl_scan(sl);
  const uint32_t above_l = readlane(pre, 63) - pre;          // keys in higher lanes
  // inside each lane, from its highest thread down: the thread whose range
  // holds the C-th largest key, if this lane's range does
  const uint32_t tv[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  uint32_t acc = above_l, q_loc = 0, above_loc = 0;
#pragma unroll
  for (int i = 7; i >= 0; --i) {
    if (acc < C && C <= acc + tv[i]) {
      q_loc = (uint32_t)i;
      above_loc = acc;
    }
    acc += tv[i];
  }
  const int L = first_lane(above_l < C && C <= above_l + sl);
  const int t_own = 8 * L + (int)readlane(q_loc, L);
  const uint32_t above2 = readlane(above_loc, L);
  // the 64 key values of that thread
  const uint32_t c = (reinterpret_cast<const uint16_t*>(s_hist))[64 * t_own + lane];
  const uint32_t pre64 = wave_incl_scan(c);
  const uint32_t above_v = above2 + readlane(pre64, 63) - pre64;
  const int bsel = first_lane(above_v < C && C <= above_v + c);
  *above = readlane(above_v, bsel);
  *equal = readlane(c, bsel);
  return (uint32_t)(64 * t_own + bsel);
}

template <int R>
__global__ __launch_bounds__(kTkThreads) void k_assign_topk(const uint16_t* __restrict__ x,
                                                            uint8_t* __restrict__ lm, int K,
                                                            TopkCuts cuts) {
  __shared__ uint32_t s_hist[kTkBins / 2];
  __shared__ __attribute__((aligned(16))) uint16_t s_key[kTkMaxK + 64 * 32];
  __shared__ __attribute__((aligned(16))) uint32_t s_tot[kTkThreads];
  __shared__ uint32_t s_cut[kCuts];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = cuts.n;
  const uint16_t* xt = x + (size_t)blockIdx.x * K;
  uint8_t* out = lm + (size_t)blockIdx.x * K;
  const int span = (K + 2047) / 2048 * 32;   // keys per lane in the tie scans; 64*span >= K

  uint32_t kw[R][4];
  load_keys<R>(xt, K, tid, kw);
  for (int i = tid; i < kTkBins / 8; i += kTkThreads) reinterpret_cast<uint4*>(s_hist)[i] = uint4{0u, 0u, 0u, 0u};
  for (int i = K + tid; i < 64 * span; i += kTkThreads) s_key[i] = 0xFFFFu;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (r * kTkChunk + 8 * tid < K)
      *reinterpret_cast<uint4*>(&s_key[r * kTkChunk + 8 * tid]) = uint4{kw[r][0], kw[r][1], kw[r][2], kw[r][3]};
  __syncthreads();
  key_histogram<R>(kw, K, tid, s_hist, s_tot);

  if (wave < n) {
    const int j = wave;
    const uint32_t C = (uint32_t)cuts.cum[j];
    uint32_t ck = 0x8000u;   // above every key: nobody is in
    int lim = 0;
    if (C > 0) {
      uint32_t above, equal;
      ck = select_key(C, s_hist, s_tot, lane, &above, &equal);
      const int need = (int)(C - above);        // >= 1 channels equal to ck
      if (need == (int)equal) {   // every channel equal to ck is in
        lim = K;
        goto store;
      }
      // channels equal to ck, in channel order: lane l scans keys [l*span, (l+1)*span)
      const int nch = span / 8;     // a multiple of 4
      int e = 0, c8 = lane % nch;   // chunks visited in rotated order (LDS banks)
      for (int i = 0; i < nch; i += 4) {
        uint4 w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          w[q] = *reinterpret_cast<const uint4*>(&s_key[lane * span + 8 * c8]);
          c8 = c8 + 1 == nch ? 0 : c8 + 1;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) e += count_eq8(w[q], ck);
      }
      const int pre_e = (int)wave_incl_scan((uint32_t)e);
      const int L2 = first_lane(pre_e - e < need && need <= pre_e);
      const int r1 = need - (int)readlane((uint32_t)(pre_e - e), L2);
      // the 8-key chunks of lane L2's span
      const int ec = lane < nch ? count_eq8(*reinterpret_cast<const uint4*>(&s_key[L2 * span + 8 * lane]), ck) : 0;
      const int pre_c = (int)wave_incl_scan((uint32_t)ec);
      const int cs = first_lane(lane < nch && pre_c - ec < r1 && r1 <= pre_c);
      int r2 = r1 - (int)readlane((uint32_t)(pre_c - ec), cs);
      const int base = L2 * span + 8 * cs;
      const uint4 w8 = *reinterpret_cast<const uint4*>(&s_key[base]);
      const uint32_t ww[4] = {w8.x, w8.y, w8.z, w8.w};
      int pos = 0, seen = 0;   // the r2-th key equal to ck in this chunk
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bool eq = ((ww[i >> 1] >> (16 * (i & 1))) & 0xFFFFu) == ck;
        seen += eq ? 1 : 0;
        if (eq && seen == r2) pos = i;
      }
      lim = base + pos + 1;
    }
  store:
    // channel k is in iff key > ck, or key == ck and k < lim: with the
    // composite key*2^16 + (65535 - k), iff composite >= ck*2^16 + 65536 - lim.
    if (lane == 0) s_cut[j] = C > 0 ? (ck << 16) + 65536u - (uint32_t)lim : 0xFFFFFFFFu;
  }
  __syncthreads();

  // level = number of cuts passed; count the cuts not passed
  uint32_t comp[R][8], miss[R][8];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t key = (kw[r][i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
      comp[r][i] = (key << 16) + (uint32_t)(65535 - (r * kTkChunk + 8 * tid + i));
      miss[r][i] = 0;
    }
  for (int j = 0; j < n; ++j) {
    const uint32_t cc = s_cut[j];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int i = 0; i < 8; ++i) miss[r][i] += comp[r][i] < cc ? 1u : 0u;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int k0 = r * kTkChunk + 8 * tid;
    if (k0 >= K) continue;
    uint32_t lv[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i) lv[i >> 2] |= ((uint32_t)n - miss[r][i]) << (8 * (i & 3));
    __builtin_memcpy(out + k0, lv, 8);
  }
}

// Offline threshold calibration (Sec. 3.2; App. A.1).  One workgroup per
// calibration sample: the two order statistics around each quantile position
// come from the same key histogram as the top-k assignment, and lane 0 of
// wave k interpolates threshold k in float64 (no contraction, so the
// rounding is the plain one of each operation).
template <int R>
__global__ __launch_bounds__(kTkThreads) void k_calibrate_sample(const uint16_t* __restrict__ x,
                                                                 int K, QuantilePos qp,
                                                                 double* __restrict__ per_sample) {
#pragma clang fp contract(off)
  __shared__ uint32_t s_hist[kTkBins / 2];
  __shared__ __attribute__((aligned(16))) uint32_t s_tot[kTkThreads];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint16_t* xt = x + (size_t)blockIdx.x * K;
  uint32_t kw[R][4];
  load_keys<R>(xt, K, tid, kw);
  for (int i = tid; i < kTkBins / 8; i += kTkThreads) reinterpret_cast<uint4*>(s_hist)[i] = uint4{0u, 0u, 0u, 0u};
  __syncthreads();
  key_histogram<R>(kw, K, tid, s_hist, s_tot);
  if (wave < qp.n) {
    uint32_t above, equal;
    // ascending rank r is the (K - r)-th largest
    const uint32_t klo = select_key((uint32_t)(K - qp.lo[wave]), s_hist, s_tot, lane, &above, &equal);
    const uint32_t khi = select_key((uint32_t)(K - qp.hi[wave]), s_hist, s_tot, lane, &above, &equal);
    if (lane == 0) {
      const double a = (double)h2f((uint16_t)klo), b = (double)h2f((uint16_t)khi);
      const double d = b - a;
      const double t = qp.frac[wave] * d;
      per_sample[(size_t)blockIdx.x * qp.n + wave] = a + t;
    }
  }
}

__global__ void k_calibrate_mean(const double* __restrict__ per_sample, int S, int n,
                                 float* __restrict__ theta) {
#pragma clang fp contract(off)
  const int k = threadIdx.x;
  if (k >= n) return;
  double acc = 0.0;
  for (int s = 0; s < S; ++s) acc += per_sample[(size_t)s * n + k];
  theta[k] = (float)(acc / (double)S);
}

int launch_calibrate(const Layer& L, const void* x, int S, const QuantilePos& qp,
                     double* per_sample, float* theta, hipStream_t s) {
  if (L.K > kTkMaxK || L.K % 8 != 0) return fail(GRINQH_EUNSUPPORTED, "calibration needs K <= %d", kTkMaxK);
  const int rounds = (L.K + kTkChunk - 1) / kTkChunk;
  const dim3 grid((unsigned)S), block(kTkThreads);
  const uint16_t* xx = (const uint16_t*)x;
  switch (rounds) {
    case 1: hipLaunchKernelGGL(k_calibrate_sample<1>, grid, block, 0, s, xx, L.K, qp, per_sample); break;
    case 2: hipLaunchKernelGGL(k_calibrate_sample<2>, grid, block, 0, s, xx, L.K, qp, per_sample); break;
    case 3: hipLaunchKernelGGL(k_calibrate_sample<3>, grid, block, 0, s, xx, L.K, qp, per_sample); break;
    default: hipLaunchKernelGGL(k_calibrate_sample<4>, grid, block, 0, s, xx, L.K, qp, per_sample); break;
  }
  int st = check_launch("calibrate (samples)");
  if (st) return st;
  hipLaunchKernelGGL(k_calibrate_mean, dim3(1), dim3(64), 0, s, per_sample, S, qp.n, theta);
  return check_launch("calibrate (mean)");
}

// Scratch of grinqh_calibrate_noalloc: the per-sample thresholds, float64
// [S][n] with S * n <= kCalibScratch, in a static array each GPU holds for
// the life of the process.  Host code never names the array in a launch or a
// copy: its device address comes from hipGetSymbolAddress, once per device,
// with that device current.  Every entry the mean reads is written by the
// sample kernel of the same call first, so nothing needs clearing; calls that
// overlap on one GPU share the array and race.
static __device__ __align__(256) double scratch[kCalibScratch];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

static int scratch_ptr(double** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(GRINQH_EHIP, "calibrate (no-alloc): hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(GRINQH_EUNSUPPORTED, "calibrate (no-alloc): device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(GRINQH_EHIP, "calibrate (no-alloc): hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = (double*)p;
  }
  *out = g_scratch_ptr[dev];
  return GRINQH_OK;
}

int launch_calibrate_noalloc(const Layer& L, const void* x, int S, const QuantilePos& qp,
                             float* theta, hipStream_t s) {
  if ((long)S * qp.n > kCalibScratch)
    return fail(GRINQH_ESIZE, "calibrate (no-alloc): S*n = %ld per-sample thresholds exceed the %d of the static scratch",
                (long)S * qp.n, kCalibScratch);
  double* per_sample = nullptr;
  const int st = scratch_ptr(&per_sample);
  if (st) return st;
  return launch_calibrate(L, x, S, qp, per_sample, theta, s);
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
  if (L.K > kTkMaxK || L.K % 8 != 0) return fail(GRINQH_EUNSUPPORTED, "top-k needs K <= %d", kTkMaxK);
  const int rounds = (L.K + kTkChunk - 1) / kTkChunk;
  const dim3 grid((unsigned)B), block(kTkThreads);
  const uint16_t* xx = (const uint16_t*)x;
  switch (rounds) {
    case 1: hipLaunchKernelGGL(k_assign_topk<1>, grid, block, 0, s, xx, level_map, L.K, cuts); break;
    case 2: hipLaunchKernelGGL(k_assign_topk<2>, grid, block, 0, s, xx, level_map, L.K, cuts); break;
    case 3: hipLaunchKernelGGL(k_assign_topk<3>, grid, block, 0, s, xx, level_map, L.K, cuts); break;
    default: hipLaunchKernelGGL(k_assign_topk<4>, grid, block, 0, s, xx, level_map, L.K, cuts); break;
  }
  return check_launch("assign (top-k)");
}

}  // namespace grinqh
