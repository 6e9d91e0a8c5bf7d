// Nested-precision decode VMM over non-uniform nested weights read through
// per-output look-up tables (Sec. 3.3: the format needs only the nested
// property, which k-means-style nested weights have; their levels are
// centred, so no midpoint bias is applied).  The codes use the packed
// layout of the uniform path; a channel at width b reads its first b/u
// planes, forms the b leading bits q_b of every output's code, and adds
// x_k * table_b[n][q_b].
//
// A workgroup owns 64 outputs of one tile (a sub-tile), a run of groups and
// one token.  It stages the run's levels and x, and copies to LDS the tables
// of its 64 outputs for the levels the run uses: for each level they are one
// contiguous block of the table array.
// 4 lanes cover a channel row's 64 outputs (16 each); the 64 row slots of
// the workgroup take two rows of each group.  Every weight is one LDS
// lookup.  Lanes holding the same outputs are reduced with shuffles, waves
// through LDS, and the sums added into y with atomics.
#include <cstdlib>

#include "grinqh_internal.h"
#include "vmm_common.h"

namespace grinqh {

namespace {

constexpr int kLutThreads = 256;
constexpr int kSub = 64;                     // outputs per workgroup
constexpr int kMaxRun = 16 * 128;            // channels per workgroup (16 groups)

__global__ __launch_bounds__(kLutThreads) void k_zero_lut(float* __restrict__ y, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = 0.0f;
}

template <int U>
__global__ __launch_bounds__(kLutThreads) void k_vmm_lut(const uint8_t* __restrict__ codes,
                                                        const uint16_t* __restrict__ luts,
                                                        const uint16_t* __restrict__ x,
                                                        const uint8_t* __restrict__ lm,
                                                        float* __restrict__ y, Layer L, LutDesc D,
                                                        int groups_per_split, int splits, int fused,
                                                        Thresholds th, uint8_t* __restrict__ lm_out) {
  constexpr uint32_t MASK = (1u << U) - 1u;
  extern __shared__ __align__(16) uint16_t s_lut[];          // [levels][kSub][2^b]
  __shared__ float s_red[kLutThreads / 64][kSub];
  __shared__ int s_cum[kMaxLevels];                           // level l's block starts at s_cum[l]
  __shared__ uint8_t s_lv[kMaxRun];                           // levels of the run's channels
  __shared__ uint16_t s_x[kMaxRun];                           // x of the run's channels
  __shared__ uint32_t s_used;                                 // bit l: level l has a channel

  // Work order: the K splits of a sub-tile, then the sub-tiles of a tile,
  // are consecutive work items, and consecutive items run on one XCD
  // (workgroup id mod 8 picks the XCD): its L2 then serves the sub-tiles'
  // shared 128-byte plane lines and the splits' shared tables.
  const int subs = L.T / kSub;
  const int nwg = gridDim.x;
  const int item = (nwg % 8 == 0) ? (int)(blockIdx.x % 8) * (nwg / 8) + (int)(blockIdx.x / 8)
                                  : (int)blockIdx.x;
  const int tile_sub = item / splits;
  const int split = item % splits;
  const int t = tile_sub / subs, sub = tile_sub % subs;
  const int tok = blockIdx.y;
  const int n0 = t * L.T + sub * kSub;       // first output of the sub-tile
  const int g0 = split * groups_per_split;
  const int g1 = min(g0 + groups_per_split, L.groups);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // LDS layout: level l's block starts at kSub * cum[l] + 4 pad (l - 1)
  // entries and holds the 64 outputs' tables as four quads of 16 outputs,
  // quad c at c (16 * 2^b + pad): the pad of 16 entries (8 banks) puts the
  // four quads a wave reads in one step on different banks (unpadded their
  // starts are 128-byte multiples apart, the same banks for every b >= 2)
  const int pad = D.quad_pad;
  if (tid < kMaxLevels) s_cum[tid] = kSub * D.cum[tid] + 4 * pad * max(tid - 1, 0);
  const int c = tid & 3;                     // outputs 16 c .. 16 c + 15 of the sub-tile
  const int rs = tid >> 2;                   // row slot: rows rs, rs + 64, ... of the run
  const int plane_bytes = L.T * U / 8;
  const int col = (sub * kSub + 16 * c) * U / 8;   // byte of the lane's outputs in a plane row
  const int n_top = L.n_levels - 1;
  const int kr0 = g0 * kGroup, nrows = (g1 - g0) * kGroup;   // the workgroup's channels

  uint32_t used = 0;
  if (tid == 0) s_used = 0;
  __syncthreads();
  // levels and x of the run's channels, staged once (<= kMaxRun channels):
  // read from the level map, or graded here from |x| against the thresholds
  // (Sec. 3.1; th.n is 0 without them), the level map then written out once
  // (by the workgroups of tile 0, sub-tile 0)
  for (int i = tid; i < nrows; i += kLutThreads) {
    const size_t k = (size_t)tok * L.K + kr0 + i;
    const uint16_t xh = x[k];
    int lv;
    if (fused) {
      const float ax = fabsf(h2f(xh));
      lv = 0;
#pragma unroll
      for (int j = 0; j < kMaxLevels - 1; ++j)   // unused thresholds are +inf: no
        lv += ax >= th.theta[j] ? 1 : 0;         // branch, all loaded up front
      lv = min(lv, n_top);
      if (lm_out && t == 0 && sub == 0) lm_out[k] = (uint8_t)lv;
    } else {
      lv = min((int)lm[k], n_top);
    }
    s_lv[i] = (uint8_t)lv;
    s_x[i] = xh;
    used |= 1u << lv;
  }
  // the levels any channel of the run uses: only their tables are copied
  // (at the paper's 4-bit budgets the 8-bit level, three quarters of the
  // table bytes, is empty)
  {
    uint32_t u = used;
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) u |= (uint32_t)__shfl_xor((int)u, m);
    if (lane == 0) atomicOr(&s_used, u);
  }
  __syncthreads();
  const uint32_t used_levels = s_used;

  float acc[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.0f;

  // Rows rs + 64 m, m = 0, 1, ..., through a ring of four register sets:
  // three rows' plane words are in flight while one row is looked up.  The
  // loads are unconditional (planes past a row's depth, and rows past the
  // run, load from no row and read zero without a memory access), so the
  // compiler counts them and waits for the row being consumed alone.
  constexpr int kWords = 8 / U;
  constexpr int R = 4;
  // 1-bit planes: the lane's two bytes are loaded as the aligned dword that
  // holds them and its half is kept when the row is consumed (plane rows and
  // sub-tiles start at multiples of four bytes)
  const uint32_t lane_off = (uint32_t)(U == 2 ? col : (col & ~3));
  const int half_sh = U == 2 ? 0 : (col & 2) * 8;
  const __amdgpu_buffer_rsrc_t rsrc = vmmdev::tile_rsrc(codes + (size_t)t * L.K * L.RB, L);
  auto fetch = [&](int i, uint32_t (&w)[kWords]) __attribute__((always_inline)) {
    const int d = i < nrows ? level_planes(L.planes_packed, s_lv[i]) : 0;
    const uint32_t row = (uint32_t)(kr0 + min(i, nrows - 1)) * (uint32_t)L.RB + lane_off;
#pragma unroll
    for (int j = 0; j < kWords; ++j)
      w[j] = vmmdev::load_plane(rsrc, j < d ? row + (uint32_t)(j * plane_bytes) : vmmdev::kNoRow);
  };
  auto consume = [&](int i, const uint32_t (&wv)[kWords]) __attribute__((always_inline)) {
    const int lvl = i < nrows ? (int)s_lv[i] : 0;
    if (lvl != 0) {
      const float xv = h2f(s_x[i]);
      const int d = level_planes(L.planes_packed, lvl);
      const int b = d * U;
      // the 16 outputs' codes left-aligned in 8 bits (planes past d were
      // loaded as zero): byte i of qw[r] is output 4 i + r; q_b is its top
      // b bits
      uint32_t m[kWords];
#pragma unroll
      for (int j = 0; j < kWords; ++j) m[j] = U == 2 ? wv[j] : (wv[j] >> half_sh) & 0xFFFFu;
      uint32_t w[4];
      if constexpr (U == 2) {
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = m[j];
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          w[j] = (vmmdev::spread_bits(m[2 * j]) << 1) | vmmdev::spread_bits(m[2 * j + 1]);
      }
      uint32_t qw[4];
      vmmdev::assemble_codes(w[0], w[1], w[2], w[3], qw);
      const int sh = 8 - b;
      // the lane's outputs' table quad of level lvl: output 16 c + e at e * 2^b
      const uint16_t* tb = s_lut + s_cum[lvl] + c * ((16 << b) + pad);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const uint32_t q8 = (qw[e & 3] >> (8 * (e >> 2))) & 0xFFu;
        acc[e] = fmaf(xv, h2f(tb[(e << b) + (q8 >> sh)]), acc[e]);
      }
    }
  };
  uint32_t wr[R][kWords];
#pragma unroll
  for (int q = 0; q < R - 1; ++q) fetch(rs + 64 * q, wr[q]);
  __builtin_amdgcn_sched_barrier(0);   // the first rows' loads go out before the table copy
  // tables of the 64 outputs: level l's are kSub * 2^b entries at
  // D.offset[l] + n0 * 2^b of the table array, 8 * 2^b pieces of 16 bytes,
  // copied quad by quad.  A thread issues eight loads before its eight
  // stores: one L2 latency per eight pieces rather than one per piece.
  for (int l = 1; l < L.n_levels; ++l) {
    if (!((used_levels >> l) & 1u)) continue;
    const int b = L.bits[l];
    const int np = 8 << b, qn = 2 << b;      // pieces of the level, of a quad
    const uint4* src = (const uint4*)(luts + D.offset[l] + ((size_t)n0 << b));
    uint16_t* dst = s_lut + kSub * D.cum[l] + 4 * pad * (l - 1);
    for (int i0 = 0; i0 < np; i0 += 8 * kLutThreads) {
      uint4 v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = src[min(i0 + tid + q * kLutThreads, np - 1)];
      __builtin_amdgcn_sched_barrier(0);     // keep the eight loads ahead of the stores
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        // (past the last piece: the last piece again, the same value to the
        // same place, so that neither loads nor stores are conditional)
        const int i = min(i0 + tid + q * kLutThreads, np - 1);
        *(uint4*)(dst + (i / qn) * ((16 << b) + pad) + 8 * (i % qn)) = v[q];
      }
    }
  }
  __syncthreads();

  for (int i = rs; i < nrows; i += 64 * R) {
#pragma unroll
    for (int q = 0; q < R; ++q) {
      fetch(i + 64 * (q + R - 1), wr[(q + R - 1) % R]);
      consume(i + 64 * q, wr[q]);
    }
  }

  // lanes with equal (lane & 3) hold the same outputs: sum over lane bits 2..5
#pragma unroll
  for (int e = 0; e < 16; ++e) {
#pragma unroll
    for (int m = 4; m < 64; m <<= 1) acc[e] += __shfl_xor(acc[e], m);
  }
  if (lane < 4) {
#pragma unroll
    for (int e = 0; e < 16; ++e) s_red[wave][16 * lane + e] = acc[e];
  }
  __syncthreads();
  if (tid < kSub) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kLutThreads / 64; ++w) v += s_red[w][tid];
    atomicAdd(&y[(size_t)tok * L.N + n0 + tid], v);
  }
}

}  // namespace

int lut_desc(const Layer& L, LutDesc* D) {
  long off = 0;
  int cum = 0;
  for (int l = 0; l < kMaxLevels; ++l) {
    D->offset[l] = off;
    D->cum[l] = cum;
    if (l >= 1 && l < L.n_levels) {
      off += (long)L.N << L.bits[l];
      cum += 1 << L.bits[l];
    }
  }
  D->entries = cum;
  // quad padding in LDS when it fits in 64 KB (see the kernel)
  const size_t padded = (size_t)kSub * cum * 2 + (size_t)4 * 16 * (L.n_levels - 1) * 2;
  D->quad_pad = padded <= 65536 ? 16 : 0;
  return GRINQH_OK;
}

int launch_vmm_lut(const Layer& L, const void* codes, const void* luts, const void* x,
                   const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out, int B,
                   float* y, int accumulate, hipStream_t s) {
  LutDesc D;
  lut_desc(L, &D);
  // <= 64 * 510 * 2 bytes (levels are distinct widths <= 8), plus the quad padding where it fits
  const size_t lds = (size_t)kSub * D.entries * 2 + (size_t)4 * D.quad_pad * (L.n_levels - 1) * 2;
  if (lds > 65536) return fail(GRINQH_EUNSUPPORTED, "LUT VMM: %d table entries per output", D.entries);
  if (!accumulate) {
    const long n = (long)B * L.N;
    hipLaunchKernelGGL(k_zero_lut, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, y, n);
  }
  // groups per workgroup: 4 on layers of up to 4096 (sub-tile, group)
  // units per token (the Llama3-8B attention projections: 8 and 16 groups
  // 5% and 30% slower), 16 above (the MLP: 45.2 us against 48.6 with 8 and
  // 59.1 with 4); fewer groups re-copy the tables too often, more leave too
  // few workgroups to hide latency
  const long subtiles = (long)L.tiles * (L.T / kSub);
  long splits;
  int gps = (long)L.groups * subtiles * B <= 4096 ? 4 : 16;
  gps = gps > L.groups ? L.groups : gps;
  if (const int v = option(&Options::lut_groups)) gps = v <= L.groups ? v : L.groups;
  gps = gps > kMaxRun / kGroup ? kMaxRun / kGroup : gps;
  splits = (L.groups + gps - 1) / gps;
  const dim3 grid((unsigned)(subtiles * splits), (unsigned)B);
  Thresholds none{};
  const Thresholds& tt = th ? *th : none;
  const int fused = th != nullptr;
  if (L.u == 2)
    hipLaunchKernelGGL(k_vmm_lut<2>, grid, dim3(kLutThreads), lds, s, (const uint8_t*)codes,
                       (const uint16_t*)luts, (const uint16_t*)x, level_map, y, L, D, gps, (int)splits,
                       fused, tt, level_map_out);
  else
    hipLaunchKernelGGL(k_vmm_lut<1>, grid, dim3(kLutThreads), lds, s, (const uint8_t*)codes,
                       (const uint16_t*)luts, (const uint16_t*)x, level_map, y, L, D, gps, (int)splits,
                       fused, tt, level_map_out);
  return check_launch("vmm_lut");
}

}  // namespace grinqh
