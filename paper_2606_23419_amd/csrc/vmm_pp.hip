// Nested-precision decode VMM at batch 1 for 2-bit planes, with a channel's
// consecutive planes merged before the multiply-add (Sec. 3.3 reconstruction
// with the midpoint bias; App. C.1 sparse bit-loading), laid out for CDNA4.
//
// A channel read to depth d planes contributes x_k * sum_j c_j 2^(8-2j).  Its
// planes are taken as items: "doubles" for the plane pairs (1,2) and (3,4)
// inside the depth, and a "single" for an odd last plane (depth 1 or 3).  A
// double's two fields merge into one 4-bit field F = 4 c_j + c_(j+1) worth
// F 2^(6-2j), so one fp16 operand carries four bits of the code instead of
// two: for 16 outputs a lane turns its two plane dwords into two dwords of
// 4-bit fields (even and odd outputs; a shift and a bit-field insert each),
// and a v_and_or_b32 with the exponent bits E = 31 - 2j - p (fp16 bias 15)
// makes the field at bit p of a half read as 2^(16-2j-p) + F 2^(6-2j).
// v_perm_b32 puts one byte of each of two channels (two fields per byte) in
// the two halves, so one v_dot2_f32_f16 with (x_k1, x_k2) adds both channels.
// Singles are consumed as 2-bit fields exactly as in the general 2-bit kernel.
//
// Work units hold four plane dwords per lane: either two doubles (two
// channels, planes j and j+1 each) or two pairs of singles.  A group's units
// are listed doubles first, each kind padded to whole batches, so every batch
// is of one kind and every unit issues the same four loads.  The offsets the
// exponent bits add are summed per lane group, one sum per kind, and taken
// out at the end of the group:
//   y_n += s_{g,n} (acc_n - f_d(n) off_d - f_s(n) off_s + beta_g),
// with f_d = 2^(-p) for doubles, f_s = 2^(4-p) for singles (p = the output's
// field position) and beta_g = sum_{k: level > 0} x_k (phi_b - 128).
//
// The prologue is spread over the four waves (each half wave grades 32 rows
// of a group; per-wave item counts are exchanged through LDS).
// With the plane-1 read-ahead, plane 1 of the first group's 128 rows is requested
// before x arrives and consumed as singles, and that group's lists start at
// plane 2: doubles (2,3) and an even last plane as a single.
#include <cstdlib>
#include <type_traits>

#include "grinqh_internal.h"
#include "vmm_common.h"

namespace grinqh {

namespace {

using namespace vmmdev;

#ifndef GRINQH_PP_DEPTH
#define GRINQH_PP_DEPTH 4
#endif

constexpr int kPPMaxGW = 4;        // groups per workgroup
constexpr int kPPMaxUnits = 160;   // per group: <= 128 double units + 32 single units, padded

// 16 outputs, two channels, planes (j, j+1) of each: w?a = plane j, w?b = j+1.
__device__ __forceinline__ void consume_double(uint32_t w1a, uint32_t w1b, uint32_t w2a,
                                               uint32_t w2b, uint32_t m0, uint32_t xp,
                                               float (&acc)[16]) {
  // 4-bit fields of the even outputs (E) and of the odd outputs (O), output
  // 2m (or 2m+1) at bits 4m..4m+3 with the plane-j field on top
  const uint32_t E1 = ((w1a << 2) & 0xCCCCCCCCu) | (w1b & 0x33333333u);
  const uint32_t O1 = (w1a & 0xCCCCCCCCu) | ((w1b >> 2) & 0x33333333u);
  const uint32_t E2 = ((w2a << 2) & 0xCCCCCCCCu) | (w2b & 0x33333333u);
  const uint32_t O2 = (w2a & 0xCCCCCCCCu) | ((w2b >> 2) & 0x33333333u);
  const uint32_t m4 = m0 - 0x10001000u;   // exponent field - 4 in both halves: p = 4
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const uint32_t S1 = s ? O1 : E1, S2 = s ? O2 : E2;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // byte 2h (outputs 8h+s, 8h+s+2) and byte 2h+1 (8h+s+4, 8h+s+6) of each
      // channel, channel 1 in the low half and channel 2 in the high half
      const uint32_t lo = __builtin_amdgcn_perm(S2, S1, h ? 0x0C060C02u : 0x0C040C00u);
      const uint32_t hi = __builtin_amdgcn_perm(S2, S1, h ? 0x0C070C03u : 0x0C050C01u);
      const int e = 8 * h + s;
      acc[e] = dot2((lo & 0x000F000Fu) | m0, xp, acc[e]);
      acc[e + 2] = dot2((lo & 0x00F000F0u) | m4, xp, acc[e + 2]);
      acc[e + 4] = dot2((hi & 0x000F000Fu) | m0, xp, acc[e + 4]);
      acc[e + 6] = dot2((hi & 0x00F000F0u) | m4, xp, acc[e + 6]);
    }
  }
}

// Offset of output e in a double unit relative to the p = 0 offset summed per
// unit: its field sits at p = 0 or p = 4.
__device__ __forceinline__ float double_offset_factor(int e) {
  return ((e >> 1) & 1) ? 0.0625f : 1.0f;
}

template <int LPR, int PB, int D, int kThreads, bool SPEC>
__global__ __launch_bounds__(kThreads) void k_vmm_pp(
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ lm, float* __restrict__ y,
    Layer L, int gw, int fused, Thresholds th, uint8_t* __restrict__ lm_out) {
  constexpr int T = LPR * 16;            // outputs of the tile
  constexpr int PLANE = T / 4;           // bytes of one plane row
  constexpr int kLaneGroups = kThreads / LPR;
  constexpr int kWaves = kThreads / 64;
  constexpr int kSlots = kLaneGroups * PB;   // units per batch

  __shared__ __align__(16) uint32_t s_units[kPPMaxGW][kPPMaxUnits][8];
  __shared__ __align__(16) uint32_t s_empty[kSlots][8];   // one all-empty batch
  __shared__ float s_beta[kPPMaxGW];
  __shared__ __align__(16) uint16_t s_scale[kPPMaxGW][T];
  __shared__ __align__(16) float s_red[kWaves][T];
  __shared__ uint32_t s_spx[kGroup / 2];   // read-ahead rows' x pairs, 0 for level 0
  __shared__ int s_cnt[kPPMaxGW][kWaves][2];   // items (doubles, singles) per group and wave
  __shared__ float s_bpart[kPPMaxGW][kWaves];  // beta_g partial sums per wave

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x % L.tiles;
  const int g0 = (blockIdx.x / L.tiles) * gw;
  const int ng = min(gw, L.groups - g0);
  // The row that empty items (padding, batches past the end) read; their
  // coefficients are zero, so only its cost matters.  With the read-ahead
  // (small grids) the tile's first row, which every workgroup of the tile
  // reads and which stays in cache; the workgroup's own first row would still
  // be in flight from the read-ahead when the first batches ask for it.
  // Without it (more workgroups) the workgroup's own first row: one row for
  // every workgroup of a tile made its cache lines a hot spot (measured
  // 13.3 against 17.0 us on a 14336 x 4096 layer).
  const uint32_t no_row = SPEC ? 0u : (uint32_t)(g0 * kGroup) * (uint32_t)L.RB;
  const int n_top = L.n_levels - 1;
  const int lg = tid / LPR, li = tid % LPR;

  // ---- prologue.  The four waves grade the rows together: in pass i, lane
  // l of wave w takes row 32w + (l & 31) of group 2i + (l >> 5), so each half
  // wave covers 32 rows of one group.  A group's items go into its unit
  // list, doubles first (item i -> unit i/2, channel slot i%2), then singles
  // (item i -> unit (doubles padded) + i/4, pair (i/2)%2, slot i%2); a half
  // wave's items follow those of the lower waves' halves of the same group,
  // whose counts are exchanged through LDS.  (Whole waves of 64 rows, two
  // waves per group, measured slower: the prologue is a chain of dependent
  // instructions, so halving the rows per wave halves its latency.)
  static_assert(kWaves == 4 && kGroup == 128, "32 rows per half wave");
  constexpr int kPasses = (kPPMaxGW + 1) / 2;
  constexpr int SH = T / 256;                // scale halves per lane and group
  const int half = lane >> 5, hl = lane & 31;
  const int row = 32 * wave + hl;            // row of the group
  // x, the level map and the scales are requested together, so the
  // prologue waits for one memory latency, not two
  uint32_t xv[kPasses], lv[kPasses];
  using ScaleWord = typename std::conditional<SH == 4, uint2, typename std::conditional<SH == 2, uint32_t, uint16_t>::type>::type;
  ScaleWord scw[kPPMaxGW];
  // (unconditional loads, so that the compiler counts them exactly and
  // waits for x alone before grading; groups past the workgroup's last one
  // read that one again, from cache)
  const uint8_t* lmsrc = fused ? (const uint8_t*)x : lm;   // in fused mode the read is ignored
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    const int k = (g0 + min(2 * i + half, ng - 1)) * kGroup + row;
    xv[i] = x[k];
    lv[i] = lmsrc[k];
  }
#pragma unroll
  for (int gg = 0; gg < kPPMaxGW; ++gg)
    scw[gg] = *(const ScaleWord*)(scales + (size_t)(g0 + min(gg, ng - 1)) * L.N + (size_t)t * T +
                                  (wave * 64 + lane) * SH);

  // Read-ahead: every channel above level 0 reads plane 1, so plane 1 of the
  // first group's 128 rows is requested now, behind x, and arrives while the
  // prologue waits for x and builds the lists; only level-0 rows' bytes are
  // fetched without need.  Unit u holds rows 4u..4u+3 (two pairs); lane group
  // lg takes units lg, lg + kLaneGroups, ...  The lists then hold the planes
  // 2..d of those rows.
  constexpr int kSpecUnits = kGroup / 4;
  constexpr int kSpecPerLG = SPEC ? kSpecUnits / kLaneGroups : 0;
  static_assert(!SPEC || kSpecUnits % kLaneGroups == 0, "read-ahead units per lane group");
  uint32_t spw[kSpecPerLG > 0 ? 4 * kSpecPerLG : 1];
  const uint8_t* tile = codes + (size_t)t * L.K * L.RB;
  const uint32_t li4 = (uint32_t)li * 4u;
  if constexpr (SPEC) {
#pragma unroll
    for (int q = 0; q < kSpecPerLG; ++q) {
      const int r = 4 * (lg + kLaneGroups * q);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        spw[4 * q + i] = __builtin_nontemporal_load(
            (const uint32_t*)(tile + ((uint32_t)(g0 * kGroup + r + i) * (uint32_t)L.RB + li4)));
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // grade, count items, local positions
  int dep[kPasses], ndb[kPasses], nsg[kPasses], dpos[kPasses], spos[kPasses];
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    if (i > 0 && 2 * i >= ng) break;         // uniform: the groups of this pass are absent
    const int gg = 2 * i + half;
    const bool valid = gg < ng;
    const float fx = h2f((uint16_t)xv[i]);
    // graded from x (th.n is 0 without thresholds) or read from the level
    // map, chosen without a branch so that the level-map load stays early
    int graded = 0;
    const float ax = fabsf(fx);
#pragma unroll
    for (int j = 0; j < kMaxLevels - 1; ++j)   // unused thresholds are +inf: no
      graded += ax >= th.theta[j] ? 1 : 0;     // branch, all loaded up front
    const int lvl = min(fused ? graded : (int)(lv[i] & 0xFFu), n_top);
    if (fused && lm_out && t == 0 && valid) lm_out[(g0 + gg) * kGroup + row] = (uint8_t)lvl;
    const int d = valid ? level_planes(L.planes_packed, lvl) : 0;
    // planes to list: all d of them, or 2..d when plane 1 was read ahead;
    // doubles of consecutive planes from the first listed one, and a single
    // for a last plane left over
    const bool sg = SPEC && gg == 0;
    const int jl = sg ? max(d - 1, 0) : d;
    dep[i] = d;
    ndb[i] = jl >> 1;
    nsg[i] = jl & 1;
    const float beta = d ? fx * phi_minus_offset(2 * d, L.bmax) : 0.0f;
    const int d1 = half_below(ndb[i] >= 1), d2 = half_below(ndb[i] >= 2);
    const int dt = half_total(ndb[i] >= 1) + half_total(ndb[i] >= 2);
    dpos[i] = d1 + d2;
    spos[i] = half_below(nsg[i] >= 1);
    const int st = half_total(nsg[i] >= 1);
    const float bs = half_sum_dpp(beta);
    if (valid && hl == 0) {
      s_cnt[gg][wave][0] = dt;
      s_cnt[gg][wave][1] = st;
      s_bpart[gg][wave] = bs;
    }
    if (sg) reinterpret_cast<uint16_t*>(s_spx)[row] = d ? (uint16_t)xv[i] : (uint16_t)0;
  }
  for (int i = tid; i < kSlots * 8; i += kThreads) {
    const int w = i % 8;
    (&s_empty[0][0])[i] = (w == 2 || w == 6) ? ((27u << 10) | (27u << 26)) : ((w & 3) == 3 ? 0u : no_row);
  }
  __syncthreads();

  // items at their places; padding and the per-group totals.  Every lane of
  // a half wave computes its group's batch counts; lanes 0 and 32 hand them
  // to the whole wave in scalar registers, so the main loop starts without
  // reading them back from LDS.
  int nb_g[kPPMaxGW] = {}, nbd_g[kPPMaxGW] = {};   // all batches, double batches
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    if (i > 0 && 2 * i >= ng) break;
    const int gg = 2 * i + half;
    int nb_v = 0, nbd_v = 0;
    if (gg < ng) {
      int dbase = 0, sbase = 0, dtot = 0, stot = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const int a = s_cnt[gg][w][0], b = s_cnt[gg][w][1];
        dbase += w < wave ? a : 0;
        sbase += w < wave ? b : 0;
        dtot += a;
        stot += b;
      }
      const int n_du = (dtot + 1) >> 1, n_su = (stot + 3) >> 2;
      const int pad_du = (n_du + kSlots - 1) / kSlots * kSlots;
      int pad_su = (n_su + kSlots - 1) / kSlots * kSlots;
      if (pad_du + pad_su == 0) pad_su = kSlots;   // an empty group still gets one batch
      uint32_t* U = &s_units[gg][0][0];
      const int k = (g0 + gg) * kGroup + row;
      const uint32_t xh = xv[i] & 0xFFFFu;
      const bool sg = SPEC && gg == 0;
      const int j0 = sg ? 2 : 1;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        if (q < ndb[i]) {
          const int j = j0 + 2 * q;                           // first plane of the pair
          const uint32_t off = (uint32_t)(k * L.RB + (j - 1) * PLANE);
          const int it = dbase + dpos[i] + q, u = it >> 1, h = it & 1;
          U[u * 8 + h] = off;
          U[u * 8 + 4 + h] = off + PLANE;
          reinterpret_cast<uint16_t*>(&U[u * 8 + 2])[h] = (uint16_t)((31 - 2 * j) << 10);
          reinterpret_cast<uint16_t*>(&U[u * 8 + 3])[h] = (uint16_t)xh;
        }
      }
      if (nsg[i]) {
        const int j = dep[i];                                 // the last plane
        const uint32_t off = (uint32_t)(k * L.RB + (j - 1) * PLANE);
        const int it = sbase + spos[i], u = pad_du + (it >> 2), sub = (it >> 1) & 1, h = it & 1;
        U[u * 8 + 4 * sub + h] = off;
        reinterpret_cast<uint16_t*>(&U[u * 8 + 4 * sub + 2])[h] = (uint16_t)((29 - 2 * j) << 10);
        reinterpret_cast<uint16_t*>(&U[u * 8 + 4 * sub + 3])[h] = (uint16_t)xh;
      }
      // empty items up to whole batches, spread over the group's 128 lanes:
      // a cached row, zero coefficient, a finite exponent word
      const int pl = row;
      for (int it = dtot + pl; it < 2 * pad_du; it += kGroup) {
        const int u = it >> 1, h = it & 1;
        U[u * 8 + h] = no_row;
        U[u * 8 + 4 + h] = no_row;
        reinterpret_cast<uint16_t*>(&U[u * 8 + 2])[h] = (uint16_t)(27 << 10);
        reinterpret_cast<uint16_t*>(&U[u * 8 + 3])[h] = 0;
      }
      for (int it = stot + pl; it < 4 * pad_su; it += kGroup) {
        const int u = pad_du + (it >> 2), sub = (it >> 1) & 1, h = it & 1;
        U[u * 8 + 4 * sub + h] = no_row;
        reinterpret_cast<uint16_t*>(&U[u * 8 + 4 * sub + 2])[h] = (uint16_t)(27 << 10);
        reinterpret_cast<uint16_t*>(&U[u * 8 + 4 * sub + 3])[h] = 0;
      }
      if (row == 0) s_beta[gg] = s_bpart[gg][0] + s_bpart[gg][1] + s_bpart[gg][2] + s_bpart[gg][3];
      nbd_v = pad_du / kSlots;
      nb_v = (pad_du + pad_su) / kSlots;
    }
    nb_g[2 * i] = __builtin_amdgcn_readlane(nb_v, 0);
    nb_g[2 * i + 1] = __builtin_amdgcn_readlane(nb_v, 32);
    nbd_g[2 * i] = __builtin_amdgcn_readlane(nbd_v, 0);
    nbd_g[2 * i + 1] = __builtin_amdgcn_readlane(nbd_v, 32);
  }
  // the scales come from HBM and arrive after x: stored last (a quarter of
  // each group's per wave)
#pragma unroll
  for (int gg = 0; gg < kPPMaxGW; ++gg)
    if (gg < ng) *(ScaleWord*)&s_scale[gg][(wave * 64 + lane) * SH] = scw[gg];
  __syncthreads();

  // ---- main loop: lane group lg takes units lg, lg + kLaneGroups, ... of
  // each batch; the (group, batch) sequence runs through four register sets,
  // three batches in flight while one is consumed.
  float yp[16], acc[16], off_d = 0.0f, off_s = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) yp[e] = acc[e] = 0.0f;

  struct Batch {
    uint32_t w[PB][4];     // plane dwords: descriptor words 0, 1, 4, 5
    uint32_t e[PB][4];     // descriptor words 2, 3, 6, 7
  };
  int bstart[kPPMaxGW + 1], bdbl[kPPMaxGW];
  bstart[0] = 0;
#pragma unroll
  for (int gg = 0; gg < kPPMaxGW; ++gg) {
    bstart[gg + 1] = bstart[gg] + nb_g[gg];
    bdbl[gg] = nbd_g[gg];
  }
  const int nbt = bstart[kPPMaxGW];
  auto group_of = [&](int b) {
    int gg = 0;
#pragma unroll
    for (int k = 1; k < kPPMaxGW; ++k) gg += (b >= bstart[k]) ? 1 : 0;
    return gg;
  };
  // Issue batch b (b >= nbt reads the all-empty batch): no test, no branch.
  auto fetch = [&](Batch& B, int b) {
    const int gg = group_of(b);
    const int u0 = (b - bstart[gg]) * kSlots;
    const uint32_t* base = b < nbt ? s_units[gg][u0] : s_empty[0];
#pragma unroll
    for (int q = 0; q < PB; ++q) {
      const uint32_t* src = base + (lg + kLaneGroups * q) * 8;
      const uint4 a = *(const uint4*)src;
      const uint4 c = *(const uint4*)(src + 4);
      B.e[q][0] = a.z;
      B.e[q][1] = a.w;
      B.e[q][2] = c.z;
      B.e[q][3] = c.w;
      B.w[q][0] = __builtin_nontemporal_load((const uint32_t*)(tile + (a.x + li4)));
      B.w[q][1] = __builtin_nontemporal_load((const uint32_t*)(tile + (a.y + li4)));
      B.w[q][2] = __builtin_nontemporal_load((const uint32_t*)(tile + (c.x + li4)));
      B.w[q][3] = __builtin_nontemporal_load((const uint32_t*)(tile + (c.y + li4)));
    }
  };
  auto consume = [&](const Batch& B, int b) {
    const int gg = group_of(b);
    const bool dbl = b < nbt && (b - bstart[gg]) < bdbl[gg];
    if (dbl) {
#pragma unroll
      for (int q = 0; q < PB; ++q) {
        off_d = dot2(B.e[q][0], B.e[q][1], off_d);
        consume_double(B.w[q][0], B.w[q][2], B.w[q][1], B.w[q][3], B.e[q][0], B.e[q][1], acc);
      }
    } else {
      float a2[1][16];
#pragma unroll
      for (int e = 0; e < 16; ++e) a2[0][e] = acc[e];
#pragma unroll
      for (int q = 0; q < PB; ++q) {
        const uint32_t xp0[1] = {B.e[q][1]}, xp1[1] = {B.e[q][3]};
        off_s = dot2(B.e[q][0], B.e[q][1], off_s);
        off_s = dot2(B.e[q][2], B.e[q][3], off_s);
        consume_pair<1, 16>(B.w[q][0], B.w[q][1], B.e[q][0], xp0, a2, 0);
        consume_pair<1, 16>(B.w[q][2], B.w[q][3], B.e[q][2], xp1, a2, 0);
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e] = a2[0][e];
    }
  };
  auto finish_group = [&](int gg) {
    float sc[16];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const uint4 v = *(const uint4*)&s_scale[gg][li * 16 + 8 * c];
      const uint32_t ww[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        sc[8 * c + 2 * h] = h2f((uint16_t)(ww[h] & 0xFFFFu));
        sc[8 * c + 2 * h + 1] = h2f((uint16_t)(ww[h] >> 16));
      }
    }
    const float beta = lg == 0 ? s_beta[gg] : 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float v = acc[e] - double_offset_factor(e) * off_d - offset_factor(e) * off_s;
      yp[e] = fmaf(sc[e], v + beta, yp[e]);
      acc[e] = 0.0f;
    }
    off_d = 0.0f;
    off_s = 0.0f;
  };
  auto after = [&](int b) {
    const int gg = group_of(b);
    if (b + 1 == bstart[gg + 1]) finish_group(gg);
  };

  // D register sets; the inner loop is unrolled so each set is a fixed group
  // of registers.  A workgroup with at most D-1 batches issues all its loads
  // before it consumes the first batch.
  Batch R[D];
#pragma unroll
  for (int i = 0; i < D - 1; ++i) fetch(R[i], i);
  if constexpr (SPEC) {
    // the read-ahead plane-1 rows of the first group, as singles (exponent
    // 29 - 2j at j = 1), while the first batches of the lists are in flight
    constexpr uint32_t e1 = (27u << 10) | (27u << 26);
    float a2[1][16];
#pragma unroll
    for (int e = 0; e < 16; ++e) a2[0][e] = acc[e];
#pragma unroll
    for (int q = 0; q < kSpecPerLG; ++q) {
      const int u = lg + kLaneGroups * q;
      const uint32_t xp0[1] = {s_spx[2 * u]}, xp1[1] = {s_spx[2 * u + 1]};
      off_s = dot2(e1, xp0[0], off_s);
      off_s = dot2(e1, xp1[0], off_s);
      consume_pair<1, 16>(spw[4 * q], spw[4 * q + 1], e1, xp0, a2, 0);
      consume_pair<1, 16>(spw[4 * q + 2], spw[4 * q + 3], e1, xp1, a2, 0);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = a2[0][e];
  }
  for (int b = 0; b < nbt; b += D) {
#pragma unroll
    for (int i = 0; i < D; ++i) {
      fetch(R[(i + D - 1) % D], b + i + D - 1);
      // a guard, not an exit: an early exit out of the unrolled body makes
      // the loop header wait for every load in flight
      if (b + i < nbt) {
        consume(R[i], b + i);
        after(b + i);
      }
    }
  }

  // ---- reduce: lane groups of a wave by lane swaps, waves through LDS, then
  // one atomic add per output
#pragma unroll
  for (int e = 0; e < 16; ++e) yp[e] = lane_group_sum<LPR>(yp[e]);
  if (lane < LPR) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      *(float4*)&s_red[wave][li * 16 + 4 * c] = make_float4(yp[4 * c], yp[4 * c + 1], yp[4 * c + 2], yp[4 * c + 3]);
  }
  __syncthreads();
  for (int o = tid; o < T; o += kThreads) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += s_red[w][o];
    atomicAdd(&y[(size_t)t * T + o], v * L.sfac);   // 8-bit code units -> b_max units
  }
}

template <int LPR>
void launch_pp(dim3 grid, hipStream_t s, const void* codes, const void* scales, const void* x,
               const uint8_t* lm, float* y, const Layer& L, int gw, int fused,
               const Thresholds& th, uint8_t* lm_out, int readahead) {
  // Plane-1 read-ahead pays where a CU holds about one workgroup, whose own
  // prologue is then the only thing to hide the first loads behind; with
  // more workgroups per CU the others hide it, and the read-ahead's level-0
  // rows only cost bandwidth.  The caller's hint decides when given (it
  // knows how many channels its budget skips); GRINQH_VMM_SPEC=0/1 forces
  // it for tests and sweeps.
  const char* forced = getenv("GRINQH_VMM_SPEC");
  const bool spec = forced ? atoi(forced) != 0 : (readahead >= 0 ? readahead != 0 : grid.x <= 384);
  if (spec)
    hipLaunchKernelGGL((k_vmm_pp<LPR, 2, GRINQH_PP_DEPTH, 256, true>), grid, dim3(256), 0, s,
                       (const uint8_t*)codes, (const uint16_t*)scales, (const uint16_t*)x, lm, y, L, gw, fused,
                       th, lm_out);
  else
    hipLaunchKernelGGL((k_vmm_pp<LPR, 2, GRINQH_PP_DEPTH, 256, false>), grid, dim3(256), 0, s,
                       (const uint8_t*)codes, (const uint16_t*)scales, (const uint16_t*)x, lm, y, L, gw, fused,
                       th, lm_out);
}

}  // namespace

bool vmm_pp_supported(const Layer& L, int B) {
  // byte offsets inside a tile are 32-bit
  return B == 1 && L.u == 2 && (L.T == 256 || L.T == 512 || L.T == 1024) &&
         (long long)L.K * L.RB < (1ll << 31);
}

int launch_vmm_pp(const Layer& L, const void* codes, const void* scales, const void* x,
                  const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out,
                  float* y, int readahead, hipStream_t s) {
  // groups per workgroup: about 512 workgroups, rounded to the nearest
  // count (896 units -> 2, 448 -> 1; measured on the Llama3-8B MLP shapes)
  int gw = (int)(((long)L.tiles * L.groups + 256) / 512);
  gw = gw < 1 ? 1 : (gw > kPPMaxGW ? kPPMaxGW : gw);
  if (const char* env = getenv("GRINQH_VMM_GW")) {
    const int v = atoi(env);
    if (v >= 1 && v <= kPPMaxGW) gw = v;
  }
  const dim3 grid((unsigned)(L.tiles * ((L.groups + gw - 1) / gw)));
  Thresholds none{};
  const Thresholds& tt = th ? *th : none;
  const int fused = th != nullptr;
  if (L.T == 256) launch_pp<16>(grid, s, codes, scales, x, level_map, y, L, gw, fused, tt, level_map_out, readahead);
  else if (L.T == 512) launch_pp<32>(grid, s, codes, scales, x, level_map, y, L, gw, fused, tt, level_map_out, readahead);
  else launch_pp<64>(grid, s, codes, scales, x, level_map, y, L, gw, fused, tt, level_map_out, readahead);
  return check_launch("vmm (plane pairs)");
}

}  // namespace grinqh
