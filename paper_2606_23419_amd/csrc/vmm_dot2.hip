// Nested-precision decode VMM for 2-bit planes (Sec. 3.3 reconstruction with
// the midpoint bias; App. C.1 sparse bit-loading), laid out for CDNA4.
//
// Work items are plane rows: (channel k, plane j) for j = 1 .. the depth that
// k's level asks for (for B > 1 tokens, the deepest of the B levels).  A
// workgroup owns one tile of T = 256*V outputs and `gw` consecutive groups of
// 128 channels.  Its prologue lists, per group, the plane rows to read and
// pairs consecutive ones; the main loop streams the pairs.
//
// A pair is consumed with v_dot2_f32_f16.  For 16 outputs a lane loads one
// dword of each plane row (sixteen 2-bit fields); v_perm_b32 puts eight
// outputs' fields of row 1 in the low half and of row 2 in the high half.  A
// field c at bit p of a half, OR-ed with the exponent bits E = 33 - 2j - p
// (fp16 bias 15), reads as the fp16 value 2^(18-2j-p) + c * 2^(8-2j): the
// field at its code-unit weight 2^(8-2j) plus an offset 2^(10-p) * 2^(8-2j).
// Fields at p in {4, 6, 8} are used as they lie, the others after a shift of
// the whole dword (<< 4 or >> 6), so eight fp16 pairs cost eight v_and_or_b32
// and two shifts.  One dot2 with the pair (x_k1, x_k2) then adds both rows'
// contributions to the output's fp32 accumulator.  The same dot2 applied to
// the bare exponent bits of position 4 (fields zero) gives 64 (x_k1 w_1 +
// x_k2 w_2), the pair's offset at p = 4; each lane group sums it alongside,
// so its partial sum can drop the offsets before anything is combined.
// Per group and output,
//   y_n += s_{g,n} * (acc_n - 2^(4-p(n)) * off_g + beta_g),
//   off_g  = sum over the group's pairs of 64 (x_k1 w_1 + x_k2 w_2),
//   beta_g = sum_{k: level > 0} x_k (phi_b - 128)  (midpoint bias, offset),
// which equals sum_k x_k s (t_k + phi - 128) with t_k the truncated code.
#include <type_traits>

#include "grinqh_internal.h"
#include "vmm_common.h"

namespace grinqh {

namespace {

using namespace vmmdev;

constexpr int kMaxGW = 4;                    // groups per workgroup (B = 1)
constexpr int max_gw(int nb) { return nb == 1 ? kMaxGW : 2; }   // LDS of the pair lists
// plane rows of a group: 128 rows x 8/U planes (4 two-bit or 8 one-bit planes)
constexpr int max_pairs(int u) { return kGroup * (8 / u) / 2; }

// Per-pair descriptor: byte offsets of the two plane chunks from the tile
// base, the fp16x2 exponent bits for field position 4, and one fp16x2
// coefficient pair per token (0 where that token does not read the plane).
template <int NB>
struct Desc {
  static constexpr int DW = NB == 1 ? 4 : 8;
};

template <int U, int V, int LPR, int NB, int PB, int kThreads>
__global__ __launch_bounds__(kThreads) void k_vmm_dot2(
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales,
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ lm, float* __restrict__ y,
    Layer L, int gw, int fused, Thresholds th, uint8_t* __restrict__ lm_out) {
  constexpr int T = LPR * 16 * V;        // outputs of the tile
  constexpr int NACC = 16 * V;           // outputs per lane
  constexpr int kLaneGroups = kThreads / LPR;
  constexpr int kWaves = kThreads / 64;
  constexpr int DW = Desc<NB>::DW;

  __shared__ __align__(16) uint32_t s_pairs[max_gw(NB)][max_pairs(U)][DW];
  __shared__ __align__(16) uint32_t s_empty[kThreads / LPR * PB][DW];   // one all-empty batch
  __shared__ float s_beta[max_gw(NB)][NB];
  __shared__ __align__(16) uint16_t s_scale[max_gw(NB)][T];
  // cross-wave sums, one token at a time (the buffer does not grow with the
  // tokens, so neither does the workgroup's LDS)
  __shared__ __align__(16) float s_red[kWaves][T];
  __shared__ int s_cnt[max_gw(NB)][kWaves][2];         // full pairs, lone items per group and wave
  __shared__ float s_bpart[max_gw(NB)][NB][kWaves];    // beta_g partial sums per wave

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x % L.tiles;
  const int g0 = (blockIdx.x / L.tiles) * gw;
  // the row that empty items read (zero coefficients): the workgroup's own
  // first row, in cache; one row shared by all workgroups of a tile made its
  // cache lines a hot spot
  const uint32_t no_row = (uint32_t)(g0 * kGroup) * (uint32_t)L.RB;
  const int ng = min(gw, L.groups - g0);
  const int n_top = L.n_levels - 1;
  const int lg = tid / LPR, li = tid % LPR;


  // ---- prologue.  The four waves grade the rows together: in pass i, lane
  // l of wave w takes row 32w + (l & 31) of group 2i + (l >> 5), so each half
  // wave covers 32 rows of one group.  A lane lists its row's plane rows
  // 1..D (D the deepest over the tokens) as the pairs (1,2), (3,4), ...; a
  // last odd plane is a lone item, and the group's lone items are paired
  // with each other after all full pairs (the second slot of an odd last one
  // repeats the first with zero coefficients).  A half wave's items follow
  // those of the lower waves' halves of the same group, whose counts are
  // exchanged through LDS.
  static_assert(kWaves == 4 && kGroup == 128, "32 rows per half wave");
  constexpr int kPasses = (max_gw(NB) + 1) / 2;
  constexpr int SH = T / 256;                // scale halves per lane and group
  constexpr int kMaxPlanes = 8 / U;
  const int half = lane >> 5, hl = lane & 31;
  const int row = 32 * wave + hl;            // row of the group
  // x, the level map and the scales are requested together, and
  // unconditionally (groups past the workgroup's last one read that one
  // again, from cache), so the compiler waits for x alone before grading
  uint32_t xv[kPasses][NB], lv[kPasses][NB];
  using ScaleWord = typename std::conditional<SH == 4, uint2, typename std::conditional<SH == 2, uint32_t, uint16_t>::type>::type;
  ScaleWord scw[max_gw(NB)];
  const uint8_t* lmsrc = fused ? (const uint8_t*)x : lm;   // in fused mode the read is ignored
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    const int k = (g0 + min(2 * i + half, ng - 1)) * kGroup + row;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      xv[i][b] = x[(size_t)b * L.K + k];
      lv[i][b] = lmsrc[(size_t)b * L.K + k];
    }
  }
#pragma unroll
  for (int gg = 0; gg < max_gw(NB); ++gg)
    scw[gg] = *(const ScaleWord*)(scales + (size_t)(g0 + min(gg, ng - 1)) * L.N + (size_t)t * T +
                                  (wave * 64 + lane) * SH);
  __builtin_amdgcn_sched_barrier(0);

  // grade, count pairs, local positions
  int dtok[kPasses][NB], dmax[kPasses], ppos[kPasses], lpos[kPasses];
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    if (i > 0 && 2 * i >= ng) break;         // uniform: the groups of this pass are absent
    const int gg = 2 * i + half;
    const bool valid = gg < ng;
    int D = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float fx = h2f((uint16_t)xv[i][b]);
      // graded from x (th.n is 0 without thresholds) or read from the level
      // map, chosen without a branch so that the level-map load stays early
      int graded = 0;
      const float ax = fabsf(fx);
#pragma unroll
      for (int j = 0; j < kMaxLevels - 1; ++j)   // unused thresholds are +inf: no
        graded += ax >= th.theta[j] ? 1 : 0;     // branch, all loaded up front
      const int lvl = min(fused ? graded : (int)(lv[i][b] & 0xFFu), n_top);
      if (fused && lm_out && t == 0 && valid) lm_out[(size_t)b * L.K + (g0 + gg) * kGroup + row] = (uint8_t)lvl;
      const int d = valid ? level_planes(L.planes_packed, lvl) : 0;
      dtok[i][b] = d;
      D = max(D, d);
      const float bs = half_sum_dpp(d ? fx * phi_minus_offset(U * d, L.bmax) : 0.0f);
      if (valid && hl == 0) s_bpart[gg][b][wave] = bs;
    }
    dmax[i] = D;
    const int np = D >> 1;                   // full pairs
    int pos = 0, tot = 0;
#pragma unroll
    for (int q = 1; q <= kMaxPlanes / 2; ++q) {
      pos += half_below(np >= q);
      tot += half_total(np >= q);
    }
    ppos[i] = pos;
    lpos[i] = half_below(D & 1);
    const int ltot = half_total(D & 1);
    if (valid && hl == 0) {
      s_cnt[gg][wave][0] = tot;
      s_cnt[gg][wave][1] = ltot;
    }
  }
  for (int i = tid; i < (kThreads / LPR * PB) * DW; i += kThreads)
    (&s_empty[0][0])[i] = (i % DW == 2) ? ((27u << 10) | (27u << 26)) : (i % DW < 2 ? no_row : 0u);
  __syncthreads();

  // pairs at their places; padding and the per-group totals.  Lanes 0 and
  // 32 hand each pass's pair counts to the whole wave in scalar registers,
  // so the main loop starts without reading them back from LDS.
  static_assert(max_gw(NB) % 2 == 0, "two groups per pass");
  int np_g[max_gw(NB)] = {};
#pragma unroll
  for (int i = 0; i < kPasses; ++i) {
    if (i > 0 && 2 * i >= ng) break;
    const int gg = 2 * i + half;
    int np_v = 0;
    if (gg < ng) {
      int base = 0, ftot = 0, lbase = 0, ltot = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const int c = s_cnt[gg][w][0], l = s_cnt[gg][w][1];
        base += w < wave ? c : 0;
        ftot += c;
        lbase += w < wave ? l : 0;
        ltot += l;
      }
      const int total = ftot + ((ltot + 1) >> 1);
      const int k = (g0 + gg) * kGroup + row;
      const int D = dmax[i];
      // plane j of width U is worth 2^(8 - U j) code units: exponent base 29 - U j
#pragma unroll
      for (int q = 0; q < kMaxPlanes / 2; ++q) {
        if (2 * q + 2 > D) break;
        const int ja = 2 * q + 1, jb = ja + 1;
        uint32_t* d = s_pairs[gg][base + ppos[i] + q];
        d[0] = (uint32_t)(k * L.RB + (ja - 1) * (T * U / 8));
        d[1] = (uint32_t)(k * L.RB + (jb - 1) * (T * U / 8));
        d[2] = ((uint32_t)(29 - U * ja) << 10) | ((uint32_t)(29 - U * jb) << 26);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const uint32_t xt = xv[i][b] & 0xFFFFu;
          const uint32_t c1 = ja <= dtok[i][b] ? xt : 0u;
          const uint32_t c2 = jb <= dtok[i][b] ? xt : 0u;
          d[3 + b] = c1 | (c2 << 16);
        }
#pragma unroll
        for (int w = 3 + NB; w < DW; ++w) d[w] = 0u;
      }
      if (D & 1) {
        // lone item li of the group: pair ftot + li/2, slot li%2 (16-bit
        // halves of the exponent and coefficient words)
        const int j = D;
        const int it = lbase + lpos[i], slot = it & 1;
        uint32_t* d = s_pairs[gg][ftot + (it >> 1)];
        const uint32_t off = (uint32_t)(k * L.RB + (j - 1) * (T * U / 8));
        const uint16_t ex = (uint16_t)((29 - U * j) << 10);
        d[slot] = off;
        reinterpret_cast<uint16_t*>(&d[2])[slot] = ex;
#pragma unroll
        for (int b = 0; b < NB; ++b)
          reinterpret_cast<uint16_t*>(&d[3 + b])[slot] = j <= dtok[i][b] ? (uint16_t)xv[i][b] : (uint16_t)0;
        if (slot == 0) {
#pragma unroll
          for (int w = 3 + NB; w < DW; ++w) d[w] = 0u;
          if (it == ltot - 1) {   // odd count: the last pair's second slot is empty (zero coefficients)
            d[1] = no_row;
            reinterpret_cast<uint16_t*>(&d[2])[1] = ex;
#pragma unroll
            for (int b = 0; b < NB; ++b) reinterpret_cast<uint16_t*>(&d[3 + b])[1] = 0;
          }
        }
      }
      // pad the list to whole batches with empty descriptors (zero
      // coefficients, a cached row, a finite exponent word), spread over the
      // group's 128 lanes, so the main loop needs no bounds tests; an empty
      // list still gets one batch (its group epilogue runs)
      constexpr int kSlots = kThreads / LPR * PB;
      const int padded = total > 0 ? (total + kSlots - 1) / kSlots * kSlots : kSlots;
      for (int it = total + row; it < padded; it += kGroup) {
        uint32_t* d = s_pairs[gg][it];
        d[0] = no_row;
        d[1] = no_row;
        d[2] = (27u << 10) | (27u << 26);
#pragma unroll
        for (int w = 3; w < DW; ++w) d[w] = 0u;
      }
      if (row == 0) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
          s_beta[gg][b] = s_bpart[gg][b][0] + s_bpart[gg][b][1] + s_bpart[gg][b][2] + s_bpart[gg][b][3];
      }
      np_v = total;
    }
    np_g[2 * i] = __builtin_amdgcn_readlane(np_v, 0);
    np_g[2 * i + 1] = __builtin_amdgcn_readlane(np_v, 32);
  }
  // the scales come from HBM and arrive after x: stored last (a quarter of
  // each group's per wave)
#pragma unroll
  for (int gg = 0; gg < max_gw(NB); ++gg)
    if (gg < ng) *(ScaleWord*)&s_scale[gg][(wave * 64 + lane) * SH] = scw[gg];
  __syncthreads();

  // ---- main loop: lane group lg takes pairs lg, lg + 16, ... of every group.
  // The (group, batch) sequence runs through four register sets, three
  // batches in flight while one is consumed, across group boundaries too.  A
  // group with no pairs still gets one (empty) batch so its epilogue runs.
  // 16 V outputs per lane.  With 1-bit planes a lane's fields are two bytes
  // of a plane row: it loads the aligned dword that holds them (its
  // neighbour's two bytes are the other half) and keeps its half when the
  // batch is consumed.  Plane rows start at multiples of four bytes.
  static_assert(U == 2 || V == 1, "1-bit planes: one 16-output word per lane");
  const int lane_byte = li * 2 * U * V;
  // (the base stays the same in every lane and the lane's part is added to
  // each 32-bit offset, so a load takes a scalar base and one offset register)
  const uint8_t* tile = codes + (size_t)t * L.K * L.RB;
  const uint32_t lane_off = (uint32_t)(U == 2 ? lane_byte : (lane_byte & ~3));
  const int half_sh = U == 2 ? 0 : (lane_byte & 2) * 8;
  float yp[NB][NACC], acc[NB][NACC], off[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    off[b] = 0.0f;
#pragma unroll
    for (int e = 0; e < NACC; ++e) yp[b][e] = acc[b][e] = 0.0f;
  }

  // A batch in flight keeps what the math needs: per pair the exponent word,
  // the coefficient pairs and the two loaded words (offsets are used at fetch)
  struct Batch {
    uint32_t m4[PB];
    uint32_t xp[PB][NB];
    uint32_t w1[PB][V], w2[PB][V];
  };
  // flattened batch sequence: group gg owns batches [bstart[gg], bstart[gg+1])
  int bstart[max_gw(NB) + 1];
  bstart[0] = 0;
#pragma unroll
  for (int gg = 0; gg < max_gw(NB); ++gg) {
    int r = gg < ng ? (np_g[gg] + kLaneGroups * PB - 1) / (kLaneGroups * PB) : 0;
    if (gg < ng && r == 0) r = 1;   // an empty group still gets its epilogue
    bstart[gg + 1] = bstart[gg] + r;
  }
  const int nbt = bstart[max_gw(NB)];
  auto group_of = [&](int b) {
    int gg = 0;
#pragma unroll
    for (int k = 1; k < max_gw(NB); ++k) gg += (b >= bstart[k]) ? 1 : 0;
    return gg;
  };
  // Issue batch b (b >= nbt reads the all-empty batch).  There is no test
  // and no branch: each group's list is padded to whole batches with empty
  // descriptors (the workgroup's first row, cached and in bounds; zero
  // coefficients; a finite exponent word, so masked fields stay finite and
  // cancel).  With straight-line loads the compiler counts them exactly and
  // waits only for the batch being consumed.
  auto fetch = [&](Batch& B, int b) {
    const int gg = group_of(b);
    const int r0 = (b - bstart[gg]) * PB;
    const uint32_t* base = b < nbt ? s_pairs[gg][r0 * kLaneGroups] : s_empty[0];
#pragma unroll
    for (int q = 0; q < PB; ++q) {
      const uint32_t* src = base + (lg + kLaneGroups * q) * DW;
      const uint4 a = *(const uint4*)src;
      B.m4[q] = a.z;
      if constexpr (DW == 4) {
        B.xp[q][0] = a.w;
      } else {
        const uint4 c = *(const uint4*)(src + 4);
        const uint32_t cw[5] = {a.w, c.x, c.y, c.z, c.w};
#pragma unroll
        for (int b = 0; b < NB; ++b) B.xp[q][b] = cw[b];
      }
#pragma unroll
      for (int v = 0; v < V; ++v) {
        B.w1[q][v] = __builtin_nontemporal_load((const uint32_t*)(tile + (a.x + lane_off + 4 * v)));
        B.w2[q][v] = __builtin_nontemporal_load((const uint32_t*)(tile + (a.y + lane_off + 4 * v)));
      }
    }
  };
  auto consume = [&](const Batch& B) {
#pragma unroll
    for (int q = 0; q < PB; ++q) {
#pragma unroll
      for (int b = 0; b < NB; ++b) off[b] = dot2(B.m4[q], B.xp[q][b], off[b]);
      if constexpr (U == 2) {
#pragma unroll
        for (int v = 0; v < V; ++v)
          consume_pair<NB, NACC>(B.w1[q][v], B.w2[q][v], B.m4[q], B.xp[q], acc, 16 * v);
      } else {
        // the lane's sixteen 1-bit fields moved to bit 2o: the 2-bit field
        // machinery then reads each as 0 or 1 at the plane's own weight
        const uint32_t w1 = spread_bits((B.w1[q][0] >> half_sh) & 0xFFFFu);
        const uint32_t w2 = spread_bits((B.w2[q][0] >> half_sh) & 0xFFFFu);
        consume_pair<NB, NACC>(w1, w2, B.m4[q], B.xp[q], acc, 0);
      }
    }
  };
  // group epilogue (no global loads): scale from LDS, bias once per output
  auto finish_group = [&](int gg) {
    float sc[NACC];
#pragma unroll
    for (int c = 0; c < NACC / 8; ++c) {
      const uint4 v = *(const uint4*)&s_scale[gg][li * NACC + 8 * c];
      const uint32_t ww[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        sc[8 * c + 2 * h] = h2f((uint16_t)(ww[h] & 0xFFFFu));
        sc[8 * c + 2 * h + 1] = h2f((uint16_t)(ww[h] >> 16));
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float beta = lg == 0 ? s_beta[gg][b] : 0.0f;
#pragma unroll
      for (int e = 0; e < NACC; ++e) {
        yp[b][e] = fmaf(sc[e], (acc[b][e] - offset_factor(e) * off[b]) + beta, yp[b][e]);
        acc[b][e] = 0.0f;
      }
      off[b] = 0.0f;
    }
  };
  auto after = [&](int b) {   // close the group whose last batch b was
    const int gg = group_of(b);
    if (b + 1 == bstart[gg + 1]) finish_group(gg);
  };

  // four register sets: batches b+1 .. b+3 are in flight while b is
  // consumed.  The inner loop is unrolled so each set is a fixed group of
  // registers, and its end is a guard rather than an exit: an exit out of the
  // unrolled body makes the loop header wait for every load in flight.
  Batch R[4];
  fetch(R[0], 0);
  fetch(R[1], 1);
  fetch(R[2], 2);
  for (int b = 0; b < nbt; b += 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fetch(R[(i + 3) % 4], b + i + 3);
      if (b + i < nbt) {
        consume(R[i]);
        after(b + i);
      }
    }
  }

  // ---- reduce: the four lane groups of a wave with lane swaps, the waves
  // through LDS, then one atomic add per output
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int e = 0; e < NACC; ++e) yp[b][e] = lane_group_sum<LPR>(yp[b][e]);
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    if (b > 0) __syncthreads();   // the previous token's sums are read
    if (lane < LPR) {
#pragma unroll
      for (int c = 0; c < NACC / 4; ++c)
        *(float4*)&s_red[wave][li * NACC + 4 * c] =
            make_float4(yp[b][4 * c], yp[b][4 * c + 1], yp[b][4 * c + 2], yp[b][4 * c + 3]);
    }
    __syncthreads();
    for (int o = tid; o < T; o += kThreads) {
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += s_red[w][o];
      atomicAdd(&y[(size_t)b * L.N + (size_t)t * T + o], v * L.sfac);   // 8-bit units -> b_max units
    }
  }
}

template <int U, int V, int LPR, int NB, int NT>
void launch_one(dim3 grid, hipStream_t s, const void* codes, const void* scales, const void* x,
                const uint8_t* lm, float* y, const Layer& L, int gw, int fused,
                const Thresholds& th, uint8_t* lm_out) {
  constexpr int PB = (V == 1 && NB <= 2) ? 4 : 2;   // pairs per batch; four batches in flight
  hipLaunchKernelGGL((k_vmm_dot2<U, V, LPR, NB, PB, NT>), grid, dim3(NT), 0, s, (const uint8_t*)codes,
                     (const uint16_t*)scales, (const uint16_t*)x, lm, y, L, gw, fused, th, lm_out);
}

}  // namespace

// Tiles of 256, 512 or 1024 outputs (512 or 1024 for 1-bit planes): 16
// outputs per lane and plane row, so 16, 32 or 64 lanes cover a plane row.
bool vmm_dot2_supported(const Layer& L) {
  if (L.u == 2) return L.T == 256 || L.T == 512 || L.T == 1024;
  return L.T == 512 || L.T == 1024;
}

int vmm_dot2_groups_per_wg(const Layer& L) {
  if (const int v = option(&Options::groups_per_wg)) return v <= kMaxGW ? v : kMaxGW;
  // 2-bit planes: about 512 workgroups (two per CU), rounded to the nearest
  // count (decode B = 2, 4 at 896 units: -4 to -10% with 2 groups).  1-bit
  // planes: one group per workgroup below 1536 units (Qwen3-8B at T = 512:
  // down, 768 units, 25% slower with 2; gate|up, 1536 units, best with 2).
  const long units = (long)L.tiles * L.groups;
  int gw = L.u == 2 ? (int)((units + 256) / 512) : (int)(units / 768);
  return gw < 1 ? 1 : (gw > kMaxGW ? kMaxGW : gw);
}

int launch_vmm_dot2(const Layer& L, const void* codes, const void* scales, const void* x,
                    const uint8_t* level_map, const Thresholds* th, uint8_t* level_map_out,
                    int B, float* y, hipStream_t s) {
  const int gw = min(vmm_dot2_groups_per_wg(L), max_gw(B));
  const dim3 grid((unsigned)(L.tiles * ((L.groups + gw - 1) / gw)));
  Thresholds none{};
  const Thresholds& tt = th ? *th : none;
  const int fused = th != nullptr;
#define GRINQH_DOT2_CASE(UU, TT, LL, NN)                                                          \
  if (L.u == UU && L.T == TT && B == NN) {                                                       \
    launch_one<UU, 1, LL, NN, 256>(grid, s, codes, scales, x, level_map, y, L, gw, fused, tt, level_map_out); \
    return check_launch("vmm (dot2)");                                                           \
  }
  GRINQH_DOT2_CASE(2, 256, 16, 1) GRINQH_DOT2_CASE(2, 256, 16, 2) GRINQH_DOT2_CASE(2, 256, 16, 3) GRINQH_DOT2_CASE(2, 256, 16, 4)
  GRINQH_DOT2_CASE(2, 512, 32, 1) GRINQH_DOT2_CASE(2, 512, 32, 2) GRINQH_DOT2_CASE(2, 512, 32, 3) GRINQH_DOT2_CASE(2, 512, 32, 4)
  GRINQH_DOT2_CASE(2, 1024, 64, 1) GRINQH_DOT2_CASE(2, 1024, 64, 2) GRINQH_DOT2_CASE(2, 1024, 64, 3) GRINQH_DOT2_CASE(2, 1024, 64, 4)
  GRINQH_DOT2_CASE(1, 512, 32, 1) GRINQH_DOT2_CASE(1, 512, 32, 2) GRINQH_DOT2_CASE(1, 512, 32, 3) GRINQH_DOT2_CASE(1, 512, 32, 4)
  GRINQH_DOT2_CASE(1, 1024, 64, 1) GRINQH_DOT2_CASE(1, 1024, 64, 2) GRINQH_DOT2_CASE(1, 1024, 64, 3) GRINQH_DOT2_CASE(1, 1024, 64, 4)
#undef GRINQH_DOT2_CASE
  return fail(GRINQH_EUNSUPPORTED, "dot2 VMM: no kernel for tile %d, B=%d", L.T, B);
}

}  // namespace grinqh
