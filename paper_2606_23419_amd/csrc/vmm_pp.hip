// Nested-precision decode VMM at batch 1 for 2-bit planes (Sec. 3.3
// reconstruction with the midpoint bias; App. C.1 sparse bit-loading), laid
// out for CDNA4.
//
// Each wave grades its own 32 rows of every group of its workgroup and sorts
// them, with two ballots, into "big" rows (3 or 4 planes to read) and "small"
// rows (1 or 2).  A batch gives each lane group either two big rows, planes
// 1-4 of each, or four small rows, planes 1-2 of each: eight plane dwords per
// lane either way.  The plane a row may lack (plane 4 of a 3-plane row,
// plane 2 of a 1-plane row) is read from an offset outside the tile's buffer
// resource, which returns zero without a memory access; a zero plane is
// exactly what truncating the code to the row's depth leaves there.  Every
// batch issues the same loads; a group's big batches come first, so the kind
// of a batch is one scalar compare.
//
// Small batches: a plane pair (j, j+1) of two channels.  The two 2-bit fields
// of an output merge into one 4-bit field F = 4 c_j + c_(j+1) worth
// F 2^(6-2j); v_perm_b32 puts one byte of each channel in the two halves of a
// dword, v_and_or_b32 adds the exponent bits E = 31 - 2j - p (fp16 bias 15)
// so the field at bit p reads as 2^(16-2j-p) + F 2^(6-2j), and one
// v_dot2_f32_f16 with (x_k1, x_k2) adds both channels.  The offsets the
// exponent bits add are summed per lane alongside and taken out at the end
// of each group:
//   y_n += s_{g,n} (acc_n - f(n) off - off8 + beta_g),
// with f = 2^(-p) for the output's field position p and beta_g = sum over the
// wave's active rows of x_k (phi_b - 128) (midpoint bias and code offset).
//
// Big batches: the four planes of two channels merge into each output's full
// 8-bit code, read with exponent bits 25 as 2^10 + F, one v_dot2_f32_f16 per
// output for both channels; their offset 2^10 per channel is summed in off8.
// The waves meet once, to sum their partial outputs.
#include "grinqh_internal.h"
#include "topk_select.h"
#include "vmm_common.h"

namespace grinqh {

namespace {

using namespace vmmdev;

// 16 outputs, two channels, planes (j, j+1) of each: w?a = plane j, w?b = j+1.
__device__ __forceinline__ void consume_double(uint32_t w1a, uint32_t w1b, uint32_t w2a,
                                               uint32_t w2b, uint32_t m0, uint32_t xp,
                                               float (&acc)[16]) {
  const uint32_t E1 = ((w1a << 2) & 0xCCCCCCCCu) | (w1b & 0x33333333u);
  const uint32_t O1 = (w1a & 0xCCCCCCCCu) | ((w1b >> 2) & 0x33333333u);
  const uint32_t E2 = ((w2a << 2) & 0xCCCCCCCCu) | (w2b & 0x33333333u);
  const uint32_t O2 = (w2a & 0xCCCCCCCCu) | ((w2b >> 2) & 0x33333333u);
  const uint32_t m4 = m0 - 0x10001000u;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const uint32_t S1 = s ? O1 : E1, S2 = s ? O2 : E2;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t lo = __builtin_amdgcn_perm(S2, S1, h ? 0x0C060C02u : 0x0C040C00u);
      const uint32_t hi = __builtin_amdgcn_perm(S2, S1, h ? 0x0C070C03u : 0x0C050C01u);
      const int e = 8 * h + s;
      acc[e] = dot2r((lo & 0x000F000Fu) | m0, xp, acc[e]);
      acc[e + 2] = dot2r((lo & 0x00F000F0u) | m4, xp, acc[e + 2]);
      acc[e + 4] = dot2r((hi & 0x000F000Fu) | m0, xp, acc[e + 4]);
      acc[e + 6] = dot2r((hi & 0x00F000F0u) | m4, xp, acc[e + 6]);
    }
  }
}

// Planes 1-4 of 16 outputs, two channels (a = first row, b = second): the
// four 2-bit fields of an output merge into its full 8-bit code
// F = 64 c_1 + 16 c_2 + 4 c_3 + c_4, which with exponent bits 25 reads as
// 2^10 + F in fp16, so one v_dot2_f32_f16 adds both channels' codes.  The
// nibble pairs (1,2) and (3,4) are merged first as in consume_double, then
// a byte takes the pair-(1,2) nibble on top of the pair-(3,4) nibble; output
// e keeps the accumulator it has in consume_double.
__device__ __forceinline__ void consume_quad(const uint32_t (&w)[8], uint32_t xp,
                                             float (&acc)[16]) {
  constexpr uint32_t kHi = 0xCCCCCCCCu, kLo = 0x33333333u, kNib = 0x0F0F0F0Fu;
  constexpr uint32_t kExp = 0x64006400u;   // exponent bits 25 in both halves
  uint32_t X[2][4];   // [channel][L_E, L_O, H_E, H_O]
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const uint32_t p1 = w[2 * c], p2 = w[2 * c + 1], p3 = w[4 + 2 * c], p4 = w[5 + 2 * c];
    const uint32_t E12 = ((p1 << 2) & kHi) | (p2 & kLo), O12 = (p1 & kHi) | ((p2 >> 2) & kLo);
    const uint32_t E34 = ((p3 << 2) & kHi) | (p4 & kLo), O34 = (p3 & kHi) | ((p4 >> 2) & kLo);
    X[c][0] = ((E12 << 4) & ~kNib) | (E34 & kNib);   // low nibbles of E bytes
    X[c][1] = ((O12 << 4) & ~kNib) | (O34 & kNib);
    X[c][2] = (E12 & ~kNib) | ((E34 >> 4) & kNib);   // high nibbles of E bytes
    X[c][3] = (O12 & ~kNib) | ((O34 >> 4) & kNib);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int s = q & 1, n = q >> 1;   // E/O set, nibble of the byte
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      // bytes 2h and 2h+1 of both channels: [a_k, b_k, a_k+1, b_k+1]
      const uint32_t G = __builtin_amdgcn_perm(X[1][q], X[0][q], h ? 0x07030602u : 0x05010400u);
      const uint32_t lo = __builtin_amdgcn_perm(kExp, G, 0x07010500u);
      const uint32_t hi = __builtin_amdgcn_perm(kExp, G, 0x07030502u);
      const int e = s + 2 * n + 8 * h;
      acc[e] = dot2r(lo, xp, acc[e]);
      acc[e + 4] = dot2r(hi, xp, acc[e + 4]);
    }
  }
}

__device__ __forceinline__ float double_offset_factor(int e) {
  return ((e >> 1) & 1) ? 0.0625f : 1.0f;
}

template <int LPR, int D, bool TOPK>
__global__ __launch_bounds__(256) void k_vmm_sr(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ lm, int gw, int groups, int fused,
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales, float* __restrict__ y,
    Layer L, Thresholds th, TopkCuts tk, uint8_t* __restrict__ lm_out) {
  constexpr int T = LPR * 16;            // outputs of the tile
  constexpr int PLANE = T / 4;           // bytes of one plane row
  constexpr int NLG = 64 / LPR;          // lane groups per wave
  constexpr int kWaves = 4;
  constexpr int MAXG = 2;                // groups per workgroup at most; gw is 1 or 2
  constexpr int BR = 2 * NLG;            // big rows per batch of a wave
  constexpr int SR = 4 * NLG;            // small rows per batch of a wave
  constexpr int MB = 32 / BR + 2;        // batches per (wave, group) at most
  // fp16 exponent bits of a merged pair's field at p = 0: 31 - 2j for the
  // pair of planes (j, j+1); 27 for empty entries (any finite value)
  constexpr uint32_t kE12 = 29u << 10, kE34 = 25u << 10, kEmpty = 27u << 10;

  // lists: per (wave, group, batch, lane group) four entries as three
  // 4-dword fields: offsets of plane j, of plane j+1, and (x | exponent << 16)
  __shared__ __align__(16) uint32_t s_ent[kWaves][MAXG][MB][NLG][3][4];
  __shared__ __align__(16) uint32_t s_empty[kWaves][3][4];
  __shared__ __align__(16) float s_red[kWaves][T];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, hl = lane & 31;
  const int t = blockIdx.x;
  const int g0 = blockIdx.y * gw;
  const int ng = min(gw, groups - g0);
  // loads first: x and the level map of this lane's row (lanes 0-31 the
  // first group, 32-63 the second).  They need no field of L, so they go
  // out before the wave waits for the layer's scalars (x, lm, gw, groups and
  // fused lead the argument list and arrive preloaded in scalar registers)
  const int gg = half;
  const bool valid = gg < ng;
  const int k = (g0 + min(gg, ng - 1)) * kGroup + 32 * wave + hl;
  const uint32_t xv = x[k];
  const uint32_t lv = (fused ? (const uint8_t*)x : lm)[k];   // ignored when graded here
  const int lg = lane / LPR, li = lane % LPR;
  const int n_top = L.n_levels - 1;
  const __amdgpu_buffer_rsrc_t rsrc = tile_rsrc(codes + (size_t)t * L.K * L.RB, L);
  const uint32_t li4 = (uint32_t)li * 4u;

  // the scales of this lane's 16 outputs for both groups (a group past the
  // last reads the last one again, from cache)
  uint4 scw[MAXG][2];
#pragma unroll
  for (int g = 0; g < MAXG; ++g) {
    const uint16_t* sp = scales + (size_t)(g0 + min(g, ng - 1)) * L.N + (size_t)t * T + li * 16;
    scw[g][0] = *(const uint4*)sp;
    scw[g][1] = *(const uint4*)(sp + 8);
  }
  if (lane < 12) (&s_empty[wave][0][0])[lane] = lane < 8 ? kNoRow : (kEmpty << 16);

  // top-k mode: the token's cuts from the whole x, the same in every workgroup
  // (top-k kernels only: the others hold no selection scratch)
  __shared__ __align__(16) uint8_t s_tk_raw[TOPK ? sizeof(topksel::Scratch) : 16];
  topksel::Scratch& s_tk = *reinterpret_cast<topksel::Scratch*>(s_tk_raw);
  if constexpr (TOPK) topksel::select_cuts(x, L.K, tk, s_tk);

  // ---- grade, sort into big and small rows, write this wave's lists
  const float fx = h2f((uint16_t)xv);
  const float ax = fabsf(fx);
  int graded = 0;
#pragma unroll
  for (int j = 0; j < kMaxLevels - 1; ++j) graded += ax >= th.theta[j] ? 1 : 0;
  const int lvl = min(fused == 1 ? graded
                      : TOPK ? topksel::level_of(xv, k, tk.n, s_tk)
                                   : (int)(lv & 0xFFu),
                      n_top);
  if (fused && lm_out && t == 0 && valid) lm_out[k] = (uint8_t)lvl;
  const int d = valid ? level_planes(L.planes_packed, lvl) : 0;
  const bool big = d >= 3, small = d == 1 || d == 2;
  const int nbig = half_total(big), nsm = half_total(small);
  const int rank = big ? half_below(big) : half_below(small);
  const int nbb = (nbig + BR - 1) / BR, nsb = (nsm + SR - 1) / SR;
  const float bs = half_sum_dpp(d ? fx * phi_minus_offset(2 * d, L.bmax) : 0.0f);
  {
    uint32_t* E = &s_ent[wave][gg][0][0][0][0];
    const uint32_t base = (uint32_t)k * (uint32_t)L.RB;
    const uint32_t xh = xv & 0xFFFFu;
    auto put = [&](int b, int lgp, int s, uint32_t o1, uint32_t o2, uint32_t xe) {
      uint32_t* p = E + (b * NLG + lgp) * 12 + s;
      p[0] = o1;
      p[4] = o2;
      p[8] = xe;
    };
    if (valid && big) {
      const int b = rank / BR, w = rank % BR;
      put(b, w >> 1, w & 1, base, base + PLANE, xh | (kE12 << 16));
      put(b, w >> 1, (w & 1) + 2, base + 2 * PLANE, d >= 4 ? base + 3 * PLANE : kNoRow, xh | (kE34 << 16));
    }
    if (valid && small) {
      const int b = nbb + rank / SR, w = rank % SR;
      put(b, w >> 2, w & 3, base, d >= 2 ? base + PLANE : kNoRow, xh | (kE12 << 16));
    }
    // empty entries up to whole batches: no memory access, zero coefficient
    if (valid) {
      for (int r = nbig + hl; r < nbb * BR; r += 32) {
        const int b = r / BR, w = r % BR;
        put(b, w >> 1, w & 1, kNoRow, kNoRow, kEmpty << 16);
        put(b, w >> 1, (w & 1) + 2, kNoRow, kNoRow, kEmpty << 16);
      }
      for (int r = nsm + hl; r < nsb * SR; r += 32) {
        const int b = nbb + r / SR, w = r % SR;
        put(b, w >> 2, w & 3, kNoRow, kNoRow, kEmpty << 16);
      }
    }
  }
  const int nb_v = valid ? nbb + nsb : 0;
  const int nbb_v = valid ? nbb : 0;
  int nb_g[MAXG];
  float beta_g[MAXG];
  nb_g[0] = __builtin_amdgcn_readlane(nb_v, 0);
  nb_g[1] = __builtin_amdgcn_readlane(nb_v, 32);
  const int nbb0 = __builtin_amdgcn_readlane(nbb_v, 0), nbb1 = __builtin_amdgcn_readlane(nbb_v, 32);
  beta_g[0] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bs), 0));
  beta_g[1] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bs), 32));
  // the lists and the empty batch are this wave's own: its LDS accesses
  // complete in order, so keeping the compiler from moving the reads above
  // the writes is enough
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // ---- main loop over this wave's (group, batch) sequence: D register sets,
  // D-1 batches in flight while one is consumed
  float yp[16], acc[16], off = 0.0f, off8 = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) yp[e] = acc[e] = 0.0f;

  struct Batch {
    uint32_t w[8];
    uint32_t xe[4];
  };
  const int bstart1 = nb_g[0], nbt = nb_g[0] + nb_g[1];
  auto fetch = [&](Batch& B, int b) {
    const int g = b >= bstart1 ? 1 : 0;
    const int lb = b - (g ? bstart1 : 0);
    const uint32_t* src = b < nbt ? &s_ent[wave][g][lb][lg][0][0] : &s_empty[wave][0][0];
    const uint4 o1 = *(const uint4*)src;
    const uint4 o2 = *(const uint4*)(src + 4);
    const uint4 xe = *(const uint4*)(src + 8);
    B.xe[0] = xe.x;
    B.xe[1] = xe.y;
    B.xe[2] = xe.z;
    B.xe[3] = xe.w;
    B.w[0] = load_plane(rsrc, o1.x + li4);
    B.w[1] = load_plane(rsrc, o2.x + li4);
    B.w[2] = load_plane(rsrc, o1.y + li4);
    B.w[3] = load_plane(rsrc, o2.y + li4);
    B.w[4] = load_plane(rsrc, o1.z + li4);
    B.w[5] = load_plane(rsrc, o2.z + li4);
    B.w[6] = load_plane(rsrc, o1.w + li4);
    B.w[7] = load_plane(rsrc, o2.w + li4);
  };
  auto consume_big = [&](const Batch& B) {
    const uint32_t xp = __builtin_amdgcn_perm(B.xe[1], B.xe[0], 0x05040100u);
    off8 = dot2r(0x64006400u, xp, off8);
    consume_quad(B.w, xp, acc);
  };
  auto consume = [&](const Batch& B) {
    // (x_k1, x_k2) from the entries' low halves, the exponent bits from the high halves
    const uint32_t xpa = __builtin_amdgcn_perm(B.xe[1], B.xe[0], 0x05040100u);
    const uint32_t m0a = __builtin_amdgcn_perm(B.xe[1], B.xe[0], 0x07060302u);
    const uint32_t xpb = __builtin_amdgcn_perm(B.xe[3], B.xe[2], 0x05040100u);
    const uint32_t m0b = __builtin_amdgcn_perm(B.xe[3], B.xe[2], 0x07060302u);
    off = dot2r(m0a, xpa, off);
    off = dot2r(m0b, xpb, off);
    consume_double(B.w[0], B.w[1], B.w[2], B.w[3], m0a, xpa, acc);
    consume_double(B.w[4], B.w[5], B.w[6], B.w[7], m0b, xpb, acc);
  };
  // the group being consumed, the end of its big batches and of all its
  // batches (a group without batches has no rows to add and is skipped)
  int cur_g = nb_g[0] > 0 ? 0 : 1;
  int cur_bigend = cur_g == 0 ? nbb0 : bstart1 + nbb1;
  int next_fin = cur_g == 0 ? bstart1 : nbt;
  auto finish_group = [&]() {
    float sc[16];
    const bool g1 = cur_g != 0;
    const uint32_t ww[8] = {g1 ? scw[1][0].x : scw[0][0].x, g1 ? scw[1][0].y : scw[0][0].y,
                            g1 ? scw[1][0].z : scw[0][0].z, g1 ? scw[1][0].w : scw[0][0].w,
                            g1 ? scw[1][1].x : scw[0][1].x, g1 ? scw[1][1].y : scw[0][1].y,
                            g1 ? scw[1][1].z : scw[0][1].z, g1 ? scw[1][1].w : scw[0][1].w};
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      sc[2 * h] = h2f((uint16_t)(ww[h] & 0xFFFFu));
      sc[2 * h + 1] = h2f((uint16_t)(ww[h] >> 16));
    }
    const float beta = lg == 0 ? (g1 ? beta_g[1] : beta_g[0]) : 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      yp[e] = fmaf(sc[e], acc[e] - double_offset_factor(e) * off - off8 + beta, yp[e]);
      acc[e] = 0.0f;
    }
    off = 0.0f;
    off8 = 0.0f;
    cur_g = 1;
    cur_bigend = bstart1 + nbb1;
    next_fin = nbt;
  };

  // the first batches in order (a scheduler free to reorder them issues
  // batch 0 last, and its consume then waits for all of them)
  Batch R[D];
#pragma unroll
  for (int i = 0; i < D - 1; ++i) {
    fetch(R[i], i);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int b = 0; b < nbt; b += D) {
#pragma unroll
    for (int i = 0; i < D; ++i) {
      fetch(R[(i + D - 1) % D], b + i + D - 1);
      __builtin_amdgcn_sched_barrier(0);   // the loads go out before the consume waits
      // a guard, not an exit: an early exit out of the unrolled body makes
      // the loop header wait for every load in flight
      if (b + i < nbt) {
        if (b + i < cur_bigend) consume_big(R[i]);
        else consume(R[i]);
        if (b + i + 1 == next_fin) finish_group();
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
  for (int o = tid; o < T; o += 256) {
    const float v = s_red[0][o] + s_red[1][o] + s_red[2][o] + s_red[3][o];
    atomicAdd(&y[(size_t)t * T + o], v * L.sfac);   // 8-bit code units -> b_max units
  }
}

// The same VMM with the lists of a workgroup shared: the four waves' rows of
// a group form one list (big rows, then small, in wave order) and the waves
// take its batches in turn (wave w: batches w, w + 4, ...).  That evens the
// waves' work and pads each list once per group rather than once per wave,
// for two workgroup barriers in the prologue; it pays on launches of two
// groups per workgroup, where each wave otherwise pads four lists.
template <int LPR, int D, bool TOPK>
__global__ __launch_bounds__(256) void k_vmm_sg(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ lm, int gw, int groups, int fused,
    const uint8_t* __restrict__ codes, const uint16_t* __restrict__ scales, float* __restrict__ y,
    Layer L, Thresholds th, TopkCuts tk, uint8_t* __restrict__ lm_out) {
  constexpr int T = LPR * 16;            // outputs of the tile
  constexpr int PLANE = T / 4;           // bytes of one plane row
  constexpr int NLG = 64 / LPR;          // lane groups per wave
  constexpr int kWaves = 4;
  constexpr int MAXG = 2;                // groups per workgroup at most; gw is 1 or 2
  constexpr int BR = 2 * NLG;            // big rows per batch
  constexpr int SR = 4 * NLG;            // small rows per batch
  constexpr int MB = kGroup / BR + 2;   // batches of one group's list at most
  constexpr int EMPTY = MAXG * MB;       // an all-empty batch after the lists
  constexpr int ENT = NLG * 12;          // dwords of one batch
  // fp16 exponent bits of a merged pair's field at p = 0: 31 - 2j for the
  // pair of planes (j, j+1); 27 for empty entries (any finite value)
  constexpr uint32_t kE12 = 29u << 10, kE34 = 25u << 10, kEmpty = 27u << 10;

  // lists: per batch and lane group four entries as three 4-dword fields:
  // offsets of plane j, of plane j+1, and (x | exponent << 16); a list's
  // batches lie back to back, group 0's then group 1's
  __shared__ __align__(16) uint32_t s_ent[EMPTY + 1][NLG][12];
  __shared__ __align__(16) float s_red[kWaves][T];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, hl = lane & 31;
  const int t = blockIdx.x;
  const int g0 = blockIdx.y * gw;
  const int ng = min(gw, groups - g0);
  // loads first: x and the level map of this lane's row (lanes 0-31 the
  // first group, 32-63 the second).  They need no field of L, so they go
  // out before the wave waits for the layer's scalars (x, lm, gw, groups and
  // fused lead the argument list and arrive preloaded in scalar registers)
  const int gg = half;
  const bool valid = gg < ng;
  const int k = (g0 + min(gg, ng - 1)) * kGroup + 32 * wave + hl;
  const uint32_t xv = x[k];
  const uint32_t lv = (fused ? (const uint8_t*)x : lm)[k];   // ignored when graded here
  const int lg = lane / LPR, li = lane % LPR;
  const int n_top = L.n_levels - 1;
  const __amdgpu_buffer_rsrc_t rsrc = tile_rsrc(codes + (size_t)t * L.K * L.RB, L);
  const uint32_t li4 = (uint32_t)li * 4u;

  // the scales of this lane's 16 outputs for both groups (a group past the
  // last reads the last one again, from cache)
  uint4 scw[MAXG][2];
#pragma unroll
  for (int g = 0; g < MAXG; ++g) {
    const uint16_t* sp = scales + (size_t)(g0 + min(g, ng - 1)) * L.N + (size_t)t * T + li * 16;
    scw[g][0] = *(const uint4*)sp;
    scw[g][1] = *(const uint4*)(sp + 8);
  }
  uint32_t* const E = &s_ent[0][0][0];
  if (wave == 0 && lane < ENT) E[EMPTY * ENT + lane] = (lane % 12) < 8 ? kNoRow : (kEmpty << 16);

  // top-k mode: the token's cuts from the whole x, the same in every workgroup
  // (top-k kernels only: the others hold no selection scratch)
  __shared__ __align__(16) uint8_t s_tk_raw[TOPK ? sizeof(topksel::Scratch) : 16];
  topksel::Scratch& s_tk = *reinterpret_cast<topksel::Scratch*>(s_tk_raw);
  if constexpr (TOPK) topksel::select_cuts(x, L.K, tk, s_tk);

  // ---- grade, sort into big and small rows
  const float fx = h2f((uint16_t)xv);
  const float ax = fabsf(fx);
  int graded = 0;
#pragma unroll
  for (int j = 0; j < kMaxLevels - 1; ++j) graded += ax >= th.theta[j] ? 1 : 0;
  const int lvl = min(fused == 1 ? graded
                      : TOPK ? topksel::level_of(xv, k, tk.n, s_tk)
                                   : (int)(lv & 0xFFu),
                      n_top);
  if (fused && lm_out && t == 0 && valid) lm_out[k] = (uint8_t)lvl;
  const int d = valid ? level_planes(L.planes_packed, lvl) : 0;
  const bool big = d >= 3, small = d == 1 || d == 2;
  const int nbig = half_total(big), nsm = half_total(small);   // this half wave's rows
  const int rank = big ? half_below(big) : half_below(small);
  const float bs = half_sum_dpp(d ? fx * phi_minus_offset(2 * d, L.bmax) : 0.0f);

  // rows of each group's list, and those of this lane's list before this wave's
  int NB[MAXG], NS[MAXG];
  int below_big = 0, below_sm = 0;
  {
    __shared__ int s_cnt[kWaves][MAXG][2];
    if (hl == 0) {
      s_cnt[wave][gg][0] = nbig;
      s_cnt[wave][gg][1] = nsm;
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < MAXG; ++g) {
      NB[g] = NS[g] = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const int cb = s_cnt[w][g][0], cs = s_cnt[w][g][1];
        if (w < wave && g == gg) {
          below_big += cb;
          below_sm += cs;
        }
        NB[g] += cb;
        NS[g] += cs;
      }
    }
  }
  const int nbb0 = (NB[0] + BR - 1) / BR, nsb0 = (NS[0] + SR - 1) / SR;
  const int nbb1 = (NB[1] + BR - 1) / BR, nsb1 = (NS[1] + SR - 1) / SR;
  const int bstart1 = nbb0 + nsb0;
  const int nbt = bstart1 + nbb1 + nsb1;

  // ---- write the lists
  {
    const uint32_t base = (uint32_t)k * (uint32_t)L.RB;
    const uint32_t xh = xv & 0xFFFFu;
    const int st = gg ? bstart1 : 0, nbb_gg = gg ? nbb1 : nbb0, nsb_gg = gg ? nsb1 : nsb0;
    auto put = [&](int b, int lgp, int sl, uint32_t o1, uint32_t o2, uint32_t xe) {
      uint32_t* p = E + b * ENT + lgp * 12 + sl;
      p[0] = o1;
      p[4] = o2;
      p[8] = xe;
    };
    if (valid && big) {
      const int r = below_big + rank;
      const int b = st + r / BR, w = r % BR;
      put(b, w >> 1, w & 1, base, base + PLANE, xh | (kE12 << 16));
      put(b, w >> 1, (w & 1) + 2, base + 2 * PLANE, d >= 4 ? base + 3 * PLANE : kNoRow,
          xh | (kE34 << 16));
    }
    if (valid && small) {
      const int r = below_sm + rank;
      const int b = st + nbb_gg + r / SR, w = r % SR;
      put(b, w >> 2, w & 3, base, d >= 2 ? base + PLANE : kNoRow, xh | (kE12 << 16));
    }
    // empty entries up to whole batches (no memory access, zero
    // coefficient), by the last wave's half of each group
    if (valid && wave == kWaves - 1) {
      const int nb_end = gg ? NB[1] : NB[0], ns_end = gg ? NS[1] : NS[0];
      for (int r = nb_end + hl; r < nbb_gg * BR; r += 32) {
        const int b = st + r / BR, w = r % BR;
        put(b, w >> 1, w & 1, kNoRow, kNoRow, kEmpty << 16);
        put(b, w >> 1, (w & 1) + 2, kNoRow, kNoRow, kEmpty << 16);
      }
      for (int r = ns_end + hl; r < nsb_gg * SR; r += 32) {
        const int b = st + nbb_gg + r / SR, w = r % SR;
        put(b, w >> 2, w & 3, kNoRow, kNoRow, kEmpty << 16);
      }
    }
  }
  float beta_g[MAXG];   // this wave's rows: it adds them with its partial sums
  beta_g[0] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bs), 0));
  beta_g[1] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bs), 32));
  __syncthreads();

  // ---- main loop over this wave's batches of the sequence (group 0 big,
  // small, group 1 big, small): D register sets, D-1 batches in flight while
  // one is consumed
  float yp[16], acc[16], off = 0.0f, off8 = 0.0f;
#pragma unroll
  for (int e = 0; e < 16; ++e) yp[e] = acc[e] = 0.0f;

  struct Batch {
    uint32_t w[8];
    uint32_t xe[4];
  };
  const uint32_t lane_ent = (uint32_t)lg * 12u;
  auto fetch = [&](Batch& B, int q) {
    const int idx = q < nbt ? q : EMPTY;
    const uint32_t* src = E + idx * ENT + lane_ent;
    const uint4 o1 = *(const uint4*)src;
    const uint4 o2 = *(const uint4*)(src + 4);
    const uint4 xe = *(const uint4*)(src + 8);
    B.xe[0] = xe.x;
    B.xe[1] = xe.y;
    B.xe[2] = xe.z;
    B.xe[3] = xe.w;
    B.w[0] = load_plane(rsrc, o1.x + li4);
    B.w[1] = load_plane(rsrc, o2.x + li4);
    B.w[2] = load_plane(rsrc, o1.y + li4);
    B.w[3] = load_plane(rsrc, o2.y + li4);
    B.w[4] = load_plane(rsrc, o1.z + li4);
    B.w[5] = load_plane(rsrc, o2.z + li4);
    B.w[6] = load_plane(rsrc, o1.w + li4);
    B.w[7] = load_plane(rsrc, o2.w + li4);
  };
  auto consume_big = [&](const Batch& B) {
    const uint32_t xp = __builtin_amdgcn_perm(B.xe[1], B.xe[0], 0x05040100u);
    off8 = dot2r(0x64006400u, xp, off8);
    consume_quad(B.w, xp, acc);
  };
  auto consume = [&](const Batch& B) {
    // (x_k1, x_k2) from the entries' low halves, the exponent bits from the high halves
    const uint32_t xpa = __builtin_amdgcn_perm(B.xe[1], B.xe[0], 0x05040100u);
    const uint32_t m0a = __builtin_amdgcn_perm(B.xe[1], B.xe[0], 0x07060302u);
    const uint32_t xpb = __builtin_amdgcn_perm(B.xe[3], B.xe[2], 0x05040100u);
    const uint32_t m0b = __builtin_amdgcn_perm(B.xe[3], B.xe[2], 0x07060302u);
    off = dot2r(m0a, xpa, off);
    off = dot2r(m0b, xpb, off);
    consume_double(B.w[0], B.w[1], B.w[2], B.w[3], m0a, xpa, acc);
    consume_double(B.w[4], B.w[5], B.w[6], B.w[7], m0b, xpb, acc);
  };
  // the group being consumed and the end of its big batches; every wave
  // finishes both groups (a group it has no batch of adds its rows' beta)
  int cur_g = 0;
  int cur_bigend = nbb0;
  auto finish_group = [&]() {
    float sc[16];
    const bool g1 = cur_g != 0;
    const uint32_t ww[8] = {g1 ? scw[1][0].x : scw[0][0].x, g1 ? scw[1][0].y : scw[0][0].y,
                            g1 ? scw[1][0].z : scw[0][0].z, g1 ? scw[1][0].w : scw[0][0].w,
                            g1 ? scw[1][1].x : scw[0][1].x, g1 ? scw[1][1].y : scw[0][1].y,
                            g1 ? scw[1][1].z : scw[0][1].z, g1 ? scw[1][1].w : scw[0][1].w};
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      sc[2 * h] = h2f((uint16_t)(ww[h] & 0xFFFFu));
      sc[2 * h + 1] = h2f((uint16_t)(ww[h] >> 16));
    }
    const float beta = lg == 0 ? (g1 ? beta_g[1] : beta_g[0]) : 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      yp[e] = fmaf(sc[e], acc[e] - double_offset_factor(e) * off - off8 + beta, yp[e]);
      acc[e] = 0.0f;
    }
    off = 0.0f;
    off8 = 0.0f;
    cur_g = 1;
    cur_bigend = bstart1 + nbb1;
  };
  constexpr int kStride = kWaves;
  const int first = wave;
  const int nbw = nbt > first ? (nbt - first + kStride - 1) / kStride : 0;   // this wave's batches
  if (first >= bstart1) finish_group();   // no batch of group 0 for this wave

  // the first batches in order (a scheduler free to reorder them issues
  // batch 0 last, and its consume then waits for all of them)
  Batch R[D];
#pragma unroll
  for (int i = 0; i < D - 1; ++i) {
    fetch(R[i], first + kStride * i);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int b = 0; b < nbw; b += D) {
#pragma unroll
    for (int i = 0; i < D; ++i) {
      fetch(R[(i + D - 1) % D], first + kStride * (b + i + D - 1));
      __builtin_amdgcn_sched_barrier(0);   // the loads go out before the consume waits
      // a guard, not an exit: an early exit out of the unrolled body makes
      // the loop header wait for every load in flight
      if (b + i < nbw) {
        const int q = first + kStride * (b + i);
        if (q < cur_bigend) consume_big(R[i]);
        else consume(R[i]);
        if (cur_g == 0 && q + kStride >= bstart1) finish_group();
      }
    }
  }
  finish_group();   // group 1 (a group past the last adds zero)

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
  for (int o = tid; o < T; o += 256) {
    const float v = s_red[0][o] + s_red[1][o] + s_red[2][o] + s_red[3][o];
    atomicAdd(&y[(size_t)t * T + o], v * L.sfac);   // 8-bit code units -> b_max units
  }
}

template <int LPR>
void launch_sr(int gw, hipStream_t s, const void* codes, const void* scales, const void* x,
               const uint8_t* lm, float* y, const Layer& L, int fused, const Thresholds& th,
               const TopkCuts& tk, uint8_t* lm_out) {
  const dim3 grid((unsigned)L.tiles, (unsigned)((L.groups + gw - 1) / gw));
  // top-k selection is its own instantiation: the other kernels carry no
  // selection code or scratch
  if (gw == 2 && fused == 2)
    hipLaunchKernelGGL((k_vmm_sg<LPR, 4, true>), grid, dim3(256), 0, s,
                       (const uint16_t*)x, lm, gw, L.groups, fused, (const uint8_t*)codes,
                       (const uint16_t*)scales, y, L, th, tk, lm_out);
  else if (gw == 2)
    hipLaunchKernelGGL((k_vmm_sg<LPR, 4, false>), grid, dim3(256), 0, s,
                       (const uint16_t*)x, lm, gw, L.groups, fused, (const uint8_t*)codes,
                       (const uint16_t*)scales, y, L, th, tk, lm_out);
  else if (fused == 2)
    hipLaunchKernelGGL((k_vmm_sr<LPR, 4, true>), grid, dim3(256), 0, s,
                       (const uint16_t*)x, lm, gw, L.groups, fused, (const uint8_t*)codes,
                       (const uint16_t*)scales, y, L, th, tk, lm_out);
  else
    hipLaunchKernelGGL((k_vmm_sr<LPR, 4, false>), grid, dim3(256), 0, s,
                       (const uint16_t*)x, lm, gw, L.groups, fused, (const uint8_t*)codes,
                       (const uint16_t*)scales, y, L, th, tk, lm_out);
}

}  // namespace

bool vmm_pp_supported(const Layer& L, int B) {
  // byte offsets inside a tile are 32-bit and stay below the empty-row offset
  return B == 1 && L.u == 2 && (L.T == 256 || L.T == 512 || L.T == 1024) &&
         (long long)L.K * L.RB < (1ll << 31);
}

int launch_vmm_pp(const Layer& L, const void* codes, const void* scales, const void* x,
                  const uint8_t* level_map, const Thresholds* th, const TopkCuts* tk,
                  uint8_t* level_map_out, float* y, hipStream_t s) {
  // groups per workgroup: about 512 workgroups, rounded to the nearest count
  // (896 (tile, group) units -> 2, 448 -> 1)
  int gw = (int)(((long)L.tiles * L.groups + 256) / 512);
  if (const int v = option(&Options::groups_per_wg)) gw = v;
  gw = gw < 1 ? 1 : (gw > 2 ? 2 : gw);
  Thresholds none{};
  TopkCuts nocuts{};
  const Thresholds& tt = th ? *th : none;
  const TopkCuts& cc = tk ? *tk : nocuts;
  const int fused = th ? 1 : (tk ? 2 : 0);   // levels graded here: thresholds, top-k
  if (L.T == 256) launch_sr<16>(gw, s, codes, scales, x, level_map, y, L, fused, tt, cc, level_map_out);
  else if (L.T == 512) launch_sr<32>(gw, s, codes, scales, x, level_map, y, L, fused, tt, cc, level_map_out);
  else launch_sr<64>(gw, s, codes, scales, x, level_map, y, L, fused, tt, cc, level_map_out);
  return check_launch("vmm (sorted rows)");
}

}  // namespace grinqh
