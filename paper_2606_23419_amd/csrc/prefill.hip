// Prefill over the nested layout: the stage-decoupled path of Sec. 3 (prefill
// reads the weights at the fixed top precision b_max and multiplies densely;
// Sec. 4 "Prefill vs. Decoding Evaluation").  For M tokens at once,
//   Y[m][n] = sum_k X[m][k] W_hat[n][k],  W_hat = s[k/128][n] (q[n][k] - 128),
// a dense contraction, on the matrix cores (v_mfma_f32_32x32x16_f16).
//
// A workgroup of WV waves computes a (64 MB) x (64 NB) tile of Y; the waves
// split it into RS row bands by WV / RS column bands, each wave's part as
// blocks of 32 x 32, so every 16-byte operand fragment read from LDS feeds
// several MFMAs.  The 256 x 256 tile runs 8 waves (two per SIMD, 128 x 64
// each): one wave's unpack and LDS waits overlap the other's MFMAs, which a
// single wave per SIMD (4 waves of 128 x 128) leaves idle.  K advances
// 64 channels per step through two LDS buffers: while the waves multiply out
// of one buffer they fill the other with the next step,
//   - X: the [64 MB rows][64 k] fp16 tile, copied;
//   - W: the codes of the tile's 64 NB outputs for 64 channels, read from the
//     bit planes (one dword of 16 outputs per channel and 2-bit plane, or a
//     16-bit word per 1-bit plane), assembled into bytes, turned into fp16
//     q - 128 (exact: 0x6400 | q reads as 1024 + q), multiplied by the fp16
//     group scale (one rounding: the dequantised weight in fp16, as a dense
//     GEMM over unpacked weights uses it), and written transposed, [n][k],
//     so that an MFMA fragment (eight consecutive k of one row) is one
//     16-byte LDS read.
// Global loads for step s + 2 are issued while step s is multiplied.  LDS
// rows are 128 bytes with XOR-swizzled 16-byte chunks, so fragment reads and
// the tile copies are free of bank conflicts and the transposed weight
// writes are at most 2-way.
#include <cstdlib>

#include "grinqh_internal.h"
#include "vmm_common.h"

namespace grinqh {

namespace {

using vmmdev::assemble_codes;
using vmmdev::spread_bits;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;

__device__ __forceinline__ uint32_t mul_half2(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, a) * __builtin_bit_cast(half2v, b));
}

// fp16 pair (q_a - 128, q_b - 128) from bytes a and b (selector byte
// indices 0..3) of the code word q: one v_perm_b32 places each code under
// an exponent byte 0x64, so a half reads 1024 + q exactly.
__device__ __forceinline__ uint32_t codes_to_half2(uint32_t q, uint32_t a, uint32_t b) {
  const uint32_t v = __builtin_amdgcn_perm(0x64646464u, q, a | 0x0400u | (b << 16) | 0x04000000u);
  const half2v h = __builtin_bit_cast(half2v, v);
  const half2v c = {(_Float16)1152.0f, (_Float16)1152.0f};
  return __builtin_bit_cast(uint32_t, h - c);
}

// LDS offsets (halves) of 16-byte chunk c of a 64-half row.  The swizzles
// make eight (or sixteen) consecutive rows at one chunk hit distinct banks;
// for weight rows bit 4 of the row also moves the chunk by 4, so that the
// transposed writes of one instruction (8 channel quads of two rows 16
// apart) fill 128 distinct bytes.  Both depend on the row's low 5 bits only:
// rows 32 apart differ by a constant offset.
__device__ __forceinline__ int x_off(int m, int c) {
  return m * kBK + 8 * (c ^ (m & 7) ^ ((m >> 3) & 1));
}
__device__ __forceinline__ int w_off(int n, int c) {
  return n * kBK + 8 * (c ^ (n & 7) ^ ((n >> 3) & 1) ^ ((n >> 2) & 4));
}

// One step's codes for one thread (CPT channels x 16 outputs as plane
// words) and the 16 outputs' fp16 scales of the step's group.
template <int U, int CPT>
struct WRegs {
  uint32_t w[CPT][8 / U];
  uint4 s[2];
};

template <int U, int MB, int NB, int WV, int RS>
__global__ __launch_bounds__(64 * WV) void k_prefill(const uint8_t* __restrict__ codes,
                                                       const uint16_t* __restrict__ scales,
                                                       const uint16_t* __restrict__ x,
                                                       float* __restrict__ y, Layer L, int M,
                                                       int accumulate, int2 win, int n_base) {
  constexpr int BM = 64 * MB, BN = 64 * NB;
  constexpr int XI = BM * kBK * 2 / 1024 / WV;     // X copy instructions per wave and step
  constexpr int WI = kBK * BN / 1024 / WV;         // code copy instructions per wave and step
  constexpr int RCH = BN / 16;                     // 16-byte chunks of one staged channel row
  constexpr int PPP = BN * U / 128;                // chunks per plane of a staged row
  constexpr int CPT = kBK * BN / 16 / (64 * WV);   // channels per thread and step
  constexpr int NCG = kBK / CPT;                   // channel groups per step
  constexpr int kWords = 8 / U;                    // plane words per channel and 16 outputs
  constexpr int MBW = 2 * MB / RS;                 // 32-row blocks per wave
  constexpr int NBW = 2 * NB * RS / WV;            // 32-column blocks per wave
  static_assert(WV == 4 || WV == 8, "waves");
  static_assert(CPT == 2 || CPT == 4, "tile width for the waves");
  static_assert(XI >= 1 && WI >= 1 && MBW >= 1 && NBW >= 1, "tile too small for the waves");
  // every thread unpacks one (channel group, 16 outputs) unit and loads its
  // scales: a thread without a unit would read scales past the tile
  static_assert(NCG * (BN / 16) == 64 * WV, "threads and unpack units");
  // separate objects per buffer: the compiler then knows that a copy in
  // flight into one buffer does not alias reads of the other
  __shared__ __align__(16) _Float16 sX0[BM * kBK];
  __shared__ __align__(16) _Float16 sX1[BM * kBK];
  __shared__ __align__(16) _Float16 sW0[BN * kBK];
  __shared__ __align__(16) _Float16 sW1[BN * kBK];
  __shared__ __align__(16) uint8_t sP0[kBK * BN];  // raw codes of a step (BN bytes per channel)
  __shared__ __align__(16) uint8_t sP1[kBK * BN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Workgroup i runs on XCD i mod 8.  The (row block, column tile) pairs are
  // taken in windows of win.x row blocks by win.y column tiles, and each XCD
  // gets a contiguous run of that order: the workgroups an XCD runs together
  // share their X rows and weight columns in its L2 (win.x = 1 when the
  // grid does not split into windows: row blocks in order).
  int rblk, ctile;
  {
    const int gx = (M + BM - 1) / BM;
    const int G = (int)gridDim.x, i = (int)blockIdx.x;
    const int xcd = i & 7, j = i >> 3, per = G >> 3, extra = G & 7;
    const int pos = xcd * per + min(xcd, extra) + j;
    const int wsz = win.x * win.y, w = pos / wsz, p = pos - w * wsz;
    const int wr = w % (gx / win.x), wc = w / (gx / win.x);
    rblk = win.x * wr + p / win.y;
    ctile = win.y * wc + p % win.y;
  }
  const int m0 = rblk * BM, n0 = n_base + ctile * BN;
  const int T = L.T, K = L.K, N = L.N;
  const int steps = K / kBK;                       // even: K is a multiple of 128
  const int tile = n0 / T, o0 = n0 - tile * T;     // BN divides T
  const int wm = (wave / (WV / RS)) * 32 * MBW, wn = (wave % (WV / RS)) * 32 * NBW;

  // X copy: instruction i of this wave fills LDS rows 8 I .. 8 I + 7, I = 4 i +
  // wave, 16 bytes per lane; lane l takes the logical chunk that the swizzle
  // puts at physical chunk l % 8 of row 8 I + l / 8.  Rows past M repeat row
  // M - 1 (never stored).
  const uint16_t* xsrc[XI];
#pragma unroll
  for (int i = 0; i < XI; ++i) {
    const int row = 8 * (WV * i + wave) + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7) ^ ((row >> 3) & 1);
    xsrc[i] = x + (size_t)min(m0 + row, M - 1) * K + 8 * c;
  }
  auto copy_x = [&](int st, _Float16* sx) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < XI; ++i)
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(xsrc[i] + st * kBK),
          (__attribute__((address_space(3))) void*)&sx[8 * kBK * (WV * i + wave)], 16, 0, 0);
  };

  // Code staging: the tile's part of a channel row is BN bytes at 8 bits
  // (every plane's BN u / 8 bytes).  Staged chunk slot v of row r (v = plane *
  // PPP + piece) sits at position v ^ ((r / CPT) & 7) of the row, so the word
  // reads below (8 channel groups x 8 output chunks per instruction) hit
  // distinct banks.  A code narrower than 8 bits (b_max = 4, 6) has only L.P
  // planes in its stored row of L.RB bytes: the slots of the missing planes
  // copy plane 1 again (in bounds) and are read as zero.
  const uint8_t* wtile = codes + (size_t)tile * K * L.RB + o0 * U / 8;
  int wsrc[WI];
#pragma unroll
  for (int i = 0; i < WI; ++i) {
    const int q = 64 * (WV * i + wave) + lane;
    const int r = q / RCH, v = (q % RCH) ^ ((r / CPT) & 7);
    const int pl = v / PPP;
    wsrc[i] = r * L.RB + (pl < L.P ? pl : 0) * (T * U / 8) + 16 * (v % PPP);
  }
  auto copy_w = [&](int st, uint8_t* sp) __attribute__((always_inline)) {
    const uint8_t* base = wtile + (size_t)st * kBK * L.RB;
#pragma unroll
    for (int i = 0; i < WI; ++i)
      __builtin_amdgcn_global_load_lds(
          (const __attribute__((address_space(1))) void*)(base + wsrc[i]),
          (__attribute__((address_space(3))) void*)&sp[1024 * (WV * i + wave)], 16, 0, 0);
  };

  // W unpack: outputs 16 j .. 16 j + 15 of the tile, channels CPT cg .. of the step
  const int cg = (lane & 7) + 8 * (wave % (NCG / 8));
  const int j = (lane >> 3) + 8 * (wave / (NCG / 8));
  const uint16_t* sbase = scales + n0 + 16 * j;
  auto load_scales = [&](int st, WRegs<U, CPT>& R) __attribute__((always_inline)) {
    const uint4* sg = (const uint4*)(sbase + (size_t)(st * kBK / kGroup) * N);
    R.s[0] = sg[0];
    R.s[1] = sg[1];
  };
  const int np = L.P;
  auto read_w = [&](const uint8_t* sp, WRegs<U, CPT>& R) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
      const int row = cg * CPT + r;
#pragma unroll
      for (int p = 0; p < kWords; ++p) {
        uint32_t wd;
        if constexpr (U == 2) {
          const int v = (p * PPP + (j >> 2)) ^ (cg & 7);
          wd = *(const uint32_t*)&sp[16 * (row * RCH + v) + 4 * (j & 3)];
        } else {
          const int v = (p * PPP + (j >> 3)) ^ (cg & 7);
          wd = *(const uint16_t*)&sp[16 * (row * RCH + v) + 2 * (j & 7)];
        }
        R.w[r][p] = p < np ? wd : 0u;   // planes past b_max are zero
      }
    }
  };
  // h[r][d][p]: fp16 weights of outputs 8p + d (low half) and 8p + 4 + d
  // (high half) of channel r
  auto unpack = [&](const WRegs<U, CPT>& R, int r, uint32_t (&h)[4][2]) __attribute__((always_inline)) {
    const uint32_t sw[8] = {R.s[0].x, R.s[0].y, R.s[0].z, R.s[0].w,
                            R.s[1].x, R.s[1].y, R.s[1].z, R.s[1].w};
    uint32_t w[4];
    if constexpr (U == 2) {
#pragma unroll
      for (int p = 0; p < 4; ++p) w[p] = R.w[r][p];
    } else {
#pragma unroll
      for (int p = 0; p < 4; ++p) w[p] = (spread_bits(R.w[r][2 * p]) << 1) | spread_bits(R.w[r][2 * p + 1]);
    }
    uint32_t q[4];
    assemble_codes(w[0], w[1], w[2], w[3], q);
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        // scale pair (s_{8p+d}, s_{8p+4+d})
        const uint32_t sp = __builtin_amdgcn_perm(sw[4 * p + 2 + (d >> 1)], sw[4 * p + (d >> 1)],
                                                  (d & 1) ? 0x07060302u : 0x05040100u);
        h[d][p] = mul_half2(codes_to_half2(q[d], 2 * p, 2 * p + 1), sp);
      }
  };
  const int kq = cg * CPT;
  // output 16 j + 4 i + d gets the thread's CPT channels, k contiguous
  auto write_w = [&](_Float16* sw, const uint32_t (&h)[CPT][4][2]) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = i >> 1;
        const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
        _Float16* dst = &sw[w_off(16 * j + 4 * i + d, kq >> 3) + (kq & 7)];
        const uint32_t lo = __builtin_amdgcn_perm(h[1][d][p], h[0][d][p], sel);
        if constexpr (CPT == 4)
          *(uint2*)dst = make_uint2(lo, __builtin_amdgcn_perm(h[3][d][p], h[2][d][p], sel));
        else
          *(uint32_t*)dst = lo;
      }
  };

  float16v acc[MBW][NBW];
#pragma unroll
  for (int a = 0; a < MBW; ++a)
#pragma unroll
    for (int b = 0; b < NBW; ++b) acc[a][b] = float16v{};

  // One step st: start the copies of X for st + 1 and of the codes for st + 2
  // (into the staging buffer that held st's codes) and the scale loads for
  // st + 2; multiply st out of (xc, wc) while unpacking st + 1 (staged in
  // pc, scales in `cur`) into (xn, wn_).  Past the last step the copies and
  // loads re-read the last step (in bounds, never used).
  auto step = [&](int st, const _Float16* xc, const _Float16* wc, _Float16* xn, _Float16* wn_,
                  const uint8_t* pc, uint8_t* pn, WRegs<U, CPT>& cur, WRegs<U, CPT>& nxt)
                  __attribute__((always_inline)) {
    copy_x(min(st + 1, steps - 1), xn);
    copy_w(min(st + 2, steps - 1), pn);
    load_scales(min(st + 2, steps - 1), nxt);
    __builtin_amdgcn_sched_barrier(0);   // issue them first: a full step of latency
    read_w(pc, cur);
    uint32_t h[CPT][4][2];
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      if (ks % (4 / CPT) == 0) unpack(cur, ks / (4 / CPT), h[ks / (4 / CPT)]);
      const int c = 2 * ks + (lane >> 5);
      half8 fa[MBW], fb[NBW];
#pragma unroll
      for (int a = 0; a < MBW; ++a) fa[a] = *(const half8*)&xc[x_off(wm + 32 * a + (lane & 31), c)];
#pragma unroll
      for (int b = 0; b < NBW; ++b) fb[b] = *(const half8*)&wc[w_off(wn + 32 * b + (lane & 31), c)];
#pragma unroll
      for (int a = 0; a < MBW; ++a)
#pragma unroll
        for (int b = 0; b < NBW; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[a], fb[b], acc[a][b], 0, 0, 0);
      // one sub-step per scheduling region: the unpack spreads over the MFMAs
      if (ks + 1 < kBK / 16) __builtin_amdgcn_sched_barrier(0);
    }
    write_w(wn_, h);
    __syncthreads();   // copies and writes for st + 1 done; st's reads done
  };

  WRegs<U, CPT> ra, rb;
  // prologue: step 0 into buffers 0, codes of step 1 staged in sP1
  copy_x(0, sX0);
  copy_w(0, sP0);
  copy_w(min(1, steps - 1), sP1);
  load_scales(0, ra);
  load_scales(min(1, steps - 1), rb);
  // consume the scale loads before the barrier: left in flight into the loop
  // they would make the compiler wait for them in every iteration
  asm volatile("" ::"v"(rb.s[0].x), "v"(rb.s[0].y), "v"(rb.s[0].z), "v"(rb.s[0].w),
               "v"(rb.s[1].x), "v"(rb.s[1].y), "v"(rb.s[1].z), "v"(rb.s[1].w));
  __syncthreads();
  read_w(sP0, ra);
  {
    uint32_t h[CPT][4][2];
#pragma unroll
    for (int r = 0; r < CPT; ++r) unpack(ra, r, h[r]);
    write_w(sW0, h);
  }
  __syncthreads();   // sP0 is free for the codes of step 2
  for (int st = 0; st < steps; st += 2) {
    step(st, sX0, sW0, sX1, sW1, sP1, sP0, rb, ra);
    step(st + 1, sX1, sW1, sX0, sW0, sP0, sP1, ra, rb);
  }

  // element e of lane l of a 32 x 32 block: row 8 (e / 4) + 4 (l / 32) + e % 4,
  // column l % 32
#pragma unroll
  for (int a = 0; a < MBW; ++a)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + wm + 32 * a + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      if (m >= M) continue;
#pragma unroll
      for (int b = 0; b < NBW; ++b) {
        float* dst = y + (size_t)m * N + n0 + wn + 32 * b + (lane & 31);
        const float v = acc[a][b][e] * L.sfac;   // 8-bit code units -> b_max units (exact)
        *dst = accumulate ? *dst + v : v;
      }
    }
}

// Output columns [n_begin, n_begin + n_cols) of Y; n_begin and n_cols are
// multiples of the tile width.
template <int U, int MB, int NB, int WV, int RS>
void launch_cfg(const Layer& L, const void* codes, const void* scales, const void* x, int M,
                float* y, int accumulate, hipStream_t s, int n_begin, int n_cols) {
  const int gx = (M + 64 * MB - 1) / (64 * MB), gy = n_cols / (64 * NB);
  // windows of up to 4 row blocks x 8 column tiles (about one XCD's worth of
  // workgroups at one per CU), the largest powers of two dividing the grid
  int2 win = make_int2(1, 1);
  while (win.x < 4 && gx % (2 * win.x) == 0) win.x *= 2;
  while (win.y < 8 && gy % (2 * win.y) == 0) win.y *= 2;
  if (win.x == 1) win.y = 1;   // one row block: the plain order already shares X
  hipLaunchKernelGGL((k_prefill<U, MB, NB, WV, RS>), dim3((unsigned)(gx * gy)), dim3(64 * WV), 0, s,
                     (const uint8_t*)codes, (const uint16_t*)scales, (const uint16_t*)x, y, L, M,
                     accumulate, win, n_begin);
}

template <int U>
void launch_u(int cfg, const Layer& L, const void* codes, const void* scales, const void* x, int M,
              float* y, int accumulate, hipStream_t s, int n_begin, int n_cols) {
  // 256 x 256: 8 waves of 128 x 64 for 2-bit planes (gate_up at 2048 tokens
  // 909 -> 939, qkv 755 -> 824 TFLOP/s); the 1-bit unpack needs more
  // registers than two waves per SIMD leave, so 4 waves of 128 x 128 there.
  // 256 x 128 and 128 x 128: 4 waves (8 waves of 64 x 64 read more LDS per
  // MFMA and were no faster).
  if (cfg == 0) launch_cfg<U, 4, 4, U == 2 ? 8 : 4, 2>(L, codes, scales, x, M, y, accumulate, s, n_begin, n_cols);
  else if (cfg == 1) launch_cfg<U, 4, 2, 4, 2>(L, codes, scales, x, M, y, accumulate, s, n_begin, n_cols);
  else launch_cfg<U, 2, 2, 4, 2>(L, codes, scales, x, M, y, accumulate, s, n_begin, n_cols);
}

// Compute units of the current device (cached per device).
int device_cus() {
  static int cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cus[dev]) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cus[dev] = v;
  }
  return cus[dev];
}

}  // namespace

// Tile choice: 256 x 256 while that gives at least ~0.6 workgroups per CU
// (one resident per CU), else 256 x 128 on the same condition, else 128 x 128
// (short prompts; two resident per CU).  GRINQH_OPT_PREFILL_TILE = 1
// (256 x 256), 2 (256 x 128) or 3 (128 x 128) forces one.
//
// At 256 x 256 the workgroups run in rounds of one per CU.  When the tiles
// leave a last round less than half full (e.g. 896 tiles on 256 CUs: three
// rounds and a half), the launch is split by columns: whole rounds of
// 256 x 256 tiles, then the remaining columns as 256 x 128 tiles, which fill
// one round that takes about half as long.  GRINQH_OPT_PREFILL_CUS sets the
// CU count the rounds are counted in (tests); 0 takes the device's.
int launch_prefill(const Layer& L, const void* codes, const void* scales, const void* x, int M,
                   float* y, int accumulate, hipStream_t s) {
  const long mb256 = (M + 255) / 256;
  int cfg = mb256 * (L.N / 256) >= 160 ? 0 : mb256 * (L.N / 128) >= 160 ? 1 : 2;
  int n_split = 0;   // columns of the 256 x 256 part when split
  if (const int v = option(&Options::prefill_tile)) {
    cfg = v - 1;
  } else if (cfg == 0) {
    const int o = option(&Options::prefill_cus);
    const long cus = o ? o : device_cus();
    const long gx = mb256, gy = L.N / 256, tiles = gx * gy;
    if (tiles > cus && tiles % cus != 0) {
      long c = gy - 1;
      while (c > 0 && (c * gx) % cus != 0) --c;
      if (c > 0 && 2 * (gy - c) * gx <= cus) n_split = (int)(256 * c);
    }
  }
  auto go = [&](int cf, int nb, int nc) {
    if (L.u == 2) launch_u<2>(cf, L, codes, scales, x, M, y, accumulate, s, nb, nc);
    else launch_u<1>(cf, L, codes, scales, x, M, y, accumulate, s, nb, nc);
  };
  if (n_split) {
    go(0, 0, n_split);
    int st = check_launch("prefill");
    if (st) return st;
    go(1, n_split, L.N - n_split);
  } else {
    go(cfg, 0, L.N);
  }
  return check_launch("prefill");
}

}  // namespace grinqh
