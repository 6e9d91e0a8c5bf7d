// Prefill over the nested layout: the stage-decoupled path of Sec. 3 (prefill
// reads the weights at the fixed top precision b_max and multiplies densely;
// Sec. 4 "Prefill vs. Decoding Evaluation").  For M tokens at once,
//   Y[m][n] = sum_g s[g][n] * sum_{k in g} X[m][k] (q[n][k] - 128),
// a dense contraction, on the matrix cores (v_mfma_f32_32x32x16_f16).
//
// A workgroup of 4 waves computes a 128 x 128 tile of Y; wave w owns the
// 64 x 64 sub-tile (w / 2, w % 2) as 2 x 2 MFMA blocks of 32 x 32.  K runs
// one quantisation group of 128 channels at a time:
//   - the X tile [128 m][128 k] is copied to LDS, k contiguous;
//   - the codes of the tile's 128 outputs and the group's 128 channels are
//     read from the bit planes (one dword of 16 outputs per channel and
//     2-bit plane, or one 16-bit word per 1-bit plane), assembled into bytes,
//     turned into the fp16 values q - 128 (exact: 0x6400 | q reads as
//     1024 + q), and written to LDS transposed, [n][k], so that each MFMA
//     operand fragment (eight consecutive k of one m or one n) is a single
//     16-byte LDS read;
//   - 8 MFMA steps of k = 16 accumulate the group's integer-weight product
//     in fp32, and s[g][n] scales it into the output sums.
// LDS rows are 256 bytes with the 16-byte chunks XOR-swizzled per row, which
// keeps both the transposed writes and the fragment reads free of bank
// conflicts beyond their minimum.  The next group's global loads are issued
// before the current group's MFMAs.
#include "grinqh_internal.h"

namespace grinqh {

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 128;
constexpr int kThreadsPF = 256;

// fp16 pair (q_a - 128, q_b - 128) from code bytes at bits 0..7 and 16..23.
__device__ __forceinline__ uint32_t codes_to_half2(uint32_t v) {
  const half2v h = __builtin_bit_cast(half2v, v | 0x64006400u);
  const half2v c = {(_Float16)1152.0f, (_Float16)1152.0f};
  return __builtin_bit_cast(uint32_t, h - c);
}

// Bit o of a 16-bit word moved to bit 2o.
__device__ __forceinline__ uint32_t spread_bits(uint32_t v) {
  v = (v | (v << 8)) & 0x00FF00FFu;
  v = (v | (v << 4)) & 0x0F0F0F0Fu;
  v = (v | (v << 2)) & 0x33333333u;
  return (v | (v << 1)) & 0x55555555u;
}

// The codes of 16 outputs from the four 2-bit plane words (output o's field
// at bit 2o, plane 1 most significant): byte i of q[d] is the code of output
// 4i + d.
__device__ __forceinline__ void assemble_codes(uint32_t w1, uint32_t w2, uint32_t w3, uint32_t w4,
                                               uint32_t (&q)[4]) {
  // 4-bit fields of the even (E) and odd (O) outputs: output 2m or 2m+1 at
  // bits 4m..4m+3, the first plane of the pair on top
  const uint32_t E12 = ((w1 << 2) & 0xCCCCCCCCu) | (w2 & 0x33333333u);
  const uint32_t O12 = (w1 & 0xCCCCCCCCu) | ((w2 >> 2) & 0x33333333u);
  const uint32_t E34 = ((w3 << 2) & 0xCCCCCCCCu) | (w4 & 0x33333333u);
  const uint32_t O34 = (w3 & 0xCCCCCCCCu) | ((w4 >> 2) & 0x33333333u);
  q[0] = ((E12 & 0x0F0F0F0Fu) << 4) | (E34 & 0x0F0F0F0Fu);
  q[1] = ((O12 & 0x0F0F0F0Fu) << 4) | (O34 & 0x0F0F0F0Fu);
  q[2] = (E12 & 0xF0F0F0F0u) | ((E34 >> 4) & 0x0F0F0F0Fu);
  q[3] = (O12 & 0xF0F0F0F0u) | ((O34 >> 4) & 0x0F0F0F0Fu);
}

// LDS element offsets (in halves) of 16-byte chunk c of row r.
__device__ __forceinline__ int x_chunk(int m, int c) { return m * kBK + 8 * (c ^ (m & 15)); }
__device__ __forceinline__ int w_chunk(int n, int c) {
  return n * kBK + 8 * (c ^ ((n & 15) ^ ((n >> 2) & 12)));
}

template <int U>
__global__ __launch_bounds__(kThreadsPF, 2) void k_prefill(const uint8_t* __restrict__ codes,
                                                       const uint16_t* __restrict__ scales,
                                                       const uint16_t* __restrict__ x,
                                                       float* __restrict__ y, Layer L, int M,
                                                       int accumulate) {
  constexpr int kWords = 8 / U;   // plane words per channel row and 16 outputs
  __shared__ __align__(16) _Float16 sX[kBM * kBK];
  __shared__ __align__(16) _Float16 sW[kBN * kBK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN;
  const int T = L.T, K = L.K, N = L.N;
  const int tile = n0 / T, o0 = n0 - tile * T;   // 128 divides T
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;

  // X copy: 16-byte chunk xc of rows 16 i + xq (rows past M repeat row M-1;
  // their outputs are never stored)
  const int xq = tid >> 4, xc = tid & 15;
  // W unpack: channels wr..wr+3 of the group, outputs wc..wc+15 of the tile
  const int wr = 4 * ((lane & 7) + 8 * wave), wc = 16 * (lane >> 3);
  const int plane_bytes = T * U / 8;
  const uint8_t* wbase = codes + ((size_t)tile * K + wr) * T + (o0 + wc) * U / 8;
  const uint16_t* sbase = scales + n0 + wn + (lane & 31);

  uint4 xv[8];
  uint32_t wv[4][kWords];
  uint16_t sv[2];
  auto load_group = [&](int g) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int m = min(m0 + 16 * i + xq, M - 1);
      xv[i] = *(const uint4*)(x + (size_t)m * K + g * kBK + 8 * xc);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint8_t* row = wbase + (size_t)(g * kBK + r) * T;
#pragma unroll
      for (int j = 0; j < kWords; ++j) {
        if constexpr (U == 2)
          wv[r][j] = *(const uint32_t*)(row + j * plane_bytes);
        else
          wv[r][j] = *(const uint16_t*)(row + j * plane_bytes);
      }
    }
    sv[0] = sbase[(size_t)g * N];
    sv[1] = sbase[(size_t)g * N + 32];
  };
  auto store_group = [&]() {
#pragma unroll
    for (int i = 0; i < 8; ++i) *(uint4*)&sX[x_chunk(16 * i + xq, xc)] = xv[i];
    // h[r][d][p]: fp16 values of outputs 8p + d (low half) and 8p + 4 + d
    // (high half) of channel wr + r
    uint32_t h[4][4][2];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      uint32_t w[4];
      if constexpr (U == 2) {
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = wv[r][j];
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (spread_bits(wv[r][2 * j]) << 1) | spread_bits(wv[r][2 * j + 1]);
      }
      uint32_t q[4];
      assemble_codes(w[0], w[1], w[2], w[3], q);
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        h[r][d][0] = codes_to_half2(__builtin_amdgcn_perm(0u, q[d], 0x0C010C00u));
        h[r][d][1] = codes_to_half2(__builtin_amdgcn_perm(0u, q[d], 0x0C030C02u));
      }
    }
    // output wc + 4i + d: its four channels' values, k contiguous
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = i >> 1;
        const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t lo = __builtin_amdgcn_perm(h[1][d][p], h[0][d][p], sel);
        const uint32_t hi = __builtin_amdgcn_perm(h[3][d][p], h[2][d][p], sel);
        *(uint2*)&sW[w_chunk(wc + 4 * i + d, wr >> 3) + (wr & 7)] = make_uint2(lo, hi);
      }
  };

  float16v acc[2][2], part[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = float16v{};

  const int groups = L.groups;
  load_group(0);
  for (int g = 0; g < groups; ++g) {
    const float s0 = h2f(sv[0]), s1 = h2f(sv[1]);
    __syncthreads();   // every wave has read the previous group's fragments
    store_group();
    __syncthreads();
    if (g + 1 < groups) load_group(g + 1);
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) part[a][b] = float16v{};
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int c = 2 * ks + (lane >> 5);
      half8 fa[2], fb[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) fa[a] = *(const half8*)&sX[x_chunk(wm + 32 * a + (lane & 31), c)];
#pragma unroll
      for (int b = 0; b < 2; ++b) fb[b] = *(const half8*)&sW[w_chunk(wn + 32 * b + (lane & 31), c)];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          part[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[a], fb[b], part[a][b], 0, 0, 0);
    }
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        acc[a][0][j] = fmaf(s0, part[a][0][j], acc[a][0][j]);
        acc[a][1][j] = fmaf(s1, part[a][1][j], acc[a][1][j]);
      }
  }

  // element j of lane l of a 32 x 32 block: row 8 (j / 4) + 4 (l / 32) + j % 4,
  // column l % 32
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int m = m0 + wm + 32 * a + 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
      if (m >= M) continue;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        float* dst = y + (size_t)m * N + n0 + wn + 32 * b + (lane & 31);
        *dst = accumulate ? *dst + acc[a][b][j] : acc[a][b][j];
      }
    }
}

}  // namespace

int launch_prefill(const Layer& L, const void* codes, const void* scales, const void* x, int M,
                   float* y, int accumulate, hipStream_t s) {
  const dim3 grid((unsigned)((M + kBM - 1) / kBM), (unsigned)(L.N / kBN));
  if (L.u == 2)
    hipLaunchKernelGGL(k_prefill<2>, grid, dim3(kThreadsPF), 0, s, (const uint8_t*)codes,
                       (const uint16_t*)scales, (const uint16_t*)x, y, L, M, accumulate);
  else
    hipLaunchKernelGGL(k_prefill<1>, grid, dim3(kThreadsPF), 0, s, (const uint8_t*)codes,
                       (const uint16_t*)scales, (const uint16_t*)x, y, L, M, accumulate);
  return check_launch("prefill");
}

}  // namespace grinqh
