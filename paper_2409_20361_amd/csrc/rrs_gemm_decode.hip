// W4A4 GEMM with Runtime Smooth for few tokens (decode: M <= 64), the same
// product as the main kernel (Section 3.2, Eq. 3, Fig. 4 step (3)):
//   Y[i, n] = fp16( alpha_i * beta_n / K * sum_b s_b * P_b[i, n] )
//   P_b[i, n] = sum_{j in group b} qx[i, j] * qw[j, n]   (exact int32)
//
// With a handful of tokens the work is streaming Wq (N x K/2 bytes) through
// the chip once; the matrix core only has to keep up. The kernel therefore
// maximizes the weight bytes in flight and never stages them in LDS:
//   - a workgroup owns two blocks of 16 output columns (rows of Wq; four
//     blocks with row-major weights from 8 tokens on and with either layout
//     above 16 tokens); its four
//     waves take every fourth smoothing group (wave w: groups w, w + 4, ...,
//     so the four read neighbouring groups of the same rows together) and
//     add their fp32 partial sums in a fixed order at the end
//     (deterministic); each wave unpacks its token codes once for both
//     blocks;
//   - tokens come in up to four blocks of 16 (TB), every block multiplied
//     with the same weight words, so the weights still stream once for up to
//     64 tokens (the 256-row tiles of the main kernel would leave most of
//     their MFMA work idle at such M);
//   - per group, lane (c, q) (c = lane % 16, q = lane / 16) takes g/8 bytes
//     of Wq row n0 + c and the same bytes of Xq row c (zero for c >= M): for
//     g = 64 bytes [8 q, 8 q + 8) of the group, for g >= 128 bytes
//     [64 h + 16 q, +16) of each 64-byte piece h of it. In the tiled Wq
//     (WqLayout) these are bytes [16 lane, +16) of the group's 1 KB tiles, so
//     every weight load instruction of a wave reads one contiguous tile
//     (512 contiguous bytes for g = 64); row-major, 16 rows x 64 bytes.
//     MFMA k-step s of the group
//     (v_mfma_i32_16x16x64_i8, 64 codes) takes the lane's bytes [8 s, 8 s + 8)
//     in that order, so each k-step stays inside one group and A and B pair
//     the same codes;
//   - loads run several groups ahead of the MFMAs (about 48 bytes of Wq per
//     lane in flight, tens of KB per CU), with no branch between a load and
//     its use, so each wait is for exactly the group about to be used.
// Codes are unpacked into the high nibble of each int8 lane (16 q), as in the
// main kernel; the 2^-8 is folded into the output scale. The group rescale
// uses the same magic-number seed: the group's first MFMA starts from the bits
// of 1.5 * 2^23, so the int32 result read as a float is 1.5 * 2^23 + 256 P
// exactly (g <= 256); for g = 512 the accumulators start at 0 and are converted.
#include "rrs_internal.h"

namespace rrs {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 waves: K quarters of the same columns
constexpr int kCols = 16;      // columns per MFMA block
constexpr int kBlocks = 2;     // column blocks per workgroup (they share the A unpack); four
                               // for larger token counts (launcher)

__device__ __forceinline__ v4i unpack_pair(uint32_t w0, uint32_t w1) {
  v4i r;
  r.x = (int)((w0 << 4) & 0xF0F0F0F0u);
  r.y = (int)(w0 & 0xF0F0F0F0u);
  r.z = (int)((w1 << 4) & 0xF0F0F0F0u);
  r.w = (int)(w1 & 0xF0F0F0F0u);
  return r;
}

// NW = g / 32 words (g / 8 bytes) per lane per group: one 8-byte piece at p
// (g = 64) or NW / 4 pieces of 16 bytes at p, p + stride, ...
template <int NW>
__device__ __forceinline__ void load_words(const uint8_t* __restrict__ p, int stride,
                                           uint32_t (&w)[NW]) {
  if constexpr (NW == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    w[0] = v.x;
    w[1] = v.y;
  } else {
#pragma unroll
    for (int c = 0; c < NW / 4; ++c) {
      const uint4 v = *reinterpret_cast<const uint4*>(p + (size_t)c * stride);
      w[4 * c] = v.x;
      w[4 * c + 1] = v.y;
      w[4 * c + 2] = v.z;
      w[4 * c + 3] = v.w;
    }
  }
}

// Groups per wave: a quarter of the groups (one each when K has fewer than
// four groups; waves past the last group get none).
__host__ __device__ inline int groups_per_wave(int K, int g) { return K / g >= 4 ? K / g / 4 : 1; }
constexpr int kMaxTokenBlocks = 4;  // up to 64 tokens

// GS = g / 64 MFMA k-steps per group; TB token blocks of 16 rows (tokens
// 16 tb .. 16 tb + 15 in block tb), all multiplied with the same weight words.
// kPartials (test hook): instead of Y, write P[b][i][n] for every group b,
// token i < M and column n, decoded from the same seeded accumulators.
template <int GS, int TB, bool kTiled, int KB, bool kPartials = false>
__global__ __launch_bounds__(kThreads) void gemm_decode_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, int M, int N, int K, uint16_t* __restrict__ Y,
    float out_scale, int32_t* __restrict__ P = nullptr) {
  constexpr WqLayout lay{kTiled};
  constexpr int g = GS * 64;
  constexpr int NW = g / 32;                  // words per lane per group and block
  constexpr int D0 = NW >= 16 ? 1 : (NW >= 8 ? 2 : 4);
  constexpr int D = TB >= 4 && D0 > 1 ? D0 / 2 : D0;  // groups in flight
  // The four waves' fp32 partial sums, added at the end.
  __shared__ __attribute__((aligned(16))) uint8_t lds[4 * TB * KB * 64 * 16];
  v4f(*part)[TB][KB][64] = reinterpret_cast<v4f(*)[TB][KB][64]>(lds);

  const int t = threadIdx.x;
  const int lane = t & 63;
  // K quarter of this wave; uniform, so group indices and scales are scalar.
  const int kq = __builtin_amdgcn_readfirstlane(t >> 6);
  const int c = lane & 15;
  const int q = lane >> 4;
  const int n0 = blockIdx.x * (KB * kCols);
  const size_t krow = (size_t)K / 2;
  const int G = K / g;
  // Wave kq takes groups kq, kq + 4, kq + 8, ...: at any time the four waves
  // read four neighbouring groups of the same rows (in the row-major Wq,
  // 4 g / 2 contiguous bytes of each row).
  const int per = groups_per_wave(K, g);  // the same for every wave
  const int nb = G > kq ? (G - kq + 3) / 4 : 0;  // groups this wave really has
  const int steps = (per + D - 1) / D * D;

  // The loop is free of branches around loads, so the compiler can count the
  // loads in flight and wait for exactly the group it needs. Steps past this
  // wave's groups load a valid group and add it with scale 0 (exactly 0: the
  // partial sums are finite). Token rows >= M load row M - 1; they only feed
  // output rows that are never stored. Column blocks past N load block 0 and
  // are never stored.
  // Byte offsets of this lane's codes inside a group: in a packed Xq row, and
  // from its Wq row's start (group b starts b gstride later, its pieces h
  // lie a tile apart).
  const int xo = g == 64 ? q * 8 : q * 16;
  constexpr int wqs = lay.quarter();
  constexpr int wts = lay.tile();
  const int wo = g == 64 ? (q >> 1) * wqs + (q & 1) * 8 : q * wqs;
  constexpr size_t gstride = kTiled ? (size_t)8 * g : (size_t)(g / 2);
  const uint8_t* pa[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) pa[tb] = Xq + (size_t)min(16 * tb + c, M - 1) * krow + xo;
  const uint8_t* pb[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) {
    const int n = n0 + j * kCols < N ? n0 + j * kCols : 0;
    pb[j] = Wq + lay.row(n + c, K) + wo;
  }

  uint32_t wa[D][TB][NW], wb[D][KB][NW];
  auto load = [&](int d, int i) {
    const int b = min(kq + 4 * i, G - 1);
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) load_words<NW>(pa[tb] + (size_t)b * (g / 2), 64, wa[d][tb]);
#pragma unroll
    for (int j = 0; j < KB; ++j) load_words<NW>(pb[j] + (size_t)b * gstride, wts, wb[d][j]);
  };

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = GS > 4 ? v4i{0, 0, 0, 0} : v4i{kMagic, kMagic, kMagic, kMagic};
  float f[TB][KB][4];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int j = 0; j < KB; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) f[tb][j][r] = 0.0f;

  auto consume = [&](int d, int i) {
    const float s = (!kPartials && i < nb) ? s_group[min(kq + 4 * i, G - 1)] : 0.0f;
    v4i acc[TB][KB];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
      for (int j = 0; j < KB; ++j) acc[tb][j] = seed;
#pragma unroll
    for (int st = 0; st < GS; ++st) {
      v4i bv[KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) bv[j] = unpack_pair(wb[d][j][2 * st], wb[d][j][2 * st + 1]);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        const v4i a = unpack_pair(wa[d][tb][2 * st], wa[d][tb][2 * st + 1]);
#pragma unroll
        for (int j = 0; j < KB; ++j)
          acc[tb][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, bv[j], acc[tb][j], 0, 0, 0);
      }
    }
    if constexpr (kPartials) {
      if (i < nb) {
        int32_t* Pg = P + (size_t)(kq + 4 * i) * (size_t)M * (size_t)N;
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
#pragma unroll
          for (int j = 0; j < KB; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = 16 * tb + 4 * q + r;
              const int col = n0 + j * kCols + c;
              const int v = acc[tb][j][r];
              if (row < M && col < N) Pg[(size_t)row * N + col] = (GS > 4 ? v : v - kMagic) >> 8;
            }
      }
      return;
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        // Bit-cast the whole vector, then index: bit-casting a single element
        // of an ext_vector is miscompiled (every element reads element 0).
        const v4f accf = __builtin_bit_cast(v4f, acc[tb][j]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pv = GS > 4 ? (float)acc[tb][j][r] : accf[r] - 12582912.0f;
          f[tb][j][r] = __builtin_fmaf(s, pv, f[tb][j][r]);
        }
      }
  };

#pragma unroll
  for (int d = 0; d < D; ++d) load(d, d);
  int i = 0;
  for (; i < steps - D; i += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      consume(d, i + d);
      load(d, i + d + D);
    }
  }
#pragma unroll
  for (int d = 0; d < D; ++d) consume(d, i + d);

  if constexpr (kPartials) return;
  // Partial sums of the four K quarters, added in a fixed order.
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int j = 0; j < KB; ++j)
      part[kq][tb][j][lane] = v4f{f[tb][j][0], f[tb][j][1], f[tb][j][2], f[tb][j][3]};
  __syncthreads();
  // Wave w stores column block w (if any): sums in the order kq = 0, 1, 2, 3.
  const int w = t >> 6;
  if (w < KB && n0 + w * kCols < N) {
    // out_scale = 2^-8 (undoes the 16 x 16 of the unpacked operands) / K (the
    // unnormalized rotation; 1 without rotation), an exact power of two.
    const float inv = out_scale;
    const int col = n0 + w * kCols + c;
    const float bcol = w_scale[col];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      v4f sum = part[0][tb][w][lane];
#pragma unroll
      for (int p = 1; p < 4; ++p) {
        const v4f x = part[p][tb][w][lane];
        sum.x += x.x;
        sum.y += x.y;
        sum.z += x.z;
        sum.w += x.w;
      }
      const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * tb + 4 * q + r;  // output row of accumulator r of this lane
        if (row < M) {
          const float sc = a_scale[row] * inv;
          Y[(size_t)row * N + col] =
              __builtin_bit_cast(uint16_t, (_Float16)((sv[r] * sc) * bcol));
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Runtime channel reorder: position block p (32 channels, 16 bytes of a packed
// row) of Xq pairs with natural block border[p] of every Wq row.
//
// The weights still stream in natural order: a sorted-order walk over the
// weight rows would use the eight 16-byte blocks of each 128-byte line at
// different times, and this streaming kernel would fetch most lines several
// times. Instead the (small, cache-resident) token codes are gathered. Wave kq
// walks its K quarter in quads of four natural blocks 4m .. 4m + 3: lane (c, q)
// loads block 4m + q of weight row n0 + 16 j + c (with the tiled Wq the wave
// reads tile m of the column block, 1 KB contiguous) and position block
// inv[4m + q] of token row c. A 4 x 4
// dword transpose through a wave-private LDS region then gives lane group q
// dword q of each of the four blocks, so that one v_mfma_i32_16x16x32_i8 per
// block and column block (lane group q holds channels 8q .. 8q + 7 of the block
// after the unpack, the same for both operands) yields the block's exact
// partial sum. It is rescaled by the scale of the group its position falls in,
// s_{inv[B] / (g/32)}: the sum over a group's blocks is taken in fp32 (K/32
// rescaled terms per output instead of K/g).
// ---------------------------------------------------------------------------
constexpr int kGatherAhead = 2;  // quads in flight per wave
constexpr int kTrStride = 20;    // dwords per row of the transpose region (conflict-free)

__device__ __forceinline__ long unpack_dword(uint32_t w) {
  const uint32_t lo = (w << 4) & 0xF0F0F0F0u;
  const uint32_t hi = w & 0xF0F0F0F0u;
  return (long)(((unsigned long)hi << 32) | lo);
}

template <bool kTiled>
__global__ __launch_bounds__(kThreads) void gemm_decode_gather_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, const int32_t* __restrict__ border, int M, int N,
    int K, int g, uint16_t* __restrict__ Y, float out_scale) {
  constexpr WqLayout lay{kTiled};
  constexpr int kMaxBlocks = 16384 / kReorderBlock;
  constexpr int kArrays = 1 + kBlocks;  // token codes and the column blocks' weights
  __shared__ int inv[kMaxBlocks];      // natural block -> byte offset of its position block
  __shared__ float sblk[kMaxBlocks];   // natural block -> scale of its position's group
  __shared__ __attribute__((aligned(16))) uint32_t tr[4][kArrays][kCols * kTrStride];
  __shared__ __attribute__((aligned(16))) v4f part[4][kBlocks][64];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int kq = __builtin_amdgcn_readfirstlane(t >> 6);
  const int c = lane & 15;
  const int q = lane >> 4;
  const int n0 = blockIdx.x * (kBlocks * kCols);
  const size_t krow = (size_t)K / 2;
  const int NB = K / kReorderBlock;
  const int quads = NB / 16;     // quads per wave (K >= 512: at least 1)
  const int b0 = kq * (NB / 4);  // first natural block of this wave
  constexpr size_t wts = (size_t)lay.tile();
  const int steps = (quads + kGatherAhead - 1) / kGatherAhead * kGatherAhead;

  // Tables. Entries are reduced modulo K/32, so any table keeps every load in
  // bounds; a table that is not a permutation leaves some blocks at scale 0.
  for (int i = t; i < NB; i += kThreads) {
    inv[i] = 0;
    sblk[i] = 0.0f;
  }
  __syncthreads();
  for (int p = t; p < NB; p += kThreads) {
    const int B = border[p] & (NB - 1);
    inv[B] = p * 16;
    sblk[B] = s_group[p / (g / kReorderBlock)];
  }
  __syncthreads();

  // Token rows >= M read row M - 1 and column blocks past N read block 0: their
  // results are never stored.
  const uint8_t* pa = Xq + (size_t)min(c, M - 1) * krow;
  const uint8_t* pb[kBlocks];
#pragma unroll
  for (int j = 0; j < kBlocks; ++j) {
    const int n = n0 + j * kCols < N ? n0 + j * kCols : 0;
    pb[j] = Wq + lay.row(n + c, K) + (size_t)q * lay.quarter();  // quad m: m tiles on
  }
  uint32_t* trw = &tr[kq][0][0];

  uint4 ld[kGatherAhead][kArrays];
  // Steps past this wave's quads reload its last quad and add it with scale 0.
  auto load = [&](int d, int i) {
    const int B0 = b0 + 4 * min(i, quads - 1);
    ld[d][0] = *reinterpret_cast<const uint4*>(pa + inv[B0 + q]);
#pragma unroll
    for (int j = 0; j < kBlocks; ++j)
      ld[d][1 + j] = *reinterpret_cast<const uint4*>(pb[j] + (size_t)(B0 >> 2) * wts);
  };

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = {kMagic, kMagic, kMagic, kMagic};
  float f[kBlocks][4];
#pragma unroll
  for (int j = 0; j < kBlocks; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) f[j][r] = 0.0f;

  // 4 x 4 transpose, first half: lane (c, q) holds dwords 0..3 of block q of
  // the quad and writes them to row c of the wave's region; the registers are
  // then free for the next loads.
  auto stash = [&](int d) {
#pragma unroll
    for (int a = 0; a < kArrays; ++a) {
      uint32_t* base = trw + a * (kCols * kTrStride) + c * kTrStride + q;
      base[0] = ld[d][a].x;
      base[4] = ld[d][a].y;
      base[8] = ld[d][a].z;
      base[12] = ld[d][a].w;
    }
  };
  // Second half: take back dword q of blocks 0..3, then one MFMA per block.
  auto consume = [&](int i) {
    uint4 tv[kArrays];
#pragma unroll
    for (int a = 0; a < kArrays; ++a)
      tv[a] = *reinterpret_cast<const uint4*>(trw + a * (kCols * kTrStride) + c * kTrStride +
                                              4 * q);
    const int B0 = b0 + 4 * min(i, quads - 1);
    const uint32_t av[4] = {tv[0].x, tv[0].y, tv[0].z, tv[0].w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float s = i < quads ? sblk[B0 + u] : 0.0f;
      const long a = unpack_dword(av[u]);
#pragma unroll
      for (int j = 0; j < kBlocks; ++j) {
        const uint32_t bw = u == 0 ? tv[1 + j].x : u == 1 ? tv[1 + j].y
                          : u == 2 ? tv[1 + j].z : tv[1 + j].w;
        // |256 P_B| <= 256 * 49 * 32 < 2^22: the magic-seeded result read as
        // a float is exactly 1.5 * 2^23 + 256 P_B.
        const v4i acc = __builtin_amdgcn_mfma_i32_16x16x32_i8(a, unpack_dword(bw), seed, 0, 0, 0);
        const v4f accf = __builtin_bit_cast(v4f, acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) f[j][r] = __builtin_fmaf(s, accf[r] - 12582912.0f, f[j][r]);
      }
    }
  };

#pragma unroll
  for (int d = 0; d < kGatherAhead; ++d) load(d, d);
  int i = 0;
  for (; i < steps - kGatherAhead; i += kGatherAhead) {
#pragma unroll
    for (int d = 0; d < kGatherAhead; ++d) {
      stash(d);
      load(d, i + d + kGatherAhead);
      consume(i + d);
    }
  }
#pragma unroll
  for (int d = 0; d < kGatherAhead; ++d) {
    stash(d);
    consume(i + d);
  }

  // Partial sums of the four K quarters, added in a fixed order (as above).
#pragma unroll
  for (int j = 0; j < kBlocks; ++j) part[kq][j][lane] = v4f{f[j][0], f[j][1], f[j][2], f[j][3]};
  __syncthreads();
  const int w = t >> 6;
  if (w < kBlocks && n0 + w * kCols < N) {
    v4f sum = part[0][w][lane];
#pragma unroll
    for (int p = 1; p < 4; ++p) {
      const v4f x = part[p][w][lane];
      sum.x += x.x;
      sum.y += x.y;
      sum.z += x.z;
      sum.w += x.w;
    }
    const float inv_s = out_scale;
    const int col = n0 + w * kCols + c;
    const float bcol = w_scale[col];
    const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 4 * q + r;
      if (row < M) {
        const float sc = a_scale[row] * inv_s;
        Y[(size_t)row * N + col] = __builtin_bit_cast(uint16_t, (_Float16)((sv[r] * sc) * bcol));
      }
    }
  }
}

}  // namespace

bool decode_kernel_fits(int M) { return M >= 1 && M <= kCols * kMaxTokenBlocks; }

hipError_t launch_w4a4_gemm_decode_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                            int K, int g, int32_t* P, hipStream_t stream) {
  // The same block and token-block choice as the row-major Y launch below.
  const int grid = (N / kCols + kBlocks - 1) / kBlocks;
  const int grid4 = (N / kCols + 3) / 4;
  const bool kb4 = M >= 8;
  const int tbs = M <= kCols ? 1 : (M <= 2 * kCols ? 2 : 4);
#define RRS_DECODE_P(GS_, TB_)                                                              \
  if (kb4)                                                                                 \
    gemm_decode_kernel<GS_, TB_, false, 4, true><<<grid4, kThreads, 0, stream>>>(            \
        Xq, nullptr, nullptr, Wq, nullptr, M, N, K, nullptr, 0.0f, P);                      \
  else                                                                                     \
    gemm_decode_kernel<GS_, TB_, false, kBlocks, true><<<grid, kThreads, 0, stream>>>(      \
        Xq, nullptr, nullptr, Wq, nullptr, M, N, K, nullptr, 0.0f, P)
#define RRS_DECODE_P_TB(GS_) \
  if (tbs == 1) {            \
    RRS_DECODE_P(GS_, 1);    \
  } else if (tbs == 2) {     \
    RRS_DECODE_P(GS_, 2);    \
  } else {                   \
    RRS_DECODE_P(GS_, 4);    \
  }
  switch (g) {
    case 64: RRS_DECODE_P_TB(1) break;
    case 128: RRS_DECODE_P_TB(2) break;
    case 256: RRS_DECODE_P_TB(4) break;
    case 512: RRS_DECODE_P_TB(8) break;
    default: return hipErrorInvalidValue;
  }
#undef RRS_DECODE_P_TB
#undef RRS_DECODE_P
  return hipGetLastError();
}
bool decode_gather_fits(int M) { return M >= 1 && M <= kCols; }

hipError_t launch_w4a4_gemm_decode(const uint8_t* Xq, const float* a_scale,
                                   const float* s_group, const uint8_t* Wq,
                                   const float* w_scale, int M, int N, int K, int g,
                                   uint16_t* Y, float out_scale, hipStream_t stream,
                                   const int32_t* border, WqLayout lay) {
  const int grid = (N / kCols + kBlocks - 1) / kBlocks;  // N % 16 == 0 (API precondition)
  // Four column blocks per workgroup (64 rows of Wq) for row-major weights
  // from 8 tokens on and for either layout above 16 tokens (at the decode
  // shape, row-major: 3 % faster at M = 8, 19 % at M = 64).
  const bool kb4 = lay.tiled ? M > kCols : M >= 8;
  const int grid4 = (N / kCols + 3) / 4;
  if (border) {
    if (M > kCols) return hipErrorInvalidValue;  // the gather kernel takes one token block
    if (lay.tiled)
      gemm_decode_gather_kernel<true><<<grid, kThreads, 0, stream>>>(
          Xq, a_scale, s_group, Wq, w_scale, border, M, N, K, g, Y, out_scale);
    else
      gemm_decode_gather_kernel<false><<<grid, kThreads, 0, stream>>>(
          Xq, a_scale, s_group, Wq, w_scale, border, M, N, K, g, Y, out_scale);
    return hipGetLastError();
  }
  const int tbs = M <= kCols ? 1 : (M <= 2 * kCols ? 2 : 4);
#define RRS_DECODE(GS_, TB_)                                                    \
  if (lay.tiled && kb4)                                                        \
    gemm_decode_kernel<GS_, TB_, true, 4><<<grid4, kThreads, 0, stream>>>(       \
        Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y, out_scale);             \
  else if (lay.tiled)                                                          \
    gemm_decode_kernel<GS_, TB_, true, kBlocks><<<grid, kThreads, 0, stream>>>(  \
        Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y, out_scale);             \
  else if (kb4)                                                                \
    gemm_decode_kernel<GS_, TB_, false, 4><<<grid4, kThreads, 0, stream>>>(      \
        Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y, out_scale);             \
  else                                                                         \
    gemm_decode_kernel<GS_, TB_, false, kBlocks><<<grid, kThreads, 0, stream>>>( \
        Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y, out_scale)
#define RRS_DECODE_TB(GS_) \
  if (tbs == 1) {          \
    RRS_DECODE(GS_, 1);    \
  } else if (tbs == 2) {   \
    RRS_DECODE(GS_, 2);    \
  } else {                 \
    RRS_DECODE(GS_, 4);    \
  }
  switch (g) {
    case 64: RRS_DECODE_TB(1) break;
    case 128: RRS_DECODE_TB(2) break;
    case 256: RRS_DECODE_TB(4) break;
    case 512: RRS_DECODE_TB(8) break;
    default: return hipErrorInvalidValue;
  }
#undef RRS_DECODE_TB
#undef RRS_DECODE
  return hipGetLastError();
}

}  // namespace rrs
