// W4A4 GEMM with Runtime Smooth fused into the K loop (Section 3.2, Eq. 3,
// Fig. 4 step (3)):
//   Y[i, n] = fp16( alpha_i * beta_n / K * sum_b s_b * P_b[i, n] )
//   P_b[i, n] = sum_{j in group b} qx[i, j] * qw[j, n]   (exact int32)
//
// Packed INT4 operands: Xq M x K/2, K contiguous; Wq row-major or tiled
// (WqLayout; a row's K tile of 32 bytes is pieces 2 kt and 2 kt + 1).
// Fallback kernel for shapes outside the main kernel's unrolling (rrs_gemm.hip).
// Tile 128 x 128 per 256-thread workgroup, four waves of 64 x 64, K step 64.
// Global -> registers (16 B per thread per operand) -> unpacked to int8 ->
// LDS (double-buffered) -> v_mfma_i32_32x32x32_i8.
//
// Unpacking: a nibble n of a packed byte is moved into the high half of an
// int8 lane, i.e. the byte holds 16 * q. Low nibbles: (w << 4) & 0xF0F0F0F0,
// high nibbles: w & 0xF0F0F0F0. Each MFMA product is then 256 q w, exact in
// int32 (|256 * 49 * 512| < 2^23); the 2^-8 is folded into the output scale.
// The unpack permutes K inside each 8-element chunk, identically for both
// operands, so every dot product is unchanged.
//
// At the end of each smoothing group the int32 accumulators are converted
// and added into fp32 accumulators with one FMA by s_b, then restart at 0.
//
// The same skeleton also runs the two baselines of the paper's kernel
// comparison (Section 4.5, Fig. 6), so that the three scale schemes differ in
// nothing else:
//   per-channel A4W4: no per-group work; the int32 accumulators run over all
//     of K (|256 P| <= 256 * 49 * 16384 < 2^31) and are converted once;
//   sub-channel A4W4: at the end of group b every accumulator is scaled by
//     fl(a[b][i] * w[b][n]) (scales of shape L x M and L x N, group-major),
//     loaded at the group's first tile.
#include "rrs_internal.h"

namespace rrs {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 64;             // INT4 elements of K per tile
constexpr int KBYTES = BK / 2;     // packed bytes per row per tile
constexpr int LROW = 2 * KBYTES + 16;  // LDS bytes per row: 64 int8 + 16 pad

__device__ __forceinline__ uint4 unpack_lo(uint4 w) {
  return make_uint4((w.x << 4) & 0xF0F0F0F0u, w.x & 0xF0F0F0F0u,
                    (w.y << 4) & 0xF0F0F0F0u, w.y & 0xF0F0F0F0u);
}
__device__ __forceinline__ uint4 unpack_hi(uint4 w) {
  return make_uint4((w.z << 4) & 0xF0F0F0F0u, w.z & 0xF0F0F0F0u,
                    (w.w << 4) & 0xF0F0F0F0u, w.w & 0xF0F0F0F0u);
}

__device__ __forceinline__ uint16_t float_to_half_bits(float x) {
  return __builtin_bit_cast(uint16_t, (_Float16)x);
}

enum Scheme { kRuntimeSmooth = 0, kPerChannel = 1, kSubChannel = 2 };

// kScheme kSubChannel: a_scale is L x M, w_scale is L x N (s_group unused);
// kPerChannel: s_group unused.
template <bool kPartials, int kScheme = kRuntimeSmooth>
__global__ __launch_bounds__(256) void gemm_small_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, int M, int N, int K, int g,
    uint16_t* __restrict__ Y, int32_t* __restrict__ P, float out_scale, WqLayout lay) {
  __shared__ __attribute__((aligned(16))) uint8_t sA[2][BM * LROW];
  __shared__ __attribute__((aligned(16))) uint8_t sB[2][BN * LROW];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int wm = wave >> 1;
  const int wn = wave & 1;
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;
  const size_t kbytes_row = (size_t)K / 2;

  // Global load slots: row t/2, bytes [16 * (t & 1), +16) of the tile's 32.
  const int lrow = t >> 1;
  const int lhalf = t & 1;
  const bool a_ok = (m0 + lrow) < M;
  const bool b_ok = (n0 + lrow) < N;
  const uint8_t* gA = Xq + (size_t)(a_ok ? m0 + lrow : 0) * kbytes_row + lhalf * 16;
  // Piece 2 kt + lhalf of the row lies (kt / 2) tile + 2 (kt % 2) quarter
  // bytes after piece lhalf.
  const uint8_t* gB = Wq + lay.piece(b_ok ? n0 + lrow : 0, lhalf, K);
  const size_t wts = (size_t)lay.tile(), wqs2 = (size_t)2 * lay.quarter();
  const int st_off = lrow * LROW + lhalf * 32;

  uint4 ra = make_uint4(0, 0, 0, 0);
  uint4 rb = make_uint4(0, 0, 0, 0);

  v16i acc[2][2];
  float f[2][2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc[i][j][r] = 0;
        f[i][j][r] = 0.0f;
      }
    }

  const int nkt = K / BK;
  const int tiles_per_group = g / BK;
  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 16;

  if (a_ok) ra = *reinterpret_cast<const uint4*>(gA);
  if (b_ok) rb = *reinterpret_cast<const uint4*>(gB);

  // Sub-channel scales of the current group: this lane's 32 rows and 2 columns.
  float sa[2][16], sb[2];
  for (int kt = 0; kt < nkt; ++kt) {
    const int st = kt & 1;
    if constexpr (kScheme == kSubChannel && !kPartials) {
      if (kt % tiles_per_group == 0) {
        const int grp = kt / tiles_per_group;
        const float* ag = a_scale + (size_t)grp * M;
        const float* wg = w_scale + (size_t)grp * N;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            sa[i][r] = ag[min(row, M - 1)];
          }
#pragma unroll
        for (int j = 0; j < 2; ++j) sb[j] = wg[min(n0 + wn * 64 + j * 32 + (lane & 31), N - 1)];
      }
    }
    *reinterpret_cast<uint4*>(&sA[st][st_off]) = unpack_lo(ra);
    *reinterpret_cast<uint4*>(&sA[st][st_off + 16]) = unpack_hi(ra);
    *reinterpret_cast<uint4*>(&sB[st][st_off]) = unpack_lo(rb);
    *reinterpret_cast<uint4*>(&sB[st][st_off + 16]) = unpack_hi(rb);
    __syncthreads();
    if (kt + 1 < nkt) {
      if (a_ok) ra = *reinterpret_cast<const uint4*>(gA + (size_t)(kt + 1) * KBYTES);
      if (b_ok)
        rb = *reinterpret_cast<const uint4*>(gB + (size_t)((kt + 1) >> 1) * wts +
                                             (size_t)((kt + 1) & 1) * wqs2);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      v4i a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const v4i*>(
            &sA[st][(wm * 64 + i * 32 + frag_row) * LROW + ks * 32 + frag_k]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const v4i*>(
            &sB[st][(wn * 64 + j * 32 + frag_row) * LROW + ks * 32 + frag_k]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if constexpr (kScheme == kPerChannel && !kPartials) continue;
    if ((kt + 1) % tiles_per_group == 0) {
      const int grp = kt / tiles_per_group;
      if constexpr (kPartials) {
        int32_t* Pg = P + (size_t)grp * (size_t)M * (size_t)N;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
              const int col = n0 + wn * 64 + j * 32 + (lane & 31);
              if (row < M && col < N) Pg[(size_t)row * N + col] = acc[i][j][r] >> 8;
            }
      } else if constexpr (kScheme == kSubChannel) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              f[i][j][r] = __builtin_fmaf(sa[i][r] * sb[j], (float)acc[i][j][r], f[i][j][r]);
      } else {
        const float s = s_group[grp];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              f[i][j][r] = __builtin_fmaf(s, (float)acc[i][j][r], f[i][j][r]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;
    }
  }

  if constexpr (kScheme == kPerChannel && !kPartials) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) f[i][j][r] = (float)acc[i][j][r];
  }
  if constexpr (kScheme == kSubChannel && !kPartials) {
    const float inv = out_scale;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < M && col < N)
            Y[(size_t)row * N + col] = float_to_half_bits(f[i][j][r] * inv);
        }
      }
  } else if constexpr (!kPartials) {
    // 2^-8 undoes the 16x16 of the unpacked operands, 1/K the unnormalized rotation.
    const float inv = out_scale;  // 2^-8 / K (2^-8 without rotation), exact
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 64 + j * 32 + (lane & 31);
        const float bcol = col < N ? w_scale[col] : 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < M && col < N) {
            const float sc = a_scale[row] * inv;
            Y[(size_t)row * N + col] = float_to_half_bits((f[i][j][r] * sc) * bcol);
          }
        }
      }
  }
}

}  // namespace

hipError_t launch_w4a4_gemm_small(const uint8_t* Xq, const float* a_scale, const float* s_group,
                            const uint8_t* Wq, const float* w_scale, int M, int N, int K,
                            int g, uint16_t* Y, float out_scale, hipStream_t stream,
                            WqLayout lay) {
  dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  gemm_small_kernel<false><<<grid, 256, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale, M, N, K,
                                                     g, Y, nullptr, out_scale, lay);
  return hipGetLastError();
}

hipError_t launch_w4a4_gemm_scheme(int scheme, const uint8_t* Xq, const float* x_scale,
                                   const float* s_group, const uint8_t* Wq, const float* w_scale,
                                   int M, int N, int K, int g, uint16_t* Y, float out_scale,
                                   hipStream_t stream, WqLayout lay) {
  dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  switch (scheme) {
    case kRuntimeSmooth:
      gemm_small_kernel<false, kRuntimeSmooth><<<grid, 256, 0, stream>>>(
          Xq, x_scale, s_group, Wq, w_scale, M, N, K, g, Y, nullptr, out_scale, lay);
      break;
    case kPerChannel:
      gemm_small_kernel<false, kPerChannel><<<grid, 256, 0, stream>>>(
          Xq, x_scale, nullptr, Wq, w_scale, M, N, K, K, Y, nullptr, out_scale, lay);
      break;
    case kSubChannel:
      gemm_small_kernel<false, kSubChannel><<<grid, 256, 0, stream>>>(
          Xq, x_scale, nullptr, Wq, w_scale, M, N, K, g, Y, nullptr, out_scale, lay);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_w4a4_gemm_partials_small(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                     int K, int g, int32_t* P, hipStream_t stream,
                                     WqLayout lay) {
  dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  gemm_small_kernel<true><<<grid, 256, 0, stream>>>(Xq, nullptr, nullptr, Wq, nullptr, M, N, K, g,
                                                    nullptr, P, 0.0f, lay);
  return hipGetLastError();
}

}  // namespace rrs
