// W4A4 GEMM with Runtime Smooth for few tokens (decode: M <= 16), the same
// product as the main kernel (Section 3.2, Eq. 3, Fig. 4 step (3)):
//   Y[i, n] = fp16( alpha_i * beta_n / K * sum_b s_b * P_b[i, n] )
//   P_b[i, n] = sum_{j in group b} qx[i, j] * qw[j, n]   (exact int32)
//
// With a handful of tokens the work is streaming Wq (N x K/2 bytes) through
// the chip once; the matrix core only has to keep up. The kernel therefore
// maximizes the weight bytes in flight and never stages them in LDS:
//   - a workgroup owns 16 output columns (16 rows of Wq); its four waves
//     split K into quarters (whole smoothing groups each) and add their
//     fp32 partial sums in a fixed order at the end (deterministic);
//   - per group, lane (c, q) (c = lane % 16, q = lane / 16) loads the g/8
//     contiguous bytes [q g/8, (q+1) g/8) of the group in Wq row n0 + c, and
//     the same bytes of Xq row c (zero for c >= M). MFMA k-step s of the group
//     (v_mfma_i32_16x16x64_i8, 64 codes) takes bytes [8 s, 8 s + 8) of every
//     lane, so each k-step stays inside one group and A and B pair the same
//     codes;
//   - loads run several groups ahead of the MFMAs (about 64 bytes of Wq per
//     lane in flight, tens of KB per CU).
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

constexpr int kThreads = 256;  // 4 waves: K quarters of the same 16 columns
constexpr int kCols = 16;

__device__ __forceinline__ v4i unpack_pair(uint32_t w0, uint32_t w1) {
  v4i r;
  r.x = (int)((w0 << 4) & 0xF0F0F0F0u);
  r.y = (int)(w0 & 0xF0F0F0F0u);
  r.z = (int)((w1 << 4) & 0xF0F0F0F0u);
  r.w = (int)(w1 & 0xF0F0F0F0u);
  return r;
}

// NW = g / 32 words (g / 8 bytes) per lane per group, read from p.
template <int NW>
__device__ __forceinline__ void load_words(const uint8_t* __restrict__ p, uint32_t (&w)[NW]) {
  if constexpr (NW == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    w[0] = v.x;
    w[1] = v.y;
  } else {
#pragma unroll
    for (int c = 0; c < NW / 4; ++c) {
      const uint4 v = reinterpret_cast<const uint4*>(p)[c];
      w[4 * c] = v.x;
      w[4 * c + 1] = v.y;
      w[4 * c + 2] = v.z;
      w[4 * c + 3] = v.w;
    }
  }
}

// GS = g / 64 MFMA k-steps per group.
template <int GS>
__global__ __launch_bounds__(kThreads) void gemm_decode_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, int M, int N, int K, uint16_t* __restrict__ Y) {
  constexpr int g = GS * 64;
  constexpr int NW = g / 32;                 // words per lane per group
  constexpr int D = NW >= 16 ? 1 : 16 / NW;  // groups in flight (64 bytes per lane)
  __shared__ v4f part[4][64];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int kq = t >> 6;  // K quarter of this wave
  const int c = lane & 15;
  const int q = lane >> 4;
  const int n0 = blockIdx.x * kCols;
  const size_t krow = (size_t)K / 2;
  const int G = K / g;
  const int per = G >= 4 ? G / 4 : 1;  // groups per wave
  const int b0 = kq * per;
  const int b1 = min(G, b0 + per);

  const uint8_t* pb = Wq + (size_t)(n0 + c) * krow + q * (g / 8);
  const bool arow = c < M;
  const uint8_t* pa = Xq + (size_t)(arow ? c : 0) * krow + q * (g / 8);

  uint32_t wb[D][NW], wa[D][NW];
  auto load = [&](int d, int b) {
    load_words<NW>(pb + (size_t)b * (g / 2), wb[d]);
    if (arow) {
      load_words<NW>(pa + (size_t)b * (g / 2), wa[d]);
    } else {
#pragma unroll
      for (int i = 0; i < NW; ++i) wa[d][i] = 0u;
    }
  };

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = GS > 4 ? v4i{0, 0, 0, 0} : v4i{kMagic, kMagic, kMagic, kMagic};
  float f[4] = {0.0f, 0.0f, 0.0f, 0.0f};

#pragma unroll
  for (int d = 0; d < D; ++d)
    if (b0 + d < b1) load(d, b0 + d);

  for (int b = b0; b < b1; b += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int bb = b + d;
      if (bb < b1) {
        const float s = s_group[bb];
        v4i acc = seed;
#pragma unroll
        for (int st = 0; st < GS; ++st)
          acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(unpack_pair(wa[d][2 * st], wa[d][2 * st + 1]),
                                                     unpack_pair(wb[d][2 * st], wb[d][2 * st + 1]),
                                                     acc, 0, 0, 0);
        if (bb + D < b1) load(d, bb + D);
        // Bit-cast the whole vector, then index: bit-casting a single element
        // of an ext_vector is miscompiled (every element reads element 0).
        const v4f accf = __builtin_bit_cast(v4f, acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pv = GS > 4 ? (float)acc[r] : accf[r] - 12582912.0f;
          f[r] = __builtin_fmaf(s, pv, f[r]);
        }
      }
    }
  }

  // Partial sums of the four K quarters, added in a fixed order.
  part[kq][lane] = v4f{f[0], f[1], f[2], f[3]};
  __syncthreads();
  if (kq == 0) {
    v4f sum = part[0][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const v4f p = part[w][lane];
      sum.x += p.x;
      sum.y += p.y;
      sum.z += p.z;
      sum.w += p.w;
    }
    // 2^-8 undoes the 16 x 16 of the unpacked operands, 1/K the unnormalized rotation.
    const float inv = __builtin_ldexpf(1.0f, -8) / (float)K;
    const int col = n0 + c;
    const float bcol = w_scale[col];
    const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 4 * q + r;  // output row of accumulator r of this lane
      if (row < M) {
        const float sc = a_scale[row] * inv;
        Y[(size_t)row * N + col] = __builtin_bit_cast(uint16_t, (_Float16)((sv[r] * sc) * bcol));
      }
    }
  }
}

}  // namespace

bool decode_kernel_fits(int M) { return M >= 1 && M <= kCols; }

hipError_t launch_w4a4_gemm_decode(const uint8_t* Xq, const float* a_scale,
                                   const float* s_group, const uint8_t* Wq,
                                   const float* w_scale, int M, int N, int K, int g,
                                   uint16_t* Y, hipStream_t stream) {
  const int grid = N / kCols;  // N % 16 == 0 is an API precondition
  switch (g) {
    case 64:
      gemm_decode_kernel<1><<<grid, kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y);
      break;
    case 128:
      gemm_decode_kernel<2><<<grid, kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y);
      break;
    case 256:
      gemm_decode_kernel<4><<<grid, kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y);
      break;
    case 512:
      gemm_decode_kernel<8><<<grid, kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rrs
