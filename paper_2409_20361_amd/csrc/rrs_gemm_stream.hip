// W4A4 GEMM with Runtime Smooth for up to 16 tokens: the same product as the
// other GEMM kernels (Section 3.2, Eq. 3, Fig. 4 step (3)):
//   Y[i, n] = fp16( alpha_i * beta_n / K * sum_b s_b * P_b[i, n] )
//   P_b[i, n] = sum_{j in group b} qx[i, j] * qw[j, n]   (exact int32)
//
// At decode sizes the whole cost is streaming Wq (N x K/2 bytes) from HBM once,
// so the kernel is built around the shape of its weight loads. A workgroup
// owns 16 output columns, i.e. 16 consecutive rows of Wq, which are one
// contiguous run of 8 K bytes in either layout; its four waves take a quarter
// of K each (wave w: packed bytes [w R, w R + R) of every row, R = K / 8),
// again one contiguous run of 16 R bytes in the tiled layout. A wave copies
// its 16 x R bytes with direct-to-LDS loads (global_load_lds_dwordx4): every
// instruction moves 1 KB of consecutive global bytes into the wave's LDS
// region without passing through registers. The MFMA operand layout wants
// lane (c, q) to hold row c, which a direct load of 1 KB cannot give; the LDS
// region turns the contiguous stream into that layout, read back with one
// ds_read_b128 per lane per 64-byte piece.
//
// LDS layout of a wave's region. Row-major Wq: a load instruction takes one
// row piece of 1 KB, or several whole row pieces when R < 1 KB; row r sits
// at r R with its 16-byte chunks permuted by chunk' = chunk ^ (r & 7), so
// that the 16 lanes reading the same chunk of 16 rows hit different banks.
// The permutation is applied on the global side (lane i of a direct load
// lands at slot i and fetches the chunk that belongs there), so each load
// instruction still covers a contiguous 1 KB range. Tiled Wq: a load
// instruction takes one 1 KB tile (16 rows x 64 bytes, quarter by quarter)
// unchanged, and the 16 lanes reading quarter q of the 16 rows read 256
// consecutive bytes. Both layouts give the same operands in the same order,
// so their results are bit-identical.
//
// The direct loads are not tracked by the compiler's wait insertion for the
// LDS reads that follow, so the kernel waits for them explicitly (vmcnt(0))
// before the first read. Each wave reads only its own region: no barrier.
//
// Token codes (M x K/2, a few KB, L2-resident) are loaded into registers:
// lane (c, q) takes the same bytes of token row c (row M - 1 for c >= M, whose
// outputs are never stored). Per group b of the wave, lane (c, q) holds
// bytes [64 h + 16 q, +16) of each 64-byte piece h of the group (g >= 128) or
// bytes [8 q, +8) (g = 64); MFMA k-step s (v_mfma_i32_16x16x64_i8) takes the
// lane's bytes [8 s, 8 s + 8) in that order for both operands, so every k-step
// stays inside one group. Codes are unpacked into the high nibble of each int8
// lane (16 q, the 2^-8 folded into the output scale) and each group's int32
// accumulators start from the bits of 1.5 * 2^23 (g <= 256), so that the
// result read as a float is exactly 1.5 * 2^23 + 256 P_b and one subtraction
// recovers 256 P_b before the FMA by s_b; for g = 512 they start from 0 and
// are converted. The four waves' fp32 sums are added in a fixed order.
//
// Needs K >= 4 g (every wave holds whole groups): K = 512 with g <= 128,
// K = 1024 with g <= 256, any g from K = 2048.
#include "rrs_internal.h"

namespace rrs {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 16;  // weight rows (output columns) per workgroup
constexpr int kMaxTokens = 16;

template <int K>
struct StreamShape {
  static constexpr int R = K / 2 / kWaves;            // packed bytes per row per wave
  static constexpr int CPR = R / 16;                  // 16-byte chunks per row per wave
  static constexpr int SW = CPR >= 8 ? 7 : CPR - 1;  // chunk permutation mask
  static constexpr int REGION = kRows * R;            // LDS bytes per wave
  static constexpr int NLD = REGION / 1024;           // direct loads of 1 KB per wave
  static_assert(REGION % 1024 == 0, "a wave's region is a whole number of 1 KB loads");
};

__device__ __forceinline__ v4i unpack_pair(uint32_t w0, uint32_t w1) {
  v4i r;
  r.x = (int)((w0 << 4) & 0xF0F0F0F0u);
  r.y = (int)(w0 & 0xF0F0F0F0u);
  r.z = (int)((w1 << 4) & 0xF0F0F0F0u);
  r.w = (int)(w1 & 0xF0F0F0F0u);
  return r;
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// kPartials (test hook): instead of Y, write P[b][i][n] for every group b,
// token i < M and column n, decoded from the same seeded accumulators.
template <int K, int GS, bool kTiled, bool kPartials>
__global__ __launch_bounds__(kThreads) void gemm_stream_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, int M, int N, uint16_t* __restrict__ Y,
    int32_t* __restrict__ P, float out_scale) {
  using S = StreamShape<K>;
  constexpr int g = GS * 64;
  constexpr int GB = g / 2;                 // packed bytes of a row per group
  constexpr int NG = S::R / GB;             // groups per wave
  constexpr int NP = GB >= 64 ? GB / 64 : 1;  // 16-byte lane pieces per group
  static_assert(NG >= 1 && S::R % GB == 0, "every wave holds whole groups");
  __shared__ __attribute__((aligned(16))) uint8_t region[kWaves * S::REGION];
  __shared__ __attribute__((aligned(16))) v4f part[kWaves][64];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int kq = __builtin_amdgcn_readfirstlane(t >> 6);  // K quarter of this wave
  const int c = lane & 15;
  const int q = lane >> 4;
  const int n0 = blockIdx.x * kRows;
  constexpr size_t krow = (size_t)K / 2;
  uint8_t* my = region + kq * S::REGION;

  // 1. The wave's 16 rows x R bytes of Wq, straight into its LDS region
  // (n0 is a multiple of 16: in the tiled layout the 16 rows are one block,
  // and the wave's quarter of K is its tiles kq R / 64 .. (kq + 1) R / 64 - 1).
  if constexpr (kTiled) {
    const uint8_t* wbase = Wq + (size_t)n0 * krow + (size_t)kq * S::R * kRows;
#pragma unroll
    for (int ii = 0; ii < S::NLD; ++ii)
      __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(wbase + 1024 * ii + 16 * lane),
                                       (lds_ptr_t)(my + 1024 * ii), 16, 0, 0);
  } else {
    const uint8_t* wbase = Wq + (size_t)n0 * krow + (size_t)kq * S::R;
#pragma unroll
    for (int ii = 0; ii < S::NLD; ++ii) {
      const int L = 64 * ii + lane;  // chunk slot in the region
      const int r = L / S::CPR;
      const int j = (L % S::CPR) ^ (r & S::SW);
      __builtin_amdgcn_global_load_lds(
          reinterpret_cast<const void*>(wbase + (size_t)r * krow + 16 * j),
          (lds_ptr_t)(my + 1024 * ii), 16, 0, 0);
    }
  }
  // LDS offset of bytes [16 jc + 8 e, +8) of row c of the wave's quarter
  // (jc: 16-byte chunk index within the quarter, e: 0 or 1).
  auto woff = [&](int jc, int e) -> int {
    if constexpr (kTiled)
      return (jc >> 2) * 1024 + ((jc & 3) * 16 + c) * 16 + 8 * e;
    else
      return c * S::R + 16 * (jc ^ (c & S::SW)) + 8 * e;
  };

  // 2. Token codes of the same bytes, and the wave's group scales (one per lane).
  const uint8_t* abase = Xq + (size_t)min(c, M - 1) * krow + (size_t)kq * S::R;
  uint32_t aw[NG][NP][4];
#pragma unroll
  for (int b = 0; b < NG; ++b) {
    if constexpr (GB >= 64) {
#pragma unroll
      for (int h = 0; h < NP; ++h) {
        const uint4 v = *reinterpret_cast<const uint4*>(abase + b * GB + 64 * h + 16 * q);
        aw[b][h][0] = v.x;
        aw[b][h][1] = v.y;
        aw[b][h][2] = v.z;
        aw[b][h][3] = v.w;
      }
    } else {
      const uint2 v = *reinterpret_cast<const uint2*>(abase + b * GB + 8 * q);
      aw[b][0][0] = v.x;
      aw[b][0][1] = v.y;
      aw[b][0][2] = 0u;
      aw[b][0][3] = 0u;
    }
  }
  float sv = 0.0f;
  if constexpr (!kPartials) sv = s_group[kq * NG + (lane < NG ? lane : 0)];

  // Every direct load of this wave has landed in LDS.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = GS > 4 ? v4i{0, 0, 0, 0} : v4i{kMagic, kMagic, kMagic, kMagic};
  float f[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int b = 0; b < NG; ++b) {
    uint32_t ww[NP][4];
#pragma unroll
    for (int h = 0; h < NP; ++h) {
      if constexpr (GB >= 64) {
        const int jc = b * (GB / 16) + 4 * h + q;
        const uint4 v = *reinterpret_cast<const uint4*>(my + woff(jc, 0));
        ww[h][0] = v.x;
        ww[h][1] = v.y;
        ww[h][2] = v.z;
        ww[h][3] = v.w;
      } else {
        const int jc = 2 * b + (q >> 1);
        const uint2 v = *reinterpret_cast<const uint2*>(my + woff(jc, q & 1));
        ww[h][0] = v.x;
        ww[h][1] = v.y;
        ww[h][2] = 0u;
        ww[h][3] = 0u;
      }
    }
    v4i acc = seed;
#pragma unroll
    for (int st = 0; st < GS; ++st) {
      const int h = st >> 1;
      const int o = 2 * (st & 1);
      acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(unpack_pair(aw[b][h][o], aw[b][h][o + 1]),
                                                  unpack_pair(ww[h][o], ww[h][o + 1]), acc, 0,
                                                  0, 0);
    }
    if constexpr (kPartials) {
      int32_t* Pg = P + (size_t)(kq * NG + b) * (size_t)M * (size_t)N;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 4 * q + r;
        if (row < M) Pg[(size_t)row * N + n0 + c] = (GS > 4 ? acc[r] : acc[r] - kMagic) >> 8;
      }
    } else {
      const float s = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                    __builtin_bit_cast(int, sv), b));
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
  if constexpr (!kPartials) {
    // The four quarters' sums, added in the order kq = 0, 1, 2, 3.
    part[kq][lane] = v4f{f[0], f[1], f[2], f[3]};
    __syncthreads();
    if (kq == 0) {
      v4f sum = part[0][lane];
#pragma unroll
      for (int p = 1; p < kWaves; ++p) {
        const v4f x = part[p][lane];
        sum.x += x.x;
        sum.y += x.y;
        sum.z += x.z;
        sum.w += x.w;
      }
      // out_scale = 2^-8 (undoes the 16 x 16 of the unpacked operands) / K (the
      // unnormalized rotation; 1 without rotation), an exact power of two.
      const int col = n0 + c;
      const float bcol = w_scale[col];
      const float sums[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 4 * q + r;
        if (row < M) {
          const float sc = a_scale[row] * out_scale;
          Y[(size_t)row * N + col] =
              __builtin_bit_cast(uint16_t, (_Float16)((sums[r] * sc) * bcol));
        }
      }
    }
  }
}

template <int K, bool kPartials>
hipError_t launch_k(const uint8_t* Xq, const float* a_scale, const float* s_group,
                    const uint8_t* Wq, const float* w_scale, int M, int N, int g, uint16_t* Y,
                    int32_t* P, float out_scale, hipStream_t stream, bool tiled) {
  const int grid = N / kRows;  // N % 16 == 0 (API precondition)
#define RRS_STREAM(GS_)                                                                   \
  if (tiled)                                                                              \
    gemm_stream_kernel<K, GS_, true, kPartials><<<grid, kThreads, 0, stream>>>(          \
        Xq, a_scale, s_group, Wq, w_scale, M, N, Y, P, out_scale);                        \
  else                                                                                    \
    gemm_stream_kernel<K, GS_, false, kPartials><<<grid, kThreads, 0, stream>>>(         \
        Xq, a_scale, s_group, Wq, w_scale, M, N, Y, P, out_scale)
  switch (g) {
    case 64: RRS_STREAM(1); break;
    case 128: RRS_STREAM(2); break;
    case 256:
      if constexpr (K >= 1024) RRS_STREAM(4);
      else return hipErrorInvalidValue;
      break;
    case 512:
      if constexpr (K >= 2048) RRS_STREAM(8);
      else return hipErrorInvalidValue;
      break;
    default: return hipErrorInvalidValue;
  }
#undef RRS_STREAM
  return hipGetLastError();
}

template <bool kPartials>
hipError_t launch_any(const uint8_t* Xq, const float* a_scale, const float* s_group,
                      const uint8_t* Wq, const float* w_scale, int M, int N, int K, int g,
                      uint16_t* Y, int32_t* P, float out_scale, hipStream_t stream,
                      bool tiled) {
  switch (K) {
#define RRS_K(K_) \
  case K_: return launch_k<K_, kPartials>(Xq, a_scale, s_group, Wq, w_scale, M, N, g, Y, P, \
                                           out_scale, stream, tiled)
    RRS_K(512);
    RRS_K(1024);
    RRS_K(2048);
    RRS_K(4096);
    RRS_K(8192);
    RRS_K(16384);
#undef RRS_K
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool stream_kernel_fits(int M, int K, int g) {
  return M >= 1 && M <= kMaxTokens && K >= 4 * g;
}

hipError_t launch_w4a4_gemm_stream(const uint8_t* Xq, const float* a_scale,
                                   const float* s_group, const uint8_t* Wq,
                                   const float* w_scale, int M, int N, int K, int g,
                                   uint16_t* Y, float out_scale, hipStream_t stream,
                                   WqLayout lay) {
  return launch_any<false>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, nullptr, out_scale,
                           stream, lay.tiled);
}

hipError_t launch_w4a4_gemm_stream_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                            int K, int g, int32_t* P, hipStream_t stream,
                                            WqLayout lay) {
  return launch_any<true>(Xq, nullptr, nullptr, Wq, nullptr, M, N, K, g, nullptr, P, 0.0f,
                          stream, lay.tiled);
}

}  // namespace rrs
