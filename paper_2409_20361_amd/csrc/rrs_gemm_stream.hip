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
// its 16 x R bytes through LDS with direct-to-LDS loads
// (global_load_lds_dwordx4): every instruction moves 1 KB of global bytes into
// LDS without passing through registers. The MFMA operand layout wants lane
// (c, q) to hold row c, which a direct load of 1 KB cannot give; LDS turns the
// stream into that layout, read back with one ds_read_b128 per lane per
// 64-byte piece.
//
// The kernel is persistent: two workgroups per compute unit, each taking the
// column blocks blockIdx.x, blockIdx.x + gridDim.x, ... A wave streams its
// quarters of those blocks as a sequence of sub-buffers of 16 rows x 512
// bytes (8 KB; smaller when R is) through a ring of 16 KB of LDS: while it
// multiplies one sub-buffer the next is in flight, and each one it has
// multiplied is refilled at once (at smaller K the ring holds more, smaller
// sub-buffers). Measured at the decode shape (M = 8, K = 8192, back-to-back
// events): 16 rows x 512 bytes in a 16 KB ring with two workgroups per
// compute unit 21.2 us; 16 x 256 bytes, four per ring, 28.3 us; 16 x 256
// bytes, eight per ring, one workgroup per compute unit 29.4 us; 16 x 128
// bytes 38.6 us: the fewer rows one load instruction touches, the faster.
// Direct loads of a sub-buffer: row-major Wq, two rows x 512 contiguous
// bytes per instruction, each row's 16-byte chunks permuted
// by chunk' = chunk ^ (r & 7) in LDS so that the 16 lanes reading the same
// chunk of 16 rows hit different banks (the permutation is applied on the
// global side: lane i of a direct load lands at slot i and fetches the chunk
// that belongs there); tiled Wq, one 1 KB tile per instruction, unchanged,
// where the 16 lanes reading quarter q of the 16 rows read 256 consecutive
// bytes. Both layouts give the same operands in the same order, so their
// results are bit-identical. The direct loads are not tracked by the
// compiler's wait insertion for the LDS reads that follow, so the kernel
// waits for them explicitly: after issuing a refill it lets the loads of the
// newer sub-buffers stay in flight (vmcnt((RS - 1) NL)) and retires the rest.
// The weight loads are non-temporal (read once).
//
// Token codes (M x K/2, a few KB, L2-resident) are loaded into registers once
// per workgroup and reused for every column block: lane (c, q) takes the
// same bytes of token row c (row M - 1 for c >= M, whose outputs are never
// stored). (Loaded per block, as 16 rows x 64 bytes per instruction, they
// cost up to 8 us at 8 to 16 tokens in a first, non-persistent version.) Per group b of the wave, lane (c, q) holds
// bytes [64 h + 16 q, +16) of each 64-byte piece h of the group (g >= 128) or
// bytes [8 q, +8) (g = 64); MFMA k-step s (v_mfma_i32_16x16x64_i8) takes the
// lane's bytes [8 s, 8 s + 8) in that order for both operands, so every k-step
// stays inside one group. Codes are unpacked into the high nibble of each int8
// lane (16 q, the 2^-8 folded into the output scale) and each group's int32
// accumulators start from the bits of 1.5 * 2^23 (g <= 256), so that the
// result read as a float is exactly 1.5 * 2^23 + 256 P_b and one subtraction
// recovers 256 P_b before the FMA by s_b; for g = 512 they start from 0 and
// are converted. The four waves' fp32 sums of a block are added in a fixed
// order, through LDS, after a workgroup barrier; each wave then stores a
// quarter of the block's outputs.
//
// Needs K >= 4 g (every wave holds whole groups): K = 512 with g <= 128,
// K = 1024 with g <= 256, any g from K = 2048 (but g >= 256 at K = 16384).
#include "rrs_stream.h"

namespace rrs {
namespace {

using namespace stream;

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
  constexpr int GB = g / 2;                   // packed bytes of a row per group
  constexpr int NG = S::R / GB;               // groups per wave (its quarter of K)
  constexpr int NGS = S::SBW / GB;            // groups per sub-buffer
  constexpr int NP = GB >= 64 ? GB / 64 : 1;  // 16-byte lane pieces per group
  static_assert(NGS >= 1 && S::SBW % GB == 0, "every sub-buffer holds whole groups");
  __shared__ __attribute__((aligned(16))) uint8_t ring[kWaves * S::RS * S::SB];
  __shared__ __attribute__((aligned(16))) v4f part[2][kWaves][64];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int kq = __builtin_amdgcn_readfirstlane(t >> 6);  // K quarter of this wave
  const int c = lane & 15;
  const int q = lane >> 4;
  constexpr size_t krow = (size_t)K / 2;
  uint8_t* my = ring + kq * S::RS * S::SB;
  const int nblk = N / kRows;
  const int mine = (nblk - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
  const int items = mine * S::SPB;  // sub-buffers this wave streams, in order

  // Direct loads of item i (sub-buffer i % SPB of column block i / SPB) into
  // ring slot i % RS. Row-major: each instruction RPI rows x SBW bytes,
  // chunks permuted; tiled: each instruction one tile (the block's 16 rows are
  // one 16-row block, n0 a multiple of 16).
  auto issue = [&](int i) {
    const int blk = (int)blockIdx.x + (i / S::SPB) * (int)gridDim.x;
    const int sp = i % S::SPB;
    uint8_t* dst = my + (i % S::RS) * S::SB;
    const uint8_t* base = Wq + (size_t)blk * kRows * krow;
    if constexpr (kTiled) {
      const uint8_t* src = base + (size_t)(kq * S::R + sp * S::SBW) * kRows;
#pragma unroll
      for (int ii = 0; ii < S::NL; ++ii)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src + 1024 * ii + 16 * lane),
                                         (lds_ptr_t)(dst + 1024 * ii), 16, 0, kWeightPolicy);
    } else {
      const uint8_t* src = base + kq * S::R + sp * S::SBW;
#pragma unroll
      for (int ii = 0; ii < S::NL; ++ii) {
        const int r = ii * S::RPI + lane / S::CPR;
        const int j = (lane % S::CPR) ^ (r & S::SW);
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src + (size_t)r * krow + 16 * j),
                                         (lds_ptr_t)(dst + 1024 * ii), 16, 0, kWeightPolicy);
      }
    }
  };
  // LDS offset, inside a sub-buffer, of bytes [16 jc + 8 e, +8) of row c
  // (jc: 16-byte chunk index within the sub-buffer's SBW bytes of a row).
  auto woff = [&](int jc, int e) -> int {
    if constexpr (kTiled)
      return (jc >> 2) * 1024 + ((jc & 3) * 16 + c) * 16 + 8 * e;
    else
      return c * S::SBW + 16 * (jc ^ (c & S::SW)) + 8 * e;
  };

  // Fill the ring: the first RS - 1 sub-buffers.
#pragma unroll
  for (int i = 0; i < S::RS - 1; ++i)
    if (i < items) issue(i);

  // Token codes of the wave's quarter (once per workgroup) and its group
  // scales (one per lane).
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

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = GS > 4 ? v4i{0, 0, 0, 0} : v4i{kMagic, kMagic, kMagic, kMagic};

  // Epilogue split: wave kq stores accumulator row kq of every lane, i.e.
  // output row 4 q + kq, so the four waves share the stores.
  const int orow = 4 * q + kq;
  float oscale = 0.0f;  // alpha of that row times out_scale
  if constexpr (!kPartials) oscale = a_scale[min(orow, M - 1)] * out_scale;

  for (int tb = 0; tb < mine; ++tb) {
    const int blk = (int)blockIdx.x + tb * (int)gridDim.x;
    float bcol = 0.0f;  // beta of this lane's column, requested early
    if constexpr (!kPartials) bcol = w_scale[blk * kRows + c];
    float f[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int sp = 0; sp < S::SPB; ++sp) {
      const int i = tb * S::SPB + sp;
      // Refill the slot freed by the previous item, then retire item i: with
      // RS - 1 items issued after it, at most (RS - 1) NL loads may remain.
      if (i + S::RS - 1 < items) {
        issue(i + S::RS - 1);
        wait_vm<(S::RS - 1) * S::NL>();
      } else {
        wait_vm<0>();
      }
      const uint8_t* buf = my + (i % S::RS) * S::SB;
#pragma unroll
      for (int bl = 0; bl < NGS; ++bl) {
        const int b = sp * NGS + bl;  // group of the wave's quarter
        uint32_t ww[NP][4];
#pragma unroll
        for (int h = 0; h < NP; ++h) {
          if constexpr (GB >= 64) {
            const uint4 v = *reinterpret_cast<const uint4*>(buf + woff(bl * (GB / 16) + 4 * h + q, 0));
            ww[h][0] = v.x;
            ww[h][1] = v.y;
            ww[h][2] = v.z;
            ww[h][3] = v.w;
          } else {
            const uint2 v = *reinterpret_cast<const uint2*>(buf + woff(2 * bl + (q >> 1), q & 1));
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
                                                      unpack_pair(ww[h][o], ww[h][o + 1]), acc,
                                                      0, 0, 0);
        }
        if constexpr (kPartials) {
          int32_t* Pg = P + (size_t)(kq * NG + b) * (size_t)M * (size_t)N;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = 4 * q + r;
            if (row < M)
              Pg[(size_t)row * N + blk * kRows + c] = (GS > 4 ? acc[r] : acc[r] - kMagic) >> 8;
          }
        } else {
          const float s =
              __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sv), b));
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
    if constexpr (!kPartials) {
      // The four quarters' sums of this block, added in the order kq = 0..3
      // (part is double-buffered, so one barrier per block suffices).
      part[tb & 1][kq][lane] = v4f{f[0], f[1], f[2], f[3]};
      __syncthreads();
      float sum = part[tb & 1][0][lane][kq];
#pragma unroll
      for (int p = 1; p < kWaves; ++p) sum += part[tb & 1][p][lane][kq];
      // out_scale = 2^-8 (undoes the 16 x 16 of the unpacked operands) / K (the
      // unnormalized rotation; 1 without rotation), an exact power of two.
      if (orow < M)
        Y[(size_t)orow * N + blk * kRows + c] =
            __builtin_bit_cast(uint16_t, (_Float16)((sum * oscale) * bcol));
    }
  }
}

template <int K, bool kPartials>
hipError_t launch_k(const uint8_t* Xq, const float* a_scale, const float* s_group,
                    const uint8_t* Wq, const float* w_scale, int M, int N, int g, uint16_t* Y,
                    int32_t* P, float out_scale, hipStream_t stream, bool tiled) {
  const int nblk = N / kRows;  // N % 16 == 0 (API precondition)
#define RRS_STREAM_T(GS_, T_)                                                             \
  {                                                                                       \
    auto kern = gemm_stream_kernel<K, GS_, T_, kPartials>;                                \
    kern<<<resident_grid(kern, nblk), kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq,    \
                                                             w_scale, M, N, Y, P,         \
                                                             out_scale);                  \
  }
#define RRS_STREAM(GS_)    \
  if (tiled)               \
    RRS_STREAM_T(GS_, true) \
  else                     \
    RRS_STREAM_T(GS_, false)
  switch (g) {
    case 64:
      if constexpr (K <= 8192) {
        RRS_STREAM(1)
      } else {
        return hipErrorInvalidValue;
      }
      break;
    case 128:
      if constexpr (K <= 8192) {
        RRS_STREAM(2)
      } else {
        return hipErrorInvalidValue;
      }
      break;
    case 256:
      if constexpr (K >= 1024) {
        RRS_STREAM(4)
      } else {
        return hipErrorInvalidValue;
      }
      break;
    case 512:
      if constexpr (K >= 2048) {
        RRS_STREAM(8)
      } else {
        return hipErrorInvalidValue;
      }
      break;
    default: return hipErrorInvalidValue;
  }
#undef RRS_STREAM
#undef RRS_STREAM_T
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

// K = 16384 with g <= 128 keeps 32 or 64 groups of token codes per wave,
// which do not fit the registers next to the loop: the few-token kernel takes
// those shapes.
bool stream_kernel_fits(int M, int K, int g) {
  return M >= 1 && M <= kMaxTokens && K >= 4 * g && !(K == 16384 && g <= 128);
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
