// W4A4 GEMM with Runtime Smooth and the runtime reorder for up to 16 tokens
// (Section 3.2, Eq. 3, Fig. 4 steps (1) and (3)), on the weight stream of
// rrs_gemm_stream.hip.
//
// Built with -mllvm -amdgpu-mfma-vgpr-form (this file only): the magic-seeded
// accumulator of every block then stays in VGPRs, where the rescale reads it;
// in the accumulation registers every block cost four extra copies.
#include "rrs_stream.h"

namespace rrs {
namespace {

using namespace stream;

// Runtime reorder (Fig. 4 step (1) taken at run time): position block p of Xq
// (channels [32 p, 32 p + 32)) pairs with natural weight block border[p]. The
// weights stream in natural order exactly as in gemm_stream_kernel; for
// natural block B the token codes come from position block inv[B], and the
// block's partial is rescaled by the scale of the group that position falls
// in. A block's channels therefore have to stay in one accumulator of their
// own: each block is one v_mfma_i32_16x16x32_i8 (lane group q holds codes
// 8 q .. 8 q + 7 of the block after the unpack, the same for both operands)
// from the magic seed, and its partial enters the fp32 sum by the exact
// two-op rescale (|256 P_B| <= 256 * 49 * 32 < 2^22). The fp32 sum runs over
// the K/32 block terms in natural block order within each wave's quarter.
// Token codes (one dword per lane and block, gathered once per workgroup) and
// the per-block scales (lane b of a wave holds block b's) stay in registers.
template <int K, bool kTiled>
__global__ __launch_bounds__(kThreads) void gemm_stream_gather_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, const int32_t* __restrict__ border, int M, int N,
    int g, uint16_t* __restrict__ Y, float out_scale) {
  using S = StreamShape<K>;
  constexpr int NB = K / kReorderBlock;  // blocks of a row
  constexpr int NBW = NB / kWaves;       // blocks of a wave's quarter
  constexpr int BPS = S::SBW / 16;       // blocks per sub-buffer
  constexpr int RPW = S::SB / (K / 2);   // token rows staged per wave
  constexpr int RPR = kWaves * RPW;      // token rows staged per round
  static_assert(RPW >= 1 && S::SB % (K / 2) == 0, "whole token rows per sub-buffer");
  static_assert(NB % 16 == 0, "the chunk swizzle stays inside a row");
  static_assert(NBW <= 64 && S::R % 16 == 0, "one lane per block of the quarter");
  static_assert(BPS % 4 == 0, "blocks of a sub-buffer in fours");
  __shared__ __attribute__((aligned(16))) uint8_t ring[kWaves * S::RS * S::SB];
  __shared__ __attribute__((aligned(16))) v4f part[2][kWaves][64];
  __shared__ int inv[NB];     // natural block -> position block
  __shared__ float sbl[NB];   // natural block -> scale of its position's group

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int kq = __builtin_amdgcn_readfirstlane(t >> 6);  // K quarter of this wave
  const int c = lane & 15;
  const int q = lane >> 4;
  constexpr size_t krow = (size_t)K / 2;
  uint8_t* my = ring + kq * S::RS * S::SB;
  uint8_t* stage = ring + (S::RS - 1) * S::SB;  // + w RS SB: wave w's staged rows
  const int nblk = N / kRows;
  const int mine = (nblk - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
  const int items = mine * S::SPB;

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
  // LDS offset, inside a sub-buffer, of dword q of 16-byte chunk jc of row c.
  auto woff = [&](int jc) -> int {
    if constexpr (kTiled)
      return (jc >> 2) * 1024 + ((jc & 3) * 16 + c) * 16 + 4 * q;
    else
      return c * S::SBW + 16 * (jc ^ (c & S::SW)) + 4 * q;
  };

  // Copy of token rows r0 + w RPW .. r0 + w RPW + RPW - 1 (those below M) into
  // the last sub-buffer of wave w's ring, by wave w. Position block j of row r
  // lands in 16-byte chunk j ^ (r & 15) of the row's copy, so that the 16 token
  // rows of one block fall in different LDS banks when gathered.
  auto stage_rows = [&](int r0) {
#pragma unroll
    for (int ii = 0; ii < S::NL; ++ii) {
      const int off = 1024 * ii + 16 * lane;  // byte of this wave's rows
      const int r = r0 + kq * RPW + off / (int)krow;
      const int j = ((off % (int)krow) >> 4) ^ (r & 15);
      if (r < M)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(Xq + (size_t)r * krow + 16 * j),
                                         (lds_ptr_t)(stage + kq * S::RS * S::SB + 1024 * ii),
                                         16, 0, 0);
    }
  };
  stage_rows(0);
#pragma unroll
  for (int i = 0; i < S::RS - 1; ++i)
    if (i < items) issue(i);

  // Tables. Entries are reduced modulo K/32, so any table keeps every load in
  // bounds; a table that is not a permutation leaves some blocks at scale 0.
  for (int i = t; i < NB; i += kThreads) {
    inv[i] = 0;
    sbl[i] = 0.0f;
  }
  __syncthreads();
  for (int p = t; p < NB; p += kThreads) {
    const int B = border[p] & (NB - 1);
    inv[B] = p;
    sbl[B] = s_group[p / (g / kReorderBlock)];
  }
  __syncthreads();

  // Token row c (row M - 1 for c >= M, never stored): dword q of the position
  // block of every natural block of this wave's quarter. The rows are copied
  // whole into LDS first, into the last sub-buffer of every wave's ring (the
  // prefetch above leaves it empty), RPW rows per wave and RPR per round;
  // gathered straight from global memory, one load touched a cache line per
  // token row and block, 16 times the lines of the whole copy.
  const int rc = min(c, M - 1);
  uint32_t aw[NBW];
  for (int r0 = 0; r0 < M; r0 += RPR) {
    if (r0 > 0) {
      __syncthreads();  // the previous round's rows have been read
      stage_rows(r0);
    }
    if (r0 == 0 && items >= S::RS - 1)
      wait_vm<(S::RS - 1) * S::NL>();  // the copy, issued before the prefetch
    else
      wait_vm<0>();
    __syncthreads();
    if (rc >= r0 && rc < r0 + RPR) {
      const uint8_t* arow = stage + ((rc - r0) / RPW) * S::RS * S::SB +
                            ((rc - r0) % RPW) * krow + 4 * q;
#pragma unroll
      for (int b = 0; b < NBW; ++b)
        aw[b] = *reinterpret_cast<const uint32_t*>(arow + 16 * (inv[kq * NBW + b] ^ (rc & 15)));
    }
  }
  __syncthreads();  // the ring's last sub-buffers are free again
  const float sv = sbl[kq * NBW + (lane < NBW ? lane : 0)];

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = {kMagic, kMagic, kMagic, kMagic};
  const int orow = 4 * q + kq;
  const float oscale = a_scale[min(orow, M - 1)] * out_scale;

  for (int tb = 0; tb < mine; ++tb) {
    const int blk = (int)blockIdx.x + tb * (int)gridDim.x;
    const float bcol = w_scale[blk * kRows + c];
    float f[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int sp = 0; sp < S::SPB; ++sp) {
      const int i = tb * S::SPB + sp;
      if (i + S::RS - 1 < items) {
        issue(i + S::RS - 1);
        wait_vm<(S::RS - 1) * S::NL>();
      } else {
        wait_vm<0>();
      }
      const uint8_t* buf = my + (i % S::RS) * S::SB;
      // Four blocks at a time: their weight words are read together and their
      // four products issued back to back, so the LDS latency and the MFMA
      // latency are paid once per four blocks; the rescales then follow in
      // natural block order (the fp32 sum's order is unchanged).
#pragma unroll
      for (int bl = 0; bl < BPS; bl += 4) {
        uint32_t w[4];
        v4i acc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) w[u] = *reinterpret_cast<const uint32_t*>(buf + woff(bl + u));
#pragma unroll
        for (int u = 0; u < 4; ++u)
          acc[u] = __builtin_amdgcn_mfma_i32_16x16x32_i8(unpack_dword(aw[sp * BPS + bl + u]),
                                                         unpack_dword(w[u]), seed, 0, 0, 0);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int b = sp * BPS + bl + u;  // natural block of the wave's quarter
          const float s = __builtin_bit_cast(
              float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sv), b));
          const v4f accf = __builtin_bit_cast(v4f, acc[u]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            f[r] = __builtin_fmaf(s, accf[r] - 12582912.0f, f[r]);
            // Pin the update here: otherwise every block's rescale sinks to
            // the end of the column block and all 64 accumulators stay live.
            asm volatile("" : "+v"(f[r]));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    part[tb & 1][kq][lane] = v4f{f[0], f[1], f[2], f[3]};
    __syncthreads();
    float sum = part[tb & 1][0][lane][kq];
#pragma unroll
    for (int p = 1; p < kWaves; ++p) sum += part[tb & 1][p][lane][kq];
    if (orow < M)
      Y[(size_t)orow * N + blk * kRows + c] =
          __builtin_bit_cast(uint16_t, (_Float16)((sum * oscale) * bcol));
  }
}

template <int K>
hipError_t launch_gather_k(const uint8_t* Xq, const float* a_scale, const float* s_group,
                           const uint8_t* Wq, const float* w_scale, const int32_t* border,
                           int M, int N, int g, uint16_t* Y, float out_scale,
                           hipStream_t stream, bool tiled) {
  const int nblk = N / kRows;
  if (tiled) {
    constexpr auto kern = gemm_stream_gather_kernel<K, true>;
    kern<<<resident_grid<kern>(nblk), kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale,
                                                             border, M, N, g, Y, out_scale);
  } else {
    constexpr auto kern = gemm_stream_gather_kernel<K, false>;
    kern<<<resident_grid<kern>(nblk), kThreads, 0, stream>>>(Xq, a_scale, s_group, Wq, w_scale,
                                                             border, M, N, g, Y, out_scale);
  }
  return hipGetLastError();
}

}  // namespace

bool stream_gather_fits(int M, int K) { return M >= 1 && M <= kMaxTokens && K <= 8192; }

hipError_t launch_w4a4_gemm_stream_gather(const uint8_t* Xq, const float* a_scale,
                                          const float* s_group, const uint8_t* Wq,
                                          const float* w_scale, const int32_t* border, int M,
                                          int N, int K, int g, uint16_t* Y, float out_scale,
                                          hipStream_t stream, WqLayout lay) {
  switch (K) {
#define RRS_GK(K_) \
  case K_: return launch_gather_k<K_>(Xq, a_scale, s_group, Wq, w_scale, border, M, N, g, Y, \
                                      out_scale, stream, lay.tiled)
    RRS_GK(512);
    RRS_GK(1024);
    RRS_GK(2048);
    RRS_GK(4096);
    RRS_GK(8192);
#undef RRS_GK
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rrs
