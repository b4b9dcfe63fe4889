// Internal pieces shared by the weight-streaming GEMM kernels
// (rrs_gemm_stream.hip, rrs_gemm_stream_gather.hip): the per-wave LDS ring
// shape, the unpack of packed codes, explicit vector-memory waits and the
// persistent grid size.
#pragma once

#include "rrs_internal.h"

namespace rrs {
namespace stream {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 16;  // weight rows (output columns) per column block
constexpr int kMaxTokens = 16;

// W waves per workgroup, each streaming a 1/W slice of K.
template <int K, int W = kWaves>
struct StreamShape {
  static constexpr int R = K / 2 / W;                 // packed bytes per row per wave
  static constexpr int SBW = R < 512 ? R : 512;        // bytes per row per sub-buffer
  static constexpr int SPB = R / SBW;                  // sub-buffers per block
  static constexpr int CPR = SBW / 16;                 // 16-byte chunks per row per sub-buffer
  static constexpr int SW = CPR >= 8 ? 7 : CPR - 1;   // chunk permutation mask (row-major)
  static constexpr int SB = kRows * SBW;               // LDS bytes per sub-buffer
  static constexpr int NL = SB / 1024;                 // direct loads of 1 KB per sub-buffer
  static constexpr int RS = 16384 / SB;                // sub-buffers in a wave's ring (16 KB)
  static constexpr int RPI = 1024 / SBW;               // rows per direct load (row-major)
  static_assert(SB % 1024 == 0, "a sub-buffer is a whole number of 1 KB loads");
  static_assert(RS >= 2 && (RS - 1) * NL <= 63, "ring depth and vmcnt immediate");
};

// Cache policy of the weight loads: non-temporal (each weight byte is read
// once; 5 % faster at the decode shape than the default policy).
constexpr int kWeightPolicy = 2;

__device__ __forceinline__ v4i unpack_pair(uint32_t w0, uint32_t w1) {
  v4i r;
  r.x = (int)((w0 << 4) & 0xF0F0F0F0u);
  r.y = (int)(w0 & 0xF0F0F0F0u);
  r.z = (int)((w1 << 4) & 0xF0F0F0F0u);
  r.w = (int)(w1 & 0xF0F0F0F0u);
  return r;
}

// Eight packed codes -> eight int8 lanes of 16 q (codes 0, 2, 4, 6 then
// 1, 3, 5, 7: the same order for both operands).
__device__ __forceinline__ long unpack_dword(uint32_t w) {
  const uint32_t lo = (w << 4) & 0xF0F0F0F0u;
  const uint32_t hi = w & 0xF0F0F0F0u;
  return (long)(((unsigned long)hi << 32) | lo);
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Waits until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}


inline int cu_count() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

// A persistent grid must not exceed the workgroups that can be resident at
// once (the surplus would wait for a whole earlier workgroup to finish):
// as many per compute unit as the runtime's occupancy query allows (two for
// most shapes: 72 KB of LDS each; one where a wave needs more than 256
// registers or the workgroup more than 80 KB of LDS), times the compute
// units. Cached per kernel (one instantiation per kernel function).
template <auto Kern>
int resident_grid(int nblk, int threads = kThreads) {
  static int per_cu = 0;
  if (per_cu == 0) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, Kern, threads, 0) != hipSuccess || n < 1)
      n = 1;
    per_cu = n;
  }
  const int cap = per_cu * cu_count();
  return nblk < cap ? nblk : cap;
}

}  // namespace stream
}  // namespace rrs
