// W4A4 GEMM with Runtime Smooth fused into the K loop (Section 3.2, Eq. 3,
// Fig. 4 step (3)):
//   Y[i, n] = fp16( alpha_i * beta_n / K * sum_b s_b * P_b[i, n] )
//   P_b[i, n] = sum_{j in group b} qx[i, j] * qw[j, n]   (exact int32)
//
// Main kernel: 512 threads (8 waves, two per SIMD), output tile 256 x 128,
// each wave 64 x 64 as 2 x 2 blocks of v_mfma_i32_32x32x32_i8. K advances in
// tiles of 128 (four MFMA k-steps of 32).
//
// Data path: packed INT4 (Xq: M x K/2, K contiguous; Wq row-major or tiled,
// see WqLayout: in the tiled layout one wave's slot of a K tile, 16 rows x 64
// bytes, is one contiguous 1 KB tile) is loaded from HBM into registers two
// tiles ahead, unpacked to int8 and stored in a
// double-buffered LDS stage whose rows are padded to 144 bytes (conflict-free
// 128-bit fragment reads at immediate offsets). The unpack and the LDS stores
// of the next tile are spread over the MFMAs of the current tile's H0 phase
// (below), so the matrix core is not idle while they run. A nibble is unpacked into the
// high half of its int8 lane (the byte holds 16 q): low nibbles are
// (w << 4) & 0xF0F0F0F0, high nibbles w & 0xF0F0F0F0, three VALU ops per
// eight codes. Products are 256 q w, exact in int32 for every group size here;
// the 2^-8 is folded into the output scale. The unpack permutes K inside each
// 16-element chunk identically for both operands, so every dot product is
// unchanged.
//
// Runtime Smooth: each group of g channels gets fresh int32 accumulators; at
// the end of the group they are converted and added into fp32 accumulators
// with one FMA by s_b. For g <= 256 the conversion is free of v_cvt_f32_i32
// (a slow instruction): the group's first MFMA starts from C = bits of
// 1.5 * 2^23 instead of 0, so the int32 result 0x4B400000 + 256 P is, read
// as a float, exactly 1.5 * 2^23 + 256 P (|256 P| <= 256 * 49 * 256 < 2^22
// keeps it in the binade whose ulp is 1), and one exact subtraction recovers
// 256 P. For g = 512 the accumulators start from 0 and are converted. That rescale costs as
// much VALU time as the group's MFMAs cost matrix time, so it must run in
// their shadow. Each wave splits its tile into two row halves (H0: rows 0-31,
// H1: rows 32-63) that take turns over every chunk of k-steps: while H0 runs
// its MFMAs, the VALU rescales H1's finished group, and the other way round.
// Only one set of int32 accumulators is live at a time (64 registers), and
// the B fragments of a chunk are read once and used by both halves.
//
// Workgroups are mapped to tiles XCD by XCD: the hardware deals workgroup ids
// round-robin to the 8 XCDs, so each XCD is given a contiguous run of tiles,
// ordered in column strips of 4 row tiles to share A and B in its L2.
#include <type_traits>

#include "rrs_internal.h"

namespace rrs {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kThreads = 512;
constexpr int BM = 256;
constexpr int BN = 128;
constexpr int BK = 128;                 // INT4 elements of K per tile
constexpr int ROWP = BK + 16;           // LDS bytes per row: 128 int8 + 16 pad
constexpr int A_BYTES = BM * ROWP;      // 36864
constexpr int B_BYTES = BN * ROWP;      // 18432
constexpr int STAGE = A_BYTES + B_BYTES;
constexpr int kGroupM = 4;              // row tiles per column strip

__device__ __forceinline__ uint4 unpack_pair(uint32_t w0, uint32_t w1) {
  return make_uint4((w0 << 4) & 0xF0F0F0F0u, w0 & 0xF0F0F0F0u, (w1 << 4) & 0xF0F0F0F0u,
                    w1 & 0xF0F0F0F0u);
}

__device__ __forceinline__ uint16_t float_to_half_bits(float x) {
  return __builtin_bit_cast(uint16_t, (_Float16)x);
}

struct TileMap {
  int m0, n0;
  bool valid;
};

// XCD-aware tile order (see the file comment).
__device__ __forceinline__ TileMap map_tile(int M, int N) {
  const int tm = (M + BM - 1) / BM;
  const int tn = (N + BN - 1) / BN;
  const int T = tm * tn;
  const int w = blockIdx.x;
  const int per = (T + 7) >> 3;
  const int lin = (w & 7) * per + (w >> 3);
  TileMap r;
  r.valid = lin < T;
  const int strip = kGroupM * tn;
  const int first_m = (lin / strip) * kGroupM;
  const int gm = min(tm - first_m, kGroupM);
  const int rem = lin % strip;
  r.m0 = (first_m + rem % gm) * BM;
  r.n0 = (rem / gm) * BN;
  return r;
}

// Row / column of accumulator register r of block (h, j) for this lane.
__device__ __forceinline__ int acc_row(int m0, int wm, int h, int r, int lane) {
  return m0 + wm * 64 + h * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
__device__ __forceinline__ int acc_col(int n0, int wn, int j, int lane) {
  return n0 + wn * 64 + j * 32 + (lane & 31);
}

// GS = g / 32 MFMA k-steps per smoothing group. kPerChannel: the per-channel
// A4W4 baseline of the paper's kernel comparison (Section 4.5) on this same
// main loop: no smoothing, so no per-group rescale; the int32 accumulators run
// over all of K (|256 P| <= 256 * 49 * 16384 < 2^31) and are converted once.
// kGather (runtime channel reorder): position block p (32 channels, 16 bytes
// of a packed row) of Xq pairs with block border[p] of every Wq row; the
// table is kept in LDS and each B slot reads its entry one tile ahead.
template <int GS, bool kPartials, bool kPerChannel, bool kGather, bool kTiled>
__global__ __launch_bounds__(kThreads, 1) void gemm_main_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, int M, int N, int K, uint16_t* __restrict__ Y,
    int32_t* __restrict__ P, float out_scale, const int32_t* __restrict__ border) {
  constexpr WqLayout lay{kTiled};
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * STAGE];
  __shared__ float scale_tab[BM + BN];  // alpha of the tile's rows, then beta of its columns
  __shared__ int btab[kGather ? 16384 / kReorderBlock : 1];

  const TileMap tile = map_tile(M, N);
  if (!tile.valid) return;
  const int m0 = tile.m0;
  const int n0 = tile.n0;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int wm = wave & 3;   // 64-row slice of the 256-row tile
  const int wn = wave >> 2;  // 64-column slice of the 128-column tile
  const size_t krow = (size_t)K / 2;

  // Global -> LDS slots. A: row t/2, 32 packed bytes; B: row t/4, 16 bytes.
  // Rows past M (or N) load the last valid row instead: their results are
  // never stored, and the loop stays free of divergent branches.
  const int arow = t >> 1;
  const int ahalf = t & 1;
  const int brow = t >> 2;
  const int bq = t & 3;
  const uint8_t* ga = Xq + (size_t)min(m0 + arow, M - 1) * krow + ahalf * 32;
  const int bn = min(n0 + brow, N - 1);
  constexpr uint32_t wts = (uint32_t)lay.tile();     // bytes from one K tile to the next
  constexpr uint32_t wqs = (uint32_t)lay.quarter();  // bytes from one 16-byte piece to the next
  const uint8_t* gb = Wq + lay.row(bn, K) + (kGather ? 0u : bq * wqs);
  const int a_st = arow * ROWP + ahalf * 64;
  const int b_st = A_BYTES + brow * ROWP + bq * 32;

  // Fragment read offsets (per lane) inside a stage.
  const int frow = lane & 31;
  const int fk = (lane >> 5) * 16;
  const int a_fr = (wm * 64 + frow) * ROWP + fk;       // H0; H1 is + 32 rows
  const int b_fr = A_BYTES + (wn * 64 + frow) * ROWP + fk;  // B0; B1 is + 32 rows

  // Packed tiles in flight: two register sets, tile kt lives in set kt & 1.
  uint4 ra0[2], ra1[2], rb0[2];
  // Byte offset from gb of this thread's B slot of tile kt: piece 4 kt + bq of
  // its row, or piece btab[4 kt + bq] with the runtime reorder.
  auto boff = [&](int kt) -> uint32_t {
    if constexpr (kGather) {
      const uint32_t p = (uint32_t)btab[kt * 4 + bq];
      return (p >> 2) * wts + (p & 3u) * wqs;
    } else {
      return (uint32_t)kt * wts;
    }
  };
  auto gload = [&](int set, int kt, uint32_t bo) {
    const uint4* p = reinterpret_cast<const uint4*>(ga + (size_t)kt * (BK / 2));
    ra0[set] = p[0];
    ra1[set] = p[1];
    rb0[set] = *reinterpret_cast<const uint4*>(gb + bo);
  };
  auto lstore = [&](int set, int stage) {
    uint8_t* s = lds + stage * STAGE;
    *reinterpret_cast<uint4*>(s + a_st) = unpack_pair(ra0[set].x, ra0[set].y);
    *reinterpret_cast<uint4*>(s + a_st + 16) = unpack_pair(ra0[set].z, ra0[set].w);
    *reinterpret_cast<uint4*>(s + a_st + 32) = unpack_pair(ra1[set].x, ra1[set].y);
    *reinterpret_cast<uint4*>(s + a_st + 48) = unpack_pair(ra1[set].z, ra1[set].w);
    *reinterpret_cast<uint4*>(s + b_st) = unpack_pair(rb0[set].x, rb0[set].y);
    *reinterpret_cast<uint4*>(s + b_st + 16) = unpack_pair(rb0[set].z, rb0[set].w);
  };
  // One sixth of lstore: piece i of this thread's six 16-byte LDS stores.
  auto lpiece = [&](int set, int stage, int i) {
    uint8_t* s = lds + stage * STAGE;
    if (i == 0) *reinterpret_cast<uint4*>(s + a_st) = unpack_pair(ra0[set].x, ra0[set].y);
    if (i == 1) *reinterpret_cast<uint4*>(s + a_st + 16) = unpack_pair(ra0[set].z, ra0[set].w);
    if (i == 2) *reinterpret_cast<uint4*>(s + b_st) = unpack_pair(rb0[set].x, rb0[set].y);
    if (i == 3) *reinterpret_cast<uint4*>(s + a_st + 32) = unpack_pair(ra1[set].x, ra1[set].y);
    if (i == 4) *reinterpret_cast<uint4*>(s + a_st + 48) = unpack_pair(ra1[set].z, ra1[set].w);
    if (i == 5) *reinterpret_cast<uint4*>(s + b_st + 16) = unpack_pair(rb0[set].z, rb0[set].w);
  };
  auto afrag = [&](int stage, int h, int ks) -> v4i {
    return *reinterpret_cast<const v4i*>(lds + stage * STAGE + a_fr + h * 32 * ROWP + ks * 32);
  };
  auto bfrag = [&](int stage, int j, int ks) -> v4i {
    return *reinterpret_cast<const v4i*>(lds + stage * STAGE + b_fr + j * 32 * ROWP + ks * 32);
  };

  // acc[h][j]: int32 accumulators of block (h, j); f[h][j][r]: fp32 results.
  v16i acc[2][2];
  float f[2][2][16];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        acc[h][j][r] = (kPerChannel || GS > 8) ? 0 : 0x4B400000;
        f[h][j][r] = 0.0f;
      }

  const int nsteps = K / 32;
  const int ntiles = K / BK;
  const v16i zero = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23 (= 12582912.0f)
  const v16i magic = {kMagic, kMagic, kMagic, kMagic, kMagic, kMagic, kMagic, kMagic,
                      kMagic, kMagic, kMagic, kMagic, kMagic, kMagic, kMagic, kMagic};

  constexpr int PH = GS < 4 ? GS : 4;            // k-steps per chunk
  constexpr int U = GS > 8 ? GS : 8;             // k-steps per unrolled loop trip
  constexpr int CONV = 32 / PH;                  // rescale elements per k-step

  // Rescale one slice of half h's accumulators: elements [q0, q0 + CONV) of 32.
  auto rescale = [&](int h, int q0, float s, int grp) {
    if constexpr (kPerChannel) {
      return;
    } else if constexpr (!kPartials) {
#pragma unroll
      for (int q = 0; q < CONV; ++q) {
        const int e = q0 + q;
        // Bit-cast the whole vector, then index: bit-casting a single element
        // of an ext_vector is miscompiled (every element reads element 0).
        const v16f accf = __builtin_bit_cast(v16f, acc[h][e >> 4]);
        const float pv = GS > 8 ? (float)acc[h][e >> 4][e & 15] : accf[e & 15] - 12582912.0f;
        f[h][e >> 4][e & 15] = __builtin_fmaf(s, pv, f[h][e >> 4][e & 15]);
        // Pin the update here: otherwise the compiler sinks all rescales of a
        // loop trip to its end, where they force copies of the accumulators.
        asm volatile("" : "+v"(f[h][e >> 4][e & 15]));
      }
    } else {
      int32_t* Pg = P + (size_t)grp * (size_t)M * (size_t)N;
#pragma unroll
      for (int q = 0; q < CONV; ++q) {
        const int e = q0 + q;
        const int row = acc_row(m0, wm, h, e & 15, lane);
        const int col = acc_col(n0, wn, e >> 4, lane);
        // The production seed: the accumulator holds 0x4B400000 + 256 P (g <= 256)
        // or 256 P (g = 512); the hook undoes exactly that encoding.
        const int32_t v = acc[h][e >> 4][e & 15];
        if (row < M && col < N) Pg[(size_t)row * N + col] = (GS > 8 ? v : v - kMagic) >> 8;
      }
    }
  };

  // Prologue: the tile's output scales into LDS (read only by the epilogue,
  // after many barriers); tile 0 staged, tiles 1 and 2 in flight, fragments
  // of chunk 0 read.
  if constexpr (!kPartials) {
    if (t < BM)
      scale_tab[t] = a_scale[min(m0 + t, M - 1)];
    else if (t < BM + BN)
      scale_tab[t] = w_scale[min(n0 + t - BM, N - 1)];
  }
  if constexpr (kGather) {
    // Entries are masked into range, so any table keeps every load in bounds.
    for (int i = t; i < K / kReorderBlock; i += kThreads)
      btab[i] = border[i] & (K / kReorderBlock - 1);
    __syncthreads();
  }
  gload(0, 0, boff(0));
  lstore(0, 0);
  gload(1, min(1, ntiles - 1), boff(min(1, ntiles - 1)));
  gload(0, min(2, ntiles - 1), boff(min(2, ntiles - 1)));
  __syncthreads();
  v4i fb[PH][2], fa0[PH], fa1[PH];
  uint32_t bnext = 0;  // gather only
#pragma unroll
  for (int s = 0; s < PH; ++s) {
    fb[s][0] = bfrag(0, 0, s);
    fb[s][1] = bfrag(0, 1, s);
    fa0[s] = afrag(0, 0, s);
  }

  for (int base = 0; base < nsteps; base += U) {
#pragma unroll
    for (int c0 = 0; c0 < U; c0 += PH) {  // one chunk of PH k-steps
      const int stage = (c0 >> 2) & 1;
      const int ks0 = c0 & 3;
      const int j0 = base + c0;             // first global k-step of the chunk
      const int grp = j0 / GS;
      const bool g_first = (c0 % GS) == 0;  // chunk opens a group (H1 closed one)
      const bool g_last = ((c0 + PH) % GS) == 0;  // chunk closes a group
      const bool tile_end = ks0 + PH == 4;
      float s_cur = 0.0f, s_prev = 0.0f;
      if constexpr (!kPartials && !kPerChannel) {
        if (g_last) s_cur = s_group[grp];
        if (g_first) s_prev = grp > 0 ? s_group[grp - 1] : 0.0f;
      }
      __builtin_amdgcn_sched_barrier(0);

      // Phase H0: MFMAs of rows 0-31; A fragments of rows 32-63 are read;
      // rescale of H1's group closed by the previous chunk (for the very
      // first chunk acc[1] and s_prev are 0); in a tile's last chunk, the
      // next tile is unpacked into the other LDS stage.
#pragma unroll
      for (int s = 0; s < PH; ++s) {
        const bool fresh = !kPerChannel && g_first && s == 0;
        acc[0][0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa0[s], fb[s][0], fresh ? (GS > 8 ? zero : magic) : acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa0[s], fb[s][1], fresh ? (GS > 8 ? zero : magic) : acc[0][1], 0, 0, 0);
        fa1[s] = afrag(stage, 1, ks0 + s);
        if (g_first) {
          if (!kPartials || grp > 0) rescale(1, s * CONV, s_prev, grp - 1);
        }
        if (tile_end) {
          const int kt = j0 >> 2;
#pragma unroll
          for (int i = s * 6 / PH; i < (s + 1) * 6 / PH; ++i) lpiece((kt + 1) & 1, stage ^ 1, i);
          // Gather: the B offset of the tile fetched after the barrier below,
          // read here so that the barrier's wait covers the LDS read.
          if (s == PH - 1) bnext = boff(min(kt + 3, ntiles - 1));
        }
        __builtin_amdgcn_sched_barrier(0);
      }

      // End of a tile: every wave has read this tile's fragments and staged
      // its pieces of the next tile (in the other stage) during phase H0;
      // after the barrier the tile after next is fetched. (On the last tile
      // this stages a duplicate that is never read.)
      if (tile_end) {
        const int kt = j0 >> 2;
        const int kn = min(kt + 3, ntiles - 1);
        __syncthreads();
        gload((kt + 1) & 1, kn, kGather ? bnext : boff(kn));
      }
      const int nstage = tile_end ? stage ^ 1 : stage;
      const int nks0 = (ks0 + PH) & 3;
      __builtin_amdgcn_sched_barrier(0);

      // Phase H1: MFMAs of rows 32-63; the next chunk's B and A0 fragments
      // are read into the registers each k-step frees; rescale of H0's group
      // if this chunk closed it.
#pragma unroll
      for (int s = 0; s < PH; ++s) {
        const bool fresh = !kPerChannel && g_first && s == 0;
        acc[1][0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa1[s], fb[s][0], fresh ? (GS > 8 ? zero : magic) : acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa1[s], fb[s][1], fresh ? (GS > 8 ? zero : magic) : acc[1][1], 0, 0, 0);
        fb[s][0] = bfrag(nstage, 0, nks0 + s);
        fb[s][1] = bfrag(nstage, 1, nks0 + s);
        fa0[s] = afrag(nstage, 0, nks0 + s);
        if (g_last) rescale(0, s * CONV, s_cur, grp);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  if constexpr (kPerChannel) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) f[h][j][r] = (float)acc[h][j][r];
  } else {  // H1's last group.
    const int G = nsteps / GS;
    const float s_last = kPartials ? 0.0f : s_group[G - 1];
#pragma unroll
    for (int s = 0; s < 32; s += CONV) rescale(1, s, s_last, G - 1);
  }

  if constexpr (!kPartials) {
    // out_scale = 2^-8 (undoes the 16 x 16 of the unpacked operands) / K (the
    // unnormalized rotation; 1 without rotation), an exact power of two.
    const float inv = out_scale;
    // Scales come from LDS, so no store waits on a global load: this lane's
    // 32 rows are eight runs of 4 consecutive ones (128-bit reads). A tile
    // that lies wholly inside Y stores without per-element bounds checks.
    float4 arow4[2][4];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        arow4[h][q] = *reinterpret_cast<const float4*>(
            &scale_tab[acc_row(0, wm, h, 4 * q, lane)]);
    float bcol2[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) bcol2[j] = scale_tab[BM + acc_col(0, wn, j, lane)];
    auto store = [&](auto full) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = acc_col(n0, wn, j, lane);
        const float bcol = bcol2[j];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = acc_row(m0, wm, h, r, lane);
            const float4 a4 = arow4[h][r >> 2];
            const float ar = (r & 3) == 0 ? a4.x : (r & 3) == 1 ? a4.y : (r & 3) == 2 ? a4.z : a4.w;
            const float sc = ar * inv;
            const uint16_t v = float_to_half_bits((f[h][j][r] * sc) * bcol);
            if (decltype(full)::value || (row < M && col < N)) Y[(size_t)row * N + col] = v;
          }
      }
    };
    if (m0 + BM <= M && n0 + BN <= N)
      store(std::true_type{});
    else
      store(std::false_type{});
  }
}

template <bool kPartials, bool kGather = false>
hipError_t launch_main(const uint8_t* Xq, const float* a_scale, const float* s_group,
                       const uint8_t* Wq, const float* w_scale, int M, int N, int K, int g,
                       uint16_t* Y, int32_t* P, float out_scale, hipStream_t stream,
                       const int32_t* border, WqLayout lay) {
  const int tm = (M + BM - 1) / BM;
  const int tn = (N + BN - 1) / BN;
  const int T = tm * tn;
  const int grid = 8 * ((T + 7) / 8);
  switch (g) {
#define RRS_LAUNCH(G_, T_)                                                                 \
  gemm_main_kernel<G_ / 32, kPartials, false, kGather, T_><<<grid, kThreads, 0, stream>>>( \
      Xq, a_scale, s_group, Wq, w_scale, M, N, K, Y, P, out_scale, border)
#define RRS_CASE(G_)          \
  case G_:                    \
    if (lay.tiled)            \
      RRS_LAUNCH(G_, true);   \
    else                      \
      RRS_LAUNCH(G_, false);  \
    break;
    RRS_CASE(64)
    RRS_CASE(128)
    RRS_CASE(256)
    RRS_CASE(512)
#undef RRS_CASE
#undef RRS_LAUNCH
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// The main kernel unrolls max(8, g / 32) k-steps per loop trip.
bool main_kernel_fits(int K, int g) {
  const int U = (g / 32 > 8) ? g / 32 : 8;
  return (K / 32) % U == 0;
}

}  // namespace

hipError_t launch_w4a4_gemm(const uint8_t* Xq, const float* a_scale, const float* s_group,
                            const uint8_t* Wq, const float* w_scale, int M, int N, int K,
                            int g, uint16_t* Y, float out_scale, hipStream_t stream,
                            WqLayout lay) {
  if (stream_kernel_fits(M, K, g))
    return launch_w4a4_gemm_stream(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, out_scale,
                                   stream, lay);
  if (decode_kernel_fits(M))
    return launch_w4a4_gemm_decode(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, out_scale,
                                   stream, nullptr, lay);
  if (!main_kernel_fits(K, g))
    return launch_w4a4_gemm_small(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, out_scale,
                                  stream, lay);
  return launch_main<false>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, nullptr,
                            out_scale, stream, nullptr, lay);
}

hipError_t launch_w4a4_gemm_per_channel(const uint8_t* Xq, const float* a_scale,
                                       const uint8_t* Wq, const float* w_scale, int M, int N,
                                       int K, uint16_t* Y, float out_scale, hipStream_t stream,
                                       WqLayout lay) {
  if (!main_kernel_fits(K, 128))
    return launch_w4a4_gemm_scheme(1, Xq, a_scale, nullptr, Wq, w_scale, M, N, K, K, Y,
                                   out_scale, stream, lay);
  const int tm = (M + BM - 1) / BM;
  const int tn = (N + BN - 1) / BN;
  const int grid = 8 * ((tm * tn + 7) / 8);
  if (lay.tiled)
    gemm_main_kernel<4, false, true, false, true><<<grid, kThreads, 0, stream>>>(
        Xq, a_scale, nullptr, Wq, w_scale, M, N, K, Y, nullptr, out_scale, nullptr);
  else
    gemm_main_kernel<4, false, true, false, false><<<grid, kThreads, 0, stream>>>(
        Xq, a_scale, nullptr, Wq, w_scale, M, N, K, Y, nullptr, out_scale, nullptr);
  return hipGetLastError();
}

hipError_t launch_w4a4_gemm_reorder(const uint8_t* Xq, const float* a_scale,
                                    const float* s_group, const uint8_t* Wq,
                                    const float* w_scale, const int32_t* border, int M, int N,
                                    int K, int g, uint16_t* Y, float out_scale,
                                    hipStream_t stream, WqLayout lay) {
  if (stream_gather_fits(M, K))
    return launch_w4a4_gemm_stream_gather(Xq, a_scale, s_group, Wq, w_scale, border, M, N, K, g,
                                          Y, out_scale, stream, lay);
  if (decode_gather_fits(M))
    return launch_w4a4_gemm_decode(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, out_scale,
                                   stream, border, lay);
  // Every shape the ABI accepts fits the main kernel (K / 32 >= 16 is a power
  // of two); the fallback kernel has no gather.
  if (!main_kernel_fits(K, g)) return hipErrorInvalidValue;
  return launch_main<false, true>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, nullptr,
                                  out_scale, stream, border, lay);
}

hipError_t launch_w4a4_gemm_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                     int K, int g, int32_t* P, hipStream_t stream,
                                     WqLayout lay) {
  // The kernel rrs_w4a4_gemm would take for this shape (row-major Wq).
  if (stream_kernel_fits(M, K, g))
    return launch_w4a4_gemm_stream_partials(Xq, Wq, M, N, K, g, P, stream, lay);
  if (decode_kernel_fits(M) && !lay.tiled)
    return launch_w4a4_gemm_decode_partials(Xq, Wq, M, N, K, g, P, stream);
  if (!main_kernel_fits(K, g))
    return launch_w4a4_gemm_partials_small(Xq, Wq, M, N, K, g, P, stream, lay);
  return launch_main<true>(Xq, nullptr, nullptr, Wq, nullptr, M, N, K, g, nullptr, P, 0.0f,
                           stream, nullptr, lay);
}

}  // namespace rrs
