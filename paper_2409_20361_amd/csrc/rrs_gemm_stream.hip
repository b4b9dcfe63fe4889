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
//
// 17 to 32 tokens at K = 8192: the same loop with eight waves, each streaming
// an eighth of K (16 rows x 512 bytes per block, the same 16 KB ring per wave)
// and holding the codes of two blocks of 16 tokens (64 registers per block,
// half of what a quarter of K would take), one workgroup of 512 threads per
// compute unit (128 KB of ring and 32 KB of partial sums), each workgroup
// streaming one contiguous range of column blocks. Every weight fragment is
// unpacked once for both token blocks; the 2 x 4 (token block, accumulator
// row) pairs of each lane are dealt to the eight waves for the fixed-order sum
// and the stores.
#include "rrs_device.h"
#include "rrs_stream.h"

namespace rrs {
namespace {

using namespace stream;

// W waves per workgroup, each streaming a 1/W slice of K; TB blocks of 16
// tokens (tokens 16 u .. 16 u + 15 in block u), all multiplied with the same
// weight operands. kPartials (test hook): instead of Y, write P[b][i][n] for
// every group b, token i < M and column n, decoded from the same seeded
// accumulators.
//
// MQ > 0 (the whole layer in one launch, MQ = M token rows of X): every
// workgroup first rotates, smooths and quantizes the MQ rows itself, with the
// arithmetic of the per-row quantizer (rrs_quant_rows.hip) and the maximum
// over the rows taken locally instead of exchanged, so the codes and scales
// are bit-identical to rrs_rotate_smooth_quant's; it works in the ring's last
// slot of every wave and the partial-sum area (one contiguous region: the
// ring is laid out slot by slot), which no load touches before the loop,
// while the first RS - 1 sub-buffers of weights stream in. (Xq, a_scale and
// s_group are intermediates of the layer and are not written.)
template <int K, int GS, int W, int TB, bool kTiled, bool kPartials, int MQ = 0>
__global__ __launch_bounds__(64 * W) void gemm_stream_kernel(
    const uint8_t* __restrict__ Xq, const float* __restrict__ a_scale,
    const float* __restrict__ s_group, const uint8_t* __restrict__ Wq,
    const float* __restrict__ w_scale, int M, int N, uint16_t* __restrict__ Y,
    int32_t* __restrict__ P, float out_scale, const uint16_t* __restrict__ X) {
  using S = StreamShape<K, W>;
  constexpr int g = GS * 64;
  constexpr int GB = g / 2;                   // packed bytes of a row per group
  constexpr int NG = S::R / GB;               // groups per wave (its slice of K)
  constexpr int NGS = S::SBW / GB;            // groups per sub-buffer
  constexpr int NP = GB >= 64 ? GB / 64 : 1;  // 16-byte lane pieces per group
  static_assert(NGS >= 1 && S::SBW % GB == 0, "every sub-buffer holds whole groups");
  static_assert(NG <= 64, "one group scale per lane");
  // The waves' fp32 sums of a block meet in `part`: double-buffered (one
  // barrier per block) when both copies fit beside the ring, else one copy
  // and a second barrier.
  constexpr int kRingBytes = W * S::RS * S::SB;
  constexpr int kPartBytes = W * TB * 64 * 16;
  constexpr int PB = kRingBytes + 2 * kPartBytes <= 163840 ? 2 : 1;
  static_assert(kRingBytes + PB * kPartBytes <= 163840, "LDS of one workgroup");
  struct alignas(16) Lds {
    uint8_t ring[kRingBytes];
    v4f part[PB][W][TB][64];  // follows the ring directly (kRingBytes % 16 == 0)
  };
  __shared__ Lds L;
  uint8_t* const ring = L.ring;
  auto& part = L.part;
  static_assert(MQ == 0 || (W == 4 && TB == 1 && !kPartials), "one-launch layer: M <= 2");
  constexpr int G = K / g;
  __shared__ float qsg[MQ > 0 ? G : 1];  // s_b (one-launch layer)
  __shared__ float qred[MQ > 0 ? 4 * MQ : 1];
  __shared__ float qa[MQ > 0 ? MQ : 1];  // alpha of the rows

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int kq = __builtin_amdgcn_readfirstlane(t >> 6);  // K slice of this wave
  const int c = lane & 15;
  const int q = lane >> 4;
  constexpr size_t krow = (size_t)K / 2;
  // Ring slot of item i of this wave: wave-major, or slot-major for MQ > 0.
  uint8_t* my = ring + kq * S::RS * S::SB;
  auto slot_of = [&](int i) -> uint8_t* {
    if constexpr (MQ > 0)
      return ring + (i % S::RS) * (W * S::SB) + kq * S::SB;
    else
      return my + (i % S::RS) * S::SB;
  };
  const int nblk = N / kRows;
  // Column blocks of this workgroup: w, w + grid, ... with four waves (two
  // workgroups per compute unit); one contiguous range with eight (one per
  // compute unit), which streams 1-2 us faster there and 1.5 us slower with
  // four (decode shape, back-to-back calls).
  constexpr bool kRange = W == 8;
  const int b_lo = kRange ? (int)(((long long)blockIdx.x * nblk) / (int)gridDim.x) : (int)blockIdx.x;
  const int b_step = kRange ? 1 : (int)gridDim.x;
  const int mine = kRange ? (int)(((long long)(blockIdx.x + 1) * nblk) / (int)gridDim.x) - b_lo
                          : (nblk - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
  const int items = mine * S::SPB;  // sub-buffers this wave streams, in order

  // Direct loads of item i (sub-buffer i % SPB of column block i / SPB) into
  // ring slot i % RS. Row-major: each instruction RPI rows x SBW bytes,
  // chunks permuted; tiled: each instruction one tile (the block's 16 rows are
  // one 16-row block, n0 a multiple of 16).
  auto issue = [&](int i) {
    const int blk = b_lo + (i / S::SPB) * b_step;
    const int sp = i % S::SPB;
    uint8_t* dst = slot_of(i);
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

  // One-launch layer: the MQ rows of X are requested first, so that waiting
  // for them (vector-memory loads retire in order) does not wait for the
  // weight loads issued after them.
  constexpr int EQ = MQ > 0 ? FwhtShape<K>::E : 8;
  uint4 xraw[MQ > 0 ? MQ : 1][EQ / 8];
  if constexpr (MQ > 0) {
#pragma unroll
    for (int r = 0; r < MQ; ++r)
#pragma unroll
      for (int w = 0; w < EQ / 8; ++w)
        xraw[r][w] = reinterpret_cast<const uint4*>(X + (size_t)r * K + (size_t)t * EQ)[w];
  }

  // Fill the ring: the first RS - 1 sub-buffers.
#pragma unroll
  for (int i = 0; i < S::RS - 1; ++i)
    if (i < items) issue(i);

  // One-launch layer: rotate, smooth and quantize the MQ rows (Section 3.3,
  // then Section 3.2, Eq. 1-2) into codes in LDS.
  const uint8_t* tok = Xq;
  if constexpr (MQ > 0) {
    constexpr int E = FwhtShape<K>::E;  // positions per thread (256 threads)
    static_assert(E >= 8 && E <= 64, "packed 8 codes at a time");
    static_assert((W * S::SB + PB * kPartBytes) >= lds_row_floats(K) * 4 &&
                      (W * S::SB + PB * kPartBytes) >= MQ * K / 2,
                  "scratch in the last ring slot and the partial sums");
    float* scr = reinterpret_cast<float*>(ring + (S::RS - 1) * (W * S::SB));
    float v[MQ][E];
#pragma unroll
    for (int r = 0; r < MQ; ++r) {
#pragma unroll
      for (int w = 0; w < E / 8; ++w) {
        const uint32_t h4[4] = {xraw[r][w].x, xraw[r][w].y, xraw[r][w].z, xraw[r][w].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          v[r][8 * w + 2 * k] = half_to_float(h4[k] & 0xFFFFu);
          v[r][8 * w + 2 * k + 1] = half_to_float(h4[k] >> 16);
        }
      }
      fwht_row<K, true>(v[r], scr, t);  // v[r][e] = y[t + 256 e]
      __syncthreads();                  // the transform's last reads are done
#pragma unroll
      for (int e = 0; e < E; ++e) scr[pos_addr<E>(t + e * kRowThreads)] = v[r][e];
      __syncthreads();
      read_positions<E>(scr, t, v[r]);  // v[r][e] = y[t E + e]
    }
    // s_b: the largest |y| of group b over the rows; a group is tps threads
    // of one wave (K >= 4 g).
    constexpr int tps = g / E;
    static_assert(tps >= 1 && tps <= 64, "a group inside one wave");
    float pm = 0.0f;
#pragma unroll
    for (int r = 0; r < MQ; ++r)
#pragma unroll
      for (int e = 0; e < E; ++e) pm = fmaxf(pm, fabsf(v[r][e]));
#pragma unroll
    for (int o = 1; o < tps; o <<= 1) pm = fmaxf(pm, __shfl_xor(pm, o, 64));
    const float rb = (pm == 0.0f) ? 0.0f : __fdiv_rn(1.0f, pm);  // r_b = fl(1 / s_b)
    if ((t & (tps - 1)) == 0) qsg[t / tps] = pm;
    // alpha_i: the largest fl(|y| r_b) of row i
#pragma unroll
    for (int r = 0; r < MQ; ++r) {
      float lm = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[r][e]));
      lm = wave_max(lm * rb);
      if (lane == 0) qred[4 * r + kq] = lm;
    }
    __syncthreads();  // qred and qsg written, every read of scr done
    uint8_t* codes = reinterpret_cast<uint8_t*>(scr);  // MQ rows of K/2 bytes
#pragma unroll
    for (int r = 0; r < MQ; ++r) {
      const float a = fmaxf(fmaxf(qred[4 * r], qred[4 * r + 1]), fmaxf(qred[4 * r + 2], qred[4 * r + 3]));
      const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
      const float m = rb * inv;  // fl(r_b * inv_i)
      uint32_t wd[E / 8];
#pragma unroll
      for (int w = 0; w < E / 8; ++w) wd[w] = quant_pack8(&v[r][8 * w], m);
      const size_t off = (size_t)r * krow + (size_t)t * (E / 2);
#pragma unroll
      for (int w = 0; w < E / 8; ++w) *reinterpret_cast<uint32_t*>(codes + off + 4 * w) = wd[w];
      if (t == 0) qa[r] = __fdiv_rn(a, 7.0f);
    }
    __syncthreads();  // codes, qa visible
    tok = codes;
  }

  // Token codes of the wave's slice (once per workgroup) and its group
  // scales (one per lane).
  uint32_t aw[TB][NG][NP][4];
#pragma unroll
  for (int u = 0; u < TB; ++u) {
    const uint8_t* abase = tok + (size_t)min(16 * u + c, M - 1) * krow + (size_t)kq * S::R;
#pragma unroll
    for (int b = 0; b < NG; ++b) {
      if constexpr (GB >= 64) {
#pragma unroll
        for (int h = 0; h < NP; ++h) {
          const uint4 v = *reinterpret_cast<const uint4*>(abase + b * GB + 64 * h + 16 * q);
          aw[u][b][h][0] = v.x;
          aw[u][b][h][1] = v.y;
          aw[u][b][h][2] = v.z;
          aw[u][b][h][3] = v.w;
        }
      } else {
        const uint2 v = *reinterpret_cast<const uint2*>(abase + b * GB + 8 * q);
        aw[u][b][0][0] = v.x;
        aw[u][b][0][1] = v.y;
        aw[u][b][0][2] = 0u;
        aw[u][b][0][3] = 0u;
      }
    }
  }
  float sv = 0.0f;
  if constexpr (MQ > 0)
    sv = qsg[kq * NG + (lane < NG ? lane : 0)];
  else if constexpr (!kPartials)
    sv = s_group[kq * NG + (lane < NG ? lane : 0)];

  constexpr int kMagic = 0x4B400000;  // bits of 1.5 * 2^23
  const v4i seed = GS > 4 ? v4i{0, 0, 0, 0} : v4i{kMagic, kMagic, kMagic, kMagic};

  // Epilogue split: the TB x 4 pairs (token block u, accumulator row r) of
  // every lane are dealt to the waves, pair x to wave x % W; pair (u, r) of
  // lane (c, q) is output row 16 u + 4 q + r. With W = 4 and one token block,
  // wave kq stores row 4 q + kq.
  constexpr int NX = (4 * TB + W - 1) / W;  // pairs per wave
  float oscale[NX];                         // alpha of the pair's row times out_scale
#pragma unroll
  for (int x = 0; x < NX; ++x) {
    const int pi = kq + x * W;
    const int row = 16 * (pi >> 2) + 4 * q + (pi & 3);
    oscale[x] = 0.0f;
    if constexpr (MQ > 0)
      oscale[x] = qa[min(row, M - 1)] * out_scale;
    else if constexpr (!kPartials)
      oscale[x] = a_scale[min(row, M - 1)] * out_scale;
  }
  // One-launch layer: every wave has read its codes before the loop's first
  // refill overwrites the scratch (the last ring slot).
  if constexpr (MQ > 0) __syncthreads();

  for (int tb = 0; tb < mine; ++tb) {
    const int blk = b_lo + tb * b_step;
    float bcol = 0.0f;  // beta of this lane's column, requested early
    if constexpr (!kPartials) bcol = w_scale[blk * kRows + c];
    float f[TB][4];
#pragma unroll
    for (int u = 0; u < TB; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) f[u][r] = 0.0f;
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
      const uint8_t* buf = slot_of(i);
#pragma unroll
      for (int bl = 0; bl < NGS; ++bl) {
        const int b = sp * NGS + bl;  // group of the wave's slice
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
        v4i acc[TB];
#pragma unroll
        for (int u = 0; u < TB; ++u) acc[u] = seed;
#pragma unroll
        for (int st = 0; st < GS; ++st) {
          const int h = st >> 1;
          const int o = 2 * (st & 1);
          const v4i wv = unpack_pair(ww[h][o], ww[h][o + 1]);
#pragma unroll
          for (int u = 0; u < TB; ++u)
            acc[u] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                unpack_pair(aw[u][b][h][o], aw[u][b][h][o + 1]), wv, acc[u], 0, 0, 0);
        }
        if constexpr (kPartials) {
          int32_t* Pg = P + (size_t)(kq * NG + b) * (size_t)M * (size_t)N;
#pragma unroll
          for (int u = 0; u < TB; ++u)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = 16 * u + 4 * q + r;
              if (row < M)
                Pg[(size_t)row * N + blk * kRows + c] =
                    (GS > 4 ? acc[u][r] : acc[u][r] - kMagic) >> 8;
            }
        } else {
          const float s =
              __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sv), b));
#pragma unroll
          for (int u = 0; u < TB; ++u) {
            // Bit-cast the whole vector, then index: bit-casting a single
            // element of an ext_vector is miscompiled (every element reads
            // element 0).
            const v4f accf = __builtin_bit_cast(v4f, acc[u]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float pv = GS > 4 ? (float)acc[u][r] : accf[r] - 12582912.0f;
              f[u][r] = __builtin_fmaf(s, pv, f[u][r]);
            }
          }
        }
      }
    }
    if constexpr (!kPartials) {
      // The W slices' sums of this block, added in the order kq = 0 .. W - 1.
      const int pb = PB == 2 ? (tb & 1) : 0;
#pragma unroll
      for (int u = 0; u < TB; ++u) part[pb][kq][u][lane] = v4f{f[u][0], f[u][1], f[u][2], f[u][3]};
      __syncthreads();
#pragma unroll
      for (int x = 0; x < NX; ++x) {
        const int pi = kq + x * W;
        if (pi < 4 * TB) {
          const int u = pi >> 2;
          const int r = pi & 3;
          float sum = part[pb][0][u][lane][r];
#pragma unroll
          for (int p = 1; p < W; ++p) sum += part[pb][p][u][lane][r];
          const int row = 16 * u + 4 * q + r;
          // out_scale = 2^-8 (undoes the 16 x 16 of the unpacked operands) / K
          // (the unnormalized rotation; 1 without rotation), an exact power of two.
          if (row < M)
            Y[(size_t)row * N + blk * kRows + c] =
                __builtin_bit_cast(uint16_t, (_Float16)((sum * oscale[x]) * bcol));
        }
      }
      if constexpr (PB == 1) __syncthreads();  // every wave has read `part`
    }
  }
}

// Shapes each form of the kernel takes (K, g powers of two, g <= 512).
// W = 4, one token block: every wave holds whole groups (K >= 4 g); K = 16384
// with g <= 128 keeps 32 or 64 groups of token codes per wave, which do not fit
// the registers next to the loop. W = 8, two token blocks: K = 8192 only. The
// form compiles without spills wherever K >= 1024, K >= 8 g and TB K <= 16384,
// but it beats the few-token kernel only where the weight stream dominates:
// at K = 8192, N = 28672 it takes 28.1 / 30.3 / 31.6 us at M = 17 / 24 / 32
// (row-major; 23.4 / 24.8 / 26.1 tiled) against 34.3 / 35.7 / 36.6 (27.3 /
// 28.8 / 30.0); at K = 4096, N = 12288 it ties up to 32 tokens and loses with
// three or four token blocks (13.7 against 12.7 us at M = 64); at K = 8192
// three or four token blocks spill.
constexpr bool stream_form_fits(int K, int W, int TB, int g) {
  return W == 4 ? (TB == 1 && K >= 4 * g && !(K == 16384 && g <= 128))
                : (W == 8 && TB == 2 && K == 8192 && K >= 8 * g);
}

template <int K, int W, int TB, bool kPartials>
hipError_t launch_k(const uint8_t* Xq, const float* a_scale, const float* s_group,
                    const uint8_t* Wq, const float* w_scale, int M, int N, int g, uint16_t* Y,
                    int32_t* P, float out_scale, hipStream_t stream, bool tiled) {
  const int nblk = N / kRows;  // N % 16 == 0 (API precondition)
#define RRS_STREAM_T(GS_, T_)                                                              \
  {                                                                                        \
    constexpr auto kern = gemm_stream_kernel<K, GS_, W, TB, T_, kPartials>;                \
    kern<<<resident_grid<kern>(nblk, 64 * W), 64 * W, 0, stream>>>(Xq, a_scale, s_group,    \
                                                                   Wq, w_scale, M, N, Y, P, \
                                                                   out_scale, nullptr);     \
  }
#define RRS_STREAM(GS_)                             \
  if constexpr (stream_form_fits(K, W, TB, GS_ * 64)) { \
    if (tiled)                                      \
      RRS_STREAM_T(GS_, true)                       \
    else                                            \
      RRS_STREAM_T(GS_, false)                      \
  } else {                                          \
    return hipErrorInvalidValue;                    \
  }
  switch (g) {
    case 64: RRS_STREAM(1) break;
    case 128: RRS_STREAM(2) break;
    case 256: RRS_STREAM(4) break;
    case 512: RRS_STREAM(8) break;
    default: return hipErrorInvalidValue;
  }
#undef RRS_STREAM
#undef RRS_STREAM_T
  return hipGetLastError();
}

template <int W, int TB, bool kPartials>
hipError_t launch_any(const uint8_t* Xq, const float* a_scale, const float* s_group,
                      const uint8_t* Wq, const float* w_scale, int M, int N, int K, int g,
                      uint16_t* Y, int32_t* P, float out_scale, hipStream_t stream,
                      bool tiled) {
  switch (K) {
#define RRS_K(K_)                                                                        \
  case K_:                                                                               \
    return launch_k<K_, W, TB, kPartials>(Xq, a_scale, s_group, Wq, w_scale, M, N, g, Y, P, \
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

// The form for M tokens: up to 16, four waves and one token block; 17 to 32,
// eight waves (one workgroup per compute unit) and two token blocks, so the
// weights still stream once.
template <bool kPartials>
hipError_t launch_tokens(const uint8_t* Xq, const float* a_scale, const float* s_group,
                         const uint8_t* Wq, const float* w_scale, int M, int N, int K, int g,
                         uint16_t* Y, int32_t* P, float out_scale, hipStream_t stream,
                         bool tiled) {
  if (M <= kMaxTokens)
    return launch_any<4, 1, kPartials>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, P,
                                       out_scale, stream, tiled);
  return launch_any<8, 2, kPartials>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, P,
                                     out_scale, stream, tiled);
}

// The one-launch layer: the same kernel with the quantizer of MQ rows in
// front of the loop (four waves, one token block).
template <int K, int MQ>
hipError_t launch_layer_k(const uint16_t* X, const uint8_t* Wq, const float* w_scale, int N,
                          int g, uint16_t* Y, float out_scale, hipStream_t stream, bool tiled) {
  const int nblk = N / kRows;
#define RRS_LAYER_T(GS_, T_)                                                                \
  {                                                                                         \
    constexpr auto kern = gemm_stream_kernel<K, GS_, 4, 1, T_, false, MQ>;                  \
    kern<<<resident_grid<kern>(nblk), kThreads, 0, stream>>>(nullptr, nullptr, nullptr, Wq, \
                                                             w_scale, MQ, N, Y, nullptr,    \
                                                             out_scale, X);                 \
  }
#define RRS_LAYER(GS_)                                 \
  if constexpr (stream_form_fits(K, 4, 1, GS_ * 64)) { \
    if (tiled)                                         \
      RRS_LAYER_T(GS_, true)                           \
    else                                               \
      RRS_LAYER_T(GS_, false)                          \
  } else {                                             \
    return hipErrorInvalidValue;                       \
  }
  switch (g) {
    case 64: RRS_LAYER(1) break;
    case 128: RRS_LAYER(2) break;
    case 256: RRS_LAYER(4) break;
    case 512: RRS_LAYER(8) break;
    default: return hipErrorInvalidValue;
  }
#undef RRS_LAYER
#undef RRS_LAYER_T
  return hipGetLastError();
}

}  // namespace

bool layer_one_launch_fits(int M, int K, int g) {
  return (M == 1 || M == 2) && (K == 2048 || K == 4096 || K == 8192) &&
         stream_form_fits(K, 4, 1, g);
}

hipError_t launch_layer_one_launch(const uint16_t* X, int M, int N, int K, int g,
                                   const uint8_t* Wq, const float* w_scale, uint16_t* Y,
                                   float out_scale, hipStream_t stream, WqLayout lay) {
  if (!layer_one_launch_fits(M, K, g)) return hipErrorInvalidValue;
#define RRS_LK(K_)                                                                          \
  case K_:                                                                                  \
    return M == 1 ? launch_layer_k<K_, 1>(X, Wq, w_scale, N, g, Y, out_scale, stream,       \
                                          lay.tiled)                                        \
                  : launch_layer_k<K_, 2>(X, Wq, w_scale, N, g, Y, out_scale, stream,       \
                                          lay.tiled)
  switch (K) {
    RRS_LK(2048);
    RRS_LK(4096);
    RRS_LK(8192);
    default: return hipErrorInvalidValue;
  }
#undef RRS_LK
}

bool stream_kernel_fits(int M, int K, int g) {
  if (M < 1 || M > 2 * kMaxTokens) return false;
  if (M <= kMaxTokens) return stream_form_fits(K, 4, 1, g);
  return stream_form_fits(K, 8, 2, g);
}

hipError_t launch_w4a4_gemm_stream(const uint8_t* Xq, const float* a_scale,
                                   const float* s_group, const uint8_t* Wq,
                                   const float* w_scale, int M, int N, int K, int g,
                                   uint16_t* Y, float out_scale, hipStream_t stream,
                                   WqLayout lay) {
  if (!stream_kernel_fits(M, K, g)) return hipErrorInvalidValue;
  return launch_tokens<false>(Xq, a_scale, s_group, Wq, w_scale, M, N, K, g, Y, nullptr,
                              out_scale, stream, lay.tiled);
}

hipError_t launch_w4a4_gemm_stream_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                            int K, int g, int32_t* P, hipStream_t stream,
                                            WqLayout lay) {
  if (!stream_kernel_fits(M, K, g)) return hipErrorInvalidValue;
  return launch_tokens<true>(Xq, nullptr, nullptr, Wq, nullptr, M, N, K, g, nullptr, P, 0.0f,
                             stream, lay.tiled);
}

}  // namespace rrs
