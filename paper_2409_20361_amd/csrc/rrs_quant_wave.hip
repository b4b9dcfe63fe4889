// Online rotate + runtime smooth + per-token INT4 quantization for K <= 4096
// (Section 3.3 then Section 3.2; Eq. 1-2; Section 2.1): one wave per row.
//
// The same two launches as for large K (see rrs_quant.hip): rot_max writes one
// row of group maxima per workgroup, quant reduces them to s_b and r_b and
// writes the codes. What differs is how a row is rotated: here a row belongs
// to R = K/64 lanes of one wave (a wave holds 64/R rows), so the whole
// transform needs no workgroup barrier:
//   layout 1: lane l of the row holds elements i = 64 l + e (e = 0..63), i.e.
//             64 contiguous values (eight 16-byte loads); FWHT stages
//             h = 1..32 are in-register butterflies;
//   layout 2: after a transpose through a wave-private LDS region, lane l
//             holds i = l + R e; stages h = 64..K/2 (index bits 6 .. log2 K - 1,
//             register bits 6 - log2 R .. 5) are in-register butterflies.
// Stage order stays h = 1, 2, ..., K/2 with one rounded fp32 add or subtract
// per butterfly output, so the result is bit-identical to the canonical
// sequential transform (and to the team kernels for large K). quant then
// transposes back to layout 1 (or gathers the statically reordered positions)
// so each lane quantizes and packs 64 consecutive codes into 32 bytes.
//
// LDS row region: element i at A(i) = i + 4 floor(i / 64) (16-byte aligned runs
// of 64, conflict-free 128-bit writes of layout 1 and 32-bit reads of layout 2);
// rows of one wave are 16 floats further apart so they start in other banks.
#include "rrs_device.h"
#include "rrs_internal.h"

namespace rrs {
namespace {

template <int K>
struct WaveRow {
  static constexpr int R = K / 64;             // lanes per row
  static constexpr int LR = ilog2(R);          // 3 .. 6
  static constexpr int RW = 64 / R;            // rows per wave
  static constexpr int RF = K + K / 16 + 16;   // LDS floats per row region
  static constexpr int LOGK = ilog2(K);
  static_assert(K >= 512 && K <= 4096 && (1 << LOGK) == K, "wave path: K in 512..4096");
};

__device__ __forceinline__ int lds_a(int i) { return i + ((i >> 6) << 2); }

// Raw halves of 64 consecutive elements (128 bytes) of a row, or zeros.
__device__ __forceinline__ void load_raw64(const uint16_t* __restrict__ src, bool live,
                                           uint4 (&raw)[8]) {
  if (live) {
#pragma unroll
    for (int c = 0; c < 8; ++c) raw[c] = reinterpret_cast<const uint4*>(src)[c];
  } else {
#pragma unroll
    for (int c = 0; c < 8; ++c) raw[c] = make_uint4(0u, 0u, 0u, 0u);
  }
}

__device__ __forceinline__ void raw_to_float(const uint4 (&raw)[8], float (&v)[64]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const uint32_t w[4] = {raw[c].x, raw[c].y, raw[c].z, raw[c].w};
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      v[c * 8 + 2 * m] = half_to_float(w[m] & 0xFFFFu);
      v[c * 8 + 2 * m + 1] = half_to_float(w[m] >> 16);
    }
  }
}

// Rotate one row held in layout 1 (v[e] = x[64 l + e]); on exit layout 2
// (v[e] = y[l + R e]; y = x when kRot is false: the same data movement without
// the butterflies, for the ablation without rotation). `row` is this row's LDS
// region (wave-private).
template <int K, bool kRot>
__device__ __forceinline__ void fwht_wave_row(float (&v)[64], float* row, int l) {
  using S = WaveRow<K>;
  if constexpr (kRot) fwht_stages<64, 0, 6>(v);
#pragma unroll
  for (int m = 0; m < 16; ++m)
    *reinterpret_cast<float4*>(row + lds_a(64 * l + 4 * m)) =
        make_float4(v[4 * m], v[4 * m + 1], v[4 * m + 2], v[4 * m + 3]);
#pragma unroll
  for (int e = 0; e < 64; ++e) v[e] = row[lds_a(l + S::R * e)];
  if constexpr (kRot) fwht_stages<64, 6 - S::LR, 6>(v);
}

// Max over the R lanes of each row of the wave (aligned groups of R lanes).
template <int R>
__device__ __forceinline__ float row_max(float x) {
#pragma unroll
  for (int o = 1; o < R; o <<= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// ---------------------------------------------------------------------------
// 1. rotate + per-workgroup group maxima (8 waves per workgroup)
// ---------------------------------------------------------------------------
constexpr int kRotWaves = 8;

template <int K, bool kRot>
__global__ __launch_bounds__(kRotWaves * 64) void rot_max_wave_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg,
    const int32_t* __restrict__ perm, float* __restrict__ gpart) {
  using S = WaveRow<K>;
  __shared__ __attribute__((aligned(16))) float rows[kRotWaves * S::RW * S::RF];
  __shared__ float red[kRotWaves * 64];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int sub = lane >> S::LR;   // row of the wave
  const int l = lane & (S::R - 1);  // lane within the row
  float* row = rows + (wave * S::RW + sub) * S::RF;

  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int per_pass = kRotWaves * S::RW;
  const int passes = (rows_per_wg + per_pass - 1) / per_pass;
  auto row_of = [&](int p) { return r0 + (p * kRotWaves + wave) * S::RW + sub; };

  float cm[64];
#pragma unroll
  for (int e = 0; e < 64; ++e) cm[e] = 0.0f;
  uint4 raw[8];
  {
    const int r = row_of(0);
    load_raw64(X + (size_t)min(r, M - 1) * K + 64 * l, r < r1, raw);
  }
  for (int p = 0; p < passes; ++p) {
    float v[64];
    raw_to_float(raw, v);
    if (p + 1 < passes) {
      const int r = row_of(p + 1);
      load_raw64(X + (size_t)min(r, M - 1) * K + 64 * l, r < r1, raw);
    }
    fwht_wave_row<K, kRot>(v, row, l);  // v[e] = y[l + R e]
#pragma unroll
    for (int e = 0; e < 64; ++e) cm[e] = fmaxf(cm[e], fabsf(v[e]));
  }
  // Rows of the same wave hold the same channels: combine them in registers.
#pragma unroll
  for (int e = 0; e < 64; ++e)
#pragma unroll
    for (int o = S::R; o < 64; o <<= 1) cm[e] = fmaxf(cm[e], __shfl_xor(cm[e], o, 64));
  // Each wave's channel maxima go into its own first row region (its rows
  // are done with it); the workgroup's maximum of channel c is then taken
  // over the waves in a fixed order (no atomics).
  if (sub == 0) {
    float* cw = rows + wave * S::RW * S::RF;
#pragma unroll
    for (int e = 0; e < 64; ++e) cw[lds_a(l + S::R * e)] = cm[e];
  }
  __syncthreads();
  auto chan_max = [&](int c) {
    float m = rows[lds_a(c)];
#pragma unroll
    for (int w = 1; w < kRotWaves; ++w) m = fmaxf(m, rows[w * S::RW * S::RF + lds_a(c)]);
    return m;
  };
  // Group maxima over the (reordered) positions: thread t covers P = K / 512
  // (at least 1) consecutive positions, all in one group (P <= 8 < g).
  constexpr int NT = kRotWaves * 64;
  constexpr int P = K >= NT ? K / NT : 1;
  static_assert(K / P == NT, "every thread covers P positions");
  float pm = 0.0f;
  if (perm) {
    int idx[P];  // all loads first, so their latencies overlap
#pragma unroll
    for (int q = 0; q < P; ++q) idx[q] = perm[tid * P + q];
#pragma unroll
    for (int q = 0; q < P; ++q) pm = fmaxf(pm, chan_max(idx[q]));
  } else {
#pragma unroll
    for (int q = 0; q < P; ++q) pm = fmaxf(pm, chan_max(tid * P + q));
  }
  red[tid] = pm;
  __syncthreads();
  const int G = K / g;
  if (tid < G) {
    const int npos = g / P;  // threads per group
    float s = 0.0f;
    for (int u = 0; u < npos; ++u) s = fmaxf(s, red[tid * npos + u]);
    gpart[(size_t)blockIdx.x * G + tid] = s;
  }
}

// ---------------------------------------------------------------------------
// 2. group scales, per-token scale, codes (4 waves per workgroup)
// ---------------------------------------------------------------------------
constexpr int kQuantWaves = 4;

// kOrder (runtime reorder): gpart holds nparts rows of K/32 block maxima; the
// workgroup ranks the blocks itself (block_order_wg), takes s_b over the
// sorted blocks of group b, and reads position j of a row from channel
// 32 sblk[j / 32] + j % 32; workgroup 0 writes s_group and block_order.
template <int K, bool kRot, bool kSmooth, bool kOrder = false>
__global__ __launch_bounds__(kQuantWaves * 64) void quant_wave_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg, int nparts,
    const int32_t* __restrict__ perm, const float* __restrict__ gpart,
    uint8_t* __restrict__ Xq, float* __restrict__ a_scale, float* __restrict__ s_group,
    int32_t* __restrict__ block_order = nullptr) {
  using S = WaveRow<K>;
  constexpr int NT = kQuantWaves * 64;
  constexpr int GMAX = K / 64;  // groups at g = 64
  constexpr int NB = K / kReorderBlock;
  __shared__ __attribute__((aligned(16))) float rows[kQuantWaves * S::RW * S::RF];
  __shared__ float rg[GMAX];
  __shared__ __attribute__((aligned(16))) float red[kOrder ? 4 * NT : NT];
  __shared__ __attribute__((aligned(16))) unsigned long long key[kOrder ? NB : 2];
  __shared__ __attribute__((aligned(16))) unsigned long long srt[kOrder ? NB : 2];
  __shared__ float skey[kOrder ? NB : 1];
  __shared__ int sblk[kOrder ? NB : 1];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int sub = lane >> S::LR;
  const int l = lane & (S::R - 1);
  float* row = rows + (wave * S::RW + sub) * S::RF;
  const int G = K / g;

  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  const int per_pass = kQuantWaves * S::RW;
  const int passes = (rows_per_wg + per_pass - 1) / per_pass;
  auto row_of = [&](int p) { return r0 + (p * kQuantWaves + wave) * S::RW + sub; };

  // This wave's first row is requested before anything else.
  uint4 raw[8];
  {
    const int r = row_of(0);
    load_raw64(X + (size_t)min(r, M - 1) * K + 64 * l, r < r1, raw);
  }

  // s_b = max over the partial rows. Thread t takes group b = t % GMAX and
  // rows t / GMAX + k NS (NS = 256 / GMAX slices) with a fixed number of
  // unconditional loads (row indices clamped to the last row, entries for
  // b >= G read neighbouring rows and are ignored: every index stays inside
  // the 256 x K/64 workspace). The loads are issued here and reduced after
  // the first row's rotation, which does not need the scales and hides their
  // latency.
  constexpr int NS = NT / GMAX;
  constexpr int NL = (256 + NS - 1) / NS;  // loads per thread for up to 256 rows
  float x[kSmooth && !kOrder ? NL : 1];
  if constexpr (kSmooth && !kOrder) {
    const int b = tid % GMAX;
    const int sl = tid / GMAX;
#pragma unroll
    for (int k = 0; k < NL; ++k) {
      const int i = min(sl + k * NS, nparts - 1);
      x[k] = gpart[(size_t)i * G + b];
    }
  }

  // Rotate row p into v (layout 2), prefetching row p + 1.
  float v[64];
  auto rotate = [&](int p) {
    raw_to_float(raw, v);
    if (p + 1 < passes) {
      const int rn = row_of(p + 1);
      load_raw64(X + (size_t)min(rn, M - 1) * K + 64 * l, rn < r1, raw);
    }
    fwht_wave_row<K, kRot>(v, row, l);  // v[e] = y[l + R e]
  };
  rotate(0);

  if constexpr (!kSmooth) {
    // Ablation without smoothing: every scale is 1 (rotation + per-token only).
    if (tid < G) {
      rg[tid] = 1.0f;
      if (blockIdx.x == 0) s_group[tid] = 1.0f;
    }
    __syncthreads();
  } else if constexpr (kOrder) {
    block_order_wg<NT, NB>(gpart, nparts, red, key, srt, sblk, skey, tid);
    if (tid < G) {
      const int per = g / kReorderBlock;
      float sv = 0.0f;
      for (int u = 0; u < per; ++u) sv = fmaxf(sv, skey[tid * per + u]);
      rg[tid] = (sv == 0.0f) ? 0.0f : __fdiv_rn(1.0f, sv);
      if (blockIdx.x == 0) s_group[tid] = sv;
    }
    if (blockIdx.x == 0)
      for (int b = tid; b < NB; b += NT) block_order[b] = sblk[b];
    __syncthreads();
  } else {
    float m = 0.0f;
#pragma unroll
    for (int k = 0; k < NL; ++k) m = fmaxf(m, x[k]);
    red[tid] = m;
    __syncthreads();
    if (tid < G) {
      float sv = red[tid];
      for (int q = 1; q < NS; ++q) sv = fmaxf(sv, red[q * GMAX + tid]);
      rg[tid] = (sv == 0.0f) ? 0.0f : __fdiv_rn(1.0f, sv);
      if (blockIdx.x == 0) s_group[tid] = sv;
    }
    __syncthreads();
  }
  // Positions 64 l .. 64 l + 63 of a row lie in one group (g >= 64).
  const float rb = rg[(64 * l) / g];

  for (int p = 0; p < passes; ++p) {
    const int r = row_of(p);
    const bool live = r < r1;
    if (p > 0) rotate(p);
    // back to layout 1 through LDS, with the static reorder applied
#pragma unroll
    for (int e = 0; e < 64; ++e) row[lds_a(l + S::R * e)] = v[e];
    if constexpr (kOrder) {
      // positions 64 l .. 64 l + 63 are blocks 2 l and 2 l + 1 (masked into
      // range, as the team kernels do)
      const int c0 = (sblk[2 * l] & (NB - 1)) * kReorderBlock;
      const int c1 = (sblk[2 * l + 1] & (NB - 1)) * kReorderBlock;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        v[e] = row[lds_a(c0 + e)];
        v[32 + e] = row[lds_a(c1 + e)];
      }
    } else if (perm) {
      const int4* pp = reinterpret_cast<const int4*>(perm + 64 * l);
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        const int4 c = pp[m];
        v[4 * m] = row[lds_a(c.x)];
        v[4 * m + 1] = row[lds_a(c.y)];
        v[4 * m + 2] = row[lds_a(c.z)];
        v[4 * m + 3] = row[lds_a(c.w)];
      }
    } else {
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        const float4 c = *reinterpret_cast<const float4*>(row + lds_a(64 * l + 4 * m));
        v[4 * m] = c.x;
        v[4 * m + 1] = c.y;
        v[4 * m + 2] = c.z;
        v[4 * m + 3] = c.w;
      }
    }
    float lm = 0.0f;
#pragma unroll
    for (int e = 0; e < 64; ++e) lm = fmaxf(lm, fabsf(v[e]));
    const float a = row_max<S::R>(lm * rb);  // max over the row's groups of fl(M_ib r_b)
    const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
    const float m = rb * inv;                // fl(r_b * inv_i)
    if (live) {
      uint32_t nib[64];
#pragma unroll
      for (int e = 0; e < 64; ++e) nib[e] = int4_nibble(v[e] * m);
      store_nibbles<64>(Xq + (size_t)r * (K / 2) + 32 * l, nib);
      if (l == 0) a_scale[r] = __fdiv_rn(a, 7.0f);
    }
  }
}

// ---------------------------------------------------------------------------
// 3. One launch (K <= 4096, up to two rows per wave): rotate every row once,
//    exchange the workgroups' group maxima, quantize the rows kept in
//    registers.
//
// The two launches above rotate every row twice (the second pass cannot
// keep the first pass's rows), and each pass is one row per wave of serial
// latency: at 2048 x 4096 they took 9.9 + 14.9 us, with the FWHT's VALU work
// twice over. Here each wave rotates its rows once, brings them back to
// layout 1 (lane l holds positions 64 l .. 64 l + 63, one group) and keeps
// them in registers (64 VGPRs per row). The workgroups (one per compute
// unit, all resident) then exchange their rows of group maxima through the
// workspace as tagged words, one per (workgroup, group), in the fence-free
// protocol of rrs_device.h (epoch tags, per-location coherence). The polls
// are bounded (max_polls rounds per thread): a wait that runs out marks the
// call as failed in the header and the workgroup writes NaN into its rows'
// alpha (workgroup 0 also into s_group), so a failed exchange shows in the
// outputs. Same arithmetic in the same order as the two-pass kernels:
// bit-identical codes and scales.
// ---------------------------------------------------------------------------
constexpr int kFusedWaves = 8;  // waves per workgroup (4 when that fills every compute unit)
constexpr int kFusedMaxPolls = 1 << 20;
constexpr int kOrderRun = 16;   // workgroups per level-1 run of the reorder exchange

// kWideG: g = 64 (K / 64 groups); otherwise g >= 128, and the exchange holds
// half as many entries per thread.
// kOrder (runtime reorder): the workgroups exchange K/32 block maxima instead
// of group maxima, in two levels (below); every workgroup ranks the blocks,
// takes s_b over the sorted blocks of group b and quantizes its kept rows over
// the sorted positions; workgroup 0 writes s_group and block_order. `tagged`
// then holds one row of block words per workgroup and `tagged2` one per level-1
// group.
template <int K, bool kRot, int SLOTS, int WAVES, bool kWideG, bool kOrder = false>
__global__ __launch_bounds__(WAVES * 64) void rot_quant_fused_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg, uint32_t* header,
    unsigned long long* tagged, int nrows, int max_polls, uint8_t* __restrict__ Xq,
    float* __restrict__ a_scale, float* __restrict__ s_group,
    unsigned long long* tagged2 = nullptr, int32_t* __restrict__ block_order = nullptr) {
  using S = WaveRow<K>;
  constexpr int NT = WAVES * 64;
  constexpr int GMAX = K / 64;  // groups at g = 64
  constexpr int NB = K / kReorderBlock;
  __shared__ __attribute__((aligned(16))) float rows[WAVES * S::RW * S::RF];
  __shared__ float wmax[WAVES][kOrder ? NB : GMAX];
  __shared__ float red[NT];
  __shared__ float rg[GMAX];
  __shared__ __attribute__((aligned(16))) unsigned long long key[kOrder ? NB : 2];
  __shared__ __attribute__((aligned(16))) unsigned long long srt[kOrder ? NB : 2];
  __shared__ float skey[kOrder ? NB : 1];
  __shared__ int sblk[kOrder ? NB : 1];
  __shared__ int missed;
  __shared__ uint32_t tag_lds;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int sub = lane >> S::LR;    // row of the wave
  const int l = lane & (S::R - 1);  // lane within the row
  float* row = rows + (wave * S::RW + sub) * S::RF;
  const int G = K / g;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  auto row_of = [&](int p) { return r0 + (p * WAVES + wave) * S::RW + sub; };
  // This call's tag (the header was written by earlier calls only): one
  // thread requests it now and hands it over in LDS before the first barrier,
  // so the load's latency hides behind the rotation.
  uint32_t epoch = 0u;
  if (tid == 0)
    epoch = __hip_atomic_load(header + kEpochWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // Phase 1: rotate, back to layout 1, per-lane maxima.
  float v[SLOTS][64];
  float lm[SLOTS];
  uint4 raw[8];
  {
    const int r = row_of(0);
    load_raw64(X + (size_t)min(r, M - 1) * K + 64 * l, r < r1, raw);
  }
#pragma unroll
  for (int p = 0; p < SLOTS; ++p) {
    raw_to_float(raw, v[p]);
    if (p + 1 < SLOTS) {
      const int rn = row_of(p + 1);
      load_raw64(X + (size_t)min(rn, M - 1) * K + 64 * l, rn < r1, raw);
    }
    fwht_wave_row<K, kRot>(v[p], row, l);  // v[e] = y[l + R e]
#pragma unroll
    for (int e = 0; e < 64; ++e) row[lds_a(l + S::R * e)] = v[p][e];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const float4 c = *reinterpret_cast<const float4*>(row + lds_a(64 * l + 4 * m));
      v[p][4 * m] = c.x;
      v[p][4 * m + 1] = c.y;
      v[p][4 * m + 2] = c.z;
      v[p][4 * m + 3] = c.w;
    }
    float x = 0.0f;
#pragma unroll
    for (int e = 0; e < 64; ++e) x = fmaxf(x, fabsf(v[p][e]));
    lm[p] = x;
  }

  if constexpr (kOrder) {
    // The workgroup's block maxima: lane l's positions 64 l .. 64 l + 63 are
    // blocks 2 l and 2 l + 1; over slots, over the wave's rows, then over the
    // waves in LDS (a fixed order, no atomics).
    float b0 = 0.0f, b1 = 0.0f;
#pragma unroll
    for (int p = 0; p < SLOTS; ++p)
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        b0 = fmaxf(b0, fabsf(v[p][e]));
        b1 = fmaxf(b1, fabsf(v[p][32 + e]));
      }
#pragma unroll
    for (int o = S::R; o < 64; o <<= 1) {
      b0 = fmaxf(b0, __shfl_xor(b0, o, 64));
      b1 = fmaxf(b1, __shfl_xor(b1, o, 64));
    }
    if (sub == 0) {
      wmax[wave][2 * l] = b0;
      wmax[wave][2 * l + 1] = b1;
    }
    if (tid == 0) {
      missed = 0;
      tag_lds = next_epoch(epoch);
    }
    __syncthreads();
    const uint32_t tag = tag_lds;
    if (tid < NB) {
      float m = wmax[0][tid];
#pragma unroll
      for (int w = 1; w < WAVES; ++w) m = fmaxf(m, wmax[w][tid]);
      publish_tagged(tagged + (size_t)blockIdx.x * NB + tid, tag, m);
    }

    // Keys over all rows, in two levels so that no workgroup reads every
    // workgroup's row of words: the first workgroup of each run of kOrderRun
    // (the run's leader) reads the run's rows and publishes their maximum as
    // the run's row in tagged2; every workgroup then reads the runs' rows. A
    // leader whose wait ran out publishes its row as failed (sign bit set:
    // keys are never negative), so the failure reaches every reader. Thread
    // t serves block t / TPB, and reads every TPB-th word of a run.
    constexpr int TPB = NT / NB < kOrderRun ? NT / NB : kOrderRun;  // threads per block
    constexpr int NW = kOrderRun / TPB;                            // words per thread
    const int bb = tid / TPB;
    const int tp = tid % TPB;
    const bool serve = bb < NB;
    const unsigned long long none = (unsigned long long)tag << 32;  // absent: 0.0
    // Maximum of the NW words this thread reads from rows[first + tp + k TPB]
    // (k < NW, row index < count) of `words`; false if a wait ran out or a
    // word was marked failed.
    auto gather = [&](const unsigned long long* words, int first, int count, float* out) {
      unsigned long long x[NW];
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const int i = tp + k * TPB;
        x[k] = (serve && i < count) ? load_tagged(words + (size_t)(first + i) * NB + bb) : none;
      }
      bool ok = false;
      for (int round = 0;; ++round) {
        ok = true;
#pragma unroll
        for (int k = 0; k < NW; ++k) ok = ok && has_tag(x[k], tag);
        if (ok || round >= max_polls) break;
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int k = 0; k < NW; ++k) {
          const int i = tp + k * TPB;
          if (!has_tag(x[k], tag)) x[k] = load_tagged(words + (size_t)(first + i) * NB + bb);
        }
      }
      float m = 0.0f;
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const uint32_t fb = (uint32_t)x[k];
        ok = ok && !(fb >> 31);
        m = fmaxf(m, __uint_as_float(fb & 0x7FFFFFFFu));
      }
      // over the TPB threads of the block (consecutive lanes)
      int okv = ok ? 1 : 0;
#pragma unroll
      for (int o = 1; o < TPB; o <<= 1) {
        m = fmaxf(m, __shfl_xor(m, o, 64));
        okv &= __shfl_xor(okv, o, 64);
      }
      *out = m;
      return okv != 0;
    };
    const int run = blockIdx.x / kOrderRun;
    const int nruns = (nrows + kOrderRun - 1) / kOrderRun;
    if (blockIdx.x % kOrderRun == 0) {
      float m1 = 0.0f;
      const int first = run * kOrderRun;
      const bool ok1 = gather(tagged, first, min(kOrderRun, nrows - first), &m1);
      if (serve && tp == 0)
        publish_tagged(tagged2 + (size_t)run * NB + bb, tag,
                       ok1 ? m1 : __uint_as_float(0x80000000u));
    }
    {
      float m2 = 0.0f;
      bool ok2 = true;
      for (int r0 = 0; r0 < nruns; r0 += kOrderRun) {
        float mm = 0.0f;
        ok2 = gather(tagged2, r0, min(kOrderRun, nruns - r0), &mm) && ok2;
        m2 = fmaxf(m2, mm);
      }
      if (!ok2) missed = 1;  // benign race: every writer writes 1
      if (serve && tp == 0) key[bb] = block_sort_key(m2, bb);
    }
    __syncthreads();
    if (tid == 0) {
      // Every word of the call has been read (or given up on): advance the
      // epoch (workgroup 0 only).
      if (missed)
        __hip_atomic_store(header + kFailWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (blockIdx.x == 0)
        __hip_atomic_store(header + kEpochWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // Blocks with a larger key, or an equal key and a smaller index, first.
    rank_blocks<NB, NT>(key, srt, sblk, skey, tid);
    const bool failed = missed != 0;  // uniform over the workgroup
    // s_b over the sorted blocks of group b.
    if (tid < G) {
      const int per = g / kReorderBlock;
      float sv = 0.0f;
      for (int u = 0; u < per; ++u) sv = fmaxf(sv, skey[tid * per + u]);
      rg[tid] = (sv == 0.0f) ? 0.0f : __fdiv_rn(1.0f, sv);
      if (blockIdx.x == 0) s_group[tid] = failed ? __builtin_nanf("") : sv;
    }
    if (blockIdx.x == 0 && tid < NB) block_order[tid] = sblk[tid];
    __syncthreads();

    // Phase 2 over the sorted positions: 64 l .. 64 l + 63 are sorted blocks
    // 2 l and 2 l + 1 (masked into range, as the other reorder kernels do),
    // gathered from the kept row through this row's LDS region.
    const float rb = rg[(64 * l) / g];
    const int c0 = (sblk[2 * l] & (NB - 1)) * kReorderBlock;
    const int c1 = (sblk[2 * l + 1] & (NB - 1)) * kReorderBlock;
#pragma unroll
    for (int p = 0; p < SLOTS; ++p) {
      const int r = row_of(p);
#pragma unroll
      for (int m = 0; m < 16; ++m)
        *reinterpret_cast<float4*>(row + lds_a(64 * l + 4 * m)) =
            make_float4(v[p][4 * m], v[p][4 * m + 1], v[p][4 * m + 2], v[p][4 * m + 3]);
      float* u = v[p];  // the natural order is in LDS now
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        const float4 x0 = *reinterpret_cast<const float4*>(row + lds_a(c0 + 4 * m));
        const float4 x1 = *reinterpret_cast<const float4*>(row + lds_a(c1 + 4 * m));
        u[4 * m] = x0.x;
        u[4 * m + 1] = x0.y;
        u[4 * m + 2] = x0.z;
        u[4 * m + 3] = x0.w;
        u[32 + 4 * m] = x1.x;
        u[32 + 4 * m + 1] = x1.y;
        u[32 + 4 * m + 2] = x1.z;
        u[32 + 4 * m + 3] = x1.w;
      }
      float x = 0.0f;
#pragma unroll
      for (int e = 0; e < 64; ++e) x = fmaxf(x, fabsf(u[e]));
      const float a = row_max<S::R>(x * rb);  // max over the row's groups of fl(M_ib r_b)
      const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
      const float mm = rb * inv;             // fl(r_b * inv_i)
      if (r < r1) {
        uint32_t wd[8];
#pragma unroll
        for (int w = 0; w < 8; ++w) wd[w] = quant_pack8(&u[8 * w], mm);
        uint4* dst = reinterpret_cast<uint4*>(Xq + (size_t)r * (K / 2) + 32 * l);
        dst[0] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
        dst[1] = make_uint4(wd[4], wd[5], wd[6], wd[7]);
        if (l == 0) a_scale[r] = failed ? __builtin_nanf("") : __fdiv_rn(a, 7.0f);
      }
    }
  } else {
    // The workgroup's group maxima: over slots, over the wave's rows (lanes with
    // the same l), over the g / 64 lanes of a group, then over the waves in LDS
    // (a fixed tree, no atomics); published as tagged entries.
    float pm = lm[0];
#pragma unroll
    for (int p = 1; p < SLOTS; ++p) pm = fmaxf(pm, lm[p]);
#pragma unroll
    for (int o = S::R; o < 64; o <<= 1) pm = fmaxf(pm, __shfl_xor(pm, o, 64));
    for (int o = 1; o < g / 64; o <<= 1) pm = fmaxf(pm, __shfl_xor(pm, o, 64));
    if (sub == 0 && (64 * l) % g == 0) wmax[wave][(64 * l) / g] = pm;
    if (tid == 0) {
      missed = 0;
      tag_lds = next_epoch(epoch);
    }
    __syncthreads();
    const uint32_t tag = tag_lds;
    if (tid < G) {
      float m = wmax[0][tid];
#pragma unroll
      for (int w = 1; w < WAVES; ++w) m = fmaxf(m, wmax[w][tid]);
      publish_tagged(tagged + (size_t)blockIdx.x * G + tid, tag, m);
    }

    float rb;  // r_b = fl(1 / s_b) of this lane's group
    // s_b = max over the nrows rows of maxima; r_b = fl(1 / s_b). Thread t takes
    // group t % G of rows t / G, t / G + NT / G, ...: the entries of a batch are
    // requested at once, and those whose tag is not set yet are requested again,
    // within a budget of max_polls rounds per batch.
    {
      // Entries per thread at most: 256 rows / (NT / G). One batch, except at
      // eight waves for g = 64 (two batches of 16: one more round trip, and the
      // words stay in registers next to the kept rows).
      constexpr int NE = 256 * (kWideG ? GMAX : GMAX / 2) / NT;
      constexpr int NEB = (WAVES == 8 && NE > 16) ? 16 : NE;
      const int b = tid % G;
      const int ns = NT / G;  // slices of rows
      const unsigned long long none = (unsigned long long)tag << 32;  // an absent row: 0.0
      float m = 0.0f;
      bool ok = true;
#pragma unroll
      for (int k0 = 0; k0 < NE; k0 += NEB) {
        unsigned long long x[NEB];
#pragma unroll
        for (int k = 0; k < NEB; ++k) {
          const int i = tid / G + (k0 + k) * ns;
          x[k] = i < nrows ? load_tagged(tagged + (size_t)i * G + b) : none;
        }
        bool bok = false;
        for (int round = 0;; ++round) {
          bok = true;
#pragma unroll
          for (int k = 0; k < NEB; ++k) bok = bok && has_tag(x[k], tag);
          if (bok || round >= max_polls) break;
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int k = 0; k < NEB; ++k) {
            const int i = tid / G + (k0 + k) * ns;
            if (!has_tag(x[k], tag)) x[k] = load_tagged(tagged + (size_t)i * G + b);
          }
        }
        ok = ok && bok;
#pragma unroll
        for (int k = 0; k < NEB; ++k) m = fmaxf(m, __uint_as_float((uint32_t)x[k]));
      }
      if (!ok) missed = 1;  // benign race: every writer writes 1
      red[tid] = m;
      __syncthreads();
      // Every word of the call has been read (or given up on): advance the epoch
      // (workgroup 0 only: one store instead of a contended one per workgroup).
      if (tid == 0) {
        if (missed)
          __hip_atomic_store(header + kFailWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (blockIdx.x == 0)
          __hip_atomic_store(header + kEpochWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      // Every lane reduces the slices of its own group (positions 64 l ..
      // 64 l + 63 lie in one group), so no barrier is needed before phase 2.
      const int gb = (64 * l) / g;
      float sv = red[gb];
      for (int q = 1; q < ns; ++q) sv = fmaxf(sv, red[q * G + gb]);
      rb = (sv == 0.0f) ? 0.0f : __fdiv_rn(1.0f, sv);
      if (blockIdx.x == 0 && tid < G) {
        float sg = red[tid];
        for (int q = 1; q < ns; ++q) sg = fmaxf(sg, red[q * G + tid]);
        s_group[tid] = missed ? __builtin_nanf("") : sg;
      }
    }
    const bool failed = missed != 0;  // uniform over the workgroup

    // Phase 2: token scale and codes of every kept row.
#pragma unroll
    for (int p = 0; p < SLOTS; ++p) {
      const int r = row_of(p);
      const float a = row_max<S::R>(lm[p] * rb);  // max over the row's groups of fl(M_ib r_b)
      const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
      const float m = rb * inv;                   // fl(r_b * inv_i)
      if (r < r1) {
        uint32_t wd[8];
#pragma unroll
        for (int w = 0; w < 8; ++w) wd[w] = quant_pack8(&v[p][8 * w], m);
        uint4* dst = reinterpret_cast<uint4*>(Xq + (size_t)r * (K / 2) + 32 * l);
        dst[0] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
        dst[1] = make_uint4(wd[4], wd[5], wd[6], wd[7]);
        if (l == 0) a_scale[r] = failed ? __builtin_nanf("") : __fdiv_rn(a, 7.0f);
      }
    }
  }
}

template <int K>
hipError_t launch_fused_k(const uint16_t* X, int M, int g, bool rot, uint8_t* Xq,
                          float* a_scale, float* s_group, void* workspace, int max_wgs,
                          int extra_rows, int max_polls, hipStream_t stream) {
  // Four waves per workgroup when one row per wave then still needs every
  // compute unit's workgroup (at 1024 x 4096 about 20 % faster than eight
  // waves on half of them) and g >= 128 (the four-wave form reads at most
  // K / 128 group maxima per row); otherwise eight waves, with two rows per
  // wave when one is not enough. One row per wave on two waves per SIMD
  // beats two rows per wave on one (at 2048 x 4096: 13.8 against 14.8 us).
  constexpr int RW = WaveRow<K>::RW;
  const bool wide = g < 128;
  const int waves = (M <= max_wgs * 4 * RW && !wide) ? 4 : kFusedWaves;
  const int per_slot = waves * RW;  // rows per workgroup per slot
  const int slots = M <= max_wgs * per_slot ? 1 : 2;
  const int rpw = slots * per_slot;
  const int wgs = (M + rpw - 1) / rpw;
  const int nrows = wgs + extra_rows;  // rows of maxima the readers wait for
  if (wgs > max_wgs || nrows > 256) return hipErrorInvalidValue;
  uint32_t* header = static_cast<uint32_t*>(workspace);
  unsigned long long* tagged =
      reinterpret_cast<unsigned long long*>(static_cast<char*>(workspace) + kQuantHeaderBytes);
  const int polls = max_polls > 0 ? max_polls : kFusedMaxPolls;
#define RRS_FUSED(R_, S_, W_, WG_)                                                 \
  rot_quant_fused_kernel<K, R_, S_, W_, WG_><<<wgs, W_ * 64, 0, stream>>>(         \
      X, M, g, rpw, header, tagged, nrows, polls, Xq, a_scale, s_group)
#define RRS_FUSED8(R_, WG_)                         \
  if (slots == 1)                                   \
    RRS_FUSED(R_, 1, kFusedWaves, WG_);             \
  else                                              \
    RRS_FUSED(R_, 2, kFusedWaves, WG_);
  if (waves == 4) {
    if (rot) RRS_FUSED(true, 1, 4, false); else RRS_FUSED(false, 1, 4, false);
  } else if (rot) {
    if (wide) { RRS_FUSED8(true, true) } else { RRS_FUSED8(true, false) }
  } else {
    if (wide) { RRS_FUSED8(false, true) } else { RRS_FUSED8(false, false) }
  }
#undef RRS_FUSED8
#undef RRS_FUSED
  return hipGetLastError();
}

// Rows of M per workgroup of `waves` waves, one row per wave where a grid of
// at most `cap` workgroups allows it; returns the grid size.
template <int K>
int wave_split(int M, int waves, int cap, int* rows_per_wg) {
  const int rows_wg_min = waves * WaveRow<K>::RW;
  int wgs = (M + rows_wg_min - 1) / rows_wg_min;
  wgs = wgs < cap ? wgs : cap;
  *rows_per_wg = (M + wgs - 1) / wgs;
  return (M + *rows_per_wg - 1) / *rows_per_wg;
}

template <int K>
hipError_t launch_wave(const uint16_t* X, int M, int g, const int32_t* perm, int flags, uint8_t* Xq,
                       float* a_scale, float* s_group, void* workspace, int max_partials,
                       int max_quant_wgs, hipStream_t stream) {
  // rot_max: at most max_partials workgroups (one partial row each).
  int rpw1 = 0, rpw2 = 0;
  const int wgs1 = wave_split<K>(M, kRotWaves, max_partials, &rpw1);
  // quant: one row per wave where the grid allows it.
  const int wgs2 = wave_split<K>(M, kQuantWaves, max_quant_wgs, &rpw2);
  float* gpart = static_cast<float*>(workspace);
  const bool rot = !(flags & kSkipRotation);
  const bool smooth = !(flags & kSkipSmoothing);
#define RRS_QUANT(R_, S_)                                                                 \
  quant_wave_kernel<K, R_, S_><<<wgs2, kQuantWaves * 64, 0, stream>>>(                    \
      X, M, g, rpw2, wgs1, perm, gpart, Xq, a_scale, s_group)
  if (smooth) {
    if (rot)
      rot_max_wave_kernel<K, true><<<wgs1, kRotWaves * 64, 0, stream>>>(X, M, g, rpw1, perm, gpart);
    else
      rot_max_wave_kernel<K, false><<<wgs1, kRotWaves * 64, 0, stream>>>(X, M, g, rpw1, perm, gpart);
  }
  if (rot && smooth) RRS_QUANT(true, true);
  else if (rot) RRS_QUANT(true, false);
  else if (smooth) RRS_QUANT(false, true);
  else RRS_QUANT(false, false);
#undef RRS_QUANT
  return hipGetLastError();
}

// Runtime reorder, pass 1: rot_max with groups of 32 natural-order channels
// writes the K / 32 block maxima per workgroup (P = K / 512 <= 8 positions per
// thread, 32 / P threads per block, K / 32 <= 128 blocks).
template <int K>
hipError_t launch_block_max_wave(const uint16_t* X, int M, bool rot, float* part,
                                 int max_partials, int* nrows, hipStream_t stream) {
  int rpw = 0;
  const int wgs = wave_split<K>(M, kRotWaves, max_partials, &rpw);
  if (rot)
    rot_max_wave_kernel<K, true><<<wgs, kRotWaves * 64, 0, stream>>>(X, M, 32, rpw, nullptr, part);
  else
    rot_max_wave_kernel<K, false><<<wgs, kRotWaves * 64, 0, stream>>>(X, M, 32, rpw, nullptr,
                                                                       part);
  *nrows = wgs;
  return hipGetLastError();
}

// Runtime reorder, pass 2: every workgroup orders the blocks from the nrows
// rows of block maxima itself, then quantizes its rows.
template <int K>
hipError_t launch_ordered_wave(const uint16_t* X, int M, int g, bool rot, const float* part,
                               int nrows, int max_quant_wgs, uint8_t* Xq, float* a_scale,
                               float* s_group, int32_t* block_order, hipStream_t stream) {
  int rpw = 0;
  const int wgs = wave_split<K>(M, kQuantWaves, max_quant_wgs, &rpw);
  if (rot)
    quant_wave_kernel<K, true, true, true><<<wgs, kQuantWaves * 64, 0, stream>>>(
        X, M, g, rpw, nrows, nullptr, part, Xq, a_scale, s_group, block_order);
  else
    quant_wave_kernel<K, false, true, true><<<wgs, kQuantWaves * 64, 0, stream>>>(
        X, M, g, rpw, nrows, nullptr, part, Xq, a_scale, s_group, block_order);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_block_maxima_wave(const uint16_t* X, int M, int K, bool rotate, float* part,
                                    int max_partials, int* nrows, hipStream_t stream) {
  switch (K) {
    case 512: return launch_block_max_wave<512>(X, M, rotate, part, max_partials, nrows, stream);
    case 1024: return launch_block_max_wave<1024>(X, M, rotate, part, max_partials, nrows, stream);
    case 2048: return launch_block_max_wave<2048>(X, M, rotate, part, max_partials, nrows, stream);
    case 4096: return launch_block_max_wave<4096>(X, M, rotate, part, max_partials, nrows, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_quantize_ordered_wave(const uint16_t* X, int M, int K, int g, bool rotate,
                                        const float* part, int nrows, int max_quant_wgs,
                                        uint8_t* Xq, float* a_scale, float* s_group,
                                        int32_t* block_order, hipStream_t stream) {
#define RRS_ORD_W(K_)                                                                     \
  launch_ordered_wave<K_>(X, M, g, rotate, part, nrows, max_quant_wgs, Xq, a_scale, s_group, \
                          block_order, stream)
  switch (K) {
    case 512: return RRS_ORD_W(512);
    case 1024: return RRS_ORD_W(1024);
    case 2048: return RRS_ORD_W(2048);
    case 4096: return RRS_ORD_W(4096);
    default: return hipErrorInvalidValue;
  }
#undef RRS_ORD_W
}

template <int K>
hipError_t launch_fused_order_k(const uint16_t* X, int M, int g, bool rot, uint8_t* Xq,
                                float* a_scale, float* s_group, int32_t* block_order,
                                uint32_t* header, unsigned long long* tagged,
                                unsigned long long* tagged2, int max_wgs, int extra_rows,
                                int max_polls, hipStream_t stream) {
  // Same shapes as the plain form (the block words need no more registers at
  // four waves than at eight).
  constexpr int RW = WaveRow<K>::RW;
  const int waves = M <= max_wgs * 4 * RW ? 4 : kFusedWaves;
  const int per_slot = waves * RW;
  const int slots = M <= max_wgs * per_slot ? 1 : 2;
  const int rpw = slots * per_slot;
  const int wgs = (M + rpw - 1) / rpw;
  const int nrows = wgs + extra_rows;  // rows of block words the readers wait for
  if (wgs > max_wgs || nrows > 256) return hipErrorInvalidValue;
  const int polls = max_polls > 0 ? max_polls : kFusedMaxPolls;
#define RRS_FUSED_O(R_, S_, W_)                                                                 \
  rot_quant_fused_kernel<K, R_, S_, W_, false, true><<<wgs, W_ * 64, 0, stream>>>(              \
      X, M, g, rpw, header, tagged, nrows, polls, Xq, a_scale, s_group, tagged2, block_order)
  if (waves == 4) {
    if (rot) RRS_FUSED_O(true, 1, 4); else RRS_FUSED_O(false, 1, 4);
  } else if (rot) {
    if (slots == 1) RRS_FUSED_O(true, 1, kFusedWaves); else RRS_FUSED_O(true, 2, kFusedWaves);
  } else {
    if (slots == 1) RRS_FUSED_O(false, 1, kFusedWaves); else RRS_FUSED_O(false, 2, kFusedWaves);
  }
#undef RRS_FUSED_O
  return hipGetLastError();
}

bool fused_quant_fits(int M, int K, int max_wgs) {
  if (K < 512 || K > 4096) return false;
  const int per_wg = 2 * kFusedWaves * (64 * 64 / K);  // two slots of rows per wave
  return M >= 1 && M <= max_wgs * per_wg;
}

hipError_t launch_rotate_smooth_quant_fused(const uint16_t* X, int M, int K, int g, bool rotate,
                                            uint8_t* Xq, float* a_scale, float* s_group,
                                            void* workspace, int max_wgs, hipStream_t stream,
                                            int extra_rows, int max_polls) {
  switch (K) {
#define RRS_FK(K_) \
  case K_: return launch_fused_k<K_>(X, M, g, rotate, Xq, a_scale, s_group, workspace, max_wgs, \
                                     extra_rows, max_polls, stream)
    RRS_FK(512);
    RRS_FK(1024);
    RRS_FK(2048);
    RRS_FK(4096);
#undef RRS_FK
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_rotate_smooth_quant_fused_order(const uint16_t* X, int M, int K, int g,
                                                  bool rotate, uint8_t* Xq, float* a_scale,
                                                  float* s_group, int32_t* block_order,
                                                  uint32_t* header, unsigned long long* tagged,
                                                  unsigned long long* tagged2, int max_wgs,
                                                  hipStream_t stream, int extra_rows,
                                                  int max_polls) {
  switch (K) {
#define RRS_FO(K_)                                                                            \
  case K_: return launch_fused_order_k<K_>(X, M, g, rotate, Xq, a_scale, s_group, block_order, \
                                           header, tagged, tagged2, max_wgs, extra_rows,       \
                                           max_polls, stream)
    RRS_FO(512);
    RRS_FO(1024);
    RRS_FO(2048);
    RRS_FO(4096);
#undef RRS_FO
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_rotate_smooth_quant_wave(const uint16_t* X, int M, int K, int g,
                                           const int32_t* perm, int flags, uint8_t* Xq,
                                           float* a_scale, float* s_group, void* workspace,
                                           int max_partials, int max_quant_wgs,
                                           hipStream_t stream) {
  switch (K) {
    case 512: return launch_wave<512>(X, M, g, perm, flags, Xq, a_scale, s_group, workspace, max_partials, max_quant_wgs, stream);
    case 1024: return launch_wave<1024>(X, M, g, perm, flags, Xq, a_scale, s_group, workspace, max_partials, max_quant_wgs, stream);
    case 2048: return launch_wave<2048>(X, M, g, perm, flags, Xq, a_scale, s_group, workspace, max_partials, max_quant_wgs, stream);
    case 4096: return launch_wave<4096>(X, M, g, perm, flags, Xq, a_scale, s_group, workspace, max_partials, max_quant_wgs, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rrs
