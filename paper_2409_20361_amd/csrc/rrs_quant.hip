// Online rotate + runtime smooth + per-token INT4 quantization
// (Section 3.3 then Section 3.2; Eq. 1-2; Section 2.1).
//
// The smoothing scale of group b is the largest |rotated activation| over
// every token of the call and every channel of the group (Eq. 1 with the
// group maximum of Section 3.2), so no token can be quantized before all
// tokens are rotated. Two launches on the caller's stream:
//   1. rot_max: each workgroup rotates its rows (FWHT, canonical stage order),
//      keeps per-channel maxima in registers, combines its teams in LDS, and
//      writes one row of per-group maxima (G floats; with a static reorder the
//      groups are formed over the reordered positions);
//   2. quant: each workgroup reduces those rows to s_b and r_b = fl(1/s_b),
//      then re-rotates its rows (identical code, identical bits; X mostly
//      comes from the MALL the second time), takes the per-token maximum of
//      fl(|y_ij| r_b), and writes alpha_i and the packed INT4 codes.
// In this file a workgroup holds 1, 2 or 4 teams of 256 threads (K = 16384,
// 8192, <= 2048: a thread's share of a row stays in registers); each team
// works on one row at a time. Cross-team and cross-wave reductions go through
// LDS, no atomics. K = 4096 (and K = 2048 with many rows) takes the
// one-wave-per-row kernels of rrs_quant_wave.hip instead.
#include "rrs_device.h"
#include "rrs_internal.h"

namespace rrs {
namespace {

constexpr int kMaxPartialRows = 256;

template <int K>
struct Teams {
  static constexpr int n = K <= 4096 ? 4 : (K == 8192 ? 2 : 1);
  static constexpr int threads = n * kRowThreads;
};

// Row slots: one padded row per team, at least 1024 floats in all, so the
// same LDS doubles as reduction scratch (indexed by channel and by thread)
// when no row is in flight.
template <int K>
constexpr int slot_floats() {
  return Teams<K>::n * lds_row_floats(K) > 1024 ? Teams<K>::n * lds_row_floats(K) : 1024;
}

// v = row r of X (this thread's E elements), or zeros past the last row r1.
template <int K>
__device__ __forceinline__ void load_row_or_zero(const uint16_t* __restrict__ X, int r, int r1,
                                                 int t, float (&v)[FwhtShape<K>::E]) {
  constexpr int E = FwhtShape<K>::E;
  if (r < r1) {
    load_halves<E>(X + (size_t)r * K + (size_t)t * E, v);
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = 0.0f;
  }
}

// Per-channel maxima cm (this thread's E channels t + 256 e) of every team
// combined into cbuf[0, K). Must be called by all threads of the workgroup;
// cbuf holds >= K floats.
template <int K, int kTeams = Teams<K>::n>
__device__ __forceinline__ void combine_teams(const float (&cm)[FwhtShape<K>::E], float* cbuf) {
  constexpr int E = FwhtShape<K>::E;
  const int tid = threadIdx.x;
  const int team = tid >> 8;
  const int t = tid & (kRowThreads - 1);
  __syncthreads();
  if (team == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) cbuf[t + e * kRowThreads] = cm[e];
  }
  __syncthreads();
  for (int tm = 1; tm < kTeams; ++tm) {
    if (team == tm) {
#pragma unroll
      for (int e = 0; e < E; ++e)
        cbuf[t + e * kRowThreads] = fmaxf(cbuf[t + e * kRowThreads], cm[e]);
    }
    __syncthreads();
  }
}

// Per-channel maxima of every team combined (combine_teams), then maxima over
// each group of g (reordered) positions. Returns, for threads tid < K / g, the
// maximum of group tid; 0 elsewhere. Must be called by all threads of the
// workgroup; cbuf holds >= K floats.
template <int K, int kTeams = Teams<K>::n>
__device__ __forceinline__ float group_maxima(const float (&cm)[FwhtShape<K>::E], float* cbuf,
                                              int g, const int32_t* __restrict__ perm) {
  constexpr int kThreads = kTeams * kRowThreads;
  const int tid = threadIdx.x;
  combine_teams<K, kTeams>(cm, cbuf);
  // The first NA threads cover P consecutive positions each, all inside one
  // group (P <= 64 <= g).
  constexpr int NA = K < kThreads ? K : kThreads;
  constexpr int P = K / NA;
  float pm = 0.0f;
  if (tid < NA) {
#pragma unroll
    for (int q = 0; q < P; ++q) {
      const int j = tid * P + q;
      pm = fmaxf(pm, cbuf[perm ? perm[j] : j]);
    }
  }
  __syncthreads();
  cbuf[tid] = pm;  // tid < kThreads <= slot_floats
  __syncthreads();
  const int G = K / g;
  float s = 0.0f;
  if (tid < G) {
    const int per = g / P;  // threads per group
    for (int u = 0; u < per; ++u) s = fmaxf(s, cbuf[tid * per + u]);
  }
  __syncthreads();  // cbuf may be reused by the caller
  return s;
}

// ---------------------------------------------------------------------------
// 1. rotate + per-workgroup group maxima
// ---------------------------------------------------------------------------
// kBlocks (runtime reorder): the row written holds instead the maxima of the
// K / 32 blocks of 32 consecutive channels, in natural order (g and perm are
// not used).
template <int K, bool kRot, bool kBlocks = false>
__global__ __launch_bounds__(Teams<K>::threads) void rot_max_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg,
    const int32_t* __restrict__ perm, float* __restrict__ gpart) {
  using S = FwhtShape<K>;
  constexpr int E = S::E;
  constexpr int RF = lds_row_floats(K);
  constexpr int kTeams = Teams<K>::n;
  __shared__ float slots[slot_floats<K>()];
  float* cbuf = slots;  // reduction scratch once the rows are done
  const int tid = threadIdx.x;
  const int team = tid >> 8;
  const int t = tid & (kRowThreads - 1);
  const int iters = (rows_per_wg + kTeams - 1) / kTeams;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  float* slot = slots + team * RF;

  float cm[E];
#pragma unroll
  for (int e = 0; e < E; ++e) cm[e] = 0.0f;
  float vn[E];  // next row, loaded while the current one is transformed
  load_row_or_zero<K>(X, r0 + team, r1, t, vn);
  for (int it = 0; it < iters; ++it) {
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = vn[e];
    if (it + 1 < iters) load_row_or_zero<K>(X, r0 + (it + 1) * kTeams + team, r1, t, vn);
    fwht_row<K, kRot>(v, slot, t);  // v[e] = y[t + 256 e]
#pragma unroll
    for (int e = 0; e < E; ++e) cm[e] = fmaxf(cm[e], fabsf(v[e]));
  }
  if constexpr (kBlocks) {
    combine_teams<K>(cm, cbuf);
    float* out = gpart + (size_t)blockIdx.x * (K / 32);
    for (int B = tid; B < K / 32; B += Teams<K>::threads) {
      float m = 0.0f;
      // start at a different channel per thread: fewer LDS bank conflicts
      for (int q = 0; q < 32; ++q) m = fmaxf(m, cbuf[B * 32 + ((q + B) & 31)]);
      out[B] = m;
    }
  } else {
    const float s = group_maxima<K>(cm, cbuf, g, perm);
    if (tid < K / g) gpart[(size_t)blockIdx.x * (K / g) + tid] = s;
  }
}

// ---------------------------------------------------------------------------
// 2. group scales, per-token scale, codes
// ---------------------------------------------------------------------------
// kOrder (runtime reorder): gpart holds nparts rows of K/32 block maxima; the
// workgroup ranks the blocks itself (block_order_wg), takes s_b over the
// sorted blocks of group b and reads position j from channel
// 32 sblk[j / 32] + j % 32; workgroup 0 writes s_group and block_order.
template <int K, bool kRot, bool kSmooth, bool kOrder = false>
__global__ __launch_bounds__(Teams<K>::threads) void quant_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg, int nparts,
    const int32_t* __restrict__ perm, const float* __restrict__ gpart,
    uint8_t* __restrict__ Xq, float* __restrict__ a_scale, float* __restrict__ s_group,
    int32_t* __restrict__ block_order = nullptr) {
  using S = FwhtShape<K>;
  constexpr int E = S::E;
  constexpr int RF = lds_row_floats(K);
  constexpr int kTeams = Teams<K>::n;
  constexpr int kThreads = Teams<K>::threads;
  constexpr int NB = K / kReorderBlock;
  __shared__ __attribute__((aligned(16))) float slots[slot_floats<K>()];
  __shared__ float rg[256];
  __shared__ float red[16];
  __shared__ __attribute__((aligned(16))) unsigned long long key[kOrder ? NB : 2];
  __shared__ __attribute__((aligned(16))) unsigned long long srt[kOrder ? NB : 2];
  __shared__ float skey[kOrder ? NB : 1];
  __shared__ int sblk[kOrder ? NB : 1];
  __shared__ __attribute__((aligned(16))) float ored[kOrder ? 4 * kThreads : 4];
  float* cbuf = slots;  // reduction scratch before the rows start
  const int tid = threadIdx.x;
  const int team = tid >> 8;
  const int t = tid & (kRowThreads - 1);
  const int G = K / g;
  float* slot = slots + team * RF;

  // This team's first row is requested before anything else, so its load
  // latency overlaps the reduction below.
  const int iters = (rows_per_wg + kTeams - 1) / kTeams;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  float vn[E];  // next row, loaded while the current one is processed
  load_row_or_zero<K>(X, r0 + team, r1, t, vn);

  if constexpr (!kSmooth) {
    // Ablation without smoothing: every scale is 1 (rotation + per-token only).
    if (tid < G) {
      rg[tid] = 1.0f;
      if (blockIdx.x == 0) s_group[tid] = 1.0f;
    }
    __syncthreads();
  } else if constexpr (kOrder) {
    block_order_wg<kThreads, NB>(gpart, nparts, ored, key, srt, sblk, skey, tid);
    if (tid < G) {
      const int per = g / kReorderBlock;
      float s = 0.0f;
      for (int u = 0; u < per; ++u) s = fmaxf(s, skey[tid * per + u]);
      rg[tid] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
      if (blockIdx.x == 0) s_group[tid] = s;
    }
    if (blockIdx.x == 0)
      for (int b = tid; b < NB; b += kThreads) block_order[b] = sblk[b];
    __syncthreads();
  } else {
    // s_b = max over the partial rows; threads split (group, row slice) and
    // issue their loads eight at a time so the latencies overlap.
    const int nsl = kThreads / G;  // G <= 256 <= kThreads
    const int b = tid % G;
    const int sl = tid / G;
    float m = 0.0f;
    if (sl < nsl) {
      int i = sl;
      for (; i + 7 * nsl < nparts; i += 8 * nsl) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = gpart[(size_t)(i + u * nsl) * G + b];
#pragma unroll
        for (int u = 0; u < 8; ++u) m = fmaxf(m, x[u]);
      }
      for (; i < nparts; i += nsl) m = fmaxf(m, gpart[(size_t)i * G + b]);
    }
    cbuf[tid] = m;
    __syncthreads();
    if (tid < G) {
      float s = cbuf[tid];
      for (int q = 1; q < nsl; ++q) s = fmaxf(s, cbuf[q * G + tid]);
      rg[tid] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
      if (blockIdx.x == 0) s_group[tid] = s;
    }
    __syncthreads();
  }
  int src[E];  // position t*E + e of the reordered row reads channel src[e]
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int j = t * E + e;
    if constexpr (kOrder)  // masked into range, whatever the partial rows held
      src[e] = (sblk[j / kReorderBlock] & (NB - 1)) * kReorderBlock + j % kReorderBlock;
    else
      src[e] = perm ? perm[j] : j;
  }
  const float rb = rg[(t * E) / g];  // this thread's positions lie in one group

  for (int it = 0; it < iters; ++it) {
    const int r = r0 + it * kTeams + team;
    const bool live = r < r1;
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = vn[e];
    if (it + 1 < iters) load_row_or_zero<K>(X, r0 + (it + 1) * kTeams + team, r1, t, vn);
    fwht_row<K, kRot>(v, slot, t);
    // back to natural order through LDS, with the static reorder applied
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) slot[lds_pad(t + e * kRowThreads)] = v[e];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = slot[lds_pad(src[e])];
    float lm = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
    lm = wave_max(lm * rb);  // fl(M_ib * r_b), max over the wave
    if ((tid & 63) == 0) red[tid >> 6] = lm;
    __syncthreads();
    const float a = fmaxf(fmaxf(red[team * 4], red[team * 4 + 1]),
                          fmaxf(red[team * 4 + 2], red[team * 4 + 3]));  // 4 waves per team
    const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
    const float m = rb * inv;  // fl(r_b * inv_i)
    if (live) {
      uint32_t nib[E];
#pragma unroll
      for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * m);
      store_nibbles<E>(Xq + (size_t)r * (K / 2) + (size_t)t * (E / 2), nib);
      if (t == 0) a_scale[r] = __fdiv_rn(a, 7.0f);
    }
  }
}

// ---------------------------------------------------------------------------
// Few tokens (M <= 16) in one launch: every workgroup rotates all M rows and
// takes the channel maxima itself (the same values in every workgroup), so no
// partial rows go through global memory and the second launch disappears.
// Team `team` of workgroup w quantizes row w * kTeams + team, which it rotated
// in iteration w of the first loop and kept in registers.
// ---------------------------------------------------------------------------
template <int K>
struct FewTeams {
  // four row teams where the registers allow it (a thread keeps three rows'
  // worth of E values: the row in flight, its channel maxima and its own row)
  static constexpr int n = K <= 4096 ? 4 : (K == 8192 ? 2 : 1);
  static constexpr int threads = n * kRowThreads;
  static constexpr int slot_floats =
      n * lds_row_floats(K) > 1024 ? n * lds_row_floats(K) : 1024;
};

// Largest M for which the one-launch kernel beats the two launches. Every
// workgroup rotates all M rows, ceil(M / teams) of them one after another,
// while the two-launch path spreads the rows over workgroups but pays a second
// launch; the crossover was measured on MI355X (events, back to back).
constexpr int few_max_rows(int K) {
  return K <= 2048 ? 16 : (K == 4096 ? 8 : (K == 8192 ? 4 : 2));
}

// Raw fp16 halves of this thread's E elements of row r (zeros past the last row).
template <int E>
__device__ __forceinline__ void load_raw_or_zero(const uint16_t* __restrict__ X, int K, int r,
                                                 int M, int t, uint32_t (&raw)[E / 2]) {
  if (r < M) {
    const uint16_t* src = X + (size_t)r * K + (size_t)t * E;
    if constexpr (E >= 8) {
#pragma unroll
      for (int c = 0; c < E / 8; ++c) {
        const uint4 w = reinterpret_cast<const uint4*>(src)[c];
        raw[4 * c] = w.x;
        raw[4 * c + 1] = w.y;
        raw[4 * c + 2] = w.z;
        raw[4 * c + 3] = w.w;
      }
    } else if constexpr (E == 4) {
      const uint2 w = *reinterpret_cast<const uint2*>(src);
      raw[0] = w.x;
      raw[1] = w.y;
    } else {
      raw[0] = *reinterpret_cast<const uint32_t*>(src);
    }
  } else {
#pragma unroll
    for (int i = 0; i < E / 2; ++i) raw[i] = 0u;
  }
}

template <int K, bool kRot>
__global__ __launch_bounds__(FewTeams<K>::threads) void quant_few_kernel(
    const uint16_t* __restrict__ X, int M, int g, const int32_t* __restrict__ perm,
    uint8_t* __restrict__ Xq, float* __restrict__ a_scale, float* __restrict__ s_group) {
  using S = FwhtShape<K>;
  constexpr int E = S::E;
  constexpr int RF = lds_row_floats(K);
  constexpr int kTeams = FewTeams<K>::n;
  __shared__ float slots[FewTeams<K>::slot_floats];
  __shared__ float rg[256];
  __shared__ float red[4 * kTeams];
  float* cbuf = slots;  // reduction scratch between the two phases
  const int tid = threadIdx.x;
  const int team = tid >> 8;
  const int t = tid & (kRowThreads - 1);
  const int G = K / g;
  float* slot = slots + team * RF;
  const int iters = (M + kTeams - 1) / kTeams;  // == gridDim.x
  const int own = blockIdx.x * kTeams + team;

  // 1. every row of the call: rotate, channel maxima; keep this team's own row
  float cm[E], keep[E];
#pragma unroll
  for (int e = 0; e < E; ++e) cm[e] = 0.0f;
  uint32_t raw[E / 2];  // next row, loaded while the current one is transformed
  load_raw_or_zero<E>(X, K, team, M, t, raw);
  for (int it = 0; it < iters; ++it) {
    float v[E];
#pragma unroll
    for (int i = 0; i < E / 2; ++i) {
      v[2 * i] = half_to_float(raw[i] & 0xFFFFu);
      v[2 * i + 1] = half_to_float(raw[i] >> 16);
    }
    if (it + 1 < iters) load_raw_or_zero<E>(X, K, (it + 1) * kTeams + team, M, t, raw);
    fwht_row<K, kRot>(v, slot, t);  // v[e] = y[t + 256 e]
#pragma unroll
    for (int e = 0; e < E; ++e) cm[e] = fmaxf(cm[e], fabsf(v[e]));
    if (it == (int)blockIdx.x) {  // uniform across the workgroup
#pragma unroll
      for (int e = 0; e < E; ++e) keep[e] = v[e];
    }
  }
  const float smax = group_maxima<K, kTeams>(cm, cbuf, g, perm);
  if (tid < G) {
    rg[tid] = (smax == 0.0f) ? 0.0f : __fdiv_rn(1.0f, smax);
    if (blockIdx.x == 0) s_group[tid] = smax;
  }
  __syncthreads();

  // 2. this team's own row, exactly as the second pass of the two-launch path
  const float rb = rg[(t * E) / g];  // this thread's positions lie in one group
#pragma unroll
  for (int e = 0; e < E; ++e) slot[lds_pad(t + e * kRowThreads)] = keep[e];
  __syncthreads();
  float v[E];
#pragma unroll
  for (int e = 0; e < E; ++e) v[e] = slot[lds_pad(perm ? perm[t * E + e] : t * E + e)];
  float lm = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
  lm = wave_max(lm * rb);  // fl(M_ib * r_b), max over the wave
  if ((tid & 63) == 0) red[tid >> 6] = lm;
  __syncthreads();
  const float a = fmaxf(fmaxf(red[team * 4], red[team * 4 + 1]),
                        fmaxf(red[team * 4 + 2], red[team * 4 + 3]));  // 4 waves per team
  const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
  const float m = rb * inv;  // fl(r_b * inv_i)
  if (own < M) {
    uint32_t nib[E];
#pragma unroll
    for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * m);
    store_nibbles<E>(Xq + (size_t)own * (K / 2) + (size_t)t * (E / 2), nib);
    if (t == 0) a_scale[own] = __fdiv_rn(a, 7.0f);
  }
}

// ---------------------------------------------------------------------------
// Sub-channel baseline (Section 2.1, Section 4.5): every (token, group of g
// channels) gets its own scale; no smoothing and no cross-token dependency,
// so one launch. y = x H_K (or x), m = max_{j in group} |y_j|,
// inv = fl(7 / m) (0 if m = 0), code = clamp(rint(fl(y * inv)), -7, 7),
// a_sub[b * M + i] = fl(m / 7) (group-major, L x M).
// ---------------------------------------------------------------------------
template <int K, bool kRot>
__global__ __launch_bounds__(Teams<K>::threads) void subchan_quant_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg, uint8_t* __restrict__ Xq,
    float* __restrict__ a_sub) {
  using S = FwhtShape<K>;
  constexpr int E = S::E;
  constexpr int RF = lds_row_floats(K);
  constexpr int kTeams = Teams<K>::n;
  __shared__ float slots[slot_floats<K>()];
  __shared__ float red[kTeams][256];
  __shared__ float gm[kTeams][256];
  const int tid = threadIdx.x;
  const int team = tid >> 8;
  const int t = tid & (kRowThreads - 1);
  const int G = K / g;
  float* slot = slots + team * RF;
  const int iters = (rows_per_wg + kTeams - 1) / kTeams;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  float vn[E];
  load_row_or_zero<K>(X, r0 + team, r1, t, vn);
  for (int it = 0; it < iters; ++it) {
    const int r = r0 + it * kTeams + team;
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = vn[e];
    if (it + 1 < iters) load_row_or_zero<K>(X, r0 + (it + 1) * kTeams + team, r1, t, vn);
    fwht_row<K, kRot>(v, slot, t);
    // back to natural order: thread t takes channels [t E, t E + E)
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) slot[lds_pad(t + e * kRowThreads)] = v[e];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = slot[lds_pad(t * E + e)];
    float lm = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
    const float m = row_group_max(lm, red[team], gm[team], t, E, g, G);
    const float inv = (m == 0.0f) ? 0.0f : __fdiv_rn(7.0f, m);
    if (r < r1) {
      uint32_t nib[E];
#pragma unroll
      for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * inv);
      store_nibbles<E>(Xq + (size_t)r * (K / 2) + (size_t)t * (E / 2), nib);
      if ((t * E) % g == 0) a_sub[(size_t)((t * E) / g) * M + r] = __fdiv_rn(m, 7.0f);
    }
  }
}

int num_cus();
inline int num_cus_sub() { return num_cus(); }

template <int K>
hipError_t launch_sub_k(const uint16_t* X, int M, int g, bool rot, uint8_t* Xq, float* a_sub,
                        hipStream_t stream) {
  constexpr int kTeams = Teams<K>::n;
  int wgs = (M + kTeams - 1) / kTeams;
  wgs = wgs < 4 * num_cus_sub() ? wgs : 4 * num_cus_sub();
  const int rpw = (M + wgs - 1) / wgs;
  wgs = (M + rpw - 1) / rpw;
  if (rot)
    subchan_quant_kernel<K, true><<<wgs, Teams<K>::threads, 0, stream>>>(X, M, g, rpw, Xq, a_sub);
  else
    subchan_quant_kernel<K, false><<<wgs, Teams<K>::threads, 0, stream>>>(X, M, g, rpw, Xq, a_sub);
  return hipGetLastError();
}

int g_num_cus = 0;

int num_cus() {
  if (g_num_cus == 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus > 0)
      g_num_cus = cus;
    else
      g_num_cus = 256;
  }
  return g_num_cus;
}

// Rows of M per workgroup for a grid of at most `cap` workgroups of kTeams
// teams (one row per team where the cap allows); returns the grid size.
// Pass 1 writes one partial row per workgroup: at most kMaxPartialRows of
// them, so the reduction every pass-2 workgroup repeats stays small. Pass 2
// has no such limit: up to 4 workgroups per CU.
template <int K>
int split_rows(int M, int cap, int* rows_per_wg) {
  constexpr int kTeams = Teams<K>::n;
  int wgs = (M + kTeams - 1) / kTeams;
  wgs = wgs < cap ? wgs : cap;
  *rows_per_wg = (M + wgs - 1) / wgs;
  return (M + *rows_per_wg - 1) / *rows_per_wg;
}

template <int K>
hipError_t launch_k(const uint16_t* X, int M, int g, const int32_t* perm, int flags, uint8_t* Xq,
                    float* a_scale, float* s_group, void* workspace, hipStream_t stream) {
  int rpw1 = 0, rpw2 = 0;
  const int wgs1 = split_rows<K>(M, kMaxPartialRows, &rpw1);
  // One pass-2 workgroup per compute unit: each re-reads the partial rows, so
  // more workgroups pay that reduction more often (measured at K = 8192,
  // M = 8192: 154.8 us for the call against 160.5 us with two per CU and
  // 173.4 us with four; K = 16384, M = 2048: 128.9 against 148.9 us).
  const int wgs2 = split_rows<K>(M, num_cus(), &rpw2);
  float* gpart = static_cast<float*>(workspace);
  const bool rot = !(flags & kSkipRotation);
  const bool smooth = !(flags & kSkipSmoothing);
#define RRS_QUANT(R_, S_)                                                                   \
  quant_kernel<K, R_, S_><<<wgs2, Teams<K>::threads, 0, stream>>>(X, M, g, rpw2, wgs1, perm, \
                                                                  gpart, Xq, a_scale, s_group)
  if (smooth) {
    if (rot)
      rot_max_kernel<K, true><<<wgs1, Teams<K>::threads, 0, stream>>>(X, M, g, rpw1, perm, gpart);
    else
      rot_max_kernel<K, false><<<wgs1, Teams<K>::threads, 0, stream>>>(X, M, g, rpw1, perm, gpart);
  }
  if (rot && smooth) RRS_QUANT(true, true);
  else if (rot) RRS_QUANT(true, false);
  else if (smooth) RRS_QUANT(false, true);
  else RRS_QUANT(false, false);
#undef RRS_QUANT
  return hipGetLastError();
}

// Runtime reorder, pass 1: block maxima rows (see rot_max_kernel's kBlocks).
template <int K>
hipError_t launch_block_max_k(const uint16_t* X, int M, bool rot, float* part, int* nrows,
                              hipStream_t stream) {
  int rpw = 0;
  const int wgs = split_rows<K>(M, kMaxPartialRows, &rpw);
  if (rot)
    rot_max_kernel<K, true, true><<<wgs, Teams<K>::threads, 0, stream>>>(X, M, 32, rpw, nullptr,
                                                                          part);
  else
    rot_max_kernel<K, false, true><<<wgs, Teams<K>::threads, 0, stream>>>(X, M, 32, rpw, nullptr,
                                                                           part);
  *nrows = wgs;
  return hipGetLastError();
}

// Runtime reorder, pass 2: quant with one given row of group maxima.
template <int K>
hipError_t launch_ordered_k(const uint16_t* X, int M, int g, bool rot, const float* part,
                            int nrows, uint8_t* Xq, float* a_scale, float* s_group,
                            int32_t* block_order, hipStream_t stream) {
  int rpw = 0;
  const int wgs = split_rows<K>(M, num_cus(), &rpw);  // as launch_k's second pass
  if (rot)
    quant_kernel<K, true, true, true><<<wgs, Teams<K>::threads, 0, stream>>>(
        X, M, g, rpw, nrows, nullptr, part, Xq, a_scale, s_group, block_order);
  else
    quant_kernel<K, false, true, true><<<wgs, Teams<K>::threads, 0, stream>>>(
        X, M, g, rpw, nrows, nullptr, part, Xq, a_scale, s_group, block_order);
  return hipGetLastError();
}

// One wave per row wins at K = 4096, and at K = 2048 once there are enough
// rows; elsewhere the team kernels are faster (measured).
bool use_wave_kernels(int M, int K) { return K == 4096 || (K == 2048 && M >= 512); }

}  // namespace

hipError_t launch_block_maxima(const uint16_t* X, int M, int K, bool rotate, float* part,
                               int* nrows, hipStream_t stream) {
  if (use_wave_kernels(M, K))
    return launch_block_maxima_wave(X, M, K, rotate, part, kMaxPartialRows, nrows, stream);
  switch (K) {
    case 512: return launch_block_max_k<512>(X, M, rotate, part, nrows, stream);
    case 1024: return launch_block_max_k<1024>(X, M, rotate, part, nrows, stream);
    case 2048: return launch_block_max_k<2048>(X, M, rotate, part, nrows, stream);
    case 8192: return launch_block_max_k<8192>(X, M, rotate, part, nrows, stream);
    case 16384: return launch_block_max_k<16384>(X, M, rotate, part, nrows, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_quantize_ordered(const uint16_t* X, int M, int K, int g, bool rotate,
                                   const float* part, int nrows, uint8_t* Xq, float* a_scale,
                                   float* s_group, int32_t* block_order, hipStream_t stream) {
  if (use_wave_kernels(M, K))
    return launch_quantize_ordered_wave(X, M, K, g, rotate, part, nrows, 2 * num_cus(), Xq,
                                        a_scale, s_group, block_order, stream);
#define RRS_ORD_K(K_) \
  launch_ordered_k<K_>(X, M, g, rotate, part, nrows, Xq, a_scale, s_group, block_order, stream)
  switch (K) {
    case 512: return RRS_ORD_K(512);
    case 1024: return RRS_ORD_K(1024);
    case 2048: return RRS_ORD_K(2048);
    case 8192: return RRS_ORD_K(8192);
    case 16384: return RRS_ORD_K(16384);
    default: return hipErrorInvalidValue;
  }
#undef RRS_ORD_K
}

int block_maxima_rows() { return kMaxPartialRows; }

hipError_t launch_quantize_sub_channel(const uint16_t* X, int M, int K, int g, int flags,
                                       uint8_t* Xq, float* a_sub, hipStream_t stream) {
  const bool rot = !(flags & kSkipRotation);
  switch (K) {
    case 512: return launch_sub_k<512>(X, M, g, rot, Xq, a_sub, stream);
    case 1024: return launch_sub_k<1024>(X, M, g, rot, Xq, a_sub, stream);
    case 2048: return launch_sub_k<2048>(X, M, g, rot, Xq, a_sub, stream);
    case 4096: return launch_sub_k<4096>(X, M, g, rot, Xq, a_sub, stream);
    case 8192: return launch_sub_k<8192>(X, M, g, rot, Xq, a_sub, stream);
    case 16384: return launch_sub_k<16384>(X, M, g, rot, Xq, a_sub, stream);
    default: return hipErrorInvalidValue;
  }
}

int quant_partial_rows(int M) { return M < kMaxPartialRows ? M : kMaxPartialRows; }

int fused_quant_wgs() { return num_cus() < kMaxPartialRows ? num_cus() : kMaxPartialRows; }

bool fused_quant_used(int M, int K, int g, const int32_t* perm, int flags) {
  (void)g;
  return !quant_rows_used(M, K, g, perm, flags) && M > few_max_rows(K) && !perm &&
         !(flags & kSkipSmoothing) && fused_quant_fits(M, K, fused_quant_wgs());
}

size_t quant_workspace_bytes(int M, int K) {
  (void)M;
  // header and tagged entries of the one-launch kernels, then the two-pass
  // kernels' partial rows (at most 256 rows of K / 64 floats)
  return quant_two_pass_offset(K) + align256((size_t)kMaxPartialRows * (K / 64) * 4);
}

namespace {

template <int K>
hipError_t launch_few_k(const uint16_t* X, int M, int g, const int32_t* perm, bool rot,
                        uint8_t* Xq, float* a_scale, float* s_group, hipStream_t stream) {
  const int grid = (M + FewTeams<K>::n - 1) / FewTeams<K>::n;
  if (rot)
    quant_few_kernel<K, true><<<grid, FewTeams<K>::threads, 0, stream>>>(X, M, g, perm, Xq,
                                                                         a_scale, s_group);
  else
    quant_few_kernel<K, false><<<grid, FewTeams<K>::threads, 0, stream>>>(X, M, g, perm, Xq,
                                                                          a_scale, s_group);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rotate_smooth_quant(const uint16_t* X, int M, int K, int g,
                                      const int32_t* perm, int flags, uint8_t* Xq,
                                      float* a_scale, float* s_group, void* workspace,
                                      hipStream_t stream) {
  // Up to 16 tokens with smoothing and no static reorder: one workgroup per
  // row, the rows' group maxima exchanged in the workspace (rrs_quant_rows.hip).
  if (quant_rows_used(M, K, g, perm, flags))
    return launch_quant_rows(X, M, K, g, !(flags & kSkipRotation), Xq, a_scale, s_group,
                             workspace, stream);
  // Few tokens with smoothing: one launch (each workgroup takes the channel
  // maxima of all rows itself).
  if (M <= few_max_rows(K) && !(flags & kSkipSmoothing)) {
    const bool rot = !(flags & kSkipRotation);
    switch (K) {
      case 512: return launch_few_k<512>(X, M, g, perm, rot, Xq, a_scale, s_group, stream);
      case 1024: return launch_few_k<1024>(X, M, g, perm, rot, Xq, a_scale, s_group, stream);
      case 2048: return launch_few_k<2048>(X, M, g, perm, rot, Xq, a_scale, s_group, stream);
      case 4096: return launch_few_k<4096>(X, M, g, perm, rot, Xq, a_scale, s_group, stream);
      case 8192: return launch_few_k<8192>(X, M, g, perm, rot, Xq, a_scale, s_group, stream);
      case 16384: return launch_few_k<16384>(X, M, g, perm, rot, Xq, a_scale, s_group, stream);
      default: return hipErrorInvalidValue;
    }
  }
  // K <= 4096 without a static reorder: one launch, every row rotated once
  // (rrs_quant_wave.hip), for up to two rows per wave on one workgroup per
  // compute unit.
  if (fused_quant_used(M, K, g, perm, flags))
    return launch_rotate_smooth_quant_fused(X, M, K, g, !(flags & kSkipRotation), Xq, a_scale,
                                            s_group, workspace, fused_quant_wgs(), stream);
  // The two-pass kernels keep their partial rows clear of the one-launch
  // kernels' header and tagged entries.
  void* tp = static_cast<char*>(workspace) + quant_two_pass_offset(K);
  if (use_wave_kernels(M, K))
    return launch_rotate_smooth_quant_wave(X, M, K, g, perm, flags, Xq, a_scale, s_group, tp,
                                           kMaxPartialRows, 2 * num_cus(), stream);
  switch (K) {
    case 512: return launch_k<512>(X, M, g, perm, flags, Xq, a_scale, s_group, tp, stream);
    case 1024: return launch_k<1024>(X, M, g, perm, flags, Xq, a_scale, s_group, tp, stream);
    case 2048: return launch_k<2048>(X, M, g, perm, flags, Xq, a_scale, s_group, tp, stream);
    case 8192: return launch_k<8192>(X, M, g, perm, flags, Xq, a_scale, s_group, tp, stream);
    case 16384: return launch_k<16384>(X, M, g, perm, flags, Xq, a_scale, s_group, tp, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rrs
