// rotate + smooth + quant for a handful of tokens (Section 3.3, then Section
// 3.2, Eq. 1-2), one workgroup per token row, in one launch. The same
// arithmetic in the same order as the two-pass kernels (rrs_quant.hip), so the
// codes and scales are bit-identical.
//
// The group scales need every row (s_b is a maximum over the tokens), so the
// rows exchange their group maxima within the launch: workgroup p rotates row
// p and publishes the row's G group maxima as tagged words in the workspace
// (the fence-free epoch protocol of rrs_device.h); every workgroup then reads
// the M rows of words, forms s_b and r_b, and quantizes its own row. With
// M <= 16 workgroups the rows are rotated in parallel instead of one after
// another as in the one-workgroup kernel. A single row needs no exchange.
// Beyond about 32 rows the M words per group the reduction reads cost more
// than the second launch they save (27.5 us against 19.7 us at M = 64,
// K = 8192, measured with an earlier, count-based exchange).
//
// The exchange needs the M workgroups to be resident together, which a plain
// launch of M <= 16 workgroups gets on an otherwise idle device but not when
// other work fills every compute unit. The polls are therefore bounded
// (kMaxPolls rounds): a wait that runs out marks the call as failed in the
// header and writes NaN into its row's alpha (and into s_group for row 0),
// so that the row's outputs come out NaN rather than silently wrong, and the
// kernel ends.
#include "rrs_device.h"
#include "rrs_internal.h"

namespace rrs {
namespace {

constexpr int kMaxRows = 16;
constexpr int kMaxPolls = 1 << 18;

// kReorder (runtime reorder, K <= 8192): the rows exchange their K/32 block
// maxima instead of their group maxima; every workgroup then ranks the blocks
// (keys largest first, equal keys in increasing block index), takes s_b over
// the sorted blocks of group b, and quantizes its row with the blocks in that
// order; workgroup 0 also writes block_order. The same order, scales and
// codes as the three-launch path (block maxima, order, given-maxima pass).
template <int K, bool kRot, bool kReorder>
__global__ __launch_bounds__(kRowThreads) void quant_rows_kernel(
    const uint16_t* __restrict__ X, int M, int g, uint8_t* __restrict__ Xq,
    float* __restrict__ a_scale, float* __restrict__ s_group, int32_t* __restrict__ block_order,
    uint32_t* header, unsigned long long* tagged, int nrows, int max_polls) {
  constexpr int E = FwhtShape<K>::E;  // this thread's channels: t + 256 e after the FWHT
  constexpr int C = E < kReorderBlock ? E : kReorderBlock;  // positions per chunk maximum
  constexpr int CH = E / C;                                 // chunks per thread (1 or 2)
  constexpr int NB = K / kReorderBlock;
  static_assert(!kReorder || NB <= kRowThreads, "one block key per thread");
  __shared__ float slot[lds_row_floats(K)];
  __shared__ float red[kRowThreads * CH];
  __shared__ float rg[256];
  __shared__ float sg[256];
  __shared__ __attribute__((aligned(16))) float key[kReorder ? NB : 4];
  __shared__ float skey[kReorder ? NB : 1];
  __shared__ int sblk[kReorder ? NB : 1];
  __shared__ int missed;
  __shared__ uint32_t tag_lds;
  const int t = threadIdx.x;
  const int p = blockIdx.x;
  const int G = K / g;
  const int span = kReorder ? kReorderBlock : g;  // positions per exchanged word
  const int W = K / span;                         // words per row
  // This call's tag (the header was written by earlier calls only): one
  // thread requests it now and hands it over in LDS after the rotation, so
  // the load's latency hides behind it.
  uint32_t epoch = 0u;
  if (t == 0 && M > 1)
    epoch = __hip_atomic_load(header + kEpochWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  float v[E];
  load_halves<E>(X + (size_t)p * K + (size_t)t * E, v);
  fwht_row<K, kRot>(v, slot, t);  // v[e] = y[t + 256 e]
  if (t == 0) {
    missed = 0;
    tag_lds = next_epoch(epoch);
  }
  __syncthreads();                // slot is free again

  // This row's maxima of the exchanged spans (groups of g channels, or blocks
  // of 32 with the runtime reorder): thread t takes positions t E .. t E + E - 1
  // as CH chunks of C, each inside one span (C <= 32 <= span).
#pragma unroll
  for (int e = 0; e < E; ++e) slot[lds_pad(t + e * kRowThreads)] = fabsf(v[e]);
  __syncthreads();
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    float pm = 0.0f;
#pragma unroll
    for (int e = 0; e < C; ++e) pm = fmaxf(pm, slot[lds_pad(t * E + k * C + e)]);
    red[t * CH + k] = pm;
  }
  __syncthreads();
  float wm = 0.0f;  // this row's maximum of span t (t < W)
  if (t < W) {
    const int per = span / C;  // chunks per span
    for (int u = 0; u < per; ++u) wm = fmaxf(wm, red[t * per + u]);
  }
  // Maxima over the rows. With more than one row, every row's maxima are
  // exchanged: thread t < W publishes span t of this row and reads span t of
  // all nrows rows (all words requested at once, those not yet tagged
  // requested again, within max_polls rounds).
  const uint32_t tag = tag_lds;  // set before the barrier after the rotation
  if (t < W) {
    float s = wm;
    if (M > 1) {
      publish_tagged(tagged + (size_t)p * W + t, tag, wm);
      unsigned long long x[kMaxRows];
#pragma unroll
      for (int i = 0; i < kMaxRows; ++i)
        x[i] = i < nrows ? load_tagged(tagged + (size_t)i * W + t) : ((unsigned long long)tag << 32);
      bool ok = false;
      for (int round = 0;; ++round) {
        ok = true;
#pragma unroll
        for (int i = 0; i < kMaxRows; ++i) ok = ok && has_tag(x[i], tag);
        if (ok || round >= max_polls) break;
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int i = 0; i < kMaxRows; ++i)
          if (i < nrows && !has_tag(x[i], tag)) x[i] = load_tagged(tagged + (size_t)i * W + t);
      }
      if (!ok) missed = 1;  // benign race: every writer writes 1
      s = 0.0f;
#pragma unroll
      for (int i = 0; i < kMaxRows; ++i) s = fmaxf(s, __uint_as_float((uint32_t)x[i]));
    }
    if constexpr (kReorder) {
      key[t] = s;  // block t's key: its largest channel maximum
    } else {
      rg[t] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);  // s_b and r_b = fl(1 / s_b)
      sg[t] = s;
    }
  }
  __syncthreads();
  if constexpr (kReorder) {
    // Rank of block t: blocks with a larger key, or an equal key and a smaller
    // index, come first (broadcast LDS reads).
    if (t < NB) {
      const float c = key[t];
      int rank = 0;
#pragma unroll 4
      for (int q = 0; q < NB / 4; ++q) {
        const float4 k4 = reinterpret_cast<const float4*>(key)[q];
        const int b = 4 * q;
        rank += (k4.x > c || (k4.x == c && b < t)) ? 1 : 0;
        rank += (k4.y > c || (k4.y == c && b + 1 < t)) ? 1 : 0;
        rank += (k4.z > c || (k4.z == c && b + 2 < t)) ? 1 : 0;
        rank += (k4.w > c || (k4.w == c && b + 3 < t)) ? 1 : 0;
      }
      sblk[rank] = t;
      skey[rank] = c;
    }
    __syncthreads();
    // s_b over the sorted blocks of group b.
    if (t < G) {
      const int per = g / kReorderBlock;
      float s = 0.0f;
      for (int u = 0; u < per; ++u) s = fmaxf(s, skey[t * per + u]);
      rg[t] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
      sg[t] = s;
    }
    if (p == 0 && t < NB) block_order[t] = sblk[t];
    __syncthreads();
  }
  const bool failed = missed != 0;  // uniform over the workgroup
  if (M > 1 && t == 0) {
    // Every word of the call has been read (or given up on): advance the epoch
    // (workgroup 0 only).
    if (failed)
      __hip_atomic_store(header + kFailWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (p == 0)
      __hip_atomic_store(header + kEpochWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (t < G && p == 0) s_group[t] = failed ? __builtin_nanf("") : sg[t];
  __syncthreads();

  // The row's codes, as the second pass: positions t E .. t E + E - 1.
  const float rb = rg[(t * E) / g];
#pragma unroll
  for (int e = 0; e < E; ++e) slot[lds_pad(t + e * kRowThreads)] = v[e];
  __syncthreads();
  if constexpr (kReorder) {
    // position j takes channel 32 sblk[j / 32] + j % 32 (masked into range:
    // with keys read from a workspace that was not zeroed, ranks could collide
    // and leave entries unset)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int j = t * E + e;
      const int b = sblk[j / kReorderBlock] & (NB - 1);
      v[e] = slot[lds_pad(b * kReorderBlock + j % kReorderBlock)];
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = slot[lds_pad(t * E + e)];
  }
  float lm = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
  lm = wave_max(lm * rb);  // fl(M_ib * r_b), max over the wave
  if ((t & 63) == 0) red[t >> 6] = lm;
  __syncthreads();
  const float a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
  const float m = rb * inv;  // fl(r_b * inv_i)
  uint32_t nib[E];
#pragma unroll
  for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * m);
  store_nibbles<E>(Xq + (size_t)p * (K / 2) + (size_t)t * (E / 2), nib);
  if (t == 0) a_scale[p] = failed ? __builtin_nanf("") : __fdiv_rn(a, 7.0f);
}

template <int K, bool kReorder>
hipError_t launch_k(const uint16_t* X, int M, int g, bool rotate, uint8_t* Xq, float* a_scale,
                    float* s_group, int32_t* block_order, uint32_t* header,
                    unsigned long long* tagged, int nrows, int max_polls, hipStream_t stream) {
  if (rotate)
    quant_rows_kernel<K, true, kReorder><<<M, kRowThreads, 0, stream>>>(
        X, M, g, Xq, a_scale, s_group, block_order, header, tagged, nrows, max_polls);
  else
    quant_rows_kernel<K, false, kReorder><<<M, kRowThreads, 0, stream>>>(
        X, M, g, Xq, a_scale, s_group, block_order, header, tagged, nrows, max_polls);
  return hipGetLastError();
}

}  // namespace

bool quant_rows_fits(int M) { return M >= 1 && M <= kMaxRows; }

size_t quant_rows_workspace_bytes(int K, int g) {
  return kQuantHeaderBytes + align256((size_t)kMaxRows * (K / g) * 8);
}

bool quant_rows_reorder_fits(int M, int K) { return quant_rows_fits(M) && K <= 8192; }

size_t quant_rows_reorder_workspace_bytes(int K) {
  return kQuantHeaderBytes + align256((size_t)kMaxRows * (K / kReorderBlock) * 8);
}

hipError_t launch_quant_rows_reorder(const uint16_t* X, int M, int K, int g, bool rotate,
                                     uint8_t* Xq, float* a_scale, float* s_group,
                                     int32_t* block_order, void* workspace, hipStream_t stream,
                                     int extra_rows, int max_polls) {
  const int nrows = M + extra_rows;  // rows of block maxima the readers wait for
  if (!quant_rows_reorder_fits(M, K) || nrows > kMaxRows) return hipErrorInvalidValue;
  const int polls = max_polls > 0 ? max_polls : kMaxPolls;
  uint32_t* header = static_cast<uint32_t*>(workspace);
  unsigned long long* tagged =
      reinterpret_cast<unsigned long long*>(static_cast<char*>(workspace) + kQuantHeaderBytes);
#define RRS_ROWS_R(K_)                                                                          \
  launch_k<K_, true>(X, M, g, rotate, Xq, a_scale, s_group, block_order, header, tagged, nrows, \
                     polls, stream)
  switch (K) {
    case 512: return RRS_ROWS_R(512);
    case 1024: return RRS_ROWS_R(1024);
    case 2048: return RRS_ROWS_R(2048);
    case 4096: return RRS_ROWS_R(4096);
    case 8192: return RRS_ROWS_R(8192);
    default: return hipErrorInvalidValue;
  }
#undef RRS_ROWS_R
}

hipError_t launch_quant_rows(const uint16_t* X, int M, int K, int g, bool rotate, uint8_t* Xq,
                             float* a_scale, float* s_group, void* workspace, hipStream_t stream,
                             int extra_rows, int max_polls) {
  uint32_t* header = static_cast<uint32_t*>(workspace);
  unsigned long long* tagged =
      reinterpret_cast<unsigned long long*>(static_cast<char*>(workspace) + kQuantHeaderBytes);
  const int nrows = M + extra_rows;  // rows of maxima the readers wait for
  if (nrows > kMaxRows) return hipErrorInvalidValue;
  const int polls = max_polls > 0 ? max_polls : kMaxPolls;
#define RRS_ROWS_K(K_)                                                                   \
  launch_k<K_, false>(X, M, g, rotate, Xq, a_scale, s_group, nullptr, header, tagged, nrows, \
                      polls, stream)
  switch (K) {
    case 512: return RRS_ROWS_K(512);
    case 1024: return RRS_ROWS_K(1024);
    case 2048: return RRS_ROWS_K(2048);
    case 4096: return RRS_ROWS_K(4096);
    case 8192: return RRS_ROWS_K(8192);
    case 16384: return RRS_ROWS_K(16384);
    default: return hipErrorInvalidValue;
  }
#undef RRS_ROWS_K
}

bool quant_rows_used(int M, int K, int g, const int32_t* perm, int flags) {
  return quant_rows_fits(M) && !perm && !(flags & kSkipSmoothing) &&
         quant_rows_workspace_bytes(K, g) <= quant_two_pass_offset(K);
}

hipError_t quant_exchange_failed(const void* workspace, hipStream_t stream, bool* failed) {
  uint32_t words[2] = {0u, 0u};
  hipError_t e = hipMemcpyAsync(words, workspace, sizeof(words), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  *failed = words[kFailWord] != 0u && words[kFailWord] == words[kEpochWord];
  return e;
}

}  // namespace rrs
