// rotate + smooth + quant for a handful of tokens (Section 3.3, then Section
// 3.2, Eq. 1-2), one workgroup per token row, in one launch. The same
// arithmetic in the same order as the two-pass kernels (rrs_quant.hip), so the
// codes and scales are bit-identical.
//
// The group scales need every row (s_b is a maximum over the tokens), so the
// rows exchange their group maxima within the launch: workgroup p rotates row
// p and publishes the row's G group maxima as tagged words in the workspace
// (the fence-free epoch protocol of rrs_device.h); every workgroup then reads
// the M rows of words, forms s_b and r_b, and quantizes its own row. The rows
// are rotated in parallel instead of one after another as in the
// one-workgroup kernel. A single row needs no exchange. The threads of a
// group share the reads of its M words (16 at most per thread), so up to 64
// rows take one launch where a group spans four threads or more: at K = 8192
// and g = 128, 8.1 to 9.1 us for 17 to 64 rows against about 19 us for the two
// launches (an earlier form, where one thread per group read every row through
// a count-based exchange, took 27.5 us at 64 rows), and at K <= 4096 0.5 to
// 0.9 us less than the fused many-token kernel.
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

constexpr int kMaxRows = 16;      // exchanged words one thread waits for
constexpr int kMaxRowsWide = 64;  // rows when a group's threads share the reads
constexpr int kMaxPolls = 1 << 18;

// kReorder (runtime reorder, K <= 8192): the rows exchange their K/32 block
// maxima instead of their group maxima; every workgroup then ranks the blocks
// (keys largest first, equal keys in increasing block index), takes s_b over
// the sorted blocks of group b, and quantizes its row with the blocks in that
// order; workgroup 0 also writes block_order. The same order, scales and
// codes as the three-launch path (block maxima, order, given-maxima pass).
//
// After the rotation the row goes once through LDS into position-major order,
// so each thread holds E consecutive positions, all in one span (a group, or
// a block of 32 with the runtime reorder; E <= span): the span maxima come
// from registers and shuffles, and the codes are packed from the same
// registers (with the runtime reorder the sorted positions are gathered from
// the position-major copy).
template <int K, bool kRot, bool kReorder>
__global__ __launch_bounds__(kRowThreads) void quant_rows_kernel(
    const uint16_t* __restrict__ X, int M, int g, uint8_t* __restrict__ Xq,
    float* __restrict__ a_scale, float* __restrict__ s_group, int32_t* __restrict__ block_order,
    uint32_t* header, unsigned long long* tagged, int nrows, int max_polls) {
  constexpr int E = FwhtShape<K>::E;  // this thread's channels: t + 256 e after the FWHT
  constexpr int NB = K / kReorderBlock;
  static_assert(!kReorder || NB <= kRowThreads, "one block key per thread");
  static_assert(E <= 64 && (!kReorder || E <= kReorderBlock), "a thread's positions in one span");
  __shared__ float slot[lds_row_floats(K)];                   // the rotation's scratch
  __shared__ __attribute__((aligned(16))) float row[K];      // position-major (pos_addr)
  __shared__ float red[4];
  __shared__ float rg[256];
  __shared__ float sg[256];
  __shared__ __attribute__((aligned(16))) unsigned long long key[kReorder ? NB : 2];
  __shared__ __attribute__((aligned(16))) unsigned long long srt[kReorder ? NB : 2];
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
#pragma unroll
  for (int e = 0; e < E; ++e) row[pos_addr<E>(t + e * kRowThreads)] = v[e];
  if (t == 0) {
    missed = 0;
    tag_lds = next_epoch(epoch);
  }
  __syncthreads();
  read_positions<E>(row, t, v);  // v[e] = y[t E + e]

  // This row's maximum of each exchanged span: over the thread's E positions,
  // then over the tps threads of the span (shuffles within a wave, LDS across
  // waves when a span is wider than a wave).
  float pm = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) pm = fmaxf(pm, fabsf(v[e]));
  const int tps = span / E;
  for (int o = 1; o < tps && o < 64; o <<= 1) pm = fmaxf(pm, __shfl_xor(pm, o, 64));
  bool owner;  // this thread publishes / reduces span b
  int b;
  if (tps <= 64) {
    owner = (t & (tps - 1)) == 0;
    b = t / tps;
  } else {
    if ((t & 63) == 0) red[t >> 6] = pm;
    __syncthreads();
    owner = t < W;
    b = t;
    if (owner) {
      const int per = tps / 64;  // waves per span
      pm = red[t * per];
      for (int u = 1; u < per; ++u) pm = fmaxf(pm, red[t * per + u]);
    }
  }

  // Maxima over the rows. With more than one row, every row's maxima are
  // exchanged: the owner of span b publishes this row's maximum, and span b
  // of all nrows rows is read (all words requested at once, those not yet
  // tagged requested again, within max_polls rounds). When a span's tps
  // threads share a wave they share the reads, thread k of the span taking
  // rows k, k + tps, ... (up to kMaxRows each), and combine them with
  // shuffles; otherwise the owner reads them all.
  const uint32_t tag = tag_lds;  // set before the barrier above
  const bool share = tps <= 64;
  const int sub = share ? (t & (tps - 1)) : 0;
  const int nsub = share ? tps : 1;
  float s = pm;
  if (M > 1 && (share || owner)) {
    if (owner) publish_tagged(tagged + (size_t)p * W + b, tag, pm);
    unsigned long long x[kMaxRows];
#pragma unroll
    for (int i = 0; i < kMaxRows; ++i) {
      const int r = sub + i * nsub;
      x[i] = r < nrows ? load_tagged(tagged + (size_t)r * W + b) : ((unsigned long long)tag << 32);
    }
    bool ok = false;
    for (int round = 0;; ++round) {
      ok = true;
#pragma unroll
      for (int i = 0; i < kMaxRows; ++i) ok = ok && has_tag(x[i], tag);
      if (ok || round >= max_polls) break;
      __builtin_amdgcn_s_sleep(1);
#pragma unroll
      for (int i = 0; i < kMaxRows; ++i) {
        const int r = sub + i * nsub;
        if (r < nrows && !has_tag(x[i], tag)) x[i] = load_tagged(tagged + (size_t)r * W + b);
      }
    }
    if (!ok) missed = 1;  // benign race: every writer writes 1
    s = 0.0f;
#pragma unroll
    for (int i = 0; i < kMaxRows; ++i) s = fmaxf(s, __uint_as_float((uint32_t)x[i]));
  }
  if (M > 1 && share)  // every lane of the wave takes part (tps is uniform)
    for (int o = 1; o < tps; o <<= 1) s = fmaxf(s, __shfl_xor(s, o, 64));
  if (owner) {
    if constexpr (kReorder) {
      key[b] = block_sort_key(s, b);  // block b's key: its largest channel maximum
    } else {
      rg[b] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);  // s_b and r_b = fl(1 / s_b)
      sg[b] = s;
    }
  }
  __syncthreads();
  if constexpr (kReorder) {
    // Blocks with a larger key, or an equal key and a smaller index, first.
    rank_blocks<NB, kRowThreads>(key, srt, sblk, skey, t);
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
    // position j takes channel 32 sblk[j / 32] + j % 32 (masked into range:
    // with keys read from a workspace that was not zeroed, ranks could collide
    // and leave entries unset)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int j = t * E + e;
      const int bl = sblk[j / kReorderBlock] & (NB - 1);
      v[e] = row[pos_addr<E>(bl * kReorderBlock + j % kReorderBlock)];
    }
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

  // The row's codes, as the second pass: positions t E .. t E + E - 1.
  const float rb = rg[(t * E) / g];
  float lm = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
  lm = wave_max(lm * rb);  // fl(M_ib * r_b), max over the wave
  if ((t & 63) == 0) red[t >> 6] = lm;
  __syncthreads();
  const float a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
  const float m = rb * inv;  // fl(r_b * inv_i)
  uint8_t* dst = Xq + (size_t)p * (K / 2) + (size_t)t * (E / 2);
  if constexpr (E >= 8) {
    uint32_t wd[E / 8];
#pragma unroll
    for (int w = 0; w < E / 8; ++w) wd[w] = quant_pack8(&v[8 * w], m);
    if constexpr (E == 8) {
      *reinterpret_cast<uint32_t*>(dst) = wd[0];
    } else if constexpr (E == 16) {
      *reinterpret_cast<uint2*>(dst) = make_uint2(wd[0], wd[1]);
    } else {
#pragma unroll
      for (int w = 0; w < E / 8; w += 4)
        *reinterpret_cast<uint4*>(dst + 4 * w) = make_uint4(wd[w], wd[w + 1], wd[w + 2], wd[w + 3]);
    }
  } else {
    uint32_t nib[E];
#pragma unroll
    for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * m);
    store_nibbles<E>(dst, nib);
  }
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

// Rows the per-row kernel takes at (K, g) without a runtime reorder: 16, or
// up to 64 where a group's threads share the reads (16 words each). From
// 17 to 64 rows it beats the alternatives at every K: the two-pass kernels
// from K = 8192 on (8.1-9.1 us against about 19 us at K = 8192, g = 128) and
// the one-launch fused kernel at K <= 4096 (8.0-8.5 against 8.6-9.1 us at
// K = 1024 to 4096; events, back-to-back calls).
int quant_rows_max(int K, int g) {
  const int tps = g / (K / kRowThreads);  // threads per group
  if (tps < 1 || tps > 64) return kMaxRows;
  return kMaxRows * tps < kMaxRowsWide ? kMaxRows * tps : kMaxRowsWide;
}

size_t quant_rows_workspace_bytes(int K, int g) {
  return kQuantHeaderBytes + align256((size_t)quant_rows_max(K, g) * (K / g) * 8);
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
  if (nrows > quant_rows_max(K, g)) return hipErrorInvalidValue;
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
  return M >= 1 && M <= quant_rows_max(K, g) && !perm && !(flags & kSkipSmoothing) &&
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
