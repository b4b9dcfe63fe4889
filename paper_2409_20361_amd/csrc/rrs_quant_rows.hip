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

template <int K, bool kRot>
__global__ __launch_bounds__(kRowThreads) void quant_rows_kernel(
    const uint16_t* __restrict__ X, int M, int g, uint8_t* __restrict__ Xq,
    float* __restrict__ a_scale, float* __restrict__ s_group, uint32_t* header,
    unsigned long long* tagged, int nrows, int max_polls) {
  constexpr int E = FwhtShape<K>::E;  // this thread's channels: t + 256 e after the FWHT
  __shared__ float slot[lds_row_floats(K)];
  __shared__ float red[kRowThreads];
  __shared__ float rg[256];
  __shared__ float sg[256];
  __shared__ int missed;
  __shared__ uint32_t tag_lds;
  const int t = threadIdx.x;
  const int p = blockIdx.x;
  const int G = K / g;
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

  // This row's group maxima: thread t takes positions t E .. t E + E - 1, all
  // in one group (E <= 64 <= g).
#pragma unroll
  for (int e = 0; e < E; ++e) slot[lds_pad(t + e * kRowThreads)] = fabsf(v[e]);
  __syncthreads();
  float pm = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) pm = fmaxf(pm, slot[lds_pad(t * E + e)]);
  red[t] = pm;
  __syncthreads();
  float gm = 0.0f;  // this row's maximum of group t (t < G)
  if (t < G) {
    const int per = g / E;  // threads per group
    for (int u = 0; u < per; ++u) gm = fmaxf(gm, red[t * per + u]);
  }
  // s_b = max over the rows, r_b = fl(1 / s_b). With more than one row, every
  // row's maxima are exchanged: thread t < G publishes group t of this row and
  // reads group t of all nrows rows (all words requested at once, those not
  // yet tagged requested again, within max_polls rounds).
  const uint32_t tag = tag_lds;  // set before the barrier after the rotation
  if (t < G) {
    float s = gm;
    if (M > 1) {
      publish_tagged(tagged + (size_t)p * G + t, tag, gm);
      unsigned long long x[kMaxRows];
#pragma unroll
      for (int i = 0; i < kMaxRows; ++i)
        x[i] = i < nrows ? load_tagged(tagged + (size_t)i * G + t) : ((unsigned long long)tag << 32);
      bool ok = false;
      for (int round = 0;; ++round) {
        ok = true;
#pragma unroll
        for (int i = 0; i < kMaxRows; ++i) ok = ok && has_tag(x[i], tag);
        if (ok || round >= max_polls) break;
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int i = 0; i < kMaxRows; ++i)
          if (i < nrows && !has_tag(x[i], tag)) x[i] = load_tagged(tagged + (size_t)i * G + t);
      }
      if (!ok) missed = 1;  // benign race: every writer writes 1
      s = 0.0f;
#pragma unroll
      for (int i = 0; i < kMaxRows; ++i) s = fmaxf(s, __uint_as_float((uint32_t)x[i]));
    }
    rg[t] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
    sg[t] = s;
  }
  __syncthreads();
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
#pragma unroll
  for (int e = 0; e < E; ++e) v[e] = slot[lds_pad(t * E + e)];
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

template <int K>
hipError_t launch_k(const uint16_t* X, int M, int g, bool rotate, uint8_t* Xq, float* a_scale,
                    float* s_group, uint32_t* header, unsigned long long* tagged, int nrows,
                    int max_polls, hipStream_t stream) {
  if (rotate)
    quant_rows_kernel<K, true><<<M, kRowThreads, 0, stream>>>(X, M, g, Xq, a_scale, s_group,
                                                              header, tagged, nrows, max_polls);
  else
    quant_rows_kernel<K, false><<<M, kRowThreads, 0, stream>>>(X, M, g, Xq, a_scale, s_group,
                                                               header, tagged, nrows, max_polls);
  return hipGetLastError();
}

}  // namespace

bool quant_rows_fits(int M) { return M >= 1 && M <= kMaxRows; }

size_t quant_rows_workspace_bytes(int K, int g) {
  return kQuantHeaderBytes + align256((size_t)kMaxRows * (K / g) * 8);
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
#define RRS_ROWS_K(K_) \
  launch_k<K_>(X, M, g, rotate, Xq, a_scale, s_group, header, tagged, nrows, polls, stream)
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
