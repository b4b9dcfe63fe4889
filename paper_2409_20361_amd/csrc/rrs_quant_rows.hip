// rotate + smooth + quant for a handful of tokens (Section 3.3, then Section
// 3.2, Eq. 1-2), one workgroup per token row, in one launch. The same
// arithmetic in the same order as the two-pass kernels (rrs_quant.hip), so the
// codes and scales are bit-identical.
//
// The group scales need every row (s_b is a maximum over the tokens), so the
// rows exchange their group maxima through the workspace: workgroup p rotates
// row p, writes the row's G group maxima, writes its caches back and counts
// itself in; when all M have arrived, each reads the M rows of maxima, forms
// s_b and r_b, and quantizes its own row. With
// M <= 16 workgroups, all resident at once, the wait is short, and the rows are
// rotated in parallel instead of one after another as in the one-workgroup
// kernel. A single row needs no exchange. Beyond about 32 rows the M loads
// per group of the reduction cost more than the second launch they save
// (27.5 us against 19.7 us at M = 64, K = 8192).
//
// The count starts from zero: a one-thread kernel launched just before clears
// it (a kernel rather than a memset, so the pair can be captured in a graph).
// Ordering: each row's maxima are written, made visible at agent scope
// (__threadfence) and then counted with a release add; the waiting thread
// polls the count with relaxed loads and, once all rows are in, takes an
// agent-scope acquire fence before the workgroup barrier, after which every
// thread of the workgroup reads the maxima with ordinary loads.
//
// The exchange needs the M workgroups to be resident together, which a plain
// launch of M <= 16 workgroups gets on an otherwise idle device but not when
// other work fills every compute unit. The wait is therefore bounded
// (kMaxPolls): a wait that runs out counts itself in the error word, writes
// NaN into its row's alpha (and into s_group for row 0) so that the row's
// outputs come out NaN rather than silently wrong, and the kernel ends.
#include "rrs_device.h"
#include "rrs_internal.h"

namespace rrs {
namespace {

constexpr int kMaxRows = 16;
constexpr int kMaxPolls = 1 << 18;
// Words at the start of the workspace (uint32): rows arrived, waits that ran out.
constexpr int kArrive = 0;
constexpr int kErr = 1;

__global__ void clear_count_kernel(uint32_t* sync) {
  if (threadIdx.x < 4) sync[threadIdx.x] = 0u;
}

__device__ bool wait_count(uint32_t* ctr, uint32_t target, int max_polls) {
  for (int i = 0; i < max_polls; ++i) {
    if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target)
      return true;
    __builtin_amdgcn_s_sleep(2);
  }
  return false;
}

template <int K, bool kRot>
__global__ __launch_bounds__(kRowThreads) void quant_rows_kernel(
    const uint16_t* __restrict__ X, int M, int g, uint8_t* __restrict__ Xq,
    float* __restrict__ a_scale, float* __restrict__ s_group, float* gpart, uint32_t* sync,
    uint32_t target, int max_polls) {
  constexpr int E = FwhtShape<K>::E;  // this thread's channels: t + 256 e after the FWHT
  __shared__ float slot[lds_row_floats(K)];
  __shared__ float red[kRowThreads];
  __shared__ float rg[256];
  __shared__ int arrived;
  const int t = threadIdx.x;
  const int p = blockIdx.x;
  const int G = K / g;

  float v[E];
  load_halves<E>(X + (size_t)p * K + (size_t)t * E, v);
  fwht_row<K, kRot>(v, slot, t);  // v[e] = y[t + 256 e]
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
  if (M > 1) {  // uniform: exchange the rows' maxima
    if (t < G) gpart[(size_t)p * G + t] = gm;
    __threadfence();  // the row of maxima reaches memory before the count
    __syncthreads();
    if (t == 0) {
      __hip_atomic_fetch_add(sync + kArrive, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      const bool ok = wait_count(sync + kArrive, target, max_polls);
      if (ok) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      } else {
        __hip_atomic_fetch_add(sync + kErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      arrived = ok ? 1 : 0;
    }
    __syncthreads();
  }
  const bool failed = M > 1 && arrived == 0;  // uniform over the workgroup

  // s_b = max over the M rows, r_b = fl(1 / s_b).
  if (t < G) {
    float s = gm;
    if (M > 1) {
      s = 0.0f;
      for (int i = 0; i < M; ++i) s = fmaxf(s, gpart[(size_t)i * G + t]);
    }
    rg[t] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
    if (p == 0) s_group[t] = failed ? __builtin_nanf("") : s;
  }
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
                    float* s_group, float* gpart, uint32_t* sync, uint32_t target, int max_polls,
                    hipStream_t stream) {
  if (rotate)
    quant_rows_kernel<K, true><<<M, kRowThreads, 0, stream>>>(X, M, g, Xq, a_scale, s_group,
                                                              gpart, sync, target, max_polls);
  else
    quant_rows_kernel<K, false><<<M, kRowThreads, 0, stream>>>(X, M, g, Xq, a_scale, s_group,
                                                               gpart, sync, target, max_polls);
  return hipGetLastError();
}

}  // namespace

bool quant_rows_fits(int M) { return M >= 1 && M <= kMaxRows; }

size_t quant_rows_workspace_bytes(int K, int g) {
  return 256 + align256((size_t)kMaxRows * (K / g) * 4);
}

hipError_t launch_quant_rows(const uint16_t* X, int M, int K, int g, bool rotate, uint8_t* Xq,
                             float* a_scale, float* s_group, void* workspace, hipStream_t stream,
                             int extra_arrivals, int max_polls) {
  uint32_t* sync = static_cast<uint32_t*>(workspace);
  float* gpart = reinterpret_cast<float*>(static_cast<char*>(workspace) + 256);
  if (M > 1) {  // one row needs no exchange and no count
    clear_count_kernel<<<1, 64, 0, stream>>>(sync);
    if (hipError_t e = hipGetLastError()) return e;
  }
  const uint32_t target = (uint32_t)M + (uint32_t)extra_arrivals;
  const int polls = max_polls > 0 ? max_polls : kMaxPolls;
#define RRS_ROWS_K(K_) \
  launch_k<K_>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, target, polls, stream)
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
         quant_rows_workspace_bytes(K, g) <= quant_workspace_bytes(M, K);
}

hipError_t quant_rows_timeouts(const void* workspace, hipStream_t stream, uint32_t* count) {
  uint32_t words[2] = {0u, 0u};
  hipError_t e = hipMemcpyAsync(words, workspace, sizeof(words), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  *count = words[kErr];
  return e;
}

}  // namespace rrs
