// rotate + smooth + quant for a handful of tokens (Section 3.3, then Section
// 3.2, Eq. 1-2), one workgroup per token row, in one launch. The same
// arithmetic in the same order as the two-pass kernels (rrs_quant.hip), so the
// codes and scales are bit-identical.
//
// The group scales need every row (s_b is a maximum over the tokens), so the
// rows exchange their group maxima through the workspace: workgroup p rotates
// row p, writes the row's G group maxima, writes its caches back and counts
// itself in; when all M have arrived, each reads the M rows of maxima with
// agent-scope atomic loads (coherent across the XCDs' L2s, so no cache
// invalidation is needed), forms s_b and r_b, and quantizes its own row. With
// M <= 16 workgroups, all resident at once, the wait is short, and the rows are
// rotated in parallel instead of one after another as in the one-workgroup
// kernel. A single row needs no exchange. Beyond about 32 rows the M coherent
// loads per group of the reduction cost more than the second launch they save
// (27.5 us against 19.7 us at M = 64, K = 8192).
//
// The count starts from zero: a one-thread kernel launched just before clears
// it (a kernel rather than a memset, so the pair can be captured in a graph).
// The wait is bounded (kMaxPolls); a wait that runs out records itself in the
// error word and goes on, so the kernel always ends.
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

__device__ bool wait_count(uint32_t* ctr, uint32_t target) {
  for (int i = 0; i < kMaxPolls; ++i) {
    if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target)
      return true;
    __builtin_amdgcn_s_sleep(2);
  }
  return false;
}

__device__ __forceinline__ float load_coherent(const float* p) {
  return __uint_as_float(__hip_atomic_load(reinterpret_cast<uint32_t*>(const_cast<float*>(p)),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

template <int K, bool kRot>
__global__ __launch_bounds__(kRowThreads) void quant_rows_kernel(
    const uint16_t* __restrict__ X, int M, int g, uint8_t* __restrict__ Xq,
    float* __restrict__ a_scale, float* __restrict__ s_group, float* gpart, uint32_t* sync) {
  constexpr int E = FwhtShape<K>::E;  // this thread's channels: t + 256 e after the FWHT
  __shared__ float slot[lds_row_floats(K)];
  __shared__ float red[kRowThreads];
  __shared__ float rg[256];
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
      if (!wait_count(sync + kArrive, (uint32_t)M))
        __hip_atomic_fetch_add(sync + kErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
  }

  // s_b = max over the M rows, r_b = fl(1 / s_b).
  if (t < G) {
    float s = gm;
    if (M > 1) {
      s = 0.0f;
      for (int i = 0; i < M; ++i) s = fmaxf(s, load_coherent(gpart + (size_t)i * G + t));
    }
    rg[t] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
    if (p == 0) s_group[t] = s;
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
  if (t == 0) a_scale[p] = __fdiv_rn(a, 7.0f);
}

template <int K>
hipError_t launch_k(const uint16_t* X, int M, int g, bool rotate, uint8_t* Xq, float* a_scale,
                    float* s_group, float* gpart, uint32_t* sync, hipStream_t stream) {
  if (rotate)
    quant_rows_kernel<K, true><<<M, kRowThreads, 0, stream>>>(X, M, g, Xq, a_scale, s_group,
                                                              gpart, sync);
  else
    quant_rows_kernel<K, false><<<M, kRowThreads, 0, stream>>>(X, M, g, Xq, a_scale, s_group,
                                                               gpart, sync);
  return hipGetLastError();
}

}  // namespace

bool quant_rows_fits(int M) { return M >= 1 && M <= kMaxRows; }

size_t quant_rows_workspace_bytes(int K, int g) {
  return 256 + align256((size_t)kMaxRows * (K / g) * 4);
}

hipError_t launch_quant_rows(const uint16_t* X, int M, int K, int g, bool rotate, uint8_t* Xq,
                             float* a_scale, float* s_group, void* workspace,
                             hipStream_t stream) {
  uint32_t* sync = static_cast<uint32_t*>(workspace);
  float* gpart = reinterpret_cast<float*>(static_cast<char*>(workspace) + 256);
  if (M > 1) {  // one row needs no exchange and no count
    clear_count_kernel<<<1, 64, 0, stream>>>(sync);
    if (hipError_t e = hipGetLastError()) return e;
  }
  switch (K) {
    case 512: return launch_k<512>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, stream);
    case 1024: return launch_k<1024>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, stream);
    case 2048: return launch_k<2048>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, stream);
    case 4096: return launch_k<4096>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, stream);
    case 8192: return launch_k<8192>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, stream);
    case 16384: return launch_k<16384>(X, M, g, rotate, Xq, a_scale, s_group, gpart, sync, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rrs
