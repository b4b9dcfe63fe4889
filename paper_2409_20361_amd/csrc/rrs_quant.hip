// Online rotate + runtime smooth + per-token INT4 quantization
// (Section 3.3 then Section 3.2; Eq. 1-2; Section 2.1).
//
// Three launches on the caller's stream:
//   1. colmax: each workgroup rotates its rows (FWHT) and keeps the running
//      per-channel max |y| in registers; it writes one partial row of K floats.
//   2. reduce: per channel, the max over the partial rows -> c_j (Eq. 1).
//   3. quant:  each workgroup derives the group scales s_b = max_{j in b} c_j
//      (Section 3.2) and r_b = 1/s_b, then re-rotates its rows (bit-identical
//      to pass 1), takes the per-token max of |y| r_b, and writes the INT4
//      codes, alpha_i and (workgroup 0) s_b.
// The channel max needs every token before any token can be quantized, hence
// the split; the second read of X mostly hits the 256 MB Infinity Cache.
#include "rrs_device.h"
#include "rrs_internal.h"

namespace rrs {
namespace {

constexpr int kMaxPartialRows = 256;
constexpr int kQuantMaxWgs = 1024;

template <int K>
__global__ __launch_bounds__(kRowThreads) void colmax_kernel(const uint16_t* __restrict__ X,
                                                             int M, int rows_per_wg,
                                                             float* __restrict__ partial) {
  using S = FwhtShape<K>;
  __shared__ float lds[lds_row_floats(K)];
  const int t = threadIdx.x;
  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  float cm[S::E];
#pragma unroll
  for (int e = 0; e < S::E; ++e) cm[e] = 0.0f;
  for (int r = r0; r < r1; ++r) {
    float v[S::E];
    load_halves<S::E>(X + (size_t)r * K + (size_t)t * S::E, v);
    fwht_row<K>(v, lds, t);
#pragma unroll
    for (int e = 0; e < S::E; ++e) cm[e] = fmaxf(cm[e], fabsf(v[e]));
  }
  float* out = partial + (size_t)blockIdx.x * K;
#pragma unroll
  for (int e = 0; e < S::E; ++e) out[t + e * kRowThreads] = cm[e];
}

// c[j] = max over the partial rows; 64 channels per workgroup, 4 row slices.
__global__ __launch_bounds__(256) void reduce_kernel(const float* __restrict__ partial,
                                                     int nparts, int K,
                                                     float* __restrict__ cmax) {
  __shared__ float red[4][64];
  const int t = threadIdx.x;
  const int j = blockIdx.x * 64 + (t & 63);
  const int slice = t >> 6;
  float m = 0.0f;
  for (int i = slice; i < nparts; i += 4) m = fmaxf(m, partial[(size_t)i * K + j]);
  red[slice][t & 63] = m;
  __syncthreads();
  if (t < 64) cmax[j] = fmaxf(fmaxf(red[0][t], red[1][t]), fmaxf(red[2][t], red[3][t]));
}

template <int K>
__global__ __launch_bounds__(kRowThreads) void quant_kernel(
    const uint16_t* __restrict__ X, int M, int g, int rows_per_wg,
    const int32_t* __restrict__ perm, const float* __restrict__ cmax,
    uint8_t* __restrict__ Xq, float* __restrict__ a_scale, float* __restrict__ s_group) {
  using S = FwhtShape<K>;
  constexpr int E = S::E;
  __shared__ float lds[lds_row_floats(K)];
  __shared__ float rgrp[kRowThreads];
  __shared__ float red[4];
  const int t = threadIdx.x;
  const int G = K / g;

  // Position j = t*E + e of the (reordered) row reads channel src[e].
  int src[E];
#pragma unroll
  for (int e = 0; e < E; ++e) src[e] = perm ? perm[t * E + e] : t * E + e;

  // Group smoothing scales: this thread's E positions lie in one group (E <= g).
  float cl = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) cl = fmaxf(cl, cmax[src[e]]);
  lds[t] = cl;
  __syncthreads();
  if (t < G) {
    const int per = g / E;
    float s = 0.0f;
    for (int u = 0; u < per; ++u) s = fmaxf(s, lds[t * per + u]);
    rgrp[t] = (s == 0.0f) ? 0.0f : __fdiv_rn(1.0f, s);
    if (blockIdx.x == 0) s_group[t] = s;
  }
  __syncthreads();
  const float rb = rgrp[(t * E) / g];

  const int r0 = blockIdx.x * rows_per_wg;
  const int r1 = min(M, r0 + rows_per_wg);
  for (int r = r0; r < r1; ++r) {
    float v[E];
    load_halves<E>(X + (size_t)r * K + (size_t)t * E, v);
    fwht_row<K>(v, lds, t);
    // back to natural order (and apply the static reorder)
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) lds[lds_pad(t + e * kRowThreads)] = v[e];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = lds[lds_pad(src[e])];

    float lm = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
    lm = lm * rb;  // fl(M_ib * r_b)
    const float a = block_max256(lm, red);
    const float inv = (a == 0.0f) ? 0.0f : __fdiv_rn(7.0f, a);
    const float m = rb * inv;  // fl(r_b * inv_i)
    uint32_t nib[E];
#pragma unroll
    for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * m);
    store_nibbles<E>(Xq + (size_t)r * (K / 2) + (size_t)t * (E / 2), nib);
    if (t == 0) a_scale[r] = __fdiv_rn(a, 7.0f);
  }
}

template <int K>
hipError_t launch_k(const uint16_t* X, int M, int g, const int32_t* perm, uint8_t* Xq,
                    float* a_scale, float* s_group, void* workspace, hipStream_t stream) {
  const int nparts = quant_partial_rows(M);
  const int rows_a = (M + nparts - 1) / nparts;
  const int grid_a = (M + rows_a - 1) / rows_a;
  float* partial = static_cast<float*>(workspace);
  float* cmax = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                         align256((size_t)kMaxPartialRows * K * 4));
  colmax_kernel<K><<<grid_a, kRowThreads, 0, stream>>>(X, M, rows_a, partial);
  reduce_kernel<<<K / 64, 256, 0, stream>>>(partial, grid_a, K, cmax);
  const int wgs_c = M < kQuantMaxWgs ? M : kQuantMaxWgs;
  const int rows_c = (M + wgs_c - 1) / wgs_c;
  const int grid_c = (M + rows_c - 1) / rows_c;
  quant_kernel<K><<<grid_c, kRowThreads, 0, stream>>>(X, M, g, rows_c, perm, cmax, Xq,
                                                      a_scale, s_group);
  return hipGetLastError();
}

}  // namespace

int quant_partial_rows(int M) { return M < kMaxPartialRows ? M : kMaxPartialRows; }

size_t quant_workspace_bytes(int M, int K) {
  (void)M;
  return align256((size_t)kMaxPartialRows * K * 4) + align256((size_t)K * 4);
}

hipError_t launch_rotate_smooth_quant(const uint16_t* X, int M, int K, int g,
                                      const int32_t* perm, uint8_t* Xq, float* a_scale,
                                      float* s_group, void* workspace, hipStream_t stream) {
  switch (K) {
    case 512: return launch_k<512>(X, M, g, perm, Xq, a_scale, s_group, workspace, stream);
    case 1024: return launch_k<1024>(X, M, g, perm, Xq, a_scale, s_group, workspace, stream);
    case 2048: return launch_k<2048>(X, M, g, perm, Xq, a_scale, s_group, workspace, stream);
    case 4096: return launch_k<4096>(X, M, g, perm, Xq, a_scale, s_group, workspace, stream);
    case 8192: return launch_k<8192>(X, M, g, perm, Xq, a_scale, s_group, workspace, stream);
    case 16384: return launch_k<16384>(X, M, g, perm, Xq, a_scale, s_group, workspace, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rrs
