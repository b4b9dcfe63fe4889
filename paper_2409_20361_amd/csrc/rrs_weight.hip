// Offline weight preparation (Section 3.3: weights are rotated offline and
// quantized per output channel; round-to-nearest stands in for GPTQ).
//
// For each output channel n (a column of W, K x N row-major):
//   u = H_K W[:, n]                 (same FWHT and stage order as activations;
//                                    u = W[:, n] for the ablation without rotation)
//   u'_j = u_{perm[j]}              (optional static reorder, Fig. 4 step (1))
//   b_n = max_j |u_j|, winv = fl(7 / b_n), beta_n = fl(b_n / 7)
//   code_j = clamp(rint(fl(u'_j * winv)), -7, 7), packed as byte j / 2 of row
//   n (low nibble even j), row-major or tiled (WqLayout).
// A workgroup stages C = 32768 / K whole columns in LDS (139 KB), then
// transforms and quantizes them one after another.
#include "rrs_device.h"
#include "rrs_internal.h"

namespace rrs {
namespace {

// kSub: the sub-channel baseline of Section 4.5: one scale per (output
// channel, group of g), w_scale[b * N + n] = fl(m_b / 7) (group-major, L x N);
// no reorder.
// Stores this thread's E codes, packed bytes [j0, j0 + E/2) of row n: one
// store inside a 16-byte piece (E <= 32), else one per piece.
template <int E>
__device__ __forceinline__ void store_wq(uint8_t* __restrict__ Wq, WqLayout lay, int n, int j0,
                                         int K, const uint32_t (&nib)[E]) {
  if constexpr (E <= 32) {
    store_nibbles<E>(Wq + lay.piece(n, j0 >> 4, K) + (j0 & 15), nib);
  } else {
#pragma unroll
    for (int c = 0; c < E / 32; ++c) {
      uint32_t part[32];
#pragma unroll
      for (int e = 0; e < 32; ++e) part[e] = nib[32 * c + e];
      store_nibbles<32>(Wq + lay.piece(n, (j0 >> 4) + c, K), part);
    }
  }
}

template <int K, bool kRot, bool kSub = false>
__global__ __launch_bounds__(kRowThreads) void prep_weight_kernel(
    const uint16_t* __restrict__ W, int N, const int32_t* __restrict__ perm,
    uint8_t* __restrict__ Wq, float* __restrict__ w_scale, int g, WqLayout lay) {
  using S = FwhtShape<K>;
  constexpr int E = S::E;
  constexpr int C = 32768 / K;
  constexpr int kCol = lds_row_floats(K);
  __shared__ float lds[C * kCol];
  __shared__ float red[kSub ? 256 : 4];
  __shared__ float gm[kSub ? 256 : 1];
  const int t = threadIdx.x;
  const int n0 = blockIdx.x * C;

  // Stage C columns, column c at lds[c * kCol + pad(k)].
  for (int idx = t; idx < K * C; idx += kRowThreads) {
    const int c = idx % C;
    const int k = idx / C;
    const int n = n0 + c;
    const float w = (n < N) ? half_to_float(W[(size_t)k * N + n]) : 0.0f;
    lds[c * kCol + lds_pad(k)] = w;
  }
  __syncthreads();

  int src[E];
#pragma unroll
  for (int e = 0; e < E; ++e) src[e] = perm ? perm[t * E + e] : t * E + e;

  for (int c = 0; c < C; ++c) {
    const int n = n0 + c;
    if (n >= N) break;  // uniform across the workgroup
    float* col = lds + c * kCol;
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = col[lds_pad(t * E + e)];
    fwht_row<K, kRot>(v, col, t);
    float lm = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
    float b = 0.0f;
    if constexpr (!kSub) b = block_max256(lm, red);  // contains barriers
#pragma unroll
    for (int e = 0; e < E; ++e) col[lds_pad(t + e * kRowThreads)] = v[e];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = col[lds_pad(src[e])];
    if constexpr (kSub) {
      // this thread's channels [t E, t E + E) lie in one group
      lm = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) lm = fmaxf(lm, fabsf(v[e]));
      b = row_group_max(lm, red, gm, t, E, g, K / g);
    }
    const float winv = (b == 0.0f) ? 0.0f : __fdiv_rn(7.0f, b);
    uint32_t nib[E];
#pragma unroll
    for (int e = 0; e < E; ++e) nib[e] = int4_nibble(v[e] * winv);
    store_wq<E>(Wq, lay, n, t * (E / 2), K, nib);
    if constexpr (kSub) {
      if ((t * E) % g == 0) w_scale[(size_t)((t * E) / g) * N + n] = __fdiv_rn(b, 7.0f);
    } else {
      if (t == 0) w_scale[n] = __fdiv_rn(b, 7.0f);
    }
  }
}

template <int K>
hipError_t launch_k(const uint16_t* W, int N, const int32_t* perm, bool rotate, uint8_t* Wq,
                    float* w_scale, int g_sub, WqLayout lay, hipStream_t stream) {
  constexpr int C = 32768 / K;
  const int grid = (N + C - 1) / C;
  if (g_sub > 0) {
    if (rotate)
      prep_weight_kernel<K, true, true><<<grid, kRowThreads, 0, stream>>>(W, N, nullptr, Wq,
                                                                          w_scale, g_sub, lay);
    else
      prep_weight_kernel<K, false, true><<<grid, kRowThreads, 0, stream>>>(W, N, nullptr, Wq,
                                                                           w_scale, g_sub, lay);
  } else if (rotate) {
    prep_weight_kernel<K, true><<<grid, kRowThreads, 0, stream>>>(W, N, perm, Wq, w_scale, 0,
                                                                   lay);
  } else {
    prep_weight_kernel<K, false><<<grid, kRowThreads, 0, stream>>>(W, N, perm, Wq, w_scale, 0,
                                                                    lay);
  }
  return hipGetLastError();
}

hipError_t launch_any_k(const uint16_t* W, int K, int N, const int32_t* perm, bool rotate,
                        uint8_t* Wq, float* w_scale, int g_sub, WqLayout lay,
                        hipStream_t stream) {
  switch (K) {
    case 512: return launch_k<512>(W, N, perm, rotate, Wq, w_scale, g_sub, lay, stream);
    case 1024: return launch_k<1024>(W, N, perm, rotate, Wq, w_scale, g_sub, lay, stream);
    case 2048: return launch_k<2048>(W, N, perm, rotate, Wq, w_scale, g_sub, lay, stream);
    case 4096: return launch_k<4096>(W, N, perm, rotate, Wq, w_scale, g_sub, lay, stream);
    case 8192: return launch_k<8192>(W, N, perm, rotate, Wq, w_scale, g_sub, lay, stream);
    case 16384: return launch_k<16384>(W, N, perm, rotate, Wq, w_scale, g_sub, lay, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prepare_weight(const uint16_t* W, int K, int N, const int32_t* perm,
                                 bool rotate, uint8_t* Wq, float* w_scale, hipStream_t stream,
                                 WqLayout lay) {
  return launch_any_k(W, K, N, perm, rotate, Wq, w_scale, 0, lay, stream);
}

hipError_t launch_prepare_weight_sub_channel(const uint16_t* W, int K, int N, int g, bool rotate,
                                             uint8_t* Wq, float* w_sub, hipStream_t stream,
                                             WqLayout lay) {
  return launch_any_k(W, K, N, nullptr, rotate, Wq, w_sub, g, lay, stream);
}

}  // namespace rrs
