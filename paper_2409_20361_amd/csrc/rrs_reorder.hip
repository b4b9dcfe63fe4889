// Runtime channel reorder (Fig. 4 step (1) taken at run time; Section 3.2):
// before the grouping, the rotated channels are sorted by this call's
// channel-wise maxima c_j (Eq. 1), so that channels of similar size share a
// smoothing scale.
//
// Channels move in blocks of 32 consecutive channels: a block is one MFMA
// k-step of the GEMM and 16 bytes of a packed INT4 row, so the GEMM can fetch
// the matching weight rows by block (one table entry per 16-byte load) from
// weights prepared once, in natural order. A block's key is its largest c_j;
// keys are sorted largest first, equal keys in increasing block index; group
// b takes the sorted blocks [b g/32, (b+1) g/32).
//
// Three launches on the caller's stream:
//   1. block maxima: the rot_max pass of the quantizer with groups of 32
//      natural-order channels, one row of K/32 maxima per workgroup;
//   2. order (this file, one workgroup): reduce the rows to the K/32 keys,
//      rank them, write block_order, the channel permutation and the sorted
//      group maxima;
//   3. quant: the second pass of the quantizer with that permutation and
//      those group maxima (one partial row), so codes, alpha and s_b follow
//      the reordered positions exactly as with a static permutation.
#include "rrs_internal.h"

namespace rrs {
namespace {

constexpr int kOrderThreads = 1024;
constexpr int kMaxBlocks = 16384 / kReorderBlock;  // 512

// part: nrows x NB block maxima; NB = K / 32 in [16, 512].
// Outputs: order[p] = block at sorted position p (NB int32); perm[j] =
// channel at position j (K int32); gmax[b] = max key of group b for b < K/g,
// 0 for K/g <= b < max(K/64, 64) (the quant pass may read that far).
__global__ __launch_bounds__(kOrderThreads) void order_kernel(
    const float* __restrict__ part, int nrows, int K, int g, int32_t* __restrict__ order,
    int32_t* __restrict__ perm, float* __restrict__ gmax) {
  __shared__ __attribute__((aligned(16))) float red[kOrderThreads * 4];
  __shared__ __attribute__((aligned(16))) float key[kMaxBlocks];
  __shared__ float skey[kMaxBlocks];
  __shared__ int sblk[kMaxBlocks];
  const int tid = threadIdx.x;
  const int NB = K / kReorderBlock;
  const int NQ = NB / 4;             // float4 columns, 4 .. 128
  const int NS = kOrderThreads / NQ;  // row slices, 8 .. 256

  // 1. keys: thread (slice, quad) takes rows slice, slice + NS, ... of four
  //    adjacent blocks, eight independent loads at a time.
  {
    const int qd = tid % NQ;
    const int sl = tid / NQ;
    float4 m = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int i = sl; i < nrows; i += 8 * NS) {
      float4 x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int r = i + u * NS;
        x[u] = r < nrows ? reinterpret_cast<const float4*>(part + (size_t)r * NB)[qd]
                         : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        m.x = fmaxf(m.x, x[u].x);
        m.y = fmaxf(m.y, x[u].y);
        m.z = fmaxf(m.z, x[u].z);
        m.w = fmaxf(m.w, x[u].w);
      }
    }
    reinterpret_cast<float4*>(red)[sl * NQ + qd] = m;
  }
  __syncthreads();
  if (tid < NB) {
    float m = 0.0f;
    for (int sl = 0; sl < NS; ++sl) m = fmaxf(m, red[sl * NB + tid]);
    key[tid] = m;
  }
  __syncthreads();

  // 2. rank of block tid: blocks with a larger key, or an equal key and a
  //    smaller index, come first (the keys are broadcast LDS reads).
  if (tid < NB) {
    const float c = key[tid];
    int rank = 0;
    for (int q = 0; q < NB / 4; ++q) {
      const float4 v = reinterpret_cast<const float4*>(key)[q];
      const int b = 4 * q;
      rank += (v.x > c || (v.x == c && b < tid)) ? 1 : 0;
      rank += (v.y > c || (v.y == c && b + 1 < tid)) ? 1 : 0;
      rank += (v.z > c || (v.z == c && b + 2 < tid)) ? 1 : 0;
      rank += (v.w > c || (v.w == c && b + 3 < tid)) ? 1 : 0;
    }
    sblk[rank] = tid;
    skey[rank] = c;
    order[rank] = tid;
  }
  __syncthreads();

  // 3. group maxima over the sorted blocks, and the channel permutation.
  const int G = K / g;
  const int per = g / kReorderBlock;
  const int GW = max(K / 64, 64);
  if (tid < GW) {
    float m = 0.0f;
    if (tid < G)
      for (int u = 0; u < per; ++u) m = fmaxf(m, skey[tid * per + u]);
    gmax[tid] = m;
  }
  for (int j = tid; j < K; j += kOrderThreads)
    perm[j] = sblk[j / kReorderBlock] * kReorderBlock + (j % kReorderBlock);
}

size_t part_bytes(int K) { return align256((size_t)block_maxima_rows() * (K / kReorderBlock) * 4); }
size_t gmax_bytes(int K) { return align256((size_t)(K / 64 > 64 ? K / 64 : 64) * 4); }
size_t perm_bytes(int K) { return align256((size_t)K * 4); }

}  // namespace

size_t reorder_workspace_bytes(int K) { return part_bytes(K) + gmax_bytes(K) + perm_bytes(K); }

hipError_t launch_rotate_smooth_quant_reorder(const uint16_t* X, int M, int K, int g, int flags,
                                              uint8_t* Xq, float* a_scale, float* s_group,
                                              int32_t* block_order, void* workspace,
                                              hipStream_t stream) {
  char* ws = static_cast<char*>(workspace);
  float* part = reinterpret_cast<float*>(ws);
  ws += part_bytes(K);
  float* gmax = reinterpret_cast<float*>(ws);
  ws += gmax_bytes(K);
  int32_t* perm = reinterpret_cast<int32_t*>(ws);
  const bool rot = !(flags & kSkipRotation);
  int nrows = 0;
  hipError_t e = launch_block_maxima(X, M, K, rot, part, &nrows, stream);
  if (e != hipSuccess) return e;
  order_kernel<<<1, kOrderThreads, 0, stream>>>(part, nrows, K, g, block_order, perm, gmax);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_quantize_given_maxima(X, M, K, g, perm, rot, gmax, Xq, a_scale, s_group, stream);
}

}  // namespace rrs
