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
// Up to 16 tokens (K <= 8192) the whole quantizer is one launch of the
// per-row kernel (rrs_quant_rows.hip), which exchanges block maxima instead
// of group maxima and ranks the blocks in every workgroup. For more tokens at
// K <= 4096 it is one launch of the one-row-per-wave kernel
// (rrs_quant_wave.hip) in its reorder form: the workgroups exchange block
// maxima in two levels (runs of 16 workgroups, then the runs), rank the
// blocks and quantize the rows they kept in registers. Otherwise two
// launches on the caller's stream:
//   1. block maxima: the rot_max pass of the quantizer with groups of 32
//      natural-order channels, one row of K/32 maxima per workgroup;
//   2. quant: the second pass of the quantizer, whose every workgroup first
//      reduces those rows to the K/32 keys and ranks them (block_order_wg in
//      rrs_device.h), then quantizes its rows over the sorted positions, so
//      codes, alpha and s_b follow the reordered positions exactly as with a
//      static permutation; workgroup 0 writes block_order and s_group.
#include "rrs_internal.h"

namespace rrs {
namespace {

size_t part_bytes(int K) { return align256((size_t)block_maxima_rows() * (K / kReorderBlock) * 4); }

// The one-launch reorder kernel for many tokens: one row of K/32 tagged words
// per workgroup (at most 256).
size_t word_rows_bytes(int K) {
  return K <= 4096 ? align256((size_t)256 * (K / kReorderBlock) * 8) : 0;
}

bool fused_order_fits(int M, int K) {
  return !quant_rows_reorder_fits(M, K) && K <= 4096 && fused_quant_fits(M, K, fused_quant_wgs());
}

}  // namespace

// Layout: the header and the per-row kernel's tagged words (16 rows of K/32;
// the many-token kernel's runs use the same rows), then the two-launch path's
// rows of block maxima (floats, a region of their own so that no tagged word
// is ever read from them), then the many-token kernel's rows of tagged words.
// All of it zero before the first use.
size_t reorder_workspace_bytes(int K) {
  return quant_rows_reorder_workspace_bytes(K) + part_bytes(K) + word_rows_bytes(K);
}

bool reorder_one_launch(int M, int K) { return quant_rows_reorder_fits(M, K) || fused_order_fits(M, K); }

hipError_t launch_reorder_one_launch(const uint16_t* X, int M, int K, int g, bool rot,
                                     uint8_t* Xq, float* a_scale, float* s_group,
                                     int32_t* block_order, void* workspace, hipStream_t stream,
                                     int extra_rows, int max_polls) {
  if (quant_rows_reorder_fits(M, K))
    return launch_quant_rows_reorder(X, M, K, g, rot, Xq, a_scale, s_group, block_order,
                                     workspace, stream, extra_rows, max_polls);
  if (!fused_order_fits(M, K)) return hipErrorInvalidValue;
  char* ws = static_cast<char*>(workspace);
  return launch_rotate_smooth_quant_fused_order(
      X, M, K, g, rot, Xq, a_scale, s_group, block_order, reinterpret_cast<uint32_t*>(ws),
      reinterpret_cast<unsigned long long*>(ws + quant_rows_reorder_workspace_bytes(K) +
                                            part_bytes(K)),
      reinterpret_cast<unsigned long long*>(ws + kQuantHeaderBytes), fused_quant_wgs(), stream,
      extra_rows, max_polls);
}

hipError_t launch_rotate_smooth_quant_reorder(const uint16_t* X, int M, int K, int g, int flags,
                                              uint8_t* Xq, float* a_scale, float* s_group,
                                              int32_t* block_order, void* workspace,
                                              hipStream_t stream) {
  const bool rot = !(flags & kSkipRotation);
  if (reorder_one_launch(M, K))
    return launch_reorder_one_launch(X, M, K, g, rot, Xq, a_scale, s_group, block_order,
                                     workspace, stream, 0, 0);
  float* part = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                         quant_rows_reorder_workspace_bytes(K));
  int nrows = 0;
  hipError_t e = launch_block_maxima(X, M, K, rot, part, &nrows, stream);
  if (e != hipSuccess) return e;
  return launch_quantize_ordered(X, M, K, g, rot, part, nrows, Xq, a_scale, s_group,
                                 block_order, stream);
}

}  // namespace rrs
