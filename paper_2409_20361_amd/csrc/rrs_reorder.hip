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
// of group maxima and ranks the blocks in every workgroup. Otherwise two
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

}  // namespace

// Layout: the one-launch kernel's header and tagged words (zero before the
// first use), then the two-launch path's rows of block maxima.
size_t reorder_workspace_bytes(int K) { return quant_rows_reorder_workspace_bytes(K) + part_bytes(K); }

bool reorder_one_launch(int M, int K) { return quant_rows_reorder_fits(M, K); }

hipError_t launch_rotate_smooth_quant_reorder(const uint16_t* X, int M, int K, int g, int flags,
                                              uint8_t* Xq, float* a_scale, float* s_group,
                                              int32_t* block_order, void* workspace,
                                              hipStream_t stream) {
  const bool rot = !(flags & kSkipRotation);
  // Up to 16 tokens (K <= 8192): one launch, one workgroup per row.
  if (reorder_one_launch(M, K))
    return launch_quant_rows_reorder(X, M, K, g, rot, Xq, a_scale, s_group, block_order,
                                     workspace, stream);
  float* part = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                         quant_rows_reorder_workspace_bytes(K));
  int nrows = 0;
  hipError_t e = launch_block_maxima(X, M, K, rot, part, &nrows, stream);
  if (e != hipSuccess) return e;
  return launch_quantize_ordered(X, M, K, g, rot, part, nrows, Xq, a_scale, s_group,
                                 block_order, stream);
}

}  // namespace rrs
