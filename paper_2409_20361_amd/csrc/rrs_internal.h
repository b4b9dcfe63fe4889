// Internal launchers called by the C ABI layer (rrs_api.cpp). Each one
// enqueues kernels on `stream` and returns hipGetLastError(). Arguments are
// already validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rrs {

// Group-max partials: one row of K / g floats per workgroup of the first pass.
int quant_partial_rows(int M);
size_t quant_workspace_bytes(int M, int K);

// Workspace of rrs_rotate_smooth_quant, three disjoint regions:
//   [0, 256)                      header of the one-launch kernels: word 0 the
//                                 exchange epoch, word 1 the epoch of the last
//                                 exchange whose wait ran out;
//   [256, 256 + tagged_bytes(K))  tagged entries of the one-launch kernels
//                                 (64 bits: epoch tag << 32 | float bits);
//   then two_pass_bytes(K)        float partials of the two-pass kernels.
// The one-launch kernels need the header and entries to hold zeros before the
// workspace's first use (every call leaves them valid for the next).
constexpr size_t kQuantHeaderBytes = 256;
inline size_t quant_tagged_bytes(int K) { return ((size_t)256 * (K / 64) * 8 + 255) & ~size_t(255); }
inline size_t quant_two_pass_offset(int K) { return kQuantHeaderBytes + quant_tagged_bytes(K); }

// Ablation switches (the public RRS_SKIP_* flags).
constexpr int kSkipRotation = 1;
constexpr int kSkipSmoothing = 2;

// Channels per block of the runtime reorder: one MFMA k-step of 32 INT4
// codes, 16 bytes of a packed row.
constexpr int kReorderBlock = 32;

// Byte layout of Wq. Row-major (the default): row n at n K/2, K contiguous.
// Tiled (RRS_WEIGHT_TILED): rows in blocks of 16, each block's K/128 tiles of
// 16 rows x 64 bytes stored one after another, the tile's four 16-byte
// quarters of the 16 rows quarter by quarter. In both, piece p (packed bytes
// [16 p, 16 p + 16)) of row n sits at row(n) + (p / 4) tile() + (p % 4) quarter().
// The hot kernels take the layout as a template argument (a constexpr
// WqLayout), so that the strides fold into the load instructions' offsets.
struct WqLayout {
  bool tiled;
  constexpr __host__ __device__ size_t row(int n, int K) const {
    return tiled ? (size_t)(n >> 4) * ((size_t)8 * K) + (size_t)(n & 15) * 16
                 : (size_t)n * (size_t)(K / 2);
  }
  constexpr __host__ __device__ int tile() const { return tiled ? 1024 : 64; }
  constexpr __host__ __device__ int quarter() const { return tiled ? 256 : 16; }
  constexpr __host__ __device__ size_t piece(int n, int p, int K) const {
    return row(n, K) + (size_t)(p >> 2) * tile() + (size_t)(p & 3) * quarter();
  }
};

hipError_t launch_rotate_smooth_quant(const uint16_t* X, int M, int K, int g,
                                      const int32_t* perm, int flags, uint8_t* Xq,
                                      float* a_scale, float* s_group, void* workspace,
                                      hipStream_t stream);

// One-wave-per-row variant for K <= 4096 (same two passes, same bits).
hipError_t launch_rotate_smooth_quant_wave(const uint16_t* X, int M, int K, int g,
                                           const int32_t* perm, int flags, uint8_t* Xq,
                                           float* a_scale, float* s_group, void* workspace,
                                           int max_partials, int max_quant_wgs,
                                           hipStream_t stream);

// One-launch rotate + smooth + quant for K <= 4096 (rrs_quant_wave.hip):
// every row rotated once and kept in registers, the workgroups' group maxima
// exchanged through the workspace (an error word at offset 0, 64-bit tagged
// entries from byte 256), at most max_wgs workgroups (one per compute unit,
// all resident), two rows per wave at most. extra_rows > 0 / max_polls > 0:
// test hook only (the readers also wait for extra_rows rows that no
// workgroup writes, so every wait runs out after max_polls polls).
bool fused_quant_fits(int M, int K, int max_wgs);
int fused_quant_wgs();  // workgroups of the fused kernel: one per compute unit, at most 256
hipError_t launch_rotate_smooth_quant_fused(const uint16_t* X, int M, int K, int g, bool rotate,
                                            uint8_t* Xq, float* a_scale, float* s_group,
                                            void* workspace, int max_wgs, hipStream_t stream,
                                            int extra_rows = 0, int max_polls = 0);

// The same one-launch kernel with the runtime reorder (K <= 4096, the shapes
// fused_quant_fits accepts): block words of each workgroup in `tagged` (256 x
// K/32), of each run of 16 workgroups in `tagged2` (16 x K/32), under `header`.
hipError_t launch_rotate_smooth_quant_fused_order(const uint16_t* X, int M, int K, int g,
                                                  bool rotate, uint8_t* Xq, float* a_scale,
                                                  float* s_group, int32_t* block_order,
                                                  uint32_t* header, unsigned long long* tagged,
                                                  unsigned long long* tagged2, int max_wgs,
                                                  hipStream_t stream, int extra_rows = 0,
                                                  int max_polls = 0);

// Every launcher that writes or reads Wq takes its layout (row-major unless
// the caller asked for RRS_WEIGHT_TILED).
hipError_t launch_prepare_weight(const uint16_t* W, int K, int N, const int32_t* perm,
                                 bool rotate, uint8_t* Wq, float* w_scale, hipStream_t stream,
                                 WqLayout lay = {false});

// out_scale multiplies every output with alpha_i beta_n: 2^-8 / K for rotated
// operands, 2^-8 without rotation (both exact powers of two).
hipError_t launch_w4a4_gemm(const uint8_t* Xq, const float* a_scale, const float* s_group,
                            const uint8_t* Wq, const float* w_scale, int M, int N, int K,
                            int g, uint16_t* Y, float out_scale, hipStream_t stream,
                            WqLayout lay = {false});

hipError_t launch_w4a4_gemm_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                     int K, int g, int32_t* P, hipStream_t stream,
                                     WqLayout lay = {false});

// Simple 128 x 128 tile kernel: the fallback for shapes the main kernel's
// unrolling does not cover (K / 32 not a multiple of max(8, g / 32); no shape
// the ABI accepts today).
hipError_t launch_w4a4_gemm_small(const uint8_t* Xq, const float* a_scale,
                                  const float* s_group, const uint8_t* Wq,
                                  const float* w_scale, int M, int N, int K, int g,
                                  uint16_t* Y, float out_scale, hipStream_t stream,
                                  WqLayout lay = {false});
hipError_t launch_w4a4_gemm_partials_small(const uint8_t* Xq, const uint8_t* Wq, int M,
                                           int N, int K, int g, int32_t* P,
                                           hipStream_t stream, WqLayout lay = {false});

// Few-token kernel (decode): streams Wq once, for M <= 64 (up to four blocks
// of 16 tokens); its runtime-reorder variant takes M <= 16.
bool decode_kernel_fits(int M);
bool decode_gather_fits(int M);
// Runtime-reorder GEMM on the weight stream (rrs_gemm_stream.hip): up to 16
// tokens, K <= 8192, any g, either layout.
bool stream_gather_fits(int M, int K);
hipError_t launch_w4a4_gemm_stream_gather(const uint8_t* Xq, const float* a_scale,
                                          const float* s_group, const uint8_t* Wq,
                                          const float* w_scale, const int32_t* border, int M,
                                          int N, int K, int g, uint16_t* Y, float out_scale,
                                          hipStream_t stream, WqLayout lay);
hipError_t launch_w4a4_gemm_decode(const uint8_t* Xq, const float* a_scale,
                                   const float* s_group, const uint8_t* Wq,
                                   const float* w_scale, int M, int N, int K, int g,
                                   uint16_t* Y, float out_scale, hipStream_t stream,
                                   const int32_t* border = nullptr, WqLayout lay = {false});

hipError_t launch_w4a4_gemm_decode_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                            int K, int g, int32_t* P, hipStream_t stream);

// Weight-streaming kernel for few tokens (rrs_gemm_stream.hip): each
// workgroup copies 16 whole rows of Wq into LDS with direct-to-LDS loads.
// Up to 16 tokens: four waves, K >= 4 g (not K = 16384 with g <= 128). 17 to
// 32 tokens at K = 8192: eight waves and two blocks of 16 tokens. Both
// layouts, bit-identical results.
bool stream_kernel_fits(int M, int K, int g);
hipError_t launch_w4a4_gemm_stream(const uint8_t* Xq, const float* a_scale,
                                   const float* s_group, const uint8_t* Wq,
                                   const float* w_scale, int M, int N, int K, int g,
                                   uint16_t* Y, float out_scale, hipStream_t stream,
                                   WqLayout lay);
hipError_t launch_w4a4_gemm_stream_partials(const uint8_t* Xq, const uint8_t* Wq, int M, int N,
                                            int K, int g, int32_t* P, hipStream_t stream,
                                            WqLayout lay);
// The whole layer for one or two tokens in one launch of the weight-streaming
// kernel: every workgroup rotates, smooths and quantizes the rows itself,
// with the arithmetic of rrs_rotate_smooth_quant, so Y is bit-identical to the
// two launches. K = 2048, 4096 or 8192, K >= 4 g, rotation and smoothing on,
// no static reorder.
bool layer_one_launch_fits(int M, int K, int g);
hipError_t launch_layer_one_launch(const uint16_t* X, int M, int N, int K, int g,
                                   const uint8_t* Wq, const float* w_scale, uint16_t* Y,
                                   float out_scale, hipStream_t stream, WqLayout lay);

// Baselines of the kernel comparison (per-channel / sub-channel A4W4).
hipError_t launch_quantize_sub_channel(const uint16_t* X, int M, int K, int g, int flags,
                                       uint8_t* Xq, float* a_sub, hipStream_t stream);
hipError_t launch_prepare_weight_sub_channel(const uint16_t* W, int K, int N, int g, bool rotate,
                                             uint8_t* Wq, float* w_sub, hipStream_t stream,
                                             WqLayout lay = {false});
// scheme: 0 Runtime Smooth, 1 per-channel, 2 sub-channel (internal numbering).
hipError_t launch_w4a4_gemm_scheme(int scheme, const uint8_t* Xq, const float* x_scale,
                                   const float* s_group, const uint8_t* Wq, const float* w_scale,
                                   int M, int N, int K, int g, uint16_t* Y, float out_scale,
                                   hipStream_t stream, WqLayout lay = {false});

// Per-channel A4W4 on the tuned main loop (no per-group rescale).
hipError_t launch_w4a4_gemm_per_channel(const uint8_t* Xq, const float* a_scale,
                                       const uint8_t* Wq, const float* w_scale, int M, int N,
                                       int K, uint16_t* Y, float out_scale, hipStream_t stream,
                                       WqLayout lay = {false});

// Runtime channel reorder (Fig. 4 step (1) at run time). Pass 1: rows of
// K / 32 block maxima (at most block_maxima_rows() rows); pass 2: the
// quantizer's second pass with a given permutation and one row of group
// maxima (K / g used, max(K / 64, 64) readable).
int block_maxima_rows();
hipError_t launch_block_maxima(const uint16_t* X, int M, int K, bool rotate, float* part,
                               int* nrows, hipStream_t stream);
hipError_t launch_block_maxima_wave(const uint16_t* X, int M, int K, bool rotate, float* part,
                                    int max_partials, int* nrows, hipStream_t stream);
// Runtime reorder, second pass: every workgroup ranks the K/32 blocks from the
// nrows rows of block maxima in `part` itself, then quantizes its rows over
// the sorted positions; workgroup 0 writes s_group and block_order.
hipError_t launch_quantize_ordered(const uint16_t* X, int M, int K, int g, bool rotate,
                                   const float* part, int nrows, uint8_t* Xq, float* a_scale,
                                   float* s_group, int32_t* block_order, hipStream_t stream);
hipError_t launch_quantize_ordered_wave(const uint16_t* X, int M, int K, int g, bool rotate,
                                        const float* part, int nrows, int max_quant_wgs,
                                        uint8_t* Xq, float* a_scale, float* s_group,
                                        int32_t* block_order, hipStream_t stream);
size_t reorder_workspace_bytes(int K);
// Whether the runtime-reorder quantizer is one launch (the per-row kernel up
// to 16 tokens, the one-row-per-wave kernel for more at K <= 4096), and that
// launch with readers that also wait for extra_rows rows of words no
// workgroup writes, polling at most max_polls rounds (0: the default).
bool reorder_one_launch(int M, int K);
hipError_t launch_reorder_one_launch(const uint16_t* X, int M, int K, int g, bool rot,
                                     uint8_t* Xq, float* a_scale, float* s_group,
                                     int32_t* block_order, void* workspace, hipStream_t stream,
                                     int extra_rows, int max_polls);
hipError_t launch_rotate_smooth_quant_reorder(const uint16_t* X, int M, int K, int g, int flags,
                                              uint8_t* Xq, float* a_scale, float* s_group,
                                              int32_t* block_order, void* workspace,
                                              hipStream_t stream);
// GEMM whose Xq position block p pairs with Wq block border[p].
hipError_t launch_w4a4_gemm_reorder(const uint8_t* Xq, const float* a_scale,
                                    const float* s_group, const uint8_t* Wq,
                                    const float* w_scale, const int32_t* border, int M, int N,
                                    int K, int g, uint16_t* Y, float out_scale,
                                    hipStream_t stream, WqLayout lay = {false});

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Library-held scratch of rrs_linear_noalloc (rrs_noalloc.hip): a device
// array of kNoAllocScratchBytes per device; noalloc_scratch returns the
// current device's copy (its address resolved once per device).
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
hipError_t noalloc_scratch(void** ptr);

// rotate + smooth + quant with one workgroup per row for M <= 16 tokens, no
// static reorder, smoothing on (rrs_quant_rows.hip); uses the header and
// tagged entries of the workspace (zero before its first use). extra_rows > 0
// and max_polls > 0 are for the test hook only: the readers also wait for
// extra_rows rows that no workgroup writes (so every wait runs out) and give
// up after max_polls rounds (0 = the default bound).
bool quant_rows_fits(int M);
int quant_rows_max(int K, int g);  // rows the per-row kernel takes (no runtime reorder)
size_t quant_rows_workspace_bytes(int K, int g);
hipError_t launch_quant_rows(const uint16_t* X, int M, int K, int g, bool rotate, uint8_t* Xq,
                             float* a_scale, float* s_group, void* workspace, hipStream_t stream,
                             int extra_rows = 0, int max_polls = 0);
// Whether launch_rotate_smooth_quant takes the per-row kernel for this call.
bool quant_rows_used(int M, int K, int g, const int32_t* perm, int flags);
// The per-row kernel with the runtime reorder (up to 16 rows, K <= 8192): the
// rows exchange their K/32 block maxima and every workgroup ranks the blocks
// itself (one launch instead of block maxima, order and given-maxima passes).
// Uses the header and quant_rows_reorder_workspace_bytes(K) bytes in all.
bool quant_rows_reorder_fits(int M, int K);
size_t quant_rows_reorder_workspace_bytes(int K);
// extra_rows, max_polls: as launch_quant_rows (test hook only).
hipError_t launch_quant_rows_reorder(const uint16_t* X, int M, int K, int g, bool rotate,
                                     uint8_t* Xq, float* a_scale, float* s_group,
                                     int32_t* block_order, void* workspace, hipStream_t stream,
                                     int extra_rows = 0, int max_polls = 0);
// Waits for `stream` and reports whether the latest one-launch exchange in
// this workspace (per-row or fused kernel) had a wait that ran out.
hipError_t quant_exchange_failed(const void* workspace, hipStream_t stream, bool* failed);
// Whether launch_rotate_smooth_quant takes the fused one-launch kernel.
bool fused_quant_used(int M, int K, int g, const int32_t* perm, int flags);

}  // namespace rrs
