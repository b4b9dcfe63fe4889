/*
 * rrs.h - C ABI of the MI355X (gfx950) Rotated Runtime Smooth W4A4 linear layer.
 *
 * Method: "Rotated Runtime Smooth: Training-Free Activation Smoother for
 * accurate INT4 inference" (arXiv 2409.20361). The online path of one linear
 * layer rotates the activations with a Hadamard matrix (Section 3.3, Eq. 4),
 * takes runtime channel maxima over the token batch as group smoothing scales
 * (Eq. 1, Section 3.2), quantizes each token to symmetric INT4 (Section 2.1,
 * Eq. 2), and multiplies against offline-rotated INT4 weights with the group
 * scale applied to each block's integer partial sum (Eq. 3, Fig. 4 step (3)).
 *
 * Orientation: X is M x K (M tokens, K input channels), W is K x N (N output
 * channels), Y = X W is M x N. (The paper writes X as N x K and W as M x K.)
 *
 * Conventions for every function below:
 *  - Pointers are DEVICE pointers unless stated otherwise. The caller allocates
 *    and owns every buffer; no function here allocates device memory or keeps
 *    a pointer after it returns.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t passed as
 *    void*; NULL = the default stream). Outputs are valid once the stream has
 *    reached that point. Calls on different streams with disjoint buffers may
 *    run concurrently; the library holds no per-call state.
 *  - Arguments are validated on the host before any device work, in this
 *    order: null pointers, shapes, group size, flags (the _ex functions),
 *    alignment, workspace size, device present, device architecture. The
 *    first failing check decides the returned code and nothing is enqueued.
 *  - Shapes: M >= 1; N >= 1 and N % 16 == 0; K a power of two with
 *    512 <= K <= 16384. Group size g: g divides K and g is one of
 *    64, 128, 256, 512. Every pointer must be 16-byte aligned.
 *  - Preconditions: inputs finite; `perm` a permutation of 0..K-1 (and
 *    `block_order` of 0..K/32-1); buffers large enough for the stated sizes;
 *    no overlap between inputs and outputs. Violations are undefined
 *    behaviour (meaningless codes, never an out-of-bounds access). With the
 *    environment variable RRS_DEBUG set to a non-zero value (read at every
 *    call) the first two are checked after the checks above: the library
 *    copies X or W, perm / block_order and the float32 scales a call reads
 *    to host memory on `stream`, waits for them, and returns
 *    RRS_ERR_PRECONDITION (nothing enqueued) on a non-finite value or a
 *    non-permutation. Debug mode synchronises the stream, so it must not be
 *    used while the stream is captured into a graph.
 *  - Device-side faults surface at the caller's next synchronisation, as with
 *    any HIP launch; launch failures are returned as RRS_ERR_HIP.
 *
 * Data layouts (fixed by this library; the paper does not specify them):
 *  - X:  M x K float16, row-major.
 *  - W:  K x N float16, row-major (the transpose of nn.Linear's weight).
 *  - Xq: M x K/2 bytes, row-major. Codes are INT4 two's complement in
 *    [-7, 7], two per byte, the low nibble holding the even channel index.
 *  - Wq: N x K/2 bytes of the same packed codes, row-major (row n = output
 *    channel n, K contiguous): packed byte j of row n at n * K/2 + j.
 *    Optional tiled layout (flag RRS_WEIGHT_TILED of the _ex functions):
 *    rows in blocks of 16, each block stored as its K/128 tiles of 16 rows x
 *    64 bytes (1 KB) one after another, and inside a tile the four 16-byte
 *    quarters of the 16 rows quarter by quarter, so packed byte j of row n
 *    sits at
 *      (n / 16) * 8K + (j / 64) * 1024 + ((j % 64) / 16) * 256
 *        + (n % 16) * 16 + j % 16.
 *    There a wave's load of one K tile of 16 channels is one contiguous 1 KB
 *    run: for 17 to 64 tokens the GEMM streams it about 15 to 20 % faster
 *    than the row-major rows (up to 16 tokens both layouts stream at about
 *    the same rate). Results are bit-identical in both layouts; a weight
 *    prepared with the flag must be multiplied with it, and one prepared
 *    without it without it.
 *  - a_scale: M float32 (per token); w_scale: N float32 (per output channel);
 *    s_group: K/g float32 (one smoothing scale per channel group).
 *  - Y:  M x N float16, row-major.
 *
 * Arithmetic: rotation, scales and epilogue in float32 with IEEE
 * round-to-nearest-even, fp32 denormals preserved; integer partial sums are
 * exact int32. The rotation is applied unnormalized (x H_K, entries +-1) and
 * the 1/K of R R^T with R = H_K / sqrt(K) is folded into the output scale.
 */
#ifndef RRS_H_
#define RRS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rrs_status;

enum {
  RRS_OK = 0,
  RRS_ERR_NULL = -1,       /* a required pointer is NULL */
  RRS_ERR_SHAPE = -2,      /* M, N or K outside the supported set */
  RRS_ERR_GROUP = -3,      /* group size unsupported or not dividing K */
  RRS_ERR_ALIGN = -4,      /* a pointer is not 16-byte aligned */
  RRS_ERR_WORKSPACE = -5,  /* workspace smaller than the query returns */
  RRS_ERR_NO_DEVICE = -6,  /* no HIP device visible */
  RRS_ERR_ARCH = -7,       /* the current device is not gfx950 */
  RRS_ERR_HIP = -8,        /* a HIP runtime call or launch failed */
  RRS_ERR_FLAGS = -9,      /* unknown or unsupported flag bits (_ex functions) */
  RRS_ERR_PRECONDITION = -10, /* RRS_DEBUG only: an input is not finite, or perm /
                                 block_order is not a permutation */
  RRS_ERR_TIMEOUT = -11       /* RRS_DEBUG only: a bounded wait between workgroups ran
                                 out (the affected outputs were written as NaN) */
};

/*
 * Ablation switches for the _ex functions (the paper's own baselines,
 * Section 3.1 and Section 2.3; Tables 1 and 4). 0 selects RRS itself.
 *  - RRS_SKIP_ROTATION: no Hadamard rotation of activations or weights
 *    (plain Runtime Smooth); the GEMM output drops the 1/K.
 *  - RRS_SKIP_SMOOTHING: every smoothing scale is 1 (rotation followed by
 *    per-token quantization only, the QuaRot scheme); rrs_rotate_smooth_quant_ex
 *    then makes one pass over X instead of two and writes s_group = 1.
 * Pass the same flags to the quantization, weight-preparation and GEMM calls
 * of one layer (weight preparation and the GEMM take only RRS_SKIP_ROTATION
 * into account; RRS_SKIP_SMOOTHING is accepted and has no effect there, except
 * that rrs_prepare_weight_ex rejects it: weights are never smoothed).
 *
 * Layout switch (not an ablation): RRS_WEIGHT_TILED selects the tiled Wq
 * layout above for every call that writes or reads Wq. Every _ex function
 * accepts it; the ones that do not touch Wq ignore it, so one flags value
 * can serve all calls of a layer.
 */
enum { RRS_SKIP_ROTATION = 1, RRS_SKIP_SMOOTHING = 2, RRS_WEIGHT_TILED = 4 };

/* Human-readable name of a status code (static storage; never NULL). */
const char* rrs_status_string(rrs_status status);

/* Library version as major*10000 + minor*100 + patch. */
int rrs_version(void);

/*
 * Bytes of device workspace rrs_rotate_smooth_quant needs for this shape
 * (a 256-byte header and up to 256 rows of K/64 tagged 8-byte words for the
 * one-launch kernels' exchange of group maxima, then up to 256 rows of K/64
 * floats for the two-pass kernels). The workspace must hold zeros before its
 * first use (e.g. allocated with hipMemsetAsync(ws, 0, bytes)); every call
 * leaves it ready for the next call, with any shape, so one workspace can
 * serve a whole model. Calls that share a workspace must not overlap.
 * Returns 0 when the shape or group size is invalid.
 */
size_t rrs_workspace_bytes(int M, int K, int group_size);

/*
 * Offline weight preparation (Section 3.3: weights are rotated offline and
 * quantized per output channel; round-to-nearest stands in for GPTQ).
 *   W       in : K x N float16, row-major.
 *   perm    in : optional K int32 (NULL = identity). Row j of the rotated
 *                weight becomes row perm[j]'s rotation (the static channel
 *                reorder of Fig. 4 step (1)); pass the same perm to
 *                rrs_rotate_smooth_quant / rrs_linear.
 *   Wq      out: N x K/2 bytes, packed INT4 codes of u = H_K W per column,
 *                row-major (tiled with RRS_WEIGHT_TILED in the _ex call).
 *   w_scale out: N float32, beta_n = max_k |u_kn| / 7.
 * Not on the timed path.
 */
rrs_status rrs_prepare_weight(const void* W, int K, int N, const int32_t* perm,
                              void* Wq, float* w_scale, void* stream);

/* rrs_prepare_weight with flags: RRS_SKIP_ROTATION quantizes W itself
 * (u = W) for the ablation without rotation; RRS_WEIGHT_TILED writes the
 * tiled layout; any other bit -> RRS_ERR_FLAGS. */
rrs_status rrs_prepare_weight_ex(const void* W, int K, int N, const int32_t* perm, int flags,
                                 void* Wq, float* w_scale, void* stream);

/*
 * Online rotate + runtime smooth + per-token INT4 quantization
 * (Section 3.3 then Section 3.2; Eq. 1-2; Section 2.1).
 *   X        in : M x K float16, row-major.
 *   perm     in : optional K int32 (NULL = identity): position j of the
 *                 rotated token takes channel perm[j].
 *   Xq       out: M x K/2 bytes, packed codes.
 *   a_scale  out: M float32, alpha_i.
 *   s_group  out: K/g float32, s_b = the largest |rotated activation| over all
 *                 M tokens and the g channels of group b.
 *   workspace   : device scratch of at least rrs_workspace_bytes(M, K, g)
 *                 bytes; contents on entry are ignored, on exit undefined.
 */
rrs_status rrs_rotate_smooth_quant(const void* X, int M, int K, int group_size,
                                   const int32_t* perm, void* Xq, float* a_scale,
                                   float* s_group, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* rrs_rotate_smooth_quant with ablation flags (RRS_SKIP_ROTATION: y = x;
 * RRS_SKIP_SMOOTHING: s_b = r_b = 1). Same buffers and workspace. */
rrs_status rrs_rotate_smooth_quant_ex(const void* X, int M, int K, int group_size,
                                      const int32_t* perm, int flags, void* Xq, float* a_scale,
                                      float* s_group, void* workspace, size_t workspace_bytes,
                                      void* stream);

/*
 * W4A4 GEMM with Runtime Smooth fused into the block loop (Section 3.2,
 * Eq. 3, Fig. 4 step (3)):
 *   Y[i, n] = fp16( a_scale[i] * w_scale[n] / K * sum_b s_group[b] * P_b[i, n] ),
 *   P_b[i, n] = sum over the g channels j of group b of q_x[i, j] * q_w[j, n],
 * with every P_b an exact integer and the sum over b in float32.
 *   Xq, a_scale, s_group: as written by rrs_rotate_smooth_quant.
 *   Wq, w_scale         : as written by rrs_prepare_weight.
 *   Y out               : M x N float16, row-major.
 */
rrs_status rrs_w4a4_gemm(const void* Xq, const float* a_scale, const float* s_group,
                         const void* Wq, const float* w_scale, int M, int N, int K,
                         int group_size, void* Y, void* stream);

/* rrs_w4a4_gemm with ablation flags: with RRS_SKIP_ROTATION the operands are
 * unrotated and the output is a_scale[i] * w_scale[n] * sum_b s_group[b] P_b
 * (no 1/K). RRS_SKIP_SMOOTHING has no effect (the scales come from s_group). */
rrs_status rrs_w4a4_gemm_ex(const void* Xq, const float* a_scale, const float* s_group,
                            const void* Wq, const float* w_scale, int M, int N, int K,
                            int group_size, int flags, void* Y, void* stream);

/*
 * Bytes of workspace rrs_linear needs: rrs_workspace_bytes plus room for Xq,
 * a_scale and s_group, each sub-buffer aligned to 256 bytes. 0 when invalid.
 * As for rrs_workspace_bytes, the workspace must hold zeros before its first
 * use (the library-held scratch of rrs_linear_noalloc starts zeroed).
 */
size_t rrs_linear_workspace_bytes(int M, int K, int group_size);

/*
 * One RRS linear layer: rrs_rotate_smooth_quant followed by rrs_w4a4_gemm,
 * with Xq, a_scale and s_group kept in the workspace. For one or two tokens
 * at K = 2048, 4096 or 8192 (K >= 4 group_size, no perm, no RRS_SKIP_*
 * flag) the layer is a single launch in which every workgroup of the
 * weight-streaming GEMM quantizes the token rows itself (Section 3.3: the
 * rotation is online, inside the layer call); Y is bit-identical to the two
 * calls, and Xq, a_scale and s_group are then not written to the workspace.
 *   X in: M x K float16; Wq, w_scale from rrs_prepare_weight (same perm);
 *   Y out: M x N float16.
 */
rrs_status rrs_linear(const void* X, const void* Wq, const float* w_scale, int M, int N,
                      int K, int group_size, const int32_t* perm, void* Y,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * rrs_linear without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). The call allocates nothing: the
 * workspace of rrs_linear is taken from a scratch array that the library
 * holds in device memory, RRS_NOALLOC_SCRATCH_BYTES (16 MiB) on each device
 * the library runs on, kept until the process ends. Arguments, layouts and
 * results as rrs_linear (bit-identical outputs).
 *   Limit: rrs_linear_workspace_bytes(M, K, group_size) must not exceed
 *   RRS_NOALLOC_SCRATCH_BYTES (about M K / 2 bytes: up to 8079 tokens at
 *   K = 4096, 3995 at K = 8192, 1950 at K = 16384, with g = 128); larger
 *   calls return RRS_ERR_WORKSPACE and enqueue nothing.
 *   Every call on one device shares that device's scratch: calls that
 *   overlap on one device (concurrent streams, or host threads using
 *   different streams of the same device) race and give undefined results;
 *   serialize them (one stream, or events). Calls on different devices are
 *   independent.
 */
#define RRS_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
rrs_status rrs_linear_noalloc(const void* X, const void* Wq, const float* w_scale, int M, int N,
                              int K, int group_size, const int32_t* perm, void* Y,
                              void* stream);

/* rrs_linear with ablation flags (quantization and GEMM as in their _ex
 * forms); Wq and w_scale must come from rrs_prepare_weight_ex with the same
 * RRS_SKIP_ROTATION and RRS_WEIGHT_TILED bits. */
rrs_status rrs_linear_ex(const void* X, const void* Wq, const float* w_scale, int M, int N,
                         int K, int group_size, const int32_t* perm, int flags, void* Y,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Test hook for the failure path of the one-launch quantizers (not for
 * computing: use rrs_rotate_smooth_quant). Without a static reorder,
 * rrs_rotate_smooth_quant runs one launch for 2 to 16 tokens (one workgroup
 * per token row; up to 64 tokens for g >= K / 64 and up to 32 for
 * g = K / 128)
 * and, at K <= 4096, for more tokens too (one workgroup per compute unit, up
 * to two rows per wave). The workgroups exchange their group
 * maxima through the workspace (Eq. 1 takes the maximum over every token),
 * each polling, with a bound, until the words it needs have arrived. That
 * needs all workgroups of the launch to be resident at the same time, which
 * holds on an otherwise idle device but not when other work fills every
 * compute unit; a wait that runs out marks the call as failed in the
 * workspace, writes NaN into its rows' a_scale (workgroup 0 also into
 * s_group) and ends, so the failure shows in the outputs.
 * This hook runs the kernel rrs_rotate_smooth_quant would choose for
 * (M, K, group_size) with the readers also waiting for extra_rows rows of
 * maxima that no workgroup writes (>= 1 makes every wait run out) and giving
 * up after max_polls polling rounds (>= 1), waits for `stream`, and stores 1
 * in *failed (host pointer) if the exchange failed, else 0. Arguments
 * otherwise as rrs_rotate_smooth_quant with perm = NULL; RRS_ERR_SHAPE when
 * no one-launch kernel serves the shape, RRS_ERR_FLAGS for extra_rows < 0,
 * max_polls < 1 or more rows in all than the per-row kernel takes for the
 * shape (16, or the 32 or 64 above; 256 for the fused one). With RRS_DEBUG set, rrs_rotate_smooth_quant(_ex) and
 * rrs_linear(_ex) make the same check after a call that used a one-launch
 * kernel and return RRS_ERR_TIMEOUT when it failed.
 */
rrs_status rrs_test_quant_rows_wait(const void* X, int M, int K, int group_size,
                                    int extra_rows, int max_polls, void* Xq, float* a_scale,
                                    float* s_group, void* workspace, size_t workspace_bytes,
                                    int32_t* failed, void* stream);

/*
 * Test hook for the failure path of the one-launch runtime-reorder quantizer
 * (not for computing: use rrs_rotate_smooth_quant_reorder). For 2 to 16 tokens
 * at K <= 8192, rrs_rotate_smooth_quant_reorder is one launch of one
 * workgroup per token row whose rows exchange their K/32 block maxima through
 * the workspace; for more tokens at K <= 4096 (as many as the one-launch
 * rrs_rotate_smooth_quant takes) one launch of at most one workgroup per
 * compute unit, whose workgroups exchange their block maxima in two levels
 * (runs of 16 workgroups, then the runs). Both run under the same residency
 * condition and bounded waits as the one-launch rrs_rotate_smooth_quant (see
 * rrs_test_quant_rows_wait). This hook runs that kernel with the readers also
 * waiting for extra_rows rows of block maxima (token rows, or workgroups in
 * the many-token form) that no workgroup writes and giving up after
 * max_polls rounds, waits for `stream`, and stores 1 in *failed (host
 * pointer) if the exchange failed, else 0; a failed call leaves NaN in
 * a_scale and s_group. Arguments otherwise as rrs_rotate_smooth_quant_reorder
 * (flags = 0); RRS_ERR_SHAPE when the shape has no one-launch reorder (M < 2,
 * K > 8192, or more than 16 tokens at K > 4096 or beyond the one-launch
 * limit), RRS_ERR_FLAGS for extra_rows < 0, max_polls < 1, more than 16 rows
 * in all (per-row form) or more than 256 workgroups' rows in all
 * (many-token form).
 */
rrs_status rrs_test_quant_reorder_wait(const void* X, int M, int K, int group_size,
                                      int extra_rows, int max_polls, void* Xq, float* a_scale,
                                      float* s_group, int32_t* block_order, void* workspace,
                                      size_t workspace_bytes, int32_t* failed, void* stream);

/*
 * Test hook: the exact int32 group partials P[b][i][n] (b < K/g, i < M,
 * n < N; G x M x N int32, row-major), before any scaling (Eq. 3's inner sums
 * per block). Wq row-major. The call runs the same kernel that rrs_w4a4_gemm
 * runs for this shape (the few-token kernels for M <= 64, the main kernel
 * above), with the same accumulator seeding, and decodes each group's
 * accumulators instead of rescaling them.
 */
rrs_status rrs_w4a4_gemm_partials(const void* Xq, const void* Wq, int M, int N, int K,
                                  int group_size, int32_t* P, void* stream);

/*
 * ------------------------------------------------------------------------
 * Baselines of the kernel-efficiency comparison (Section 4.5, Fig. 6).
 * Per-channel A4W4 (one scale per token and per output channel, the setting
 * of QuaRot and SpinQuant), Runtime Smooth A4W4 (the same plus one smoothing
 * scale per group) and sub-channel A4W4 (one scale per (token, group) and per
 * (output channel, group)) run on one shared GEMM skeleton (128 x 128 tiles)
 * that differs between the three only in how scales are applied, so their
 * times compare the schemes, not the kernels. rrs_w4a4_gemm is the tuned
 * Runtime Smooth kernel and is not part of this comparison.
 * ------------------------------------------------------------------------
 */
enum {
  RRS_SCHEME_PER_CHANNEL = 0,
  RRS_SCHEME_RUNTIME_SMOOTH = 1,
  RRS_SCHEME_SUB_CHANNEL = 2
};

/*
 * Sub-channel quantization of activations: y = x H_K (x itself with
 * RRS_SKIP_ROTATION); for token i and group b of g channels,
 * m = max_j |y_ij|, inv = fl(7/m) (0 if m = 0), q = clamp(rint(fl(y inv)), -7, 7).
 *   X in      : M x K float16, row-major.
 *   Xq out    : M x K/2 bytes, packed as for rrs_rotate_smooth_quant.
 *   a_sub out : L x M float32, a_sub[b * M + i] = fl(m / 7), L = K / g (group-major).
 * One launch; no workspace. Shapes and errors as rrs_rotate_smooth_quant
 * (flags: RRS_SKIP_ROTATION; RRS_WEIGHT_TILED is accepted and ignored).
 */
rrs_status rrs_quantize_sub_channel(const void* X, int M, int K, int group_size, int flags,
                                    void* Xq, float* a_sub, void* stream);

/*
 * Sub-channel weight preparation: u = H_K W (W with RRS_SKIP_ROTATION), then
 * for output channel n and group b the same RTN as above.
 *   W in      : K x N float16, row-major.
 *   Wq out    : N x K/2 bytes, as rrs_prepare_weight_ex (RRS_WEIGHT_TILED
 *               for the tiled layout).
 *   w_sub out : L x N float32, w_sub[b * N + n] (group-major).
 */
rrs_status rrs_prepare_weight_sub_channel(const void* W, int K, int N, int group_size,
                                          int flags, void* Wq, float* w_sub, void* stream);

/*
 * GEMM of one scheme on the comparison skeleton; Y out M x N float16. With
 * norm = K (1 with RRS_SKIP_ROTATION):
 *   RRS_SCHEME_PER_CHANNEL   : Y = x_scale[i] w_scale[n] / norm * sum_j q_x q_w
 *                              (x_scale M, w_scale N; s_group unused, may be NULL;
 *                              inputs from rrs_rotate_smooth_quant_ex with
 *                              RRS_SKIP_SMOOTHING and rrs_prepare_weight_ex);
 *   RRS_SCHEME_RUNTIME_SMOOTH: Y as rrs_w4a4_gemm (x_scale M, s_group L, w_scale N);
 *   RRS_SCHEME_SUB_CHANNEL   : Y = 1 / norm * sum_b fl(x_scale[b M + i] w_scale[b N + n]) P_b
 *                              (x_scale L x M, w_scale L x N; s_group unused).
 * group_size is ignored by RRS_SCHEME_PER_CHANNEL (pass any valid one).
 * Errors as rrs_w4a4_gemm_ex; an unknown scheme is RRS_ERR_FLAGS.
 */
rrs_status rrs_w4a4_gemm_scheme(int scheme, const void* Xq, const float* x_scale,
                                const float* s_group, const void* Wq, const float* w_scale,
                                int M, int N, int K, int group_size, int flags, void* Y,
                                void* stream);

/*
 * Per-channel A4W4 GEMM (one scale per token and per output channel, no
 * smoothing; the setting of QuaRot and SpinQuant, Section 2.1) on the same
 * tuned main loop as rrs_w4a4_gemm, without its per-group rescale:
 *   Y[i, n] = fp16( a_scale[i] * w_scale[n] / norm * sum_j q_x[i, j] q_w[j, n] ),
 * norm = K (1 with RRS_SKIP_ROTATION). Inputs from rrs_rotate_smooth_quant_ex
 * with RRS_SKIP_SMOOTHING (its s_group is all ones and unused here) and
 * rrs_prepare_weight_ex. Shapes, alignment and errors as rrs_w4a4_gemm_ex.
 */
rrs_status rrs_w4a4_gemm_per_channel(const void* Xq, const float* a_scale, const void* Wq,
                                     const float* w_scale, int M, int N, int K, int flags,
                                     void* Y, void* stream);

/*
 * ------------------------------------------------------------------------
 * Runtime channel reorder (Fig. 4 step (1) taken at run time, Section 3.2):
 * before the grouping, the rotated channels are sorted by this call's
 * channel-wise maxima c_j = max_i |y_ij| (Eq. 1), so that channels of similar
 * size share a smoothing scale. Channels move in blocks of 32 consecutive
 * channels (RRS_REORDER_BLOCK): a block's key is its largest c_j, keys are
 * sorted largest first, equal keys keep increasing block index, and group b
 * takes the sorted blocks [b g/32, (b+1) g/32). The weights are prepared once
 * in natural order (rrs_prepare_weight with perm = NULL); the GEMM fetches
 * the weight block that belongs to each position.
 * ------------------------------------------------------------------------
 */
enum { RRS_REORDER_BLOCK = 32 };

/*
 * Bytes of device workspace rrs_rotate_smooth_quant_reorder needs (0 for
 * invalid arguments). It holds the one-launch kernels' header and exchanged
 * block maxima (16 rows of K/32 tagged words), then up to 256 rows of K/32
 * block maxima for the two-launch path, then, at K <= 4096, 256 rows of K/32
 * tagged words for the many-token one-launch kernel. As for
 * rrs_workspace_bytes, the workspace must hold zeros before its first use and
 * may then be reused by later calls (calls sharing one must not overlap).
 */
size_t rrs_reorder_workspace_bytes(int M, int K, int group_size);

/*
 * rrs_rotate_smooth_quant with the runtime reorder:
 *   X in            : M x K float16.
 *   Xq out          : M x K/2 bytes; position j of a row holds rotated channel
 *                     32 block_order[j / 32] + j % 32.
 *   a_scale out     : M float32; s_group out: K/g float32, over the reordered
 *                     positions (so s_group never increases with b).
 *   block_order out : K/32 int32, a permutation of 0..K/32-1.
 *   workspace       : at least rrs_reorder_workspace_bytes(M, K, g) bytes.
 * flags: RRS_SKIP_ROTATION (reorder the unrotated channels: Runtime Smooth
 * with its reorder step); RRS_SKIP_SMOOTHING -> RRS_ERR_FLAGS (without
 * smoothing the order changes nothing); RRS_WEIGHT_TILED is accepted and
 * ignored. Up to 16 tokens at K <= 8192 the call is one launch (one workgroup
 * per token row; the rows exchange their K/32 block maxima in the workspace
 * and every workgroup ranks the blocks itself); for more tokens at K <= 4096,
 * as many as the one-launch rrs_rotate_smooth_quant takes, also one launch
 * (workgroups exchange block maxima in two levels, rank the blocks and
 * quantize the rows they kept). Both under the same residency condition and
 * bounded waits as the one-launch rrs_rotate_smooth_quant (RRS_ERR_TIMEOUT
 * under RRS_DEBUG). Otherwise two launches (block maxima, then quantization,
 * whose every workgroup ranks the blocks itself).
 */
rrs_status rrs_rotate_smooth_quant_reorder(const void* X, int M, int K, int group_size,
                                           int flags, void* Xq, float* a_scale,
                                           float* s_group, int32_t* block_order,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream);

/*
 * rrs_w4a4_gemm whose position block p of Xq (channels [32 p, 32 p + 32))
 * pairs with block block_order[p] of every Wq row:
 *   Y[i, n] = fp16( alpha_i beta_n / norm * sum_b s_b sum_{j in group b}
 *                   q_x[i, j] q_w[32 block_order[j / 32] + j % 32, n] ),
 * norm = K (1 with RRS_SKIP_ROTATION). Wq, w_scale from rrs_prepare_weight
 * without perm; Xq, a_scale, s_group, block_order from
 * rrs_rotate_smooth_quant_reorder. block_order is read on the device and each
 * entry is reduced modulo K/32 (loads stay in bounds for any table; a table
 * that is not a permutation gives meaningless results). flags:
 * RRS_SKIP_ROTATION, RRS_WEIGHT_TILED. Other errors as rrs_w4a4_gemm_ex.
 */
rrs_status rrs_w4a4_gemm_reorder(const void* Xq, const float* a_scale, const float* s_group,
                                 const void* Wq, const float* w_scale,
                                 const int32_t* block_order, int M, int N, int K,
                                 int group_size, int flags, void* Y, void* stream);

/* Workspace of rrs_linear_reorder: the quantizer's workspace plus Xq,
 * a_scale, s_group and block_order (0 for invalid arguments). Zero before its
 * first use, as the quantizer's. */
size_t rrs_linear_reorder_workspace_bytes(int M, int K, int group_size);

/*
 * One RRS linear layer with the runtime reorder:
 * rrs_rotate_smooth_quant_reorder followed by rrs_w4a4_gemm_reorder, the
 * intermediates kept in the workspace. W prepared by rrs_prepare_weight
 * (perm = NULL, same RRS_SKIP_ROTATION and RRS_WEIGHT_TILED bits). Errors as
 * the two calls.
 */
rrs_status rrs_linear_reorder(const void* X, const void* Wq, const float* w_scale, int M,
                              int N, int K, int group_size, int flags, void* Y, void* workspace,
                              size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RRS_H_ */
