// C ABI of the RRS W4A4 linear layer: host-side validation, device and
// architecture checks, workspace layout, and launches on the caller's stream.
// Every check runs on the host before any device work is enqueued.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cmath>
#include <cstring>
#include <vector>

#include "rrs.h"
#include "rrs_internal.h"

namespace {

constexpr int kVersion = 601;  // 0.6.1: one-launch runtime-reorder quantizer for up to 16 tokens
constexpr int kMaxDevices = 64;

bool is_aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_k(int K) { return K >= 512 && K <= 16384 && (K & (K - 1)) == 0; }
bool valid_m(int M) { return M >= 1; }
bool valid_n(int N) { return N >= 1 && (N % 16) == 0; }
bool valid_group(int K, int g) {
  return (g == 64 || g == 128 || g == 256 || g == 512) && K % g == 0;
}
bool valid_flags(int flags, int allowed) { return (flags & ~allowed) == 0; }
// Every _ex function accepts RRS_WEIGHT_TILED, so that one flags value can
// serve all calls of a layer; only the calls that read or write Wq use it.
constexpr int kQuantFlags = RRS_SKIP_ROTATION | RRS_SKIP_SMOOTHING;
constexpr int kAllFlags = kQuantFlags | RRS_WEIGHT_TILED;
constexpr int kRotationFlags = RRS_SKIP_ROTATION | RRS_WEIGHT_TILED;
static_assert(RRS_SKIP_ROTATION == rrs::kSkipRotation && RRS_SKIP_SMOOTHING == rrs::kSkipSmoothing,
              "public and internal flag values agree");

rrs::WqLayout layout(int flags) { return rrs::WqLayout{(flags & RRS_WEIGHT_TILED) != 0}; }

// Output scale of the GEMM: 2^-8 undoes the 16 x 16 of the unpacked int8
// operands, 1/K the unnormalized rotation (absent without rotation).
float out_scale(int K, int flags) {
  const float s = std::ldexp(1.0f, -8);
  return (flags & RRS_SKIP_ROTATION) ? s : s / (float)K;
}

// RRS_DEBUG is read at every call (a getenv, far below a launch's cost), so a
// process can switch the checks on and off between calls.
bool debug_enabled() {
  const char* v = std::getenv("RRS_DEBUG");
  return v != nullptr && v[0] != '\0' && v[0] != '0';
}

// ---------------------------------------------------------------------------
// RRS_DEBUG precondition checks. They run after the regular validation (so
// the pointers are non-null and aligned and the device is a gfx950), copy
// the checked input to host memory on the caller's stream and wait for it,
// so they must not be used while the stream is being captured into a graph.
// ---------------------------------------------------------------------------

// Copies `bytes` bytes of device memory to `host` on `st` and waits.
rrs_status debug_fetch(void* host, const void* dev, size_t bytes, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (bytes == 0) return RRS_OK;
  if (hipMemcpyAsync(host, dev, bytes, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_HIP;
  }
  return RRS_OK;
}

// `perm` (n entries) holds every value of 0..n-1 exactly once.
rrs_status debug_check_perm(const int32_t* perm, int n, const char* what, void* stream) {
  if (!perm) return RRS_OK;
  std::vector<int32_t> h((size_t)n);
  if (rrs_status e = debug_fetch(h.data(), perm, (size_t)n * 4, stream)) return e;
  std::vector<unsigned char> seen((size_t)n, 0);
  for (int j = 0; j < n; ++j) {
    const int32_t v = h[(size_t)j];
    if (v < 0 || v >= n || seen[(size_t)v]) {
      std::fprintf(stderr, "[rrs] RRS_DEBUG: %s is not a permutation of 0..%d (entry %d = %d)\n",
                   what, n - 1, j, (int)v);
      return RRS_ERR_PRECONDITION;
    }
    seen[(size_t)v] = 1;
  }
  return RRS_OK;
}

// Every float16 of the count at `p` is finite (exponent field not all ones).
rrs_status debug_check_finite_f16(const void* p, size_t count, const char* what, void* stream) {
  std::vector<uint16_t> h(count);
  if (rrs_status e = debug_fetch(h.data(), p, count * 2, stream)) return e;
  for (size_t i = 0; i < count; ++i) {
    if ((h[i] & 0x7C00u) == 0x7C00u) {
      std::fprintf(stderr, "[rrs] RRS_DEBUG: %s[%zu] is not finite (bits 0x%04x)\n", what, i,
                   (unsigned)h[i]);
      return RRS_ERR_PRECONDITION;
    }
  }
  return RRS_OK;
}

// After a quantizer launch under RRS_DEBUG: waits for the stream and fails
// when a one-launch kernel (per-row or fused, used for this shape) reported a
// wait that ran out in its exchange.
rrs_status debug_check_quant_wait(int M, int K, int g, const int32_t* perm, int flags,
                                  const void* workspace, void* stream) {
  const bool rows = rrs::quant_rows_used(M, K, g, perm, flags & kQuantFlags) && M >= 2;
  if (!rows && !rrs::fused_quant_used(M, K, g, perm, flags & kQuantFlags)) return RRS_OK;
  bool failed = false;
  if (rrs::quant_exchange_failed(workspace, static_cast<hipStream_t>(stream), &failed) !=
      hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_HIP;
  }
  if (failed) {
    std::fprintf(stderr, "[rrs] RRS_DEBUG: a wait between workgroups ran out in the quantizer\n");
    return RRS_ERR_TIMEOUT;
  }
  return RRS_OK;
}

// The same check for the runtime-reorder quantizer, which is one launch (an
// exchange between the row workgroups) for up to 16 tokens at K <= 8192.
rrs_status debug_check_reorder_wait(int M, int K, const void* workspace, void* stream) {
  if (M < 2 || !rrs::reorder_one_launch(M, K)) return RRS_OK;
  bool failed = false;
  if (rrs::quant_exchange_failed(workspace, static_cast<hipStream_t>(stream), &failed) !=
      hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_HIP;
  }
  if (failed) {
    std::fprintf(stderr, "[rrs] RRS_DEBUG: a wait between workgroups ran out in the quantizer\n");
    return RRS_ERR_TIMEOUT;
  }
  return RRS_OK;
}

// Every float32 of the count at `p` is finite.
rrs_status debug_check_finite_f32(const float* p, size_t count, const char* what,
                                  void* stream) {
  std::vector<float> h(count);
  if (rrs_status e = debug_fetch(h.data(), p, count * 4, stream)) return e;
  for (size_t i = 0; i < count; ++i) {
    if (!std::isfinite(h[i])) {
      std::fprintf(stderr, "[rrs] RRS_DEBUG: %s[%zu] is not finite (%g)\n", what, i,
                   (double)h[i]);
      return RRS_ERR_PRECONDITION;
    }
  }
  return RRS_OK;
}

// 0 = unknown, 1 = gfx950, 2 = other architecture.
std::atomic<int> g_arch_cache[kMaxDevices];

rrs_status check_device() {
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) {
    (void)hipGetLastError();
    return RRS_ERR_NO_DEVICE;
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_NO_DEVICE;
  }
  int cached = (dev >= 0 && dev < kMaxDevices) ? g_arch_cache[dev].load() : 0;
  if (cached == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
      (void)hipGetLastError();
      return RRS_ERR_HIP;
    }
    cached = (std::strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
    if (dev >= 0 && dev < kMaxDevices) g_arch_cache[dev].store(cached);
  }
  return cached == 1 ? RRS_OK : RRS_ERR_ARCH;
}

rrs_status from_hip(hipError_t e) { return e == hipSuccess ? RRS_OK : RRS_ERR_HIP; }

size_t linear_ws_bytes(int M, int K, int g) {
  return rrs::quant_workspace_bytes(M, K) + rrs::align256((size_t)M * (K / 2)) +
         rrs::align256((size_t)M * 4) + rrs::align256((size_t)(K / g) * 4);
}

static_assert(RRS_REORDER_BLOCK == rrs::kReorderBlock, "public and internal block sizes agree");

size_t linear_reorder_ws_bytes(int M, int K, int g) {
  return rrs::reorder_workspace_bytes(K) + rrs::align256((size_t)M * (K / 2)) +
         rrs::align256((size_t)M * 4) + rrs::align256((size_t)(K / g) * 4) +
         rrs::align256((size_t)(K / RRS_REORDER_BLOCK) * 4);
}

rrs_status linear_run(const void* X, const void* Wq, const float* w_scale, int M, int N, int K,
                      int group_size, const int32_t* perm, int flags, void* Y, void* workspace,
                      void* stream);

}  // namespace

extern "C" {

const char* rrs_status_string(rrs_status s) {
  switch (s) {
    case RRS_OK: return "RRS_OK";
    case RRS_ERR_NULL: return "RRS_ERR_NULL: a required pointer is NULL";
    case RRS_ERR_SHAPE:
      return "RRS_ERR_SHAPE: need M >= 1, N >= 1 with N % 16 == 0, K a power of two in "
             "[512, 16384]";
    case RRS_ERR_GROUP: return "RRS_ERR_GROUP: group size must be 64, 128, 256 or 512 and divide K";
    case RRS_ERR_ALIGN: return "RRS_ERR_ALIGN: every pointer must be 16-byte aligned";
    case RRS_ERR_WORKSPACE: return "RRS_ERR_WORKSPACE: workspace smaller than required";
    case RRS_ERR_NO_DEVICE: return "RRS_ERR_NO_DEVICE: no HIP device visible";
    case RRS_ERR_ARCH: return "RRS_ERR_ARCH: current device is not gfx950";
    case RRS_ERR_HIP: return "RRS_ERR_HIP: a HIP call or kernel launch failed";
    case RRS_ERR_FLAGS: return "RRS_ERR_FLAGS: unknown or unsupported flag bits";
    case RRS_ERR_TIMEOUT:
      return "RRS_ERR_TIMEOUT: (RRS_DEBUG) a bounded wait between workgroups ran out; the "
             "affected outputs are NaN";
    case RRS_ERR_PRECONDITION:
      return "RRS_ERR_PRECONDITION: (RRS_DEBUG) an input is not finite or a permutation is "
             "not one";
    default: return "RRS_ERR_UNKNOWN";
  }
}

int rrs_version(void) { return kVersion; }

size_t rrs_workspace_bytes(int M, int K, int group_size) {
  if (!valid_m(M) || !valid_k(K) || !valid_group(K, group_size)) return 0;
  return rrs::quant_workspace_bytes(M, K);
}

size_t rrs_linear_workspace_bytes(int M, int K, int group_size) {
  if (!valid_m(M) || !valid_k(K) || !valid_group(K, group_size)) return 0;
  return linear_ws_bytes(M, K, group_size);
}

rrs_status rrs_prepare_weight_ex(const void* W, int K, int N, const int32_t* perm, int flags,
                                 void* Wq, float* w_scale, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] prepare_weight W=%p K=%d N=%d perm=%p flags=%d Wq=%p w_scale=%p\n", W,
                 K, N, (const void*)perm, flags, Wq, (void*)w_scale);
  if (!W || !Wq || !w_scale) return RRS_ERR_NULL;
  if (!valid_k(K) || !valid_n(N)) return RRS_ERR_SHAPE;
  if (!valid_flags(flags, kRotationFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(W) || !is_aligned(Wq) || !is_aligned(w_scale) || (perm && !is_aligned(perm)))
    return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_finite_f16(W, (size_t)K * N, "W", stream)) return s;
    if (rrs_status s = debug_check_perm(perm, K, "perm", stream)) return s;
  }
  return from_hip(rrs::launch_prepare_weight(
      static_cast<const uint16_t*>(W), K, N, perm, !(flags & RRS_SKIP_ROTATION),
      static_cast<uint8_t*>(Wq), w_scale, static_cast<hipStream_t>(stream), layout(flags)));
}

rrs_status rrs_prepare_weight(const void* W, int K, int N, const int32_t* perm, void* Wq,
                              float* w_scale, void* stream) {
  return rrs_prepare_weight_ex(W, K, N, perm, 0, Wq, w_scale, stream);
}

rrs_status rrs_rotate_smooth_quant_ex(const void* X, int M, int K, int group_size,
                                      const int32_t* perm, int flags, void* Xq, float* a_scale,
                                      float* s_group, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] rotate_smooth_quant X=%p M=%d K=%d g=%d perm=%p flags=%d Xq=%p a=%p "
                 "s=%p ws=%p (%zu B)\n",
                 X, M, K, group_size, (const void*)perm, flags, Xq, (void*)a_scale,
                 (void*)s_group, workspace, workspace_bytes);
  if (!X || !Xq || !a_scale || !s_group || !workspace) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kAllFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(s_group) ||
      !is_aligned(workspace) || (perm && !is_aligned(perm)))
    return RRS_ERR_ALIGN;
  if (workspace_bytes < rrs::quant_workspace_bytes(M, K)) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_finite_f16(X, (size_t)M * K, "X", stream)) return s;
    if (rrs_status s = debug_check_perm(perm, K, "perm", stream)) return s;
  }
  const rrs_status st = from_hip(rrs::launch_rotate_smooth_quant(
      static_cast<const uint16_t*>(X), M, K, group_size, perm, flags & kQuantFlags,
      static_cast<uint8_t*>(Xq), a_scale, s_group, workspace, static_cast<hipStream_t>(stream)));
  if (st == RRS_OK && debug_enabled())
    return debug_check_quant_wait(M, K, group_size, perm, flags, workspace, stream);
  return st;
}

rrs_status rrs_rotate_smooth_quant(const void* X, int M, int K, int group_size,
                                   const int32_t* perm, void* Xq, float* a_scale,
                                   float* s_group, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  return rrs_rotate_smooth_quant_ex(X, M, K, group_size, perm, 0, Xq, a_scale, s_group,
                                    workspace, workspace_bytes, stream);
}

rrs_status rrs_w4a4_gemm_ex(const void* Xq, const float* a_scale, const float* s_group,
                            const void* Wq, const float* w_scale, int M, int N, int K,
                            int group_size, int flags, void* Y, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] w4a4_gemm Xq=%p a=%p s=%p Wq=%p w=%p M=%d N=%d K=%d g=%d flags=%d "
                 "Y=%p\n",
                 Xq, (const void*)a_scale, (const void*)s_group, Wq, (const void*)w_scale, M, N,
                 K, group_size, flags, Y);
  if (!Xq || !a_scale || !s_group || !Wq || !w_scale || !Y) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kAllFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(s_group) || !is_aligned(Wq) ||
      !is_aligned(w_scale) || !is_aligned(Y))
    return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_finite_f32(a_scale, (size_t)M, "a_scale", stream)) return s;
    if (rrs_status s = debug_check_finite_f32(s_group, (size_t)(K / group_size), "s_group", stream))
      return s;
    if (rrs_status s = debug_check_finite_f32(w_scale, (size_t)N, "w_scale", stream)) return s;
  }
  return from_hip(rrs::launch_w4a4_gemm(
      static_cast<const uint8_t*>(Xq), a_scale, s_group, static_cast<const uint8_t*>(Wq),
      w_scale, M, N, K, group_size, static_cast<uint16_t*>(Y), out_scale(K, flags),
      static_cast<hipStream_t>(stream), layout(flags)));
}

rrs_status rrs_w4a4_gemm(const void* Xq, const float* a_scale, const float* s_group,
                         const void* Wq, const float* w_scale, int M, int N, int K,
                         int group_size, void* Y, void* stream) {
  return rrs_w4a4_gemm_ex(Xq, a_scale, s_group, Wq, w_scale, M, N, K, group_size, 0, Y, stream);
}

rrs_status rrs_linear_ex(const void* X, const void* Wq, const float* w_scale, int M, int N,
                         int K, int group_size, const int32_t* perm, int flags, void* Y,
                         void* workspace, size_t workspace_bytes, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] linear X=%p Wq=%p w=%p M=%d N=%d K=%d g=%d perm=%p flags=%d Y=%p ws=%p "
                 "(%zu B)\n",
                 X, Wq, (const void*)w_scale, M, N, K, group_size, (const void*)perm, flags, Y,
                 workspace, workspace_bytes);
  if (!X || !Wq || !w_scale || !Y || !workspace) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kAllFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Wq) || !is_aligned(w_scale) || !is_aligned(Y) ||
      !is_aligned(workspace) || (perm && !is_aligned(perm)))
    return RRS_ERR_ALIGN;
  if (workspace_bytes < linear_ws_bytes(M, K, group_size)) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_finite_f16(X, (size_t)M * K, "X", stream)) return s;
    if (rrs_status s = debug_check_perm(perm, K, "perm", stream)) return s;
    if (rrs_status s = debug_check_finite_f32(w_scale, (size_t)N, "w_scale", stream)) return s;
  }
  return linear_run(X, Wq, w_scale, M, N, K, group_size, perm, flags, Y, workspace, stream);
}

}  // extern "C"

namespace {

// The layer on a validated call: quantizer then GEMM, with Xq, alpha and s in
// the workspace (rrs_linear_workspace_bytes bytes).
rrs_status linear_run(const void* X, const void* Wq, const float* w_scale, int M, int N, int K,
                      int group_size, const int32_t* perm, int flags, void* Y, void* workspace,
                      void* stream) {
  char* ws = static_cast<char*>(workspace);
  void* qws = ws;
  ws += rrs::quant_workspace_bytes(M, K);
  uint8_t* xq = reinterpret_cast<uint8_t*>(ws);
  ws += rrs::align256((size_t)M * (K / 2));
  float* a = reinterpret_cast<float*>(ws);
  ws += rrs::align256((size_t)M * 4);
  float* s = reinterpret_cast<float*>(ws);

  hipStream_t st = static_cast<hipStream_t>(stream);
  // One or two tokens: the whole layer in one launch (no exchange, so no
  // wait to check).
  if (!perm && (flags & kQuantFlags) == 0 && rrs::layer_one_launch_fits(M, K, group_size))
    return from_hip(rrs::launch_layer_one_launch(
        static_cast<const uint16_t*>(X), M, N, K, group_size, static_cast<const uint8_t*>(Wq),
        w_scale, static_cast<uint16_t*>(Y), out_scale(K, flags), st, layout(flags)));
  hipError_t e = rrs::launch_rotate_smooth_quant(static_cast<const uint16_t*>(X), M, K,
                                                 group_size, perm, flags & kQuantFlags, xq, a,
                                                 s, qws, st);
  if (e != hipSuccess) return RRS_ERR_HIP;
  const rrs_status r = from_hip(rrs::launch_w4a4_gemm(
      xq, a, s, static_cast<const uint8_t*>(Wq), w_scale, M, N, K, group_size,
      static_cast<uint16_t*>(Y), out_scale(K, flags), st, layout(flags)));
  if (r == RRS_OK && debug_enabled())
    return debug_check_quant_wait(M, K, group_size, perm, flags, qws, stream);
  return r;
}

}  // namespace

extern "C" {

rrs_status rrs_linear(const void* X, const void* Wq, const float* w_scale, int M, int N,
                      int K, int group_size, const int32_t* perm, void* Y, void* workspace,
                      size_t workspace_bytes, void* stream) {
  return rrs_linear_ex(X, Wq, w_scale, M, N, K, group_size, perm, 0, Y, workspace,
                       workspace_bytes, stream);
}

rrs_status rrs_linear_noalloc(const void* X, const void* Wq, const float* w_scale, int M, int N,
                              int K, int group_size, const int32_t* perm, void* Y,
                              void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] linear_noalloc X=%p Wq=%p w=%p M=%d N=%d K=%d g=%d perm=%p Y=%p\n", X,
                 Wq, (const void*)w_scale, M, N, K, group_size, (const void*)perm, Y);
  if (!X || !Wq || !w_scale || !Y) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!is_aligned(X) || !is_aligned(Wq) || !is_aligned(w_scale) || !is_aligned(Y) ||
      (perm && !is_aligned(perm)))
    return RRS_ERR_ALIGN;
  // The library-held scratch takes the place of the workspace.
  if (linear_ws_bytes(M, K, group_size) > rrs::kNoAllocScratchBytes) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_finite_f16(X, (size_t)M * K, "X", stream)) return s;
    if (rrs_status s = debug_check_perm(perm, K, "perm", stream)) return s;
    if (rrs_status s = debug_check_finite_f32(w_scale, (size_t)N, "w_scale", stream)) return s;
  }
  void* ws = nullptr;
  if (rrs::noalloc_scratch(&ws) != hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_HIP;
  }
  return linear_run(X, Wq, w_scale, M, N, K, group_size, perm, 0, Y, ws, stream);
}

rrs_status rrs_quantize_sub_channel(const void* X, int M, int K, int group_size, int flags,
                                    void* Xq, float* a_sub, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr, "[rrs] quantize_sub_channel X=%p M=%d K=%d g=%d flags=%d Xq=%p a=%p\n",
                 X, M, K, group_size, flags, Xq, (void*)a_sub);
  if (!X || !Xq || !a_sub) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kRotationFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Xq) || !is_aligned(a_sub)) return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled())
    if (rrs_status s = debug_check_finite_f16(X, (size_t)M * K, "X", stream)) return s;
  return from_hip(rrs::launch_quantize_sub_channel(
      static_cast<const uint16_t*>(X), M, K, group_size, flags & RRS_SKIP_ROTATION,
      static_cast<uint8_t*>(Xq), a_sub,
      static_cast<hipStream_t>(stream)));
}

rrs_status rrs_prepare_weight_sub_channel(const void* W, int K, int N, int group_size,
                                          int flags, void* Wq, float* w_sub, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr, "[rrs] prepare_weight_sub_channel W=%p K=%d N=%d g=%d flags=%d\n", W, K,
                 N, group_size, flags);
  if (!W || !Wq || !w_sub) return RRS_ERR_NULL;
  if (!valid_k(K) || !valid_n(N)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kRotationFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(W) || !is_aligned(Wq) || !is_aligned(w_sub)) return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled())
    if (rrs_status s = debug_check_finite_f16(W, (size_t)K * N, "W", stream)) return s;
  return from_hip(rrs::launch_prepare_weight_sub_channel(
      static_cast<const uint16_t*>(W), K, N, group_size, !(flags & RRS_SKIP_ROTATION),
      static_cast<uint8_t*>(Wq), w_sub, static_cast<hipStream_t>(stream), layout(flags)));
}

rrs_status rrs_w4a4_gemm_scheme(int scheme, const void* Xq, const float* x_scale,
                                const float* s_group, const void* Wq, const float* w_scale,
                                int M, int N, int K, int group_size, int flags, void* Y,
                                void* stream) {
  if (debug_enabled())
    std::fprintf(stderr, "[rrs] w4a4_gemm_scheme %d M=%d N=%d K=%d g=%d flags=%d\n", scheme, M,
                 N, K, group_size, flags);
  if (scheme != RRS_SCHEME_PER_CHANNEL && scheme != RRS_SCHEME_RUNTIME_SMOOTH &&
      scheme != RRS_SCHEME_SUB_CHANNEL)
    return RRS_ERR_FLAGS;
  const bool need_s = scheme == RRS_SCHEME_RUNTIME_SMOOTH;
  if (!Xq || !x_scale || !Wq || !w_scale || !Y || (need_s && !s_group)) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kAllFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(Xq) || !is_aligned(x_scale) || (need_s && !is_aligned(s_group)) ||
      !is_aligned(Wq) || !is_aligned(w_scale) || !is_aligned(Y))
    return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  const int internal = scheme == RRS_SCHEME_PER_CHANNEL ? 1
                       : scheme == RRS_SCHEME_SUB_CHANNEL ? 2
                                                          : 0;
  return from_hip(rrs::launch_w4a4_gemm_scheme(
      internal, static_cast<const uint8_t*>(Xq), x_scale, s_group,
      static_cast<const uint8_t*>(Wq), w_scale, M, N, K, group_size, static_cast<uint16_t*>(Y),
      out_scale(K, flags), static_cast<hipStream_t>(stream), layout(flags)));
}

rrs_status rrs_w4a4_gemm_per_channel(const void* Xq, const float* a_scale, const void* Wq,
                                     const float* w_scale, int M, int N, int K, int flags,
                                     void* Y, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr, "[rrs] w4a4_gemm_per_channel M=%d N=%d K=%d flags=%d\n", M, N, K, flags);
  if (!Xq || !a_scale || !Wq || !w_scale || !Y) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_flags(flags, kAllFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(Wq) || !is_aligned(w_scale) ||
      !is_aligned(Y))
    return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  return from_hip(rrs::launch_w4a4_gemm_per_channel(
      static_cast<const uint8_t*>(Xq), a_scale, static_cast<const uint8_t*>(Wq), w_scale, M, N, K,
      static_cast<uint16_t*>(Y), out_scale(K, flags), static_cast<hipStream_t>(stream),
      layout(flags)));
}

size_t rrs_reorder_workspace_bytes(int M, int K, int group_size) {
  if (!valid_m(M) || !valid_k(K) || !valid_group(K, group_size)) return 0;
  return rrs::reorder_workspace_bytes(K);
}

size_t rrs_linear_reorder_workspace_bytes(int M, int K, int group_size) {
  if (!valid_m(M) || !valid_k(K) || !valid_group(K, group_size)) return 0;
  return linear_reorder_ws_bytes(M, K, group_size);
}

rrs_status rrs_rotate_smooth_quant_reorder(const void* X, int M, int K, int group_size,
                                           int flags, void* Xq, float* a_scale,
                                           float* s_group, int32_t* block_order,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] rotate_smooth_quant_reorder X=%p M=%d K=%d g=%d flags=%d Xq=%p a=%p "
                 "s=%p order=%p ws=%p (%zu B)\n",
                 X, M, K, group_size, flags, Xq, (void*)a_scale, (void*)s_group,
                 (void*)block_order, workspace, workspace_bytes);
  if (!X || !Xq || !a_scale || !s_group || !block_order || !workspace) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kRotationFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(s_group) ||
      !is_aligned(block_order) || !is_aligned(workspace))
    return RRS_ERR_ALIGN;
  if (workspace_bytes < rrs::reorder_workspace_bytes(K)) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled())
    if (rrs_status s = debug_check_finite_f16(X, (size_t)M * K, "X", stream)) return s;
  const rrs_status r = from_hip(rrs::launch_rotate_smooth_quant_reorder(
      static_cast<const uint16_t*>(X), M, K, group_size, flags & RRS_SKIP_ROTATION,
      static_cast<uint8_t*>(Xq), a_scale, s_group, block_order, workspace,
      static_cast<hipStream_t>(stream)));
  if (r == RRS_OK && debug_enabled()) return debug_check_reorder_wait(M, K, workspace, stream);
  return r;
}

rrs_status rrs_w4a4_gemm_reorder(const void* Xq, const float* a_scale, const float* s_group,
                                 const void* Wq, const float* w_scale,
                                 const int32_t* block_order, int M, int N, int K,
                                 int group_size, int flags, void* Y, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr, "[rrs] w4a4_gemm_reorder M=%d N=%d K=%d g=%d flags=%d order=%p\n", M,
                 N, K, group_size, flags, (const void*)block_order);
  if (!Xq || !a_scale || !s_group || !Wq || !w_scale || !block_order || !Y) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kRotationFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(s_group) || !is_aligned(Wq) ||
      !is_aligned(w_scale) || !is_aligned(block_order) || !is_aligned(Y))
    return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_perm(block_order, K / RRS_REORDER_BLOCK, "block_order", stream))
      return s;
    if (rrs_status s = debug_check_finite_f32(a_scale, (size_t)M, "a_scale", stream)) return s;
    if (rrs_status s = debug_check_finite_f32(s_group, (size_t)(K / group_size), "s_group", stream))
      return s;
    if (rrs_status s = debug_check_finite_f32(w_scale, (size_t)N, "w_scale", stream)) return s;
  }
  return from_hip(rrs::launch_w4a4_gemm_reorder(
      static_cast<const uint8_t*>(Xq), a_scale, s_group, static_cast<const uint8_t*>(Wq),
      w_scale, block_order, M, N, K, group_size, static_cast<uint16_t*>(Y), out_scale(K, flags),
      static_cast<hipStream_t>(stream), layout(flags)));
}

rrs_status rrs_linear_reorder(const void* X, const void* Wq, const float* w_scale, int M,
                              int N, int K, int group_size, int flags, void* Y, void* workspace,
                              size_t workspace_bytes, void* stream) {
  if (debug_enabled())
    std::fprintf(stderr,
                 "[rrs] linear_reorder X=%p Wq=%p w=%p M=%d N=%d K=%d g=%d flags=%d Y=%p ws=%p "
                 "(%zu B)\n",
                 X, Wq, (const void*)w_scale, M, N, K, group_size, flags, Y, workspace,
                 workspace_bytes);
  if (!X || !Wq || !w_scale || !Y || !workspace) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!valid_flags(flags, kRotationFlags)) return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Wq) || !is_aligned(w_scale) || !is_aligned(Y) ||
      !is_aligned(workspace))
    return RRS_ERR_ALIGN;
  if (workspace_bytes < linear_reorder_ws_bytes(M, K, group_size)) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  if (debug_enabled()) {
    if (rrs_status s = debug_check_finite_f16(X, (size_t)M * K, "X", stream)) return s;
    if (rrs_status s = debug_check_finite_f32(w_scale, (size_t)N, "w_scale", stream)) return s;
  }

  char* ws = static_cast<char*>(workspace);
  void* qws = ws;
  ws += rrs::reorder_workspace_bytes(K);
  uint8_t* xq = reinterpret_cast<uint8_t*>(ws);
  ws += rrs::align256((size_t)M * (K / 2));
  float* a = reinterpret_cast<float*>(ws);
  ws += rrs::align256((size_t)M * 4);
  float* s = reinterpret_cast<float*>(ws);
  ws += rrs::align256((size_t)(K / group_size) * 4);
  int32_t* order = reinterpret_cast<int32_t*>(ws);

  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = rrs::launch_rotate_smooth_quant_reorder(
      static_cast<const uint16_t*>(X), M, K, group_size, flags & RRS_SKIP_ROTATION, xq, a, s,
      order, qws, st);
  if (e != hipSuccess) return RRS_ERR_HIP;
  const rrs_status r = from_hip(rrs::launch_w4a4_gemm_reorder(
      xq, a, s, static_cast<const uint8_t*>(Wq), w_scale, order, M, N, K, group_size,
      static_cast<uint16_t*>(Y), out_scale(K, flags), st, layout(flags)));
  if (r == RRS_OK && debug_enabled()) return debug_check_reorder_wait(M, K, qws, stream);
  return r;
}

rrs_status rrs_test_quant_rows_wait(const void* X, int M, int K, int group_size,
                                    int extra_rows, int max_polls, void* Xq, float* a_scale,
                                    float* s_group, void* workspace, size_t workspace_bytes,
                                    int32_t* failed, void* stream) {
  if (!X || !Xq || !a_scale || !s_group || !workspace || !failed) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  const bool rows = M >= 2 && rrs::quant_rows_used(M, K, group_size, nullptr, 0);
  const bool fused = rrs::fused_quant_used(M, K, group_size, nullptr, 0);
  if (!rows && !fused) return RRS_ERR_SHAPE;
  if (extra_rows < 0 || max_polls < 1 ||
      (rows && M + extra_rows > rrs::quant_rows_max(K, group_size)))
    return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(s_group) ||
      !is_aligned(workspace))
    return RRS_ERR_ALIGN;
  if (workspace_bytes < rrs::quant_workspace_bytes(M, K)) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e =
      rows ? rrs::launch_quant_rows(static_cast<const uint16_t*>(X), M, K, group_size, true,
                                    static_cast<uint8_t*>(Xq), a_scale, s_group, workspace, st,
                                    extra_rows, max_polls)
           : rrs::launch_rotate_smooth_quant_fused(static_cast<const uint16_t*>(X), M, K,
                                                   group_size, true, static_cast<uint8_t*>(Xq),
                                                   a_scale, s_group, workspace,
                                                   rrs::fused_quant_wgs(), st, extra_rows,
                                                   max_polls);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e == hipErrorInvalidValue ? RRS_ERR_FLAGS : RRS_ERR_HIP;
  }
  bool f = false;
  if (rrs::quant_exchange_failed(workspace, st, &f) != hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_HIP;
  }
  *failed = f ? 1 : 0;
  return RRS_OK;
}

rrs_status rrs_test_quant_reorder_wait(const void* X, int M, int K, int group_size,
                                      int extra_rows, int max_polls, void* Xq, float* a_scale,
                                      float* s_group, int32_t* block_order, void* workspace,
                                      size_t workspace_bytes, int32_t* failed, void* stream) {
  if (!X || !Xq || !a_scale || !s_group || !block_order || !workspace || !failed)
    return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (M < 2 || !rrs::reorder_one_launch(M, K)) return RRS_ERR_SHAPE;
  if (extra_rows < 0 || max_polls < 1) return RRS_ERR_FLAGS;
  if (rrs::quant_rows_reorder_fits(M, K) && M + extra_rows > 16) return RRS_ERR_FLAGS;
  if (!is_aligned(X) || !is_aligned(Xq) || !is_aligned(a_scale) || !is_aligned(s_group) ||
      !is_aligned(block_order) || !is_aligned(workspace))
    return RRS_ERR_ALIGN;
  if (workspace_bytes < rrs::reorder_workspace_bytes(K)) return RRS_ERR_WORKSPACE;
  if (rrs_status s = check_device()) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e = rrs::launch_reorder_one_launch(
      static_cast<const uint16_t*>(X), M, K, group_size, true, static_cast<uint8_t*>(Xq),
      a_scale, s_group, block_order, workspace, st, extra_rows, max_polls);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e == hipErrorInvalidValue ? RRS_ERR_FLAGS : RRS_ERR_HIP;
  }
  bool f = false;
  if (rrs::quant_exchange_failed(workspace, st, &f) != hipSuccess) {
    (void)hipGetLastError();
    return RRS_ERR_HIP;
  }
  *failed = f ? 1 : 0;
  return RRS_OK;
}

rrs_status rrs_w4a4_gemm_partials(const void* Xq, const void* Wq, int M, int N, int K,
                                  int group_size, int32_t* P, void* stream) {
  if (!Xq || !Wq || !P) return RRS_ERR_NULL;
  if (!valid_m(M) || !valid_n(N) || !valid_k(K)) return RRS_ERR_SHAPE;
  if (!valid_group(K, group_size)) return RRS_ERR_GROUP;
  if (!is_aligned(Xq) || !is_aligned(Wq) || !is_aligned(P)) return RRS_ERR_ALIGN;
  if (rrs_status s = check_device()) return s;
  return from_hip(rrs::launch_w4a4_gemm_partials(static_cast<const uint8_t*>(Xq),
                                                 static_cast<const uint8_t*>(Wq), M, N, K,
                                                 group_size, P, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
