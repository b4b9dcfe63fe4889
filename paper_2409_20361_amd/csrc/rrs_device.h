// Internal device helpers shared by the rotate/quantize and weight-preparation
// kernels: fp16 row loads, the register/LDS fast Walsh-Hadamard transform and
// workgroup max reductions. gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rrs {

// Threads per workgroup for the row kernels: one row of K elements is spread
// over 256 threads, E = K / 256 consecutive elements per thread.
constexpr int kRowThreads = 256;
constexpr int kLogRowThreads = 8;

constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x >> 1); }

// LDS row buffer: one pad word per 16 floats keeps the strided transposes of
// the FWHT free of bank conflicts.
__device__ __forceinline__ int lds_pad(int p) { return p + (p >> 4); }
constexpr int lds_row_floats(int K) { return K + K / 16; }

__device__ __forceinline__ float half_to_float(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

// v[e] = float(src[e]) for e < E; src aligned to min(16, 2E) bytes.
template <int E>
__device__ __forceinline__ void load_halves(const uint16_t* __restrict__ src, float (&v)[E]) {
  if constexpr (E >= 8) {
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
#pragma unroll
    for (int c = 0; c < E / 8; ++c) {
      const uint4 w = s4[c];
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        v[c * 8 + 2 * m] = half_to_float(ws[m] & 0xFFFFu);
        v[c * 8 + 2 * m + 1] = half_to_float(ws[m] >> 16);
      }
    }
  } else if constexpr (E == 4) {
    const uint2 w = *reinterpret_cast<const uint2*>(src);
    v[0] = half_to_float(w.x & 0xFFFFu);
    v[1] = half_to_float(w.x >> 16);
    v[2] = half_to_float(w.y & 0xFFFFu);
    v[3] = half_to_float(w.y >> 16);
  } else {
    static_assert(E == 2, "E must be a power of two >= 2");
    const uint32_t w = *reinterpret_cast<const uint32_t*>(src);
    v[0] = half_to_float(w & 0xFFFFu);
    v[1] = half_to_float(w >> 16);
  }
}

// ---------------------------------------------------------------------------
// Fast Walsh-Hadamard transform of one row (y = x H_K, unnormalized).
//
// Stage order is h = 1, 2, 4, ..., K/2 and every butterfly output is a single
// rounded fp32 add or subtract, so the result is bit-identical to the
// canonical sequential definition. The K = 2^(8+L) indices are covered by
// "windows" of L = log2(E) index bits: in the window starting at bit `lo`,
// thread t holds the E elements
//   p(t, e) = (t mod 2^lo) | (e << lo) | ((t >> lo) << (lo + L)),
// so the window's stages are in-register butterflies. Windows advance through
// the bits in increasing order (the last one is shifted down to end at bit
// log2 K and only applies the stages not yet done); between windows the row
// goes through LDS.
// ---------------------------------------------------------------------------

template <int E, int J>
__device__ __forceinline__ void fwht_stage(float (&v)[E]) {
  constexpr int h = 1 << J;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    if ((e & h) == 0) {
      const float a = v[e];
      const float b = v[e + h];
      v[e] = a + b;
      v[e + h] = a - b;
    }
  }
}

template <int E, int J0, int J1>
__device__ __forceinline__ void fwht_stages(float (&v)[E]) {
  if constexpr (J0 < J1) {
    fwht_stage<E, J0>(v);
    fwht_stages<E, J0 + 1, J1>(v);
  }
}

__device__ __forceinline__ int window_index(int t, int e, int lo, int L) {
  return (t & ((1 << lo) - 1)) | (e << lo) | ((t >> lo) << (lo + L));
}

template <int K>
struct FwhtShape {
  static constexpr int E = K / kRowThreads;
  static constexpr int L = ilog2(E);
  static constexpr int LOGK = ilog2(K);
  static constexpr int kWindows = (LOGK + L - 1) / L;
  static constexpr int kFinalLo = LOGK - L;  // == kLogRowThreads
  static_assert(E >= 2 && (1 << L) == E, "K must be 2^(8+L), L >= 1");
};

template <int K, int W, bool kRot>
__device__ __forceinline__ void fwht_windows(float (&v)[FwhtShape<K>::E], float* lds, int t) {
  using S = FwhtShape<K>;
  if constexpr (W < S::kWindows) {
    constexpr int prev_lo = (W - 1) * S::L;
    constexpr int lo = (W * S::L < S::LOGK - S::L) ? W * S::L : S::LOGK - S::L;
    constexpr int first = W * S::L - lo;  // first e-bit not yet transformed
    __syncthreads();  // earlier readers of lds are done
#pragma unroll
    for (int e = 0; e < S::E; ++e) lds[lds_pad(window_index(t, e, prev_lo, S::L))] = v[e];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < S::E; ++e) v[e] = lds[lds_pad(window_index(t, e, lo, S::L))];
    if constexpr (kRot) fwht_stages<S::E, first, S::L>(v);
    fwht_windows<K, W + 1, kRot>(v, lds, t);
  }
}

// On entry v[e] holds element t*E + e of the row. On exit v[e] holds element
// t + e * 256 of x H_K (of x itself when kRot is false: the same data
// movement without the butterflies, for the ablation without rotation).
// `lds` must hold lds_row_floats(K) floats; it is clobbered. Must be called by
// all 256 threads of the workgroup.
template <int K, bool kRot = true>
__device__ __forceinline__ void fwht_row(float (&v)[FwhtShape<K>::E], float* lds, int t) {
  using S = FwhtShape<K>;
  if constexpr (kRot) fwht_stages<S::E, 0, S::L>(v);
  fwht_windows<K, 1, kRot>(v, lds, t);
}

// LDS address of position q of the rotated row in position-major order: row
// a = q / E (E floats) holds positions [a E, a E + E), thread a's share; its
// 4-float chunks are permuted by h(a) so that both the strided writes of the
// rotation's output (position t + 256 e from thread t) and the 128-bit chunk
// reads of the owner are free of bank conflicts.
template <int E>
__device__ __forceinline__ int pos_addr(int q) {
  constexpr int CH = E < 4 ? E : 4;  // floats per chunk
  constexpr int NCH = E / CH;        // chunks per row
  constexpr int S = ilog2(64 / E);   // rows per 64 banks = 2^S
  const int a = q / E;
  const int b = q % E;
  const int h = NCH > 1 ? (a >> S) & (NCH - 1) : 0;
  return a * E + ((b / CH) ^ h) * CH + b % CH;
}

// Thread t's E consecutive positions [t E, t E + E) of a row stored with
// pos_addr<E>, read as 128-bit chunks in the permuted order (E >= 4) or one
// by one.
template <int E>
__device__ __forceinline__ void read_positions(const float* row, int t, float (&v)[E]) {
  constexpr int CH = E < 4 ? E : 4;
  constexpr int NCH = E / CH;
  const int h = NCH > 1 ? (t >> ilog2(64 / E)) & (NCH - 1) : 0;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const float* src = row + t * E + (c ^ h) * CH;
    if constexpr (CH == 4) {
      const float4 x = *reinterpret_cast<const float4*>(src);
      v[4 * c] = x.x;
      v[4 * c + 1] = x.y;
      v[4 * c + 2] = x.z;
      v[4 * c + 3] = x.w;
    } else {
#pragma unroll
      for (int i = 0; i < CH; ++i) v[CH * c + i] = src[i];
    }
  }
}

// ---------------------------------------------------------------------------
// Reductions (values are non-negative and finite, so fmaxf is exact).
// ---------------------------------------------------------------------------

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// Max over the 256 threads of the workgroup; `red` is 4 floats of LDS.
__device__ __forceinline__ float block_max256(float x, float* red) {
  x = wave_max(x);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// Sub-channel quantization helper. On entry each of the 256 threads of a row
// team holds E consecutive channels [t E, t E + E) of the row, all inside one
// group of g (E <= 64 <= g), and lm = their largest |value|. Returns the
// largest |value| of this thread's group. `red` is 256 floats and `gm` K / g
// floats of LDS private to the team; contains workgroup barriers, so every
// thread of the workgroup must call it.
__device__ __forceinline__ float row_group_max(float lm, float* red, float* gm, int t, int E,
                                               int g, int G) {
  red[t] = lm;
  __syncthreads();
  const int per = g / E;  // threads per group
  if (t < G) {
    float m = 0.0f;
    for (int u = 0; u < per; ++u) m = fmaxf(m, red[t * per + u]);
    gm[t] = m;
  }
  __syncthreads();
  const float r = gm[(t * E) / g];
  __syncthreads();  // red and gm may be rewritten for the next row
  return r;
}

// ---------------------------------------------------------------------------
// Exchange between the workgroups of one launch (the one-launch quantizers).
//
// Each exchanged float travels as one 64-bit word, a tag in the high half and
// the float's bits in the low half, written with a single relaxed
// agent-scope atomic store; a reader polls the words it needs with relaxed
// agent-scope atomic loads until the tag is this call's. Each value carries
// its own tag, so the exchange rests on per-location coherence alone: no
// fence, no arrival count, no L2 write-back or invalidation (an agent-scope
// release / acquire pair per workgroup cost about 40 us at 256 workgroups in
// a probe; a count-based barrier with coherent data 6 us; tagged words 4 us).
//
// Tags come from an epoch word in the workspace header, zero before the
// workspace's first use: every workgroup reads the epoch E at its start and
// tags with T = next_epoch(E) (never 0, so zeroed words never match); once
// workgroup 0 has read every word of the call it stores T as the new epoch
// (all workgroups had read E before publishing, so none can see T too early).
// Words of earlier calls carry older tags; the
// tag repeats only after 2^32 - 1 calls. A wait that runs out stores T in
// header word 1 instead, so that a host check can see that the latest call
// failed (word 1 == word 0).
// ---------------------------------------------------------------------------
constexpr int kEpochWord = 0;
constexpr int kFailWord = 1;

__device__ __forceinline__ uint32_t next_epoch(uint32_t e) { return e + 1u == 0u ? 1u : e + 1u; }

__device__ __forceinline__ void publish_tagged(unsigned long long* w, uint32_t tag, float v) {
  __hip_atomic_store(w, ((unsigned long long)tag << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned long long load_tagged(const unsigned long long* w) {
  return __hip_atomic_load(const_cast<unsigned long long*>(w), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool has_tag(unsigned long long x, uint32_t tag) {
  return (uint32_t)(x >> 32) == tag;
}

// Symmetric INT4 code of v: clamp(rint(v), -7, 7) as a 4-bit two's complement nibble.
__device__ __forceinline__ uint32_t int4_nibble(float v) {
  const float q = fminf(fmaxf(__builtin_rintf(v), -7.0f), 7.0f);
  return (uint32_t)((int)q) & 0xFu;
}

// Codes of v[0..7] * m packed into one word, low nibble = even index:
// bit-identical to packing int4_nibble(v[e] * m) (same two roundings, same
// clamp). fl(fl(v m) + 1.5 * 2^23) is fl(v m) rounded to an integer, half to
// even (the binade of 1.5 * 2^23 has ulp 1), held in the low bits of the
// float's bit pattern, 0x4B400000 + q; clamping those bits to
// 0x4B400000 +- 7 (v_med3_i32) clamps q to [-7, 7], and the low nibble of
// 0x4B400000 + q is q's two's-complement nibble. Values far outside the
// binade clamp to +-7 as well; NaN (excluded by the preconditions) would
// not. 3 VALU ops per code plus 11 per word, against about 8 per code for
// rint / clamp / convert / pack.
__device__ __forceinline__ uint32_t quant_pack8(const float* v, float m) {
  int b[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int x = __builtin_bit_cast(int, __fadd_rn(__fmul_rn(v[e], m), 12582912.0f));
    b[e] = min(max(x, 0x4B400000 - 7), 0x4B400000 + 7);
  }
  uint32_t p[4];  // byte k in the low 8 bits: codes 2k (low nibble) and 2k + 1
#pragma unroll
  for (int k = 0; k < 4; ++k) p[k] = ((uint32_t)b[2 * k + 1] << 4) | ((uint32_t)b[2 * k] & 0xFu);
  const uint32_t lo = __builtin_amdgcn_perm(p[1], p[0], 0x0C0C0400u);  // bytes 0, 1
  const uint32_t hi = __builtin_amdgcn_perm(p[3], p[2], 0x04000C0Cu);  // bytes 2, 3
  return lo | hi;
}

// The order of the runtime reorder as one unsigned 64-bit sort key per block:
// the block key's bits above the complemented block index. Keys are
// non-negative and finite, so their bit patterns order as the keys do, and a
// larger sort key means a larger key, or an equal key and a smaller index.
__device__ __forceinline__ unsigned long long block_sort_key(float key, int b) {
  return ((unsigned long long)__float_as_uint(key) << 32) |
         (unsigned long long)(0xFFFFFFFFu - (uint32_t)b);
}
__device__ __forceinline__ float sort_key_value(unsigned long long k) {
  return __uint_as_float((uint32_t)(k >> 32));
}

// Rank of sort key `me` among the NB sort keys in LDS: how many are larger
// (two keys per 128-bit broadcast read, one 64-bit compare each; the rank of
// the float keys with their tie rule took about five operations per key).
template <int NB>
__device__ __forceinline__ int block_rank(const unsigned long long* sk, unsigned long long me) {
  static_assert(NB % 2 == 0, "pairs of keys");
  int rank = 0;
#pragma unroll 8
  for (int q = 0; q < NB / 2; ++q) {
    const uint4 v = reinterpret_cast<const uint4*>(sk)[q];
    const unsigned long long k0 = ((unsigned long long)v.y << 32) | v.x;
    const unsigned long long k1 = ((unsigned long long)v.w << 32) | v.z;
    rank += (k0 > me) ? 1 : 0;
    rank += (k1 > me) ? 1 : 0;
  }
  return rank;
}

// Count of the entries of A larger than x, for A of L distinct sort keys in
// LDS in decreasing order (L a power of two): a binary search, log2(L) + 1
// dependent reads.
template <int L>
__device__ __forceinline__ int count_greater(const unsigned long long* A, unsigned long long x) {
  int lo = 0;  // A[0 .. lo - 1] > x
#pragma unroll
  for (int s = L / 2; s >= 1; s >>= 1)
    if (A[lo + s - 1] > x) lo += s;
  return lo + (A[lo] > x ? 1 : 0);
}

// The runtime reorder's ranking: key holds the NB sort keys (block_sort_key);
// on return sblk[p] is the block at sorted position p and skey[p] its key. The
// blocks fall into lists of L = min(NB, 64); a block's rank is the number of
// larger sort keys in its own list (block_rank, broadcast reads) plus, for
// every other list, the number of larger ones in that list once sorted
// (count_greater). The sort keys are distinct, so the ranks are a permutation
// and equal to the count over all NB keys. srt is NB entries of LDS scratch.
// All NT threads of the workgroup call it; it ends with a barrier.
template <int NB, int NT>
__device__ __forceinline__ void rank_blocks(const unsigned long long* key, unsigned long long* srt,
                                            int* sblk, float* skey, int tid) {
  constexpr int L = NB < 64 ? NB : 64;
  constexpr int NL = NB / L;
  constexpr int PER = (NB + NT - 1) / NT;  // blocks per thread
  static_assert(NB % L == 0 && (L & (L - 1)) == 0, "lists of a power of two");
  unsigned long long me[PER];
  int r[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int b = tid + i * NT;
    me[i] = 0;
    r[i] = 0;
    if (b < NB) {
      me[i] = key[b];
      r[i] = block_rank<L>(key + (b / L) * L, me[i]);
      if constexpr (NL > 1) srt[(b / L) * L + r[i]] = me[i];
    }
  }
  if constexpr (NL > 1) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = tid + i * NT;
      if (b < NB) {
        const int own = b / L;
#pragma unroll
        for (int w = 0; w < NL; ++w)
          if (w != own) r[i] += count_greater<L>(srt + w * L, me[i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int b = tid + i * NT;
    if (b < NB) {
      sblk[r[i]] = b;
      skey[r[i]] = sort_key_value(me[i]);
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Runtime reorder (Fig. 4 step (1) at run time), computed by every workgroup
// of the quantizer's second pass: the key of block b (32 consecutive
// channels) is the largest of the nrows partial rows part[r][b] (r < nrows,
// NB = K / 32 entries per row); keys are ranked largest first, equal keys in
// increasing block index. On return (after a barrier) sblk[p] is the block at
// sorted position p and skey[p] its key. `red` holds at least 4 NT floats,
// `key` and `srt` NB entries each. All NT threads of the workgroup must call it.
// ---------------------------------------------------------------------------
template <int NT, int NB>
__device__ __forceinline__ void block_order_wg(const float* __restrict__ part, int nrows,
                                               float* red, unsigned long long* key,
                                               unsigned long long* srt, int* sblk, float* skey,
                                               int tid) {
  static_assert(NB % 4 == 0 && NB / 4 <= NT, "float4 columns, one per thread at least");
  constexpr int NQ = NB / 4;   // float4 columns of a partial row
  constexpr int NS = NT / NQ;  // row slices
  const int qd = tid % NQ;
  const int sl = tid / NQ;
  float4 m = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (sl < NS) {
    int i = sl;
    // eight independent loads at a time so their latencies overlap
    for (; i + 7 * NS < nrows; i += 8 * NS) {
      float4 x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = reinterpret_cast<const float4*>(part + (size_t)(i + u * NS) * NB)[qd];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        m.x = fmaxf(m.x, x[u].x);
        m.y = fmaxf(m.y, x[u].y);
        m.z = fmaxf(m.z, x[u].z);
        m.w = fmaxf(m.w, x[u].w);
      }
    }
    for (; i < nrows; i += NS) {
      const float4 x = reinterpret_cast<const float4*>(part + (size_t)i * NB)[qd];
      m.x = fmaxf(m.x, x.x);
      m.y = fmaxf(m.y, x.y);
      m.z = fmaxf(m.z, x.z);
      m.w = fmaxf(m.w, x.w);
    }
    reinterpret_cast<float4*>(red)[sl * NQ + qd] = m;
  }
  __syncthreads();
  for (int b = tid; b < NB; b += NT) {
    float k = red[b];
    for (int q = 1; q < NS; ++q) k = fmaxf(k, red[q * NB + b]);
    key[b] = block_sort_key(k, b);
  }
  __syncthreads();
  rank_blocks<NB, NT>(key, srt, sblk, skey, tid);
}

template <int E>
__device__ __forceinline__ void store_nibbles(uint8_t* __restrict__ dst, const uint32_t (&nib)[E]) {
  if constexpr (E >= 8) {
    uint32_t words[E / 8];
#pragma unroll
    for (int w = 0; w < E / 8; ++w) {
      uint32_t x = 0;
#pragma unroll
      for (int n = 0; n < 8; ++n) x |= nib[w * 8 + n] << (4 * n);
      words[w] = x;
    }
    if constexpr (E == 8) {
      *reinterpret_cast<uint32_t*>(dst) = words[0];
    } else if constexpr (E == 16) {
      *reinterpret_cast<uint2*>(dst) = make_uint2(words[0], words[1]);
    } else {
#pragma unroll
      for (int c = 0; c < E / 32; ++c)
        reinterpret_cast<uint4*>(dst)[c] =
            make_uint4(words[4 * c], words[4 * c + 1], words[4 * c + 2], words[4 * c + 3]);
    }
  } else if constexpr (E == 4) {
    const uint32_t x = nib[0] | (nib[1] << 4) | (nib[2] << 8) | (nib[3] << 12);
    *reinterpret_cast<uint16_t*>(dst) = (uint16_t)x;
  } else {
    *dst = (uint8_t)(nib[0] | (nib[1] << 4));
  }
}

}  // namespace rrs
