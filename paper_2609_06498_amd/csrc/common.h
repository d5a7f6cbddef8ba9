// Shared device helpers of the DFlow HIP library (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include "gemm.h"

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
// global-address-space view of 16-byte fragments (loads compile to global_load_dwordx4)
typedef const __attribute__((address_space(1))) u32x4_t gu4;
typedef const __attribute__((address_space(1))) float gf32;

namespace dflow {

constexpr int WAVE = 64;
constexpr int PAGE = 64;          // KV page size in tokens (also the attention sub-chunk)
constexpr int SSQ_LD = 512;       // row stride of the RMSNorm partial sums [row][strip] (d <= 16 * SSQ_LD)
// Keys per attention split (fixed absolute positions): at most 4 pages bf16, 2
// pages fp32, so the staged K+V pages of a split fit the 160 KB LDS of a CU.
// Split size of a context, from its dimensions only (never from a batch): the
// largest split (fewest partials to merge, every split re-reads the query
// rows) unless a full-capacity round launch with it -- max_batch sequences
// at max_keys, one workgroup per kv head and split -- would leave compute
// units idle (fewer workgroups than the MI355X's 256 units), then 128 keys
// (Qwen3-1.7B shape at context 1024: attention 16.5 -> 13.8 us per layer;
// Qwen3-8B shape at context 4096, b = 1: 19.3 -> 18.7 us; at 8 sequences the
// 256-key chunks of the multi-chunk splits win).
constexpr int SPLIT_RULE_CUS = 256;
inline int split_keys_for(bool bf16, int max_batch, int n_kv_heads, int max_keys) {
  if (!bf16) return 128;
  return (long long)max_batch * n_kv_heads * ((max_keys + 255) / 256) >= SPLIT_RULE_CUS ? 256 : 128;
}

// Chunks per attention split in the round calls (verify and draft).  One chunk
// (split = split_keys_for keys) while a full-capacity round launch -- every
// sequence at max_keys, batch x kv heads x splits workgroups -- fits one
// workgroup per compute unit; beyond, each split streams that many chunks
// (running softmax across them) so the full-capacity launch keeps about one
// workgroup per unit and the partials to merge shrink accordingly (8 ragged
// Qwen3-8B-shape sequences: attention + merge 72.4 -> 58.2 us per layer).  At
// most 64 pages per split (one page-id lane each).  Fixed per context, so a
// row's split and chunk boundaries never depend on the batch.
inline int round_chunks_for(int max_batch, int n_kv_heads, int max_keys, int chunk_keys, int cus) {
  const long long items = (long long)max_batch * n_kv_heads * ((max_keys + chunk_keys - 1) / chunk_keys);
  const long long c = cus > 0 ? (items + cus - 1) / cus : 1;
  const int cap = 64 * PAGE / chunk_keys;
  return c < 1 ? 1 : (c > cap ? cap : (int)c);
}

// ------------------------------------------------------------------ bf16 storage
struct bf16 { uint16_t u; };

__device__ __host__ inline float bf2f(uint16_t u) {
  union { uint32_t i; float f; } c;
  c.i = (uint32_t)u << 16;
  return c.f;
}
// fp32 -> bf16 round-to-nearest-even with the gfx950 conversion instruction
// (v_cvt_pk_bf16_f32; bit-identical to the integer RNE formula on every
// finite input, and NaN stays NaN)
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_hw_t __attribute__((ext_vector_type(2)));
__device__ inline uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// two values packed low | high << 16 in one instruction
__device__ inline uint32_t f2bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_hw_t));
}


// Storage-type traits.  A "lane fragment" is the 16 bytes one lane feeds to
// the matrix core per tile: 8 bf16 or 4 fp32 consecutive k values.
template <typename T> struct TT;
template <> struct TT<bf16> {
  static constexpr int KL = 8;          // elements per 16-byte lane fragment
  static constexpr int KT = 32;         // k extent of a 16x(KT) weight tile
  __device__ static inline float ld(const bf16* p, size_t i) { return bf2f(p[i].u); }
  __device__ static inline void st(bf16* p, size_t i, float v) { p[i].u = f2bf(v); }
  __device__ static inline float rnd(float v) { return bf2f(f2bf(v)); }
};
template <> struct TT<float> {
  static constexpr int KL = 4;
  static constexpr int KT = 16;
  __device__ static inline float ld(const float* p, size_t i) { return p[i]; }
  __device__ static inline void st(float* p, size_t i, float v) { p[i] = v; }
  __device__ static inline float rnd(float v) { return v; }
};

// Matrix-core operand order of an activation block [rows][K] (the A operand
// of a skinny projection): 16-row tiles of KT columns, 1 KB per (row tile, k
// tile), lane l holding KL consecutive k values of row l%16 at k chunk l/16 --
// one contiguous 16-byte load per lane, the k tiles of a row tile adjacent.
// A producer that feeds a projection writes this copy besides its row-major
// output; ktiles = K/KT of the consumer and c0 the
// producer's first column within the consumer's K (the capture layers write
// their slices of the W_c input).
template <typename T>
__device__ inline size_t afrag_off(int m, int c, int ktiles) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  return ((((size_t)(m >> 4) * ktiles + c / KT) * 64 + ((c % KT) / KL) * 16 + (m & 15)) * KL) + (c % KL);
}
template <typename T>
__device__ inline void frag_st(const FragOut& f, int m, int c, float v) {
  if (f.p) TT<T>::st(reinterpret_cast<T*>(f.p), afrag_off<T>(m, f.c0 + c, f.ktiles), v);
}

// 16 consecutive elements (16-byte aligned) <-> fp32, stores rounded to the storage type
// n consecutive values of row m from column c (c and n multiples of KL, the
// producer's c0 too) as whole 16-byte lane fragments of the copy
template <typename T>
__device__ inline void frag_st_run(const FragOut& f, int m, int c, const float* v, int n) {
  if (!f.p) return;
  constexpr int KL = TT<T>::KL;
  for (int q = 0; q < n; q += KL) {
    uint4 u;
    if constexpr (sizeof(T) == 2) {
      u = make_uint4(f2bf2(v[q], v[q + 1]), f2bf2(v[q + 2], v[q + 3]), f2bf2(v[q + 4], v[q + 5]),
                     f2bf2(v[q + 6], v[q + 7]));
    } else {
      u = make_uint4(__float_as_uint(v[q]), __float_as_uint(v[q + 1]), __float_as_uint(v[q + 2]),
                     __float_as_uint(v[q + 3]));
    }
    *reinterpret_cast<uint4*>(reinterpret_cast<T*>(f.p) + afrag_off<T>(m, f.c0 + c + q, f.ktiles)) = u;
  }
}

template <typename T> struct Row16;
template <> struct Row16<bf16> {
  __device__ static inline void load(const bf16* p, float* v) {
    const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint4 u = q[h];
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) { v[8 * h + 2 * i] = bf2f(w[i] & 0xFFFF); v[8 * h + 2 * i + 1] = bf2f(w[i] >> 16); }
    }
  }
  __device__ static inline void store(bf16* p, const float* v) {
    uint4* q = reinterpret_cast<uint4*>(p);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = f2bf2(v[8 * h + 2 * i], v[8 * h + 2 * i + 1]);
      q[h] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
};
template <> struct Row16<float> {
  __device__ static inline void load(const float* p, float* v) {
    const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const float4 u = q[h];
      v[4 * h] = u.x; v[4 * h + 1] = u.y; v[4 * h + 2] = u.z; v[4 * h + 3] = u.w;
    }
  }
  __device__ static inline void store(float* p, const float* v) {
    float4* q = reinterpret_cast<float4*>(p);
#pragma unroll
    for (int h = 0; h < 4; ++h) q[h] = make_float4(v[4 * h], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]);
  }
};

// acc(16x16) += A(16 x k) * B(k x 16) over one 16-byte lane fragment pair.
// Lane l supplies row (l%16) of A and column (l%16) of B, k-group l/16.
__device__ inline f32x4_t mma_frag(bf16, const uint4& a, const uint4& b, f32x4_t acc) {
  bf16x8_t av = __builtin_bit_cast(bf16x8_t, a);
  bf16x8_t bv = __builtin_bit_cast(bf16x8_t, b);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
}
__device__ inline f32x4_t mma_frag(bf16, const u32x4_t& a, const u32x4_t& b, f32x4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 acc, 0, 0, 0);
}
__device__ inline f32x4_t mma_frag(float, const u32x4_t& a, const u32x4_t& b, f32x4_t acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  return acc;
}
__device__ inline f32x4_t mma_frag(float, const uint4& a, const uint4& b, f32x4_t acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  return acc;
}

// Wave reductions (64 lanes)
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum with a fixed combination order (wave partials summed 0..n-1).
__device__ inline float block_sum(float v, float* sh /* >= 32 floats */) {
  v = wave_sum(v);
  const int w = threadIdx.x / WAVE, nw = blockDim.x / WAVE;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += sh[i];
  return s;
}

// Device status bits (OR-ed by kernels; read by the host after a sync)
enum : int {
  ST_BAD_TOKEN = 1,        // token id outside [0, V)
  ST_CAPACITY = 2,         // a position beyond the sequence's page table
  ST_BAD_PAGE = 4,         // page id outside the pool
};
__device__ inline void set_status(int* status, int bit) { atomicOr(status, bit); }

__device__ inline float silu(float x) { return x / (1.f + __expf(-x)); }

// ordered 64-bit key: larger float first, then lower index
__device__ inline uint64_t argmax_key(float v, int idx) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx);
}
__device__ inline int argmax_key_index(uint64_t k) { return (int)(0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFu)); }


}  // namespace dflow
