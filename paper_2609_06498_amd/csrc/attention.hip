// Block attention over the paged KV cache with split-KV and GQA row packing.
//
// Verification (causal = 1): block row j at position t+j attends to keys
// 0..t+j.  Drafting (causal = 0): every block row attends to every key below
// t+B (committed-context keys followed by the block's own keys).
//
// Work item = (sequence, kv head, split of 256 keys at fixed absolute
// positions, group of 16 attention rows), where the attention rows of a kv
// head are (block row j, query head g of the group) pairs.  Each of the four
// waves of a workgroup takes one 64-key page of the split: it computes
// S^T = K Q^T on the matrix cores (so the softmax'd scores already sit in the
// A-operand layout of P V), applies the mask, and accumulates P V.  The four
// waves are merged in LDS in wave order, the splits by the combine kernel in
// split order: a row's arithmetic depends only on its own visible keys.
#include "common.h"
#include "kernels.h"

namespace dflow {

template <typename T>
__device__ inline f32x4_t mma_pv(const float p[4], const void* vrow, f32x4_t acc);

// P (4 consecutive keys of row l%16) times V^T fragment (same 4 keys, channel l%16)
template <>
__device__ inline f32x4_t mma_pv<bf16>(const float p[4], const void* vrow, f32x4_t acc) {
  const uint2 vb = *reinterpret_cast<const uint2*>(vrow);
  short4_t a, b;
  a[0] = (short)f2bf(p[0]); a[1] = (short)f2bf(p[1]); a[2] = (short)f2bf(p[2]); a[3] = (short)f2bf(p[3]);
  b[0] = (short)(vb.x & 0xFFFF); b[1] = (short)(vb.x >> 16); b[2] = (short)(vb.y & 0xFFFF); b[3] = (short)(vb.y >> 16);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc, 0, 0, 0);
}
template <>
__device__ inline f32x4_t mma_pv<float>(const float p[4], const void* vrow, f32x4_t acc) {
  const float4 vb = *reinterpret_cast<const float4*>(vrow);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[0], vb.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[1], vb.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[2], vb.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[3], vb.w, acc, 0, 0, 0);
  return acc;
}

template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_kernel(AttnParams p) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  constexpr int KS = DH / KT;          // k steps of S^T
  constexpr int DT = DH / 16;          // output channel tiles
  __shared__ float sh_o[4][16][DH];
  __shared__ float sh_m[4][16], sh_l[4][16];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // XCD-aware item mapping: the row groups of one (seq, head, split) share an XCD (and its L2).
  const int L = blockIdx.x;
  const int xcd = L & 7, slot = L >> 3;
  const int rgi = slot % p.rg;
  const int item = xcd + 8 * (slot / p.rg);
  const int n_items = p.nseq * p.Hkv * p.nsplit;
  if (item >= n_items) return;
  const int split = item % p.nsplit;
  const int kvh = (item / p.nsplit) % p.Hkv;
  const int s = item / (p.nsplit * p.Hkv);

  const int t0 = p.start_pos[s];
  const int kv_len = t0 + p.Bq;
  if (split * SPLIT_KEYS >= kv_len) return;
  const int G = p.Hq / p.Hkv;
  const int R = p.Bq * G;
  const float scale = rsqrtf((float)DH);

  // this lane's attention row (as column of S^T / B operand)
  const int ar = rgi * 16 + (lane & 15);
  const bool row_ok = ar < R;
  const int jrow = row_ok ? ar / G : 0;
  const int grow = row_ok ? ar % G : 0;
  const int pos_row = t0 + jrow;
  const T* qrow = reinterpret_cast<const T*>(p.Q) + ((size_t)(s * p.Bq + jrow) * p.Hq + kvh * G + grow) * DH;
  uint4 qf[KS];
#pragma unroll
  for (int k = 0; k < KS; ++k)
    qf[k] = row_ok ? *reinterpret_cast<const uint4*>(qrow + k * KT + (lane >> 4) * KL) : make_uint4(0, 0, 0, 0);

  const int kp0 = split * SPLIT_KEYS + w * PAGE;   // first key of this wave's page
  float mrow = -INFINITY, lrow = 0.f;
  f32x4_t o[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int pidx = kp0 / PAGE;
  const int page = (kp0 < kv_len && pidx < p.max_pages) ? p.page_table[(size_t)s * p.max_pages + pidx] : -1;
  if (page >= 0 && page < p.num_pages) {
    const T* kb = reinterpret_cast<const T*>(p.kpool) + ((size_t)page * p.Hkv + kvh) * PAGE * DH;
    const T* vb = reinterpret_cast<const T*>(p.vpool) + ((size_t)page * p.Hkv + kvh) * DH * PAGE;
    float sc[4][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const T* krow = kb + (size_t)(kt * 16 + (lane & 15)) * DH + (lane >> 4) * KL;
#pragma unroll
      for (int k = 0; k < KS; ++k) acc = mma_frag(T(), *reinterpret_cast<const uint4*>(krow + k * KT), qf[k], acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kp0 + kt * 16 + 4 * (lane >> 4) + r;
        const bool vis = row_ok && key < kv_len && (!p.causal || key <= pos_row);
        sc[kt][r] = vis ? acc[r] * scale : -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[kt][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float ls = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = (mx == -INFINITY || sc[kt][r] == -INFINITY) ? 0.f : __expf(sc[kt][r] - mx);
        sc[kt][r] = e;
        ls += e;
      }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    mrow = mx;
    lrow = ls;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const T* vrow = vb + (size_t)(dt * 16 + (lane & 15)) * PAGE + kt * 16 + 4 * (lane >> 4);
        o[dt] = mma_pv<T>(sc[kt], vrow, o[dt]);
      }
  }

  // ---- merge the four waves (fixed order)
  if (lane < 16) { sh_m[w][lane] = mrow; sh_l[w][lane] = lrow; }
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 4; ++r) sh_o[w][4 * (lane >> 4) + r][dt * 16 + (lane & 15)] = o[dt][r];
  __syncthreads();
  const size_t pi = (((size_t)s * p.Hkv + kvh) * p.rg + rgi) * p.nsplit + split;
  float* po = p.part_o + pi * 16 * DH;
  float* pml = p.part_ml + pi * 32;
  for (int e = threadIdx.x; e < 16 * DH; e += blockDim.x) {
    const int r = e / DH, d = e - r * DH;
    float M = -INFINITY;
    for (int ww = 0; ww < 4; ++ww) M = fmaxf(M, sh_m[ww][r]);
    float acc = 0.f, lsum = 0.f;
    for (int ww = 0; ww < 4; ++ww) {
      const float f = (sh_m[ww][r] == -INFINITY) ? 0.f : __expf(sh_m[ww][r] - M);
      acc += f * sh_o[ww][r][d];
      lsum += f * sh_l[ww][r];
    }
    po[e] = acc;
    if (d == 0) { pml[2 * r] = M; pml[2 * r + 1] = lsum; }
  }
}

// out[row, head, :] = sum_split e^(m_s - M) O_s / sum_split e^(m_s - M) l_s
// (split order fixed; the split loads are independent and unrolled)
template <typename T, int DH>
__global__ void __launch_bounds__(DH) attn_combine_kernel(AttnParams p) {
  const int row = blockIdx.x;           // s*Bq + j
  const int hq = blockIdx.y;
  const int d = threadIdx.x;
  const int s = row / p.Bq, j = row - s * p.Bq;
  const int G = p.Hq / p.Hkv;
  const int kvh = hq / G, g = hq - kvh * G;
  const int ar = j * G + g;
  const int rgi = ar >> 4, r = ar & 15;
  const int kv_len = p.start_pos[s] + p.Bq;
  int ns = (kv_len + SPLIT_KEYS - 1) / SPLIT_KEYS;
  if (ns > p.nsplit) ns = p.nsplit;
  const size_t base = (((size_t)s * p.Hkv + kvh) * p.rg + rgi) * p.nsplit;
  const float* ml = p.part_ml + base * 32 + 2 * r;
  const float* po = p.part_o + (base * 16 + r) * DH + d;
  float M = -INFINITY;
#pragma unroll 8
  for (int sp = 0; sp < ns; ++sp) M = fmaxf(M, ml[(size_t)sp * 32]);
  float acc = 0.f, lsum = 0.f;
#pragma unroll 8
  for (int sp = 0; sp < ns; ++sp) {
    const float m = ml[(size_t)sp * 32];
    const float f = (m == -INFINITY) ? 0.f : __expf(m - M);
    acc += f * po[(size_t)sp * 16 * DH];
    lsum += f * ml[(size_t)sp * 32 + 1];
  }
  const float v = lsum > 0.f ? acc / lsum : 0.f;
  TT<T>::st(reinterpret_cast<T*>(p.out), (size_t)row * p.Hq * DH + hq * DH + d, v);
}

template <typename T, int DH>
static hipError_t launch_dh(const AttnParams& p, hipStream_t st) {
  const int n_items = p.nseq * p.Hkv * p.nsplit;
  const int blocks = ((n_items + 7) / 8) * 8 * p.rg;
  hipLaunchKernelGGL((attn_kernel<T, DH>), dim3(blocks), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), dim3(p.nseq * p.Bq, p.Hq), dim3(DH), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_attention(bool bf16, const AttnParams& p, hipStream_t st) {
  if (p.Dh == 128) return bf16 ? launch_dh<dflow::bf16, 128>(p, st) : launch_dh<float, 128>(p, st);
  if (p.Dh == 64) return bf16 ? launch_dh<dflow::bf16, 64>(p, st) : launch_dh<float, 64>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace dflow
