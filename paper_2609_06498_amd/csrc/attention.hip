// Block attention over the paged KV cache with split-KV and GQA row packing.
//
// Verification (causal = 1): block row j at position t+j attends to keys
// 0..t+j.  Drafting (causal = 0): every block row attends to every key below
// t+B (committed-context keys followed by the block's own keys).
//
// Workgroup = (sequence, kv head, split of keys at fixed absolute positions:
// 256 keys for bf16, 128 for fp32).  The split's K and V pages (stored in
// matrix-core fragment order) are staged into LDS once with 16-byte loads;
// each wave then owns whole groups of 16 attention rows -- (block row j,
// query head g of the group) pairs, so the query heads of a group share every
// K/V byte -- and sweeps the staged pages with an online softmax: S^T = K Q^T
// on the matrix cores (the exponentiated scores already sit in the A-operand
// layout of P V), mask, running max/sum, P V.  Splits are merged by the
// combine kernel in split order, so a row's arithmetic depends only on its
// own visible keys, at any batch composition.
#include "common.h"
#include "kernels.h"

namespace dflow {

// Fragment of 4 consecutive keys of one value channel (8 bytes bf16, 16 bytes fp32)
template <typename T> struct VFrag;
template <> struct VFrag<bf16> { typedef uint2 type; };
template <> struct VFrag<float> { typedef float4 type; };

template <typename T>
__device__ inline f32x4_t mma_pv_frag(const float p[4], const typename VFrag<T>::type& v, f32x4_t acc);
template <>
__device__ inline f32x4_t mma_pv_frag<bf16>(const float p[4], const uint2& vb, f32x4_t acc) {
  short4_t a, b;
  a[0] = (short)f2bf(p[0]); a[1] = (short)f2bf(p[1]); a[2] = (short)f2bf(p[2]); a[3] = (short)f2bf(p[3]);
  b[0] = (short)(vb.x & 0xFFFF); b[1] = (short)(vb.x >> 16); b[2] = (short)(vb.y & 0xFFFF); b[3] = (short)(vb.y >> 16);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, acc, 0, 0, 0);
}
template <>
__device__ inline f32x4_t mma_pv_frag<float>(const float p[4], const float4& vb, f32x4_t acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[0], vb.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[1], vb.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[2], vb.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[3], vb.w, acc, 0, 0, 0);
  return acc;
}

template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_kernel(AttnParams p) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  constexpr int KS = DH / KT;                 // k steps of S^T
  constexpr int DT = DH / 16;                 // output channel tiles
  constexpr int NPG = SplitKeys<T>::value / PAGE;   // pages per split
  constexpr int PG = PAGE * DH;               // elements of one K (or V) page block
  typedef typename VFrag<T>::type vfrag_t;
  extern __shared__ __align__(16) unsigned char smem[];
  T* lk = reinterpret_cast<T*>(smem);         // [2][PG] keys, fragment order (double buffer)
  T* lv = lk + (size_t)2 * PG;                // [2][PG] values, fragment order
  __shared__ int s_page[NPG];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int item = blockIdx.x;                // (seq, kv head, split), split fastest
  const int split = item % p.nsplit;
  const int kvh = (item / p.nsplit) % p.Hkv;
  const int s = item / (p.nsplit * p.Hkv);
  const int G = p.Hq / p.Hkv;
  const int R = p.Bq * G;
  const float scale = rsqrtf((float)DH);
  const int key0 = split * SplitKeys<T>::value;
  const int t0 = p.start_pos[s];
  const int kv_len = t0 + p.Bq;
  if (key0 >= kv_len) return;                 // uniform over the workgroup

  // ---- pages stream through two LDS buffers: page i+1 is fetched into
  // registers while page i is used, then stored into the other buffer.
  if (threadIdx.x < NPG) {
    const int pidx = min(key0 / PAGE + (int)threadIdx.x, p.max_pages - 1);
    const int pg = p.page_table[(size_t)s * p.max_pages + pidx];
    s_page[threadIdx.x] = (key0 + (int)threadIdx.x * PAGE < kv_len && pg >= 0 && pg < p.num_pages) ? pg : -1;
  }
  __syncthreads();
  constexpr int V16 = PG * (int)sizeof(T) / 16;       // 16-byte vectors per page block
  constexpr int PER = V16 / 256;                      // per thread, K and V each
  static_assert(V16 % 256 == 0, "page staging assumes 256 threads");
  u32x4_t kr[PER], vr[PER];
  // absent pages read page 0 of the pool (always valid); their copy is never used
  auto fetch = [&](int pi) {
    const int pg = max(s_page[pi], 0);
    const size_t off = ((size_t)pg * p.Hkv + kvh) * PG;
    const gu4* gk = (const gu4*)(reinterpret_cast<const T*>(p.kpool) + off);
    const gu4* gv = (const gu4*)(reinterpret_cast<const T*>(p.vpool) + off);
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      kr[it] = gk[threadIdx.x + it * 256];
      vr[it] = gv[threadIdx.x + it * 256];
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      reinterpret_cast<u32x4_t*>(lk + (size_t)buf * PG)[threadIdx.x + it * 256] = kr[it];
      reinterpret_cast<u32x4_t*>(lv + (size_t)buf * PG)[threadIdx.x + it * 256] = vr[it];
    }
  };
  // ---- each wave owns up to RGW whole 16-row groups per pass over the pages.
  // The pass and page loops are uniform over the workgroup: every thread
  // stages every page and reaches every barrier, with or without rows.
  constexpr int RGW = 2;
  const int nrg = (R + 15) / 16;
  const int npass = (nrg + 4 * RGW - 1) / (4 * RGW);
  for (int pass = 0; pass < npass; ++pass) {
    int rgs[RGW];
    bool rgv[RGW];
    u32x4_t qf[RGW][KS];
    float mrow[RGW], lrow[RGW];
    f32x4_t o[RGW][DT];
#pragma unroll
    for (int g = 0; g < RGW; ++g) {
      rgs[g] = pass * 4 * RGW + 4 * g + w;
      rgv[g] = rgs[g] < nrg;
      const int ar = min(rgs[g], nrg - 1) * 16 + (lane & 15);
      const int jrow = ar < R ? ar / G : 0, grow = ar < R ? ar % G : 0;
      const T* qrow = reinterpret_cast<const T*>(p.Q) + ((size_t)(s * p.Bq + jrow) * p.Hq + kvh * G + grow) * DH;
#pragma unroll
      for (int k = 0; k < KS; ++k) qf[g][k] = *(const gu4*)(qrow + k * KT + (lane >> 4) * KL);
      mrow[g] = -INFINITY;
      lrow[g] = 0.f;
#pragma unroll
      for (int i = 0; i < DT; ++i) o[g][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    fetch(0);
    __syncthreads();                          // buffer 0 is free (previous pass finished with it)
    store(0);
    __syncthreads();
    for (int pi = 0; pi < NPG; ++pi) {
      const int buf = pi & 1;
      if (pi + 1 < NPG) fetch(pi + 1);        // uniform; lands while this page is used
      if (s_page[pi] >= 0) {                  // uniform
        const int kp0 = key0 + pi * PAGE;
        const u32x4_t* kb = reinterpret_cast<const u32x4_t*>(lk + (size_t)buf * PG);
        const vfrag_t* vb = reinterpret_cast<const vfrag_t*>(lv + (size_t)buf * PG);
#pragma unroll
        for (int g = 0; g < RGW; ++g) {
          if (!rgv[g]) continue;              // uniform per wave; no barrier inside
          const int ar = rgs[g] * 16 + (lane & 15);
          const bool row_ok = ar < R;
          const int pos_row = t0 + (row_ok ? ar / G : 0);
          float sc[4][4];
#pragma unroll
          for (int kt = 0; kt < 4; ++kt) {
            f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < KS; ++k) acc = mma_frag(T(), kb[(kt * KS + k) * 64 + lane], qf[g][k], acc);
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
          // rows with nothing visible so far keep m = -inf, l = 0 and a zero output;
          // control flow stays uniform (the matrix-core ops and shuffles need all lanes)
          const float mnew = fmaxf(mrow[g], mx);
          const float alpha = (mrow[g] == -INFINITY) ? (mnew == -INFINITY ? 1.f : 0.f) : __expf(mrow[g] - mnew);
          float ls = 0.f;
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float e = (sc[kt][r] == -INFINITY) ? 0.f : __expf(sc[kt][r] - mnew);
              sc[kt][r] = e;
              ls += e;
            }
          ls += __shfl_xor(ls, 16, 64);
          ls += __shfl_xor(ls, 32, 64);
          lrow[g] = lrow[g] * alpha + ls;
          mrow[g] = mnew;
          float al[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) al[r] = __shfl(alpha, 4 * (lane >> 4) + r, 64);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 4; ++r) o[g][dt][r] *= al[r];
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[g][dt] = mma_pv_frag<T>(sc[kt], vb[(kt * DT + dt) * 64 + lane], o[g][dt]);
        }
      }
      if (pi + 1 < NPG) {
        // the other buffer was last read in iteration pi-1, which every wave
        // finished before the barrier that ended that iteration
        store(buf ^ 1);
        __syncthreads();
      }
    }
    // ---- this split's partials of the wave's row groups
#pragma unroll
    for (int g = 0; g < RGW; ++g) {
      if (!rgv[g]) continue;
      const size_t pidx = (((size_t)s * p.Hkv + kvh) * p.rg + rgs[g]) * p.nsplit + split;
      float* po = p.part_o + pidx * 16 * DH;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) po[(4 * (lane >> 4) + r) * DH + dt * 16 + (lane & 15)] = o[g][dt][r];
      if (lane < 16) {
        p.part_ml[pidx * 32 + 2 * lane] = mrow[g];
        p.part_ml[pidx * 32 + 2 * lane + 1] = lrow[g];
      }
    }
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
  int ns = (kv_len + SplitKeys<T>::value - 1) / SplitKeys<T>::value;
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
  const int blocks = p.nseq * p.Hkv * p.nsplit;
  const size_t lds = 2 * 2 * (size_t)PAGE * DH * sizeof(T);   // two page buffers, K and V
  if (lds > 160 * 1024) return hipErrorInvalidConfiguration;
  static bool lds_set = false;   // allow more than the default dynamic LDS once per instantiation
  if (!lds_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<T, DH>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    lds_set = true;
  }
  hipLaunchKernelGGL((attn_kernel<T, DH>), dim3(blocks), dim3(256), lds, st, p);
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
