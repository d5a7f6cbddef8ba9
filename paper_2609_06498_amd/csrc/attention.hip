// Block attention over the paged KV cache with split-KV and GQA row packing,
// fused with QK-norm + RoPE of the block's queries and keys and the KV-cache
// write of the block's rows.
//
// Verification (causal = 1): block row j at position t+j attends to keys
// 0..t+j.  Drafting (causal = 0): every block row attends to every key below
// t+B (committed-context keys followed by the block's own keys).
//
// Attention rows are (block row j, query head g of a kv group) pairs packed
// 16 to a matrix-core tile, so the query heads of a group share every K/V
// byte.  Splits are merged by the combine kernel in split order, so a row's
// arithmetic depends only on its own visible keys, at any batch composition.
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
  const uint2 pa = make_uint2(f2bf2(p[0], p[1]), f2bf2(p[2], p[3]));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(short4_t, pa), __builtin_bit_cast(short4_t, vb),
                                                  acc, 0, 0, 0);
}
template <>
__device__ inline f32x4_t mma_pv_frag<float>(const float p[4], const float4& vb, f32x4_t acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[0], vb.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[1], vb.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[2], vb.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(p[3], vb.w, acc, 0, 0, 0);
  return acc;
}

// One workgroup of NW waves per (sequence, kv head, split of SplitKeys keys at
// fixed absolute positions).
//  1. The split's K/V pages are staged into LDS, all loads in flight at once.
//     Meanwhile the waves apply QK-norm + RoPE to the group's R = Bq * G query
//     rows (one row per wave and pass, one rotate-half pair per lane) into an
//     LDS query tile, and to the block's own key rows that fall into this
//     split (V copied).
//  2. The block rows' keys and values are written into the staged tiles and
//     into the paged cache.
//  3. Work units are (16-row group, page subset): with nrg row groups, WPR =
//     min(pages, NW / nrg) waves share a row group and take pages part,
//     part + WPR, ... with an online softmax (S^T = K Q^T on the matrix cores,
//     mask, running max/sum, P V).  Their partials are merged through LDS in
//     part order and written as this split's partial (m, l, O); with WPR = 1
//     each wave owns whole row groups and writes directly.
// WPR depends only on (Bq, G), so a row's arithmetic does not depend on the
// batch it is part of.
template <typename T, int DH, int NW, bool FUSED>
__global__ void __launch_bounds__(NW * 64) attn_kernel(AttnParams p) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  constexpr int KS = DH / KT;                 // k steps of S^T
  constexpr int DT = DH / 16;                 // output channel tiles
  constexpr int SK = SplitKeys<T>::value;
  constexpr int NPG = SK / PAGE;              // pages per split
  constexpr int PG = PAGE * DH;               // elements of one K (or V) page block
  constexpr int NT = NW * 64;
  constexpr int HALF = DH / 2;
  typedef typename VFrag<T>::type vfrag_t;
  constexpr int QLD = DH + KL;                // padded row of the query tile
  constexpr int MAXB = 4;                     // block rows per wave held in registers (Bq <= 64)
  extern __shared__ __align__(16) unsigned char smem[];
  T* lk = reinterpret_cast<T*>(smem);         // [NPG][PG] keys, fragment order
  T* lv = lk + (size_t)NPG * PG;              // [NPG][PG] values, fragment order
  T* lq = lv + (size_t)NPG * PG;              // [R][QLD] queries after QK-norm + RoPE
  float* mo = reinterpret_cast<float*>(smem); // merge area [NW][16][DH], reuses the K/V tiles after use
  float* s_ml = reinterpret_cast<float*>(lq); // merge (m, l) [NW][16][2], reuses the query tile after use
  __shared__ int s_page[NPG];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int item = blockIdx.x;                // (seq, kv head, split), split fastest
  const int split = item % p.nsplit;
  const int kvh = (item / p.nsplit) % p.Hkv;
  const int s = item / (p.nsplit * p.Hkv);
  const int G = p.Hq / p.Hkv;
  const int R = p.Bq * G;
  const int nrg = (R + 15) / 16;
  const float sl2 = rsqrtf((float)DH) * 1.4426950408889634f;   // softmax scale x log2(e)
  const int key0 = split * SK;
  const int t0 = p.start_pos[s];
  const int kv_len = t0 + p.Bq;
  const int cap = p.max_pages * PAGE;
  if (threadIdx.x == 0 && split == 0 && kv_len > cap) set_status(p.status, ST_CAPACITY);
  if (key0 >= kv_len) return;                 // uniform over the workgroup

  if (threadIdx.x < NPG) {
    const int pidx = min(key0 / PAGE + (int)threadIdx.x, p.max_pages - 1);
    const int pg = p.page_table[(size_t)s * p.max_pages + pidx];
    s_page[threadIdx.x] = (key0 + (int)threadIdx.x * PAGE < kv_len && pg >= 0 && pg < p.num_pages) ? pg : -1;
  }
  __syncthreads();

  // ---- 1. stage all pages (absent pages read page 0 of the pool; never used) ...
  constexpr int V16 = PG * (int)sizeof(T) / 16;   // 16-byte vectors per page block
  constexpr int PER = (NPG * V16 + NT - 1) / NT;  // per thread, K and V each (the last one partial)
  u32x4_t kr[PER], vr[PER];
#pragma unroll
  for (int it = 0; it < PER; ++it) {
    const int idx = min(threadIdx.x + it * NT, NPG * V16 - 1);   // a clamped duplicate is never stored
    const int pi = idx / V16, vi = idx - pi * V16;
    const size_t off = ((size_t)max(s_page[pi], 0) * p.Hkv + kvh) * PG;
    kr[it] = ((const gu4*)(reinterpret_cast<const T*>(p.kpool) + off))[vi];
    vr[it] = ((const gu4*)(reinterpret_cast<const T*>(p.vpool) + off))[vi];
  }
  // ... while the query rows get QK-norm + RoPE (lane i < DH/2 owns channels i, i + DH/2)
  const T* qkv = reinterpret_cast<const T*>(p.qkv);
  if constexpr (FUSED) {
    const T* gq = reinterpret_cast<const T*>(p.q_norm);
    const float g1 = lane < HALF ? TT<T>::ld(gq, lane) : 0.f;
    const float g2 = lane < HALF ? TT<T>::ld(gq, lane + HALF) : 0.f;
    constexpr int QB = 4;                      // rows per wave per batch: all their loads in flight together
    for (int rr0 = w; rr0 < R; rr0 += QB * NW) {   // uniform per wave
      float x1[QB], x2[QB];
      float2 c[QB];
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        const int rr = min(rr0 + b * NW, R - 1);   // clamped rows are computed and not stored
        const int j = rr / G, g = rr - j * G;
        const T* src = qkv + (size_t)(s * p.Bq + j) * p.ld_qkv + (size_t)(kvh * G + g) * DH;
        const int pos = min(t0 + j, cap - 1);     // past capacity: status set above
        const int l = lane < HALF ? lane : 0;
        x1[b] = TT<T>::ld(src, l);
        x2[b] = TT<T>::ld(src, l + HALF);
        c[b] = p.rope[(size_t)pos * HALF + l];
      }
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        const int rr = rr0 + b * NW;
        const float v1 = lane < HALF ? x1[b] : 0.f, v2 = lane < HALF ? x2[b] : 0.f;
        const float r = rsqrtf(wave_sum(v1 * v1 + v2 * v2) / (float)DH + p.eps);
        if (rr < R && lane < HALF) {
          const float y1 = v1 * r * g1;
          const float y2 = v2 * r * g2;
          TT<T>::st(lq, (size_t)rr * QLD + lane, y1 * c[b].x - y2 * c[b].y);
          TT<T>::st(lq, (size_t)rr * QLD + lane + HALF, y2 * c[b].x + y1 * c[b].y);
        }
      }
    }
  }
  // ... and the block's own key rows in this split (wave w: rows jlo + w + NW * b)
  const int jlo = max(0, key0 - t0), jhi = min(p.Bq, key0 + SK - t0);
  float nk1[MAXB], nk2[MAXB], nv1[MAXB], nv2[MAXB];
  if constexpr (FUSED) {
    const T* gk = reinterpret_cast<const T*>(p.k_norm);
#pragma unroll
    for (int b = 0; b < MAXB; ++b) {
      const int j = jlo + w + NW * b;
      if (j >= jhi) break;                     // uniform per wave
      const int pos = min(t0 + j, cap - 1);
      const T* src = qkv + (size_t)(s * p.Bq + j) * p.ld_qkv + (size_t)p.Hq * DH + (size_t)kvh * DH;
      const T* vsrc = src + (size_t)p.Hkv * DH;
      float x1 = 0.f, x2 = 0.f;
      if (lane < HALF) { x1 = TT<T>::ld(src, lane); x2 = TT<T>::ld(src, lane + HALF); }
      const float r = rsqrtf(wave_sum(x1 * x1 + x2 * x2) / (float)DH + p.eps);
      nk1[b] = nk2[b] = 0.f;
      if (lane < HALF) {
        const float2 c = p.rope[(size_t)pos * HALF + lane];
        const float y1 = x1 * r * TT<T>::ld(gk, lane);
        const float y2 = x2 * r * TT<T>::ld(gk, lane + HALF);
        nk1[b] = y1 * c.x - y2 * c.y;
        nk2[b] = y2 * c.x + y1 * c.y;
      }
      nv1[b] = TT<T>::ld(vsrc, lane);
      nv2[b] = lane + 64 < DH ? TT<T>::ld(vsrc, lane + 64) : 0.f;
    }
  }
#pragma unroll
  for (int it = 0; it < PER; ++it) {
    const int idx = threadIdx.x + it * NT;
    if ((NPG * V16) % NT == 0 || idx < NPG * V16) {
      reinterpret_cast<u32x4_t*>(lk)[idx] = kr[it];
      reinterpret_cast<u32x4_t*>(lv)[idx] = vr[it];
    }
  }
  __syncthreads();

  // ---- 2. the block rows' keys and values into the staged tiles and the cache
#pragma unroll
  for (int b = 0; b < (FUSED ? MAXB : 0); ++b) {
    const int j = jlo + w + NW * b;
    if (j >= jhi) break;                       // uniform per wave
    const int pos = t0 + j;
    if (pos >= cap) continue;                  // status set above
    const int pi = (pos - key0) / PAGE, slot = pos % PAGE;
    const int gpage = s_page[pi];
    if (lane == 0 && gpage < 0) set_status(p.status, ST_BAD_PAGE);
    T* kt_l = lk + (size_t)pi * PG;
    T* vt_l = lv + (size_t)pi * PG;
    T* kt_g = gpage >= 0 ? reinterpret_cast<T*>(p.kpool) + ((size_t)gpage * p.Hkv + kvh) * PG : nullptr;
    T* vt_g = gpage >= 0 ? reinterpret_cast<T*>(p.vpool) + ((size_t)gpage * p.Hkv + kvh) * PG : nullptr;
    auto koff = [&](int d) -> int {
      return (((slot / 16) * KS + d / KT) * 64 + ((d % KT) / KL) * 16 + slot % 16) * KL + d % KL;
    };
    auto voff = [&](int e) -> int {
      return (((slot / 16) * DT + e / 16) * 64 + ((slot % 16) / 4) * 16 + e % 16) * 4 + slot % 4;
    };
    if (lane < HALF) {
      TT<T>::st(kt_l, koff(lane), nk1[b]);
      TT<T>::st(kt_l, koff(lane + HALF), nk2[b]);
      if (kt_g) {
        TT<T>::st(kt_g, koff(lane), nk1[b]);
        TT<T>::st(kt_g, koff(lane + HALF), nk2[b]);
      }
    }
    TT<T>::st(vt_l, voff(lane), nv1[b]);
    if (vt_g) TT<T>::st(vt_g, voff(lane), nv1[b]);
    if (lane + 64 < DH) {
      TT<T>::st(vt_l, voff(lane + 64), nv2[b]);
      if (vt_g) TT<T>::st(vt_g, voff(lane + 64), nv2[b]);
    }
  }
  __syncthreads();

  // ---- 3. row groups x page subsets
  // merge area (units x 16 x DH fp32) must fit in the K/V tiles it reuses
  constexpr int MAXU = (2 * NPG * PG * (int)sizeof(T)) / (16 * DH * 4) < NW ? (2 * NPG * PG * (int)sizeof(T)) / (16 * DH * 4) : NW;
  int wpr = MAXU / nrg < NPG ? MAXU / nrg : NPG;
  if (wpr < 1) wpr = 1;
  const int units = nrg * wpr;                 // waves with work in a pass (merge) or row groups (wpr = 1)
  auto run_unit = [&](int rg, int part, u32x4_t (&qf)[KS], float& mrow, float& lrow, f32x4_t (&o)[DT]) {
    {
      const int qr = min(rg * 16 + (lane & 15), R - 1);
      if constexpr (FUSED) {
#pragma unroll
        for (int k = 0; k < KS; ++k)
          qf[k] = *reinterpret_cast<const u32x4_t*>(lq + (size_t)qr * QLD + k * KT + (lane >> 4) * KL);
      } else {
        const int j = qr / G, g = qr - j * G;
        const T* qrow = reinterpret_cast<const T*>(p.q) + ((size_t)(s * p.Bq + j) * p.Hq + kvh * G + g) * DH;
#pragma unroll
        for (int k = 0; k < KS; ++k) qf[k] = *(const gu4*)(qrow + k * KT + (lane >> 4) * KL);
      }
    }
    mrow = -INFINITY;
    lrow = 0.f;
#pragma unroll
    for (int i = 0; i < DT; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int ar = rg * 16 + (lane & 15);
    const bool row_ok = ar < R;
    const int pos_row = t0 + (row_ok ? ar / G : 0);
    bool first = true;                        // uniform: the unit's first present page
    for (int pi = part; pi < NPG; pi += wpr) {
      if (s_page[pi] < 0) continue;          // uniform
      const int kp0 = key0 + pi * PAGE;
      const u32x4_t* kb = reinterpret_cast<const u32x4_t*>(lk + (size_t)pi * PG);
      const vfrag_t* vb = reinterpret_cast<const vfrag_t*>(lv + (size_t)pi * PG);
      // every key of the page precedes the block and every row is valid: no mask
      const bool full = kp0 + PAGE <= t0 && rg * 16 + 16 <= R;   // uniform
      // scores in log2 units (scale folded with log2 e), so the softmax uses exp2
      float sc[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < KS; ++k) acc = mma_frag(T(), kb[(kt * KS + k) * 64 + lane], qf[k], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[kt][r] = acc[r] * sl2;
      }
      if (!full) {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = kp0 + kt * 16 + 4 * (lane >> 4) + r;
            const bool vis = row_ok && key < kv_len && (!p.causal || key <= pos_row);
            if (!vis) sc[kt][r] = -INFINITY;
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
      const float mnew = first ? mx : fmaxf(mrow, mx);
      float ls = 0.f;
      if (full) {                              // mnew is finite and no score is masked
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            sc[kt][r] = exp2f(sc[kt][r] - mnew);
            ls += sc[kt][r];
          }
      } else {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float e = (sc[kt][r] == -INFINITY) ? 0.f : exp2f(sc[kt][r] - mnew);
            sc[kt][r] = e;
            ls += e;
          }
      }
      ls += __shfl_xor(ls, 16, 64);
      ls += __shfl_xor(ls, 32, 64);
      if (first) {                             // the output is still zero: nothing to rescale
        lrow = ls;
      } else {
        const float alpha = (mrow == -INFINITY) ? (mnew == -INFINITY ? 1.f : 0.f) : exp2f(mrow - mnew);
        lrow = lrow * alpha + ls;
        float al[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) al[r] = __shfl(alpha, 4 * (lane >> 4) + r, 64);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 4; ++r) o[dt][r] *= al[r];
      }
      mrow = mnew;
      first = false;
      if constexpr (KL == 8) {
        // P V with 32 keys per matrix-core op: lane group g supplies keys
        // 4g..4g+3 of key tiles 2c and 2c+1, and the same keys of V
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const u32x4_t pa = {f2bf2(sc[2 * c][0], sc[2 * c][1]), f2bf2(sc[2 * c][2], sc[2 * c][3]),
                              f2bf2(sc[2 * c + 1][0], sc[2 * c + 1][1]), f2bf2(sc[2 * c + 1][2], sc[2 * c + 1][3])};
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const uint2 v0 = reinterpret_cast<const uint2*>(vb)[((2 * c) * DT + dt) * 64 + lane];
            const uint2 v1 = reinterpret_cast<const uint2*>(vb)[((2 * c + 1) * DT + dt) * 64 + lane];
            const u32x4_t vv = {v0.x, v0.y, v1.x, v1.y};
            o[dt] = mma_frag(T(), pa, vv, o[dt]);
          }
        }
      } else {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[dt] = mma_pv_frag<T>(sc[kt], vb[(kt * DT + dt) * 64 + lane], o[dt]);
      }
    }
  };
  auto write_partial = [&](int rg, float mrow, float lrow, const f32x4_t (&o)[DT]) {
    const size_t pidx = (((size_t)s * p.Hkv + kvh) * p.rg + rg) * p.nsplit + split;
    float* po = p.part_o + pidx * 16 * DH;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) po[(4 * (lane >> 4) + r) * DH + dt * 16 + (lane & 15)] = o[dt][r];
    if (lane < 16) {
      p.part_ml[pidx * 32 + 2 * lane] = mrow;
      p.part_ml[pidx * 32 + 2 * lane + 1] = lrow;
    }
  };

  u32x4_t qf[KS];
  float mrow, lrow;
  f32x4_t o[DT];
  if (wpr == 1) {
    for (int rg = w; rg < nrg; rg += NW) {     // uniform per wave; no barrier inside
      run_unit(rg, 0, qf, mrow, lrow, o);
      write_partial(rg, mrow, lrow, o);
    }
    return;
  }
  const bool active = w < units;
  const int rg = w % nrg, part = w / nrg;
  if (active) run_unit(rg, part, qf, mrow, lrow, o);
  __syncthreads();                             // every wave is done with the K/V tiles
  if (active) {
    float* mw = mo + (size_t)w * 16 * DH;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r)   // 16-column blocks XOR-swizzled by row/4: conflict-free stores
        mw[(4 * (lane >> 4) + r) * DH + ((dt * 16 + (lane & 15)) ^ ((lane >> 4) << 4))] = o[dt][r];
    if (lane < 16) {
      s_ml[(w * 16 + lane) * 2] = mrow;
      s_ml[(w * 16 + lane) * 2 + 1] = lrow;
    }
  }
  __syncthreads();
  // merge the wpr partials of each row group in part order; lane handles 4
  // consecutive channels, all partial loads in flight together
  for (int e4 = threadIdx.x; e4 < nrg * 4 * DH; e4 += NT) {
    const int e = e4 * 4;
    const int g = e / (16 * DH), rem = e - g * 16 * DH, row = rem / DH, dd = rem - row * DH;
    float mq[NPG], lq4[NPG];
    float4 oq[NPG];
#pragma unroll
    for (int q = 0; q < NPG; ++q) {
      if (q < wpr) {                               // uniform
        const int u = q * nrg + g;
        mq[q] = s_ml[(u * 16 + row) * 2];
        lq4[q] = s_ml[(u * 16 + row) * 2 + 1];
        oq[q] = *reinterpret_cast<const float4*>(mo + ((size_t)u * 16 + row) * DH + (dd ^ (((row >> 2) & 3) << 4)));
      } else {
        mq[q] = -INFINITY;
        lq4[q] = 0.f;
        oq[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < NPG; ++q) M = fmaxf(M, mq[q]);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float l = 0.f;
#pragma unroll
    for (int q = 0; q < NPG; ++q) {
      const float f = (mq[q] == -INFINITY) ? 0.f : exp2f(mq[q] - M);
      acc.x += f * oq[q].x;
      acc.y += f * oq[q].y;
      acc.z += f * oq[q].z;
      acc.w += f * oq[q].w;
      l += f * lq4[q];
    }
    const size_t pidx = (((size_t)s * p.Hkv + kvh) * p.rg + g) * p.nsplit + split;
    *reinterpret_cast<float4*>(p.part_o + (pidx * 16 + row) * DH + dd) = acc;
    if (dd == 0) {
      p.part_ml[pidx * 32 + 2 * row] = M;
      p.part_ml[pidx * 32 + 2 * row + 1] = l;
    }
  }
}

// out[row, head, :] = sum_split 2^(m_s - M) O_s / sum_split 2^(m_s - M) l_s (m in log2 units)
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
    const float f = (m == -INFINITY) ? 0.f : exp2f(m - M);   // partial maxima are in log2 units
    acc += f * po[(size_t)sp * 16 * DH];
    lsum += f * ml[(size_t)sp * 32 + 1];
  }
  const float v = lsum > 0.f ? acc / lsum : 0.f;
  TT<T>::st(reinterpret_cast<T*>(p.out), (size_t)row * p.Hq * DH + hq * DH + d, v);
}

constexpr int ATTN_WAVES = 16;

// Dynamic LDS of the attention kernel: the split's K and V pages plus the
// query tile (fused variant) or the merge statistics.
template <typename T, int DH>
static size_t attn_lds(bool fused, int R) {
  const size_t tile = fused ? (size_t)R * (DH + TT<T>::KL) * sizeof(T) : 0;
  const size_t ml = (size_t)ATTN_WAVES * 16 * 2 * sizeof(float);
  return 2 * (size_t)SplitKeys<T>::value * DH * sizeof(T) + (tile > ml ? tile : ml);
}
static constexpr size_t ATTN_LDS_MAX = 159 * 1024;

template <typename T, int DH>
static bool fuses_dh(int Bq, int G) {
  return Bq <= 4 * ATTN_WAVES && attn_lds<T, DH>(true, Bq * G) <= ATTN_LDS_MAX;
}

template <typename T, int DH, bool FUSED>
static hipError_t launch_k(const AttnParams& p, hipStream_t st) {
  constexpr int NW = ATTN_WAVES;
  const size_t lds = attn_lds<T, DH>(FUSED, p.Bq * (p.Hq / p.Hkv));
  if (lds > ATTN_LDS_MAX) return hipErrorInvalidConfiguration;
  static bool lds_set = false;   // allow the largest dynamic LDS once per instantiation
  if (!lds_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<T, DH, NW, FUSED>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)ATTN_LDS_MAX);
    if (e != hipSuccess) return e;
    lds_set = true;
  }
  hipLaunchKernelGGL((attn_kernel<T, DH, NW, FUSED>), dim3(p.nseq * p.Hkv * p.nsplit), dim3(NW * 64), lds, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), dim3(p.nseq * p.Bq, p.Hq), dim3(DH), 0, st, p);
  return hipGetLastError();
}

template <typename T, int DH>
static hipError_t launch_dh(const AttnParams& p, hipStream_t st) {
  if (p.fused) {
    if (!fuses_dh<T, DH>(p.Bq, p.Hq / p.Hkv)) return hipErrorInvalidConfiguration;
    return launch_k<T, DH, true>(p, st);
  }
  return launch_k<T, DH, false>(p, st);
}

bool attention_fuses_rope(bool bf16, int Bq, int G, int Dh) {
  if (Dh == 128) return bf16 ? fuses_dh<dflow::bf16, 128>(Bq, G) : fuses_dh<float, 128>(Bq, G);
  if (Dh == 64) return bf16 ? fuses_dh<dflow::bf16, 64>(Bq, G) : fuses_dh<float, 64>(Bq, G);
  return false;
}

hipError_t launch_attention(bool bf16, const AttnParams& p, hipStream_t st) {
  if (p.Dh == 128) return bf16 ? launch_dh<dflow::bf16, 128>(p, st) : launch_dh<float, 128>(p, st);
  if (p.Dh == 64) return bf16 ? launch_dh<dflow::bf16, 64>(p, st) : launch_dh<float, 64>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace dflow
