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

// 16 bytes of storage-type values <-> fp32
template <typename T> struct Chunk;
template <> struct Chunk<bf16> {
  __device__ static inline void unpack(const u32x4_t& u, float* x) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = bf2f(u[i] & 0xFFFFu);
      x[2 * i + 1] = bf2f(u[i] >> 16);
    }
  }
  __device__ static inline u32x4_t pack(const float* x) {
    return u32x4_t{f2bf2(x[0], x[1]), f2bf2(x[2], x[3]), f2bf2(x[4], x[5]), f2bf2(x[6], x[7])};
  }
  __device__ static inline bf16 elem(const u32x4_t& u, int i) {
    return bf16{(uint16_t)((i & 1) ? (u[i >> 1] >> 16) : (u[i >> 1] & 0xFFFFu))};
  }
};
template <> struct Chunk<float> {
  __device__ static inline void unpack(const u32x4_t& u, float* x) {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(u[i]);
  }
  __device__ static inline u32x4_t pack(const float* x) {
    return u32x4_t{__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3])};
  }
  __device__ static inline float elem(const u32x4_t& u, int i) { return __uint_as_float(u[i]); }
};

// Offsets of element (slot, e) of a page block in matrix-core fragment order.
template <typename T, int DH>
__device__ inline int kfrag_off(int slot, int e) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT, KS = DH / KT;
  return (((slot / 16) * KS + e / KT) * 64 + ((e % KT) / KL) * 16 + slot % 16) * KL + e % KL;
}
// V: a lane fragment holds KL keys of one channel: keys 4g..4g+3 of the
// KL/4 consecutive 16-key tiles of a 4*KL-key group, g = lane/16.
template <typename T, int DH>
__device__ inline int vfrag_off(int slot, int e) {
  constexpr int KL = TT<T>::KL, DT = DH / 16, VG = 4 * KL;
  return (((slot / VG) * DT + e / 16) * 64 + ((slot % 16) / 4) * 16 + e % 16) * KL + ((slot % VG) / 16) * 4 + slot % 4;
}

// One workgroup of NW waves per (sequence, kv head, split at fixed absolute
// positions); a split is one or more chunks of NPG pages, the pages resident
// in LDS at once.  Wave w owns the 16-row groups w, w + NW, ...  Attention
// rows of a group are (block row j, query head g) pairs, R = Bq * G.
//  1. Loads are issued in the order their consumers need them and all stay in
//     flight together: the split's page ids (one vector load), the query rows
//     and the block's own key/value rows of this split (fused variant), then
//     the first chunk's K/V pages, page by page, into registers.  Vector loads
//     complete in issue order, so the query math below waits only for the
//     query loads.
//  2. Fused variant: QK-norm + RoPE of the R query rows into an LDS query
//     tile; QK-norm + RoPE of the block rows' keys, written to the paged
//     cache and to an LDS row tile together with their values.
//  3. Chunk by chunk, page by page in key order: the staged page goes to LDS
//     (its registers then take the next chunk's page), the block rows replace
//     their (stale) slots, and every wave computes the masked scores of its
//     first row group against the page (S^T = K Q^T on the matrix cores) and
//     takes one running-softmax step over them: the row maximum so far, the
//     rescale of the running sum and output by 2^(m_old - m_new), exp2 of the
//     scores and P V on the matrix cores.  Early pages are consumed while
//     later ones still arrive; after the last page the split partial (m, l,
//     O) of the row group is written.
//  4. A wave's further row groups (single-chunk splits only) then run over
//     the resident pages.  The combine kernel merges the splits in split
//     order.
// A row's arithmetic depends only on its own visible keys and the fixed split
// boundaries (and page order within them), never on the batch it is part of.
// MC = 0 instantiates single-chunk splits only (no chunk loop).

// Prefetch workgroup wg of an attention launch: plain 16-byte loads of its
// slice of p.pf (eight in flight per thread), which allocate in the
// memory-side cache; the loaded values only feed an empty asm statement.
// These workgroups run on the compute units the attention workgroups leave
// idle (the launch's LDS size keeps the two kinds off each other's units).
// They first sleep about 8K clocks (a few microseconds), so the attention
// workgroups' latency-bound first loads go out ahead of the prefetch stream:
// without the pause the attention launch grew by 0.6-1.5 us at the 8B shape.
template <int NT>
__device__ __forceinline__ void attn_prefetch(const AttnParams& p, int wg) {
  __builtin_amdgcn_s_sleep(127);
  const size_t b0 = (size_t)wg * p.pf_per;
  const size_t b1 = b0 + p.pf_per < p.pf_bytes ? b0 + p.pf_per : p.pf_bytes;
  const gu4* src = (const gu4*)(p.pf);
  u32x4_t x = u32x4_t{0u, 0u, 0u, 0u};
  size_t i = b0 / 16 + threadIdx.x;
  const size_t e = b1 / 16;
  for (; i + 7 * NT < e; i += 8 * NT) {
    u32x4_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = src[i + (size_t)u * NT];
#pragma unroll
    for (int u = 0; u < 8; ++u) x ^= v[u];
  }
  for (; i < e; i += NT) x ^= src[i];
  asm volatile("" ::"v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]));
}

template <typename T, int DH, int NW, bool FUSED, int NPART, int NPG, bool MC>
__global__ void __launch_bounds__(NW * 64) attn_kernel(AttnParams p) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  constexpr int KS = DH / KT;                 // k steps of S^T
  constexpr int DT = DH / 16;                 // output channel tiles
  constexpr int SK = NPG * PAGE;              // keys per chunk
  constexpr int PG = PAGE * DH;               // elements of one K (or V) page block
  constexpr int NT = NW * 64;
  constexpr int HALF = DH / 2;
  constexpr int V16 = PG * (int)sizeof(T) / 16;   // 16-byte vectors per page block
  constexpr int PER = V16 / NT;                   // per thread, page and K or V
  static_assert(V16 % NT == 0, "page blocks split evenly over the workgroup");
  typedef typename VFrag<T>::type vfrag_t;
  constexpr int QLD = DH + KL;                // padded row of the query tile
  constexpr int CE = 16 / (int)sizeof(T);     // channels per 16-byte chunk
  constexpr int LPR = DH / CE;                // lanes per head row
  constexpr int RPI = 64 / LPR;               // head rows per wave and pass
  constexpr int QI = FUSED ? (64 + NW * RPI - 1) / (NW * RPI) : 1;   // query passes per wave (R <= 64)
  constexpr int RC = CE * 8 / 16;             // 16-byte chunks of the lane's CE (cos, sin) pairs
  static_assert(CE == KL, "a key chunk is one fragment run of the paged layout");
  constexpr int NQ = CE / 4;                  // 16-byte fp32 loads per chunk and projection part
  extern __shared__ __align__(16) unsigned char smem[];
  T* lk = reinterpret_cast<T*>(smem);         // [NPG][PG] keys, fragment order
  T* lv = lk + (size_t)NPG * PG;              // [NPG][PG] values, fragment order

  if ((int)blockIdx.x >= p.nseq * p.Hkv * p.nsplit) {   // prefetch workgroup (uniform)
    attn_prefetch<NW * 64>(p, (int)blockIdx.x - p.nseq * p.Hkv * p.nsplit);
    return;
  }
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
  const int SPK = p.split_keys;               // keys per split: p.chunks chunks of SK keys
  const int key0 = split * SPK;
  const int t0 = p.start_pos[s];
  const int kv_len = t0 + p.Bq;
  const int cap = p.max_pages * PAGE;
  if (threadIdx.x == 0 && split == 0 && kv_len > cap) set_status(p.status, ST_CAPACITY);
  if (key0 >= kv_len) return;                 // uniform over the workgroup
  const int nch = MC ? min(p.chunks, (kv_len - key0 + SK - 1) / SK) : 1;   // chunks holding keys of the sequence
  T* lq = lv + (size_t)NPG * PG;              // [R][QLD] queries after QK-norm + RoPE (fused)
  T* ln = lq + (size_t)(FUSED ? R : 0) * QLD; // [rows][2][DH] block rows' keys and values (fused)

  // ---- 1. loads, in this order: page ids; query rows and the block rows of
  // the split as raw storage values (clamped rows are loaded and never
  // stored); then, once the page ids are in, the first chunk's K/V pages.
  // Nothing between the first load and the last K/V load waits on memory.
  // (one vector load: lane i reads page i of the split, i < p.chunks * NPG <= 64)
  const int npl = p.chunks * NPG;
  const int pvl = p.page_table[(size_t)s * p.max_pages + min(key0 / PAGE + (lane < npl ? lane : 0), p.max_pages - 1)];
  // Head rows (queries, block keys/values) are handled as 16-byte chunks: LPR
  // lanes per row, lane chunk cl holds channels [cl*CE, cl*CE + CE); its
  // rotate-half partner chunk sits LPR/2 lanes away and shares its RoPE angles.
  // The projection rows arrive as NPART fp32 partial sums (K parts of the QKV
  // projection) that are added here and rounded to the storage type.
  const float* qkv = p.qkv;
  const int cl = lane % LPR, rl = lane / LPR;
  const int rc0 = (cl % (LPR / 2)) * CE;      // RoPE angle index of the chunk's first channel
  u32x4_t qraw[QI][NPART][NQ], qrope[QI][RC];
  if constexpr (FUSED) {
#pragma unroll
    for (int it = 0; it < QI; ++it) {
      const int rr = min((w + NW * it) * RPI + rl, R - 1);   // clamped rows are computed and not stored
      const int j = rr / G, g = rr - j * G;
      const float* src = qkv + (size_t)(s * p.Bq + j) * p.ld_qkv + (size_t)(kvh * G + g) * DH + cl * CE;
#pragma unroll
      for (int k = 0; k < NPART; ++k)
#pragma unroll
        for (int c = 0; c < NQ; ++c) qraw[it][k][c] = *(const gu4*)(src + k * p.qkv_part + 4 * c);
      const gu4* rp = (const gu4*)(p.rope + (size_t)min(t0 + j, cap - 1) * HALF + rc0);   // past capacity: status set above
#pragma unroll
      for (int c = 0; c < RC; ++c) qrope[it][c] = rp[c];
    }
  }
  const int jlo = max(0, key0 - t0), jhi = min(p.Bq, key0 + SPK - t0);   // block rows in this split
  u32x4_t kraw[NPART][NQ], vraw[NPART][NQ], krope[RC];
  auto load_rows = [&](int it) {
    const int j = max(0, min(jlo + (w + NW * it) * RPI + rl, jhi - 1));   // clamped rows are not stored
    const float* src = qkv + (size_t)(s * p.Bq + j) * p.ld_qkv + (size_t)p.Hq * DH + (size_t)kvh * DH + cl * CE;
#pragma unroll
    for (int k = 0; k < NPART; ++k)
#pragma unroll
      for (int c = 0; c < NQ; ++c) {
        kraw[k][c] = *(const gu4*)(src + k * p.qkv_part + 4 * c);
        vraw[k][c] = *(const gu4*)(src + (size_t)p.Hkv * DH + k * p.qkv_part + 4 * c);
      }
    const gu4* rp = (const gu4*)(p.rope + (size_t)min(t0 + j, cap - 1) * HALF + rc0);
#pragma unroll
    for (int c = 0; c < RC; ++c) krope[c] = rp[c];
  };
  // the lane's CE channels: sum of the parts, rounded to the storage type
  auto combine = [&](const u32x4_t (&raw)[NPART][NQ], float (&x)[CE]) {
#pragma unroll
    for (int c = 0; c < NQ; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = __uint_as_float(raw[0][c][e]);
#pragma unroll
        for (int k = 1; k < NPART; ++k) v += __uint_as_float(raw[k][c][e]);
        x[4 * c + e] = TT<T>::rnd(v);
      }
  };
  // query fragments of row group rg from the query rows after QK-norm + RoPE (unfused variant)
  auto load_q_global = [&](int rg, u32x4_t (&qf)[KS]) {
    const int qr = min(rg * 16 + (lane & 15), R - 1);
    const int j = qr / G, g = qr - j * G;
    const T* qrow = reinterpret_cast<const T*>(p.q) + ((size_t)(s * p.Bq + j) * p.Hq + kvh * G + g) * DH;
#pragma unroll
    for (int k = 0; k < KS; ++k) qf[k] = *(const gu4*)(qrow + k * KT + (lane >> 4) * KL);
  };
  u32x4_t gq, gk;                             // QK-norm gains of the lane's chunk
  if constexpr (FUSED) {
    if (jlo < jhi) load_rows(0);              // uniform: only splits holding block rows
    gq = *(const gu4*)(reinterpret_cast<const T*>(p.q_norm) + cl * CE);
    gk = *(const gu4*)(reinterpret_cast<const T*>(p.k_norm) + cl * CE);
  }
  __builtin_amdgcn_sched_barrier(0);
  // a page of the split holding keys of the sequence with an invalid id sets
  // the status (once, here: the chunk loop below issues no conditional stores)
  {
    const bool bad = lane < npl && key0 + lane * PAGE < kv_len && (pvl < 0 || pvl >= p.num_pages);
    if (__builtin_amdgcn_ballot_w64(bad) != 0 && threadIdx.x == 0) set_status(p.status, ST_BAD_PAGE);
  }
  // page ids of chunk c: absent pages (past the sequence or invalid ids) read
  // page 0 of the pool and are never used
  auto chunk_pages = [&](int c, int (&pg)[NPG]) {
    unsigned pres = 0;
#pragma unroll
    for (int i = 0; i < NPG; ++i) {
      const int pv = __builtin_amdgcn_readlane(pvl, c * NPG + i);
      const bool ok = key0 + (c * NPG + i) * PAGE < kv_len && pv >= 0 && pv < p.num_pages;
      pg[i] = ok ? pv : 0;
      pres |= ok ? (1u << i) : 0u;
    }
    return pres;
  };
  u32x4_t kr[NPG][PER], vr[NPG][PER];
  auto issue_page = [&](int i, int pgid) {
    const size_t off = ((size_t)pgid * p.Hkv + kvh) * PG;
    const gu4* kg = (const gu4*)(reinterpret_cast<const T*>(p.kpool) + off);
    const gu4* vg = (const gu4*)(reinterpret_cast<const T*>(p.vpool) + off);
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      kr[i][it] = __builtin_nontemporal_load(&kg[threadIdx.x + it * NT]);   // each page is read once per launch
      vr[i][it] = __builtin_nontemporal_load(&vg[threadIdx.x + it * NT]);
    }
  };
  u32x4_t qf[KS];                             // the wave's first row group's query fragments
  const bool own = w < nrg;                    // uniform: the wave has a row group
  if constexpr (!FUSED) {
    if (own) load_q_global(w, qf);
  }
  int pgid[NPG];
  unsigned present = chunk_pages(0, pgid);    // pages holding keys of the sequence, with valid ids
#pragma unroll
  for (int i = 0; i < NPG; ++i) {
    issue_page(i, pgid[i]);
    __builtin_amdgcn_sched_barrier(0);        // issue order = page order = consumption order
  }

  // ---- 2. query tile; block rows to the cache and the row tile
  // RMSNorm over the row's LPR lanes, gain, then RoPE against the partner chunk
  auto norm_rope = [&](float (&x)[CE], const u32x4_t& gain, const u32x4_t (&rope)[RC], u32x4_t& out) {
    float g[CE], y[CE], cs[2 * CE];
    Chunk<T>::unpack(gain, g);
#pragma unroll
    for (int c = 0; c < RC; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) cs[4 * c + e] = __uint_as_float(rope[c][e]);
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < CE; ++i) ss += x[i] * x[i];
#pragma unroll
    for (int o = LPR / 2; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
    const float r = rsqrtf(ss / (float)DH + p.eps);
#pragma unroll
    for (int i = 0; i < CE; ++i) y[i] = x[i] * r * g[i];
    const bool lo = cl < LPR / 2;
#pragma unroll
    for (int i = 0; i < CE; ++i) {
      const float q = __shfl_xor(y[i], LPR / 2, 64);
      x[i] = lo ? y[i] * cs[2 * i] - q * cs[2 * i + 1] : y[i] * cs[2 * i] + q * cs[2 * i + 1];
    }
    out = Chunk<T>::pack(x);
  };
  if constexpr (FUSED) {
#pragma unroll
    for (int it = 0; it < QI; ++it) {
      const int rr = (w + NW * it) * RPI + rl;
      u32x4_t y;
      float x[CE];
      combine(qraw[it], x);
      norm_rope(x, gq, qrope[it], y);
      if (rr < R) *reinterpret_cast<u32x4_t*>(lq + (size_t)rr * QLD + cl * CE) = y;
    }
    for (int it = 0; jlo + (w + NW * it) * RPI < jhi; ++it) {   // uniform per wave
      if (it > 0) load_rows(it);
      u32x4_t y, vchunk;
      float x[CE];
      combine(kraw, x);
      norm_rope(x, gk, krope, y);
      combine(vraw, x);
      vchunk = Chunk<T>::pack(x);
      const int j = jlo + (w + NW * it) * RPI + rl;
      const int pos = t0 + j;
      // the cache page of the row (page index within the split, a lane of pvl)
      const int gp = __shfl(pvl, min(max((pos - key0) / PAGE, 0), 63), 64);
      if (j >= jhi) continue;
      T* row = ln + (size_t)(j - jlo) * 2 * DH;
      *reinterpret_cast<u32x4_t*>(row + cl * CE) = y;
      *reinterpret_cast<u32x4_t*>(row + DH + cl * CE) = vchunk;
      if (pos >= cap) continue;                // status set above
      if (gp < 0 || gp >= p.num_pages) continue;   // status set when the page's chunk is staged
      const int slot = pos % PAGE;
      T* kt_g = reinterpret_cast<T*>(p.kpool) + ((size_t)gp * p.Hkv + kvh) * PG;
      T* vt_g = reinterpret_cast<T*>(p.vpool) + ((size_t)gp * p.Hkv + kvh) * PG;
      *reinterpret_cast<u32x4_t*>(kt_g + kfrag_off<T, DH>(slot, cl * CE)) = y;   // CE = KL consecutive channels
#pragma unroll
      for (int i = 0; i < CE; ++i) vt_g[vfrag_off<T, DH>(slot, cl * CE + i)] = Chunk<T>::elem(vchunk, i);
    }
  }

  // ---- 3. page by page: scores as pages land, then one softmax step per chunk
  // The softmax runs in log2 units (scale folded with log2 e) with exp2; the
  // split partial is (M, sum 2^(s - M), sum 2^(s - M) v) with M the row's
  // maximum over the split's visible keys, reached chunk by chunk.
  typedef float score_t[4][4];               // [key tile][key within the lane's group of 4]
  auto scores = [&](int rg, int pi, int kc0, const u32x4_t (&qf)[KS], score_t& sc) {
    const int ar = rg * 16 + (lane & 15);
    const bool row_ok = ar < R;
    const int pos_row = t0 + (row_ok ? ar / G : 0);
    const int kp0 = kc0 + pi * PAGE;
    const u32x4_t* kb = reinterpret_cast<const u32x4_t*>(lk + (size_t)pi * PG);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < KS; ++k) acc = mma_frag(T(), kb[(kt * KS + k) * 64 + lane], qf[k], acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[kt][r] = acc[r];
    }
    // every key of the page precedes the block and every row is valid: no mask
    const bool full = kp0 + PAGE <= t0 && rg * 16 + 16 <= R;   // uniform
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
  };
  // one softmax step over page pi's scores: running maximum m (log2 units)
  // and sum l of row lane&15, running output o (row 4*(lane>>4)+r of
  // o[dt][r]); the state starts at m = -inf, l = 0, o = 0, and a step rescales
  // it by 2^(m_old - m_new) before adding the page's terms
  auto step = [&](score_t& sc, int pi, float& m, float& l, f32x4_t (&o)[DT]) {
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[kt][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    // scores are raw dot products; in log2 units a score is s * sl2 and the
    // row maximum is mx * sl2 (sl2 > 0).  A row with no visible key so far
    // keeps m = -inf, l = 0 and a zero output: its scores are all -inf and
    // exponentiate to 0 against a finite reference.
    const float mn = fmaxf(m, mx * sl2);
    const float mref = mn == -INFINITY ? 0.f : mn;
    const float f = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mref);
    m = mn;
    float ls = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // hardware 2^x: arguments are <= 0; results below 2^-126 flush to 0
        const float e = __builtin_amdgcn_exp2f(fmaf(sc[kt][r], sl2, -mref));
        sc[kt][r] = e;
        ls += e;
      }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    l = fmaf(l, f, ls);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float fr = __shfl(f, 4 * (lane >> 4) + r, 64);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt][r] *= fr;
    }
    if constexpr (KL == 8) {
      // P V with 32 keys per matrix-core op: lane group g supplies keys
      // 4g..4g+3 of key tiles 2c and 2c+1, and V holds the same keys in
      // one 16-byte fragment
      const u32x4_t* vb = reinterpret_cast<const u32x4_t*>(lv + (size_t)pi * PG);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const float (&a)[4] = sc[2 * c];
        const float (&b)[4] = sc[2 * c + 1];
        const u32x4_t pa = {f2bf2(a[0], a[1]), f2bf2(a[2], a[3]), f2bf2(b[0], b[1]), f2bf2(b[2], b[3])};
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] = mma_frag(T(), pa, vb[(c * DT + dt) * 64 + lane], o[dt]);
      }
    } else {
      const vfrag_t* vb = reinterpret_cast<const vfrag_t*>(lv + (size_t)pi * PG);
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] = mma_pv_frag<T>(sc[kt], vb[(kt * DT + dt) * 64 + lane], o[dt]);
    }
  };
  auto write_partial = [&](int rg, float m, float l, const f32x4_t (&o)[DT]) {
    const size_t pidx = (((size_t)s * p.Hkv + kvh) * p.rg + rg) * p.nsplit + split;
    float* po = p.part_o + pidx * 16 * DH;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) po[(4 * (lane >> 4) + r) * DH + dt * 16 + (lane & 15)] = o[dt][r];
    if (lane < 16) {
      p.part_ml[pidx * 32 + 2 * lane] = m;
      p.part_ml[pidx * 32 + 2 * lane + 1] = l;
    }
  };
  auto load_q = [&](int rg, u32x4_t (&qf)[KS]) {
    if constexpr (FUSED) {
      const int qr = min(rg * 16 + (lane & 15), R - 1);
#pragma unroll
      for (int k = 0; k < KS; ++k)
        qf[k] = *reinterpret_cast<const u32x4_t*>(lq + (size_t)qr * QLD + k * KT + (lane >> 4) * KL);
    } else {
      load_q_global(rg, qf);
    }
  };

  score_t sc;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o_run[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i) o_run[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // the staged pages of chunk c: to LDS page by page (each page's registers
  // then take the same page of the next chunk when `next`), block-row patch,
  // scores of the wave's first row group.  The vector-memory operations of a
  // chunk are exactly its prefetch loads, so the waits stay exact per page.
  auto chunk = [&](int c, bool next, const int (&pg_next)[NPG]) {
    const int kc0 = key0 + c * SK;
#pragma unroll
    for (int pi = 0; pi < NPG; ++pi) {
#pragma unroll
      for (int it = 0; it < PER; ++it) {
        reinterpret_cast<u32x4_t*>(lk + (size_t)pi * PG)[threadIdx.x + it * NT] = kr[pi][it];
        reinterpret_cast<u32x4_t*>(lv + (size_t)pi * PG)[threadIdx.x + it * NT] = vr[pi][it];
      }
      if (next) issue_page(pi, pg_next[pi]);   // the next chunk's page streams in meanwhile
      __syncthreads();
      if constexpr (FUSED) {
        // block rows of this page replace the slots staged from the cache
        const int jp0 = max(jlo, kc0 + pi * PAGE - t0), jp1 = min(jhi, kc0 + (pi + 1) * PAGE - t0);
        if (jp0 < jp1) {                       // uniform
          T* kt_l = lk + (size_t)pi * PG;
          T* vt_l = lv + (size_t)pi * PG;
          for (int e = threadIdx.x; e < (jp1 - jp0) * DH; e += NT) {
            const int j = jp0 + e / DH, d = e % DH;
            const int slot = (t0 + j) % PAGE;
            const T* row = ln + (size_t)(j - jlo) * 2 * DH;
            kt_l[kfrag_off<T, DH>(slot, d)] = row[d];
            vt_l[vfrag_off<T, DH>(slot, d)] = row[DH + d];
          }
          __syncthreads();
        }
        if (c == 0 && pi == 0 && own) load_q(w, qf);   // LDS reads only
      }
      if (own && ((present >> pi) & 1u)) {   // uniform
        scores(w, pi, kc0, qf, sc);
        step(sc, pi, m_run, l_run, o_run);
      }
    }
  };
  // Fused multi-chunk splits: a chunk's pages are staged first, then the two
  // halves of the workgroup (waves w and w + 4, same row group) take the
  // even and the odd pages, each with a running softmax of its own, and the
  // two states are merged at the end -- twice the waves on the matrix cores
  // and the exponentials while the next chunk streams in.
  if constexpr (MC && FUSED) {
    static_assert(NW == 8, "fused launches have eight waves");
    const int rgw = w & 3, par = w >> 2;
    const bool own2 = rgw < nrg;              // uniform (R <= 64: at most four row groups)
    auto chunk2 = [&](int c, bool next, const int (&pg_next)[NPG]) {
      const int kc0 = key0 + c * SK;
#pragma unroll
      for (int pi = 0; pi < NPG; ++pi) {
#pragma unroll
        for (int it = 0; it < PER; ++it) {
          reinterpret_cast<u32x4_t*>(lk + (size_t)pi * PG)[threadIdx.x + it * NT] = kr[pi][it];
          reinterpret_cast<u32x4_t*>(lv + (size_t)pi * PG)[threadIdx.x + it * NT] = vr[pi][it];
        }
        if (next) issue_page(pi, pg_next[pi]);   // the next chunk's page streams in meanwhile
      }
      __syncthreads();
      // block rows of this chunk replace the slots staged from the cache
      const int jc0 = max(jlo, kc0 - t0), jc1 = min(jhi, kc0 + SK - t0);
      if (jc0 < jc1) {                         // uniform
        for (int e = threadIdx.x; e < (jc1 - jc0) * DH; e += NT) {
          const int j = jc0 + e / DH, d = e % DH;
          const int pos = t0 + j, pi = (pos - kc0) / PAGE, slot = pos % PAGE;
          const T* row = ln + (size_t)(j - jlo) * 2 * DH;
          lk[(size_t)pi * PG + kfrag_off<T, DH>(slot, d)] = row[d];
          lv[(size_t)pi * PG + vfrag_off<T, DH>(slot, d)] = row[DH + d];
        }
        __syncthreads();
      }
      if (c == 0 && own2) load_q(rgw, qf);     // LDS reads only
#pragma unroll
      for (int pi = 0; pi < NPG; ++pi)
        if ((pi & 1) == par && own2 && ((present >> pi) & 1u)) {   // uniform
          scores(rgw, pi, kc0, qf, sc);
          step(sc, pi, m_run, l_run, o_run);
        }
    };
    for (int c = 0; c + 1 < nch; ++c) {        // uniform
      int pg_next[NPG];
      const unsigned pres_next = chunk_pages(c + 1, pg_next);
      if (c > 0) __syncthreads();              // every wave is done with the previous chunk's pages
      chunk2(c, true, pg_next);
      present = pres_next;
    }
    if (nch > 1) __syncthreads();
    chunk2(nch - 1, false, pgid);
    // merge: the odd-page state of each row group through LDS into the even-page one
    __syncthreads();                           // the pages are no longer read
    float* scr = reinterpret_cast<float*>(lk);     // [4][DT][4][64] outputs, then [4][16][2] (m, l)
    float* sml = scr + 4 * DT * 4 * 64;
    static_assert((4 * DT * 4 * 64 + 4 * 16 * 2) * sizeof(float) <= 2 * NPG * PG * sizeof(T),
                  "the merge scratch fits in the chunk's key and value pages");
    if (own2 && par == 1) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) scr[((rgw * DT + dt) * 4 + r) * 64 + lane] = o_run[dt][r];
      if (lane < 16) {
        sml[(rgw * 16 + lane) * 2] = m_run;
        sml[(rgw * 16 + lane) * 2 + 1] = l_run;
      }
    }
    __syncthreads();
    if (own2 && par == 0) {
      const float m1 = sml[(rgw * 16 + (lane & 15)) * 2], l1 = sml[(rgw * 16 + (lane & 15)) * 2 + 1];
      const float M = fmaxf(m_run, m1);
      const float Mref = M == -INFINITY ? 0.f : M;
      const float f0 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - Mref);
      const float f1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - Mref);
      const float l = fmaf(l_run, f0, l1 * f1);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float g0 = __shfl(f0, 4 * (lane >> 4) + r, 64), g1 = __shfl(f1, 4 * (lane >> 4) + r, 64);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          o_run[dt][r] = fmaf(o_run[dt][r], g0, scr[((rgw * DT + dt) * 4 + r) * 64 + lane] * g1);
      }
      write_partial(rgw, M, l, o_run);
    }
    return;
  }
  // chunks 0 .. nch-2 prefetch the next one unconditionally; the last chunk is peeled
  if constexpr (MC) {
    for (int c = 0; c + 1 < nch; ++c) {        // uniform
      int pg_next[NPG];
      const unsigned pres_next = chunk_pages(c + 1, pg_next);
      if (c > 0) __syncthreads();              // every wave is done with the previous chunk's pages
      chunk(c, true, pg_next);
      present = pres_next;
    }
    if (nch > 1) __syncthreads();
  }
  chunk(nch - 1, false, pgid);
  if (own) write_partial(w, m_run, l_run, o_run);
  // further row groups: single-chunk splits only (the host launches no others
  // with more row groups than waves); pages resident, no barrier
  for (int rg = w + NW; rg < nrg; rg += NW) {  // uniform per wave
    float m = -INFINITY, l = 0.f;
    f32x4_t o[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    load_q(rg, qf);
    unsigned pres0 = 0;
#pragma unroll
    for (int i = 0; i < NPG; ++i) {
      const int pv = __builtin_amdgcn_readlane(pvl, i);
      pres0 |= (key0 + i * PAGE < kv_len && pv >= 0 && pv < p.num_pages) ? (1u << i) : 0u;
    }
#pragma unroll
    for (int pi = 0; pi < NPG; ++pi)
      if ((pres0 >> pi) & 1u) {
        scores(rg, pi, key0, qf, sc);
        step(sc, pi, m, l, o);
      }
    write_partial(rg, m, l, o);
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
  int ns = (kv_len + p.split_keys - 1) / p.split_keys;
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
  frag_st<T>(p.outf, row, hq * DH + d, v);
}

// Dynamic LDS of the attention kernel: the split's K and V pages, plus the
// query tile and the block rows' key/value tile in the fused variant.
template <typename T, int DH>
static size_t attn_lds(bool fused, int Bq, int G, int sk) {
  const size_t pages = 2 * (size_t)sk * DH * sizeof(T);
  if (!fused) return pages;
  const int rows = Bq < sk ? Bq : sk;
  return pages + ((size_t)Bq * G * (DH + TT<T>::KL) + (size_t)rows * 2 * DH) * sizeof(T);
}
static constexpr size_t ATTN_LDS_MAX = 159 * 1024;

// Fused: R = Bq * G <= 64 rows, at most four 16-row groups.  Eight waves: the
// four without a row group share the loads and the query / block-row prologue
// (two waves per SIMD hide each other's latency; 8B shape at context 4096:
// 19.8 -> 18.7 us per layer, 8 ragged sequences 76.9 -> 71.8 us).
template <typename T, int DH>
static bool fuses_dh(int Bq, int G, int sk) {
  return Bq * G <= 64 && attn_lds<T, DH>(true, Bq, G, sk) <= ATTN_LDS_MAX;
}

template <typename T, int DH, int NW, bool FUSED, int NPART, int NPG, bool MC>
static hipError_t launch_kn(const AttnParams& p, hipStream_t st) {
  const size_t lds = attn_lds<T, DH>(FUSED, p.Bq, p.Hq / p.Hkv, NPG * PAGE);   // one chunk resident
  if (lds > ATTN_LDS_MAX) return hipErrorInvalidConfiguration;
  // allow the largest dynamic LDS, once per instantiation (thread-safe static initialisation)
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&attn_kernel<T, DH, NW, FUSED, NPART, NPG, MC>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)ATTN_LDS_MAX);
  if (attr != hipSuccess) return attr;
  if (p.pf_wgs < 0 || (p.pf_wgs > 0 && (!p.pf || p.pf_per % 16 || p.pf_bytes % 16 ||
                                        (size_t)p.pf_wgs * p.pf_per < p.pf_bytes)))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL((attn_kernel<T, DH, NW, FUSED, NPART, NPG, MC>), dim3(p.nseq * p.Hkv * p.nsplit + p.pf_wgs),
                     dim3(NW * 64),
                     lds, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), dim3(p.nseq * p.Bq, p.Hq), dim3(DH), 0, st, p);
  return hipGetLastError();
}

// chunk sizes: 128 keys, and 256 for bf16 (four fp32 pages exceed the LDS)
template <typename T, int DH, int NW, bool FUSED, int NPART>
static hipError_t launch_k(const AttnParams& p, hipStream_t st) {
  if (p.chunks < 1 || p.split_keys % p.chunks) return hipErrorInvalidValue;
  const int ck = p.split_keys / p.chunks;
  if (ck * p.chunks > 64 * PAGE) return hipErrorInvalidValue;   // one page-id lane per page of a split
  if (p.chunks > 1 && (p.Bq * (p.Hq / p.Hkv) + 15) / 16 > NW) return hipErrorInvalidValue;
  if (ck == 2 * PAGE)
    return p.chunks > 1 ? launch_kn<T, DH, NW, FUSED, NPART, 2, true>(p, st)
                        : launch_kn<T, DH, NW, FUSED, NPART, 2, false>(p, st);
  if constexpr (sizeof(T) == 2)
    if (ck == 4 * PAGE)
      return p.chunks > 1 ? launch_kn<T, DH, NW, FUSED, NPART, 4, true>(p, st)
                          : launch_kn<T, DH, NW, FUSED, NPART, 4, false>(p, st);
  return hipErrorInvalidValue;
}

template <typename T, int DH>
static hipError_t launch_dh(const AttnParams& p, hipStream_t st) {
  if (p.fused) {
    if (p.chunks < 1 || !fuses_dh<T, DH>(p.Bq, p.Hq / p.Hkv, p.split_keys / p.chunks))
      return hipErrorInvalidConfiguration;
    if (p.qkv_ks == 2) return launch_k<T, DH, 8, true, 2>(p, st);
    if (p.qkv_ks == 1) return launch_k<T, DH, 8, true, 1>(p, st);
    return hipErrorInvalidValue;
  }
  // one wave per 16-row group up to eight; beyond, waves take several groups
  if (p.Bq * (p.Hq / p.Hkv) <= 64) return launch_k<T, DH, 4, false, 1>(p, st);
  return launch_k<T, DH, 8, false, 1>(p, st);
}

int attention_waves(bool fused, int Bq, int G) { return fused || Bq * G > 64 ? 8 : 4; }

bool attention_fuses_rope(bool bf16, int Bq, int G, int Dh, int sk) {
  if (Dh == 128) return bf16 ? fuses_dh<dflow::bf16, 128>(Bq, G, sk) : fuses_dh<float, 128>(Bq, G, sk);
  if (Dh == 64) return bf16 ? fuses_dh<dflow::bf16, 64>(Bq, G, sk) : fuses_dh<float, 64>(Bq, G, sk);
  return false;
}

hipError_t launch_attention(bool bf16, const AttnParams& p, hipStream_t st) {
  if (p.Dh == 128) return bf16 ? launch_dh<dflow::bf16, 128>(p, st) : launch_dh<float, 128>(p, st);
  if (p.Dh == 64) return bf16 ? launch_dh<dflow::bf16, 64>(p, st) : launch_dh<float, 64>(p, st);
  return hipErrorInvalidValue;
}

}  // namespace dflow
