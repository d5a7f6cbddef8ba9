// Row-wise and integer kernels of the DFlow round: embedding gather, RMSNorm,
// fused QK-norm + RoPE + paged KV write, relay gather / reject-conditioned
// input build, acceptance scan, argmax reduction, KV commit and the
// measurement-only forced-draft builder.
#include "common.h"
#include "kernels.h"
#include "round_state.h"

namespace dflow {

// ---------------------------------------------------------------- embedding
// Also writes the per-16-column-strip sums of squares of the row (the
// RMSNorm row scale of the next projection), ssq[row * ssq_ld + c].
template <typename T>
__global__ void embed_kernel(const int* tok, const T* E, int V, int d, T* out, int* status, float* ssq, int ssq_ld,
                             FragOut of) {
  const int row = blockIdx.x;
  int t = tok[row];
  const bool ok = t >= 0 && t < V;
  if (!ok && threadIdx.x == 0) set_status(status, ST_BAD_TOKEN);
  for (int c = threadIdx.x; c < d / 16; c += blockDim.x) {
    float sq = 0.f, vs[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const size_t i = (size_t)c * 16 + e;
      const float v = ok ? TT<T>::ld(E, (size_t)t * d + i) : 0.f;
      TT<T>::st(out, (size_t)row * d + i, v);
      vs[e] = v;
      sq += v * v;
    }
    frag_st_run<T>(of, row, c * 16, vs, 16);
    if (ssq) ssq[(size_t)row * ssq_ld + c] = sq;
  }
}

hipError_t launch_embed(bool isbf, const int* tok, int M, const void* E, int V, int d, void* out, int* status,
                        float* ssq, int ssq_ld, FragOut of, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (d % 16) return hipErrorInvalidValue;
  if (isbf)
    hipLaunchKernelGGL(embed_kernel<bf16>, dim3(M), dim3(256), 0, s, tok, (const bf16*)E, V, d, (bf16*)out, status,
                       ssq, ssq_ld, of);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, s, tok, (const float*)E, V, d, (float*)out,
                       status, ssq, ssq_ld, of);
  return hipGetLastError();
}

// ---------------------------------------------------------------- RMSNorm
// One block per row.  Each thread keeps up to RV 16-byte input vectors in
// registers between the sum of squares and the scaled write.
template <typename TI> struct Vec16;
template <> struct Vec16<bf16> {
  static constexpr int N = 8;
  __device__ static inline void load(const bf16* p, float* v) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) { v[2 * i] = bf2f(w[i] & 0xFFFF); v[2 * i + 1] = bf2f(w[i] >> 16); }
  }
};
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ static inline void load(const float* p, float* v) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
};

template <typename T, typename TI>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const TI* x, int ldx, int d, const T* g, float eps, T* out,
                                                      int ldo, FragOut of) {
  constexpr int VN = Vec16<TI>::N;
  constexpr int RV = 4;                       // vectors held per thread (d <= 256*RV*VN)
  __shared__ float sh[32];
  const int row = blockIdx.x;
  const TI* xr = x + (size_t)row * ldx;
  const int nv = d / VN;
  float v[RV][VN];
  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < RV; ++r) {
    const int i = threadIdx.x + r * blockDim.x;
    if (i < nv) {
      Vec16<TI>::load(xr + (size_t)i * VN, v[r]);
#pragma unroll
      for (int e = 0; e < VN; ++e) ss += v[r][e] * v[r][e];
    }
  }
  for (int i = threadIdx.x + RV * blockDim.x; i < nv; i += blockDim.x) {   // rows wider than the register budget
    float t[VN];
    Vec16<TI>::load(xr + (size_t)i * VN, t);
#pragma unroll
    for (int e = 0; e < VN; ++e) ss += t[e] * t[e];
  }
  ss = block_sum(ss, sh);
  const float rs = rsqrtf(ss / (float)d + eps);
  T* o = out + (size_t)row * ldo;
#pragma unroll
  for (int r = 0; r < RV; ++r) {
    const int i = threadIdx.x + r * blockDim.x;
    if (i < nv) {
      float y[VN];
#pragma unroll
      for (int e = 0; e < VN; ++e) {
        y[e] = v[r][e] * rs * TT<T>::ld(g, (size_t)i * VN + e);
        TT<T>::st(o, (size_t)i * VN + e, y[e]);
      }
      frag_st_run<T>(of, row, i * VN, y, VN);
    }
  }
  for (int i = threadIdx.x + RV * blockDim.x; i < nv; i += blockDim.x) {
    float t[VN];
    Vec16<TI>::load(xr + (size_t)i * VN, t);
    float y[VN];
#pragma unroll
    for (int e = 0; e < VN; ++e) {
      y[e] = t[e] * rs * TT<T>::ld(g, (size_t)i * VN + e);
      TT<T>::st(o, (size_t)i * VN + e, y[e]);
    }
    frag_st_run<T>(of, row, i * VN, y, VN);
  }
}

hipError_t launch_rmsnorm(bool isbf, bool in_f32, const void* x, int ldx, int M, int d, const void* g, float eps,
                          void* out, int ldo, FragOut of, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if ((d & 7) || (ldx & 7)) return hipErrorInvalidValue;   // 16-byte row vectors
  if (isbf && in_f32)
    hipLaunchKernelGGL((rmsnorm_kernel<bf16, float>), dim3(M), dim3(256), 0, s, (const float*)x, ldx, d,
                       (const bf16*)g, eps, (bf16*)out, ldo, of);
  else if (isbf)
    hipLaunchKernelGGL((rmsnorm_kernel<bf16, bf16>), dim3(M), dim3(256), 0, s, (const bf16*)x, ldx, d,
                       (const bf16*)g, eps, (bf16*)out, ldo, of);
  else
    hipLaunchKernelGGL((rmsnorm_kernel<float, float>), dim3(M), dim3(256), 0, s, (const float*)x, ldx, d,
                       (const float*)g, eps, (float*)out, ldo, of);
  return hipGetLastError();
}

// ---------------------------------------------------------------- QK-norm + RoPE + KV write
// Block (row, head): head < nq is a query head, then Hkv key heads, then Hkv value heads.
template <typename T>
__global__ void qk_rope_kernel(RopeParams p) {
  const int row = blockIdx.x;
  const int h = blockIdx.y;
  const int s = row / p.Bq, j = row - s * p.Bq;
  if (p.row_limit && j > p.row_limit[s]) return;
  const int Dh = p.Dh, half = Dh / 2;
  const int pos = p.start_pos[s] + j;
  const int layer = blockIdx.z;
  const size_t off = (size_t)row * p.ld + (size_t)layer * p.layer_cols + (size_t)h * Dh;
  const T* src = reinterpret_cast<const T*>(p.qkv) + off;
  const float* src32 = p.qkv32 ? p.qkv32 + off : nullptr;
  // element e of the head row as a storage-type value (fp32 parts: sum, rounded)
  auto val = [&](int e) -> float {
    if (!src32) return TT<T>::ld(src, e);
    return TT<T>::rnd(p.part ? src32[e] + src32[p.part + e] : src32[e]);
  };
  const bool is_q = h < p.nq;
  const bool is_k = !is_q && h < p.nq + p.Hkv;
  const int kvh = is_q ? 0 : (is_k ? h - p.nq : h - p.nq - p.Hkv);

  size_t page_base = 0;
  const int pidx = pos / PAGE;
  if (pos < 0 || pidx >= p.max_pages) {      // also bounds the RoPE table
    if (threadIdx.x == 0) set_status(p.status, ST_CAPACITY);
    return;
  }
  if (!is_q) {
    const int page = p.page_table[(size_t)s * p.max_pages + pidx];
    if (page < 0 || page >= p.num_pages) {
      if (threadIdx.x == 0) set_status(p.status, ST_BAD_PAGE);
      return;
    }
    page_base = ((size_t)page * p.Hkv + kvh) * PAGE * Dh;
  }
  const int slot = pos % PAGE;
  const int i = threadIdx.x;   // pair (i, i + half)
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  const int KS = Dh / KT, DT = Dh / 16;
  if (!is_q && !is_k) {        // value head, fragment order (see kernels.h)
    T* vp = reinterpret_cast<T*>(p.vpool) + (size_t)layer * p.pool_stride + page_base;
    const int vg = slot / (4 * KL), q = (slot % 16) / 4, r = ((slot % (4 * KL)) / 16) * 4 + slot % 4;
    for (int e = i; e < Dh; e += blockDim.x)
      TT<T>::st(vp, ((size_t)(vg * DT + e / 16) * 64 + q * 16 + e % 16) * KL + r, val(e));
    return;
  }
  // key element d of this slot, fragment order (see kernels.h)
  auto koff = [&](int d) -> size_t {
    return ((size_t)((slot / 16) * KS + d / KT) * 64 + ((d % KT) / KL) * 16 + slot % 16) * KL + d % KL;
  };
  const T* gain = reinterpret_cast<const T*>(is_q ? p.q_norm : (p.k_norms ? p.k_norms[layer] : p.k_norm));
  float x1 = 0.f, x2 = 0.f;
  if (i < half) { x1 = val(i); x2 = val(i + half); }
  const float ss = wave_sum(x1 * x1 + x2 * x2);
  const float r = rsqrtf(ss / (float)Dh + p.eps);
  if (i < half) {
    const float y1 = x1 * r * TT<T>::ld(gain, i);
    const float y2 = x2 * r * TT<T>::ld(gain, i + half);
    const float2 cs = p.rope[(size_t)pos * half + i];
    const float o1 = y1 * cs.x - y2 * cs.y;
    const float o2 = y2 * cs.x + y1 * cs.y;
    if (is_q) {
      T* q = reinterpret_cast<T*>(p.q_out) + (size_t)row * p.nq * Dh + (size_t)h * Dh;
      TT<T>::st(q, i, o1);
      TT<T>::st(q, i + half, o2);
    } else {
      T* kp = reinterpret_cast<T*>(p.kpool) + (size_t)layer * p.pool_stride + page_base;
      TT<T>::st(kp, koff(i), o1);
      TT<T>::st(kp, koff(i + half), o2);
    }
  }
}

hipError_t launch_qk_rope_write(bool isbf, const RopeParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (p.Dh > 128 || (p.Dh & 1)) return hipErrorInvalidValue;
  if (p.nlayers < 1 || (p.nlayers > 1 && p.nq != 0)) return hipErrorInvalidValue;
  dim3 grid(p.M, p.nq + 2 * p.Hkv, p.nlayers);
  if (isbf) hipLaunchKernelGGL(qk_rope_kernel<bf16>, grid, dim3(64), 0, s, p);
  else hipLaunchKernelGGL(qk_rope_kernel<float>, grid, dim3(64), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------- argmax
// Keys are [group][M].  Workgroup b takes a contiguous range of groups; its
// lane t reads row t%16 (+16 per row batch) of groups t/16, t/16 + 16, ...,
// so 16 consecutive lanes read one contiguous 128-byte run.  Each workgroup
// leaves its per-row maxima in part[b][m]; the last workgroup to arrive
// (device-scope counter, reset by that workgroup) reduces the partials and
// writes the indices.  Max is order-independent, so the result does not
// depend on arrival order.
__global__ void __launch_bounds__(256) argmax_reduce_kernel(const uint64_t* amax, int groups, int M, uint64_t* part,
                                                            unsigned* counter, int* out, DraftOut dr) {
  __shared__ uint64_t sh[16][17];
  __shared__ bool s_last;
  const int r16 = threadIdx.x & 15, slice = threadIdx.x >> 4;
  const int per = (groups + gridDim.x - 1) / gridDim.x;
  const int g0 = blockIdx.x * per, g1 = min(groups, g0 + per);
  for (int m0 = 0; m0 < M; m0 += 16) {
    const int m = m0 + r16, mc = min(m, M - 1);
    uint64_t best = 0;
#pragma unroll 4
    for (int g = g0 + slice; g < g1; g += 16) {
      const uint64_t k = amax[(size_t)g * M + mc];
      best = k > best ? k : best;
    }
    sh[slice][r16] = best;
    __syncthreads();
    if (threadIdx.x < 16 && m < M) {
      uint64_t b = sh[0][r16];
      for (int i = 1; i < 16; ++i) b = sh[i][r16] > b ? sh[i][r16] : b;
      part[(size_t)blockIdx.x * M + m] = b;
    }
    __syncthreads();
  }
  // publish this workgroup's partials, then count arrivals
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(counter, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  // lane (slice, r16) folds partials of workgroups slice, slice + 16, ... (independent loads)
  for (int m0 = 0; m0 < M; m0 += 16) {
    const int m = m0 + r16, mc = min(m, M - 1);
    uint64_t best = 0;
#pragma unroll
    for (int w = slice; w < ARGMAX_SPLITS; w += 16) {
      if (w < (int)gridDim.x) {
        const uint64_t k = __hip_atomic_load(part + (size_t)w * M + mc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        best = k > best ? k : best;
      }
    }
    sh[slice][r16] = best;
    __syncthreads();
    if (threadIdx.x < 16 && m < M) {
      uint64_t b = sh[0][r16];
      for (int i = 1; i < 16; ++i) b = sh[i][r16] > b ? sh[i][r16] : b;
      const int v = argmax_key_index(b);
      if (out) out[m] = v;
      if (dr.B > 0) {
        const int sq = m / dr.B, j = m - sq * dr.B;
        if (dr.block_out) dr.block_out[m] = j == 0 ? dr.anchor[sq] : v;
        if (dr.draft_tok && j > 0) dr.draft_tok[(size_t)sq * (dr.B - 1) + j - 1] = v;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

hipError_t launch_argmax_reduce(const uint64_t* amax, int groups, int M, uint64_t* part, unsigned* counter, int* out,
                                const DraftOut* draft, hipStream_t s) {
  if (M <= 0 || groups <= 0) return hipSuccess;
  DraftOut dr{nullptr, 0, nullptr, nullptr};
  if (draft) {
    if (draft->B < 1 || M % draft->B || !draft->anchor) return hipErrorInvalidValue;
    dr = *draft;
  }
  const int nb = groups < ARGMAX_SPLITS ? groups : ARGMAX_SPLITS;
  hipLaunchKernelGGL(argmax_reduce_kernel, dim3(nb), dim3(256), 0, s, amax, groups, M, part, counter, out, dr);
  return hipGetLastError();
}

// ---------------------------------------------------------------- acceptance scan
// a = number of leading drafts d_i (block index i) equal to the target argmax of row i-1;
// bonus = argmax of row a.
__global__ void accept_kernel(const int* block, const int* g, int nseq, int B, int carry_window, int* accept_len,
                              int* bonus, int* committed, int* n_carry, int* carry_rec) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= nseq) return;
  const int K = B - 1;
  const int* blk = block + (size_t)s * B;
  const int* gs = g + (size_t)s * B;
  int a = 0;
  while (a < K && blk[a + 1] == gs[a]) ++a;
  write_accept_outcome(s, a, gs[a], blk, B, carry_window, accept_len, bonus, committed, n_carry, carry_rec);
}

hipError_t launch_accept(const int* block, const int* g, int nseq, int B, int carry_window, int* accept_len,
                         int* bonus, int* committed, int* n_carry, int* carry_rec, hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3((nseq + 63) / 64), dim3(64), 0, s, block, g, nseq, B, carry_window,
                     accept_len, bonus, committed, n_carry, carry_rec);
  return hipGetLastError();
}

// ---------------------------------------------------------------- relay
// u[s*B + i] = [E(b); E(y_rej); f[s*B + rec[1] + i - 1]] for relayed block indices rec[4]..rec[0], else 0.
// One workgroup per (row, segment), 16-byte copies (d * sizeof(T) is a multiple of 16).
template <typename T>
__global__ void relay_gather_kernel(int carry_on, const int* rec, const T* E, const T* f, int B, int d, int V, T* u,
                                    FragOut of) {
  const int row = blockIdx.x, seg = blockIdx.y;
  const int s = row / B, i = row - s * B;
  const int* r = rec + (size_t)s * CARRY_REC;
  const bool valid = carry_on && i >= 1 && i >= r[4] && i <= r[0] && r[0] < B && r[1] >= 1 &&
                     r[1] + r[0] <= B && r[2] >= 0 && r[2] < V && r[3] >= 0 && r[3] < V;
  uint4* dst = reinterpret_cast<uint4*>(u + ((size_t)row * 3 + seg) * d);
  const int nvec = d * (int)sizeof(T) / 16;
  constexpr int EV = 16 / (int)sizeof(T);   // elements per 16-byte vector
  static_assert(EV == TT<T>::KL, "a 16-byte vector is one lane fragment");
  // one vector is one lane fragment of the matrix-core-order copy
  auto fdst = [&](int v) {
    return reinterpret_cast<uint4*>(reinterpret_cast<T*>(of.p) + afrag_off<T>(row, of.c0 + seg * d + v * EV, of.ktiles));
  };
  if (!valid) {
    for (int v = threadIdx.x; v < nvec; v += blockDim.x) {
      dst[v] = make_uint4(0u, 0u, 0u, 0u);
      if (of.p) *fdst(v) = make_uint4(0u, 0u, 0u, 0u);
    }
    return;
  }
  const T* src = seg == 0 ? E + (size_t)r[2] * d : seg == 1 ? E + (size_t)r[3] * d
                                                            : f + ((size_t)s * B + r[1] + i - 1) * d;
  const uint4* sv = reinterpret_cast<const uint4*>(src);
  for (int v = threadIdx.x; v < nvec; v += blockDim.x) {
    const uint4 x = sv[v];
    dst[v] = x;
    if (of.p) *fdst(v) = x;
  }
}

hipError_t launch_relay_gather(bool isbf, int carry_on, const int* carry_rec, const void* E, const void* f, int nseq,
                               int B, int d, int V, void* u, FragOut of, hipStream_t s) {
  if (d % 16) return hipErrorInvalidValue;
  if (isbf)
    hipLaunchKernelGGL(relay_gather_kernel<bf16>, dim3(nseq * B, 3), dim3(256), 0, s, carry_on, carry_rec,
                       (const bf16*)E, (const bf16*)f, B, d, V, (bf16*)u, of);
  else
    hipLaunchKernelGGL(relay_gather_kernel<float>, dim3(nseq * B, 3), dim3(256), 0, s, carry_on, carry_rec,
                       (const float*)E, (const float*)f, B, d, V, (float*)u, of);
  return hipGetLastError();
}

// x[s*B + 0] = E(anchor); relayed rows: E_mask + beta * LN(h) + gamma; others E_mask.
// Also writes the per-16-column-strip sums of squares of the stored row.
// Thread t owns the 16-column chunks t, t + 256, ... (d <= 16 * 256 * RC);
// the carried state is read once and kept in registers for both LayerNorm passes.
template <typename T>
__global__ void __launch_bounds__(256) relay_input_kernel(int carry_on, const int* rec, const int* anchor, const T* E,
                                                          const T* e_mask, const T* f,
                                                          const float* bg, const T* ln_g, const T* ln_b, float ln_eps,
                                                          int B, int d, int V, T* x, int* status, float* ssq,
                                                          int ssq_ld, FragOut of) {
  constexpr int RC = 2;
  __shared__ float sh[32];
  const int row = blockIdx.x;
  const int s = row / B, i = row - s * B;
  const int nc = d / 16;
  T* xr = x + (size_t)row * d;
  const int* r = rec + (size_t)s * CARRY_REC;
  const bool relay = i > 0 && carry_on && i >= r[4] && i <= r[0] && r[0] < B && r[1] >= 1 && r[1] + r[0] <= B &&
                     r[2] >= 0 && r[2] < V && r[3] >= 0 && r[3] < V;
  int src_tok = -1;                  // row 0: the anchor's embedding
  if (i == 0) {
    src_tok = anchor[s];
    if (src_tok < 0 || src_tok >= V) {
      if (threadIdx.x == 0) set_status(status, ST_BAD_TOKEN);
      src_tok = -2;                  // zero row
    }
  }
  float hv[RC][16];
  float mu = 0.f, rs = 0.f;
  const T* h = nullptr;
  if (relay) {                       // LayerNorm statistics of the carried state (uniform per workgroup)
    h = f + ((size_t)s * B + r[1] + i - 1) * d;
    float sm = 0.f;
#pragma unroll
    for (int k = 0; k < RC; ++k) {
      const int c = threadIdx.x + 256 * k;
      if (c < nc) {
        Row16<T>::load(h + (size_t)c * 16, hv[k]);
#pragma unroll
        for (int e = 0; e < 16; ++e) sm += hv[k][e];
      }
    }
    mu = block_sum(sm, sh) / (float)d;
    float sv = 0.f;
#pragma unroll
    for (int k = 0; k < RC; ++k) {
      const int c = threadIdx.x + 256 * k;
      if (c < nc)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float t = hv[k][e] - mu;
          sv += t * t;
        }
    }
    rs = rsqrtf(block_sum(sv, sh) / (float)d + ln_eps);
  }
  const float* bgr = bg + (size_t)row * 2 * d;
#pragma unroll
  for (int k = 0; k < RC; ++k) {
    const int c = threadIdx.x + 256 * k;
    if (c >= nc) continue;
    float v[16];
    if (i == 0) {
      if (src_tok >= 0) Row16<T>::load(E + (size_t)src_tok * d + (size_t)c * 16, v);
      else
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = 0.f;
    } else {
      Row16<T>::load(e_mask + (size_t)c * 16, v);
      if (relay) {
        float g[16], b[16];
        Row16<T>::load(ln_g + (size_t)c * 16, g);
        Row16<T>::load(ln_b + (size_t)c * 16, b);
        const float4* be = reinterpret_cast<const float4*>(bgr + (size_t)c * 16);
        const float4* ga = reinterpret_cast<const float4*>(bgr + d + (size_t)c * 16);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 bq = be[q], gq = ga[q];
          const float bb[4] = {bq.x, bq.y, bq.z, bq.w}, gg[4] = {gq.x, gq.y, gq.z, gq.w};
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4) {
            const int e = 4 * q + e4;
            const float ln = (hv[k][e] - mu) * rs * g[e] + b[e];
            v[e] = TT<T>::rnd(v[e] + bb[e4] * ln + gg[e4]);
          }
        }
      }
    }
    Row16<T>::store(xr + (size_t)c * 16, v);
    frag_st_run<T>(of, row, c * 16, v, 16);
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) sq += v[e] * v[e];
    if (ssq) ssq[(size_t)row * ssq_ld + c] = sq;
  }
}

hipError_t launch_relay_input(bool isbf, int carry_on, const int* carry_rec, const int* anchor, const void* E,
                              const void* e_mask, const void* f, const float* bg, const void* ln_g,
                              const void* ln_b, float ln_eps, int nseq, int B, int d, int V, void* x, int* status,
                              float* ssq, int ssq_ld, FragOut of, hipStream_t s) {
  if (d % 16 || d > 16 * 256 * 2) return hipErrorInvalidValue;
  if (isbf)
    hipLaunchKernelGGL(relay_input_kernel<bf16>, dim3(nseq * B), dim3(256), 0, s, carry_on, carry_rec, anchor,
                       (const bf16*)E, (const bf16*)e_mask, (const bf16*)f, bg, (const bf16*)ln_g,
                       (const bf16*)ln_b, ln_eps, B, d, V, (bf16*)x, status, ssq, ssq_ld, of);
  else
    hipLaunchKernelGGL(relay_input_kernel<float>, dim3(nseq * B), dim3(256), 0, s, carry_on, carry_rec, anchor,
                       (const float*)E, (const float*)e_mask, (const float*)f, bg, (const float*)ln_g,
                       (const float*)ln_b, ln_eps, B, d, V, (float*)x, status, ssq, ssq_ld, of);
  return hipGetLastError();
}

// ---------------------------------------------------------------- commit
__global__ void commit_kernel(const int* accept_len, int nseq, int* seq_len) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s < nseq) seq_len[s] += accept_len[s] + 1;
}

hipError_t launch_commit(const int* accept_len, int nseq, int* seq_len, hipStream_t s) {
  hipLaunchKernelGGL(commit_kernel, dim3((nseq + 63) / 64), dim3(64), 0, s, accept_len, nseq, seq_len);
  return hipGetLastError();
}

// ---------------------------------------------------------------- forced drafts (measurement only)
__global__ void force_kernel(const int* traj, int stride, int traj_len, const signed char* mode, const int* tok,
                             const int* anchor, const int* start_pos, int B, int V, int* block_tok) {
  const int s = blockIdx.x;
  const int t = start_pos[s];
  for (int j = threadIdx.x; j < B; j += blockDim.x) {
    int v;
    const int m = mode[(size_t)s * B + j];
    const int u = tok[(size_t)s * B + j];
    const int p = t + j;
    const int tv = (p >= 0 && p < traj_len) ? traj[(size_t)s * stride + p] : 0;
    if (j == 0) v = anchor[s];
    else if (m == 1) v = tv;
    else if (m == 2) v = (int)(((long long)tv + 1 + u) % V);
    else v = u;
    block_tok[(size_t)s * B + j] = v;
  }
}

hipError_t launch_force(const int* traj, int traj_stride, int traj_len, const signed char* mode, const int* tok,
                        const int* anchor, const int* start_pos, int nseq, int B, int V, int* block_tok,
                        hipStream_t s) {
  hipLaunchKernelGGL(force_kernel, dim3(nseq), dim3(64), 0, s, traj, traj_stride, traj_len, mode, tok, anchor,
                     start_pos, B, V, block_tok);
  return hipGetLastError();
}

// ---------------------------------------------------------------- small utilities
__global__ void set_int_kernel(int* dst, int v) { *dst = v; }
hipError_t launch_set_int(int* dst, int value, hipStream_t s) {
  hipLaunchKernelGGL(set_int_kernel, dim3(1), dim3(1), 0, s, dst, value);
  return hipGetLastError();
}
__global__ void fill_u32_kernel(uint32_t* dst, uint32_t v, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = v;
}
hipError_t launch_fill_u32(uint32_t* dst, uint32_t value, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, dst, value, n);
  return hipGetLastError();
}

}  // namespace dflow
