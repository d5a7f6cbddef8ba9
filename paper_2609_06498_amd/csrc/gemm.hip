// Skinny-M GEMM for weight-streaming projections: Y[M, N] = A[M, K] W[N, K]^T.
//
// Weights are pre-packed into 1 KB tiles of 16 output columns x KT k values
// (KT = 32 bf16 or 16 fp32) laid out so that lane l of a wavefront loads the
// 16 contiguous bytes W[n0 + l%16][k0 + (l/16)*KL ..] with one dwordx4 load;
// the tiles of one 16-column strip are contiguous along k.  One workgroup owns
// NG strips and the full K range; its waves split K into equal contiguous
// ranges that depend only on (N, K), and the wave partials are summed in LDS
// in wave order.  Every output element therefore sees the same reduction
// order whatever M is, which keeps results batch- and position-invariant.
#include "common.h"
#include "kernels.h"

namespace dflow {

template <typename T, int NG, int MT, int EPI>
__global__ void __launch_bounds__(1024) gemm_kernel(GemmParams p) {
  constexpr int KL = TT<T>::KL;
  constexpr int KT = TT<T>::KT;
  constexpr int U = (MT >= 4) ? 1 : (MT == 2 ? 2 : 4);   // k tiles per pipeline stage
  extern __shared__ float lds[];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int g = blockIdx.x;
  const int nt0 = g * NG;
  const int nvalid = min(NG, p.ntiles - nt0);
  const int kper = (p.ktiles + nw - 1) / nw;
  const int kb = min(p.ktiles, w * kper);
  const int ke = min(p.ktiles, kb + kper);
  const int M = p.M;
  const int mtiles = (M + 15) >> 4;

  const uint4* Wp = reinterpret_cast<const uint4*>(p.W);
  const T* Ap = reinterpret_cast<const T*>(p.A);
  const uint4 zero = make_uint4(0, 0, 0, 0);

  f32x4_t acc[MT][NG];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NG; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  size_t wrow[NG];
#pragma unroll
  for (int j = 0; j < NG; ++j) wrow[j] = (size_t)(nt0 + j) * p.ktiles * 64 + lane;
  const T* arow[MT];
  bool aval[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int m = i * 16 + (lane & 15);
    aval[i] = (i < mtiles) && (m < M);
    arow[i] = Ap + (size_t)(aval[i] ? m : 0) * p.lda + (lane >> 4) * KL;
  }

  uint4 bq[2][U][NG];
  uint4 aq[2][U][MT];
  auto load = [&](int st, int kt) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kt + u;
      const bool kv = k < ke;
#pragma unroll
      for (int j = 0; j < NG; ++j)
        bq[st][u][j] = (kv && j < nvalid) ? Wp[wrow[j] + (size_t)k * 64] : zero;
#pragma unroll
      for (int i = 0; i < MT; ++i)
        aq[st][u][i] = (kv && aval[i]) ? *reinterpret_cast<const uint4*>(arow[i] + (size_t)k * KT) : zero;
    }
  };
  auto compute = [&](int st) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NG; ++j) acc[i][j] = mma_frag(T(), aq[st][u][i], bq[st][u][j], acc[i][j]);
  };

  if (kb < ke) {
    load(0, kb);
    int kt = kb;
    for (;;) {
      const int k1 = kt + U;
      if (k1 < ke) load(1, k1);
      compute(0);
      if (k1 >= ke) break;
      const int k2 = k1 + U;
      if (k2 < ke) load(0, k2);
      compute(1);
      if (k2 >= ke) break;
      kt = k2;
    }
  }

  // ---- cross-wave reduction in fixed wave order, one m tile at a time
  float* red = lds;                                 // [nw][NG][64][4]
  constexpr int CW = NG * 16 + 1;                   // padded C-tile row
  float* ct = lds + (size_t)nw * NG * 256;          // [MT*16][CW]
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    if (i >= mtiles) break;
#pragma unroll
    for (int j = 0; j < NG; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((w * NG + j) * 64 + lane) * 4 + r] = acc[i][j][r];
    __syncthreads();
    for (int e = threadIdx.x; e < NG * 256; e += blockDim.x) {
      float s = 0.f;
      for (int ww = 0; ww < nw; ++ww) s += red[(size_t)ww * NG * 256 + e];
      const int j = e >> 8, l = (e >> 2) & 63, r = e & 3;
      ct[(i * 16 + 4 * (l >> 4) + r) * CW + j * 16 + (l & 15)] = s;
    }
    __syncthreads();
  }

  // ---- epilogue
  const int ncols = nvalid * 16;
  const int colbase = p.col0 + nt0 * 16;
  if constexpr (EPI == EPI_ARGMAX) {
    for (int e = threadIdx.x; e < M * ncols; e += blockDim.x) {
      const int m = e / ncols, n = e - m * ncols;
      if (p.logits) p.logits[(size_t)m * p.ldl + colbase + n] = ct[m * CW + n];
    }
    for (int m = threadIdx.x; m < M; m += blockDim.x) {
      float best = ct[m * CW];
      int bi = 0;
      for (int n = 1; n < ncols; ++n) {
        const float v = ct[m * CW + n];
        if (v > best) { best = v; bi = n; }
      }
      p.amax[(size_t)g * p.amax_ld + m] = argmax_key(best, colbase + bi);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int half = ncols / 2;
    const int obase = (p.col0 + nt0 * 16) / 2;
    for (int e = threadIdx.x; e < M * half; e += blockDim.x) {
      const int m = e / half, c = e - m * half;
      const int pair = c >> 4, cc = c & 15;
      const float gt = ct[m * CW + pair * 32 + cc];
      const float up = ct[m * CW + pair * 32 + 16 + cc];
      TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + obase + c, silu(gt) * up);
    }
  } else {
    for (int e = threadIdx.x; e < M * ncols; e += blockDim.x) {
      const int m = e / ncols, n = e - m * ncols;
      const int col = colbase + n;
      float v = ct[m * CW + n];
      if constexpr (EPI == EPI_STORE_T) {
        TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, v);
      } else if constexpr (EPI == EPI_STORE_F32) {
        reinterpret_cast<float*>(p.Y)[(size_t)m * p.ldy + col] = v;
      } else if constexpr (EPI == EPI_RESID) {
        v += TT<T>::ld(reinterpret_cast<const T*>(p.R), (size_t)m * p.ldr + col);
        TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, v);
        if (p.Y2) TT<T>::st(reinterpret_cast<T*>(p.Y2), (size_t)m * p.ldy2 + col, v);
      } else if constexpr (EPI == EPI_BIAS_SILU) {
        v += TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
        TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, silu(v));
      } else if constexpr (EPI == EPI_BIAS_F32) {
        v += TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
        reinterpret_cast<float*>(p.Y)[(size_t)m * p.ldy + col] = v;
      }
    }
  }
}

// Column-strip count per workgroup is tied to the epilogue; the wave count
// (the K split) depends only on the K extent, never on M.
GemmShape gemm_shape(int ntiles, int ktiles, int epi) {
  GemmShape s;
  s.ng = (epi == EPI_SWIGLU) ? 2 : (epi == EPI_ARGMAX ? 4 : 1);
  int waves = ktiles / 16;
  if (waves < 1) waves = 1;
  if (waves > 16) waves = 16;
  s.waves = waves;
  s.groups = (ntiles + s.ng - 1) / s.ng;
  return s;
}

template <typename T, int NG, int EPI>
static hipError_t launch_mt(const GemmParams& p, const GemmShape& sh, hipStream_t st) {
  const int mt = (p.M + 15) / 16;
  const int cw = NG * 16 + 1;
  auto go = [&](auto kern, int MTv) {
    const size_t lds = ((size_t)sh.waves * NG * 256 + (size_t)MTv * 16 * cw) * sizeof(float);
    if (lds > 65536) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(kern, dim3(sh.groups), dim3(sh.waves * 64), lds, st, p);
    return hipGetLastError();
  };
  if (mt <= 1) return go(gemm_kernel<T, NG, 1, EPI>, 1);
  if (mt <= 2) return go(gemm_kernel<T, NG, 2, EPI>, 2);
  if (mt <= 4) return go(gemm_kernel<T, NG, 4, EPI>, 4);
  if (mt <= 8) return go(gemm_kernel<T, NG, 8, EPI>, 8);
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t launch_t(int epi, const GemmParams& p, hipStream_t st) {
  const GemmShape sh = gemm_shape(p.ntiles, p.ktiles, epi);
  switch (epi) {
    case EPI_STORE_T: return launch_mt<T, 1, EPI_STORE_T>(p, sh, st);
    case EPI_STORE_F32: return launch_mt<T, 1, EPI_STORE_F32>(p, sh, st);
    case EPI_RESID: return launch_mt<T, 1, EPI_RESID>(p, sh, st);
    case EPI_SWIGLU: return launch_mt<T, 2, EPI_SWIGLU>(p, sh, st);
    case EPI_BIAS_SILU: return launch_mt<T, 1, EPI_BIAS_SILU>(p, sh, st);
    case EPI_BIAS_F32: return launch_mt<T, 1, EPI_BIAS_F32>(p, sh, st);
    case EPI_ARGMAX: return launch_mt<T, 4, EPI_ARGMAX>(p, sh, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(bool bf16, int epi, const GemmParams& p, hipStream_t st) {
  if (p.M <= 0 || p.ntiles <= 0 || p.ktiles <= 0) return hipSuccess;
  return bf16 ? launch_t<dflow::bf16>(epi, p, st) : launch_t<float>(epi, p, st);
}

// ------------------------------------------------------------------ packing
// out tile (nt, kt) lane l element e <- W[src_row(nt, l%16)][kt*KT + (l/16)*KL + e]
// gate_up: W is [2F, K] = [gate; up]; packed strip 2i is gate strip i, 2i+1 is up strip i.
template <typename T>
__global__ void pack_kernel(const T* __restrict__ W, int N, int K, int gate_up, T* __restrict__ out) {
  constexpr int KL = TT<T>::KL, KT = TT<T>::KT;
  const int ktiles = K / KT;
  const size_t total = (size_t)N * K;
  for (size_t o = (size_t)blockIdx.x * blockDim.x + threadIdx.x; o < total; o += (size_t)gridDim.x * blockDim.x) {
    const int e = (int)(o % KL);
    const size_t lt = o / KL;
    const int l = (int)(lt % 64);
    const size_t tile = lt / 64;
    const int kt = (int)(tile % ktiles);
    const int nt = (int)(tile / ktiles);
    int strip = nt;
    if (gate_up) strip = (nt & 1) ? (N / 32 + (nt >> 1)) : (nt >> 1);
    const size_t row = (size_t)strip * 16 + (l & 15);
    const size_t col = (size_t)kt * KT + (l >> 4) * KL + e;
    out[o] = W[row * K + col];
  }
}

hipError_t launch_pack(bool bf16, const void* w, int N, int K, int gate_up, void* out, hipStream_t s) {
  const int threads = 256;
  const size_t total = (size_t)N * K;
  int blocks = (int)((total + threads - 1) / threads);
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    hipLaunchKernelGGL(pack_kernel<dflow::bf16>, dim3(blocks), dim3(threads), 0, s,
                       (const dflow::bf16*)w, N, K, gate_up, (dflow::bf16*)out);
  else
    hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(threads), 0, s, (const float*)w, N, K, gate_up,
                       (float*)out);
  return hipGetLastError();
}

}  // namespace dflow
