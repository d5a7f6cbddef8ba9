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
#include <cmath>

#include "common.h"
#include "gemm.h"

namespace dflow {

template <typename T, int NG, int MT, int EPI, bool NORM>
__global__ void __launch_bounds__(512) gemm_kernel(GemmParams p) {
  constexpr int KL = TT<T>::KL;
  constexpr int KT = TT<T>::KT;
  // k tiles per pipeline stage: 4 fragments of weights per stage and buffer
  constexpr int U = (MT * NG >= 8) ? 1 : 8 / (MT * NG);
  extern __shared__ float lds[];
  const int lane = threadIdx.x & 63;
  // wave index as a scalar: keeps the k-range bounds and the pipeline control uniform
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nw = blockDim.x >> 6;
  // workgroup (strip group g, K part h): the K parts of a group sit on adjacent workgroups
  const int ks = p.ksplit > 1 ? p.ksplit : 1;
  const int g = blockIdx.x / ks, h = blockIdx.x - g * ks;
  const int nt0 = g * NG;
  const int nvalid = min(NG, p.ntiles - nt0);
  const int kpart = (p.ktiles + ks - 1) / ks;
  const int k0 = min(p.ktiles, h * kpart), k1 = min(p.ktiles, k0 + kpart);
  const int kper = (k1 - k0 + nw - 1) / nw;
  const int kb = min(k1, k0 + w * kper);
  const int ke = min(k1, kb + kper);
  const int M = p.M;
  const int mtiles = (M + 15) >> 4;

  // Explicit global address space: generic (flat) loads would also count
  // against the LDS counter and defeat the load pipelining below.  Weight
  // tiles are read by exactly one wave, once: they are loaded non-temporally,
  // so the weight stream does not evict the A rows, which every workgroup
  // re-reads from L2 (at the 8B down projection this takes a launch from
  // 23.8 to 20.2 us).
  const gu4* Wp = (const gu4*)(p.W);
  const T* Ap = reinterpret_cast<const T*>(p.A);

  f32x4_t acc[MT][NG];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NG; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Out-of-range strips and rows are clamped to valid addresses instead of
  // being predicated, so the main loop is straight-line code; their results
  // land in columns/rows the epilogue never stores.
  const gu4* wrow[NG];
#pragma unroll
  for (int j = 0; j < NG; ++j) wrow[j] = Wp + (size_t)min(nt0 + j, p.ntiles - 1) * p.ktiles * 64 + lane;
  const gu4* arow[MT];
  // one k tile of A: 16 bytes per lane, 4 apart along a row-major row (16 row
  // pieces per load), or 64 apart in the matrix-core-order copy (1 KB contiguous)
  const int ast = p.Af ? 64 : KT * (int)sizeof(T) / 16;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    if (p.Af) {   // rows past M in the last row tile are read and never stored
      arow[i] = (const gu4*)(p.Af) + (size_t)min(i, mtiles - 1) * p.ktiles * 64 + lane;
    } else {
      const int m = min(i * 16 + (lane & 15), M - 1);
      arow[i] = (const gu4*)(Ap + (size_t)m * p.lda + (lane >> 4) * KL);
    }
  }

  u32x4_t bq[2][U][NG];
  u32x4_t aq[2][U][MT];
#define DFLOW_LOAD(st, kt)                                                             \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                       \
    _Pragma("unroll") for (int j = 0; j < NG; ++j) bq[st][u][j] = __builtin_nontemporal_load(&wrow[j][(size_t)((kt) + u) * 64]); \
    _Pragma("unroll") for (int i = 0; i < MT; ++i) aq[st][u][i] = arow[i][(size_t)((kt) + u) * ast]; \
  }                                                                                     \
  __builtin_amdgcn_sched_barrier(0);
#define DFLOW_COMPUTE(st)                                                              \
  _Pragma("unroll") for (int u = 0; u < U; ++u)                                         \
    _Pragma("unroll") for (int i = 0; i < MT; ++i)                                      \
      _Pragma("unroll") for (int j = 0; j < NG; ++j) acc[i][j] = mma_frag(T(), aq[st][u][i], bq[st][u][j], acc[i][j]);

  // RMSNorm row scales.  The norm gain is folded into the packed weight, so
  // the normalised projection is rs[m] * (x W'^T) and the scale is applied in
  // the epilogue.  rs comes from the per-strip sums of squares ssq[m][c] that
  // the producer of x left behind: lane q of a 16-lane group sums strips
  // c = q (mod 16) in increasing c, then a fixed butterfly over the group --
  // the same order for every row, batch and launch shape.  Group g owns rows
  // g + k * ngrp; the partials of strips c < 256 for its first two rows are
  // loaded early (see below) and consumed after the main loop, so the
  // reduction costs no latency on the critical path.
  constexpr int EL = 16;                  // early partials per lane and row
  const int q16 = threadIdx.x & 15, grp = threadIdx.x >> 4, ngrp = blockDim.x >> 4;
  float ea[NORM ? EL : 1], eb[NORM ? EL : 1];
  // The epilogue's own operand -- the residual rows (written by the previous
  // launch, so an L2 miss) or the bias -- for this thread's first PF outputs,
  // loaded early instead of after the main loop.
  constexpr bool EPF = EPI == EPI_RESID || EPI == EPI_BIAS_SILU || EPI == EPI_BIAS_F32;
  constexpr int PF = EPF ? 4 : 1;
  const int ncols = nvalid * 16;
  const int colbase = p.col0 + nt0 * 16;
  float pre[PF];
  // Early operand loads (row-scale partials, epilogue operand).  Loads
  // complete in order, so they are issued after the first matrix-core ops:
  // ahead of them they would hold up the pipeline start (the 8B QKV launch's
  // first stage landed 3.7 instead of 1.6 us after its start).
  auto prefetch = [&]() {
    if constexpr (NORM) {
      // rows of a group are clamped to valid rows and strips read the padded
      // row (ssq_ld >= 256 entries), so every load is unconditional
      gf32* ra = (gf32*)(p.ssq) + (size_t)min(grp, M - 1) * p.ssq_ld + q16;
      gf32* rb = (gf32*)(p.ssq) + (size_t)min(grp + ngrp, M - 1) * p.ssq_ld + q16;
#pragma unroll
      for (int it = 0; it < EL; ++it) {
        ea[it] = ra[16 * it];
        eb[it] = rb[16 * it];
      }
      __builtin_amdgcn_sched_barrier(0);
    }

    if constexpr (EPF) {
#pragma unroll
      for (int it = 0; it < PF; ++it) {
        const int e = threadIdx.x + it * (int)blockDim.x;
        const int m = min(e / ncols, M - 1), col = colbase + e % ncols;   // clamped: never used past M
        pre[it] = EPI == EPI_RESID ? TT<T>::ld(reinterpret_cast<const T*>(p.R), (size_t)m * p.ldr + col)
                                   : TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
      }
    }
  };

  // Full stages of U tiles, double-buffered.  Inside the steady-state loop
  // every load is unconditional, so the compiler's wait before each compute
  // covers only the stage being consumed, never the prefetch just issued.
  const int nst = (ke - kb) / U;
  int kt = kb;
  if (nst > 2) {
    // first iteration peeled: the early loads go out after its first stage
    DFLOW_LOAD(0, kt);
    DFLOW_LOAD(1, kt + U);
    DFLOW_COMPUTE(0);
    prefetch();
    DFLOW_LOAD(0, kt + 2 * U);
    DFLOW_COMPUTE(1);
    kt += 2 * U;
    int left = nst - 2;
    while (left > 2) {
      DFLOW_LOAD(1, kt + U);
      DFLOW_COMPUTE(0);
      DFLOW_LOAD(0, kt + 2 * U);
      DFLOW_COMPUTE(1);
      kt += 2 * U;
      left -= 2;
    }
    if (left == 2) {
      DFLOW_LOAD(1, kt + U);
      DFLOW_COMPUTE(0);
      DFLOW_COMPUTE(1);
      kt += 2 * U;
    } else {
      DFLOW_COMPUTE(0);
      kt += U;
    }
  } else {   // short range (a few stages)
    prefetch();
    if (nst > 0) {
      DFLOW_LOAD(0, kt);
      if (nst == 2) {
        DFLOW_LOAD(1, kt + U);
        DFLOW_COMPUTE(0);
        DFLOW_COMPUTE(1);
        kt += 2 * U;
      } else {
        DFLOW_COMPUTE(0);
        kt += U;
      }
    }
  }
  // ragged tail (fewer than U tiles)
  for (; kt < ke; ++kt) {
    u32x4_t b1[NG], a1[MT];
#pragma unroll
    for (int j = 0; j < NG; ++j) b1[j] = __builtin_nontemporal_load(&wrow[j][(size_t)kt * 64]);
#pragma unroll
    for (int i = 0; i < MT; ++i) a1[i] = arow[i][(size_t)kt * ast];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NG; ++j) acc[i][j] = mma_frag(T(), a1[i], b1[j], acc[i][j]);
  }
#undef DFLOW_LOAD
#undef DFLOW_COMPUTE

  __shared__ float s_rs[NORM ? MT * 16 : 1];
  if constexpr (NORM) {
    const int np = p.ssq_parts;
    for (int m0 = grp; m0 < MT * 16; m0 += 2 * ngrp) {
      const int ma = min(m0, M - 1), mb = min(m0 + ngrp, M - 1);
      float sa = 0.f, sb = 0.f;
      if (m0 == grp) {
#pragma unroll
        for (int it = 0; it < EL; ++it) {
          const bool ok = q16 + 16 * it < np;
          sa += ok ? ea[it] : 0.f;
          sb += ok ? eb[it] : 0.f;
        }
      } else {
        gf32* ra = (gf32*)(p.ssq) + (size_t)ma * p.ssq_ld + q16;
        gf32* rb = (gf32*)(p.ssq) + (size_t)mb * p.ssq_ld + q16;
        float la[EL], lb[EL];
#pragma unroll
        for (int it = 0; it < EL; ++it) {
          la[it] = ra[16 * it];
          lb[it] = rb[16 * it];
        }
#pragma unroll
        for (int it = 0; it < EL; ++it) {
          const bool ok = q16 + 16 * it < np;
          sa += ok ? la[it] : 0.f;
          sb += ok ? lb[it] : 0.f;
        }
      }
      for (int c = q16 + 16 * EL; c < np; c += 16) {   // strips beyond the early window (d > 4096)
        sa += p.ssq[(size_t)ma * p.ssq_ld + c];
        sb += p.ssq[(size_t)mb * p.ssq_ld + c];
      }
#pragma unroll
      for (int x = 8; x >= 1; x >>= 1) {
        sa += __shfl_xor(sa, x, 16);
        sb += __shfl_xor(sb, x, 16);
      }
      if (q16 == 0) {
        s_rs[m0] = rsqrtf(sa / (float)(np * 16) + p.eps);
        if (m0 + ngrp < MT * 16) s_rs[m0 + ngrp] = rsqrtf(sb / (float)(np * 16) + p.eps);
      }
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
  if constexpr (EPI == EPI_ARGMAX) {
    for (int e = threadIdx.x; e < M * ncols; e += blockDim.x) {
      const int m = e / ncols, n = e - m * ncols;
      float v = ct[m * CW + n];
      if constexpr (NORM) ct[m * CW + n] = v = v * s_rs[m];
      if (p.logits) p.logits[(size_t)m * p.ldl + colbase + n] = v;
    }
    __syncthreads();
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
    // each packed strip holds 8 gate columns followed by the matching 8 up columns
    const int half = ncols / 2;
    const int obase = (p.col0 + nt0 * 16) / 2;
    for (int e = threadIdx.x; e < M * half; e += blockDim.x) {
      const int m = e / half, c = e - m * half;
      const int strip = c >> 3, cc = c & 7;
      float gt = ct[m * CW + strip * 16 + cc];
      float up = ct[m * CW + strip * 16 + 8 + cc];
      if constexpr (NORM) {
        gt *= s_rs[m];
        up *= s_rs[m];
      }
      const float y = silu(gt) * up;
      TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + obase + c, y);
      frag_st<T>(p.yf, m, obase + c, y);
    }
  } else {
    // output e of this thread; x = the residual or bias value of its column
    auto out1 = [&](int e, float x) {
      const int m = e / ncols, n = e - m * ncols;
      const int col = colbase + n;
      float v = ct[m * CW + n];
      if constexpr (NORM) v *= s_rs[m];
      if constexpr (EPI == EPI_STORE_T) {
        TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, v);
      } else if constexpr (EPI == EPI_STORE_F32) {
        reinterpret_cast<float*>(p.Y)[(size_t)h * p.y_part + (size_t)m * p.ldy + col] = v;
      } else if constexpr (EPI == EPI_RESID) {
        v = TT<T>::rnd(v + x);
        TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, v);
        if (p.Y2) TT<T>::st(reinterpret_cast<T*>(p.Y2), (size_t)m * p.ldy2 + col, v);
        frag_st<T>(p.yf, m, col, v);
        frag_st<T>(p.y2f, m, col, v);
        ct[m * CW + n] = v;
      } else if constexpr (EPI == EPI_BIAS_SILU) {
        v += x;
        TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, silu(v));
        frag_st<T>(p.yf, m, col, silu(v));
      } else if constexpr (EPI == EPI_BIAS_F32) {
        v += x;
        reinterpret_cast<float*>(p.Y)[(size_t)m * p.ldy + col] = v;
      }
    };
    const int nout = M * ncols;
#pragma unroll
    for (int it = 0; it < PF; ++it) {
      const int e = threadIdx.x + it * (int)blockDim.x;
      if (e < nout) out1(e, pre[it]);
    }
    for (int e = threadIdx.x + PF * (int)blockDim.x; e < nout; e += blockDim.x) {
      const int col = colbase + e % ncols;
      float x = 0.f;
      if constexpr (EPI == EPI_RESID)
        x = TT<T>::ld(reinterpret_cast<const T*>(p.R), (size_t)(e / ncols) * p.ldr + col);
      else if constexpr (EPI == EPI_BIAS_SILU || EPI == EPI_BIAS_F32)
        x = TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
      out1(e, x);
    }
    if constexpr (EPI == EPI_RESID) {
      if (p.ssq_out) {   // sum of squares of the stored values, per row and 16-column strip
        __syncthreads();
        for (int e = threadIdx.x; e < M * nvalid; e += blockDim.x) {
          const int m = e / nvalid, j = e - m * nvalid;
          float sq = 0.f;
#pragma unroll
          for (int c = 0; c < 16; ++c) {
            const float v = ct[m * CW + j * 16 + c];
            sq += v * v;
          }
          p.ssq_out[(size_t)m * p.ssq_out_ld + nt0 + j] = sq;
        }
      }
    }
  }
}

// ------------------------------------------------------------------ large M
// Tiled GEMM for M > 128 rows (serving batches, prefill chunks): A and W
// staged through LDS in MFMA fragment order.  The K loop runs the same contiguous ranges as the weight-
// streaming kernel's waves (gemm_shape's wave count for this N, K) and folds
// each range's MFMA chain into the running sum in range order, starting from
// zero, so every output element is bit-identical to what the weight-streaming
// kernel computes for it at any M: the result of a row never depends on the
// batch it is part of.  The M tiles of one strip tile are dispatched to the
// same XCD (round-robin placement, id mod 8), so its weights are fetched from
// HBM once and shared through that XCD's L2.
// Same row scale as the weight-streaming kernel: lane q of a 16-lane group
// sums strips c = q (mod 16) in increasing c, then the fixed butterfly.
__device__ inline float norm_row_scale(const GemmParams& p, int m, int q16) {
  constexpr int EL = 16;
  const int np = p.ssq_parts;
  gf32* r = (gf32*)(p.ssq) + (size_t)m * p.ssq_ld + q16;
  float v[EL];
#pragma unroll
  for (int it = 0; it < EL; ++it) v[it] = r[16 * it];   // padded rows: ssq_ld >= 256 entries
  float sa = 0.f;
#pragma unroll
  for (int it = 0; it < EL; ++it) sa += (q16 + 16 * it < np) ? v[it] : 0.f;
  for (int c = q16 + 16 * EL; c < np; c += 16) sa += p.ssq[(size_t)m * p.ssq_ld + c];
#pragma unroll
  for (int x = 8; x >= 1; x >>= 1) sa += __shfl_xor(sa, x, 16);
  return rsqrtf(sa / (float)(np * 16) + p.eps);
}

constexpr int TILE_BM = 128, TILE_BS = 8, TILE_CW = TILE_BS * 16 + 4;
constexpr size_t TILE_LDS = (size_t)TILE_BM * TILE_CW * sizeof(float);   // C tile (widest); >= 2 staging buffers

// Workgroup tile 128 rows x BS strips (BS = 8: 128 columns; 4 for narrow
// weights, so that enough workgroups exist), four waves of 64 rows x BS/2
// strips.  Per k tile the workgroup stages 8 KB of A and BS KB of W; loads
// run TILE_D - 1 k tiles ahead in registers and the LDS is double buffered.
// About 250 registers per lane and at most 68 KB of LDS, so two workgroups
// share a compute unit.
constexpr int TILE_D = 4;
// NTW: the weight tiles are loaded non-temporally (a launch with one M tile
// reads each weight byte once; with several, the M tiles of a strip tile share
// it through L2 and the loads stay temporal).
template <typename T, int EPI, bool NORM, int BS, bool NTW>
__global__ void __launch_bounds__(256, 2) gemm_tile_kernel(GemmParams p, int nw, int mt, int units) {
  constexpr int KL = TT<T>::KL;
  constexpr int KT = TT<T>::KT;
  constexpr int D = TILE_D;
  constexpr int WS = BS / 2;                  // strips per wave
  constexpr int NWC = BS / 4;                 // W chunks per thread and k tile
  constexpr int CW = BS * 16 + 4;             // padded C-tile row
  extern __shared__ float lds[];
  __shared__ float s_rs[NORM ? TILE_BM : 1];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  // block -> (m tile, unit = strip tile x K part); the m tiles of a unit share an XCD
  const int x8 = blockIdx.x & 7, y = blockIdx.x >> 3;
  const int mtile = y % mt, unit = (y / mt) * 8 + x8;
  if (unit >= units) return;                                  // padding of the dispatch grid
  const int ks = p.ksplit > 1 ? p.ksplit : 1;
  const int stile = unit / ks, h = unit - stile * ks;
  const int nt0 = stile * BS;
  const int nvalid = min(BS, p.ntiles - nt0);
  const int m0 = mtile * TILE_BM;
  const int rows = min(TILE_BM, p.M - m0);
  const int kpart = (p.ktiles + ks - 1) / ks;
  const int k0 = min(p.ktiles, h * kpart), k1 = min(p.ktiles, k0 + kpart);
  const int kper = (k1 - k0 + nw - 1) / nw;                  // the weight-streaming kernel's wave ranges
  const T* Ap = reinterpret_cast<const T*>(p.A);
  const gu4* Wp = (const gu4*)(p.W);

  if constexpr (NORM) {
    const int q16 = threadIdx.x & 15, grp = threadIdx.x >> 4;   // 16 groups of 16 lanes
    for (int r = grp; r < TILE_BM; r += 16) {
      const float rs = norm_row_scale(p, m0 + min(r, rows - 1), q16);
      if (q16 == 0) s_rs[r] = rs;
    }
  }

  // staging: A chunk c (row c/4, quarter c%4 of its KT values) goes to the
  // fragment slot of its m tile, XOR-swizzled within the quarter's 16 slots
  // (slot q*16 + (r ^ 2q)) so that the eight lanes of one 16-byte LDS write
  // pass (two rows x four quarters) hit distinct banks; the reader undoes the
  // swizzle.  W chunk c is lane c%64 of strip c/64.
  u32x4_t* sa = reinterpret_cast<u32x4_t*>(lds);             // [buffer][8 m tiles][64]
  u32x4_t* sw = sa + 2 * 512;                                 // [buffer][BS strips][64]
  // From the matrix-core-order copy (p.Af) chunk c is lane c%64 of the 1 KB
  // tile of m tile c/64: contiguous loads and LDS slots, no swizzle needed
  // (rows past M in the last 16-row tile are loaded and never stored).
  const bool af = p.Af != nullptr;
  const gu4* asrc[2];
  const gu4* wsrc[NWC];
  int adst[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (af) {
      const int mtg = min(m0 / 16 + (c >> 6), (p.M + 15) / 16 - 1);
      asrc[i] = (const gu4*)(p.Af) + (size_t)mtg * p.ktiles * 64 + (c & 63);
      adst[i] = c;
    } else {
      const int r = c >> 2, q = c & 3;
      asrc[i] = (const gu4*)(Ap + (size_t)(m0 + min(r, rows - 1)) * p.lda + q * KL);   // clamped rows are not stored
      adst[i] = (r >> 4) * 64 + q * 16 + ((r & 15) ^ (2 * q));
    }
  }
#pragma unroll
  for (int i = 0; i < NWC; ++i) {
    const int c = threadIdx.x + 256 * i;
    wsrc[i] = Wp + (size_t)min(nt0 + (c >> 6), p.ntiles - 1) * p.ktiles * 64 + (c & 63);   // clamped strips: not stored
  }
  constexpr int AST = KT * (int)sizeof(T) / 16;              // 16-byte chunks per k tile along an A row
  const int ast = af ? 64 : AST;
  u32x4_t ra[D][2], rw[D][NWC];                               // register slots
  auto load = [&](int slot, int kt) {                         // clamped: a load past the end is never used
    kt = min(kt, k1 - 1);
#pragma unroll
    for (int i = 0; i < 2; ++i) ra[slot][i] = asrc[i][(size_t)kt * ast];
#pragma unroll
    for (int i = 0; i < NWC; ++i)
      rw[slot][i] = NTW ? __builtin_nontemporal_load(&wsrc[i][(size_t)kt * 64]) : wsrc[i][(size_t)kt * 64];
  };
  auto store = [&](int slot, int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) sa[buf * 512 + adst[i]] = ra[slot][i];
#pragma unroll
    for (int i = 0; i < NWC; ++i) sw[buf * BS * 64 + threadIdx.x + 256 * i] = rw[slot][i];
  };

  f32x4_t acc[4][WS], tot[4][WS];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < WS; ++j) acc[i][j] = tot[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  int folds = 0;
  auto fold = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WS; ++j) {
#pragma unroll
        for (int r = 0; r < 4; ++r) tot[i][j][r] += acc[i][j][r];
        acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
    ++folds;
  };
  auto compute = [&](int buf) {
    u32x4_t a[4], b[WS];
    const int aslot = af ? lane : (lane & 48) | ((lane & 15) ^ (2 * (lane >> 4)));   // fragment lane -> slot
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = sa[buf * 512 + (wm * 4 + i) * 64 + aslot];
#pragma unroll
    for (int j = 0; j < WS; ++j) b[j] = sw[buf * BS * 64 + (wn * WS + j) * 64 + lane];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WS; ++j) acc[i][j] = mma_frag(T(), a[i], b[j], acc[i][j]);
  };
  // k tile t sits in LDS buffer (t - k0) & 1 and, before that, in register
  // slot (t - k0) % D; step t stores t + 1, loads t + D, multiplies t
  auto step = [&](int t, int j) {
    store((j + 1) % D, ((t - k0) & 1) ^ 1);
    load(j, t + D);
    compute((t - k0) & 1);
    if ((t - k0 + 1) % kper == 0 || t + 1 == k1) fold();     // end of a range
    __syncthreads();
  };

  if (k0 < k1) {
#pragma unroll
    for (int j = 0; j < D; ++j) load(j, k0 + j);
    store(0, 0);
  }
  __syncthreads();
  int kt = k0;
  for (; kt + D <= k1; kt += D) {                             // uniform
#pragma unroll
    for (int j = 0; j < D; ++j) step(kt + j, j);
  }
#pragma unroll
  for (int j = 0; j < D; ++j)                                 // the last k1 - kt < D tiles
    if (kt + j < k1) step(kt + j, j);
  while (folds < nw) fold();                                  // empty ranges add +0, as their waves do
  __syncthreads();                                            // staging buffers free for the C tile

  // C tile to LDS (the staging buffers are free), then the epilogue
  float* ct = lds;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < WS; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        ct[(wm * 64 + i * 16 + 4 * (lane >> 4) + r) * CW + (wn * WS + j) * 16 + (lane & 15)] = tot[i][j][r];
  __syncthreads();
  const int ncols = nvalid * 16;
  const int colbase = p.col0 + nt0 * 16;
  if constexpr (EPI == EPI_ARGMAX) {
    for (int e = threadIdx.x; e < rows * ncols; e += blockDim.x) {
      const int m = e / ncols, n = e - m * ncols;
      float v = ct[m * CW + n];
      if constexpr (NORM) ct[m * CW + n] = v = v * s_rs[m];
      if (p.logits) p.logits[(size_t)(m0 + m) * p.ldl + colbase + n] = v;
    }
    __syncthreads();
    // one key per row and group of two strips, as the weight-streaming kernel's workgroups
    const int ngrp = (nvalid + 1) / 2;
    for (int e = threadIdx.x; e < rows * ngrp; e += blockDim.x) {
      const int m = e / ngrp, gi = e - m * ngrp;
      const int c0 = gi * 32, c1 = min(ncols, c0 + 32);
      float best = ct[m * CW + c0];
      int bi = c0;
      for (int n = c0 + 1; n < c1; ++n) {
        const float v = ct[m * CW + n];
        if (v > best) { best = v; bi = n; }
      }
      p.amax[(size_t)(nt0 / 2 + gi) * p.amax_ld + m0 + m] = argmax_key(best, colbase + bi);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int half = ncols / 2;
    const int obase = (p.col0 + nt0 * 16) / 2;
    for (int e = threadIdx.x; e < rows * half; e += blockDim.x) {
      const int m = e / half, c = e - m * half;
      const int strip = c >> 3, cc = c & 7;
      float gt = ct[m * CW + strip * 16 + cc];
      float up = ct[m * CW + strip * 16 + 8 + cc];
      if constexpr (NORM) {
        gt *= s_rs[m];
        up *= s_rs[m];
      }
      const float y = silu(gt) * up;
      TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)(m0 + m) * p.ldy + obase + c, y);
      frag_st<T>(p.yf, m0 + m, obase + c, y);
    }
  } else {
    for (int e = threadIdx.x; e < rows * ncols; e += blockDim.x) {
      const int m = e / ncols, n = e - m * ncols;
      const int col = colbase + n;
      const size_t gm = (size_t)(m0 + m);
      float v = ct[m * CW + n];
      if constexpr (NORM) v *= s_rs[m];
      if constexpr (EPI == EPI_STORE_T) {
        TT<T>::st(reinterpret_cast<T*>(p.Y), gm * p.ldy + col, v);
      } else if constexpr (EPI == EPI_STORE_F32) {
        reinterpret_cast<float*>(p.Y)[(size_t)h * p.y_part + gm * p.ldy + col] = v;
      } else if constexpr (EPI == EPI_RESID) {
        v = TT<T>::rnd(v + TT<T>::ld(reinterpret_cast<const T*>(p.R), gm * p.ldr + col));
        TT<T>::st(reinterpret_cast<T*>(p.Y), gm * p.ldy + col, v);
        if (p.Y2) TT<T>::st(reinterpret_cast<T*>(p.Y2), gm * p.ldy2 + col, v);
        frag_st<T>(p.yf, (int)gm, col, v);
        frag_st<T>(p.y2f, (int)gm, col, v);
        ct[m * CW + n] = v;
      } else if constexpr (EPI == EPI_BIAS_SILU) {
        v += TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
        TT<T>::st(reinterpret_cast<T*>(p.Y), gm * p.ldy + col, silu(v));
        frag_st<T>(p.yf, (int)gm, col, silu(v));
      } else if constexpr (EPI == EPI_BIAS_F32) {
        v += TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
        reinterpret_cast<float*>(p.Y)[gm * p.ldy + col] = v;
      }
    }
    if constexpr (EPI == EPI_RESID) {
      if (p.ssq_out) {
        __syncthreads();
        for (int e = threadIdx.x; e < rows * nvalid; e += blockDim.x) {
          const int m = e / nvalid, j = e - m * nvalid;
          float sq = 0.f;
#pragma unroll
          for (int c = 0; c < 16; ++c) {
            const float v = ct[m * CW + j * 16 + c];
            sq += v * v;
          }
          p.ssq_out[(size_t)(m0 + m) * p.ssq_out_ld + nt0 + j] = sq;
        }
      }
    }
  }
}

template <typename T, int EPI, bool NORM, int BS, bool NTW>
static hipError_t launch_tile_bs(const GemmParams& p, const GemmShape& sh, int ks, int mt, hipStream_t st) {
  const int units = (p.ntiles + BS - 1) / BS * ks;
  const int blocks = (units + 7) / 8 * 8 * mt;
  // the C tile needs more than the default dynamic LDS; set once per
  // instantiation (thread-safe static initialisation)
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&gemm_tile_kernel<T, EPI, NORM, BS, NTW>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)TILE_LDS);
  if (attr != hipSuccess) return attr;
  const size_t lds = (size_t)TILE_BM * (BS * 16 + 4) * sizeof(float);
  hipLaunchKernelGGL((gemm_tile_kernel<T, EPI, NORM, BS, NTW>), dim3(blocks), dim3(256), lds, st, p, sh.waves, mt,
                     units);
  return hipGetLastError();
}

// Tile width from (N, M): 8 strips unless that leaves fewer workgroups than
// compute units.  The arithmetic of an output element does not depend on it.
template <typename T, int EPI, bool NORM>
static hipError_t launch_tile(const GemmParams& p, const GemmShape& sh, int ks, hipStream_t st) {
  const int mt = (p.M + TILE_BM - 1) / TILE_BM;
  const int wide = (p.ntiles + TILE_BS - 1) / TILE_BS * ks * mt;
  if (mt == 1) {
    if (wide < 256) return launch_tile_bs<T, EPI, NORM, 4, true>(p, sh, ks, mt, st);
    return launch_tile_bs<T, EPI, NORM, 8, true>(p, sh, ks, mt, st);
  }
  if (wide < 256) return launch_tile_bs<T, EPI, NORM, 4, false>(p, sh, ks, mt, st);
  return launch_tile_bs<T, EPI, NORM, 8, false>(p, sh, ks, mt, st);
}

// Launch shape from (N, K) (and the K parts) only, never from M.  Wide weights (>= 1024
// strips) and the LM head take two 16-column strips per workgroup (the A
// fragments are reused across both); narrower ones take one so that enough
// workgroups exist.  The wave count (the K split) is the smallest power of
// two in 2..8 that puts at least 1024 waves in flight while leaving each wave
// at least 8 k tiles.  Chosen from a sweep over the 8B-shape projections at
// M = 16 with weights streamed from HBM.
GemmShape gemm_shape(int ntiles, int ktiles, int epi, int ksplit) {
  GemmShape s;
  s.ng = (epi == EPI_ARGMAX || ntiles >= 1024) ? 2 : 1;
  s.groups = (ntiles + s.ng - 1) / s.ng * ksplit;   // workgroups: strip groups x K parts
  const int kpart = (ktiles + ksplit - 1) / ksplit;
  int waves = 2;
  while (waves < 8 && (long long)s.groups * waves < 1024 && kpart / (2 * waves) >= 8) waves *= 2;
  s.waves = waves;
  return s;
}

// K parts for a projection whose consumer adds fp32 partial outputs: two when
// that spreads the strip groups more evenly over the compute units (every
// unit streams weights at about the same rate, so the slowest unit sets the
// time), one otherwise.  Depends only on (N, K) and the device.
int gemm_ksplit(int ntiles, int ktiles, int cus) {
  const GemmShape s = gemm_shape(ntiles, ktiles, EPI_STORE_F32, 1);
  if (cus < 1 || ktiles < 8) return 1;
  auto imbalance = [&](int ks) {
    const double per = (double)s.groups * ks / cus;
    return std::ceil(per) / per;
  };
  return imbalance(2) < imbalance(1) - 1e-9 ? 2 : 1;
}

template <typename T, int NG, int EPI, bool NORM>
static hipError_t launch_mtn(const GemmParams& p, const GemmShape& sh, hipStream_t st) {
  const int mt = (p.M + 15) / 16;
  const int cw = NG * 16 + 1;
  auto go = [&](auto kern, int MTv) {
    const size_t lds = ((size_t)sh.waves * NG * 256 + (size_t)MTv * 16 * cw) * sizeof(float);
    if (lds > 65536) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(kern, dim3(sh.groups), dim3(sh.waves * 64), lds, st, p);
    return hipGetLastError();
  };
  // the tiled kernel for more than 128 rows, and from 64 rows for weights wide
  // enough to give it a workgroup per compute unit or so (measured crossover:
  // the weight-streaming kernel re-reads A from L2 once per strip group)
  const int ks = p.ksplit > 1 ? p.ksplit : 1;
  const bool tile = mt > 8 || (mt >= 4 && (p.ntiles + TILE_BS - 1) / TILE_BS * ks >= 96);
  if (tile) return launch_tile<T, EPI, NORM>(p, sh, ks, st);
  if (mt <= 1) return go(gemm_kernel<T, NG, 1, EPI, NORM>, 1);
  if (mt <= 2) return go(gemm_kernel<T, NG, 2, EPI, NORM>, 2);
  if (mt <= 4) return go(gemm_kernel<T, NG, 4, EPI, NORM>, 4);
  return go(gemm_kernel<T, NG, 8, EPI, NORM>, 8);
}

// The RMSNorm row scale is instantiated only for the projections that follow a norm.
template <int EPI> struct HasNorm {
  static constexpr bool value = EPI == EPI_STORE_T || EPI == EPI_STORE_F32 || EPI == EPI_SWIGLU || EPI == EPI_ARGMAX;
};

template <typename T, int NG, int EPI>
static hipError_t launch_mt(const GemmParams& p, const GemmShape& sh, hipStream_t st) {
  if constexpr (HasNorm<EPI>::value) {
    if (p.norm) return launch_mtn<T, NG, EPI, true>(p, sh, st);
  } else {
    if (p.norm) return hipErrorInvalidValue;
  }
  return launch_mtn<T, NG, EPI, false>(p, sh, st);
}

template <typename T, int EPI>
static hipError_t launch_ng(const GemmParams& p, const GemmShape& sh, hipStream_t st) {
  return sh.ng == 2 ? launch_mt<T, 2, EPI>(p, sh, st) : launch_mt<T, 1, EPI>(p, sh, st);
}

// Residual epilogue of the K-split path: one thread per (row, 16-column
// strip) adds the fp32 parts in part order from +0 -- the order in which the
// weight-streaming kernel adds its waves' ranges, so each row is bit-identical
// to that kernel's -- then applies its EPI_RESID epilogue: rnd(sum + R) to Y
// (and Y2) and the strip's sum of squares of the stored values.
// The KS parts (KS > 0: all loads in flight at once; KS = 0: a loop over ks)
// of a thread's 16 columns, summed in part order from +0.
template <int KS>
__device__ inline void sum_parts16(const float* part, size_t part_stride, int ks, size_t off, float (&s)[16]) {
#pragma unroll
  for (int c = 0; c < 16; ++c) s[c] = 0.f;
  if constexpr (KS > 0) {
    float v[KS][16];
#pragma unroll
    for (int h = 0; h < KS; ++h) Row16<float>::load(part + h * part_stride + off, v[h]);
#pragma unroll
    for (int h = 0; h < KS; ++h)
#pragma unroll
      for (int c = 0; c < 16; ++c) s[c] += v[h][c];
  } else {
    for (int h = 0; h < ks; ++h) {
      float v[16];
      Row16<float>::load(part + h * part_stride + off, v);
#pragma unroll
      for (int c = 0; c < 16; ++c) s[c] += v[c];
    }
  }
}

template <typename T, int KS>
__global__ void __launch_bounds__(256) resid_reduce_kernel(const float* part, size_t part_stride, int ks, int M,
                                                           int N, const T* R, int ldr, T* Y, int ldy, T* Y2, int ldy2,
                                                           float* ssq_out, int ssq_ld, int strip0, FragOut yf,
                                                           FragOut y2f) {
  const int nstrips = N / 16;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= M * nstrips) return;
  const int m = e / nstrips, j = e - m * nstrips;
  float r[16], s[16];
  Row16<T>::load(R + (size_t)m * ldr + j * 16, r);
  sum_parts16<KS>(part, part_stride, ks, (size_t)m * N + j * 16, s);
  float sq = 0.f;
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    s[c] = TT<T>::rnd(s[c] + r[c]);
    sq += s[c] * s[c];
  }
  Row16<T>::store(Y + (size_t)m * ldy + j * 16, s);
  if (Y2) Row16<T>::store(Y2 + (size_t)m * ldy2 + j * 16, s);
  frag_st_run<T>(yf, m, j * 16, s, 16);
  frag_st_run<T>(y2f, m, j * 16, s, 16);
  if (ssq_out) ssq_out[(size_t)m * ssq_ld + strip0 + j] = sq;
}

int split_parts(int epi, int ntiles, int ktiles) { return gemm_shape(ntiles, ktiles, epi, 1).waves; }

// SwiGLU epilogue of the K-split path: one thread per (row, 16-column strip of
// 8 gate + 8 up columns), parts added in part order from +0, then the
// weight-streaming kernel's epilogue (row scale, silu(gate) * up, rounding).
// Every 16-lane group computes the row scale (the same value) before any lane
// leaves.
template <typename T, bool NORM, int KS>
__global__ void __launch_bounds__(256) swiglu_reduce_kernel(GemmParams p, const float* part, size_t part_stride,
                                                            int ks, int N) {
  const int m = blockIdx.y;
  float rs = 1.f;
  if constexpr (NORM) rs = norm_row_scale(p, m, threadIdx.x & 15);
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= N / 16) return;
  float s[16];
  sum_parts16<KS>(part, part_stride, ks, (size_t)m * N + j * 16, s);
  float y[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    float gt = s[c], up = s[8 + c];
    if constexpr (NORM) {
      gt *= rs;
      up *= rs;
    }
    y[c] = silu(gt) * up;
    TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + j * 8 + c, y[c]);
  }
  frag_st_run<T>(p.yf, m, j * 8, y, 8);
}

// The gate/up projection between SPLIT_MIN_ROWS and SWIGLU_SPLIT_MAX_ROWS
// rows, when K parts (the weight-streaming kernel's ranges) lower the bytes
// the busiest compute unit streams by a sixth or more: for the 8B shape at
// 64-256 rows the single-part launch puts two 4-strip workgroups on half the
// units, the split one two 8-strip half-K workgroups on every unit (a third
// fewer bytes each, against the parts' round trip).
template <typename T>
static hipError_t launch_swiglu_split(const GemmParams& p, hipStream_t st) {
  const int ks = split_parts(EPI_SWIGLU, p.ntiles, p.ktiles);
  GemmParams q = p;   // the parts read A (or its matrix-core-order copy); the reduce writes the copies
  q.yf = q.y2f = FragOut{nullptr, 0, 0};
  q.ksplit = ks;
  q.norm = 0;
  q.Y = p.part_ws;
  q.ldy = p.ntiles * 16;
  q.y_part = (size_t)p.M * q.ldy;
  q.col0 = 0;
  GemmShape sh{};
  sh.waves = 1;   // one K range per part
  hipError_t e = launch_tile<T, EPI_STORE_F32, false>(q, sh, ks, st);
  if (e != hipSuccess) return e;
  const dim3 grid((p.ntiles + 255) / 256, p.M);
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(256), 0, st, p, p.part_ws, q.y_part, ks, q.ldy);
    return hipGetLastError();
  };
  // the part count as a template argument where it is one of the wave counts, so all loads are in flight at once
  if (p.norm) {
    if (ks == 2) return go(swiglu_reduce_kernel<T, true, 2>);
    if (ks == 4) return go(swiglu_reduce_kernel<T, true, 4>);
    if (ks == 8) return go(swiglu_reduce_kernel<T, true, 8>);
    return go(swiglu_reduce_kernel<T, true, 0>);
  }
  if (ks == 2) return go(swiglu_reduce_kernel<T, false, 2>);
  if (ks == 4) return go(swiglu_reduce_kernel<T, false, 4>);
  if (ks == 8) return go(swiglu_reduce_kernel<T, false, 8>);
  return go(swiglu_reduce_kernel<T, false, 0>);
}

// A narrow weight (O, down) at more than SPLIT_MIN_ROWS rows: the weight-
// streaming kernel would re-read the whole A block from L2 for every strip
// group, so the tiled kernel computes each of the weight-streaming kernel's K
// ranges as a part of its own (fp32 partial sums, no row scale), and the
// reduce kernel adds them and applies the residual epilogue.
template <typename T>
static hipError_t launch_resid_split(const GemmParams& p, hipStream_t st) {
  const int ks = split_parts(EPI_RESID, p.ntiles, p.ktiles);
  GemmParams q = p;   // the parts read A (or its matrix-core-order copy); the reduce writes the copies
  q.yf = q.y2f = FragOut{nullptr, 0, 0};
  q.ksplit = ks;
  q.Y = p.part_ws;
  q.ldy = p.ntiles * 16;
  q.y_part = (size_t)p.M * q.ldy;
  q.R = nullptr;
  q.Y2 = nullptr;
  q.ssq_out = nullptr;
  q.col0 = 0;
  GemmShape sh{};
  sh.waves = 1;   // one K range per part
  hipError_t e = launch_tile<T, EPI_STORE_F32, false>(q, sh, ks, st);
  if (e != hipSuccess) return e;
  const int items = p.M * p.ntiles;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3((items + 255) / 256), dim3(256), 0, st, p.part_ws, q.y_part, ks, p.M, q.ldy,
                       reinterpret_cast<const T*>(p.R), p.ldr, reinterpret_cast<T*>(p.Y), p.ldy,
                       reinterpret_cast<T*>(p.Y2), p.ldy2, p.ssq_out, p.ssq_out_ld, 0, p.yf, p.y2f);
    return hipGetLastError();
  };
  if (ks == 2) return go(resid_reduce_kernel<T, 2>);
  if (ks == 4) return go(resid_reduce_kernel<T, 4>);
  if (ks == 8) return go(resid_reduce_kernel<T, 8>);
  return go(resid_reduce_kernel<T, 0>);
}

// Range split of the narrow drafter-side projections (W_c, relay MLP,
// drafter context K/V: plain, fp32, bias + SiLU and bias epilogues) between
// SPLIT_MIN_ROWS + 1 and SWIGLU_SPLIT_MAX_ROWS rows, where a tiled launch
// would have too few workgroups and the weight-streaming kernel re-reads the
// whole A block for every strip group: the tiled kernel computes each of the
// weight-streaming kernel's wave ranges as a part of its own, and this kernel
// folds the parts in range order from +0 -- that kernel's wave fold -- and
// applies its epilogue.  One workgroup row per output row (every 16-lane group
// computes the row scale); four columns per thread.
template <typename T, int EPI, bool NORM, int KS>
__global__ void __launch_bounds__(256) range_reduce_kernel(GemmParams p, const float* part, size_t part_stride,
                                                           int nw, int N) {
  const int m = blockIdx.y;
  float rs = 1.f;
  if constexpr (NORM) rs = norm_row_scale(p, m, threadIdx.x & 15);
  const int c4 = blockIdx.x * 256 + threadIdx.x;
  if (c4 >= N / 4) return;
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  const float* src = part + (size_t)m * N + 4 * c4;
  if constexpr (KS > 0) {   // all parts' loads in flight at once, summed in part order
    float4 v[KS];
#pragma unroll
    for (int w = 0; w < KS; ++w) v[w] = *reinterpret_cast<const float4*>(src + (size_t)w * part_stride);
#pragma unroll
    for (int w = 0; w < KS; ++w) {
      s[0] += v[w].x;
      s[1] += v[w].y;
      s[2] += v[w].z;
      s[3] += v[w].w;
    }
  } else {
    for (int w = 0; w < nw; ++w) {
      const float4 v = *reinterpret_cast<const float4*>(src + (size_t)w * part_stride);
      s[0] += v.x;
      s[1] += v.y;
      s[2] += v.z;
      s[3] += v.w;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int col = 4 * c4 + i;
    float v = s[i];
    if constexpr (NORM) v *= rs;
    if constexpr (EPI == EPI_STORE_T) {
      TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, v);
    } else if constexpr (EPI == EPI_STORE_F32) {
      reinterpret_cast<float*>(p.Y)[(size_t)m * p.ldy + col] = v;
    } else if constexpr (EPI == EPI_BIAS_SILU) {
      v += TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
      TT<T>::st(reinterpret_cast<T*>(p.Y), (size_t)m * p.ldy + col, silu(v));
      frag_st<T>(p.yf, m, col, silu(v));
    } else if constexpr (EPI == EPI_BIAS_F32) {
      v += TT<T>::ld(reinterpret_cast<const T*>(p.bias), col);
      reinterpret_cast<float*>(p.Y)[(size_t)m * p.ldy + col] = v;
    }
  }
}

bool range_split_applies(int epi, int M, int ntiles, int ksplit) {
  return (epi == EPI_STORE_T || epi == EPI_STORE_F32 || epi == EPI_BIAS_SILU || epi == EPI_BIAS_F32) &&
         ksplit <= 1 && M > SPLIT_MIN_ROWS && M <= SWIGLU_SPLIT_MAX_ROWS && (ntiles + TILE_BS - 1) / TILE_BS < 96;
}

template <typename T, int EPI, bool NORM>
static hipError_t launch_range_reduce(const GemmParams& p, size_t part_stride, int nw, int N, hipStream_t st) {
  const dim3 grid((N / 4 + 255) / 256, p.M);
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(256), 0, st, p, p.part_ws, part_stride, nw, N);
    return hipGetLastError();
  };
  if (nw == 2) return go(range_reduce_kernel<T, EPI, NORM, 2>);
  if (nw == 4) return go(range_reduce_kernel<T, EPI, NORM, 4>);
  if (nw == 8) return go(range_reduce_kernel<T, EPI, NORM, 8>);
  return go(range_reduce_kernel<T, EPI, NORM, 0>);
}

template <typename T>
static hipError_t launch_range_split(int epi, const GemmParams& p, hipStream_t st) {
  const int nw = split_parts(epi, p.ntiles, p.ktiles);
  GemmParams q = p;   // the parts read A (or its matrix-core-order copy); the reduce writes the copies
  q.yf = q.y2f = FragOut{nullptr, 0, 0};
  q.ksplit = nw;
  q.norm = 0;
  q.Y = p.part_ws;
  q.ldy = p.ntiles * 16;
  q.y_part = (size_t)p.M * q.ldy;
  q.R = nullptr;
  q.Y2 = nullptr;
  q.ssq_out = nullptr;
  q.col0 = 0;
  GemmShape sh{};
  sh.waves = 1;   // one range per part
  hipError_t e = launch_tile<T, EPI_STORE_F32, false>(q, sh, nw, st);
  if (e != hipSuccess) return e;
  const bool n = p.norm != 0;
  switch (epi) {
    case EPI_STORE_T:
      return n ? launch_range_reduce<T, EPI_STORE_T, true>(p, q.y_part, nw, q.ldy, st)
               : launch_range_reduce<T, EPI_STORE_T, false>(p, q.y_part, nw, q.ldy, st);
    case EPI_STORE_F32:
      return n ? launch_range_reduce<T, EPI_STORE_F32, true>(p, q.y_part, nw, q.ldy, st)
               : launch_range_reduce<T, EPI_STORE_F32, false>(p, q.y_part, nw, q.ldy, st);
    case EPI_BIAS_SILU:
      return n ? hipErrorInvalidValue : launch_range_reduce<T, EPI_BIAS_SILU, false>(p, q.y_part, nw, q.ldy, st);
    case EPI_BIAS_F32:
      return n ? hipErrorInvalidValue : launch_range_reduce<T, EPI_BIAS_F32, false>(p, q.y_part, nw, q.ldy, st);
  }
  return hipErrorInvalidValue;
}

// Bytes the busiest compute unit streams in a tiled launch with ks K parts:
// workgroups per unit (rounded up) x (A and W bytes of one workgroup's k
// tiles), with the strip count launch_tile would pick.
static double tile_unit_bytes(int ntiles, int ktiles, int M, int ks, int cus, int kt_bytes) {
  const int mt = (M + TILE_BM - 1) / TILE_BM;
  const int bs = (ntiles + TILE_BS - 1) / TILE_BS * ks * mt < 256 ? 4 : 8;
  const long long wgs = (long long)((ntiles + bs - 1) / bs) * ks * mt;
  const int kpart = (ktiles + ks - 1) / ks;
  const double per_wg = (double)kpart * (TILE_BM + bs * 16) * kt_bytes;
  return (double)((wgs + cus - 1) / cus) * per_wg;
}

template <typename T>
static bool swiglu_split_pays(const GemmParams& p) {
  if (p.cus < 1) return false;
  const int ks = split_parts(EPI_SWIGLU, p.ntiles, p.ktiles);
  if (ks < 2) return false;
  const int ktb = TT<T>::KT * (int)sizeof(T);   // bytes of one row's k tile
  return tile_unit_bytes(p.ntiles, p.ktiles, p.M, ks, p.cus, ktb) <
         (5.0 / 6.0) * tile_unit_bytes(p.ntiles, p.ktiles, p.M, 1, p.cus, ktb);
}

template <typename T>
static hipError_t launch_t(int epi, const GemmParams& p, hipStream_t st) {
  const int ks = p.ksplit > 1 ? p.ksplit : 1;
  if (epi == EPI_RESID && p.M > SPLIT_MIN_ROWS && p.part_ws && !p.norm && p.col0 == 0)
    return launch_resid_split<T>(p, st);
  if (epi == EPI_SWIGLU && p.M > SPLIT_MIN_ROWS && p.M <= SWIGLU_SPLIT_MAX_ROWS && p.part_ws && p.col0 == 0 &&
      swiglu_split_pays<T>(p))
    return launch_swiglu_split<T>(p, st);
  if (p.part_ws && p.col0 == 0 && range_split_applies(epi, p.M, p.ntiles, ks)) return launch_range_split<T>(epi, p, st);
  if (ks > 1 && epi != EPI_STORE_F32) return hipErrorInvalidValue;   // only partial fp32 outputs are split
  const GemmShape sh = gemm_shape(p.ntiles, p.ktiles, epi, ks);
  switch (epi) {
    case EPI_STORE_T: return launch_ng<T, EPI_STORE_T>(p, sh, st);
    case EPI_STORE_F32: return launch_ng<T, EPI_STORE_F32>(p, sh, st);
    case EPI_RESID: return launch_ng<T, EPI_RESID>(p, sh, st);
    case EPI_SWIGLU: return launch_ng<T, EPI_SWIGLU>(p, sh, st);
    case EPI_BIAS_SILU: return launch_ng<T, EPI_BIAS_SILU>(p, sh, st);
    case EPI_BIAS_F32: return launch_ng<T, EPI_BIAS_F32>(p, sh, st);
    case EPI_ARGMAX: return launch_mt<T, 2, EPI_ARGMAX>(p, sh, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(bool bf16, int epi, const GemmParams& p, hipStream_t st) {
  if (p.M <= 0 || p.ntiles <= 0 || p.ktiles <= 0) return hipSuccess;
  return bf16 ? launch_t<dflow::bf16>(epi, p, st) : launch_t<float>(epi, p, st);
}

// ------------------------------------------------------------------ packing
// out tile (nt, kt) lane l element e <- W[src_row(nt, l%16)][kt*KT + (l/16)*KL + e] * gain[col]
// gate_up: W is [2F, K] = [gate; up]; packed strip i holds gate rows 8i..8i+7
// followed by up rows 8i..8i+7, so one strip yields 8 SwiGLU outputs.  The
// optional column gain (the RMSNorm gain of the rows this weight multiplies)
// is applied in fp32 and rounded once to the storage type.
template <typename T>
__global__ void pack_kernel(const T* __restrict__ W, int N, int K, int gate_up, const T* __restrict__ gain,
                            T* __restrict__ out) {
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
    const int r16 = l & 15;
    size_t row = (size_t)nt * 16 + r16;
    if (gate_up) row = (r16 < 8) ? (size_t)nt * 8 + r16 : (size_t)N / 2 + (size_t)nt * 8 + (r16 - 8);
    const size_t col = (size_t)kt * KT + (l >> 4) * KL + e;
    if (gain)
      TT<T>::st(out, o, TT<T>::ld(W, row * K + col) * TT<T>::ld(gain, col));
    else
      out[o] = W[row * K + col];
  }
}

hipError_t launch_pack(bool bf16, const void* w, int N, int K, int gate_up, const void* col_gain, void* out,
                       hipStream_t s) {
  const int threads = 256;
  const size_t total = (size_t)N * K;
  int blocks = (int)((total + threads - 1) / threads);
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    hipLaunchKernelGGL(pack_kernel<dflow::bf16>, dim3(blocks), dim3(threads), 0, s, (const dflow::bf16*)w, N, K,
                       gate_up, (const dflow::bf16*)col_gain, (dflow::bf16*)out);
  else
    hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(threads), 0, s, (const float*)w, N, K, gate_up,
                       (const float*)col_gain, (float*)out);
  return hipGetLastError();
}

}  // namespace dflow
