// Internal launch interface of the weight-streaming and tiled GEMMs.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dflow {

// Matrix-core-order copy of an activation block (afrag_off): written by the
// producer of a projection's A operand besides its row-major output, read by
// the projection in whole 16-row tiles (buffers hold the launch's rows rounded
// up to 16).  p null: no copy.
struct FragOut {
  void* p;
  int ktiles;   // K / KT of the consuming projection
  int c0;       // first column of the producer's output within that K
};

enum Epi : int {
  EPI_STORE_T = 0,   // Y = acc                       (storage type)
  EPI_STORE_F32,     // Y = acc                       (fp32)
  EPI_RESID,         // Y = R + acc; optional copy Y2 (storage type)
  EPI_SWIGLU,        // Y = silu(gate) * up           (gate/up tiles interleaved)
  EPI_BIAS_SILU,     // Y = silu(acc + bias)          (storage type)
  EPI_BIAS_F32,      // Y = acc + bias                (fp32)
  EPI_ARGMAX,        // per-row best (value, lowest index) over the group's columns
  EPI_COUNT
};

struct GemmParams {
  const void* A; int lda;           // activations [M, lda], storage type
  const void* W;                    // packed weight tiles of this column range
  int M, ntiles, ktiles;            // ntiles = N/16 of the range, ktiles = K/KT
  void* Y; int ldy;
  const void* R; int ldr;
  void* Y2; int ldy2;
  const void* bias;
  uint64_t* amax; int amax_ld;      // [workgroup][amax_ld] argmax keys
  float* logits; int ldl;           // optional fp32 logits
  int col0;                         // first output column of this range (argmax indices, bias)
  // RMSNorm row scale (norm = 1): A rows are the raw x, the norm gain is
  // folded into W, and every output of row m is scaled by rs[m] =
  // (sum_c ssq[m * ssq_ld + c] / (16 ssq_parts) + eps)^(-1/2).  Rows are
  // padded: ssq_ld >= max(256, ssq_parts) entries are readable.
  int norm;
  const float* ssq; int ssq_ld; int ssq_parts;
  float eps;
  // EPI_RESID: per-16-column-strip sums of squares of the stored rows, [m * ssq_out_ld + strip]
  float* ssq_out; int ssq_out_ld;
  // EPI_STORE_F32 only: K split into ksplit parts; part h writes its partial
  // sums at Y + h * y_part (floats), and the consumer adds the parts
  int ksplit; size_t y_part;
  // EPI_RESID above SPLIT_MIN_ROWS rows, EPI_SWIGLU from SPLIT_MIN_ROWS + 1
  // to SWIGLU_SPLIT_MAX_ROWS rows: fp32 scratch of split_parts(epi, ntiles,
  // ktiles) x M x N floats for the K-part partial sums; the narrow plain,
  // fp32 and bias projections under range_split_applies the same (null: no
  // split)
  float* part_ws;
  int cus;                          // compute units (0: unknown, no balance-driven split)
  // A read from its matrix-core-order copy (afrag_off; null: from A), and
  // copies of the outputs Y / Y2 written in that order for the next
  // projection (every path and epilogue that writes Y / Y2 honours them).
  const void* Af;
  FragOut yf, y2f;
};

constexpr int SPLIT_MIN_ROWS = 48, SWIGLU_SPLIT_MAX_ROWS = 256;

struct GemmShape { int ng; int waves; int groups; };
GemmShape gemm_shape(int ntiles, int ktiles, int epi, int ksplit = 1);
int gemm_ksplit(int ntiles, int ktiles, int cus);
// K parts of a split residual or SwiGLU GEMM (the weight-streaming kernel's
// wave count for (N, K), so every part is one of its K ranges)
int split_parts(int epi, int ntiles, int ktiles);
// Whether a plain, fp32, bias + SiLU or bias projection (no K parts) of M rows
// takes the range split: SPLIT_MIN_ROWS < M <= SWIGLU_SPLIT_MAX_ROWS and a
// weight too narrow for the tiled kernel's workgroup count; it needs
// split_parts(epi, ntiles, ktiles) x M x N floats of part_ws
bool range_split_applies(int epi, int M, int ntiles, int ksplit);
hipError_t launch_gemm(bool bf16, int epi, const GemmParams& p, hipStream_t s);
hipError_t launch_pack(bool bf16, const void* w, int N, int K, int gate_up, const void* col_gain, void* out,
                       hipStream_t s);

}  // namespace dflow
