// Speculative sampling at temperature T > 0 (gfx950 / CDNA4).
//
// The rule (speculative decoding of Leviathan, Kalman and Matias, cited in
// Sec. 1; Table 1 reports DFlow under it at T = 1): drafts d_i ~ q_i, the
// drafter's softmax(logits / T) at block row i; d_i is kept while
// u_i < p_{i-1}(d_i) / q_i(d_i), p_j the target's softmax(logits / T) at
// verify row j; at the first rejection (a < K) the token at block index a+1
// is drawn from the positive part of p_a - q_{a+1}; when all K drafts are
// kept the bonus is drawn from p_K.
//
// Randomness: Philox4x64-10 (Salmon et al., SC 2011) keyed by (seed, stream
// of the sequence); counter (t, block index, purpose, column / 4), output
// word column % 4; purposes 0 draft, 1 acceptance, 2 correction/bonus.  A
// word x gives u = ((x >> 41) + 1/2) 2^-23.  Draws use the Gumbel-max trick:
// argmax_v (w_v - log(-log u_v)), lowest index on ties (the argmax key of
// common.h), so a draw over V columns splits into independent column chunks
// whose maxima combine in any order.
//
// Arithmetic is fp32 with contraction off, in the order: z = logit * (1/T);
// lse = m + log(sum exp(z - m)) from per-chunk (max, sum) pairs;
// log p = z - lse; acceptance log u < log p - log q; correction weights
// log(exp(log p) - exp(log q)) where positive (all non-positive: drawn from z_p).
//
// Launch shapes: every kernel over logits takes one workgroup of 256 lanes per
// (1024-column chunk, row); a lane handles one group of four columns (one
// Philox block and one 16-byte load), so a Qwen3 vocabulary row spreads over
// 149 workgroups.  Chunk partials are folded by one wave per row or sequence.
#include <mutex>

#include "common.h"
#include "kernels.h"
#include "round_state.h"

#pragma clang fp contract(off)

namespace dflow {

namespace {

constexpr int CH = SAMP_CHUNK;            // columns per workgroup
constexpr int GPW = CH / 4;               // four-column groups per workgroup
constexpr uint64_t PH_M0 = 0xD2E7470EE14C6C93ull, PH_M1 = 0xCA5A826395121157ull;
constexpr uint64_t PH_W0 = 0x9E3779B97F4A7C15ull, PH_W1 = 0xBB67AE8584CAA73Bull;
constexpr uint32_t NEG_INF_ORD = 0x007FFFFFu;   // high word of argmax_key(-inf, .)

struct Words { uint64_t w[4]; };

__device__ inline Words philox(uint64_t k0, uint64_t k1, uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += PH_W0;
      k1 += PH_W1;
    }
    const uint64_t hi0 = __umul64hi(PH_M0, c0), lo0 = PH_M0 * c0;
    const uint64_t hi1 = __umul64hi(PH_M1, c2), lo1 = PH_M1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return Words{{c0, c1, c2, c3}};
}

__device__ inline float unif(uint64_t x) { return ((float)(uint32_t)(x >> 41) + 0.5f) * 0x1p-23f; }
__device__ inline float gumbel(uint64_t x) { return -logf(-logf(unif(x))); }

__device__ inline uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o, 64);
    v = w > v ? w : v;
  }
  return v;
}
__device__ inline float wave_max_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// workgroup max of a u64 key (four waves); every lane gets the result
__device__ inline uint64_t block_max_u64(uint64_t v, uint64_t* sh) {
  v = wave_max_u64(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t r = sh[0];
  for (int i = 1; i < 4; ++i) r = sh[i] > r ? sh[i] : r;
  return r;
}

struct SampP {
  float inv_t;
  uint64_t seed;
  const uint64_t* stream;   // [nseq]
  const int* pos;           // [nseq] anchor positions t
  int V, B, chunks;
};

// rows drawn by draw_kernel: row r is block index i = r % K + i0 of sequence
// s = r / K, logits row s * B + i, counter (t_s, i, purpose, column / 4)
struct DrawRows { int K, i0, purpose; };

// ---------------------------------------------------------------- drafts (and the first token)
// grid (chunk, row r): partial Gumbel-max key of one logits row over one chunk
__global__ void __launch_bounds__(256) draw_kernel(const float* dlog, SampP p, DrawRows dr, uint64_t* part) {
  __shared__ uint64_t sh[4];
  const int c = blockIdx.x, r = blockIdx.y;
  const int s = r / dr.K, i = r - s * dr.K + dr.i0;
  const float* row = dlog + (size_t)(s * p.B + i) * p.V;
  const uint64_t key1 = p.stream[s], t = (uint64_t)p.pos[s];
  const int g0 = c * GPW, g1 = min(p.V / 4, g0 + GPW);
  uint64_t best = 0;
  for (int g = g0 + threadIdx.x; g < g1; g += 256) {
    const float4 x = *(const float4*)(row + 4 * (size_t)g);
    const Words w = philox(p.seed, key1, t, (uint64_t)i, (uint64_t)dr.purpose, (uint64_t)g);
    const float xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float z = xs[j] * p.inv_t;
      const uint64_t k = argmax_key(z + gumbel(w.w[j]), 4 * g + j);
      best = k > best ? k : best;
    }
  }
  best = block_max_u64(best, sh);
  if (threadIdx.x == 0) part[(size_t)r * p.chunks + c] = best;
}

// one wave per drawn row: fold the chunk keys (lanes stride the chunks, then
// a wave max); out[r] = the token and, for drafts (K = B - 1, i0 = 1),
// block_out = [anchor, drafts]
__global__ void __launch_bounds__(256) draw_finish_kernel(const uint64_t* part, int rows, int chunks, int B,
                                                          const int* anchor, int* draft_tok, int* block_out) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= rows) return;
  uint64_t best = 0;
  for (int c = lane; c < chunks; c += 64) {
    const uint64_t k = part[(size_t)r * chunks + c];
    best = k > best ? k : best;
  }
  best = wave_max_u64(best);
  if (lane) return;
  const int v = argmax_key_index(best);
  if (draft_tok) draft_tok[r] = v;
  if (block_out) {
    const int K = B - 1, s = r / K, i = r - s * K + 1;
    block_out[(size_t)s * B + i] = v;
    if (i == 1) block_out[(size_t)s * B] = anchor[s];
  }
}

// ---------------------------------------------------------------- log-sum-exp partials
// grid (chunk, y): y < R target row y, else drafter row y - R (R = nseq * B);
// ml[(y * chunks + c) * 2 + {0, 1}] = (max z, sum exp(z - max z)) over the chunk
__global__ void __launch_bounds__(256) lse_part_kernel(const float* logits, const float* dlog, SampP p, int R,
                                                       float* ml) {
  __shared__ float sh[4];
  const int c = blockIdx.x, y = blockIdx.y;
  if (y >= R && (y - R) % p.B == 0) return;   // drafter row 0 (the anchor row) is not used
  const float* row = y < R ? logits + (size_t)y * p.V : dlog + (size_t)(y - R) * p.V;
  const int g0 = c * GPW, g1 = min(p.V / 4, g0 + GPW);
  float z[GPW / 256][4];
  float m = -INFINITY;
#pragma unroll
  for (int k = 0; k < GPW / 256; ++k) {
    const int g = g0 + threadIdx.x + 256 * k;
    float4 x = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    if (g < g1) x = *(const float4*)(row + 4 * (size_t)g);
    z[k][0] = x.x * p.inv_t;
    z[k][1] = x.y * p.inv_t;
    z[k][2] = x.z * p.inv_t;
    z[k][3] = x.w * p.inv_t;
    m = fmaxf(m, fmaxf(fmaxf(z[k][0], z[k][1]), fmaxf(z[k][2], z[k][3])));
  }
  m = wave_max_f(m);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3]));
  __syncthreads();
  float sum = 0.f;
  if (m != -INFINITY) {
#pragma unroll
    for (int k = 0; k < GPW / 256; ++k)
#pragma unroll
      for (int j = 0; j < 4; ++j) sum += expf(z[k][j] - m);
  }
  sum = wave_sum_f(sum);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    float* o = ml + ((size_t)y * p.chunks + c) * 2;
    o[0] = m;
    o[1] = (sh[0] + sh[1]) + (sh[2] + sh[3]);
  }
}

constexpr int FOLD_IT = 4;    // chunk partials per lane: vocabularies up to 64 * 4 * 1024 columns
constexpr int FOLD_ROWS = 8;  // rows a wave folds at once (their loads issue together)

// log-sum-exp of up to FOLD_ROWS rows (row offsets rowoff[j], j < n) from
// their chunk partials (max, sum): the row max by a lane-local max over chunks
// lane + 64 k and a shuffle tree, then the sum of the partial sums rescaled to
// it, lane-local in k order and by a shuffle tree; lse[j]
__device__ inline void wave_fold_rows(const float* ml, int chunks, const int* rowoff, int n, float* lse) {
  const int lane = threadIdx.x & 63;
  float2 v[FOLD_ROWS][FOLD_IT];
#pragma unroll
  for (int j = 0; j < FOLD_ROWS; ++j)
#pragma unroll
    for (int k = 0; k < FOLD_IT; ++k) {
      const int c = lane + 64 * k;
      v[j][k] = (j < n && c < chunks) ? *(const float2*)(ml + ((size_t)rowoff[j] * chunks + c) * 2)
                                      : make_float2(-INFINITY, 0.f);
    }
#pragma unroll
  for (int j = 0; j < FOLD_ROWS; ++j) {
    float m = v[j][0].x;
#pragma unroll
    for (int k = 1; k < FOLD_IT; ++k) m = fmaxf(m, v[j][k].x);
    m = wave_max_f(m);
    float sum = 0.f;
    if (m != -INFINITY) {
#pragma unroll
      for (int k = 0; k < FOLD_IT; ++k)
        if (v[j][k].x != -INFINITY) sum += v[j][k].y * expf(v[j][k].x - m);
    }
    sum = wave_sum_f(sum);
    lse[j] = m == -INFINITY ? -INFINITY : m + logf(sum);
  }
}

// ---------------------------------------------------------------- acceptance + correction
// grid (chunk, s).  Every workgroup of a sequence runs the (cheap) acceptance
// scan, then its chunk of the correction draw; keys[(s * chunks + c) * 2] =
// (residual key, fallback key); acc[s] = a (written by chunk 0).
__global__ void __launch_bounds__(256) accept_sample_kernel(const float* logits, const float* dlog, const int* block,
                                                            SampP p, int R, const float* ml, uint64_t* keys,
                                                            int* acc, int* status) {
  __shared__ float lse_p[64], lse_q[64];
  __shared__ int s_a;
  __shared__ uint64_t sh[4];
  const int c = blockIdx.x, s = blockIdx.y, B = p.B, K = B - 1;
  const uint64_t key1 = p.stream[s], t = (uint64_t)p.pos[s];
  const int tid = threadIdx.x;
  // acceptance operands first (they need no log-sum-exp): lane i = 1..K of
  // wave 0 reads d_i, z_p(d_i) of verify row i-1, z_q(d_i) of drafter row i, u_i
  float xp = 0.f, xq = 0.f, logu = 0.f;
  if (tid >= 1 && tid <= K) {
    int x = block[(size_t)s * B + tid];
    if (x < 0 || x >= p.V) {
      if (c == 0) set_status(status, ST_BAD_TOKEN);
      x = x < 0 ? 0 : p.V - 1;
    }
    xp = logits[(size_t)(s * B + tid - 1) * p.V + x];
    xq = dlog[(size_t)(s * B + tid) * p.V + x];
    logu = logf(unif(philox(p.seed, key1, t, (uint64_t)tid, 1, 0).w[0]));
  }
  // wave w folds rows w, w + 4, ... of [target rows 0..B-1, drafter rows 1..B-1]
  for (int y0 = tid >> 6; y0 < 2 * B - 1; y0 += 4 * FOLD_ROWS) {
    int off[FOLD_ROWS];
    int n = 0;
#pragma unroll
    for (int j = 0; j < FOLD_ROWS; ++j) {
      const int y = y0 + 4 * j;
      if (y < 2 * B - 1) n = j + 1;
      off[j] = y < B ? s * B + y : R + s * B + (y - B + 1);
    }
    float l[FOLD_ROWS];
    wave_fold_rows(ml, p.chunks, off, n, l);
    if ((tid & 63) == 0) {
#pragma unroll
      for (int j = 0; j < FOLD_ROWS; ++j) {
        const int y = y0 + 4 * j;
        if (y < B) lse_p[y] = l[j];
        else if (y < 2 * B - 1) lse_q[y - B + 1] = l[j];
      }
    }
  }
  __syncthreads();
  if (tid < 64) {
    // lane i (1..K): d_i is kept when log u_i < log p_{i-1}(d_i) - log q_i(d_i)
    bool rej = false;
    if (tid >= 1 && tid <= K) {
      const float lp = xp * p.inv_t - lse_p[tid - 1];
      const float lq = xq * p.inv_t - lse_q[tid];
      rej = !(logu < lp - lq);
    }
    const uint64_t mask = __ballot(rej);
    if (tid == 0) s_a = mask ? __ffsll((unsigned long long)mask) - 2 : K;
  }
  __syncthreads();
  const int a = s_a;
  const float* rp = logits + (size_t)(s * B + a) * p.V;
  const float* rq = dlog + (size_t)(s * B + (a < K ? a + 1 : a)) * p.V;
  const float lsp = lse_p[a], lsq = a < K ? lse_q[a + 1] : 0.f;
  const int g0 = c * GPW, g1 = min(p.V / 4, g0 + GPW);
  uint64_t b1 = 0, b2 = 0;
  for (int g = g0 + tid; g < g1; g += 256) {
    const float4 xp = *(const float4*)(rp + 4 * (size_t)g);
    float4 xq = xp;
    if (a < K) xq = *(const float4*)(rq + 4 * (size_t)g);
    const Words w = philox(p.seed, key1, t, (uint64_t)(a + 1), 2, (uint64_t)g);
    const float ps[4] = {xp.x, xp.y, xp.z, xp.w}, qs[4] = {xq.x, xq.y, xq.z, xq.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float zp = ps[j] * p.inv_t;
      const float gj = gumbel(w.w[j]);
      float w1 = zp;
      if (a < K) {
        const float d = expf(zp - lsp) - expf(qs[j] * p.inv_t - lsq);
        w1 = d > 0.f ? logf(d) : -INFINITY;
      }
      const uint64_t k1 = argmax_key(w1 + gj, 4 * g + j), k2 = argmax_key(zp + gj, 4 * g + j);
      b1 = k1 > b1 ? k1 : b1;
      b2 = k2 > b2 ? k2 : b2;
    }
  }
  b1 = block_max_u64(b1, sh);
  b2 = block_max_u64(b2, sh);
  if (tid == 0) {
    keys[((size_t)s * p.chunks + c) * 2] = b1;
    keys[((size_t)s * p.chunks + c) * 2 + 1] = b2;
    if (c == 0) acc[s] = a;
  }
}

// one wave per sequence: fold the chunk keys into the correction / bonus token
// and write the round's outcome and carry record (as the greedy scan does)
__global__ void __launch_bounds__(256) accept_finish_kernel(const uint64_t* keys, const int* acc, const int* block,
                                                            int nseq, int B, int chunks, int carry_window,
                                                            int* accept_len, int* bonus, int* committed,
                                                            int* n_carry, int* carry_rec) {
  const int s = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (s >= nseq) return;
  uint64_t b1 = 0, b2 = 0;
  for (int c = lane; c < chunks; c += 64) {
    const uint64_t k1 = keys[((size_t)s * chunks + c) * 2], k2 = keys[((size_t)s * chunks + c) * 2 + 1];
    b1 = k1 > b1 ? k1 : b1;
    b2 = k2 > b2 ? k2 : b2;
  }
  b1 = wave_max_u64(b1);
  b2 = wave_max_u64(b2);
  if (lane) return;
  const int a = acc[s];
  const bool empty = (uint32_t)(b1 >> 32) <= NEG_INF_ORD;   // every residual weight was -inf
  const int tok = argmax_key_index(empty ? b2 : b1);
  write_accept_outcome(s, a, tok, block + (size_t)s * B, B, carry_window, accept_len, bonus, committed, n_carry,
                       carry_rec);
}

SampP make_params(const SampleArgs& a, int B) {
  SampP p;
  p.inv_t = a.inv_t;
  p.seed = a.seed;
  p.stream = a.stream;
  p.pos = a.pos;
  p.V = a.V;
  p.B = B;
  p.chunks = samp_chunks(a.V);
  return p;
}

// ---------------------------------------------------------------- rollout (trajectory transitions, loss)
// tgt[s * B + j] = traj[s][start[s] + j + 1], j = 0..B-1: with these as the
// "target predictions", the acceptance scan's a is the number of leading
// drafts equal to the trajectory and its bonus the trajectory token at the
// first mismatch.  Past the trajectory's end: -1 and a status bit.
__global__ void traj_targets_kernel(const int* traj, int stride, int len, const int* start, int nseq, int B,
                                    int* tgt, int* status) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= nseq * B) return;
  const int s = e / B, j = e - s * B;
  const int p = start[s] + j + 1;
  int v = -1;
  if (p >= 0 && p < len) v = traj[(size_t)s * stride + p];
  else set_status(status, ST_CAPACITY);
  tgt[e] = v;
}

// one workgroup per sequence: loss[s] = sum_i w_i CE_i / sum_i w_i over drafter
// rows i = 1..K, CE_i = lse(z_i) - z_i[traj[s][start[s] + i]], w_i = exp(-(i-1)/gamma);
// the log-sum-exp rows come from lse_part_kernel's chunk partials
__global__ void __launch_bounds__(256) draft_loss_kernel(const float* dlog, const float* ml, int chunks, int V,
                                                         int B, const int* traj, int stride, int len,
                                                         const int* start, float gamma, float* loss,
                                                         int* status) {
  __shared__ float ce[64];
  const int s = blockIdx.x, K = B - 1, tid = threadIdx.x;
  // label logits first (lane i of wave 0)
  float zl = 0.f;
  if (tid >= 1 && tid <= K) {
    const int p = start[s] + tid;
    int lab = (p >= 0 && p < len) ? traj[(size_t)s * stride + p] : -1;
    if (lab < 0 || lab >= V) {
      set_status(status, ST_BAD_TOKEN);
      lab = lab < 0 ? 0 : V - 1;
    }
    zl = dlog[(size_t)(s * B + tid) * V + lab];
  }
  for (int y0 = tid >> 6; y0 < K; y0 += 4 * FOLD_ROWS) {
    int off[FOLD_ROWS];
    int n = 0;
#pragma unroll
    for (int j = 0; j < FOLD_ROWS; ++j) {
      const int y = y0 + 4 * j;
      if (y < K) n = j + 1;
      off[j] = s * B + 1 + y;
    }
    float l[FOLD_ROWS];
    wave_fold_rows(ml, chunks, off, n, l);
    if ((tid & 63) == 0) {
#pragma unroll
      for (int j = 0; j < FOLD_ROWS; ++j)
        if (y0 + 4 * j < K) ce[1 + y0 + 4 * j] = l[j];
    }
  }
  __syncthreads();
  if (tid >= 1 && tid <= K) ce[tid] -= zl;
  __syncthreads();
  if (tid == 0) {
    float num = 0.f, den = 0.f;
    for (int i = 1; i <= K; ++i) {
      const float w = expf(-(float)(i - 1) / gamma);
      num += w * ce[i];
      den += w;
    }
    loss[s] = num / den;
  }
}

}  // namespace

hipError_t launch_traj_targets(const int* traj, int stride, int len, const int* start, int nseq, int B, int* tgt,
                               int* status, hipStream_t st) {
  if (nseq <= 0) return hipSuccess;
  const int n = nseq * B;
  hipLaunchKernelGGL(traj_targets_kernel, dim3((n + 255) / 256), dim3(256), 0, st, traj, stride, len, start, nseq, B,
                     tgt, status);
  return hipGetLastError();
}

hipError_t launch_draft_loss(const float* dlog, int V, int nseq, int B, const int* traj, int stride, int len,
                             const int* start, float gamma, float* loss, int* status, void* ws, hipStream_t st) {
  if (nseq <= 0) return hipSuccess;
  if (B < 2 || B > 64 || V < 4 || (V & 3) || samp_chunks(V) > 64 * FOLD_IT || !(gamma > 0.f))
    return hipErrorInvalidValue;
  SampleArgs a;
  a.inv_t = 1.f;
  a.seed = 0;
  a.stream = nullptr;
  a.pos = nullptr;
  a.V = V;
  const SampP p = make_params(a, B);
  const int R = nseq * B;
  float* ml = (float*)ws;
  hipLaunchKernelGGL(lse_part_kernel, dim3(p.chunks, R), dim3(256), 0, st, dlog, dlog, p, R, ml);
  hipLaunchKernelGGL(draft_loss_kernel, dim3(nseq), dim3(256), 0, st, dlog, ml, p.chunks, V, B, traj, stride, len,
                     start, gamma, loss, status);
  return hipGetLastError();
}

size_t samp_workspace_bytes(int V, int rows, int nseq) {
  const size_t ch = (size_t)samp_chunks(V);
  return 2 * (size_t)rows * ch * 2 * 4      // (max, sum) pairs of target and drafter rows
         + (size_t)rows * ch * 8            // draft keys
         + (size_t)nseq * ch * 16           // correction keys
         + (size_t)nseq * 4 + 256;          // acceptance lengths
}

hipError_t launch_sample_draft(const float* dlog, const SampleArgs& a, int nseq, int B, const int* anchor,
                               int* draft_tok, int* block_out, void* ws, hipStream_t st) {
  if (nseq <= 0) return hipSuccess;
  if (B < 2 || B > 64 || a.V < 4 || (a.V & 3) || samp_chunks(a.V) > 64 * FOLD_IT) return hipErrorInvalidValue;
  const SampP p = make_params(a, B);
  const int rows = nseq * (B - 1);
  uint64_t* part = (uint64_t*)ws;
  hipLaunchKernelGGL(draw_kernel, dim3(p.chunks, rows), dim3(256), 0, st, dlog, p, DrawRows{B - 1, 1, 0}, part);
  hipLaunchKernelGGL(draw_finish_kernel, dim3((rows + 3) / 4), dim3(256), 0, st, part, rows, p.chunks, B,
                     anchor, draft_tok, block_out);
  return hipGetLastError();
}

// The allocation-free draft sampling call keeps its draw keys here instead of
// in a context workspace.  The name is a host-side stand-in for the device
// array: host code only ever passes the address hipGetSymbolAddress returns.
static __device__ __align__(256) uint64_t scratch[SAMPLE_SCRATCH_BYTES / sizeof(uint64_t)];

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[SCRATCH_MAX_DEVICES] = {};
}  // namespace

hipError_t sample_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {   // first use on this device: resolve the device's own copy
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_sample_first(const float* row, const SampleArgs& a, int* out, void* ws, hipStream_t st) {
  if (a.V < 4 || (a.V & 3) || samp_chunks(a.V) > 64 * FOLD_IT) return hipErrorInvalidValue;
  const SampP p = make_params(a, 1);
  uint64_t* part = (uint64_t*)ws;
  hipLaunchKernelGGL(draw_kernel, dim3(p.chunks, 1), dim3(256), 0, st, row, p, DrawRows{1, 0, 2}, part);
  hipLaunchKernelGGL(draw_finish_kernel, dim3(1), dim3(256), 0, st, part, 1, p.chunks, 1, nullptr, out, nullptr);
  return hipGetLastError();
}

hipError_t launch_accept_sampled(const float* logits, const float* dlog, const int* block, const SampleArgs& a,
                                 int nseq, int B, int carry_window, int* accept_len, int* bonus, int* committed,
                                 int* n_carry, int* carry_rec, int* status, void* ws, hipStream_t st) {
  if (nseq <= 0) return hipSuccess;
  if (B < 2 || B > 64 || a.V < 4 || (a.V & 3) || samp_chunks(a.V) > 64 * FOLD_IT) return hipErrorInvalidValue;
  const SampP p = make_params(a, B);
  const int R = nseq * B;
  char* b = (char*)ws;
  float* ml = (float*)b;
  b += 2 * (size_t)R * p.chunks * 2 * 4;
  uint64_t* keys = (uint64_t*)b;
  b += (size_t)nseq * p.chunks * 16;
  int* acc = (int*)b;
  hipLaunchKernelGGL(lse_part_kernel, dim3(p.chunks, 2 * R), dim3(256), 0, st, logits, dlog, p, R, ml);
  hipLaunchKernelGGL(accept_sample_kernel, dim3(p.chunks, nseq), dim3(256), 0, st, logits, dlog, block, p, R, ml,
                     keys, acc, status);
  hipLaunchKernelGGL(accept_finish_kernel, dim3((nseq + 3) / 4), dim3(256), 0, st, keys, acc, block, nseq, B,
                     p.chunks, carry_window, accept_len, bonus, committed, n_carry, carry_rec);
  return hipGetLastError();
}

}  // namespace dflow
