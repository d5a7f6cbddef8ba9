// Internal launch interface between the C-ABI layer and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm.h"

namespace dflow {

// Paged KV layout (per layer pool): [page][kv_head][64 keys x Dh] where the
// 64 x Dh block of a page is stored in matrix-core fragment order:
//   K element (key, d): ((kt*KS + ks)*64 + q*16 + key%16)*KL + d%KL
//       with kt = key/16, ks = d/KT, q = (d%KT)/KL, KS = Dh/KT
//   V element (key, d): ((vg*DT + dt)*64 + q*16 + d%16)*KL + (key%(4 KL))/16*4 + key%4
//       with vg = key/(4 KL), q = (key%16)/4, dt = d/16, DT = Dh/16
//       (a lane fragment holds KL keys of one channel)
// (KL, KT: 8, 32 for bf16 and 4, 16 for fp32.)
struct AttnParams {
  int fused;                 // 1: QK-norm + RoPE + the block's KV write done here from qkv
  const void* q;             // fused = 0: [nseq*Bq, Hq*Dh] queries after QK-norm + RoPE
  // fused = 1: raw projection rows [q heads | k heads | v heads] x Dh as qkv_ks
  // fp32 partial sums (K parts) qkv_part floats apart, added by the kernel
  const float* qkv; int ld_qkv; int qkv_ks; size_t qkv_part;
  const void* q_norm;        // [Dh] QK-norm gains
  const void* k_norm;        // [Dh]
  const float2* rope;        // [max_pages*64][Dh/2] (cos, sin)
  float eps;
  int* status;
  void* kpool;               // this layer's pools (the block's own rows are written)
  void* vpool;
  const int* page_table;     // [nseq][max_pages]
  int max_pages;
  const int* start_pos;      // [nseq] absolute position of block row 0
  int nseq, Bq, Hq, Hkv, Dh;
  int causal;                // 1: row j sees keys <= start+j; 0: all keys < start+Bq
  int split_keys;            // keys per split: `chunks` chunks of split_keys_for keys, at most 64 pages
  int chunks;                // chunks per split (resident in LDS one after another); 1 when the
                             // launch has more 16-row groups than attention_waves
  int nsplit;                // split slots per sequence for this launch (grid and partial stride)
  int num_pages;             // pages per layer pool (page ids are checked)
  int rg;                    // 16-row groups per (seq, kv head)
  float* part_o;             // [nseq][Hkv][rg][nsplit][16][Dh]
  float* part_ml;            // [nseq][Hkv][rg][nsplit][16][2]
  void* out;                 // [nseq*Bq, Hq*Dh] storage type
  FragOut outf;              // matrix-core-order copy of out for the O projection (skinny launches)
  // pf_wgs extra workgroups (after the nseq*Hkv*nsplit attention ones) read
  // bytes [0, pf_bytes) of pf, pf_per bytes each (multiples of 16), with
  // plain loads that leave them in the memory-side cache for a following
  // launch's non-temporal weight stream; pf_wgs = 0: none
  const void* pf; size_t pf_bytes; size_t pf_per; int pf_wgs;
};
// Bytes one prefetch workgroup of an attention launch reads: what a compute
// unit pulls in between the workgroup's pause and the end of a skinny round's
// attention (8B shape: 192 KB per unit, 21.5 MB over 112 idle units; 256 KB
// stretched the launch by 0.5-0.9 us for less than that gained).
constexpr size_t ATTN_PF_WG_BYTES = 192 * 1024;
hipError_t launch_attention(bool bf16, const AttnParams& p, hipStream_t s);
// Waves per attention workgroup (each owns one 16-row group; more groups need chunks = 1).
int attention_waves(bool fused, int Bq, int G);
// Whether the fused variant fits (block rows per wave, LDS) for this shape.
bool attention_fuses_rope(bool bf16, int Bq, int G, int Dh, int split_keys);

}  // namespace dflow

namespace dflow {

struct RopeParams {
  const void* qkv; int ld;        // rows: [q heads (nq)][k heads][v heads] x Dh, storage type
  // or, when qkv32 is set, the same rows as fp32 partial sums: part k at
  // qkv32 + k * part (parts = 2 when part > 0), added and rounded here
  const float* qkv32; size_t part;
  int M, Bq;                      // rows, rows per sequence
  int nq, Hkv, Dh;                // nq = query heads present (0 for context rows)
  const void* q_norm;             // [Dh]
  const void* k_norm;             // [Dh]
  const float2* rope;             // [max_pos][Dh/2] (cos, sin)
  const int* start_pos;           // [nseq] position of row 0 of each sequence
  const int* row_limit;           // nullable [nseq]: only rows j <= row_limit[s] are written
  void* q_out;                    // [M, nq*Dh]
  void* kpool; void* vpool;       // this layer's pools
  const int* page_table; int max_pages; int num_pages;
  int* status;
  float eps;
  // several layers in one launch (grid z): layer l reads columns from l * layer_cols,
  // writes the pools at l * pool_stride elements and takes its K-norm gain from k_norms[l]
  int nlayers; int layer_cols; size_t pool_stride; const void* const* k_norms;
};

hipError_t launch_embed(bool bf16, const int* tok, int M, const void* E, int V, int d, void* out, int* status,
                        float* ssq, int ssq_ld, FragOut of, hipStream_t s);
hipError_t launch_rmsnorm(bool bf16, bool in_f32, const void* x, int ldx, int M, int d, const void* g, float eps,
                          void* out, int ldo, FragOut of, hipStream_t s);
hipError_t launch_qk_rope_write(bool bf16, const RopeParams& p, hipStream_t s);
constexpr int ARGMAX_SPLITS = 32;   // workgroups of the argmax reduction
// Optional drafter layout of the row argmaxes (rows s*B + j): block_out[s][j] =
// anchor[s] for j = 0 else the argmax; draft_tok[s][j-1] = the argmax of rows j >= 1.
struct DraftOut { const int* anchor; int B; int* draft_tok; int* block_out; };
hipError_t launch_argmax_reduce(const uint64_t* amax, int groups, int M, uint64_t* part, unsigned* counter, int* out,
                                const DraftOut* draft, hipStream_t s);
hipError_t launch_accept(const int* block, const int* g, int nseq, int B, int carry_window, int* accept_len,
                         int* bonus, int* committed, int* n_carry, int* carry_rec, hipStream_t s);
hipError_t launch_relay_gather(bool bf16, int carry_on, const int* carry_rec, const void* E, const void* f, int nseq,
                               int B, int d, int V, void* u, FragOut of, hipStream_t s);
hipError_t launch_relay_input(bool bf16, int carry_on, const int* carry_rec, const int* anchor, const void* E,
                              const void* e_mask, const void* f, const float* bg, const void* ln_g,
                              const void* ln_b, float ln_eps, int nseq, int B, int d, int V, void* x, int* status,
                              float* ssq, int ssq_ld, FragOut of, hipStream_t s);
hipError_t launch_commit(const int* accept_len, int nseq, int* seq_len, hipStream_t s);
hipError_t launch_force(const int* traj, int traj_stride, int traj_len, const signed char* mode, const int* tok,
                        const int* anchor, const int* start_pos, int nseq, int B, int V, int* block_tok,
                        hipStream_t s);
hipError_t launch_set_int(int* dst, int value, hipStream_t s);
hipError_t launch_fill_u32(uint32_t* dst, uint32_t value, size_t n, hipStream_t s);

// ---- speculative sampling (sampling.hip)
constexpr int SAMP_CHUNK = 1024;   // columns per workgroup of the vocabulary passes (one 4-column group per lane)
inline int samp_chunks(int V) { return (V + SAMP_CHUNK - 1) / SAMP_CHUNK; }
struct SampleArgs {
  float inv_t;              // 1/T rounded to fp32
  uint64_t seed;            // Philox key word 0
  const uint64_t* stream;   // [nseq] Philox key word 1 per sequence
  const int* pos;           // [nseq] anchor position t of the round
  int V;                    // vocabulary (multiple of 4); logits rows have stride V
};
size_t samp_workspace_bytes(int V, int rows, int nseq);
// drafts d_i ~ softmax(z_i) of drafter logits rows s*B + i (i = 1..K)
hipError_t launch_sample_draft(const float* dlog, const SampleArgs& a, int nseq, int B, const int* anchor,
                               int* draft_tok, int* block_out, void* ws, hipStream_t st);
// Fixed scratch of the allocation-free draft sampling call: the draw keys in a
// file-scope device array (one copy per GPU).  sample_scratch resolves the
// array's device address on the current device (once per device, cached) and
// returns it with its size in bytes.
constexpr size_t SAMPLE_SCRATCH_BYTES = (size_t)1 << 20;
hipError_t sample_scratch(void** ptr);
// first token after a prompt: out[0] ~ softmax(row / T), counter (pos[0], 0, 2, column / 4)
hipError_t launch_sample_first(const float* row, const SampleArgs& a, int* out, void* ws, hipStream_t st);
// rollout: trajectory tokens as acceptance targets, and the decayed drafter loss
hipError_t launch_traj_targets(const int* traj, int stride, int len, const int* start, int nseq, int B, int* tgt,
                               int* status, hipStream_t st);
hipError_t launch_draft_loss(const float* dlog, int V, int nseq, int B, const int* traj, int stride, int len,
                             const int* start, float gamma, float* loss, int* status, void* ws, hipStream_t st);
// acceptance, correction / bonus draw and the outcome of every sequence
hipError_t launch_accept_sampled(const float* logits, const float* dlog, const int* block, const SampleArgs& a,
                                 int nseq, int B, int carry_window, int* accept_len, int* bonus, int* committed,
                                 int* n_carry, int* carry_rec, int* status, void* ws, hipStream_t st);

}  // namespace dflow
