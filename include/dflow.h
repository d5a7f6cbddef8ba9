/*
 * dflow.h - C ABI of the MI355X (gfx950) DFlow speculative-decoding round.
 *
 * One round of block-diffusion speculative decoding with verifier information
 * relay (DFlow):
 *   dflow_draft_block       block drafting: drafter inputs built from the mask
 *                           embedding and the relayed verifier states
 *                           (Sec. 4.2, eqs. reject_conditioning, dflow_input),
 *                           one parallel drafter forward conditioned on fused
 *                           target features (Sec. 3, eqs. dflash_context,
 *                           dflash_drafting);
 *   dflow_verify_block      target forward over the block against the KV cache
 *                           (Sec. 3, exact-match verification);
 *   dflow_accept_and_carry  longest-prefix acceptance, bonus token, block
 *                           partition (Sec. 3, eq. verification_partition),
 *                           joint W_c projection of the verifier states and
 *                           the shifted carry record (Sec. 4.2, verifier
 *                           representation alignment);
 *   kv_commit               commit of the accepted prefix plus bonus; the
 *                           rejected positions are rolled back (Sec. 3; Sec. 1
 *                           on the rejection boundary as the commit boundary).
 *
 * Conventions
 *  - Every data pointer argument is a DEVICE pointer owned by the caller unless
 *    stated otherwise; the library never allocates or frees device memory.
 *    Weight, cache, page-table, workspace and status pointers registered at
 *    dflow_create must stay valid until dflow_destroy.
 *  - Every call is asynchronous on the given hipStream_t (0 = null stream) and
 *    performs no host synchronisation, except dflow_read_status.  The calls
 *    on one context share its workspace and per-sequence state, so they must
 *    execute in order: issue them on one stream (or order the streams with
 *    events); contexts are independent of each other.
 *  - Return value: DFLOW_OK (0) or a negative DFLOW_E* code; the thread-local
 *    message of the last failure is available from dflow_last_error().  Host-
 *    checkable errors are reported before any launch.  Conditions that depend
 *    on device-resident values (a token id out of range, a position past the
 *    sequence's page table) set bits of the device status word instead and the
 *    offending writes are skipped; read it with dflow_read_status.
 *  - Storage type: DFLOW_BF16 (weights, activations and KV in bf16, fp32
 *    accumulation, fp32 logits) or DFLOW_F32.  Token ids are int32.
 *  - Shape constraints: d, ffn, relay_hidden, n_heads*head_dim and vocab must
 *    be multiples of 16; d, ffn and n_heads*head_dim multiples of 32 (bf16) or
 *    16 (f32); head_dim is 64 or 128; block <= 64.
 *  - Batch: b sequences (slots 0..b-1), each with the same block size B.
 *    Per-sequence positions, acceptance lengths and carry sizes are device
 *    arrays, so sequences may be ragged.
 *
 * Layouts
 *  - Linear weights are [out, in] row-major in the source and must be
 *    converted with dflow_pack_linear into the library's tile layout (same
 *    byte size).  The target/drafter QKV weight is the row concatenation
 *    [Wq; Wk; Wv]; the gate/up weight is [W_gate; W_up] packed with
 *    gate_up = 1.  A projection that reads RMSNorm(x) (QKV after the
 *    attention norm, gate/up after the FFN norm, the LM heads after the
 *    final norms) is packed with that norm's gain as col_gain: the library
 *    applies the per-row 1/rms scale itself and never materialises the
 *    normalised rows.  QK-norm gains, g_c, biases, embeddings and E_mask
 *    stay plain.
 *  - KV pools, one per layer, consecutive: [layer][num_pages][n_kv_heads]
 *    [64 x head_dim block].  Position p of sequence s lives in page
 *    page_table[s*max_pages + p/64], slot p%64.  Inside a block the keys and
 *    values are stored in matrix-core fragment order (KL, KT = 8, 32 for
 *    bf16; 4, 16 for f32):
 *      K (slot, e): ((slot/16 * head_dim/KT + e/KT) * 64 + (e%KT)/KL * 16
 *                    + slot%16) * KL + e%KL
 *      V (slot, e): ((slot/(4 KL) * head_dim/16 + e/16) * 64 + (slot%16)/4 * 16
 *                    + e%16) * KL + (slot%(4 KL))/16 * 4 + slot%4
 *    The drafter's context cache has the same layout with n_draft_layers
 *    layers and shares the page table.
 */
#ifndef DFLOW_H
#define DFLOW_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DFLOW_OK 0
#define DFLOW_EINVAL (-1)       /* null pointer, bad enum value, bad index */
#define DFLOW_ESHAPE (-2)       /* a dimension violates the shape constraints */
#define DFLOW_EDTYPE (-3)       /* unsupported storage type */
#define DFLOW_ECAPACITY (-4)    /* rows/sequences beyond what the context was created for */
#define DFLOW_EHIP (-5)         /* a HIP runtime call failed */
#define DFLOW_EUNSUPPORTED (-6) /* valid request the library does not implement */

#define DFLOW_F32 0
#define DFLOW_BF16 1

/* Which verifier rows are relayed (Sec. 4.2).  Next-round block index i takes
 * verify row a+i (the state at the position before the index's position).
 * SUFFIX: rows a+1..K-1, the states that predict the rejected-suffix
 * positions, at indices 1..K-1-a.  SUFFIX_TAIL: rows a+1..K (also the state
 * after the last draft), at indices 1..K-a.  SUFFIX_INPUTS: rows a+2..K, the
 * states whose inputs are the rejected suffix, at indices 2..K-a (index 1
 * keeps the mask embedding). */
#define DFLOW_CARRY_SUFFIX 0
#define DFLOW_CARRY_SUFFIX_TAIL 1
#define DFLOW_CARRY_SUFFIX_INPUTS 2

/* device status bits */
#define DFLOW_STATUS_BAD_TOKEN 1
#define DFLOW_STATUS_CAPACITY 2
#define DFLOW_STATUS_BAD_PAGE 4

typedef struct dflow_dims {
  int dtype;              /* DFLOW_F32 or DFLOW_BF16 */
  int d;                  /* hidden size */
  int n_layers;           /* target decoder layers */
  int n_heads;            /* query heads */
  int n_kv_heads;         /* key/value heads (divides n_heads) */
  int head_dim;           /* 64 or 128 */
  int ffn;                /* SwiGLU intermediate size */
  int vocab;
  int n_draft_layers;     /* drafter decoder layers (Sec. 5.1: five) */
  int n_capture;          /* m, number of target layers feeding W_c */
  int capture_layers[16]; /* 0-based target layer indices, increasing */
  int relay_hidden;       /* MLP_phi hidden width */
  int block;              /* B = anchor + K drafted tokens */
  int max_batch;          /* sequences per call; max_batch * block <= 1024 */
  int max_rows;           /* rows per prefill chunk (block..1024) */
  int max_pages;          /* page-table row length per sequence */
  int num_pages;          /* pages in each layer pool */
  int carry_window;       /* DFLOW_CARRY_* */
  float rope_theta;       /* RoPE base (1e6 for Qwen3) */
  float rms_eps;          /* RMSNorm epsilon */
  float ln_eps;           /* relay LayerNorm epsilon */
} dflow_dims;

typedef struct dflow_layer {
  const void* wqkv;       /* packed [(n_heads+2*n_kv_heads)*head_dim, d], col_gain = attention-norm gain */
  const void* q_norm;     /* [head_dim] */
  const void* k_norm;     /* [head_dim] */
  const void* wo;         /* packed [d, n_heads*head_dim] */
  const void* wgu;        /* packed (gate_up=1) [2*ffn, d], col_gain = FFN-norm gain */
  const void* wdown;      /* packed [d, ffn] */
} dflow_layer;

typedef struct dflow_weights {
  const void* embed;            /* [vocab, d] plain row-major (shared by target, drafter and relay) */
  const void* lm_head;          /* packed [vocab, d], col_gain = target final-norm gain */
  const dflow_layer* layers;    /* HOST array [n_layers] */
  const dflow_layer* draft_layers; /* HOST array [n_draft_layers] */
  const void* draft_lm_head;    /* the shared LM head packed with col_gain = drafter final-norm gain */
  const void* draft_wkv_ctx;    /* packed [n_draft_layers*2*n_kv_heads*head_dim, d], no gain: for each drafter
                                   layer l its [Wk; Wv] (rows from l*2*n_kv_heads*head_dim), projecting the
                                   context features F into that layer's K/V (Sec. 3, eq. dflash_context) */
  const void* e_mask;           /* [d] mask embedding E_mask */
  const void* w_c;              /* packed [d, n_capture*d] feature projection W_c */
  const void* g_c;              /* [d] RMSNorm gain after W_c */
  const void* relay_w1;         /* packed [relay_hidden, 3d] */
  const void* relay_c1;         /* [relay_hidden] */
  const void* relay_w2;         /* packed [2d, relay_hidden] -> [beta; gamma] */
  const void* relay_c2;         /* [2d] */
  const void* relay_ln_g;       /* [d] LayerNorm gain */
  const void* relay_ln_b;       /* [d] LayerNorm bias */
} dflow_weights;

typedef struct dflow_cache {
  void* k_pool;                 /* target K pools, n_layers consecutive */
  void* v_pool;                 /* target V pools */
  void* ck_pool;                /* drafter context K pools, n_draft_layers consecutive */
  void* cv_pool;                /* drafter context V pools */
  const int32_t* page_table;    /* [max_batch][max_pages] page ids in [0, num_pages) */
} dflow_cache;

typedef struct dflow_ctx dflow_ctx;

/* Thread-local description of the last error of this thread ("" if none). */
const char* dflow_last_error(void);

/* Bytes of one packed linear weight of shape [N, K] (equal to N*K*elt). */
size_t dflow_packed_bytes(int dtype, int N, int K);

/* Rearranges a row-major [N, K] weight into the tile layout the GEMM kernels
 * stream.  gate_up = 1 treats w as [W_gate; W_up] and makes every packed
 * 16-row strip hold 8 gate rows followed by the same 8 up rows.  col_gain
 * (nullable, device [K] in the storage type) multiplies column k by
 * col_gain[k] (fp32 product rounded once to the storage type): the gain of
 * the RMSNorm that precedes the projection.  `w` and `out` are device buffers
 * of dflow_packed_bytes. */
int dflow_pack_linear(hipStream_t stream, int dtype, const void* w, int N, int K, int gate_up, const void* col_gain,
                      void* out);

/* Bytes of device workspace a context needs for these dims (0 if the dims are
 * invalid).  The workspace holds the round's activations, the carry record
 * between rounds, split partials, the RoPE table and reduction counters. */
size_t dflow_workspace_bytes(const dflow_dims* dims);

/* Validates dims and registers the (device) weight and cache pointers, the
 * caller's workspace (device, at least dflow_workspace_bytes(dims) bytes,
 * 256-byte aligned) and the caller's status word (device int32, the
 * DFLOW_STATUS_* bits of device-detected conditions).  Set-up: clears the
 * workspace and the status word and uploads the RoPE table (angles
 * p * theta^(-2i/head_dim) evaluated in double) on `stream`, then waits for
 * that stream.  The library allocates no device memory, here or in any
 * other call.  *out receives the context (host memory, freed by
 * dflow_destroy; the workspace and status stay the caller's). */
int dflow_create(const dflow_dims* dims, const dflow_weights* w, const dflow_cache* cache, void* workspace,
                 size_t workspace_bytes, int32_t* status, hipStream_t stream, dflow_ctx** out);
int dflow_destroy(dflow_ctx* ctx);

/* Number of K parts the context streams each QKV projection in (1 or 2):
 * with two, the projection writes two fp32 partial sums that the attention
 * (or QK-norm/RoPE) kernel adds.  Fixed at create from (d, q/kv widths) and
 * the device's compute-unit count; for byte accounting.  Returns -1 on a
 * null context. */
int dflow_qkv_parts(const dflow_ctx* ctx);

/* Attention work split of the round calls (verify and draft): *chunk_keys
 * receives the keys of one LDS-resident chunk (128 or 256) and *chunks the
 * chunks per split (a split covers chunks * chunk_keys keys at fixed absolute
 * positions, the running softmax carried across its chunks; prefill, and a
 * call whose query rows need more row groups than one workgroup has waves,
 * use one chunk per split).  Fixed at create from max_batch, the kv heads and the
 * capacity; for tests and byte accounting.  Returns 0, or DFLOW_EINVAL on a
 * null argument. */
int dflow_attention_split(const dflow_ctx* ctx, int* chunk_keys, int* chunks);

/* Prompt processing for sequence slot `seq` (set-up, not part of the round):
 * target KV for positions 0..len-1, fused features and drafter context K/V
 * for the same positions, and first_anchor[0] = the target's greedy token
 * after the prompt.  Clears the slot's carry record.  tok: device [len]. */
int dflow_prefill(dflow_ctx* ctx, hipStream_t stream, int seq, const int32_t* tok, int len, int32_t* first_anchor);

/* Prompt processing of nseq sequences in slots 0..nseq-1: dflow_prefill of
 * each.  tok: device, the prompts back to back (sum of len tokens); len: HOST
 * [nseq] prompt lengths (the host plans the row chunks, so the lengths are
 * host values); first_anchor: device [nseq].  Every length is checked before
 * anything is launched. */
int dflow_prefill_batch(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* tok, const int32_t* len,
                        int32_t* first_anchor);

/* Block drafting (Sec. 3 eq. dflash_drafting; Sec. 4.2 eq. dflow_input).
 * Block row 0 is anchor_tok[s] at position anchor_pos[s]; rows 1..K start
 * from E_mask, except rows 1..n_carry[s] of the previous accept_and_carry,
 * which take E_mask + beta*LN(h) + gamma when carry_on != 0.  Every block row
 * attends to the drafter context (positions < anchor_pos) and to the whole
 * block.  Writes draft_tok [b, K] (argmax of rows 1..K) and, if non-null,
 * block_out [b, B] = [anchor, drafts] and, if non-null, the fp32 drafter
 * logits of every block row, draft_logits [b*B, vocab].  With draft_logits
 * given, draft_tok and block_out may both be NULL (sampling decoding draws
 * the drafts with dflow_sample_draft).
 * The block's K/V are written to the drafter context cache at
 * anchor_pos..anchor_pos+K as scratch and are overwritten by kv_commit. */
int dflow_draft_block(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* anchor_tok,
                      const int32_t* anchor_pos, int carry_on, int32_t* draft_tok, int32_t* block_out,
                      float* draft_logits);

/* Exact-match verification forward (Sec. 3).  block_tok [b, B] holds the
 * anchor followed by the K proposals, at positions start_pos[s]..+K.  Writes
 * the target KV of all B positions (speculatively; kv_commit rolls back the
 * rejected ones), the target argmax per row tgt_argmax [b, B] (lowest id on
 * ties), optional fp32 logits [b, B, vocab] (tgt_argmax and logits may each
 * be NULL; with both NULL the LM head is skipped), and the residual outputs of the
 * capture layers, which accept_and_carry projects (hcap: pass NULL to use
 * the internal buffer; otherwise a device [b*B, n_capture*d] copy). */
int dflow_verify_block(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* block_tok,
                       const int32_t* start_pos, int32_t* tgt_argmax, float* logits, void* hcap);

/* Acceptance and relay preparation (Sec. 3 eq. verification_partition;
 * Sec. 4.2).  a = number of leading proposals equal to the target argmax of
 * the previous row; bonus = argmax of row a; committed [b, B] = d_1..d_a,
 * bonus, then -1.  Projects every verified row with the shared W_c + RMSNorm
 * (rows 0..a become drafter context at kv_commit, rows a+1.. are the relay
 * source) and records the carry for the next dflow_draft_block.  Launches no
 * target-layer kernel.  feat (nullable): device [b*B, d] copy of the
 * projected features. */
int dflow_accept_and_carry(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* block_tok,
                           const int32_t* tgt_argmax, int32_t* accept_len, int32_t* bonus, int32_t* committed,
                           int32_t* n_carry, void* feat);

/* Commit (rollback = truncation): seq_len[s] += accept_len[s] + 1, where
 * seq_len[s] must equal the start_pos used by the verify.  Appends the drafter
 * context K/V of the projected rows 0..accept_len[s] at positions
 * seq_len..seq_len+accept_len (the name follows the paper's round contract). */
int kv_commit(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* accept_len, int32_t* seq_len);

/* ---- Sampling decoding at temperature T > 0 (Table 1 reports T = 1).
 * Verification then follows speculative sampling (Leviathan, Kalman and
 * Matias, ICML 2023, cited in Sec. 1), which keeps the target's output
 * distribution: with p_j = softmax(target logits of verify row j / T) and
 * q_i = softmax(drafter logits of block row i / T),
 *   drafts    d_i ~ q_i (i = 1..K);
 *   accept    d_i while u_i < p_{i-1}(d_i) / q_i(d_i) (a = leading accepted);
 *   token     at block index a+1: drawn from max(0, p_a - q_{a+1})
 *             normalised when a < K, from p_K when a = K.
 * The round is then: dflow_draft_block (draft_logits non-null), then
 * dflow_sample_draft, dflow_verify_block (logits non-null),
 * dflow_accept_sampled, kv_commit.
 * Random numbers: Philox4x64-10 (Salmon et al., SC 2011) with key (seed,
 * stream[s]) and counter (anchor_pos[s], block index, purpose, column / 4),
 * output word column % 4, purposes 0 = draft, 1 = acceptance, 2 = correction
 * or bonus; a word x gives u = ((x >> 41) + 1/2) * 2^-23.  Draws use
 * argmax_v (log-weight_v - log(-log u_v)), lowest id on ties.  A sequence's
 * tokens therefore depend only on (seed, its stream id, its state), never on
 * its slot or on the other sequences of the batch.  All arithmetic is fp32. */
typedef struct dflow_sampler {
  float temperature;        /* T: positive and finite */
  uint64_t seed;            /* Philox key word 0 */
  const uint64_t* stream;   /* device [b]: Philox key word 1 of each sequence (e.g. a request id) */
} dflow_sampler;

/* Draws d_i ~ q_i for rows i = 1..K of every sequence from draft_logits
 * [b*B, vocab] (fp32, as written by dflow_draft_block; row s*B holds the
 * anchor row and is not read).  Writes draft_tok [b, K] and, if non-null,
 * block_out [b, B] = [anchor_tok[s], drafts].  anchor_pos [b] is the round's
 * anchor position t (the counter word 0).  Host checks: smp non-null with a
 * valid temperature, vocab a multiple of 4. */
int dflow_sample_draft(dflow_ctx* ctx, hipStream_t stream, int nseq, const float* draft_logits,
                       const int32_t* anchor_tok, const int32_t* anchor_pos, const dflow_sampler* smp,
                       int32_t* draft_tok, int32_t* block_out);

/* Allocation-free variant of dflow_sample_draft, for callers that cannot
 * allocate or provide device memory for a call's scratch (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation).  Same
 * arguments, outputs and random-number addressing as dflow_sample_draft, and
 * bit-identical drafts; the per-chunk draw keys (nseq * (block - 1) *
 * ceil(vocab / 1024) 8-byte keys) go to a fixed device array of the library,
 * DFLOW_SAMPLE_SCRATCH_BYTES on every GPU it runs on, held until the process
 * ends, instead of the context's workspace.  A request needing more returns
 * DFLOW_ECAPACITY before any launch (at the Qwen3 vocabulary: up to 879 drawn
 * rows, 58 sequences at block 16).  The call allocates nothing.  Every call on
 * one GPU shares that GPU's array, which keeps the last call's keys: calls
 * that overlap on one GPU (streams not ordered against each other) race on it
 * and must not be issued. */
#define DFLOW_SAMPLE_SCRATCH_BYTES (1u << 20)
int dflow_sample_draft_noalloc(dflow_ctx* ctx, hipStream_t stream, int nseq, const float* draft_logits,
                               const int32_t* anchor_tok, const int32_t* anchor_pos, const dflow_sampler* smp,
                               int32_t* draft_tok, int32_t* block_out);

/* Prompt processing for sampling decoding: dflow_prefill, except that the
 * first token is drawn from softmax(z / T) of the prompt's last row with the
 * Philox counter (len - 1, 0, 2, column / 4) and key (seed, smp->stream[0]):
 * pass this sequence's stream id as a one-element device array.  The rounds'
 * counters start at t = len, so no number is drawn twice. */
int dflow_prefill_sampled(dflow_ctx* ctx, hipStream_t stream, int seq, const int32_t* tok, int len,
                          const dflow_sampler* smp, int32_t* first_token);

/* Speculative-sampling acceptance: the counterpart of dflow_accept_and_carry
 * for T > 0, with the same outputs (accept_len, bonus = the token at block
 * index a+1, committed [b, B], n_carry, the carry record, the projected
 * features and the optional feat copy).  logits [b*B, vocab]: verify rows of
 * dflow_verify_block; draft_logits [b*B, vocab]: the drafter logits the drafts
 * were drawn from (rows 1..K read); block_tok [b, B] = [anchor, d_1..d_K];
 * anchor_pos [b] and smp as in dflow_sample_draft.  A draft id outside
 * [0, vocab) sets DFLOW_STATUS_BAD_TOKEN and is tested at the nearest valid id. */
int dflow_accept_sampled(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* block_tok,
                         const int32_t* anchor_pos, const float* logits, const float* draft_logits,
                         const dflow_sampler* smp, int32_t* accept_len, int32_t* bonus, int32_t* committed,
                         int32_t* n_carry, void* feat);

/* ---- Forward-only multi-round rollout (Sec. 4.3, Multi-Round Self-Conditioned
 * Training, without the optimizer).  From an anchor on a precomputed target
 * trajectory, round 0 drafts from mask embeddings (dflow_draft_block with
 * carry_on = 0) and rounds 1..k are reject-conditioned (carry_on = 1); each
 * round's actual proposals are verified (dflow_verify_block; with tgt_argmax
 * and logits both NULL the LM head is skipped: the rollout needs only the KV
 * and the captured states), and the transition to the next round follows
 * the trajectory, not the verifier: dflow_trajectory_targets writes the
 * trajectory tokens as the acceptance targets, so dflow_accept_and_carry
 * finds a = leading drafts equal to the trajectory and takes the trajectory
 * token at the first mismatch as the next anchor (Sec. 4.3, target
 * trajectory transition), while the relayed states still come from the
 * verification of the actual proposals.  kv_commit then keeps the target KV
 * of the accepted prefix, which equals the trajectory's.
 *
 * traj: device int32 [b, traj_stride], row s = sequence s's trajectory
 * (tokens at absolute positions 0..traj_len-1).  tgt [b, B]: tgt[s][j] =
 * traj[s][start_pos[s] + j + 1]; a position at or past traj_len gives -1 and
 * sets DFLOW_STATUS_CAPACITY. */
int dflow_trajectory_targets(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* traj, int traj_stride,
                             int traj_len, const int32_t* start_pos, int32_t* tgt);

/* Decayed cross entropy of one round's drafts against the trajectory
 * (following DFlash, Sec. 4.3): loss[s] = sum_i w_i CE_i / sum_i w_i over
 * block rows i = 1..K, w_i = exp(-(i-1)/gamma), CE_i = logsumexp(z_i) -
 * z_i[traj[s][start_pos[s] + i]], z_i the fp32 drafter logits of row s*B + i
 * in draft_logits [b*B, vocab] (from dflow_draft_block).  The rollout's
 * objective is the sum of the rounds' losses (eq. dflow_training_objective).
 * loss: device float [b].  A label outside [0, vocab) or past traj_len sets
 * DFLOW_STATUS_BAD_TOKEN and is read at the nearest valid id. */
int dflow_draft_loss(dflow_ctx* ctx, hipStream_t stream, int nseq, const float* draft_logits, const int32_t* traj,
                     int traj_stride, int traj_len, const int32_t* start_pos, float gamma, float* loss);

/* Serving support (continuous batching keeps the active sequences in slots
 * 0..nseq-1): moves the per-sequence state the library keeps between rounds
 * -- the carry record and the projected feature rows of the last verify, which
 * the next dflow_draft_block relays (Sec. 4.2) -- from slot `from` to slot `to`
 * (overwriting it).  The caller moves its own per-slot state: the page-table
 * row (the KV and drafter-context pages follow it), sequence length and anchor.
 * Slots must be in 0..max_batch-1; asynchronous on `stream`. */
int dflow_move_slot(dflow_ctx* ctx, hipStream_t stream, int from, int to);

/* Measurement construct (not part of the method): builds the verified block
 * [anchor, forced drafts] from a target trajectory traj [b, traj_stride]
 * (absolute positions, traj_len valid entries) and this round's plan
 * mode/tok [b, B]: mode 1 -> traj[t+j], 2 -> (traj[t+j] + 1 + tok) mod vocab,
 * 0 -> tok, with t = start_pos[s]. */
int dflow_bench_force_drafts(dflow_ctx* ctx, hipStream_t stream, int nseq, const int32_t* traj, int traj_stride,
                             int traj_len, const int8_t* mode, const int32_t* tok, const int32_t* anchor,
                             const int32_t* start_pos, int32_t* block_tok);

/* Kernel timing (tracing aid, not part of the method).  While enabled, every
 * weight-streaming GEMM launch and every attention launch is bracketed by HIP
 * events recorded on the launch's stream (up to 16384 launches between reads;
 * timing-only events, created without the system-scope fence, so a record
 * adds no cache writeback to the launch it brackets).  Synchronise the
 * stream before reading.  dflow_profile_read waits for the recorded events
 * and aggregates them per
 * kernel class (GEMM epilogue and shape, or attention): summed elapsed
 * milliseconds, launches and algorithmic bytes (GEMM: each weight, input and
 * output byte once; attention: 0, its key count is device-resident), and
 * the entry point that issued them (phase).  Writes up to max_entries
 * entries, sets *n_entries, then clears the record. */
#define DFLOW_PHASE_OTHER 0
#define DFLOW_PHASE_DRAFT 1     /* dflow_draft_block */
#define DFLOW_PHASE_VERIFY 2    /* dflow_verify_block */
#define DFLOW_PHASE_ACCEPT 3    /* dflow_accept_and_carry, dflow_accept_sampled */
#define DFLOW_PHASE_COMMIT 4    /* kv_commit */
#define DFLOW_PHASE_PREFILL 5   /* dflow_prefill, dflow_prefill_batch, dflow_prefill_sampled */
typedef struct dflow_prof_entry {
  char name[32];   /* "gemm.store", "gemm.resid", "gemm.swiglu", "gemm.argmax", ..., "attention" */
  int N, K, M;     /* GEMM shape (0 for attention) */
  int phase;       /* DFLOW_PHASE_* */
  int launches;
  double ms;
  double bytes;
} dflow_prof_entry;
int dflow_profile(dflow_ctx* ctx, int enable);
int dflow_profile_read(dflow_ctx* ctx, dflow_prof_entry* out, int max_entries, int* n_entries);

/* Synchronises `stream`, copies the device status word to *host_status and,
 * if clear != 0, resets it (on `stream`, then waits for it). */
int dflow_read_status(dflow_ctx* ctx, hipStream_t stream, int32_t* host_status, int clear);

#ifdef __cplusplus
}
#endif
#endif /* DFLOW_H */
