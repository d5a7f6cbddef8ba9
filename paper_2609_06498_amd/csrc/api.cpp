// C ABI of the DFlow round: context, workspace and the call sequences of the
// four round calls (draft, verify, accept-and-carry, commit) plus prefill.
// Every computation is a HIP kernel launch on the caller's stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/dflow.h"
#include "common.h"
#include "kernels.h"
#include "round_state.h"

using namespace dflow;

namespace {
thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIPCHK(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) return fail(DFLOW_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
}  // namespace

struct dflow_ctx {
  dflow_dims dm;
  bool bf;
  size_t elt;
  int KT;
  int q_dim, kv_dim, qkv_n;
  int mmax, rows_round;
  int G, nsplit, part_items;
  int split_keys;            // keys per attention chunk (split_keys_for)
  int round_chunks;          // attention chunks per split in the round calls (prefill: 1)
  int lm_groups;
  int qkv_ks;                // K parts of the QKV projection (fp32 partial sums, added by the consumers)
  int cus;                   // compute units of the device (launch balance decisions)

  dflow_weights w;
  std::vector<dflow_layer> layers, dlayers;
  dflow_cache c;
  size_t pool_layer_elems;   // elements of one layer pool (K or V)

  void* ws = nullptr;         // caller-owned workspace (dflow_workspace_bytes)
  size_t ws_bytes = 0;
  int phase = DFLOW_PHASE_OTHER;   // entry point being issued (tags the kernel-timing record)
  // workspace views
  void *x, *xn, *qkv, *q, *attn, *act, *hcap, *f, *fpre, *u, *hid;
  float *fproj, *bg, *part_o, *part_ml;
  float2* rope;
  uint64_t* amax;
  int *carry_rec, *status, *tmp_pos, *tmp_argmax;
  float* ssq;   // [mmax][SSQ_LD] sums of squares of x per 16-column strip (RMSNorm row scales)
  uint64_t* amax_part;   // [ARGMAX_SPLITS][mmax]
  unsigned* counters;    // arrival counters of last-workgroup reductions; every launch leaves them at 0
  void* ctxkv;           // [mmax][n_draft_layers * 2 * kv_dim] drafter-context K/V projections
  const void** dknorm;   // device [n_draft_layers] K-norm gain pointers of the drafter layers
  void* samp;            // sampling decoding partials
  float* samp_row;       // [vocab] logits of the last prompt row (dflow_prefill_sampled)
  float* kpart;          // K-part partial sums of the split residual and gate/up GEMMs
  // Matrix-core-order copies of the projections' A operands (the round's
  // max_batch * block rows, rounded up to 16): x (QKV, gate/up, LM heads),
  // attention output (O), SwiGLU / relay hidden (down, relay W2), captured
  // states (W_c), relay input (W1), projected features (drafter context K/V).
  // Used by the round's calls (frag; prefill reads row-major A); a copy is read
  // only by the call that wrote it, or -- captured states, features -- by the
  // next call of the round (accept after verify, commit after accept).
  void *xf, *attnf, *actf, *hcapf, *uf, *ff;
  bool frag = false;

  // kernel timing record (dflow_profile)
  bool prof = false;
  std::vector<hipEvent_t> ev0, ev1;
  struct Rec { int cls, N, K, M, phase; double bytes; };
  std::vector<Rec> ev_rec;
  int n_ev = 0;
};

static const char* kClassName[] = {"gemm.store", "gemm.store_f32", "gemm.resid", "gemm.swiglu",
                                   "gemm.bias_silu", "gemm.bias_f32", "gemm.argmax", "attention"};
static constexpr int CLS_ATTN = 7;
// rows of one call (b x B per round, a prefill chunk); up to 128 the weight-streaming GEMM, beyond the tiled one
static constexpr int MAX_ROWS = 1024;

static constexpr int PROF_MAX = 16384;
static_assert(DFLOW_SAMPLE_SCRATCH_BYTES == SAMPLE_SCRATCH_BYTES, "the header states the scratch size");

extern "C" const char* dflow_last_error(void) { return g_err.c_str(); }

extern "C" size_t dflow_packed_bytes(int dtype, int N, int K) {
  return (size_t)N * (size_t)K * (dtype == DFLOW_BF16 ? 2 : 4);
}

extern "C" int dflow_pack_linear(hipStream_t stream, int dtype, const void* w, int N, int K, int gate_up,
                                 const void* col_gain, void* out) {
  if (!w || !out) return fail(DFLOW_EINVAL, "pack: null pointer");
  if (dtype != DFLOW_F32 && dtype != DFLOW_BF16) return fail(DFLOW_EDTYPE, "pack: dtype %d", dtype);
  const int KT = dtype == DFLOW_BF16 ? 32 : 16;
  if (N <= 0 || K <= 0 || N % 16 || K % KT || (gate_up && N % 32))
    return fail(DFLOW_ESHAPE, "pack: N=%d K=%d must be multiples of 16 and %d", N, K, KT);
  HIPCHK(launch_pack(dtype == DFLOW_BF16, w, N, K, gate_up, col_gain, out, stream));
  return DFLOW_OK;
}

namespace {

int validate(const dflow_dims* d) {
  if (!d) return fail(DFLOW_EINVAL, "dims is null");
  if (d->dtype != DFLOW_F32 && d->dtype != DFLOW_BF16) return fail(DFLOW_EDTYPE, "dtype %d", d->dtype);
  const int KT = d->dtype == DFLOW_BF16 ? 32 : 16;
  const int qd = d->n_heads * d->head_dim;
  if (d->head_dim != 64 && d->head_dim != 128) return fail(DFLOW_ESHAPE, "head_dim %d (64 or 128)", d->head_dim);
  if (d->n_heads <= 0 || d->n_kv_heads <= 0 || d->n_heads % d->n_kv_heads)
    return fail(DFLOW_ESHAPE, "heads %d / kv heads %d", d->n_heads, d->n_kv_heads);
  if (d->d <= 0 || d->d % KT || qd % KT || d->ffn <= 0 || d->ffn % KT || d->relay_hidden <= 0 ||
      d->relay_hidden % KT)
    return fail(DFLOW_ESHAPE, "d=%d q_dim=%d ffn=%d relay_hidden=%d must be multiples of %d", d->d, qd, d->ffn,
                d->relay_hidden, KT);
  if (d->vocab <= 0 || d->vocab % 16) return fail(DFLOW_ESHAPE, "vocab %d must be a multiple of 16", d->vocab);
  if (d->d > 16 * SSQ_LD) return fail(DFLOW_ESHAPE, "d = %d: RMSNorm row scales support d <= %d", d->d, 16 * SSQ_LD);
  if (d->n_layers <= 0 || d->n_draft_layers <= 0) return fail(DFLOW_ESHAPE, "layer counts");
  if (d->n_capture < 1 || d->n_capture > 16) return fail(DFLOW_ESHAPE, "n_capture %d", d->n_capture);
  for (int i = 0; i < d->n_capture; ++i) {
    if (d->capture_layers[i] < 0 || d->capture_layers[i] >= d->n_layers ||
        (i && d->capture_layers[i] <= d->capture_layers[i - 1]))
      return fail(DFLOW_ESHAPE, "capture_layers must be increasing layer indices");
  }
  if (d->block < 2 || d->block > 64) return fail(DFLOW_ESHAPE, "block %d (2..64)", d->block);
  if (d->max_batch < 1 || d->max_batch * d->block > MAX_ROWS)
    return fail(DFLOW_ECAPACITY, "max_batch*block = %d exceeds %d rows", d->max_batch * d->block, MAX_ROWS);
  if (d->max_rows < d->block || d->max_rows > MAX_ROWS)
    return fail(DFLOW_ECAPACITY, "max_rows %d (block..%d)", d->max_rows, MAX_ROWS);
  if (d->max_pages < 1 || d->num_pages < 1) return fail(DFLOW_ECAPACITY, "page counts");
  if (d->carry_window != DFLOW_CARRY_SUFFIX && d->carry_window != DFLOW_CARRY_SUFFIX_TAIL &&
      d->carry_window != DFLOW_CARRY_SUFFIX_INPUTS)
    return fail(DFLOW_EINVAL, "carry_window %d", d->carry_window);
  return DFLOW_OK;
}

struct Layout {
  size_t off[40];
  size_t total;
};

// Workspace carve-up; identical for dflow_workspace_bytes and dflow_create.
Layout plan(const dflow_dims* d, int* nsplit_out, int* part_items_out, int* lm_groups_out) {
  const size_t elt = d->dtype == DFLOW_BF16 ? 2 : 4;
  const int qd = d->n_heads * d->head_dim, kvd = d->n_kv_heads * d->head_dim;
  const int qkvn = qd + 2 * kvd;
  const int rows_round = d->max_batch * d->block;
  const int mmax = rows_round > d->max_rows ? rows_round : d->max_rows;
  const int G = d->n_heads / d->n_kv_heads;
  const int split_keys = split_keys_for(d->dtype == DFLOW_BF16, d->max_batch, d->n_kv_heads, d->max_pages * PAGE);
  const int nsplit = (d->max_pages * PAGE + split_keys - 1) / split_keys;
  const int rg_round = (d->block * G + 15) / 16, rg_pre = (d->max_rows * G + 15) / 16;
  int items = d->max_batch * rg_round;
  if (rg_pre > items) items = rg_pre;
  const int lm_groups = (d->vocab / 16 + 1) / 2;   // gemm_shape: two strips per argmax workgroup
  Layout L;
  size_t o = 0;
  int i = 0;
  auto add = [&](size_t bytes) { L.off[i++] = o; o += align256(bytes); };
  add((size_t)mmax * d->d * elt);                      // 0 x
  add((size_t)mmax * 3 * d->d * elt);                  // 1 xn (also relay u rows)
  add((size_t)2 * mmax * qkvn * 4);                    // 2 qkv: up to two fp32 K parts
  add((size_t)mmax * qd * elt);                        // 3 q
  add((size_t)mmax * qd * elt);                        // 4 attn
  add((size_t)mmax * (d->ffn > d->relay_hidden ? d->ffn : d->relay_hidden) * elt);  // 5 act / relay hidden
  add((size_t)mmax * d->n_capture * d->d * elt);       // 6 hcap
  add((size_t)rows_round * d->d * elt);                // 7 f (projected features of the last verify)
  add((size_t)mmax * d->d * elt);                      // 8 fpre (prefill features)
  add((size_t)mmax * d->d * 4);                        // 9 fproj
  add((size_t)rows_round * 2 * d->d * 4);              // 10 bg
  add((size_t)items * d->n_kv_heads * nsplit * 16 * d->head_dim * 4);  // 11 part_o
  add((size_t)items * d->n_kv_heads * nsplit * 32 * 4);               // 12 part_ml
  add((size_t)d->max_pages * PAGE * (d->head_dim / 2) * sizeof(float2));  // 13 rope
  add((size_t)lm_groups * mmax * 8);                   // 14 amax: [lm_groups][rows] argmax keys
  add((size_t)d->max_batch * CARRY_REC * 4);           // 15 carry_rec
  add(4);                                              // 16 unused (the status word is the caller's)
  add((size_t)(d->max_batch + 1) * 4);                 // 17 tmp_pos
  add((size_t)mmax * 4);                               // 18 tmp_argmax
  add((size_t)mmax * SSQ_LD * 4);                      // 19 ssq: per-strip sums of squares of the residual rows
  add((size_t)ARGMAX_SPLITS * mmax * 8);               // 20 amax_part: [split][row] partial argmax keys
  add(256);                                            // 21 counters (zero between launches)
  add((size_t)mmax * d->n_draft_layers * 2 * kvd * elt);   // 22 ctxkv: drafter-context K/V rows of all drafter layers
  add((size_t)(d->n_draft_layers > 0 ? d->n_draft_layers : 1) * sizeof(void*));   // 23 drafter K-norm gain pointers
  add(samp_workspace_bytes(d->vocab, mmax, d->max_batch));   // 24 sampling partials (log-sum-exp, draw keys)
  add((size_t)d->vocab * 4);                           // 25 fp32 logits of a prompt's last row (sampled prefill)
  {   // 26 K-part partial sums of the split GEMMs: residual (O, down), gate/up and the range-split projections
    const int kt = d->dtype == DFLOW_BF16 ? TT<bf16>::KT : TT<float>::KT;
    const int po = split_parts(EPI_RESID, d->d / 16, qd / kt), pd = split_parts(EPI_RESID, d->d / 16, d->ffn / kt);
    const size_t resid = (size_t)(po > pd ? po : pd) * mmax * d->d * 4;
    const int ps = split_parts(EPI_SWIGLU, 2 * d->ffn / 16, d->d / kt);
    const size_t rows_split = mmax < SWIGLU_SPLIT_MAX_ROWS ? mmax : SWIGLU_SPLIT_MAX_ROWS;
    const size_t swiglu = (size_t)ps * rows_split * 2 * d->ffn * 4;
    size_t need = resid > swiglu ? resid : swiglu;
    // range split of the narrow plain / fp32 / bias projections: QKV (when in
    // one part), W_c, drafter context K/V, relay MLP
    const int nc = d->n_draft_layers * 2 * kvd;
    const int rs_epi[5] = {EPI_STORE_F32, EPI_STORE_F32, EPI_STORE_T, EPI_BIAS_SILU, EPI_BIAS_F32};
    const int rs_n[5] = {qkvn, d->d, nc, d->relay_hidden, 2 * d->d};
    const int rs_k[5] = {d->d, d->n_capture * d->d, d->d, 3 * d->d, d->relay_hidden};
    for (int i = 0; i < 5; ++i) {
      if (rs_n[i] <= 0 || rs_k[i] <= 0) continue;
      const size_t r = (size_t)split_parts(rs_epi[i], rs_n[i] / 16, rs_k[i] / kt) * rows_split * rs_n[i] * 4;
      if (r > need) need = r;
    }
    add(need);
  }
  {   // 27..32 matrix-core-order operand copies of the round's rows
    const size_t fr = (size_t)((rows_round + 15) / 16 * 16) * elt;
    add(fr * d->d);                                       // 27 x
    add(fr * qd);                                         // 28 attention output
    add(fr * (d->ffn > d->relay_hidden ? d->ffn : d->relay_hidden));   // 29 SwiGLU / relay hidden
    add(fr * d->n_capture * d->d);                        // 30 captured states
    add(fr * 3 * d->d);                                   // 31 relay input
    add(fr * d->d);                                       // 32 projected features
  }
  L.total = o;
  if (nsplit_out) *nsplit_out = nsplit;
  if (part_items_out) *part_items_out = items;
  if (lm_groups_out) *lm_groups_out = lm_groups;
  return L;
}

}  // namespace

extern "C" size_t dflow_workspace_bytes(const dflow_dims* dims) {
  if (validate(dims) != DFLOW_OK) return 0;
  return plan(dims, nullptr, nullptr, nullptr).total;
}

extern "C" int dflow_create(const dflow_dims* dims, const dflow_weights* w, const dflow_cache* cache,
                            void* workspace, size_t workspace_bytes, int32_t* status, hipStream_t stream,
                            dflow_ctx** out) {
  int rc = validate(dims);
  if (rc) return rc;
  if (!w || !cache || !out || !workspace || !status) return fail(DFLOW_EINVAL, "create: null argument");
  if (((uintptr_t)workspace & 255) || ((uintptr_t)status & 3))
    return fail(DFLOW_EINVAL, "create: workspace must be 256-byte and status 4-byte aligned");
  {
    const size_t need = plan(dims, nullptr, nullptr, nullptr).total;
    if (workspace_bytes < need)
      return fail(DFLOW_ECAPACITY, "create: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  }
  const void* req[] = {w->embed, w->lm_head, w->layers, w->draft_layers, w->draft_lm_head, w->draft_wkv_ctx,
                       w->e_mask, w->w_c, w->g_c, w->relay_w1, w->relay_c1, w->relay_w2, w->relay_c2,
                       w->relay_ln_g, w->relay_ln_b, cache->k_pool, cache->v_pool, cache->ck_pool, cache->cv_pool,
                       cache->page_table};
  for (size_t i = 0; i < sizeof(req) / sizeof(req[0]); ++i)
    if (!req[i]) return fail(DFLOW_EINVAL, "create: required pointer #%zu is null", i);
  auto chk_layer = [](const dflow_layer& L) {
    return L.wqkv && L.q_norm && L.k_norm && L.wo && L.wgu && L.wdown;
  };
  for (int l = 0; l < dims->n_layers; ++l)
    if (!chk_layer(w->layers[l])) return fail(DFLOW_EINVAL, "create: null pointer in target layer %d", l);
  for (int l = 0; l < dims->n_draft_layers; ++l)
    if (!chk_layer(w->draft_layers[l])) return fail(DFLOW_EINVAL, "create: null pointer in drafter layer %d", l);

  dflow_ctx* c = new dflow_ctx();
  c->dm = *dims;
  c->bf = dims->dtype == DFLOW_BF16;
  c->elt = c->bf ? 2 : 4;
  c->KT = c->bf ? 32 : 16;
  c->q_dim = dims->n_heads * dims->head_dim;
  c->kv_dim = dims->n_kv_heads * dims->head_dim;
  c->qkv_n = c->q_dim + 2 * c->kv_dim;
  c->rows_round = dims->max_batch * dims->block;
  c->mmax = c->rows_round > dims->max_rows ? c->rows_round : dims->max_rows;
  c->G = dims->n_heads / dims->n_kv_heads;
  {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                hipSuccess) {
      delete c;
      return fail(DFLOW_EHIP, "create: no device attributes");
    }
    c->qkv_ks = gemm_ksplit(c->qkv_n / 16, dims->d / c->KT, cus);
    c->cus = cus;
  }
  c->w = *w;
  c->layers.assign(w->layers, w->layers + dims->n_layers);
  c->dlayers.assign(w->draft_layers, w->draft_layers + dims->n_draft_layers);
  c->w.layers = c->layers.data();
  c->w.draft_layers = c->dlayers.data();
  c->c = *cache;
  c->pool_layer_elems = (size_t)dims->num_pages * dims->n_kv_heads * PAGE * dims->head_dim;

  Layout L = plan(dims, &c->nsplit, &c->part_items, &c->lm_groups);
  c->split_keys = split_keys_for(c->bf, dims->max_batch, dims->n_kv_heads, dims->max_pages * PAGE);
  c->round_chunks = round_chunks_for(dims->max_batch, dims->n_kv_heads, dims->max_pages * PAGE, c->split_keys, c->cus);
  c->ws = workspace;
  c->ws_bytes = L.total;
  char* b = (char*)c->ws;
  c->x = b + L.off[0];
  c->xn = b + L.off[1];
  c->qkv = b + L.off[2];
  c->q = b + L.off[3];
  c->attn = b + L.off[4];
  c->act = b + L.off[5];
  c->hcap = b + L.off[6];
  c->f = b + L.off[7];
  c->fpre = b + L.off[8];
  c->fproj = (float*)(b + L.off[9]);
  c->bg = (float*)(b + L.off[10]);
  c->part_o = (float*)(b + L.off[11]);
  c->part_ml = (float*)(b + L.off[12]);
  c->rope = (float2*)(b + L.off[13]);
  c->amax = (uint64_t*)(b + L.off[14]);
  c->carry_rec = (int*)(b + L.off[15]);
  c->status = status;
  c->tmp_pos = (int*)(b + L.off[17]);
  c->tmp_argmax = (int*)(b + L.off[18]);
  c->ssq = (float*)(b + L.off[19]);
  c->amax_part = (uint64_t*)(b + L.off[20]);
  c->counters = (unsigned*)(b + L.off[21]);
  c->ctxkv = b + L.off[22];
  c->dknorm = (const void**)(b + L.off[23]);
  c->samp = b + L.off[24];
  c->samp_row = (float*)(b + L.off[25]);
  c->kpart = (float*)(b + L.off[26]);
  c->xf = b + L.off[27];
  c->attnf = b + L.off[28];
  c->actf = b + L.off[29];
  c->hcapf = b + L.off[30];
  c->uf = b + L.off[31];
  c->ff = b + L.off[32];
  c->u = c->xn;
  c->hid = c->act;

  // RoPE table: angle p * theta^(-2i/Dh) evaluated in double
  const int half = dims->head_dim / 2;
  const size_t npos = (size_t)dims->max_pages * PAGE;
  std::vector<float2> tab(npos * half);
  for (int i = 0; i < half; ++i) {
    const double inv = std::pow((double)dims->rope_theta, -2.0 * i / dims->head_dim);
    for (size_t p = 0; p < npos; ++p) {
      const double a = (double)p * inv;
      tab[p * half + i] = make_float2((float)std::cos(a), (float)std::sin(a));
    }
  }
  {   // the device address of the allocation-free sampling call's scratch, resolved on this device now
    void* sp = nullptr;
    const hipError_t es = sample_scratch(&sp);
    if (es != hipSuccess) {
      delete c;
      return fail(DFLOW_EHIP, "create: scratch symbol: %s", hipGetErrorString(es));
    }
  }
  // set-up on the caller's stream: clear the workspace and the status word,
  // upload the RoPE table and the drafter K-norm pointers, then wait for it
  // (the host buffers are local)
  std::vector<const void*> kn(dims->n_draft_layers > 0 ? dims->n_draft_layers : 0);
  for (int l = 0; l < dims->n_draft_layers; ++l) kn[l] = c->dlayers[l].k_norm;
  hipError_t e = launch_fill_u32((uint32_t*)c->ws, 0u, c->ws_bytes / 4, stream);
  if (e == hipSuccess) e = launch_fill_u32((uint32_t*)c->status, 0u, 1, stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess && !kn.empty())
    e = hipMemcpyAsync(c->dknorm, kn.data(), kn.size() * sizeof(void*), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    delete c;
    return fail(DFLOW_EHIP, "create: %s", hipGetErrorString(e));
  }
  *out = c;
  return DFLOW_OK;
}

extern "C" int dflow_destroy(dflow_ctx* c) {
  if (!c) return fail(DFLOW_EINVAL, "destroy: null context");
  for (auto ev : c->ev0) (void)hipEventDestroy(ev);
  for (auto ev : c->ev1) (void)hipEventDestroy(ev);
  delete c;   // the workspace and the status word belong to the caller
  return DFLOW_OK;
}

// ------------------------------------------------------------------ internals
namespace {

struct NormIn {            // RMSNorm of the A rows: per-strip sums of squares; the gain is in the packed weight
  const float* ssq = nullptr;
};

struct Frag {              // matrix-core-order A operand and output copies (skinny launches only)
  const void* a = nullptr;
  FragOut y{}, y2{};
};

// copy of `cols` columns at c0 of a K-wide consumer operand, when the call uses them
FragOut fout(const dflow_ctx* c, void* buf, int K, int c0 = 0) {
  return c->frag ? FragOut{buf, K / c->KT, c0} : FragOut{nullptr, 0, 0};
}

hipError_t gemm(dflow_ctx* c, hipStream_t st, int epi, const void* A, int lda, const void* W, int M, int N, int K,
                void* Y, int ldy, const void* R = nullptr, int ldr = 0, void* Y2 = nullptr, int ldy2 = 0,
                const void* bias = nullptr, float* logits = nullptr, int ldl = 0, NormIn nin = NormIn(),
                float* ssq_out = nullptr, int ksplit = 1, Frag fr = Frag()) {
  GemmParams p{};
  p.Af = fr.a;
  p.yf = fr.y;
  p.y2f = fr.y2;
  p.ksplit = ksplit;
  p.y_part = (size_t)M * ldy;
  if (nin.ssq) {
    p.norm = 1;
    p.ssq = nin.ssq;
    p.ssq_ld = SSQ_LD;
    p.ssq_parts = c->dm.d / 16;
    p.eps = c->dm.rms_eps;
  }
  p.ssq_out = ssq_out;
  p.ssq_out_ld = SSQ_LD;
  p.A = A;
  p.lda = lda;
  p.W = W;
  p.M = M;
  p.ntiles = N / 16;
  p.ktiles = K / c->KT;
  p.Y = Y;
  p.ldy = ldy;
  p.R = R;
  p.ldr = ldr;
  p.Y2 = Y2;
  p.ldy2 = ldy2;
  p.bias = bias;
  p.amax = c->amax;
  p.amax_ld = M;   // keys [group][row], compact for this launch
  p.logits = logits;
  p.ldl = ldl;
  p.col0 = 0;
  p.part_ws = (epi == EPI_RESID || epi == EPI_SWIGLU || range_split_applies(epi, M, N / 16, ksplit)) ? c->kpart
                                                                                                    : nullptr;
  p.cus = c->cus;
  const bool rec = c->prof && c->n_ev < PROF_MAX;
  if (rec) {
    hipError_t e = hipEventRecord(c->ev0[c->n_ev], st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = launch_gemm(c->bf, epi, p, st);
  if (e != hipSuccess) return e;
  if (rec) {
    if ((e = hipEventRecord(c->ev1[c->n_ev], st)) != hipSuccess) return e;
    const double out_elt = (epi == EPI_ARGMAX) ? 0.0 : ((epi == EPI_STORE_F32 || epi == EPI_BIAS_F32) ? 4.0 : c->elt);
    const double n_out = (epi == EPI_SWIGLU) ? N / 2.0 : N;
    c->ev_rec[c->n_ev] = {epi, N, K, M, c->phase,
                          (double)N * K * c->elt + (double)M * K * c->elt + (double)M * n_out * out_elt * ksplit};
    ++c->n_ev;
  }
  return hipSuccess;
}

void* pool_layer(dflow_ctx* c, void* pool, int l) { return (char*)pool + (size_t)l * c->pool_layer_elems * c->elt; }

// Attention of `nseq` sequences x Bq rows over one layer's pools.  With
// `fused`, from the raw QKV projection rows (QK-norm, RoPE and the block's
// KV-cache write happen inside); otherwise from c->q after qk_rope.
hipError_t attention(dflow_ctx* c, hipStream_t st, const dflow_layer& L, int nseq, int Bq, const int* start_pos,
                     const int* page_table, void* kpool, void* vpool, int causal, bool fused) {
  AttnParams a{};
  a.fused = fused ? 1 : 0;
  a.q = c->q;
  a.qkv = reinterpret_cast<const float*>(c->qkv);
  a.ld_qkv = c->qkv_n;
  a.qkv_ks = c->qkv_ks;
  a.qkv_part = (size_t)nseq * Bq * c->qkv_n;
  a.q_norm = L.q_norm;
  a.k_norm = L.k_norm;
  a.rope = c->rope;
  a.eps = c->dm.rms_eps;
  a.status = c->status;
  a.kpool = kpool;
  a.vpool = vpool;
  a.page_table = page_table;
  a.max_pages = c->dm.max_pages;
  a.start_pos = start_pos;
  a.nseq = nseq;
  a.Bq = Bq;
  a.Hq = c->dm.n_heads;
  a.Hkv = c->dm.n_kv_heads;
  a.Dh = c->dm.head_dim;
  a.causal = causal;
  {
    const int nw = attention_waves(fused, Bq, c->G), nrg = (Bq * c->G + 15) / 16;
    a.chunks = (c->phase != DFLOW_PHASE_PREFILL && nrg <= nw) ? c->round_chunks : 1;
    a.split_keys = c->split_keys * a.chunks;
    a.nsplit = (c->dm.max_pages * PAGE + a.split_keys - 1) / a.split_keys;   // <= c->nsplit
  }
  // Round launches that leave compute units idle pull weights of a following
  // projection into the memory-side cache meanwhile, at most ATTN_PF_WG_BYTES
  // per idle unit: the O projection's when they fit in that budget, else the
  // start of the gate/up projection's, whose long HBM-bound stream gains more
  // per prefetched byte (8B shape, same box: O 4.400 -> 4.377 ms/round,
  // gate/up 4.392 -> 4.359; 1.7B shape: O 1.932 -> 1.897, gate/up 1.898 ->
  // 1.917, its shorter attention stretched by the larger prefetch).
  if (c->phase != DFLOW_PHASE_PREFILL && L.wo && L.wgu && c->cus > nseq * a.Hkv * a.nsplit) {
    const int idle = c->cus - nseq * a.Hkv * a.nsplit;
    const size_t cap = (size_t)idle * ATTN_PF_WG_BYTES;
    const size_t wo_bytes = (size_t)c->dm.d * c->q_dim * c->elt;
    const size_t gu_bytes = (size_t)2 * c->dm.ffn * c->dm.d * c->elt;
    const bool o_fits = wo_bytes <= cap;
    a.pf = o_fits ? L.wo : L.wgu;
    a.pf_bytes = (o_fits ? wo_bytes : (gu_bytes < cap ? gu_bytes : cap)) / 16 * 16;
    a.pf_per = ((a.pf_bytes + idle - 1) / idle + 15) / 16 * 16;
    a.pf_wgs = idle;
  }
  a.num_pages = c->dm.num_pages;
  a.rg = (Bq * c->G + 15) / 16;
  a.part_o = c->part_o;
  a.part_ml = c->part_ml;
  a.out = c->attn;
  a.outf = fout(c, c->attnf, c->q_dim);
  const bool rec = c->prof && c->n_ev < PROF_MAX;
  hipError_t e;
  if (rec && (e = hipEventRecord(c->ev0[c->n_ev], st)) != hipSuccess) return e;
  if ((e = launch_attention(c->bf, a, st)) != hipSuccess) return e;
  if (rec) {
    if ((e = hipEventRecord(c->ev1[c->n_ev], st)) != hipSuccess) return e;
    c->ev_rec[c->n_ev++] = {CLS_ATTN, 0, 0, nseq * Bq, c->phase, 0.0};
  }
  return hipSuccess;
}

// QK-norm + RoPE + KV write for rows of `nseq` x Bq.
RopeParams rope_params(dflow_ctx* c, const dflow_layer& L, int nseq, int Bq, int nq, const int* start_pos,
                       const int* row_limit, const int* page_table, void* kpool, void* vpool) {
  RopeParams r{};
  r.M = nseq * Bq;
  r.Bq = Bq;
  r.nq = nq;
  r.Hkv = c->dm.n_kv_heads;
  r.Dh = c->dm.head_dim;
  r.q_norm = L.q_norm;
  r.k_norm = L.k_norm;
  r.rope = c->rope;
  r.start_pos = start_pos;
  r.row_limit = row_limit;
  r.q_out = c->q;
  r.kpool = kpool;
  r.vpool = vpool;
  r.page_table = page_table;
  r.max_pages = c->dm.max_pages;
  r.num_pages = c->dm.num_pages;
  r.status = c->status;
  r.eps = c->dm.rms_eps;
  r.nlayers = 1;
  return r;
}

// One Qwen3-style decoder layer over x (M = nseq*Bq rows) in place.
hipError_t decoder_layer(dflow_ctx* c, hipStream_t st, const dflow_layer& L, int nseq, int Bq, const int* start_pos,
                         const int* page_table, void* kpool, void* vpool, int causal, void* capture,
                         FragOut capf = FragOut{nullptr, 0, 0}) {
  const dflow_dims& d = c->dm;
  const int M = nseq * Bq;
  hipError_t e;
  // The attention and FFN RMSNorms are applied by the QKV and gate/up
  // projections (gain folded into the packed weight, 1/rms from the sums of
  // squares that the producer of x -- embedding, relay input or the residual
  // epilogue -- left in c->ssq).
  NormIn attn_n, ffn_n;
  attn_n.ssq = c->ssq;
  ffn_n.ssq = c->ssq;
  // QKV projection as fp32 partial sums over qkv_ks K parts (spreads the
  // weight stream evenly over the compute units); its consumers add them
  // matrix-core-order operands (skinny rounds): x from its producer, the
  // attention output from the combine kernel, the SwiGLU output from gate/up
  Frag fq, fo, fgu, fdn;
  if (c->frag) {
    fq.a = c->xf;
    fo.a = c->attnf;
    fo.y = fout(c, c->xf, d.d);
    fgu.a = c->xf;
    fgu.y = fout(c, c->actf, d.ffn);
    fdn.a = c->actf;
    fdn.y = fout(c, c->xf, d.d);
    fdn.y2 = capf;
  }
  if ((e = gemm(c, st, EPI_STORE_F32, c->x, d.d, L.wqkv, M, c->qkv_n, d.d, c->qkv, c->qkv_n, nullptr, 0, nullptr, 0,
                nullptr, nullptr, 0, attn_n, nullptr, c->qkv_ks, fq)))
    return e;
  const bool fused = attention_fuses_rope(c->bf, Bq, c->G, d.head_dim, c->split_keys);
  if (!fused) {
    RopeParams r = rope_params(c, L, nseq, Bq, d.n_heads, start_pos, nullptr, page_table, kpool, vpool);
    r.qkv32 = reinterpret_cast<const float*>(c->qkv);
    r.ld = c->qkv_n;
    r.part = c->qkv_ks == 2 ? (size_t)M * c->qkv_n : 0;
    if ((e = launch_qk_rope_write(c->bf, r, st))) return e;
  }
  if ((e = attention(c, st, L, nseq, Bq, start_pos, page_table, kpool, vpool, causal, fused))) return e;
  if ((e = gemm(c, st, EPI_RESID, c->attn, c->q_dim, L.wo, M, d.d, c->q_dim, c->x, d.d, c->x, d.d, nullptr, 0,
                nullptr, nullptr, 0, NormIn(), c->ssq, 1, fo)))
    return e;
  if ((e = gemm(c, st, EPI_SWIGLU, c->x, d.d, L.wgu, M, 2 * d.ffn, d.d, c->act, d.ffn, nullptr, 0, nullptr, 0,
                nullptr, nullptr, 0, ffn_n, nullptr, 1, fgu)))
    return e;
  const int capld = d.n_capture * d.d;
  if ((e = gemm(c, st, EPI_RESID, c->act, d.ffn, L.wdown, M, d.d, d.ffn, c->x, d.d, c->x, d.d, capture, capld,
                nullptr, nullptr, 0, NormIn(), c->ssq, 1, fdn)))
    return e;
  return hipSuccess;
}

// Target forward over block rows already embedded in x; argmax of every row into `argmax_out`.
hipError_t target_forward(dflow_ctx* c, hipStream_t st, int nseq, int Bq, const int* start_pos,
                          const int* page_table, int* argmax_out, float* logits, int lm_row0 = 0, int lm_rows = -1) {
  const dflow_dims& d = c->dm;
  const int M = nseq * Bq;
  hipError_t e;
  int ci = 0;
  for (int l = 0; l < d.n_layers; ++l) {
    void* cap = nullptr;
    FragOut capf{nullptr, 0, 0};
    if (ci < d.n_capture && d.capture_layers[ci] == l) {
      capf = fout(c, c->hcapf, d.n_capture * d.d, ci * d.d);
      cap = (char*)c->hcap + (size_t)ci++ * d.d * c->elt;
    }
    if ((e = decoder_layer(c, st, c->layers[l], nseq, Bq, start_pos, page_table, pool_layer(c, c->c.k_pool, l),
                           pool_layer(c, c->c.v_pool, l), 1, cap, capf)))
      return e;
  }
  if (!argmax_out && !logits) return hipSuccess;
  // LM head (final RMSNorm folded in) over rows lm_row0 .. lm_row0+lm_rows-1 only
  if (lm_rows < 0) lm_rows = M;
  const size_t off = (size_t)lm_row0 * d.d * c->elt;
  NormIn fin;
  fin.ssq = c->ssq + (size_t)lm_row0 * SSQ_LD;
  Frag flm;
  if (c->frag && lm_row0 == 0) flm.a = c->xf;
  if ((e = gemm(c, st, EPI_ARGMAX, (char*)c->x + off, d.d, c->w.lm_head, lm_rows, d.vocab, d.d, nullptr, 0, nullptr,
                0, nullptr, 0, nullptr, logits, d.vocab, fin, nullptr, 1, flm)))
    return e;
  if (!argmax_out) return hipSuccess;
  return launch_argmax_reduce(c->amax, c->lm_groups, lm_rows, c->amax_part, c->counters, argmax_out, nullptr, st);
}

// F = RMSNorm(W_c [captured states]) for M rows -> fout (storage type)
hipError_t project(dflow_ctx* c, hipStream_t st, int M, void* out) {
  const dflow_dims& d = c->dm;
  hipError_t e;
  const int K = d.n_capture * d.d;
  Frag fr;
  if (c->frag) fr.a = c->hcapf;
  if ((e = gemm(c, st, EPI_STORE_F32, c->hcap, K, c->w.w_c, M, d.d, K, c->fproj, d.d, nullptr, 0, nullptr, 0,
                nullptr, nullptr, 0, NormIn(), nullptr, 1, fr)))
    return e;
  return launch_rmsnorm(c->bf, true, c->fproj, d.d, M, d.d, c->w.g_c, d.rms_eps, out, d.d, fout(c, c->ff, d.d),
                        st);
}

// Drafter context K/V of feature rows (nseq x Bq) at start_pos + j for rows j <= row_limit[s].
// All drafter layers at once: one GEMM over the stacked [Wk; Wv] of every
// layer, then K-norm + RoPE + paged write for every layer in one launch.
hipError_t ctx_append(dflow_ctx* c, hipStream_t st, const void* feat, int nseq, int Bq, const int* start_pos,
                      const int* row_limit, const int* page_table) {
  const dflow_dims& d = c->dm;
  if (d.n_draft_layers < 1) return hipSuccess;
  const int M = nseq * Bq;
  const int ncols = d.n_draft_layers * 2 * c->kv_dim;
  hipError_t e;
  Frag fr;
  if (c->frag) fr.a = c->ff;
  if ((e = gemm(c, st, EPI_STORE_T, feat, d.d, c->w.draft_wkv_ctx, M, ncols, d.d, c->ctxkv, ncols, nullptr, 0,
                nullptr, 0, nullptr, nullptr, 0, NormIn(), nullptr, 1, fr)))
    return e;
  RopeParams r{};
  r.qkv = c->ctxkv;
  r.ld = ncols;
  r.M = M;
  r.Bq = Bq;
  r.nq = 0;
  r.Hkv = d.n_kv_heads;
  r.Dh = d.head_dim;
  r.rope = c->rope;
  r.start_pos = start_pos;
  r.row_limit = row_limit;
  r.kpool = c->c.ck_pool;
  r.vpool = c->c.cv_pool;
  r.page_table = page_table;
  r.max_pages = d.max_pages;
  r.num_pages = d.num_pages;
  r.status = c->status;
  r.eps = d.rms_eps;
  r.nlayers = d.n_draft_layers;
  r.layer_cols = 2 * c->kv_dim;
  r.pool_stride = c->pool_layer_elems;
  r.k_norms = c->dknorm;
  return launch_qk_rope_write(c->bf, r, st);
}

int check_nseq(dflow_ctx* c, int nseq) {
  if (!c) return fail(DFLOW_EINVAL, "null context");
  if (nseq < 1 || nseq > c->dm.max_batch) return fail(DFLOW_ECAPACITY, "nseq %d outside 1..%d", nseq, c->dm.max_batch);
  return DFLOW_OK;
}

}  // namespace

namespace {
int sampler_args(const dflow_ctx* c, const dflow_sampler* smp, const int32_t* pos, SampleArgs* a);

// Prompt processing in chunks of max_rows; the last chunk's final row gives
// the first token: its argmax, or a draw at temperature T when smp is given.
int prefill_impl(dflow_ctx* c, hipStream_t st, int seq, const int32_t* tok, int len, const dflow_sampler* smp,
                 int32_t* first) {
  if (!c || !tok || !first) return fail(DFLOW_EINVAL, "prefill: null argument");
  if (seq < 0 || seq >= c->dm.max_batch) return fail(DFLOW_EINVAL, "prefill: seq %d", seq);
  if (len < 1) return fail(DFLOW_ESHAPE, "prefill: len %d", len);
  if ((long long)len + c->dm.block > (long long)c->dm.max_pages * PAGE)
    return fail(DFLOW_ECAPACITY, "prefill: %d tokens exceed the page table (%d)", len, c->dm.max_pages * PAGE);
  c->phase = DFLOW_PHASE_PREFILL;
  c->frag = false;
  SampleArgs sa;
  if (smp) {
    // counter word 0 of the first draw: the prompt's last position (held in tmp_pos[1])
    int rc = sampler_args(c, smp, c->tmp_pos + 1, &sa);
    if (rc) return rc;
  }
  const dflow_dims& d = c->dm;
  const int* pt = c->c.page_table + (size_t)seq * d.max_pages;
  for (int p0 = 0; p0 < len; p0 += d.max_rows) {
    const int n = (len - p0) < d.max_rows ? (len - p0) : d.max_rows;
    const bool last = p0 + n >= len;
    HIPCHK(launch_set_int(c->tmp_pos, p0, st));
    HIPCHK(launch_embed(c->bf, tok + p0, n, c->w.embed, d.vocab, d.d, c->x, c->status, c->ssq, SSQ_LD,
                        FragOut{nullptr, 0, 0}, st));
    int* amax = last && !smp ? c->tmp_argmax : nullptr;
    float* lrow = last && smp ? c->samp_row : nullptr;
    HIPCHK(target_forward(c, st, 1, n, c->tmp_pos, pt, amax, lrow, n - 1, 1));
    HIPCHK(project(c, st, n, c->fpre));
    HIPCHK(ctx_append(c, st, c->fpre, 1, n, c->tmp_pos, nullptr, pt));
    if (last && !smp) HIPCHK(hipMemcpyAsync(first, c->tmp_argmax, 4, hipMemcpyDeviceToDevice, st));
  }
  if (smp) {
    HIPCHK(launch_set_int(c->tmp_pos + 1, len - 1, st));
    HIPCHK(launch_sample_first(c->samp_row, sa, first, c->samp, st));
  }
  HIPCHK(launch_fill_u32((uint32_t*)(c->carry_rec + (size_t)seq * CARRY_REC), 0u, CARRY_REC, st));
  return DFLOW_OK;
}
}  // namespace

// ------------------------------------------------------------------ entry points
extern "C" int dflow_prefill(dflow_ctx* c, hipStream_t st, int seq, const int32_t* tok, int len,
                             int32_t* first_anchor) {
  return prefill_impl(c, st, seq, tok, len, nullptr, first_anchor);
}

extern "C" int dflow_prefill_batch(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* tok, const int32_t* len,
                                   int32_t* first_anchor) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!tok || !len || !first_anchor) return fail(DFLOW_EINVAL, "prefill_batch: null argument");
  for (int s = 0; s < nseq; ++s)   // every length is checked before anything is launched
    if (len[s] < 1 || (long long)len[s] + c->dm.block > (long long)c->dm.max_pages * PAGE)
      return fail(len[s] < 1 ? DFLOW_ESHAPE : DFLOW_ECAPACITY, "prefill_batch: sequence %d has %d tokens", s, len[s]);
  size_t off = 0;
  for (int s = 0; s < nseq; ++s) {
    if ((rc = prefill_impl(c, st, s, tok + off, len[s], nullptr, first_anchor + s))) return rc;
    off += (size_t)len[s];
  }
  return DFLOW_OK;
}

extern "C" int dflow_prefill_sampled(dflow_ctx* c, hipStream_t st, int seq, const int32_t* tok, int len,
                                     const dflow_sampler* smp, int32_t* first_token) {
  if (!smp) return fail(DFLOW_EINVAL, "prefill_sampled: null sampler");
  return prefill_impl(c, st, seq, tok, len, smp, first_token);
}

extern "C" int dflow_draft_block(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* anchor_tok,
                                 const int32_t* anchor_pos, int carry_on, int32_t* draft_tok, int32_t* block_out,
                                 float* draft_logits) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!anchor_tok || !anchor_pos || (!draft_tok && !block_out && !draft_logits))
    return fail(DFLOW_EINVAL, "draft_block: null argument");
  c->phase = DFLOW_PHASE_DRAFT;
  const dflow_dims& d = c->dm;
  const int B = d.block, M = nseq * B;
  c->frag = true;
  if (carry_on) {
    Frag f1, f2;
    if (c->frag) {
      f1.a = c->uf;
      f1.y = fout(c, c->actf, d.relay_hidden);
      f2.a = c->actf;
    }
    HIPCHK(launch_relay_gather(c->bf, 1, c->carry_rec, c->w.embed, c->f, nseq, B, d.d, d.vocab, c->u,
                               fout(c, c->uf, 3 * d.d), st));
    HIPCHK(gemm(c, st, EPI_BIAS_SILU, c->u, 3 * d.d, c->w.relay_w1, M, d.relay_hidden, 3 * d.d, c->hid,
                d.relay_hidden, nullptr, 0, nullptr, 0, c->w.relay_c1, nullptr, 0, NormIn(), nullptr, 1, f1));
    HIPCHK(gemm(c, st, EPI_BIAS_F32, c->hid, d.relay_hidden, c->w.relay_w2, M, 2 * d.d, d.relay_hidden, c->bg,
                2 * d.d, nullptr, 0, nullptr, 0, c->w.relay_c2, nullptr, 0, NormIn(), nullptr, 1, f2));
  }
  HIPCHK(launch_relay_input(c->bf, carry_on ? 1 : 0, c->carry_rec, anchor_tok, c->w.embed, c->w.e_mask, c->f, c->bg,
                            c->w.relay_ln_g, c->w.relay_ln_b, d.ln_eps, nseq, B, d.d, d.vocab, c->x, c->status,
                            c->ssq, SSQ_LD, fout(c, c->xf, d.d), st));
  for (int l = 0; l < d.n_draft_layers; ++l)
    HIPCHK(decoder_layer(c, st, c->dlayers[l], nseq, B, anchor_pos, c->c.page_table, pool_layer(c, c->c.ck_pool, l),
                         pool_layer(c, c->c.cv_pool, l), 0, nullptr));
  NormIn fin;
  fin.ssq = c->ssq;
  Frag flm;
  if (c->frag) flm.a = c->xf;
  HIPCHK(gemm(c, st, EPI_ARGMAX, c->x, d.d, c->w.draft_lm_head, M, d.vocab, d.d, nullptr, 0, nullptr, 0, nullptr, 0,
              nullptr, draft_logits, d.vocab, fin, nullptr, 1, flm));
  if (!draft_tok && !block_out) return DFLOW_OK;
  const DraftOut dr{anchor_tok, B, draft_tok, block_out};
  HIPCHK(launch_argmax_reduce(c->amax, c->lm_groups, M, c->amax_part, c->counters, nullptr, &dr, st));
  return DFLOW_OK;
}

extern "C" int dflow_verify_block(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* block_tok,
                                  const int32_t* start_pos, int32_t* tgt_argmax, float* logits, void* hcap) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!block_tok || !start_pos) return fail(DFLOW_EINVAL, "verify_block: null argument");
  c->phase = DFLOW_PHASE_VERIFY;
  const dflow_dims& d = c->dm;
  const int B = d.block, M = nseq * B;
  c->frag = true;
  HIPCHK(launch_embed(c->bf, block_tok, M, c->w.embed, d.vocab, d.d, c->x, c->status, c->ssq, SSQ_LD,
                      fout(c, c->xf, d.d), st));
  HIPCHK(target_forward(c, st, nseq, B, start_pos, c->c.page_table, tgt_argmax, logits));
  if (hcap)
    HIPCHK(hipMemcpyAsync(hcap, c->hcap, (size_t)M * d.n_capture * d.d * c->elt, hipMemcpyDeviceToDevice, st));
  return DFLOW_OK;
}

extern "C" int dflow_accept_and_carry(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* block_tok,
                                      const int32_t* tgt_argmax, int32_t* accept_len, int32_t* bonus,
                                      int32_t* committed, int32_t* n_carry, void* feat) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!block_tok || !tgt_argmax || !accept_len || !committed)
    return fail(DFLOW_EINVAL, "accept_and_carry: null argument");
  c->phase = DFLOW_PHASE_ACCEPT;
  const dflow_dims& d = c->dm;
  const int B = d.block, M = nseq * B;
  c->frag = true;
  HIPCHK(launch_accept(block_tok, tgt_argmax, nseq, B, d.carry_window, accept_len, bonus, committed, n_carry,
                       c->carry_rec, st));
  HIPCHK(project(c, st, M, c->f));
  if (feat) HIPCHK(hipMemcpyAsync(feat, c->f, (size_t)M * d.d * c->elt, hipMemcpyDeviceToDevice, st));
  return DFLOW_OK;
}

namespace {
int sampler_args(const dflow_ctx* c, const dflow_sampler* smp, const int32_t* pos, SampleArgs* a) {
  if (!smp || !smp->stream || !pos) return fail(DFLOW_EINVAL, "sampling: null sampler, stream or position array");
  const float T = smp->temperature;
  if (!(T > 0.f) || !std::isfinite(T)) return fail(DFLOW_EINVAL, "sampling: temperature %g (must be positive)", T);
  a->inv_t = 1.0f / T;
  a->seed = smp->seed;
  a->stream = smp->stream;
  a->pos = pos;
  a->V = c->dm.vocab;
  return DFLOW_OK;
}
}  // namespace

extern "C" int dflow_sample_draft(dflow_ctx* c, hipStream_t st, int nseq, const float* draft_logits,
                                  const int32_t* anchor_tok, const int32_t* anchor_pos, const dflow_sampler* smp,
                                  int32_t* draft_tok, int32_t* block_out) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!draft_logits || !anchor_tok || !draft_tok) return fail(DFLOW_EINVAL, "sample_draft: null argument");
  SampleArgs a;
  if ((rc = sampler_args(c, smp, anchor_pos, &a))) return rc;
  HIPCHK(launch_sample_draft(draft_logits, a, nseq, c->dm.block, anchor_tok, draft_tok, block_out, c->samp, st));
  return DFLOW_OK;
}

extern "C" int dflow_sample_draft_noalloc(dflow_ctx* c, hipStream_t st, int nseq, const float* draft_logits,
                                          const int32_t* anchor_tok, const int32_t* anchor_pos,
                                          const dflow_sampler* smp, int32_t* draft_tok, int32_t* block_out) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!draft_logits || !anchor_tok || !draft_tok) return fail(DFLOW_EINVAL, "sample_draft_noalloc: null argument");
  SampleArgs a;
  if ((rc = sampler_args(c, smp, anchor_pos, &a))) return rc;
  const size_t need = (size_t)nseq * (c->dm.block - 1) * samp_chunks(c->dm.vocab) * sizeof(uint64_t);
  if (need > SAMPLE_SCRATCH_BYTES)
    return fail(DFLOW_ECAPACITY, "sample_draft_noalloc: %zu bytes of draw keys (%d sequences x %d rows x %d chunks) "
                                 "exceed the fixed scratch of %zu bytes", need, nseq, c->dm.block - 1,
                samp_chunks(c->dm.vocab), SAMPLE_SCRATCH_BYTES);
  void* ws = nullptr;
  HIPCHK(sample_scratch(&ws));
  HIPCHK(launch_sample_draft(draft_logits, a, nseq, c->dm.block, anchor_tok, draft_tok, block_out, ws, st));
  return DFLOW_OK;
}

extern "C" int dflow_accept_sampled(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* block_tok,
                                    const int32_t* anchor_pos, const float* logits, const float* draft_logits,
                                    const dflow_sampler* smp, int32_t* accept_len, int32_t* bonus,
                                    int32_t* committed, int32_t* n_carry, void* feat) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!block_tok || !logits || !draft_logits || !accept_len || !committed)
    return fail(DFLOW_EINVAL, "accept_sampled: null argument");
  c->phase = DFLOW_PHASE_ACCEPT;
  SampleArgs a;
  if ((rc = sampler_args(c, smp, anchor_pos, &a))) return rc;
  const dflow_dims& d = c->dm;
  const int B = d.block, M = nseq * B;
  c->frag = true;
  HIPCHK(launch_accept_sampled(logits, draft_logits, block_tok, a, nseq, B, d.carry_window, accept_len, bonus,
                               committed, n_carry, c->carry_rec, c->status, c->samp, st));
  HIPCHK(project(c, st, M, c->f));
  if (feat) HIPCHK(hipMemcpyAsync(feat, c->f, (size_t)M * d.d * c->elt, hipMemcpyDeviceToDevice, st));
  return DFLOW_OK;
}

extern "C" int dflow_trajectory_targets(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* traj,
                                        int traj_stride, int traj_len, const int32_t* start_pos, int32_t* tgt) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!traj || !start_pos || !tgt) return fail(DFLOW_EINVAL, "trajectory_targets: null argument");
  if (traj_len < 1 || traj_stride < traj_len) return fail(DFLOW_ESHAPE, "trajectory_targets: len %d stride %d",
                                                          traj_len, traj_stride);
  HIPCHK(launch_traj_targets(traj, traj_stride, traj_len, start_pos, nseq, c->dm.block, tgt, c->status, st));
  return DFLOW_OK;
}

extern "C" int dflow_draft_loss(dflow_ctx* c, hipStream_t st, int nseq, const float* draft_logits,
                                const int32_t* traj, int traj_stride, int traj_len, const int32_t* start_pos,
                                float gamma, float* loss) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!draft_logits || !traj || !start_pos || !loss) return fail(DFLOW_EINVAL, "draft_loss: null argument");
  if (traj_len < 1 || traj_stride < traj_len) return fail(DFLOW_ESHAPE, "draft_loss: len %d stride %d", traj_len,
                                                          traj_stride);
  if (!(gamma > 0.f) || !std::isfinite(gamma)) return fail(DFLOW_EINVAL, "draft_loss: gamma %g", gamma);
  HIPCHK(launch_draft_loss(draft_logits, c->dm.vocab, nseq, c->dm.block, traj, traj_stride, traj_len, start_pos,
                           gamma, loss, c->status, c->samp, st));
  return DFLOW_OK;
}

extern "C" int kv_commit(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* accept_len, int32_t* seq_len) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!accept_len || !seq_len) return fail(DFLOW_EINVAL, "kv_commit: null argument");
  c->phase = DFLOW_PHASE_COMMIT;
  c->frag = true;
  HIPCHK(ctx_append(c, st, c->f, nseq, c->dm.block, seq_len, accept_len, c->c.page_table));
  HIPCHK(launch_commit(accept_len, nseq, seq_len, st));
  return DFLOW_OK;
}

extern "C" int dflow_qkv_parts(const dflow_ctx* c) { return c ? c->qkv_ks : fail(DFLOW_EINVAL, "qkv_parts: null context"); }

extern "C" int dflow_attention_split(const dflow_ctx* c, int* chunk_keys, int* chunks) {
  if (!c || !chunk_keys || !chunks) return fail(DFLOW_EINVAL, "attention_split: null argument");
  *chunk_keys = c->split_keys;
  *chunks = c->round_chunks;
  return DFLOW_OK;
}

extern "C" int dflow_move_slot(dflow_ctx* c, hipStream_t st, int from, int to) {
  if (!c) return fail(DFLOW_EINVAL, "move_slot: null context");
  if (from < 0 || from >= c->dm.max_batch || to < 0 || to >= c->dm.max_batch)
    return fail(DFLOW_EINVAL, "move_slot: slots %d -> %d outside 0..%d", from, to, c->dm.max_batch - 1);
  if (from == to) return DFLOW_OK;
  const size_t frow = (size_t)c->dm.block * c->dm.d * c->elt;
  HIPCHK(hipMemcpyAsync(c->carry_rec + (size_t)to * CARRY_REC, c->carry_rec + (size_t)from * CARRY_REC,
                        CARRY_REC * sizeof(int), hipMemcpyDeviceToDevice, st));
  HIPCHK(hipMemcpyAsync((char*)c->f + (size_t)to * frow, (const char*)c->f + (size_t)from * frow, frow,
                        hipMemcpyDeviceToDevice, st));
  return DFLOW_OK;
}

extern "C" int dflow_bench_force_drafts(dflow_ctx* c, hipStream_t st, int nseq, const int32_t* traj,
                                        int traj_stride, int traj_len, const int8_t* mode, const int32_t* tok,
                                        const int32_t* anchor, const int32_t* start_pos, int32_t* block_tok) {
  int rc = check_nseq(c, nseq);
  if (rc) return rc;
  if (!traj || !mode || !tok || !anchor || !start_pos || !block_tok)
    return fail(DFLOW_EINVAL, "force_drafts: null argument");
  if (traj_len > traj_stride || traj_len < 1) return fail(DFLOW_ESHAPE, "force_drafts: traj_len %d stride %d",
                                                          traj_len, traj_stride);
  HIPCHK(launch_force(traj, traj_stride, traj_len, (const signed char*)mode, tok, anchor, start_pos, nseq,
                      c->dm.block, c->dm.vocab, block_tok, st));
  return DFLOW_OK;
}

extern "C" int dflow_profile(dflow_ctx* c, int enable) {
  if (!c) return fail(DFLOW_EINVAL, "profile: null context");
  if (enable && c->ev0.empty()) {
    c->ev0.resize(PROF_MAX);
    c->ev1.resize(PROF_MAX);
    c->ev_rec.resize(PROF_MAX);
    // timing-only events: no system-scope fence (cache writeback and
    // invalidation) at each record, which would lengthen the bracketed launch
    for (int i = 0; i < PROF_MAX; ++i) {
      HIPCHK(hipEventCreateWithFlags(&c->ev0[i], hipEventDisableSystemFence));
      HIPCHK(hipEventCreateWithFlags(&c->ev1[i], hipEventDisableSystemFence));
    }
  }
  c->prof = enable != 0;
  return DFLOW_OK;
}

extern "C" int dflow_profile_read(dflow_ctx* c, dflow_prof_entry* out, int max_entries, int* n_entries) {
  if (!c || !n_entries || (max_entries > 0 && !out)) return fail(DFLOW_EINVAL, "profile_read: null argument");
  std::vector<dflow_prof_entry> agg;
  for (int i = 0; i < c->n_ev; ++i) {
    HIPCHK(hipEventSynchronize(c->ev1[i]));
    float t = 0.f;
    HIPCHK(hipEventElapsedTime(&t, c->ev0[i], c->ev1[i]));
    const auto& r = c->ev_rec[i];
    size_t k = 0;
    for (; k < agg.size(); ++k)
      if (!strcmp(agg[k].name, kClassName[r.cls]) && agg[k].N == r.N && agg[k].K == r.K && agg[k].M == r.M &&
          agg[k].phase == r.phase)
        break;
    if (k == agg.size()) {
      dflow_prof_entry e{};
      snprintf(e.name, sizeof(e.name), "%s", kClassName[r.cls]);
      e.N = r.N;
      e.K = r.K;
      e.M = r.M;
      e.phase = r.phase;
      agg.push_back(e);
    }
    agg[k].launches += 1;
    agg[k].ms += t;
    agg[k].bytes += r.bytes;
  }
  const int n = (int)agg.size() < max_entries ? (int)agg.size() : max_entries;
  for (int i = 0; i < n; ++i) out[i] = agg[i];
  *n_entries = (int)agg.size();
  c->n_ev = 0;
  return DFLOW_OK;
}

extern "C" int dflow_read_status(dflow_ctx* c, hipStream_t st, int32_t* host_status, int clear) {
  if (!c || !host_status) return fail(DFLOW_EINVAL, "read_status: null argument");
  HIPCHK(hipStreamSynchronize(st));
  HIPCHK(hipMemcpy(host_status, c->status, 4, hipMemcpyDeviceToHost));
  if (clear) {
    HIPCHK(launch_fill_u32((uint32_t*)c->status, 0u, 1, st));
    HIPCHK(hipStreamSynchronize(st));
  }
  return DFLOW_OK;
}
