"""ctypes binding of libdflow.so.

Argument marshalling only: device buffers are torch CUDA tensors whose
pointers are passed to the C ABI, and every call runs on torch's current
HIP stream.  There is no CPU fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB = None

DFLOW_F32, DFLOW_BF16 = 0, 1
CARRY_WINDOWS = {"suffix": 0, "suffix+tail": 1, "suffix-inputs": 2}
PAGE = 64


class DFlowError(RuntimeError):
    pass


def library_path() -> str:
    return os.path.join(_PKG, "libdflow.so")


class Dims(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("d", ctypes.c_int), ("n_layers", ctypes.c_int),
                ("n_heads", ctypes.c_int), ("n_kv_heads", ctypes.c_int), ("head_dim", ctypes.c_int),
                ("ffn", ctypes.c_int), ("vocab", ctypes.c_int), ("n_draft_layers", ctypes.c_int),
                ("n_capture", ctypes.c_int), ("capture_layers", ctypes.c_int * 16), ("relay_hidden", ctypes.c_int),
                ("block", ctypes.c_int), ("max_batch", ctypes.c_int), ("max_rows", ctypes.c_int),
                ("max_pages", ctypes.c_int), ("num_pages", ctypes.c_int), ("carry_window", ctypes.c_int),
                ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float), ("ln_eps", ctypes.c_float)]


class Layer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("wqkv", "q_norm", "k_norm", "wo", "wgu", "wdown")]


class Weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(Layer)), ("draft_layers", ctypes.POINTER(Layer)),
                ("draft_lm_head", ctypes.c_void_p), ("draft_wkv_ctx", ctypes.c_void_p),
                ("e_mask", ctypes.c_void_p), ("w_c", ctypes.c_void_p),
                ("g_c", ctypes.c_void_p), ("relay_w1", ctypes.c_void_p), ("relay_c1", ctypes.c_void_p),
                ("relay_w2", ctypes.c_void_p), ("relay_c2", ctypes.c_void_p), ("relay_ln_g", ctypes.c_void_p),
                ("relay_ln_b", ctypes.c_void_p)]


class Cache(ctypes.Structure):
    _fields_ = [("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p), ("ck_pool", ctypes.c_void_p),
                ("cv_pool", ctypes.c_void_p), ("page_table", ctypes.c_void_p)]


class Sampler(ctypes.Structure):
    """dflow_sampler: temperature, Philox seed, device pointer to the per-sequence stream ids."""
    _fields_ = [("temperature", ctypes.c_float), ("seed", ctypes.c_uint64), ("stream", ctypes.c_void_p)]


EXPORTS = {
    "dflow_last_error": (ctypes.c_char_p, []),
    "dflow_packed_bytes": (ctypes.c_size_t, [ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "dflow_pack_linear": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                         ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(Dims)]),
    "dflow_create": (ctypes.c_int, [ctypes.POINTER(Dims), ctypes.POINTER(Weights), ctypes.POINTER(Cache),
                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.POINTER(ctypes.c_void_p)]),
    "dflow_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "dflow_prefill": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                     ctypes.c_void_p]),
    "dflow_prefill_batch": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                           ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p]),
    "dflow_draft_block": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p]),
    "dflow_verify_block": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_accept_and_carry": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_prefill_sampled": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                             ctypes.c_int, ctypes.POINTER(Sampler), ctypes.c_void_p]),
    "dflow_sample_draft": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(Sampler),
                                          ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_sample_draft_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(Sampler),
                                                  ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_accept_sampled": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.POINTER(Sampler), ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_trajectory_targets": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                                ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_draft_loss": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_float,
                                        ctypes.c_void_p]),
    "kv_commit": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_qkv_parts": (ctypes.c_int, [ctypes.c_void_p]),
    "dflow_attention_split": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int),
                                             ctypes.POINTER(ctypes.c_int)]),
    "dflow_move_slot": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int]),
    "dflow_bench_force_drafts": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                                ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "dflow_read_status": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                         ctypes.c_int]),
    "dflow_profile": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int]),
    "dflow_profile_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                          ctypes.POINTER(ctypes.c_int)]),
}


class ProfEntry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("N", ctypes.c_int), ("K", ctypes.c_int), ("M", ctypes.c_int),
                ("phase", ctypes.c_int), ("launches", ctypes.c_int), ("ms", ctypes.c_double),
                ("bytes", ctypes.c_double)]


PHASES = {0: "other", 1: "draft", 2: "verify", 3: "accept", 4: "commit", 5: "prefill"}


def load_library(path: Optional[str] = None):
    """Loads libdflow.so (built by __graft_entry__.build or build.py)."""
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    p = path or library_path()
    if not os.path.exists(p):
        raise DFlowError(f"{p} is missing: build the HIP library first (python -m paper_2609_06498_amd.build)")
    lib = ctypes.CDLL(p)
    for name, (res, args) in EXPORTS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _LIB = lib
    return lib


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class Runtime:
    """One DFlow context: uploaded/packed weights, paged KV pools, page table."""

    def __init__(self, dims, block: int, max_batch: int, max_ctx: int, weights: Dict[str, np.ndarray],
                 carry_window: str = "suffix", max_rows: int = 128, device: str = "cuda:0"):
        import torch
        if not torch.cuda.is_available():
            raise DFlowError("no HIP device available; the DFlow runtime has no CPU path")
        self.lib = load_library()
        self.torch = torch
        self.dims = dims
        self.block = block
        self.max_batch = max_batch
        self.device = torch.device(device)
        self.dtype_code = DFLOW_BF16 if dims.dtype == "bf16" else DFLOW_F32
        self.elt_torch = torch.int16 if dims.dtype == "bf16" else torch.float32
        self.max_pages = (max_ctx + 2 * block + PAGE - 1) // PAGE
        self.num_pages = self.max_pages * max_batch
        self._keep: List = []

        d = Dims()
        d.dtype = self.dtype_code
        d.d, d.n_layers, d.n_heads, d.n_kv_heads = dims.d, dims.n_layers, dims.n_heads, dims.n_kv_heads
        d.head_dim, d.ffn, d.vocab, d.n_draft_layers = dims.head_dim, dims.ffn, dims.vocab, dims.n_draft_layers
        d.n_capture = len(dims.capture_layers)
        for i, l in enumerate(dims.capture_layers):
            d.capture_layers[i] = l
        d.relay_hidden = dims.d_h
        d.block, d.max_batch, d.max_rows = block, max_batch, max_rows
        d.max_pages, d.num_pages = self.max_pages, self.num_pages
        d.carry_window = CARRY_WINDOWS[carry_window]
        d.rope_theta, d.rms_eps, d.ln_eps = dims.rope_theta, dims.rms_eps, dims.ln_eps
        self.cdims = d

        up = self._upload
        W = Weights()
        W.embed = up(weights["embed"])
        # RMSNorm gains that precede a projection are folded into its packed weight
        W.lm_head = self._packed(weights["lm_head"], gain=weights["final_norm"])
        self.layers = (Layer * dims.n_layers)(*[self._layer(weights, f"layers.{l}") for l in range(dims.n_layers)])
        self.dlayers = (Layer * dims.n_draft_layers)(
            *[self._layer(weights, f"draft.layers.{l}") for l in range(dims.n_draft_layers)])
        W.layers = self.layers
        W.draft_layers = self.dlayers
        W.draft_lm_head = self._packed(weights["lm_head"], gain=weights["draft.final_norm"])
        # the context features enter each drafter layer's K/V without its attention norm
        W.draft_wkv_ctx = self._packed(np.concatenate(
            [np.concatenate([weights[f"draft.layers.{l}.wk"], weights[f"draft.layers.{l}.wv"]])
             for l in range(dims.n_draft_layers)]))
        W.e_mask = up(weights["draft.e_mask"])
        W.w_c = self._packed(weights["draft.w_c"])
        W.g_c = up(weights["draft.g_c"])
        W.relay_w1 = self._packed(weights["relay.w1"])
        W.relay_c1 = up(weights["relay.c1"])
        W.relay_w2 = self._packed(weights["relay.w2"])
        W.relay_c2 = up(weights["relay.c2"])
        W.relay_ln_g = up(weights["relay.ln_g"])
        W.relay_ln_b = up(weights["relay.ln_b"])
        self.cweights = W

        pool = self.num_pages * dims.n_kv_heads * PAGE * dims.head_dim
        z = lambda n: torch.zeros(n, dtype=self.elt_torch, device=self.device)
        self.k_pool, self.v_pool = z(dims.n_layers * pool), z(dims.n_layers * pool)
        self.ck_pool, self.cv_pool = z(dims.n_draft_layers * pool), z(dims.n_draft_layers * pool)
        pt = np.arange(self.num_pages, dtype=np.int32).reshape(max_batch, self.max_pages)
        self.page_table = torch.from_numpy(pt).to(self.device)
        C = Cache()
        C.k_pool, C.v_pool = self.k_pool.data_ptr(), self.v_pool.data_ptr()
        C.ck_pool, C.cv_pool = self.ck_pool.data_ptr(), self.cv_pool.data_ptr()
        C.page_table = self.page_table.data_ptr()
        self.ccache = C
        # workspace and status word: device memory owned here (torch), registered with the context
        ws_bytes = int(self.lib.dflow_workspace_bytes(ctypes.byref(d)))
        if ws_bytes == 0:
            self._check(-2, "dflow_workspace_bytes")
        self.workspace = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=self.device)
        self.status_word = torch.zeros(1, dtype=torch.int32, device=self.device)
        ws_ptr = (self.workspace.data_ptr() + 255) // 256 * 256
        torch.cuda.synchronize(self.device)
        ctx = ctypes.c_void_p()
        self._check(self.lib.dflow_create(ctypes.byref(d), ctypes.byref(W), ctypes.byref(C), ws_ptr, ws_bytes,
                                          self.status_word.data_ptr(), _stream(), ctypes.byref(ctx)), "dflow_create")
        self.ctx = ctx

    # ------------------------------------------------------------ weights
    def _upload(self, a: np.ndarray):
        t = self._to_dev(a)
        self._keep.append(t)
        return t.data_ptr()

    def _to_dev(self, a: np.ndarray):
        torch = self.torch
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(self.device)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.device)

    def _packed(self, a: np.ndarray, gate_up: int = 0, gain: Optional[np.ndarray] = None):
        N, K = a.shape
        src = self._to_dev(a)
        g = self._to_dev(gain) if gain is not None else None
        out = self.torch.empty_like(src)
        self._check(self.lib.dflow_pack_linear(_stream(), self.dtype_code, src.data_ptr(), N, K, gate_up,
                                               g.data_ptr() if g is not None else None, out.data_ptr()),
                    "dflow_pack_linear")
        self.torch.cuda.current_stream().synchronize()
        del src, g
        self._keep.append(out)
        return out.data_ptr()

    def _layer(self, w, p) -> Layer:
        L = Layer()
        L.wqkv = self._packed(np.concatenate([w[f"{p}.wq"], w[f"{p}.wk"], w[f"{p}.wv"]]),
                              gain=w[f"{p}.attn_norm"])
        L.q_norm = self._upload(w[f"{p}.q_norm"])
        L.k_norm = self._upload(w[f"{p}.k_norm"])
        L.wo = self._packed(w[f"{p}.wo"])
        L.wgu = self._packed(np.concatenate([w[f"{p}.w_gate"], w[f"{p}.w_up"]]), gate_up=1,
                             gain=w[f"{p}.ffn_norm"])
        L.wdown = self._packed(w[f"{p}.w_down"])
        return L

    # ------------------------------------------------------------ calls
    def _check(self, rc: int, what: str):
        if rc != 0:
            msg = self.lib.dflow_last_error().decode()
            raise DFlowError(f"{what} failed ({rc}): {msg}")

    def prefill(self, seq: int, tokens, first_anchor):
        self._check(self.lib.dflow_prefill(self.ctx, _stream(), seq, _ptr(tokens), int(tokens.numel()),
                                           _ptr(first_anchor)), "dflow_prefill")

    def prefill_batch(self, tokens, lengths, first_anchor):
        """tokens: device int32 prompts back to back; lengths: host ints; first_anchor: device int32 [nseq]."""
        n = len(lengths)
        lens = (ctypes.c_int32 * n)(*[int(x) for x in lengths])
        self._check(self.lib.dflow_prefill_batch(self.ctx, _stream(), n, _ptr(tokens), lens, _ptr(first_anchor)),
                    "dflow_prefill_batch")

    def draft_block(self, nseq, anchor_tok, anchor_pos, carry_on, draft_tok=None, block_out=None, draft_logits=None):
        self._check(self.lib.dflow_draft_block(self.ctx, _stream(), nseq, _ptr(anchor_tok), _ptr(anchor_pos),
                                               int(bool(carry_on)), _ptr(draft_tok), _ptr(block_out),
                                               _ptr(draft_logits)), "dflow_draft_block")

    def verify_block(self, nseq, block_tok, start_pos, tgt_argmax, logits=None, hcap=None):
        self._check(self.lib.dflow_verify_block(self.ctx, _stream(), nseq, _ptr(block_tok), _ptr(start_pos),
                                                _ptr(tgt_argmax), _ptr(logits), _ptr(hcap)), "dflow_verify_block")

    def accept_and_carry(self, nseq, block_tok, tgt_argmax, accept_len, bonus, committed, n_carry, feat=None):
        self._check(self.lib.dflow_accept_and_carry(self.ctx, _stream(), nseq, _ptr(block_tok), _ptr(tgt_argmax),
                                                    _ptr(accept_len), _ptr(bonus), _ptr(committed), _ptr(n_carry),
                                                    _ptr(feat)), "dflow_accept_and_carry")

    @staticmethod
    def sampler(temperature: float, seed: int, stream) -> Sampler:
        """stream: device uint64 (torch int64) tensor of per-sequence stream ids, kept alive by the caller."""
        return Sampler(float(temperature), int(seed) & (2**64 - 1), _ptr(stream))

    def prefill_sampled(self, seq: int, tokens, sampler, first_token):
        """sampler.stream must point at this sequence's one stream id."""
        self._check(self.lib.dflow_prefill_sampled(self.ctx, _stream(), seq, _ptr(tokens), int(tokens.numel()),
                                                   ctypes.byref(sampler), _ptr(first_token)),
                    "dflow_prefill_sampled")

    def sample_draft(self, nseq, draft_logits, anchor_tok, anchor_pos, sampler, draft_tok, block_out=None):
        self._check(self.lib.dflow_sample_draft(self.ctx, _stream(), nseq, _ptr(draft_logits), _ptr(anchor_tok),
                                                _ptr(anchor_pos), ctypes.byref(sampler), _ptr(draft_tok),
                                                _ptr(block_out)), "dflow_sample_draft")

    def sample_draft_noalloc(self, nseq, draft_logits, anchor_tok, anchor_pos, sampler, draft_tok, block_out=None):
        """dflow_sample_draft with the draw keys in the library's fixed device scratch (no workspace)."""
        self._check(self.lib.dflow_sample_draft_noalloc(self.ctx, _stream(), nseq, _ptr(draft_logits),
                                                        _ptr(anchor_tok), _ptr(anchor_pos), ctypes.byref(sampler),
                                                        _ptr(draft_tok), _ptr(block_out)),
                    "dflow_sample_draft_noalloc")

    def accept_sampled(self, nseq, block_tok, anchor_pos, logits, draft_logits, sampler, accept_len, bonus,
                       committed, n_carry, feat=None):
        self._check(self.lib.dflow_accept_sampled(self.ctx, _stream(), nseq, _ptr(block_tok), _ptr(anchor_pos),
                                                  _ptr(logits), _ptr(draft_logits), ctypes.byref(sampler),
                                                  _ptr(accept_len), _ptr(bonus), _ptr(committed), _ptr(n_carry),
                                                  _ptr(feat)), "dflow_accept_sampled")

    def trajectory_targets(self, nseq, traj, traj_len, start_pos, tgt):
        self._check(self.lib.dflow_trajectory_targets(self.ctx, _stream(), nseq, _ptr(traj), int(traj.shape[1]),
                                                      int(traj_len), _ptr(start_pos), _ptr(tgt)),
                    "dflow_trajectory_targets")

    def draft_loss(self, nseq, draft_logits, traj, traj_len, start_pos, gamma, loss):
        self._check(self.lib.dflow_draft_loss(self.ctx, _stream(), nseq, _ptr(draft_logits), _ptr(traj),
                                              int(traj.shape[1]), int(traj_len), _ptr(start_pos), float(gamma),
                                              _ptr(loss)), "dflow_draft_loss")

    def kv_commit(self, nseq, accept_len, seq_len):
        self._check(self.lib.kv_commit(self.ctx, _stream(), nseq, _ptr(accept_len), _ptr(seq_len)), "kv_commit")

    @property
    def qkv_parts(self) -> int:
        """K parts of the QKV projection (fp32 partial sums added by its consumers)."""
        return int(self.lib.dflow_qkv_parts(self.ctx))

    @property
    def attention_split(self) -> tuple:
        """(keys per LDS chunk, chunks per attention split) of the round calls."""
        ck, nc = ctypes.c_int(), ctypes.c_int()
        self._check(self.lib.dflow_attention_split(self.ctx, ctypes.byref(ck), ctypes.byref(nc)),
                    "dflow_attention_split")
        return ck.value, nc.value

    def move_slot(self, src: int, dst: int):
        self._check(self.lib.dflow_move_slot(self.ctx, _stream(), int(src), int(dst)), "dflow_move_slot")

    def force_drafts(self, nseq, traj, traj_len, mode, tok, anchor, start_pos, block_tok):
        self._check(self.lib.dflow_bench_force_drafts(self.ctx, _stream(), nseq, _ptr(traj), int(traj.shape[1]),
                                                      traj_len, _ptr(mode), _ptr(tok), _ptr(anchor),
                                                      _ptr(start_pos), _ptr(block_tok)), "dflow_bench_force_drafts")

    def status(self, clear: bool = True) -> int:
        out = ctypes.c_int32(0)
        self._check(self.lib.dflow_read_status(self.ctx, _stream(), ctypes.byref(out), int(clear)),
                    "dflow_read_status")
        return out.value

    def profile(self, enable: bool):
        self._check(self.lib.dflow_profile(self.ctx, int(bool(enable))), "dflow_profile")

    def profile_read(self):
        """List of dicts (name, N, K, M, phase, launches, ms, bytes) per kernel class and issuing entry point."""
        buf = (ProfEntry * 128)()
        n = ctypes.c_int(0)
        self._check(self.lib.dflow_profile_read(self.ctx, buf, 128, ctypes.byref(n)), "dflow_profile_read")
        return [{"name": e.name.decode(), "N": e.N, "K": e.K, "M": e.M, "phase": PHASES.get(e.phase, str(e.phase)),
                 "launches": e.launches, "ms": e.ms, "bytes": e.bytes} for e in buf[:min(n.value, 128)]]

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.dflow_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
