"""Oracle model primitives, target forward and drafter forward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The target is the Qwen3 decoder evaluated in the paper (Sec. 5.1): RMSNorm,
per-head RMSNorm of q and k (QK-norm), rotate-half RoPE with theta = 1e6 at
absolute positions, grouped-query attention, SwiGLU feed-forward, no biases.
The drafter is the block-diffusion drafter of Sec. 3 (eq. dflash_drafting)
whose key and value projections in every layer also take the fused target
feature (Sec. 3, text after eq. dflash_context).

Pins (tests/test_oracle_pins.py, tests/test_oracle_primitives.py):
  * target_block / logits: transformers.Qwen3ForCausalLM on CPU with the same
    weights (fp64), plus block-vs-stepwise-vs-full-recompute agreement;
  * attention with all keys visible: torch scaled_dot_product_attention;
  * layer_norm: torch.nn.functional.layer_norm;
  * relay MLP: torch Linear -> SiLU -> Linear with the same weights;
  * drafter numeric values as a whole: parity unpinned (no published values).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from workload.configs import ModelDims
from workload.synth import bf16_bits_to_f32

from .numerics import Mode


class OracleModel:
    def __init__(self, dims: ModelDims, raw: Dict[str, np.ndarray], mode: Mode, cache: bool = True):
        self.dims = dims
        self.raw = raw
        self.mode = mode
        self.cache = cache
        self._conv: Dict[str, np.ndarray] = {}
        Dh = dims.head_dim
        # RoPE inverse frequencies theta^(-2i/Dh), i < Dh/2, in fp64
        self.inv_freq = dims.rope_theta ** (-(np.arange(0, Dh // 2, dtype=np.float64) * 2.0) / Dh)

    # ------------------------------------------------------------ weights
    def w(self, name: str) -> np.ndarray:
        if name in self._conv:
            return self._conv[name]
        a = self.raw[name]
        if a.dtype == np.uint16:
            a = bf16_bits_to_f32(a)
        a = np.asarray(a, dtype=self.mode.dt)
        if self.cache:
            self._conv[name] = a
        return a

    # ------------------------------------------------------------ primitives
    def rms_norm(self, x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
        """x * (mean(x^2) + eps)^(-1/2) * g over the last axis."""
        dt = self.mode.dt
        x = np.asarray(x, dtype=dt)
        ms = np.mean(x * x, axis=-1, keepdims=True)
        return x / np.sqrt(ms + dt(eps)) * g

    def layer_norm(self, x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
        """LayerNorm over the last axis with biased variance, gain and bias."""
        dt = self.mode.dt
        x = np.asarray(x, dtype=dt)
        mu = np.mean(x, axis=-1, keepdims=True)
        var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
        return (x - mu) / np.sqrt(var + dt(eps)) * g + b

    def silu(self, x: np.ndarray) -> np.ndarray:
        return x / (self.mode.dt(1) + np.exp(-x))

    def linear(self, x: np.ndarray, wname: str) -> np.ndarray:
        return np.asarray(x, dtype=self.mode.dt) @ self.w(wname).T

    def rope(self, x: np.ndarray, pos: np.ndarray) -> np.ndarray:
        """Rotate-half RoPE: pair (i, i + Dh/2) rotated by angle pos * inv_freq[i].
        x: [n, H, Dh], pos: [n]."""
        ang = np.asarray(pos, dtype=np.float64)[:, None] * self.inv_freq[None, :]
        cos = np.cos(ang).astype(self.mode.dt)[:, None, :]
        sin = np.sin(ang).astype(self.mode.dt)[:, None, :]
        h = x.shape[-1] // 2
        x1, x2 = x[..., :h], x[..., h:]
        return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)

    def attention(self, q: np.ndarray, k: np.ndarray, v: np.ndarray, visible: np.ndarray) -> np.ndarray:
        """softmax(q k^T / sqrt(Dh)) v per query head; head h reads KV head
        floor(h * Hkv / Hq), i.e. the G = Hq / Hkv consecutive query heads of
        a group share one KV head.  q: [n, Hq, Dh]; k, v: [m, Hkv, Dh];
        visible: [n, m] bool.  Returns [n, Hq * Dh].  Evaluated one KV head
        at a time (one group of query heads) to bound the score arrays."""
        dm = self.dims
        dt = self.mode.dt
        n, Hq, Dh = q.shape
        G = Hq // dm.n_kv_heads
        hidden = ~np.asarray(visible, bool)
        out = np.empty((n, Hq, Dh), dt)
        for j in range(dm.n_kv_heads):
            qj = np.ascontiguousarray(q[:, j * G:(j + 1) * G, :].transpose(1, 0, 2))   # [G, n, Dh]
            s = np.matmul(qj, np.ascontiguousarray(k[:, j, :].T))                      # [G, n, m]
            np.divide(s, dt(np.sqrt(Dh)), out=s)
            s[:, hidden] = -np.inf
            s -= s.max(axis=-1, keepdims=True)
            np.exp(s, out=s)
            s /= s.sum(axis=-1, keepdims=True)
            out[:, j * G:(j + 1) * G, :] = np.matmul(s, np.ascontiguousarray(v[:, j, :])).transpose(1, 0, 2)
        return out.reshape(n, Hq * Dh)

    # ------------------------------------------------------------ decoder layer pieces
    def _qkv(self, prefix: str, h: np.ndarray, pos: np.ndarray):
        dm, st = self.dims, self.mode.st
        n = h.shape[0]
        q = st(self.linear(h, f"{prefix}.wq")).reshape(n, dm.n_heads, dm.head_dim)
        k = st(self.linear(h, f"{prefix}.wk")).reshape(n, dm.n_kv_heads, dm.head_dim)
        v = st(self.linear(h, f"{prefix}.wv")).reshape(n, dm.n_kv_heads, dm.head_dim)
        q = st(self.rope(self.rms_norm(q, self.w(f"{prefix}.q_norm"), dm.rms_eps), pos))
        k = st(self.rope(self.rms_norm(k, self.w(f"{prefix}.k_norm"), dm.rms_eps), pos))
        return q, k, v

    def _ffn(self, prefix: str, x: np.ndarray) -> np.ndarray:
        st = self.mode.st
        h = st(self.rms_norm(x, self.w(f"{prefix}.ffn_norm"), self.dims.rms_eps))
        a = st(self.silu(self.linear(h, f"{prefix}.w_gate")) * self.linear(h, f"{prefix}.w_up"))
        return st(x + self.linear(a, f"{prefix}.w_down"))

    def decoder_layer(self, prefix: str, x: np.ndarray, pos: np.ndarray,
                      k_past: np.ndarray, v_past: np.ndarray, past_pos: np.ndarray,
                      causal: bool):
        """One Qwen3-style decoder layer over n rows.  Keys are the past
        entries followed by the rows' own keys.  causal: row i sees keys at
        positions <= pos[i]; otherwise it sees every key.
        Returns (x_out, k_rows, v_rows)."""
        st = self.mode.st
        h = st(self.rms_norm(x, self.w(f"{prefix}.attn_norm"), self.dims.rms_eps))
        q, k, v = self._qkv(prefix, h, pos)
        K = np.concatenate([k_past, k], axis=0)
        Vv = np.concatenate([v_past, v], axis=0)
        kpos = np.concatenate([past_pos, pos])
        if causal:
            visible = kpos[None, :] <= pos[:, None]
        else:
            visible = np.ones((len(pos), len(kpos)), dtype=bool)
        o = st(self.attention(q, K, Vv, visible))
        x = st(x + self.linear(o, f"{prefix}.wo"))
        return self._ffn(prefix, x), k, v

    # ------------------------------------------------------------ target
    def embed(self, tokens: Sequence[int]) -> np.ndarray:
        return self.w("embed")[np.asarray(tokens, dtype=np.int64)]

    def logits(self, x: np.ndarray, norm: str) -> np.ndarray:
        """LM head over the final-normed rows (fp32 logits in bf16 mode)."""
        h = self.mode.st(self.rms_norm(x, self.w(norm), self.dims.rms_eps))
        return self.linear(h, "lm_head")

    def target_block(self, tokens: Sequence[int], pos0: int,
                     k_cache: List[np.ndarray], v_cache: List[np.ndarray], logit_rows: slice = slice(None)):
        """Causal target forward of rows tokens[j] at positions pos0 + j against
        a cache holding positions 0..pos0-1 of every layer.
        Returns (logits of the rows logit_rows selects (all by default) [n', V],
        k_rows[L], v_rows[L], hidden[L] residual outputs)."""
        dm = self.dims
        n = len(tokens)
        pos = np.arange(pos0, pos0 + n)
        x = self.embed(tokens)
        ks, vs, hid = [], [], []
        for l in range(dm.n_layers):
            past_pos = np.arange(k_cache[l].shape[0])
            x, k, v = self.decoder_layer(f"layers.{l}", x, pos, k_cache[l], v_cache[l], past_pos, True)
            ks.append(k)
            vs.append(v)
            hid.append(x)
        return self.logits(x[logit_rows], "final_norm"), ks, vs, hid

    # ------------------------------------------------------------ drafter
    def fuse(self, hcat: np.ndarray) -> np.ndarray:
        """Fused target feature RMSNorm(W_c [H^l1; ...; H^lm]) (Sec. 3, eq.
        dflash_context); also the verifier-state alignment of Sec. 4.2, which
        reuses W_c and the RMSNorm.  hcat: [n, m*d]."""
        return self.mode.st(self.rms_norm(self.linear(hcat, "draft.w_c"), self.w("draft.g_c"),
                                          self.dims.rms_eps))

    def ctx_kv(self, l: int, F: np.ndarray, pos: np.ndarray):
        """Key/value rows that the fused features contribute to drafter layer l
        (Sec. 3: the feature feeds the key and value projections of each draft
        layer).  The feature is already RMS-normalised by the fusion."""
        dm, st = self.dims, self.mode.st
        p = f"draft.layers.{l}"
        n = F.shape[0]
        k = st(self.linear(F, f"{p}.wk")).reshape(n, dm.n_kv_heads, dm.head_dim)
        v = st(self.linear(F, f"{p}.wv")).reshape(n, dm.n_kv_heads, dm.head_dim)
        k = st(self.rope(self.rms_norm(k, self.w(f"{p}.k_norm"), dm.rms_eps), pos))
        return k, v

    def drafter_block(self, x: np.ndarray, pos0: int,
                      ctx_k: List[np.ndarray], ctx_v: List[np.ndarray]) -> np.ndarray:
        """One parallel drafter forward (Sec. 3, eq. dflash_drafting) over the
        B block rows at positions pos0..pos0+B-1.  Every row attends to the
        context keys (positions < pos0) and to every row of the block.
        Returns logits [B, V]."""
        dm = self.dims
        B = x.shape[0]
        pos = np.arange(pos0, pos0 + B)
        for l in range(dm.n_draft_layers):
            past_pos = np.arange(ctx_k[l].shape[0])
            x, _, _ = self.decoder_layer(f"draft.layers.{l}", x, pos, ctx_k[l], ctx_v[l], past_pos, False)
        return self.logits(x, "draft.final_norm")

    def relay(self, bonus: int, y_rej: int, h: np.ndarray) -> np.ndarray:
        """Reject-conditioned draft initialisation (Sec. 4.2):
        [beta; gamma] = MLP_phi([E(b); E(y_rej); h_i])   (eq. reject_conditioning)
        x_i = E_mask + beta * LN(h_i) + gamma             (eq. dflow_input)
        h: [n_c, d] aligned verifier representations.  Returns [n_c, d]."""
        dm, st = self.dims, self.mode.st
        d, n = dm.d, h.shape[0]
        E = self.w("embed")
        u = np.concatenate([np.repeat(E[bonus][None], n, 0), np.repeat(E[y_rej][None], n, 0),
                            np.asarray(h, dtype=self.mode.dt)], axis=1)
        hid = st(self.silu(self.linear(u, "relay.w1") + self.w("relay.c1")))
        bg = self.linear(hid, "relay.w2") + self.w("relay.c2")
        beta, gamma = bg[:, :d], bg[:, d:]
        ln = self.layer_norm(h, self.w("relay.ln_g"), self.w("relay.ln_b"), dm.ln_eps)
        return st(self.w("draft.e_mask")[None, :] + beta * ln + gamma)
