"""Oracle round algorithm of DFlow.

TEST INFRASTRUCTURE ONLY (see the package docstring).

State of one sequence: the committed tokens y_0..y_{n-1}; the anchor is the
last one, at position t = n-1; the target KV cache and the fused context
features F hold positions 0..t-1; the carry record holds the aligned
verifier representations of the previous round's rejected suffix.

One round (Sec. 3 and Sec. 4.2):
  1. draft   - drafter inputs [E(anchor), E_mask, ...] with relayed rows at
               the reusable positions (eq. dflow_input), one parallel drafter
               forward, argmax at block rows 1..K (eq. dflash_drafting);
  2. verify  - causal target forward of [anchor, d_1..d_K] at t..t+K;
  3. accept  - a = longest prefix with d_i == argmax of row i-1; the bonus
               is the target's prediction at the first rejection, or after
               the last row when every draft matches (eq.
               verification_partition and the text after it);
  4. project - f_j = RMSNorm(W_c [S^l1_j; ...; S^lm_j]) for every block row
               (eq. dflash_context; Sec. 4.2 projects the suffix jointly);
  5. commit  - keep KV and F for positions 0..t+a, append d_1..d_a and the
               bonus to the committed tokens (rollback = truncation);
  6. carry   - the verifier state at position q-1 predicts position q, so
               next-round block index i (position t+a+1+i) takes row a+i
               (Sec. 4.2, shift alignment); rows a+1..K-1 cover the rejected
               suffix positions t+a+2..t+K, so n_c = max(0, K-1-a).

At temperature T > 0 (round_sampled) steps 1 and 3 draw the drafts from the
drafter and accept them by speculative sampling (oracle.sampling); the other
steps are unchanged, the corrected token taking the bonus' place.

Pins: accept/commit/carry index maps are brute-forced and checked against
position arithmetic; the whole loop is pinned by losslessness against plain
greedy decoding and by KV/F equality with a fresh prefill
(tests/test_oracle_invariants.py).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from . import sampling
from .model import OracleModel

CARRY_WINDOWS = ("suffix", "suffix+tail", "suffix-inputs")


@dataclass
class Carry:
    n: int                      # number of relayed positions (block indices i0..i0+n-1)
    h: np.ndarray               # [n, d] aligned verifier representations
    bonus: int                  # b, the target correction at the first rejection
    y_rej: int                  # first rejected proposal d_{a+1}
    i0: int = 1                 # first relayed block index


@dataclass
class SeqState:
    tokens: List[int]
    k: List[np.ndarray]         # per target layer [t, Hkv, Dh]
    v: List[np.ndarray]
    F: np.ndarray               # [t, d] fused context features
    ck: List[np.ndarray]        # per drafter layer [t, Hkv, Dh] context keys
    cv: List[np.ndarray]
    carry: Optional[Carry] = None
    last_logits: Optional[np.ndarray] = None   # [V] logits of the prompt's last row (set by prefill)

    @property
    def t(self) -> int:
        return len(self.tokens) - 1

    @property
    def anchor(self) -> int:
        return self.tokens[-1]


@dataclass
class RoundResult:
    t: int                      # anchor position of the round
    x_in: np.ndarray            # [B, d] drafter input rows
    n_relay: int                # block indices 1..n_relay used relayed inputs
    draft: np.ndarray           # [K] drafter argmax d'_1..d'_K
    draft_logits: np.ndarray    # [K, V] drafter logits of rows 1..K
    block: np.ndarray           # [B] verified tokens [anchor, d_1..d_K]
    logits: np.ndarray          # [B, V] target logits
    g: np.ndarray               # [B] target argmax per row
    hcap: np.ndarray            # [B, m*d] captured verifier states
    f: np.ndarray               # [B, d] projected features
    a: int
    bonus: int
    committed: List[int]
    n_carry: int


def argmax_lowest(x: np.ndarray) -> np.ndarray:
    """Row-wise argmax; np.argmax returns the first (lowest) index on ties."""
    return np.argmax(x, axis=-1)


def forced_block(anchor: int, t: int, traj: np.ndarray, mode: np.ndarray, tok: np.ndarray, V: int) -> np.ndarray:
    """Measurement construct: the block fed to verification when drafts are
    forced from a target trajectory (mode 1), a guaranteed mismatch (mode 2)
    or a uniform token (mode 0).  Index 0 is always the anchor."""
    B = len(mode)
    out = np.empty(B, np.int64)
    out[0] = anchor
    for j in range(1, B):
        if mode[j] == 1:
            out[j] = traj[t + j]
        elif mode[j] == 2:
            out[j] = (int(traj[t + j]) + 1 + int(tok[j])) % V
        else:
            out[j] = tok[j]
    return out


class OracleDFlow:
    def __init__(self, model: OracleModel, block: int, carry_window: str = "suffix", prefill_chunk: int = 256):
        if carry_window not in CARRY_WINDOWS:
            raise ValueError(carry_window)
        self.m = model
        self.B = block
        self.K = block - 1
        self.carry_window = carry_window
        self.prefill_chunk = prefill_chunk

    # ------------------------------------------------------------ prefill
    def empty_state(self) -> SeqState:
        dm = self.m.dims
        dt = self.m.mode.dt
        e = lambda: np.zeros((0, dm.n_kv_heads, dm.head_dim), dt)
        return SeqState(tokens=[], k=[e() for _ in range(dm.n_layers)], v=[e() for _ in range(dm.n_layers)],
                        F=np.zeros((0, dm.d), dt), ck=[e() for _ in range(dm.n_draft_layers)],
                        cv=[e() for _ in range(dm.n_draft_layers)])

    def _append_target(self, s: SeqState, tokens: Sequence[int], keep: int, logit_rows: slice = slice(None)):
        """Run the target over tokens at positions t.. and keep the first
        `keep` rows in the caches; returns (logits of logit_rows, hcat, fused f)."""
        pos0 = s.k[0].shape[0]
        logits, ks, vs, hid = self.m.target_block(tokens, pos0, s.k, s.v, logit_rows)
        hcat = np.concatenate([hid[l] for l in self.m.dims.capture_layers], axis=1)
        f = self.m.fuse(hcat)
        for l in range(self.m.dims.n_layers):
            s.k[l] = np.concatenate([s.k[l], ks[l][:keep]])
            s.v[l] = np.concatenate([s.v[l], vs[l][:keep]])
        self._append_ctx(s, f[:keep])
        return logits, hcat, f

    def _append_ctx(self, s: SeqState, f: np.ndarray):
        t0 = s.F.shape[0]
        pos = np.arange(t0, t0 + f.shape[0])
        s.F = np.concatenate([s.F, f])
        for l in range(self.m.dims.n_draft_layers):
            k, v = self.m.ctx_kv(l, f, pos)
            s.ck[l] = np.concatenate([s.ck[l], k])
            s.cv[l] = np.concatenate([s.cv[l], v])

    def prefill(self, prompt: Sequence[int], sampler=None) -> SeqState:
        """Target KV and fused features for every prompt position; the first
        anchor is the target's greedy token after the prompt or, with
        sampler = (T, seed, stream), a draw from softmax(z / T) of the last
        row (oracle.sampling.sample_first)."""
        s = self.empty_state()
        prompt = [int(x) for x in prompt]
        logits = None
        for c in range(0, len(prompt), self.prefill_chunk):
            chunk = prompt[c:c + self.prefill_chunk]
            last = c + self.prefill_chunk >= len(prompt)   # only the prompt's last row is scored
            logits, _, _ = self._append_target(s, chunk, len(chunk), slice(-1, None) if last else slice(0, 0))
        if sampler is None:
            first = int(argmax_lowest(logits[-1]))
        else:
            T, seed, stream = sampler
            first = sampling.sample_first(logits[-1], sampling.inv_temperature(T), seed, stream, len(prompt) - 1)
        s.tokens = prompt + [first]
        s.last_logits = np.asarray(logits[-1])
        return s

    # ------------------------------------------------------------ round steps
    def draft_inputs(self, s: SeqState, carry_on: bool):
        """Drafter input rows: E(anchor) at index 0, mask embedding elsewhere,
        and relayed verifier information at the reusable positions
        (Sec. 4.2, eq. dflow_input; plain masks in the first round, when the
        suffix is empty, or when relay is disabled)."""
        dm = self.m.dims
        x = np.repeat(self.m.w("draft.e_mask")[None, :], self.B, axis=0).astype(self.m.mode.dt)
        x[0] = self.m.embed([s.anchor])[0]
        n_relay = 0
        c = s.carry
        if carry_on and c is not None and c.n > 0:
            x[c.i0:c.i0 + c.n] = self.m.relay(c.bonus, c.y_rej, c.h)
            n_relay = c.n
        return x, n_relay

    def draft(self, s: SeqState, carry_on: bool):
        x, n_relay = self.draft_inputs(s, carry_on)
        lg = self.m.drafter_block(x, s.t, s.ck, s.cv)[1:]
        return argmax_lowest(lg), lg, x, n_relay

    def verify(self, s: SeqState, block: Sequence[int]):
        """Target forward of the block at positions t..t+K (no cache update)."""
        logits, ks, vs, hid = self.m.target_block(block, s.t, s.k, s.v)
        hcat = np.concatenate([hid[l] for l in self.m.dims.capture_layers], axis=1)
        return logits, argmax_lowest(logits), hcat, ks, vs

    @staticmethod
    def accept(block: Sequence[int], g: Sequence[int]):
        """a = number of leading proposals equal to the target's prediction at
        the previous row; bonus = g[a]; committed = d_1..d_a, bonus."""
        K = len(block) - 1
        a = 0
        while a < K and int(block[a + 1]) == int(g[a]):
            a += 1
        bonus = int(g[a])
        return a, bonus, [int(x) for x in block[1:a + 1]] + [bonus]

    def carry_map(self, a: int):
        """(n_c, source block rows) of the relay for acceptance length a.
        Next-round block index i takes the verify row a+i (the row whose
        position predicts the index's position); the window picks the rows:
        'suffix' a+1..K-1 (predictions of the rejected-suffix positions),
        'suffix+tail' a+1..K (also the prediction after the block),
        'suffix-inputs' a+2..K (the rows whose inputs are the rejected suffix;
        index 1 keeps the mask)."""
        K = self.K
        lo, hi = {"suffix": (a + 1, K - 1), "suffix+tail": (a + 1, K), "suffix-inputs": (a + 2, K)}[self.carry_window]
        rows = list(range(lo, hi + 1))
        return len(rows), rows

    def round(self, s: SeqState, carry_on: bool = True, block: Optional[Sequence[int]] = None,
              force=None, decide: Optional[Sequence[int]] = None) -> RoundResult:
        """One drafting/verification round.  `block` replaces the verified
        tokens; `force=(traj, mode, tok)` builds them with forced_block.  The
        drafter runs in full either way.  `decide(a, bonus, logits)` may
        replace the acceptance outcome; parity tests use it to follow the
        device through a near-tie that the numerical tolerance cannot
        decide."""
        t = s.t
        d, dlg, x, n_relay = self.draft(s, carry_on)
        if block is None and force is not None:
            traj, mode, tok = force
            block = forced_block(s.anchor, t, traj, mode, tok, self.m.dims.vocab)
        if block is None:
            block = np.concatenate([[s.anchor], d])
        block = np.asarray(block, dtype=np.int64)
        assert block[0] == s.anchor and len(block) == self.B
        logits, g, hcat, ks, vs = self.verify(s, block)
        a, bonus, committed = self.accept(block, g)
        if decide is not None:
            a, bonus = (int(v) for v in decide(a, bonus, logits))
            committed = [int(x) for x in block[1:a + 1]] + [bonus]
        f, n_c = self._commit(s, block, a, committed, hcat, ks, vs)
        return RoundResult(t=t, x_in=x, n_relay=n_relay, draft=d, draft_logits=dlg, block=block, logits=logits,
                           g=g, hcap=hcat, f=f, a=a, bonus=bonus, committed=committed, n_carry=n_c)

    def _commit(self, s: SeqState, block, a: int, committed, hcat, ks, vs):
        """Keep positions t..t+a in the caches (t+a+1.. are rolled back),
        append the committed tokens and record the relay of the suffix."""
        f = self.m.fuse(hcat)
        for l in range(self.m.dims.n_layers):
            s.k[l] = np.concatenate([s.k[l], ks[l][:a + 1]])
            s.v[l] = np.concatenate([s.v[l], vs[l][:a + 1]])
        self._append_ctx(s, f[:a + 1])
        s.tokens += committed
        n_c, rows = self.carry_map(a)
        s.carry = Carry(n_c, f[rows].copy(), committed[-1], int(block[a + 1]) if a < self.K else -1,
                        rows[0] - a if rows else 1)
        return f, n_c

    def round_sampled(self, s: SeqState, temperature: float, seed: int, stream: int, carry_on: bool = True,
                      draft: Optional[Sequence[int]] = None, decide=None):
        """One round decoded by speculative sampling at temperature T (see
        oracle.sampling): the drafter samples its block, verification keeps
        the target's distribution.  `draft` replaces the sampled drafts and
        `decide(dec)` the (a, token) outcome; parity tests use them to follow
        the device through decisions within the numerical tolerance.
        Returns (RoundResult, drafter z-scores, drafter Gumbel noise,
        SampledDecision)."""
        t = s.t
        inv_t = sampling.inv_temperature(temperature)
        x, n_relay = self.draft_inputs(s, carry_on)
        dlg = self.m.drafter_block(x, t, s.ck, s.cv)[1:]
        d, zq, gq = sampling.sample_drafts(dlg, inv_t, seed, stream, t)
        if draft is not None:
            d = np.asarray(draft, np.int64)
        block = np.concatenate([[s.anchor], d]).astype(np.int64)
        logits, g, hcat, ks, vs = self.verify(s, block)
        dec = sampling.accept_sampled(block, logits, dlg, inv_t, seed, stream, t)
        a, bonus = dec.a, dec.bonus
        if decide is not None:
            a, bonus = (int(v) for v in decide(dec))
        committed = [int(v) for v in block[1:a + 1]] + [bonus]
        f, n_c = self._commit(s, block, a, committed, hcat, ks, vs)
        res = RoundResult(t=t, x_in=x, n_relay=n_relay, draft=d, draft_logits=dlg, block=block, logits=logits,
                          g=g, hcap=hcat, f=f, a=a, bonus=bonus, committed=committed, n_carry=n_c)
        return res, zq, gq, dec

    # ------------------------------------------------------------ plain greedy (losslessness reference)
    def greedy_decode(self, prompt: Sequence[int], n_new: int) -> List[int]:
        """Plain autoregressive greedy decoding with an incremental KV cache."""
        dm = self.m.dims
        dt = self.m.mode.dt
        e = lambda: np.zeros((0, dm.n_kv_heads, dm.head_dim), dt)
        k = [e() for _ in range(dm.n_layers)]
        v = [e() for _ in range(dm.n_layers)]
        toks = [int(x) for x in prompt]
        lg, ks, vs, _ = self.m.target_block(toks, 0, k, v)
        k = [np.concatenate([k[l], ks[l]]) for l in range(dm.n_layers)]
        v = [np.concatenate([v[l], vs[l]]) for l in range(dm.n_layers)]
        out = []
        nxt = int(argmax_lowest(lg[-1]))
        while len(out) < n_new:
            out.append(nxt)
            lg, ks, vs, _ = self.m.target_block([nxt], len(toks) + len(out) - 1, k, v)
            k = [np.concatenate([k[l], ks[l]]) for l in range(dm.n_layers)]
            v = [np.concatenate([v[l], vs[l]]) for l in range(dm.n_layers)]
            nxt = int(argmax_lowest(lg[-1]))
        return out

    def full_logits(self, tokens: Sequence[int]) -> np.ndarray:
        """No-cache causal forward over the whole sequence."""
        dm = self.m.dims
        dt = self.m.mode.dt
        e = lambda: np.zeros((0, dm.n_kv_heads, dm.head_dim), dt)
        lg, _, _, _ = self.m.target_block(list(tokens), 0, [e() for _ in range(dm.n_layers)],
                                          [e() for _ in range(dm.n_layers)])
        return lg
