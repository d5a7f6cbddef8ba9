"""Speculative sampling at temperature T > 0 for the oracle round.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper reports sampling decoding at T = 1 next to greedy decoding (Table 1)
and, for the verification rule, relies on speculative decoding as introduced
by Leviathan, Kalman and Matias (ICML 2023, cited in Sec. 1), whose rule keeps
the output distribution of the target exactly.  For one block with anchor at
position t, target distributions p_0..p_K (block rows 0..K of the verify
forward) and drafter distributions q_1..q_K (block rows 1..K of the drafter
forward), all softmax(logits / T):
  * draft   d_i ~ q_i for i = 1..K (the drafter samples its block);
  * accept  d_i while u_i < p_{i-1}(d_i) / q_i(d_i), u_i uniform in (0, 1);
            a = number of leading accepted drafts (the same alignment as
            greedy verification: row i-1 of the verify forward scores d_i);
  * correct at the first rejection (a < K) the token at block index a+1 is
            drawn from the positive part of p_a - q_{a+1}, normalised; when
            every draft is accepted (a = K) the bonus is drawn from p_K.
The committed tokens d_1..d_a, bonus then have the distribution of sampling
the target token by token.

Random numbers: Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011), a counter-based generator,
implemented here from its definition: key (k0, k1), counter (c0..c3); ten
rounds, each two 64x64 -> 128-bit products of c0 and c2 by the round
multipliers, recombined with c1, c3 and the key, and the key advanced by the
Weyl increments between rounds.  A draw is addressed by key = (seed, stream
of the sequence) and counter = (t, block index, purpose, column // 4), using
output word column % 4; purposes: 0 = drafter sample, 1 = acceptance test,
2 = correction / bonus sample.  A 64-bit word x gives
u = ((x >> 41) + 1/2) * 2^-23, exact in fp32 and strictly inside (0, 1).

Arithmetic, all fp32 (the precision of the device path):
  z = logits * (1/T)  with 1/T rounded to fp32 once;
  lse(z) = max z + log(sum exp(z - max z));   log p = z - lse(z);
  sampling with log-weights w: argmax_v (w_v + g_v), g_v = -log(-log u_v)
  (the Gumbel-max trick), lowest index on ties; drafts use w = z_q, the bonus
  w = z_p;
  acceptance: log u_i < log p_{i-1}(d_i) - log q_i(d_i);
  correction: w_v = log(p_a(v) - q_{a+1}(v)) where positive, else -inf; if
  no column is positive (rounding only; p = q exactly rejects nothing) the
  correction is drawn from p_a.

Pins (tests/test_oracle_sampling.py): Philox against numpy's Philox bit
generator; the rule by the exact output distribution, which must equal p for
arbitrary p and q (a dropped min, an unnormalised or wrong residual fails
it); the implemented block rule by chi-square tests of the emitted tokens
over many streams against p_0 and, after an acceptance, p_1; the Gumbel-max
sampler against softmax(z).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence, Tuple

import numpy as np

M64 = (1 << 64) - 1
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B

DRAFT, ACCEPT, RESAMPLE = 0, 1, 2


# ------------------------------------------------------------------ Philox4x64-10
def philox4x64_10(key: Tuple[int, int], ctr: Tuple[int, int, int, int]) -> Tuple[int, int, int, int]:
    """One block with Python integers (the definition written out)."""
    k0, k1 = key[0] & M64, key[1] & M64
    c0, c1, c2, c3 = (c & M64 for c in ctr)
    for r in range(10):
        if r > 0:
            k0 = (k0 + PHILOX_W0) & M64
            k1 = (k1 + PHILOX_W1) & M64
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> 64, p0 & M64
        hi1, lo1 = p1 >> 64, p1 & M64
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a: int, b: np.ndarray):
    """(high, low) 64-bit halves of the 128-bit product a * b, a a constant."""
    b = np.asarray(b, np.uint64)
    a_lo, a_hi = np.uint64(a & 0xFFFFFFFF), np.uint64(a >> 32)
    b_lo, b_hi = b & _M32, b >> _S32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> _S32) + (lh & _M32) + (hl & _M32)
    hi = hh + (lh >> _S32) + (hl >> _S32) + (mid >> _S32)
    lo = (mid << _S32) | (ll & _M32)
    return hi, lo


def philox_np(k0, k1, c0, c1, c2, c3) -> np.ndarray:
    """The same block vectorised over broadcast uint64 arrays; [..., 4]."""
    with np.errstate(over="ignore"):
        k0, k1, c0, c1, c2, c3 = np.broadcast_arrays(*(np.asarray(v, np.uint64) for v in (k0, k1, c0, c1, c2, c3)))
        k0, k1 = k0.copy(), k1.copy()
        for r in range(10):
            if r > 0:
                k0 = k0 + np.uint64(PHILOX_W0)
                k1 = k1 + np.uint64(PHILOX_W1)
            hi0, lo0 = _mulhilo(PHILOX_M0, c0)
            hi1, lo1 = _mulhilo(PHILOX_M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1)


def uniform_from_bits(x) -> np.ndarray:
    x = np.asarray(x, np.uint64)
    return (((x >> np.uint64(41)).astype(np.float64) + 0.5) * 2.0 ** -23).astype(np.float32)


def uniforms(seed: int, stream: int, pos: int, row: int, purpose: int, n: int) -> np.ndarray:
    """u[v] for columns v = 0..n-1 of one (position, block index, purpose)."""
    blocks = philox_np(seed, stream, pos, row, purpose, np.arange((n + 3) // 4, dtype=np.uint64))
    return uniform_from_bits(blocks.reshape(-1)[:n])


def gumbel(u: np.ndarray) -> np.ndarray:
    u = np.asarray(u, np.float32)
    return (-np.log(-np.log(u))).astype(np.float32)


# ------------------------------------------------------------------ distributions (fp32)
def inv_temperature(temperature: float) -> np.float32:
    if not (temperature > 0 and np.isfinite(temperature)):
        raise ValueError("temperature must be positive and finite")
    return np.float32(1.0) / np.float32(temperature)


def scaled(logits: np.ndarray, inv_t: np.float32) -> np.ndarray:
    return (np.asarray(logits, np.float32) * np.float32(inv_t)).astype(np.float32)


def lse(z: np.ndarray) -> np.ndarray:
    """Row-wise log-sum-exp in fp32 (max-shifted)."""
    z = np.asarray(z, np.float32)
    m = z.max(axis=-1, keepdims=True)
    s = np.exp(z - m).sum(axis=-1, dtype=np.float32, keepdims=True)
    return (m + np.log(s)).astype(np.float32)[..., 0]


def gumbel_argmax(w: np.ndarray, g: np.ndarray) -> int:
    """argmax (w + g), lowest index on ties."""
    return int(np.argmax((np.asarray(w, np.float32) + np.asarray(g, np.float32)).astype(np.float32)))


def residual_logw(lp: np.ndarray, lq: np.ndarray) -> np.ndarray:
    """log(p - q) where positive, else -inf (unnormalised: the Gumbel-max
    draw needs no normaliser)."""
    d = (np.exp(np.asarray(lp, np.float32)) - np.exp(np.asarray(lq, np.float32))).astype(np.float32)
    out = np.full(d.shape, -np.inf, np.float32)
    pos = d > 0
    out[pos] = np.log(d[pos])
    return out


# ------------------------------------------------------------------ the block rule
@dataclass
class SampledDecision:
    a: int
    bonus: int
    log_u: np.ndarray          # [K] log u_i of the acceptance tests
    ratio: np.ndarray          # [K] log p_{i-1}(d_i) - log q_i(d_i)
    lp: np.ndarray             # [B, V] log p of the verify rows
    lq: np.ndarray             # [K, V] log q of drafter rows 1..K
    w: np.ndarray              # [V] log-weights of the final draw
    g: np.ndarray              # [V] its Gumbel noise
    fallback: bool             # correction drawn from p_a (empty residual)


def sample_drafts(draft_logits: np.ndarray, inv_t, seed: int, stream: int, t: int):
    """d_i = argmax(z_q,i + g(t, i, draft)) for drafter rows i = 1..K
    (draft_logits holds rows 1..K).  Returns (d [K], z [K, V], g [K, V])."""
    z = scaled(draft_logits, inv_t)
    K, V = z.shape
    g = np.stack([gumbel(uniforms(seed, stream, t, i, DRAFT, V)) for i in range(1, K + 1)])
    d = np.array([gumbel_argmax(z[i], g[i]) for i in range(K)], np.int64)
    return d, z, g


def sample_first(logits_row: np.ndarray, inv_t, seed: int, stream: int, t_last: int) -> int:
    """The token after a prompt whose last position is t_last, drawn from
    softmax(z / T) with counter (t_last, 0, correction purpose); rounds
    address t >= t_last + 1, so no number is reused."""
    z = scaled(logits_row, inv_t)
    return gumbel_argmax(z, gumbel(uniforms(seed, stream, t_last, 0, RESAMPLE, z.shape[-1])))


def accept_sampled(block: Sequence[int], logits: np.ndarray, draft_logits: np.ndarray, inv_t, seed: int,
                   stream: int, t: int) -> SampledDecision:
    """Speculative-sampling acceptance of block = [anchor, d_1..d_K] with
    target logits of block rows 0..K and drafter logits of rows 1..K."""
    block = [int(x) for x in block]
    B = len(block)
    K = B - 1
    zp = scaled(logits, inv_t)
    zq = scaled(draft_logits, inv_t)
    V = zp.shape[1]
    lp = (zp - lse(zp)[:, None]).astype(np.float32)
    lq = (zq - lse(zq)[:, None]).astype(np.float32)
    log_u = np.array([np.log(uniforms(seed, stream, t, i, ACCEPT, 1)[0]) for i in range(1, K + 1)], np.float32)
    ratio = np.array([lp[i - 1, block[i]] - lq[i - 1, block[i]] for i in range(1, K + 1)], np.float32)
    a = 0
    while a < K and log_u[a] < ratio[a]:
        a += 1
    g = gumbel(uniforms(seed, stream, t, a + 1, RESAMPLE, V))
    fallback = False
    if a == K:
        w = zp[K]
    else:
        w = residual_logw(lp[a], lq[a])
        if not np.isfinite(w).any():
            w, fallback = zp[a], True
    return SampledDecision(a, gumbel_argmax(w, g), log_u, ratio, lp, lq, w, g, fallback)


# ------------------------------------------------------------------ exact law (for the pins)
def exact_output_distribution(p: np.ndarray, q: np.ndarray) -> np.ndarray:
    """P(first emitted token = v), enumerating the draft x ~ q:
    sum_x q(x) [min(1, p(x)/q(x)) 1{x = v} + (1 - min(1, p(x)/q(x))) r(v)],
    r the normalised positive part of p - q."""
    p = np.asarray(p, np.float64)
    q = np.asarray(q, np.float64)
    acc = np.where(q > 0, np.minimum(1.0, p / np.where(q > 0, q, 1.0)), 0.0)
    r = np.maximum(p - q, 0.0)
    rs = r.sum()
    r = r / rs if rs > 0 else np.zeros_like(r)
    reject = float((q * (1.0 - acc)).sum())
    return q * acc + reject * r
