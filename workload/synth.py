"""Seeded synthetic inputs: weights, prompts and acceptance-forcing schedules.

Everything here is input data.  It is consumed identically by the CPU oracle
and by the GPU path and implements none of the method's arithmetic.

Weights follow the PyTorch ``Linear`` convention ``[out_features,
in_features]``.  Linear weights, embeddings, the LM head, the mask embedding,
the feature projection ``W_c`` and every relay parameter except the LayerNorm
gain are drawn with mean 0 and std 0.02.  Norm gains are ``1 + 0.02 z`` so that
a dropped gain changes results.  bf16 weights are produced by round-to-nearest-
even from the fp32 draw and stored as ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import hashlib
import os
import subprocess
import threading
from typing import Dict, Iterator, List, Tuple

import numpy as np

from .configs import ModelDims, Workload

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "wlgen.c")
_LIB_PATH = os.path.join(_HERE, "_wlgen.so")
_lib = None
_lib_lock = threading.Lock()


def build_generator(force: bool = False) -> str:
    """Compile the counter-based generator helper (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _gen():
    global _lib
    with _lib_lock:
        if _lib is None:
            lib = ctypes.CDLL(build_generator())
            for fn, ptr_t in (("wl_fill_f32", ctypes.c_void_p), ("wl_fill_bf16", ctypes.c_void_p)):
                f = getattr(lib, fn)
                f.argtypes = [ptr_t, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float, ctypes.c_float]
                f.restype = None
            lib.wl_bf16_to_f32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
            lib.wl_bf16_to_f32.restype = None
            _lib = lib
    return _lib


def tensor_key(seed: int, name: str) -> int:
    h = hashlib.blake2b(f"{seed}/{name}".encode(), digest_size=8).digest()
    return int.from_bytes(h, "little")


def fill(shape, key: int, mean: float, std: float, dtype: str) -> np.ndarray:
    n = int(np.prod(shape))
    lib = _gen()
    if dtype == "f32":
        out = np.empty(n, np.float32)
        lib.wl_fill_f32(out.ctypes.data, n, key, mean, std)
    elif dtype == "bf16":
        out = np.empty(n, np.uint16)
        lib.wl_fill_bf16(out.ctypes.data, n, key, mean, std)
    else:
        raise ValueError(dtype)
    return out.reshape(shape)


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    a = np.ascontiguousarray(a, dtype=np.uint16)
    out = np.empty(a.shape, np.float32)
    _gen().wl_bf16_to_f32(a.ctypes.data, out.ctypes.data, a.size)
    return out


# ---------------------------------------------------------------- weights
GAIN, LINEAR = "gain", "linear"


def _layer_specs(prefix: str, dm: ModelDims) -> List[Tuple[str, Tuple[int, ...], str]]:
    d, F = dm.d, dm.ffn
    return [
        (f"{prefix}.attn_norm", (d,), GAIN),
        (f"{prefix}.wq", (dm.q_dim, d), LINEAR),
        (f"{prefix}.wk", (dm.kv_dim, d), LINEAR),
        (f"{prefix}.wv", (dm.kv_dim, d), LINEAR),
        (f"{prefix}.q_norm", (dm.head_dim,), GAIN),
        (f"{prefix}.k_norm", (dm.head_dim,), GAIN),
        (f"{prefix}.wo", (d, dm.q_dim), LINEAR),
        (f"{prefix}.ffn_norm", (d,), GAIN),
        (f"{prefix}.w_gate", (F, d), LINEAR),
        (f"{prefix}.w_up", (F, d), LINEAR),
        (f"{prefix}.w_down", (d, F), LINEAR),
    ]


def weight_specs(dm: ModelDims) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, kind) of every parameter of the target, drafter and relay."""
    d, V = dm.d, dm.vocab
    specs = [("embed", (V, d), LINEAR)]
    for l in range(dm.n_layers):
        specs += _layer_specs(f"layers.{l}", dm)
    specs += [("final_norm", (d,), GAIN), ("lm_head", (V, d), LINEAR)]
    for l in range(dm.n_draft_layers):
        specs += _layer_specs(f"draft.layers.{l}", dm)
    specs += [
        ("draft.final_norm", (d,), GAIN),
        ("draft.e_mask", (d,), LINEAR),
        ("draft.w_c", (d, dm.m * d), LINEAR),
        ("draft.g_c", (d,), GAIN),
        ("relay.w1", (dm.d_h, 3 * d), LINEAR),
        ("relay.c1", (dm.d_h,), LINEAR),
        ("relay.w2", (2 * d, dm.d_h), LINEAR),
        ("relay.c2", (2 * d,), LINEAR),
        ("relay.ln_g", (d,), GAIN),
        ("relay.ln_b", (d,), LINEAR),
    ]
    return specs


def make_tensor(dm: ModelDims, seed: int, name: str, shape, kind: str) -> np.ndarray:
    mean = 1.0 if kind == GAIN else 0.0
    return fill(shape, tensor_key(seed, name), mean, 0.02, dm.dtype)


def iter_weights(dm: ModelDims, seed: int) -> Iterator[Tuple[str, np.ndarray]]:
    for name, shape, kind in weight_specs(dm):
        yield name, make_tensor(dm, seed, name, shape, kind)


def make_weights(dm: ModelDims, seed: int) -> Dict[str, np.ndarray]:
    return dict(iter_weights(dm, seed))


def weight_bytes(dm: ModelDims) -> int:
    elt = 4 if dm.dtype == "f32" else 2
    return sum(int(np.prod(s)) for _, s, _ in weight_specs(dm)) * elt


# ---------------------------------------------------------------- prompts / schedules
def _rng(seed: int, *tag) -> np.random.Generator:
    key = tensor_key(seed, "/".join(str(t) for t in tag))
    return np.random.Generator(np.random.Philox(key=[key & 0xFFFFFFFFFFFFFFFF, 0x5EED]))


def context_lengths(wl: Workload) -> List[int]:
    lo, hi = wl.ctx
    if lo == hi:
        return [lo] * wl.batch
    r = _rng(wl.seed_prompt, "ctxlen")
    return [int(x) for x in r.integers(lo, hi + 1, size=wl.batch)]


def make_prompts(wl: Workload) -> List[np.ndarray]:
    """Uniform token ids in [0, V) for each sequence (stand-ins for the
    benchmark prompts of Sec. 5.1, whose items are not used)."""
    out = []
    for s, n in enumerate(context_lengths(wl)):
        r = _rng(wl.seed_prompt, "prompt", s)
        out.append(r.integers(0, wl.dims.vocab, size=n).astype(np.int32))
    return out


def balanced_capped_geometric(rng: np.random.Generator, R: int, q: float, cap: int) -> np.ndarray:
    """R draws of a = min(G, cap), P(G = k) = (1-q) q^k, arranged so that every
    prefix of the rounds realises close to the distribution's mean.

    The values are the distribution's quantiles at the stratified points
    u_i = (i + 1/2) / R (through the inverse CDF G = floor(log(1-u) / log q));
    they are then ordered greedily, each round taking the remaining value that
    keeps the running sum closest to n times their mean (ties broken by a
    seeded shuffle).  The multiset follows the law; the order bounds the
    prefix error by cap / n, so a short timed run measures the configured
    acceptance instead of whatever a few pseudo-random draws happened to be.
    """
    u = (np.arange(R) + 0.5) / R
    vals = np.minimum(np.floor(np.log1p(-u) / np.log(q)), cap).astype(np.int64)
    target = vals.mean()
    pool = [int(v) for v in rng.permutation(vals)]
    out = np.empty(R, np.int64)
    s = 0
    for n in range(R):
        i = min(range(len(pool)), key=lambda j: abs(s + pool[j] - (n + 1) * target))
        out[n] = pool.pop(i)
        s += int(out[n])
    return out


# forcing modes for draft position j of round r, sequence s
FORCE_RANDOM, FORCE_TRAJ, FORCE_MISMATCH = 0, 1, 2


def make_schedule(wl: Workload, rounds: int | None = None) -> Dict[str, np.ndarray]:
    """Per (round, sequence, block index) forcing plan.

    ``mode[r,s,j]``: 1 -> the draft at block index j is the trajectory token
    at its position, 2 -> the trajectory token shifted by ``1 + tok`` modulo V
    (a guaranteed mismatch, tok in [0, V-2]), 0 -> the uniform token ``tok``.
    Index 0 is the anchor and is never forced.  ``accept`` holds the intended
    prefix length for geometric schedules (-1 for Bernoulli).
    """
    R = wl.rounds if rounds is None else rounds
    b, B, V, K = wl.batch, wl.block, wl.dims.vocab, wl.K
    r = _rng(wl.seed_sched, "schedule", wl.schedule)
    tok = r.integers(0, V, size=(R, b, B)).astype(np.int32)
    mode = np.zeros((R, b, B), np.int8)
    accept = np.full((R, b), -1, np.int32)
    if wl.schedule == "bernoulli":
        coin = r.random(size=(R, b, B))
        mode[:] = np.where(coin < wl.sched_param, FORCE_TRAJ, FORCE_RANDOM)
    elif wl.schedule == "geometric":
        q = wl.sched_param / (1.0 + wl.sched_param)
        a = np.stack([balanced_capped_geometric(r, R, q, K) for _ in range(b)], axis=1).astype(np.int32)
        accept[:] = a
        j = np.arange(B)[None, None, :]
        mode[:] = np.where(j <= a[..., None], FORCE_TRAJ,
                           np.where(j == a[..., None] + 1, FORCE_MISMATCH, FORCE_RANDOM))
        tok = np.where(mode == FORCE_MISMATCH, tok % (V - 1), tok).astype(np.int32)
    else:
        raise ValueError(wl.schedule)
    mode[:, :, 0] = FORCE_TRAJ
    return {"mode": mode, "tok": tok, "accept": accept}


def trajectory_length_needed(wl: Workload, sched: Dict[str, np.ndarray]) -> List[int]:
    """Upper bound on trajectory positions each sequence can touch."""
    R, b, B = sched["mode"].shape
    ctx = context_lengths(wl)
    if wl.schedule == "geometric":
        tot = (sched["accept"] + 1).sum(axis=0)
        return [int(ctx[s] + tot[s] + B + 1) for s in range(b)]
    return [int(ctx[s] + R * B + B + 1) for s in range(b)]
