"""Helpers shared by the GPU tests: build a runtime and an oracle on the same
seeded inputs, and numeric comparison utilities."""
import numpy as np

from workload import get_config
from workload.synth import make_prompts, make_schedule, make_weights, trajectory_length_needed

TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_rows(x, ref):
    x = np.asarray(x, np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, np.float64).reshape(ref.shape[0], -1)
    return np.linalg.norm(x - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)


def margin_rel(logits):
    """(top1 - top2) / max|l| per row."""
    l = np.asarray(logits, np.float64)
    part = np.partition(l, -2, axis=-1)
    return (part[..., -1] - part[..., -2]) / np.abs(l).max(axis=-1)


def bf16_bits(t):
    """torch int16 bit patterns -> float32 numpy."""
    a = t.cpu().numpy().view(np.uint16).astype(np.uint32) << 16
    return a.view(np.float32)


def dev_values(t, dtype):
    return bf16_bits(t) if dtype == "bf16" else t.cpu().numpy()


def check_argmax(gpu_idx, ref_logits, tol, err_abs=None):
    """Rows whose argmax must agree: margin above tol (and above 4x observed error)."""
    mr = margin_rel(ref_logits)
    ok = gpu_idx == np.argmax(ref_logits, axis=-1)
    need = mr > tol
    bad = need & ~ok
    assert not bad.any(), f"argmax mismatch at rows {np.where(bad)[0]} margins {mr[bad]}"
    if err_abs is not None:
        l = np.asarray(ref_logits, np.float64)
        part = np.partition(l, -2, axis=-1)
        gap = part[..., -1] - part[..., -2]
        strong = gap > 4 * err_abs
        assert not (strong & ~ok).any(), "argmax mismatch on a row with a clear margin"
    return int((~need).sum())


def gpu_trajectory(rt, sess, prompts, need):
    """The target's greedy continuation of every prompt, produced on the GPU by
    junk-draft rounds through the round kernels (each commits at least the
    bonus token); returns int32 [b, max(need)] with the prompts in front."""
    import torch
    b, B = len(prompts), rt.block
    sess.prefill(prompts)
    P = [len(p) for p in prompts]
    L = max(need)
    traj = torch.zeros(b, L, dtype=torch.int32, device="cuda")
    zmode = torch.zeros(b, B, dtype=torch.int8, device="cuda")
    ztok = torch.zeros(b, B, dtype=torch.int32, device="cuda")
    first = sess.anchor.cpu().numpy().copy()
    hist = []
    while int((sess.seq_len.cpu().numpy() - np.array(P)).min()) < max(n - p for n, p in zip(need, P)):
        pos = sess.seq_len.cpu().numpy().copy()
        rt.force_drafts(b, traj, 1, zmode, ztok, sess.anchor, sess.seq_len, sess.block)
        rt.verify_block(b, sess.block, sess.seq_len, sess.tgt)
        rt.accept_and_carry(b, sess.block, sess.tgt, sess.accept, sess.anchor, sess.committed, sess.n_carry)
        rt.kv_commit(b, sess.accept, sess.seq_len)
        hist.append((pos, sess.accept.cpu().numpy().copy(), sess.committed.cpu().numpy().copy()))
    out = np.zeros((b, L), np.int32)
    for s in range(b):
        out[s, :P[s]] = prompts[s]
        out[s, P[s]] = first[s]
    for pos, acc, com in hist:
        for s in range(b):
            for j in range(acc[s] + 1):
                if pos[s] + 1 + j < L:
                    out[s, pos[s] + 1 + j] = com[s, j]
    return out
