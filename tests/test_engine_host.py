"""Host logic of the serving engine, on the CPU: admission, truncation at the
token budget, retirement and slot compaction, checked against a stand-in
runtime with the same call surface.

The stand-in keeps each sequence's tokens in pages addressed through the
engine's page table and computes a toy deterministic "target" from them, so a
wrong page-table swap changes the output; its per-slot library state records
the sequence length it belongs to, so a missing or wrong dflow_move_slot is
caught at the next draft.  Its drafter proposes a varying number of correct
tokens, so rounds commit several tokens and cross the budget mid-block.
"""
from types import SimpleNamespace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_06498_amd.engine import Engine  # noqa: E402
from paper_2609_06498_amd.runtime import PAGE, DFlowError  # noqa: E402

V = 997


def toy_next(seq):
    """The stand-in target's greedy token after `seq`."""
    a = int(seq[-1])
    b = int(seq[-2]) if len(seq) > 1 else 0
    return (a * 131 + b * 71 + len(seq) * 17 + 3) % V


def toy_greedy(prompt, n):
    seq = [int(x) for x in prompt]
    out = []
    while len(out) < n:
        t = toy_next(seq)
        out.append(t)
        seq.append(t)
    return out


class FakeRuntime:
    def __init__(self, block, max_batch, max_ctx):
        self.torch = torch
        self.device = torch.device("cpu")
        self.block, self.max_batch = block, max_batch
        self.max_pages = (max_ctx + 2 * block + PAGE - 1) // PAGE
        self.dims = SimpleNamespace(vocab=V)
        n = self.max_pages * max_batch
        perm = np.random.default_rng(3).permutation(n).astype(np.int32)
        self.page_table = torch.from_numpy(perm.reshape(max_batch, self.max_pages).copy())
        self.pages = np.full((n, PAGE), -1, np.int64)
        self.slot_len = [None] * max_batch        # library per-slot state
        self.moves = 0

    # tokens of slot s at positions [0, n) through the page table
    def _read(self, s, n):
        pt = self.page_table[s].numpy()
        return [int(self.pages[pt[p // PAGE], p % PAGE]) for p in range(n)]

    def _write(self, s, pos, toks):
        pt = self.page_table[s].numpy()
        for i, t in enumerate(toks):
            p = pos + i
            self.pages[pt[p // PAGE], p % PAGE] = int(t)

    def prefill(self, s, tok, first_anchor):
        toks = tok.numpy().tolist()
        self._write(s, 0, toks)
        first_anchor[0] = toy_next(toks)
        self.slot_len[s] = len(toks)

    def draft_block(self, n, anchor, seq_len, carry_on, draft_tok, block):
        B = self.block
        for s in range(n):
            t = int(seq_len[s])
            assert self.slot_len[s] == t, f"slot {s}: library state of a sequence at {self.slot_len[s]}, not {t}"
            seq = self._read(s, t) + [int(anchor[s])]
            good = (t * 7) % B
            for j in range(1, B):
                nxt = toy_next(seq) if j <= good else (toy_next(seq) + 1) % V
                block[s, j] = nxt
                draft_tok[s, j - 1] = nxt
                seq.append(nxt)
            block[s, 0] = anchor[s]

    def force_drafts(self, n, traj, traj_len, mode, tok, anchor, seq_len, block):
        for s in range(n):
            t = int(seq_len[s])
            for j in range(1, self.block):
                m = int(mode[s, j])
                tr = int(traj[s, t + j])
                block[s, j] = tr if m == 1 else ((tr + 1 + int(tok[s, j])) % V if m == 2 else int(tok[s, j]))

    def verify_block(self, n, block, seq_len, tgt):
        for s in range(n):
            t = int(seq_len[s])
            self._write(s, t, block[s].tolist())
            seq = self._read(s, t)
            for j in range(self.block):
                seq.append(int(block[s, j]))
                tgt[s, j] = toy_next(seq)

    def accept_and_carry(self, n, block, tgt, accept, bonus, committed, n_carry):
        for s in range(n):
            a = 0
            while a < self.block - 1 and int(block[s, a + 1]) == int(tgt[s, a]):
                a += 1
            accept[s] = a
            bonus[s] = tgt[s, a]
            committed[s, :a] = block[s, 1:a + 1]
            committed[s, a] = tgt[s, a]
            n_carry[s] = max(0, self.block - 2 - a)

    def kv_commit(self, n, accept, seq_len):
        for s in range(n):
            seq_len[s] += int(accept[s]) + 1
            self.slot_len[s] = int(seq_len[s])

    def move_slot(self, src, dst):
        self.slot_len[dst] = self.slot_len[src]
        self.moves += 1

    def status(self):
        return 0


def _prompts(n, seed=1):
    r = np.random.default_rng(seed)
    return [r.integers(0, V, size=int(r.integers(1, 150))).astype(np.int32) for _ in range(n)]


@pytest.mark.parametrize("slots", [1, 2, 4])
def test_engine_outputs_are_greedy(slots):
    prompts = _prompts(9)
    budgets = [1, 5, 16, 17, 40, 2, 33, 9, 64]
    rt = FakeRuntime(block=8, max_batch=4, max_ctx=300)
    pt0 = sorted(rt.page_table.numpy().ravel().tolist())
    eng = Engine(rt, max_active=slots)
    rids = [eng.submit(p, n) for p, n in zip(prompts, budgets)]
    outs = eng.run()
    for rid, p, n in zip(rids, prompts, budgets):
        assert outs[rid] == toy_greedy(p, n), rid
    assert max(eng.active_hist) == min(slots, len(prompts))
    assert sorted(rt.page_table.numpy().ravel().tolist()) == pt0
    assert not eng.slots and not eng.queue
    if slots > 1:
        assert rt.moves > 0
    assert sum(r.accepted for r in eng.done.values()) > 0


def test_engine_forced_acceptance_is_greedy():
    prompts = _prompts(6, seed=2)
    budgets = [3, 30, 12, 1, 25, 18]
    rt = FakeRuntime(block=8, max_batch=3, max_ctx=300)
    eng = Engine(rt, force_mean=4.0, seed=9)
    for p, n in zip(prompts, budgets):
        eng.submit(p, n, traj=np.concatenate([p, toy_greedy(p, n + 9)]))
    outs = eng.run()
    for rid, (p, n) in enumerate(zip(prompts, budgets)):
        assert outs[rid] == toy_greedy(p, n)
    assert sum(r.accepted for r in eng.done.values()) > 0


@pytest.mark.parametrize("slots", [1, 3])
def test_engine_stop_token(slots):
    """A request ends right after its stop token (first occurrence), or at
    its budget; a stop token absent from the output changes nothing."""
    prompts = _prompts(6, seed=4)
    budgets = [40, 40, 40, 5, 40, 1]
    rt = FakeRuntime(block=8, max_batch=3, max_ctx=300)
    eng = Engine(rt, max_active=slots)
    plan = []
    for i, (p, n) in enumerate(zip(prompts, budgets)):
        g = toy_greedy(p, n)
        stop = g[[7, 0, 22, 2, 0, 0][i]] if i != 4 else -5      # -5 never occurs
        exp = g[:g.index(stop) + 1] if stop in g else g
        plan.append((eng.submit(p, n, stop=stop), exp))
    outs = eng.run()
    for rid, exp in plan:
        assert outs[rid] == exp, rid
    assert not eng.slots and not eng.queue


def test_engine_rejects_bad_requests():
    rt = FakeRuntime(block=8, max_batch=2, max_ctx=100)
    eng = Engine(rt)
    with pytest.raises(DFlowError):
        eng.submit(np.zeros(0, np.int32), 4)
    with pytest.raises(DFlowError):
        eng.submit(np.zeros(10, np.int32), 0)
    with pytest.raises(DFlowError):
        eng.submit(np.zeros(eng.capacity, np.int32), 1)
    with pytest.raises(DFlowError):
        eng.submit(np.zeros(10, np.int32), 4, traj=np.zeros(40, np.int32))
    forced = Engine(rt, force_mean=2.0)
    with pytest.raises(DFlowError):
        forced.submit(np.zeros(10, np.int32), 4)
    with pytest.raises(DFlowError):
        forced.submit(np.zeros(10, np.int32), 4, traj=np.zeros(12, np.int32))
    for bad in (0.0, -1.0):
        with pytest.raises(DFlowError):
            Engine(rt, temperature=bad)
    with pytest.raises(DFlowError):
        Engine(rt, temperature=1.0, force_mean=2.0)
