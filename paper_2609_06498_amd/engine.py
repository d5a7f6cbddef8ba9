"""Continuous-batching serving loop over the round entry points.

Active requests occupy slots 0..n-1 of one context; a slot owns one row of
the page table, and with it the target KV pages and the drafter-context
pages of its sequence.  A round runs draft_block -> verify_block ->
accept_and_carry -> kv_commit over the n active slots with the drafter's own
proposals (Sec. 4: anchor plus K drafts, greedy longest-prefix acceptance,
commit of the accepted prefix and the bonus token).  After the round the host
reads the acceptance lengths and committed tokens, appends them to the
requests' outputs, retires every request that reached its token budget and
fills the hole by moving the last active slot into it (page-table rows are
swapped, so the pages stay a permutation; the library's own per-slot state
moves with dflow_move_slot).  Queued requests are admitted into free slots by
a prefill, whose argmax is the request's first output token.

With a temperature T > 0 the engine decodes by speculative sampling: the
first token is drawn at the prefill (dflow_prefill_sampled), and a round is
draft_block (drafter logits) -> sample_draft -> verify_block (logits) ->
accept_sampled -> kv_commit.  Each request draws from its own Philox stream
(its request id under the engine's sampling seed), so its tokens do not
depend on its slot or on the requests that share its rounds.

Every step runs in the library's kernels; this layer only sequences calls
and keeps the per-request bookkeeping.  The one host synchronisation per
round reads the committed tokens, which the retirement decision needs.
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from .runtime import PAGE, DFlowError, Runtime


@dataclass
class Request:
    rid: int
    prompt: np.ndarray
    max_new: int
    traj: Optional[np.ndarray] = None      # forcing trajectory (measurement construct only)
    stop: Optional[int] = None             # end-of-sequence token: generation ends after it
    out: List[int] = field(default_factory=list)
    rounds: int = 0
    accepted: int = 0                      # drafted tokens accepted over all rounds


class Engine:
    """DFlow serving of many requests through one Runtime: greedy decoding,
    or speculative sampling at `temperature` (Philox key (sample_seed,
    request id)).

    max_active caps the concurrently decoded requests (at most the runtime's
    max_batch).  With force_mean set, every round's block is rebuilt from the
    request's `traj` by dflow_bench_force_drafts with a geometric accepted
    prefix of that mean (a measurement construct for random-weight models,
    whose drafter proposals are never accepted); outputs stay the target's
    greedy continuation either way.
    """

    def __init__(self, rt: Runtime, max_active: Optional[int] = None, carry_on: bool = True,
                 force_mean: Optional[float] = None, seed: int = 0, temperature: Optional[float] = None,
                 sample_seed: int = 0):
        torch = rt.torch
        self.rt, self.B, self.carry_on = rt, rt.block, carry_on
        self.max_active = min(max_active or rt.max_batch, rt.max_batch)
        if self.max_active < 1:
            raise DFlowError("max_active must be at least 1")
        self.capacity = rt.max_pages * PAGE
        n, B, dev = rt.max_batch, self.B, rt.device
        i32 = lambda *s: torch.zeros(*s, dtype=torch.int32, device=dev)
        self.seq_len, self.anchor = i32(n), i32(n)
        self.draft_tok, self.block, self.tgt = i32(n, B - 1), i32(n, B), i32(n, B)
        self.accept, self.committed, self.n_carry = i32(n), i32(n, B), i32(n)
        self.force_mean = force_mean
        self.seed = seed
        self.temperature = temperature
        if temperature is not None:
            if not temperature > 0:
                raise DFlowError("temperature must be positive (greedy decoding: temperature=None)")
            if force_mean is not None:
                raise DFlowError("forced drafts are a greedy-decoding measurement construct")
            V = rt.dims.vocab
            self.streams = torch.zeros(n, dtype=torch.int64, device=dev)
            self.sampler = rt.sampler(temperature, sample_seed, self.streams)
            self.dl = torch.empty(n * B, V, dtype=torch.float32, device=dev)
            self.lg = torch.empty(n * B, V, dtype=torch.float32, device=dev)
        self.traj = None
        self.slots: List[Request] = []
        self.queue: deque = deque()
        self.done: Dict[int, Request] = {}
        self._next = 0
        self.rounds = 0
        self.active_hist: List[int] = []

    # ------------------------------------------------------------ requests
    def submit(self, prompt, max_new: int, traj=None, stop: Optional[int] = None) -> int:
        """Queues a request: at most max_new generated tokens, fewer when the
        `stop` token is generated (it is the last output token then)."""
        prompt = np.ascontiguousarray(prompt, dtype=np.int32).reshape(-1)
        if prompt.size < 1 or max_new < 1:
            raise DFlowError("a request needs at least one prompt token and one new token")
        if prompt.size + max_new + self.B > self.capacity:
            raise DFlowError(f"prompt {prompt.size} + {max_new} new tokens exceed the context capacity "
                             f"{self.capacity - self.B}")
        if (self.force_mean is None) != (traj is None):
            raise DFlowError("forcing needs a trajectory per request and an engine built with force_mean")
        if traj is not None:
            traj = np.ascontiguousarray(traj, dtype=np.int32).reshape(-1)
            if traj.size < prompt.size + max_new + self.B:
                raise DFlowError("forcing trajectory shorter than prompt + max_new + block")
        rid = self._next
        self._next += 1
        self.queue.append(Request(rid, prompt, int(max_new), traj, None if stop is None else int(stop)))
        return rid

    def run(self) -> Dict[int, List[int]]:
        """Serves until every submitted request is finished; returns the
        generated tokens per request id."""
        while self.queue or self.slots:
            self.step()
        return {rid: r.out for rid, r in self.done.items()}

    # ------------------------------------------------------------ scheduling
    def step(self):
        self._admit()
        if self.slots:
            self._round()

    def _admit(self):
        torch, rt = self.rt.torch, self.rt
        new = []
        while self.queue and len(self.slots) < self.max_active:
            req = self.queue.popleft()
            s = len(self.slots)
            tok = torch.from_numpy(req.prompt).to(rt.device)
            if self.temperature is None:
                rt.prefill(s, tok, self.anchor[s:s + 1])
            else:
                self.streams[s:s + 1].fill_(req.rid)
                one = rt.sampler(self.temperature, self.sampler.seed, self.streams[s:s + 1])
                rt.prefill_sampled(s, tok, one, self.anchor[s:s + 1])
            self.seq_len[s:s + 1].fill_(int(req.prompt.size))
            if req.traj is not None:
                self._traj_row(s, req.traj)
            self.slots.append(req)
            new.append(s)
        if new:
            first = self.anchor[:len(self.slots)].cpu().numpy()
            for s in new:
                self._emit(self.slots[s], [int(first[s])])
            self._retire()

    def _traj_row(self, s: int, traj: np.ndarray):
        torch = self.rt.torch
        if self.traj is None or self.traj.shape[1] < traj.size:
            L = max(traj.size, 0 if self.traj is None else self.traj.shape[1])
            t = torch.zeros(self.rt.max_batch, L, dtype=torch.int32, device=self.rt.device)
            if self.traj is not None:
                t[:, :self.traj.shape[1]] = self.traj
            self.traj = t
        self.traj[s].zero_()
        self.traj[s, :traj.size] = torch.from_numpy(traj).to(self.rt.device)

    def _force_plan(self):
        """Per request and round (seeded by both, so the plan does not depend
        on which requests share the round): a geometric accepted prefix a of
        mean force_mean, capped at K; block index j <= a takes the trajectory
        token, j = a + 1 a guaranteed mismatch, the rest uniform tokens."""
        B, V = self.B, self.rt.dims.vocab
        q = self.force_mean / (1.0 + self.force_mean)
        mode = np.zeros((len(self.slots), B), np.int8)
        tok = np.zeros((len(self.slots), B), np.int32)
        j = np.arange(B)
        for s, req in enumerate(self.slots):
            r = np.random.default_rng([self.seed, req.rid, req.rounds])
            a = min(int(r.geometric(1.0 - q)) - 1, B - 1)
            mode[s] = np.where(j <= a, 1, np.where(j == a + 1, 2, 0))
            tok[s] = r.integers(0, V - 1, size=B)
        return mode, tok

    def _round(self):
        rt, torch, n = self.rt, self.rt.torch, len(self.slots)
        if self.temperature is not None:
            rt.draft_block(n, self.anchor, self.seq_len, self.carry_on, None, None, self.dl)
            rt.sample_draft(n, self.dl, self.anchor, self.seq_len, self.sampler, self.draft_tok, self.block)
            rt.verify_block(n, self.block, self.seq_len, None, self.lg)
            rt.accept_sampled(n, self.block, self.seq_len, self.lg, self.dl, self.sampler, self.accept, self.anchor,
                              self.committed, self.n_carry)
            rt.kv_commit(n, self.accept, self.seq_len)
            return self._collect(n)
        rt.draft_block(n, self.anchor, self.seq_len, self.carry_on, self.draft_tok, self.block)
        if self.force_mean is not None:
            mode, tok = self._force_plan()
            mode_d = torch.from_numpy(mode).to(rt.device)
            tok_d = torch.from_numpy(tok).to(rt.device)
            rt.force_drafts(n, self.traj, self.traj.shape[1], mode_d, tok_d, self.anchor, self.seq_len, self.block)
        rt.verify_block(n, self.block, self.seq_len, self.tgt)
        rt.accept_and_carry(n, self.block, self.tgt, self.accept, self.anchor, self.committed, self.n_carry)
        rt.kv_commit(n, self.accept, self.seq_len)
        self._collect(n)

    def _collect(self, n: int):
        acc = self.accept[:n].cpu().numpy()
        com = self.committed[:n].cpu().numpy()
        for s, req in enumerate(self.slots):
            a = int(acc[s])
            self._emit(req, [int(x) for x in com[s, :a + 1]])
            req.rounds += 1
            req.accepted += a
        self.rounds += 1
        self.active_hist.append(n)
        self._retire()

    def _emit(self, req: Request, toks: List[int]):
        """Appends committed tokens up to the budget and the stop token."""
        for x in toks:
            if self._finished(req):
                return
            req.out.append(x)

    @staticmethod
    def _finished(req: Request) -> bool:
        return len(req.out) >= req.max_new or (req.stop is not None and bool(req.out) and req.out[-1] == req.stop)

    def _retire(self):
        for s in range(len(self.slots) - 1, -1, -1):
            if self._finished(self.slots[s]):
                self._remove(s)

    def _remove(self, s: int):
        """Finishes the request in slot s; the last active slot moves into s."""
        rt = self.rt
        req = self.slots[s]
        self.done[req.rid] = req
        last = len(self.slots) - 1
        if s != last:
            pt = rt.page_table
            idx = [s, last]
            pt[idx] = pt[[last, s]]
            self.seq_len[s:s + 1].copy_(self.seq_len[last:last + 1])
            self.anchor[s:s + 1].copy_(self.anchor[last:last + 1])
            if self.traj is not None:
                self.traj[s].copy_(self.traj[last])
            if self.temperature is not None:
                self.streams[s:s + 1].copy_(self.streams[last:last + 1])
            rt.move_slot(last, s)
            self.slots[s] = self.slots[last]
        self.slots.pop()
