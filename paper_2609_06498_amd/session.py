"""Round loop over a Runtime: device-resident state, no per-round host sync.

State per sequence slot: seq_len (KV length = anchor position) and the
anchor token (the previous round's bonus).  One round is
draft_block -> [measurement-only forcing] -> verify_block ->
accept_and_carry -> kv_commit; at temperature T > 0 (round_sampled) it is
draft_block (logits) -> sample_draft -> verify_block (logits) ->
accept_sampled -> kv_commit.  A forward-only multi-round rollout (rollout)
chains rounds whose transitions follow a target trajectory.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np

from .runtime import Runtime


class Session:
    def __init__(self, rt: Runtime, nseq: int):
        torch = rt.torch
        self.rt, self.nseq, self.B = rt, nseq, rt.block
        dev = rt.device
        i32 = lambda *s: torch.zeros(*s, dtype=torch.int32, device=dev)
        self.seq_len = i32(nseq)
        self.anchor = i32(nseq)
        self.draft_tok = i32(nseq, self.B - 1)
        self.block = i32(nseq, self.B)
        self.tgt = i32(nseq, self.B)
        self.accept = i32(nseq)
        self.committed = i32(nseq, self.B)
        self.n_carry = i32(nseq)
        self._dl = self._lg = None

    def logit_buffers(self):
        """fp32 [b*B, vocab] drafter and verify logits of sampling decoding (allocated once)."""
        if self._dl is None:
            torch = self.rt.torch
            shape = (self.nseq * self.B, self.rt.dims.vocab)
            self._dl = torch.empty(shape, dtype=torch.float32, device=self.rt.device)
            self._lg = torch.empty(shape, dtype=torch.float32, device=self.rt.device)
        return self._dl, self._lg

    def prefill(self, prompts: List[np.ndarray]):
        torch = self.rt.torch
        assert len(prompts) == self.nseq
        tok = torch.from_numpy(np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts])).to(self.rt.device)
        self.rt.prefill_batch(tok, [len(p) for p in prompts], self.anchor)
        self.seq_len.copy_(torch.tensor([len(p) for p in prompts], dtype=torch.int32))

    def round(self, carry_on: bool = True, force=None, draft_logits=None, logits=None, hcap=None, feat=None):
        """force = (traj [b, L] int32 device, traj_len, mode [b, B] int8, tok [b, B] int32) for this round."""
        rt, b = self.rt, self.nseq
        rt.draft_block(b, self.anchor, self.seq_len, carry_on, self.draft_tok, self.block, draft_logits)
        if force is not None:
            traj, traj_len, mode, tok = force
            rt.force_drafts(b, traj, traj_len, mode, tok, self.anchor, self.seq_len, self.block)
        rt.verify_block(b, self.block, self.seq_len, self.tgt, logits, hcap)
        rt.accept_and_carry(b, self.block, self.tgt, self.accept, self.anchor, self.committed, self.n_carry, feat)
        rt.kv_commit(b, self.accept, self.seq_len)

    def capture_round(self, carry_on: bool = True, force=None):
        """Records one greedy round (the launches of `round`) into a HIP graph
        and returns replay(mode=None, tok=None), which re-issues the whole
        round as one graph launch on the current stream: no per-kernel host
        launch cost.  With force = (traj, traj_len) the round is recorded with
        the forcing step reading fixed plan buffers, and replay first copies
        that round's plan (mode, tok; device [b, B]) into them.  The graph
        holds kernel launches only (no memset nodes); the recorded state
        buffers are the session's own, so replays continue from whatever
        state the session is in.  Run one eager round first: launch-attribute
        set-up happens at a kernel's first launch, outside any capture."""
        torch = self.rt.torch
        f = None
        if force is not None:
            traj, traj_len = force
            self._gmode = torch.zeros(self.nseq, self.B, dtype=torch.int8, device=self.rt.device)
            self._gtok = torch.zeros(self.nseq, self.B, dtype=torch.int32, device=self.rt.device)
            f = (traj, traj_len, self._gmode, self._gtok)
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize(self.rt.device)
        with torch.cuda.graph(graph):
            self.round(carry_on, force=f)
        torch.cuda.synchronize(self.rt.device)

        def replay(mode=None, tok=None):
            if f is not None:
                self._gmode.copy_(mode, non_blocking=True)
                self._gtok.copy_(tok, non_blocking=True)
            graph.replay()
        replay.graph = graph
        return replay

    def round_sampled(self, sampler, carry_on: bool = True, draft_logits=None, logits=None, hcap=None, feat=None):
        """One round decoded by speculative sampling; `sampler` from Runtime.sampler."""
        rt, b = self.rt, self.nseq
        if draft_logits is None or logits is None:
            draft_logits, logits = self.logit_buffers()
        rt.draft_block(b, self.anchor, self.seq_len, carry_on, None, None, draft_logits)
        rt.sample_draft(b, draft_logits, self.anchor, self.seq_len, sampler, self.draft_tok, self.block)
        rt.verify_block(b, self.block, self.seq_len, None, logits, hcap)
        rt.accept_sampled(b, self.block, self.seq_len, logits, draft_logits, sampler, self.accept, self.anchor,
                          self.committed, self.n_carry, feat)
        rt.kv_commit(b, self.accept, self.seq_len)

    def rollout(self, traj, traj_len: int, k: int, gamma: float, carry_on: bool = True, draft_logits=None,
                on_round=None):
        """Forward-only multi-round rollout (Sec. 4.3) from the current state,
        whose anchors must be traj[s][seq_len[s]] with no carry (a prefill of
        the trajectory prefix with the anchor set): round 0 from mask
        embeddings, rounds 1..k reject-conditioned when carry_on; transitions
        follow the trajectory.  Returns the losses [k + 1, b] (device fp32);
        their sum over rounds is the objective.  on_round(q) runs after each
        round's commit."""
        rt, b, torch = self.rt, self.nseq, self.rt.torch
        if draft_logits is None:
            draft_logits = self.logit_buffers()[0]
        losses = torch.empty(k + 1, b, dtype=torch.float32, device=rt.device)
        for q in range(k + 1):
            rt.draft_block(b, self.anchor, self.seq_len, carry_on and q > 0, self.draft_tok, self.block, draft_logits)
            rt.draft_loss(b, draft_logits, traj, traj_len, self.seq_len, gamma, losses[q])
            rt.verify_block(b, self.block, self.seq_len, None, None)
            rt.trajectory_targets(b, traj, traj_len, self.seq_len, self.tgt)
            rt.accept_and_carry(b, self.block, self.tgt, self.accept, self.anchor, self.committed, self.n_carry)
            rt.kv_commit(b, self.accept, self.seq_len)
            if on_round is not None:
                on_round(q)
        return losses

