"""Round loop over a Runtime: device-resident state, no per-round host sync.

State per sequence slot: seq_len (KV length = anchor position) and the
anchor token (the previous round's bonus).  One round is
draft_block -> [measurement-only forcing] -> verify_block ->
accept_and_carry -> kv_commit.
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

    def prefill(self, prompts: List[np.ndarray]):
        torch = self.rt.torch
        assert len(prompts) == self.nseq
        for s, p in enumerate(prompts):
            tok = torch.from_numpy(np.ascontiguousarray(p, dtype=np.int32)).to(self.rt.device)
            self.rt.prefill(s, tok, self.anchor[s:s + 1])
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
