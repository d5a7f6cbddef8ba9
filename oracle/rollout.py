"""Forward-only multi-round rollout with trajectory-guided transitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 4.3 (Multi-Round Self-Conditioned Training) unfolds, from an anchor
sampled on a target trajectory, an initial mask-prediction round followed by
k reject-conditioned rounds (k = 2 in the paper's experiments), all with the
same drafter:
  * round 0 predicts the block from mask embeddings (a DFlash round);
  * each round's proposals are verified by the frozen target, and the
    verifier states of the rejected suffix are relayed to the next round
    (Sec. 4.2's relay, unchanged);
  * the transition to the next round does not use the verifier's acceptance:
    the proposals are matched exactly against the precomputed target
    trajectory, a = number of leading proposals equal to the trajectory
    tokens, and the next anchor is the trajectory token at the first
    mismatch (position t + a + 1), so every round stays on the trajectory and
    the accepted prefix's target KV is the trajectory's own;
  * the verifier information that is carried still comes from verifying the
    actual proposals.
The objective sums the rounds' losses (eq. dflow_training_objective); each
round's loss is a cross entropy against the trajectory tokens with an
exponential decay over the draft position (following DFlash).

Readings (the paper gives no formula for the decay or the normalisation):
block loss L = sum_i w_i CE_i / sum_i w_i over draft positions i = 1..K,
w_i = exp(-(i - 1) / gamma), CE_i = logsumexp(z_i) - z_i[traj[t + i]] with z_i
the drafter logits of block row i (natural log).  The reject-conditioned
rounds relay with the window of the inference path (carry_window).

Pins (tests/test_oracle_rollout.py): the transition by brute force and, on
the target's own greedy trajectory, equal to greedy verification; the loss
against torch's weighted cross entropy; commits follow the trajectory and the
caches after the rollout equal a fresh prefill of the trajectory prefix;
relay off gives the plain mask drafter in every round; a planted trajectory
is reproduced on replay.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from .dflow import OracleDFlow, SeqState


def decay_weights(K: int, gamma: float) -> np.ndarray:
    """w_i = exp(-(i - 1) / gamma), i = 1..K."""
    return np.exp(-np.arange(K, dtype=np.float64) / float(gamma))


def block_loss(draft_logits: np.ndarray, labels: Sequence[int], gamma: float) -> float:
    """Decayed cross entropy of drafter rows 1..K against their labels (fp64)."""
    z = np.asarray(draft_logits, np.float64)
    m = z.max(axis=1)
    lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
    ce = lse - z[np.arange(z.shape[0]), np.asarray(labels, np.int64)]
    w = decay_weights(z.shape[0], gamma)
    return float((w * ce).sum() / w.sum())


def transition(drafts: Sequence[int], traj: Sequence[int], t: int):
    """(a, next anchor): a = leading drafts d_i equal to traj[t + i]; the next
    anchor is traj[t + a + 1] (the trajectory token at the first mismatch)."""
    K = len(drafts)
    a = 0
    while a < K and int(drafts[a]) == int(traj[t + 1 + a]):
        a += 1
    return a, int(traj[t + a + 1])


def anchor_state(o: OracleDFlow, traj: Sequence[int], t: int) -> SeqState:
    """Target context of a training sample: KV and features of traj[:t], anchor traj[t]."""
    s = o.prefill([int(x) for x in traj[:t]])
    s.tokens[-1] = int(traj[t])
    return s


@dataclass
class RolloutRound:
    t: int
    drafts: np.ndarray
    draft_logits: np.ndarray
    a: int
    bonus: int
    n_relay: int
    n_carry: int
    loss: float


def rollout(o: OracleDFlow, s: SeqState, traj: Sequence[int], k: int, gamma: float, carry_on: bool = True,
            drafts: Optional[List[Sequence[int]]] = None) -> List[RolloutRound]:
    """k + 1 rounds from state s (anchor = traj[s.t], no carry): round 0 from
    mask embeddings, rounds 1..k reject-conditioned when carry_on.  `drafts`
    may replace a round's proposals (parity tests follow the device through a
    near-tie of the drafter's argmax)."""
    traj = np.asarray(traj, np.int64)
    assert s.carry is None and s.anchor == int(traj[s.t])
    out = []
    for q in range(k + 1):
        t = s.t
        hold = {}

        def decide(a, bonus, logits, hold=hold):
            return hold["tr"]

        d, dlg, x, n_relay = o.draft(s, carry_on and q > 0)
        if drafts is not None and drafts[q] is not None:
            d = np.asarray(drafts[q], np.int64)
        hold["tr"] = transition(d, traj, t)
        rr = o.round(s, carry_on and q > 0, block=np.concatenate([[s.anchor], d]), decide=decide)
        loss = block_loss(dlg, traj[t + 1:t + 1 + o.K], gamma)
        out.append(RolloutRound(t, np.asarray(d), dlg, rr.a, rr.bonus, n_relay, rr.n_carry, loss))
    return out


def objective(rounds: Sequence[RolloutRound]) -> float:
    """L_DFlow = L^(0) + sum_q L^(q) (eq. dflow_training_objective)."""
    return float(sum(r.loss for r in rounds))


def plant_trajectory(o: OracleDFlow, prompt: Sequence[int], k: int, accept: Sequence[int],
                     carry_on: bool = True, seed: int = 0) -> np.ndarray:
    """A trajectory on which rollout round q accepts exactly accept[q] drafts:
    starting from the target's greedy token after the prompt, each round's
    first accept[q] proposals are written into the trajectory, followed by a
    token different from the next proposal and by seeded tokens.  Later
    rounds read only positions already fixed, so a replay of the rollout on
    the returned trajectory reproduces the plan.  Length: prompt + (k + 1) *
    (K + 1) + 1."""
    V = o.m.dims.vocab
    K = o.K
    rng = np.random.default_rng(seed)
    P = len(prompt)
    L = P + (k + 1) * (K + 1) + 1
    traj = np.zeros(L, np.int64)
    traj[:P] = prompt
    s = o.prefill(prompt)
    traj[P] = s.anchor
    for q in range(k + 1):
        t = s.t
        d, _, _, _ = o.draft(s, carry_on and q > 0)
        j = int(accept[q])
        assert 0 <= j <= K
        traj[t + 1:t + 1 + j] = d[:j]
        traj[t + 1 + j:t + 2 + K] = rng.integers(0, V, size=K + 1 - j)   # the anchor after and beyond
        if j < K:
            traj[t + 1 + j] = (int(d[j]) + 1 + int(rng.integers(0, V - 1))) % V   # != d_{j+1}
        a, nxt = transition(d, traj, t)
        assert a == j
        o.round(s, carry_on and q > 0, block=np.concatenate([[s.anchor], d]),
                decide=lambda *_a, a=a, nxt=nxt: (a, nxt))
    return traj
