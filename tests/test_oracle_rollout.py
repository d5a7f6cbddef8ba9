"""Pins of the forward-only multi-round rollout (oracle/rollout.py), CPU only.

* transition: brute force over planted matches; on the target's own greedy
  trajectory it equals greedy verification's acceptance and bonus (the case
  the paper describes as usually agreeing with the verifier);
* loss: against torch's cross entropy with per-position weights, and the
  decay weights' closed form;
* the rollout stays on the trajectory: the committed tokens are the
  trajectory prefix and the caches equal a fresh prefill of it (rollback);
* relay off: every round is the plain mask-embedding drafter;
* a planted trajectory is reproduced on replay (acceptance lengths as
  planned), with relays in the reject-conditioned rounds;
* planted mistakes (bonus = the drafted token, off-by-one labels) fail.
"""
import numpy as np
import pytest
import torch

import oracle.rollout as ro
from oracle import Mode, OracleDFlow, OracleModel
from workload import get_config
from workload.synth import make_prompts, make_weights


@pytest.fixture(scope="module")
def tiny():
    wl = get_config("tiny-f32")
    w = make_weights(wl.dims, wl.seed_w)
    o = OracleDFlow(OracleModel(wl.dims, w, Mode("fp64")), wl.block)
    return wl, o, make_prompts(wl)[0][:40]


def test_transition_brute_force():
    rng = np.random.default_rng(0)
    for _ in range(200):
        K = int(rng.integers(1, 9))
        t = int(rng.integers(0, 5))
        traj = rng.integers(0, 4, size=t + K + 2)
        d = rng.integers(0, 4, size=K)
        a, nxt = ro.transition(d, traj, t)
        ref = next((i for i in range(K) if d[i] != traj[t + 1 + i]), K)
        assert a == ref and nxt == traj[t + 1 + ref]
        assert all(d[i] == traj[t + 1 + i] for i in range(a))


def test_transition_on_greedy_trajectory_is_verification(tiny):
    wl, o, prompt = tiny
    g = o.greedy_decode(prompt, 3 * wl.block)
    traj = np.array(list(prompt) + g, np.int64)
    s = o.prefill(prompt)
    rng = np.random.default_rng(1)
    for r in range(3):
        t = s.t
        n = int(rng.integers(0, wl.K + 1))
        d = np.concatenate([traj[t + 1:t + 1 + n], rng.integers(0, wl.dims.vocab, wl.K - n)])
        rr = o.round(s, True, block=np.concatenate([[s.anchor], d]))
        assert ro.transition(d, traj, t) == (rr.a, rr.bonus)


def test_decay_and_loss_against_torch():
    rng = np.random.default_rng(2)
    z = rng.normal(size=(7, 11)) * 3
    lab = rng.integers(0, 11, size=7)
    gamma = 4.0
    w = ro.decay_weights(7, gamma)
    assert w[0] == 1.0 and np.allclose(w[1:] / w[:-1], np.exp(-1 / gamma))
    ce = torch.nn.functional.cross_entropy(torch.from_numpy(z), torch.from_numpy(lab), reduction="none").numpy()
    assert abs(ro.block_loss(z, lab, gamma) - (w * ce).sum() / w.sum()) < 1e-12


def test_rollout_stays_on_the_trajectory(tiny):
    wl, o, prompt = tiny
    g = o.greedy_decode(prompt, 4 * wl.block)
    traj = np.array(list(prompt) + g, np.int64)
    t0 = len(prompt) + 3
    s = ro.anchor_state(o, traj, t0)
    rounds = ro.rollout(o, s, traj, 2, 7.0)
    assert [r.t for r in rounds] == [t0, t0 + rounds[0].a + 1, t0 + rounds[0].a + rounds[1].a + 2]
    assert s.tokens == [int(x) for x in traj[:s.t + 1]]
    assert rounds[0].n_relay == 0
    fresh = o.prefill(s.tokens[:-1])
    for a, b in [(s.F, fresh.F)] + list(zip(s.k, fresh.k)) + list(zip(s.v, fresh.v)) + \
            list(zip(s.ck, fresh.ck)) + list(zip(s.cv, fresh.cv)):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
    assert abs(ro.objective(rounds) - sum(r.loss for r in rounds)) == 0
    assert all(np.isfinite(r.loss) and r.loss > 0 for r in rounds)


def test_relay_off_is_the_mask_drafter(tiny):
    wl, o, prompt = tiny
    traj = ro.plant_trajectory(o, prompt, 2, [1, 0, 3], carry_on=False)
    s = ro.anchor_state(o, traj, len(prompt))
    rounds = ro.rollout(o, s, traj, 2, 7.0, carry_on=False)
    m = o.m
    s2 = ro.anchor_state(o, traj, len(prompt))
    for r in rounds:
        assert r.n_relay == 0
        x = np.stack([m.w("embed")[s2.anchor]] + [m.w("draft.e_mask")] * wl.K)
        lg = m.drafter_block(x, s2.t, s2.ck, s2.cv)[1:]
        np.testing.assert_array_equal(r.drafts, np.argmax(lg, axis=1))
        o.round(s2, False, block=np.concatenate([[s2.anchor], r.drafts]),
                decide=lambda *_a, r=r: (r.a, r.bonus))


@pytest.mark.parametrize("plan", [[2, 0, 5], [7, 7, 1], [0, 3, 7]])
def test_planted_trajectory_replays(tiny, plan):
    wl, o, prompt = tiny
    traj = ro.plant_trajectory(o, prompt, 2, plan, seed=sum(plan))
    s = ro.anchor_state(o, traj, len(prompt))
    rounds = ro.rollout(o, s, traj, 2, 7.0)
    assert [r.a for r in rounds] == plan
    for q, r in enumerate(rounds):
        assert r.bonus == traj[r.t + r.a + 1]
        if q > 0:
            prev = rounds[q - 1]
            assert r.n_relay == max(0, wl.K - 1 - prev.a)


def test_mutation_bonus_from_draft(tiny, monkeypatch):
    wl, o, prompt = tiny
    traj = ro.plant_trajectory(o, prompt, 2, [2, 1, 0], seed=3)
    real = ro.transition

    def bad(d, tr, t):
        a, _ = real(d, tr, t)
        return a, int(d[a]) if a < len(d) else int(tr[t + a + 1])

    monkeypatch.setattr(ro, "transition", bad)
    s = ro.anchor_state(o, traj, len(prompt))
    ro.rollout(o, s, traj, 2, 7.0)
    assert s.tokens != [int(x) for x in traj[:s.t + 1]]


def test_mutation_label_shift(tiny, monkeypatch):
    """Labels traj[t + i + 1] instead of traj[t + i] change the loss."""
    wl, o, prompt = tiny
    traj = ro.plant_trajectory(o, prompt, 0, [3], seed=4)
    s = ro.anchor_state(o, traj, len(prompt))
    r = ro.rollout(o, s, traj, 0, 7.0)[0]
    shifted = ro.block_loss(r.draft_logits, traj[r.t + 2:r.t + 2 + wl.K], 7.0)
    assert abs(shifted - r.loss) > 1e-6
    # with drafts equal to the labels, the loss is below the uniform-prediction loss
    assert r.loss < np.log(wl.dims.vocab) + 1.0
