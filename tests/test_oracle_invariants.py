"""Invariants that pin the oracle's round algorithm (CPU only).

1. Block verification gives the same logits as one-token-at-a-time decoding
   and as a no-cache full recompute (B = 1 is plain decoding).
2. Losslessness: the committed stream equals plain greedy decoding for any
   draft source, with relay on or off (exact-match verification, Sec. 3).
3. Drafts equal to the target's greedy tokens are all accepted; a wrong
   draft at index a+1 gives acceptance length a and bonus = greedy token.
4. Relay disabled reproduces the mask-embedding drafter; a zero relay
   output layer makes relay-on bitwise equal to relay-off.
Also: KV / fused features after several rounds equal a fresh prefill of the
committed tokens (rollback), and the carry index map agrees with position
arithmetic for every acceptance length.
"""
import numpy as np
import pytest

from oracle import Mode, OracleDFlow, OracleModel
from oracle.dflow import forced_block
from workload import get_config
from workload.synth import make_prompts, make_schedule, make_weights


def _setup(mode, wl_name="tiny-f32", w=None, **kw):
    wl = get_config(wl_name)
    if w is None:
        w = make_weights(wl.dims, wl.seed_w)
    m = OracleModel(wl.dims, w, Mode(mode))
    return wl, m, OracleDFlow(m, wl.block, **kw)


@pytest.mark.parametrize("mode,tol", [("fp64", 1e-12), ("fp32", 2e-5)])
def test_block_verify_equals_stepwise_and_full(mode, tol):
    wl, m, o = _setup(mode)
    prompt = make_prompts(wl)[0][:50]
    s = o.prefill(prompt)
    rng = np.random.default_rng(0)
    block = np.concatenate([[s.anchor], rng.integers(0, wl.dims.vocab, wl.K)])
    lg_block, _, _, _, _ = o.verify(s, block)
    # stepwise: feed block rows one at a time through a B=1 verify
    s1 = o.prefill(prompt)
    step = []
    for j in range(wl.block):
        lg, _, _, ks, vs = o.verify(s1, [int(block[j])])
        step.append(lg[0])
        for l in range(wl.dims.n_layers):
            s1.k[l] = np.concatenate([s1.k[l], ks[l]])
            s1.v[l] = np.concatenate([s1.v[l], vs[l]])
        s1.tokens.append(int(block[j + 1]) if j + 1 < wl.block else 0)
    step = np.array(step)
    full = o.full_logits(list(prompt) + [int(x) for x in block])[len(prompt):]
    for other in (step, full):
        rel = np.linalg.norm(lg_block - other, axis=1) / np.linalg.norm(other, axis=1)
        assert rel.max() < tol, rel.max()


@pytest.mark.parametrize("mode", ["fp64", "fp32"])
@pytest.mark.parametrize("source", ["drafter", "forced", "random", "oracle_greedy"])
@pytest.mark.parametrize("carry_on", [True, False])
def test_lossless_against_plain_greedy(mode, source, carry_on):
    wl, m, o = _setup(mode)
    prompt = make_prompts(wl)[0]
    R = 8
    ref = o.greedy_decode(prompt, R * wl.block + wl.block)
    traj = np.array(list(prompt) + ref, np.int64)
    sched = make_schedule(wl, R)
    rng = np.random.default_rng(1)
    s = o.prefill(prompt)
    accepted = []
    for r in range(R):
        if source == "drafter":
            rr = o.round(s, carry_on)
        elif source == "forced":
            rr = o.round(s, carry_on, force=(traj, sched["mode"][r, 0], sched["tok"][r, 0]))
        elif source == "random":
            rr = o.round(s, carry_on, block=np.concatenate([[s.anchor], rng.integers(0, wl.dims.vocab, wl.K)]))
        else:
            rr = o.round(s, carry_on, block=traj[s.t:s.t + wl.block])
        accepted.append(rr.a)
    gen = s.tokens[len(prompt):]
    assert gen == ref[:len(gen)]
    if source == "oracle_greedy":
        assert all(a == wl.K for a in accepted)


def test_acceptance_brute_force():
    wl, m, o = _setup("fp64")
    prompt = make_prompts(wl)[0][:40]
    ref = o.greedy_decode(prompt, wl.block + 1)
    V, K = wl.dims.vocab, wl.K
    for a in range(K + 1):
        s = o.prefill(prompt)
        block = np.array([s.anchor] + ref[1:K + 1])
        if a < K:
            block[a + 1] = (block[a + 1] + 1) % V
        rr = o.round(s, True, block=block)
        assert rr.a == a
        assert rr.bonus == ref[a + 1]
        assert rr.committed == ref[1:a + 2]
        assert s.t == len(prompt) + a + 1
        assert s.k[0].shape[0] == s.t and s.F.shape[0] == s.t and s.ck[0].shape[0] == s.t


@pytest.mark.parametrize("window", ["suffix", "suffix+tail", "suffix-inputs"])
def test_carry_index_map_against_positions(window):
    """Next-round block index i sits at position t' + i with t' = t + a + 1.
    The drafter predicts the token at its own position; the verifier row at
    position p predicts p + 1.  So index i must take the row at position
    t' + i - 1, i.e. block row a + i, and only rows whose input was a
    verified proposal (index <= K) qualify; 'suffix' additionally requires
    the predicted position to lie inside the verified block (<= t + K), and
    'suffix-inputs' requires the row's input to be a rejected-suffix token
    (after the first rejected proposal d_{a+1})."""
    wl, m, o = _setup("fp64", carry_window=window)
    K, t = wl.K, 100
    for a in range(K + 1):
        n, rows = o.carry_map(a)
        t_next = t + a + 1
        expect = []
        for i in range(1, K + 1):
            src_pos = t_next + i - 1
            row = src_pos - t
            if row <= a or row > K:
                continue
            if window == "suffix" and src_pos + 1 > t + K:
                continue
            if window == "suffix-inputs" and row < a + 2:
                continue
            expect.append((i, row))
        assert n == len(expect)
        assert [(r - a, r) for r in rows] == expect


@pytest.mark.parametrize("mode", ["fp64", "fp32"])
def test_rollback_matches_fresh_prefill(mode):
    wl, m, o = _setup(mode)
    prompt = make_prompts(wl)[0][:64]
    ref = o.greedy_decode(prompt, 6 * wl.block)
    traj = np.array(list(prompt) + ref, np.int64)
    sched = make_schedule(wl, 5)
    s = o.prefill(prompt)
    for r in range(5):
        o.round(s, True, force=(traj, sched["mode"][r, 0], sched["tok"][r, 0]))
    fresh = o.prefill(s.tokens[:-1])
    assert fresh.tokens == s.tokens
    tol = 1e-12 if mode == "fp64" else 2e-5
    for a, b in [(s.F, fresh.F)] + list(zip(s.k, fresh.k)) + list(zip(s.v, fresh.v)) + \
            list(zip(s.ck, fresh.ck)) + list(zip(s.cv, fresh.cv)):
        assert a.shape == b.shape
        np.testing.assert_allclose(a, b, rtol=tol, atol=tol)


def test_relay_off_is_mask_embedding_drafter():
    """Invariant 4: with relay disabled, drafter inputs are E(anchor) followed
    by the mask embedding, built here directly, and the drafts are those of
    the plain mask-embedding drafter."""
    wl, m, o = _setup("fp64")
    prompt = make_prompts(wl)[0][:48]
    s = o.prefill(prompt)
    rng = np.random.default_rng(3)
    o.round(s, True, block=np.concatenate([[s.anchor], rng.integers(0, wl.dims.vocab, wl.K)]))
    assert s.carry.n > 0
    d_off, lg_off, x_off, n_relay = o.draft(s, carry_on=False)
    assert n_relay == 0
    x = np.stack([m.w("embed")[s.anchor]] + [m.w("draft.e_mask")] * wl.K)
    np.testing.assert_array_equal(x_off, x)
    lg = m.drafter_block(x, s.t, s.ck, s.cv)[1:]
    np.testing.assert_array_equal(lg_off, lg)
    d_on, lg_on, _, n_on = o.draft(s, carry_on=True)
    assert n_on == s.carry.n and np.abs(lg_on - lg_off).max() > 1e-6


@pytest.mark.parametrize("mode", ["fp64", "fp32"])
def test_zero_relay_output_equals_relay_off(mode, tiny_weights):
    wl, w = tiny_weights
    w2 = dict(w)
    w2["relay.w2"] = np.zeros_like(w["relay.w2"])
    w2["relay.c2"] = np.zeros_like(w["relay.c2"])
    _, m, o = _setup(mode, w=w2)
    prompt = make_prompts(wl)[0][:48]
    s_on, s_off = o.prefill(prompt), o.prefill(prompt)
    rng = np.random.default_rng(4)
    for r in range(4):
        blk = np.concatenate([[s_on.anchor], rng.integers(0, wl.dims.vocab, wl.K)])
        r_on = o.round(s_on, True, block=blk)
        r_off = o.round(s_off, False, block=blk)
        np.testing.assert_array_equal(r_on.x_in, r_off.x_in)
        np.testing.assert_array_equal(r_on.draft_logits, r_off.draft_logits)
        assert r_on.committed == r_off.committed


def test_forced_block_rule():
    traj = np.arange(100, 200)
    mode = np.array([1, 1, 1, 2, 0, 0, 1, 1])
    tok = np.array([0, 0, 0, 5, 7, 8, 0, 0])
    blk = forced_block(42, 10, traj, mode, tok, 4096)
    assert list(blk) == [42, 111, 112, (113 + 1 + 5) % 4096, 7, 8, 116, 117]


@pytest.mark.parametrize("window", ["suffix", "suffix+tail", "suffix-inputs"])
def test_relay_window_placement_and_losslessness(window):
    """The relayed rows land at the block indices the window names (the
    others keep the mask embedding), the committed stream stays the plain
    greedy one, and the relay changes the drafts."""
    wl, m, o = _setup("fp64", carry_window=window)
    prompt = make_prompts(wl)[0][:40]
    ref = o.greedy_decode(prompt, 5 * wl.block)
    traj = np.array(list(prompt) + ref, np.int64)
    s = o.prefill(prompt)
    K = wl.K
    for a in [1, 3, 0, K - 1]:
        t = s.t
        block = np.concatenate([[s.anchor], traj[t + 1:t + 1 + a], [(traj[t + 1 + a] + 1) % wl.dims.vocab],
                                np.zeros(K - a - 1, np.int64)])[:wl.block]
        rr = o.round(s, True, block=block)
        assert rr.a == a
        n, rows = o.carry_map(a)
        x, n_relay = o.draft_inputs(s, True)
        idx = [r - a for r in rows]
        assert n_relay == n and s.carry.i0 == (idx[0] if idx else 1)
        mask = m.w("draft.e_mask")
        for i in range(1, wl.block):
            if i in idx:
                assert not np.array_equal(x[i], mask), (window, a, i)
            else:
                np.testing.assert_array_equal(x[i], mask)
    assert s.tokens == [int(v) for v in traj[:s.t + 1]]
