"""Pins of the oracle's speculative sampling (oracle/sampling.py), CPU only.

* Philox4x64-10 against numpy's Philox bit generator (numpy advances its
  counter before producing a block, so its block from counter c is ours at
  c + 1), and the vectorised form against the definition in Python integers.
* The rule's law: for arbitrary p and q the first emitted token has law p
  exactly (enumeration of draft and acceptance), the defining property of
  speculative sampling (Leviathan et al., cited in Sec. 1).
* The implemented block rule, run over many independent streams: the first
  emitted token follows p_0, the second (after an acceptance) p_1,
  chi-square at a fixed seed; the Gumbel-max sampler follows softmax(z / T).
* The first token after a prompt (sample_first): its law softmax(z / T) over
  many streams, and its counter address, which no round reuses.
* Special cases: drafter = target accepts every draft; a draft the target
  gives probability 0 is always rejected and never emitted; a tiny
  temperature reduces sampling to the argmax.
* Planted mistakes (a wrong residual, wrong noise, a dropped temperature, a
  shifted verify row) fail these checks.
"""
import numpy as np
import pytest
from scipy import stats

import oracle.sampling as sp

V = 6
N_TRIALS = 4000


def test_philox_matches_numpy():
    rng = np.random.default_rng(5)
    for _ in range(20):
        key = [int(x) for x in rng.integers(0, 2**63, size=2, dtype=np.int64)]
        ctr = [int(x) for x in rng.integers(0, 2**62, size=4, dtype=np.int64)]
        bg = np.random.Philox(key=np.array(key, np.uint64), counter=np.array(ctr, np.uint64))
        raw = [int(x) for x in bg.random_raw(8)]
        c1 = (ctr[0] + 1,) + tuple(ctr[1:])
        c2 = (ctr[0] + 2,) + tuple(ctr[1:])
        assert list(sp.philox4x64_10(tuple(key), c1)) == raw[:4]
        assert list(sp.philox4x64_10(tuple(key), c2)) == raw[4:]


def test_philox_vectorised_equals_definition():
    rng = np.random.default_rng(6)
    k = rng.integers(0, 2**64, size=(50, 2), dtype=np.uint64)
    c = rng.integers(0, 2**64, size=(50, 4), dtype=np.uint64)
    out = sp.philox_np(k[:, 0], k[:, 1], c[:, 0], c[:, 1], c[:, 2], c[:, 3])
    for i in range(50):
        ref = sp.philox4x64_10((int(k[i, 0]), int(k[i, 1])), tuple(int(x) for x in c[i]))
        assert tuple(int(x) for x in out[i]) == ref


def test_uniforms_open_interval_and_addressing():
    u = sp.uniforms(3, 9, 100, 4, sp.DRAFT, 4001)
    assert u.dtype == np.float32 and u.min() > 0 and u.max() < 1
    assert abs(float(u.mean()) - 0.5) < 0.02
    # the extremes of the 23-bit grid
    assert sp.uniform_from_bits(0) == np.float32(2.0 ** -24)
    assert sp.uniform_from_bits(2**64 - 1) == np.float32(1 - 2.0 ** -24)
    # column v uses word v % 4 of block v // 4
    blk = sp.philox4x64_10((3, 9), (100, 4, sp.DRAFT, 1000))
    assert u[4000] == sp.uniform_from_bits(blk[0])
    # purposes and rows address different numbers
    assert not np.array_equal(u[:8], sp.uniforms(3, 9, 100, 4, sp.ACCEPT, 8))
    assert not np.array_equal(u[:8], sp.uniforms(3, 9, 100, 5, sp.DRAFT, 8))


@pytest.mark.parametrize("case", range(6))
def test_exact_law_is_target(case):
    r = np.random.default_rng(case)
    p = r.dirichlet(np.ones(9) * 0.5)
    q = r.dirichlet(np.ones(9) * 0.5)
    if case == 1:
        q[2] = 0.0
        q /= q.sum()
    if case == 2:
        p[4] = 0.0
        p /= p.sum()
    if case == 3:
        q = p.copy()
    np.testing.assert_allclose(sp.exact_output_distribution(p, q), p, atol=1e-14)


def test_exact_law_rejects_wrong_rules():
    r = np.random.default_rng(11)
    p, q = r.dirichlet(np.ones(7)), r.dirichlet(np.ones(7))
    acc = np.minimum(1, p / q)
    reject = (q * (1 - acc)).sum()
    # the correction drawn from p instead of the residual
    bad = q * acc + reject * p
    assert np.abs(bad - p).max() > 1e-3
    # the correction drawn from the unclipped, renormalised difference
    d = (p - q) / (p - q).sum() if abs((p - q).sum()) > 1e-9 else p
    assert np.abs(q * acc + reject * d - p).max() > 1e-3


def _rows(seed, n, scale=1.2):
    return (np.random.default_rng(seed).normal(size=(n, V)) * scale).astype(np.float32)


def _softmax64(z):
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max())
    return e / e.sum()


def _chi2_p(samples, probs):
    counts = np.bincount(samples, minlength=len(probs)).astype(np.float64)
    exp = probs * counts.sum()
    keep = exp > 0
    assert counts[~keep].sum() == 0, "a token of probability zero was sampled"
    return stats.chisquare(counts[keep], exp[keep] * counts[keep].sum() / exp[keep].sum()).pvalue


def test_gumbel_max_sampler_law():
    z = _rows(1, 1)[0]
    T = 0.7
    inv_t = sp.inv_temperature(T)
    s = [sp.gumbel_argmax(sp.scaled(z, inv_t), sp.gumbel(sp.uniforms(21, st, 50, 3, sp.DRAFT, V)))
         for st in range(N_TRIALS)]
    assert _chi2_p(np.array(s), _softmax64(z / T)) > 1e-3


def _block_trials(T=1.0, seed=17, n=N_TRIALS):
    """K = 2 block with fixed synthetic verify rows p_0..p_2 and drafter rows
    q_1, q_2 over independent streams; returns the emitted sequences."""
    tgt = _rows(2, 3)
    drf = (tgt[:2] + _rows(3, 2, scale=0.8)).astype(np.float32)   # q_i near p_{i-1}
    inv_t = sp.inv_temperature(T)
    out = []
    for st in range(n):
        d, _, _ = sp.sample_drafts(drf, inv_t, seed, st, 40)
        block = [7 % V] + [int(x) for x in d]
        dec = sp.accept_sampled(block, tgt, drf, inv_t, seed, st, 40)
        out.append(block[1:dec.a + 1] + [dec.bonus])
    return tgt, out


def _law_pvalues(tgt, out, T=1.0):
    first = np.array([o[0] for o in out])
    second = np.array([o[1] for o in out if len(o) >= 2])
    assert len(second) > len(out) // 4
    return _chi2_p(first, _softmax64(tgt[0] / T)), _chi2_p(second, _softmax64(tgt[1] / T))


def test_block_rule_keeps_target_law():
    tgt, out = _block_trials()
    p1, p2 = _law_pvalues(tgt, out)
    assert p1 > 1e-3 and p2 > 1e-3, (p1, p2)
    # all three outcomes occur: early rejection, one acceptance, full acceptance
    lens = np.bincount([len(o) for o in out], minlength=4)
    assert (lens[1:4] > 100).all(), lens


def test_block_rule_at_temperature():
    T = 0.6
    tgt, out = _block_trials(T=T, seed=23)
    p1, p2 = _law_pvalues(tgt, out, T=T)
    assert p1 > 1e-3 and p2 > 1e-3, (p1, p2)


def test_drafter_equal_to_target_accepts_everything():
    tgt = _rows(4, 4)
    for st in range(50):
        d, _, _ = sp.sample_drafts(tgt[:3], np.float32(1), 5, st, 9)
        # the drafter's row i equals the target's row i-1
        dec = sp.accept_sampled([0] + list(d), tgt, tgt[:3], np.float32(1), 5, st, 9)
        assert dec.a == 3


def test_zero_probability_draft_is_rejected():
    tgt = _rows(5, 2)
    tgt[0, 2] = -np.inf                  # p_0(2) = 0
    drf = _rows(6, 1)
    for st in range(200):
        dec = sp.accept_sampled([1, 2], tgt, drf, np.float32(1), 8, st, 3)
        assert dec.a == 0 and dec.bonus != 2


def test_low_temperature_is_argmax():
    z = np.array([[0.3, 1.9, -0.4, 1.2, 0.0, 1.85]], np.float32)
    for st in range(50):
        d, _, _ = sp.sample_drafts(z, sp.inv_temperature(1e-3), 2, st, 0)
        assert d[0] == 1


def test_temperature_must_be_positive():
    for bad in (0.0, -1.0, float("inf"), float("nan")):
        with pytest.raises(ValueError):
            sp.inv_temperature(bad)


# ------------------------------------------------------------ the first token after a prompt
def _first_and_round(seed, stream, z, t_last):
    """The prompt's first token (sample_first at position t_last) and the first
    draft of the round that follows (anchor at t_last + 1), both drawn from
    the same logits row."""
    inv_t = sp.inv_temperature(1.0)
    first = sp.sample_first(z, inv_t, seed, stream, t_last)
    d, _, _ = sp.sample_drafts(z[None], inv_t, seed, stream, t_last + 1)
    return first, int(d[0])


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_sample_first_law(T):
    """The first token after a prompt follows softmax(z / T) over independent
    streams (chi-square), and a vanishing temperature makes it the argmax."""
    z = _rows(31, 1)[0]
    inv_t = sp.inv_temperature(T)
    s = np.array([sp.sample_first(z, inv_t, 13, st, 77) for st in range(N_TRIALS)])
    assert _chi2_p(s, _softmax64(z / T)) > 1e-3
    assert all(sp.sample_first(z, sp.inv_temperature(1e-4), 13, st, 77) == int(np.argmax(z)) for st in range(20))


def test_sample_first_counter_is_disjoint_from_the_rounds(monkeypatch):
    """The first token's random numbers are addressed at (t_last, 0, correction),
    which no round addresses: rounds start at t_last + 1 and draw corrections
    at block indices >= 1.  Recorded over a sampled round, no counter repeats,
    and over many streams the first token and the following round's first
    draft (same logits row) agree at the rate of independent draws, sum p^2,
    not always as shared numbers would make them."""
    seen = []
    real = sp.uniforms
    monkeypatch.setattr(sp, "uniforms", lambda seed, stream, pos, row, purpose, n:
                        seen.append((pos, row, purpose)) or real(seed, stream, pos, row, purpose, n))
    z = _rows(32, 1)[0]
    sp.sample_first(z, np.float32(1), 3, 0, 40)
    first_addr = set(seen)
    seen.clear()
    tgt = _rows(33, 4)
    d, _, _ = sp.sample_drafts(tgt[:3], np.float32(1), 3, 0, 41)
    sp.accept_sampled([1] + list(d), tgt, tgt[:3], np.float32(1), 3, 0, 41)
    assert first_addr == {(40, 0, sp.RESAMPLE)} and not first_addr & set(seen)
    monkeypatch.setattr(sp, "uniforms", real)
    p = _softmax64(z)
    same = np.mean([a == b for a, b in (_first_and_round(5, st, z, 40) for st in range(N_TRIALS))])
    assert abs(same - (p * p).sum()) < 0.03, (same, (p * p).sum())


def test_mutation_first_token_reuses_the_rounds_numbers(monkeypatch):
    """Planted mistake: the first token addressed like the next round's first
    draft.  The agreement-rate pin catches it."""
    monkeypatch.setattr(sp, "sample_first", lambda z, inv_t, seed, stream, t_last: int(
        sp.sample_drafts(np.asarray(z)[None], inv_t, seed, stream, t_last + 1)[0][0]))
    z = _rows(32, 1)[0]
    p = _softmax64(z)
    same = np.mean([a == b for a, b in (_first_and_round(5, st, z, 40) for st in range(500))])
    assert abs(same - (p * p).sum()) > 0.3


# ------------------------------------------------------------ planted mistakes
def _mut_residual_is_p(lp, lq):
    return np.asarray(lp, np.float32)


def _mut_exponential_noise(u):
    return (-np.log(np.asarray(u, np.float32))).astype(np.float32)


def test_mutation_residual(monkeypatch):
    monkeypatch.setattr(sp, "residual_logw", _mut_residual_is_p)
    tgt, out = _block_trials(n=2000)
    assert min(_law_pvalues(tgt, out)) < 1e-6


def test_mutation_noise(monkeypatch):
    monkeypatch.setattr(sp, "gumbel", _mut_exponential_noise)
    tgt, out = _block_trials(n=2000)
    assert min(_law_pvalues(tgt, out)) < 1e-6


def test_mutation_dropped_temperature(monkeypatch):
    monkeypatch.setattr(sp, "inv_temperature", lambda T: np.float32(1))
    tgt, out = _block_trials(T=0.6, n=2000)
    assert min(_law_pvalues(tgt, out, T=0.6)) < 1e-6


def test_mutation_verify_row_shift(monkeypatch):
    """Scoring d_i with p_i instead of p_{i-1}."""
    real = sp.accept_sampled

    def shifted(block, logits, draft_logits, *a, **k):
        lg = np.concatenate([logits[1:], logits[-1:]])
        return real(block, lg, draft_logits, *a, **k)

    monkeypatch.setattr(sp, "accept_sampled", shifted)
    tgt, out = _block_trials(n=2000)
    assert min(_law_pvalues(tgt, out)) < 1e-6


# ------------------------------------------------------------ whole rounds on the tiny model
def _tiny(mode="fp32"):
    from oracle import Mode, OracleDFlow, OracleModel
    from workload import get_config
    from workload.synth import make_prompts, make_weights
    wl = get_config("tiny-f32")
    w = make_weights(wl.dims, wl.seed_w)
    return wl, OracleDFlow(OracleModel(wl.dims, w, Mode(mode)), wl.block), make_prompts(wl)[0][:48]


def test_vanishing_temperature_is_the_greedy_round():
    """At T -> 0 the drafter samples its argmax, the target's distributions are
    one-hot, and the rule accepts exactly the drafts equal to the target's
    argmax and corrects with it: the round equals the greedy round."""
    wl, o, prompt = _tiny()
    s1, s2 = o.prefill(prompt), o.prefill(prompt)
    for r in range(3):
        g = o.round(s1, True)
        res, _, _, dec = o.round_sampled(s2, 1e-6, seed=4, stream=r)
        assert list(res.draft) == list(g.draft)
        assert (res.a, res.committed) == (g.a, g.committed)
        assert not dec.fallback
    assert s1.tokens == s2.tokens


def test_sampled_rounds_roll_back_like_a_fresh_prefill():
    wl, o, prompt = _tiny()
    s = o.prefill(prompt)
    lens = []
    for r in range(4):
        res, zq, gq, dec = o.round_sampled(s, 1.0, seed=9, stream=3)
        assert res.committed[:-1] == [int(x) for x in res.block[1:res.a + 1]]
        assert 0 <= res.bonus < wl.dims.vocab
        lens.append(res.a)
    assert s.carry is not None
    fresh = o.prefill(s.tokens[:-1])
    for a, b in [(s.F, fresh.F)] + list(zip(s.k, fresh.k)) + list(zip(s.v, fresh.v)):
        assert a.shape == b.shape
        np.testing.assert_allclose(a, b, rtol=2e-5, atol=2e-5)
