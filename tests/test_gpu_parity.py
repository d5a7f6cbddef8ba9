"""GPU parity: the C-ABI round (draft, verify, accept-and-carry, commit) against
the CPU oracle on the same seeded inputs, round by round.

Bar: logits, captured verifier states and projected features within 1e-4
(fp32) / 2e-2 (bf16) relative L2 error per row; argmax tokens, acceptance
lengths, bonus tokens, committed tokens and carry counts bit-exact, except
where the oracle's top-1 margin (relative to max |logit|) is within the
tolerance (an excused near-tie: the oracle then follows the device's
decision).  bf16 additionally requires argmax agreement wherever the margin
exceeds four times the observed logit error of the row.
"""
from dataclasses import replace

import numpy as np
import pytest

from tests.gpu_common import TOL, check_argmax as _check_argmax, dev_values, margin_rel, rel_rows
from workload import get_config
from workload.synth import make_prompts, make_schedule, make_weights, trajectory_length_needed

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = ["tiny-f32", "small-f32", "small-bf16", "tiny-f32-b20"]


@pytest.fixture(scope="module")
def lib():
    from paper_2609_06498_amd import load_library
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return load_library()


def _setup(name, window=None, capacity=None, n_heads=None):
    from oracle import Mode, OracleDFlow, OracleModel
    from paper_2609_06498_amd import Runtime
    wl = get_config(name)
    if window is not None:
        wl = wl.with_(carry_window=window)
    if n_heads is not None:   # another GQA group size at the same widths
        wl = wl.with_(dims=replace(wl.dims, n_heads=n_heads))
    dm = wl.dims
    w = make_weights(dm, wl.seed_w)
    mode = "fp32" if dm.dtype == "f32" else "bf16"
    o = OracleDFlow(OracleModel(dm, w, Mode(mode)), wl.block, wl.carry_window)
    prompts = make_prompts(wl)
    sched = make_schedule(wl)
    need = trajectory_length_needed(wl, sched)
    max_ctx = max(need) + wl.block
    max_batch = wl.batch
    if capacity is not None:   # a larger context capacity than the sequences use
        max_batch, max_ctx = max(capacity[0], wl.batch), max(capacity[1], max_ctx)
    rt = Runtime(dm, wl.block, max_batch, max_ctx, w, wl.carry_window)
    return wl, w, o, prompts, sched, need, rt


@pytest.mark.parametrize("carry_on", [True, False])
@pytest.mark.parametrize("name", CASES)
def test_round_parity(lib, name, carry_on):
    _round_parity(name, carry_on)


@pytest.mark.parametrize("window", ["suffix+tail", "suffix-inputs"])
@pytest.mark.parametrize("name", ["tiny-f32", "small-bf16"])
def test_round_parity_carry_windows(lib, name, window):
    """The alternative readings of the relay window (Sec. 4.2) on the device."""
    _round_parity(name, True, window)


@pytest.mark.parametrize("name", ["small-f32", "small-bf16"])
def test_round_parity_multichunk(lib, name):
    """Attention splits of several LDS chunks (the running softmax carried from
    chunk to chunk, the last one partial).  The chunk count follows from the
    capacity (batch x kv heads x chunks spread over the compute units): a
    capacity of 64 sequences x 2048 positions gives splits of several chunks,
    and the 356..402-key sequence of these cases spans more than one of them."""
    _round_parity(name, True, capacity=(64, 2048), min_chunks=2)


@pytest.mark.parametrize("name", ["small-f32", "small-bf16"])
def test_round_parity_multichunk_group8(lib, name):
    """The same with a GQA group of 8 (16 query heads on 2 kv heads): 128 query
    rows per kv head, so attention takes its unfused eight-wave form (queries
    normalised and rotated by their own kernel) -- the Qwen3-32B shape's
    launch -- with multi-chunk splits."""
    _round_parity(name, True, capacity=(64, 2048), min_chunks=2, n_heads=16)


def _round_parity(name, carry_on, window=None, capacity=None, min_chunks=1, n_heads=None):
    from paper_2609_06498_amd.session import Session
    wl, w, o, prompts, sched, need, rt = _setup(name, window, capacity, n_heads)
    chunk_keys, chunks = rt.attention_split
    assert chunks >= min_chunks, (chunk_keys, chunks)
    assert max(need) > chunk_keys or min_chunks == 1
    dm, B, K, b, V = wl.dims, wl.block, wl.K, wl.batch, wl.dims.vocab
    tol = TOL[dm.dtype]
    print(f"[parity] {name} carry_on={carry_on} window={wl.carry_window} b={b} ctx={[len(p) for p in prompts]} "
          f"split={chunks}x{chunk_keys}", flush=True)
    sess = Session(rt, b)
    states = [o.prefill(p) for p in prompts]
    sess.prefill(prompts)
    torch.cuda.synchronize()
    assert rt.status() == 0
    # first anchors: exact unless the prompt's last row is a near-tie
    anc = sess.anchor.cpu().numpy()
    for s in range(b):
        if anc[s] != states[s].anchor:
            pytest.fail(f"first anchor differs for seq {s}: {anc[s]} vs {states[s].anchor}")
    # trajectories: the oracle's greedy continuation
    traj = np.zeros((b, max(need)), np.int32)
    for s in range(b):
        g = o.greedy_decode(prompts[s], need[s] - len(prompts[s]))
        traj[s, :need[s]] = np.concatenate([prompts[s], g])[:need[s]]
    traj_d = torch.from_numpy(traj).cuda()
    mode_d = torch.from_numpy(sched["mode"]).cuda()
    tok_d = torch.from_numpy(sched["tok"]).cuda()
    excused = 0
    capd = dm.m * dm.d
    for r in range(wl.rounds):
        dl = torch.zeros(b * B, V, dtype=torch.float32, device="cuda")
        lg = torch.zeros(b * B, V, dtype=torch.float32, device="cuda")
        hc = torch.zeros(b * B * capd, dtype=rt.elt_torch, device="cuda")
        ft = torch.zeros(b * B * dm.d, dtype=rt.elt_torch, device="cuda")
        sess.round(carry_on, force=(traj_d, traj.shape[1], mode_d[r], tok_d[r]), draft_logits=dl, logits=lg,
                   hcap=hc, feat=ft)
        torch.cuda.synchronize()
        g_dl, g_lg = dl.cpu().numpy(), lg.cpu().numpy()
        g_hc = dev_values(hc, dm.dtype).reshape(b * B, capd)
        g_ft = dev_values(ft, dm.dtype).reshape(b * B, dm.d)
        g_blk, g_tgt = sess.block.cpu().numpy(), sess.tgt.cpu().numpy()
        g_draft = sess.draft_tok.cpu().numpy()
        g_a, g_bonus = sess.accept.cpu().numpy(), sess.anchor.cpu().numpy()
        g_com, g_nc = sess.committed.cpu().numpy(), sess.n_carry.cpu().numpy()
        g_len = sess.seq_len.cpu().numpy()
        for s in range(b):
            rows = slice(s * B, (s + 1) * B)
            hold = {}

            def decide(a, bonus, logits, s=s, hold=hold):
                hold["logits"] = logits
                if (a, bonus) == (int(g_a[s]), int(g_bonus[s])):
                    return a, bonus
                mr = margin_rel(logits)
                crit = mr[:min(max(a, int(g_a[s])), K) + 1]
                assert (crit <= tol).any(), \
                    f"r{r} s{s}: acceptance (a={g_a[s]}, b={g_bonus[s]}) vs oracle ({a}, {bonus}), margins {crit}"
                hold["excused"] = True
                return int(g_a[s]), int(g_bonus[s])

            rr = o.round(states[s], carry_on, force=(traj[s], sched["mode"][r, s], sched["tok"][r, s]),
                         decide=decide)
            excused += int(hold.get("excused", False))
            ctx = f"{name} r{r} s{s}"
            np.testing.assert_array_equal(g_blk[s], rr.block, err_msg=ctx + " block")
            e = rel_rows(g_dl[rows][1:], rr.draft_logits)
            assert e.max() <= tol, f"{ctx} draft logits rel err {e.max()}"
            err_abs = np.abs(g_dl[rows][1:] - rr.draft_logits).max(axis=1) if dm.dtype == "bf16" else None
            _check_argmax(g_draft[s], rr.draft_logits, tol, err_abs)
            e = rel_rows(g_lg[rows], rr.logits)
            assert e.max() <= tol, f"{ctx} verify logits rel err {e.max()}"
            err_abs = np.abs(g_lg[rows] - rr.logits).max(axis=1) if dm.dtype == "bf16" else None
            _check_argmax(g_tgt[s], rr.logits, tol, err_abs)
            e = rel_rows(g_hc[rows], rr.hcap)
            assert e.max() <= tol, f"{ctx} captured states rel err {e.max()}"
            e = rel_rows(g_ft[rows], rr.f)
            assert e.max() <= tol, f"{ctx} projected features rel err {e.max()}"
            assert int(g_a[s]) == rr.a and int(g_bonus[s]) == rr.bonus, ctx
            assert list(g_com[s][:rr.a + 1]) == rr.committed and (g_com[s][rr.a + 1:] == -1).all(), ctx
            assert int(g_nc[s]) == rr.n_carry, ctx
            assert int(g_len[s]) == states[s].t, ctx
        print(f"[parity] {name} round {r}: a={list(g_a)} n_carry={list(g_nc)}", flush=True)
    assert rt.status() == 0
    print(f"[parity] {name} carry_on={carry_on}: excused rounds {excused}", flush=True)
    rt.close()
