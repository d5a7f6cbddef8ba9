"""GPU properties at the full batched shapes, where the oracle cannot follow:

* qwen3-8b-b8: the Qwen3-8B shape with 8 sequences of ragged contexts
  (2048..8192 positions), M = 128 verify rows;
* qwen3-32b: the Qwen3-32B shape (64 + 5 layers, d 5120, GQA group 8),
  4 sequences of 16384 positions;
* small-bf16-b24: 24 sequences, M = 384 rows, so the batched run takes the
  tiled GEMM and each sequence alone the weight-streaming one; the same model
  at 4 and 16 sequences (M = 64 and 256, the first row counts above and the
  last row count within the K-split and range-split paths).

Batch invariance: every kernel's arithmetic for a row depends only on that
row's own data (K reductions split by (N, K) only, attention splits at fixed
absolute positions, work units fixed by (B, G)), so one sequence run alone
must reproduce its rows of the batched run bit for bit -- logits, draft
tokens, verify argmax, acceptance, committed tokens and carry -- round after
round with ragged acceptance, ragged KV rollback and ragged carry.  The
drafts are forced from the target's own greedy trajectory (made on the GPU by
junk-draft rounds) with the workload's seeded geometric acceptance, and the
realised acceptance must follow the schedule exactly (the forced prefix is
accepted, the forced mismatch rejected), which also checks losslessness
against the GPU's own greedy decode."""
import numpy as np
import pytest

from tests.gpu_common import gpu_trajectory
from workload import get_config
from workload.synth import make_prompts, make_schedule, make_weights, trajectory_length_needed

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name, rounds, alone", [("qwen3-8b-b8", 3, "extremes"), ("qwen3-32b", 2, "extremes"),
                                                 ("small-bf16-b24", 3, "all"), ("small-bf16-b24@4", 3, "all"),
                                                 ("small-bf16-b24@16", 2, "extremes")])
def test_batch_invariance(name, rounds, alone):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.session import Session
    base, _, nb = name.partition("@")
    wl = get_config(base)
    if nb:   # the same workload at another sequence count
        wl = wl.with_(name=name, batch=int(nb))
    dm, B, b, V = wl.dims, wl.block, wl.batch, wl.dims.vocab
    prompts = make_prompts(wl)
    sched = make_schedule(wl, rounds)
    need = trajectory_length_needed(wl, sched)
    print(f"[invariance] {name}: b={b} ctx={[len(p) for p in prompts]} rounds={rounds}", flush=True)
    w = make_weights(dm, wl.seed_w)
    P = [len(p) for p in prompts]   # trajectory rounds advance all sequences together
    rt = Runtime(dm, B, b, max(P) + max(n - q for n, q in zip(need, P)) + 2 * B, w, wl.carry_window)
    del w
    sess = Session(rt, b)
    traj = gpu_trajectory(rt, sess, prompts, need)
    traj_d = torch.from_numpy(traj).cuda()
    L = traj.shape[1]
    mode_d = torch.from_numpy(sched["mode"]).cuda()
    tok_d = torch.from_numpy(sched["tok"]).cuda()
    assert rt.status() == 0

    def run(sess, seqs, r):
        lg = torch.zeros(len(seqs) * B, V, dtype=torch.float32, device="cuda")
        dl = torch.zeros(len(seqs) * B, V, dtype=torch.float32, device="cuda")
        idx = torch.tensor(seqs, device="cuda")
        sess.round(True, force=(traj_d[idx].contiguous(), L, mode_d[r][idx].contiguous(), tok_d[r][idx].contiguous()),
                   draft_logits=dl, logits=lg)
        torch.cuda.synchronize()
        return {"logits": lg.cpu().numpy(), "draft_logits": dl.cpu().numpy(), "block": sess.block.cpu().numpy(),
                "tgt": sess.tgt.cpu().numpy(), "draft": sess.draft_tok.cpu().numpy(),
                "accept": sess.accept.cpu().numpy(), "committed": sess.committed.cpu().numpy(),
                "n_carry": sess.n_carry.cpu().numpy(), "seq_len": sess.seq_len.cpu().numpy()}

    sess.prefill(prompts)
    batched = [run(sess, list(range(b)), r) for r in range(rounds)]
    for r in range(rounds):
        np.testing.assert_array_equal(batched[r]["accept"], sched["accept"][r], err_msg=f"r{r} schedule")
    print(f"[invariance] batched accept per round {[list(x['accept']) for x in batched]}", flush=True)
    lens = [len(p) for p in prompts]
    picks = sorted({int(np.argmin(lens)), int(np.argmax(lens))}) if alone == "extremes" else list(range(b))
    for s in picks:
        one = Session(rt, 1)
        one.prefill([prompts[s]])
        for r in range(rounds):
            got = run(one, [s], r)
            rows = slice(s * B, (s + 1) * B)
            for key in ("logits", "draft_logits"):
                ok = np.array_equal(got[key], batched[r][key][rows])
                assert ok, f"{name} seq {s} round {r}: {key} differ alone vs batched " \
                           f"(max abs {np.abs(got[key] - batched[r][key][rows]).max()})"
            for key in ("block", "tgt", "draft", "committed"):
                np.testing.assert_array_equal(got[key][0], batched[r][key][s], err_msg=f"seq {s} r{r} {key}")
            for key in ("accept", "n_carry", "seq_len"):
                assert int(got[key][0]) == int(batched[r][key][s]), f"seq {s} r{r} {key}"
        print(f"[invariance] seq {s} (ctx {lens[s]}) alone == batched for {rounds} rounds", flush=True)
    assert rt.status() == 0
    rt.close()
