"""HIP-graph replay of the round (Session.capture_round): one recorded graph
of draft_block, the forcing step, verify_block, accept_and_carry and
kv_commit, replayed once per round with that round's forcing plan copied in,
must reproduce the eager rounds bit for bit -- drafts, verified blocks,
target argmax, acceptance lengths, bonus tokens, committed tokens, carry
counts, sequence lengths -- and leave the same KV and drafter-context
caches.  Between replays the test synchronises and runs unrelated eager
work (the graph holds kernel launches only, no memset nodes).  Workloads:
tiny-f32 (fp32) and small-bf16 (three ragged sequences), relay on."""
import numpy as np
import pytest

from tests.gpu_common import gpu_trajectory
from workload import get_config
from workload.synth import make_prompts, make_schedule, make_weights, trajectory_length_needed

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

OUT = ("draft_tok", "block", "tgt", "accept", "anchor", "committed", "n_carry", "seq_len")


@pytest.mark.parametrize("name", ["tiny-f32", "small-bf16"])
def test_graph_replay_equals_eager(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.session import Session
    wl = get_config(name)
    dm, B, b = wl.dims, wl.block, wl.batch
    R = 6
    w = make_weights(dm, wl.seed_w)
    prompts = make_prompts(wl)
    sched = make_schedule(wl, R)
    need = trajectory_length_needed(wl, sched)
    rt = Runtime(dm, B, b, max(need) + 2 * B, w, wl.carry_window)
    sess = Session(rt, b)
    print(f"[graph] {name}: b={b}, {R} rounds", flush=True)
    traj = torch.from_numpy(gpu_trajectory(rt, sess, prompts, need)).cuda()
    L = traj.shape[1]
    mode = torch.from_numpy(sched["mode"]).cuda()
    tok = torch.from_numpy(sched["tok"]).cuda()

    sess.prefill(prompts)
    eager = []
    for r in range(R):
        sess.round(True, force=(traj, L, mode[r], tok[r]))
        torch.cuda.synchronize()
        eager.append({k: getattr(sess, k).cpu().numpy().copy() for k in OUT})
    caches = [t.clone() for t in (rt.k_pool, rt.v_pool, rt.ck_pool, rt.cv_pool)]
    assert rt.status() == 0

    sess.prefill(prompts)
    replay = sess.capture_round(True, force=(traj, L))
    scratch = torch.randn(1 << 16, device="cuda")
    for r in range(R):
        replay(mode[r], tok[r])
        torch.cuda.synchronize()
        scratch.mul_(0.5).add_(1.0)      # eager work between replays
        torch.cuda.synchronize()
        for k in OUT:
            np.testing.assert_array_equal(getattr(sess, k).cpu().numpy(), eager[r][k], err_msg=f"round {r} {k}")
    for a, e in zip((rt.k_pool, rt.v_pool, rt.ck_pool, rt.cv_pool), caches):
        assert torch.equal(a, e)
    assert rt.status() == 0
    print(f"[graph] {name}: {R} replays equal the eager rounds; accept per round "
          f"{[e['accept'].tolist() for e in eager]}", flush=True)
    rt.close()
