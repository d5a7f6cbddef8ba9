"""GPU serving: the continuous-batching engine over the C-ABI round calls.

Requests outnumber the engine's slots, so admissions happen while other
requests are mid-decode and finished requests are compacted away (page-table
row swaps plus dflow_move_slot).  Bars:
  * lossless greedy decoding (Sec. 4: greedy verification commits exactly the
    target's greedy continuation): every generated token is the oracle's
    argmax given the device's own prefix, checked with one teacher-forced
    oracle forward over prompt + output; a token may differ only where the
    oracle's top-1 margin is within the dtype tolerance;
  * the output of a request does not depend on which requests share its
    rounds: serving at concurrency 3 and at concurrency 1 gives bit-identical
    tokens.
Both with the drafter's own proposals and with forced acceptances (a
geometric accepted prefix from the oracle's greedy trajectory), which drives
multi-token commits, truncation at the token budget and non-empty relays.
Sampling decoding (T > 0) is served too: per-request Philox streams make its
tokens independent of concurrency as well.
"""
import numpy as np
import pytest

from tests.gpu_common import TOL, check_argmax
from workload import get_config
from workload.synth import make_weights

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

MAX_NEW = [1, 7, 33, 20, 48]
SLOTS = 3


@pytest.fixture(scope="module")
def lib():
    from paper_2609_06498_amd import load_library
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return load_library()


def _requests(wl, n):
    r = np.random.default_rng([wl.seed_prompt, 77])
    lo, hi = 40, 300
    out = []
    for i in range(n):
        P = int(r.integers(lo, hi + 1))
        out.append(r.integers(0, wl.dims.vocab, size=P).astype(np.int32))
    return out


_CACHE = {}


def _setup(name):
    if name in _CACHE:
        return _CACHE[name]
    from oracle import Mode, OracleDFlow, OracleModel
    wl = get_config(name)
    dm = wl.dims
    w = make_weights(dm, wl.seed_w)
    o = OracleDFlow(OracleModel(dm, w, Mode("fp32" if dm.dtype == "f32" else "bf16")), wl.block, wl.carry_window)
    prompts = _requests(wl, len(MAX_NEW))
    trajs = []
    for p, n in zip(prompts, MAX_NEW):
        g = o.greedy_decode(p, n + wl.block + 1)
        trajs.append(np.concatenate([p, np.asarray(g, np.int32)]))
    _CACHE[name] = (wl, w, o, prompts, trajs)
    return _CACHE[name]


def _serve(name, slots, force, carry_on=True):
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.engine import Engine
    wl, w, o, prompts, trajs = _setup(name)
    max_ctx = max(len(p) + n for p, n in zip(prompts, MAX_NEW)) + 2 * wl.block
    rt = Runtime(wl.dims, wl.block, SLOTS, max_ctx, w, wl.carry_window)
    eng = Engine(rt, max_active=slots, carry_on=carry_on, force_mean=4.0 if force else None, seed=5)
    rids = [eng.submit(p, n, traj=t if force else None) for p, n, t in zip(prompts, MAX_NEW, trajs)]
    outs = eng.run()
    torch.cuda.synchronize()
    assert rt.status() == 0
    stats = {"rounds": eng.rounds, "max_active": max(eng.active_hist),
             "accepted": sum(r.accepted for r in eng.done.values())}
    rt.close()
    return [outs[i] for i in rids], stats


@pytest.mark.parametrize("force", [False, True])
@pytest.mark.parametrize("name", ["tiny-f32", "small-f32", "small-bf16"])
def test_serving_is_greedy(lib, name, force):
    wl, w, o, prompts, trajs = _setup(name)
    print(f"[serving] {name} force={force} slots={SLOTS} requests={len(prompts)}", flush=True)
    outs, stats = _serve(name, SLOTS, force)
    assert stats["max_active"] == SLOTS
    if force:
        assert stats["accepted"] > 0
    tol = TOL[wl.dims.dtype]
    excused = 0
    for p, n, y in zip(prompts, MAX_NEW, outs):
        assert len(y) == n
        seq = np.concatenate([p, np.asarray(y, np.int32)])
        lg = o.full_logits(seq[:-1])[len(p) - 1:]
        excused += check_argmax(np.asarray(y), lg, tol)
    print(f"[serving] {name} force={force} rounds={stats['rounds']} accepted={stats['accepted']} "
          f"near-ties={excused}", flush=True)


@pytest.mark.parametrize("force", [False, True])
def test_serving_concurrency_invariant(lib, force):
    print(f"[serving] small-bf16 concurrency invariance force={force}", flush=True)
    one, _ = _serve("small-bf16", 1, force)
    many, stats = _serve("small-bf16", SLOTS, force)
    assert stats["max_active"] == SLOTS
    for i, (a, b) in enumerate(zip(one, many)):
        assert a == b, f"request {i}: outputs differ at concurrency 1 and {SLOTS}"


def test_serving_many_slots_invariant(lib):
    """30 requests through 24 slots (up to 384 rows per round, the tiled
    GEMM) give the same tokens as through one slot (16 rows)."""
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.engine import Engine
    wl = get_config("small-bf16")
    w = make_weights(wl.dims, wl.seed_w)
    r = np.random.default_rng([wl.seed_prompt, 91])
    prompts = [r.integers(0, wl.dims.vocab, size=int(r.integers(20, 200))).astype(np.int32) for _ in range(30)]
    budgets = [int(x) for x in r.integers(1, 24, size=30)]
    print(f"[serving] small-bf16 30 requests, 24 slots vs 1", flush=True)
    rt = Runtime(wl.dims, wl.block, 24, 200 + 24 + 2 * wl.block, w, wl.carry_window)
    outs = {}
    for slots in (24, 1):
        eng = Engine(rt, max_active=slots)
        rids = [eng.submit(p, n) for p, n in zip(prompts, budgets)]
        res = eng.run()
        torch.cuda.synchronize()
        assert rt.status() == 0
        assert max(eng.active_hist) == slots
        outs[slots] = [res[i] for i in rids]
    rt.close()
    for i, (a, b) in enumerate(zip(outs[1], outs[24])):
        assert a == b, f"request {i}: outputs differ with 1 and 24 slots"


def _serve_sampled(name, slots, T, n_req=None, budgets=None):
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.engine import Engine
    wl, w, o, prompts, trajs = _setup(name)
    budgets = budgets or MAX_NEW
    max_ctx = max(len(p) + n for p, n in zip(prompts, budgets)) + 2 * wl.block
    rt = Runtime(wl.dims, wl.block, SLOTS, max_ctx, w, wl.carry_window)
    eng = Engine(rt, max_active=slots, temperature=T, sample_seed=11)
    rids = [eng.submit(p, n) for p, n in zip(prompts, budgets)]
    outs = eng.run()
    torch.cuda.synchronize()
    assert rt.status() == 0
    stats = {"rounds": eng.rounds, "max_active": max(eng.active_hist),
             "accepted": sum(r.accepted for r in eng.done.values())}
    rt.close()
    return [outs[i] for i in rids], rids, stats


@pytest.mark.parametrize("T", [1.0, 0.3])
def test_serving_sampled(lib, T):
    """Speculative-sampling serving: a request's tokens are the same at
    concurrency 1 and 3 (its own Philox stream, batch-invariant logits), its
    first token is the oracle's draw from the prompt's last row, and the
    output is not the greedy one."""
    import oracle.sampling as sp
    name = "small-bf16"
    wl, w, o, prompts, trajs = _setup(name)
    print(f"[serving] {name} sampled T={T}", flush=True)
    one, rids, _ = _serve_sampled(name, 1, T)
    many, _, stats = _serve_sampled(name, SLOTS, T)
    assert stats["max_active"] == SLOTS
    for i, (a, b) in enumerate(zip(one, many)):
        assert a == b, f"request {i}: sampled outputs differ at concurrency 1 and {SLOTS}"
    tol = TOL[wl.dims.dtype]
    differs = 0
    for p, n, y, rid, t in zip(prompts, MAX_NEW, many, rids, trajs):
        assert len(y) == n
        lg = o.full_logits(p)[-1]
        inv_t = sp.inv_temperature(T)
        z = sp.scaled(lg, inv_t)
        g = sp.gumbel(sp.uniforms(11, rid, len(p) - 1, 0, sp.RESAMPLE, z.size))
        sc = z + g
        ref = int(np.argmax(sc))
        if y[0] != ref:
            assert sc[ref] - sc[y[0]] <= 2 * tol * float(np.abs(z).max()), f"request {rid}: first token"
        differs += int(list(y) != list(t[len(p):len(p) + n]))
    assert differs > 0, "sampled outputs equal the greedy continuation"
    print(f"[serving] sampled T={T}: rounds {stats['rounds']} accepted {stats['accepted']}", flush=True)
