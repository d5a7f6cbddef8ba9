"""The allocation-free draft sampling call (dflow_sample_draft_noalloc)
against the workspace call it varies (dflow_sample_draft), through the C-ABI
on the same seeded synthetic drafter logits at the Qwen3 vocabulary: drafts
and block rows bit-identical on two calls in a row, the first at the largest
batch the fixed scratch holds (58 sequences x 15 rows x 149 chunks of keys),
the second with fewer sequences and other logits and positions; a request
beyond the scratch is rejected before any launch."""
import numpy as np
import pytest

from workload.configs import ModelDims
from workload.synth import make_weights

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

V, B = 151936, 16


def _logits(nseq, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randn(nseq * B, V, generator=g, device="cuda") * 2.0


def _call(rt, fn, nseq, dl, pos, anc, smp):
    draft = torch.full((nseq, B - 1), -7, dtype=torch.int32, device="cuda")
    block = torch.full((nseq, B), -7, dtype=torch.int32, device="cuda")
    fn(nseq, dl, anc, pos, smp, draft, block)
    torch.cuda.synchronize()
    return draft.cpu().numpy(), block.cpu().numpy()


def test_noalloc_sample_draft_equals_workspace_call():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.runtime import DFlowError
    dims = ModelDims("f32", 256, 2, 4, 2, 64, 768, V, 1, (0, 1))
    rt = Runtime(dims, B, 64, 256, make_weights(dims, 1), "suffix")
    streams = torch.arange(64, dtype=torch.int64, device="cuda") * 13 + 5
    smp = rt.sampler(0.8, 0x5EED_0002, streams)
    chunks = (V + 1023) // 1024
    n_max = (1 << 20) // (8 * (B - 1) * chunks)
    assert n_max == 58
    for call, (nseq, seed) in enumerate([(n_max, 11), (3, 12)]):
        dl = _logits(nseq, seed)
        pos = torch.randint(0, 5000, (nseq,), dtype=torch.int32, device="cuda", generator=torch.Generator(
            device="cuda").manual_seed(seed + 100))
        anc = torch.arange(nseq, dtype=torch.int32, device="cuda") * 31 + call
        d_ws, b_ws = _call(rt, rt.sample_draft, nseq, dl, pos, anc, smp)
        d_na, b_na = _call(rt, rt.sample_draft_noalloc, nseq, dl, pos, anc, smp)
        np.testing.assert_array_equal(d_na, d_ws, err_msg=f"call {call}: drafts")
        np.testing.assert_array_equal(b_na, b_ws, err_msg=f"call {call}: block rows")
        assert (b_na[:, 0] == anc.cpu().numpy()).all() and (d_na >= 0).all() and (d_na < V).all()
        print(f"[noalloc] call {call}: {nseq} sequences, {nseq * (B - 1)} drawn rows equal", flush=True)
    with pytest.raises(DFlowError, match="exceed the fixed scratch"):
        big = torch.empty(1, dtype=torch.float32, device="cuda")   # never read: rejected before any launch
        rt.sample_draft_noalloc(n_max + 1, big, anc, pos, smp,
                                torch.empty((n_max + 1, B - 1), dtype=torch.int32, device="cuda"))
    assert rt.status() == 0
    rt.close()
