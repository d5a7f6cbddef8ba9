"""Planted mistakes in the oracle (CPU only) must be caught by the pins.

Each case monkeypatches one oracle function with a plausible error and checks
that the corresponding pin comparison no longer holds."""
import numpy as np
import pytest
import torch

import oracle.model as om
from oracle import Mode, OracleDFlow, OracleModel
from workload import get_config
from workload.synth import make_prompts, make_weights

from .test_oracle_pins import _hf_model


@pytest.fixture(scope="module")
def setup():
    wl = get_config("tiny-f32")
    w = make_weights(wl.dims, wl.seed_w)
    prompt = make_prompts(wl)[0][:64]
    hf = _hf_model(wl.dims, w)
    with torch.no_grad():
        ref = hf(torch.from_numpy(prompt.astype(np.int64))[None]).logits[0].numpy()
    return wl, w, prompt, ref


def _hf_err(wl, w, prompt, ref):
    o = OracleDFlow(OracleModel(wl.dims, w, Mode("fp64")), wl.block)
    lg = o.full_logits(prompt)
    return (np.linalg.norm(lg - ref, axis=1) / np.linalg.norm(ref, axis=1)).max()


def test_unmutated_passes(setup):
    assert _hf_err(*setup) < 1e-5


def _rope_sign(self, x, pos):
    ang = np.asarray(pos, np.float64)[:, None] * self.inv_freq[None, :]
    cos, sin = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    h = x.shape[-1] // 2
    return np.concatenate([x[..., :h] * cos + x[..., h:] * sin, x[..., h:] * cos - x[..., :h] * sin], -1)


def _rms_no_gain(self, x, g, eps):
    x = np.asarray(x, self.mode.dt)
    return x / np.sqrt(np.mean(x * x, -1, keepdims=True) + eps)


def _gqa_modulo(self, q, k, v, visible):
    n, Hq, Dh = q.shape
    kv_of = np.arange(Hq) % self.dims.n_kv_heads
    s = np.einsum("nhd,mhd->hnm", q, k[:, kv_of]) / np.sqrt(Dh)
    s = np.where(visible[None], s, -np.inf)
    p = np.exp(s - s.max(-1, keepdims=True))
    p /= p.sum(-1, keepdims=True)
    return np.einsum("hnm,mhd->nhd", p, v[:, kv_of]).reshape(n, -1)


def _no_causal(self, prefix, x, pos, k_past, v_past, past_pos, causal):
    return _orig_layer(self, prefix, x, pos, k_past, v_past, past_pos, False)


_orig_layer = om.OracleModel.decoder_layer


@pytest.mark.parametrize("name,fn", [("rope", _rope_sign), ("rms_norm", _rms_no_gain),
                                     ("attention", _gqa_modulo), ("decoder_layer", _no_causal)])
def test_target_mutations_caught_by_hf_pin(setup, monkeypatch, name, fn):
    monkeypatch.setattr(om.OracleModel, name, fn)
    assert _hf_err(*setup) > 1e-3


def test_carry_shift_mutation_caught():
    from .test_oracle_invariants import test_carry_index_map_against_positions
    orig = OracleDFlow.carry_map

    def shifted(self, a):
        n, rows = orig(self, a)
        return n, [r + 1 for r in rows]
    OracleDFlow.carry_map = shifted
    try:
        with pytest.raises(AssertionError):
            test_carry_index_map_against_positions("suffix")
    finally:
        OracleDFlow.carry_map = orig


def test_bonus_mutation_caught():
    from .test_oracle_invariants import test_acceptance_brute_force
    orig = OracleDFlow.accept

    def wrong(block, g):
        a, bonus, c = orig(block, g)
        return a, int(g[min(a + 1, len(g) - 1)]), c[:-1] + [int(g[min(a + 1, len(g) - 1)])]
    OracleDFlow.accept = staticmethod(wrong)
    try:
        with pytest.raises(AssertionError):
            test_acceptance_brute_force()
    finally:
        OracleDFlow.accept = staticmethod(orig)


def test_relay_swap_mutation_caught(monkeypatch):
    from . import test_oracle_primitives as tp
    orig = om.OracleModel.relay

    def swapped(self, bonus, y_rej, h):   # beta and gamma exchanged
        w2 = self.raw["relay.w2"]
        d = self.dims.d
        self._conv.pop("relay.w2", None)
        self._conv.pop("relay.c2", None)
        self.raw = dict(self.raw)
        self.raw["relay.w2"] = np.concatenate([w2[d:], w2[:d]])
        c2 = self.raw["relay.c2"]
        self.raw["relay.c2"] = np.concatenate([c2[d:], c2[:d]])
        out = orig(self, bonus, y_rej, h)
        self.raw["relay.w2"], self.raw["relay.c2"] = w2, c2
        self._conv.pop("relay.w2", None)
        self._conv.pop("relay.c2", None)
        return out
    monkeypatch.setattr(om.OracleModel, "relay", swapped)
    wl = get_config("tiny-f32")
    m = OracleModel(wl.dims, make_weights(wl.dims, wl.seed_w), Mode("fp64"))
    with pytest.raises(AssertionError):
        tp.test_relay_mlp_vs_torch(m)


def test_ctx_input_norm_mutation_caught(monkeypatch):
    from .test_oracle_pins import test_drafter_with_context_matches_hf_cache
    orig = om.OracleModel.ctx_kv

    def normed(self, l, F, pos):
        return orig(self, l, self.rms_norm(F, self.w(f"draft.layers.{l}.attn_norm"), self.dims.rms_eps), pos)
    monkeypatch.setattr(om.OracleModel, "ctx_kv", normed)
    wl = get_config("tiny-f32")
    with pytest.raises(AssertionError):
        test_drafter_with_context_matches_hf_cache((wl, make_weights(wl.dims, wl.seed_w)))
