"""Oracle primitives pinned against library routines (CPU only)."""
import numpy as np
import pytest
import torch

from oracle import Mode, OracleModel
from oracle.numerics import round_bf16
from workload import get_config
from workload.configs import ModelDims, replace
from workload.synth import make_weights


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-8, 8, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -3.0e38, 1e-40], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(round_bf16(x), ref)


@pytest.fixture(scope="module")
def tiny64():
    wl = get_config("tiny-f32")
    return OracleModel(wl.dims, make_weights(wl.dims, wl.seed_w), Mode("fp64"))


def test_layer_norm_vs_torch(tiny64):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 256)) * 3 + 0.5
    g, b = rng.standard_normal(256), rng.standard_normal(256)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (256,), torch.from_numpy(g), torch.from_numpy(b),
                                         eps=1e-5).numpy()
    np.testing.assert_allclose(tiny64.layer_norm(x, g, b, 1e-5), ref, rtol=1e-12, atol=1e-12)


def test_rms_norm_vs_torch(tiny64):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 256)) * 2
    g = rng.standard_normal(256)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (256,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(tiny64.rms_norm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("visible_all", [True, False])
def test_attention_vs_sdpa(tiny64, visible_all):
    rng = np.random.default_rng(3)
    n, m, Hq, Hkv, Dh = 6, 11, 4, 2, 64
    q = rng.standard_normal((n, Hq, Dh))
    k = rng.standard_normal((m, Hkv, Dh))
    v = rng.standard_normal((m, Hkv, Dh))
    if visible_all:
        vis = np.ones((n, m), bool)
    else:   # block-causal: row j sees keys 0..m-n+j
        vis = np.arange(m)[None, :] <= (m - n + np.arange(n))[:, None]
    out = tiny64.attention(q, k, v, vis)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(vis),
                                                           enable_gqa=True)
    ref = ref[0].permute(1, 0, 2).reshape(n, Hq * Dh).numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)


def test_rope_properties(tiny64):
    """Position 0 is the identity; each (i, i+Dh/2) pair keeps its norm; the
    score of rotated q,k depends only on the position difference."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 2, 64))
    np.testing.assert_allclose(tiny64.rope(x, np.zeros(3)), x, rtol=0, atol=0)
    y = tiny64.rope(x, np.array([5, 77, 1000]))
    np.testing.assert_allclose(y[..., :32] ** 2 + y[..., 32:] ** 2, x[..., :32] ** 2 + x[..., 32:] ** 2, rtol=1e-12)
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    s1 = np.sum(tiny64.rope(q, np.array([10])) * tiny64.rope(k, np.array([3])))
    s2 = np.sum(tiny64.rope(q, np.array([107])) * tiny64.rope(k, np.array([100])))
    assert abs(s1 - s2) < 1e-10
    # frequency of the first pair is 1 rad/position, last pair theta^(-(Dh-2)/Dh)
    assert tiny64.inv_freq[0] == 1.0
    np.testing.assert_allclose(tiny64.inv_freq[-1], 1e6 ** (-62 / 64), rtol=1e-14)


def test_relay_mlp_vs_torch(tiny64):
    """MLP_phi = Linear(3d->d_h) -> SiLU -> Linear(d_h->2d), checked through the
    relay output with the LayerNorm replaced by torch's."""
    m = tiny64
    d = m.dims.d
    rng = np.random.default_rng(5)
    h = rng.standard_normal((3, d))
    bonus, y_rej = 17, 4000
    x = m.relay(bonus, y_rej, h)
    E = torch.from_numpy(m.w("embed"))
    u = torch.cat([E[bonus].expand(3, d), E[y_rej].expand(3, d), torch.from_numpy(h)], dim=1)
    l1 = torch.nn.Linear(3 * d, m.dims.d_h).double()
    l2 = torch.nn.Linear(m.dims.d_h, 2 * d).double()
    with torch.no_grad():
        l1.weight.copy_(torch.from_numpy(m.w("relay.w1")))
        l1.bias.copy_(torch.from_numpy(m.w("relay.c1")))
        l2.weight.copy_(torch.from_numpy(m.w("relay.w2")))
        l2.bias.copy_(torch.from_numpy(m.w("relay.c2")))
        bg = l2(torch.nn.functional.silu(l1(u)))
        ln = torch.nn.functional.layer_norm(torch.from_numpy(h), (d,), torch.from_numpy(m.w("relay.ln_g")),
                                            torch.from_numpy(m.w("relay.ln_b")), eps=1e-5)
        ref = torch.from_numpy(m.w("draft.e_mask")) + bg[:, :d] * ln + bg[:, d:]
    np.testing.assert_allclose(x, ref.numpy(), rtol=1e-11, atol=1e-12)


def test_relay_special_cases(tiny_weights):
    """Zero second layer and zero bias -> beta = gamma = 0 -> x = E_mask
    exactly; W2 = 0 with c2 = [1; 0] -> x = E_mask + LN(h)."""
    wl, w = tiny_weights
    d = wl.dims.d
    w2 = dict(w)
    w2["relay.w2"] = np.zeros_like(w["relay.w2"])
    w2["relay.c2"] = np.zeros_like(w["relay.c2"])
    for mode in ("fp64", "fp32"):
        m = OracleModel(wl.dims, w2, Mode(mode))
        h = np.random.default_rng(6).standard_normal((4, d)).astype(m.mode.dt)
        x = m.relay(3, 9, h)
        np.testing.assert_array_equal(x, np.repeat(m.w("draft.e_mask")[None], 4, 0))
    c2 = np.concatenate([np.ones(d, np.float32), np.zeros(d, np.float32)])
    w2["relay.c2"] = c2
    m = OracleModel(wl.dims, w2, Mode("fp64"))
    h = np.random.default_rng(7).standard_normal((4, d))
    ln = torch.nn.functional.layer_norm(torch.from_numpy(h), (d,), torch.from_numpy(m.w("relay.ln_g")),
                                        torch.from_numpy(m.w("relay.ln_b")), eps=1e-5).numpy()
    np.testing.assert_allclose(m.relay(3, 9, h), m.w("draft.e_mask")[None] + ln, rtol=1e-12, atol=1e-13)
