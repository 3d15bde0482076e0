"""The U-Net of Sec. 5 on the GPU against the oracle.

Every unit is checked teacher-forced: the oracle runs the unit on the GPU's
own input to that unit and the GPU's output must match it at the layer
tolerance.  In the fused network each unit's output is written already
pre-activated for its consumers (and the skip half of a decoder input
straight into the concatenation buffer), so every such destination is
checked against the oracle's convolution followed by that destination's
affine map and ReLU.
The small network is also compared end to end with the oracle's own
composition; at 256^3 x 8 scenes every output row of the level-0 units is
checked and 2048 sampled rows of each deeper unit, and all rule books of
levels 1-4 (level 0 is checked in the rule-book tests) bit-exactly.
"""
import numpy as np
import pytest
import torch

from oracle import sscn_oracle as O
from paper_1711_10275_amd import sscn, unet
from paper_1711_10275_amd import synthetic as S
from tests.gpu_common import assert_same_rulebook, dev, host, oracle_levels
from tests.parity import assert_close, assert_close_head

pytestmark = pytest.mark.gpu

TD = {"f32": torch.float32, "bf16": torch.bfloat16}


def _draw(dtype):
    return lambda name, k, cin, cout: S.layer_params(name, k, cin, cout, bf16=dtype == "bf16")


def _oracle_rb(levels, u):
    if u.kind == "ssc":
        return levels[u.level][2]
    if u.kind == "sc":
        return levels[u.level - 1][3]
    return O.transpose(levels[u.level][3])


def _check_geometry(geom, levels, first_level=0):
    for l in range(first_level, len(levels)):
        coords, size, ossc, osc = levels[l]
        np.testing.assert_array_equal(host(geom.coords[l]), coords)
        assert geom.sizes[l] == tuple(size)
        assert_same_rulebook(geom.ssc[l], ossc, f"level {l} ssc")
        if osc is not None:
            assert_same_rulebook(geom.down[l], osc, f"level {l} sc")
            assert_same_rulebook(geom.up[l], O.transpose(osc), f"level {l} dc")


def _teacher_forced(trace, levels, dtype, rows=None, seed=0, fused=True, full_levels=()):
    """fused: trace entries (unit, convolution input, [(dest, scale, shift)]);
    each destination must hold the oracle's convolution of that input with
    the destination's pre-activation (affine + ReLU, or none) applied.
    Unfused: (unit, unit input, output); the oracle pre-activates the input
    with the unit's own parameters and rounds it to the stored dtype."""
    rng = np.random.default_rng(seed)
    draw = _draw(dtype)
    rnd = O.round_bf16 if dtype == "bf16" else (lambda a: a)
    for u, inp, outs in trace:
        rb = _oracle_rb(levels, u)
        scale, shift, W = draw(u.name, u.k, u.cin, u.cout)
        if fused:
            a = host(inp)
        else:
            a = rnd(O.affine_relu(host(inp), scale, shift))
            outs = [(outs, None, None)]
        sample = rows is not None and u.level not in full_levels
        pick = rng.choice(rb.n_out, size=min(rows, rb.n_out), replace=False) if sample else None
        ref = O.forward(a, W, rb) if pick is None else O.forward_rows(a, W, rb, pick)
        for i, (dest, hs, hb) in enumerate(outs):
            got = host(dest)
            assert got.shape == (rb.n_out, u.cout), u.name
            g = got if pick is None else got[pick]
            if hs is None:
                assert_close(g, ref, dtype, f"{u.name} head {i}")
            else:
                assert_close_head(g, ref, host(hs), host(hb), dtype, f"{u.name} head {i}")


@pytest.mark.parametrize("fused", [True, False], ids=["fused", "unfused"])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_unet_small_scenes(dtype, fused):
    """64^3 x 2 scenes, five levels 64 -> 4, channels 32 .. 160."""
    levels = oracle_levels("scenes_small", 5)
    coords, size = levels[0][0], levels[0][1]
    geom = unet.Geometry(dev(coords), size)
    _check_geometry(geom, levels)
    X = S.features(coords.shape[0], 32, S.SEED_FEAT + 13, bf16=dtype == "bf16")
    params = unet.device_params(dtype=TD[dtype], draw=_draw(dtype))
    trace = []
    y = unet.forward(dev(X, TD[dtype]), geom, params, trace=trace, fused=fused)
    assert len(trace) == len(unet.units())
    _teacher_forced(trace, levels, dtype, fused=fused)
    ref = O.unet_forward(coords, size, X, _draw(dtype), unet.CHANNELS, round_to_bf16=dtype == "bf16")
    got = host(y)
    err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert err < (2e-2 if dtype == "bf16" else 1e-4), err


@pytest.mark.timeout(900)
def test_unet_scenes256():
    """256^3 x 8 scenes (about 2M level-0 sites), bf16, the benchmarked network:
    every output row of the level-0 units (enc0a, enc0b, up0, dec0a, dec0b),
    2048 sampled rows of the units of levels 1-4."""
    levels = oracle_levels("scenes256", 5)
    coords, size = levels[0][0], levels[0][1]
    geom = unet.Geometry(dev(coords), size)
    _check_geometry(geom, levels, first_level=1)
    X = S.features(coords.shape[0], 32, S.SEED_FEAT + 3, bf16=True)
    params = unet.device_params(dtype=torch.bfloat16, draw=_draw("bf16"))
    trace = []
    y = unet.forward(dev(X, torch.bfloat16), geom, params, trace=trace)
    assert tuple(y.shape) == (coords.shape[0], 32)
    assert torch.isfinite(y.float()).all()
    _teacher_forced(trace, levels, "bf16", rows=2048, seed=3, full_levels=(0,))
