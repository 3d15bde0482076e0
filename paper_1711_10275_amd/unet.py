"""Submanifold sparse U-Net forward pass (Sec. 5) composed from the library's layers.

Every arithmetic step runs in libsscn.so: the rule books (SSC per level,
SC(2, 2) between levels, their transposes for the upsampling DC layers),
the pre-activation (inference-form batch normalisation + ReLU on active
sites), the convolutions and the skip concatenation.  This module only
orders the calls.

Network (five levels by default, channels 32 (l + 1) at level l):

* encoder, level l: two units BN-ReLU-SSC(3) with C_l -> C_l; the result is
  kept as the skip tensor of level l; below the last level a unit
  BN-ReLU-SC(2, 2) with C_l -> C_{l+1} moves to level l + 1;
* decoder, level l (from the second-lowest level up): a unit BN-ReLU-DC(2, 2)
  with C_{l+1} -> C_l over the transposed SC rule book of level l, the
  concatenation [skip_l, up_l] (2 C_l channels), then BN-ReLU-SSC(3) with
  2 C_l -> C_l and BN-ReLU-SSC(3) with C_l -> C_l.

Every unit's input is first mapped per channel by the unit's affine (scale,
shift) and ReLU, then convolved.  SC output sites of level l are the active
sites of level l + 1; SSC keeps each level's active set (Sec. 4.1), so the
decoder's output sites are the input sites.
"""
from __future__ import annotations

import dataclasses

import torch

from . import sscn

CHANNELS = (32, 64, 96, 128, 160)


@dataclasses.dataclass(frozen=True)
class Unit:
    name: str      # parameter name
    kind: str      # "ssc", "sc" or "dc"
    level: int     # level of the unit's output sites
    k: int         # filter offsets (27 for SSC(3), 8 for SC / DC(2, 2))
    cin: int
    cout: int


def units(channels=CHANNELS):
    """All units of the network in execution order."""
    L = len(channels)
    out = []
    for l in range(L):
        c = channels[l]
        out += [Unit(f"enc{l}a", "ssc", l, 27, c, c), Unit(f"enc{l}b", "ssc", l, 27, c, c)]
        if l < L - 1:
            out.append(Unit(f"down{l}", "sc", l + 1, 8, c, channels[l + 1]))
    for l in reversed(range(L - 1)):
        c = channels[l]
        out += [Unit(f"up{l}", "dc", l, 8, channels[l + 1], c),
                Unit(f"dec{l}a", "ssc", l, 27, 2 * c, c), Unit(f"dec{l}b", "ssc", l, 27, c, c)]
    return out


class Geometry:
    """Active sites and rule books of every level, built on the GPU.

    ssc[l]: SSC(3) rule book of level l; down[l]: SC(2, 2) rule book from
    level l to l + 1; up[l]: its transpose (DC from level l + 1 to l).
    """

    def __init__(self, coords, spatial_size, levels=len(CHANNELS)):
        self.coords, self.sizes, self.ssc, self.down, self.up = [coords], [tuple(spatial_size)], [], [], []
        c, size = coords, tuple(spatial_size)
        for l in range(levels):
            self.ssc.append(sscn.ssc_rulebook_build(c, size, 3))
            if l < levels - 1:
                d = sscn.sc_rulebook_build(c, size, 2, 2)
                self.down.append(d)
                self.up.append(d.transpose())
                c, size = d.out_coords(), d.out_size
                self.coords.append(c)
                self.sizes.append(size)

    @property
    def levels(self):
        return len(self.ssc)

    def rulebook(self, unit):
        if unit.kind == "ssc":
            return self.ssc[unit.level]
        if unit.kind == "sc":
            return self.down[unit.level - 1]
        return self.up[unit.level]

    def n_pairs(self, unit):
        return self.rulebook(unit).n_pairs


def forward(x, geom, params, channels=CHANNELS, trace=None, fused=True):
    """Run the network on level-0 features x (n_0 x channels[0]).

    params[name] = (scale, shift, W): device fp32 scale and shift over the
    unit's input channels, W [k][cin][cout] in x's dtype.

    fused (default): every unit writes its output already pre-activated for
    the unit(s) that consume it (the convolution's write-out applies their
    affine map and ReLU), and the skip and upsampled halves of each decoder
    concatenation are written straight into one buffer; only the network
    input is pre-activated separately.  If `trace` is a list, (unit, the
    convolution's input, [(destination, scale, shift), ...]) is appended
    for every unit.

    fused=False: one pre-activation, convolution and concatenation call
    after another; `trace` receives (unit, unit input before its
    pre-activation, unit output).
    """
    if len(channels) != geom.levels:
        raise ValueError("channel list and geometry disagree on the number of levels")
    if fused:
        return _forward_fused(x, geom, params, channels, trace)

    def run(u, inp):
        scale, shift, w = params[u.name]
        if tuple(w.shape) != (u.k, u.cin, u.cout):
            raise ValueError(f"{u.name}: weights {tuple(w.shape)}, expected {(u.k, u.cin, u.cout)}")
        y = sscn.sparse_conv_forward(sscn.affine_relu(inp, scale, shift), w, geom.rulebook(u))
        if trace is not None:
            trace.append((u, inp, y))
        return y

    skips = {}
    for u in units(channels):
        if u.name.startswith("enc"):
            x = run(u, x)
            if u.name.endswith("b"):
                skips[u.level] = x
        elif u.kind == "sc":
            x = run(u, x)
        elif u.kind == "dc":
            up = run(u, x)
            x = sscn.concat_cols(skips.pop(u.level), up)
        else:
            x = run(u, x)
    return x


def _forward_fused(x, geom, params, channels, trace):
    L = len(channels)
    by_name = {u.name: u for u in units(channels)}

    def new(level, c):
        return torch.empty((geom.coords[level].shape[0], c), dtype=x.dtype, device=x.device)

    def act(name, lo=None, hi=None):
        scale, shift, _ = params[name]
        return scale[lo:hi], shift[lo:hi]

    def conv(name, inp, heads):
        u = by_name[name]
        w = params[name][2]
        if tuple(w.shape) != (u.k, u.cin, u.cout):
            raise ValueError(f"{name}: weights {tuple(w.shape)}, expected {(u.k, u.cin, u.cout)}")
        sscn.sparse_conv_forward_heads(inp, w, geom.rulebook(u), heads)
        if trace is not None:
            trace.append((u, inp, heads))
        return [h[0] for h in heads]

    s0, b0 = act("enc0a")
    cur = sscn.affine_relu(x, s0, b0)
    cat = {}
    for l in range(L):
        c = channels[l]
        (y,) = conv(f"enc{l}a", cur, [(new(l, c), *act(f"enc{l}b"))])
        if l < L - 1:
            cat[l] = new(l, 2 * c)
            a_down, _ = conv(f"enc{l}b", y, [(new(l, c), *act(f"down{l}")),
                                             (cat[l][:, :c], *act(f"dec{l}a", 0, c))])
            (cur,) = conv(f"down{l}", a_down, [(new(l + 1, channels[l + 1]), *act(f"enc{l + 1}a"))])
        else:
            (cur,) = conv(f"enc{l}b", y, [(new(l, c), *act(f"up{l - 1}"))]) if L > 1 else \
                conv(f"enc{l}b", y, [(new(l, c), None, None)])
    if L == 1:
        return cur
    for l in reversed(range(L - 1)):
        c = channels[l]
        conv(f"up{l}", cur, [(cat[l][:, c:], *act(f"dec{l}a", c, 2 * c))])
        (z,) = conv(f"dec{l}a", cat.pop(l), [(new(l, c), *act(f"dec{l}b"))])
        if l > 0:
            (cur,) = conv(f"dec{l}b", z, [(new(l, c), *act(f"up{l - 1}"))])
        else:
            (cur,) = conv(f"dec{l}b", z, [(new(l, c), None, None)])
    return cur


def flops(geom, channels=CHANNELS):
    """Useful flops of one forward pass: 2 C_in C_out per rule-book pair (Table 2)."""
    return sum(2 * u.cin * u.cout * geom.n_pairs(u) for u in units(channels))


def device_params(channels=CHANNELS, dtype=torch.bfloat16, device="cuda:0", draw=None):
    """Parameters for every unit from `draw(name, k, cin, cout)` -> numpy (scale, shift, W)."""
    out = {}
    for u in units(channels):
        scale, shift, w = draw(u.name, u.k, u.cin, u.cout)
        out[u.name] = (torch.from_numpy(scale).to(device), torch.from_numpy(shift).to(device),
                       torch.from_numpy(w).to(dtype).to(device))
    return out
