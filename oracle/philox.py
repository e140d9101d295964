"""Counter-based candidate stream of the oracle.

The paper draws the mutated parameter and the increment at random (Eq. 1:
``w -> w + delta * rand`` with rand uniform on [-1, 1]) and, for discrete
weights, a jump to another discrete state (Eq. 12).  It does not fix a
generator.  Both the oracle and the HIP path therefore implement the same
published counter-based generator, Philox4x64-10 (Salmon, Moraes, Dror, Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3", SC'11), each from that
definition, so that draw (seed, step t, candidate k) is the same number on
both sides.

Decoding of one 4x64-bit block (w0, w1, w2, w3):

* which parameter:  flat = floor(w0 * P / 2^64) over all P parameters in
  canonical order; in "layer" mode the layer is floor(w1 * L / 2^64) and the
  position inside it floor(w0 * size_l / 2^64);
* continuous increment: r = (w2 >> 40) * 2^-23 - 1 in [-1, 1 - 2^-23] (exact in
  fp32), d = fl32(delta * r), new value fl32(w + d);
* ternary jump: bit b = w3 >> 63 picks the b-th of the two codes other than
  the current one, in ascending order (Eq. 12 with W_ij in {-1, 0, +1}).

The Metropolis rule (Eq. 7) needs one more uniform per candidate: word w0
of the block at counter (t, k, 1, 0), U = (w0 >> 11) * 2^-53 in [0, 1).

A channel mutation (Sec. 2.3) draws one unit per layer of the net, input to
output, and for the re-draw scheme one value per weight on that path.  Its
words are those of the blocks at counters (t, k, 2 + b, 0), b = 0, 1, ...,
taken in order (four per block): word m picks the path's unit of layer m,
units[m] = floor(word_m * n_m / 2^64), m = 0..L (units[L] a class); word
L + 1 + m re-draws the weight of layer m on the path as
fl32(a_m * r), r = unit_r(word), a_m = fl32(sqrt(8 / n_m)) the He amplitude
of its fan-in (the initialisation scale of Sec. 2.2).
"""
from __future__ import annotations

from dataclasses import dataclass

import math

import numpy as np

MASK64 = (1 << 64) - 1
# Philox4x64 multipliers and Weyl key increments (SC'11, Table/Sec. 5).
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B


def philox4x64(ctr, key, rounds: int = 10):
    """One Philox4x64-R block: 4 counter words, 2 key words -> 4 output words.

    Each round multiplies words 0 and 2 by the two multipliers; the new state
    is (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1, lo(M0 x0)); the key
    is bumped by the Weyl increments before every round but the first.
    """
    x0, x1, x2, x3 = (int(v) & MASK64 for v in ctr)
    k0, k1 = (int(v) & MASK64 for v in key)
    for r in range(rounds):
        if r:
            k0 = (k0 + PHILOX_W0) & MASK64
            k1 = (k1 + PHILOX_W1) & MASK64
        p0 = PHILOX_M0 * x0
        p1 = PHILOX_M1 * x2
        x0, x1, x2, x3 = ((p1 >> 64) ^ x1 ^ k0, p1 & MASK64,
                          (p0 >> 64) ^ x3 ^ k1, p0 & MASK64)
    return x0, x1, x2, x3


def mulhi64(a: int, n: int) -> int:
    """floor(a * n / 2^64): maps a uniform 64-bit word onto [0, n)."""
    return (int(a) * int(n)) >> 64


def unit_r(w2: int) -> np.float32:
    """rand of Eq. 1 on the 2^-23 grid of [-1, 1 - 2^-23]; every step is exact in fp32."""
    m = np.float32(int(w2) >> 40)
    return np.float32(m * np.float32(2.0 ** -23)) - np.float32(1.0)


def draw(seed: int, tag: int, t: int, k: int):
    """The block for candidate k of step t: key (seed, tag), counter (t, k, 0, 0)."""
    return philox4x64((t, k, 0, 0), (seed, tag))


def accept_uniform(seed: int, tag: int, t: int, k: int) -> float:
    """The acceptance uniform of candidate k of step t (Eq. 7): exact in fp64."""
    w0 = philox4x64((t, k, 1, 0), (seed, tag))[0]
    return float(w0 >> 11) * 2.0 ** -53


@dataclass(frozen=True)
class Candidate:
    """A single-parameter mutation: parameter `flat` = tensor `layer`, row j,
    column i; `d` the fp32 increment (continuous) or fl32(w' - w) (ternary,
    pruning); `code` the new ternary code (0 for continuous weights); `prune`
    a pruning move (w' = 0)."""
    flat: int
    layer: int
    j: int
    i: int
    d: np.float32
    code: int = 0
    prune: bool = False  # set the weight to zero (Sec. 2.2): w' = 0, d = -w


def ternary_next(code: int, bit: int) -> int:
    """The bit-th (0 or 1) of the two codes in {-1, 0, 1} other than `code`."""
    others = [c for c in (-1, 0, 1) if c != code]
    return others[bit]


def locate(flat: int, sizes):
    """Tensor index and offset of flat index `flat` in the canonical order."""
    off = 0
    for l, s in enumerate(sizes):
        if flat < off + s:
            return l, flat - off
        off += s
    raise IndexError(flat)


def decode(words, shapes, delta: float, mode: str = "weight",
           codes=None, scales=None) -> Candidate:
    """Turn one Philox block into a Candidate.

    shapes: list of parameter tensor shapes in canonical order (2-D as
    (rows, cols), 1-D as (n,)).  mode "weight": uniform over all parameters;
    "layer": uniform layer, then uniform inside it.  codes/scales: the
    committed ternary codes (int8 arrays) and per-layer fp32 scales, or None
    for continuous weights.
    """
    w0, w1, w2, w3 = words
    sizes = [int(np.prod(s)) for s in shapes]
    if mode == "weight":
        flat = mulhi64(w0, sum(sizes))
        layer, off = locate(flat, sizes)
    elif mode == "layer":
        layer = mulhi64(w1, len(sizes))
        off = mulhi64(w0, sizes[layer])
        flat = sum(sizes[:layer]) + off
    else:
        raise ValueError(mode)
    shp = shapes[layer]
    if len(shp) == 2:
        j, i = divmod(off, shp[1])
    else:
        j, i = off, 0
    if codes is None:
        d = np.float32(np.float32(delta) * unit_r(w2))
        return Candidate(flat, layer, j, i, d, 0)
    cur = int(codes[layer][j, i])
    new = ternary_next(cur, w3 >> 63)
    s = np.float32(scales[layer])
    d = np.float32(np.float32(new) * s - np.float32(cur) * s)
    return Candidate(flat, layer, j, i, d, new)


@dataclass(frozen=True)
class Channel:
    """A multi-parameter channel mutation (Sec. 2.3): one weight per layer on a
    path from an input to an output unit.  units[m] is the path's unit in
    layer m (units[0] an input, units[L] a class), so the path's weight of
    layer m is W_m[units[m + 1], units[m]]; w_new[m] is its proposed fp32 value."""
    units: tuple
    w_new: tuple


def channel_words(seed: int, tag: int, t: int, k: int, n: int):
    """The first n words of channel candidate k of step t: blocks at counters
    (t, k, 2 + b, 0) under key (seed, tag), four words each, in order."""
    out = []
    b = 0
    while len(out) < n:
        out.extend(philox4x64((t, k, 2 + b, 0), (seed, tag)))
        b += 1
    return out[:n]


def he_amplitude(fan_in: int) -> np.float32:
    """fl32(sqrt(8 / fan_in)): the amplitude of a re-drawn weight (Sec. 2.2's
    He initialisation scale, used by Sec. 2.3's re-draw scheme)."""
    return np.float32(math.sqrt(8.0 / fan_in))


def decode_channel(words, widths, scheme: str) -> Channel:
    """A channel of a net with widths (n_0 .. n_L) from 2L + 1 words: the path
    (one unit per layer), then, for scheme "redraw", the new weights
    fl32(a_m * r_m); for scheme "zero" every path weight becomes 0."""
    L = len(widths) - 1
    units = tuple(mulhi64(words[m], widths[m]) for m in range(L + 1))
    if scheme == "zero":
        w_new = tuple(np.float32(0.0) for _ in range(L))
    elif scheme == "redraw":
        w_new = tuple(np.float32(he_amplitude(widths[m]) * unit_r(words[L + 1 + m]))
                      for m in range(L))
    else:
        raise ValueError(scheme)
    return Channel(units, w_new)
