"""Inputs that make the one-pass Cauchy-Schwarz bracket ambiguous.

The library settles a row's Cauchy-Schwarz exponent from per-chunk records
reduced against each chunk's own maximum; when a chunk's maximum lies one
binade below the row's, its exact share of the sum of squares is only known
within an interval, and a row whose interval straddles a power of 4 is summed
again from the data.  These vectors are built so that this happens: their
exact sum U (the rule's definition, against the row maximum) sits at a power
of 4, and the chunks without the row maximum leave it unsettled.

Layout of a vector (parts: the real parts, and for complex vectors the
imaginary parts too):
* exact region: anchors 1.0 at every `stride`-th position (max exponent
  E = 1, each contributes (2^19)^2), fillers y 2^-19 (contributing y^2
  exactly) in the remaining parts of the region;
* one-binade region: real parts 0.5 + 2^-21 ("low": the interval's lower end
  is loose, its upper end exact; U = 4^j + 1) or 0.5 + 3 2^-21 ("high": the
  lower end exact, the upper loose; U = 4^j), i.e. a max exponent of 0.

Every chunk of a width dividing `stride` that meets the exact region holds an
anchor, and every chunk inside the one-binade region holds none, so the
construction does not depend on how the library chunks a row.  The values are
exact in fp32 as well.  No arithmetic of the method is done here beyond
choosing the fillers (the tests check the construction against the rule's
definition)."""
from __future__ import annotations

import math

import numpy as np

ANCHOR = 1.0                       # E = 1: y = 2^19 at the row maximum
ONE_BINADE = {"low": 0.5 + 2.0 ** -21, "high": 0.5 + 3 * 2.0 ** -21}
SHARE_AT_E = (2 ** 18 + 1) ** 2    # ceil(v 2^19)^2 for both one-binade values


def _squares(r: int, cap: int) -> list[int]:
    """r as a sum of squares of integers in [1, cap] (greedy)."""
    out = []
    while r > 0:
        y = min(math.isqrt(r), cap)
        out.append(y)
        r -= y * y
    return out


def straddle_vector(length: int, kind: str, complex_: bool = True, exact=(0, 128), binade=(128, 192),
                    stride: int = 16, dtype=None) -> np.ndarray:
    """A vector of `length` entries whose Cauchy-Schwarz sum sits at a power of
    4 (see the module docstring); entries outside both regions are zero."""
    assert exact[1] <= binade[0] and binade[1] <= length and exact[1] - exact[0] >= stride
    anchors = list(range(exact[0], exact[1], stride))
    n1 = binade[1] - binade[0]
    fixed = len(anchors) * (2 ** 19) ** 2 + n1 * SHARE_AT_E
    j = 1
    while 4 ** j + 1 - fixed < 0:
        j += 1
    # leave the fillers room below the cap of the slots
    slots = [(c, 1) for c in range(*exact)] if complex_ else []
    slots += [(c, 0) for c in range(*exact) if c not in anchors]
    target = 4 ** j + (1 if kind == "low" else 0)
    while True:
        rest = target - fixed
        full, r = divmod(rest, (2 ** 19) ** 2)
        ys = [2 ** 19] * full + _squares(r, 2 ** 19 - 1)
        if rest >= 0 and len(ys) <= len(slots):
            break
        j += 1
        target = 4 ** j + (1 if kind == "low" else 0)
    re = np.zeros(length)
    im = np.zeros(length)
    for c in anchors:
        re[c] = ANCHOR
    for c in range(*binade):
        re[c] = ONE_BINADE[kind]
    for (c, part), y in zip(slots, ys):
        (im if part else re)[c] = y * 2.0 ** -19
    if not complex_:
        return re.astype(dtype or np.float64)
    return (re + 1j * im).astype(dtype or np.complex128)


def exact_sum(parts, E: int) -> int:
    """U = sum over the nonzero parts of ceil(|v| 2^(20 - E))^2, in integers."""
    U = 0
    for v in parts:
        if v == 0:
            continue
        n, d = abs(float(v)).as_integer_ratio()
        if 20 - E >= 0:
            n <<= 20 - E
        else:
            d <<= E - 20
        y = -((-n) // d)
        U += y * y
    return U


def frexp_exp(parts) -> int:
    """The exponent e with max |v| < 2^e (frexp's), 0 for all zeros."""
    m = max((abs(float(v)) for v in parts), default=0.0)
    return math.frexp(m)[1] if m != 0 else 0
