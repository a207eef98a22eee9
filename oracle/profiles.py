"""Per-layer coefficients lambda^(l) from a depth profile (section 3.3, Eq. (6)).

TEST INFRASTRUCTURE ONLY (see the package docstring).

A profile gives a latent value a(l) for every layer l = 0..n_layers-1 and the coefficient is
lambda^(l) = sinh(a(l)); the same mapping is used for lambda1 and lambda2 in every family.
  * Global:   a(l) = a0                                   (one parameter)
  * Segments: a(l) = a[floor(n_seg * l / n_layers)]       (n_seg parameters; the paper's default is
              three: shallow, middle and deep thirds, i.e. layers 0-10 / 11-21 / 22-31 of 32)
  * Curve:    a(l) = c0 + c1 t + c2 t^2, t = l / (n_layers - 1)   (three parameters)
Reading for a single layer (n_layers = 1): t = 0.
"""
from __future__ import annotations

import math
from typing import List, Sequence

GLOBAL = "global"
SEGMENTS = "segments"
CURVE = "curve"


def latent(family: str, params: Sequence[float], layer: int, n_layers: int) -> float:
    """a(layer) of one family (section 3.3, Eq. (6) and the family definitions before it)."""
    if not 0 <= layer < n_layers:
        raise ValueError("layer out of range")
    if family == GLOBAL:
        if len(params) != 1:
            raise ValueError("Global takes one parameter")
        return float(params[0])
    if family == SEGMENTS:
        n_seg = len(params)
        if n_seg < 1 or n_seg > n_layers:
            raise ValueError("Segments needs 1..n_layers parameters")
        return float(params[(n_seg * layer) // n_layers])
    if family == CURVE:
        if len(params) != 3:
            raise ValueError("Curve takes three parameters")
        t = 0.0 if n_layers == 1 else layer / (n_layers - 1)
        return float(params[0]) + float(params[1]) * t + float(params[2]) * t * t
    raise ValueError(f"unknown profile family {family!r}")


def layer_lambdas(family: str, params: Sequence[float], n_layers: int) -> List[float]:
    """lambda^(l) = sinh(a(l)) for l = 0..n_layers-1 (Eq. (6)), in float64."""
    return [math.sinh(latent(family, params, layer, n_layers)) for layer in range(n_layers)]
