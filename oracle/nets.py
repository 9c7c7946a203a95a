"""Multi-layer perceptrons of the actor and the twin critics (float64).

Layer l maps in_l -> out_l with z = x W^T + b; hidden layers apply ReLU, the last
layer is linear. Parameters of one network are kept as a list of [W, b] with
W of shape [out, in]; the flat layout (used to compare with the device) is, layer
by layer, W row-major followed by b.

Shapes (Section 3.2.2 names the networks; sizes come from the workload):
  actor  (SAC): obs -> hidden... -> 2*act (mean | log-std)
  actor  (TD3): obs -> hidden... -> act
  critic      : obs+act -> hidden... -> 1

For bf16 workloads every matrix-product operand (inputs, activations, weights and
back-propagated gradients) is passed through `rnd` (bfloat16 rounding); bias
adds, ReLU and everything outside the products stay in float64.
"""
from __future__ import annotations

from typing import Callable, List

import numpy as np

from .philox import init_uniform

NET_ACTOR, NET_CRITIC1, NET_CRITIC2 = 0, 1, 2


def layer_dims(kind: str, obs_dim: int, act_dim: int, hidden, algo: str):
    """[(in, out), ...] for 'actor' or 'critic'."""
    if kind == "actor":
        dims = [obs_dim] + list(hidden) + [2 * act_dim if algo == "sac" else act_dim]
    else:
        dims = [obs_dim + act_dim] + list(hidden) + [1]
    return list(zip(dims[:-1], dims[1:]))


def init_net(seed: int, net_id: int, dims) -> List[List[np.ndarray]]:
    """Fan-in uniform init; tensor id = net*16 + layer*2 + (0 for W, 1 for b)."""
    layers = []
    for l, (fi, fo) in enumerate(dims):
        w = init_uniform(seed, net_id * 16 + 2 * l, fo * fi, fi).reshape(fo, fi)
        b = init_uniform(seed, net_id * 16 + 2 * l + 1, fo, fi)
        layers.append([w.astype(np.float64), b.astype(np.float64)])
    return layers


def flatten(layers) -> np.ndarray:
    return np.concatenate([np.concatenate([w.ravel(), b.ravel()]) for w, b in layers])


def unflatten(flat: np.ndarray, dims) -> List[List[np.ndarray]]:
    out, o = [], 0
    for fi, fo in dims:
        w = np.array(flat[o:o + fo * fi], dtype=np.float64).reshape(fo, fi)
        o += fo * fi
        b = np.array(flat[o:o + fo], dtype=np.float64)
        o += fo
        out.append([w, b])
    assert o == flat.size
    return out


def count(dims) -> int:
    return sum(fi * fo + fo for fi, fo in dims)


def forward(layers, x, rnd: Callable):
    """Returns (z_last, xs) where xs[l] is the (rounded) operand fed to layer l."""
    xs = []
    h = x
    z = None
    for l, (w, b) in enumerate(layers):
        xo = rnd(h)
        xs.append(xo)
        z = xo @ rnd(w).T + b
        if l + 1 < len(layers):
            h = np.maximum(z, 0.0)
    return z, xs


def backward(layers, xs, dz, rnd: Callable, want_wgrad: bool = True, want_dx: bool = False):
    """Back-propagate dL/dz_last. Returns (grads, dx).

    grads[l] = (dW, db) with dW = rnd(dZ)^T X, db = sum_b rnd(dZ) (None when
    want_wgrad is False); dx = rnd(dZ_0) rnd(W_0) is dL/dx for the first layer's
    input when want_dx. ReLU'(0) = 0.
    """
    L = len(layers)
    grads = [None] * L
    dx = None
    for l in reversed(range(L)):
        w, _ = layers[l]
        dzo = rnd(dz)
        if want_wgrad:
            grads[l] = (dzo.T @ xs[l], dzo.sum(axis=0))
        if l > 0 or want_dx:
            d_in = dzo @ rnd(w)
            if l > 0:
                dz = d_in * (xs[l] > 0.0)
            else:
                dx = d_in
    return grads, dx
