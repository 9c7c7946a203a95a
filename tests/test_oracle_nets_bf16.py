"""Pins for the oracle's bfloat16 operand semantics (the bf16-GEMM workloads).

The paper leaves the numeric precision open (Section 4.1 names only the hardware);
the bf16 workloads are read as "every matrix-product operand rounded to bfloat16
(round to nearest, ties to even), float32 accumulation and float32 everything
else". The oracle applies that rounding at four points of oracle/nets.py:

  * forward:  the layer input (x, or the stored activation) and the weight;
  * backward: the back-propagated pre-activation gradient dZ (weight gradient,
    bias gradient and input gradient all take the rounded dZ) and the weight
    of the input-gradient product.

Two pins, neither of which shares code with the oracle's layer loop:

1. A two-layer micro net whose inputs sit on or next to bf16 rounding ties, with
   every forward and backward value worked out by hand (comments give the
   arithmetic). All values are exact binary fractions, so the comparison is exact.
2. torch autograd in float64 on small random nets: custom autograd functions
   round operands with torch's own bf16 converter in the forward pass and round
   the incoming gradient of each pre-activation in the backward pass; autograd,
   not a hand-written loop, does the back-propagation.

Mutation checks remove each rounding point from the real oracle code (a rounding
call identified by its source line is turned into the identity), and replace the
bias gradient by the sum of the unrounded dZ; each such mistake fails both pins.
"""
import linecache
import sys

import numpy as np
import pytest

import oracle.nets as nets
from oracle.bf16 import identity, round_bf16

# --------------------------------------------------------------------------- micro net
# Inputs of the hand-worked example. bf16 keeps 8 significant bits: spacing 2^-7 in
# [1, 2), 2^-6 in [2, 4); ties round to the even neighbour.
X = np.array([[1 + 2 ** -8 + 2 ** -12, 3.0]])        # rb -> [1 + 2^-7, 3] (just above a tie: up)
W0 = np.array([[1 + 2 ** -9, 0.5],                   # rb -> [1, 0.5] (below half a spacing: down)
               [-1.0, 1 + 3 * 2 ** -8]])             # rb -> [-1, 1 + 2^-6] (a tie: to even)
B0 = np.array([0.25, -5.0])
W1 = np.array([[1.5 + 2 ** -9, 7.0]])                # rb -> [1.5, 7]
B1 = np.array([0.125])
DZ1 = np.array([[1 + 2 ** -8 + 2 ** -11]])           # rb -> 1 + 2^-7

# Forward, by hand:
#   z0[0] = (1 + 2^-7) * 1 + 3 * 0.5 + 0.25        = 2.75 + 2^-7   -> ReLU keeps it
#   z0[1] = -(1 + 2^-7) + 3 (1 + 2^-6) - 5         = -3 + 5 * 2^-7 -> ReLU gives 0
#   rb(h) = [rb(2.75 + 2^-7), 0] = [2.75, 0]   (a tie between 2.75 and 2.75 + 2^-6: even)
#   z1    = 2.75 * 1.5 + 0 * 7 + 0.125             = 4.25
Z1 = 4.25
H_ROUNDED = [2.75, 0.0]
# Backward from dz1 = DZ1 (rb -> 1 + 2^-7):
#   dW1 = rb(dz1) * rb(h)                           = [2.75 (1 + 2^-7), 0]
#   db1 = rb(dz1)                                   = 1 + 2^-7
#   dh  = rb(dz1) * rb(W1)                          = [1.5 + 3 * 2^-8, 7 (1 + 2^-7)]
#   dz0 = dh * [h > 0]                              = [1.5 + 3 * 2^-8, 0]
#   rb(dz0) = [1.5 + 2^-6, 0]   (a tie between 1.5 + 2^-7 and 1.5 + 2^-6: even)
#   dW0 = rb(dz0)^T rb(x)                           = [[(1.5 + 2^-6)(1 + 2^-7), 3 (1.5 + 2^-6)], [0, 0]]
#   db0 = rb(dz0)                                   = [1.5 + 2^-6, 0]
#   dx  = rb(dz0) rb(W0)                            = [1.5 + 2^-6, 0.5 (1.5 + 2^-6)]
DW1 = [[2.75 * (1 + 2 ** -7), 0.0]]
DB1 = [1 + 2 ** -7]
DW0 = [[(1.5 + 2 ** -6) * (1 + 2 ** -7), 3 * (1.5 + 2 ** -6)], [0.0, 0.0]]
DB0 = [1.5 + 2 ** -6, 0.0]
DX = [[1.5 + 2 ** -6, 0.5 * (1.5 + 2 ** -6)]]


def micro_layers():
    return [[W0.copy(), B0.copy()], [W1.copy(), B1.copy()]]


def micro_pin(fwd=None, bwd=None, rnd=round_bf16):
    """Raise AssertionError unless forward/backward reproduce the hand-worked values."""
    fwd = fwd or nets.forward
    bwd = bwd or nets.backward
    layers = micro_layers()
    z, xs = fwd(layers, X, rnd)
    assert z[0, 0] == Z1, z
    assert list(xs[1][0]) == H_ROUNDED, xs[1]
    grads, dx = bwd(layers, xs, DZ1, rnd, want_wgrad=True, want_dx=True)
    assert np.array_equal(grads[1][0], DW1), grads[1][0]
    assert np.array_equal(grads[1][1], DB1), grads[1][1]
    assert np.array_equal(grads[0][0], DW0), grads[0][0]
    assert np.array_equal(grads[0][1], DB0), grads[0][1]
    assert np.array_equal(dx, DX), dx


def test_micro_net_hand_values():
    micro_pin()


def test_micro_net_fp32_mode_differs():
    """The example is sensitive to rounding at all: without it every value moves."""
    with pytest.raises(AssertionError):
        micro_pin(rnd=identity)


# --------------------------------------------------------------------------- torch autograd
torch = pytest.importorskip("torch")


def t_round(x):
    return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)


class RoundOperand(torch.autograd.Function):
    """Operand rounding: bf16 in the forward pass, gradient passed on unchanged."""

    @staticmethod
    def forward(ctx, x):
        return t_round(x)

    @staticmethod
    def backward(ctx, g):
        return g


class RoundGradient(torch.autograd.Function):
    """Identity in the forward pass; the incoming gradient is rounded to bf16."""

    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return t_round(g)


def torch_reference(layers, x, dz_last):
    """Forward z and (dW, db) per layer plus dx, by autograd with bf16 operand rounding."""
    ws = [torch.tensor(w, dtype=torch.float64, requires_grad=True) for w, _ in layers]
    bs = [torch.tensor(b, dtype=torch.float64, requires_grad=True) for _, b in layers]
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    h = xt
    z = None
    for l in range(len(layers)):
        # the gradient reaching the pre-activation (bias included) is rounded
        z = RoundGradient.apply(RoundOperand.apply(h) @ RoundOperand.apply(ws[l]).T + bs[l])
        if l + 1 < len(layers):
            h = torch.relu(z)
    z.backward(torch.tensor(dz_last, dtype=torch.float64))
    grads = [(w.grad.numpy(), b.grad.numpy()) for w, b in zip(ws, bs)]
    return z.detach().numpy(), grads, xt.grad.numpy()


def random_case(seed, dims, batch):
    r = np.random.default_rng(seed)
    layers = [[r.standard_normal((fo, fi)) * 0.7, r.standard_normal(fo) * 0.3] for fi, fo in dims]
    x = r.standard_normal((batch, dims[0][0]))
    dz = r.standard_normal((batch, dims[-1][1])) * 0.01
    return layers, x, dz


CASES = [(0, [(3, 4), (4, 1)], 6), (1, [(5, 7), (7, 6), (6, 2)], 9), (2, [(11, 8), (8, 8), (8, 34)], 5)]


def torch_pin(fwd=None, bwd=None):
    """Raise AssertionError unless the oracle agrees with the autograd reference."""
    fwd = fwd or nets.forward
    bwd = bwd or nets.backward
    for seed, dims, batch in CASES:
        layers, x, dz = random_case(seed, dims, batch)
        z_ref, g_ref, dx_ref = torch_reference(layers, x, dz)
        z, xs = fwd(layers, x, round_bf16)
        grads, dx = bwd(layers, xs, dz, round_bf16, want_wgrad=True, want_dx=True)
        np.testing.assert_allclose(z, z_ref, rtol=1e-12, atol=1e-15)
        for l, ((gw, gb), (rw, rbias)) in enumerate(zip(grads, g_ref)):
            np.testing.assert_allclose(gw, rw, rtol=1e-12, atol=1e-15, err_msg="dW layer %d" % l)
            np.testing.assert_allclose(gb, rbias, rtol=1e-12, atol=1e-15, err_msg="db layer %d" % l)
        np.testing.assert_allclose(dx, dx_ref, rtol=1e-12, atol=1e-15)


def test_matches_torch_autograd_with_bf16_operands():
    torch_pin()


# --------------------------------------------------------------------------- mutations
# Rounding calls of oracle/nets.py, identified by the text of their source line.
SITES = {"fwd_input": "xo = rnd(h)", "fwd_weight": "rnd(w).T", "bwd_dz": "dzo = rnd(dz)",
         "bwd_weight": "dzo @ rnd(w)"}


def selective_rnd(skip=None, hits=None):
    """round_bf16, except at the call site `skip`, where the value passes unrounded."""
    def rnd(x):
        fr = sys._getframe(1)
        line = linecache.getline(fr.f_code.co_filename, fr.f_lineno)
        site = [k for k, s in SITES.items() if s in line]
        assert len(site) == 1, line
        if hits is not None:
            hits.add(site[0])
        return identity(x) if site[0] == skip else round_bf16(x)
    return rnd


def with_rnd(rnd):
    """forward / backward of the oracle with `rnd` in place of the rounding they are given."""
    return (lambda layers, x, _r: nets.forward(layers, x, rnd),
            lambda layers, xs, dz, _r, **kw: nets.backward(layers, xs, dz, rnd, **kw))


def test_every_rounding_site_is_reached():
    hits = set()
    fwd, bwd = with_rnd(selective_rnd(hits=hits))
    micro_pin(fwd, bwd)
    torch_pin(fwd, bwd)
    assert hits == set(SITES), hits


@pytest.mark.parametrize("site", sorted(SITES))
def test_mutation_dropped_rounding_is_caught(site):
    fwd, bwd = with_rnd(selective_rnd(skip=site))
    with pytest.raises(AssertionError):
        micro_pin(fwd, bwd)
    with pytest.raises(AssertionError):
        torch_pin(fwd, bwd)


def test_mutation_bias_gradient_from_unrounded_dz_is_caught():
    def bad_backward(layers, xs, dz, rnd, want_wgrad=True, want_dx=False):
        grads, dx = [None] * len(layers), None
        for l in reversed(range(len(layers))):
            dzo = rnd(dz)
            grads[l] = (dzo.T @ xs[l], dz.sum(axis=0))          # planted: unrounded dZ
            d_in = dzo @ rnd(layers[l][0])
            if l > 0:
                dz = d_in * (xs[l] > 0.0)
            elif want_dx:
                dx = d_in
        return grads, dx
    with pytest.raises(AssertionError):
        micro_pin(bwd=bad_backward)
    with pytest.raises(AssertionError):
        torch_pin(bwd=bad_backward)
