"""Shared set-up for parity tests: one workload, the HIP learner and the oracle on
the same seeded inputs (synthetic rows from `synth`, library seed, data seed)."""
from __future__ import annotations

import sys

import numpy as np

import synth
from oracle import Oracle

NET_KEYS = ("actor", "critic1", "critic2")


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def fill_rows(w, n_rows, data_seed, sinks, chunk=1 << 18):
    """Push rows 0..n_rows-1 of the synthetic stream into every sink (in order)."""
    for r0 in range(0, n_rows, chunk):
        rows = synth.workload_rows(w, r0, min(chunk, n_rows - r0), data_seed)
        for push in sinks:
            push(*rows)


def make_oracle(w, seed=1, data_seed=0, virtual_rows=None):
    hp = w.hparams()
    if virtual_rows is not None:
        o = Oracle(w.obs_dim, w.act_dim, w.hidden, w.batch, hp, seed,
                   row_source=lambda idx: synth.workload_rows_at(w, idx, data_seed))
        o.set_virtual_size(virtual_rows)
        return o
    return Oracle(w.obs_dim, w.act_dim, w.hidden, w.batch, hp, seed)


def make_gpu(w, seed=1, n_streams=2):
    from paper_2312_06126_amd import Spz
    return Spz(w.obs_dim, w.act_dim, w.hidden, w.batch, w.hparams(), seed, n_streams=n_streams)


def make_pair(w, n_rows, seed=1, data_seed=0, n_streams=2, virtual=False):
    g = make_gpu(w, seed, n_streams)
    if virtual:
        o = make_oracle(w, seed, data_seed, virtual_rows=n_rows)
        fill_rows(w, n_rows, data_seed, [g.buffer_push])
    else:
        o = make_oracle(w, seed, data_seed)
        fill_rows(w, n_rows, data_seed, [g.buffer_push, o.push])
    return g, o


def state_keys(algo):
    keys = ["actor", "critic1", "critic2", "tcritic1", "tcritic2", "log_alpha"]
    if algo == "td3":
        keys.append("tactor")
    keys += ["m_actor", "m_critic1", "m_critic2", "m_log_alpha", "v_actor", "v_critic1", "v_critic2",
             "v_log_alpha"]
    return keys


def teacher_force(o, g):
    """Round the oracle's state to float32, keep that in the oracle, and write it to the GPU."""
    for k in state_keys(o.algo):
        v = o.params(k).astype(np.float32)
        o.set_params(k, v.astype(np.float64))
        g.write_params(k, v)
    g.set_step(o.t)


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def oracle_grad_flat(o, key):
    gr = o.last_grads[key]
    return np.concatenate([np.concatenate([gw.ravel(), gb.ravel()]) for gw, gb in gr])


def per_tensor_rel(o, key, flat_gpu, flat_ref):
    """Largest per-tensor relative L2 difference over the W and b tensors of one net."""
    worst = 0.0
    off = 0
    for fi, fo in o.dims(key):
        for n in (fi * fo, fo):
            worst = max(worst, rel(flat_gpu[off:off + n], flat_ref[off:off + n]))
            off += n
    return worst


# ---------------------------------------------------------------- multi-step parameter parity
# An Adam update m_hat / (sqrt(v_hat) + eps) changes by about delta / sqrt(v_hat)
# when the gradient changes by delta. For an element whose whole gradient history
# is tiny next to its tensor's typical gradient (at step 1: |g| itself, since the
# first step is lr * sign(g)), the direction is set by rounding -- mostly by ReLU
# decisions on pre-activations within float32 rounding of zero, which float32
# and float64 can take differently. Such elements are identified from the
# oracle's gradients alone (sqrt(v_hat) < AMBIGUOUS * rms(g) of the tensor at a
# step), counted per element over the steps, excluded from the norm comparison
# and held to the bound their ambiguous steps allow: each such step can move the
# two runs apart by at most two Adam steps (one each way). Adam's moments m and v
# are continuous in g and are compared without exclusions.
AMBIGUOUS = 3e-3


def tensor_slices(o, key):
    off, out = 0, []
    for fi, fo in o.dims(key):
        for n in (fi * fo, fo):
            out.append(slice(off, off + n))
            off += n
    return out


def ambiguous_steps(o, key, grad_history, beta1=0.9, beta2=0.999):
    """Per element of `key`'s flat layout: the number of Adam steps at which it was
    sign-ambiguous (grad_history: flat oracle gradients per Adam step), and the bound
    on one Adam step's size |m_hat| / sqrt(v_hat) over those steps (at most about 1)."""
    n = o.param_count(key)
    cnt = np.zeros(n, np.int64)
    v = np.zeros(n)
    for t, gflat in enumerate(grad_history, start=1):
        v = beta2 * v + (1.0 - beta2) * gflat * gflat
        root_vhat = np.sqrt(v / (1.0 - beta2 ** t))
        for sl in tensor_slices(o, key):
            gt = gflat[sl]
            rms = np.sqrt(np.mean(gt * gt))
            cnt[sl] += ((root_vhat[sl] < AMBIGUOUS * rms) & (root_vhat[sl] > 0.0)).astype(np.int64)
    return cnt


def adam_step_bound(steps, beta1=0.9, beta2=0.999):
    """Largest |m_hat_t| / sqrt(v_hat_t) over t <= steps for any gradient sequence.

    m_hat_t = sum_k a_k g_k and v_hat_t = sum_k b_k g_k^2 with a_k = (1 - beta1)
    beta1^(t-k) / (1 - beta1^t) and b_k = (1 - beta2) beta2^(t-k) / (1 - beta2^t), so
    by Cauchy-Schwarz the ratio is at most sqrt(sum_k a_k^2 / b_k), with equality for
    g_k proportional to a_k / b_k (1 at t = 1, about 1.04 at t = 10)."""
    best = 0.0
    for t in range(1, steps + 1):
        j = np.arange(t)
        a = (1.0 - beta1) * beta1 ** j / (1.0 - beta1 ** t)
        b = (1.0 - beta2) * beta2 ** j / (1.0 - beta2 ** t)
        best = max(best, float(np.sqrt(np.sum(a * a / b))))
    return best


def check_param_parity(o, key, pg, pr, amb_steps, tol, lr, steps, p0=None, max_frac=0.05):
    """Per-tensor rel L2 <= tol over the elements never sign-ambiguous. Ambiguous ones
    must be rare (<= max_frac of a tensor) and stay within two Adam steps per ambiguous
    step: |p_gpu - p_ref| <= 2 lr n_ambiguous adam_step_bound(steps). With p0 (the common
    start), an element whose net motion has opposite signs in the two runs (both moves
    larger than lr / 10) must be one of the ambiguous elements."""
    worst = 0.0
    amb = amb_steps > 0
    step_bound = adam_step_bound(steps)
    for sl in tensor_slices(o, key):
        a, b, m = pg[sl].astype(np.float64), pr[sl], ~amb[sl]
        if m.any():
            worst = max(worst, rel(a[m], b[m]))
        if (~m).any():
            assert (~m).mean() <= max_frac, (key, (~m).mean())
            bound = 2.0 * step_bound * lr * amb_steps[sl][~m] + tol * np.abs(b[~m]) + 1e-12
            assert np.all(np.abs(a[~m] - b[~m]) <= bound), key
    if p0 is not None:
        dg, dr = pg.astype(np.float64) - p0, pr - p0
        big = (np.abs(dg) > 0.1 * lr) & (np.abs(dr) > 0.1 * lr)
        flipped = big & (np.sign(dg) != np.sign(dr))
        assert not np.any(flipped & ~amb), (key, int(np.sum(flipped & ~amb)))
    assert worst <= tol, (key, worst)
    return worst


# ---------------------------------------------------------------- the twin-minimum choice
# The SAC actor loss's min(Q1, Q2) picks a critic per row: where the two values are
# within accumulation-order error of each other, float32 and float64 can pick
# differently, and the row's whole gradient then moves to the other critic (one such
# row changes a first-layer weight gradient at batch 131072 by about 1/sqrt(batch) of
# its size). Comparisons of one step take the GPU's choice into the oracle and check it.

def gpu_min_choice(g):
    """The GPU's twin-minimum choice (critic 1 where qp1 <= qp2) of its last actor step."""
    qpi = g.debug_rows("qpi")
    return qpi[0] <= qpi[1]


def check_min_choice(o, take1, tol):
    """The oracle's own choice of its last step agrees with take1 wherever its two critic
    values differ by more than tol times their rms. Returns the number of rows taken over."""
    own = o.last_min_choice
    qp1, qp2 = o.last_qpi
    scale = float(np.sqrt(np.mean(qp1 * qp1)))
    diff = own != np.asarray(take1, bool)
    assert np.all(np.abs(qp1 - qp2)[diff] <= tol * scale), np.abs(qp1 - qp2)[diff].max() / scale
    return int(diff.sum())
