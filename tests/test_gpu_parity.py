"""GPU parity: the HIP learner (through the C ABI) against the CPU oracle.

Bars (spec tolerances):
  * replay indices and the step-0 parameters: bit-exact;
  * fp32 GEMM workloads: losses within rel 1e-4 per step; parameters within
    per-tensor rel 1e-4 (||p_gpu - p_ref|| / ||p_ref|| for every W and b) after
    10 steps, over the elements whose Adam direction the arithmetic determines
    (sign-ambiguous elements, found from the oracle's gradients alone, are
    counted, must be under 5% of a tensor, and must stay within Adam's step
    bound); gradients of a teacher-forced step within per-tensor rel 1e-4;
  * bf16 GEMM workloads: losses within rel 2e-2.
Loss values near zero use an absolute floor of 1e-6 (L_alpha is exactly 0 at
log(alpha) = 0, the first step of every learned-temperature workload).
"""
import numpy as np
import pytest

import synth
from oracle import philox
from synth.workloads import Workload

from .helpers import (NET_KEYS, ambiguous_steps, check_min_choice, check_param_parity, gpu_min_choice, log, make_gpu, make_oracle, make_pair,
                      oracle_grad_flat, per_tensor_rel, state_keys, teacher_force)

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS
# Ragged shapes: batch not a multiple of 256, widths not multiples of 32.
RAGGED = Workload("ragged_sac", "sac", 13, 5, (100, 70), 1000, 5000, "fp32", 10, target_entropy=-5.0)
RAGGED_TD3 = Workload("ragged_td3", "td3", 13, 5, (100, 70), 1000, 5000, "fp32", 10, learn_alpha=False,
                      alpha_init=0.0)
RAGGED_BF16 = RAGGED.replace(name="ragged_sac_bf16", prec="bf16", zero_mod=10, obs_dim=45)
DEEP = Workload("deep_sac", "sac", 29, 3, (96, 64, 160), 600, 3000, "fp32", 10, target_entropy=-3.0)
# bf16 shapes on the large-tile kernel with every fused epilogue (ReLU masks as bits,
# critic output layer folded into the last hidden product): 256- and 128-wide
# column tiles, a ragged batch (500 of 512 rows) and a three-layer variant.
FUSED_BF16 = RAGGED_BF16.replace(name="fused_sac_bf16", hidden=(256, 128), batch=500)
FUSED_BF16_DEEP = RAGGED_BF16.replace(name="fused_sac_bf16_deep", hidden=(128, 256, 384), batch=768)
FUSED_TD3_BF16 = RAGGED_TD3.replace(name="fused_td3_bf16", prec="bf16", zero_mod=10, hidden=(256, 256), batch=256)

# Sequential update ordering (critics step first, the actor sees the updated critics).
SEQ_SAC = RAGGED.replace(name="ragged_sac_seq", ordering="sequential")
SEQ_TD3 = RAGGED_TD3.replace(name="ragged_td3_seq", ordering="sequential")
SEQ_BF16 = FUSED_BF16.replace(name="fused_sac_bf16_seq", ordering="sequential")

FP32_TOL = 1e-4
BF16_LOSS_TOL = 2e-2


def check_losses(rec_gpu, rec_ref, tol, what=""):
    cols = [0, 1, 2, 3, 4, 5]
    for c in cols:
        a, b = rec_gpu[:, c].astype(np.float64), rec_ref[:, c]
        err = np.abs(a - b) / np.maximum(np.abs(b), 1e-6 / tol)
        assert np.all(err <= tol), "%s loss column %d: gpu %s ref %s" % (what, c, a, b)
    assert np.array_equal(rec_gpu[:, 6], rec_ref[:, 6])
    assert np.array_equal(rec_gpu[:, 7], rec_ref[:, 7])


# ---------------------------------------------------------------------------- bit-exact pieces
@pytest.mark.parametrize("w", [W["sac_small"], RAGGED_TD3, RAGGED_BF16, W["sac_large_bf16"].replace(batch=256,
                                                                                              capacity=1000)],
                         ids=lambda w: w.name)
def test_init_params_bit_exact(w):
    log("init parity %s" % w.name)
    g = make_gpu(w, seed=123)
    o = make_oracle(w, seed=123)
    for k in ["actor", "critic1", "critic2", "tcritic1", "tcritic2", "log_alpha"] + (["tactor"] if w.algo == "td3" else []):
        assert np.array_equal(g.read_params(k), o.params(k).astype(np.float32)), k
    g.close()


def test_indices_bit_exact_small():
    w = W["sac_small"]
    log("indices sac_small")
    g = make_gpu(w, seed=7)
    synth_rows = synth.workload_rows(w, 0, 777, 0)
    g.buffer_push(*synth_rows)
    for t in range(1, 6):
        g.update(1)
        assert np.array_equal(g.debug_indices(), philox.indices(7, t, w.batch, 777).astype(np.int32))
    g.close()


def test_indices_bit_exact_full_size_large():
    """Full batch (131072) over a full 4M-row ring; indices depend only on the ring size."""
    w = W["sac_large_bf16"]
    log("indices sac_large_bf16 full size")
    g = make_gpu(w, seed=1)
    chunk = 1 << 18
    zeros = (np.zeros((chunk, w.obs_dim), np.float32), np.zeros((chunk, w.act_dim), np.float32),
             np.zeros(chunk, np.float32), np.zeros(chunk, np.float32), np.zeros((chunk, w.obs_dim), np.float32))
    n = 0
    while n < w.capacity:
        m = min(chunk, w.capacity - n)
        g.buffer_push(*[z[:m] for z in zeros])
        n += m
    assert g.buffer_size() == w.capacity
    g.update(1)
    idx = g.debug_indices()
    assert np.array_equal(idx, philox.indices(1, 1, w.batch, w.capacity).astype(np.int32))
    rec = g.read_losses(1, 1)[0]
    assert rec[6] == 0.0 and np.all(np.isfinite(rec))
    g.close()


def _rms_err(gpu, ref):
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(np.asarray(gpu, np.float64) - ref)) / max(np.sqrt(np.mean(ref * ref)), 1e-30))


# Per-row values differ by bf16 rounding flips between fp32 and float64 accumulation:
# a flipped operand moves a 1024-term dot product by about 1e-4 of its size. Forward
# values see about one flip per net (observed max error / rms 3e-7 to 4e-5); the action
# gradient goes through three rounded layers of dz, one flip per 1024 elements each, and
# its max runs over 17 components per row (observed 1.8e-3). A dropped term, a wrong
# sign or a wrong critic for a row gives errors of order 1.
ROW_TOL_BF16 = 1e-3
ROW_TOL_BF16_GRAD = 1e-2
# A ReLU mask is a floating-point decision: a hidden unit whose pre-activation lies within
# accumulation error of zero may be active on one side and not on the other. Such a flip
# leaves the forward values alone (the unit's value is next to zero either way) but moves
# the action gradient by one unit's share of a 1024-term sum (a few percent). Candidates
# are units with |z| <= MASK_AMBIG * sum_i |x_i w_i| + |b| (fp32 accumulation of 1024
# terms plus one bf16 flip of an upstream operand stay far below this bound).
MASK_AMBIG = 2.0 ** -12
MASK_FLIP_ROWS = 5   # at most this many of the 96 sampled rows may need a flipped mask


def _critic_dx(o, key, x_row, dq_row, flips=()):
    """dL/dx of one row of critic `key` (oracle arithmetic) with the ReLU masks of the
    listed (operand layer, unit) pairs inverted."""
    from oracle.nets import backward, forward
    _, xs = forward(o.net[key], x_row[None, :], o.rnd)
    xs = [v.copy() for v in xs]
    for l, u in flips:
        xs[l][0, u] = 0.0 if xs[l][0, u] > 0.0 else 1e-30
    _, dx = backward(o.net[key], xs, np.array([[dq_row]]), o.rnd, want_wgrad=False, want_dx=True)
    return dx[0]


def _mask_candidates(o, key, x_row):
    """(operand layer, unit) pairs of critic `key` on one row whose ReLU decision is
    within MASK_AMBIG of zero, nearest first."""
    from oracle.nets import forward
    _, xs = forward(o.net[key], x_row[None, :], o.rnd)
    cand = []
    for l, (w, b) in enumerate(o.net[key][:-1]):
        wr = o.rnd(w)
        z = xs[l][0] @ wr.T + b
        scale = np.abs(xs[l][0]) @ np.abs(wr).T + np.abs(b)
        m = np.abs(z) / np.maximum(scale, 1e-300)
        cand += [(float(m[u]), l + 1, int(u)) for u in np.nonzero(m <= MASK_AMBIG)[0]]
    return [(l, u) for _, l, u in sorted(cand)]


def _explained_by_mask_flip(o, x_row, dq_row, got_row, ref_row, rms, tol):
    """Whether the GPU's action gradient of one row equals the oracle's with the ReLU
    decisions of one or two near-zero units inverted (within tol of the gradient rms)."""
    import itertools
    A = got_row.size
    keys = [k for k, v in dq_row.items() if v != 0.0]
    base = {k: _critic_dx(o, k, x_row, dq_row[k])[-A:] for k in keys}
    for k in keys:
        cand = _mask_candidates(o, k, x_row)[:12]
        others = sum(base[j] for j in keys if j != k)
        for n in (1, 2):
            for flips in itertools.combinations(cand, n):
                alt = others + _critic_dx(o, k, x_row, dq_row[k], flips)[-A:]
                if np.max(np.abs(got_row - alt)) <= tol * rms:
                    log("    row explained by the mask of %s unit(s) %s of %s" % (n, flips, k))
                    return True
    return False


@pytest.mark.parametrize("name", ["sac_large_bf16", "td3_ant"])
def test_full_size_sampled_rows(name):
    """A workload at its full batch and widths, in bench's launch configuration (one
    stream; for SAC the actor row split): after 3 steps the oracle takes the GPU's
    state, and step 4's per-row values (TD target, q1, q2, the critics on (s, a~),
    log pi, the actor loss's gradient to the action) are checked on 96 sampled rows,
    each computed by the oracle on those rows alone. The ring holds 200000 rows (the
    ring size only changes which rows are drawn)."""
    from oracle.nets import forward
    from oracle.update import tanh_gaussian
    from .helpers import fill_rows, state_keys
    rows = 200_000
    w = W[name].replace(capacity=rows)
    sac = w.algo == "sac"
    tol = ROW_TOL_BF16 if w.prec == "bf16" else FP32_TOL
    tol_grad = ROW_TOL_BF16_GRAD if w.prec == "bf16" else FP32_TOL
    log("sampled rows %s full size" % name)
    g = make_gpu(w, n_streams=1)
    fill_rows(w, rows, 0, [g.buffer_push])
    g.update(3)
    o = make_oracle(w, virtual_rows=rows)
    for k in state_keys(o.algo):
        o.set_params(k, g.read_params(k).astype(np.float64))
    g.update(1)
    t, B, A = 4, w.batch, w.act_dim
    idx = philox.indices(1, t, B, rows)
    assert np.array_equal(g.debug_indices(), idx.astype(np.int32))
    got = {k: g.debug_rows(k) for k in ("td_target", "q", "qpi", "daction") + (("logpi",) if sac else ())}
    g.close()

    R = np.sort(np.random.default_rng(5).choice(B, 96, replace=False))
    s, a, r, d, s2 = o._gather(idx[R])
    eps_tgt = philox.normals(1, t, philox.PURPOSE_NOISE_TGT, B * A).reshape(B, A)[R]
    x = np.concatenate([s, a], axis=1)
    q = [forward(o.net[k], x, o.rnd)[0][:, 0] for k in ("critic1", "critic2")]
    z, _ = forward(o.net["actor"], s, o.rnd)
    ref = {}
    if sac:
        alpha = float(np.exp(o.log_alpha[0]))
        y, _ = o.sac_target(s2, r, d, eps_tgt, alpha)
        eps_pol = philox.normals(1, t, philox.PURPOSE_NOISE_POL, B * A).reshape(B, A)[R]
        pol = tanh_gaussian(z, eps_pol, A, w.log_std_min, w.log_std_max)
        a_pi = pol["a"]
        ref["logpi"] = (got["logpi"][R], pol["logp"])
    else:
        y, _ = o.td3_target(s2, r, d, eps_tgt)
        a_pi = np.tanh(z)
    xa = np.concatenate([s, a_pi], axis=1)
    qp = [forward(o.net[k], xa, o.rnd)[0][:, 0] for k in ("critic1", "critic2")]
    if sac:
        # The minimum critic is a floating-point decision: take the GPU's, and check that
        # the oracle's own agrees wherever the two values are not within the bar.
        take1 = got["qpi"][0][R] <= got["qpi"][1][R]
        close = np.abs(qp[0] - qp[1]) <= 2 * tol * np.sqrt(np.mean(qp[0] ** 2))
        assert np.all((take1 == (qp[0] <= qp[1])) | close)
        assert 0 < take1.sum() < len(R)
        dq = {"critic1": np.where(take1, -1.0 / B, 0.0), "critic2": np.where(take1, 0.0, -1.0 / B)}
        ref["qpi2"] = (got["qpi"][1][R], qp[1])
    else:
        dq = {"critic1": np.full(len(R), -1.0 / B)}
    da = o._critic_action_grad(s, a_pi, dq)
    ref.update(td_target=(got["td_target"][R], y), q1=(got["q"][0][R], q[0]), q2=(got["q"][1][R], q[1]),
               qpi1=(got["qpi"][0][R], qp[0]), daction=(got["daction"][R], da))
    if w.prec == "bf16":
        # Rows whose action gradient is off by more than the bar must be explained by
        # inverting the ReLU decision of one or two near-zero hidden units of a critic.
        gd, rd = ref["daction"]
        rms = float(np.sqrt(np.mean(rd * rd)))
        bad = np.nonzero(np.max(np.abs(gd - rd), axis=1) > tol_grad * rms)[0]
        log("  rows of the action gradient above the bar: %d" % len(bad))
        assert len(bad) <= MASK_FLIP_ROWS, len(bad)
        for i in bad:
            dq_row = {k: float(v[i]) for k, v in dq.items()}
            assert _explained_by_mask_flip(o, xa[i], dq_row, gd[i], rd[i], rms, tol_grad), (
                int(R[i]), float(np.max(np.abs(gd[i] - rd[i])) / rms))
        keep = np.setdiff1d(np.arange(len(R)), bad)
        ref["daction"] = (gd[keep], rd[keep])
    errs = {k: _rms_err(gv, rv) for k, (gv, rv) in ref.items()}
    log("  per-row max error / rms: " + " ".join("%s %.2e" % kv for kv in errs.items()))
    for k, e in errs.items():
        assert e <= (tol_grad if k == "daction" else tol), (k, e)


# ---------------------------------------------------------------------------- teacher-forced steps
def teacher_forced(w, n_rows, steps_before=0, virtual=False, tol_grad=FP32_TOL, tol_loss=FP32_TOL,
                   n_steps=1):
    g, o = make_pair(w, n_rows, virtual=virtual)
    if steps_before:
        o.update(steps_before)
    teacher_force(o, g)
    for _ in range(n_steps):
        if _:
            teacher_force(o, g)
        g.update(1)
        actor_step = w.algo == "sac" or (o.t + 1) % w.policy_delay == 0
        if w.algo == "sac":
            o.forced_min_choice = take1 = gpu_min_choice(g)
        o.update(1)
        if w.algo == "sac":
            check_min_choice(o, take1, tol_grad)
        assert np.array_equal(g.debug_indices(), o.last_idx.astype(np.int32))
        for k in NET_KEYS:
            if o.last_grads[k] is None:
                continue
            gg = g.read_params("g_" + k)
            gr = oracle_grad_flat(o, k)
            e = per_tensor_rel(o, k, gg, gr)
            # Adam's moments after the step from the same start: continuous in g
            em = max(per_tensor_rel(o, k, g.read_params(mv + k), o.params(mv + k)) for mv in ("m_", "v_"))
            log("  %s step %d grad %s rel %.2e, moments %.2e" % (w.name, o.t, k, e, em))
            assert e <= tol_grad, (k, e)
            assert em <= tol_grad, (k, em)
        assert actor_step == (o.last_grads["actor"] is not None)
        check_losses(g.read_losses(o.t, 1), o.losses()[-1:], tol_loss, w.name)
    g.close()


@pytest.mark.parametrize("w,rows,before", [(W["sac_small"], 10_000, 0), (RAGGED, 5000, 3), (DEEP, 3000, 2)],
                         ids=["sac_small", "ragged_sac", "deep_sac"])
def test_teacher_forced_sac_fp32(w, rows, before):
    log("teacher-forced %s" % w.name)
    teacher_forced(w, rows, steps_before=before)


# 2A = 80 actor outputs: wider than the head product's fused epilogue takes (at most 64
# columns), so these run the SAC head as its own kernel.
WIDE_ACT = RAGGED.replace(name="wide_action_sac", act_dim=40, target_entropy=-40.0)
WIDE_ACT_BF16 = RAGGED_BF16.replace(name="wide_action_sac_bf16", act_dim=40, target_entropy=-40.0)


@pytest.mark.parametrize("w,fused", [(RAGGED, True), (RAGGED_BF16, True), (WIDE_ACT, False), (WIDE_ACT_BF16, False)],
                         ids=["ragged_fp32", "ragged_bf16", "wide_fp32", "wide_bf16"])
def test_sac_head_paths(w, fused):
    """The SAC head runs inside the actor's output product where 2A fits its tile and as its
    own kernel otherwise (checked from the kernel records); both paths give the oracle's
    gradients, moments and losses on a teacher-forced step."""
    log("SAC head path %s" % w.name)
    g = make_gpu(w)
    g.buffer_push(*synth.workload_rows(w, 0, 5000, 0))
    g.profile_enable(True, 100)
    g.update(1)
    names = {s["name"] for s in g.profile_read()}
    g.close()
    assert ("sac_head" not in names) == fused, names
    bf16 = w.prec == "bf16"
    teacher_forced(w, 5000, steps_before=1, tol_grad=1e-3 if bf16 else FP32_TOL,
                   tol_loss=BF16_LOSS_TOL if bf16 else FP32_TOL)


def test_teacher_forced_td3_fp32():
    log("teacher-forced ragged_td3")
    teacher_forced(RAGGED_TD3, 5000, steps_before=1, n_steps=2)


def test_teacher_forced_bf16():
    log("teacher-forced ragged_sac_bf16")
    teacher_forced(RAGGED_BF16, 5000, steps_before=1, tol_grad=1e-3, tol_loss=BF16_LOSS_TOL)


@pytest.mark.parametrize("w,n_steps", [(FUSED_BF16, 1), (FUSED_BF16_DEEP, 1), (FUSED_TD3_BF16, 2)],
                         ids=lambda x: getattr(x, "name", str(x)))
def test_teacher_forced_bf16_fused(w, n_steps):
    log("teacher-forced %s" % w.name)
    teacher_forced(w, 5000, steps_before=1, tol_grad=1e-3, tol_loss=BF16_LOSS_TOL, n_steps=n_steps)


@pytest.mark.parametrize("w,n_steps,tol", [(SEQ_SAC, 2, FP32_TOL), (SEQ_TD3, 2, FP32_TOL), (SEQ_BF16, 1, 1e-3)],
                         ids=["sac_fp32", "td3_fp32", "sac_bf16_fused"])
def test_teacher_forced_sequential(w, n_steps, tol):
    log("teacher-forced %s" % w.name)
    teacher_forced(w, 5000, steps_before=1, tol_grad=tol, tol_loss=FP32_TOL if tol == FP32_TOL else BF16_LOSS_TOL,
                   n_steps=n_steps)


def test_teacher_forced_log_std_clamp_active():
    """Push the log-std head beyond both clamp bounds through write_params."""
    w = RAGGED
    log("clamp ragged_sac")
    g, o = make_pair(w, 5000)
    flat = o.params("actor")
    dims = o.dims("actor")
    off = sum(fi * fo + fo for fi, fo in dims[:-1])
    fi, fo = dims[-1]
    b_off = off + fi * fo
    flat[b_off + w.act_dim: b_off + w.act_dim + 2] = [2.5, -21.0]   # two log-std heads out of range
    flat[off:off + fi * fo] *= 0.1
    o.set_params("actor", flat)
    teacher_force(o, g)
    g.update(1)
    o.update(1)
    for k in NET_KEYS:
        assert per_tensor_rel(o, k, g.read_params("g_" + k), oracle_grad_flat(o, k)) <= FP32_TOL, k
    g.close()


# ---------------------------------------------------------------------------- 10-step runs
def ten_steps(w, rows, steps=10, virtual=False, n_streams=2):
    g, o = make_pair(w, rows, virtual=virtual, n_streams=n_streams)
    p0 = {k: o.params(k) for k in NET_KEYS}
    hist = {k: [] for k in NET_KEYS}
    for _ in range(steps):
        g.update(1)
        o.update(1)
        for k in NET_KEYS:
            if o.last_grads[k] is not None:
                hist[k].append(oracle_grad_flat(o, k))
    rg, ro = g.read_losses(1, steps), o.losses()
    out = {k: (g.read_params(k), o.params(k)) for k in state_keys(w.algo)}
    out["p0"] = p0
    g.close()
    return rg, ro, out, o, hist


def check_ten_step_params(w, params, o, hist, steps):
    """Free-running runs: parameters and targets against the oracle, sign-ambiguous
    elements held to their Adam bound. Adam's moments integrate the gradients, which
    jump apart where a ReLU decision within float32 rounding of zero falls differently;
    they are compared step by step in the teacher-forced trajectories."""
    p0 = params.get("p0", {})
    for k, val in params.items():
        if k == "p0":
            continue
        pg, pr = val
        if k in ("log_alpha", "m_log_alpha", "v_log_alpha"):
            assert abs(pg[0] - pr[0]) <= FP32_TOL * max(abs(pr[0]), 1e-2 if k == "log_alpha" else 1e-12), (k, pg, pr)
            continue
        if k.startswith(("m_", "v_")):
            # compared step by step in the teacher-forced trajectories; logged here
            log("  %s %s rel %.2e (free-running)" % (w.name, k, per_tensor_rel(o, k[2:], pg, pr)))
            continue
        net = k[1:] if k.startswith("t") else k
        amb = ambiguous_steps(o, net, hist[net])
        lr = w.lr_actor if net == "actor" else w.lr_critic
        e = check_param_parity(o, net, pg, pr, amb, FP32_TOL, lr, steps, p0=p0.get(k))
        log("  %s %s param rel %.2e (ambiguous %d of %d)" % (w.name, k, e, int((amb > 0).sum()), amb.size))


@pytest.mark.parametrize("w,rows,virtual", [(W["sac_small"], 10_000, False), (RAGGED, 5000, False),
                                            (RAGGED_TD3, 5000, False), (W["sac_walker"], 1_000_000, True)],
                         ids=["sac_small", "ragged_sac", "ragged_td3", "sac_walker_full"])
def test_ten_step_parity_fp32(w, rows, virtual):
    log("10-step %s" % w.name)
    rg, ro, params, o, hist = ten_steps(w, rows, virtual=virtual)
    check_losses(rg, ro, FP32_TOL, w.name)
    check_ten_step_params(w, params, o, hist, 10)


@pytest.mark.parametrize("w,rows,n_steps", [
    (W["sac_small"], 10_000, 10), (RAGGED, 5000, 10), (RAGGED_TD3, 5000, 10), (SEQ_SAC, 5000, 10),
    (DEEP, 3000, 10)], ids=["sac_small", "ragged_sac", "ragged_td3", "sequential_sac", "deep_sac"])
def test_teacher_forced_trajectory_fp32(w, rows, n_steps):
    """Every step of a 10-step oracle trajectory, the GPU started from the oracle's state
    each time: gradients, Adam moments m and v (with their real histories and bias
    corrections at t = 1..10) and the losses of each step within rel 1e-4.

    A ReLU decision on a pre-activation within float32 rounding of zero may fall either
    way; where it does, a weight gradient moves by about 1 / sqrt(batch x width) of its
    size (measured 9.7e-4 at batch 8192 x 256 units, 4.8e-4 at 32768 x 400), above this
    bar. At these sizes (up to 1000 x 160 per layer) no such decision arises in these
    seeded runs; at the full batch sizes the free-running parameter checks and the
    full-size bf16 step (whose bars cover it) take over."""
    log("teacher-forced trajectory %s" % w.name)
    teacher_forced(w, rows, n_steps=n_steps)


@pytest.mark.parametrize("w", [SEQ_SAC, SEQ_TD3], ids=["sac", "td3"])
def test_ten_step_parity_sequential(w):
    log("10-step %s" % w.name)
    rg, ro, params, o, hist = ten_steps(w, 5000)
    check_losses(rg, ro, FP32_TOL, w.name)
    check_ten_step_params(w, params, o, hist, 10)


@pytest.mark.slow
def test_td3_full_batch_parity():
    w = W["td3_ant"].replace(capacity=200_000)
    log("4-step td3_ant full batch")
    rg, ro, params, o, hist = ten_steps(w, 200_000, steps=4, virtual=True)
    check_losses(rg, ro, FP32_TOL, w.name)
    check_ten_step_params(w, params, o, hist, 4)


@pytest.mark.parametrize("w,rows,steps", [(RAGGED_BF16, 5000, 10), (FUSED_BF16, 5000, 10),
                                          (W["sac_humanoid_bf16"].replace(capacity=100_000), 100_000, 4),
                                          (W["sac_large_bf16"].replace(batch=1024, capacity=20_000), 20_000, 3)],
                         ids=["ragged_bf16", "fused_bf16", "humanoid_bf16", "large_bf16_b1024"])
def test_bf16_loss_parity(w, rows, steps):
    log("bf16 %s" % w.name)
    rg, ro, _, _, _ = ten_steps(w, rows, steps=steps, virtual=rows > 50_000)
    check_losses(rg, ro, BF16_LOSS_TOL, w.name)


# ---------------------------------------------------------------------------- invariances
@pytest.mark.parametrize("w,rows,steps", [
    (RAGGED, 5000, 10), (FUSED_BF16, 5000, 4), (FUSED_TD3_BF16, 5000, 4),
    (W["sac_large_bf16"].replace(batch=2560, capacity=20_000), 20_000, 3)],
    ids=["ragged_fp32", "fused_bf16_row_split", "fused_td3_bf16", "large_b2560"])
def test_stream_and_chunk_invariance_bit_exact(w, rows, steps):
    """One stream (where the actor part reuses the critic operand and, for SAC bf16,
    takes the row split) and two concurrent streams give bit-identical parameters,
    targets, Adam moments and loss records; so do different update() chunkings."""
    log("invariance %s" % w.name)
    half = steps // 2
    runs = []
    for n_streams, chunks in ((2, [steps]), (1, [steps]), (2, [half, steps - half]), (1, [1] * steps)):
        g = make_gpu(w, n_streams=n_streams)
        g.buffer_push(*synth.workload_rows(w, 0, rows, 0))
        for c in chunks:
            g.update(c)
        keys = ["actor", "critic1", "critic2", "tcritic1", "tcritic2", "log_alpha", "m_critic1", "v_actor"]
        runs.append({k: g.read_params(k) for k in keys + (["tactor"] if w.algo == "td3" else [])})
        runs[-1]["rec"] = g.read_losses(1, steps)
        g.close()
    for r in runs[1:]:
        for k in r:
            assert np.array_equal(r[k], runs[0][k]), k


def test_profile_only_times_one_kernel_and_keeps_results():
    """Kernel timing restricted to one family and shape records only those launches,
    and timing (all launches or one kernel) leaves the update bit-identical."""
    w = FUSED_BF16
    log("profile filter")
    runs = []
    for mode in ("off", "all", "one"):
        g = make_gpu(w)
        g.buffer_push(*synth.workload_rows(w, 0, 5000, 0))
        if mode != "off":
            g.profile_enable(True, 100)
        if mode == "one":
            g.profile_only("gemm_fwd", 512, 128, 256)
        g.update(3)
        stats = g.profile_read() if mode != "off" else []
        if mode == "all":
            assert {s["name"] for s in stats} >= {"gemm_fwd", "gemm_dgrad", "gemm_wgrad", "gather", "adam_polyak"}
            n_fwd = [s["launches"] for s in stats if (s["name"], s["M"], s["N"], s["K"]) == ("gemm_fwd", 512, 128, 256)]
            assert n_fwd and n_fwd[0] > 0
        if mode == "one":
            assert [(s["name"], s["M"], s["N"], s["K"]) for s in stats] == [("gemm_fwd", 512, 128, 256)]
            assert stats[0]["launches"] == n_fwd[0] and stats[0]["total_ms"] > 0
        runs.append({k: g.read_params(k) for k in ("actor", "critic1", "critic2")})
        g.close()
    for r in runs[1:]:
        for k in r:
            assert np.array_equal(r[k], runs[0][k]), k


def test_profile_stride_times_every_kth_step():
    """With a profile stride of 3, only steps 3 and 6 of 7 carry timed launches."""
    w = FUSED_BF16
    g = make_gpu(w)
    g.buffer_push(*synth.workload_rows(w, 0, 5000, 0))
    g.profile_enable(True, 1000)
    g.profile_stride(3)
    g.update(7)
    st = {s["name"]: s["launches"] for s in g.profile_read()}
    g.profile_enable(True, 1000)
    g.profile_stride(1)
    g.update(1)
    one = {s["name"]: s["launches"] for s in g.profile_read()}
    g.close()
    assert st["gather"] == 2 and st["finish"] == 2, st
    assert st == {k: 2 * v for k, v in one.items()}, (st, one)


def test_sequential_runs_on_one_stream_and_differs_from_snapshot():
    """The sequential ordering ignores the second stream (bit-identical runs) and
    moves the actor differently from the snapshot ordering."""
    runs = []
    for w, n_streams in ((SEQ_SAC, 2), (SEQ_SAC, 1), (RAGGED, 1)):
        g = make_gpu(w, n_streams=n_streams)
        g.buffer_push(*synth.workload_rows(w, 0, 5000, 0))
        g.update(3)
        runs.append({k: g.read_params(k) for k in ("actor", "critic1", "log_alpha")})
        g.close()
    for k in runs[0]:
        assert np.array_equal(runs[0][k], runs[1][k]), k
    assert not np.array_equal(runs[0]["actor"], runs[2]["actor"])


def _split_runs(w, rows, steps, tie=False):
    from paper_2312_06126_amd import Spz
    out = []
    for split in (0, 1):
        g = Spz(w.obs_dim, w.act_dim, w.hidden, w.batch, dict(w.hparams(), actor_row_split=split), 1)
        g.buffer_push(*synth.workload_rows(w, 0, rows, 0))
        if tie:
            # Equal critics: min(Q1, Q2) is a tie on every row and all rows go to critic 1.
            g.write_params("critic2", g.read_params("critic1"))
        g.profile_enable(True, 4096)
        g.update(steps)
        names = {s["name"] for s in g.profile_read()}
        assert ("minq_split" in names) == bool(split), names
        out.append({k: g.read_params(k) for k in ("actor", "critic1", "critic2", "log_alpha")})
        out[-1]["rec"] = g.read_losses(1, steps)
        g.close()
    return out


@pytest.mark.parametrize("w,rows,steps,tie", [
    (FUSED_BF16, 5000, 4, False), (FUSED_BF16_DEEP, 5000, 3, False), (SEQ_BF16, 5000, 3, False),
    (FUSED_BF16, 5000, 1, True), (W["sac_large_bf16"].replace(batch=2560, capacity=20_000), 20_000, 2, False),
    # one row (one list empty); all 700 rows to critic 1 (padded length capped at Bp = 768)
    (FUSED_BF16.replace(batch=1), 1000, 3, False), (FUSED_BF16.replace(batch=700), 5000, 1, True)],
    ids=["fused", "deep", "sequential", "all_ties", "large_b2560", "batch1", "ties_b700_cap"])
def test_actor_row_split_bit_exact(w, rows, steps, tie):
    """Each critic's gradient to the action taken only on the rows where it attains
    min(Q1, Q2) (padded row lists, device-side row counts) gives exactly what taking
    both critics over every row gives, including the all-ties case (one list empty)."""
    log("row split %s" % w.name)
    a, b = _split_runs(w, rows, steps, tie)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("w,created", [(RAGGED.replace(batch=600), 1000), (FUSED_BF16, 1000)],
                         ids=["fp32", "bf16_fused"])
def test_set_batch_equals_created_batch_bit_exact(w, created):
    """A context created with a larger batch and set to w.batch computes exactly
    what a context created with w.batch computes."""
    log("set_batch %s" % w.name)
    out = []
    for b in (created, w.batch):
        g = make_gpu(w.replace(batch=b))
        g.buffer_push(*synth.workload_rows(w, 0, 5000, 0))
        if b != w.batch:
            g.set_batch(w.batch)
        assert g.batch == w.batch
        g.update(3)
        out.append({k: g.read_params(k) for k in ("actor", "critic1", "tcritic2", "log_alpha")})
        out[-1]["rec"] = g.read_losses(1, 3)
        out[-1]["idx"] = g.debug_indices()
        g.close()
    for k in out[0]:
        assert np.array_equal(out[0][k], out[1][k]), k


def test_batch_changes_mid_run_parity():
    """Grow and shrink the batch between steps; the oracle follows the same sizes
    (rows past the batch left by a larger earlier batch must not leak in)."""
    w = RAGGED.replace(batch=1000)
    log("batch changes %s" % w.name)
    g, o = make_pair(w, 5000)
    p0 = {k: o.params(k) for k in NET_KEYS}
    hist = {k: [] for k in NET_KEYS}
    for b, n in ((1000, 2), (300, 2), (777, 1), (1000, 1), (40, 2)):
        g.set_batch(b)
        o.set_batch(b)
        for _ in range(n):
            g.update(1)
            o.update(1)
            assert np.array_equal(g.debug_indices(), o.last_idx.astype(np.int32))
            for k in NET_KEYS:
                hist[k].append(oracle_grad_flat(o, k))
    check_losses(g.read_losses(1, o.t), o.losses(), FP32_TOL, w.name)
    params = {k: (g.read_params(k), o.params(k)) for k in state_keys(w.algo)}
    params["p0"] = p0
    check_ten_step_params(w, params, o, hist, o.t)
    g.close()


def test_autotune_batch_probes_geometrically():
    """The controller probes b_min * 2^k up to the created batch (stopping at
    saturation), picks one of the probed sizes, sets it, and its probes are real
    update steps."""
    from paper_2312_06126_amd.spz import SpzError
    w = RAGGED.replace(batch=4096, capacity=20000)
    g = make_gpu(w, n_streams=1)
    g.buffer_push(*synth.workload_rows(w, 0, 20000, 0))
    chosen, probes = g.autotune_batch(256, 3, 0.05)
    log("autotune probes %s chosen %d" % (probes, chosen))
    sizes = [b for b, _ in probes]
    assert sizes[0] == 256
    assert all(sizes[i + 1] == min(2 * sizes[i], 4096) for i in range(len(sizes) - 1))
    assert chosen in sizes and g.batch == chosen
    assert all(r > 0 for _, r in probes)
    assert g.step() == 4 * len(probes)
    rec = g.read_losses(1, g.step())
    assert np.all(rec[:, 6] == 0)
    with pytest.raises(SpzError):
        g.autotune_batch(8192, 3, 0.05)
    with pytest.raises(SpzError):
        g.set_batch(4097)
    g.close()


@pytest.mark.parametrize("w", [RAGGED, RAGGED_BF16, FUSED_BF16, RAGGED_TD3], ids=lambda w: w.name)
def test_sampler_actions_parity(w):
    """spz_act against the oracle's actor after a few updates: mean and sampled
    actions, batches below, at and above the created batch (chunked)."""
    log("act %s" % w.name)
    g, o = make_pair(w, 5000)
    g.update(2)
    o.update(2)
    teacher_force(o, g)
    tol = 1e-5 if w.prec == "fp32" else 2e-2
    for n in (1, 37, w.batch, 2 * w.batch + 5):
        obs = synth.workload_rows(w, 100, n, 7)[0]
        for stochastic in ((False, True) if w.algo == "sac" else (False,)):
            got = g.act(obs, stochastic=stochastic, counter=9)
            ref = o.act(obs.astype(np.float64), stochastic, 9)
            err = np.abs(got - ref).max()
            assert err <= tol, (n, stochastic, err)
    if w.algo == "td3":
        from paper_2312_06126_amd.spz import SpzError
        with pytest.raises(SpzError):
            g.act(obs, stochastic=True)
    g.close()


@pytest.mark.parametrize("use_stream", [False, True], ids=["null_stream", "side_stream"])
def test_async_push_equals_sync_push_bit_exact(use_stream):
    """The same sequence of pushes and updates gives identical results with
    asynchronous and synchronous pushes: rows are seen by exactly the steps
    enqueued after the push. Covers several staging slots (more rows than four
    slots hold), a wrapping ring, and a torch side stream for the updates."""
    import torch
    w = RAGGED.replace(capacity=300_000)
    rows = synth.workload_rows(w, 0, 600_000, 0)
    part = lambda a, b: [x[a:b] for x in rows]
    plan = [("push", 0, 3000), ("update", 2), ("push", 3000, 4500), ("update", 2), ("push", 4500, 5000),
            ("push", 5000, 5200), ("update", 3), ("push", 5200, 600_000), ("update", 2)]
    stream = torch.cuda.Stream() if use_stream else None
    out = []
    for async_ in (False, True):
        g = make_gpu(w)
        sizes = []
        for op in plan:
            if op[0] == "push":
                (g.buffer_push_async if async_ else g.buffer_push)(*part(op[1], op[2]))
                sizes.append(g.buffer_size())
            else:
                g.update(op[1], stream)
        g.synchronize()
        if stream is not None:
            stream.synchronize()
        st = {k: g.read_params(k) for k in ("actor", "critic1", "tcritic2", "log_alpha", "m_critic2")}
        st["rec"] = g.read_losses(1, 9)
        st["idx"] = g.debug_indices()
        st["sizes"] = np.array(sizes)
        out.append(st)
        g.close()
    assert list(out[0]["sizes"]) == [3000, 4500, 5000, 5200, 300_000]
    for k in out[0]:
        assert np.array_equal(out[0][k], out[1][k]), k


def _full_state(g, w, n_steps):
    st = {k: g.read_params(k) for k in state_keys(w.algo)}
    st["rec"] = g.read_losses(1, n_steps)
    st["idx"] = g.debug_indices()
    st["step"] = g.step()
    return st


@pytest.mark.parametrize("w", [RAGGED, FUSED_TD3_BF16], ids=["sac_fp32", "td3_bf16_fused"])
def test_checkpoint_resume_bit_exact(w, tmp_path):
    """Save after 3 steps, continue 4 steps; a fresh context (other seed, empty or
    identically filled ring) that loads the file and runs 4 steps ends bit-identical."""
    from paper_2312_06126_amd.spz import SPZ_EIO, SpzError
    log("checkpoint %s" % w.name)
    rows = synth.workload_rows(w, 0, 5000, 0)
    for ring in (True, False):
        path = str(tmp_path / ("ckpt_%d.spz" % ring))
        g = make_gpu(w)
        g.buffer_push(*rows)
        g.update(3)
        g.save(path, ring=ring)
        g.update(4)
        ref = _full_state(g, w, 7)
        g.close()
        h = make_gpu(w, seed=99)
        if not ring:
            h.buffer_push(*rows)
        h.load(path)
        assert h.step() == 3 and h.buffer_size() == 5000
        h.update(4)
        got = _full_state(h, w, 7)
        h.close()
        for k in ref:
            assert np.array_equal(np.asarray(ref[k]), np.asarray(got[k])), (ring, k)
    other = make_gpu(w.replace(hidden=(256, 64)))
    with pytest.raises(SpzError) as e:
        other.load(str(tmp_path / "ckpt_1.spz"))
    assert e.value.code == SPZ_EIO
    with pytest.raises(SpzError) as e:
        other.load(str(tmp_path / "missing.spz"))
    assert e.value.code == SPZ_EIO
    other.close()


def test_tau_one_targets_equal_online_bit_exact():
    w = RAGGED.replace(tau=1.0)
    g = make_gpu(w)
    g.buffer_push(*synth.workload_rows(w, 0, 2000, 0))
    g.update(3)
    for k in ("critic1", "critic2"):
        assert np.array_equal(g.read_params("t" + k), g.read_params(k))
    g.close()


# ---------------------------------------------------------------------------- edge cases
def test_error_codes():
    from paper_2312_06126_amd.spz import SPZ_EEMPTY, SPZ_EINVAL, SPZ_ESIZE, SpzError
    w = RAGGED
    g = make_gpu(w)
    with pytest.raises(SpzError) as e:
        g.update(1)
    assert e.value.code == SPZ_EEMPTY
    with pytest.raises(SpzError) as e:
        g.read_params("tactor")
    assert e.value.code == SPZ_EINVAL
    with pytest.raises(SpzError) as e:
        g.write_params("actor", np.zeros(3, np.float32))
    assert e.value.code == SPZ_ESIZE
    with pytest.raises(SpzError) as e:
        g.read_losses(1, 1)
    assert e.value.code == SPZ_EINVAL
    g.buffer_push(*synth.workload_rows(w, 0, 10, 0))
    g.update(0)
    assert g.step() == 0
    g.close()


def test_tiny_ring_wraps_and_batch_one():
    """Capacity 7 with 10 rows pushed (FIFO overwrite), then batch 1 over a 1-row ring."""
    w = RAGGED.replace(capacity=7, batch=64)
    g, o = make_pair(w, 10)
    assert g.buffer_size() == 7
    g.update(2)
    o.update(2)
    check_losses(g.read_losses(1, 2), o.losses(), FP32_TOL, "wrap")
    g.close()
    w1 = RAGGED.replace(capacity=1, batch=1)
    g, o = make_pair(w1, 1)
    g.update(3)
    o.update(3)
    assert np.array_equal(g.debug_indices(), np.zeros(1, np.int32))
    check_losses(g.read_losses(1, 3), o.losses(), FP32_TOL, "batch1")
    g.close()


def test_terminal_and_zero_discount():
    """done = 1 everywhere and gamma = 0 both make the target equal to the reward."""
    w = RAGGED.replace(gamma=0.0)
    g, o = make_pair(w, 3000)
    g.update(2)
    o.update(2)
    check_losses(g.read_losses(1, 2), o.losses(), FP32_TOL, "gamma0")
    g.close()
    w = RAGGED.replace(p_done=1.0)
    g, o = make_pair(w, 3000)
    g.update(2)
    o.update(2)
    check_losses(g.read_losses(1, 2), o.losses(), FP32_TOL, "done1")
    g.close()
