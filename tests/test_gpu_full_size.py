"""The whole update step of the large-batch SAC workload at its full size, against
the oracle (Section 3.2.1's large-batch update at the largest configuration: obs 376,
act 17, 3 x 1024 ReLU MLPs, batch 131072, bf16 operands, fp32 master weights and
Adam), in the launch configuration the benchmark times: one stream, the actor's
gradient through each critic on that critic's rows only.

The GPU runs two steps from the seeded start; the oracle then takes the GPU's whole
state (parameters, targets, Adam moments, temperature, step counters) and both run
step 3, the oracle taking the GPU's twin-minimum choice per row (a floating-point
decision of a discrete choice; validated: wherever the oracle's own choice differs,
its two critic values are within 1e-3 of their rms). Compared with the oracle:
  * the loss record (rel 2e-2, the bf16 loss bar; every value also logged);
  * every gradient tensor of the actor, both critics and log(alpha), whole tensors
    summed over all 131072 rows: this covers the split-K weight gradients over the
    batch, the bias gradients from the fused column sums and the row-split input
    gradients. Critics and log(alpha): per-tensor rel 1e-3, the teacher-forced bf16
    bar. Actor: 1e-2, the bar of the per-row action gradient it is built from (three
    more rounded layers of dz inside the critics; bf16 rounding flips between float32
    and float64 accumulation move it by about 1e-3 per row), which a weight gradient
    whose rows cancel -- the first layer's, over N(0, 1) observations -- inherits
    (observed 1.6e-3 there, 1e-4 to 2e-4 elsewhere);
  * the parameters, targets and Adam moments after the step (parameters and targets
    per-tensor rel 1e-4 over elements that are not sign-ambiguous for Adam, which
    stay within their step bound; m and v per tensor within their net's gradient bar,
    since the step's gradient enters them with weight 1 - beta).
The ring holds 200000 rows (its size only changes which rows are drawn). The
oracle's float64 step at this size takes about a minute of host time.
"""
import numpy as np
import pytest

import synth

from .helpers import (AMBIGUOUS, check_min_choice, check_param_parity, fill_rows, gpu_min_choice, log, make_gpu,
                      make_oracle, per_tensor_rel, state_keys, tensor_slices)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

BF16_LOSS_TOL = 2e-2
GRAD_TOL = 1e-3
ACTOR_GRAD_TOL = 1e-2
PARAM_TOL = 1e-4


def adopt_gpu_state(o, g):
    """The oracle takes the GPU's state after g.step() SAC steps."""
    for k in state_keys(o.algo):
        o.set_params(k, g.read_params(k).astype(np.float64))
    t = g.step()
    o.t = t
    o.opt_actor.t = o.opt_critic.t = o.opt_alpha.t = t


@pytest.mark.timeout(1800)
def test_full_size_teacher_forced_step_sac_large():
    rows = 200_000
    w = synth.workload("sac_large_bf16").replace(capacity=rows)
    log("full-size step %s batch %d (one stream, row split)" % (w.name, w.batch))
    g = make_gpu(w, n_streams=1)
    fill_rows(w, rows, 0, [g.buffer_push])
    g.update(2)
    o = make_oracle(w, virtual_rows=rows)
    adopt_gpu_state(o, g)
    g.update(1)
    rec_g = g.read_losses(3, 1)[0].astype(np.float64)
    grads_g = {k: g.read_params("g_" + k) for k in ("actor", "critic1", "critic2", "log_alpha")}
    state_g = {k: g.read_params(k) for k in state_keys(o.algo)}
    idx_g = g.debug_indices()
    take1 = gpu_min_choice(g)
    g.close()
    log("  GPU step done; oracle step (float64, batch %d)" % w.batch)
    o.progress = lambda what: log("  oracle " + what)
    o.forced_min_choice = take1
    o.update(1)
    assert np.array_equal(idx_g, o.last_idx.astype(np.int32))
    log("  twin-minimum rows taken from the GPU where the oracle decided otherwise: %d"
        % check_min_choice(o, take1, 1e-3))

    rec_o = o.losses()[-1]
    err = np.abs(rec_g[:6] - rec_o[:6]) / np.maximum(np.abs(rec_o[:6]), 1e-6 / BF16_LOSS_TOL)
    log("  losses gpu %s oracle %s rel %s" % (rec_g[:6], rec_o[:6], err))
    assert np.all(err <= BF16_LOSS_TOL), err
    assert rec_g[6] == rec_o[6] == 0.0 and rec_g[7] == rec_o[7] == 1.0

    for k in ("actor", "critic1", "critic2"):
        gr = np.concatenate([np.concatenate([gw.ravel(), gb.ravel()]) for gw, gb in o.last_grads[k]])
        e = per_tensor_rel(o, k, grads_g[k], gr)
        log("  gradient %s worst per-tensor rel %.2e" % (k, e))
        assert e <= (ACTOR_GRAD_TOL if k == "actor" else GRAD_TOL), (k, e)
    ga = o.last_grads["log_alpha"]
    assert abs(grads_g["log_alpha"][0] - ga) <= GRAD_TOL * max(abs(ga), 1e-6), (grads_g["log_alpha"], ga)

    b2, t = w.beta2, o.t
    for k in state_keys(o.algo):
        pg, pr = state_g[k], o.params(k)
        if k in ("log_alpha", "m_log_alpha", "v_log_alpha"):
            assert abs(pg[0] - pr[0]) <= GRAD_TOL * max(abs(pr[0]), 1e-12), (k, pg, pr)
            continue
        if k.startswith(("m_", "v_")):
            e = per_tensor_rel(o, k[2:], pg, pr)
            log("  %s worst per-tensor rel %.2e" % (k, e))
            assert e <= (ACTOR_GRAD_TOL if k[2:] == "actor" else GRAD_TOL), (k, e)
            continue
        # Elements whose whole gradient history (the oracle's v after the step) is tiny
        # next to the tensor's gradient take their Adam direction from rounding.
        net = k[1:] if k.startswith("t") else k
        v_hat = o.params("v_" + net) / (1.0 - b2 ** t)
        gflat = np.concatenate([np.concatenate([gw.ravel(), gb.ravel()]) for gw, gb in o.last_grads[net]])
        amb = np.zeros(v_hat.size, np.int64)
        for sl in tensor_slices(o, net):
            rms = np.sqrt(np.mean(gflat[sl] ** 2))
            root = np.sqrt(v_hat[sl])   # exactly 0: no gradient ever (zeroed observation columns)
            amb[sl] = ((root < AMBIGUOUS * rms) & (root > 0.0)).astype(np.int64) * t
        lr = w.lr_actor if net == "actor" else w.lr_critic
        e = check_param_parity(o, net, pg, pr, amb, PARAM_TOL, lr, t)
        log("  %s worst per-tensor rel %.2e (ambiguous %d of %d)" % (k, e, int((amb > 0).sum()), amb.size))
