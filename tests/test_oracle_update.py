"""Pins for the oracle's update step (CPU, float64).

* finite-difference gradients on tiny nets for the critic, SAC actor, TD3 actor
  and temperature losses (central differences, h = 1e-6);
* the tanh-Gaussian log-density against scipy's normal log-pdf plus the
  change-of-variables term, and its closed form at mu = logstd = eps = 0;
* closed-form TD targets and critic losses on hand-built nets whose outputs are
  constants;
* Adam against torch.optim.Adam and against the scalar first step;
* Polyak invariants (tau = 1 copies bit-for-bit, tau = 0 keeps), TD3's delay;
* mutation checks: plausible mistakes planted in the oracle make a pin fail.
"""
import copy
import math

import numpy as np
import pytest
from scipy import stats

import oracle.update as U
from oracle import Oracle, philox

HP = dict(algo="sac", gemm_prec="fp32", capacity=64, gamma=0.99, tau=0.005, lr_actor=3e-4,
          lr_critic=3e-4, lr_alpha=3e-4, beta1=0.9, beta2=0.999, eps=1e-8, alpha_init=0.7,
          learn_alpha=True, target_entropy=-2.0, log_std_min=-20.0, log_std_max=2.0,
          policy_noise=0.2, noise_clip=0.5, policy_delay=2)
O, A, H, B = 3, 2, (4, 4), 5


def tiny(algo="sac", **kw):
    hp = dict(HP, algo=algo, **kw)
    return Oracle(O, A, H, B, hp, seed=11)


def batch(seed=0):
    r = np.random.default_rng(seed)
    return (r.standard_normal((B, O)), r.uniform(-1, 1, (B, A)), r.standard_normal(B),
            (r.uniform(size=B) < 0.4).astype(np.float64), r.standard_normal((B, O)))


def fd_check(orc, net_keys, loss_fn, analytic, h=1e-6, rtol=1e-5, atol=1e-9):
    """Central differences of loss_fn() w.r.t. every element of orc.net[k] for k in net_keys."""
    for k in net_keys:
        for l, (w, b) in enumerate(orc.net[k]):
            for ti, tens in enumerate((w, b)):
                g = analytic[k][l][ti]
                flat = tens.reshape(-1)
                fd = np.empty(flat.size)
                for i in range(flat.size):
                    old = flat[i]
                    flat[i] = old + h
                    lp = loss_fn()
                    flat[i] = old - h
                    lm = loss_fn()
                    flat[i] = old
                    fd[i] = (lp - lm) / (2 * h)
                np.testing.assert_allclose(np.asarray(g).reshape(-1), fd, rtol=rtol, atol=atol,
                                           err_msg="%s layer %d %s" % (k, l, "Wb"[ti]))


# ------------------------------------------------------------------ gradients

def test_fd_critic_loss():
    o = tiny()
    s, a, r, d, s2 = batch(1)
    y = np.random.default_rng(2).standard_normal(B)
    _, cg = o._critic_grads(s, a, y)
    fd_check(o, ("critic1", "critic2"), lambda: o._critic_grads(s, a, y)[0], cg)


@pytest.mark.parametrize("logstd_bias", [0.0, 2.5, -20.5])
def test_fd_sac_actor_loss(logstd_bias):
    o = tiny()
    # push some log-std heads across the clamp bounds to exercise the mask
    o.net["actor"][-1][1][A:] += logstd_bias
    s = batch(3)[0]
    eps = np.random.default_rng(4).standard_normal((B, A))
    alpha = 0.37
    _, ag, pol = o.sac_actor(s, eps, alpha)
    fd_check(o, ("actor",), lambda: o.sac_actor(s, eps, alpha)[0], {"actor": ag})
    if logstd_bias == 2.5:
        assert np.any(pol["l"] > 2.0)


def test_fd_td3_actor_loss():
    o = tiny("td3")
    s = batch(5)[0]
    _, ag = o.td3_actor(s)
    fd_check(o, ("actor",), lambda: o.td3_actor(s)[0], {"actor": ag})


def test_temperature_gradient_fd():
    o = tiny()
    s, a, r, d, s2 = batch(6)
    o.push(s, a, r, d, s2)
    o.update(1)
    g = o.last_grads["log_alpha"]
    lp = o.last_grads["logp"]
    la0 = math.log(HP["alpha_init"])
    loss = lambda la: -la * float(np.mean(lp + HP["target_entropy"]))
    h = 1e-6
    assert np.isclose(g, (loss(la0 + h) - loss(la0 - h)) / (2 * h), rtol=1e-7)
    rec = o.losses()[0]
    assert np.isclose(rec[U.REC_LALPHA], loss(la0), rtol=1e-12)
    assert np.isclose(rec[U.REC_ALPHA], HP["alpha_init"], rtol=1e-12)


# ------------------------------------------------------------------ forward closed forms

def test_logp_matches_change_of_variables():
    rng = np.random.default_rng(7)
    z = rng.standard_normal((64, 2 * 3))
    z[:, 3:] *= 0.5
    eps = rng.standard_normal((64, 3))
    pol = U.tanh_gaussian(z, eps, 3, -20.0, 2.0)
    mu, sig = z[:, :3], np.exp(np.clip(z[:, 3:], -20, 2))
    u = mu + sig * eps
    ref = np.sum(stats.norm.logpdf(u, loc=mu, scale=sig) - np.log(1.0 - np.tanh(u) ** 2), axis=1)
    np.testing.assert_allclose(pol["logp"], ref, rtol=1e-10, atol=1e-10)
    np.testing.assert_array_equal(pol["a"], np.tanh(u))


def test_logp_closed_form_at_zero_and_stable_tail():
    pol = U.tanh_gaussian(np.zeros((2, 6)), np.zeros((2, 3)), 3, -20.0, 2.0)
    np.testing.assert_allclose(pol["logp"], -1.5 * math.log(2 * math.pi), rtol=0, atol=1e-15)
    # |u| = 30: 1 - tanh^2 underflows in float64 but the stable form stays finite
    z = np.array([[30.0, 0.0]])
    pol = U.tanh_gaussian(z, np.zeros((1, 1)), 1, -20.0, 2.0)
    assert np.isfinite(pol["logp"][0])
    assert np.isclose(pol["logp"][0], -0.5 * math.log(2 * math.pi) - (math.log(4.0) - 60.0), rtol=1e-12)


def _constant_head(layers, bias):
    layers[-1][0][...] = 0.0
    layers[-1][1][...] = bias


def test_sac_td_target_closed_form():
    o = tiny()
    c1, c2 = 0.8, -0.3
    _constant_head(o.net["tcritic1"], c1)
    _constant_head(o.net["tcritic2"], c2)
    m0, l0 = np.array([0.2, -0.4]), np.array([-0.5, 0.3])
    _constant_head(o.net["actor"], np.concatenate([m0, l0]))
    s, a, r, d, s2 = batch(8)
    eps = np.random.default_rng(9).standard_normal((B, A))
    alpha = 0.25
    y, _ = o.sac_target(s2, r, d, eps, alpha)
    u = m0 + np.exp(l0) * eps
    logp = np.sum(stats.norm.logpdf(u, m0, np.exp(l0)) - np.log(1 - np.tanh(u) ** 2), axis=1)
    np.testing.assert_allclose(y, r + 0.99 * (1 - d) * (min(c1, c2) - alpha * logp), rtol=1e-12)
    # terminal rows bootstrap nothing; gamma = 0 gives y = r
    assert np.array_equal(y[d == 1], r[d == 1])
    o.hp["gamma"] = 0.0
    assert np.array_equal(o.sac_target(s2, r, d, eps, alpha)[0], r)


def test_sampler_actions_closed_form():
    """Actor with a constant head: the mean action is tanh(mu); the stochastic
    action is tanh(mu + exp(clip(l)) eps) with eps the purpose-4 normals of the
    counter, row-major over (row, action); TD3 gives tanh(z)."""
    o = tiny()
    m0, l0 = np.array([0.2, -0.4]), np.array([-0.5, 25.0])   # second log-std beyond the clamp
    _constant_head(o.net["actor"], np.concatenate([m0, l0]))
    obs = np.random.default_rng(3).standard_normal((7, O))
    np.testing.assert_allclose(o.act(obs, False, 0), np.tile(np.tanh(m0), (7, 1)), rtol=1e-15)
    eps = philox.normals(o.seed, 123, philox.PURPOSE_ACT, 7 * A).reshape(7, A)
    want = np.tanh(m0 + np.exp(np.minimum(l0, HP["log_std_max"])) * eps)
    np.testing.assert_allclose(o.act(obs, True, 123), want, rtol=1e-15)
    assert not np.array_equal(o.act(obs, True, 124), want)
    t = tiny("td3")
    _constant_head(t.net["actor"], np.array([0.3, -1.2]))
    np.testing.assert_allclose(t.act(obs, False, 0), np.tile(np.tanh([0.3, -1.2]), (7, 1)), rtol=1e-15)
    with pytest.raises(ValueError):
        t.act(obs, True, 0)


def test_critic_loss_closed_form():
    o = tiny()
    _constant_head(o.net["critic1"], 1.5)
    _constant_head(o.net["critic2"], -0.5)
    s, a, r, d, s2 = batch(10)
    y = np.array([0.0, 1.0, 2.0, -1.0, 0.5])
    lq, cg = o._critic_grads(s, a, y)
    assert np.isclose(lq, np.mean((1.5 - y) ** 2) + np.mean((-0.5 - y) ** 2), rtol=1e-14)
    # with a zero last layer, the head bias gradient is the mean residual times 2
    assert np.isclose(cg["critic1"][-1][1][0], 2 * np.mean(1.5 - y), rtol=1e-14)


def test_td3_target_smoothing_closed_form():
    o = tiny("td3")
    _constant_head(o.net["tactor"], 50.0)        # tanh saturates at +1
    _constant_head(o.net["tcritic1"], 2.0)
    _constant_head(o.net["tcritic2"], 3.0)
    s, a, r, d, s2 = batch(11)
    eps = np.array([[3.0, -3.0], [0.5, -0.5], [0.0, 1.0], [-10.0, 10.0], [1.0, -1.0]])
    y, a2 = o.td3_target(s2, r, d, eps)
    want = np.array([[1.0, 0.5], [1.0, 0.9], [1.0, 1.0], [0.5, 1.0], [1.0, 0.8]])
    np.testing.assert_allclose(a2, want, rtol=0, atol=1e-15)
    np.testing.assert_allclose(y, r + 0.99 * (1 - d) * 2.0, rtol=1e-15)


# ------------------------------------------------------------------ optimizer and targets

def test_adam_against_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(12)
    p0 = rng.standard_normal(50)
    grads = [rng.standard_normal(50) * 10.0 ** rng.integers(-3, 2) for _ in range(6)]
    p = p0.copy()
    m, v = np.zeros(50), np.zeros(50)
    opt = U.Adam(3e-4, 0.9, 0.999, 1e-8)
    tp = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    topt = torch.optim.Adam([tp], lr=3e-4, betas=(0.9, 0.999), eps=1e-8)
    for g in grads:
        opt.step([p], [g], [m], [v])
        tp.grad = torch.tensor(g)
        topt.step()
    np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-16)


def test_adam_scalar_first_steps_by_hand():
    opt = U.Adam(0.1, 0.9, 0.999, 1e-8)
    p, m, v = np.array([1.0]), np.zeros(1), np.zeros(1)
    opt.step([p], [np.array([0.5])], [m], [v])
    # m = 0.05, v = 0.00025; corrected: 0.5 and 0.25; step = 0.1 * 0.5 / (0.5 + 1e-8)
    assert np.isclose(m[0], 0.05, rtol=1e-15) and np.isclose(v[0], 0.00025, rtol=1e-15)
    assert np.isclose(p[0], 1.0 - 0.1 * 0.5 / (0.5 + 1e-8), rtol=1e-15)
    opt.step([p], [np.array([-0.25])], [m], [v])
    # m = 0.045 - 0.025 = 0.02; v = 0.00024975 + 0.0000625 = 0.00031225
    assert np.isclose(m[0], 0.02, rtol=1e-14) and np.isclose(v[0], 0.00031225, rtol=1e-14)
    # corrected: 0.02 / 0.19 and 0.00031225 / 0.001999
    step2 = 0.1 * (0.02 / 0.19) / (math.sqrt(0.00031225 / 0.001999) + 1e-8)
    assert np.isclose(p[0], 1.0 - 0.1 * 0.5 / (0.5 + 1e-8) - step2, rtol=1e-14)


def _filled(algo="sac", n=40, **kw):
    o = tiny(algo, **kw)
    s, a, r, d, s2 = (np.random.default_rng(13).standard_normal((n, O)),
                      np.random.default_rng(14).uniform(-1, 1, (n, A)),
                      np.random.default_rng(15).standard_normal(n),
                      (np.random.default_rng(16).uniform(size=n) < 0.1).astype(np.float64),
                      np.random.default_rng(17).standard_normal((n, O)))
    o.push(s, a, r, d, s2)
    return o


def test_polyak_tau_one_copies_exactly_and_tau_zero_keeps():
    o = _filled(tau=1.0)
    o.update(3)
    for k in ("critic1", "critic2"):
        assert np.array_equal(o.params("t" + k), o.params(k))
    o = _filled(tau=0.0)
    t0 = o.params("tcritic1").copy()
    o.update(3)
    assert np.array_equal(o.params("tcritic1"), t0)
    assert not np.array_equal(o.params("critic1"), t0)


def test_polyak_half_by_hand():
    tb, th = [np.array([1.0, -2.0])], [np.array([3.0, 4.0])]
    U.polyak(tb, th, 0.5)
    assert np.array_equal(tb[0], np.array([2.0, 1.0]))


def test_td3_delay_trace():
    o = _filled("td3", tau=0.5)
    hist = [(o.params("actor").copy(), o.params("tactor").copy(), o.params("critic1").copy(),
             o.params("tcritic1").copy())]
    for _ in range(4):
        o.update(1)
        hist.append((o.params("actor").copy(), o.params("tactor").copy(), o.params("critic1").copy(),
                     o.params("tcritic1").copy()))
    for k in range(1, 5):
        moved = [not np.array_equal(hist[k][i], hist[k - 1][i]) for i in range(4)]
        assert moved[2], "critic updates every step"
        assert moved[0] == moved[1] == moved[3] == (k % 2 == 0), (k, moved)
    rec = o.losses()
    assert list(rec[:, U.REC_ACTOR]) == [0, 1, 0, 1]
    assert rec[0, U.REC_LPI] == 0.0 and rec[1, U.REC_LPI] != 0.0
    assert o.opt_actor.t == 2 and o.opt_critic.t == 4


def test_snapshot_semantics_actor_reads_step_start_critic():
    o = _filled()
    snap = copy.deepcopy(o)
    o.update(1)
    idx = o.last_idx
    s = o.last_batch[0]
    eps = philox.normals(o.seed, 1, philox.PURPOSE_NOISE_POL, B * A).reshape(B, A)
    lpi, _, _ = snap.sac_actor(s, eps, HP["alpha_init"])
    assert np.isclose(o.losses()[0, U.REC_LPI], lpi, rtol=1e-14)
    assert np.array_equal(idx, philox.indices(o.seed, 1, B, 40))


def test_sequential_with_frozen_critics_equals_snapshot():
    """With lr_critic = 0 the critics' Adam step leaves them unchanged, so the two
    update orderings must agree bit for bit over several steps (SAC and TD3)."""
    for algo in ("sac", "td3"):
        a = _filled(algo, lr_critic=0.0)
        b = _filled(algo, lr_critic=0.0, ordering="sequential")
        a.update(4)
        b.update(4)
        keys = ["actor", "critic1", "critic2", "tcritic1", "tcritic2"] + (["tactor"] if algo == "td3" else [])
        for k in keys:
            assert np.array_equal(a.params(k), b.params(k)), (algo, k)
        assert np.array_equal(a.losses(), b.losses()), algo


def test_sequential_sac_actor_reads_updated_critics():
    """Sequential ordering: the critic side of the step is the snapshot one, and the
    actor loss and gradient are the snapshot formulas evaluated at the critics after
    this step's critic update (and differ from the step-start ones)."""
    o = _filled(ordering="sequential")
    start = copy.deepcopy(o)
    twin = _filled()
    o.update(1)
    twin.update(1)
    for k in ("critic1", "critic2", "tcritic1", "tcritic2"):
        assert np.array_equal(o.params(k), twin.params(k)), k
    assert o.losses()[0, U.REC_LQ] == twin.losses()[0, U.REC_LQ]
    s = o.last_batch[0]
    eps = philox.normals(o.seed, 1, philox.PURPOSE_NOISE_POL, B * A).reshape(B, A)
    ref = copy.deepcopy(start)
    for k in ("critic1", "critic2"):
        ref.set_params(k, o.params(k))
    lpi_new, ag_new, pol = ref.sac_actor(s, eps, HP["alpha_init"])
    lpi_old, _, _ = start.sac_actor(s, eps, HP["alpha_init"])
    assert np.isclose(o.losses()[0, U.REC_LPI], lpi_new, rtol=1e-14)
    assert abs(lpi_new - lpi_old) > 1e-9 * abs(lpi_old)
    for l, (gw, gb) in enumerate(ag_new):
        np.testing.assert_allclose(o.last_grads["actor"][l][0], gw, rtol=1e-13, atol=1e-300)
        np.testing.assert_allclose(o.last_grads["actor"][l][1], gb, rtol=1e-13, atol=1e-300)
    # the temperature still sees the step-start actor sample
    assert np.isclose(o.losses()[0, U.REC_LOGPI], np.mean(pol["logp"]), rtol=1e-14)
    assert o.losses()[0, U.REC_LOGPI] == twin.losses()[0, U.REC_LOGPI]


def test_sequential_td3_actor_reads_updated_critic():
    """TD3: on the delayed step the actor gradient goes through the critic after that
    step's critic update; on the other steps only the critics move, as in snapshot."""
    o = _filled("td3", ordering="sequential")
    o.update(1)
    start = copy.deepcopy(o)
    o.update(1)                       # step 2: critic update, then actor update
    s = o.last_batch[0]
    ref = copy.deepcopy(start)
    ref.t = 2
    for k in ("critic1", "critic2"):
        ref.set_params(k, o.params(k))
    lpi_new, ag_new = ref.td3_actor(s)
    lpi_old, _ = start.td3_actor(s)
    assert np.isclose(o.losses()[1, U.REC_LPI], lpi_new, rtol=1e-14)
    assert abs(lpi_new - lpi_old) > 1e-9 * abs(lpi_old)
    for l, (gw, gb) in enumerate(ag_new):
        np.testing.assert_allclose(o.last_grads["actor"][l][0], gw, rtol=1e-13, atol=1e-300)
    assert o.opt_actor.t == 1 and o.opt_critic.t == 2


def test_set_batch_equals_created_batch():
    """An oracle created with batch 5 and set to 3 equals one created with batch 3:
    indices and noise of a row depend only on (seed, step, row)."""
    a = _filled()
    a.set_batch(3)
    b = Oracle(O, A, H, 3, dict(HP), seed=11)
    b.push(*[np.asarray(x) for x in (a.buf_obs[:40], a.buf_act[:40], a.buf_rew[:40], a.buf_done[:40],
                                     a.buf_nobs[:40])])
    a.update(3)
    b.update(3)
    assert np.array_equal(a.losses(), b.losses())
    for k in ("actor", "critic1", "tcritic2", "log_alpha"):
        assert np.array_equal(a.params(k), b.params(k)), k


def test_step_zero_params_are_the_fanin_init():
    o = tiny()
    w0 = o.net["critic2"][0][0]
    np.testing.assert_array_equal(w0.reshape(-1), philox.init_uniform(11, 2 * 16 + 0, w0.size, O + A))
    assert np.array_equal(o.params("tcritic2"), o.params("critic2"))


def test_ring_fifo_and_empty():
    o = tiny(capacity=4)
    with pytest.raises(RuntimeError):
        o.update(1)
    rows = lambda lo, n: (np.arange(lo, lo + n)[:, None] * np.ones((1, O)), np.zeros((n, A)),
                          np.arange(lo, lo + n, dtype=float), np.zeros(n), np.zeros((n, O)))
    o.push(*rows(0, 3))
    assert o.size == 3 and o.ptr == 3
    o.push(*rows(3, 3))          # slots 3, 0, 1 overwritten by 3, 4, 5
    assert o.size == 4 and o.ptr == 2
    assert list(o.buf_rew) == [4, 5, 2, 3]
    o.push(*rows(10, 9))         # only the last 4 rows survive: 15..18 land in slots 3,0,1,2
    assert list(o.buf_rew) == [16, 17, 18, 15] and o.ptr == 3


# ------------------------------------------------------------------ the pins have teeth

def test_mutation_dropped_entropy_gradient_is_caught():
    """Plant a dropped term (the 2*tanh(u) entropy gradient) in the oracle: FD must fail."""
    o = tiny()
    s = batch(3)[0]
    eps = np.random.default_rng(4).standard_normal((B, A))
    alpha = 0.37
    z, xs_a = U.forward(o.net["actor"], s, o.rnd)
    pol = U.tanh_gaussian(z, eps, A, -20.0, 2.0)
    xa = np.concatenate([s, pol["a"]], 1)
    qp1 = U.forward(o.net["critic1"], xa, o.rnd)[0][:, 0]
    qp2 = U.forward(o.net["critic2"], xa, o.rnd)[0][:, 0]
    take1 = qp1 <= qp2
    da = o._critic_action_grad(s, pol["a"], {"critic1": np.where(take1, -1.0 / B, 0.0),
                                             "critic2": np.where(take1, 0.0, -1.0 / B)})
    g_u = da * (1.0 - pol["a"] ** 2)                      # planted: + (alpha/B) 2 tanh(u) dropped
    d_l = g_u * pol["sigma"] * eps - alpha / B
    ag_bad, _ = U.backward(o.net["actor"], xs_a, np.concatenate([g_u, d_l], 1), o.rnd)
    with pytest.raises(AssertionError):
        fd_check(o, ("actor",), lambda: o.sac_actor(s, eps, alpha)[0], {"actor": ag_bad})


def test_mutation_transposed_operand_is_caught(monkeypatch):
    """Plant a transposed weight in the backward pass (square 4x4 layer): FD must fail."""
    o = tiny()
    s, a, r, d, s2 = batch(1)
    y = np.random.default_rng(2).standard_normal(B)

    def bad_backward(layers, xs, dz, rnd, want_wgrad=True, want_dx=False):
        grads, dx = [None] * len(layers), None
        for l in reversed(range(len(layers))):
            w = layers[l][0]
            grads[l] = (rnd(dz).T @ xs[l], rnd(dz).sum(0))
            if l > 0:
                wl = w.T if w.shape[0] == w.shape[1] else w           # planted transpose
                dz = (rnd(dz) @ rnd(wl)) * (xs[l] > 0)
        return grads, dx
    monkeypatch.setattr(U, "backward", bad_backward)
    _, cg_bad = o._critic_grads(s, a, y)
    monkeypatch.undo()
    with pytest.raises(AssertionError):
        fd_check(o, ("critic1",), lambda: o._critic_grads(s, a, y)[0], cg_bad)


def test_mutation_wrong_sign_in_target_is_caught():
    o = tiny()
    c1, c2 = 0.8, -0.3
    _constant_head(o.net["tcritic1"], c1)
    _constant_head(o.net["tcritic2"], c2)
    s, a, r, d, s2 = batch(8)
    eps = np.zeros((B, A))
    alpha = 0.25
    y, pol2 = o.sac_target(s2, r, d, eps, alpha)
    wrong = r + 0.99 * (1 - d) * (min(c1, c2) + alpha * pol2["logp"])   # sign flipped
    assert not np.allclose(y[d == 0], wrong[d == 0])


def test_nan_reward_sets_nonfinite_flag():
    """A NaN reward in a sampled row makes the step's losses NaN and sets the
    non-finite flag (the loss record's contract); min(Q1', Q2') propagates a NaN."""
    o = _filled(n=40)
    idx = philox.indices(o.seed, 1, o.B, o.size)
    o.buf_rew[idx[0]] = np.nan
    with np.errstate(invalid="ignore"):
        o.update(1)
    rec = o.losses()[0]
    assert np.isnan(rec[U.REC_LQ]) and rec[U.REC_NONFINITE] == 1.0
    assert np.isnan(np.minimum(np.nan, 1.0)) and np.isnan(np.minimum(1.0, np.nan))
    clean = _filled(n=40)
    clean.update(1)
    assert clean.losses()[0][U.REC_NONFINITE] == 0.0


def test_forced_min_choice_hook():
    """The twin-minimum test hook: forcing the oracle's own choice changes nothing;
    forcing the opposite choice on every row changes the actor's step but not the
    critics' (they do not see the actor loss), and the hook applies to one step only."""
    a, b, c = _filled(n=40), _filled(n=40), _filled(n=40)
    for o in (a, b, c):
        o.set_batch(32)
    a.update(1)
    own = a.last_min_choice.copy()
    b.forced_min_choice = own
    b.update(1)
    for k in ("actor", "critic1", "critic2", "log_alpha"):
        assert np.array_equal(a.params(k), b.params(k)), k
    c.forced_min_choice = ~own
    c.update(1)
    assert np.array_equal(c.last_min_choice, own)
    assert not np.array_equal(a.params("actor"), c.params("actor"))
    for k in ("critic1", "critic2", "log_alpha"):
        assert np.array_equal(a.params(k), c.params(k)), k
    assert c.forced_min_choice is None
