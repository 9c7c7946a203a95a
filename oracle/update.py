"""One network-update step of the actor-critic learner, float64, step by step.

The paper's learner (Section 3.2) draws a large uniform batch from the shared
replay pool (Section 3.3.2) and updates the actor and the double-Q critics with
their target networks, the actor and the critics being updated independently
(Section 3.2.2). SAC is its worked example; TD3 runs in the same framework
(Section 4.2.4, Fig. 8). The paper prints no update equations, so the steps below
follow the published algorithms:

  SAC  Haarnoja et al., "Soft Actor-Critic Algorithms and Applications", 2018:
       soft TD target with twin-Q minimum and target critics, reparameterised
       tanh-Gaussian policy with its change-of-variables log-density, learned
       temperature against a target entropy, Polyak-averaged target critics.
  TD3  Fujimoto et al., "Addressing Function Approximation Error in Actor-Critic
       Methods", 2018: clipped double-Q target, target policy smoothing,
       delayed actor and target updates.

Readings taken where the paper is silent (each is also stated where used):
  * Snapshot semantics: every loss of step t reads the parameters as they were at
    the start of step t (actor, critics, targets, temperature); all Adam and
    Polyak writes happen after both the critic and the actor gradients exist.
    This is the reading of "actor and critics updated independently".
  * Critic loss L_Q = mean_b (q1 - y)^2 + mean_b (q2 - y)^2 (no 1/2 factor).
  * log pi = sum_j [-eps_j^2/2 - logstd_j - ln(2 pi)/2 - 2(ln 2 - u_j - softplus(-2 u_j))],
    using eps directly; the clamp of log-std passes gradient on the closed interval.
  * min(q1, q2) routes its gradient to q1 on ties; ReLU'(0) = 0.
  * Temperature loss L_a = -log(alpha) * mean(log pi + H_target), alpha = exp(log alpha),
    and alpha enters the critic and actor losses as a constant.
  * Adam with bias correction, one step counter per optimizer; Polyak
    tbar <- (1 - tau) * tbar + tau * theta after Adam, every step (SAC) or on
    delayed steps only (TD3, together with the target actor).
  * TD3's delayed step fires when the global step k satisfies k % delay == 0.
  * Ordering "sequential" (hp["ordering"], default "snapshot"): the order of the
    published SAC and TD3 algorithms instead. The critics take their Adam step
    first and the actor loss of the same step is taken through the updated
    critics; the temperature loss still uses the step-start actor sample and
    alpha, and the target networks move after both updates as above.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, Optional

import numpy as np

from . import philox
from .bf16 import identity, round_bf16
from .nets import (NET_ACTOR, NET_CRITIC1, NET_CRITIC2, backward, count, flatten, forward,
                   init_net, layer_dims, unflatten)

LN2 = math.log(2.0)
HALF_LN_2PI = 0.5 * math.log(2.0 * math.pi)

# Loss record columns.
REC_LQ, REC_LPI, REC_LALPHA, REC_ALPHA, REC_LOGPI, REC_Q1, REC_NONFINITE, REC_ACTOR = range(8)


def softplus(x):
    return np.logaddexp(0.0, x)


def tanh_gaussian(z, eps, act_dim: int, lmin: float, lmax: float):
    """Reparameterised tanh-Gaussian sample and log-density from the actor head z.

    z = [mu | l]; lc = clip(l, lmin, lmax); sigma = exp(lc); u = mu + sigma * eps;
    a = tanh(u); log pi(a) = sum_j [N(eps_j; 0, 1) log-density - lc_j - log(1 - tanh^2 u_j)],
    with log(1 - tanh^2 u) written in the overflow-free form 2(ln 2 - u - softplus(-2u)).
    """
    mu, l = z[:, :act_dim], z[:, act_dim:2 * act_dim]
    lc = np.clip(l, lmin, lmax)
    sigma = np.exp(lc)
    u = mu + sigma * eps
    a = np.tanh(u)
    log1m_tanh2 = 2.0 * (LN2 - u - softplus(-2.0 * u))
    logp = np.sum(-0.5 * eps * eps - lc - HALF_LN_2PI - log1m_tanh2, axis=1)
    return dict(mu=mu, l=l, lc=lc, sigma=sigma, u=u, a=a, logp=logp)


class Adam:
    """Kingma & Ba Adam with bias correction; no weight decay, no clipping."""

    def __init__(self, lr: float, b1: float, b2: float, eps: float):
        self.lr, self.b1, self.b2, self.eps = lr, b1, b2, eps
        self.t = 0

    def step(self, params, grads, m, v):
        """params/grads/m/v: parallel lists of arrays; updated in place."""
        self.t += 1
        c1 = 1.0 - self.b1 ** self.t
        c2 = 1.0 - self.b2 ** self.t
        for p, g, mm, vv in zip(params, grads, m, v):
            mm *= self.b1
            mm += (1.0 - self.b1) * g
            vv *= self.b2
            vv += (1.0 - self.b2) * g * g
            p -= self.lr * (mm / c1) / (np.sqrt(vv / c2) + self.eps)


def polyak(targets, online, tau: float):
    """tbar <- (1 - tau) * tbar + tau * theta (tau = 1 copies exactly, tau = 0 keeps)."""
    for tb, th in zip(targets, online):
        tb *= (1.0 - tau)
        tb += tau * th


def _tensors(layers):
    return [x for wb in layers for x in wb]


class Oracle:
    """CPU reference of the update.

    Parameters mirror spz_create: obs_dim, act_dim, hidden widths, batch, a dict of
    hyper-parameters (keys of synth.Workload.hparams()) and the library seed.
    `row_source`, if given, replaces the stored replay ring by a callable
    idx -> (obs, act, rew, done, next_obs) for a ring filled in order from empty;
    call `set_virtual_size` to state how many rows it holds.
    """

    def __init__(self, obs_dim: int, act_dim: int, hidden, batch: int, hp: Dict, seed: int,
                 row_source: Optional[Callable] = None):
        self.O, self.A, self.hidden, self.B = obs_dim, act_dim, tuple(hidden), batch
        self.hp = dict(hp)
        self.seed = int(seed)
        self.algo = hp["algo"]
        self.sequential = hp.get("ordering", "snapshot") == "sequential"
        self.rnd = round_bf16 if hp["gemm_prec"] == "bf16" else identity
        self.dims_actor = layer_dims("actor", obs_dim, act_dim, hidden, self.algo)
        self.dims_critic = layer_dims("critic", obs_dim, act_dim, hidden, self.algo)
        self.net = {
            "actor": init_net(seed, NET_ACTOR, self.dims_actor),
            "critic1": init_net(seed, NET_CRITIC1, self.dims_critic),
            "critic2": init_net(seed, NET_CRITIC2, self.dims_critic),
        }
        self.net["tcritic1"] = [[w.copy(), b.copy()] for w, b in self.net["critic1"]]
        self.net["tcritic2"] = [[w.copy(), b.copy()] for w, b in self.net["critic2"]]
        if self.algo == "td3":
            self.net["tactor"] = [[w.copy(), b.copy()] for w, b in self.net["actor"]]
        self.log_alpha = np.array([math.log(hp["alpha_init"])]) if self.algo == "sac" else np.zeros(1)
        self.m = {k: [np.zeros_like(x) for x in _tensors(self.net[k])] for k in ("actor", "critic1", "critic2")}
        self.v = {k: [np.zeros_like(x) for x in _tensors(self.net[k])] for k in ("actor", "critic1", "critic2")}
        self.m["log_alpha"] = [np.zeros(1)]
        self.v["log_alpha"] = [np.zeros(1)]
        b1, b2, e = hp["beta1"], hp["beta2"], hp["eps"]
        self.opt_actor = Adam(hp["lr_actor"], b1, b2, e)
        self.opt_critic = Adam(hp["lr_critic"], b1, b2, e)
        self.opt_alpha = Adam(hp["lr_alpha"], b1, b2, e)
        self.t = 0
        self.records = []
        self.last_idx = None
        self.last_batch = None
        self.last_grads = None
        # optional callable(str), told when each part of a step is done (progress of
        # long steps in tests; no effect on the arithmetic)
        self.progress = None
        # Test hook for a floating-point decision of a discrete choice: when set to a
        # bool per batch row, the next SAC step's actor loss takes critic 1 on exactly
        # those rows instead of deciding qp1 <= qp2 itself (the values differ only by
        # accumulation order where two implementations disagree). The oracle's own
        # decision and both critic values stay in last_min_choice / last_qpi.
        self.forced_min_choice = None
        self.last_min_choice = None
        self.last_qpi = None
        # replay ring
        self.capacity = int(hp["capacity"])
        self.row_source = row_source
        self.ptr = 0
        self.size = 0
        if row_source is None:
            self.buf_obs = np.zeros((0, obs_dim), np.float32)
            self._alloc_ring()

    # ---------------------------------------------------------------- replay ring
    def _alloc_ring(self):
        n, O, A = self.capacity, self.O, self.A
        self.buf_obs = np.zeros((n, O), np.float32)
        self.buf_act = np.zeros((n, A), np.float32)
        self.buf_rew = np.zeros(n, np.float32)
        self.buf_done = np.zeros(n, np.float32)
        self.buf_nobs = np.zeros((n, O), np.float32)

    def push(self, obs, act, rew, done, next_obs):
        """FIFO ring: row i goes to slot (ptr + i) mod capacity; size saturates."""
        assert self.row_source is None
        n = len(rew)
        skip = max(0, n - self.capacity)       # rows overwritten within this same push
        slots = (self.ptr + np.arange(skip, n)) % self.capacity
        self.buf_obs[slots] = np.asarray(obs)[skip:]
        self.buf_act[slots] = np.asarray(act)[skip:]
        self.buf_rew[slots] = np.asarray(rew)[skip:]
        self.buf_done[slots] = np.asarray(done)[skip:]
        self.buf_nobs[slots] = np.asarray(next_obs)[skip:]
        self.ptr = (self.ptr + n) % self.capacity
        self.size = min(self.size + n, self.capacity)

    def set_virtual_size(self, size: int):
        assert self.row_source is not None and size <= self.capacity
        self.size = int(size)
        self.ptr = self.size % self.capacity

    def _gather(self, idx):
        if self.row_source is not None:
            o, a, r, d, n = self.row_source(idx)
        else:
            o, a, r, d, n = (self.buf_obs[idx], self.buf_act[idx], self.buf_rew[idx],
                             self.buf_done[idx], self.buf_nobs[idx])
        f = lambda x: np.asarray(x, dtype=np.float64)
        return f(o), f(a), f(r), f(d), f(n)

    # ---------------------------------------------------------------- parameters
    def dims(self, which: str):
        return self.dims_actor if "actor" in which else self.dims_critic

    def params(self, which: str) -> np.ndarray:
        if which == "log_alpha":
            return self.log_alpha.copy()
        if which.startswith("m_") or which.startswith("v_"):
            store = self.m if which[0] == "m" else self.v
            return np.concatenate([x.ravel() for x in store[which[2:]]])
        return flatten(self.net[which])

    def set_params(self, which: str, flat):
        flat = np.asarray(flat, dtype=np.float64)
        if which == "log_alpha":
            self.log_alpha[:] = flat
            return
        if which.startswith("m_") or which.startswith("v_"):
            store = self.m if which[0] == "m" else self.v
            o = 0
            for x in store[which[2:]]:
                x[...] = flat[o:o + x.size].reshape(x.shape)
                o += x.size
            return
        self.net[which] = unflatten(flat, self.dims(which))

    def param_count(self, which: str) -> int:
        if which == "log_alpha" or which in ("m_log_alpha", "v_log_alpha"):
            return 1
        key = which[2:] if which[:2] in ("m_", "v_") else which
        return count(self.dims(key))

    # ---------------------------------------------------------------- the step
    def act(self, obs, stochastic: bool, counter: int):
        """Actions of the current actor for sampler observations (the policy acting
        for the sampling processes, Section 3.1.1; deterministic for test and
        visualisation, Section 3.1.2). SAC: tanh(mu), or tanh(mu + sigma eps) with
        eps from purpose ACT at step word `counter`; TD3: tanh(z)."""
        hp = self.hp
        obs = np.asarray(obs, np.float64)
        n = obs.shape[0]
        z, _ = forward(self.net["actor"], obs, self.rnd)
        A = self.A
        if self.algo == "td3":
            if stochastic:
                raise ValueError("TD3 actions are deterministic")
            return np.tanh(z)
        mu = z[:, :A]
        if not stochastic:
            return np.tanh(mu)
        eps = philox.normals(self.seed, counter, philox.PURPOSE_ACT, n * A).reshape(n, A)
        lc = np.clip(z[:, A:2 * A], hp["log_std_min"], hp["log_std_max"])
        return np.tanh(mu + np.exp(lc) * eps)

    def set_batch(self, batch: int):
        """Batch size of the following steps; a row's index and noise depend only on
        (seed, step, row), so this equals a learner created with that batch."""
        if batch < 1:
            raise ValueError("batch must be >= 1")
        self.B = int(batch)

    def update(self, n_steps: int):
        if self.size == 0:
            raise RuntimeError("replay buffer is empty")
        for _ in range(n_steps):
            self.t += 1
            if self.algo == "sac":
                self._sac_step(self.t)
            else:
                self._td3_step(self.t)

    def _note(self, what: str):
        if self.progress is not None:
            self.progress(what)

    def _sample(self, t: int):
        B, A = self.B, self.A
        idx = philox.indices(self.seed, t, B, self.size)
        batch = self._gather(idx)
        self.last_idx = idx
        self.last_batch = batch
        eps_tgt = philox.normals(self.seed, t, philox.PURPOSE_NOISE_TGT, B * A).reshape(B, A)
        eps_pol = philox.normals(self.seed, t, philox.PURPOSE_NOISE_POL, B * A).reshape(B, A)
        return batch, eps_tgt, eps_pol

    def _critic_grads(self, s, a, y):
        """Online twin critics on (s, a) against the fixed target y."""
        B, rnd = self.B, self.rnd
        x = np.concatenate([s, a], axis=1)
        out = {}
        lq = 0.0
        for k in ("critic1", "critic2"):
            q, xs = forward(self.net[k], x, rnd)
            q = q[:, 0]
            lq += np.mean((q - y) ** 2)
            dq = (2.0 / B) * (q - y)
            grads, _ = backward(self.net[k], xs, dq[:, None], rnd)
            out[k] = grads
            out["q_" + k] = q
        return lq, out

    def _critic_action_grad(self, s, a_pi, dq_by_net):
        """dL/da for L = sum_i <dq_i, Q_i(s, a)> at the current critic parameters (held fixed)."""
        rnd = self.rnd
        x = np.concatenate([s, a_pi], axis=1)
        da = np.zeros_like(a_pi)
        for k, dq in dq_by_net.items():
            _, xs = forward(self.net[k], x, rnd)
            _, dx = backward(self.net[k], xs, dq[:, None], rnd, want_wgrad=False, want_dx=True)
            da += dx[:, self.O:]
        return da

    def sac_target(self, s2, r, d, eps_tgt, alpha):
        """Soft TD target with the target critics; next action from the current actor."""
        hp, rnd = self.hp, self.rnd
        z2, _ = forward(self.net["actor"], s2, rnd)
        pol2 = tanh_gaussian(z2, eps_tgt, self.A, hp["log_std_min"], hp["log_std_max"])
        x2 = np.concatenate([s2, pol2["a"]], axis=1)
        qt1 = forward(self.net["tcritic1"], x2, rnd)[0][:, 0]
        qt2 = forward(self.net["tcritic2"], x2, rnd)[0][:, 0]
        y = r + hp["gamma"] * (1.0 - d) * (np.minimum(qt1, qt2) - alpha * pol2["logp"])
        return y, pol2

    def sac_actor(self, s, eps_pol, alpha, take1=None):
        """Actor loss and gradient: reparameterised sample on s, twin-Q minimum at the
        current critics (step-start under snapshot ordering, updated under sequential).
        take1 (bool per row, optional) replaces the choice qp1 <= qp2 of the minimum.
        Returns (L_pi, actor grads, policy dict)."""
        hp, B, A, rnd = self.hp, self.B, self.A, self.rnd
        lmin, lmax = hp["log_std_min"], hp["log_std_max"]
        z, xs_a = forward(self.net["actor"], s, rnd)
        pol = tanh_gaussian(z, eps_pol, A, lmin, lmax)
        xa = np.concatenate([s, pol["a"]], axis=1)
        qp1 = forward(self.net["critic1"], xa, rnd)[0][:, 0]
        qp2 = forward(self.net["critic2"], xa, rnd)[0][:, 0]
        own = qp1 <= qp2
        self.last_min_choice, self.last_qpi = own, (qp1, qp2)
        take1 = own if take1 is None else np.asarray(take1, dtype=bool)
        lpi = float(np.mean(alpha * pol["logp"] - np.where(take1, qp1, qp2)))
        dq1 = np.where(take1, -1.0 / B, 0.0)
        dq2 = np.where(take1, 0.0, -1.0 / B)
        da = self._critic_action_grad(s, pol["a"], {"critic1": dq1, "critic2": dq2})
        # d log pi/du = 2 tanh u, du/dmu = 1, du/dlc = sigma*eps, and log pi has -lc directly.
        th = pol["a"]
        g_u = da * (1.0 - th * th) + (alpha / B) * 2.0 * th
        d_lc = g_u * pol["sigma"] * eps_pol - alpha / B
        d_l = d_lc * ((pol["l"] >= lmin) & (pol["l"] <= lmax))
        dz = np.concatenate([g_u, d_l], axis=1)
        ag, _ = backward(self.net["actor"], xs_a, dz, rnd)
        return lpi, ag, pol

    def td3_target(self, s2, r, d, eps_tgt):
        """Clipped double-Q target with target-policy smoothing from the target actor."""
        hp, rnd = self.hp, self.rnd
        z2, _ = forward(self.net["tactor"], s2, rnd)
        noise = np.clip(hp["policy_noise"] * eps_tgt, -hp["noise_clip"], hp["noise_clip"])
        a2 = np.clip(np.tanh(z2) + noise, -1.0, 1.0)
        x2 = np.concatenate([s2, a2], axis=1)
        qt1 = forward(self.net["tcritic1"], x2, rnd)[0][:, 0]
        qt2 = forward(self.net["tcritic2"], x2, rnd)[0][:, 0]
        return r + hp["gamma"] * (1.0 - d) * np.minimum(qt1, qt2), a2

    def td3_actor(self, s):
        """Deterministic policy gradient through Q1 at the current critic."""
        B, rnd = self.B, self.rnd
        z, xs_a = forward(self.net["actor"], s, rnd)
        ap = np.tanh(z)
        xa = np.concatenate([s, ap], axis=1)
        qp1 = forward(self.net["critic1"], xa, rnd)[0][:, 0]
        lpi = -float(np.mean(qp1))
        da = self._critic_action_grad(s, ap, {"critic1": np.full(B, -1.0 / B)})
        ag, _ = backward(self.net["actor"], xs_a, da * (1.0 - ap * ap), rnd)
        return lpi, ag

    def _step_critics(self, cg):
        self.opt_critic.step(_tensors(self.net["critic1"]) + _tensors(self.net["critic2"]),
                             _tensors(cg["critic1"]) + _tensors(cg["critic2"]),
                             self.m["critic1"] + self.m["critic2"], self.v["critic1"] + self.v["critic2"])

    def _sac_step(self, t: int):
        hp = self.hp
        (s, a, r, d, s2), eps_tgt, eps_pol = self._sample(t)
        log_alpha = float(self.log_alpha[0])
        alpha = math.exp(log_alpha)

        y, _ = self.sac_target(s2, r, d, eps_tgt, alpha)
        self._note("step %d: TD target" % t)
        lq, cg = self._critic_grads(s, a, y)
        self._note("step %d: critic gradients" % t)
        if self.sequential:
            self._step_critics(cg)
        forced, self.forced_min_choice = self.forced_min_choice, None
        lpi, ag, pol = self.sac_actor(s, eps_pol, alpha, take1=forced)
        self._note("step %d: actor gradient" % t)
        mean_lp_h = float(np.mean(pol["logp"] + hp["target_entropy"]))
        l_alpha = -log_alpha * mean_lp_h
        g_alpha = -mean_lp_h
        self.last_grads = {"actor": ag, "critic1": cg["critic1"], "critic2": cg["critic2"],
                           "log_alpha": g_alpha, "y": y, "logp": pol["logp"]}

        # Snapshot semantics: optimizer writes happen after both gradients exist.
        if not self.sequential:
            self._step_critics(cg)
        self.opt_actor.step(_tensors(self.net["actor"]), _tensors(ag), self.m["actor"], self.v["actor"])
        if hp["learn_alpha"]:
            self.opt_alpha.step([self.log_alpha], [np.array([g_alpha])], self.m["log_alpha"],
                                self.v["log_alpha"])
        for k in ("critic1", "critic2"):
            polyak(_tensors(self.net["t" + k]), _tensors(self.net[k]), hp["tau"])

        rec = np.zeros(8)
        rec[REC_LQ], rec[REC_LPI], rec[REC_LALPHA] = lq, lpi, l_alpha
        rec[REC_ALPHA], rec[REC_LOGPI] = alpha, float(np.mean(pol["logp"]))
        rec[REC_Q1] = float(np.mean(cg["q_critic1"]))
        rec[REC_NONFINITE] = float(not np.all(np.isfinite(rec[:6])))
        rec[REC_ACTOR] = 1.0
        self.records.append(rec)

    def _td3_step(self, k: int):
        hp = self.hp
        (s, a, r, d, s2), eps_tgt, _ = self._sample(k)
        y, _ = self.td3_target(s2, r, d, eps_tgt)
        lq, cg = self._critic_grads(s, a, y)
        actor_step = (k % hp["policy_delay"]) == 0
        if self.sequential:
            self._step_critics(cg)
        lpi, ag = self.td3_actor(s) if actor_step else (0.0, None)
        self.last_grads = {"actor": ag, "critic1": cg["critic1"], "critic2": cg["critic2"], "y": y}

        if not self.sequential:
            self._step_critics(cg)
        if actor_step:
            self.opt_actor.step(_tensors(self.net["actor"]), _tensors(ag), self.m["actor"], self.v["actor"])
            for key in ("critic1", "critic2", "actor"):
                polyak(_tensors(self.net["t" + key]), _tensors(self.net[key]), hp["tau"])

        rec = np.zeros(8)
        rec[REC_LQ], rec[REC_LPI] = lq, lpi
        rec[REC_Q1] = float(np.mean(cg["q_critic1"]))
        rec[REC_NONFINITE] = float(not np.all(np.isfinite(rec[:6])))
        rec[REC_ACTOR] = 1.0 if actor_step else 0.0
        self.records.append(rec)

    def losses(self) -> np.ndarray:
        return np.array(self.records).reshape(-1, 8)
