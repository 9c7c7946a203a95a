"""The five update workloads: network shapes, batch, buffer size, data recipe and
hyper-parameters.

The paper fixes neither network sizes nor algorithm constants (it cites SAC and
TD3 by reference, Section 3.2.2 and Section 4.2.4); these values are the workload
definitions this implementation is measured on. Hyper-parameters follow the
published SAC / TD3 defaults (discount 0.99, Polyak 0.005, Adam 3e-4 with
betas 0.9/0.999, eps 1e-8, log-std clamp [-20, 2], TD3 smoothing noise 0.2
clipped to 0.5 and policy delay 2).
"""
from __future__ import annotations

import dataclasses
from typing import Tuple


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    algo: str                 # "sac" | "td3"
    obs_dim: int
    act_dim: int
    hidden: Tuple[int, ...]
    batch: int
    capacity: int
    prec: str                 # GEMM operand precision: "fp32" | "bf16"
    steps: int
    learn_alpha: bool = True
    alpha_init: float = 1.0
    target_entropy: float = 0.0
    zero_mod: int = 0         # obs column j is exactly 0 when j % zero_mod == 0 (0: none)
    p_done: float = 0.01
    gamma: float = 0.99
    tau: float = 0.005
    lr_actor: float = 3e-4
    lr_critic: float = 3e-4
    lr_alpha: float = 3e-4
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    log_std_min: float = -20.0
    log_std_max: float = 2.0
    policy_noise: float = 0.2
    noise_clip: float = 0.5
    policy_delay: int = 2
    ordering: str = "snapshot"  # "snapshot" | "sequential" (update order within a step)

    def hparams(self) -> dict:
        """Hyper-parameters as a plain dict (the key names of the C struct spz_hparams)."""
        return dict(algo=self.algo, gemm_prec=self.prec, capacity=self.capacity, gamma=self.gamma,
                    tau=self.tau, lr_actor=self.lr_actor, lr_critic=self.lr_critic,
                    lr_alpha=self.lr_alpha, beta1=self.beta1, beta2=self.beta2, eps=self.eps,
                    alpha_init=self.alpha_init, learn_alpha=self.learn_alpha,
                    target_entropy=self.target_entropy, log_std_min=self.log_std_min,
                    log_std_max=self.log_std_max, policy_noise=self.policy_noise,
                    noise_clip=self.noise_clip, policy_delay=self.policy_delay, ordering=self.ordering)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # Small SAC case: 8-d observations, 2-d actions, 2x64 ReLU, fixed temperature 0.2.
    "sac_small": Workload("sac_small", "sac", 8, 2, (64, 64), 256, 10_000, "fp32", 10,
                          learn_alpha=False, alpha_init=0.2, target_entropy=-2.0),
    # Walker2D-shaped SAC (17-d obs, 6-d actions), 2x256, batch 8192, learned temperature.
    "sac_walker": Workload("sac_walker", "sac", 17, 6, (256, 256), 8192, 1_000_000, "fp32", 1000,
                           target_entropy=-6.0),
    # Humanoid-shaped SAC (376-d obs, 17-d actions), 2x256, batch 16384, bf16 GEMM operands.
    "sac_humanoid_bf16": Workload("sac_humanoid_bf16", "sac", 376, 17, (256, 256), 16384, 1_000_000,
                                  "bf16", 1000, target_entropy=-17.0, zero_mod=10),
    # Ant-shaped TD3 (111-d obs, 8-d actions), 400->300, batch 32768.
    "td3_ant": Workload("td3_ant", "td3", 111, 8, (400, 300), 32768, 2_000_000, "fp32", 1000,
                        learn_alpha=False, alpha_init=0.0),
    # Large-batch SAC stress case: 3x1024, batch 131072, 4M-row buffer, bf16 GEMM operands.
    "sac_large_bf16": Workload("sac_large_bf16", "sac", 376, 17, (1024, 1024, 1024), 131072,
                               4_000_000, "bf16", 500, target_entropy=-17.0, zero_mod=10),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
