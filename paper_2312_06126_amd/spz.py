"""ctypes binding of libspz.so (include/spz.h): argument marshalling only.

Every step of the update runs in the HIP library. If the library is missing the
import of this module fails; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspz.so")

SPZ_OK, SPZ_EINVAL, SPZ_ENOMEM, SPZ_EEMPTY, SPZ_ESIZE, SPZ_EHIP, SPZ_EIO = 0, -1, -2, -3, -4, -5, -6
ALGOS = {"sac": 0, "td3": 1}
PRECS = {"fp32": 0, "bf16": 1}
ORDERINGS = {"snapshot": 0, "sequential": 1}
SELECTORS = {
    "actor": 0, "critic1": 1, "critic2": 2, "tcritic1": 3, "tcritic2": 4, "tactor": 5, "log_alpha": 6,
    "m_actor": 7, "m_critic1": 8, "m_critic2": 9, "m_log_alpha": 10,
    "v_actor": 11, "v_critic1": 12, "v_critic2": 13, "v_log_alpha": 14,
    "g_actor": 15, "g_critic1": 16, "g_critic2": 17, "g_log_alpha": 18,
}
DBG_INDICES = 0
DBG_BATCH = 6
# Per-row values of the last step: selector -> rows of the array (None: act_dim columns).
DEBUG_ROWS = {"td_target": (1, 1), "q": (2, 2), "qpi": (3, 2), "logpi": (4, 1), "daction": (5, None)}
REC_WIDTH = 8
EXPORTS = ["spz_hparams_default", "spz_create", "spz_destroy", "spz_buffer_push", "spz_buffer_size",
           "spz_update", "spz_synchronize", "spz_step", "spz_set_step", "spz_param_count",
           "spz_read_params", "spz_write_params", "spz_read_losses", "spz_debug_read", "spz_last_error",
           "spz_profile_enable", "spz_profile_only", "spz_profile_stride", "spz_profile_read", "spz_set_batch", "spz_batch", "spz_autotune_batch",
           "spz_save", "spz_load", "spz_act", "spz_buffer_push_async", "spz_act_noalloc"]


class SpzError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("spz error %d: %s" % (code, msg))
        self.code = code


class Hparams(ctypes.Structure):
    _fields_ = [("algo", ctypes.c_int32), ("gemm_prec", ctypes.c_int32), ("capacity", ctypes.c_int64),
                ("gamma", ctypes.c_float), ("tau", ctypes.c_float), ("lr_actor", ctypes.c_float),
                ("lr_critic", ctypes.c_float), ("lr_alpha", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float), ("alpha_init", ctypes.c_float),
                ("learn_alpha", ctypes.c_int32), ("target_entropy", ctypes.c_float),
                ("log_std_min", ctypes.c_float), ("log_std_max", ctypes.c_float),
                ("policy_noise", ctypes.c_float), ("noise_clip", ctypes.c_float),
                ("policy_delay", ctypes.c_int32), ("device", ctypes.c_int32), ("n_streams", ctypes.c_int32),
                ("ordering", ctypes.c_int32), ("actor_row_split", ctypes.c_int32), ("graphs", ctypes.c_int32)]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("M", ctypes.c_int32), ("N", ctypes.c_int32),
                ("K", ctypes.c_int32), ("bf16", ctypes.c_int32), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libspz.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError("libspz.so not built (run paper_2312_06126_amd/build.py or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    P, fp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_float)
    sig = {
        "spz_hparams_default": (None, [ctypes.POINTER(Hparams)]),
        "spz_create": (P, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                           ctypes.c_int32, ctypes.POINTER(Hparams), ctypes.c_uint64]),
        "spz_destroy": (None, [P]),
        "spz_buffer_push": (ctypes.c_int, [P, fp, fp, fp, fp, fp, ctypes.c_int64]),
        "spz_buffer_size": (ctypes.c_int64, [P]),
        "spz_buffer_push_async": (ctypes.c_int, [P, fp, fp, fp, fp, fp, ctypes.c_int64]),
        "spz_update": (ctypes.c_int, [P, ctypes.c_int32, P]),
        "spz_synchronize": (ctypes.c_int, [P]),
        "spz_set_batch": (ctypes.c_int, [P, ctypes.c_int32]),
        "spz_save": (ctypes.c_int, [P, ctypes.c_char_p, ctypes.c_int32]),
        "spz_act": (ctypes.c_int, [P, fp, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, fp]),
        "spz_act_noalloc": (ctypes.c_int, [P, P, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, P, P]),
        "spz_load": (ctypes.c_int, [P, ctypes.c_char_p]),
        "spz_batch": (ctypes.c_int32, [P]),
        "spz_autotune_batch": (ctypes.c_int, [P, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, P,
                                              ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                              ctypes.POINTER(ctypes.c_float), ctypes.c_int32,
                                              ctypes.POINTER(ctypes.c_int32)]),
        "spz_step": (ctypes.c_int64, [P]),
        "spz_set_step": (ctypes.c_int, [P, ctypes.c_int64]),
        "spz_param_count": (ctypes.c_int64, [P, ctypes.c_int32]),
        "spz_read_params": (ctypes.c_int, [P, ctypes.c_int32, fp, ctypes.c_int64]),
        "spz_write_params": (ctypes.c_int, [P, ctypes.c_int32, fp, ctypes.c_int64]),
        "spz_read_losses": (ctypes.c_int, [P, fp, ctypes.c_int64, ctypes.c_int32]),
        "spz_debug_read": (ctypes.c_int, [P, ctypes.c_int32, P, ctypes.c_int64]),
        "spz_last_error": (ctypes.c_char_p, [P]),
        "spz_profile_enable": (ctypes.c_int, [P, ctypes.c_int32, ctypes.c_int64]),
        "spz_profile_only": (ctypes.c_int, [P, ctypes.c_char_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
        "spz_profile_stride": (ctypes.c_int, [P, ctypes.c_int32]),
        "spz_profile_read": (ctypes.c_int, [P, ctypes.POINTER(KernelStat), ctypes.c_int32,
                                            ctypes.POINTER(ctypes.c_int32)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def default_hparams() -> Hparams:
    hp = Hparams()
    load().spz_hparams_default(ctypes.byref(hp))
    return hp


def make_hparams(d: dict, device: int = 0, n_streams: int = 2) -> Hparams:
    hp = default_hparams()
    for k, v in d.items():
        if k == "algo":
            v = ALGOS[v]
        elif k == "gemm_prec":
            v = PRECS[v]
        elif k in ("learn_alpha", "actor_row_split", "graphs"):
            v = int(bool(v))
        elif k == "ordering":
            v = ORDERINGS[v]
        setattr(hp, k, v)
    hp.device = device
    hp.n_streams = n_streams
    return hp


def _fptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _stream_handle(stream) -> Optional[int]:
    if stream is None or isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)   # torch.cuda.Stream


class Spz:
    """One learner context (spz_create ... spz_destroy)."""

    def __init__(self, obs_dim: int, act_dim: int, hidden, batch: int, hp: dict, seed: int,
                 device: int = 0, n_streams: int = 2):
        self.lib = load()
        self.obs_dim, self.act_dim, self.batch = obs_dim, act_dim, batch
        h = (ctypes.c_int32 * len(hidden))(*hidden)
        self.hp = make_hparams(hp, device, n_streams)
        self.ctx = self.lib.spz_create(obs_dim, act_dim, h, len(hidden), batch, ctypes.byref(self.hp), seed)
        if not self.ctx:
            raise SpzError(SPZ_EINVAL, self.lib.spz_last_error(None).decode())

    def _check(self, rc: int):
        if rc != SPZ_OK:
            raise SpzError(rc, self.lib.spz_last_error(self.ctx).decode())

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.spz_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- calls with the C names ------------------------------------------------------
    def buffer_push(self, obs, act, rew, done, next_obs):
        arrs = [np.ascontiguousarray(x, dtype=np.float32) for x in (obs, act, rew, done, next_obs)]
        n = arrs[2].shape[0]
        assert arrs[0].shape == (n, self.obs_dim) and arrs[4].shape == (n, self.obs_dim)
        assert arrs[1].shape == (n, self.act_dim) and arrs[3].shape == (n,)
        self._check(self.lib.spz_buffer_push(self.ctx, *map(_fptr, arrs), n))

    def buffer_push_async(self, obs, act, rew, done, next_obs):
        arrs = [np.ascontiguousarray(x, dtype=np.float32) for x in (obs, act, rew, done, next_obs)]
        n = arrs[2].shape[0]
        assert arrs[0].shape == (n, self.obs_dim) and arrs[4].shape == (n, self.obs_dim)
        assert arrs[1].shape == (n, self.act_dim) and arrs[3].shape == (n,)
        self._check(self.lib.spz_buffer_push_async(self.ctx, *map(_fptr, arrs), n))

    def buffer_size(self) -> int:
        return int(self.lib.spz_buffer_size(self.ctx))

    def update(self, n_steps: int, stream=None):
        self._check(self.lib.spz_update(self.ctx, int(n_steps), _stream_handle(stream)))

    def synchronize(self):
        self._check(self.lib.spz_synchronize(self.ctx))

    def act(self, obs, stochastic: bool = False, counter: int = 0) -> np.ndarray:
        """Actions of the current policy for sampler observations [n, obs_dim]."""
        obs = np.ascontiguousarray(obs, dtype=np.float32)
        n = obs.shape[0]
        assert obs.shape == (n, self.obs_dim)
        out = np.empty((n, self.act_dim), np.float32)
        self._check(self.lib.spz_act(self.ctx, _fptr(obs), n, 1 if stochastic else 0, int(counter) & 0xFFFFFFFF,
                                     _fptr(out)))
        return out

    def act_noalloc(self, obs_ptr: int, n: int, act_ptr: int, stochastic: bool = False, counter: int = 0,
                    stream=None):
        """spz_act_noalloc on device buffers (addresses, e.g. torch tensors' data_ptr()):
        obs float32 [n, obs_dim] in, act float32 [n, act_dim] out; asynchronous on stream."""
        self._check(self.lib.spz_act_noalloc(self.ctx, obs_ptr, int(n), 1 if stochastic else 0,
                                             int(counter) & 0xFFFFFFFF, act_ptr, _stream_handle(stream)))

    def save(self, path: str, ring: bool = True):
        """Whole learner state to a file (with the replay ring unless ring=False)."""
        self._check(self.lib.spz_save(self.ctx, os.fsencode(path), 1 if ring else 0))

    def load(self, path: str):
        self._check(self.lib.spz_load(self.ctx, os.fsencode(path)))

    def set_batch(self, batch: int):
        self._check(self.lib.spz_set_batch(self.ctx, int(batch)))
        self.batch = int(self.lib.spz_batch(self.ctx))

    def autotune_batch(self, b_min: int, probe_steps: int, tolerance: float = 0.05, stream=None, max_probes: int = 32):
        """Adaptive batch size; returns (chosen, [(batch, frames/s), ...])."""
        chosen = ctypes.c_int32(0)
        n = ctypes.c_int32(0)
        bs = (ctypes.c_int32 * max_probes)()
        fr = (ctypes.c_float * max_probes)()
        self._check(self.lib.spz_autotune_batch(self.ctx, b_min, probe_steps, tolerance, _stream_handle(stream),
                                                ctypes.byref(chosen), bs, fr, max_probes, ctypes.byref(n)))
        self.batch = int(self.lib.spz_batch(self.ctx))
        return int(chosen.value), [(int(bs[i]), float(fr[i])) for i in range(min(n.value, max_probes))]

    def step(self) -> int:
        return int(self.lib.spz_step(self.ctx))

    def set_step(self, step: int):
        self._check(self.lib.spz_set_step(self.ctx, int(step)))

    def param_count(self, which: str) -> int:
        n = int(self.lib.spz_param_count(self.ctx, SELECTORS[which]))
        if n < 0:
            raise SpzError(n, "bad selector %s" % which)
        return n

    def read_params(self, which: str) -> np.ndarray:
        out = np.empty(self.param_count(which), np.float32)
        self._check(self.lib.spz_read_params(self.ctx, SELECTORS[which], _fptr(out), out.size))
        return out

    def write_params(self, which: str, values):
        a = np.ascontiguousarray(values, dtype=np.float32)
        self._check(self.lib.spz_write_params(self.ctx, SELECTORS[which], _fptr(a), a.size))

    def read_losses(self, first_step: int, n: int) -> np.ndarray:
        out = np.empty((n, REC_WIDTH), np.float32)
        self._check(self.lib.spz_read_losses(self.ctx, _fptr(out), int(first_step), int(n)))
        return out

    def debug_indices(self) -> np.ndarray:
        out = np.empty(self.batch, np.int32)
        self._check(self.lib.spz_debug_read(self.ctx, DBG_INDICES, out.ctypes.data_as(ctypes.c_void_p),
                                            out.nbytes))
        return out

    def debug_batch(self):
        """The last step's gathered transitions as (s, a, s', r, d) float32 arrays."""
        O, A = self.obs_dim, self.act_dim
        out = np.empty((self.batch, 2 * O + A + 2), np.float32)
        self._check(self.lib.spz_debug_read(self.ctx, DBG_BATCH, out.ctypes.data_as(ctypes.c_void_p), out.nbytes))
        return out[:, :O], out[:, O:O + A], out[:, O + A:2 * O + A], out[:, -2], out[:, -1]

    def debug_rows(self, what: str) -> np.ndarray:
        """Per-row float32 values of the last step: "td_target" [batch], "q" and "qpi"
        [2, batch], "logpi" [batch], "daction" [batch, act_dim]."""
        sel, n = DEBUG_ROWS[what]
        out = np.empty((self.batch, self.act_dim) if n is None else (n, self.batch), np.float32)
        self._check(self.lib.spz_debug_read(self.ctx, sel, out.ctypes.data_as(ctypes.c_void_p), out.nbytes))
        return out[0] if n == 1 else out

    def profile_enable(self, on: bool = True, reserve_launches: int = 0):
        self._check(self.lib.spz_profile_enable(self.ctx, 1 if on else 0, int(reserve_launches)))

    def profile_only(self, name=None, M: int = 0, N: int = 0, K: int = 0):
        """Time only launches of kernel family `name` with shape (M, N, K); None: all."""
        self._check(self.lib.spz_profile_only(self.ctx, name.encode() if name else None, int(M), int(N), int(K)))

    def profile_stride(self, stride: int):
        """Time launches only in update steps whose number is a multiple of stride."""
        self._check(self.lib.spz_profile_stride(self.ctx, int(stride)))

    def profile_read(self, max_entries: int = 256):
        """Aggregated kernel timings: list of dicts sorted by total time (largest first)."""
        arr = (KernelStat * max_entries)()
        n = ctypes.c_int32(0)
        self._check(self.lib.spz_profile_read(self.ctx, arr, max_entries, ctypes.byref(n)))
        out = []
        for k in arr[:min(n.value, max_entries)]:
            out.append(dict(name=k.name.decode(), M=k.M, N=k.N, K=k.K, bf16=k.bf16, launches=k.launches,
                            total_ms=k.total_ms, flops=k.flops, bytes=k.bytes,
                            avg_ms=k.total_ms / max(k.launches, 1)))
        return out
