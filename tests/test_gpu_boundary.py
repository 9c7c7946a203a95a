"""GPU tests of the boundary calls against the oracle: the gathered batch, the
non-finite flag of the loss record, asynchronous ingestion interleaved with
updates (Section 3.3.2) and checkpoint resume (Section 3.3.1).

Bars as in test_gpu_parity: gathered rows bit-exact (bf16 workloads: the oracle's
rows rounded to bfloat16, the ring's storage type); fp32 losses within rel 1e-4
per step and parameters within per-tensor rel 1e-4 (Adam moments without
exclusions) after the whole sequence.
"""
import numpy as np
import pytest

import synth
from oracle import philox
from oracle.bf16 import round_bf16

from .helpers import NET_KEYS, log, make_gpu, make_oracle, make_pair, oracle_grad_flat, state_keys
from .test_gpu_parity import FP32_TOL, FUSED_BF16, RAGGED, RAGGED_TD3, check_losses, check_ten_step_params

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


# ---------------------------------------------------------------------------- gathered batch
def expected_batch(w, idx, data_seed=0):
    """The oracle's gathered rows (s, a, s', r, d) for replay rows idx, in the ring's
    storage precision (bf16 workloads keep s, a, s' as bfloat16)."""
    s, a, r, d, s2 = synth.workload_rows_at(w, idx, data_seed)
    cast = round_bf16 if w.prec == "bf16" else (lambda x: np.asarray(x, np.float64))
    return cast(s), cast(a), cast(s2), np.asarray(r, np.float64), np.asarray(d, np.float64)


@pytest.mark.parametrize("w,rows,n_streams", [
    (W["sac_small"], 10_000, 1), (W["sac_small"], 10_000, 2),
    (W["sac_large_bf16"].replace(capacity=1_000_000), 1_000_000, 1),
    (W["sac_large_bf16"].replace(batch=2560, capacity=50_000), 50_000, 2),
    (W["td3_ant"].replace(batch=4096, capacity=50_000), 50_000, 1)],
    ids=["sac_small_1stream", "sac_small_2streams", "sac_large_bf16_full_batch", "large_bf16_b2560_2streams",
         "td3_ant_b4096"])
def test_gathered_batch_bit_exact(w, rows, n_streams):
    """Every row the step gathered (s, a, s', r, d), as the update's kernels read it,
    equals the oracle's row of the sampled replay index bit for bit, over two steps."""
    log("gather %s rows %d streams %d" % (w.name, rows, n_streams))
    g = make_gpu(w, n_streams=n_streams)
    for r0 in range(0, rows, 1 << 18):
        g.buffer_push(*synth.workload_rows(w, r0, min(1 << 18, rows - r0), 0))
    for t in (1, 2):
        g.update(1)
        idx = philox.indices(1, t, w.batch, rows)
        assert np.array_equal(g.debug_indices(), idx.astype(np.int32))
        got = g.debug_batch()
        want = expected_batch(w, idx)
        for name, a, b in zip(("s", "a", "s'", "r", "d"), got, want):
            assert np.array_equal(a.astype(np.float64), b), (t, name, int(np.sum(a != b)))
    g.close()


# ---------------------------------------------------------------------------- non-finite values
@pytest.mark.parametrize("w", [RAGGED, FUSED_BF16], ids=["fp32", "bf16_fused"])
def test_nan_reward_sets_nonfinite_flag(w):
    """A NaN reward in a sampled transition makes the step's loss record non-finite:
    both the GPU and the oracle set SPZ_REC_NONFINITE and the update call succeeds."""
    log("nan reward %s" % w.name)
    rows = synth.workload_rows(w, 0, 5000, 0)
    idx = philox.indices(1, 1, w.batch, 5000)
    rows[2][idx[0]] = np.nan
    g = make_gpu(w)
    o = make_oracle(w)
    g.buffer_push(*rows)
    o.push(*rows)
    with np.errstate(invalid="ignore", over="ignore"):
        for _ in range(2):
            g.update(1)
            o.update(1)
    rec_g, rec_o = g.read_losses(1, 2), o.losses()
    g.close()
    assert np.all(rec_o[:, 6] == 1.0), rec_o
    assert np.all(rec_g[:, 6] == 1.0), rec_g
    assert np.isnan(rec_g[0, 0]) and np.isnan(rec_o[0, 0])


def test_nan_in_one_target_critic_propagates_to_td_target():
    """min(Q1', Q2') with one target critic NaN is NaN (no silent fallback to the other
    critic): the TD target and the critic loss are NaN on both sides and flagged."""
    w = RAGGED
    log("nan target critic")
    g, o = make_pair(w, 3000)
    bad = o.params("tcritic2")
    bad[-1] = np.nan                       # output bias of target critic 2
    o.set_params("tcritic2", bad)
    g.write_params("tcritic2", bad.astype(np.float32))
    with np.errstate(invalid="ignore"):
        g.update(1)
        o.update(1)
    y = g.debug_rows("td_target")
    rec_g, rec_o = g.read_losses(1, 1)[0], o.losses()[0]
    g.close()
    assert np.all(np.isnan(y))
    assert np.all(np.isnan(o.last_grads["y"]))
    assert rec_g[6] == 1.0 and rec_o[6] == 1.0
    assert np.isnan(rec_g[0]) and np.isnan(rec_o[0])


# ---------------------------------------------------------------------------- ingestion
@pytest.mark.parametrize("use_stream", [False, True], ids=["null_stream", "side_stream"])
def test_async_push_interleaved_with_updates_matches_oracle(use_stream):
    """Asynchronous pushes between updates (Section 3.3.2's experience pool fed while
    the learner runs), against the oracle fed the same pushes and updates in the same
    order: every step's losses and the parameters after 10 steps. The last push wraps
    the ring."""
    import torch
    w = RAGGED.replace(capacity=8000)
    log("async ingestion vs oracle (%s)" % ("side stream" if use_stream else "null stream"))
    rows = synth.workload_rows(w, 0, 14_000, 0)
    part = lambda a, b: [x[a:b] for x in rows]
    plan = [("push", 0, 3000), ("update", 2), ("push", 3000, 4500), ("update", 2), ("push", 4500, 5000),
            ("push", 5000, 5200), ("update", 3), ("push", 5200, 14_000), ("update", 3)]
    stream = torch.cuda.Stream() if use_stream else None
    g = make_gpu(w)
    o = make_oracle(w)
    p0 = {k: o.params(k) for k in NET_KEYS}
    hist = {k: [] for k in NET_KEYS}
    for op in plan:
        if op[0] == "push":
            g.buffer_push_async(*part(op[1], op[2]))
            o.push(*part(op[1], op[2]))
            assert g.buffer_size() == o.size
            continue
        g.update(op[1], stream)
        for _ in range(op[1]):
            o.update(1)
            for k in NET_KEYS:
                hist[k].append(oracle_grad_flat(o, k))
    g.synchronize()
    if stream is not None:
        stream.synchronize()
    assert np.array_equal(g.debug_indices(), o.last_idx.astype(np.int32))
    check_losses(g.read_losses(1, 10), o.losses(), FP32_TOL, "async")
    params = {k: (g.read_params(k), o.params(k)) for k in state_keys(w.algo)}
    params["p0"] = p0
    g.close()
    check_ten_step_params(w, params, o, hist, 10)


# ---------------------------------------------------------------------------- checkpoints
@pytest.mark.parametrize("w,ring", [(RAGGED, True), (RAGGED, False), (RAGGED_TD3, True)],
                         ids=["sac_with_ring", "sac_without_ring", "td3_with_ring"])
def test_checkpoint_resume_matches_uninterrupted_oracle(w, ring, tmp_path):
    """Save after 3 steps, load into a fresh context (another seed; without the ring in
    the file, the same rows pushed again), run 4 more steps: the 7 loss records and the
    final state match an oracle that ran 7 steps without interruption."""
    log("checkpoint vs oracle %s ring=%s" % (w.name, ring))
    rows = synth.workload_rows(w, 0, 5000, 0)
    path = str(tmp_path / "ckpt.spz")
    g = make_gpu(w)
    g.buffer_push(*rows)
    g.update(3)
    g.save(path, ring=ring)
    g.close()
    h = make_gpu(w, seed=99)
    if not ring:
        h.buffer_push(*rows)
    h.load(path)
    h.update(4)
    o = make_oracle(w)
    o.push(*rows)
    p0 = {k: o.params(k) for k in NET_KEYS}
    hist = {k: [] for k in NET_KEYS}
    for _ in range(7):
        o.update(1)
        for k in NET_KEYS:
            if o.last_grads[k] is not None:
                hist[k].append(oracle_grad_flat(o, k))
    assert h.step() == 7
    assert np.array_equal(h.debug_indices(), o.last_idx.astype(np.int32))
    check_losses(h.read_losses(1, 7), o.losses(), FP32_TOL, "resume")
    params = {k: (h.read_params(k), o.params(k)) for k in state_keys(w.algo)}
    params["p0"] = p0
    h.close()
    check_ten_step_params(w, params, o, hist, 7)
