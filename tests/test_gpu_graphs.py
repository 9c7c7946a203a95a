"""Update steps replayed from captured HIP graphs (spz_hparams.graphs) against the
same steps launched kernel by kernel: bit-identical parameters, targets, Adam moments,
loss records and replay indices after every update call.

Each graph is replayed many times with the program's own eager work (a torch product,
synchronizations, synchronous and asynchronous pushes, a batch-size change, parameter
reads) between the replays, and every replay is checked. The pushes change the ring's
fill level and the batch change the shapes, both kernel arguments fixed at capture,
so those calls also exercise re-capture.
"""
import numpy as np
import pytest

import synth

from .helpers import log, state_keys
from .test_gpu_parity import FUSED_BF16, FUSED_TD3_BF16, RAGGED, RAGGED_TD3, SEQ_SAC

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


def _make(w, graphs, n_streams):
    from paper_2312_06126_amd import Spz
    return Spz(w.obs_dim, w.act_dim, w.hidden, w.batch, dict(w.hparams(), graphs=graphs), 1, n_streams=n_streams)


def _state(g, w, first, n):
    st = {k: g.read_params(k) for k in state_keys(w.algo)}
    st["rec"] = g.read_losses(first, n)
    st["idx"] = g.debug_indices()
    return st


@pytest.mark.parametrize("w,n_streams", [
    (W["sac_small"], 1), (RAGGED, 1), (RAGGED, 2), (RAGGED_TD3, 1), (FUSED_BF16, 1), (FUSED_TD3_BF16, 2),
    (SEQ_SAC, 1)],
    ids=["sac_small", "ragged_sac_1stream", "ragged_sac_2streams", "ragged_td3", "fused_bf16_row_split",
         "fused_td3_bf16_2streams", "sequential_sac"])
def test_graph_replay_bit_exact(w, n_streams):
    import torch
    log("graphs %s streams %d" % (w.name, n_streams))
    w = w.replace(capacity=6000)
    rows = synth.workload_rows(w, 0, 6000, 0)
    part = lambda a, b: [x[a:b] for x in rows]
    small = max(1, w.batch // 3)
    plan = [("push", 0, 3000), ("update", 3), ("eager",), ("update", 5), ("update", 1), ("push_async", 3000, 3500),
            ("update", 4), ("eager",), ("batch", small), ("update", 3), ("batch", w.batch), ("update", 2),
            ("push", 3500, 6000), ("update", 6)]
    runs = [_make(w, 0, n_streams), _make(w, 1, n_streams)]
    x = torch.randn(512, 512, device="cuda")
    t = 0
    for op in plan:
        for g in runs:
            if op[0] == "push":
                g.buffer_push(*part(op[1], op[2]))
            elif op[0] == "push_async":
                g.buffer_push_async(*part(op[1], op[2]))
            elif op[0] == "batch":
                g.set_batch(op[1])
            elif op[0] == "eager":
                y = x @ x
                torch.cuda.synchronize()
                g.synchronize()
                assert torch.isfinite(y).all()
            else:
                g.update(op[1])
        if op[0] == "update":
            first = t + 1
            t += op[1]
            a, b = (_state(g, w, first, op[1]) for g in runs)
            for k in a:
                assert np.array_equal(a[k], b[k]), (op, k)
    assert runs[1].step() == t
    for g in runs:
        g.close()
