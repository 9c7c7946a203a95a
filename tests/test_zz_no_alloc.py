"""The allocation-free sampler-action call (spz_act_noalloc) against spz_act.

spz_act_noalloc keeps its intermediate values in the library's per-GPU scratch array
instead of the context's buffers and takes device pointers; it runs the same kernels,
so its actions must equal spz_act's bit for bit. Two calls in a row, the second with
fewer rows (the scratch keeps the first call's contents), for fp32 and bf16 actors
(the bf16 one at the large network's widths, near the scratch limit), SAC mean and
sampled actions and TD3; plus the size limit and argument errors.
"""
import numpy as np
import pytest

import synth

from .helpers import log, make_gpu
from .test_gpu_parity import FUSED_BF16, RAGGED, RAGGED_TD3

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS


@pytest.mark.parametrize("w,n_first,n_second", [
    (RAGGED, 2000, 37), (FUSED_BF16, 1500, 256), (RAGGED_TD3, 900, 1),
    (W["sac_large_bf16"].replace(batch=4096, capacity=20_000), 12_800, 513)],
    ids=["sac_fp32", "sac_bf16_fused", "td3_fp32", "sac_large_widths"])
def test_act_noalloc_equals_act(w, n_first, n_second):
    import torch
    from paper_2312_06126_amd.spz import SPZ_EINVAL, SpzError
    log("act_noalloc %s: %d then %d rows" % (w.name, n_first, n_second))
    g = make_gpu(w)
    g.buffer_push(*synth.workload_rows(w, 0, min(w.capacity, 20_000), 0))
    g.update(2)
    g.synchronize()
    stream = torch.cuda.current_stream()
    modes = (False, True) if w.algo == "sac" else (False,)
    for n in (n_first, n_second):
        obs = synth.workload_rows(w, 50_000, n, 3)[0]
        obs_d = torch.from_numpy(obs).cuda()
        for stochastic in modes:
            out_d = torch.full((n, w.act_dim), float("nan"), dtype=torch.float32, device="cuda")
            g.act_noalloc(obs_d.data_ptr(), n, out_d.data_ptr(), stochastic=stochastic, counter=11, stream=stream)
            torch.cuda.synchronize()
            got = out_d.cpu().numpy()
            ref = g.act(obs, stochastic=stochastic, counter=11)
            assert np.array_equal(got, ref), (n, stochastic, np.abs(got - ref).max())
    with pytest.raises(SpzError) as e:
        g.act_noalloc(obs_d.data_ptr(), 10 ** 8, out_d.data_ptr())
    assert e.value.code == SPZ_EINVAL and "exceed" in str(e.value)
    with pytest.raises(SpzError) as e:
        g.act_noalloc(0, 5, out_d.data_ptr())
    assert e.value.code == SPZ_EINVAL
    g.act_noalloc(0, 0, 0)
    if w.algo == "td3":
        with pytest.raises(SpzError):
            g.act_noalloc(obs_d.data_ptr(), 1, out_d.data_ptr(), stochastic=True)
    g.close()
