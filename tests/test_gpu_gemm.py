"""GPU unit tests of the matrix-product kernels through the test hook spzt_gemm.

The reference is a float64 CPU product of the same (already bf16-rounded, for
bf16) operands. Products of two bf16 values are exact in float32, so the kernel
differs from the reference only by float32 accumulation order: float32 outputs
agree to rel 1e-5 (norm) and bf16 outputs to one bf16 ulp per element.
Shapes cover the large-tile kernel (256-row tiles, 256/128-wide column tiles,
k-contiguous and transposing LDS reads), its ragged column remainder handled by
the generic kernel, the generic kernel alone, and split-K weight gradients.
"""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = pytest.importorskip("torch")
    from paper_2312_06126_amd import spz
    lib = spz.load()
    f = lib.spzt_gemm
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    f.argtypes = [I32, I32, I32, I32, I32, I32, P, I64, P, I64, P, I64, P, P, I64, I32, I32]
    f.restype = ctypes.c_int
    return torch, f


def to_dev(torch, a, bf16):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).cuda() if bf16 else t.cuda()


def rounded(torch, a, bf16):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return (t.to(torch.bfloat16) if bf16 else t).to(torch.float64).numpy()


def run(env, bf16, mode, M, N, K, splits=1, relu=0, out_f32=0, use_bias=False, use_mask=False, seed=0):
    torch, f = env
    rng = np.random.default_rng(seed)
    if mode == 2:
        A = rng.standard_normal((K, M)).astype(np.float32)
    else:
        A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((N, K) if mode == 0 else (K, N)).astype(np.float32)
    bias = rng.standard_normal(N).astype(np.float32) if use_bias else None
    mask = (rng.standard_normal((M, N)) * (rng.uniform(size=(M, N)) < 0.5)).astype(np.float32) if use_mask else None
    dA, dB = to_dev(torch, A, bf16), to_dev(torch, B, bf16)
    dbias = torch.from_numpy(bias).cuda() if use_bias else None
    dmask = to_dev(torch, mask, bf16) if use_mask else None
    f32_out = out_f32 or mode == 2 or not bf16
    dC = torch.zeros((M, N), dtype=torch.float32 if f32_out else torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    rc = f(1 if bf16 else 0, mode, M, N, K, splits, dA.data_ptr(), dA.shape[1], dB.data_ptr(), dB.shape[1],
           dC.data_ptr(), N, dbias.data_ptr() if use_bias else None, dmask.data_ptr() if use_mask else None,
           N, relu, out_f32)
    assert rc == 0, rc
    got = dC.to(torch.float64).cpu().numpy()
    Ar, Br = rounded(torch, A, bf16), rounded(torch, B, bf16)
    if mode == 0:
        ref = Ar @ Br.T
        if use_bias:
            ref = ref + bias
        if relu:
            ref = np.maximum(ref, 0.0)
    elif mode == 1:
        ref = Ar @ Br
        if use_mask:
            ref = ref * (rounded(torch, mask, bf16) > 0)
    else:
        ref = Ar.T @ Br
    if f32_out:
        err = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert err < 1e-5, err
    else:
        ref_b = rounded(torch, ref, True)
        ulp = np.abs(ref_b) * 2.0 ** -7 + 1e-30
        bad = np.abs(got - ref_b) > ulp * 1.01
        assert bad.mean() < 1e-3 and np.all(np.abs(got - ref_b) <= 2 * ulp + 1e-6), bad.mean()
    return got


@pytest.mark.parametrize("M,N,K", [(512, 512, 96), (256, 1024, 1024), (512, 384, 64), (512, 416, 416)])
@pytest.mark.parametrize("variant", ["relu_bf16", "plain_f32", "bias_bf16"])
def test_forward_bf16(env, M, N, K, variant):
    run(env, True, 0, M, N, K, relu=variant == "relu_bf16", out_f32=variant == "plain_f32",
        use_bias=variant != "plain_f32")


@pytest.mark.parametrize("M,N,K", [(512, 512, 64), (256, 1024, 1024), (512, 416, 96), (256, 32, 1024)])
@pytest.mark.parametrize("masked", [True, False])
def test_dgrad_bf16(env, M, N, K, masked):
    run(env, True, 1, M, N, K, use_mask=masked, out_f32=not masked)


@pytest.mark.parametrize("M,N,K,splits", [(256, 256, 512, 1), (512, 1024, 2048, 4), (1024, 416, 1024, 2),
                                          (1024, 384, 512, 2), (64, 1024, 1024, 4), (256, 128, 256, 1)])
def test_wgrad_bf16(env, M, N, K, splits):
    run(env, True, 2, M, N, K, splits=splits)


@pytest.mark.parametrize("mode,M,N,K,splits", [(0, 256, 416, 96, 1), (1, 256, 320, 416, 1), (2, 416, 96, 512, 2),
                                               (0, 128, 32, 32, 1), (2, 32, 64, 256, 1)])
def test_fp32_generic(env, mode, M, N, K, splits):
    run(env, False, mode, M, N, K, splits=splits, relu=mode == 0, use_bias=mode == 0, use_mask=mode == 1)


def test_rejects_bad_shapes(env):
    torch, f = env
    d = torch.zeros(1024, device="cuda")
    assert f(1, 0, 100, 64, 64, 1, d.data_ptr(), 64, d.data_ptr(), 64, d.data_ptr(), 64, None, None, 0, 0, 1) != 0
