"""GPU unit tests of the matrix-product kernels through the test hook spzt_gemm.

The reference is a float64 CPU product of the same (already bf16-rounded, for
bf16) operands. Products of two bf16 values are exact in float32, so the kernel
differs from the reference only by float32 accumulation order: float32 outputs
agree to rel 1e-5 (norm) and bf16 outputs to one bf16 ulp per element.
Shapes cover the large-tile kernel (256-row tiles, 256/128-wide column tiles,
k-contiguous and transposing LDS reads, ragged last column tiles for any
N % 8 == 0), the generic kernel alone, and split-K weight gradients.
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
    elif mode in (1, 3):
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


@pytest.mark.parametrize("M,N,K", [(512, 512, 96), (256, 1024, 1024), (512, 384, 64), (512, 416, 416),
                                   (512, 64, 1024), (256, 200, 96), (512, 136, 64)])
@pytest.mark.parametrize("variant", ["relu_bf16", "plain_f32", "bias_bf16"])
def test_forward_bf16(env, M, N, K, variant):
    run(env, True, 0, M, N, K, relu=variant == "relu_bf16", out_f32=variant == "plain_f32",
        use_bias=variant != "plain_f32")


@pytest.mark.parametrize("M,N,K", [(512, 512, 64), (256, 1024, 1024), (512, 416, 96), (256, 32, 1024),
                                   (512, 280, 64)])
@pytest.mark.parametrize("masked", [True, False])
def test_dgrad_bf16(env, M, N, K, masked):
    run(env, True, 1, M, N, K, use_mask=masked, out_f32=not masked)


@pytest.mark.parametrize("M,N,K,splits", [(256, 256, 512, 1), (512, 1024, 2048, 4), (1024, 416, 1024, 2),
                                          (1024, 384, 512, 2), (64, 1024, 1024, 4), (256, 128, 256, 1),
                                          (256, 160, 512, 2), (512, 264, 256, 1),
                                          # many slices of a small output: grouped slice reduction
                                          (64, 1024, 8192, 32), (128, 96, 5120, 40)])
def test_wgrad_bf16(env, M, N, K, splits):
    run(env, True, 2, M, N, K, splits=splits)


# Ragged last tiles (the widest tile wasting at most 10%): N = 416 and 352 take 64- and
# 128-wide tiles past the last column, M = 416 / 320 weight-gradient row tiles likewise.
@pytest.mark.parametrize("mode,M,N,K,splits", [(0, 256, 416, 96, 1), (1, 256, 320, 416, 1), (2, 416, 96, 512, 2),
                                               (0, 128, 32, 32, 1), (2, 32, 64, 256, 1),
                                               (1, 1024, 416, 320, 1), (0, 1024, 416, 160, 1), (1, 512, 352, 96, 1),
                                               (2, 416, 160, 2048, 4), (2, 320, 416, 4096, 8), (0, 32768, 416, 160, 1)])
def test_fp32_generic(env, mode, M, N, K, splits):
    run(env, False, mode, M, N, K, splits=splits, relu=mode == 0, use_bias=mode == 0, use_mask=mode == 1)


# bf16 shapes the large-tile kernel refuses (M % 256, N < 128): the generic kernel
# with the transposed image.
@pytest.mark.parametrize("M,N,K", [(128, 416, 96), (384, 64, 256), (128, 1024, 64)])
def test_bf16_dgrad_transposed_generic(env, M, N, K):
    run(env, True, 3, M, N, K, use_mask=True)


def test_rejects_bad_shapes(env):
    torch, f = env
    d = torch.zeros(1024, device="cuda")
    assert f(1, 0, 100, 64, 64, 1, d.data_ptr(), 64, d.data_ptr(), 64, d.data_ptr(), 64, None, None, 0, 0, 1) != 0


# ----------------------------------------------------------------------------- fused epilogues
@pytest.fixture(scope="module")
def fused(env):
    torch, _ = env
    from paper_2312_06126_amd import spz
    lib = spz.load()
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    f = lib.spzt_gemm_fused
    f.argtypes = [I32, I32, I32, I32, P, I64, P, I64, P, I64, P, P, P, I64, P, P, I64, I32, P, I64]
    f.restype = ctypes.c_int
    lib.spzt_rdot_cols.argtypes = [I32, I32]
    lib.spzt_rdot_cols.restype = ctypes.c_int
    return torch, f, lib.spzt_rdot_cols


def unpack_bits(words, M, N):
    """words [N/32, M] uint32 -> bool [M, N]: bit c % 32 of word (c / 32, r)."""
    w = words.astype(np.uint64)
    cols = [((w[c // 32] >> np.uint64(c % 32)) & np.uint64(1)).astype(bool) for c in range(N)]
    return np.stack(cols, axis=1)


def dev_ptr(t):
    return t.data_ptr() if t is not None else None


# (16384, 1024, 256): a grid with a workgroup per CU, where the kernel takes 256-wide column
# tiles; the smaller products take 128-wide ones.
@pytest.mark.parametrize("M,N,K", [(512, 512, 96), (256, 384, 64), (768, 1024, 416), (16384, 1024, 256)])
@pytest.mark.parametrize("bits,rdot,no_store", [(True, False, False), (False, True, False), (False, True, True),
                                                (True, True, False), (True, True, True)])
def test_forward_fused_epilogue(fused, M, N, K, bits, rdot, no_store):
    """ReLU forward with mask bits / row dots: C matches the plain product (one
    bf16 ulp), the bits are exactly C > 0 of the stored C, and the row-dot partials
    are the column-group sums of stored C times w (float32 accumulation)."""
    torch, f, rdot_cols = fused
    rng = np.random.default_rng(M + N + K)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((N, K)).astype(np.float32)
    bias = rng.standard_normal(N).astype(np.float32)
    w = rng.standard_normal(N).astype(np.float32)
    dA, dB = to_dev(torch, A, True), to_dev(torch, B, True)
    dbias = torch.from_numpy(bias).cuda()
    dw = to_dev(torch, w, True)
    dC = torch.full((M, N), 7.0, dtype=torch.bfloat16, device="cuda")
    dbits = torch.zeros((N // 32, M), dtype=torch.int32, device="cuda") if bits else None
    cols = rdot_cols(M, N)
    parts = N // cols
    dpart = torch.zeros((parts, M), dtype=torch.float32, device="cuda") if rdot else None
    rc = f(0, M, N, K, dA.data_ptr(), K, dB.data_ptr(), K, dC.data_ptr(), N, dbias.data_ptr(), dev_ptr(dbits), None,
           M, dev_ptr(dw) if rdot else None, dev_ptr(dpart), M, int(no_store), None, 0)
    assert rc == 0, rc
    pre = rounded(torch, A, True) @ rounded(torch, B, True).T + bias
    ref = np.maximum(pre, 0.0)
    ref_b = rounded(torch, ref, True)
    got = dC.to(torch.float64).cpu().numpy()
    # ReLU of a pre-activation within float32 accumulation error of zero may fall either
    # way (a few of the 16.7M values of the largest shape)
    near0 = np.abs(pre) <= 1e-4 * np.sqrt(np.mean(pre * pre))
    if no_store:
        assert np.all(got == 7.0)
        # the stored values the epilogue used are not visible: compare the row dots
        # with the reference product instead (bf16 ulp-level differences allowed)
        cval = ref_b
    else:
        ulp = np.abs(ref_b) * 2.0 ** -7 + 1e-30
        assert np.all((np.abs(got - ref_b) <= 2 * ulp + 1e-6) | near0)
        cval = got
    if bits:
        words = dbits.cpu().numpy().view(np.uint32)
        mask = unpack_bits(words, M, N)
        if no_store:
            # sign decisions near zero may differ from the float64 reference
            assert (mask != (ref_b > 0)).mean() < 1e-3
        else:
            assert np.array_equal(mask, got > 0)
    if rdot:
        wr = rounded(torch, w, True)
        part = dpart.cpu().numpy().astype(np.float64)
        want = np.stack([(cval[:, p * cols:(p + 1) * cols] * wr[p * cols:(p + 1) * cols]).sum(1)
                         for p in range(parts)])
        scale = np.abs(cval[:, :]).max() * np.abs(wr).max() * cols
        tol = 1e-5 if not no_store else 2.0 ** -7
        assert np.abs(part - want).max() <= tol * scale, np.abs(part - want).max() / scale


@pytest.mark.parametrize("M,N,K", [(512, 512, 64), (256, 1024, 1024), (512, 384, 96), (16384, 1024, 256)])
@pytest.mark.parametrize("colsum", [False, True])
def test_dgrad_bits_equal_mask(env, fused, M, N, K, colsum):
    """A dgrad masked by bits is bit-identical to the same dgrad masked by a bf16
    tensor with the same sign pattern; the fused column sums are those of the
    stored result over each 256-row tile."""
    torch, gemm = env
    _, f, _ = fused
    rng = np.random.default_rng(M * 7 + N + K)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    pos = rng.uniform(size=(M, N)) < 0.5
    mask = np.where(pos, rng.uniform(0.1, 2.0, size=(M, N)), -rng.uniform(0.0, 2.0, size=(M, N))).astype(np.float32)
    words = np.zeros((N // 32, M), dtype=np.uint32)
    for c in range(N):
        words[c // 32] |= (pos[:, c].astype(np.uint32) << np.uint32(c % 32))
    dA, dB = to_dev(torch, A, True), to_dev(torch, B, True)
    dmask = to_dev(torch, mask, True)
    dbits = torch.from_numpy(words.view(np.int32)).cuda()
    dC1 = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
    dC2 = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
    dcs = torch.zeros((M // 256, N), dtype=torch.float32, device="cuda") if colsum else None
    rc = gemm(1, 1, M, N, K, 1, dA.data_ptr(), K, dB.data_ptr(), N, dC1.data_ptr(), N, None, dmask.data_ptr(), N, 0, 0)
    assert rc == 0
    rc = f(1, M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, dC2.data_ptr(), N, None, None, dbits.data_ptr(), M,
           None, None, 0, 0, dev_ptr(dcs), N)
    assert rc == 0
    assert torch.equal(dC1.view(torch.int16), dC2.view(torch.int16))
    if colsum:
        c = dC2.to(torch.float64).cpu().numpy().reshape(M // 256, 256, N).sum(1)
        got = dcs.cpu().numpy()
        assert np.abs(got - c).max() <= 1e-5 * np.abs(c).max() + 1e-6


def test_fused_rejects_bad_use(fused):
    """Fused epilogues need the whole product on the large-tile kernel."""
    torch, f, _ = fused
    d = torch.zeros(1 << 20, device="cuda")
    p = d.data_ptr()
    # N not a multiple of 128
    assert f(0, 256, 96, 64, p, 64, p, 64, p, 96, None, p, None, 256, None, None, 0, 0, None, 0) != 0
    # no_store without a row dot
    assert f(0, 256, 128, 64, p, 64, p, 64, p, 128, None, p, None, 256, None, None, 0, 1, None, 0) != 0
    # dgrad without bits
    assert f(1, 256, 128, 64, p, 64, p, 128, p, 128, None, None, None, 256, None, None, 0, 0, None, 0) != 0
    # bits leading dimension shorter than M
    assert f(0, 512, 128, 64, p, 64, p, 64, p, 128, None, p, None, 256, None, None, 0, 0, None, 0) != 0


def test_bf16_rounding_exhaustive(env):
    """The device float32 -> bf16 conversion (hardware instruction) rounds every
    float32 bit pattern to nearest-even exactly as the integer definition does."""
    from paper_2312_06126_amd import spz
    lib = spz.load()
    lib.spzt_bf16_round_check.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint64)]
    lib.spzt_bf16_round_check.restype = ctypes.c_int
    bad = ctypes.c_uint64(0)
    assert lib.spzt_bf16_round_check(0, 1 << 32, ctypes.byref(bad)) == 0
    assert bad.value == 0, bad.value


# ----------------------------------------------------------------------------- device-side row count
@pytest.mark.parametrize("bf16,M,N,K,bits,out_f32", [(True, 1024, 256, 512, True, False),
                                                      (True, 1024, 1024, 256, True, False),
                                                      (True, 1024, 128, 256, False, True),
                                                      (True, 1024, 32, 1024, False, True),
                                                      (False, 512, 64, 128, False, True)],
                         ids=["large_bits", "large_bits_n1024", "large_f32", "generic_n32", "fp32"])
def test_dgrad_device_row_count(env, bf16, M, N, K, bits, out_f32):
    """An input-gradient product limited to the first m rows by a device-side count
    gives exactly the rows of the unlimited product and leaves the other rows as they
    were (m = 0, a middle multiple of 256, M); a count that is not a multiple of 256
    is refused."""
    torch, _ = env
    from paper_2312_06126_amd import spz
    lib = spz.load()
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    f = lib.spzt_gemm_dgrad_rows
    f.argtypes = [I32, I32, I32, I32, P, I64, P, I64, P, I64, P, I64, I32, I32]
    f.restype = ctypes.c_int
    rng = np.random.default_rng(M + N + K)
    dA = to_dev(torch, rng.standard_normal((M, K)), bf16)
    dB = to_dev(torch, rng.standard_normal((K, N)), bf16)
    dbits = (torch.from_numpy(rng.integers(0, 1 << 32, size=(N // 32, M), dtype=np.uint64).astype(np.uint32)
                              .view(np.int32)).cuda() if bits else None)
    ctype = torch.float32 if (out_f32 or not bf16) else torch.bfloat16
    outs = {}
    for m in (M, 0, 256 if M > 256 else 0, M // 2):
        dC = torch.full((M, N), 3.0, dtype=ctype, device="cuda")
        torch.cuda.synchronize()
        rc = f(int(bf16), M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, dC.data_ptr(), N,
               dbits.data_ptr() if bits else None, M, int(out_f32), m)
        assert rc == 0, (m, rc)
        outs[m] = dC.to(torch.float64).cpu().numpy()
    full = outs[M]
    assert not np.all(full == 3.0)
    for m, got in outs.items():
        assert np.array_equal(got[:m], full[:m]), m
        assert np.all(got[m:] == 3.0), m
    dC = torch.zeros((M, N), dtype=ctype, device="cuda")
    assert f(int(bf16), M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, dC.data_ptr(), N,
             dbits.data_ptr() if bits else None, M, int(out_f32), 128) == spz.SPZ_EINVAL
