"""The C-ABI library loads and exports every entry point include/spz.h declares.

No compute calls: these run without a GPU. The struct layout of spz_hparams is
checked by reading back the library's defaults through the binding's mirror.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spz.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spz_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2312_06126_amd import spz
    if not os.path.exists(spz.LIB_PATH):
        pytest.fail("libspz.so is not built; run __graft_entry__.build()")
    return spz.load()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    from paper_2312_06126_amd import spz
    assert sorted(spz.EXPORTS) == names


def test_hparams_defaults_roundtrip_layout(lib):
    from paper_2312_06126_amd import spz
    hp = spz.default_hparams()
    assert hp.algo == 0 and hp.gemm_prec == 0 and hp.capacity == 1_000_000
    assert abs(hp.gamma - 0.99) < 1e-7 and abs(hp.tau - 0.005) < 1e-9
    assert abs(hp.lr_actor - 3e-4) < 1e-10 and abs(hp.beta2 - 0.999) < 1e-7
    assert hp.learn_alpha == 1 and hp.log_std_min == -20.0 and hp.log_std_max == 2.0
    assert abs(hp.policy_noise - 0.2) < 1e-7 and hp.policy_delay == 2
    assert hp.device == 0 and hp.n_streams == 2 and hp.ordering == 0 and hp.actor_row_split == 1


def test_selector_table_matches_header(lib):
    from paper_2312_06126_amd import spz
    text = open(HEADER).read()
    for name, val in spz.SELECTORS.items():
        m = re.search(r"#define SPZ_%s (\d+)" % name.upper(), text)
        assert m and int(m.group(1)) == val, name


def test_debug_selectors_match_header(lib):
    from paper_2312_06126_amd import spz
    text = open(HEADER).read()
    for name, (val, _) in spz.DEBUG_ROWS.items():
        m = re.search(r"#define SPZ_DBG_%s (\d+)" % name.upper(), text)
        assert m and int(m.group(1)) == val, name
    for name, val in (("INDICES", spz.DBG_INDICES), ("BATCH", spz.DBG_BATCH)):
        m = re.search(r"#define SPZ_DBG_%s (\d+)" % name, text)
        assert m and int(m.group(1)) == val, name


def test_null_arguments_fail_cleanly(lib):
    """Argument validation happens before any device call."""
    from paper_2312_06126_amd import spz
    hp = spz.default_hparams()
    h = (ctypes.c_int32 * 1)(4)
    assert not lib.spz_create(3, 2, None, 1, 8, ctypes.byref(hp), 1)
    assert b"NULL" in lib.spz_last_error(None)
    assert not lib.spz_create(0, 2, h, 1, 8, ctypes.byref(hp), 1)
    assert b"dimensions" in lib.spz_last_error(None)
    assert lib.spz_update(None, 1, None) == spz.SPZ_EINVAL
    assert lib.spz_profile_stride(None, 1) == spz.SPZ_EINVAL
    assert lib.spz_buffer_push(None, None, None, None, None, None, 0) == spz.SPZ_EINVAL
    assert lib.spz_param_count(None, 0) == spz.SPZ_EINVAL


def test_only_the_c_abi_is_exported(lib):
    """The dynamic symbol table holds the spz_* calls of include/spz.h and the spzt_*
    test hooks of include/spz_testing.h, nothing else (no C++ internals, no helpers)."""
    import shutil
    import subprocess
    from paper_2312_06126_amd import spz
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm (binutils) not installed")
    out = subprocess.run([nm, "-D", "--defined-only", spz.LIB_PATH], capture_output=True, text=True, check=True)
    names = sorted(line.split()[-1] for line in out.stdout.splitlines() if line.strip())
    testing = open(os.path.join(ROOT, "include", "spz_testing.h")).read()
    testing = re.sub(r"/\*.*?\*/", "", testing, flags=re.S)
    hooks = sorted(set(re.findall(r"\b(spzt_[a-z0-9_]+)\s*\(", testing)))
    assert names == sorted(declared_functions() + hooks), [n for n in names if not n.startswith("spz")]
