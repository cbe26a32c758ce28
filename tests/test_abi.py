"""The C ABI library loads and exports every symbol include/pgsr.h declares;
host-side validation answers without touching a GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pgsr.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pgsr_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def native():
    from paper_2609_04875_amd import _native
    return _native


def test_header_declares_the_hot_path():
    names = declared_functions()
    for must in ("pgsr_kv_crop", "pgsr_replay_prefill", "pgsr_full_reset_prefill"):
        assert must in names


def test_every_declared_symbol_is_exported(native):
    names = declared_functions()
    raw = ctypes.CDLL(native.LIB_PATH)
    missing = [n for n in names if not hasattr(raw, n)]
    assert not missing, missing
    assert set(names) == set(native.EXPORTS)


def test_checked_build_exports_the_same_symbols(native):
    """The checked build (block ids validated on the device) has the same C ABI."""
    path = os.path.join(os.path.dirname(native.LIB_PATH), "libpgsr_checked.so")
    if not os.path.exists(path):
        pytest.skip("checked build not built")
    raw = ctypes.CDLL(path)
    missing = [n for n in declared_functions() if not hasattr(raw, n)]
    assert not missing, missing
    raw.pgsr_abi_version.restype = ctypes.c_int
    assert raw.pgsr_abi_version() == native.lib.pgsr_abi_version()


def test_abi_version_and_workspace_size(native):
    assert native.lib.pgsr_abi_version() == 2
    assert native.lib.pgsr_workspace_bytes(32, 128, 2048, 4) == 2048 * 32 * 4 * 130 * 4
    assert native.lib.pgsr_workspace_bytes(32, 128, 2048, 1) == 0


def test_create_rejects_bad_geometry_before_any_device_call(native):
    out = ctypes.c_void_p()
    fake = ctypes.c_void_p(16)   # never dereferenced: validation fails first
    args = dict(n_layers=1, hq=32, hkv=8, d=128, B=16, dt=native.BF16, nb=64, ms=2, mbps=8)

    def create(**kw):
        a = {**args, **kw}
        return native.lib.pgsr_pool_create(a["n_layers"], a["hq"], a["hkv"], a["d"], a["B"], a["dt"],
                                           a["nb"], a["ms"], a["mbps"], fake, fake, fake, fake, fake,
                                           fake, fake, None, 0, None, None, ctypes.byref(out))
    assert create(d=96) == native.EUNSUPPORTED
    assert create(B=8) == native.EUNSUPPORTED
    assert create(hq=30) == native.EUNSUPPORTED
    assert create(hq=33, hkv=1) == native.EUNSUPPORTED       # bf16: at most 32 query heads per KV head
    assert create(dt=7) == native.EUNSUPPORTED
    assert create(dt=native.FP8_E4M3, hq=33, hkv=1) == native.EUNSUPPORTED   # fp8 runs the bf16 kernel
    assert create(nb=0) == native.EINVAL
    order = native.int32_array([0, 1, 1] + list(range(3, 64)))
    assert native.lib.pgsr_pool_create(1, 32, 8, 128, 16, native.BF16, 64, 2, 8, fake, fake, fake,
                                       fake, fake, fake, fake, None, 0, order, None,
                                       ctypes.byref(out)) == native.EINVAL
    assert b"permutation" in native.lib.pgsr_last_error()
    assert not out.value
    # a missing ref_counts array is rejected before any device call
    assert native.lib.pgsr_pool_create(1, 32, 8, 128, 16, native.BF16, 64, 2, 8, fake, fake, fake,
                                       fake, fake, fake, None, None, 0, None, None,
                                       ctypes.byref(out)) == native.EINVAL


def test_null_pool_and_gemm_validation(native):
    assert native.lib.pgsr_kv_crop(None, 0, None, None, 0, None) == native.EINVAL
    assert native.lib.pgsr_kv_fork(None, 0, None, None, None) == native.EINVAL
    one = (ctypes.c_float * 1)(1.0)
    assert native.lib.pgsr_pool_set_kv_scales(None, one, one) == native.EINVAL
    assert native.lib.pgsr_gemm_bf16(4, 12, 16, None, None, None, None, None) == native.EUNSUPPORTED
    assert native.lib.pgsr_gemm_bf16(0, 16, 16, None, None, None, None, None) == native.OK
    assert native.lib.pgsr_gemm_bf16(4, 16, 16, None, None, None, None, None) == native.EINVAL


def test_prefill_kernel_choice_is_validated(native):
    assert native.lib.pgsr_pool_set_prefill_kernel(None, 0) == native.EINVAL


def test_binding_rejects_tensors_of_the_wrong_size_or_device():
    """The C ABI takes raw pointers, so the binding checks what it cannot:
    exact element counts for the call's token total, and the pool's device."""
    import torch
    from paper_2609_04875_amd.pool import _dev_ptr, prefill_sizes

    assert prefill_sizes(32, 8, 128, [3, 0, 5]) == (8 * 32 * 128, 8 * 8 * 128)
    q = torch.zeros((7, 32, 128), dtype=torch.bfloat16)      # one token short of 3 + 0 + 5
    nq, nkv = prefill_sizes(32, 8, 128, [3, 0, 5])
    with pytest.raises(ValueError, match="exactly"):
        _dev_ptr(q, torch.bfloat16, "q", None, nq)
    with pytest.raises(ValueError, match="exactly"):
        _dev_ptr(torch.zeros((9, 8, 128), dtype=torch.bfloat16), torch.bfloat16, "k", None, nkv)
    with pytest.raises(ValueError, match="needed"):
        _dev_ptr(None, torch.bfloat16, "o", None, nq)
    with pytest.raises(ValueError, match="CUDA"):              # right size, but host memory
        _dev_ptr(torch.zeros((8, 32, 128), dtype=torch.bfloat16), torch.bfloat16, "q", None, nq)

    class OnOtherDevice:                                      # stands in for a tensor on cuda:1
        is_cuda = True
        dtype = torch.bfloat16
        device = torch.device("cuda", 1)

        def numel(self):
            return nq

        def is_contiguous(self):
            return True

    with pytest.raises(ValueError, match="cuda:1"):
        _dev_ptr(OnOtherDevice(), torch.bfloat16, "q", 0, nq)
