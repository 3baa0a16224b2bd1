"""The C ABI library loads and exports every declared entry point; argument
validation rejects bad calls before any HIP call (CPU only, no GPU needed)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "rgd.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(rgd_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


def test_every_declared_symbol_is_exported(rgd):
    names = _declared()
    assert len(names) >= 19
    for n in names:
        assert hasattr(rgd.lib, n), n
    assert set(names) == set(rgd.EXPORTS)


def test_version_and_empty_error(rgd):
    assert b"gfx950" in rgd.lib.rgd_version()


def _code(rc):
    return int(rc)


def test_model_create_rejects_nulls_and_bad_config(rgd):
    h = C.c_void_p()
    assert _code(rgd.lib.rgd_model_create(None, None, 1, C.byref(h))) == 1
    assert b"null" in rgd.lib.rgd_last_error()
    cfg = rgd.ModelConfig(1, 256, 4, 3, 64, 1024, 8192, 0, 1e-5, 5e5, 128)   # 4 % 3 != 0
    w = rgd.Weights()
    assert _code(rgd.lib.rgd_model_create(C.byref(cfg), C.byref(w), 1, C.byref(h))) == 4
    cfg = rgd.ModelConfig(1, 256, 4, 2, 64, 1024, 8192, 7, 1e-5, 5e5, 128)   # bad dtype
    assert _code(rgd.lib.rgd_model_create(C.byref(cfg), C.byref(w), 1, C.byref(h))) == 1
    cfg = rgd.ModelConfig(1, 4096, 32, 8, 64, 14336, 128256, 1, 1e-5, 5e5, 128)  # bf16 needs D=128
    assert _code(rgd.lib.rgd_model_create(C.byref(cfg), C.byref(w), 1, C.byref(h))) == 4
    cfg = rgd.ModelConfig(1, 256, 4, 2, 64, 1024, 8192, 0, 1e-5, 5e5, 128)
    assert _code(rgd.lib.rgd_model_create(C.byref(cfg), C.byref(w), 0, C.byref(h))) == 1
    assert _code(rgd.lib.rgd_model_create(C.byref(cfg), C.byref(w), 4, C.byref(h))) == 1  # null weights


def test_table_validation(rgd):
    h = C.c_void_p()
    off = np.array([1, 2], np.int32)
    tok = np.array([5, 6], np.int32)
    P = C.POINTER(C.c_int32)
    rc = rgd.lib.rgd_table_create(off.ctypes.data_as(P), tok.ctypes.data_as(P), 1, None, 2, C.byref(h))
    assert rc == 1 and b"offsets[0]" in rgd.lib.rgd_last_error()
    off = np.array([0, 3, 2], np.int32)
    rc = rgd.lib.rgd_table_create(off.ctypes.data_as(P), tok.ctypes.data_as(P), 2, None, 2, C.byref(h))
    assert rc == 1
    off = np.array([0, 2], np.int32)
    rc = rgd.lib.rgd_table_create(off.ctypes.data_as(P), tok.ctypes.data_as(P), 1, None, 0, C.byref(h))
    assert rc == 1
    own = np.array([-2], np.int32)
    rc = rgd.lib.rgd_table_create(off.ctypes.data_as(P), tok.ctypes.data_as(P), 1, own.ctypes.data_as(P), 2,
                                  C.byref(h))
    assert rc == 1
    assert rgd.lib.rgd_table_create(None, None, -1, None, 2, C.byref(h)) == 1


def test_entry_points_reject_null_handles(rgd):
    P = C.POINTER(C.c_int32)
    one = np.zeros(4, np.int32)
    p = one.ctypes.data_as(P)
    assert rgd.lib.rgd_prefill_kv(None, None, None, 1, 1, 0, None, None) == 1
    assert rgd.lib.rgd_probe(None, None, None, None, 1, 1, 1, -1, None, None, None, None) == 1
    assert rgd.lib.rgd_gate(None, None, 1, p, p, p, None) == 1
    assert rgd.lib.rgd_sample_continuations(None, None, None, p, 1, 1, 1, 1.0, 0.1, None, None, None,
                                            None, None) == 1
    assert rgd.lib.rgd_sample_continuations_pless(None, None, None, p, 1, 1, 1, 1.0, None, None, None,
                                                  None, None) == 1
    assert rgd.lib.rgd_kv_create(None, 1, 1, 1, 16, None, None, None, None, C.byref(C.c_void_p())) == 1
    assert rgd.lib.rgd_kv_set_prefix_len(None, 0, 0) == 1
    assert rgd.lib.rgd_check_status(None, None) == 1
    assert rgd.lib.rgd_kernel_lm_head(None, None, 1, None, None) == 1
    assert rgd.lib.rgd_kernel_attention(None, None, 1, p, p, None, None, 1, 1, None, None, 16, None, 1,
                                        0, 0, None, None) == 1


def test_kernel_sampler_validation(rgd):
    fake = C.c_void_p(256)   # never dereferenced: validation fails first
    assert rgd.lib.rgd_kernel_sample(fake, 2, 8, 0.0, 0.1, fake, 0, 0, 1, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample(fake, 2, 8, 1.0, 1.5, fake, 0, 0, 1, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample(fake, 2, 6, 1.0, 0.1, fake, 0, 0, 1, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample(fake, 2, 8, 1.0, 0.1, fake, 0, 0, 0, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample(fake, 2, 8, 1.0, 0.1, fake, 0, 0, 1, C.c_void_p(260), fake, None) == 1
    assert rgd.lib.rgd_kernel_sample_pless(fake, 2, 8, 0.0, fake, 0, 0, 1, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample_pless(fake, 2, 6, 1.0, fake, 0, 0, 1, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample_pless(None, 2, 8, 1.0, fake, 0, 0, 1, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_sample_pless(fake, 2, 8, 1.0, fake, 0, 0, 1, C.c_void_p(260), fake, None) == 1
    assert rgd.lib.rgd_kernel_argmax(None, 2, 8, fake, fake, None) == 1
    assert rgd.lib.rgd_kernel_argmax(fake, 0, 8, fake, fake, None) == 1
    assert rgd.lib.rgd_sampler_workspace_bytes(4, 152064) >= 8 * 4 + 4 * 4 + 16 * 4 * 38
    assert rgd.lib.rgd_sampler_workspace_bytes(0, 8) == 0


def test_noalloc_sampler_rejects_before_any_hip_call(rgd):
    """The no-allocation sampler validates sizes (against its fixed scratch)
    and arguments before touching the GPU, so this runs without one."""
    fake = C.c_void_p(0x1000)
    assert _code(rgd.lib.rgd_kernel_sample_noalloc(None, 4, 8, 1.0, 0.1, fake, 0, 0, 1, fake, None)) == 1
    assert _code(rgd.lib.rgd_kernel_sample_noalloc(fake, 4096, 152064, 1.0, 0.1, fake, 0, 0, 1, fake, None)) == 1
    assert b"scratch" in rgd.lib.rgd_last_error()
    assert _code(rgd.lib.rgd_kernel_sample_noalloc(fake, 4, 8, 0.0, 0.1, fake, 0, 0, 1, fake, None)) == 1
    assert _code(rgd.lib.rgd_kernel_sample_noalloc(fake, 4, 8, 1.0, 1.5, fake, 0, 0, 1, fake, None)) == 1
    assert rgd.sampler_workspace_bytes(160, 152064) <= rgd.NOALLOC_SCRATCH_BYTES
