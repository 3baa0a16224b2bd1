"""rgd_kernel_sample_noalloc (the sampler for callers that cannot allocate)
against rgd_kernel_sample with a caller workspace, through the C ABI: two calls
in a row, the second on a smaller input, each bit-identical to the workspace
entry point's draws on the same logits and seeds (same kernels; the scratch
keeps the first call's contents, which the second must not depend on).  A
call beyond the fixed scratch is rejected."""
import numpy as np
import pytest

import synth
from tests.gpu_common import seeds_tensor, torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


def _both(rgd, z_np, T, pmin, seeds, ctr, stream0, draws):
    t = torch()
    z = t.from_numpy(np.ascontiguousarray(z_np, dtype=np.float32)).cuda()
    R, V = z.shape
    sd = seeds_tensor(seeds)
    ws = t.empty(rgd.sampler_workspace_bytes(R, V), dtype=t.uint8, device="cuda")
    a = t.full((R, draws), -1, dtype=t.int32, device="cuda")
    b = t.full((R, draws), -2, dtype=t.int32, device="cuda")
    rgd.kernel_sample(z, T, pmin, sd, ctr, stream0, draws, ws, a)
    rgd.kernel_sample_noalloc(z, T, pmin, sd, ctr, stream0, draws, b)
    t.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy()


def test_noalloc_matches_workspace_sampler_on_two_calls(rgd):
    # first call: 160 rows of the sampler-sweep logits (one workgroup per row,
    # 3 draws per row); second: 24 rows of a smaller vocabulary (chunk kernels)
    z1 = synth.sweep_logits(synth.SWEEP, rows=160)
    assert rgd.sampler_workspace_bytes(160, z1.shape[1]) <= rgd.NOALLOC_SCRATCH_BYTES
    a, b = _both(rgd, z1, 2.0, 0.05, np.arange(160, dtype=np.uint64) + 9, 4, 1, 3)
    assert (a >= 0).all() and np.array_equal(a, b)
    z2 = np.ascontiguousarray(z1[:24, :12288 + 4])
    a, b = _both(rgd, z2, 1.5, 0.1, np.arange(24, dtype=np.uint64) + 70, 2, 0, 2)
    assert (a >= 0).all() and np.array_equal(a, b)


def test_noalloc_rejects_inputs_beyond_the_scratch(rgd):
    """Rejected before any HIP call: the buffers are never touched."""
    import ctypes as C
    t = torch()
    R, V = 4096, 152064
    assert rgd.sampler_workspace_bytes(R, V) > rgd.NOALLOC_SCRATCH_BYTES
    small = t.zeros(16, dtype=t.float32, device="cuda")
    p = C.c_void_p(small.data_ptr())
    rc = rgd.lib.rgd_kernel_sample_noalloc(p, R, V, 1.0, 0.1, p, 0, 0, 1, p, None)
    assert rc == 1 and b"scratch" in rgd.lib.rgd_last_error()
    # the entry point still works afterwards
    test_noalloc_matches_workspace_sampler_on_two_calls(rgd)
