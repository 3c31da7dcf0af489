"""hstu_attn_fwd_noalloc (the forward with its scratch in the library's
static device array) through the C ABI against hstu_attn_fwd with a
caller workspace: bitwise equal outputs on two calls in a row, the second
on a smaller batch (the static array keeps the first call's contents),
plus the size limit, which is rejected before anything is launched."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2402_17152_amd import inputs
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hs():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2402_17152_amd import hstu
    return hstu


def _pair(hs, batch):
    d = gu.dev_inputs(batch)
    ref = gu.gpu_fwd(hs, d, batch)
    out = torch.full_like(ref, float("nan"))
    hs.hstu_attn_fwd_noalloc(d["q"], d["k"], d["v"], d["seq_offsets"], d["timestamps"],
                             d["rab_pos"], d["rab_time"], batch.spec.max_seq_len, out,
                             num_targets=d["num_targets"])
    torch.cuda.synchronize()
    return out, ref


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_forward(hs, oracle_mod, dtype):
    big = inputs.make_batch(3, seed=81, lengths=(700, 1, 0, 513, 2049, 64), num_heads=2,
                            d_qk=64, d_v=64, max_seq_len=2049, dtype=dtype,
                            num_targets=(0, 0, 0, 13, 0, 64))
    small = inputs.make_batch(3, seed=82, lengths=(129, 5), num_heads=2, d_qk=64, d_v=64,
                              max_seq_len=256, dtype=dtype)
    for batch in (big, small):
        out, ref = _pair(hs, batch)
        assert torch.equal(out, ref), "no-alloc forward differs from the workspace forward"
    # and the smaller call is right on its own terms
    gu.assert_close("O", gu.to_f64(out), gu.oracle_fwd(oracle_mod, small), gu.tol(small), dtype)


def test_noalloc_long_workload(hs):
    """The long workload (T = 48118, B = 8), then a 3-sequence batch."""
    for batch in (inputs.make_batch("long"),
                  inputs.make_batch(3, seed=83, lengths=(300, 17, 1000), max_seq_len=8192)):
        out, ref = _pair(hs, batch)
        assert torch.equal(out, ref)


def test_noalloc_rejects_oversize(hs):
    """A problem whose work list would not fit the static scratch returns
    HSTU_ERR_UNSUPPORTED with a message; nothing is dereferenced (the
    device pointers are never used)."""
    B, T = 1024, 80_000_000
    p = hs.make_problem(B, T, 8192, 1, 32, 32, 128, hs.HSTU_BF16)
    fake = 0x10000
    j = hs.Jagged(fake, fake, None, fake, fake)
    P = ctypes.c_void_p
    st = hs.lib.hstu_attn_fwd_noalloc(ctypes.byref(p), ctypes.byref(j), P(fake), 32, P(fake), 32,
                                      P(fake), 32, P(fake), None)
    assert st == 2, hs.hstu_last_error()
    assert "static" in hs.hstu_last_error()
