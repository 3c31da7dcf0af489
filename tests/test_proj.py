"""GPU parity of the layer's linear maps (Eq. 1 with phi_1, Eq. 3's f_2 and
the residual) and of the whole layer they close, through the C ABI
against the fp64 oracle on the same stored inputs.

Criterion as in the attention tests: per output tensor, max_i (|gpu_i -
ref_i| - u |ref_i|)_+ <= tau RMS(ref), tau = 2e-2 (bf16) / 1e-4 (fp32),
u the storage rounding of the output.

* small shapes: every output, both dtypes, token counts that leave ragged
  row tiles, output widths that leave partial column tiles, T = 1;
* the training shape (T = 60383 tokens, D = 512, h = 8, d = 64, F = 2048):
  sampled token rows of z, z_pre, y, dx, dg, and sampled rows of the
  weight gradients (each a sum over all tokens, computed by the oracle for
  those rows alone);
* the whole layer, x -> x_next and back, on a small jagged batch."""
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


def _dev(P):
    return {k: inputs.array_to_device(v) for k, v in P.items()}


def _f64(P):
    return {k: inputs.stored_f64(v) for k, v in P.items()}


def _tau(dtype):
    return 2e-2 if dtype == "bf16" else 1e-4


def _dz_parts(dz, h, dqk, dv):
    """[du | dv | dq | dk] of dz [T, F] as dense [T, h, d] device tensors."""
    T = dz.shape[0]
    hv, hq = h * dv, h * dqk
    cuts = [(0, hv, dv), (hv, 2 * hv, dv), (2 * hv, 2 * hv + hq, dqk), (2 * hv + hq, 2 * hv + 2 * hq, dqk)]
    return [dz[:, a:b].contiguous().view(T, h, d) for a, b, d in cuts]


SMALL = [
    # (T, D, h, d_qk, d_v)
    (300, 64, 2, 32, 32),
    (1000, 128, 2, 64, 32),
    (257, 256, 4, 32, 64),
    (1, 64, 1, 32, 64),
    # 128-wide heads, widths that are not multiples of the 128 / 256 tiles
    (513, 384, 3, 128, 64),
    (130, 192, 1, 128, 128),
    # a longer contraction (f_1 over D = 1024, f_2 over h d_v = 512)
    (700, 1024, 8, 64, 64),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("case", range(len(SMALL)))
def test_proj_small(hs, oracle_mod, dtype, case):
    T, D, h, dqk, dv = SMALL[case]
    P = inputs.make_proj(T, D, h, dqk, dv, dtype=dtype, seed=40 + case)
    d, r = _dev(P), _f64(P)
    tau, st = _tau(dtype), dtype
    z, z_pre = hs.hstu_proj_in_fwd(d["x"], d["w1"], d["b1"], h, dqk, dv)
    y = hs.hstu_proj_out_fwd(d["g"], d["w2"], d["b2"], d["x"], h, dqk, dv)
    dx, dw1, db1 = hs.hstu_proj_in_bwd(d["x"], d["w1"], z_pre, *_dz_parts(d["dz"], h, dqk, dv),
                                       h, dqk, dv, dx_add=d["dy"])
    dg, dw2, db2 = hs.hstu_proj_out_bwd(d["g"], d["w2"], d["dy"], h, dqk, dv)
    torch.cuda.synchronize()
    rz, rpre = oracle_mod.proj_in_fwd(r["x"], r["w1"], r["b1"])
    ry = oracle_mod.proj_out_fwd(r["g"], r["w2"], r["b2"], residual=r["x"])
    # z_pre as stored feeds the backward; the oracle recomputes its own.
    rdx, rdw1, rdb1 = oracle_mod.proj_in_bwd(r["x"], r["w1"], r["b1"], r["dz"])
    rdg, rdw2, rdb2 = oracle_mod.proj_out_bwd(r["g"], r["w2"], r["dy"])
    for name, got, ref, store in (("z", z, rz, st), ("z_pre", z_pre, rpre, st), ("y", y, ry, st),
                                  ("dx", dx, rdx + r["dy"], st), ("dw1", dw1, rdw1, "f32"),
                                  ("db1", db1, rdb1, "f32"), ("dg", dg, rdg, st),
                                  ("dw2", dw2, rdw2, "f32"), ("db2", db2, rdb2, "f32")):
        e = gu.assert_close(name, gu.to_f64(got), ref, tau, store)
        print(f"\n  {name}: {e[0]:.3e} raw {e[1]:.3e}", end="")


def test_proj_empty(hs):
    """No tokens: nothing to compute, weight and bias gradients are zero."""
    P = inputs.make_proj(0, 64, 2, 32, 32, seed=3)
    d = _dev(P)
    z, z_pre = hs.hstu_proj_in_fwd(d["x"], d["w1"], d["b1"], 2, 32, 32)
    dz = torch.zeros((0, 256), dtype=torch.bfloat16, device="cuda")
    dx, dw1, db1 = hs.hstu_proj_in_bwd(d["x"], d["w1"], z_pre, *_dz_parts(dz, 2, 32, 32), 2, 32,
                                       32)
    dg, dw2, db2 = hs.hstu_proj_out_bwd(d["g"], d["w2"], d["dy"], 2, 32, 32)
    torch.cuda.synchronize()
    for t in (dw1, db1, dw2, db2):
        assert torch.count_nonzero(t).item() == 0


def test_proj_rejects_bad_shapes(hs):
    P = inputs.make_proj(8, 96, 2, 32, 32, seed=4)  # D = 96: not a multiple of 64
    d = _dev(P)
    with pytest.raises(RuntimeError, match="multiples of 64"):
        hs.hstu_proj_in_fwd(d["x"], d["w1"], d["b1"], 2, 32, 32)


def test_proj_training_shape(hs, oracle_mod):
    """Training shape: T = 60383 tokens (the training workload's), D = 512,
    h = 8, d = 64.  Token rows sampled for the row-wise outputs, rows of
    the weight gradients sampled (each an exact sum over all tokens)."""
    T = int(inputs.make_batch("training").seq_offsets[-1])
    D, h, dqk, dv = 512, 8, 64, 64
    P = inputs.make_proj(T, D, h, dqk, dv, dtype="bf16", seed=7)
    d = _dev(P)
    z, z_pre = hs.hstu_proj_in_fwd(d["x"], d["w1"], d["b1"], h, dqk, dv)
    y = hs.hstu_proj_out_fwd(d["g"], d["w2"], d["b2"], d["x"], h, dqk, dv)
    dx, dw1, db1 = hs.hstu_proj_in_bwd(d["x"], d["w1"], z_pre, *_dz_parts(d["dz"], h, dqk, dv),
                                       h, dqk, dv, dx_add=d["dy"])
    dg, dw2, db2 = hs.hstu_proj_out_bwd(d["g"], d["w2"], d["dy"], h, dqk, dv)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    rows = np.unique(np.r_[0, T - 1, rng.integers(0, T, 62)])
    r = {k: inputs.stored_f64(P[k][rows]) for k in ("x", "g", "dz", "dy")}
    w1, w2 = inputs.stored_f64(P["w1"]), inputs.stored_f64(P["w2"])
    rz, rpre = oracle_mod.proj_in_fwd(r["x"], w1, P["b1"])
    ry = oracle_mod.proj_out_fwd(r["g"], w2, P["b2"], residual=r["x"])
    rdx = oracle_mod.proj_in_bwd(r["x"], w1, P["b1"], r["dz"])[0] + r["dy"]
    rdg = oracle_mod.proj_out_bwd(r["g"], w2, r["dy"])[0]
    for name, got, ref in (("z", z, rz), ("z_pre", z_pre, rpre), ("y", y, ry), ("dx", dx, rdx),
                           ("dg", dg, rdg)):
        e = gu.assert_close(name, gu.to_f64(got[torch.from_numpy(rows).cuda()]), ref, 2e-2, "bf16")
        print(f"\n  {name}: {e[0]:.3e} raw {e[1]:.3e}", end="")
    # Weight-gradient rows: f in fs of dw1 / db1, c in cs of dw2 / db2.
    fs = np.unique(np.r_[0, w1.shape[0] - 1, rng.integers(0, w1.shape[0], 14)])
    cs = np.unique(np.r_[0, D - 1, rng.integers(0, D, 14)])
    x = inputs.stored_f64(P["x"])
    _, rdw1, rdb1 = oracle_mod.proj_in_bwd(x, w1[fs], P["b1"][fs], inputs.stored_f64(P["dz"][:, fs]))
    _, rdw2, rdb2 = oracle_mod.proj_out_bwd(inputs.stored_f64(P["g"]), w2[cs],
                                            inputs.stored_f64(P["dy"][:, cs]))
    for name, got, ref in (("dw1", dw1.cpu().numpy()[fs], rdw1), ("db1", db1.cpu().numpy()[fs], rdb1),
                           ("dw2", dw2.cpu().numpy()[cs], rdw2), ("db2", db2.cpu().numpy()[cs], rdb2)):
        e = gu.assert_close(name, got, ref, 2e-2, "f32")
        print(f"\n  {name}: {e[0]:.3e} raw {e[1]:.3e}", end="")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_full_layer(hs, oracle_mod, dtype):
    """x -> Eq. 1 -> Eq. 2 -> Eq. 3 -> x + f_2(.) and back through the C ABI,
    on a jagged batch with a target-aware sequence and ragged tiles."""
    h, dqk, dv = 2, 64, 32
    D = 128
    lengths = [300, 1, 129, 77]
    batch = inputs.make_batch("training", seed=11, lengths=lengths, num_targets=[40, 0, 0, 5],
                              num_heads=h, d_qk=dqk, d_v=dv, max_seq_len=320, dtype=dtype)
    T = int(batch.seq_offsets[-1])
    P = inputs.make_proj(T, D, h, dqk, dv, dtype=dtype, seed=12)
    rng = np.random.default_rng(13)
    lw = (1.0 + 0.1 * rng.standard_normal(h * dv)).astype(np.float32)
    lb = (0.1 * rng.standard_normal(h * dv)).astype(np.float32)
    d, jd = _dev(P), gu.dev_inputs(batch)
    lwd, lbd = torch.from_numpy(lw).cuda(), torch.from_numpy(lb).cuda()
    N = batch.spec.max_seq_len
    z, z_pre = hs.hstu_proj_in_fwd(d["x"], d["w1"], d["b1"], h, dqk, dv)
    u, v, q, k = hs.split_uvqk(z, h, dqk, dv)
    args = (jd["seq_offsets"], jd["timestamps"], jd["rab_pos"], jd["rab_time"], N)
    attn_out, g, mean, rstd = hs.hstu_layer_fwd(q, k, v, u, *args, num_targets=jd["num_targets"],
                                                ln_weight=lwd, ln_bias=lbd)
    xn = hs.hstu_proj_out_fwd(g, d["w2"], d["b2"], d["x"], h, dqk, dv)
    dxn = d["dy"]
    dg, dw2, db2 = hs.hstu_proj_out_bwd(g, d["w2"], dxn, h, dqk, dv)
    dq, dk, dvv, du, dlw, dlb, drp, drt = hs.hstu_layer_bwd(
        q, k, v, u, attn_out, mean, rstd, dg, *args, num_targets=jd["num_targets"],
        ln_weight=lwd, ln_bias=lbd)
    dx, dw1, db1 = hs.hstu_proj_in_bwd(d["x"], d["w1"], z_pre, du, dvv, dq, dk, h, dqk, dv,
                                       dx_add=dxn)
    torch.cuda.synchronize()
    r = _f64(P)
    oargs = (batch.seq_offsets, N, batch.timestamps, batch.rab_pos, batch.rab_time, r["x"],
             r["w1"], P["b1"], r["w2"], P["b2"], h, dqk, dv)
    # The oracle rounds the tensors the calls hand to each other (Z, its
    # pre-activation, g, dg, dz) to the problem's storage type, as the
    # calls store them; all its arithmetic is fp64.
    f = oracle_mod.layer_full_fwd(*oargs, num_targets=batch.num_targets, ln_weight=lw, ln_bias=lb,
                                  store=dtype)
    b = oracle_mod.layer_full_bwd(*oargs, r["dy"], num_targets=batch.num_targets, ln_weight=lw,
                                  ln_bias=lb, store=dtype)
    tau = _tau(dtype)
    for name, got, ref, store in (
            ("x_next", xn, f["x_next"], dtype), ("dx", dx, b["dx"], dtype),
            ("dw1", dw1, b["dw1"], "f32"), ("db1", db1, b["db1"], "f32"),
            ("dw2", dw2, b["dw2"], "f32"), ("db2", db2, b["db2"], "f32"),
            ("d_ln_weight", dlw, b["d_ln_weight"], "f32"), ("d_ln_bias", dlb, b["d_ln_bias"], "f32"),
            ("d_rab_pos", drp, b["d_rab_pos"], "f32"), ("d_rab_time", drt, b["d_rab_time"], "f32")):
        e = gu.assert_close(name, gu.to_f64(got), ref, tau, store)
        print(f"\n  {name}: {e[0]:.3e} raw {e[1]:.3e}", end="")
