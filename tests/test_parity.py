"""GPU parity: the HIP path through the C ABI against the fp64 oracle on
the same seeded inputs.  Criterion per output tensor (over the jagged
rows that exist): max |gpu - oracle| <= tau * RMS(oracle), tau = 1e-4 for
the fp32 path and 2e-2 for bf16; time buckets and offsets bit-exact.

Stored outputs carry their storage type's own rounding (half an ulp:
2^-8 |x| for bf16) on top of the computation's error; the criterion
takes that term out per element: max_i (|gpu_i - ref_i| - u|ref_i|)_+ <=
tau * RMS(ref).

Small shapes compare every element and span several tiles plus ragged
tails; the five workload shapes run at full size, compared in full
where the oracle finishes in seconds and otherwise on whole sampled
sequences (sequences are independent, so a sub-batch of them is an
exact oracle for those rows) plus properties of the full batch."""
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


def _check_fwd(hs, oracle, batch):
    d = gu.dev_inputs(batch)
    out = gu.gpu_fwd(hs, d, batch)
    torch.cuda.synchronize()
    ref = gu.oracle_fwd(oracle, batch)
    e = gu.assert_close("O", gu.to_f64(out), ref, gu.tol(batch), batch.spec.dtype)
    print(f"\n  O err {e[0]:.3e} raw {e[1]:.3e}")
    return e


def _check_bwd(hs, oracle, batch):
    d = gu.dev_inputs(batch)
    got = gu.gpu_bwd(hs, d, batch)
    torch.cuda.synchronize()
    ref = gu.oracle_bwd(oracle, batch)
    errs = {}
    for name, g, r in zip(("dq", "dk", "dv", "d_rab_pos", "d_rab_time"), got, ref):
        store = "f32" if name.startswith("d_rab") else batch.spec.dtype
        errs[name] = gu.assert_close(name, gu.to_f64(g), r, gu.tol(batch), store)
        print(f"  {name} err {errs[name][0]:.3e} raw {errs[name][1]:.3e}")
    return errs


SMALL = [
    # (lengths, h, d_qk, d_v, N, num_targets)
    ((1, 37, 200, 129, 300, 0, 64), 2, 64, 64, 320, None),
    ((300, 5, 257), 1, 128, 128, 300, None),
    ((33, 160, 95), 3, 32, 32, 160, None),
    ((130, 77), 2, 32, 128, 160, None),
    ((130, 77), 2, 128, 64, 160, None),
    ((250, 190, 64), 2, 128, 128, 256, (70, 190, 1)),   # target-aware, incl. all-candidate
    ((129, 128, 127), 1, 64, 64, 129, (3, 0, 127)),
    # N too large for the backward's LDS position accumulator: global-atomic path
    ((300, 100), 1, 128, 128, 12000, None),
]


def test_bwd_bf16_dq_dk_dv_deterministic(hs):
    """bf16 hstu_attn_bwd sums dQ from per-key-block partials in a fixed
    order (no atomics), so dQ, dK and dV are bitwise reproducible; the
    bias gradients use atomics and are only compared within tolerance."""
    for lengths, h, dqk, dv, N in (((1, 37, 200, 129, 300, 0, 64), 2, 64, 64, 320),
                                   ((700, 5, 513), 3, 128, 128, 768)):
        batch = inputs.make_batch(3, seed=11, lengths=lengths, num_heads=h, d_qk=dqk,
                                  d_v=dv, max_seq_len=N, dtype="bf16")
        d = gu.dev_inputs(batch)
        a = gu.gpu_bwd(hs, d, batch)
        b = gu.gpu_bwd(hs, d, batch)
        torch.cuda.synchronize()
        for name, x, y in zip(("dq", "dk", "dv"), a[:3], b[:3]):
            assert torch.equal(x, y), f"{name} differs between two identical calls"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_parity(hs, oracle_mod, dtype, case):
    lengths, h, dqk, dv, N, nt = SMALL[case]
    batch = inputs.make_batch(3, seed=100 + case, lengths=lengths, num_heads=h, d_qk=dqk, d_v=dv,
                              max_seq_len=N, dtype=dtype, num_targets=nt)
    _check_fwd(hs, oracle_mod, batch)
    _check_bwd(hs, oracle_mod, batch)


def test_bwd_bf16_reduce_two_rounds(hs, oracle_mod):
    """Every output of a 2200-token sequence (18 key blocks of 128, so the
    bf16 dQ reduce sums its partial blocks over two rounds of loads) and a
    ragged 45-token one.  bf16 only: the fp32 kernels have no reduce, and
    at this length their time-table gradient (sums of ~2.4M pairs per
    bucket, with heavy cancellation) sits at 1.3e-4 of its RMS."""
    batch = inputs.make_batch(3, seed=150, lengths=(2200, 45), num_heads=1, d_qk=32, d_v=32,
                              max_seq_len=2200, dtype="bf16")
    _check_fwd(hs, oracle_mod, batch)
    _check_bwd(hs, oracle_mod, batch)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_small_parity_wide_timestamps(hs, oracle_mod, dtype):
    """Timestamps spanning more than 2^31 (and unsorted within a sequence):
    the exact 64-bit time-bucket path of the kernels."""
    rng = np.random.default_rng(17)
    lengths = (200, 77, 130)
    T = sum(lengths)
    ts = rng.integers(0, 1 << 60, size=T)
    ts[200:277] = np.sort(ts[200:277])
    batch = inputs.make_batch(3, seed=31, lengths=lengths, num_heads=2, d_qk=64, d_v=64,
                              max_seq_len=256, dtype=dtype, timestamps=ts)
    _check_fwd(hs, oracle_mod, batch)
    _check_bwd(hs, oracle_mod, batch)


def test_workload_tiny_full(hs, oracle_mod):
    """fp32 tiny workload (B=4, h=2, d=32, N=128): every output in full."""
    batch = inputs.make_batch("tiny")
    _check_fwd(hs, oracle_mod, batch)
    _check_bwd(hs, oracle_mod, batch)


def test_workload_medium_full(hs, oracle_mod):
    """bf16 medium workload (B=32 Zipf lengths, h=4, d=64, N=1024), forward in full."""
    batch = inputs.make_batch("medium")
    _check_fwd(hs, oracle_mod, batch)


def _sampled(hs, oracle_mod, batch, seqs, backward):
    """Full-size batch on the GPU; the oracle on the sampled sequences."""
    d = gu.dev_inputs(batch)
    out = gu.to_f64(gu.gpu_fwd(hs, d, batch))
    sub = gu.sub_batch(batch, seqs)
    rows = gu.token_rows(batch, seqs)
    tau = gu.tol(batch)
    st = batch.spec.dtype
    gu.assert_close("O", out[rows], gu.oracle_fwd(oracle_mod, sub), tau, st)
    if backward:
        g = [gu.to_f64(x) for x in gu.gpu_bwd(hs, d, batch)]
        r = gu.oracle_bwd(oracle_mod, sub)
        for name, gi, ri in zip(("dq", "dk", "dv"), g[:3], r[:3]):
            gu.assert_close(name, gi[rows], ri, tau, st)
        # bias gradients of the sampled sequences alone, same launch shape
        ds = gu.dev_inputs(sub)
        gs = [gu.to_f64(x) for x in gu.gpu_bwd(hs, ds, sub)]
        gu.assert_close("d_rab_pos", gs[3], r[3], tau)
        gu.assert_close("d_rab_time", gs[4], r[4], tau)
        # full-batch properties: both tables sum to the same total; offsets
        # j > i and unpopulated buckets get exactly zero
        N = batch.spec.max_seq_len
        drp, drt = g[3], g[4]
        assert np.all(drp[N:] == 0.0)
        tot = np.abs(drp).sum()
        assert abs(drp.sum() - drt.sum()) <= 1e-3 * tot
        assert np.all(drt[64:] == 0.0)


def test_workload_training_sampled(hs, oracle_mod):
    """bf16 training workload (B=64, h=8, d=64, N=4096) at full size."""
    batch = inputs.make_batch("training")
    L = batch.lengths
    seqs = [int(np.argmax(L)), int(np.argmin(L)), 7]
    _sampled(hs, oracle_mod, batch, seqs, backward=True)


def test_workload_long_sampled(hs, oracle_mod):
    """bf16 long workload (B=8, L in [4096, 8192], h=4, d=128, N=8192) at full size."""
    batch = inputs.make_batch("long")
    _sampled(hs, oracle_mod, batch, [int(np.argmin(batch.lengths))], backward=True)


def test_workload_target_sampled(hs, oracle_mod):
    """bf16 target-aware workload (16 x (2048 + 1024), h=4, d=128, N=3072)."""
    batch = inputs.make_batch("target")
    _sampled(hs, oracle_mod, batch, [0, 11], backward=False)


def test_bucketize_bit_exact(hs, oracle_mod):
    """Standalone bucketisation equals the oracle byte for byte, including
    empty sequences, length 1, the clamp (B_t = 9), a ragged total, rows
    past one 4096-column slab and spans beyond 2^31 (the 64-bit path)."""
    rng = np.random.default_rng(9)
    lens = np.array([0, 1, 17, 300, 0, 45, 1024, 3, 5000, 4100], dtype=np.int64)
    offs = np.concatenate([[0], np.cumsum(lens)])
    T = int(offs[-1])
    ts = np.empty(T, dtype=np.int64)
    for b in range(len(lens)):
        s, e = offs[b], offs[b + 1]
        ts[s:e] = rng.integers(0, 1 << 40) + np.cumsum(rng.integers(0, 1 << int(rng.integers(1, 30)), e - s))
    ts[offs[6]:offs[7]] = rng.permutation(ts[offs[6]:offs[7]])   # unsorted sequence
    # two column slabs on the 64-bit path (span ~ 2^41)
    ts[offs[9]:offs[10]] = (1 << 50) + np.cumsum(rng.integers(0, 1 << 30, int(lens[9])))
    for nb in (128, 9):
        po_ref, bk_ref = oracle_mod.time_bucketize(offs, ts, nb)
        so = torch.from_numpy(offs).cuda()
        po = hs.hstu_pair_offsets(so)
        assert np.array_equal(po.cpu().numpy(), po_ref)
        bk = hs.hstu_time_bucketize(so, torch.from_numpy(ts).cuda(), nb, pair_offsets=po)
        assert np.array_equal(bk.cpu().numpy(), bk_ref)


def test_bucketize_long_workload(hs, oracle_mod):
    """Standalone bucketisation of the long workload (302 MB of buckets),
    bit-exact against the oracle."""
    batch = inputs.make_batch("long")
    po_ref, bk_ref = oracle_mod.time_bucketize(batch.seq_offsets, batch.timestamps, 128)
    so = torch.from_numpy(batch.seq_offsets).cuda()
    bk = hs.hstu_time_bucketize(so, torch.from_numpy(batch.timestamps).cuda(), 128)
    assert bk.numel() == bk_ref.size
    assert torch.equal(bk.cpu(), torch.from_numpy(bk_ref))


def test_complete_cumsum(hs, oracle_mod):
    rng = np.random.default_rng(2)
    for n in (1, 5, 1023, 1024, 1025, 5000):
        x = rng.integers(0, 1 << 40, size=n)
        got = hs.hstu_complete_cumsum(torch.from_numpy(x).cuda()).cpu().numpy()
        assert np.array_equal(got, oracle_mod.complete_cumsum(x))


def _ln_params(D, seed):
    rng = np.random.default_rng(seed)
    w = (1 + 0.1 * rng.standard_normal(D)).astype(np.float32)
    b = (0.1 * rng.standard_normal(D)).astype(np.float32)
    return w, b


def _ln_tol(dtype):
    # mean / rstd of the stored attention output: exact up to fp32 for the
    # fp32 path; the bf16 path normalises the bf16-rounded output
    return 1e-5 if dtype == "f32" else 2e-2


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_layer_fwd_epilogue(hs, oracle_mod, dtype):
    """hstu_layer_fwd = attention then LayerNorm(A V) (.) U (Eq. 3), with a
    random affine; attn_out, y, mean and rstd against the oracle's own
    attention output and epilogue."""
    batch = inputs.make_batch(2, seed=21, lengths=(300, 1, 129, 64), num_heads=4, d_qk=64, d_v=64,
                              max_seq_len=300, dtype=dtype)
    d = gu.dev_inputs(batch)
    D = 4 * 64
    w, b = _ln_params(D, 3)
    ao, y, mu, rs = hs.hstu_layer_fwd(d["q"], d["k"], d["v"], d["u"], d["seq_offsets"],
                                      d["timestamps"], d["rab_pos"], d["rab_time"], 300,
                                      ln_weight=torch.from_numpy(w).cuda(),
                                      ln_bias=torch.from_numpy(b).cuda(), ln_eps=1e-5)
    torch.cuda.synchronize()
    tau = gu.tol(batch)
    ref_o = gu.oracle_fwd(oracle_mod, batch).reshape(-1, D)
    gu.assert_close("attn_out", gu.to_f64(ao), ref_o, tau, dtype)
    ry, rmu, rrs = oracle_mod.ln_gate(ref_o, batch.f64("u").reshape(-1, D), w, b, 1e-5)
    gu.assert_close("y", gu.to_f64(y), ry, tau, dtype)
    gu.assert_close("mean", gu.to_f64(mu), rmu, _ln_tol(dtype))
    gu.assert_close("rstd", gu.to_f64(rs), rrs, _ln_tol(dtype))


def test_layer_fwd_training_workload(hs, oracle_mod):
    """Epilogue at the training workload's full size (T=60383, D=512); the
    oracle on three whole sampled sequences."""
    batch = inputs.make_batch("training")
    d = gu.dev_inputs(batch)
    ao, y, mu, rs = hs.hstu_layer_fwd(d["q"], d["k"], d["v"], d["u"], d["seq_offsets"],
                                      d["timestamps"], d["rab_pos"], d["rab_time"], 4096)
    torch.cuda.synchronize()
    D = 512
    L = batch.lengths
    seqs = [int(np.argmax(L)), int(np.argmin(L)), 7]
    sub = gu.sub_batch(batch, seqs)
    rows = gu.token_rows(batch, seqs)
    ref_o = gu.oracle_fwd(oracle_mod, sub).reshape(-1, D)
    ry, rmu, rrs = oracle_mod.ln_gate(ref_o, sub.f64("u").reshape(-1, D))
    gu.assert_close("y", gu.to_f64(y)[rows], ry, 2e-2, "bf16")
    gu.assert_close("rstd", gu.to_f64(rs)[rows], rrs, 2e-2)


def _layer_bwd_check(hs, oracle_mod, batch, seqs=None, affine=True):
    """hstu_layer_fwd then hstu_layer_bwd with dY = the batch's seeded dO
    draw, against the oracle chain: its own attention output, the
    epilogue backward (dU, d attn_out, d gamma, d beta), then the
    attention backward from that d attn_out.  With `seqs`, the oracle runs
    on those whole sequences and parameter gradients are checked on a
    launch over them alone."""
    N = batch.spec.max_seq_len
    H, dv = batch.spec.num_heads, batch.spec.d_v
    D = H * dv
    dt = batch.spec.dtype
    tau = gu.tol(batch)
    w, b = _ln_params(D, 5)

    def gpu(bt):
        d = gu.dev_inputs(bt)
        wt = torch.from_numpy(w).cuda() if affine else None
        bb = torch.from_numpy(b).cuda() if affine else None
        ao, y, mu, rs = hs.hstu_layer_fwd(d["q"], d["k"], d["v"], d["u"], d["seq_offsets"],
                                          d["timestamps"], d["rab_pos"], d["rab_time"], N,
                                          num_targets=d["num_targets"], ln_weight=wt,
                                          ln_bias=bb, ln_eps=1e-5)
        dy = d["do"].reshape(-1, D)
        g = hs.hstu_layer_bwd(d["q"], d["k"], d["v"], d["u"], ao, mu, rs, dy, d["seq_offsets"],
                              d["timestamps"], d["rab_pos"], d["rab_time"], N,
                              num_targets=d["num_targets"], ln_weight=wt, ln_bias=bb,
                              want_ln_grads=True)
        torch.cuda.synchronize()
        return [None if x is None else gu.to_f64(x) for x in g]

    def oracle(bt):
        o = gu.oracle_fwd(oracle_mod, bt).reshape(-1, D)
        dx, du, dg, db = oracle_mod.ln_gate_bwd(o, bt.f64("u").reshape(-1, D),
                                                bt.f64("do").reshape(-1, D),
                                                w if affine else np.ones(D),
                                                b if affine else np.zeros(D), 1e-5)
        T = o.shape[0]
        dq, dk, dvv, drp, drt = oracle_mod.attn_bwd(
            bt.seq_offsets, N, bt.timestamps, bt.rab_pos, bt.rab_time, bt.f64("q"),
            bt.f64("k"), bt.f64("v"), dx.reshape(T, H, dv), num_targets=bt.num_targets)
        return dq, dk, dvv, du, dg, db, drp, drt

    got = gpu(batch)
    sub = batch if seqs is None else gu.sub_batch(batch, seqs)
    ref = oracle(sub)
    rows = slice(None) if seqs is None else gu.token_rows(batch, seqs)
    for name, gi, ri in zip(("dq", "dk", "dv", "du"), got[:4], ref[:4]):
        e = gu.assert_close(name, gi.reshape(gi.shape[0], -1)[rows], ri.reshape(ri.shape[0], -1),
                            tau, dt)
        print(f"  {name} err {e[0]:.3e} raw {e[1]:.3e}")
    gs = got if seqs is None else gpu(sub)
    for name, gi, ri in zip(("d_ln_weight", "d_ln_bias", "d_rab_pos", "d_rab_time"),
                            gs[4:], ref[4:]):
        e = gu.assert_close(name, gi, ri, tau)
        print(f"  {name} err {e[0]:.3e} raw {e[1]:.3e}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("affine", [True, False])
def test_layer_bwd_small(hs, oracle_mod, dtype, affine):
    """hstu_layer_bwd (epilogue backward then attention backward) on a
    small jagged batch with ragged tails, an empty and a length-1 sequence,
    candidates, and both affine settings."""
    batch = inputs.make_batch(2, seed=23, lengths=(300, 0, 1, 129, 70), num_targets=(0, 0, 0, 17, 5),
                              num_heads=4, d_qk=64, d_v=64, max_seq_len=300, dtype=dtype)
    _layer_bwd_check(hs, oracle_mod, batch, affine=affine)


def test_layer_bwd_training_sampled(hs, oracle_mod):
    """hstu_layer_bwd at the training workload's full size (T=60383, h=8,
    d=64, N=4096); the oracle on three whole sequences."""
    batch = inputs.make_batch("training")
    L = batch.lengths
    _layer_bwd_check(hs, oracle_mod, batch, seqs=[int(np.argmax(L)), int(np.argmin(L)), 7])