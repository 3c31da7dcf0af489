"""Helpers shared by the GPU parity tests: move a seeded Batch to the
device, run the C ABI through the binding, run the oracle on the same
stored values, and compare with the max-abs / RMS criterion."""
import numpy as np
import torch

from paper_2402_17152_amd import inputs


def dev_inputs(batch: inputs.Batch):
    return inputs.to_device(batch)


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def tol(batch) -> float:
    return 1e-4 if batch.spec.dtype == "f32" else 2e-2


# Relative rounding bound of the output's own storage type: a value
# stored in bf16 carries up to half an ulp, 2^-8 |x|, whatever the
# arithmetic before it; fp32 storage 2^-24 |x|.
STORE_ROUNDING = {"bf16": 2.0 ** -8, "f32": 2.0 ** -24}


def rel_err(got: np.ndarray, ref: np.ndarray, store_u: float = 0.0) -> float:
    """max_i max(0, |got_i - ref_i| - store_u |ref_i|) / RMS(ref): the error
    of the computation beyond the rounding of the stored output."""
    got = np.asarray(got, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    if not ref.size:
        return 0.0
    err = float(np.max(np.maximum(np.abs(got - ref) - store_u * np.abs(ref), 0.0)))
    if rms == 0.0:
        return 0.0 if err == 0.0 else float("inf")
    return err / rms


def _round_store(ref, store):
    import oracle
    return oracle.round_store(ref, store)


def assert_close(name, got, ref, tau, store="f32"):
    """Criterion: max_i (|got_i - ref_i| - u |ref_i|)_+ <= tau * RMS(ref), u
    the storage rounding of `store`, and a guard on taking that term out:
    if the plain max|err| / RMS exceeds tau, the oracle's own values
    rounded to the storage type ("floor") must reach at least tau / 2, i.e.
    storage rounding alone uses half the budget or more on that tensor.
    Everywhere else the plain bound applies.  `ref` must be the oracle's
    (unrounded) result.  Returns (criterion, raw)."""
    e = rel_err(got, ref, STORE_ROUNDING[store])
    raw = rel_err(got, ref, 0.0)
    assert e <= tau, f"{name}: (max|err| - rounding)/RMS = {e:.3e} > {tau:.1e} (raw {raw:.3e})"
    if raw > tau:
        floor = rel_err(_round_store(np.asarray(ref, dtype=np.float64), store), ref, 0.0)
        assert floor >= tau / 2, (f"{name}: raw max|err|/RMS = {raw:.3e} > {tau:.1e} while the "
                                  f"oracle rounded to {store} uses only {floor:.3e}")
        print(f"  [{name}: raw {raw:.3e} > {tau:.0e}; oracle rounded to {store}: {floor:.3e}]")
    return e, raw


def gpu_fwd(hs, d, batch):
    return hs.hstu_attn_fwd(d["q"], d["k"], d["v"], d["seq_offsets"], d["timestamps"],
                            d["rab_pos"], d["rab_time"], batch.spec.max_seq_len,
                            num_targets=d["num_targets"])


def gpu_bwd(hs, d, batch):
    return hs.hstu_attn_bwd(d["q"], d["k"], d["v"], d["do"], d["seq_offsets"], d["timestamps"],
                            d["rab_pos"], d["rab_time"], batch.spec.max_seq_len,
                            num_targets=d["num_targets"])


def oracle_fwd(oracle, batch):
    return oracle.attn_fwd(batch.seq_offsets, batch.spec.max_seq_len, batch.timestamps,
                           batch.rab_pos, batch.rab_time, batch.f64("q"), batch.f64("k"),
                           batch.f64("v"), num_targets=batch.num_targets)


def oracle_bwd(oracle, batch):
    return oracle.attn_bwd(batch.seq_offsets, batch.spec.max_seq_len, batch.timestamps,
                           batch.rab_pos, batch.rab_time, batch.f64("q"), batch.f64("k"),
                           batch.f64("v"), batch.f64("do"), num_targets=batch.num_targets)


def sub_batch(batch: inputs.Batch, seqs) -> inputs.Batch:
    """Sequences are independent, so every per-token output of the
    sub-batch equals the full batch's rows."""
    return inputs.sub_batch(batch, seqs)


def token_rows(batch: inputs.Batch, seqs):
    offs = batch.seq_offsets
    return np.concatenate([np.arange(offs[b], offs[b + 1]) for b in seqs])
