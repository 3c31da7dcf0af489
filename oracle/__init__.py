"""CPU oracle for the HSTU jagged-attention path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU
baseline may import this package.  The product path never routes
through it.

The arithmetic lives in ``hstu_oracle.c`` (plain fp64 loops); this module
compiles it with gcc and marshals numpy arrays through ctypes.  Every
float input is widened to float64 before the call, so the oracle sees
exactly the stored (fp32 or bf16) values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hstu_oracle.c")
_LIB = os.path.join(_HERE, "libhstu_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (never hipcc)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
               "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_time_bucket.argtypes = [i64, i32]
        lib.oracle_time_bucket.restype = i32
        lib.oracle_complete_cumsum.argtypes = [i32, P, P]
        lib.oracle_time_bucketize.argtypes = [i32, P, P, i32, P, P]
        lib.oracle_attn_fwd.argtypes = [i32, P, i32, i32, i32, i32, P, P, P, P,
                                        i32, P, P, P, P]
        lib.oracle_attn_bwd.argtypes = [i32, P, i32, i32, i32, i32, P, P, P, P,
                                        i32, P, P, P, P, P, P, P, P, P]
        lib.oracle_ln_gate.argtypes = [i64, i32, P, P, P, P, f64, P, P, P]
        lib.oracle_ln_gate_bwd.argtypes = [i64, i32, P, P, P, P, P, f64, P, P, P, P]
        lib.oracle_num_threads.restype = i32
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _i64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int64)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def time_bucket(dt: int, num_buckets: int) -> int:
    return int(_load().oracle_time_bucket(int(dt), int(num_buckets)))


def complete_cumsum(x) -> np.ndarray:
    x = _i64(x)
    out = np.empty(len(x) + 1, dtype=np.int64)
    _load().oracle_complete_cumsum(len(x), _p(x), _p(out))
    return out


def time_bucketize(seq_offsets, timestamps, num_buckets):
    """Returns (pair_offsets [B+1], buckets uint8 [sum L_b^2])."""
    offs, ts = _i64(seq_offsets), _i64(timestamps)
    lens = np.diff(offs)
    pair_offsets = complete_cumsum(lens * lens)
    out = np.zeros(int(pair_offsets[-1]), dtype=np.uint8)
    _load().oracle_time_bucketize(len(lens), _p(offs), _p(ts), int(num_buckets),
                                  _p(pair_offsets), _p(out))
    return pair_offsets, out


def _check(offs, ts, nt, N, rp, T):
    """Data preconditions of the definition: offsets start at 0 and do not
    decrease, every L_b <= N (so every signed offset has a rab_pos entry),
    0 <= n_t <= L_b, timestamps in [0, 2^62)."""
    lens = np.diff(offs)
    if offs[0] != 0 or offs[-1] != T or (lens < 0).any():
        raise ValueError("bad seq_offsets")
    if len(lens) and lens.max() > N:
        raise ValueError("sequence longer than max_seq_len")
    if len(rp) != 2 * N - 1:
        raise ValueError("rab_pos must have 2N-1 entries")
    if nt is not None and ((nt < 0).any() or (nt > lens).any()):
        raise ValueError("num_targets out of range")
    if len(ts) != T or (T and (ts.min() < 0 or ts.max() >= (1 << 62))):
        raise ValueError("timestamps out of range")


def attn_fwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time, q, k, v,
             num_targets=None):
    """O [T, h, d_v] = (1/N) sum_j SiLU(q_i.k_j + rab(i,j)) v_j over kept pairs."""
    offs, ts, nt = _i64(seq_offsets), _i64(timestamps), _i64(num_targets)
    q, k, v = _f64(q), _f64(k), _f64(v)
    rp, rt = _f64(rab_pos), _f64(rab_time)
    T, H, dqk = q.shape
    dv = v.shape[2]
    _check(offs, ts, nt, int(max_seq_len), rp, T)
    out = np.empty((T, H, dv), dtype=np.float64)
    _load().oracle_attn_fwd(len(offs) - 1, _p(offs), int(max_seq_len), H, dqk, dv,
                            _p(ts), _p(nt), _p(rp), _p(rt), len(rt),
                            _p(q), _p(k), _p(v), _p(out))
    return out


def attn_bwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time, q, k, v,
             d_out, num_targets=None):
    """Returns (dq, dk, dv, d_rab_pos, d_rab_time) for the loss <O, d_out>."""
    offs, ts, nt = _i64(seq_offsets), _i64(timestamps), _i64(num_targets)
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(d_out)
    rp, rt = _f64(rab_pos), _f64(rab_time)
    T, H, dqk = q.shape
    dvd = v.shape[2]
    _check(offs, ts, nt, int(max_seq_len), rp, T)
    dq = np.empty_like(q)
    dk = np.empty_like(k)
    dv = np.empty_like(v)
    drp = np.empty_like(rp)
    drt = np.empty_like(rt)
    _load().oracle_attn_bwd(len(offs) - 1, _p(offs), int(max_seq_len), H, dqk, dvd,
                            _p(ts), _p(nt), _p(rp), _p(rt), len(rt),
                            _p(q), _p(k), _p(v), _p(do), _p(dq), _p(dk), _p(dv),
                            _p(drp), _p(drt))
    return dq, dk, dv, drp, drt


def ln_gate(x, u, gamma=None, beta=None, eps=1e-5):
    """Y = LayerNorm(x) * u per row; returns (y, mean, rstd)."""
    x = _f64(x)
    T = x.shape[0]
    x = x.reshape(T, -1)
    D = x.shape[1]
    u = _f64(u).reshape(T, D)
    g, b = _f64(gamma), _f64(beta)
    y = np.empty((T, D), dtype=np.float64)
    mean = np.empty(T, dtype=np.float64)
    rstd = np.empty(T, dtype=np.float64)
    _load().oracle_ln_gate(T, D, _p(x), _p(u), _p(g), _p(b), float(eps), _p(y),
                           _p(mean), _p(rstd))
    return y, mean, rstd


def ln_gate_bwd(x, u, dy, gamma=None, beta=None, eps=1e-5):
    """Gradient of <ln_gate(x, u, gamma, beta), dy> (Eq. 3 epilogue);
    returns (dx, du, dgamma, dbeta), dgamma / dbeta None when gamma / beta
    are None."""
    x = _f64(x)
    T = x.shape[0]
    x = x.reshape(T, -1)
    D = x.shape[1]
    u = _f64(u).reshape(T, D)
    dy = _f64(dy).reshape(T, D)
    g, b = _f64(gamma), _f64(beta)
    dx = np.empty((T, D), dtype=np.float64)
    du = np.empty((T, D), dtype=np.float64)
    dg = np.empty(D, dtype=np.float64) if g is not None else None
    db = np.empty(D, dtype=np.float64) if b is not None else None
    _load().oracle_ln_gate_bwd(T, D, _p(x), _p(u), _p(dy), _p(g), _p(b), float(eps), _p(dx),
                               _p(du), _p(dg), _p(db))
    return dx, du, dg, db


def mfalcon_fwd(seq_offsets, num_targets, b_m, max_seq_len, timestamps, rab_pos, rab_time,
                q, k, v):
    """Algorithm 1 (M-FALCON) for one attention layer.  Sequence b of the
    merged batch holds its n_b prefix tokens followed by its m_b candidates
    (m_b = num_targets[b]).  The candidates are taken b_m at a time: pass i
    runs the target-aware attention (candidates see the prefix and
    themselves, never each other) over prefix ++ candidates
    [i b_m, min((i+1) b_m, m_b)) of every sequence, and keeps the outputs of
    those candidates.  Returns O of the candidate rows, in the order of the
    merged batch ([sum m_b, h, d_v]); the prefix rows are not outputs."""
    offs, nt, ts = _i64(seq_offsets), _i64(num_targets), _i64(timestamps)
    q, k, v = _f64(q), _f64(k), _f64(v)
    B = len(offs) - 1
    if b_m < 1:
        raise ValueError("b_m must be >= 1")
    lens = np.diff(offs)
    nh = lens - nt
    cand_start = np.concatenate([[0], np.cumsum(nt)])
    out = np.full((int(cand_start[-1]), q.shape[1], v.shape[2]), np.nan)
    passes = (int(nt.max()) + b_m - 1) // b_m if B and nt.max() > 0 else 0
    for i in range(passes):
        rows, keep, counts = [], [], []
        for b in range(B):
            c0, c1 = min(i * b_m, int(nt[b])), min((i + 1) * b_m, int(nt[b]))
            rows.append(np.arange(offs[b], offs[b] + nh[b]))
            rows.append(np.arange(offs[b] + nh[b] + c0, offs[b] + nh[b] + c1))
            keep.append(cand_start[b] + np.arange(c0, c1))
            counts.append(c1 - c0)
        counts = np.asarray(counts, dtype=np.int64)
        sub_offs = np.concatenate([[0], np.cumsum(nh + counts)])
        r = np.concatenate(rows)
        o = attn_fwd(sub_offs, max_seq_len, ts[r], rab_pos, rab_time, q[r], k[r], v[r],
                     num_targets=counts)
        # Candidate rows of the pass, in sequence order.
        sel = np.concatenate([np.arange(sub_offs[b] + nh[b], sub_offs[b + 1]) for b in range(B)])
        out[np.concatenate(keep)] = o[sel]
    return out


# ------------------------------------------------ projections (Eq. 1, Eq. 3)
# f_1 and f_2 are single linear layers (Sec. 3.1, after Eq. 3): a weight
# matrix stored [out][in] and a bias.  Plain definitions in fp64 numpy.

def _silu(x):
    return x / (1.0 + np.exp(-x))


def _silu_grad(x):
    s = 1.0 / (1.0 + np.exp(-x))
    return s * (1.0 + x * (1.0 - s))


def proj_in_fwd(x, w1, b1=None):
    """Eq. 1: pre = x W1^T + b1, Z = SiLU(pre) per token row, Z = [U | V | Q | K]
    (the split of the fused projection output, notation table entry for
    Split).  x [T, D], w1 [F, D], b1 [F].  Returns (Z, pre), both [T, F]."""
    x, w1 = _f64(x), _f64(w1)
    pre = x @ w1.T
    if b1 is not None:
        pre = pre + _f64(b1)[None, :]
    return _silu(pre), pre


def split_uvqk(z, num_heads, d_qk, d_v):
    """U, V, Q, K views of Z [T, F] as [T, h, d]: U first, then V, Q, K."""
    T = z.shape[0]
    hv, hq = num_heads * d_v, num_heads * d_qk
    u = z[:, :hv].reshape(T, num_heads, d_v)
    v = z[:, hv:2 * hv].reshape(T, num_heads, d_v)
    q = z[:, 2 * hv:2 * hv + hq].reshape(T, num_heads, d_qk)
    k = z[:, 2 * hv + hq:2 * hv + 2 * hq].reshape(T, num_heads, d_qk)
    return u, v, q, k


def proj_in_bwd(x, w1, b1, dz, pre=None):
    """Gradient of <Z, dZ> for Z = SiLU(x W1^T + b1): returns (dx, dw1, db1).
    ``pre`` (optional): the pre-activation to differentiate SiLU at, e.g.
    as the layer stored it; recomputed from x, w1, b1 when None."""
    x, w1, dz = _f64(x), _f64(w1), _f64(dz)
    if pre is None:
        _, pre = proj_in_fwd(x, w1, b1)
    dpre = dz * _silu_grad(_f64(pre))
    return dpre @ w1, dpre.T @ x, dpre.sum(axis=0)


def proj_out_fwd(g, w2, b2=None, residual=None):
    """Eq. 3's f_2 plus the residual connection between layers (Sec. 3.1):
    Y = g W2^T + b2 (+ residual).  g [T, h d_v], w2 [D, h d_v]."""
    g, w2 = _f64(g), _f64(w2)
    y = g @ w2.T
    if b2 is not None:
        y = y + _f64(b2)[None, :]
    if residual is not None:
        y = y + _f64(residual)
    return y


def proj_out_bwd(g, w2, dy):
    """Gradient of <Y, dY> for Y = g W2^T + b2: returns (dg, dw2, db2)."""
    g, w2, dy = _f64(g), _f64(w2), _f64(dy)
    return dy @ w2, dy.T @ g, dy.sum(axis=0)


def round_store(a, store):
    """Storage rounding of an interface tensor: None keeps fp64, "f32" rounds
    to float32, "bf16" to bfloat16 (round to nearest even, via float32)."""
    if store is None:
        return a
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    if store == "f32":
        return a32.astype(np.float64)
    if store != "bf16":
        raise ValueError(f"unknown storage type {store}")
    u = a32.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def layer_full_fwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time, x, w1, b1, w2, b2,
                   num_heads, d_qk, d_v, num_targets=None, ln_weight=None, ln_bias=None,
                   eps=1e-5, store=None):
    """One whole HSTU layer with its residual (Sec. 3.1): Eq. 1, Eq. 2, Eq. 3,
    x_next = x + f_2(Norm(A V) * U).  Returns the intermediates and x_next.
    ``store``: storage type of the tensors a layer built from separate calls
    hands from one call to the next (Z and its pre-activation, the gated
    output g); they are rounded to it, everything else stays fp64."""
    x = _f64(x)
    T = x.shape[0]
    z, pre = proj_in_fwd(x, w1, b1)
    z, pre = round_store(z, store), round_store(pre, store)
    u, v, q, k = split_uvqk(z, num_heads, d_qk, d_v)
    o = attn_fwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time, q, k, v,
                 num_targets=num_targets)
    g, mean, rstd = ln_gate(o.reshape(T, -1), u.reshape(T, -1), ln_weight, ln_bias, eps)
    g = round_store(g, store)
    xn = proj_out_fwd(g, w2, b2, residual=x)
    return {"z": z, "pre": pre, "o": o, "g": g, "mean": mean, "rstd": rstd, "x_next": xn}


def layer_full_bwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time, x, w1, b1, w2, b2,
                   num_heads, d_qk, d_v, d_x_next, num_targets=None, ln_weight=None,
                   ln_bias=None, eps=1e-5, store=None):
    """Gradients of <x_next, d_x_next> for layer_full_fwd: dx (residual
    included), dw1, db1, dw2, db2, d_ln_weight, d_ln_bias, d_rab_pos,
    d_rab_time, and the intermediate gradients dg, do, dz.  With ``store``
    the gradients handed between calls (dg, dz) are rounded to it as well
    and SiLU is differentiated at the stored pre-activation."""
    x = _f64(x)
    T = x.shape[0]
    f = layer_full_fwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time, x, w1, b1, w2, b2,
                       num_heads, d_qk, d_v, num_targets, ln_weight, ln_bias, eps, store)
    dxn = _f64(d_x_next)
    dg, dw2, db2 = proj_out_bwd(f["g"], w2, dxn)
    dg = round_store(dg, store)
    u, v, q, k = split_uvqk(f["z"], num_heads, d_qk, d_v)
    do, du, dlw, dlb = ln_gate_bwd(f["o"].reshape(T, -1), u.reshape(T, -1), dg, ln_weight,
                                   ln_bias, eps)
    dq, dk, dv, drp, drt = attn_bwd(seq_offsets, max_seq_len, timestamps, rab_pos, rab_time,
                                    q, k, v, do.reshape(T, num_heads, d_v),
                                    num_targets=num_targets)
    dz = np.concatenate([du.reshape(T, -1), dv.reshape(T, -1), dq.reshape(T, -1),
                         dk.reshape(T, -1)], axis=1)
    dz = round_store(dz, store)
    dx, dw1, db1 = proj_in_bwd(x, w1, b1, dz, pre=f["pre"])
    return {"dx": dx + dxn, "dw1": dw1, "db1": db1, "dw2": dw2, "db2": db2,
            "d_ln_weight": dlw, "d_ln_bias": dlb, "d_rab_pos": drp, "d_rab_time": drt,
            "dg": dg, "do": do, "dz": dz}


# -------------------------------------------- Stochastic Length (Eq. 4)
# Random draws are inputs: u_keep [B] ~ U[0, 1) decides whether a long
# history is kept whole; e_rand [T] ~ Exp(1) per token drives the random
# and feature-weighted selections.

SL_GREEDY, SL_RANDOM, SL_WEIGHTED = 0, 1, 2


def sl_subseq_len(max_seq_len, alpha):
    """L = N_c^(alpha/2) of Eq. 4 (floor, with N_c the maximum length): the
    length of the subsequence, and the history length up to which a
    sequence is always kept whole (n <= N_c^(alpha/2) iff n <= L for an
    integer n)."""
    return int(np.floor(float(max_seq_len) ** (alpha / 2.0) + 1e-9))


def sl_keep_numerator(max_seq_len, alpha):
    """N_c^alpha of Eq. 4: a history of n > L tokens is kept whole with
    probability N_c^alpha / n^2 (fp64)."""
    return float(max_seq_len) ** float(alpha)


def _sl_keys(ts, e, mode):
    """Selection keys of one history (smaller = chosen first), following the
    subsequence selection appendix: greedy takes the most recent items
    (f_i = t_n - t_i, t_n the latest timestamp); random takes items
    uniformly (exponential-race keys E_i); feature-weighted takes items with
    probability proportional to w_i = 1 - f_i / sum_k f_k, by
    exponential-race keys E_i / w_i, ordered identically as E_i / (F - f_i)
    with F = sum_k f_k (Efraimidis and Spirakis' weighted sampling without
    replacement).  Greedy keys are integers; the others fp64."""
    f = [int(ts.max()) - int(t) for t in ts] if len(ts) else []
    if mode == SL_GREEDY:
        return f
    e = [float(x) if x > 0 else 0.0 for x in e]  # an Exp(1) draw is >= 0
    if mode == SL_RANDOM:
        return e
    F = sum(f)
    if F >= (1 << 53):
        raise ValueError("feature-weighted selection needs the elapsed-time sum below 2^53")
    keys = []
    for ei, fi in zip(e, f):
        den = F - fi
        if F == 0:
            keys.append(float(ei))      # all weights equal
        elif den == 0:
            keys.append(float("inf"))   # weight 0: never chosen before the others
        else:
            keys.append(float(ei) / float(den))
    return keys


def stochastic_length(seq_offsets, timestamps, num_targets, subseq_len, keep_num, mode, u_keep,
                      e_rand):
    """Eq. 4 per sequence: with n_h history tokens (the candidates, if any,
    are always kept after them), keep the sequence whole if n_h <= L or
    u_keep[b] < keep_num / n_h^2 (keep_num = N_c^alpha, fp64); otherwise
    keep L = subseq_len history tokens chosen by the
    selection keys (the L smallest; equal keys: the later token first),
    in their original order.  Returns (new_offsets [B+1], gather [T'] of
    original token indices)."""
    offs = _i64(seq_offsets)
    ts = _i64(timestamps)
    B = len(offs) - 1
    L = int(subseq_len)
    if L < 1:
        raise ValueError("subseq_len must be >= 1")
    keep_num = float(keep_num)
    u = np.asarray(u_keep, dtype=np.float64)
    e = None if e_rand is None else np.asarray(e_rand, dtype=np.float64)
    gather, lens = [], []
    for b in range(B):
        o, n = int(offs[b]), int(offs[b + 1] - offs[b])
        nt = 0 if num_targets is None else int(num_targets[b])
        nh = n - nt
        if nh <= L or u[b] < keep_num / float(nh * nh):
            sel = list(range(o, o + n))
        else:
            keys = _sl_keys(ts[o:o + nh], None if e is None else e[o:o + nh], mode)
            order = sorted(range(nh), key=lambda i: (keys[i], -i))
            sel = [o + i for i in sorted(order[:L])] + list(range(o + nh, o + n))
        gather += sel
        lens.append(len(sel))
    new_offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return new_offs, np.asarray(gather, dtype=np.int64)


def sl_sparsity(lengths, max_seq_len):
    """The two metrics of the appendix on the impact of Stochastic Length on
    sequence sparsity.  sparsity = 1 - mean length / maximum length N.
    s2 is the same measure taken over the attention matrices: the share of
    the B padded N x N score matrices that lies outside the sequences,
    1 - sum_b n_b^2 / (B N^2).  The appendix's prose words s2 as the
    complement of the attention matrix's sparsity, but every pair of its
    printed tables (60-day and 90-day histories) has s2 above sparsity,
    which only this form admits (for n_b <= N it lies between sparsity and
    1 - (1 - sparsity)^2), so the tables decide."""
    n = np.asarray(lengths, dtype=np.float64)
    N = float(max_seq_len)
    return 1.0 - n.mean() / N, 1.0 - float((n * n).sum() / (len(n) * N * N))
