"""Dense per-sequence brute force in NumPy (fp64), used to pin the oracle
and, with `rnd`, to emulate the rounding of the matrix-core operands.  It
is written in matrix form, independently of the oracle's loops: an
explicit L x L mask built the way Algorithm 1 builds it (lower-triangular
matrix, then candidate rows/columns cleared off the diagonal), the full
score matrix, and the backward as matrix products."""
import numpy as np


def mask_alg1(L, n_t):
    """Algorithm 1: start from the lower-triangular matrix L_{n+b_m}
    (diagonal kept), then forbid (i, j) with i, j >= n and i != j."""
    m = np.tril(np.ones((L, L), dtype=bool))
    n = L - n_t
    for i in range(n, L):
        for j in range(n, L):
            if i != j:
                m[i, j] = False
    return m


def bucket_matrix(ts, num_buckets):
    d = np.abs(ts[:, None].astype(object) - ts[None, :].astype(object))
    out = np.empty(d.shape, dtype=np.int64)
    for idx, x in np.ndenumerate(d):
        x = max(int(x), 1)
        out[idx] = min(num_buckets - 1, x.bit_length() - 1)
    return out


def position_index(L, n_t, N):
    n = L - n_t
    p = np.minimum(np.arange(L), n)
    return (N - 1) + p[None, :] - p[:, None]


def silu(x):
    return x / (1.0 + np.exp(-x))


def dsilu(x):
    s = 1.0 / (1.0 + np.exp(-x))
    return s * (1.0 + x * (1.0 - s))


def _exact(x):
    return x


def seq_dense(q, k, v, ts, rab_pos, rab_time, N, n_t, d_out=None, rnd=_exact):
    """One sequence, all heads.  q,k: [L,h,dqk]; v,d_out: [L,h,dv].
    Returns O [L,h,dv] and, if d_out is given, the gradients.  `rnd` is
    applied to SiLU(S) and to dP SiLU'(S) (both before the 1/N) where they
    enter the products with V, dO, K and Q."""
    L, H, _ = q.shape
    M = mask_alg1(L, n_t)
    bias = rab_pos[position_index(L, n_t, N)] + rab_time[bucket_matrix(ts, len(rab_time))]
    O = np.zeros((L, H, v.shape[2]))
    grads = None
    if d_out is not None:
        dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
        drp, drt = np.zeros_like(rab_pos), np.zeros_like(rab_time)
    for a in range(H):
        S = q[:, a, :] @ k[:, a, :].T + bias
        A = np.where(M, silu(S) / N, 0.0)
        Ar = np.where(M, rnd(silu(S)), 0.0) / N
        O[:, a, :] = Ar @ v[:, a, :]
        if d_out is not None:
            G = d_out[:, a, :]
            dA = G @ v[:, a, :].T
            dS = np.where(M, dA * dsilu(S) / N, 0.0)
            dSr = np.where(M, rnd(dA * dsilu(S)), 0.0) / N
            dv[:, a, :] = Ar.T @ G
            dq[:, a, :] = dSr @ k[:, a, :]
            dk[:, a, :] = dSr.T @ q[:, a, :]
            np.add.at(drp, position_index(L, n_t, N)[M], dS[M])
            np.add.at(drt, bucket_matrix(ts, len(rab_time))[M], dS[M])
    if d_out is not None:
        grads = (dq, dk, dv, drp, drt)
    return O, grads


def jagged_dense(batch_offsets, ts, rab_pos, rab_time, N, q, k, v, num_targets=None, d_out=None,
                 rnd=_exact):
    B = len(batch_offsets) - 1
    O = np.zeros((q.shape[0], q.shape[1], v.shape[2]))
    tot = None
    for b in range(B):
        s, e = int(batch_offsets[b]), int(batch_offsets[b + 1])
        if e == s:
            continue
        nt = 0 if num_targets is None else int(num_targets[b])
        o, g = seq_dense(q[s:e], k[s:e], v[s:e], ts[s:e], rab_pos, rab_time, N, nt,
                         None if d_out is None else d_out[s:e], rnd)
        O[s:e] = o
        if g is not None:
            if tot is None:
                tot = [np.zeros_like(q), np.zeros_like(k), np.zeros_like(v),
                       np.zeros_like(rab_pos), np.zeros_like(rab_time)]
            tot[0][s:e] += g[0]
            tot[1][s:e] += g[1]
            tot[2][s:e] += g[2]
            tot[3] += g[3]
            tot[4] += g[4]
    if d_out is not None and tot is None:
        tot = [np.zeros_like(q), np.zeros_like(k), np.zeros_like(v),
               np.zeros_like(rab_pos), np.zeros_like(rab_time)]
    return O, tot
