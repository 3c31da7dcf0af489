"""C ABI checks that need no GPU: the library loads, exports every entry
point include/hstu.h declares, and rejects bad arguments on the host
before anything is launched (every call below fails validation, so no
device work is attempted)."""
import ctypes
import os
import re
import threading

import pytest

from tests.conftest import ROOT

HEADER = os.path.join(ROOT, "include", "hstu.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hstu_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def hs():
    from paper_2402_17152_amd import hstu
    return hstu


def test_header_symbols_exported(hs):
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(hs.lib, n), n
    assert sorted(hs.EXPORTED) == names


def test_abi_version(hs):
    assert hs.hstu_abi_version() == 1


def _problem(hs, **kw):
    a = dict(num_seqs=8, total_tokens=48118, max_seq_len=8192, num_heads=4, d_qk=128, d_v=128,
             num_time_buckets=128, dtype=hs.HSTU_BF16)
    a.update(kw)
    return hs.make_problem(**a)


def test_workspace_bytes(hs):
    p = _problem(hs)
    n = hs.hstu_workspace_bytes(p)
    # work lists + fp32 dQ accumulator [T][h][d_qk]
    assert n >= 48118 * 4 * 128 * 4
    assert n % 256 == 0
    assert hs.hstu_workspace_bytes(_problem(hs, d_qk=48)) == 0
    assert hs.hstu_workspace_bytes(_problem(hs, num_heads=0)) == 0
    assert hs.hstu_workspace_bytes(_problem(hs, max_seq_len=70000)) == 0
    f = hs.hstu_workspace_bytes(_problem(hs, dtype=hs.HSTU_F32))
    assert 0 < f < n


def _partial_slots(lengths):
    """Slots of the bf16 backward's partial dQ blocks: one per 32-row step
    of every 128-key block (rows from the block's first key to the end)."""
    n = 0
    for L in lengths:
        for j0 in range(0, L, 128):
            n += (L - j0 + 31) // 32
    return n


@pytest.mark.parametrize("N,B,extra", [(8192, 8, 0), (4096, 64, 0), (129, 5, 0), (127, 3, 50),
                                       (1, 40, 0), (300, 7, 299), (3072, 16, 0)])
def test_workspace_covers_partial_dq(hs, N, B, extra):
    """The workspace bound (computed from T, B and N only) holds the partial
    dQ blocks of the worst jagged batch with that T: as many sequences of
    length N as fit, the remainder in one more (the slot count is convex in
    L, so that is its maximum)."""
    lengths = [N] * B + ([extra] if extra else [])
    T = sum(lengths)
    for h, d in ((4, 128), (8, 64), (2, 32)):
        p = _problem(hs, num_seqs=len(lengths), total_tokens=T, max_seq_len=N, num_heads=h, d_qk=d,
                     d_v=d)
        need = _partial_slots(lengths) * h * d * 32 * 2
        assert hs.hstu_workspace_bytes(p) >= need


FAKE = 0x10000  # 64 KiB-aligned, never dereferenced: every call fails validation first


def _jagged(hs, **kw):
    a = dict(seq_offsets=FAKE, timestamps=FAKE, num_targets=None, rab_pos=FAKE, rab_time=FAKE)
    a.update(kw)
    return hs.Jagged(**a)


def _fwd(hs, p, j, q=FAKE, qs=512, k=FAKE, ks=512, v=FAKE, vs=512, out=FAKE, ws=FAKE, wsb=None):
    if wsb is None:
        wsb = 1 << 40
    P = ctypes.c_void_p
    return hs.lib.hstu_attn_fwd(None if p is None else ctypes.byref(p),
                                None if j is None else ctypes.byref(j), P(q), qs, P(k), ks, P(v), vs,
                                P(out), P(ws), wsb, None)


@pytest.mark.parametrize("case,status,needle", [
    (dict(p=None), 1, "problem"),
    (dict(j=None), 1, "jagged"),
    (dict(pkw=dict(d_qk=48)), 2, "d_qk"),
    (dict(pkw=dict(num_heads=65)), 2, "num_heads"),
    (dict(pkw=dict(num_time_buckets=300)), 2, "num_time_buckets"),
    (dict(pkw=dict(num_seqs=0)), 1, "num_seqs"),
    (dict(jkw=dict(rab_pos=None)), 1, "rab_pos"),
    (dict(jkw=dict(timestamps=None)), 1, "timestamps"),
    (dict(q=None), 1, "q is NULL"),
    (dict(q=FAKE + 8), 1, "aligned"),
    (dict(qs=256), 1, "q_stride"),
    (dict(vs=516), 1, "multiple of 16"),
    (dict(ws=None), 3, "workspace"),
    (dict(wsb=100), 3, "too small"),
])
def test_fwd_argument_errors(hs, case, status, needle):
    p = None if "p" in case else _problem(hs, **case.get("pkw", {}))
    j = None if "j" in case else _jagged(hs, **case.get("jkw", {}))
    kw = {k: v for k, v in case.items() if k in ("q", "qs", "k", "ks", "v", "vs", "out", "ws", "wsb")}
    st = _fwd(hs, p, j, **kw)
    assert st == status
    assert needle in hs.hstu_last_error()


def test_error_message_is_thread_local(hs):
    st = _fwd(hs, _problem(hs, d_qk=48), _jagged(hs))
    assert st == 2
    seen = []

    def other():
        seen.append(hs.hstu_last_error())

    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen == [""]
    assert "d_qk" in hs.hstu_last_error()


def test_other_entry_points_validate(hs):
    P = ctypes.c_void_p
    assert hs.lib.hstu_complete_cumsum(-1, P(FAKE), P(FAKE), None) == 1
    assert hs.lib.hstu_pair_offsets(0, P(FAKE), P(FAKE), None) == 1
    assert hs.lib.hstu_time_bucketize(1, 10, 300, P(FAKE), P(FAKE), P(FAKE), 100, P(FAKE), None) == 2
    assert hs.lib.hstu_time_bucketize(1, 10, 128, P(FAKE), P(FAKE), P(FAKE), 100, P(FAKE + 1), None) == 1
    assert hs.lib.hstu_validate(None, None, None) == 1
    p = _problem(hs, num_heads=64, d_v=128)   # D = 8192 > 4096 for the epilogue
    j = _jagged(hs)
    st = hs.lib.hstu_layer_fwd(ctypes.byref(p), ctypes.byref(j), P(FAKE), 8192, P(FAKE), 8192,
                               P(FAKE), 8192, P(FAKE), 8192, None, None, 1e-5, P(FAKE), P(FAKE),
                               None, None, P(FAKE), 1 << 40, None)
    assert st == 2 and "4096" in hs.hstu_last_error()
    p = _problem(hs)
    st = hs.lib.hstu_attn_bwd(ctypes.byref(p), ctypes.byref(j), P(FAKE), 512, P(FAKE), 512,
                              P(FAKE), 512, P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE),
                              P(FAKE), 1 << 40, None)
    assert st == 1 and "dv" in hs.hstu_last_error()


def test_projection_entry_points_validate(hs):
    """f_1 / f_2 calls reject bad shapes, pointers and workspaces on the host."""
    P = ctypes.c_void_p
    p = _problem(hs, num_heads=8, d_qk=64, d_v=64, total_tokens=1000)
    pf = _problem(hs, num_heads=8, d_qk=64, d_v=64, total_tokens=1000, dtype=hs.HSTU_F32)
    L = hs.lib
    assert L.hstu_proj_workspace_bytes(ctypes.byref(p), 512) > 0
    assert L.hstu_proj_workspace_bytes(ctypes.byref(p), 96) == 0     # bf16: multiple of 64
    assert L.hstu_proj_workspace_bytes(ctypes.byref(pf), 12) == 0    # multiple of 8
    assert L.hstu_proj_workspace_bytes(ctypes.byref(pf), 24) > 0
    cases = [
        (lambda: L.hstu_proj_in_fwd(ctypes.byref(p), 96, P(FAKE), 96, P(FAKE), None, P(FAKE), None,
                                    None), 2, "multiples of 64"),
        (lambda: L.hstu_proj_in_fwd(ctypes.byref(pf), 12, P(FAKE), 12, P(FAKE), None, P(FAKE), None,
                                    None), 2, "multiple of 8"),
        (lambda: L.hstu_proj_in_fwd(ctypes.byref(p), 512, None, 512, P(FAKE), None, P(FAKE), None,
                                    None), 1, "x is NULL"),
        (lambda: L.hstu_proj_in_fwd(ctypes.byref(p), 512, P(FAKE), 256, P(FAKE), None, P(FAKE), None,
                                    None), 1, "x_stride"),
        (lambda: L.hstu_proj_in_fwd(ctypes.byref(p), 512, P(FAKE), 512, P(FAKE), P(FAKE + 4),
                                    P(FAKE), None, None), 1, "b1"),
        (lambda: L.hstu_proj_out_fwd(ctypes.byref(p), 512, P(FAKE), 512, P(FAKE), None, None, None,
                                     None), 1, "y is NULL"),
        (lambda: L.hstu_proj_out_bwd(ctypes.byref(p), 512, P(FAKE), 512, P(FAKE), P(FAKE), P(FAKE),
                                     P(FAKE), None, None, 0, None), 3, "workspace"),
        (lambda: L.hstu_proj_in_bwd(ctypes.byref(p), 512, P(FAKE), 512, P(FAKE), P(FAKE), P(FAKE),
                                    P(FAKE), P(FAKE), None, None, P(FAKE), P(FAKE), None, P(FAKE),
                                    100, None), 1, "dk is NULL"),
        (lambda: L.hstu_proj_in_bwd(ctypes.byref(p), 512, P(FAKE), 512, P(FAKE), P(FAKE), P(FAKE),
                                    P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), P(FAKE), None, P(FAKE),
                                    100, None), 3, "too small"),
    ]
    big = _problem(hs, num_heads=8, d_qk=64, d_v=64, total_tokens=600000)  # T*F*2 >= 2^31
    cases.append((lambda: L.hstu_proj_in_fwd(ctypes.byref(big), 512, P(FAKE), 512, P(FAKE), None,
                                             P(FAKE), None, None), 2, "2 GiB"))
    for call, status, needle in cases:
        assert call() == status, needle
        assert needle in hs.hstu_last_error(), (needle, hs.hstu_last_error())


def test_stochastic_length_entry_points_validate(hs):
    P = ctypes.c_void_p
    L = hs.lib
    assert hs.hstu_sl_workspace_bytes(0) == 0 and hs.hstu_sl_workspace_bytes(64) > 0
    assert hs.hstu_sl_subseq_len(4096, 2.5) == 0 and hs.hstu_sl_subseq_len(0, 1.6) == 0
    assert hs.hstu_sl_keep_numerator(4096, 2.5) == 0.0
    assert hs.hstu_sl_keep_numerator(4096, 1.6) == 4096.0 ** 1.6

    def sl(B=8, Ls=16, mode=1, e=FAKE, ws=FAKE, wsb=1 << 20, offs=FAKE, kn=256.0):
        return L.hstu_stochastic_length(B, P(offs), P(FAKE), None, Ls, kn, mode, P(FAKE),
                                        P(e) if e else None, P(FAKE), P(FAKE), P(ws) if ws else None,
                                        wsb, None)
    for kw, status, needle in ((dict(B=0), 1, "num_seqs"), (dict(Ls=0), 1, "subseq_len"),
                               (dict(mode=5), 1, "selection"), (dict(e=None), 1, "e_rand"),
                               (dict(kn=-1.0), 1, "keep_numerator"),
                               (dict(kn=float("inf")), 1, "keep_numerator"),
                               (dict(kn=float("nan")), 1, "keep_numerator"),
                               (dict(offs=0), 1, "NULL"), (dict(ws=None), 3, "workspace"),
                               (dict(wsb=16), 3, "too small"), (dict(ws=FAKE + 64), 3, "aligned")):
        assert sl(**kw) == status, kw
        assert needle in hs.hstu_last_error(), (needle, hs.hstu_last_error())
    assert L.hstu_gather_rows(P(FAKE), 8, 6, P(FAKE), P(FAKE), 10, P(FAKE), 8, None) == 1
    assert "4-byte" in hs.hstu_last_error()
    assert L.hstu_gather_rows(P(FAKE), 4, 8, P(FAKE), P(FAKE), 10, P(FAKE), 8, None) == 1
    assert "stride" in hs.hstu_last_error()
    assert L.hstu_gather_rows(P(FAKE), 8, 8, P(FAKE), P(FAKE), 0, P(FAKE), 8, None) == 0
    sp, s2 = ctypes.c_double(), ctypes.c_double()
    assert L.hstu_sl_sparsity(0, P(FAKE), 16, ctypes.byref(sp), ctypes.byref(s2)) == 1


def test_cached_pass_validates(hs):
    P = ctypes.c_void_p
    L = hs.lib
    p = _problem(hs, num_seqs=16, total_tokens=4096, max_seq_len=3072)
    pf = _problem(hs, num_seqs=16, total_tokens=4096, max_seq_len=3072, dtype=hs.HSTU_F32)
    j = _jagged(hs)
    assert L.hstu_attn_fwd_cached_workspace_bytes(ctypes.byref(p)) > 0
    assert L.hstu_attn_fwd_cached_workspace_bytes(ctypes.byref(_problem(hs, d_qk=48))) == 0

    def cached(pp=p, co=FAKE, ct=100, ws=FAKE, wsb=1 << 40):
        return L.hstu_attn_fwd_cached(ctypes.byref(pp), ctypes.byref(j), P(FAKE), 512, P(FAKE), 512,
                                      P(FAKE), 512, P(co) if co else None, P(FAKE), ct, P(FAKE), 512,
                                      P(FAKE), 512, P(FAKE), P(ws) if ws else None, wsb, None)
    for kw, status, needle in ((dict(pp=pf), 2, "bf16"), (dict(co=0), 1, "cache_offsets"),
                               (dict(ct=-1), 1, "cache_tokens"), (dict(ws=None), 3, "workspace"),
                               (dict(wsb=1000), 3, "too small")):
        assert cached(**kw) == status, kw
        assert needle in hs.hstu_last_error(), (needle, hs.hstu_last_error())
