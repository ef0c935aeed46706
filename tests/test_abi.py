"""The C ABI without a GPU: exported symbols, host-side validation (which
returns before any HIP call) and the host rotary-table builder."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import brute
from paper_2609_35110_amd import sol

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
P = ctypes.c_void_p


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sol.LIB_PATH):
        from paper_2609_35110_amd import build
        build.build()
    return sol.lib()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "sol.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sol_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_function_is_exported(L):
    names = declared_functions()
    assert {"sol_attn_fwd", "sol_rope3d", "sol_rope3d_table", "sol_rope3d_table_floats"} <= set(names)
    for n in names:
        assert hasattr(L, n), "libsol.so does not export %s" % n


def test_status_strings(L):
    assert sol.sol_status_string(0) == "ok"
    for s in (-1, -2, -3):
        assert sol.sol_status_string(s) not in ("ok", "unknown status")
    assert sol.sol_version() == 200


# Fake, 16-byte aligned device addresses: every call below is rejected on the
# host before anything would dereference them.
A, Bp, C, Dp, TAB = (P(0x100000 * i) for i in range(1, 6))


def attn(q=A, k=Bp, v=C, out=Dp, B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, tab=TAB):
    return sol.sol_attn_fwd(q, k, v, out, B, H, N, D, T, Hl, Wl, tab, None)


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(q=None), -1, "NULL"),
    (dict(out=None), -1, "NULL"),
    (dict(D=64), -2, "head dim"),
    (dict(N=0), -1, ">= 1"),
    (dict(B=0), -1, ">= 1"),
    (dict(T=-1), -1, "negative"),
    (dict(T=4), -1, "more tokens"),
    (dict(N=(1 << 23) + 1, T=1, Hl=1, Wl=1), -2, "exceeds"),
    (dict(q=P(0x100008)), -1, "aligned"),
    (dict(out=P(0x500004)), -1, "aligned"),
    (dict(tab=P(0x500008)), -1, "aligned"),
    (dict(out=A), -1, "overlaps"),
    (dict(out=P(0x100000 + 1024)), -1, "overlaps"),
])
def test_attn_fwd_rejects_before_any_hip_call(L, kw, status, fragment):
    st = attn(**kw)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


WS = P(0x10000000)


def attn_ws(q=A, k=Bp, v=C, out=Dp, B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, tab=TAB, ws=WS,
            ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = sol.sol_attn_workspace_bytes(B, H, N, D)
    return sol.sol_attn_fwd_ws(q, k, v, out, B, H, N, D, T, Hl, Wl, tab, ws, ws_bytes, None)


def test_workspace_size(L):
    # 3488 tiles of 32 keys per slab (the last one padded), 8 KB of K and 8 KB of V each
    assert sol.sol_prepared_kv_bytes(1, 40, 111600, 128) == 40 * 3488 * 32 * 128 * 2
    assert sol.sol_attn_workspace_bytes(1, 40, 111600, 128) == 2 * 40 * 3488 * 32 * 128 * 2
    assert sol.sol_prepared_kv_bytes(2, 3, 33, 128) == 2 * 3 * 2 * 32 * 128 * 2
    assert sol.sol_attn_workspace_bytes(0, 1, 1, 128) == 0
    assert sol.sol_prepared_kv_bytes(1, 1, 1, 64) == 0


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(ws=None), -1, "workspace is NULL"),
    (dict(ws=P(0x10000008)), -1, "aligned"),
    (dict(ws_bytes=1000), -1, "workspace needs"),
    (dict(ws=P(0x100000 - 4096)), -1, "workspace overlaps"),
    (dict(D=64), -2, "head dim"),
    (dict(out=Bp), -1, "overlaps"),
    (dict(T=9), -1, "more tokens"),
])
def test_attn_fwd_ws_rejects_before_any_hip_call(L, kw, status, fragment):
    st = attn_ws(**kw)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(k=None), -1, "NULL"),
    (dict(k_prep=P(0x100008)), -1, "aligned"),
    (dict(k_prep=Bp), -1, "overlap"),
    (dict(v_prep=P(0x300000 + 4096)), -1, "overlap"),
    (dict(D=32), -2, "head dim"),
])
def test_prepare_kv_rejects_before_any_hip_call(L, kw, status, fragment):
    args = dict(k=A, v=Bp, k_prep=C, v_prep=Dp, B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, tab=TAB)
    args.update(kw)
    st = sol.sol_prepare_kv(args["k"], args["v"], args["k_prep"], args["v_prep"], args["B"], args["H"],
                            args["N"], args["D"], args["T"], args["Hl"], args["Wl"], args["tab"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(q=None), -1, "NULL"),
    (dict(out=C), -1, "overlaps"),
    (dict(v_prep=P(0x300008)), -1, "aligned"),
    (dict(N=100, T=9), -1, "more tokens"),
])
def test_attn_fwd_prepared_rejects_before_any_hip_call(L, kw, status, fragment):
    args = dict(q=A, k_prep=Bp, v_prep=C, out=Dp, B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, tab=TAB)
    args.update(kw)
    st = sol.sol_attn_fwd_prepared(args["q"], args["k_prep"], args["v_prep"], args["out"], args["B"],
                                   args["H"], args["N"], args["D"], args["T"], args["Hl"], args["Wl"],
                                   args["tab"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), -1),
    (dict(D=96), -2),
    (dict(T=5), -1),
    (dict(tab=None), -1),
    (dict(y=P(0x100000 + 4096)), -1),   # partial overlap (in place is allowed)
])
def test_rope3d_rejects_before_any_hip_call(L, kw, status):
    args = dict(x=A, y=Bp, B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, tab=TAB)
    args.update(kw)
    st = sol.sol_rope3d(args["x"], args["y"], args["B"], args["H"], args["N"], args["D"],
                        args["T"], args["Hl"], args["Wl"], args["tab"], None)
    assert st == status, sol.sol_last_error()


G = P(0x20000000)  # fake, aligned device address of normalisation weights


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(key0=-1), -1, "do not fit"),
    (dict(key0=100, n_kv=291), -1, "do not fit"),     # 100 + 192 > 291
    (dict(n_kv=0), -1, "n_kv"),
    (dict(n_kv=(1 << 23) + 1), -2, "n_kv"),
    (dict(gamma=P(0x20000004)), -1, "gamma must be 16-byte aligned"),
    (dict(eps=-1e-6), -1, "eps"),
    (dict(eps=float("nan")), -1, "eps"),
    (dict(k_prep=P(0x200000 + 4096)), -1, "overlap"),   # k_prep inside v
    (dict(T=9), -1, "more tokens"),
    (dict(sp=(4, 48, 48)), -1, "multiple of 8"),
    (dict(sp=(-8, 48, 48)), -1, "non-negative multiple of 8"),
    (dict(sp=(32, 48, 56)), -1, "exceeds the head dim"),
])
def test_prepare_kv_ex_rejects_before_any_hip_call(L, kw, status, fragment):
    args = dict(k=A, v=Bp, k_prep=P(0x1000000), v_prep=P(0x2000000), B=1, H=2, N=192, key0=0,
                n_kv=192, D=128, T=3, Hl=8, Wl=8, sp=(32, 48, 48), tab=TAB, gamma=G, eps=1e-6)
    args.update(kw)
    st = sol.sol_prepare_kv_ex(args["k"], args["v"], args["k_prep"], args["v_prep"], args["B"],
                               args["H"], args["N"], args["key0"], args["n_kv"], args["D"], args["T"],
                               args["Hl"], args["Wl"], *args["sp"], args["tab"], args["gamma"],
                               args["eps"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(n_kv=0), -1, "n_kv"),
    (dict(gamma=P(0x20000008)), -1, "gamma must be 16-byte aligned"),
    (dict(eps=float("inf")), -1, "eps"),
    (dict(out=P(0x1000000 + 256)), -1, "overlaps"),   # out inside k_prep of 1000 keys
    (dict(D=64), -2, "head dim"),
    (dict(fmt=3), -1, "out_format"),
    (dict(fmt=-1), -1, "out_format"),
    (dict(out=P(0x100000 - 49152)), -1, "overlaps"),   # 96 KB of bf16 out would reach q
    (dict(out=P(0x100000 - 49152 + 16), fmt=1), -1, "overlaps"),  # 48 KB of E4M3 out reaches q
    (dict(out=P(0x100000 - 55296 + 16), fmt=2), -1, "overlaps"),  # 54 KB of records reach q
    (dict(sp=(4, 48, 48)), -1, "multiple of 8"),
    (dict(sp=(-8, 48, 48)), -1, "non-negative multiple of 8"),
    (dict(sp=(32, 48, 56)), -1, "exceeds the head dim"),
])
def test_attn_fwd_prepared_ex_rejects_before_any_hip_call(L, kw, status, fragment):
    args = dict(q=A, k_prep=P(0x1000000), v_prep=P(0x2000000), out=Dp, B=1, H=2, N=192, n_kv=1000,
                D=128, T=3, Hl=8, Wl=8, sp=(32, 48, 48), tab=TAB, gamma=G, eps=1e-6, fmt=0)
    args.update(kw)
    st = sol.sol_attn_fwd_prepared_ex(args["q"], args["k_prep"], args["v_prep"], args["out"],
                                      args["B"], args["H"], args["N"], args["n_kv"], args["D"],
                                      args["T"], args["Hl"], args["Wl"], *args["sp"], args["tab"],
                                      args["gamma"], args["eps"], args["fmt"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(gamma=P(0x20000002)), -1),
    (dict(eps=-0.5), -1),
    (dict(tab=None), -1),
    (dict(D=96), -2),
    (dict(sp=(4, 48, 48)), -1),
    (dict(sp=(32, 48, -8)), -1),
    (dict(sp=(64, 64, 8)), -1),
])
def test_qknorm_rope3d_rejects_before_any_hip_call(L, kw, status):
    args = dict(x=A, y=Bp, B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, sp=(32, 48, 48), tab=TAB, gamma=G,
                eps=1e-6)
    args.update(kw)
    st = sol.sol_qknorm_rope3d(args["x"], args["y"], args["B"], args["H"], args["N"], args["D"],
                               args["T"], args["Hl"], args["Wl"], *args["sp"], args["tab"],
                               args["gamma"], args["eps"], None)
    assert st == status, sol.sol_last_error()


def test_sparse_workspace_size(L):
    nqb, nkb = 436, 872  # N = 111,600
    up = lambda x: (x + 255) // 256 * 256
    o1 = up(40 * nqb * 4)
    o2 = up(o1 + 40 * nqb * nkb * 2)
    o3 = up(o2 + 40 * nqb * 128 * 4)
    assert sol.sol_sparse_workspace_bytes(1, 40, 111600, 128) == up(o3 + 40 * nkb * 128 * 4)
    assert sol.sol_sparse_workspace_bytes(1, 1, 8064 * 128 + 1, 128) == 0
    assert sol.sol_sparse_workspace_bytes(1, 1, 8064 * 128, 128) > 0
    assert sol.sol_sparse_workspace_bytes(1, 1, 100, 64) == 0


WSS = P(0x30000000)


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(N=8064 * 128 + 1, T=1, Hl=1, Wl=1), -2, "N <= "),
    (dict(ws=None), -1, "workspace is NULL"),
    (dict(ws_bytes=100), -1, "workspace needs"),
    (dict(ws=P(0x30000004)), -1, "aligned"),
    (dict(ws=P(0x100000 - 4096)), -1, "workspace overlaps"),
    (dict(tau=float("nan")), -1, "tau"),
    (dict(tau=float("inf")), -1, "tau"),
    (dict(gamma=P(0x20000004)), -1, "gamma"),
    (dict(k_prep=None), -1, "NULL"),
    (dict(sp=(4, 48, 48)), -1, "multiple of 8"),
    (dict(sp=(-8, 48, 48)), -1, "non-negative multiple of 8"),
    (dict(sp=(32, 48, 56)), -1, "exceeds the head dim"),
])
def test_sparse_route_rejects_before_any_hip_call(L, kw, status, fragment):
    args = dict(q=A, k_prep=P(0x1000000), B=1, H=2, N=1000, D=128, T=1, Hl=10, Wl=100, sp=(32, 48, 48),
                tab=TAB, gamma=None, eps=1e-6, tau=1.0, ws=WSS, ws_bytes=None)
    args.update(kw)
    if args["ws_bytes"] is None:
        args["ws_bytes"] = sol.sol_sparse_workspace_bytes(args["B"], args["H"], min(args["N"], 1 << 20), 128)
    st = sol.sol_sparse_route(args["q"], args["k_prep"], args["B"], args["H"], args["N"], args["D"],
                              args["T"], args["Hl"], args["Wl"], *args["sp"], args["tab"], args["gamma"],
                              args["eps"], args["tau"], args["ws"], args["ws_bytes"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(out=P(0x30000000 + 64)), -1, "overlaps"),
    (dict(fmt=3), -1, "out_format"),
    (dict(v_prep=None), -1, "NULL"),
    (dict(ws_bytes=10), -1, "workspace needs"),
    (dict(sp=(4, 48, 48)), -1, "multiple of 8"),
    (dict(sp=(-8, 48, 48)), -1, "non-negative multiple of 8"),
    (dict(sp=(32, 48, 56)), -1, "exceeds the head dim"),
])
def test_attn_fwd_sparse_rejects_before_any_hip_call(L, kw, status, fragment):
    args = dict(q=A, k_prep=P(0x1000000), v_prep=P(0x2000000), out=Dp, B=1, H=2, N=1000, D=128, T=1,
                Hl=10, Wl=100, sp=(32, 48, 48), tab=TAB, gamma=None, eps=1e-6, ws=WSS, ws_bytes=None,
                fmt=0)
    args.update(kw)
    if args["ws_bytes"] is None:
        args["ws_bytes"] = sol.sol_sparse_workspace_bytes(1, 2, 1000, 128)
    st = sol.sol_attn_fwd_sparse(args["q"], args["k_prep"], args["v_prep"], args["out"], args["B"],
                                 args["H"], args["N"], args["D"], args["T"], args["Hl"], args["Wl"],
                                 *args["sp"], args["tab"], args["gamma"], args["eps"], args["ws"],
                                 args["ws_bytes"], args["fmt"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


def test_qkv_record_bytes(L):
    assert sol.sol_qkv_record_bytes(1, 2, 192) == 192 * 2 * 400
    assert sol.sol_qkv_record_bytes(2, 40, 111600) == 2 * 40 * 111600 * 400
    assert sol.sol_qkv_record_bytes(0, 2, 192) == 0
    assert sol.sol_qkv_record_bytes(1, 2, (1 << 23) + 1) == 0


# records of B=1, H=2, N=192: 153,600 bytes
@pytest.mark.parametrize("kw,status,fragment", [
    (dict(q=None), -1, "NULL"),
    (dict(D=64), -2, "head dim"),
    (dict(rec=P(0x1000008)), -1, "aligned"),
    (dict(rec=P(0x100000 + 512)), -1, "overlaps"),   # records over q
    (dict(qg=P(0x20000004)), -1, "gamma"),
    (dict(kg=P(0x20000004)), -1, "gamma"),
    (dict(eps=-1.0), -1, "eps"),
    (dict(T=9), -1, "more tokens"),
    (dict(tab=P(0x500008)), -1, "aligned"),
])
def test_qkv_encode_rejects_before_any_hip_call(L, kw, status, fragment):
    a = dict(q=A, k=Bp, v=C, rec=P(0x1000000), B=1, H=2, N=192, D=128, T=3, Hl=8, Wl=8, tab=TAB,
             qg=G, kg=G, eps=1e-6)
    a.update(kw)
    st = sol.sol_qkv_encode(a["q"], a["k"], a["v"], a["rec"], a["B"], a["H"], a["N"], a["D"], a["T"],
                            a["Hl"], a["Wl"], a["tab"], a["qg"], a["kg"], a["eps"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,fragment", [
    (dict(sb=-8), "strides"),
    (dict(sh=12), "strides"),
    (dict(sn=4), "strides"),
    (dict(rec=P(0x100000 + 3 * 128 * 2 + 16)), "overlaps"),  # inside the packed span of q
])
def test_qkv_encode_strided_rejects_before_any_hip_call(L, kw, fragment):
    # packed [1, 192, 3, 2, 128] at A: q = A, k = A + 256 elements, v = A + 512
    a = dict(rec=P(0x1000000), sb=192 * 3 * 2 * 128, sh=128, sn=3 * 2 * 128)
    a.update(kw)
    st = sol.sol_qkv_encode_strided(A, P(0x100000 + 512), P(0x100000 + 1024), a["sb"], a["sh"], a["sn"],
                                    a["rec"], 1, 2, 192, 128, 0, 0, 0, None, None, None, 0.0, None)
    assert st == -1, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(rec=None), -1, "NULL"),
    (dict(D=64), -2, "head dim"),
    (dict(N=0), -1, ">= 1"),
    (dict(k=P(0x400000 - 64)), -1, "overlap"),        # k (96 KB) runs into v
    (dict(q=P(0x100000 + 1024)), -1, "overlap"),      # q inside the records
    (dict(v=P(0x300008)), -1, "aligned"),
])
def test_qkv_decode_rejects_before_any_hip_call(L, kw, status, fragment):
    a = dict(rec=A, q=Bp, k=C, v=Dp, B=1, H=2, N=192, D=128)
    a.update(kw)
    st = sol.sol_qkv_decode(a["rec"], a["q"], a["k"], a["v"], a["B"], a["H"], a["N"], a["D"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(rec=None), -1, "NULL"),
    (dict(key0=-1), -1, "do not fit"),
    (dict(key0=100, n_kv=291), -1, "do not fit"),
    (dict(n_kv=0), -1, "n_kv"),
    (dict(n_kv=(1 << 23) + 1), -2, "n_kv"),
    (dict(k_prep=P(0x1000008)), -1, "aligned"),
    (dict(k_prep=P(0x100000 + 4096)), -1, "overlap"),  # k_prep over the records
    (dict(D=256), -2, "head dim"),
])
def test_prepare_kv_records_rejects_before_any_hip_call(L, kw, status, fragment):
    a = dict(rec=A, k_prep=P(0x1000000), v_prep=P(0x2000000), B=1, H=2, N=192, key0=0, n_kv=192,
             D=128)
    a.update(kw)
    st = sol.sol_prepare_kv_records(a["rec"], a["k_prep"], a["v_prep"], a["B"], a["H"], a["N"],
                                    a["key0"], a["n_kv"], a["D"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,status,fragment", [
    (dict(out=None), -1, "NULL"),
    (dict(n_kv=0), -1, "n_kv"),
    (dict(fmt=3), -1, "out_format"),
    (dict(out=P(0x100000 + 2048)), -1, "overlaps"),    # out over the records
    (dict(out=P(0x1000000 + 256)), -1, "overlaps"),    # out inside k_prep
    (dict(D=64), -2, "head dim"),
    (dict(out=P(0x400004)), -1, "aligned"),
])
def test_attn_fwd_records_rejects_before_any_hip_call(L, kw, status, fragment):
    a = dict(rec=A, k_prep=P(0x1000000), v_prep=P(0x2000000), out=Dp, B=1, H=2, N=192, n_kv=1000,
             D=128, fmt=0)
    a.update(kw)
    st = sol.sol_attn_fwd_records(a["rec"], a["k_prep"], a["v_prep"], a["out"], a["B"], a["H"], a["N"],
                                  a["n_kv"], a["D"], a["fmt"], None)
    assert st == status, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


@pytest.mark.parametrize("kw,fragment", [
    (dict(ops=None), "NULL"),
    (dict(wg=0), "out of range"),
    (dict(iters=0), "out of range"),
    (dict(iters=(1 << 24) + 1), "out of range"),
    (dict(out=P(0x100008)), "aligned"),
    (dict(out=P(0x200000 - 1024)), "overlaps"),   # 256 floats per workgroup reach the operands
])
def test_mfma_probe_rejects_before_any_hip_call(L, kw, fragment):
    a = dict(ops=P(0x200000), out=P(0x100000), wg=4, iters=10)
    a.update(kw)
    st = sol.sol_mfma_probe(a["ops"], a["out"], a["wg"], a["iters"], None)
    assert st == -1, sol.sol_last_error()
    assert fragment in sol.sol_last_error()


def test_binding_rejects_wrong_dtype_and_device():
    import torch
    x = torch.zeros(1, 1, 4, 128, dtype=torch.float32)
    with pytest.raises(TypeError):
        sol.attn_fwd(x, x, x, 1, 1, 1)
    xb = x.to(torch.bfloat16)
    with pytest.raises(ValueError):
        sol.attn_fwd(xb, xb, xb, 1, 1, 1)  # CPU tensors are not device memory


# ------------------------------------------------------------ rotary table

def test_table_size(L):
    assert sol.sol_rope3d_table_floats(128, 31, 45, 80) == 4 * (31 * 16 + 45 * 24 + 80 * 24)
    assert sol.sol_rope3d_table_floats(100, 1, 1, 1) == 0
    tab = np.zeros(10, np.float32)
    st = sol.sol_rope3d_table(tab.ctypes.data_as(P), 10, 128, 3, 8, 8, 10000.0)
    assert st == -1 and "needs" in sol.sol_last_error()


def _check_planes(tab, ang):
    """Plane 0 of a table holds the float32 rounding of each (cos, sin) of
    the numpy twin's angles (within 1 float32 ulp: libm vs numpy), plane 1
    what that rounding lost: hi + lo within 2^-46 of numpy's double (two libm
    results 1 ulp apart, plus lo's own rounding at 2^-48), |lo| at most half
    an fp32 ulp of hi."""
    hi, lo = tab.reshape(2, -1, 2)
    exact = np.stack([np.cos(ang), np.sin(ang)], -1)
    want = exact.astype(np.float32)
    assert hi.shape == want.shape
    ulps = np.abs(hi.view(np.int32).astype(np.int64) - want.view(np.int32).astype(np.int64))
    assert np.all((ulps <= 1) | (np.abs(hi - want) <= 1e-7))
    assert np.all(np.abs(hi.astype(np.float64) + lo - exact) <= 2.0 ** -46)
    assert np.all(np.abs(lo.astype(np.float64)) <= np.spacing(np.abs(hi)) / 2)
    assert np.abs(lo).max() > 0  # the second plane is not a copy of zeros


def test_table_matches_oracle_angles(L):
    """Both planes of the default table against the oracle's angle for each
    axis position and pair."""
    T, Hl, Wl = 5, 7, 9
    tab = sol.rope3d_table_host(T, Hl, Wl)
    # the oracle's angle of every pair at every position of each axis alone
    sections = []
    for axis, (ext, lo, width) in enumerate([(T, 0, 32), (Hl, 32, 48), (Wl, 80, 48)]):
        pos = np.zeros((ext, 3), np.int64)
        pos[:, axis] = np.arange(ext)
        ang = brute.rope_angles(pos)[:, lo // 2:(lo + width) // 2]
        sections.append(ang.reshape(-1))
    _check_planes(tab, np.concatenate(sections))


SPLITS = [(32, 48, 48), (16, 24, 24), (0, 64, 64), (8, 0, 0), (64, 0, 64)]


@pytest.mark.parametrize("split", SPLITS)
def test_split_table_matches_oracle_angles(L, split):
    """The table of any rotary split (partial RoPE: dims past dt+dh+dw pass
    through): one section per axis of width > 0 in each plane, as above."""
    T, Hl, Wl = 4, 6, 5
    dt, dh, dw = split
    n = sol.sol_rope3d_table_floats_ex(128, T, Hl, Wl, dt, dh, dw)
    assert n == 4 * (T * dt // 2 + Hl * dh // 2 + Wl * dw // 2)
    tab = sol.rope3d_table_host(T, Hl, Wl, split=split)
    assert tab.size == n
    sections, off = [], 0
    for axis, (ext, width) in enumerate([(T, dt), (Hl, dh), (Wl, dw)]):
        pos = np.zeros((ext, 3), np.int64)
        pos[:, axis] = np.arange(ext)
        ang = brute.rope_angles(pos, split=split)[:, off // 2:(off + width) // 2]
        sections.append(ang.reshape(-1))
        off += width
    _check_planes(tab, np.concatenate(sections))
    if split == (32, 48, 48):  # the default split is the table every other entry point takes
        assert np.array_equal(tab, sol.rope3d_table_host(T, Hl, Wl))


@pytest.mark.parametrize("split", [(4, 48, 48), (32, 48, 56), (-8, 64, 64), (32, 12, 48)])
def test_split_table_rejects_invalid_splits(L, split):
    assert sol.sol_rope3d_table_floats_ex(128, 3, 8, 8, *split) == 0
    tab = np.zeros(4096, np.float32)
    st = sol.sol_rope3d_table_ex(tab.ctypes.data_as(P), tab.size, 128, 3, 8, 8, *split, 10000.0)
    assert st == -1 and "split" in sol.sol_last_error()


def test_binding_rejects_a_table_of_another_grid():
    """The C ABI receives only the table's pointer; the binding checks its
    length against the grid and split before any launch (a 720p call given the
    low-resolution table would read past its end; the reverse would find its
    second plane in the wrong place)."""
    import torch
    low = torch.from_numpy(sol.rope3d_table_host(8, 30, 52))
    dev = low.device
    assert sol._table_ptr(low, dev, 128, 8, 30, 52) is not None
    with pytest.raises(ValueError, match="need"):
        sol._table_ptr(low, dev, 128, 31, 45, 80)
    big = torch.from_numpy(sol.rope3d_table_host(31, 45, 80))
    with pytest.raises(ValueError, match="need"):
        sol._table_ptr(big, dev, 128, 8, 30, 52)
    part = torch.from_numpy(sol.rope3d_table_host(8, 30, 52, split=(16, 24, 24)))
    with pytest.raises(ValueError, match="need"):
        sol._table_ptr(part, dev, 128, 8, 30, 52)  # the default split needs twice as many floats
    assert sol._table_ptr(part, dev, 128, 8, 30, 52, split=(16, 24, 24)) is not None


# ------------------------------------------------------- sol_attn_fwd's plan

def _plan_rule(S, N, D=128):
    """The schedule sol.h states, written out: chunks front to back, each the
    largest c whose prepared K and V (2 ceil(N/32) 32 D fp16 values per slab)
    fit in the S - s - c out slabs (N D bf16 each) after it; then the prefix
    of chunks with the least modelled time, a launch over x workgroups
    (ceil(N/256) per slab) costing ceil(x / 256) rounds, 1.4 times as long on
    the fused kernel, which takes every slab after the prefix, and each chunk
    0.1 round more."""
    region = N * D * 2
    kv = 2 * ((N + 31) // 32) * 32 * D * 2
    nq = (N + 255) // 256
    rounds = lambda slabs: -(-slabs * nq // 256)
    chunks, s = [], 0
    while s < S and len(chunks) < 64:
        c = max([t for t in range(0, S - s + 1) if t * kv <= (S - s - t) * region])
        if c == 0:
            break
        chunks.append(c)
        s += c
    best, best_cov = 1.4 * rounds(S), 0
    t, cov = 0, 0
    for c in chunks:
        t += rounds(c) + 0.1
        cov += c
        total = t + (1.4 * rounds(S - cov) if cov < S else 0)
        if total < best:
            best, best_cov = total, cov
    return best_cov


def test_attn_fwd_plan(L):
    assert sol.sol_attn_fwd_plan(1, 40, 111600, 128) == _plan_rule(40, 111600) > 30  # 720p: most slabs in place
    assert sol.sol_attn_fwd_plan(1, 24, 12480, 128) == 0     # low resolution: chunks too small to fill the chip
    assert sol.sol_attn_fwd_plan(1, 2, 192, 128) == 0        # two slabs: no room for any chunk
    assert _plan_rule(3, 192) == 0
    for B, H, N in [(2, 5, 112112), (1, 24, 12480), (3, 7, 466), (1, 1, 1), (4, 16, 1000), (1, 200, 64),
                    (1, 40, 48360), (2, 20, 200000), (8, 40, 4096)]:
        assert sol.sol_attn_fwd_plan(B, H, N, 128) == _plan_rule(B * H, N), (B, H, N)
    assert sol.sol_attn_fwd_plan(1, 2, 0, 128) < 0
    assert sol.sol_attn_fwd_plan(1, 2, 64, 64) < 0
