"""Host-side checks of libh2o.so: it loads, exports every function the header
declares, and rejects bad arguments before touching the device.

Fake (aligned, never dereferenced) pointers are used only for calls that must
fail host validation; the one call that passes validation runs only where no
device is visible and must report H2O_ENODEVICE.
"""
import ctypes
import os
import re
import subprocess

import pytest
import torch

from paper_2608_19920_amd import h2o as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "h2o.h")
P = 0x10000          # an aligned fake address; validation fails before any use
MIS = 0x10004        # misaligned


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(h2o_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(H.LIB_PATH):
        pytest.skip("libh2o.so not built")
    return H.lib()


def test_header_and_exports_agree(L):
    fns = header_functions()
    assert set(fns) == set(H.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", H.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (h2o_\w+)", out))
    for f in fns:
        assert f in exported, f
        assert hasattr(L, f)


def test_version(L):
    assert "gfx950" in H.h2o_version()


def _sdpa(L, **kw):
    a = dict(q=P, kc=P, vc=P, kn=P, vn=P, out=P, lse=P, wsum=P, ws=P, wsb=1 << 40, B=1, Hq=4,
             Hkv=2, T=8, M=16, d=64, scale=0.125, dt=1, st=None)
    a.update(kw)
    return L.h2o_sdpa_chunk(a["q"], a["kc"], a["vc"], a["kn"], a["vn"], a["out"], a["lse"],
                            a["wsum"], a["ws"], a["wsb"], a["B"], a["Hq"], a["Hkv"], a["T"],
                            a["M"], a["d"], a["scale"], a["dt"], a["st"])


@pytest.mark.parametrize("kw,code", [
    (dict(dt=7), H.H2O_EDTYPE),
    (dict(Hq=3, Hkv=2), H.H2O_ESHAPE),
    (dict(d=96), H.H2O_ESHAPE),
    (dict(B=0), H.H2O_ESHAPE),
    (dict(T=0), H.H2O_EINVAL),
    (dict(M=-1), H.H2O_EINVAL),
    (dict(q=None), H.H2O_EINVAL),
    (dict(wsum=None), H.H2O_EINVAL),
    (dict(kc=None), H.H2O_EINVAL),
    (dict(scale=float("nan")), H.H2O_EINVAL),
    (dict(scale=-1.0), H.H2O_EINVAL),
    (dict(out=MIS), H.H2O_EALIGN),
    (dict(vc=MIS), H.H2O_EALIGN),
    (dict(wsb=16), H.H2O_EWORKSPACE),
    (dict(M=1 << 30, d=128), H.H2O_ESHAPE),
])
def test_sdpa_rejects(L, kw, code):
    assert _sdpa(L, **kw) == code
    assert len(L.h2o_last_error()) > 0


def test_workspace_bytes(L):
    assert L.h2o_workspace_bytes(1, 4, 2, 64, 256, 64, 0) > 0
    assert L.h2o_workspace_bytes(1, 4, 2, 64, 256, 65, 0) == 0
    assert L.h2o_workspace_bytes(1, 4, 3, 64, 256, 64, 1) == 0
    assert L.h2o_workspace_bytes(1, 4, 2, 64, 256, 64, 5) == 0


def _evict(L, **kw):
    a = dict(kc=P, vc=P, sc=P, tp=P, kn=P, vn=P, w=P, idx=P, B=1, Hkv=2, M=16, T=4, d=64, k=4,
             pos0=16, dt=1, st=None)
    a.update(kw)
    return L.h2o_evict_insert(a["kc"], a["vc"], a["sc"], a["tp"], a["kn"], a["vn"], a["w"],
                              a["idx"], a["B"], a["Hkv"], a["M"], a["T"], a["d"], a["k"],
                              a["pos0"], a["dt"], a["st"])


@pytest.mark.parametrize("kw,code", [
    (dict(k=3), H.H2O_EINVAL),
    (dict(M=3), H.H2O_EINVAL),
    (dict(dt=2), H.H2O_EDTYPE),
    (dict(d=32), H.H2O_ESHAPE),
    (dict(Hkv=0), H.H2O_ESHAPE),
    (dict(sc=None), H.H2O_EINVAL),
    (dict(idx=None), H.H2O_EINVAL),
    (dict(tp=MIS), H.H2O_EALIGN),
    (dict(T=0, k=0), H.H2O_EINVAL),
])
def test_evict_rejects(L, kw, code):
    assert _evict(L, **kw) == code


def _evict_policy(L, **kw):
    a = dict(kc=P, vc=P, sc=P, tp=P, kn=P, vn=P, w=P, idx=P, B=2, Hkv=2, M=16, T=4, d=64, k=4,
             pos0=16, dt=1, pol=1, ws=P, wsb=1 << 20, st=None)
    a.update(kw)
    return L.h2o_evict_insert_policy(a["kc"], a["vc"], a["sc"], a["tp"], a["kn"], a["vn"],
                                     a["w"], a["idx"], a["B"], a["Hkv"], a["M"], a["T"], a["d"],
                                     a["k"], a["pos0"], a["dt"], a["pol"], a["ws"], a["wsb"],
                                     a["st"])


def test_evict_workspace_bytes(L):
    # h2o: none; norm: B*Hkv*M floats; orig: Hkv*M floats + Hkv*k indices (256-B sections)
    assert L.h2o_evict_workspace_bytes(2, 2, 16, 4, 0) == 0
    assert L.h2o_evict_workspace_bytes(2, 2, 1000, 4, 1) == 16128
    assert L.h2o_evict_workspace_bytes(2, 2, 1000, 4, 2) == 8192 + 256
    assert L.h2o_evict_workspace_bytes(2, 2, 16, 4, 7) == 0
    assert L.h2o_evict_workspace_bytes(0, 2, 16, 4, 1) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(pol=3), H.H2O_EINVAL),
    (dict(pol=-1), H.H2O_EINVAL),
    (dict(pol=1, tp=None), H.H2O_EINVAL),
    (dict(pol=1, wsb=64), H.H2O_EWORKSPACE),
    (dict(pol=2, wsb=64), H.H2O_EWORKSPACE),
    (dict(pol=2, ws=None), H.H2O_EINVAL),
    (dict(pol=1, ws=MIS), H.H2O_EALIGN),
    (dict(pol=2, k=3), H.H2O_EINVAL),
    (dict(pol=1, dt=5), H.H2O_EDTYPE),
    (dict(pol=2, sc=None), H.H2O_EINVAL),
])
def test_evict_policy_rejects(L, kw, code):
    assert _evict_policy(L, **kw) == code
    assert len(L.h2o_last_error()) > 0


STEP_FNS = ["h2o_chunk_step", "h2o_chunk_step_attend", "h2o_chunk_step_evict"]


def _step(L, fn="h2o_chunk_step", **kw):
    a = dict(q=P, kc=P, vc=P, sc=P, tp=P, kn=P, vn=P, out=P, lse=P, w=P, idx=P, ws=P,
             wsb=1 << 40, B=1, Hq=4, Hkv=2, T=4, M=16, d=64, scale=0.125, pos0=16, dt=1, st=None)
    a.update(kw)
    return getattr(L, fn)(a["q"], a["kc"], a["vc"], a["sc"], a["tp"], a["kn"], a["vn"],
                          a["out"], a["lse"], a["w"], a["idx"], a["ws"], a["wsb"], a["B"],
                          a["Hq"], a["Hkv"], a["T"], a["M"], a["d"], a["scale"], a["pos0"],
                          a["dt"], a["st"])


@pytest.mark.parametrize("kw,code", [
    (dict(dt=3), H.H2O_EDTYPE),
    (dict(Hq=6, Hkv=4), H.H2O_ESHAPE),
    (dict(M=3), H.H2O_EINVAL),
    (dict(sc=None), H.H2O_EINVAL),
    (dict(idx=None), H.H2O_EINVAL),
    (dict(q=None), H.H2O_EINVAL),
    (dict(scale=0.0), H.H2O_EINVAL),
    (dict(tp=MIS), H.H2O_EALIGN),
    (dict(sc=MIS), H.H2O_EALIGN),
    (dict(lse=MIS), H.H2O_EALIGN),
    (dict(wsb=8), H.H2O_EWORKSPACE),
])
@pytest.mark.parametrize("fn", STEP_FNS)
def test_chunk_step_rejects(L, kw, code, fn):
    assert _step(L, fn, **kw) == code
    assert len(L.h2o_last_error()) > 0


def _noalloc(L, **kw):
    a = dict(q=P, kc=P, vc=P, sc=P, tp=P, kn=P, vn=P, out=P, lse=P, w=P, idx=P, B=1, Hq=4,
             Hkv=2, T=4, M=16, d=64, scale=0.125, pos0=16, dt=1, st=None)
    a.update(kw)
    return L.h2o_chunk_step_noalloc(a["q"], a["kc"], a["vc"], a["sc"], a["tp"], a["kn"],
                                    a["vn"], a["out"], a["lse"], a["w"], a["idx"], a["B"],
                                    a["Hq"], a["Hkv"], a["T"], a["M"], a["d"], a["scale"],
                                    a["pos0"], a["dt"], a["st"])


def test_noalloc_scratch_limit(L):
    """The allocation-free step has a fixed 32 MiB scratch array: a shape
    whose workspace exceeds it (the long-cache shape needs 66 MiB) is refused
    on the host before anything else; the decode shape fits."""
    assert L.h2o_noalloc_scratch_bytes() == 32 << 20
    assert L.h2o_workspace_bytes(4, 32, 8, 512, 32768, 128, 1) > 32 << 20
    assert _noalloc(L, B=4, Hq=32, Hkv=8, T=512, M=32768, d=128) == H.H2O_EWORKSPACE
    assert b"h2o_chunk_step_noalloc" in L.h2o_last_error()
    assert L.h2o_workspace_bytes(8, 32, 8, 1, 4096, 64, 1) <= 32 << 20
    assert _noalloc(L, dt=3) == H.H2O_EDTYPE
    assert _noalloc(L, Hq=6, Hkv=4) == H.H2O_ESHAPE


def _cache(L, **kw):
    a = dict(q=P, kc=P, vc=P, tp=P, out=P, lse=P, w=P, ws=P, wsb=1 << 40, B=1, Hq=4, Hkv=2, T=8,
             M=16, d=64, scale=0.125, pos0=100, dt=1, st=None)
    a.update(kw)
    return L.h2o_sdpa_cache(a["q"], a["kc"], a["vc"], a["tp"], a["out"], a["lse"], a["w"],
                            a["ws"], a["wsb"], a["B"], a["Hq"], a["Hkv"], a["T"], a["M"], a["d"],
                            a["scale"], a["pos0"], a["dt"], a["st"])


def _step_if(L, **kw):
    a = dict(q=P, kc=P, vc=P, sc=P, tp=P, kn=P, vn=P, out=P, lse=P, w=P, idx=P, ws=P,
             wsb=1 << 40, B=1, Hq=4, Hkv=2, T=4, M=16, d=64, scale=0.125, pos0=16, dt=1, pol=0,
             st=None)
    a.update(kw)
    return L.h2o_chunk_step_insert_first(
        a["q"], a["kc"], a["vc"], a["sc"], a["tp"], a["kn"], a["vn"], a["out"], a["lse"],
        a["w"], a["idx"], a["ws"], a["wsb"], a["B"], a["Hq"], a["Hkv"], a["T"], a["M"], a["d"],
        a["scale"], a["pos0"], a["dt"], a["pol"], a["st"])


def test_cache_workspace_bytes(L):
    base = L.h2o_cache_workspace_bytes(2, 8, 2, 16, 1000, 64, 1, 0)
    assert base > 0 and base % 256 == 0
    # the policy's eviction scratch comes on top (h2o_norm: B*Hkv*M floats)
    assert L.h2o_cache_workspace_bytes(2, 8, 2, 16, 1000, 64, 1, 1) == base + 16128
    assert L.h2o_cache_workspace_bytes(2, 8, 2, 16, 0, 64, 1, 0) == 0      # M >= 1
    assert L.h2o_cache_workspace_bytes(2, 8, 2, 16, 1000, 64, 1, 5) == 0   # policy
    assert L.h2o_cache_workspace_bytes(2, 8, 3, 16, 1000, 64, 1, 0) == 0   # Hq % Hkv


@pytest.mark.parametrize("kw,code", [
    (dict(tp=None), H.H2O_EINVAL),
    (dict(M=0), H.H2O_EINVAL),
    (dict(q=None), H.H2O_EINVAL),
    (dict(w=None), H.H2O_EINVAL),
    (dict(tp=MIS), H.H2O_EALIGN),
    (dict(lse=MIS), H.H2O_EALIGN),
    (dict(dt=4), H.H2O_EDTYPE),
    (dict(d=80), H.H2O_ESHAPE),
    (dict(scale=float("inf")), H.H2O_EINVAL),
    (dict(wsb=32), H.H2O_EWORKSPACE),
])
def test_sdpa_cache_rejects(L, kw, code):
    assert _cache(L, **kw) == code
    assert len(L.h2o_last_error()) > 0


@pytest.mark.parametrize("kw,code", [
    (dict(tp=None), H.H2O_EINVAL),
    (dict(sc=None), H.H2O_EINVAL),
    (dict(kn=None), H.H2O_EINVAL),
    (dict(idx=None), H.H2O_EINVAL),
    (dict(M=3), H.H2O_EINVAL),
    (dict(pol=9), H.H2O_EINVAL),
    (dict(sc=MIS), H.H2O_EALIGN),
    (dict(vn=MIS), H.H2O_EALIGN),
    (dict(pol=1, wsb=64), H.H2O_EWORKSPACE),
    (dict(dt=2), H.H2O_EDTYPE),
])
def test_step_insert_first_rejects(L, kw, code):
    assert _step_if(L, **kw) == code
    assert len(L.h2o_last_error()) > 0


def _bwd(L, **kw):
    a = dict(q=P, kc=P, vc=P, kn=P, vn=P, tp=None, lse=P, do=P, dq=P, dkc=P, dvc=P, dkn=P,
             dvn=P, ws=P, wsb=1 << 40, B=1, Hq=4, Hkv=2, T=8, M=16, d=64, scale=0.125, pos0=0,
             dt=1, st=None)
    a.update(kw)
    return L.h2o_sdpa_chunk_backward(
        a["q"], a["kc"], a["vc"], a["kn"], a["vn"], a["tp"], a["lse"], a["do"],
        a["dq"], a["dkc"], a["dvc"], a["dkn"], a["dvn"], a["ws"], a["wsb"], a["B"], a["Hq"],
        a["Hkv"], a["T"], a["M"], a["d"], a["scale"], a["pos0"], a["dt"], a["st"])


def test_backward_workspace_bytes(L):
    # one float per query row (B*Hkv*G*T = 2*8*16 rows), in 256-byte units: too
    # few key tiles (4) for a key-range split
    assert L.h2o_backward_workspace_bytes(2, 8, 2, 16, 100, 64, 1) == 1024
    assert L.h2o_backward_workspace_bytes(2, 8, 2, 16, 100, 64, 0) == 1024
    assert L.h2o_backward_workspace_bytes(2, 8, 3, 16, 100, 64, 1) == 0
    # B1 Hq32 Hkv8 d128 M8192 T1024: 128 blocks of 256 rows (8-wave blocks,
    # one per CU on 256 CUs), so both bf16 rows passes split the keys 2 ways
    # to fill one round: the D pass's two planes plus a plane for their sum,
    # and the dq pass's float32 partials; float32 keeps one float per row
    rows = 8 * 4096
    assert L.h2o_backward_workspace_bytes(1, 32, 8, 1024, 8192, 128, 1) == \
        (2 + 1) * rows * 4 + 2 * rows * 128 * 4
    assert L.h2o_backward_workspace_bytes(1, 32, 8, 1024, 8192, 128, 0) == rows * 4


@pytest.mark.parametrize("kw,code", [
    (dict(dt=3), H.H2O_EDTYPE),
    (dict(d=48), H.H2O_ESHAPE),
    (dict(Hq=5), H.H2O_ESHAPE),
    (dict(dq=None), H.H2O_EINVAL),
    (dict(dkn=None), H.H2O_EINVAL),
    (dict(lse=None), H.H2O_EINVAL),
    (dict(tp=P, M=0), H.H2O_EINVAL),
    (dict(do=MIS), H.H2O_EALIGN),
    (dict(tp=MIS), H.H2O_EALIGN),
    (dict(wsb=16), H.H2O_EWORKSPACE),
    (dict(scale=0.0), H.H2O_EINVAL),
])
def test_backward_rejects(L, kw, code):
    assert _bwd(L, **kw) == code
    assert len(L.h2o_last_error()) > 0


@pytest.mark.parametrize("fn", ["h2o_kv_gather", "h2o_kv_scatter"])
def test_kv_copy_rejects(L, fn):
    f = getattr(L, fn)
    assert f(P, P, P, 1, 2, 16, 17, 64, 1, None) == H.H2O_ESHAPE     # k > M
    assert f(P, P, P, 1, 2, 16, 4, 32, 1, None) == H.H2O_ESHAPE      # d
    assert f(P, P, P, 1, 2, 16, 4, 64, 7, None) == H.H2O_EDTYPE
    assert f(None, P, P, 1, 2, 16, 4, 64, 1, None) == H.H2O_EINVAL
    assert f(P, MIS, P, 1, 2, 16, 4, 64, 1, None) == H.H2O_EALIGN


@pytest.mark.parametrize("args,code", [
    ((P, 4, 10, 11, P, None), H.H2O_EINVAL),
    ((P, 4, 10, -1, P, None), H.H2O_EINVAL),
    ((None, 4, 10, 3, P, None), H.H2O_EINVAL),
    ((MIS, 4, 10, 3, P, None), H.H2O_EALIGN),
])
def test_bottomk_rejects(L, args, code):
    assert L.h2o_bottomk(*args) == code


def test_accumulate_rejects(L):
    assert L.h2o_accumulate_scores(None, P, 1, 2, 8, 1, None) == H.H2O_EINVAL
    assert L.h2o_accumulate_scores(P, P, 0, 2, 8, 1, None) == H.H2O_ESHAPE
    assert L.h2o_accumulate_scores(P, MIS, 1, 2, 8, 1, None) == H.H2O_EALIGN


def test_debug_path_hook(L):
    assert L.h2o_debug_force_path(5) == H.H2O_EINVAL
    assert L.h2o_debug_force_path(-1) == H.H2O_OK


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a device is visible")
def test_no_device_is_reported(L):
    assert _sdpa(L) == H.H2O_ENODEVICE
    assert _evict(L) == H.H2O_ENODEVICE
    assert L.h2o_bottomk(P, 4, 10, 3, P, None) == H.H2O_ENODEVICE
    assert L.h2o_accumulate_scores(P, P, 1, 2, 8, 1, None) == H.H2O_ENODEVICE
    for fn in STEP_FNS:
        assert _step(L, fn) == H.H2O_ENODEVICE
    for pol in (0, 1, 2):
        assert _evict_policy(L, pol=pol) == H.H2O_ENODEVICE
    assert _evict_policy(L, pol=0, ws=None, wsb=0) == H.H2O_ENODEVICE
    assert _evict_policy(L, pol=2, tp=None) == H.H2O_ENODEVICE
    assert _cache(L) == H.H2O_ENODEVICE
    assert _bwd(L) == H.H2O_ENODEVICE
    assert _bwd(L, tp=P, kn=None, vn=None, dkn=None, dvn=None) == H.H2O_ENODEVICE
    assert L.h2o_kv_gather(P, P, P, 1, 2, 16, 4, 64, 1, None) == H.H2O_ENODEVICE
    assert L.h2o_kv_scatter(P, P, P, 1, 2, 16, 4, 64, 1, None) == H.H2O_ENODEVICE
    for pol in (0, 1, 2):
        assert _step_if(L, pol=pol) == H.H2O_ENODEVICE
    assert _noalloc(L) == H.H2O_ENODEVICE
    assert _noalloc(L, B=8, Hq=32, Hkv=8, T=1, M=4096, d=64) == H.H2O_ENODEVICE


def test_binding_raises_typed_errors(L):
    with pytest.raises(H.H2OError) as e:
        H._check(L.h2o_debug_force_path(9))
    assert e.value.status == H.H2O_EINVAL and "H2O_EINVAL" in str(e.value)


def test_binding_refuses_host_tensors():
    q = torch.zeros(1, 2, 4, 64)
    kc = torch.zeros(1, 1, 8, 64)
    with pytest.raises(ValueError):
        H.h2o_sdpa_chunk(q, kc, kc, q[:, :1], q[:, :1], q, torch.zeros(1, 2, 4),
                         torch.zeros(1, 1, 12), torch.zeros(16, dtype=torch.uint8))
