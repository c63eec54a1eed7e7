"""The C-ABI library loads on a CPU-only host, exports every entry point declared in
include/pearl_attn.h, and rejects bad host arguments synchronously (no GPU work is launched:
every call below fails validation before any HIP call)."""
import ctypes
import os
import re

import pytest

import paper_2609_35158_amd as pa
from paper_2609_35158_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pearl_attn.h")

FAKE = 0x10000          # aligned non-NULL device address: never dereferenced by these calls


def declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(pearl_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    from paper_2609_35158_amd import pd
    lib = pa.load()
    names = declared_functions()
    assert set(names) == set(bd.EXPORTED) | set(pd.EXPORTED), names
    assert "pearl_pd_decide" in names and "pearl_kv_pack" in names
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version_and_status_strings():
    assert pa.abi_version() == 1
    lib = pa.load()
    assert lib.pearl_status_str(0) == b"PEARL_OK"
    assert lib.pearl_status_str(3) == b"PEARL_ERR_WORKSPACE"
    assert lib.pearl_status_str(99) == b"PEARL_ERR_UNKNOWN"


def shape(hq=32, hkv=8, d=128, ps=16, n=1000):
    return bd.KvShape(hq, hkv, d, ps, n)


def desc(batch=4, stride=64, cu=None, total=None, max_q=1, max_kv=1000):
    total = batch if total is None else total
    return bd.SeqDesc(FAKE, stride, FAKE, cu, batch, total, max_q, max_kv)


def ws_bytes(s, d):
    return pa.load().pearl_attn_workspace_bytes(ctypes.byref(s), ctypes.byref(d))


def test_workspace_bytes():
    small = ws_bytes(shape(), desc())
    big = ws_bytes(shape(), desc(batch=64, stride=2100, max_kv=33000))
    assert 0 < small < big
    assert small % 256 == 0 and big % 256 == 0
    assert ws_bytes(shape(hkv=6), desc()) == 0 and "multiple" in pa.last_error()
    assert ws_bytes(shape(), desc(stride=10, max_kv=1000)) == 0 and "bt_stride" in pa.last_error()


def call(fn, s, d, q=FAKE, kp=FAKE, vp=FAKE, scale=0.1, out=FAKE, lse=None, ws=FAKE, wsb=1 << 30):
    f = getattr(pa.load(), fn)
    st = f(None if s is None else ctypes.byref(s), None if d is None else ctypes.byref(d), q, kp, vp,
           scale, out, lse, ws, wsb, None)
    return st, pa.last_error()


INVALID, UNSUPPORTED, WORKSPACE = 1, 2, 3


@pytest.mark.parametrize("fn", ["pearl_attn_prefill_append", "pearl_attn_decode", "pearl_attn_mixed"])
def test_attention_host_validation(fn):
    cu = FAKE if fn != "pearl_attn_decode" else None
    good = dict(cu=cu)
    assert call(fn, None, desc(**good))[0] == INVALID
    assert call(fn, shape(), None)[0] == INVALID
    assert call(fn, shape(hkv=6), desc(**good))[0] == INVALID
    assert call(fn, shape(hq=32, hkv=2), desc(**good))[0] == UNSUPPORTED       # G = 16
    assert call(fn, shape(d=96), desc(**good))[0] == UNSUPPORTED
    assert call(fn, shape(ps=32), desc(**good))[0] == UNSUPPORTED
    assert call(fn, shape(), desc(batch=0, **good))[0] == INVALID
    assert call(fn, shape(), desc(stride=2, max_kv=1000, **good))[0] == INVALID
    assert call(fn, shape(), desc(**good), q=None)[0] == INVALID
    assert call(fn, shape(), desc(**good), out=FAKE + 2)[0] == INVALID        # misaligned
    assert call(fn, shape(), desc(**good), scale=0.0)[0] == INVALID
    assert call(fn, shape(), desc(**good), scale=float("nan"))[0] == INVALID
    assert call(fn, shape(), desc(**good), ws=None)[0] == WORKSPACE
    assert call(fn, shape(), desc(**good), wsb=16)[0] == WORKSPACE
    assert call(fn, shape(), desc(**good), ws=FAKE + 128)[0] == WORKSPACE      # not 256-aligned


def test_mode_specific_validation():
    st, msg = call("pearl_attn_decode", shape(), desc(cu=FAKE))
    assert st == INVALID and "cu_q_lens" in msg
    st, msg = call("pearl_attn_mixed", shape(), desc(cu=None))
    assert st == INVALID and "cu_q_lens" in msg
    st, msg = call("pearl_attn_decode", shape(), desc(total=5))
    assert st == INVALID and "total_q" in msg


def test_kv_append_host_validation():
    lib = pa.load()
    s, d = shape(), desc()
    f = lib.pearl_kv_append
    assert f(ctypes.byref(s), ctypes.byref(d), None, FAKE, FAKE, FAKE, None) == INVALID
    assert f(ctypes.byref(s), ctypes.byref(d), FAKE + 4, FAKE, FAKE, FAKE, None) == INVALID
    assert f(ctypes.byref(shape(d=80)), ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None) == UNSUPPORTED
    assert f(None, ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None) == INVALID


@pytest.mark.parametrize("fn", ["pearl_kv_pack", "pearl_kv_unpack"])
def test_kv_transfer_host_validation(fn):
    f = getattr(pa.load(), fn)
    s, d = shape(), desc()
    assert f(ctypes.byref(s), ctypes.byref(d), FAKE, FAKE, None, None) == INVALID
    assert f(ctypes.byref(s), ctypes.byref(d), FAKE, FAKE + 8, FAKE, None) == INVALID   # misaligned
    assert f(ctypes.byref(shape(d=80)), ctypes.byref(d), FAKE, FAKE, FAKE, None) == UNSUPPORTED
    assert f(ctypes.byref(s), ctypes.byref(desc(batch=0)), FAKE, FAKE, FAKE, None) == INVALID
    assert f(None, ctypes.byref(d), FAKE, FAKE, FAKE, None) == INVALID
    assert f(ctypes.byref(s), ctypes.byref(desc(max_q=1 << 22, total=1 << 22, cu=FAKE, max_kv=1 << 23,
                                                stride=1 << 19)), FAKE, FAKE, FAKE, None) == UNSUPPORTED
    # nothing to move: succeeds without touching the GPU
    assert f(ctypes.byref(s), ctypes.byref(desc(total=0, cu=FAKE, max_q=0)), FAKE, FAKE, FAKE, None) == 0


def test_python_layer_refuses_cpu_tensors():
    import torch
    q = torch.zeros(2, 4, 64, dtype=torch.bfloat16)
    with pytest.raises((ValueError, TypeError)):
        pa.decode(q, q.view(2, 1, 4, 64), q.view(2, 1, 4, 64), torch.zeros(2, 1, dtype=torch.int32),
                  torch.zeros(2, dtype=torch.int32), 1)


def test_hbm_probe_host_validation():
    """The measurement kernels of include/pearl_bench.h reject bad arguments before any HIP call
    and do nothing for zero bytes."""
    lib = pa.load()
    assert lib.pearl_hbm_copy(FAKE, FAKE + 4096, 0, None) == 0
    assert lib.pearl_hbm_fill(FAKE, 0, 7, None) == 0
    assert lib.pearl_hbm_copy(FAKE, FAKE + 4096, 24, None) == INVALID and "multiple of 16" in pa.last_error()
    assert lib.pearl_hbm_copy(None, FAKE, 32, None) == INVALID and "null" in pa.last_error()
    assert lib.pearl_hbm_copy(FAKE, None, 32, None) == INVALID
    assert lib.pearl_hbm_read(FAKE + 8, 32, FAKE, None) == INVALID and "aligned" in pa.last_error()
    assert lib.pearl_hbm_read(FAKE, 32, FAKE + 4, None) == INVALID and "aligned" in pa.last_error()
    assert lib.pearl_hbm_read(FAKE, 32, None, None) == INVALID
    assert lib.pearl_hbm_read_nt(FAKE, 0, FAKE, None) == 0
    assert lib.pearl_hbm_read_nt(FAKE + 8, 32, FAKE, None) == INVALID and "aligned" in pa.last_error()
    assert lib.pearl_hbm_read_nt(FAKE, 24, FAKE, None) == INVALID and "multiple of 16" in pa.last_error()
    assert lib.pearl_hbm_fill(None, 32, 0, None) == INVALID
    assert lib.pearl_hbm_fill(FAKE, 40, 0, None) == INVALID


def call_static(s, d, q=FAKE, kp=FAKE, vp=FAKE, scale=0.1, out=FAKE, lse=None):
    st = pa.load().pearl_attn_decode_static(None if s is None else ctypes.byref(s),
                                            None if d is None else ctypes.byref(d), q, kp, vp, scale, out, lse, None)
    return st, pa.last_error()


def test_decode_static_host_validation():
    """The allocation-free decode checks its arguments like pearl_attn_decode, and rejects a batch
    whose workspace exceeds its static limit, all before any HIP call."""
    lib = pa.load()
    assert lib.pearl_attn_decode_static_max_bytes() == 32 << 20
    assert call_static(None, desc())[0] == INVALID
    assert call_static(shape(), None)[0] == INVALID
    assert call_static(shape(hq=32, hkv=2), desc())[0] == UNSUPPORTED
    assert call_static(shape(), desc(batch=0))[0] == INVALID
    assert call_static(shape(), desc(), q=None)[0] == INVALID
    assert call_static(shape(), desc(), out=FAKE + 2)[0] == INVALID
    assert call_static(shape(), desc(), scale=0.0)[0] == INVALID
    st, msg = call_static(shape(), desc(cu=FAKE))
    assert st == INVALID and "cu_q_lens" in msg
    # 2048 sequences of up to 32K keys need far more than 32 MiB of split partials
    big = desc(batch=2048, stride=2100, max_kv=33000)
    assert ws_bytes(shape(), big) > lib.pearl_attn_decode_static_max_bytes()
    st, msg = call_static(shape(), big)
    assert st == UNSUPPORTED and "static limit" in msg


def test_decode_append_host_validation():
    """The fused append-and-decode checks k_new / v_new and the decode layout before any HIP call."""
    lib = pa.load()

    def fused(s, d, k_new=FAKE, v_new=FAKE, ws=FAKE, wsb=1 << 30):
        st = lib.pearl_attn_decode_append(ctypes.byref(s), ctypes.byref(d), FAKE, k_new, v_new, FAKE, FAKE, 0.1,
                                          FAKE, None, ws, wsb, None)
        return st, pa.last_error()

    assert fused(shape(), desc(), k_new=None)[0] == INVALID
    assert fused(shape(), desc(), v_new=None)[0] == INVALID
    assert fused(shape(), desc(), k_new=FAKE + 8)[0] == INVALID
    st, msg = fused(shape(), desc(cu=FAKE))
    assert st == INVALID and "cu_q_lens" in msg
    assert fused(shape(hq=32, hkv=2), desc())[0] == UNSUPPORTED
    assert fused(shape(), desc(), wsb=16)[0] == WORKSPACE
