"""The C-ABI library: it loads, exports every entry point include/frog.h
declares, and rejects bad arguments on the host before touching a GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2608_16491_amd as F
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "frog.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(frog_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = F.lib()
    names = _declared()
    assert len(names) >= 15
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(F.SYMBOLS)


def test_param_defaults_follow_the_paper():
    p = F.build_params(128)
    assert (p.m, p.ef_c, p.n_inv, p.patience) == (16, 128, 7, 30)
    assert (p.beta, p.gamma) == (0.2, 0.5)
    p = F.build_params(960)
    assert (p.m, p.ef_c, p.n_inv) == (32, 256, 6)
    s = F.search_params()
    assert (s.epn, s.budget, s.epn_frac) == (16, 16, 0.0)
    # the struct's tail fields as the library fills them (layout check)
    assert (s.hash_log2, s.entry_mode, s.hotspot_mode, s.eager_check) == (10, 0, 0, 0)


def _small_index(n=400, d=8):
    rng = np.random.default_rng(0)
    X = rng.standard_normal((n, d)).astype(np.float32)
    attr = rng.permutation(n).astype(np.float64)
    return X, attr


def test_build_rejects_bad_arguments():
    X, attr = _small_index()
    bad = attr.copy()
    bad[3] = np.nan
    with pytest.raises(F.FrogError) as e:
        F.Index.build(X, bad)
    assert e.value.code == -1 and "NaN" in str(e.value)
    with pytest.raises(F.FrogError):
        F.Index.build(X, attr, m=0)
    with pytest.raises(F.FrogError):
        F.Index.build(X, attr, m=16, ef_c=8)
    with pytest.raises(F.FrogError):
        F.Index.build(X, attr, beta=1.5)


def test_from_arrays_validates():
    X, attr = _small_index(64, 4)
    perm = np.arange(64, dtype=np.int32)
    E = -np.ones((64, 2, 4), np.int32)
    ix = F.Index.from_arrays(X, np.sort(attr), perm, E)
    assert ix.info() == (64, 4, 2, 4)
    with pytest.raises(F.FrogError):
        F.Index.from_arrays(X, attr, perm, E)                   # not ascending
    p2 = perm.copy(); p2[5] = 7
    with pytest.raises(F.FrogError):
        F.Index.from_arrays(X, np.sort(attr), p2, E)            # not a permutation
    E2 = E.copy(); E2[3, 1, 2] = 64
    with pytest.raises(F.FrogError):
        F.Index.from_arrays(X, np.sort(attr), perm, E2)         # entry out of range


def test_device_calls_need_an_uploaded_index():
    X, attr = _small_index()
    ix = F.Index.build(X, attr)
    L = F.lib()
    ids = np.zeros(10, np.int32)
    rc = L.frog_search(ix.handle, None, 1, None, None, 10, 64, None, None, None)
    assert rc == -5 and b"uploaded" in L.frog_last_error()
    rc = L.frog_bruteforce_filtered(ix.handle, None, 1, None, None, 10, None, None, None, None)
    assert rc == -5
    rc = L.frog_index_prepare_sample(ix.handle, 0)
    assert rc == -5 and b"uploaded" in L.frog_last_error()
    rc = L.frog_search(None, None, 1, None, None, 10, 64, None, None, None)
    assert rc == -1


def test_gpu_build_rejects_unsupported_shapes_on_the_host():
    # checked before any device is touched
    X, attr = _small_index(64, 4)
    with pytest.raises(F.FrogError) as e:
        F.Index.build(X, attr, device=0, m=64, ef_c=128)
    assert e.value.code == -7
    with pytest.raises(F.FrogError) as e:
        F.Index.build(X, attr, device=0, m=16, ef_c=512)
    assert e.value.code == -7
    with pytest.raises(F.FrogError) as e:
        F.Index.build(X, attr, device=0, beta=1.5)
    assert e.value.code == -1


def test_16bit_upload_rejects_on_the_host():
    # checked before any device is touched: unknown storage, d > 128, a
    # value that rounds past the largest binary16 (65504)
    L = F.lib()
    X, attr = _small_index(64, 4)
    ix = F.Index.from_arrays(X, np.sort(attr), np.arange(64, dtype=np.int32), -np.ones((64, 2, 4), np.int32))
    assert L.frog_index_upload_ex(ix.handle, 0, 7) == -1
    assert b"storage" in L.frog_last_error()
    with pytest.raises(ValueError):
        ix.upload(0, storage="fp8")
    X2 = X.copy()
    X2[10, 2] = 65520.0          # rounds to infinity
    ix2 = F.Index.from_arrays(X2, np.sort(attr), np.arange(64, dtype=np.int32), -np.ones((64, 2, 4), np.int32))
    assert L.frog_index_upload_ex(ix2.handle, 0, F.STORAGE_F16) == -7
    assert b"fp16 range" in L.frog_last_error()
    Xw = np.zeros((64, 130), np.float32)
    ix3 = F.Index.from_arrays(Xw, np.sort(attr), np.arange(64, dtype=np.int32), -np.ones((64, 2, 4), np.int32))
    assert L.frog_index_upload_ex(ix3.handle, 0, F.STORAGE_F16) == -7
    assert b"d <= 128" in L.frog_last_error()
    # bf16: a value that rounds to infinity (above the largest bf16,
    # (2 - 2^-7) 2^127) and a non-finite value
    X4 = X.copy()
    X4[3, 1] = np.float32(3.4028235e38)
    ix4 = F.Index.from_arrays(X4, np.sort(attr), np.arange(64, dtype=np.int32), -np.ones((64, 2, 4), np.int32))
    assert L.frog_index_upload_ex(ix4.handle, 0, F.STORAGE_BF16) == -7
    assert b"bf16 range" in L.frog_last_error()
    X5 = X.copy()
    X5[7, 0] = np.inf
    ix5 = F.Index.from_arrays(X5, np.sort(attr), np.arange(64, dtype=np.int32), -np.ones((64, 2, 4), np.int32))
    assert L.frog_index_upload_ex(ix5.handle, 0, F.STORAGE_BF16) == -7


def test_save_load_roundtrip_and_corruption(tmp_path):
    w = workloads.make("tiny", n=1500, nq=1)
    ix = F.Index.build(w.X, w.attr)
    path = str(tmp_path / "a.frog")
    ix.save(path)
    ix2 = F.Index.load(path)
    a, b = ix.export(), ix2.export()
    for key in a:
        assert (a[key] == b[key]).all(), key
    raw = bytearray(open(path, "rb").read())
    raw[100] ^= 0x40
    bad = str(tmp_path / "b.frog")
    open(bad, "wb").write(bytes(raw))
    with pytest.raises(F.FrogError) as e:
        F.Index.load(bad)
    assert e.value.code == -4
    open(bad, "wb").write(bytes(raw[:500]))
    with pytest.raises(F.FrogError) as e:
        F.Index.load(bad)
    assert e.value.code == -4
    with pytest.raises(F.FrogError) as e:
        F.Index.load(str(tmp_path / "missing.frog"))
    assert e.value.code == -6
