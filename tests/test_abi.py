"""C-ABI checks that need no GPU: the library loads, exports every function the
header declares, validates arguments before touching the device, and its host
logic (knapsack item quantisation) matches the oracle bit for bit."""
import ctypes as C
import math
import os
import re

import numpy as np
import pytest

import workloads as W
from oracle import additive as A
import paper_2602_20217_amd as PKG
from paper_2602_20217_amd import _lib as K


def _declared():
    src = open(PKG.HEADER_PATH).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ks_[a-z_0-9]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 20
    for n in names:
        assert hasattr(K.lib, n), n
    assert sorted(K.EXPORTS) == names


def _desc(**kw):
    d = dict(L=4, d=256, hq=4, hkv=2, hd=64, ffn=1024, vocab=1024, n_max=512, qk_norm=0,
             dtype=K.KS_F32, eps=1e-6, rope_theta=1e4)
    d.update(kw)
    return K.ModelDesc(*[d[f] for f, _ in K.ModelDesc._fields_])


def test_sizes_and_validation():
    lim = K.Limits(4, 5, 64, 64)
    d = _desc()
    assert K.ks_kv_cache_bytes(C.byref(d)) == 4 * 2 * 2 * 512 * 64 * 4
    assert K.ks_workspace_bytes(C.byref(d), C.byref(lim)) > 0
    for bad in (dict(hd=128), dict(hq=3), dict(d=100), dict(vocab=1000), dict(n_max=1),
                dict(dtype=7), dict(L=0), dict(dtype=K.KS_BF16, hd=64)):
        assert K.ks_kv_cache_bytes(C.byref(_desc(**bad))) == 0, bad
        assert K.last_error()
    for bad in (K.Limits(16, 5, 64, 64), K.Limits(4, 0, 64, 64), K.Limits(4, 5, 0, 64),
                K.Limits(4, 5, 64, 10)):
        assert K.ks_workspace_bytes(C.byref(d), C.byref(bad)) == 0


def test_null_and_range_errors_before_any_launch():
    with pytest.raises(K.KsError) as e:
        K.ks_create(None, None, None, None, 0, None, 0, None, None)
    assert e.value.status == K.KS_EINVAL
    with pytest.raises(K.KsError) as e:
        K.ks_pack_matrix(None, None, 16, 32, K.KS_BF16, None)
    assert e.value.status == K.KS_EINVAL
    with pytest.raises(K.KsError):
        K.ks_hidden_cos(None, None, 1, 1, 1, None, None)
    fake = C.c_void_p(16)  # never dereferenced: validation fails first
    with pytest.raises(K.KsError) as e:
        K.ks_knapsack_batch(fake, fake, 1, 72, 9000, 10, fake, fake, None)
    assert "C must be" in str(e.value)
    with pytest.raises(K.KsError):
        K.ks_knapsack_batch_select(fake, fake, fake, fake, 1, 200, 64, 10, fake, fake, fake, fake,
                                   None)
    with pytest.raises(K.KsError):
        K.ks_knapsack_batch(fake, fake, 1, 72, 64, -1, fake, fake, None)
    with pytest.raises(K.KsError) as e:  # a timing bracket needs both events
        K.ks_time_launches(fake, None)
    assert e.value.status == K.KS_EINVAL
    K.ks_time_launches(None, None)  # closing with nothing open: no HIP call


def test_sampling_calls_validate_before_any_launch():
    fake = C.c_void_p(16)  # never dereferenced: validation fails first
    ok = K.Sampling(0.7, 50, 0.95, 1)
    ws = K.ks_sample_workspace_bytes(2, 128256, 50)
    assert ws > 0 and K.ks_sample_workspace_bytes(2, 128256, 128) > 0
    for rows, vocab, k in ((0, 1000, 5), (1, 0, 5), (1, 40, 50), (1, 1000, 0), (1, 1000, 129),
                           (1, 600000, 128)):
        assert K.ks_sample_workspace_bytes(rows, vocab, k) == 0, (rows, vocab, k)
    for s in (K.Sampling(0.0, 50, 0.95, 1), K.Sampling(float("inf"), 50, 0.95, 1),
              K.Sampling(0.7, 0, 0.95, 1), K.Sampling(0.7, 129, 0.95, 1),
              K.Sampling(0.7, 50, 0.0, 1), K.Sampling(0.7, 50, 1.01, 1)):
        with pytest.raises(K.KsError) as e:
            K.ks_sample_filter(fake, 2, 128256, 128256, C.byref(s), 0, 2, fake, fake, fake, None,
                               None, fake, ws, None)
        assert e.value.status == K.KS_EINVAL
    with pytest.raises(K.KsError) as e:  # workspace too small
        K.ks_sample_filter(fake, 2, 128256, 128256, C.byref(ok), 0, 2, fake, fake, fake, None,
                           None, fake, ws - 1, None)
    assert e.value.status == K.KS_ENOMEM
    with pytest.raises(K.KsError):  # row stride below the vocabulary
        K.ks_sample_filter(fake, 2, 128256, 1000, C.byref(ok), 0, 2, fake, fake, fake, None,
                           None, fake, ws, None)
    with pytest.raises(K.KsError):
        K.ks_sample_filter(None, 2, 128256, 128256, C.byref(ok), 0, 2, fake, fake, fake, None,
                           None, fake, ws, None)
    with pytest.raises(K.KsError):
        K.ks_spec_accept(fake, fake, fake, fake, fake, fake, fake, 2000, 0, 0, fake, None)
    with pytest.raises(K.KsError):
        K.ks_spec_accept(fake, fake, fake, None, None, None, None, 3, 0, 0, fake, None)
    with pytest.raises(K.KsError):
        K.ks_sample_uniforms(0, fake, -1, 0, fake, None)
    K.ks_sample_uniforms(0, None, 0, 0, None, None)  # nothing to do: no launch


def test_knapsack_quantize_matches_oracle_bit_exact():
    inst = W.knapsack_instances(B=64, n_items=72, seed=2)
    w0, q0 = A.quantize_items(inst["t"], inst["s"], 4096)
    t = np.ascontiguousarray(inst["t"])
    s = np.ascontiguousarray(inst["s"])
    w = np.zeros_like(w0)
    q = np.zeros_like(q0)
    K.ks_knapsack_quantize(t.ctypes.data, s.ctypes.data, 64, 72, 4096, w.ctypes.data, q.ctypes.data)
    np.testing.assert_array_equal(w, w0)
    np.testing.assert_array_equal(q, q0)
    bad = t.copy()
    bad[0, 0] = -1.0
    with pytest.raises(K.KsError):
        K.ks_knapsack_quantize(bad.ctypes.data, s.ctypes.data, 64, 72, 4096, w.ctypes.data,
                               q.ctypes.data)


def test_product_package_does_not_touch_oracle():
    root = os.path.dirname(PKG.__file__)
    for dirpath, _, files in os.walk(root):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in txt and "from oracle" not in txt, f
                assert "workloads" not in txt, f


def test_single_hip_runtime_in_process():
    """The library binds to the HIP runtime torch loaded: exactly one libamdhip64 and
    one libhsa-runtime64 are mapped after import."""
    maps = open("/proc/self/maps").read().splitlines()
    hip = {l.split()[-1] for l in maps if "libamdhip64" in l}
    hsa = {l.split()[-1] for l in maps if "libhsa-runtime64" in l}
    assert len(hip) == 1 and len(hsa) == 1, (hip, hsa)
