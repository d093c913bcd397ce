"""ks_sample_filter_noalloc (the sampling filter for callers that cannot
allocate: its scratch is a fixed array of the library) against ks_sample_filter
with a caller-allocated workspace, through the C ABI: identical tables, counts,
top-1 probabilities and draws on two calls in a row, the second on a smaller
input, and a refusal, before any launch, of a call that needs more scratch than
the array holds."""
import ctypes as C

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _noalloc(K, logits, temperature, top_k, top_p, seed, pos0):
    R, V = logits.shape
    s = K.Sampling(temperature, top_k, top_p, seed)
    dev = logits.device
    ids = torch.full((R, K.KS_SAMPLE_KMAX), -7, dtype=torch.int32, device=dev)
    probs = torch.full((R, K.KS_SAMPLE_KMAX), -7.0, dtype=torch.float32, device=dev)
    cnt = torch.full((R,), -7, dtype=torch.int32, device=dev)
    top1 = torch.full((R,), -7.0, dtype=torch.float32, device=dev)
    tok = torch.full((R,), -7, dtype=torch.int32, device=dev)
    K.ks_sample_filter_noalloc(logits.data_ptr(), R, V, logits.stride(0), C.byref(s), pos0, 2,
                               ids.data_ptr(), probs.data_ptr(), cnt.data_ptr(), top1.data_ptr(),
                               tok.data_ptr(), torch.cuda.current_stream().cuda_stream)
    return ids, probs, cnt, top1, tok


def _same(a, b):
    ids0, p0, c0, t0, k0 = [x.cpu().numpy() for x in a]
    ids1, p1, c1, t1, k1 = [x.cpu().numpy() for x in b]
    np.testing.assert_array_equal(c1, c0)
    for r in range(len(c0)):
        n = int(c0[r])
        np.testing.assert_array_equal(ids1[r, :n], ids0[r, :n])
        np.testing.assert_array_equal(p1[r, :n], p0[r, :n])
    np.testing.assert_array_equal(t1, t0)
    np.testing.assert_array_equal(k1, k0)


def test_noalloc_filter_equals_workspace_filter():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd import _lib as K
    from paper_2602_20217_amd.engine import sample_filter
    cases = [(3, 128256, 50, 0.7, 0.95, 11, 8192),  # the paper's sampling setting, 8B head
             (1, 4096, 8, 1.1, 0.6, 12, 5)]          # then a smaller call
    for R, V, k, T, p, seed, pos0 in cases:
        print(f"[noalloc] rows {R} vocab {V} top_k {k}", flush=True)
        lg = torch.from_numpy(W.synthetic_logits(R, V, seed=seed, index=R)).cuda()
        ref = sample_filter(lg, T, k, p, seed=seed, pos0=pos0)
        got = _noalloc(K, lg, T, k, p, seed, pos0)
        torch.cuda.synchronize()
        _same(ref, got)
    # a call that needs more scratch than the array holds is refused before any launch
    R, V, k = 300, 128256, 128
    assert K.ks_sample_workspace_bytes(R, V, k) > 4 << 20
    lg = torch.zeros(R, V, device="cuda")
    with pytest.raises(K.KsError) as e:
        _noalloc(K, lg, 0.7, k, 0.95, 1, 0)
    assert e.value.status == K.KS_ENOMEM
