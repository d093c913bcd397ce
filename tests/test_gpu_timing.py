"""Kernel timing brackets (ks_time_launches): launches made while a bracket is
open carry its events, so the elapsed time spans the bracket's kernels."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def K():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd import _lib
    return _lib


def _pair():
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    b.record()
    return a, b


def test_bracket_spans_its_launches(K):
    nb = 256 << 20
    buf = torch.empty(4 * nb, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    for k in range(4):  # clocks settle
        K.ks_stream_read(buf.data_ptr() + k * nb, nb, sink.data_ptr(), st)
    one, two = [], []
    for r in range(6):
        a, b = _pair()
        K.ks_time_launches(a.cuda_event, b.cuda_event)
        K.ks_stream_read(buf.data_ptr() + (r % 4) * nb, nb, sink.data_ptr(), st)
        K.ks_time_launches(None, None)
        c, d = _pair()
        K.ks_time_launches(c.cuda_event, d.cuda_event)
        K.ks_stream_read(buf.data_ptr() + ((r + 1) % 4) * nb, nb, sink.data_ptr(), st)
        K.ks_stream_read(buf.data_ptr() + ((r + 2) % 4) * nb, nb, sink.data_ptr(), st)
        K.ks_time_launches(None, None)
        one.append((a, b))
        two.append((c, d))
    torch.cuda.synchronize()
    t1 = sorted(a.elapsed_time(b) for a, b in one)[3]
    t2 = sorted(a.elapsed_time(b) for a, b in two)[3]
    # a 256 MiB read takes tens of microseconds at any rate this GPU reaches
    # (at most 8 TB/s: >= 33 us); two in one bracket take about twice as long
    assert 0.03 < t1 < 1.0, t1
    assert 1.5 * t1 < t2 < 2.6 * t1, (t1, t2)


def test_launches_after_a_closed_bracket_leave_its_events(K):
    nb = 64 << 20
    buf = torch.empty(nb, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    a, b = _pair()
    K.ks_time_launches(a.cuda_event, b.cuda_event)
    K.ks_stream_read(buf.data_ptr(), nb, sink.data_ptr(), st)
    K.ks_time_launches(None, None)
    torch.cuda.synchronize()
    t = a.elapsed_time(b)
    for _ in range(20):  # outside the bracket: the events keep their times
        K.ks_stream_read(buf.data_ptr(), nb, sink.data_ptr(), st)
    torch.cuda.synchronize()
    assert a.elapsed_time(b) == t


def test_decode_profile_launch_counts_and_times(K):
    """The decode-step profile (its launches carry their class's events): every
    class of a bf16 decode step has the launch count the step's structure fixes,
    positive times, and the classes add up to at most the step's own time."""
    import numpy as np
    import workloads as W
    from gpu_helpers import build
    cfg, dm, _ = build("small_bf16", n_max=160, gamma_max=4)
    try:
        dm.prefill(np.arange(40, dtype=np.int32) % cfg.vocab)
        pr = dm.profile_decode(None, 4, per_kernel=True)
        L = cfg.L
        want = {"embed": 1, "gemm_qkv": L, "attn": L, "combine": L, "gemm_o": L,
                "gemm_gate_up": L, "gemm_down": L, "gemm_head": 1, "argmax": 1}
        for name, n in want.items():
            assert pr["launches"][name] == n, (name, pr["launches"][name])
            assert pr["ms"][name] > 0, name
        total = sum(pr["ms"][k] * pr["launches"][k] for k in pr["ms"])
        assert 0 < total <= pr["ms_step"] * 1.02, (total, pr["ms_step"])
        # a mask that skips every attention sublayer drops their launches
        exec_mask = np.ones(2 * L, dtype=bool)
        exec_mask[0::2] = False
        pm = dm.profile_decode(exec_mask, 2, per_kernel=True)
        assert pm["launches"]["attn"] == 0 and pm["launches"]["gemm_qkv"] == 0
        assert pm["launches"]["gemm_gate_up"] == L
    finally:
        dm.close()
