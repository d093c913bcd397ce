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
