"""GPU vs oracle: ks_hidden_cos, the mean row cosine of Section 2 (cos(x, y) of
two rows; for matrices the mean over their rows) of every [r, d] group of X
against Y, through the C ABI, against ``oracle.select.cos_matrix``.

Shapes: the selection's own (49 budgets x 25 history rows x 4096), a single
row, d not a multiple of 4 (the scalar path), unaligned pointers (the scalar
path with aligned sizes), zero-norm rows (which score 0), r at the 8192 limit,
no groups at all, and X rows that are small perturbations of Y (cosines near 1,
as in the selection).  The device accumulates in float64 and rounds the mean
to float32, so the tolerance is 1e-6 absolute on values in [-1, 1]."""
import numpy as np
import pytest

from oracle import select as SEL

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = 1e-6


@pytest.fixture(scope="module")
def E():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd import engine
    return engine


def _inputs(G, r, d, seed, near=False):
    g = np.random.default_rng(seed)
    Y = g.standard_normal((r, d)).astype(np.float32)
    if near:
        X = Y[None] + np.float32(0.05) * g.standard_normal((G, r, d)).astype(np.float32)
    else:
        X = g.standard_normal((G, r, d)).astype(np.float32)
    return X.astype(np.float32), Y


def _check(E, X, Y, tag):
    G, r, d = X.shape
    out = E.hidden_cos(torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()).cpu().numpy()
    ref = np.array([SEL.cos_matrix(X[k], Y) for k in range(G)])
    err = float(np.max(np.abs(out - ref))) if G else 0.0
    print(f"[cos {tag}] G {G} r {r} d {d}: max abs err {err:.2e}", flush=True)
    assert out.shape == (G,)
    assert err < TOL, (tag, err)
    return out, ref


@pytest.mark.parametrize("G,r,d,near", [
    (49, 25, 4096, True),      # the selection's cells x history rows at d = 4096
    (49, 25, 4096, False),
    (65, 35, 4096, True),      # the 32K workload's history (gamma 6)
    (3, 1, 4096, False),       # one row per group
    (7, 5, 1001, False),       # d not a multiple of 4: scalar loads
    (4, 3, 6, True),           # d below one wave
    (2, 8192, 64, False),      # r at its upper limit
])
def test_hidden_cos_matches_oracle(E, G, r, d, near):
    X, Y = _inputs(G, r, d, seed=G * 7 + r + d, near=near)
    _check(E, X, Y, f"{'near' if near else 'random'}")


def test_hidden_cos_zero_rows_and_no_groups(E):
    X, Y = _inputs(6, 9, 256, seed=3)
    X[1, 4] = 0.0           # a zero row of X
    X[2] = 0.0              # a whole group of zero rows scores 0
    Y[7] = 0.0              # a zero row of Y: that row scores 0 in every group
    out, ref = _check(E, X, Y, "zero rows")
    assert out[2] == 0.0
    # no groups: nothing is written
    from paper_2602_20217_amd import _lib as K
    y = torch.from_numpy(Y).cuda()
    out = torch.full((1,), 7.0, device="cuda")
    K.ks_hidden_cos(y.data_ptr(), y.data_ptr(), 0, 9, 256, out.data_ptr(),
                    torch.cuda.current_stream().cuda_stream)
    assert out.item() == 7.0


def test_hidden_cos_unaligned_pointers(E):
    """X and Y one float past a 16-byte boundary: the kernel must take its
    scalar path and still match."""
    G, r, d = 5, 6, 512
    X, Y = _inputs(G, r, d, seed=9, near=True)
    xb = torch.zeros(G * r * d + 4, dtype=torch.float32, device="cuda")
    yb = torch.zeros(r * d + 4, dtype=torch.float32, device="cuda")
    xb[1:1 + G * r * d] = torch.from_numpy(X.reshape(-1)).cuda()
    yb[1:1 + r * d] = torch.from_numpy(Y.reshape(-1)).cuda()
    out = torch.empty(G, dtype=torch.float32, device="cuda")
    from paper_2602_20217_amd import _lib as K
    K.ks_hidden_cos(xb.data_ptr() + 4, yb.data_ptr() + 4, G, r, d, out.data_ptr(),
                    torch.cuda.current_stream().cuda_stream)
    got = out.cpu().numpy()
    ref = np.array([SEL.cos_matrix(X[k], Y) for k in range(G)])
    assert float(np.max(np.abs(got - ref))) < TOL


def test_hidden_cos_refuses_bad_sizes(E):
    from paper_2602_20217_amd import _lib as K
    x = torch.zeros(16, device="cuda")
    out = torch.zeros(1, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    for G, r, d in ((1, 0, 4), (1, 8193, 1), (-1, 1, 4), (1, 1, 0)):
        with pytest.raises(K.KsError) as e:
            K.ks_hidden_cos(x.data_ptr(), x.data_ptr(), G, r, d, out.data_ptr(), s)
        assert e.value.status == K.KS_EINVAL
