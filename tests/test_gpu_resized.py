"""A second context over the same uploaded weights (DeviceModel.resized) with
a larger KV cache generates exactly the tokens of a model built from scratch
with that cache size (speculative and autoregressive), and the first context
keeps working.  Through the C ABI."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_helpers import build

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def test_resized_context_matches_fresh_model():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_20217_amd.engine import select_params
    cfg, small, _ = build("small_bf16", n_max=1500)
    big = small.resized(14000)
    _, fresh, _ = build("small_bf16", n_max=14000)
    prompt = W.prompt_ids(cfg.vocab, 200, 5)
    params = select_params((1.0, 0.01, 0.2), "paper_min", 0)
    out = []
    for dm in (big, fresh):
        ar, _, _ = dm.generate(prompt, 24, gamma=0)
        sd, _, _ = dm.generate(prompt, 24, gamma=3, reselect_every=8, params=params)
        np.testing.assert_array_equal(sd, ar)
        out.append(ar)
    np.testing.assert_array_equal(out[0], out[1])
    ar_small, _, _ = small.generate(prompt, 8, gamma=0)
    assert len(ar_small) == 8
    for dm in (big, fresh, small):
        dm.close()
