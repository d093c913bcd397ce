"""Shared set-up of the GPU parity tests: seeded weights from ``workloads`` are
uploaded through the C ABI and also handed to the oracle."""
import numpy as np

import workloads as W
from oracle import model as M


def rel_err(a, b):
    """Row-wise ||a - b|| / ||b|| (max over rows)."""
    a = np.asarray(a, dtype=np.float64).reshape(-1, np.shape(b)[-1])
    b = np.asarray(b, dtype=np.float64).reshape(-1, np.shape(b)[-1])
    num = np.linalg.norm(a - b, axis=1)
    den = np.maximum(np.linalg.norm(b, axis=1), 1e-300)
    return float(np.max(num / den))


def build(name, n_max, gamma_max=6, m_rounds=5, cap_max=128, prefill_chunk=64, seed=0):
    from paper_2602_20217_amd.engine import DeviceModel
    cfg = W.config(name)
    weights = W.generate_weights(cfg, seed=seed)
    dm = DeviceModel(cfg, n_max=n_max, gamma_max=gamma_max, m_rounds=m_rounds,
                     cap_max=cap_max, prefill_chunk=prefill_chunk).upload_all(weights)
    return cfg, dm, M.Model(cfg, weights)


def margin(logits_row):
    """Top-1 minus top-2 logit."""
    s = np.sort(np.asarray(logits_row))
    return float(s[-1] - s[-2])
