"""CPU oracle of the optimiser step: Adam (Kingma and Ba, "Adam: A Method for
Stochastic Optimization", Algorithm 1) in float64, as the paper's training
pipeline applies it (supplementary implementation details): one learning rate
per parameter channel, a second-moment decay of its own per parameter tensor
(0.99 for the decoder weights), every Gaussian updated whether or not it was
visible in the iteration, fp32 master values with a binary16 copy for the
passes that evaluate in half precision.

TEST INFRASTRUCTURE ONLY: imported by the test-suite and by the benchmark's
CPU-baseline leg; it imports nothing from the GPU package.

The step is written exactly in Algorithm 1's order and notation:
    m_t = b1 m_{t-1} + (1 - b1) g_t
    v_t = b2 v_{t-1} + (1 - b2) g_t^2
    mhat_t = m_t / (1 - b1^t),   vhat_t = v_t / (1 - b2^t)
    theta_t = theta_{t-1} - alpha mhat_t / (sqrt(vhat_t) + eps)
with alpha the learning rate of the element's row (planar [rows][n] layout:
the row is the channel).
"""
from __future__ import annotations

import numpy as np


def adam_step(theta, g, m, v, lr_rows, beta1: float, beta2: float, eps: float, t: int):
    """One step on planar [rows][n] arrays; returns (theta_t, m_t, v_t) in float64.
    lr_rows has one learning rate per row."""
    theta = np.asarray(theta, np.float64)
    g = np.asarray(g, np.float64)
    m = np.asarray(m, np.float64)
    v = np.asarray(v, np.float64)
    alpha = np.asarray(lr_rows, np.float64).reshape(-1, 1)
    assert theta.ndim == 2 and alpha.shape[0] == theta.shape[0] and t >= 1
    m_t = beta1 * m + (1.0 - beta1) * g
    v_t = beta2 * v + (1.0 - beta2) * g * g
    mhat = m_t / (1.0 - beta1 ** t)
    vhat = v_t / (1.0 - beta2 ** t)
    theta_t = theta - alpha * mhat / (np.sqrt(vhat) + eps)
    return theta_t, m_t, v_t


def half_copy(theta32: np.ndarray) -> np.ndarray:
    """The binary16 copy of fp32 values (round to nearest even), as raw bits."""
    return np.asarray(theta32, np.float32).astype(np.float16).view(np.uint16)
