"""Server update after the backward: Adam and replica averaging.

Test infrastructure only (see the package docstring).

* Adam (Kingma & Ba, "Adam: A Method for Stochastic Optimization", 2015,
  Algorithm 1) is the optimizer the paper trains with (Section 4.1.4,
  Parameter Settings: Adam, learning rate 2e-2, batch size 1, no warmup, no
  weight decay).  The paper does not give beta1, beta2 or epsilon; the
  defaults of the Adam paper (0.9, 0.999, 1e-8) are used.
* Replica averaging is the aggregation of the server-hierarchical strategy
  (Section 3.3, Parallel Acceleration: one server-side model per client,
  parameters averaged at the end of each training period; the appendix on
  the averaging period uses periods of 50 and 100 steps).  The average is
  the unweighted elementwise mean of the replicas' parameters; optimizer
  state is not averaged (the paper averages parameters only).

float64 unless the caller passes float32 arrays and ``dtype``.
"""

from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np

ADAM_LR = 2e-2
ADAM_BETA1 = 0.9
ADAM_BETA2 = 0.999
ADAM_EPS = 1e-8


def adam_step(param: np.ndarray, grad: np.ndarray, exp_avg: np.ndarray, exp_avg_sq: np.ndarray, step: int,
              lr: float = ADAM_LR, beta1: float = ADAM_BETA1, beta2: float = ADAM_BETA2, eps: float = ADAM_EPS,
              dtype=np.float64) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One Adam update at time step ``step`` (1 for the first update).

    Algorithm 1 of the Adam paper, in its order: biased first moment
    m_t = b1 m + (1 - b1) g, biased second raw moment v_t = b2 v + (1 - b2) g^2,
    bias-corrected m_hat = m_t / (1 - b1^t) and v_hat = v_t / (1 - b2^t),
    then theta_t = theta - lr m_hat / (sqrt(v_hat) + eps).
    Returns (param, exp_avg, exp_avg_sq) after the step, as new arrays."""
    if step < 1:
        raise ValueError("Adam time steps start at 1")
    p = np.asarray(param, dtype)
    g = np.asarray(grad, dtype)
    m = beta1 * np.asarray(exp_avg, dtype) + (1 - beta1) * g
    v = beta2 * np.asarray(exp_avg_sq, dtype) + (1 - beta2) * g * g
    m_hat = m / (1 - beta1 ** step)
    v_hat = v / (1 - beta2 ** step)
    p = p - lr * m_hat / (np.sqrt(v_hat) + eps)
    return p.astype(dtype), m.astype(dtype), v.astype(dtype)


def average_replicas(replicas: Sequence[np.ndarray], dtype=np.float64) -> np.ndarray:
    """Elementwise mean of M replicas of one parameter tensor (Section 3.3,
    server-hierarchical strategy): the sum over replicas, in order, divided
    by M."""
    if len(replicas) == 0:
        raise ValueError("no replicas")
    acc = np.zeros(np.shape(replicas[0]), dtype)
    for r in replicas:
        acc = acc + np.asarray(r, dtype)
    return acc / len(replicas)
