"""Closed-form values behind the hand-worked adaptive-gamma cases in
ada_hand.json (Phase 4, Eq. gamma_estimator; Algorithm 2 UpdateGamma).

Written from the definitions, not from the oracle or the kernel:
  - a request alone on an idle server (default engine: base 5000 us, 2 us per
    token, context / 100) takes one prefill iteration of 5000 + 2P + P // 100
    us, then one decode iteration per further token j of 5002 + (P + j) // 100
    us, so its end-to-end latency is L(P, D);
  - the estimator is gamma_hat = tau ln(0.05 / 0.01) / max(t99 - t95, eps)
    with tau = 5000 us per token and nearest-rank t95, t99 of the window;
  - the EMA is gamma <- (1 - beta) gamma + beta gamma_hat per iteration, then
    the clip to [gamma_min, gamma_max].

    python tests/golden/ada_hand_calc.py      # prints the values
"""
from __future__ import annotations

import math

TAU = 5000.0
LN5 = math.log(0.05) - math.log(0.01)


def alone(P: int, D: int) -> int:
    """End-to-end latency (us) of a request alone on an idle server."""
    t = 5000 + 2 * P + P // 100
    for j in range(1, D):
        t += 5002 + (P + j) // 100
    return t


def nearest_rank(values, q: int) -> int:
    s = sorted(values)
    return s[(q * len(s) + 99) // 100 - 1]


def estimate(window, eps_us: float) -> float:
    d = float(nearest_rank(window, 99) - nearest_rank(window, 95))
    return TAU * LN5 / max(d, eps_us)


def expected():
    """Expected final gamma per case (and the isolated-request latencies)."""
    lat20 = [alone(100, d) for d in (7, 13, 1, 20, 4, 16, 9, 2, 18, 11, 5, 14, 19, 3, 10, 6,
                                      17, 8, 12, 15)]
    g = estimate(lat20, 1000.0)  # t99 - t95 = L(100, 20) - L(100, 19) = 5003
    ema1 = 0.75 * 1e-3 + 0.25 * g  # two iterations see the full window
    ema2 = 0.75 * ema1 + 0.25 * g
    flat = [alone(100, 5)] * 20
    low = [alone(1, 1)] * 19 + [alone(100, 1600)]
    return {
        "ada_estimator": {"gamma_final": g, "ttlt_alone": lat20},
        "ada_ema": {"gamma_final": ema2},
        "ada_eps_floor": {"gamma_final": estimate(flat, 1000.0)},
        "ada_clip_high": {"gamma_final": min(estimate(flat, 1000.0), 5.0)},
        "ada_clip_low": {"gamma_final": max(estimate(low, 1000.0), 0.002)},
        "ada_min_samples": {"gamma_final": 1e-3},
        # requests 0-2 overlap; their completions enter the window in batch
        # order, which puts t99 - t95 at 6000 us
        "ada_window_batch_order": {"gamma_final": TAU * LN5 / 6000.0},
    }


if __name__ == "__main__":
    for name, v in expected().items():
        print(name, v)
