"""The paper's decoding-latency model (appendix "Breakdown of Decoding Latency").

With t the target's forward-pass latency, t_bar the draft's per-pass latency,
d the draft rollout depth and tau the acceptance length, autoregressive
decoding of N tokens costs N*t and speculative decoding (N/tau)*(t + d*t_bar),
so the speedup is tau * t / (t + d*t_bar).  The paper's worked example
(t = 25 ms, t_bar = 1.5 ms, d = 6, tau = 5) gives about 3.68.
"""


def speedup_ratio(t: float, t_bar: float, d: int, tau: float) -> float:
    return t / (t + d * t_bar) * tau


def total_latency(n_tokens: int, t: float, t_bar: float = 0.0, d: int = 0,
                  tau: float = 1.0) -> float:
    """Latency of generating n_tokens: autoregressive when tau == 1 and d == 0."""
    return n_tokens / tau * (t + d * t_bar)
