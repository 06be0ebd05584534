"""Benchmark placeholder: the full harness lands with the HIP path."""


def mean_gain(t_opt: float, t_base: float) -> float:
    """The paper's mean gain G = 1 - E[T_opt] / E[T_base] (Section IV-G, Evaluation)."""
    return 1.0 - float(t_opt) / float(t_base)
