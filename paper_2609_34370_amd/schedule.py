"""Host-side closed forms of the scheduling model around selective speculation (Sec. 5).

With a drop ratio alpha, a pipeline of N stages and a batch budget B, the total batch size of
speculative-parallel execution follows B_{t+1} = alpha B_{t+1-N} + (1 - alpha) B_t (Eq. 3) and
settles at B*_alpha = B / (1 + alpha (N - 1)).  Counting only accepted work, with Theta_alpha the
speculation accuracy of the drafts that are kept, the effective batch is (Eq. 4)
    B*_eff,alpha = alpha B*_alpha + (1 - alpha) B*_alpha / (N - Theta_alpha (N - 1)).
"""


def steady_batch(B: float, alpha: float, N: int) -> float:
    """B*_alpha of Eq. 3."""
    if not (0.0 <= alpha < 1.0) or N < 1:
        raise ValueError("alpha must be in [0, 1) and N >= 1")
    return B / (1.0 + alpha * (N - 1))


def effective_batch(B: float, alpha: float, N: int, theta_alpha: float) -> float:
    """B*_eff,alpha of Eq. 4 for the speculation accuracy theta_alpha of the kept drafts."""
    if not (0.0 <= theta_alpha <= 1.0):
        raise ValueError("theta_alpha must be in [0, 1]")
    bs = steady_batch(B, alpha, N)
    return alpha * bs + (1.0 - alpha) * bs / (N - theta_alpha * (N - 1))
