"""Learning-rate schedules of the paper's training runs (host scalars passed
to Network.optimizer_step each step).

Methods / "Implementation" and the hyper-parameter tables: on Yin-Yang both
learning rates decay at the end of every epoch (factor 0.998 per epoch); on
SHD and SSC the weight learning rate eases in, starting at 0.001 times its
final value and growing at the end of every batch (factor 1.05 per batch)
until it reaches that value; the delay learning rate is constant there.
"""


def epoch_decay(base: float, epoch: int, factor: float = 0.998) -> float:
    """base * factor**epoch (Yin-Yang weights and delays)."""
    if epoch < 0:
        raise ValueError("epoch must be >= 0")
    return base * factor ** epoch


def ease_in(base: float, batch: int, start: float = 1e-3, growth: float = 1.05) -> float:
    """min(base, base * start * growth**batch) (SHD / SSC weights)."""
    if batch < 0:
        raise ValueError("batch must be >= 0")
    if not (0.0 < start <= 1.0) or growth < 1.0:
        raise ValueError("need 0 < start <= 1 and growth >= 1")
    return min(base, base * start * growth ** batch)
