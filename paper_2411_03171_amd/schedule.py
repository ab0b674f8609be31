"""Host-side schedules of the training loop around the library's calls.

SET topology updates run every ``interval`` steps and stop after a fraction of
the total steps (the appendix on DST settings: the topology is updated until
66 % of the training steps).  The auxiliary cluster head's loss carries a
weight that starts at ``w0`` and decays to zero at a cut-off epoch (Sec. 2.3;
the study of auxiliary cut-off epochs).  The paper does not give the decay's
shape: it is taken as linear in (fractional) epochs, and without a cut-off the
weight stays ``w0`` for the whole run.  At weight zero the head need not run
at all.

Steps are 1-based Adam step numbers t (the first update is t = 1); SET runs
after the update of step t.
"""
from __future__ import annotations

from typing import Optional

TOPOLOGY_STOP_FRAC = 0.66


def set_due(step: int, interval: int, total_steps: int, stop_frac: float = TOPOLOGY_STOP_FRAC) -> bool:
    """Whether SET runs after step ``step``: a multiple of the interval, and
    not past ``stop_frac`` of the total steps."""
    if interval < 1 or step < 1:
        return False
    return step % interval == 0 and step <= int(stop_frac * total_steps + 1e-9)


def set_round(step: int, interval: int) -> int:
    """Round counter of the SET draw stream for the update after ``step``
    (1 for the first update, 2 for the second, ...)."""
    return step // interval


def aux_weight(epoch: float, w0: float, cutoff_epoch: Optional[float]) -> float:
    """Weight of the auxiliary loss at (fractional) ``epoch``: w0 decaying
    linearly to 0 at ``cutoff_epoch``; 0 from then on; w0 throughout without a
    cut-off (None); 0 for a cut-off of 0 (no auxiliary loss)."""
    if cutoff_epoch is None:
        return float(w0)
    if cutoff_epoch <= 0 or epoch >= cutoff_epoch:
        return 0.0
    return float(w0) * (1.0 - max(0.0, float(epoch)) / float(cutoff_epoch))
