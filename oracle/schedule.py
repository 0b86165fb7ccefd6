"""Integer schedule of the publisher/subscriber training loop.

Test infrastructure only (see ``oracle/__init__.py``).

The paper keys every embedding and gradient by the id of its batch and lets a
publisher run ahead of its subscriber (Section 4.1, "System Design"); a
channel holds at most p entries (buffer mechanism) and a gradient may be
computed at a parameter version up to the delay bound old (Assumption 4 and
the update rule of the Theorem).  Deterministic reading used here, with
staleness s:

* tick t: the passive party B publishes batch group t (while t < n_groups);
  the active party A consumes group u = t - s and returns its gradient; B
  back-propagates group u and updates its parameters.  Inside a tick, B's
  forward comes before B's update.
* ring slot of group g: g mod (s + 1) (s + 1 <= p slots are ever live).
* B's parameter version used by the forward of group g: max(0, g - s);
  delay of the update made with group u: min(u, s).
"""
from __future__ import annotations

TRACE_FIELDS = ("tick", "fwd_group", "fwd_slot", "fwd_version",
                "bwd_group", "bwd_slot", "version_after")


def tick_record(t: int, s: int, n_groups: int):
    """One trace row: (tick, group published or -1, its slot or -1, B's
    version used by that forward or -1, group consumed or -1, its slot or -1,
    B's version after this tick's update or -1)."""
    fwd = t if t < n_groups else -1
    u = t - s
    bwd = u if 0 <= u < n_groups else -1
    return (t,
            fwd, fwd % (s + 1) if fwd >= 0 else -1, max(0, fwd - s) if fwd >= 0 else -1,
            bwd, bwd % (s + 1) if bwd >= 0 else -1, bwd + 1 if bwd >= 0 else -1)


def trace(s: int, n_groups: int):
    """All trace rows of a run of ``n_groups`` groups (n_groups + s ticks)."""
    return [tick_record(t, s, n_groups) for t in range(n_groups + s)]
