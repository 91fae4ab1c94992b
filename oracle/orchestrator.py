"""The job orchestrator's choice between Weight-as-a-Service and
Compute-as-a-Service, written out plainly. Test infrastructure only.

§4.3 "Consistent mode switching": one central orchestrator decides the mode
for every engine of the data-parallel group, so all ranks agree on each
layer's communication pattern. It watches how many sequences each engine
still has active; while the effective batch stays at or above the
hardware-specific threshold B_th (the smallest batch whose forward time hides
a layer's weight fetch, from offline profiling) WaS stays; when it
persistently falls below, the group switches to CaS. Switches happen only at
coarse boundaries and with hysteresis, so the mode does not flap.

Readings (the paper gives no formulas):
  - effective batch of an iteration: the mean number of active sequences over
    all engines of the group (engines that ran out count as 0, they are the
    underutilised ones);
  - "persistently": the condition holds for `window` consecutive iterations;
  - hysteresis: back from CaS to WaS only when the effective batch is at least
    B_th * (1 + hysteresis) for `window` consecutive iterations;
  - a decision taken after iteration t applies from iteration t + 1; the job
    starts in WaS.
"""

WAS, CAS = 0, 1


def effective_batch(active):
    """Mean active sequences over the group's engines."""
    return sum(active) / len(active)


def mode_schedule(batches, b_th, hysteresis, window):
    """Mode of every iteration for a trace `batches` (one list of per-engine
    active counts per iteration): element t is the mode iteration t runs in."""
    mode, run, modes = WAS, 0, []
    for active in batches:
        modes.append(mode)
        b = effective_batch(active)
        if mode == WAS:
            run = run + 1 if b < b_th else 0
        else:
            run = run + 1 if b >= b_th * (1 + hysteresis) else 0
        if run >= window:
            mode, run = (CAS if mode == WAS else WAS), 0
    return modes
