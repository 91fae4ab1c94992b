"""Order of weight-cache operations in Weight-as-a-Service, written out
plainly. Test infrastructure only.

§4.2 "Asynchronous one-sided reading" and "Asynchronous buffer management":
a rank keeps a small set of pre-allocated cache slots; for each layer it
reserves a slot, issues the reads into it ahead of time (a lookahead window),
attaches a completion notification that the compute waits on just before it
uses the layer, and the slot is freed once compute on it has signalled done.
Layers are visited in a fixed order, so the schedule is static (§4.2, last
sentence of that paragraph; §4.4: event-driven, no CPU barrier).

Reading for one GPU with n_slots slots: layers are numbered globally across
decode iterations, g = step * L + l. Layer g uses slot g mod n_slots. The
first n_slots layers are filled up front; the fill of layer g + n_slots into
slot g mod n_slots waits for the compute of layer g to be done with it. Each
compute waits for its own fill. The copy stream always runs n_slots layers
ahead of compute, also across the end of an iteration: after the last layers
of iteration t, the first layers of iteration t + 1 are already being fetched.

Operations (tuples):
  ("fill", g, slot)         copy layer g mod L from the pool into slot
  ("wait_fill", g, slot)    compute stream waits for that fill
  ("compute", g, slot)      compute layer g mod L from slot
  ("done", g, slot)         compute stream signals the slot is free
  ("wait_done", g, slot)    copy stream waits for that signal
Listed per stream, in issue order.
"""


def was_schedule(num_layers, steps, n_slots=2):
    """Per-stream issue order for `steps` decode iterations of `num_layers`
    layers. Returns (copy_ops, compute_ops)."""
    total = num_layers * steps
    copy_ops, compute_ops = [], []
    if total == 0:
        return copy_ops, compute_ops
    for g in range(n_slots):
        copy_ops.append(("fill", g, g % n_slots))
    for g in range(total):
        s = g % n_slots
        compute_ops += [("wait_fill", g, s), ("compute", g, s), ("done", g, s)]
        copy_ops += [("wait_done", g, s), ("fill", g + n_slots, s)]
    return copy_ops, compute_ops
