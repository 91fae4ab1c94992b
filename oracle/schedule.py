"""Order of weight-cache operations in Weight-as-a-Service, written out
plainly. Test infrastructure only.

§4.2 "Asynchronous one-sided reading" and "Asynchronous buffer management":
a rank keeps a small set of pre-allocated cache slots; for each layer it
reserves a slot, issues the reads into it ahead of time (a lookahead window),
attaches notifications that the compute waits on just before it uses the
layer, and the slot is freed once compute on it has signalled done. A slot
holds a layer's "tensor tiles", each read with its own notification. Layers
are visited in a fixed order, so the schedule is static (§4.2, end of that
paragraph; §4.4: event-driven, no CPU barrier).

Reading for one GPU with 2 slots: layers are numbered globally across decode
iterations, g = step * L + l, and layer g uses slot g mod 2. While layer g
computes, layer g + 1 is read into the other slot as two tiles: tile A as soon
as layer g - 1 has released that slot, tile B once layer g's attention half
has been issued (so that it overlaps layer g's projections). Layer g + 1's
compute waits for tile B's notification. Before the first layer, layer 0 is
read whole. The copy stream therefore always runs one layer ahead, also across
the end of an iteration.

Operations, in host issue order, as (kind, g, slot):
  ("fill_a", g, s)     copy tile A of layer g mod L into slot s
  ("fill_b", g, s)     copy tile B, then notify "filled"
  ("wait_fill", g, s)  compute waits for layer g's "filled"
  ("attn", g, s)       attention half of layer g
  ("mid", g, s)        compute notifies that the attention half is issued
  ("proj", g, s)       projection half of layer g
  ("done", g, s)       compute notifies that slot s is free
  ("wait_done", g, s)  copy waits for layer g's "done"
  ("wait_mid", g, s)   copy waits for layer g's "mid"
"""


def was_schedule(num_layers, steps):
    """Issue order of the ring operations for `steps` decode iterations of
    `num_layers` layers."""
    total = num_layers * steps
    ops = []
    if total == 0:
        return ops
    ops += [("fill_a", 0, 0), ("fill_b", 0, 0)]
    for g in range(total):
        s, n = g % 2, (g + 1) % 2
        if g > 0:
            ops.append(("wait_done", g - 1, n))
        ops += [("fill_a", g + 1, n), ("wait_fill", g, s), ("attn", g, s), ("mid", g, s),
                ("wait_mid", g, s), ("fill_b", g + 1, n), ("proj", g, s), ("done", g, s)]
    return ops
