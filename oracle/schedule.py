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

Layers owned by this rank (§4.1: each rank keeps the FFN weights of the
layers it owns, layer l being owned by rank l mod d when d ranks pool their
weights) are computed straight from the local pool: no read, no slot. The
ring above then runs over the layers this rank does not own, g counting only
those (g = step * Ls + j for the j-th non-owned layer of a step, Ls of them
per step), and an owned layer's compute sits between the ring operations of
its neighbours in layer order.

Operations, in host issue order, as (kind, g, slot):
  ("fill_a", g, s)     copy tile A of layer g mod L into slot s
  ("fill_b", g, s)     copy tile B, then notify "filled"
  ("wait_fill", g, s)  compute waits for the part of layer g's fill that its
                       attention half reads
  ("attn", g, s)       attention half of layer g
  ("mid", g, s)        compute notifies that the attention half is issued
  ("proj", g, s)       projection half of layer g (each projection first
                       waits for the part of the fill holding its weights;
                       the last of them waits for "filled")
  ("done", g, s)       compute notifies that slot s is free
  ("wait_done", g, s)  copy waits for layer g's "done"
  ("wait_mid", g, s)   copy waits for layer g's "mid"
  ("local", n, -1)     compute of owned layer n (n = step * L + l), from the pool
"""


def owned(layer, ranks, rank):
    """Whether this rank owns `layer` (ranks = 0: it owns none)."""
    return ranks > 0 and layer % ranks == rank


def was_schedule(num_layers, steps, ranks=0, rank=0):
    """Issue order of the ring operations for `steps` decode iterations of
    `num_layers` layers, on rank `rank` of `ranks` pooling ranks."""
    streamed = [l for l in range(num_layers) if not owned(l, ranks, rank)]
    total = len(streamed) * steps
    ops = []
    if total > 0:
        ops += [("fill_a", 0, 0), ("fill_b", 0, 0)]
    g = 0
    for step in range(steps):
        for l in range(num_layers):
            if owned(l, ranks, rank):
                ops.append(("local", step * num_layers + l, -1))
                continue
            s, n = g % 2, (g + 1) % 2
            if g > 0:
                ops.append(("wait_done", g - 1, n))
            ops += [("fill_a", g + 1, n), ("wait_fill", g, s), ("attn", g, s), ("mid", g, s),
                    ("wait_mid", g, s), ("fill_b", g + 1, n), ("proj", g, s), ("done", g, s)]
            g += 1
    return ops


def streamed_layer(g, num_layers, ranks=0, rank=0):
    """The layer (0 .. L-1) that ring instance g computes."""
    streamed = [l for l in range(num_layers) if not owned(l, ranks, rank)]
    return streamed[g % len(streamed)]


def peak_shift_order(num_layers, ranks, rank):
    """§4.2 "Peak shifting": the order in which rank `rank` of `ranks` (d)
    pulls the layers it does not own during one decode iteration. Layers form
    cycles of d consecutive indices; in the cycle starting at layer c the rank
    starts at layer c + rank and walks the cycle with wrap-around, skipping the
    layer it owns (§4.1: layer l belongs to rank l mod d). Layers past the end
    of the stack (a short last cycle) are left out. Returns a list of
    (layer, owner) pairs, owner = layer mod d.

    Reading: the text starts the walk at c + rank, which is the rank's own
    layer when cycles start at multiples of d, so the first pull is c + rank + 1."""
    d = ranks
    order = []
    for c in range(0, num_layers, d):
        for k in range(d):
            layer = c + (rank + k) % d
            if layer >= num_layers or owned(layer, d, rank):
                continue
            order.append((layer, layer % d))
    return order
