"""Paged KV cache bookkeeping, written out plainly. Test infrastructure only.

The paper's engine keeps per-request KV state (§2.2) and its capacity model
counts KV in tokens (§1, K = B*S); it does not fix a block policy. Reading:
16-token blocks; the physical blocks are handed out in the order of a seeded
random permutation so that a sequence's blocks are scattered, as in a
long-running engine:

  * the random stream is splitmix64 (S. Vigna, public-domain reference
    implementation "splitmix64.c"): state += 0x9E3779B97F4A7C15, then the
    output is state mixed by two xor-shift-multiply rounds and a final
    xor-shift;
  * the permutation is the Fisher-Yates shuffle in Durstenfeld's form: for
    i = n-1 down to 1, draw r and swap entries i and r mod (i + 1);
  * sequence b = 0, 1, ... takes the next ceil((ctx_b + reserve) / 16)
    entries of the permutation as its logical blocks 0, 1, ...; unused
    table entries are -1.

A token at position p of sequence b lives at slot
block_table[b][p // block_size] * block_size + p % block_size.
"""

MASK64 = (1 << 64) - 1


def splitmix64_stream(seed, n):
    """The first n outputs of splitmix64 seeded with `seed` (Python ints)."""
    state = seed & MASK64
    out = []
    for _ in range(n):
        state = (state + 0x9E3779B97F4A7C15) & MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        out.append(z ^ (z >> 31))
    return out


def fisher_yates(n, seed):
    """Durstenfeld's shuffle of [0, n) driven by splitmix64(seed)."""
    a = list(range(n))
    draws = splitmix64_stream(seed, max(n - 1, 0))
    for step, i in enumerate(range(n - 1, 0, -1)):
        j = draws[step] % (i + 1)
        a[i], a[j] = a[j], a[i]
    return a


def allocate_block_tables(ctx_lens, reserve, num_phys_blocks, max_blocks, seed, block_size=16):
    """Block tables (list of lists, -1 padded to max_blocks) or None when the
    physical blocks or the table width do not suffice."""
    perm = fisher_yates(num_phys_blocks, seed)
    tables, nxt = [], 0
    for ctx in ctx_lens:
        need = -(-(int(ctx) + int(reserve)) // block_size)
        if need > max_blocks or nxt + need > num_phys_blocks:
            return None
        row = perm[nxt:nxt + need] + [-1] * (max_blocks - need)
        nxt += need
        tables.append(row)
    return tables


def slot_of(block_table_row, pos, block_size=16):
    """Physical slot of token `pos` of one sequence."""
    return block_table_row[pos // block_size] * block_size + pos % block_size
