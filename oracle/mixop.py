"""Oracle of the swap-integrity test op MIX (test infrastructure).

MIX is not part of the paper's method: it is an integer function used to
check that every byte a function reads after arbitrary swaps is the byte the
sequence last wrote.  The last variable y is written; every other variable
(and y itself when it is also read) is read:
y[j] = seed ^ (j * 2654435761 mod 2^32) ^ (sum over read x of x[j mod len(x)]) mod 2^32.
"""

import numpy as np


def mix(reads, y_len, seed):
    j = np.arange(y_len, dtype=np.uint64)
    acc = np.zeros(y_len, dtype=np.uint64)
    for x in reads:
        acc += x[j % len(x)].astype(np.uint64)
    acc &= 0xFFFFFFFF
    h = (j * np.uint64(2654435761)) & np.uint64(0xFFFFFFFF)
    return (np.uint64(seed) ^ h ^ acc).astype(np.uint32)


def run(var_words, var_kinds, fns, init):
    """Executes a MIX-only sequence: fns = [(vars, accesses, seed)], init = {var: uint32 array}
    for the variables that hold a value at the start.  Returns every variable's final words."""
    val = {v: np.array(a, dtype=np.uint32) for v, a in init.items()}
    for vs, acc, seed in fns:
        y = vs[-1]
        reads = [val[v] for v in vs[:-1]]
        if acc[-1] & 1:
            reads.append(val[y])
        val[y] = mix(reads, var_words[y], seed)
    return val
