"""Float64 oracle of the streaming codebook synchronisation (test
infrastructure, see oracle/__init__).

Sec. 3.5 ("Codebook Synchronization") and App. F: sender and receiver keep
identical codebooks by sending, with each micro-batch, a random subset of
the codewords instead of the whole codebook; the codebook is partitioned
into random subsets and one subset travels per micro-batch (a 1/5 fraction
in the hyperparameter table of App. H).  The random partition is an input
here (a permutation of the K codeword indices per round, split into
`parts` consecutive pieces); the sender gathers the chosen rows, the
receiver writes them into its copy.
"""
import numpy as np


def partition(perm, parts):
    """Split a permutation of range(K) into `parts` consecutive subsets,
    the first K % parts of them one element longer."""
    perm = np.asarray(perm)
    return np.array_split(perm, parts)


def pack(C, rows):
    """Sender: buf[l, i] = C[l, rows[l, i]] for rows [L, n]."""
    C = np.asarray(C)
    rows = np.asarray(rows)
    return np.stack([C[l][rows[l]] for l in range(C.shape[0])])


def unpack(C_recv, buf, rows):
    """Receiver: its copy with C_recv[l, rows[l, i]] = buf[l, i]; other rows
    unchanged.  Rows of one round must be distinct."""
    out = np.array(C_recv, copy=True)
    rows = np.asarray(rows)
    for l in range(out.shape[0]):
        out[l][rows[l]] = buf[l]
    return out
