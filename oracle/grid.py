"""Toroidal grid and 5-cell von Neumann neighbourhoods (Section 2, spatial
coevolution: one centre plus four adjacent cells; Section 3, Figure 1(b); the
grid wraps around, i.e. it is a torus).

Cell id c = r * cols + col.  Slot order is [centre, north, south, west, east];
on grids with fewer than 3 rows or columns the same cell can occupy several
slots and every occurrence is kept as its own slot.
"""
import numpy as np

N_SLOTS = 5


def neighbours(rows, cols):
    nbr = np.empty((rows * cols, N_SLOTS), dtype=np.int64)
    for r in range(rows):
        for q in range(cols):
            c = r * cols + q
            nbr[c] = [c,
                      ((r - 1) % rows) * cols + q,
                      ((r + 1) % rows) * cols + q,
                      r * cols + (q - 1) % cols,
                      r * cols + (q + 1) % cols]
    return nbr
