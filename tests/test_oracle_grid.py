import os

import numpy as np

from oracle import grid


def test_neighbours_hand_enumerated(golden_dir):
    with open(os.path.join(golden_dir, "neighbours.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            head, tail = line.split(":")
            r, c, cell = map(int, head.split())
            assert list(grid.neighbours(r, c)[cell]) == list(map(int, tail.split()))


def test_every_cell_fills_five_slots():
    for r, c in [(1, 1), (1, 4), (2, 2), (2, 3), (3, 3), (4, 4), (5, 7), (8, 8), (12, 12)]:
        nbr = grid.neighbours(r, c)
        assert nbr.shape == (r * c, 5)
        assert np.all(nbr[:, 0] == np.arange(r * c))
        assert np.all(np.bincount(nbr.ravel(), minlength=r * c) == 5)


def test_neighbour_relation_is_symmetric_on_large_grids():
    nbr = grid.neighbours(4, 5)
    for c in range(20):
        assert nbr[nbr[c, 1], 2] == c and nbr[nbr[c, 2], 1] == c
        assert nbr[nbr[c, 3], 4] == c and nbr[nbr[c, 4], 3] == c
