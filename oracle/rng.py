"""Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers: As
Easy as 1, 2, 3", SC 2011), written from its published definition, and the
draws the coevolutionary algorithm makes from it.

Round function on a 4x32-bit counter (c0, c1, c2, c3) with key (k0, k1):
    (hi0, lo0) = M0 * c0,  (hi1, lo1) = M1 * c2        (32x32 -> 64-bit products)
    c' = (hi1 ^ c1 ^ k0,  lo1,  hi0 ^ c3 ^ k1,  lo0)
ten rounds, with the key advanced by the Weyl constants (W0, W1) between rounds.

Stream layout used by every draw of the method (both sides implement it):
    key     = (seed mod 2^32, seed >> 32)
    counter = (element // 4, cell, (gen << 16) | step_field, tag)
    word    = element % 4 of the 4-word output
step_field is 0 for the evaluation minibatch and s+1 for training step s.
"""
import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)
PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint64(0x9E3779B9)
PHILOX_W1 = np.uint64(0xBB67AE85)

TAG = dict(IDX=1, Z=2, TOURN_G=3, TOURN_D=4, LRMUT_G=5, LRMUT_D=6,
           MIXN=7, MIXZ=8, PROJ=9, INIT_G=10, INIT_D=11, NES_G=12, NES_D=13)


def philox4x32_10(ctr, key):
    """Philox4x32-10 block function.

    ctr: integer array [..., 4] of 32-bit counter words; key: (k0, k1).
    Returns a uint64 array [..., 4] holding the four 32-bit output words.
    """
    ctr = np.asarray(ctr, dtype=np.uint64)
    c0, c1, c2, c3 = ctr[..., 0], ctr[..., 1], ctr[..., 2], ctr[..., 3]
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = c0 * PHILOX_M0
        p1 = c2 * PHILOX_M1
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1)


def seed_key(seed):
    seed = int(seed)
    return (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)


def raw_words(seed, n, cell, gen, step_field, tag):
    """The first n 32-bit words of stream (cell, gen, step_field, tag)."""
    nb = (n + 3) // 4
    ctr = np.zeros((nb, 4), dtype=np.uint64)
    ctr[:, 0] = np.arange(nb, dtype=np.uint64)
    ctr[:, 1] = cell
    ctr[:, 2] = (int(gen) << 16) | int(step_field)
    ctr[:, 3] = TAG[tag] if isinstance(tag, str) else int(tag)
    return philox4x32_10(ctr, seed_key(seed)).reshape(-1)[:n]


def to_uniform(words):
    """Map 32-bit words to (0, 1): ((w >> 9) + 0.5) * 2^-23, a value in
    [2^-24, 1 - 2^-24] that is exact in fp32 as well as fp64."""
    return ((np.asarray(words, dtype=np.uint64) >> np.uint64(9)).astype(np.float64) + 0.5) * 2.0 ** -23


def uniforms(seed, n, cell, gen, step_field, tag):
    return to_uniform(raw_words(seed, n, cell, gen, step_field, tag))


def box_muller(u):
    """Four normals per 4 uniforms: (u0, u1) -> r cos, r sin with r = sqrt(-2 ln u0),
    angle 2 pi u1; likewise (u2, u3)."""
    u = np.asarray(u, dtype=np.float64).reshape(-1, 4)
    r01 = np.sqrt(-2.0 * np.log(u[:, 0]))
    r23 = np.sqrt(-2.0 * np.log(u[:, 2]))
    t01 = 2.0 * np.pi * u[:, 1]
    t23 = 2.0 * np.pi * u[:, 3]
    return np.stack([r01 * np.cos(t01), r01 * np.sin(t01),
                     r23 * np.cos(t23), r23 * np.sin(t23)], axis=1).reshape(-1)


def normals(seed, n, cell, gen, step_field, tag):
    nb = (n + 3) // 4
    return box_muller(uniforms(seed, 4 * nb, cell, gen, step_field, tag))[:n]


def indices(seed, n, n_samples, cell, gen, step_field, tag="IDX"):
    """Uniform integers in [0, n_samples): floor(w * n_samples / 2^32)."""
    w = raw_words(seed, n, cell, gen, step_field, tag)
    return ((w * np.uint64(n_samples)) >> np.uint64(32)).astype(np.int64)
