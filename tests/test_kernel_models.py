"""CPU models of two steps of the prep pass, written in the order the kernel
takes them, checked against plain definitions (CPU only).

- The inverse T = (I + A)^-1 of the strictly lower-triangular A of a 64-token
  tile (the UT transform of the chunkwise form, A_ri = beta_r D_ri k_r . k_i
  for i < r): 16 x 16 diagonal blocks by forward substitution, each row's dot
  product split over four partial sums (terms i = p mod 4), then the
  off-diagonal blocks in two levels of the 2 x 2 block inverse
  [[T11, 0], [T21, T22]] with T21 = -T22 A21 T11 -- first the two 32 x 32
  halves, then the lower-left quarter as Y = A_[23][01] T_[01][01] and
  T_[23][01] = -T_[23][23] Y, block by block as four workgroup waves form it.
- The inclusive prefix sum of the gates over a 64-lane wave: row shifts by
  1, 2, 4, 8 inside rows of 16 lanes (lanes shifted in from outside a row read
  0), then the last lane of row 0 into row 1 and of row 2 into row 3, then
  the last lane of row 1 into rows 2 and 3.
"""
import numpy as np
import pytest


def blocked_unit_lower_inverse(A, dtype=np.float64):
    """(I + A)^-1 for strictly lower-triangular 64 x 64 A, in the kernel's order."""
    A = A.astype(dtype)
    T = np.zeros((64, 64), dtype)
    blk = lambda M, i, j: M[16 * i:16 * i + 16, 16 * j:16 * j + 16]
    # diagonal blocks: lane (c, p) holds the terms i = p mod 4 of row r's sum
    for b in range(4):
        Ab = blk(A, b, b)
        for c in range(16):
            x = np.zeros(16, dtype)
            for r in range(16):
                ps = np.zeros(4, dtype)
                for p in range(4):
                    for m in range((r + 3) // 4):
                        i = 4 * m + p
                        if i < 16:
                            ps[p] += Ab[r, i] * x[i]
                total = (ps[0] + ps[1]) + (ps[2] + ps[3])
                x[r] = (1.0 if r == c else 0.0) - total
            blk(T, b, b)[:, c] = x
    # first level: T_{2u+1,2u} = -T_{2u+1,2u+1} (A_{2u+1,2u} T_{2u,2u})
    for u in range(2):
        bi, bj = 2 * u + 1, 2 * u
        y = blk(A, bi, bj) @ blk(T, bj, bj)
        blk(T, bi, bj)[:] = -(blk(T, bi, bi) @ y)
    # second level: Y_ij = sum_{k = j..1} A_ik T_kj, then T_ij = -sum_{m = 2..i} T_im Y_mj
    Y = {}
    for i in (2, 3):
        for j in (0, 1):
            y = blk(A, i, j) @ blk(T, j, j)
            if j == 0:
                y = y + blk(A, i, 1) @ blk(T, 1, 0)
            Y[i, j] = y
    for i in (2, 3):
        for j in (0, 1):
            t = blk(T, i, 2) @ Y[2, j]
            if i == 3:
                t = t + blk(T, 3, 3) @ Y[3, j]
            blk(T, i, j)[:] = -t
    return T


def tile_A(rng, decay_scale=1.0, repeat=False):
    """A of one tile from unit keys, beta in (0, 1) and log decays g <= 0."""
    k = rng.standard_normal((64, 128))
    if repeat:  # keys repeated inside the tile (re-presented tokens): k_r . k_i near 1
        k[1::2] = k[0::2] + 0.05 * rng.standard_normal((32, 128))
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal(64)))
    g = -np.log1p(np.exp(rng.standard_normal(64))) * decay_scale
    gam = np.cumsum(g)
    D = np.exp(gam[:, None] - gam[None, :])
    return np.tril(beta[:, None] * D * (k @ k.T), -1)


@pytest.mark.parametrize("decay_scale,repeat", [(1.0, False), (1e-4, False), (1e-4, True), (0.0, True)])
def test_blocked_inverse_matches_definition(decay_scale, repeat):
    rng = np.random.default_rng(17)
    for _ in range(3):
        A = tile_A(rng, decay_scale, repeat)
        ref = np.linalg.inv(np.eye(64) + A)
        T = blocked_unit_lower_inverse(A)
        assert np.allclose(np.tril(T), T)
        assert np.allclose(np.diag(T), 1.0)
        assert np.max(np.abs(T - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref)))
        # in fp32, as the kernel computes it: well inside the fp16 rounding the
        # T fragments get afterwards (2^-11 relative)
        T32 = blocked_unit_lower_inverse(A, np.float32).astype(np.float64)
        err = np.linalg.norm(T32 - ref) / np.linalg.norm(ref)
        assert err <= 1e-5, err


def test_blocked_inverse_catches_a_wrong_level_formula():
    """The check above fails for a plausible slip in the second level (the
    first-level block T_32 left out of T_30), so it tests the order taken."""
    rng = np.random.default_rng(3)
    A = tile_A(rng, 1e-4, True)
    ref = np.linalg.inv(np.eye(64) + A)
    T = blocked_unit_lower_inverse(A)
    bad = T.copy()
    Y30 = A[48:64, 0:16] @ T[0:16, 0:16] + A[48:64, 16:32] @ T[16:32, 0:16]
    bad[48:64, 0:16] = -(T[48:64, 48:64] @ Y30)   # missing T_32 Y_20
    assert np.max(np.abs(bad - ref)) > 1e-3
    assert np.max(np.abs(T - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref)))


def wave_prefix_sum(x):
    v = np.array(x, dtype=np.float64)
    lanes = np.arange(64)

    def row_shr(v, n):
        out = np.zeros(64)
        src = lanes - n
        ok = src >= (lanes // 16) * 16
        out[ok] = v[src[ok]]
        return out
    for n in (1, 2, 4, 8):
        v = v + row_shr(v, n)
    b = np.zeros(64)
    rows13 = np.isin(lanes // 16, (1, 3))
    b[rows13] = v[(lanes[rows13] // 16) * 16 - 1]   # lane 15 of the row before
    v = v + b
    b = np.zeros(64)
    rows23 = lanes >= 32
    b[rows23] = v[31]
    return v + b


def test_wave_prefix_sum_is_the_inclusive_scan():
    rng = np.random.default_rng(5)
    for _ in range(20):
        x = rng.standard_normal(64)
        assert np.allclose(wave_prefix_sum(x), np.cumsum(x), rtol=0, atol=1e-12)
    x = np.zeros(64)
    x[[0, 15, 16, 31, 47, 63]] = 1.0
    assert np.array_equal(wave_prefix_sum(x), np.cumsum(x))
