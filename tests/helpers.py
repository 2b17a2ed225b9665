"""Shared test helpers: tolerance rules and the per-octant view of the
sibling-group neighbour table (for comparison with the oracle's per-octant
hash search)."""
import numpy as np

# fp32 features and input gradients vs the float64 oracle
RTOL, ATOL = 1e-4, 1e-5
# bf16 inputs/weights, fp32 accumulation, vs the fp32-input oracle
BF16_REL = 2e-2


def assert_f32_close(got, ref, what="", rtol=RTOL, atol=ATOL):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    err = np.abs(got - ref)
    bad = err > atol + rtol * np.abs(ref)
    if bad.any():
        i = np.argmax(err - (atol + rtol * np.abs(ref)))
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {bad.size} outside |g-r| <= {atol} + {rtol}|r|; "
            f"worst at {np.unravel_index(i, err.shape)}: got {got.flat[i]!r} ref {ref.flat[i]!r}")


def assert_dw_close(got, ref, what=""):
    """Elementwise rule first; if an entry near zero fails it, the scaled rule
    |g-r| <= 1e-5 max(1, rms(r)) + 1e-4 |r| (each dW entry sums over every
    output row, so relative error of near-zero sums is unbounded for any
    fp32 summation order).  Returns the name of the rule that passed."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    if np.all(err <= ATOL + RTOL * np.abs(ref)):
        return "elementwise"
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    tol = 1e-5 * max(1.0, rms) + RTOL * np.abs(ref)
    bad = err > tol
    if bad.any():
        i = np.argmax(err - tol)
        raise AssertionError(f"{what}: {int(bad.sum())} dW entries fail the scaled rule; worst "
                             f"got {got.flat[i]!r} ref {ref.flat[i]!r} rms {rms}")
    return "scaled"


def assert_bf16_close(got, ref, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rel2 = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    relmax = np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-300)
    assert rel2 <= BF16_REL and relmax <= BF16_REL, (what, rel2, relmax)


def per_octant_neighbors(nbr_groups, K):
    """Expand NB [G][27] (first-child rows of the 27 parent neighbours) into the
    per-octant table [8G][K^3] with the weight layout's tap order."""
    nbr_groups = np.asarray(nbr_groups, np.int64)
    G = nbr_groups.shape[0]
    r = (K - 1) // 2
    out = np.full((8 * G, K ** 3), -1, np.int64)
    k = 0
    for dx in range(-r, r + 1):
        for dy in range(-r, r + 1):
            for dz in range(-r, r + 1):
                for c in range(8):
                    ux, uy, uz = (c >> 2) + dx, ((c >> 1) & 1) + dy, (c & 1) + dz
                    o = ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)
                    base = nbr_groups[:, o]
                    child = 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1)
                    out[c::8, k] = np.where(base >= 0, base + child, -1)
                k += 1
    return out


def bf16_round(a):
    """Round float32 values to bfloat16 (nearest-even) and back, via torch."""
    import torch
    return torch.as_tensor(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()
