"""The budget manager's rotation policy: the reference (oracle/pool.py)
pinned to the paper's properties, and the library's host-side policy
(cas_pool_plan_rotation) against it."""
import numpy as np

from oracle import pool


def test_b1_rotation_properties():
    """B1: with the paper's B = 20 and phi = 0.5, every rotation swaps 10;
    the admitted cartridges are never more trained than any offloaded one left
    behind, the evicted never less than any active one kept; over many
    rotations of R steps the step counts stay within a few R of each other
    (uniform coverage), and every cartridge gets trained."""
    N, B, R, phi = 90, 20, 10, 0.5
    steps = [0] * N
    active = set(pool.first_active(steps, B))
    assert active == set(range(B))
    for _ in range(60):
        for c in active:
            steps[c] += R
        mask = [c in active for c in range(N)]
        ev, ad = pool.plan_rotation(steps, mask, B, phi)
        assert len(ev) == len(ad) == 10
        assert set(ev) <= active and not (set(ad) & active)
        kept = active - set(ev)
        assert min(steps[c] for c in ev) >= max(steps[c] for c in kept)
        left = set(range(N)) - active - set(ad)
        assert max(steps[c] for c in ad) <= min(steps[c] for c in left)
        active = kept | set(ad)
    assert min(steps) > 0 and max(steps) - min(steps) <= 3 * R


def test_b2_edge_cases():
    """B2: nothing to swap when every cartridge is active or phi = 0; ties go
    to the lower id; phi * B is rounded down."""
    assert pool.plan_rotation([5, 5, 5], [True] * 3, 3, 0.5) == ([], [])
    assert pool.plan_rotation([1, 2, 3, 0], [True, True, False, False], 2, 0.0) == ([], [])
    assert pool.plan_rotation([4, 4, 0, 0, 0], [True, True, False, False, False], 2, 0.99) == ([0], [2])
    assert pool.plan_rotation([4, 4, 0, 0], [True, True, False, False], 2, 1.0) == ([0, 1], [2, 3])


def test_b3_library_policy_matches():
    import paper_2606_04557_amd as cas
    r = np.random.default_rng(3)
    for _ in range(200):
        N = int(r.integers(1, 40))
        B = int(r.integers(1, N + 1))
        phi = float(r.choice([0.0, 0.25, 0.5, 0.7, 1.0]))
        steps = [int(x) for x in r.integers(0, 5, N)]
        act = [False] * N
        for c in r.permutation(N)[:B]:
            act[int(c)] = True
        assert cas.plan_rotation(steps, act, B, phi) == pool.plan_rotation(steps, act, B, phi)
