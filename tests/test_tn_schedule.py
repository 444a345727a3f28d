"""Host check of the work split of the 256 x 256 weight-gradient kernel
(gemm_tnw.hip): G workgroups first run whole items (item g + k G while full
rounds remain), then equal shares of the (item, step) space of the rest.
A segment of an item shared by several workgroups goes to its workgroup's
partial slot, and a second pass (tnw_reduce_kernel) adds the segments of
each shared item from those slots.

The arithmetic below restates the kernel's (share boundaries floor(Lw q / G),
the workgroup of a position, slot 0 for a share's first segment and 1 for its
last, workgroups with an empty share skipped) and checks the properties the
kernels rely on: every (item, step) is computed exactly once, no two
segments write the same slot, and the second pass finds exactly the item's
segments, in token order, each in the slot its writer used.  CPU only."""
import pytest


def share_of(x, Lw, G):
    q = (x * G) // Lw
    while q + 1 < G and (Lw * (q + 1)) // G <= x:
        q += 1
    while q > 0 and (Lw * q) // G > x:
        q -= 1
    return q


def segments(I, S, G):
    """(workgroup, item, s0, s1, whole, which) in each workgroup's order."""
    full, left = divmod(I, G)
    Lw = left * S
    out = []
    for g in range(G):
        for rd in range(full):
            out.append((g, rd * G + g, 0, S, True, 0))
        r0, r1 = Lw * g // G, Lw * (g + 1) // G
        x = r0
        while x < r1:
            li, s0 = divmod(x, S)
            s1 = min(S, s0 + (r1 - x))
            out.append((g, full * G + li, s0, s1, s0 == 0 and s1 == S, 0 if x == r0 else 1))
            x += s1 - s0
    return out


CASES = [(272, 256, 256), (272, 64, 256), (208, 256, 256), (208, 64, 256), (208, 512, 208),
         (192, 33, 192), (1, 1, 256),
         (3, 2, 256), (255, 7, 256), (256, 5, 256), (257, 5, 256), (513, 33, 256),
         (1000, 129, 256), (17, 1000, 256), (64, 128, 256), (5, 3, 8)]


@pytest.mark.parametrize("I,S,G", CASES)
def test_every_step_once_and_slots_consistent(I, S, G):
    segs = segments(I, S, G)
    full, left = divmod(I, G)
    Lw = left * S
    seen = [[0] * S for _ in range(I)]
    slots = {}
    per_item = {}
    for g, item, s0, s1, whole, which in segs:
        assert 0 <= item < I and 0 <= s0 < s1 <= S
        for t in range(s0, s1):
            seen[item][t] += 1
        if not whole:
            assert item >= full * G, "only the remaining items are shared"
            assert (g, which) not in slots, "two segments in one slot"
            slots[(g, which)] = (item, s0, s1)
            per_item.setdefault(item, []).append((g, s0))
    assert all(c == 1 for row in seen for c in row)
    for item, parts in per_item.items():
        li = item - full * G
        g_first = share_of(li * S, Lw, G)
        g_last = share_of((li + 1) * S - 1, Lw, G)
        # The workgroups in [g_first, g_last] with a non-empty share hold the
        # item's segments, in token order.
        has = [gk for gk in range(g_first, g_last + 1) if (Lw * (gk + 1)) // G > (Lw * gk) // G]
        assert sorted(g for g, _ in parts) == has
        assert [s0 for _g, s0 in sorted(parts)] == sorted(s0 for _g, s0 in parts)
        for gk in has:
            wk = 0 if (Lw * gk) // G >= li * S else 1
            assert slots[(gk, wk)][0] == item, "reader looks in the wrong slot"


@pytest.mark.parametrize("I,S,G", CASES)
def test_equal_shares(I, S, G):
    """Every workgroup gets the same number of steps, up to one."""
    steps = [0] * G
    for g, _item, s0, s1, _w, _which in segments(I, S, G):
        steps[g] += s1 - s0
    assert max(steps) - min(steps) <= 1
    assert sum(steps) == I * S
