"""The windowed kernel's per-lane ready lists as a plain model (no GPU).

A lane keeps the ready nodes of its SMs in a near list (at most four
entries, all below the window end H) and a far list.  At a window start the
far entries below H move to near; those that do not fit go to the front of
the far list, so it reads [due | later | pushed since the window start].  A
local step then looks only at near, the due part, and -- once a due entry
was pushed while near was full -- the pushed part.  Taking an entry from the
due part moves the last due, later and pushed entries down one place each.

This model restates those list operations in Python, step for step as the
kernel takes them, and checks them against the plain rule they must keep:
each step selects, for every SM, the smallest entry below H among all of
that lane's entries (what a scan of every entry selects), and no entry is
lost or duplicated.  Random pushes, windows and steps over many seeds.
"""
import random

import pytest

K_NEAR = 4   # near entries per lane
SLOTS = 3    # SMs per lane


class Lane:
    def __init__(self):
        self.near, self.far = [], []
        self.fh = self.fa = 0        # end of the due part, start of the pushed part
        self.pushed_due = False
        self.live = set()

    def push(self, key, h_near):
        """A release (or root) entering the lists: below h_near it is due in
        the running window's local phase (h_near = 0 outside it)."""
        self.live.add(key)
        if key[0] < h_near:
            if len(self.near) < K_NEAR:
                self.near.append(key)
                return
            self.pushed_due = True
        self.far.append(key)

    def rebuild(self, H):
        """Window start: far entries below H to near, the rest that are below
        H first, in place (writes at or below the entry at hand)."""
        if self.far and min(k[0] for k in self.far) < H:
            orig, arr = list(self.far), list(self.far)
            kp = h = 0
            for i, k in enumerate(orig):
                if k[0] < H and len(self.near) < K_NEAR:
                    self.near.append(k)
                    continue
                if k[0] < H:
                    if h != kp:
                        arr[kp] = arr[h]
                    if h != i:
                        arr[h] = k
                    h += 1
                elif kp != i:
                    arr[kp] = k
                kp += 1
            self.far, self.fh, self.fa = arr[:kp], h, kp
        else:
            self.fh, self.fa = 0, len(self.far)
        self.pushed_due = False

    def candidates(self):
        out = [(k, ("n", i)) for i, k in enumerate(self.near)]
        if self.fh or self.pushed_due:
            out += [(self.far[i], ("f", i)) for i in range(self.fh)]
            if self.pushed_due:
                out += [(self.far[i], ("f", i)) for i in range(self.fa, len(self.far))]
        return out

    def take(self, where):
        kind, i = where
        if kind == "n":
            self.live.discard(self.near[i])
            self.near[i] = self.near[-1]
            self.near.pop()
            return
        far, fn = self.far, len(self.far)
        self.live.discard(far[i])
        if i >= self.fa:
            far[i] = far[fn - 1]
        else:
            v1, v2, v3 = far[self.fh - 1], far[self.fa - 1], far[fn - 1]
            if i != self.fh - 1:
                far[i] = v1
            if self.fh != self.fa:
                far[self.fh - 1] = v2
            if self.fa != fn:
                far[self.fa - 1] = v3
            self.fh -= 1
            self.fa -= 1
        far.pop()


def run(seed, windows=200):
    rnd = random.Random(seed)
    lane = Lane()
    serial = [0]

    def key(cycle):
        serial[0] += 1
        return (cycle, rnd.randrange(SLOTS), serial[0])  # (cycle, SM slot, node)

    T = 0
    for _ in range(windows):
        for _ in range(rnd.randrange(4)):  # completions and dispatch: far only
            lane.push(key(T + rnd.randrange(300)), 0)
        Lm = rnd.randrange(1, 60)
        H = T + Lm
        lane.rebuild(H)
        assert all(k[0] < H for k in lane.far[:lane.fh])
        assert all(k[0] >= H for k in lane.far[lane.fh:lane.fa])
        for _ in range(rnd.randrange(1, 10)):
            best = {}
            for k, where in lane.candidates():
                if k[0] < H and (k[1] not in best or k < best[k[1]][0]):
                    best[k[1]] = (k, where)
            plain = {}
            for k in lane.near + lane.far:
                if k[0] < H and (k[1] not in plain or k < plain[k[1]]):
                    plain[k[1]] = k
            assert {s: v[0] for s, v in best.items()} == plain
            if not plain:
                break
            # far entries before near ones, highest index first
            for where in sorted((v[1] for v in best.values()), key=lambda w: (w[0] == "f", w[1]), reverse=True):
                lane.take(where)
            for _ in range(rnd.randrange(5)):  # releases of the issued nodes
                lane.push(key(T + rnd.randrange(2 * Lm + 5)), H)
            assert sorted(lane.near + lane.far) == sorted(lane.live)
        T = H


@pytest.mark.parametrize("chunk", range(4))
def test_due_part_selects_as_a_full_scan(chunk):
    for seed in range(chunk * 25, chunk * 25 + 25):
        run(seed)
