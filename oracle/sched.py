"""Oracle of slice scheduling across GPUs and of bursty preemption control.

Test infrastructure only (see the package header).

Scheduling (section 5.2, Appendix C): m GPUs, one slice per unordered pair
{i, j} of `units` units. Every unit a request of GPU i needs goes, one unit at
a time, to the incident slice {i, j} (j != i) whose total use -- both users'
units -- is lowest (Greedy-Least-Loaded); readings taken where the paper is
silent: ties go to the lowest j; a slice with no free unit, or on which GPU i is
capped and at its cap, is skipped; a unit no slice can take is refused (peer
-1). A release frees the request's most recently placed units first.

Bursty preemption control (section 5.3): when GPU i is preempted on slice
{i, j} while holding more than half of it, its units there are capped at the
level it held, for a window of T ticks; a further such preemption inside the
window restarts it and lowers the cap if its level is lower; without one the
cap lifts when the window ends. T = 0 means no caps.
"""


class SchedOracle:
    def __init__(self, m, units, window):
        self.m, self.units, self.window = m, units, window
        self.use = [[0] * m for _ in range(m)]          # use[i][j]: GPU i's units on {i, j}
        self.cap = [[None] * m for _ in range(m)]       # (level, until) or None
        self.held = {}                                  # (gpu, req) -> list of peers, in order

    def total(self, i, j):
        return self.use[i][j] + self.use[j][i]

    def active_cap(self, i, j, t):
        c = self.cap[i][j]
        if c is not None and t < c[1]:
            return c[0]
        return None

    def place(self, gpu, req, n, t):
        peers = []
        for _ in range(n):
            choice = None
            for j in range(self.m):
                if j == gpu or self.total(gpu, j) >= self.units:
                    continue
                c = self.active_cap(gpu, j, t)
                if c is not None and self.use[gpu][j] >= c:
                    continue
                if choice is None or self.total(gpu, j) < self.total(gpu, choice):
                    choice = j
            if choice is None:
                peers.append(-1)
                continue
            self.use[gpu][choice] += 1
            self.held.setdefault((gpu, req), []).append(choice)
            peers.append(choice)
        return peers

    def release(self, gpu, req, n):
        held = self.held.get((gpu, req), [])
        if n > len(held):
            raise ValueError("release: more units than the request holds")
        for _ in range(n):
            self.use[gpu][held.pop()] -= 1
        if not held:
            self.held.pop((gpu, req), None)

    def preempted(self, gpu, peer, t):
        if self.window == 0:
            return
        level = self.use[gpu][peer]
        if 2 * level <= self.units:
            return
        c = self.active_cap(gpu, peer, t)
        new_level = level if c is None or level < c else c
        self.cap[gpu][peer] = (new_level, t + self.window)
