"""A deliberately naive brute-force model of the cache policy, used only to
cross-check the C oracle on tiny inputs.

It is written from the rules of the paper (arXiv 2407.15264, Sec. 4.2 levels and
static tie-break, Sec. 4.3.1 victim-buffer enqueue, Sec. 4.3.2 level swap) with
different data structures from the oracle: Python lists of (node, inserted_at)
pairs per set, the victim ring as a plain list searched linearly, the window as
the list of announced Python sets scanned at every update of the dynamic
information (a dict of recorded next uses per resident node), victim queues as
a dict of lists keyed by iteration, and victim selection by sorting all
candidates.  The set-index function is injected.
"""
from __future__ import annotations

NEAR, FAR, RECENT, NONE = "near", "far", "recent", "none"


class NaiveCache:
    def __init__(self, num_nodes, num_sets, ways, victim_rows, lookahead, static, set_of,
                 near_threshold=0, policy="hybrid", victim_mode="fifo", refresh_period=1):
        self.N, self.S, self.W, self.V, self.L = num_nodes, num_sets, ways, victim_rows, lookahead
        self.T = near_threshold or max(1, lookahead // 8)
        self.static = list(static)
        self.set_of = set_of
        self.sets = [[None] * ways for _ in range(num_sets)]  # (node, inserted_at) | None
        self.ring = [None] * victim_rows
        self.tail = 0
        self.announced = []
        self.t = 0
        self.policy = policy
        self.pointer = [0] * num_sets  # round-robin: next way to evict
        self.queues = victim_mode == "queues"
        self.C = victim_rows // (lookahead + 1) if self.queues else 0
        self.q = {}  # queue mode: reuse iteration j -> evicted nodes, in eviction order
        self.U = refresh_period
        self.t_upd = 0
        self.info = {}  # node -> next reuse iteration seen at the last update (resident nodes only)

    def advance(self, ids):
        if len(self.announced) > self.t + self.L:
            return "E_WINDOW"
        if any(not (0 <= x < self.N) for x in ids):
            return "E_RANGE"
        self.announced.append(set(int(x) for x in ids))
        return "OK"

    def _update(self):
        self.t_upd = self.t
        self.info = {}
        for ways in self.sets:
            for e in ways:
                if e is not None:
                    uses = [j for j in range(self.t + 1, self.t + self.L + 1)
                            if j < len(self.announced) and e[0] in self.announced[j]]
                    self.info[e[0]] = min(uses) if uses else None

    def _class(self, entry):
        node, at = entry
        if at >= self.t_upd:
            return RECENT  # no dynamic information yet
        r = self.info.get(node)
        if r is None:
            return NONE
        if r <= self.t:
            return RECENT  # its recorded reuse has come
        return NEAR if r - self.t <= self.T else FAR

    def _level(self, cls):
        order = [FAR, NONE, RECENT, NEAR] if self.V > 0 else [NONE, FAR, RECENT, NEAR]
        return order.index(cls)

    def gather(self, ids):
        if any(not (0 <= x < self.N) for x in ids):
            return "E_RANGE", None
        uniq = sorted(set(int(x) for x in ids))
        if self.t % self.U == 0:
            self._update()
        st = dict(hits=0, victim_hits=0, misses=0, evictions=0, enqueued=0, dropped=0)
        outcome = []
        for x in uniq:
            ways = self.sets[self.set_of(x)]
            if any(e is not None and e[0] == x for e in ways):
                st["hits"] += 1
                outcome.append("H")
                continue
            if self.queues and x in self.q.get(self.t, []):
                st["victim_hits"] += 1
                outcome.append("V")
            elif not self.queues and x in self.ring:
                self.ring[self.ring.index(x)] = None
                st["victim_hits"] += 1
                outcome.append("V")
            else:
                st["misses"] += 1
                outcome.append("M")
            empties = [w for w, e in enumerate(ways) if e is None]
            if empties:
                w = empties[0]
            else:
                w = self._victim(self.set_of(x), ways)
                cls = self._class(ways[w])
                st["evictions"] += 1
                if self.queues and self.C > 0 and cls in (FAR, NEAR):
                    j = self.info[ways[w][0]]
                    if len(self.q.setdefault(j, [])) < self.C:
                        self.q[j].append(ways[w][0])
                        self.tail += 1
                        st["enqueued"] += 1
                    else:
                        st["dropped"] += 1
                elif not self.queues and self.V > 0 and cls in (FAR, NEAR):
                    self.ring[self.tail % self.V] = ways[w][0]
                    self.tail += 1
                    st["enqueued"] += 1
                else:
                    st["dropped"] += 1
            ways[w] = (x, self.t)
        self.q.pop(self.t, None)
        self.t += 1
        return "OK", dict(uniq=uniq, outcome="".join(outcome), **st)

    def _next_use(self, entry):
        """Distance to the recorded reuse, or None without usable information."""
        node, at = entry
        r = self.info.get(node)
        if at >= self.t_upd or r is None or r <= self.t:
            return None
        return r - self.t

    def _victim(self, s, ways):
        if self.policy == "hybrid":
            return sorted((self._level(self._class(e)), self.static[e[0]], w) for w, e in enumerate(ways))[0][2]
        if self.policy == "static":
            return sorted((self.static[e[0]], w) for w, e in enumerate(ways))[0][1]
        if self.policy == "dynamic":
            # no announced use counts as further than any announced one
            far = [(self.L + 1 if self._next_use(e) is None else self._next_use(e)) for e in ways]
            return sorted((-f, w) for w, f in enumerate(far))[0][1]
        w = self.pointer[s]
        self.pointer[s] = (w + 1) % self.W
        return w

    def tags(self):
        return [[-1 if e is None else e[0] for e in s] for s in self.sets]

    def ring_tags(self):
        if not self.queues:
            return [-1 if r is None else r for r in self.ring]
        out = [-1] * self.V
        for j, nodes in self.q.items():
            slot = j % (self.L + 1)
            out[slot * self.C: slot * self.C + len(nodes)] = nodes
        return out
