"""Brute-force checkers used only to pin the oracle itself."""
import numpy as np


def loop_matvec(W, x):
    """y[i] = sum_j W[i][j] x[j] with Python loops."""
    return [sum(float(W[i][j]) * float(x[j]) for j in range(len(x))) for i in range(len(W))]


def loop_swiglu(x, wg, wu, wd):
    """Textbook SwiGLU MLP with Python loops and math.exp."""
    import math
    a = loop_matvec(wg, x)
    b = loop_matvec(wu, x)
    act = [ai / (1.0 + math.exp(-ai)) * bi for ai, bi in zip(a, b)]
    return loop_matvec(wd, act)


def sort_topk(z_row, k):
    """Top-k by a full Python sort with an explicit (value desc, id asc) key."""
    return [e for _, e in sorted(((-float(v), e) for e, v in enumerate(z_row)))][:k]


def dense_moe(x, ids, w, expert_fn, n_experts, act_bf16, swiglu):
    """Evaluate every expert on every token and mask by the routing weights."""
    T, k = ids.shape
    y = np.zeros((T, x.shape[1]))
    for e in range(n_experts):
        mask = np.zeros(T)
        for t in range(T):
            for r in range(k):
                if ids[t, r] == e:
                    mask[t] += w[t, r]
        y += mask[:, None] * swiglu(x, *expert_fn(e), act_bf16)
    return y


class NaiveLRU:
    """The same cache rules restated over an access log: residency is a dict, the
    LRU victim is found by re-scanning the whole log for each resident expert's
    latest access, and fill order by scanning for its latest fill."""

    def __init__(self, n_experts, slots, warm=True, pinned=0):
        self.E, self.C, self.pinned = n_experts, slots, pinned
        self.where = {}          # expert -> slot
        self.log = []            # (kind, expert), kind in {"touch", "fill"}
        if warm:
            for s in range(min(slots, n_experts)):
                self.where[s] = s
                self.log.append(("touch", s))
        self.warm_set = set(self.where)
        self.spec_pending = set()
        self.c = {k: 0 for k in ("prec_access", "hit", "miss", "spec_issued", "spec_resident",
                                 "spec_used", "spec_wasted", "evict", "pred_n", "pred_correct")}
        self.predicted = []      # the last prediction not yet followed by a route

    def _last(self, e, kinds):
        for i in range(len(self.log) - 1, -1, -1):
            if self.log[i][1] == e and self.log[i][0] in kinds:
                return i
        return -1

    def _free_or_lru(self, keep=frozenset()):
        # slots below `pinned` are never given away, nor experts in `keep`
        used = set(self.where.values())
        free = [s for s in range(self.pinned, self.C) if s not in used]
        if free:
            return free[0], None
        movable = [e for e in self.where if self.where[e] >= self.pinned and e not in keep]
        if not movable:
            return -1, None
        v = min(movable, key=lambda e: self._last(e, ("touch", "fill")))
        return self.where[v], v

    def _bring(self, e, speculative, keep=frozenset()):
        s, v = self._free_or_lru(keep)
        if s < 0:
            return -1, None
        if v is not None:
            self.c["evict"] += 1
            if v in self.spec_pending:
                self.c["spec_wasted"] += 1
                self.spec_pending.discard(v)
            del self.where[v]
        self.where[e] = s
        self.log.append(("fill", e))
        if speculative:
            self.spec_pending.add(e)
        else:
            self.spec_pending.discard(e)
        return s, v

    def spec(self, Q, budget=-1, predicted=True, voted=None):
        """Touch the list's resident members, then bring the others in list
        order, never evicting a list member or an expert in `voted`."""
        if predicted:
            self.predicted = list(Q)
            self.c["pred_n"] += len(Q)
        keep = frozenset(Q) | frozenset(voted or ())
        resident_before = {e: self.where[e] for e in Q if e in self.where}
        for e in Q:
            if e in resident_before:
                self.log.append(("touch", e))
                self.c["spec_resident"] += 1
        out = []
        brought = 0
        for e in Q:
            if e in resident_before:
                out.append((e, resident_before[e], False))
                continue
            s = -1
            if not (budget >= 0 and brought >= budget):
                s, _ = self._bring(e, True, keep)
            if s < 0:
                out.append((e, -1, False))
                continue
            brought += 1
            self.c["spec_issued"] += 1
            out.append((e, s, True))
        return out

    def _fill_time(self, e):
        i = self._last(e, ("fill",))
        return i if i >= 0 else -1   # warm experts were never filled: earliest

    def _use(self, e):
        self.log.append(("touch", e))
        self.c["hit"] += 1
        if e in self.spec_pending:
            self.c["spec_used"] += 1
            self.spec_pending.discard(e)
        return self.where[e]

    def precise(self, P, reorder=True):
        P = sorted(set(P))
        self.c["pred_correct"] += sum(1 for e in self.predicted if e in P)
        self.predicted = []
        if not reorder:
            # one access at a time, in id order
            slots = []
            for e in P:
                if e in self.where:
                    slots.append(self._use(e))
                else:
                    s, _ = self._bring(e, False)
                    self.c["miss"] += 1
                    slots.append(s)
            self.c["prec_access"] += len(P)
            return P, slots
        hits = [e for e in P if e in self.where]
        miss = [e for e in P if e not in self.where]
        hits.sort(key=lambda e: (self._fill_time(e), e))
        order = hits + miss
        slots = [self._use(e) for e in hits]
        for e in miss:
            s, _ = self._bring(e, False)
            self.c["miss"] += 1
            slots.append(s)
        self.c["prec_access"] += len(P)
        return order, slots
