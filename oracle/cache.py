"""Logical per-layer expert cache of the prefetcher (Sec. "Coordination of
Prefetching and Inference": Alg. 1 prefetch worker, Alg. 2 PushPredictedExperts
/ PushPreciseExperts, "Reordered Inference"; Sec. "Cache Implementation":
a standard per-layer LRU in which both prefetch and inference count as
accesses, and prefetching touches experts that are already cached).

Deterministic reading.  The paper replaces a slot when the worker copies an
expert's first chunk and counts a hit only once a chunk has arrived; both
depend on copy timing.  Here the *logical* state (slot assignment, LRU order,
counters) changes in program order when a plan is made; the physical copies
follow.  Any slot-assigned expert counts as resident.

State of one layer: slot_expert[C] (-1 free), slot_of[E], stamp[C] from a
per-layer clock, fetch_seq[C] (order in which slots were (re)filled),
spec_unused[C] (filled by a prediction and not yet used).
Warm start: experts 0..C-1 in slots 0..C-1, stamp = slot index, fetch_seq 0.

spec_plan(Q)      -- PushPredictedExperts: first every resident member of Q is
                     touched, in Q order; then, in Q order, each non-resident
                     member takes the lowest free slot or the least recently
                     stamped one, evicts, assigns, is marked speculative and
                     queues its three chunks at low priority.  Touches first:
                     Alg. 2 counts the hits while it pushes the list, and the
                     worker of Alg. 1 replaces a slot only when it starts a
                     copy, after the whole list has been pushed; so a fill never
                     evicts a member of its own list (|Q| <= C).
                     A fill never evicts an expert the same prediction names
                     (``voted``: every expert with a vote, of which Q is the
                     first C; default Q): when every candidate victim is
                     predicted, the rest of the list is skipped.  The paper
                     pushes one token's list, where this never binds; for a
                     batch whose votes cover the cache, trading one predicted
                     expert for another only adds copies (a design reading).
                     With a budget b >= 0 at most b experts per plan are filled
                     (later non-resident members are skipped): the paper's
                     worker replaces a slot only when a copy starts, and when
                     copies are the bottleneck only the first few predicted
                     experts of a layer start before the layer's route drops
                     the rest.
precise_plan(P)   -- PushPreciseExperts: P = the distinct experts the layer's
                     tokens chose, ascending.  Low-priority work of the layer is
                     dropped (physical only).  Order = resident experts by
                     (fetch_seq, id) ascending -- earliest filled first, which on
                     one FIFO copy queue is the most-complete-first order of the
                     paper's sort by ready chunks -- followed by the missing
                     experts in id order.  Resident ones are touched (hits);
                     missing ones get a victim slot exactly as above (misses) and
                     are queued at high priority.  A victim that is itself an
                     earlier member of this order must finish computing before
                     its slot is overwritten: its position is recorded as
                     ``after``.
precise_plan(P, reorder=False)
                  -- the order frameworks use without reordered inference:
                     ascending expert id, each expert classified at its turn.
                     An earlier miss may evict a later member of P, which then
                     misses in its turn (the cache thrashing of "Reordered
                     Inference"); a victim that is a later member needs no wait.

Prediction accuracy (Sec. "A New Prediction Metric: GoodPred": the share of
predicted experts that are correct).  A predictor-driven spec plan of a layer
records its list Q (pred_n += |Q|); the layer's next precise plan counts
pred_correct += |Q & P| and forgets Q.  With one token, Q is the token's k
predicted experts, so pred_correct / pred_n is exactly the per-token accuracy;
with several tokens it is the accuracy of the merged list.  Lists pushed by the
caller are not predictions and are not counted.

Static cache (the paper's static baseline, Sec. "Evaluation"): the first
``pinned`` slots keep their warm experts for good; victims are chosen among the
remaining slots only (with C - pinned = 2 staging buffers, as the paper's static
baseline uses).  pinned = 0 is the LRU cache above.
"""
from dataclasses import dataclass

COUNTERS = ("prec_access", "hit", "miss", "spec_issued", "spec_resident", "spec_used", "spec_wasted", "evict",
            "pred_n", "pred_correct")


@dataclass
class SpecEntry:
    expert: int
    slot: int            # -1 when skipped
    new: bool
    victim: int          # expert evicted (-1 none)
    skipped: bool = False  # non-resident, over the fill budget


@dataclass
class PreciseEntry:
    expert: int
    slot: int            # slot this position computes from
    miss: bool
    victim: int          # expert evicted for a miss (-1 none)
    after: int           # position in the order whose compute must precede the fill (-1 none)


class LayerCache:
    def __init__(self, n_experts: int, slots: int, warm: bool = True, pinned: int = 0):
        assert 0 <= pinned < slots
        self.E, self.C, self.pinned = n_experts, slots, pinned
        self.slot_expert = [-1] * slots
        self.slot_of = [-1] * n_experts
        self.stamp = [0] * slots
        self.fetch_seq = [0] * slots
        self.spec_unused = [False] * slots
        self.clock = slots - 1
        self.fseq = 0
        self.pred_set = set()
        self.count = {c: 0 for c in COUNTERS}
        if warm:
            for s in range(min(slots, n_experts)):
                self.slot_expert[s] = s
                self.slot_of[s] = s
                self.stamp[s] = s

    # -- helpers
    def _victim(self, spare=()) -> int:
        """Lowest free slot, else the least recently stamped one whose expert is
        not in `spare`; -1 when there is none."""
        cand = range(self.pinned, self.C)
        for s in cand:
            if self.slot_expert[s] < 0:
                return s
        cand = [s for s in cand if self.slot_expert[s] not in spare]
        return min(cand, key=lambda s: self.stamp[s]) if cand else -1

    def _evict(self, s: int) -> int:
        v = self.slot_expert[s]
        if v >= 0:
            self.count["evict"] += 1
            if self.spec_unused[s]:
                self.count["spec_wasted"] += 1
            self.slot_of[v] = -1
            self.slot_expert[s] = -1
        return v

    def _touch(self, s: int) -> None:
        self.clock += 1
        self.stamp[s] = self.clock

    def _fill(self, e: int, s: int, speculative: bool) -> None:
        self.slot_expert[s] = e
        self.slot_of[e] = s
        self.fseq += 1
        self.fetch_seq[s] = self.fseq
        self.spec_unused[s] = speculative
        self._touch(s)

    # -- plans
    def spec_plan(self, Q, budget: int = -1, predicted: bool = True, voted=None):
        Q = [int(e) for e in Q]
        if predicted:
            self.pred_set = set(Q)
            self.count["pred_n"] += len(self.pred_set)
        spare = set(Q) | set(int(e) for e in (voted if voted is not None else ()))
        out = [None] * len(Q)
        for i, e in enumerate(Q):          # the list's hits
            s = self.slot_of[e]
            if s >= 0:
                self._touch(s)
                self.count["spec_resident"] += 1
                out[i] = SpecEntry(e, s, False, -1)
        fills = 0
        for i, e in enumerate(Q):          # then its fills
            if out[i] is not None:
                continue
            s = -1 if 0 <= budget <= fills else self._victim(spare)
            if s < 0:
                out[i] = SpecEntry(e, -1, False, -1, True)
                continue
            fills += 1
            v = self._evict(s)
            self._fill(e, s, True)
            self.count["spec_issued"] += 1
            out[i] = SpecEntry(e, s, True, v)
        return out

    def _hit(self, e: int) -> PreciseEntry:
        s = self.slot_of[e]
        self._touch(s)
        self.count["hit"] += 1
        if self.spec_unused[s]:
            self.count["spec_used"] += 1
            self.spec_unused[s] = False
        return PreciseEntry(e, s, False, -1, -1)

    def _miss(self, e: int, pos: int, pos_of) -> PreciseEntry:
        s = self._victim()
        v = self._evict(s)
        self._fill(e, s, False)
        self.count["miss"] += 1
        after = pos_of[v] if v >= 0 and pos_of.get(v, pos) < pos else -1
        return PreciseEntry(e, s, True, v, after)

    def precise_plan(self, P, reorder: bool = True):
        P = sorted(set(int(e) for e in P))
        self.count["pred_correct"] += len(self.pred_set & set(P))
        self.pred_set = set()
        if not reorder:
            pos_of = {e: i for i, e in enumerate(P)}
            entries = [self._hit(e) if self.slot_of[e] >= 0 else self._miss(e, i, pos_of) for i, e in enumerate(P)]
            self.count["prec_access"] += len(P)
            return P, entries
        hits = [e for e in P if self.slot_of[e] >= 0]
        missing = [e for e in P if self.slot_of[e] < 0]
        hits.sort(key=lambda e: (self.fetch_seq[self.slot_of[e]], e))
        order = hits + missing
        pos_of = {e: i for i, e in enumerate(order)}
        entries = [self._hit(e) for e in hits]
        entries += [self._miss(e, len(hits) + i, pos_of) for i, e in enumerate(missing)]
        self.count["prec_access"] += len(P)
        return order, entries

    def resident(self):
        return {e for e in self.slot_expert if e >= 0}


class Cache:
    """One LayerCache per layer (layers are independent)."""

    def __init__(self, n_layers: int, n_experts: int, slots: int, warm: bool = True, pinned: int = 0):
        self.layers = [LayerCache(n_experts, slots, warm, pinned) for _ in range(n_layers)]

    def totals(self):
        t = {c: 0 for c in COUNTERS}
        for lc in self.layers:
            for c in COUNTERS:
                t[c] += lc.count[c]
        return t
