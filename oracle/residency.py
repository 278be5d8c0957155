"""Oracle: per-layer HBM cache of expert slots and the copies each step needs.

Test infrastructure only.

The paper keeps one buffer per layer that receives the prefetched set K_p, is used,
and is evicted before the next layer (Sec. V-C, per-token budget distribution), and
says the method supports batching (Sec. V-B) without further detail.  The workloads
instead give every layer a persistent cache of C slots and keep the other experts in
host memory.  Reading used here (deterministic, a pure function of the K_p history):

* at start, slot s holds expert s (s < C) and every expert's last-use step is -1;
* each step, P = union of the batch's prefetched sets; an expert's count is the number
  of tokens whose set holds it and its best rank the smallest position it takes in
  them; the target T is P when |P| <= C, else the first C of P ordered by
  (count descending, best rank ascending, id ascending);
* experts of T already resident stay; the others are copied in that same order into
  free slots taken as empty slots (ascending) first, then the slots of resident
  experts outside T ordered by (last use ascending, id ascending);
* every expert of T gets last use = this step.

Under the paper's own memory model (batch 1, cache emptied every layer) the resident
set after the step is exactly K_p.
"""
from __future__ import annotations


class Residency:
    def __init__(self, E: int, C: int):
        self.E, self.C = E, C
        self.expert_of_slot = [s if s < E else -1 for s in range(C)]
        self.last_used = [-1] * E

    def resident(self):
        return set(e for e in self.expert_of_slot if e >= 0)

    def slot_of_expert(self):
        table = [-1] * self.E
        for s, e in enumerate(self.expert_of_slot):
            if e >= 0:
                table[e] = s
        return table

    def target(self, pf_lists):
        count, best = {}, {}
        for lst in pf_lists:
            for pos, e in enumerate(lst):
                e = int(e)
                if e < 0:
                    continue
                count[e] = count.get(e, 0) + 1
                best[e] = min(best.get(e, pos), pos)
        prio = sorted(count, key=lambda e: (-count[e], best[e], e))
        return prio[:self.C]

    def plan(self, pf_lists, step: int):
        """Advance one step; returns the copies [(expert, slot), ...] in issue order."""
        T = self.target(pf_lists)
        R = self.resident()
        new = [e for e in T if e not in R]
        Tset = set(T)
        empty = [s for s, e in enumerate(self.expert_of_slot) if e < 0]
        evict = sorted((e for e in R if e not in Tset), key=lambda e: (self.last_used[e], e))
        slot_of = self.slot_of_expert()
        free = empty + [slot_of[e] for e in evict]
        copies = []
        for e, s in zip(new, free):
            self.expert_of_slot[s] = e
            copies.append((e, s))
        for e in T:
            self.last_used[e] = step
        return copies
