"""Oracle: prefix-aware refinement of the in-context demonstrations (test infrastructure).

What is computed (InferLog, section 3.2.1 "Prefix-Aware ICL Refinement" and
section 3.2.2 "ICL Table Management", with the figure of matching, modifying
and reordering):

* a demonstration set DS is an ordered list of N demonstrations, each a
  labelled (log, template) pair; here a demonstration is the pair
  (template id, demonstration id), the demonstration id standing for the
  concrete log text (and so for its tokens);
* the ICL table keeps the demonstration sets of past requests, oldest first;
* prefix-matching count PMC(H, C) of a past set H against the current set C:
  the number of leading demonstrations of H whose templates all occur in C.
  A demonstration of C serves at most one of H's (so two leading H entries
  of one template need two such entries in C);
* matching: the past set with the largest PMC is the target;
* modifying: each of the target's first PMC demonstrations replaces the
  current demonstration of the same template (the first one in current order
  not yet replaced), so both carry identical tokens;
* reordering: the final set is the target's first PMC demonstrations in the
  target's order, then the remaining current demonstrations in their order;
* table update after the request:
  (1) PMC = N: the current set becomes the target set; the target moves to
      the tail (most recently used);
  (2) PMC = 0: the current set is kept unchanged and appended at the tail;
  (3) 0 < PMC < N: the modified and reordered set is appended at the tail;
      the target keeps its place;
  when the table holds more sets than its capacity, the head (least recently
  used) is evicted.

Readings taken where the paper is silent:

* ties between past sets of equal PMC go to the one nearest the tail (the most
  recently used, whose KV is the most likely still held);
* with no past set at all the PMC is 0 (rule 2);
* the table holds each demonstration sequence once: appending a sequence that
  is already present moves that entry to the tail instead.

Plain Python lists and an OrderedDict, no shortcuts.
"""
from __future__ import annotations

from collections import OrderedDict


def pmc(hist, cur) -> int:
    """Prefix-matching count of past set `hist` against current set `cur`.

    Both are sequences of (template, demo) pairs.
    """
    avail = {}
    for t, _ in cur:
        avail[t] = avail.get(t, 0) + 1
    k = 0
    for t, _ in hist:
        if avail.get(t, 0) == 0:
            break
        avail[t] -= 1
        k += 1
    return k


def refine(target, cur, k):
    """Modify and reorder `cur` against the first `k` entries of `target`."""
    used = [False] * len(cur)
    head = []
    for t, d in target[:k]:
        for i, (ct, _) in enumerate(cur):
            if not used[i] and ct == t:
                used[i] = True
                break
        else:  # cannot happen when k <= pmc(target, cur)
            raise ValueError("target prefix does not match the current set")
        head.append((t, d))
    tail = [cur[i] for i in range(len(cur)) if not used[i]]
    return head + tail


class PairTableRef:
    """The ICL table with its three update rules and LRU eviction."""

    def __init__(self, capacity: int, n_demos: int):
        if capacity < 1 or n_demos < 1:
            raise ValueError("capacity and n_demos must be positive")
        self.capacity, self.n = capacity, n_demos
        self.table: OrderedDict[tuple, None] = OrderedDict()

    def entries(self):
        """Demonstration sets, head (least recently used) first."""
        return [list(k) for k in self.table]

    def _append(self, ds):
        key = tuple(ds)
        if key in self.table:
            self.table.move_to_end(key)
        else:
            self.table[key] = None
            while len(self.table) > self.capacity:
                self.table.popitem(last=False)

    def process(self, cur):
        """Refine one request's demonstration set; returns (final set, PMC).

        `cur` is a list of N (template, demo) pairs.  The table is updated as
        after the request completed.
        """
        cur = [tuple(x) for x in cur]
        if len(cur) != self.n:
            raise ValueError("demonstration set of the wrong size")
        best, best_k = None, 0
        for hist in self.table:  # head to tail: a later equal PMC wins
            k = pmc(hist, cur)
            if k > 0 and k >= best_k:
                best, best_k = hist, k
        if best_k == self.n:  # rule (1)
            final = list(best)
            self.table.move_to_end(best)
        elif best_k == 0:  # rule (2)
            final = list(cur)
            self._append(final)
        else:  # rule (3)
            final = refine(list(best), cur, best_k)
            self._append(final)
        return final, best_k
