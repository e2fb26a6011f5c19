"""Block-grained scheduling and compute-aware admission (reference).

Passages followed: Algorithm 1 (admit while the cost fits, execute one
block-cycle, advance every active request by one block, evict requests that
reached K_i blocks or produced EOS); Eq. 1 (the cost of an active set is its
size times its widest row p_i + (b_i + 1) L); paragraph "Compute-aware
admission control" (the pending queue is sorted by prompt length; the refill
searches for candidates whose initial row width p + L fits inside the current
bounding box -- "sand filling" -- and admits a candidate only if the cost of
the enlarged set stays within the token budget); Experimental setup (the
Fixed variant replaces the budget rule by a batch-size cap); Eq. 2 (effective
compute ratio).

Readings where the paper is silent:
* the queue order is ascending prompt length by default (ties: arrival order);
  descending and arrival order are options (the sorting ablation compares
  sorted with unsorted queues);
* a refill alternates two moves until neither admits anything: scan the
  whole queue for sand-filling candidates (p + L no wider than the current
  box) and admit each one whose admission keeps the cost within budget; then
  admit the head of the queue if its admission keeps the cost within budget
  (it may widen the box, which can make further queued requests sand fills);
  it stops when the head does not fit;
* the Fixed policy admits from the head of the queue while fewer than the cap
  are active;
* an admitted request also needs a free row of the physical box (the lowest
  free row is taken); a request whose p + g exceeds the box's columns, or
  (budget policy) whose p + L alone exceeds the budget, is rejected when it
  is submitted, so no request can block the queue forever;
* a block-cycle ends when every active request's block is fully unmasked.

Test infrastructure: the oracle, not the product path.
"""
from __future__ import annotations

from dataclasses import dataclass, field

BUDGET, FIXED = 0, 1
ASCENDING, DESCENDING, ARRIVAL = 0, 1, 2


@dataclass
class Req:
    id: int
    p: int
    g: int
    L: int
    b: int = 0
    row: int = -1
    seq: int = 0          # arrival order

    @property
    def K(self) -> int:
        return -(-self.g // self.L)

    def width(self) -> int:
        """Eq. 1 row width: prompt plus completed and current blocks."""
        return self.p + (self.b + 1) * self.L


def cost(active, extra=None) -> int:
    """Eq. 1 for `active` (plus one candidate at block 0 when given)."""
    widths = [r.width() for r in active]
    if extra is not None:
        widths.append(extra.p + extra.L)
    return len(widths) * max(widths) if widths else 0


@dataclass
class Scheduler:
    L: int
    policy: int = BUDGET
    budget: int = 0
    fixed_batch: int = 0
    rows: int = 1
    width: int = 1
    order: int = ASCENDING
    pending: list = field(default_factory=list)
    active: list = field(default_factory=list)
    finished: list = field(default_factory=list)
    active_counts: list = field(default_factory=list)
    _seq: int = 0

    def submit(self, reqs):
        """reqs: iterable of (id, p, g)."""
        reqs = [(int(a), int(b), int(c)) for a, b, c in reqs]
        for rid, p, g in reqs:
            if p < 0 or g < 1 or p + g > self.width or (self.policy == BUDGET and p + self.L > self.budget):
                raise ValueError(f"request {rid} cannot be served by this box/budget")
        for rid, p, g in reqs:
            self.pending.append(Req(rid, p, g, self.L, seq=self._seq))
            self._seq += 1
        key = {ASCENDING: lambda r: (r.p, r.seq), DESCENDING: lambda r: (-r.p, r.seq),
               ARRIVAL: lambda r: r.seq}[self.order]
        self.pending.sort(key=key)

    def _free_row(self):
        used = {r.row for r in self.active}
        for row in range(self.rows):
            if row not in used:
                return row
        return -1

    def _take(self, i):
        r = self.pending.pop(i)
        r.row = self._free_row()
        self.active.append(r)
        return r.id

    def admit(self):
        """Refill at a block boundary; returns the admitted ids in admission order."""
        out = []
        if self.policy == FIXED:
            while self.pending and len(self.active) < self.fixed_batch and self._free_row() >= 0:
                out.append(self._take(0))
            return out
        while True:
            # sand filling: candidates that do not widen the box, anywhere in the queue
            box = max((r.width() for r in self.active), default=0)
            i = 0
            while i < len(self.pending) and self._free_row() >= 0:
                c = self.pending[i]
                if c.p + self.L <= box and cost(self.active, c) <= self.budget:
                    out.append(self._take(i))
                else:
                    i += 1
            # then the head of the queue, if the enlarged set fits
            if not self.pending or self._free_row() < 0 or cost(self.active, self.pending[0]) > self.budget:
                return out
            out.append(self._take(0))

    def active_sorted(self):
        """Active requests in row order (the order their descriptors take)."""
        return sorted(self.active, key=lambda r: r.row)

    def complete_cycle(self, eos_ids=()):
        """After a block-cycle: every active request advances one block; those at
        K blocks or reporting EOS leave. Returns the evicted ids."""
        self.active_counts.append(len(self.active))
        eos = set(int(x) for x in eos_ids)
        keep, gone = [], []
        for r in self.active:
            r.b += 1
            if r.b >= r.K or r.id in eos:
                gone.append(r.id)
                self.finished.append(r)
            else:
                keep.append(r)
        self.active = keep
        return gone

    def cost(self) -> int:
        return cost(self.active)

    def done(self) -> bool:
        return not self.pending and not self.active
