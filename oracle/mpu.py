"""Reference of the Maximum Pipeline Utilization (MPU) wave planner, in plain Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, with the passages it follows (Design of WavePP, "Pipeline Scheduling"):

* The executor keeps a ring of R = 2P waves for P stages; the planner targets S = R + (F - 1) P
  waves, F - 1 being the number of extra waiting pipeline fills.
* Candidate budgets come from repeated halving of the maximum wave budget M, aligned down to the
  block size B and floored at b_min (Eq. 6).
* W counts the not-yet-scheduled suffix tokens of the admitted requests plus, for each of them,
  its most recently committed chunk while that chunk's wave is still in the ring.  For a
  candidate budget b, N_{>b/2} counts the pieces (remaining suffixes and those in-flight chunks)
  larger than b/2, and the available waves are n(b) = max(W / b, N_{>b/2}) (Eq. 7).
* The planner takes the largest budget with n(b) >= S, else b_min.  Once a budget already
  supplies R waves, halving it further is refused when the pieces it would newly split (larger
  than the smaller budget but not larger than this one) exceed 12.5 % of W.
* A larger budget is adopted at once when it is at least two halvings up (a burst); one halving
  up must be asked for R/2 decisions in a row; a smaller budget must be asked for R decisions in
  a row and pass the hysteresis check.  The first decision has no budget to hold on to and takes
  its target directly.
* Waves are packed first-come-first-served, at most one chunk per request and at most
  max_lanes requests per wave.  A fragment of a request that does not fit whole is not placed in
  a leftover space smaller than max(b_min, b/2).
* While the ring is busy, a wave holding a single request below half the budget waits one
  planning iteration if another request is in admission.
* The scheduler may accept less than proposed: positions advance only by the accepted spans.

Readings where the text leaves details open (each also listed in the design notes):
* Packing stops at the first request it cannot place (strict FCFS, no overtaking).
* The hysteresis check for a decrease: the current budget must fall at least one wave short of
  the target, n(b_current) <= S - 1.
* Budgets are compared as ladder positions; a "one-step" increase is one halving.
* n(b) >= X is evaluated exactly in integers: W >= X * b or N_{>b/2} >= X.
* Nothing is planned while the ring already holds R waves.

All arithmetic is on integers, so the C++ planner must agree decision for decision.
"""
from __future__ import annotations

from dataclasses import dataclass, field


def budget_ladder(max_budget: int, min_budget: int, block: int) -> list[int]:
    """Eq. 6: b_0 = M, b_{j+1} = max(b_min, alignDown_B(b_j / 2)), stopping at b_min."""
    if not (block > 0 and max_budget % block == 0 and min_budget % block == 0
            and block <= min_budget <= max_budget):
        raise ValueError("need B | M, B | b_min and B <= b_min <= M")
    ladder = [max_budget]
    while ladder[-1] > min_budget:
        halved = (ladder[-1] // 2) // block * block
        ladder.append(max(min_budget, halved))
    return ladder


def waves_at_least(W: int, pieces: list[int], b: int, x: int) -> bool:
    """n(b) >= x with n(b) = max(W / b, N_{>b/2}) (Eq. 7), exactly: W >= x b or N_{>b/2} >= x."""
    n_big = sum(1 for p in pieces if 2 * p > b)
    return W >= x * b or n_big >= x


def waves_at_most(W: int, pieces: list[int], b: int, x: int) -> bool:
    """n(b) <= x, exactly: W <= x b and N_{>b/2} <= x."""
    n_big = sum(1 for p in pieces if 2 * p > b)
    return W <= x * b and n_big <= x


def choose_budget(ladder: list[int], W: int, pieces: list[int], S: int, R: int, split_permille: int) -> int:
    """The largest budget with n(b) >= S, with thinning stopped when it would mainly split pieces
    that fit the current budget; b_min when none qualifies."""
    for j, b in enumerate(ladder):
        if waves_at_least(W, pieces, b, S):
            return b
        if j + 1 < len(ladder) and waves_at_least(W, pieces, b, R):
            nxt = ladder[j + 1]
            newly_split = sum(p for p in pieces if nxt < p <= b)
            if newly_split * 1000 > split_permille * W:
                return b
    return ladder[-1]


@dataclass
class Request:
    rid: int
    pos: int          # next token to schedule
    end: int          # one past the last token of the prompt
    last_chunk: tuple | None = None    # (wave serial, length) of the most recent committed chunk


@dataclass
class Planner:
    max_budget: int
    min_budget: int
    block: int
    stages: int
    fills: int
    max_lanes: int
    split_permille: int = 125
    count_inflight: bool = True
    ladder: list = field(default_factory=list)
    queue: list = field(default_factory=list)    # admitted requests, admission order
    ring: list = field(default_factory=list)     # serials of in-flight waves, oldest first
    budget: int = 0
    up_count: int = 0
    down_count: int = 0
    waited: bool = False
    next_serial: int = 1

    def __post_init__(self):
        self.ladder = budget_ladder(self.max_budget, self.min_budget, self.block)
        self.budget = 0                  # no decision yet

    @property
    def R(self) -> int:
        return 2 * self.stages

    @property
    def S(self) -> int:
        return self.R + (self.fills - 1) * self.stages

    # -- admission and bookkeeping ------------------------------------------------------------
    def admit(self, rid: int, start: int, end: int):
        if any(r.rid == rid for r in self.queue):
            raise ValueError("request already admitted")
        if not 0 <= start < end:
            raise ValueError("need 0 <= start < end")
        self.queue.append(Request(rid, start, end))

    def _inflight(self, r: Request) -> int:
        if self.count_inflight and r.last_chunk is not None and r.last_chunk[0] in self.ring:
            return r.last_chunk[1]
        return 0

    def work(self):
        """(W, pieces): remaining suffixes and in-flight latest chunks of the admitted requests."""
        W, pieces = 0, []
        for r in self.queue:
            rem = r.end - r.pos
            inf = self._inflight(r)
            W += rem + inf
            if rem > 0:
                pieces.append(rem)
            if inf > 0:
                pieces.append(inf)
        return W, pieces

    # -- one planning decision ----------------------------------------------------------------
    def _update_budget(self, target: int, W: int, pieces: list[int]):
        if self.budget == 0:
            self.budget = target
            return
        cur_i, tgt_i = self.ladder.index(self.budget), self.ladder.index(target)
        if tgt_i == cur_i:
            self.up_count = self.down_count = 0
        elif tgt_i < cur_i:                                # larger budget wanted
            self.down_count = 0
            if cur_i - tgt_i >= 2:
                self.budget, self.up_count = target, 0
            else:
                self.up_count += 1
                if self.up_count >= self.R // 2:
                    self.budget, self.up_count = target, 0
        else:                                              # smaller budget wanted
            self.up_count = 0
            self.down_count += 1
            short = waves_at_most(W, pieces, self.budget, self.S - 1)     # a full wave short
            if self.down_count >= self.R and short:
                self.budget, self.down_count = target, 0

    def plan(self, admission_pending: bool = False):
        """Propose the next wave: a list of (request id, start, length) and the budget used.
        An empty list means nothing to schedule now (ring full, no work, or a lone small wave
        waiting one iteration)."""
        if len(self.ring) >= self.R:
            return [], self.budget
        W, pieces = self.work()
        if W == 0:
            return [], self.budget
        target = choose_budget(self.ladder, W, pieces, self.S, self.R, self.split_permille)
        self._update_budget(target, W, pieces)
        b = self.budget
        spans, space = [], b
        floor = max(self.min_budget, b // 2)
        for r in self.queue:
            rem = r.end - r.pos
            if rem == 0:
                continue
            if len(spans) == self.max_lanes or space == 0:
                break
            take = min(rem, space)
            if take < rem and take < floor:
                break
            spans.append((r.rid, r.pos, take))
            space -= take
        if (len(spans) == 1 and 2 * spans[0][2] < b and self.ring and admission_pending and not self.waited):
            self.waited = True
            return [], b
        return spans, b

    def commit(self, accepted):
        """Record the spans the scheduler accepted as one wave entering the ring."""
        if len(self.ring) >= self.R:
            raise ValueError("ring full")
        serial = self.next_serial
        by_id = {r.rid: r for r in self.queue}
        seen = set()
        for rid, start, length in accepted:
            r = by_id.get(rid)
            if r is None or rid in seen:
                raise ValueError("unknown or repeated request")
            if start != r.pos:
                raise ValueError("span does not start at the request's position")
            if not 0 < length <= r.end - r.pos:
                raise ValueError("bad span length")
            seen.add(rid)
        for rid, start, length in accepted:
            r = by_id[rid]
            r.pos += length
            r.last_chunk = (serial, length)
        self.next_serial += 1
        self.ring.append(serial)
        self.waited = False
        return serial

    def retire(self):
        """The oldest in-flight wave left the last stage."""
        if not self.ring:
            raise ValueError("ring empty")
        self.ring.pop(0)
        self.queue = [r for r in self.queue if r.pos < r.end or self._inflight(r) > 0]
