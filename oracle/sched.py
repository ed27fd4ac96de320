"""Scheduler oracle for D-STACK (arxiv 2304.13541), integer arithmetic only.

TEST INFRASTRUCTURE ONLY (see the package docstring).  This is the plain,
slow statement of the decisions the library's scheduler must reproduce
bit-exactly from the same timing table.

Units: times are integer microseconds; GPU share is counted in *slots*.  A
slot is one CU on each XCD (8 CUs of 256), so ``s`` slots = ``s/32`` of the
GPU.  Every decision depends only on the timing table ``L[b][s]`` (median
latency in us of batch ``b`` on ``s`` slots).

Readings taken where the paper is silent (each one is restated in the design
notes):
* efficacy (Sec. 5, Eq. efficiencySquareLatency): eta = b / (L^2 * GPU%),
  compared exactly as b1*L2^2*s2 > b2*L1^2*s1;
* knee (Sec. 4.3, Eq. first_order_derivative read as the magnitude
  1/(E_t^2 S)): argmax over swept slots of eta, ties to fewer slots;
* over-provisioning (Sec. 5, "Estimation of the Knee"): deployed slots =
  knee + 2 slots (6.25%), clamped to the total;
* batch optimisation (Sec. 5.1, Eqs. max_batch_size, meet_slo,
  meet_half_slo): maximise eta s.t. 1 <= b <= Bmax, L + C(b) <= SLO,
  L <= floor(SLO/2); C(b) = ceil(b*1e6/rate) with an arrival rate, else
  482*b us (one 224x224x3 fp32 image per ~481.7 us on 10 Gb/s, Sec. 5.1);
  ties: higher eta, then fewer slots, then larger batch; if nothing is
  feasible: b = 1 with its lowest-latency slot count, flagged infeasible;
* session plan (Sec. 6.1 and 6.1.1): jobs k = 0..ceil(T/SLO)-1 in fixed
  windows [k*SLO, min((k+1)*SLO, T)); EDF order (deadline, SLO, model, k);
  even k start as early as possible, odd k as late as possible ("as far
  apart as possible"); a start is feasible when the summed slots of
  overlapping jobs plus the job's own stay within the total at every
  instant (no over-subscription, Sec. 6); failing that, retry at the
  un-over-provisioned knee, then at each smaller swept slot count
  ("below the knee", Sec. 6.1.1); failing that the job is missed;
* slot ids: placed jobs, in (start, placement order), take the
  lowest-numbered slots free at their start; an interval set whose load
  never exceeds the total can always be coloured this way;
* utilisation = sum over placed jobs of s * L / (total * T) (the paper's
  knee% x busy-time accounting, Sec. 6.1);
* home placement (an alternative to lowest free ids, for a launcher that
  gives every model one fixed set of CUs, as a GPU% fixed per model
  process does in Sec. 6): every model owns one contiguous slot range of
  its deployed size; models in order of decreasing size (then index) take
  the offset in [0, total - size] whose summed overlap with the ranges
  already placed is least, lowest offset on ties; a job runs on its whole
  home range only (no smaller fallback) and may start when no overlapping
  placed job's range meets its own.
"""
from dataclasses import dataclass, field
from typing import Dict, List, Optional

BATCH_GRID = (1, 2, 4, 8, 16, 32)
TOTAL_SLOTS = 32
OVERPROVISION_SLOTS = 2
ASSEMBLY_US_PER_ITEM = 482


def ceil_div(a, b):
    return -(-a // b)


def eta_gt(b1, L1, s1, b2, L2, s2):
    """eta(b1, L1, s1) > eta(b2, L2, s2) for eta = b / (L^2 * s)."""
    return b1 * L2 * L2 * s2 > b2 * L1 * L1 * s1


def latency_at(row: Dict[int, int], s: int) -> Optional[int]:
    """Latency for ``s`` slots: the measurement at the largest swept count <= s."""
    keys = [k for k in row if k <= s]
    return row[max(keys)] if keys else None


def knee(row: Dict[int, int], b: int) -> int:
    """Slot count maximising eta = b/(L^2 s) over a row ``{s: L}``; ties to fewer slots."""
    best = None
    for s in sorted(row):
        L = row[s]
        if best is None or eta_gt(b, L, s, b, row[best], best):
            best = s
    return best


def knee_search(latency, b: int, candidates, start: int):
    """Knee of a model without a profile (Sec. 3.6: start at a nominal 30%,
    binary search on the latency).  Reading: over the ascending GPU% grid
    `candidates` (slot counts) eta(s) = b / (L(s)^2 s) is taken as unimodal;
    keep the index interval [lo, hi] = [0, n - 1], probe candidates mid and
    mid + 1 (mid = the last candidate <= start first, then the midpoint,
    clamped into [lo, hi - 1]); if eta rises from mid to mid + 1 the knee is
    above mid, else at or below it.  On a fine GPU% grid the latency falls
    in steps (whole rounds of workgroups), so eta can have a local maximum
    where the bisection stops; the result is then confirmed against its grid
    neighbours k-2, k-1, k+1, k+2 (in that order): while one of them has a
    higher eta (or an equal eta with fewer slots) the search moves to the
    best of them and confirms again.  latency(s) is called once per slot
    count.  Returns (knee slots, probes)."""
    c = list(candidates)
    seen = {}
    probes = []

    def L(i):
        if i not in seen:
            seen[i] = latency(c[i])
            probes.append((c[i], seen[i]))
        return seen[i]

    lo, hi = 0, len(c) - 1
    mid = max([i for i in range(len(c)) if c[i] <= start], default=0)
    while lo < hi:
        mid = min(max(mid, lo), hi - 1)
        a, d = L(mid), L(mid + 1)
        if eta_gt(b, d, c[mid + 1], b, a, c[mid]):
            lo = mid + 1
        else:
            hi = mid
        mid = (lo + hi) // 2
    k = lo

    def better(j, i):  # higher eta, or equal eta on fewer slots
        return eta_gt(b, L(j), c[j], b, L(i), c[i]) or (not eta_gt(b, L(i), c[i], b, L(j), c[j]) and c[j] < c[i])

    while True:
        best = k
        for j in (k - 2, k - 1, k + 1, k + 2):
            if 0 <= j < len(c) and better(j, best):
                best = j
        if best == k:
            return c[k], probes
        k = best


def deployed_slots(knee_s: int, overprov=OVERPROVISION_SLOTS, total=TOTAL_SLOTS) -> int:
    return min(total, knee_s + overprov)


def home_offsets(sizes: List[int], total: int = TOTAL_SLOTS) -> List[int]:
    """Offset of each model's fixed slot range (home placement)."""
    offs = [0] * len(sizes)
    placed = []
    for i in sorted(range(len(sizes)), key=lambda i: (-sizes[i], i)):
        best = None
        for o in range(total - sizes[i] + 1):
            overlap = sum(max(0, min(o + sizes[i], po + ps) - max(o, po)) for po, ps in placed)
            if best is None or overlap < best[0]:
                best = (overlap, o)
        offs[i] = best[1]
        placed.append((offs[i], sizes[i]))
    return offs


def range_mask(offset: int, size: int) -> int:
    return ((1 << size) - 1) << offset


def assembly_us(b: int, rate: int) -> int:
    if rate and rate > 0:
        return ceil_div(b * 1000000, rate)
    return ASSEMBLY_US_PER_ITEM * b


@dataclass
class Choice:
    batch: int
    slots: int
    latency: int
    feasible: bool


def optimize(table: Dict[int, Dict[int, int]], slo: int, bmax: int, rate: int = 0) -> Choice:
    """SLO-constrained efficacy maximisation over the measured (b, s) grid."""
    best = None
    for b in BATCH_GRID:
        if b > bmax or b not in table:
            continue
        C = assembly_us(b, rate)
        for s in sorted(table[b]):
            L = table[b][s]
            if L + C > slo or L > slo // 2:
                continue
            if best is None:
                best = (b, s, L)
                continue
            bb, bs, bL = best
            if eta_gt(b, L, s, bb, bL, bs):
                best = (b, s, L)
            elif eta_gt(bb, bL, bs, b, L, s):
                pass
            elif s < bs or (s == bs and b > bb):
                best = (b, s, L)
    if best is not None:
        return Choice(best[0], best[1], best[2], True)
    b = min(table) if 1 not in table else 1
    row = table[b]
    s = min(sorted(row), key=lambda k: (row[k], k))
    return Choice(b, s, row[s], False)


@dataclass
class PlanModel:
    slo: int               # us
    knee: int              # slots at the efficacy optimum (no over-provision)
    slots: int             # deployed slots
    row: Dict[int, int]    # {swept slots: latency us} at the chosen batch
    batch: int = 1


@dataclass
class Job:
    model: int
    k: int
    release: int
    deadline: int
    start: int = 0
    duration: int = 0
    slots: int = 0
    missed: bool = False
    slot_mask: int = 0
    order: int = 0

    @property
    def end(self) -> int:
        return self.start + self.duration


def _max_load(placed: List[Job], t0: int, t1: int) -> int:
    """Largest summed slots of placed jobs at any instant of [t0, t1)."""
    points = [t0] + [p.start for p in placed if t0 < p.start < t1]
    best = 0
    for tau in points:
        load = sum(p.slots for p in placed if p.start <= tau < p.end)
        best = max(best, load)
    return best


def _conflicts(placed: List[Job], t0: int, t1: int, mask: int) -> bool:
    """Does a placed job overlapping [t0, t1) in time use a slot of mask?"""
    return any(p.start < t1 and t0 < p.end and (p.slot_mask & mask) for p in placed)


def _find_start(placed, ws, we, L, s, latest, total, home_mask=None):
    if L > we - ws:
        return None
    cands = {ws, we - L}
    for p in placed:
        cands.add(p.end)
        cands.add(p.start - L)
    cands = sorted(c for c in cands if ws <= c <= we - L)
    if latest:
        cands.reverse()
    for t in cands:
        if home_mask is None:
            if _max_load(placed, t, t + L) + s <= total:
                return t
        elif not _conflicts(placed, t, t + L, home_mask):
            return t
    return None


def plan(models: List[PlanModel], period: int, total: int = TOTAL_SLOTS, homes: Optional[List[int]] = None) -> List[Job]:
    """Spatio-temporal session plan; returns jobs in placement (EDF) order.
    homes: per-model range offsets for home placement (None: lowest free ids)."""
    jobs = []
    for i, m in enumerate(models):
        r = ceil_div(period, m.slo)
        for k in range(r):
            ws = k * m.slo
            we = min((k + 1) * m.slo, period)
            jobs.append(Job(model=i, k=k, release=ws, deadline=we))
    jobs.sort(key=lambda j: (j.deadline, models[j.model].slo, j.model, j.k))
    placed = []
    for order, j in enumerate(jobs):
        j.order = order
        m = models[j.model]
        options = [m.slots]
        if homes is None:
            if m.knee != m.slots:
                options.append(m.knee)
            options += [s for s in sorted(m.row, reverse=True) if s < m.knee]
        hm = None if homes is None else range_mask(homes[j.model], m.slots)
        for s in options:
            L = latency_at(m.row, s)
            if L is None:
                continue
            t = _find_start(placed, j.release, j.deadline, L, s, j.k % 2 == 1, total, hm)
            if t is not None:
                j.start, j.duration, j.slots = t, L, s
                if hm is not None:
                    j.slot_mask = hm
                placed.append(j)
                break
        else:
            j.start, j.duration, j.slots, j.missed = j.release, 0, 0, True
    if homes is not None:
        return jobs
    # slot ids: lowest free ids at each start, in (start, placement order)
    busy = []  # (end, mask)
    for j in sorted(placed, key=lambda p: (p.start, p.order)):
        used = 0
        for end, mask in busy:
            if end > j.start:
                used |= mask
        mask, need = 0, j.slots
        for sid in range(total):
            if need == 0:
                break
            if not (used >> sid) & 1:
                mask |= 1 << sid
                need -= 1
        assert need == 0, "load invariant violated"
        j.slot_mask = mask
        busy.append((j.end, mask))
    return jobs


def utilisation_ppm(jobs: List[Job], period: int, total: int = TOTAL_SLOTS) -> int:
    """Sum of s*L over placed jobs / (total*T), in parts per million (floor)."""
    num = sum(j.slots * j.duration for j in jobs if not j.missed)
    return num * 1000000 // (total * period)


def temporal_utilisation(slos_and_shares):
    """Temporal sharing (Sec. 6.1): slices proportional to SLO, each model
    using its knee share while it holds the whole GPU; returns the
    slice-weighted mean share."""
    num = sum(slo * share for slo, share in slos_and_shares)
    den = sum(slo for slo, _ in slos_and_shares)
    return num / den


def schedule(models, period, total=TOTAL_SLOTS, overprov=OVERPROVISION_SLOTS, placement="lowest"):
    """Per-model optimisation followed by the session plan.

    models: list of dicts {slo_us, max_batch, rate_per_s, table: {b: {s: L}}};
    placement: "lowest" (lowest free slot ids) or "home" (fixed ranges).
    Returns (choices, jobs, utilisation_ppm, feasible_all)."""
    choices = [optimize(m["table"], m["slo_us"], m["max_batch"], m.get("rate_per_s", 0)) for m in models]
    pms = [PlanModel(slo=m["slo_us"], knee=c.slots, slots=deployed_slots(c.slots, overprov, total),
                     row=m["table"][c.batch], batch=c.batch) for m, c in zip(models, choices)]
    homes = home_offsets([pm.slots for pm in pms], total) if placement == "home" else None
    jobs = plan(pms, period, total, homes)
    ok = all(c.feasible for c in choices) and not any(j.missed for j in jobs)
    return choices, jobs, utilisation_ppm(jobs, period, total), ok


# ---------------------------------------------------------------------------
# Launcher simulation: the session plan repeated every period, plus the fair,
# opportunistic, dynamic (FOD) fill of Sec. 6.1.2, on a virtual integer-us
# clock driven by the timing table (a TimingTable-driven stand-in for the GPU).
#
# Readings (restated in the design notes):
# * planned job (model i, start p*T + st): takes up to b_i of the oldest
#   queued requests; with none queued it does not run; it runs for the
#   planned duration;
# * FOD is triggered by every request arrival and every job completion; the
#   candidates are models with no running job and >= 1 queued request,
#   ordered by (runs in the current and previous 9 sessions, cumulative busy
#   us, model index) -- "fewest runs" (Sec. 6.1.2) then "least time" (Sec. 6.3);
#   the first candidate that fits is launched (at most one per trigger):
#   it takes the lowest-numbered s_i slots free now (s_i = its deployed
#   slots) -- with home placement, its own range, which must be all free;
#   its gap ends at the first planned start at or after now whose
#   slots meet them, or at its own model's next planned start (a planned job
#   at this very instant may not have been processed yet); its batch is the largest
#   b in {1,2,4,8,16,32} with b <= max_batch, b <= queued and L(b, s_i) <= gap;
# * events at one instant: completions, then planned starts, then arrivals
#   (each group by model, then by issue order); FOD runs after each
#   completion and each arrival;
# * a served request violates its SLO if completion - arrival > SLO; no job
#   starts at or after the end of the trace, and requests still queued when
#   the last started job ends are unserved (also violations); utilisation
#   counts slot-time inside [0, duration);
# * runs/busy time are charged at job start; the session of time t is t // T;
# * a planned start that finds an empty queue or its model running is skipped
#   (counted per model).
# ---------------------------------------------------------------------------

FNV_OFFSET = 0xcbf29ce484222325
FNV_PRIME = 0x100000001b3


def _fnv(h, v):
    v &= (1 << 64) - 1
    for i in range(8):
        h ^= (v >> (8 * i)) & 0xff
        h = (h * FNV_PRIME) & ((1 << 64) - 1)
    return h


def _nearest_rank(sorted_vals, pct):
    if not sorted_vals:
        return 0
    k = max(1, -(-pct * len(sorted_vals) // 100))
    return sorted_vals[k - 1]


def simulate(models, period, duration, arrivals, total=TOTAL_SLOTS, overprov=OVERPROVISION_SLOTS, fod=True,
             sessions_window=10, placement="lowest", policy="dstack", slice_cycle=0, replay_events=None,
             resize_violations=0):
    """models: as for schedule(); arrivals: per model sorted list of integer us in [0, duration).
    Returns dict with per-model counters, utilisation_ppm and a hash of the job log.

    policy "dstack": the session plan plus the FOD fill (Sec. 6.1.2).  The
    comparators of Sec. 6.3 run the same fill with no plan and another order
    of the candidates (a reading: each is a non-preemptive greedy fill at the
    model's deployed share and largest queued grid batch):
    "maxthroughput" -- least runtime first (the model's SLO-optimal latency
    at its deployed slots, then index), the schedule that favours the sum of
    throughputs; "maxmin" -- smallest demand first (deployed slots, then
    busy time, then index), max-min fairness over GPU% demands.

    "temporal": the time-sliced full-GPU baseline of Sec. 6.1 and Sec. 7
    (temporal sharing, "T"): one model at a time holds the whole GPU during
    its time slice, slices proportional to the models' SLOs.  Reading: the
    slices repeat every C = slice_cycle us (0: the smallest SLO, so that every
    model gets a turn within every one of its SLO intervals); model i's slice is [off_i, off_i +
    len_i) of each cycle with len_i = floor(C * SLO_i / sum of SLOs) and the
    offsets in model order (the remainder of the cycle idles).  At every slice
    start, completion and arrival, if no job runs and the instant lies in a
    slice whose model has queued requests, that model starts a job on all
    the slots with the largest grid batch (<= max_batch, <= queued) whose
    table latency at all the slots ends by its slice's end (the adaptive
    batch of the slice); none fits: it waits.  No plan, no FOD.

    resize_violations > 0 (D-STACK with home placement): a GPU% change on
    SLO violations (Sec. 3.5's dynamic reconfiguration, the trigger count a
    parameter).  A request that arrived at or after its model's last change
    (earlier ones waited through the previous size) counts once: when its
    job starts, if it has waited more than half its SLO by then (the share
    Eq. meet_half_slo leaves to waiting), else when its job completes past
    its SLO.  At the completion that brings the count to the trigger the
    model moves to the next larger column of its table (over all batches)
    that has a latency at its plan batch, keeping its home offset if the
    range fits, else ending at the last slot -- it stays, and the count
    restarts, when there is none or when the larger range would meet another
    model's range that the current one does not meet; from then on its
    planned and FOD jobs use that range and the table latency there.  A
    planned start runs only if its slots are free.

    replay_events: instead of the virtual clock, the triggers a live launcher
    handled, in its order, as dicts (kind, t_us, model, value_us, slot_mask):
    kind 0 a completion seen (the model's job ends), 1 a planned start due
    (value_us its planned time, slot_mask its slots; temporal: a slice
    start), 2 an arrival admitted (value_us its trace time), 3 a GPU% change
    took effect (the live launcher builds the model's new stream meanwhile:
    from the completion that triggers the change until this event the model
    starts no job, and its late-request count restarts here); each decision
    is taken at t_us with the same rules (a planned start also needs its
    slots free, since a measured job may overrun its table time).  The jobs
    started are then in "log" as (start, table end, model, mask, kind,
    batch)."""
    import collections
    import heapq
    choices, jobs, _, _ = schedule(models, period, total, overprov, placement)
    n = len(models)
    dep = [deployed_slots(c.slots, overprov, total) for c in choices]
    homes = home_offsets(dep, total) if placement == "home" else None
    planned = [j for j in jobs if not j.missed] if policy == "dstack" else []
    if policy != "dstack":
        fod = True
    assert resize_violations == 0 or (policy == "dstack" and homes is not None)
    cur_dep = list(dep)
    cur_home = list(homes) if homes is not None else [0] * n
    viol = [0] * n
    resizes = [0] * n
    changed_at = [0] * n  # time of each model's last GPU% change
    job_start = [0] * n   # start of each model's current (or last) job
    unavailable = set()   # replay of a live run: models whose new stream is not ready yet
    columns = [sorted(set().union(*[set(r) for r in m["table"].values()])) for m in models]
    if policy == "temporal":
        cycle = slice_cycle if slice_cycle > 0 else min(m["slo_us"] for m in models)
        slo_sum = sum(m["slo_us"] for m in models)
        slice_len = [cycle * m["slo_us"] // slo_sum for m in models]
        slice_off = [sum(slice_len[:i]) for i in range(n)]
    # next planned start of each model after time t (over all periods)
    n_periods = ceil_div(duration, period)

    def lat(i, b, s):
        row = models[i]["table"].get(b)
        return latency_at(row, s) if row else None

    # events: (time, kind, model, seq, payload); kind 0 completion, 1 planned start, 2 arrival
    ev = []
    seq = 0
    for p in range(n_periods):
        for j in planned:
            t = p * period + j.start
            if t < duration:
                heapq.heappush(ev, (t, 1, j.model, seq, (j.slot_mask, j.duration)))
                seq += 1
    if policy == "temporal":  # slice starts take the place of planned starts
        for k in range(ceil_div(duration, cycle)):
            for i in range(n):
                t = k * cycle + slice_off[i]
                if slice_len[i] > 0 and t < duration:
                    heapq.heappush(ev, (t, 1, i, seq, None))
                    seq += 1
    for i in range(n):
        for a in arrivals[i]:
            heapq.heappush(ev, (a, 2, i, seq, None))
            seq += 1
    planned_starts = sorted((p * period + j.start, j.model, j.slot_mask) for p in range(n_periods)
                            for j in planned if p * period + j.start < duration)

    queue = [collections.deque() for _ in range(n)]
    running = {}  # model -> (end, mask)
    used = 0
    runs = [collections.Counter() for _ in range(n)]
    busy = [0] * n
    served = [0] * n
    late = [0] * n
    lats = [[] for _ in range(n)]
    planned_runs = [0] * n
    fod_runs = [0] * n
    plan_skips = [0] * n
    slot_us = 0
    h = FNV_OFFSET
    last_end = 0
    log = []

    def start_job(t, i, mask, dur, b, kind):
        nonlocal used, seq, slot_us, h, last_end
        reqs = [queue[i].popleft() for _ in range(b)]
        job_start[i] = t
        if policy == "dstack" and resize_violations > 0:
            # requests (since the last change) that have waited more than half
            # their SLO when their job starts count towards the next change now
            viol[i] += sum(1 for a in reqs if a >= changed_at[i] and 2 * (t - a) > models[i]["slo_us"])
        running[i] = (t + dur, mask, reqs)
        used |= mask
        heapq.heappush(ev, (t + dur, 0, i, seq, reqs))
        seq += 1
        runs[i][t // period] += 1
        busy[i] += dur
        slot_us += bin(mask).count("1") * (min(t + dur, duration) - t)
        last_end = max(last_end, t + dur)
        for v in (t, i, b, mask, dur, kind):
            h = _fnv(h, v)
        log.append((t, t + dur, i, mask, kind, b))
        if kind == 0:
            planned_runs[i] += 1
        else:
            fod_runs[i] += 1

    def current(i, mask, dur):
        """A planned job of model i as it runs now (its size may have changed)."""
        if not resizes[i]:
            return mask, dur
        return range_mask(cur_home[i], cur_dep[i]), lat(i, choices[i].batch, cur_dep[i])

    def note_late(i, t, reqs):
        """GPU% change on SLO violations (Sec. 3.5): the job of model i that
        ended at t adds its requests (since the last change) that completed
        past their SLO and were not counted at its start; the change is
        decided once the count reaches the threshold."""
        if policy != "dstack" or resize_violations <= 0:
            return
        slo = models[i]["slo_us"]
        viol[i] += sum(1 for a in reqs if t - a > slo and a >= changed_at[i] and 2 * (job_start[i] - a) <= slo)
        if viol[i] < resize_violations:
            return
        viol[i] = 0
        nxt = [c for c in columns[i] if cur_dep[i] < c <= total and lat(i, choices[i].batch, c)]
        if not nxt:
            return
        home = total - nxt[0] if cur_home[i] + nxt[0] > total else cur_home[i]
        now, grown = range_mask(cur_home[i], cur_dep[i]), range_mask(home, nxt[0])
        # no change that would make the model contend with one whose range its current range does not meet
        if any(grown & range_mask(cur_home[j], cur_dep[j]) and not now & range_mask(cur_home[j], cur_dep[j])
               for j in range(n) if j != i):
            return
        cur_dep[i] = nxt[0]
        cur_home[i] = home
        resizes[i] += 1
        changed_at[i] = t
        if replay_events is not None:  # live: the model waits for its new stream (an event of kind 3)
            unavailable.add(i)

    def temporal_pass(t):
        if t >= duration or running:
            return
        r = t % cycle
        owner = [i for i in range(n) if slice_off[i] <= r < slice_off[i] + slice_len[i]]
        if not owner or not queue[owner[0]]:
            return
        i = owner[0]
        left = slice_off[i] + slice_len[i] - r
        best = None
        for b in BATCH_GRID:
            if b > models[i]["max_batch"] or b > len(queue[i]):
                continue
            L = lat(i, b, total)
            if L is not None and L <= left:
                best = (b, L)
        if best is not None:
            start_job(t, i, range_mask(0, total), best[1], best[0], 0)

    def fod_pass(t):
        if policy == "temporal":
            temporal_pass(t)
            return
        if t >= duration:  # nothing starts once the trace has ended
            return
        cands = [i for i in range(n) if i not in running and queue[i] and i not in unavailable]
        cur = t // period
        if policy == "maxthroughput":
            cands.sort(key=lambda i: (choices[i].latency, i))
        elif policy == "maxmin":
            cands.sort(key=lambda i: (dep[i], busy[i], i))
        else:
            cands.sort(key=lambda i: (sum(runs[i][s] for s in range(cur - sessions_window + 1, cur + 1)), busy[i], i))
        for i in cands:
            s = cur_dep[i]
            if homes is not None:  # its own range, all of it free
                mask = range_mask(cur_home[i], s)
                if used & mask:
                    continue
            else:  # the lowest-numbered free slots
                free = [sid for sid in range(total) if not (used >> sid) & 1]
                if len(free) < s:
                    continue
                mask = 0
                for sid in free[:s]:
                    mask |= 1 << sid
            gap = None
            for (ps, pm, pmask) in planned_starts:
                pmask = current(pm, pmask, 0)[0]
                if ps >= t and ((pmask & mask) or pm == i):
                    gap = ps - t
                    break
            best = None
            for b in BATCH_GRID:
                if b > models[i]["max_batch"] or b > len(queue[i]):
                    continue
                L = lat(i, b, s)
                if L is None or (gap is not None and L > gap):
                    continue
                best = (b, L)
            if best is None:
                continue
            start_job(t, i, mask, best[1], best[0], 1)
            return

    if replay_events is not None:
        plan_dur = {(p * period + j.start, j.model): (j.slot_mask, j.duration) for p in range(n_periods)
                    for j in planned}
        for e in replay_events:
            t, i = e["t_us"], e["model"]
            if e["kind"] == 0:
                _, mask, reqs = running.pop(i)
                used &= ~mask
                note_late(i, t, reqs)
                if fod:
                    fod_pass(t)
            elif e["kind"] == 1 and policy == "temporal":
                temporal_pass(t)
            elif e["kind"] == 1:
                key = (e["value_us"], i)
                mask, dur = current(i, *plan_dur[key])
                if queue[i] and i not in running and i not in unavailable and not used & mask:
                    start_job(t, i, mask, dur, min(choices[i].batch, len(queue[i])), 0)
                else:
                    plan_skips[i] += 1
            elif e["kind"] == 3:  # a GPU% change took effect: the model runs again, its count restarts now
                unavailable.discard(i)
                changed_at[i] = t
                if fod:
                    fod_pass(t)
            else:
                queue[i].append(e["value_us"])
                if fod:
                    fod_pass(t)
        return dict(log=log, plan_skips=plan_skips, job_hash=h, resizes=resizes, final_slots=cur_dep)

    events = []  # the triggers in the order handled, in the form replay_events takes
    while ev:
        t, kind, i, _, payload = heapq.heappop(ev)
        events.append(dict(kind=kind, t_us=t, model=i, value_us=0 if kind == 0 else t,
                           slot_mask=payload[0] if kind == 1 and payload else
                           (range_mask(0, total) if kind == 1 else 0)))
        if kind == 0:
            end, mask, _ = running.pop(i)
            used &= ~mask
            job_late = 0
            for a in payload:
                served[i] += 1
                lats[i].append(t - a)
                if t - a > models[i]["slo_us"]:
                    job_late += 1
            late[i] += job_late
            note_late(i, t, payload)
            if fod:
                fod_pass(t)
        elif kind == 1 and policy == "temporal":
            temporal_pass(t)
        elif kind == 1:
            mask, dur = current(i, *payload)
            if queue[i] and i not in running and not used & mask:
                start_job(t, i, mask, dur, min(choices[i].batch, len(queue[i])), 0)
            else:
                plan_skips[i] += 1
        else:
            queue[i].append(t)
            if fod:
                fod_pass(t)
    out = []
    for i in range(n):
        L = sorted(lats[i])
        out.append(dict(served=served[i], violations=late[i] + len(queue[i]), unserved=len(queue[i]),
                        planned_runs=planned_runs[i], fod_runs=fod_runs[i], busy_us=busy[i],
                        p50_us=_nearest_rank(L, 50), p99_us=_nearest_rank(L, 99), plan_skips=plan_skips[i],
                        resizes=resizes[i], final_slots=total if policy == "temporal" else cur_dep[i]))
    return dict(models=out, utilisation_ppm=slot_us * 1000000 // (total * max(duration, 1)), job_hash=h,
                last_end_us=last_end, log=log, events=events)


def simulate_ideal(models, horizon, slot, total=TOTAL_SLOTS):
    """The ideal spatio-temporal schedule of Sec. 6.2 (Eqs. maximization and
    constraints), time-slotted at kernel granularity with preemption.

    models: dicts with "slots" and "dur" (per kernel of one forward: its knee
    share and its duration there, integer us), "batch" and "slo_us".  Closed
    loop: a model's next forward is released when the previous one ends.
    In every slot [t, t + slot) the eligible kernels are each model's current
    kernel (its predecessors done: kernels of a model run in order); among
    all subsets whose shares sum to at most `total`, the one with the largest
    sum runs (exhaustive search), ties going to the subset that includes the
    earliest-deadline models (the inclusion bits in (deadline, index) order,
    read as a number, largest first).  A running kernel's remaining time
    drops by the slot length; when it reaches 0 the model moves to its next
    kernel in the next slot (the rest of the slot stays unused by it); after
    the last kernel the forward completes at the slot's end (late if that
    is past release + SLO).  Utilisation = sum over slots of the used shares
    / (total x number of slots)."""
    n = len(models)
    k = [0] * n
    rem = [models[i]["dur"][0] for i in range(n)]
    release = [0] * n
    deadline = [models[i]["slo_us"] for i in range(n)]
    items = [0] * n
    forwards = [0] * n
    late = [0] * n
    busy = [0] * n
    used_sum = 0
    n_slots = 0
    h = FNV_OFFSET
    t = 0
    while t < horizon:
        order = sorted(range(n), key=lambda i: (deadline[i], i))
        best_key, best = None, 0
        for sub in range(1 << n):
            s = sum(models[i]["slots"][k[i]] for i in range(n) if (sub >> i) & 1)
            if s > total:
                continue
            bits = 0
            for i in order:
                bits = (bits << 1) | ((sub >> i) & 1)
            key = (s, bits)
            if best_key is None or key > best_key:
                best_key, best = key, sub
        used_sum += best_key[0]
        n_slots += 1
        h = _fnv(h, t)
        h = _fnv(h, best)
        end = t + slot
        for i in range(n):
            if not (best >> i) & 1:
                continue
            busy[i] += models[i]["slots"][k[i]] * slot
            rem[i] -= slot
            if rem[i] <= 0:
                k[i] += 1
                if k[i] == len(models[i]["dur"]):
                    forwards[i] += 1
                    items[i] += models[i]["batch"]
                    if end > deadline[i]:
                        late[i] += 1
                    k[i] = 0
                    release[i] = end
                    deadline[i] = end + models[i]["slo_us"]
                rem[i] = models[i]["dur"][k[i]]
        t = end
    return dict(items=items, forwards=forwards, late=late, busy_slot_us=busy,
                utilisation_ppm=used_sum * 1000000 // (total * max(n_slots, 1)), hash=h)

