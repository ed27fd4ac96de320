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
  knee% x busy-time accounting, Sec. 6.1).
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


def deployed_slots(knee_s: int, overprov=OVERPROVISION_SLOTS, total=TOTAL_SLOTS) -> int:
    return min(total, knee_s + overprov)


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


def _find_start(placed, ws, we, L, s, latest, total):
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
        if _max_load(placed, t, t + L) + s <= total:
            return t
    return None


def plan(models: List[PlanModel], period: int, total: int = TOTAL_SLOTS) -> List[Job]:
    """Spatio-temporal session plan; returns jobs in placement (EDF) order."""
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
        if m.knee != m.slots:
            options.append(m.knee)
        options += [s for s in sorted(m.row, reverse=True) if s < m.knee]
        for s in options:
            L = latency_at(m.row, s)
            if L is None:
                continue
            t = _find_start(placed, j.release, j.deadline, L, s, j.k % 2 == 1, total)
            if t is not None:
                j.start, j.duration, j.slots = t, L, s
                placed.append(j)
                break
        else:
            j.start, j.duration, j.slots, j.missed = j.release, 0, 0, True
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


def schedule(models, period, total=TOTAL_SLOTS, overprov=OVERPROVISION_SLOTS):
    """Per-model optimisation followed by the session plan.

    models: list of dicts {slo_us, max_batch, rate_per_s, table: {b: {s: L}}}.
    Returns (choices, jobs, utilisation_ppm, feasible_all)."""
    choices = [optimize(m["table"], m["slo_us"], m["max_batch"], m.get("rate_per_s", 0)) for m in models]
    pms = [PlanModel(slo=m["slo_us"], knee=c.slots, slots=deployed_slots(c.slots, overprov, total),
                     row=m["table"][c.batch], batch=c.batch) for m, c in zip(models, choices)]
    jobs = plan(pms, period, total)
    ok = all(c.feasible for c in choices) and not any(j.missed for j in jobs)
    return choices, jobs, utilisation_ppm(jobs, period, total), ok
