"""Oracle of the TempoKV claim / commitment controller and a discrete-event
model of the runtime and staging device it serves -- TEST INFRASTRUCTURE ONLY
(imported by tests and the benchmark's CPU baseline, never by the library).

Plain Python, one event at a time, written from the paper's Section 3 (claims,
two-sided timing, commitment, replanning, protected capacity, shared staging,
lifecycle) and Section 5 (policies, the cost metric C).  The runtime and the
device are a model of this library's own (the paper's are vLLM and an SSD-
backed CXL device); every modelling choice is stated below.

Model
-----
Objects o (staged chunks) of bytes[o].  Fast tier of `capacity` bytes with a
protected budget `budget` <= capacity.  An object is resident or not, may have
a staging read outstanding (completion time ready_at[o]), and a protection
count prot[o] (committed, unreleased claims that need it).  Reserved capacity
P(t) = sum of bytes[o] over objects with prot[o] > 0: objects held under
protection, whether resident or still being staged, each shared object
counted once (Section 5, "Metrics").

Staging device: one FIFO server at `stage_rate` bytes/s (concurrent reads
share an aggregate rate, Section 3.1); busy_until is when its queue drains.

Runtime: requests arrive at arrival[i] with an ordered manifest of objects,
uncached tokens and output tokens; FCFS with at most `max_active` active
requests.  A request admitted to a slot requests retrieval of its claim
(Section 3.2).  Retrieval = transfer of the manifest's bytes at `gpu_rate`,
then prefill (uncached tokens x prefill_s), first token, then decode (output
tokens x decode_s); the slot frees at the end.

Claims (one per request, Section 3): reported PLANNED at arrival; eligible when
the policy says so or retrieval is requested; committed through the
commitment rule (eligible; total bytes <= budget and newly reserved bytes <=
budget - P) else BLOCKED (stays PLANNED) or, if retrieval was requested,
ORDINARY.  Commitment protects every manifest object (prot += 1) and queues a
staging read for each one neither resident nor already queued (coalescing);
the claim is STAGEREADY once all its objects are resident, TRANSFERRING when
its transfer starts, RELEASED when the transfer ends (prot -= 1; an object
left with prot == 0 stays resident, evictable, Section 3.2 "Shared staging and
resource lifecycle").  A commitment is never revoked.  An ORDINARY request
reads its non-resident objects through the same server without protection,
then transfers.

Residency: an object becoming resident evicts least-recently-released
unprotected resident objects (ties by id) until it fits; an unprotected object
that cannot fit is not retained.

Policies (Section 5 "Policies"): DEMAND (eligible only when retrieval is
requested), IMMEDIATE (when reported), QUEUE_K (when at most K-1 waiting
requests are ahead of it), TEMPO_STATIC (TTU <= TTR with TTR = non-resident bytes /
static_rate, in isolation), TEMPO (TTU <= TTR with TTR from a projection of
the staging queue: already-queued objects keep their completion times, new
reads are appended in manifest order; the last object decides, Section 3.1).
TTU (Section 3.1): projection of the FCFS slots assuming the target and the
requests ahead of it are stage-ready: each active request frees its slot at
its projected end, each waiting request ahead takes the earliest free slot for
its service time; TTU = target's start - now.

Control points: after every event (arrival, staging completion, fetch end,
transfer end, request end) and every `tick` seconds (Section 5: event-driven
plus a 50 ms tick).  Each control point first admits requests to free slots,
then evaluates PLANNED claims: requested ones first in admission order, then
waiting ones in FCFS order (Section 3.2 "Commitment and replanning"), then
starts transfers and ordinary reads.  Events with equal times run in the order
they were scheduled.

Cost: C = (integral of P dt from t=0 until the last request ends) / N, in
GiB*s per request (Section 5).
"""
from __future__ import annotations

import heapq
import math
from dataclasses import dataclass
from typing import Dict, List, Sequence

import oracle

DEMAND, IMMEDIATE, QUEUE_K, TEMPO_STATIC, TEMPO = range(5)
POLICY_NAMES = ["demand", "immediate", "queue_k", "tempo_static", "tempo"]
PLANNED, STAGING, STAGEREADY, TRANSFERRING, RELEASED, ORDINARY = range(6)
# event kinds
EV_ARRIVAL, EV_OBJ_READY, EV_FETCH_END, EV_TRANSFER_END, EV_REQ_END, EV_TICK = range(6)
# active-request phases
PH_WAIT, PH_FETCH, PH_RUN = range(3)
GIB = float(1 << 30)


@dataclass
class SimConfig:
    budget: float
    capacity: float
    stage_rate: float
    static_rate: float
    gpu_rate: float
    prefill_s: float
    decode_s: float
    max_active: int = 4
    tick: float = 0.05
    policy: int = TEMPO
    queue_k: int = 4


def ttr_static_of(objs, obj_bytes, resident, static_rate):
    """Static TTR (Section 5, TempoKV-Static): the claim's non-resident bytes
    over a fixed staging rate, as if it were staged alone."""
    return sum(obj_bytes[o] for o in objs if not resident[o]) / static_rate


def ttr_state_aware_of(objs, obj_bytes, resident, queued, ready_at, now, busy_until, stage_rate):
    """State-aware TTR (Section 3.1, "Storage-estimated time-to-ready"): the
    staging queue projected from `now`.  Objects already queued keep their
    completion times; the claim's other non-resident objects are appended, in
    claim order, behind the queue's tail at the aggregate staging rate; the
    last object to become resident decides."""
    t_end = now
    tail = max(busy_until, now)
    for o in objs:
        if resident[o]:
            continue
        if queued[o]:
            t_end = max(t_end, ready_at[o])
        else:
            tail = tail + obj_bytes[o] / stage_rate
            t_end = max(t_end, tail)
    return t_end - now


def simulate(cfg: SimConfig, obj_bytes: Sequence[float], arrival: Sequence[float],
             manifests: Sequence[Sequence[int]], uncached: Sequence[int], out_tokens: Sequence[int]) -> Dict:
    N, O = len(arrival), len(obj_bytes)
    resident = [False] * O
    queued = [False] * O
    ready_at = [0.0] * O
    prot = [0] * O
    lru = [0.0] * O
    busy_until = 0.0
    state = [PLANNED] * N
    requested = [False] * N
    ever_blocked = [False] * N
    # unique objects of each manifest, in manifest order
    uniq = []
    for m in manifests:
        seen, u = set(), []
        for o in m:
            if o not in seen:
                seen.add(o)
                u.append(o)
        uniq.append(u)
    total = [sum(obj_bytes[o] for o in u) for u in uniq]
    svc = [total[i] / cfg.gpu_rate + uncached[i] * cfg.prefill_s + out_tokens[i] * cfg.decode_s for i in range(N)]
    waiting: List[int] = []
    active: List[int] = []          # admission order
    phase = [PH_WAIT] * N
    fetch_end = [0.0] * N
    req_end = [0.0] * N
    first_token = [math.nan] * N
    done = [math.nan] * N
    arrived = [False] * N
    P = 0.0
    P_max = 0.0
    area = 0.0
    now = 0.0
    heap: list = []
    seq = [0]
    trace: list = []

    def push(t, kind, a):
        heapq.heappush(heap, (t, seq[0], kind, a))
        seq[0] += 1

    def make_resident(o, protected):
        if resident[o]:
            lru[o] = now
            return
        used = sum(obj_bytes[x] for x in range(O) if resident[x])
        if used + obj_bytes[o] > cfg.capacity:
            victims = sorted([x for x in range(O) if resident[x] and prot[x] == 0 and x != o],
                             key=lambda x: (lru[x], x))
            for x in victims:
                if used + obj_bytes[o] <= cfg.capacity:
                    break
                resident[x] = False
                used -= obj_bytes[x]
                trace.append((now, "evict", x))
        if used + obj_bytes[o] <= cfg.capacity or protected:
            resident[o] = True
            lru[o] = now

    def ttr_static(i):
        return ttr_static_of(uniq[i], obj_bytes, resident, cfg.static_rate)

    def ttr_state(i):
        return ttr_state_aware_of(uniq[i], obj_bytes, resident, queued, ready_at, now, busy_until, cfg.stage_rate)

    def projected_end(i):
        if phase[i] == PH_RUN:
            return req_end[i]
        if phase[i] == PH_FETCH:
            return fetch_end[i] + svc[i]
        if state[i] == STAGING:
            r = now
            for o in uniq[i]:
                if not resident[o] and queued[o]:
                    r = max(r, ready_at[o])
            return r + svc[i]
        return now + svc[i]

    def ttus():
        slots = [projected_end(a) for a in active] + [now] * (cfg.max_active - len(active))
        heapq.heapify(slots)
        out = {}
        for w in waiting:
            s0 = max(slots[0], now)
            out[w] = s0 - now
            heapq.heapreplace(slots, s0 + svc[w])
        return out

    def commit(i):
        nonlocal P, P_max, busy_until
        for o in uniq[i]:
            if prot[o] == 0:
                P += obj_bytes[o]
                P_max = max(P_max, P)
            prot[o] += 1
            if not resident[o] and not queued[o]:
                start = max(now, busy_until)
                ready_at[o] = start + obj_bytes[o] / cfg.stage_rate
                busy_until = ready_at[o]
                queued[o] = True
                push(ready_at[o], EV_OBJ_READY, o)
        state[i] = STAGEREADY if all(resident[o] for o in uniq[i]) else STAGING
        trace.append((now, "commit", i))

    def decide(i, pos, ttu_map):
        new = sum(obj_bytes[o] for o in uniq[i] if prot[o] == 0)
        req = requested[i]
        pol = cfg.policy
        if pol == DEMAND:
            ttu, ttr = math.inf, 0.0
        elif pol == IMMEDIATE:
            ttu, ttr = -math.inf, 0.0
        elif pol == QUEUE_K:
            ttu, ttr = (-math.inf if (pos is not None and pos < cfg.queue_k) else math.inf), 0.0
        elif pol == TEMPO_STATIC:
            ttu, ttr = (ttu_map[i] if i in ttu_map else math.inf), ttr_static(i)
        else:
            ttu, ttr = (ttu_map[i] if i in ttu_map else math.inf), ttr_state(i)
        return oracle.commit_should_stage(ttu, ttr, int(cfg.budget - P), int(new), int(total[i]), int(cfg.budget), req)

    def control():
        nonlocal busy_until
        while waiting and len(active) < cfg.max_active:
            i = waiting.pop(0)
            active.append(i)
            requested[i] = True
            phase[i] = PH_WAIT
            trace.append((now, "admit", i))
        order = [i for i in active if state[i] == PLANNED] + [i for i in waiting if state[i] == PLANNED]
        ttu_map = ttus() if cfg.policy in (TEMPO, TEMPO_STATIC) else {}
        pos = {w: k for k, w in enumerate(waiting)}
        for i in order:
            d = decide(i, pos.get(i), ttu_map)
            if d == oracle.COMMIT:
                commit(i)
                if cfg.policy in (TEMPO, TEMPO_STATIC):
                    ttu_map = ttus()
            elif d == oracle.ORDINARY:
                state[i] = ORDINARY
                trace.append((now, "ordinary", i))
            elif d == oracle.BLOCKED:
                ever_blocked[i] = True
        for i in list(active):
            if phase[i] != PH_WAIT:
                continue
            if state[i] == STAGEREADY:
                state[i] = TRANSFERRING
                phase[i] = PH_RUN
                t_x = now + total[i] / cfg.gpu_rate
                first_token[i] = t_x + uncached[i] * cfg.prefill_s
                req_end[i] = first_token[i] + out_tokens[i] * cfg.decode_s
                push(t_x, EV_TRANSFER_END, i)
                push(req_end[i], EV_REQ_END, i)
                trace.append((now, "transfer", i))
            elif state[i] == ORDINARY:
                phase[i] = PH_FETCH
                nonres = sum(obj_bytes[o] for o in uniq[i] if not resident[o])
                fetch_end[i] = max(now, busy_until) + nonres / cfg.stage_rate
                busy_until = fetch_end[i]
                push(fetch_end[i], EV_FETCH_END, i)
                trace.append((now, "fetch", i))

    for i in range(N):
        push(float(arrival[i]), EV_ARRIVAL, i)
    push(0.0, EV_TICK, 0)
    n_done = 0
    while heap and n_done < N:
        t, _, kind, a = heapq.heappop(heap)
        area += P * (t - now)
        now = t
        if kind == EV_ARRIVAL:
            arrived[a] = True
            waiting.append(a)
            trace.append((now, "arrive", a))
        elif kind == EV_OBJ_READY:
            queued[a] = False
            make_resident(a, True)
            trace.append((now, "ready", a))
            for i in range(N):
                if state[i] == STAGING and all(resident[o] for o in uniq[i]):
                    state[i] = STAGEREADY
                    trace.append((now, "stageready", i))
        elif kind == EV_FETCH_END:
            for o in uniq[a]:
                if not resident[o]:
                    make_resident(o, False)
            phase[a] = PH_RUN
            t_x = now + total[a] / cfg.gpu_rate
            first_token[a] = t_x + uncached[a] * cfg.prefill_s
            req_end[a] = first_token[a] + out_tokens[a] * cfg.decode_s
            push(t_x, EV_TRANSFER_END, a)
            push(req_end[a], EV_REQ_END, a)
        elif kind == EV_TRANSFER_END:
            if state[a] == TRANSFERRING:
                state[a] = RELEASED
                for o in uniq[a]:
                    prot[o] -= 1
                    if prot[o] == 0:
                        P -= obj_bytes[o]
                        lru[o] = now
                trace.append((now, "release", a))
        elif kind == EV_REQ_END:
            done[a] = now
            active.remove(a)
            n_done += 1
            trace.append((now, "done", a))
        elif kind == EV_TICK:
            push((a + 1) * cfg.tick, EV_TICK, a + 1)
        control()
    ttft = [first_token[i] - arrival[i] for i in range(N)]
    return dict(ttft=ttft, first_token=first_token, done=done, area=area, C=area / GIB / N, end=now, P_max=P_max,
                final_state=list(state),
                trace=trace, blocked=sum(ever_blocked), ordinary=sum(1 for s in state if s == ORDINARY),
                committed=sum(1 for x in trace if x[1] == "commit"))
