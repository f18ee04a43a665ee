"""Brute-force event-driven serving simulator -- TEST INFRASTRUCTURE ONLY.

An independent formulation of the serving model for tiny traces (a dozen
requests).  Where the C oracle uses the max-plus recurrence on per-stage free
times, this one simulates the devices: every pipeline stage of a group is a
single server with a FIFO queue, a global clock advances through a heap of
stage-completion and stage-arrival events (the paper's simulator is described
as a continuous-time discrete-event simulator with a global clock, Sec. 5), and
the controller's decisions are made from the simulated timelines:

  - dispatch (Sec. 4.3): for each group hosting the model, replay its admitted
    requests and read the time at which stage 0 finishes the most recently
    admitted one (0.0 for a group that admitted nothing); pick the smallest,
    lowest group index on ties;
  - admission (Sec. 4.3, Sec. 3.2): replay the chosen group's admitted
    requests plus the new one; admit iff the new request leaves the last stage
    no later than arrival + slo_scale * d_single (a finish at the deadline is
    on time).  Under FCFS a later request never delays an earlier one, so the
    replayed finish time is final.

Service of a request at a stage starts when both the request has left the
previous stage and the server has released the previous request, so every
start time is one of those two event times and every completion is that start
plus the stage latency: the same fp64 operations as the recurrence, reached by
a different route.  Cost grows like O(n^2 * S) events; meant for n <= ~20.
"""
from __future__ import annotations

import heapq

import numpy as np


def _replay(requests, lat_rows):
    """Event-driven run of one group's tandem queue.

    requests: list of arrival times in FCFS (admission) order.
    lat_rows: list of per-request stage-latency lists (same length S each).
    Returns per-request list of stage departure times.
    """
    n = len(requests)
    if n == 0:
        return []
    S = len(lat_rows[0])
    depart = [[None] * S for _ in range(n)]
    busy = [False] * S
    queues = [[] for _ in range(S)]  # FIFO of request ids waiting at each stage
    heap = []
    seq = 0
    # event kinds: 0 = completion (processed first at equal time), 1 = arrival at a stage
    for r, a in enumerate(requests):
        heapq.heappush(heap, (a, 1, seq, r, 0))
        seq += 1
    while heap:
        now, kind, _, r, s = heapq.heappop(heap)
        if kind == 1:  # request r arrives at stage s
            queues[s].append(r)
        else:  # request r completes stage s
            busy[s] = False
            depart[r][s] = now
            if s + 1 < S:
                heapq.heappush(heap, (now, 1, seq, r, s + 1))
                seq += 1
        # start service wherever a server is idle and its FIFO head is waiting
        for st in range(S):
            if not busy[st] and queues[st]:
                # FCFS: the head must be the lowest waiting id (arrival order)
                queues[st].sort()
                nxt = queues[st].pop(0)
                busy[st] = True
                heapq.heappush(heap, (now + lat_rows[nxt][st], 0, seq, nxt, st))
                seq += 1
    return depart


def simulate(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask, slo_scale,
             return_groups=False):
    """Simulate one job.  Returns (served, finish[n]) with finish = departure time
    of accepted requests, -1.0 for rejected and -2.0 for unhosted models; with
    return_groups, also group[n]: the group the controller chose for each
    request (-1 when no group hosts the model)."""
    t = [float(x) for x in t]
    model = [int(x) for x in model]
    n = len(t)
    G = len(group_cfg)
    admitted = {g: ([], []) for g in range(G)}  # g -> (arrival times, latency rows)
    finish = np.empty(n, dtype=np.float64)
    chosen = np.full(n, -1, dtype=np.int64)
    served = 0
    for i in range(n):
        m, a = model[i], t[i]
        hosts = [g for g in range(G) if (int(host_mask[m]) >> g) & 1]
        if not hosts:
            finish[i] = -2.0
            continue
        best, best_key = None, None
        for g in hosts:
            arr, rows = admitted[g]
            dep = _replay(arr, rows)
            key = dep[-1][0] if dep else 0.0
            if best is None or key < best_key:
                best, best_key = g, key
        chosen[i] = best
        c = int(group_cfg[best])
        S = int(cfg_stages[c])
        row = [float(stage_lat[m][c][s]) for s in range(S)]
        arr, rows = admitted[best]
        dep = _replay(arr + [a], rows + [row])
        f = dep[-1][S - 1]
        deadline = a + float(slo_scale) * float(d_single[m])
        if f > deadline:
            finish[i] = -1.0
        else:
            arr.append(a)
            rows.append(row)
            finish[i] = f
            served += 1
    if return_groups:
        return served, finish, chosen
    return served, finish


def _mix64(z):
    M64 = (1 << 64) - 1
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def simulate_batched(t, model, d_single, cfg_stages, stage_lat, group_cfg, host_mask, slo_scale,
                     max_batch, beta, on_queue=None):
    """Dynamic batching (Sec. 6.5) as an event-driven simulation: a global clock
    walks through arrival events and group-idle events; every group keeps the
    list of batches it ran, and its stage timelines come from replaying them
    through explicit stage servers (a batch is one unit whose stage latencies
    are the model's times (1 + beta (b - 1))).  Rules as in the C oracle's
    batched simulation.  Returns (served, finish[n], batch[n], digest).
    on_queue(m, queue, i, at_once), if given, sees model m's queue (trace
    indices) at each hosted arrival i: after the request joins it, or, when
    the request runs (or is dropped) at once, as it stands (it changes
    nothing)."""
    t = [float(x) for x in t]
    model = [int(x) for x in model]
    n, G = len(t), len(group_cfg)
    ran = {g: ([], []) for g in range(G)}  # g -> (batch start times, latency rows)
    queue = {m: [] for m in range(len(d_single))}
    finish = np.array([-2.0 if int(host_mask[m]) == 0 else -1.0 for m in model], dtype=np.float64)
    batch = np.zeros(n, dtype=np.int32)

    def rows(g, m, b):
        c = int(group_cfg[g])
        fac = 1.0 + float(beta) * float(b - 1)
        return [float(stage_lat[m][c][s]) * fac for s in range(int(cfg_stages[c]))]

    def free0(g):
        starts, lat = ran[g]
        dep = _replay(starts, lat)
        return dep[-1][0] if dep else 0.0

    def run(g, m, b, x):
        starts, lat = ran[g]
        dep = _replay(starts + [x], lat + [rows(g, m, b)])
        return dep[-1][-1]

    def commit(g, m, b, x):
        ran[g][0].append(x)
        ran[g][1].append(rows(g, m, b))

    def hosts(m, g):
        return (int(host_mask[m]) >> g) & 1

    i = 0
    while True:
        # next idle event among groups with queued work for a hosted model
        ev = None
        for g in range(G):
            if int(group_cfg[g]) < 0 or not any(queue[m] and hosts(m, g) for m in queue):
                continue
            x = free0(g)
            if ev is None or x < ev[0]:
                ev = (x, g)
        if ev is not None and (i >= n or ev[0] <= t[i]):
            tau, g = ev
            while True:
                cands = [m for m in queue if queue[m] and hosts(m, g)]
                if not cands:
                    break
                m = min(cands, key=lambda mm: queue[mm][0])
                head = queue[m][0]
                dl = t[head] + float(slo_scale) * float(d_single[m])
                best = 0
                for b in range(1, min(max_batch, len(queue[m])) + 1):
                    if run(g, m, b, tau) > dl:
                        break
                    best = b
                if best == 0:
                    queue[m].pop(0)
                    continue
                fin = run(g, m, best, tau)
                commit(g, m, best, tau)
                for r in queue[m][:best]:
                    finish[r] = fin
                    batch[r] = best
                del queue[m][:best]
                break
            continue
        if i >= n:
            break
        m = model[i]
        if int(host_mask[m]) != 0:
            avail = [(free0(g), g) for g in range(G) if hosts(m, g) and free0(g) <= t[i]]
            if avail:
                if on_queue:
                    on_queue(m, tuple(queue[m]), i, True)
                _, g = min(avail)
                fin = run(g, m, 1, t[i])
                if not fin > t[i] + float(slo_scale) * float(d_single[m]):
                    commit(g, m, 1, t[i])
                    finish[i] = fin
                    batch[i] = 1
            else:
                queue[m].append(i)
                if on_queue:
                    on_queue(m, tuple(queue[m]), i, False)
        i += 1
    served = int((batch > 0).sum())
    h = 0
    fs = 0
    for r in range(n):
        if batch[r] > 0:
            h = (h + _mix64(r)) & ((1 << 64) - 1)
            fs = (fs + int(np.float64(finish[r]).view(np.uint64))) & ((1 << 64) - 1)
    return served, finish, batch, (h, fs)
