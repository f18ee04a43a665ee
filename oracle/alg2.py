"""Alg. 2 of the paper (Sec. 4.2) scored by the C oracle -- TEST INFRASTRUCTURE ONLY.

Enumeration-based group partition and model-parallel configuration selection:
for every model-bucket partition and every device-bucket split, each bucket
picks its best (group partition, parallel configuration) by running Alg. 1
(beam search, or the fast heuristic) on the bucket's models and devices with
the whole workload, the placement is the concatenation of the buckets'
choices, and the search keeps the best placement.  Written loop by loop in
the order Alg. 2 states it, without the sharing of repeated bucket problems
that the native driver does.

Readings (each one also stated in the design notes):
  - model buckets: the models sorted by single-device latency (ties by id)
    are cut into contiguous runs -- a bucket holds models of similar latency
    -- and every cut into at most max_buckets runs whose latency span is at
    most bucket_threshold is a potential bucket partition, so models whose
    latencies differ by more than the threshold always land in different
    buckets; cuts are taken by run count, then in lexicographic order;
  - device buckets: every split of the devices into the buckets in multiples
    of device_unit, lexicographic; a split is dropped when the largest bucket
    load exceeds balance_ratio times the smallest, where a bucket's load is
    the sum over its models of (requests in the trace x d_single), divided by
    its devices (the pace at which it must serve, compared across buckets);
  - group partitions / parallel configurations: for each configuration c that
    fits the bucket, equal groups of c's device count and one last group of
    the remaining devices, configured with the configuration of that device
    count whose pipeline is deepest without exceeding c's (lowest index on
    ties; c is skipped if none exists or more than 64 groups would result);
    each group holds (its devices x device memory) MiB;
  - a bucket's option is scored by the requests it serves (other buckets'
    models are never placed there); plm_i* starts empty (0 served) and is
    replaced only by a strictly better option, best_plm likewise.
"""
from __future__ import annotations

import numpy as np

from . import greedy


def model_bucket_cuts(d_single, max_buckets, threshold):
    """Potential model buckets: (order, list of cuts); a cut is the list of
    run start positions in `order` (models sorted by latency, ties by id)."""
    d = np.asarray(d_single, dtype=np.float64)
    order = sorted(range(len(d)), key=lambda m: (d[m], m))
    M = len(order)
    cuts = []

    def rec(pos, left, starts):
        if pos == M:
            if left == 0:
                cuts.append(list(starts))
            return
        if left == 0:
            return
        for end in range(pos + 1, M + 1):
            if d[order[end - 1]] - d[order[pos]] > threshold:
                break
            rec(end, left - 1, starts + [pos])

    for k in range(1, min(max_buckets, M) + 1):
        rec(0, k, [])
    return order, cuts


def device_splits(units, k):
    """Compositions of `units` into k positive parts, lexicographic."""
    out = []

    def rec(left, parts, acc):
        if parts == 1:
            out.append(acc + [left])
            return
        for x in range(1, left - (parts - 1) + 1):
            rec(left - x, parts - 1, acc + [x])

    if units >= k:
        rec(units, k, [])
    return out


def bucket_options(H, cfg_devices, cfg_stages, device_mem_mib):
    """(c, group_cfg, group_mem) for every configuration option of a bucket
    with H devices."""
    out = []
    C = len(cfg_devices)
    for c in range(C):
        size = int(cfg_devices[c])
        if size > H:
            continue
        nfull, rem = divmod(H, size)
        groups = [c] * nfull
        if rem > 0:
            last = None
            for c2 in range(C):
                if int(cfg_devices[c2]) == rem and cfg_stages[c2] <= cfg_stages[c]:
                    if last is None or cfg_stages[c2] > cfg_stages[last]:
                        last = c2
            if last is None:
                continue
            groups.append(last)
        if len(groups) > 64:
            continue
        mem = [int(cfg_devices[g]) * int(device_mem_mib) for g in groups]
        out.append((c, np.array(groups, np.int32), np.array(mem, np.int64)))
    return out


def placement_search(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat, cfg_devices, n_devices,
                     device_unit, device_mem_mib, bucket_threshold, balance_ratio, max_buckets, beam,
                     slo_scale):
    """Alg. 2.  beam >= 1: Alg. 1 with that beam; beam == 0: the fast
    heuristic.  Returns dict(served, buckets=[dict(models, devices, cfg,
    group_cfg, mask, served)], n_bucket_configs, n_device_splits,
    n_kept_splits)."""
    M = len(d_single)
    d = np.asarray(d_single, dtype=np.float64)
    nreq = np.bincount(np.asarray(model, dtype=np.int64), minlength=M)
    order, cuts = model_bucket_cuts(d, max_buckets, bucket_threshold)
    best = {"served": 0, "buckets": []}
    n_splits = n_kept = 0
    for starts in cuts:
        k = len(starts)
        buckets = [order[starts[b]:(starts[b + 1] if b + 1 < k else M)] for b in range(k)]
        for split in device_splits(n_devices // device_unit, k):
            n_splits += 1
            H = [x * device_unit for x in split]
            if balance_ratio != float("inf"):
                rhos = []
                for b in range(k):
                    load = 0.0
                    for m in buckets[b]:
                        load += float(nreq[m]) * d[m]
                    rhos.append(load / float(H[b]))
                if not (max(rhos) <= balance_ratio * min(rhos)):
                    continue
            n_kept += 1
            plm = []
            total = 0
            for b in range(k):
                star = None
                for (c, gcfg, gmem) in bucket_options(H[b], cfg_devices, cfg_stages, device_mem_mib):
                    if beam == 0:
                        r = greedy.fast_selection(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat,
                                                  gcfg, gmem, slo_scale, models=buckets[b])
                    else:
                        r = greedy.beam_selection(lib, t, model, d_single, weight_mib, cfg_stages, stage_lat,
                                                  gcfg, gmem, slo_scale, beam=beam, models=buckets[b])
                    if r["best_served"] > (0 if star is None else star["served"]):
                        star = {"cfg": c, "group_cfg": gcfg, "mask": r["best_mask"], "served": r["best_served"]}
                entry = {"models": sorted(buckets[b]), "devices": H[b]}
                entry.update(star if star is not None else
                             {"cfg": -1, "group_cfg": np.zeros(0, np.int32), "mask": np.zeros(M, np.uint64),
                              "served": 0})
                plm.append(entry)
                total += entry["served"]
            if total > best["served"]:
                best = {"served": total, "buckets": plm}
    best["n_bucket_configs"] = len(cuts)
    best["n_device_splits"] = n_splits
    best["n_kept_splits"] = n_kept
    return best

