"""Brute-force event-driven simulation of tiny traces (test infrastructure).

An independent second implementation of the same serial-service model as the
C oracle, written the other way round: instead of fixing every event time at
admission, it keeps a time-ordered heap of events (arrival, prefill done, KV
arrived at decode, decode done), explicit per-instance queues and an
in-flight ledger, and lets servers pick their next request as they free up.
The router reads the live state at each arrival; its "committed work"
(backlog) is obtained by projecting each instance's current queue forward.

Model (paper, Section III-D simulator and Section VI serial-service model):
  * a prefill instance serves its queue one request at a time in arrival
    order; a request's KV moves to its decode instance after a transfer delay;
  * a decode instance serves its assigned requests one at a time in admission
    order and idles until the KV of the request at the head of its queue has
    arrived;
  * at equal times completions and KV arrivals precede arrivals, so a request
    that ends at t no longer counts at an arrival at t; equal arrival times
    are routed in index order.

The cost equation (Section III-A) is evaluated in numpy float32, one rounding
per operation, in the written order.  Only small traces are practical.
"""
from __future__ import annotations

import heapq
from collections import deque
from typing import Dict, List

import numpy as np

F = np.float32
NS = F(1e-9)

ARRIVE, KV_AT, DONE = 2, 1, 0  # heap priority at equal times


def _key(c: np.float32) -> int:
    c = F(c)
    if np.isnan(c):
        return 0x7FC00000
    if c == 0:
        return 0
    return int(np.frombuffer(c.tobytes(), np.uint32)[0])


def _cost(pt: Dict, backlog: np.float32, work: np.float32, sg: np.float32, kv: int, k: int, inv: np.float32,
          q: int) -> np.float32:
    press = F(kv + k) * inv
    load = F(pt["w_b"]) * backlog * sg
    size = work * (F(1.0) + F(pt["rho"]) * press) * sg
    return load + size + F(pt["w_q"]) * F(q)


def _pair(u: int, v: int, n: int):
    """The sampled policy's two candidates among n instances from words u, v:
    u picks one of the n, v one of the n - 1 others (counted past the first)."""
    a = (int(u) * n) >> 32
    if n < 2:
        return a, a
    b = (int(v) * (n - 1)) >> 32
    return a, (b if b < a else b + 1)


def simulate(pt: Dict, arrival, prompt, out, pred, cls, words=None) -> Dict[str, np.ndarray]:
    n = len(arrival)
    P, D = int(pt["n_prefill"]), int(pt["n_decode"])
    s_pre = [int(pt["pre_base_ns"]) + int(prompt[r]) * int(pt["pre_tok_ns"]) for r in range(n)]
    s_dec = [(int(out[r]) - 1) * int(pt["dec_tok_ns"]) for r in range(n)]
    xfer = [int(prompt[r]) * int(pt["xfer_tok_ns"]) for r in range(n)]

    pre_wait: List[deque] = [deque() for _ in range(P)]
    pre_cur: List = [None] * P  # (rid, end)
    dec_wait: List[List[int]] = [[] for _ in range(D)]
    dec_cur: List = [None] * D
    led_pre: List[List[int]] = [[] for _ in range(P)]
    led_dec: List[List[int]] = [[] for _ in range(D)]
    kv_ready = [False] * n
    kv_at = [None] * n
    pf_end = [None] * n
    dec_end = [None] * n
    i_pre = [-1] * n
    i_dec = [-1] * n

    heap = []
    seq = 0

    def push(t, prio, kind, rid):
        nonlocal seq
        heapq.heappush(heap, (t, prio, seq, kind, rid))
        seq += 1

    for r in range(n):
        push(int(arrival[r]), ARRIVE, "arrive", r)

    def start_pre(j, t):
        if pre_cur[j] is None and pre_wait[j]:
            r = pre_wait[j].popleft()
            pre_cur[j] = (r, t + s_pre[r])
            push(t + s_pre[r], DONE, "pf_done", r)

    def start_dec(j, t):
        if dec_cur[j] is None and dec_wait[j] and kv_ready[dec_wait[j][0]]:
            r = dec_wait[j].pop(0)
            dec_cur[j] = (r, t + s_dec[r])
            push(t + s_dec[r], DONE, "dec_done", r)

    def projected_pf_end(now):
        """Finish time of every request still held by a prefill instance."""
        proj = {}
        for j in range(P):
            t = pre_cur[j][1] if pre_cur[j] is not None else now
            if pre_cur[j] is not None:
                proj[pre_cur[j][0]] = pre_cur[j][1]
            for r in pre_wait[j]:
                t = t + s_pre[r]
                proj[r] = t
        return proj

    def busy_until_pre(j, now):
        if pre_cur[j] is None:
            return now
        t = pre_cur[j][1]
        for r in pre_wait[j]:
            t += s_pre[r]
        return t

    def busy_until_dec(j, now, proj):
        t = dec_cur[j][1] if dec_cur[j] is not None else now
        for r in dec_wait[j]:
            ready = kv_at[r] if kv_at[r] is not None else proj[r] + xfer[r]
            t = max(t, ready) + s_dec[r]
        return t

    def backlog(pool, j, now, proj):
        if pt["backlog_mode"] == "true":
            b = busy_until_pre(j, now) if pool == 0 else busy_until_dec(j, now, proj)
            return F(max(b - now, 0)) * NS
        led = led_pre[j] if pool == 0 else led_dec[j]
        if pool == 0:
            pend = sum(int(prompt[r]) for r in led)
            return F(pt["tau_pre_s"]) * F(pend) + F(pt["pre_base_s"]) * F(len(led))
        pend = sum(int(pred[r]) for r in led)
        return F(pt["tau_dec_s"]) * F(pend)

    def decide(pool, r, now, proj):
        n_inst = P if pool == 0 else D
        led = led_pre if pool == 0 else led_dec
        if pt["policy"] == "round_robin":
            return r % n_inst
        if pt["policy"] == "least_loaded":
            qs = [len(led[j]) for j in range(n_inst)]
            return int(np.argmin(qs))  # first minimum = lowest index
        if pt["policy"] == "length_threshold":
            part = list(range(n_inst))
            if pool == 1 and n_inst > 1:
                h = (n_inst + 1) // 2
                part = part[h:] if int(pred[r]) >= int(pt["len_threshold"]) else part[:h]
            qs = [len(led[j]) for j in part]
            return part[int(np.argmin(qs))]
        sg = F(pt["sigma"][int(cls[r])])
        if pool == 0:
            work = F(pt["w_s"]) * F(int(prompt[r])) * F(pt["tau_pre_s"])
            k = int(prompt[r])
            inv = F(1.0) / F(pt["kv_cap_pre"])
            fp = lambda x: int(prompt[x])
        else:
            work = F(pt["w_s"]) * F(int(pred[r])) * F(pt["tau_dec_s"])
            k = int(prompt[r]) + int(pred[r])
            inv = F(1.0) / F(pt["kv_cap_dec"])
            fp = lambda x: int(prompt[x]) + int(out[x])
        offered = range(n_inst)
        if pt["policy"] == "learned_sampled":
            offered = sorted(set(_pair(words[r][2 * pool], words[r][2 * pool + 1], n_inst)))
        best, best_key = 0, None
        for j in offered:
            kv = sum(fp(x) for x in led[j])
            c = _cost(pt, backlog(pool, j, now, proj), work, sg, kv, k, inv, len(led[j]))
            kk = _key(c)
            if best_key is None or kk < best_key:
                best, best_key = j, kk
        return best

    while heap:
        t, _, _, kind, r = heapq.heappop(heap)
        if kind == "arrive":
            proj = projected_pf_end(t)
            ip = decide(0, r, t, proj)
            idd = decide(1, r, t, proj)
            i_pre[r], i_dec[r] = ip, idd
            pre_wait[ip].append(r)
            led_pre[ip].append(r)
            dec_wait[idd].append(r)
            led_dec[idd].append(r)
            start_pre(ip, t)
        elif kind == "pf_done":
            j = i_pre[r]
            pre_cur[j] = None
            led_pre[j].remove(r)
            pf_end[r] = t
            kv_at[r] = t + xfer[r]
            push(t + xfer[r], KV_AT, "kv_at", r)
            start_pre(j, t)
        elif kind == "kv_at":
            kv_ready[r] = True
            start_dec(i_dec[r], t)
        elif kind == "dec_done":
            j = i_dec[r]
            dec_cur[j] = None
            led_dec[j].remove(r)
            dec_end[r] = t
            start_dec(j, t)

    ttft = np.array([pf_end[r] - int(arrival[r]) for r in range(n)], np.int64)
    span = np.array([dec_end[r] - pf_end[r] for r in range(n)], np.int64)
    return dict(i_pre=np.array(i_pre, np.int32), i_dec=np.array(i_dec, np.int32), ttft_ns=ttft,
                decode_span_ns=span)
