"""Brute-force simulation of the continuous-batching service model
(test infrastructure).

A second, independent implementation of the model the C oracle's
orc_sim_replica_batched follows (Section VI: both stages batched
continuously, each request slowed by 1 + beta (b - 1) while b requests share an
instance), written the other way round: instead of a virtual clock per
instance it keeps every request's remaining stand-alone work and, between
consecutive events, takes dt / (1 + beta (b - 1)) off each request of every
busy instance.  The next event is found by scanning every instance for the
request with the least remaining work.

With ``exact=True`` all times and works are Python Fractions (beta is taken
as the exact value of its float), so the result is the model's exact answer;
otherwise plain Python floats.  Only small traces are practical.

Event order at equal times: completions, then KV landings, then arrivals in
index order.  The router reads, at each arrival, the instance's requests in
flight, cache tokens, and either the stand-alone work still owed (clock
backlog: the remaining work of the batch plus, on a decode instance, the full
decode work of requests routed there that have not joined) or the in-flight
ledger (proxy backlog).  The cost equation is evaluated in numpy float32 in
the written order.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Dict

import numpy as np

from .des_heap import F, NS, _cost, _key, _pair


def simulate_batched(pt: Dict, arrival, prompt, out, pred, cls, words=None, exact: bool = False) -> Dict:
    num = Fraction if exact else float
    n = len(arrival)
    P, D = int(pt["n_prefill"]), int(pt["n_decode"])
    beta = (num(pt["beta_pre"]), num(pt["beta_dec"]))
    w_pre = [int(pt["pre_base_ns"]) + int(prompt[r]) * int(pt["pre_tok_ns"]) for r in range(n)]
    w_dec = [(int(out[r]) - 1) * int(pt["dec_tok_ns"]) for r in range(n)]
    xfer = [int(prompt[r]) * int(pt["xfer_tok_ns"]) for r in range(n)]

    # remaining stand-alone work of the requests each instance is serving
    batch = ([{} for _ in range(P)], [{} for _ in range(D)])
    # requests routed to a decode instance that have not joined, and the
    # landing time of those whose prefill has ended
    routed = [set() for _ in range(D)]
    landing: Dict[int, object] = {}
    # the router's in-flight ledger: admitted and not yet done, per pool
    ledger = ([[] for _ in range(P)], [[] for _ in range(D)])
    pf_end = [None] * n
    dec_end = [None] * n
    i_pre = [-1] * n
    i_dec = [-1] * n
    zero = num(0)

    def factor(pool, b):
        return 1 + beta[pool] * (b - 1)

    def completion_in():
        """Time from now to each busy instance's next completion."""
        return {(pool, j): min(jobs.values()) * factor(pool, len(jobs))
                for pool in (0, 1) for j, jobs in enumerate(batch[pool]) if jobs}

    def advance(dt):
        if dt == 0:
            return
        for pool in (0, 1):
            for jobs in batch[pool]:
                if jobs:
                    s = factor(pool, len(jobs))
                    for r in jobs:
                        jobs[r] -= dt / s

    def owed(pool, j):
        w = sum(batch[pool][j].values(), zero)
        if pool == 1:
            w += sum(w_dec[r] for r in routed[j])
        return w

    def decide(pool, r):
        n_inst = P if pool == 0 else D
        led = ledger[pool]
        pol = pt["policy"]
        if pol == "round_robin":
            return r % n_inst
        if pol in ("least_loaded", "length_threshold"):
            part = list(range(n_inst))
            if pol == "length_threshold" and pool == 1 and n_inst > 1:
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
        if pol == "learned_sampled":
            offered = sorted(set(_pair(words[r][2 * pool], words[r][2 * pool + 1], n_inst)))
        best, best_key = 0, None
        for j in offered:
            if pt["backlog_mode"] == "true":
                bl = F(float(owed(pool, j))) * NS
            elif pool == 0:
                bl = F(pt["tau_pre_s"]) * F(sum(int(prompt[x]) for x in led[j])) + F(pt["pre_base_s"]) * F(len(led[j]))
            else:
                bl = F(pt["tau_dec_s"]) * F(sum(int(pred[x]) for x in led[j]))
            kv = sum(fp(x) for x in led[j])
            c = _cost(pt, bl, work, sg, kv, k, inv, len(led[j]))
            if best_key is None or _key(c) < best_key:
                best, best_key = j, _key(c)
        return best

    t = zero
    r_next = 0
    while True:
        cin = completion_in()
        tc = t + min(cin.values()) if cin else None
        tl = min(landing.values()) if landing else None
        ta = num(int(arrival[r_next])) if r_next < n else None
        if tc is None and tl is None and ta is None:
            break
        if tc is not None and (tl is None or tc <= tl) and (ta is None or tc <= ta):
            # completions: on each instance whose next completion is the
            # earliest, every request with the least remaining work leaves
            dt = min(cin.values())
            advance(tc - t)
            t = tc
            for (pool, j), ci in cin.items():
                if ci != dt:
                    continue
                jobs = batch[pool][j]
                m = min(jobs.values())
                for r in [x for x, w in jobs.items() if w == m]:
                    del jobs[r]
                    ledger[pool][j].remove(r)
                    if pool == 0:
                        pf_end[r] = t
                        landing[r] = t + xfer[r]
                    else:
                        dec_end[r] = t
            continue
        if tl is not None and (ta is None or tl <= ta):
            advance(tl - t)
            t = tl
            for r in sorted(x for x, v in landing.items() if v == t):
                del landing[r]
                d = i_dec[r]
                routed[d].discard(r)
                batch[1][d][r] = num(w_dec[r])
            continue
        # the arrival of request r_next
        advance(ta - t)
        t = ta
        r = r_next
        r_next += 1
        ip, idd = decide(0, r), decide(1, r)
        i_pre[r], i_dec[r] = ip, idd
        batch[0][ip][r] = num(w_pre[r])
        ledger[0][ip].append(r)
        ledger[1][idd].append(r)
        routed[idd].add(r)

    def rnd(x):
        return int(round(x))  # nearest, ties to even (Fraction and float alike)

    ex_ttft = [pf_end[r] - int(arrival[r]) for r in range(n)]
    ex_span = [dec_end[r] - pf_end[r] for r in range(n)]
    return dict(i_pre=np.array(i_pre, np.int32), i_dec=np.array(i_dec, np.int32),
                ttft_ns=np.array([rnd(x) for x in ex_ttft], np.int64),
                decode_span_ns=np.array([rnd(x) for x in ex_span], np.int64),
                exact=dict(ttft_ns=ex_ttft, decode_span_ns=ex_span))
