"""Token-at-a-time reference scheduler, used only to pin the C oracle.

It builds each token batch by handing out the token budget ONE TOKEN AT A TIME
(not in chunks), and accumulates the batch-time features per token from their
descriptions in Sec. 4.1 (token-batch processing time):
  * each decode token reads the KV cache of its sequence: C gets the sequence's
    context length c before the batch;
  * the k-th prefill token of a chunk attends to the context already present plus
    the chunk's preceding tokens and itself: A gets c + k.
Python floats are binary64 with round-to-nearest-even and no fused
multiply-add.  The logic is written independently of ``oracle/sfs_oracle.c``.
"""

from __future__ import annotations

import numpy as np


class Req:
    __slots__ = ("rp", "rd", "cx", "query", "prompt")

    def __init__(self, rp, rd, cx, query=-1):
        self.rp, self.rd, self.cx = int(rp), int(rd), int(cx)
        self.query = int(query)     # index of the routed query, -1 for residents
        self.prompt = int(rp) if cx == 0 else -1

    def tup(self):
        return (self.rp, self.rd, self.cx)


class BFInstance:
    def __init__(self, a, b, c, d, e, budget, max_seqs, rp=(), rd=(), cx=(), clock=0.0):
        self.coef = (float(a), float(b), float(c), float(d), float(e))
        self.B, self.M = int(budget), int(max_seqs)
        self.reqs = [Req(x, y, z) for x, y, z in zip(rp, rd, cx)]
        self.clock = float(clock)

    def copy(self):
        o = BFInstance(*self.coef, self.B, self.M, clock=self.clock)
        o.reqs = []
        for r in self.reqs:
            x = Req(*r.tup(), query=r.query)
            x.prompt = r.prompt
            o.reqs.append(x)
        return o

    # -- one batch, token by token ---------------------------------------------------
    def batch(self):
        """Return (T, features, per-request tokens) of the next batch; do not apply it."""
        budget = self.B
        given_pre = [0] * len(self.reqs)
        given_dec = [0] * len(self.reqs)
        in_service = [r.cx > 0 for r in self.reqs]
        slots = sum(in_service)
        P = D = Cf = A = 0
        for i, r in enumerate(self.reqs):           # one decode token per decoding sequence
            if r.cx > 0 and r.rp == 0 and budget > 0:
                given_dec[i] = 1
                budget -= 1
                D += 1
                Cf += r.cx
        while budget > 0:                            # then prefill, one token at a time
            nxt = None
            for i, r in enumerate(self.reqs):
                if r.rp - given_pre[i] > 0:
                    nxt = i
                    break
            if nxt is None:
                break
            if not in_service[nxt]:
                if slots >= self.M:
                    break                            # head of line cannot get a slot
                in_service[nxt] = True
                slots += 1
            given_pre[nxt] += 1
            budget -= 1
            P += 1
            A += self.reqs[nxt].cx + given_pre[nxt]
        a, b, c, d, e = self.coef
        T = a
        T = T + b * float(P)
        T = T + c * float(D)
        T = T + d * float(Cf)
        T = T + e * float(A)
        return T, (P, D, Cf, A), given_pre, given_dec

    def apply(self, given_pre, given_dec):
        keep = []
        for i, r in enumerate(self.reqs):
            r.cx += given_pre[i] + given_dec[i]
            r.rp -= given_pre[i]
            r.rd -= given_dec[i]
            if r.rd > 0:
                keep.append(r)
        self.reqs = keep

    def step(self, first_token=None, reading=0):
        """One batch.  first_token(query, end_time) is called for every routed query
        whose first token the batch produces: under reading 0 a query that decodes
        while its context is still exactly its prompt (it has not decoded before);
        under reading 1 a query whose remaining prefill reaches 0 in the batch."""
        T, f, gp, gd = self.batch()
        self.clock = self.clock + T
        if first_token is not None:
            for i, r in enumerate(self.reqs):
                if r.query < 0:
                    continue
                if reading == 1:
                    hit = r.rp > 0 and r.rp - gp[i] == 0
                else:
                    hit = gd[i] == 1 and r.cx == r.prompt
                if hit:
                    first_token(r.query, self.clock)
        self.apply(gp, gd)
        return T, f

    def advance(self, t, first_token=None, reading=0):
        while self.reqs and self.clock < t:
            self.step(first_token, reading)
        if not self.reqs and self.clock < t:
            self.clock = float(t)

    def append(self, p, d, query=-1):
        self.reqs.append(Req(p, max(int(d), 1), 0, query))

    def estimate(self, p, d, t, reading=0):
        w = self.copy()
        w.append(p, d)
        q = w.reqs[-1]
        E = w.clock
        n = 0
        feats = []
        while True:
            T, f, gp, gd = w.batch()
            me = len(w.reqs) - 1
            if reading == 1:
                done = gp[me] > 0 and gp[me] == q.rp
            else:
                done = gd[me] == 1
            E = E + T
            n += 1
            feats.append(f)
            w.apply(gp, gd)
            if done:
                return E - t, n, feats

    def state(self):
        return [r.tup() for r in self.reqs]


def instances_of(wl):
    out = []
    sched = getattr(wl, "sched", None)
    for j in range(wl.n_inst):
        rp, rd, cx = wl.instance_requests(j)
        if sched is None:
            out.append(BFInstance(wl.a[j], wl.b[j], wl.c[j], wl.d[j], wl.e[j], wl.budget[j],
                                  wl.max_seqs[j], rp, rd, cx, wl.clock_ms[j]))
        else:
            out.append(BFSchedInstance(wl.a[j], wl.b[j], wl.c[j], wl.d[j], wl.e[j],
                                       wl.budget[j], wl.max_seqs[j], sched[j], rp, rd, cx,
                                       wl.clock_ms[j]))
    return out


def _pick_constrained(row, util, tau):
    """Eq. 3 restated: the feasible instance with the best (utility, -index), or, if no
    instance meets the target, the one with the smallest (TTFT, index)."""
    feas = [j for j in range(len(row)) if row[j] <= tau]
    if feas:
        return max(feas, key=lambda j: (util[j], -j))
    return min(range(len(row)), key=lambda j: (row[j], j))


def trace(wl, scenario=0, n_q=None, reading=0, tau=None, realized=None):
    """Sequential trace with the route computed by numpy (first maximum wins), or by
    the constrained rule of Eq. 3 when per-query targets ``tau`` are given.

    With an array ``realized`` [N], the replay records each query's first-token
    time minus its arrival; queries without it at the end get it from a copy of
    their instance run on with no further arrivals."""
    insts = instances_of(wl)
    N = wl.n_q if n_q is None else n_q
    col = np.asarray(wl.col)
    wc, wlat = float(wl.w_cost[scenario]), float(wl.w_lat_ms[scenario])
    choices, rows = [], []
    ft = None
    if realized is not None:
        realized[:N] = np.nan

        def ft(q, end):
            assert np.isnan(realized[q]), "a query got two first tokens"
            realized[q] = end - float(wl.q_t_ms[q])
    if N:
        for x in insts:
            x.advance(wl.q_t_ms[0], ft, reading)
    for i in range(N):
        p, d, t = int(wl.q_prefill[i]), int(wl.q_decode[i]), float(wl.q_t_ms[i])
        row = np.array([x.estimate(p, d, t, reading)[0] for x in insts])
        acc = wl.acc[i][col]
        cost = wl.cost[i][col]
        if tau is None:
            u = (acc - wc * cost) - wlat * row
            m = int(np.argmax(u))
        else:
            m = _pick_constrained(row, acc - wc * cost, float(tau[i]))
        choices.append(m)
        rows.append(row)
        insts[m].append(p, d, query=i if ft else -1)
        t_next = float(wl.q_t_ms[i + 1]) if i + 1 < N else t
        for x in insts:
            x.advance(t_next, ft, reading)
    if ft is not None:
        for j, x in enumerate(insts):
            mine = [i for i in range(N) if choices[i] == j]
            w = x.copy()
            while any(np.isnan(realized[i]) for i in mine):
                w.step(ft, reading)
    return np.array(choices, np.int32), np.array(rows), insts


# ------------------------------------------------------------------ scheduler limits
class SReq:
    __slots__ = ("rp", "rd", "cx", "query", "prompt", "blocks", "kv", "first_done")

    def __init__(self, rp, rd, cx, query=-1):
        self.rp, self.rd, self.cx = int(rp), int(rd), int(cx)
        self.query = int(query)
        self.prompt = int(rp) if cx == 0 else -1
        self.blocks = []        # ids of the KV blocks held
        self.kv = 0             # tokens those blocks hold
        self.first_done = False

    def clone(self):
        x = SReq(self.rp, self.rd, self.cx, self.query)
        x.prompt, x.blocks, x.kv, x.first_done = self.prompt, list(self.blocks), self.kv, \
            self.first_done
        return x


class BFSchedInstance:
    """The batch under scheduler limits, restated token by token with its own
    bookkeeping: running requests (in admission order) and waiting requests (in queue
    order) are two lists; the KV cache is a pool of numbered blocks of S slots, each
    running request owning a list of block ids that it fills one token at a time,
    taking a block from the pool whenever its last one is full; when the pool is
    empty, the last running request is popped and pushed to the front of the
    waiting list with its blocks returned.  The context limit ends a decoding
    request when its context reaches it (the predicted decode is not cut)."""

    def __init__(self, a, b, c, d, e, budget, max_seqs, lim, rp=(), rd=(), cx=(), clock=0.0):
        self.coef = (float(a), float(b), float(c), float(d), float(e))
        self.B, self.M = int(budget), int(max_seqs)
        H, K, S, X = (int(v) for v in lim)
        self.H = H if H > 0 else None
        self.K, self.S, self.X = K, (S if K > 0 else 1), X
        self.pool = list(range(K - 1, -1, -1)) if K > 0 else None
        self.running, self.waiting = [], []
        self.clock = float(clock)
        self.preemptions = 0
        for x, y, z in zip(rp, rd, cx):
            r = SReq(x, y, z)
            if r.cx > 0:
                self.running.append(r)
                for _ in range(r.cx):
                    assert self._slot(r, allow_preempt=False)
            else:
                self.waiting.append(r)

    def copy(self):
        o = BFSchedInstance(*self.coef, self.B, self.M, (0, 0, 1, 0), clock=self.clock)
        o.H, o.K, o.S, o.X = self.H, self.K, self.S, self.X
        o.pool = None if self.pool is None else list(self.pool)
        o.running = [r.clone() for r in self.running]
        o.waiting = [r.clone() for r in self.waiting]
        o.preemptions = self.preemptions
        return o

    def requests(self):
        return self.running + self.waiting

    # one KV slot for one more token of r; False if r itself had to be preempted
    def _slot(self, r, allow_preempt=True):
        if self.pool is not None and r.kv == len(r.blocks) * self.S:
            while not self.pool:
                assert allow_preempt
                if self._preempt_last() is r:
                    return False
            r.blocks.append(self.pool.pop())
        r.kv += 1
        return True

    def _preempt_last(self):
        v = self.running.pop()
        if self.pool is not None:
            self.pool.extend(v.blocks)
        v.blocks, v.kv = [], 0
        self._left += self._given.pop(id(v), (None, 0))[1]
        v.rp, v.cx = v.rp + v.cx, 0
        self.waiting.insert(0, v)
        self._preempted = True
        self.preemptions += 1
        return v

    def batch(self):
        """Build and apply one batch; return (T, (P, D, C, A), events), events being
        (request, 'dec' | 'pre', tokens) for every request served."""
        self._left, self._given, self._preempted = self.B, {}, False
        for r in list(self.running):                 # decode tokens, running order
            if r not in self.running:
                break
            if r.rp != 0:
                continue
            if not self._slot(r):
                break
            self._given[id(r)] = ("dec", 1)
            self._left -= 1
        for r in list(self.running):                 # chunks of partial prefills
            if r not in self.running:
                break
            if r.rp == 0:
                continue
            g = min(r.rp, self._left) if self.H is None else min(r.rp, self.H, self._left)
            if g == 0:
                continue
            ok = True
            for _ in range(g):
                if not self._slot(r):
                    ok = False
                    break
            if not ok:
                break
            self._given[id(r)] = ("pre", g)
            self._left -= g
        if not self._preempted:                      # admissions, FCFS
            while self.waiting and self._left > 0 and len(self.running) < self.M:
                w = self.waiting[0]
                g = min(w.rp, self._left) if self.H is None else min(w.rp, self.H, self._left)
                if self.pool is not None and -(-g // self.S) > len(self.pool):
                    break
                self.waiting.pop(0)
                self.running.append(w)
                for _ in range(g):
                    assert self._slot(w, allow_preempt=False)
                self._given[id(w)] = ("pre", g)
                self._left -= g
        # features, token by token, then apply
        P = D = Cf = A = 0
        events = []
        for r in self.running:
            kind, n = self._given.get(id(r), (None, 0))
            if kind == "dec":
                D += 1
                Cf += r.cx
            elif kind == "pre":
                for k in range(1, n + 1):
                    P += 1
                    A += r.cx + k
            if kind:
                events.append((r, kind, n))
        a, b, c, d, e = self.coef
        T = a
        T = T + b * float(P)
        T = T + c * float(D)
        T = T + d * float(Cf)
        T = T + e * float(A)
        keep = []
        for r in self.running:
            kind, n = self._given.get(id(r), (None, 0))
            if kind == "dec":
                r.cx += 1
                r.rd -= 1
            elif kind == "pre":
                r.cx += n
                r.rp -= n
            if r.rd == 0 or (self.X > 0 and r.rp == 0 and r.cx == self.X):
                if self.pool is not None:
                    self.pool.extend(r.blocks)
                continue
            keep.append(r)
        self.running = keep
        return T, (P, D, Cf, A), events

    def step(self, first_token=None, reading=0):
        T, f, events = self.batch()
        self.clock = self.clock + T
        if first_token is not None:
            for r, kind, n in events:
                if r.query < 0 or r.first_done:
                    continue
                hit = (kind == "pre" and r.rp == 0) if reading == 1 else kind == "dec"
                if hit:
                    r.first_done = True
                    first_token(r.query, self.clock)
        return T, f

    @property
    def reqs(self):
        return self.running + self.waiting

    def advance(self, t, first_token=None, reading=0):
        while self.reqs and self.clock < t:
            self.step(first_token, reading)
        if not self.reqs and self.clock < t:
            self.clock = float(t)

    def append(self, p, d, query=-1):
        self.waiting.append(SReq(p, max(int(d), 1), 0, query))

    def estimate(self, p, d, t, reading=0):
        w = self.copy()
        w.append(p, d)
        q = w.waiting[-1]
        E = w.clock
        n = 0
        while True:
            T, f, events = w.batch()
            E = E + T
            n += 1
            mine = [kind for r, kind, _ in events if r is q]
            if reading == 1:
                done = mine == ["pre"] and q.rp == 0
            else:
                done = mine == ["dec"]
            if done:
                return E - t, n

    def state(self):
        """(rp, rd, cx) in list order, the predicted decode cut to the context limit
        as the oracle keeps it."""
        out = []
        for r in self.running + self.waiting:
            rd = r.rd if self.X <= 0 else min(r.rd, self.X - (r.cx + r.rp))
            out.append((r.rp, rd, r.cx))
        return out
