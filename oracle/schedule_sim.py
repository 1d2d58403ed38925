"""Independent safety oracle for decode-step task schedules (test
infrastructure only: the product path never imports it).

The library's static checker (paper §4, paragraph "The invariants validate()
proves" and Table "Static checks") must reject every schedule that could
deadlock or race before it is launched.  The paper measures that promise
against mutants and random task graphs labelled by an oracle that does not
call the checker (§5, Table "Validator soundness").  This module is such an
oracle, written from the task semantics alone, in plain Python:

* structural labels: operation, queue, counter and range bounds, the per-task
  row cap and the wait-slot cap;
* a dynamic label: the schedule is executed on a model of the device (one
  in-order queue per workgroup; a task starts once each of its counters has
  reached its wait count, finishes later, then increments its signal counter;
  an inline task runs right after the producer whose increment completes its
  single wait counter) under many random interleavings.  An execution that
  stops with tasks left is a deadlock; a task that starts reading a value
  whose writer has not finished is a race; a value written twice, or an
  output of the step never written, is an output error.

A schedule is unsafe if any label says so.  Like the paper's counter-driven
oracle, the dynamic part only observes races that some sampled interleaving
exhibits (a wait count below the producer count, for instance, is unsafe
only in interleavings where the waiting task starts early), so it can miss
hazards the static checker proves; half the sampled runs are therefore
adversarial (slow producers, eager consumers).  The test asks for zero false
accepts: no schedule this oracle finds unsafe may be accepted by the checker.

``find_cycle`` is an independent depth-first search for a cycle in the
ordering graph (queue order plus counter edges), compared with the
library's Kahn-based check on random task graphs.

Pinned by hand-built schedules whose verdict is known by construction (a
safe one, a cross-queue deadlock, an unsatisfiable wait, a race, a partial
wait, a double write, a missing output, a self wait and a longer cycle) in
the soundness tests.
"""
from __future__ import annotations

import random
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

# operation codes of the task descriptor
QKV, ATTN, COMBINE, O, GATEUP, DOWN, LMHEAD, ARGMAX = range(1, 9)
INLINE = -1
MAX_WAITS = 4


@dataclass
class Task:
    op: int
    layer: int
    cu: int
    seq: int
    begin: int
    end: int
    aux: int
    waits: List[Tuple[int, int]]  # (counter, count)
    signal: int
    chain: int


@dataclass
class Shape:
    """The step's dimensions a schedule refers to."""
    H: int
    L: int
    nq: int
    nkv: int
    hd: int
    I: int
    V: int
    nsplit: int
    max_jobs: int
    npg: int  # QKV tasks per KV group (producers of a group's QKV counter)

    @property
    def group(self) -> int:
        return self.nq // self.nkv

    @property
    def half(self) -> int:
        return self.hd // 2

    @property
    def units(self) -> int:
        return (self.nq + 2 * self.nkv) * self.half

    @property
    def gunits(self) -> int:
        return (self.group + 2) * self.half


def from_descriptors(descs: Sequence) -> List[Task]:
    """Tasks from amk_task_t-like objects (fields op, layer, cu, seq, begin,
    end, aux, n_wait, wait_counter, wait_count, signal_counter,
    chain_counter).  n_wait values outside [0, MAX_WAITS] are kept as given
    (clipped for reading the arrays) so the structural label sees them."""
    out = []
    for d in descs:
        nw = int(d.n_wait)
        waits = [(int(d.wait_counter[i]), int(d.wait_count[i])) for i in range(max(0, min(nw, MAX_WAITS)))]
        t = Task(int(d.op), int(d.layer), int(d.cu), int(d.seq), int(d.begin), int(d.end), int(d.aux), waits,
                 int(d.signal_counter), int(d.chain_counter))
        t.n_wait_raw = nw
        out.append(t)
    return out


# ---------------------------------------------------------------- values a task reads and writes
# A value is (buffer name, element index range).  Buffers: x<i> residual
# stream i (x0: the embedding row, an input), q<l> (RoPE row-pair units of
# the queries), kv<l> (appended K then V row-pair units), part<l> (attention
# split records), o<l> (attention output), a<l>, logits, argp, next.

def _units_of_qkv(s: Shape, t: Task):
    """Query units and K/V units a QKV task writes (unit u of KV group g is
    head slot u // half of the group: its query heads, then K, then V)."""
    q, kv = [], []
    for u in range(t.begin, t.end):
        slot, i = divmod(u, s.half)
        g, r = divmod(slot, s.group + 2)
        if r < s.group:
            q.append((g * s.group + r) * s.half + i)
        elif r == s.group:
            kv.append(g * s.half + i)
        else:
            kv.append((s.nkv + g) * s.half + i)
    return q, kv


def _ranges(idx: List[int]):
    """Sorted indices -> half-open runs."""
    out = []
    for v in sorted(idx):
        if out and out[-1][1] == v:
            out[-1][1] = v + 1
        else:
            out.append([v, v + 1])
    return [tuple(r) for r in out]


def accesses(s: Shape, t: Task, n_lm: int):
    """(reads, writes): lists of (buffer, lo, hi)."""
    l = t.layer
    rd, wr = [], []
    if t.op == QKV:
        rd.append((f"x{2 * l}", 0, s.H))
        q, kv = _units_of_qkv(s, t)
        wr += [(f"q{l}", a, b) for a, b in _ranges(q)]
        wr += [(f"kv{l}", a, b) for a, b in _ranges(kv)]
    elif t.op == ATTN:
        g = t.aux
        rd.append((f"q{l}", g * s.group * s.half, (g + 1) * s.group * s.half))
        rd.append((f"kv{l}", g * s.half, (g + 1) * s.half))
        rd.append((f"kv{l}", (s.nkv + g) * s.half, (s.nkv + g + 1) * s.half))
        if t.cu == INLINE:
            wr.append((f"o{l}", g * s.group * s.hd, (g + 1) * s.group * s.hd))
        else:
            wr.append((f"part{l}", g * s.nsplit + t.begin, g * s.nsplit + t.begin + 1))
    elif t.op == COMBINE:
        g0, g1 = t.begin // s.group, (t.end - 1) // s.group + 1
        rd.append((f"part{l}", g0 * s.nsplit, g1 * s.nsplit))
        wr.append((f"o{l}", t.begin * s.hd, t.end * s.hd))
    elif t.op == O:
        if t.aux == 1:
            rd.append((f"q{l}", 0, s.nq * s.half))
            rd.append((f"kv{l}", 0, 2 * s.nkv * s.half))
        else:
            rd.append((f"o{l}", 0, s.nq * s.hd))
        rd.append((f"x{2 * l}", t.begin, t.end))
        wr.append((f"x{2 * l + 1}", t.begin, t.end))
    elif t.op == GATEUP:
        rd.append((f"x{2 * l + 1}", 0, s.H))
        wr.append((f"a{l}", t.begin, t.end))
    elif t.op == DOWN:
        rd.append((f"a{l}", 0, s.I))
        rd.append((f"x{2 * l + 1}", t.begin, t.end))
        wr.append((f"x{2 * l + 2}", t.begin, t.end))
    elif t.op == LMHEAD:
        rd.append((f"x{2 * s.L}", 0, s.H))
        wr.append(("logits", t.begin, t.end))
        wr.append(("argp", t.aux, t.aux + 1))
    elif t.op == ARGMAX:
        rd.append(("argp", t.begin, t.end))
        wr.append(("next", 0, 1))
    return rd, wr


def required_outputs(s: Shape, n_lm: int) -> Dict[str, int]:
    """Every value one step must produce exactly once: buffer -> size."""
    req = {f"x{i}": s.H for i in range(1, 2 * s.L + 1)}
    for l in range(s.L):
        req[f"q{l}"] = s.nq * s.half
        req[f"kv{l}"] = 2 * s.nkv * s.half
        req[f"o{l}"] = s.nq * s.hd
        req[f"a{l}"] = s.I
    req["logits"] = s.V
    req["argp"] = n_lm
    req["next"] = 1
    return req


# ---------------------------------------------------------------- structural label
def structural(s: Shape, tasks: List[Task], n_cu: int, n_counters: int) -> Optional[str]:
    """A reason the schedule is malformed, or None."""
    n_lm = sum(1 for t in tasks if t.op == LMHEAD)
    limits = {QKV: s.units, COMBINE: s.nq, O: s.H, DOWN: s.H, GATEUP: s.I, LMHEAD: s.V, ARGMAX: n_lm}
    rows = {QKV: 2, GATEUP: 2, O: 1, DOWN: 1, LMHEAD: 1}
    for i, t in enumerate(tasks):
        if not QKV <= t.op <= ARGMAX:
            return f"task {i}: op {t.op}"
        if t.cu != INLINE and not 0 <= t.cu < n_cu:
            return f"task {i}: queue {t.cu}"
        if getattr(t, "n_wait_raw", len(t.waits)) > MAX_WAITS or getattr(t, "n_wait_raw", 0) < 0:
            return f"task {i}: {t.n_wait_raw} waits"
        for c, k in t.waits:
            if not 0 <= c < n_counters:
                return f"task {i}: wait counter {c}"
        for c in (t.signal, t.chain):
            if not -1 <= c < n_counters:
                return f"task {i}: counter {c}"
        if t.op <= DOWN and not 0 <= t.layer < s.L:
            return f"task {i}: layer {t.layer}"
        if t.op == ATTN:
            if not 0 <= t.aux < s.nkv:
                return f"task {i}: KV head {t.aux}"
            if t.cu == INLINE and (t.begin, t.end) != (0, 1):
                return f"task {i}: inline attention range"
            if t.cu != INLINE and not (t.end == s.nsplit and 0 <= t.begin < s.nsplit):
                return f"task {i}: attention split"
        elif not (0 <= t.begin < t.end <= limits[t.op]):
            return f"task {i}: range [{t.begin}, {t.end}) beyond {limits[t.op]}"
        if t.op in rows and (t.end - t.begin) * rows[t.op] > s.max_jobs:
            return f"task {i}: {(t.end - t.begin) * rows[t.op]} rows over the cap {s.max_jobs}"
        if t.op == QKV and not (0 <= t.aux < s.nkv and t.begin // s.gunits == t.aux == (t.end - 1) // s.gunits):
            return f"task {i}: QKV units outside KV group {t.aux}"
        if t.op == O and t.aux not in (0, 1):
            return f"task {i}: O aux {t.aux}"
        if t.op == LMHEAD and not 0 <= t.aux < n_lm:
            return f"task {i}: argmax slot {t.aux}"
        if t.op == COMBINE and t.end - t.begin > 64:
            return f"task {i}: combine of {t.end - t.begin} heads"
    # queue positions 0..len-1, each once; inline tasks at position 0
    seen: Dict[int, set] = {}
    for i, t in enumerate(tasks):
        if t.cu == INLINE:
            if t.seq != 0 or t.op not in (ATTN, COMBINE):
                return f"task {i}: inline task"
            continue
        if t.seq in seen.setdefault(t.cu, set()):
            return f"task {i}: queue position repeated"
        seen[t.cu].add(t.seq)
    for c, ps in seen.items():
        if ps != set(range(len(ps))):
            return f"queue {c}: positions not contiguous"
    return None


# ---------------------------------------------------------------- dynamic label
def _inline_index(tasks: List[Task]) -> Dict[int, List[int]]:
    by_ctr: Dict[int, List[int]] = {}
    for i, t in enumerate(tasks):
        if t.cu == INLINE and len(t.waits) == 1:
            by_ctr.setdefault(t.waits[0][0], []).append(i)
    return by_ctr


# Element states of the simulated buffers: an input nobody writes, a value
# whose writer has not started, one being written, one written.
_INPUT, _PENDING, _RUNNING, _DONE = 0, 1, 2, 3


def _check_writes_once(acc) -> Optional[str]:
    """A value written by two tasks of the schedule, or None."""
    owner: Dict[str, Dict[int, int]] = {}
    for i, (_, wr) in enumerate(acc):
        for buf, lo, hi in wr:
            d = owner.setdefault(buf, {})
            for e in range(lo, hi):
                if e in d:
                    return f"{buf}[{e}] written by tasks {d[e]} and {i}"
                d[e] = i
    return None


def simulate(s: Shape, tasks: List[Task], n_cu: int, n_counters: int, rng: random.Random,
             eager: float = 0.0) -> Optional[str]:
    """One random execution; a reason it went wrong, or None.  Each step picks
    one enabled action (start a queue's ready head task, or finish a running
    task) uniformly.  With `eager` > 0 the run is adversarial: a random third
    of the tasks are slow (they finish only when nothing else can happen),
    and with probability `eager` a step picks among the starts only, when
    there are any; consumers then start as early as their waits allow while
    some producers are still running, which exposes a too-weak wait in fewer
    runs.  Every execution sampled either way is one the device can perform."""
    n_lm = sum(1 for t in tasks if t.op == LMHEAD)
    queues: Dict[int, List[int]] = {}
    for i, t in enumerate(tasks):
        if t.cu != INLINE:
            queues.setdefault(t.cu, []).append(i)
    for q in queues.values():
        q.sort(key=lambda i: tasks[i].seq)
    inline_of = _inline_index(tasks)
    acc = [accesses(s, t, n_lm) for t in tasks]
    err = _check_writes_once(acc)
    if err:
        return err
    # every buffer a task touches, sized to the largest index touched, each
    # element INPUT until some task is found to write it (then PENDING)
    size: Dict[str, int] = {}
    for rd, wr in acc:
        for buf, lo, hi in rd + wr:
            size[buf] = max(size.get(buf, 0), hi)
    state = {buf: bytearray(n) for buf, n in size.items()}
    for _, wr in acc:
        for buf, lo, hi in wr:
            state[buf][lo:hi] = bytes([_PENDING]) * (hi - lo)
    counters = [0] * n_counters
    head = {c: 0 for c in queues}
    running: Dict[int, int] = {}  # queue -> task running on it
    done = [False] * len(tasks)
    inline_run = set()
    slow = set(rng.sample(range(len(tasks)), len(tasks) // 3)) if eager else set()

    def ready(i):
        return all(counters[c] >= k for c, k in tasks[i].waits)

    def start_reads(i):
        for buf, lo, hi in acc[i][0]:
            st = state[buf]
            for bad, what in ((_RUNNING, "while its writer runs"), (_PENDING, "before it is written")):
                e = st.find(bad, lo, hi)
                if e >= 0:
                    return f"task {i} reads {buf}[{e}] {what}"
        return None

    def set_writes(i, val):
        for buf, lo, hi in acc[i][1]:
            state[buf][lo:hi] = bytes([val]) * (hi - lo)

    def finish(i):
        set_writes(i, _DONE)
        done[i] = True
        t = tasks[i]
        if t.signal >= 0:
            counters[t.signal] += 1
            # the device: the producer whose increment brings its counter to the
            # producer count it assumes (QKV tasks of a KV group, or the
            # attention splits of one) runs the inline task waiting on that
            # counter, then increments its own chain counter
            expected = s.npg if t.op == QKV else s.nsplit
            if t.chain >= 0 and counters[t.signal] == expected:
                for j in inline_of.get(t.signal, []):
                    if j in inline_run:
                        continue
                    inline_run.add(j)
                    err = start_reads(j)
                    if err:
                        return err
                    set_writes(j, _DONE)
                    done[j] = True
                counters[t.chain] += 1
        return None

    while True:
        actions = []
        for c, h in head.items():
            if c in running:
                actions.append(("finish", c))
            elif h < len(queues[c]) and ready(queues[c][h]):
                actions.append(("start", c))
        if not actions:
            break
        if slow:
            fast = [a for a in actions if a[0] == "start" or running[a[1]] not in slow]
            actions = fast or actions
        starts = [a for a in actions if a[0] == "start"]
        if starts and eager and rng.random() < eager:
            actions = starts
        kind, c = rng.choice(actions)
        if kind == "start":
            i = queues[c][head[c]]
            err = start_reads(i)
            if err:
                return err
            set_writes(i, _RUNNING)
            running[c] = i
        else:
            i = running.pop(c)
            head[c] += 1
            err = finish(i)
            if err:
                return err
    left = [i for i, d in enumerate(done) if not d]
    if left:
        return f"deadlock: {len(left)} tasks never ran (first {left[0]})"
    req = required_outputs(s, n_lm)
    read_bufs = {buf for rd, _ in acc for buf, _, _ in rd}
    for l in range(s.L):
        if f"o{l}" not in read_bufs:  # the tiny schedule computes attention inside the O tasks
            req.pop(f"o{l}", None)
    for buf, n in req.items():
        st = state.get(buf, bytearray())
        have = st[:n].count(_DONE) if len(st) >= n else st.count(_DONE)
        if len(st) != n or have != n:
            return f"{buf}: {have} of {n} values written"
    return None


def find_cycle(tasks: List[Task]) -> Optional[List[int]]:
    """A cycle of the schedule's ordering graph (task indices), or None.

    Edges: each queued task to the next one on its queue, and every task
    that signals a counter to every task waiting on that counter (a wait
    completes only after all of the counter's producers ran).  Iterative
    depth-first search with three colours; independent of the library's
    Kahn-based check."""
    n = len(tasks)
    succ: List[List[int]] = [[] for _ in range(n)]
    by_queue: Dict[int, List[int]] = {}
    for i, t in enumerate(tasks):
        if t.cu != INLINE:
            by_queue.setdefault(t.cu, []).append(i)
    for q in by_queue.values():
        q.sort(key=lambda i: tasks[i].seq)
        for a, b in zip(q, q[1:]):
            succ[a].append(b)
    prod: Dict[int, List[int]] = {}
    for i, t in enumerate(tasks):
        if t.signal >= 0:
            prod.setdefault(t.signal, []).append(i)
    for i, t in enumerate(tasks):
        for c, _ in t.waits:
            for p in prod.get(c, []):
                succ[p].append(i)
    WHITE, GREY, BLACK = 0, 1, 2
    colour = [WHITE] * n
    parent = [-1] * n
    for root in range(n):
        if colour[root] != WHITE:
            continue
        stack = [(root, 0)]
        colour[root] = GREY
        while stack:
            v, k = stack[-1]
            if k < len(succ[v]):
                stack[-1] = (v, k + 1)
                w = succ[v][k]
                if colour[w] == WHITE:
                    colour[w] = GREY
                    parent[w] = v
                    stack.append((w, 0))
                elif colour[w] == GREY:
                    cyc = [w]
                    u = v
                    while u != w:
                        cyc.append(u)
                        u = parent[u]
                    return cyc[::-1]
            else:
                colour[v] = BLACK
                stack.pop()
    return None


def label(s: Shape, tasks: List[Task], n_cu: int, n_counters: int, runs: int = 8, seed: int = 0) -> Optional[str]:
    """None if the schedule is safe as far as this oracle can tell, else why not."""
    why = structural(s, tasks, n_cu, n_counters)
    if why:
        return why
    rng = random.Random(seed)
    for r in range(runs):
        # alternate uniform interleavings with eager-start ones
        why = simulate(s, tasks, n_cu, n_counters, rng, eager=0.9 if r % 2 else 0.0)
        if why:
            return why
    return None
