"""Soundness of the static schedule check against an independent oracle
(paper §5, Table "Validator soundness"): single-injection mutants of the
eight unsafe classes the paper uses, plus random multi-field mutations,
are labelled by oracle/schedule_sim.py, which executes a schedule on a model
of the device under random interleavings and never calls the checker.  No
schedule the oracle finds unsafe may be accepted (zero false accepts), and
every real lowering must be accepted and found safe.  CPU only."""
import ctypes
import random

import pytest

import synth
from oracle import schedule_sim as sim
from paper_2606_09682_amd import amk

N_CU = 16


@pytest.fixture(scope="module")
def lib():
    import os
    if not os.path.exists(amk.LIB_PATH):
        from paper_2606_09682_amd import build
        build.build()
    return amk.load()


def cfg_of(name):
    c = synth.get(name)
    return amk.make_config(c.hidden, c.n_layers, c.n_heads, c.n_kv_heads, c.head_dim, c.intermediate, c.vocab,
                           c.seq_capacity, c.rope_theta, c.rms_eps, c.tied_embeddings, "bf16")


def shape_of(name, tasks):
    c = synth.get(name)
    splits = [t for t in tasks if t.op == amk.AMK_OP_ATTN and t.cu != amk.AMK_CU_INLINE]
    nsplit = splits[0].end if splits else max(1, min(64, N_CU // c.n_kv_heads))
    npg = sum(1 for t in tasks if t.op == amk.AMK_OP_QKV and t.layer == 0 and t.aux == 0)
    return sim.Shape(c.hidden, c.n_layers, c.n_heads, c.n_kv_heads, c.head_dim, c.intermediate, c.vocab, nsplit,
                     1024, npg)


def clone(tasks):
    arr = (amk.amk_task_t * len(tasks))()
    ctypes.memmove(arr, tasks, ctypes.sizeof(amk.amk_task_t) * len(tasks))
    return arr


def checker_accepts(cfg, tasks, nc, n_cu=N_CU):
    return amk.amk_schedule_check(cfg, n_cu, tasks, nc).ok == 1


VARIANTS = [amk.AMK_SCHEDULE_SHORT, amk.AMK_SCHEDULE_LONG, amk.AMK_SCHEDULE_TINY]


@pytest.mark.parametrize("name", ["tiny", "smollm2_135m"])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("n_cu", [16, 13])
@pytest.mark.parametrize("assign", [amk.AMK_ASSIGN_ROUND_ROBIN, amk.AMK_ASSIGN_LPT])
def test_real_lowerings_safe_and_accepted(lib, name, variant, n_cu, assign):
    cfg = cfg_of(name)
    tuning = amk.amk_tuning_t()
    tuning.queue_assign = assign
    tasks, nc = amk.amk_schedule_export(cfg, n_cu, tuning, variant=variant)
    s = shape_of(name, tasks)
    s.nsplit = max(1, min(64, n_cu // synth.get(name).n_kv_heads))
    assert sim.label(s, sim.from_descriptors(tasks), n_cu, nc, runs=4) is None
    assert sim.find_cycle(sim.from_descriptors(tasks)) is None
    assert checker_accepts(cfg, tasks, nc, n_cu)


# ---------------------------------------------------------------- the oracle's own labels
# Hand-built schedules of a one-layer micro decoder whose verdict is known by
# construction pin what oracle/schedule_sim.label reports: a safe schedule,
# a deadlock, a read racing its writer, a value written twice, an output
# never written, and a wait that counts too few producers.
MICRO = sim.Shape(H=4, L=1, nq=1, nkv=1, hd=4, I=4, V=4, nsplit=1, max_jobs=1024, npg=1)
MICRO_UNITS = MICRO.units  # 6 QKV row-pair units: 2 query, 2 key, 2 value


def micro_tasks():
    """The tiny-style step on two queues: QKV -> O (attention inside) ->
    gate/up -> down -> LM head -> argmax, alternating queues, one counter per
    stage (c0 .. c4)."""
    T = sim.Task
    return [
        T(sim.QKV, 0, 0, 0, 0, MICRO_UNITS, 0, [], 0, -1),
        T(sim.O, 0, 1, 0, 0, 4, 1, [(0, 1)], 1, -1),
        T(sim.GATEUP, 0, 0, 1, 0, 4, 0, [(1, 1)], 2, -1),
        T(sim.DOWN, 0, 1, 1, 0, 4, 0, [(2, 1)], 3, -1),
        T(sim.LMHEAD, 0, 0, 2, 0, 4, 0, [(3, 1)], 4, -1),
        T(sim.ARGMAX, 0, 1, 2, 0, 1, 0, [(4, 1)], -1, -1),
    ]


def micro_label(tasks, n_counters=5, runs=32):
    return sim.label(MICRO, tasks, 2, n_counters, runs=runs, seed=7)


def test_oracle_label_safe_schedule():
    assert micro_label(micro_tasks()) is None
    assert sim.find_cycle(micro_tasks()) is None


def test_oracle_label_cross_queue_deadlock():
    t = micro_tasks()
    t[0].waits = [(1, 1)]  # QKV waits for O, which waits for QKV: two queues block each other
    why = micro_label(t)
    assert why is not None and why.startswith("deadlock"), why
    assert set(sim.find_cycle(t)) == {0, 1}


def test_oracle_label_unsatisfiable_wait_deadlocks():
    t = micro_tasks()
    t[1].waits = [(0, 2)]  # two signals expected, one producer
    why = micro_label(t)
    assert why is not None and why.startswith("deadlock"), why


def test_oracle_label_race():
    t = micro_tasks()
    t[1].waits = []  # O reads q / K / V with no order after the QKV task that writes them
    why = micro_label(t)
    assert why is not None and " reads q0[" in why or " reads kv0[" in why, why


def test_oracle_label_partial_wait_races():
    t = micro_tasks()
    # QKV split over both queues: two producers of c0; O waits for one of them
    t[0].end = 3
    t.insert(1, sim.Task(sim.QKV, 0, 1, 0, 3, MICRO_UNITS, 0, [], 0, -1))
    for x in t[2:]:
        if x.cu == 1:
            x.seq += 1
    assert t[2].op == sim.O and t[2].waits == [(0, 1)]
    why = micro_label(t)
    assert why is not None and " reads " in why, why
    t[2].waits = [(0, 2)]  # the all-join fixes it
    assert micro_label(t) is None


def test_oracle_label_double_write():
    t = micro_tasks()
    t.append(sim.Task(sim.DOWN, 0, 0, 3, 2, 4, 0, [(2, 1)], -1, -1))  # x2[2:4] written again
    why = micro_label(t)
    assert why is not None and "x2[2] written by tasks 3 and 6" in why, why


def test_oracle_label_missing_output():
    t = micro_tasks()
    t[2].end = 3  # a0[3] is never written (down still reads it as an input value)
    why = micro_label(t)
    assert why == "a0: 3 of 4 values written", why


def test_oracle_label_self_wait_and_long_cycle():
    t = micro_tasks()
    t[2].waits = [(1, 1), (2, 1)]  # gate/up waits for its own signal
    assert micro_label(t).startswith("deadlock")
    assert sim.find_cycle(t) == [2]
    t = micro_tasks()
    t[0].waits = [(3, 1)]  # QKV waits for down, which runs after gate/up, queued after QKV
    assert micro_label(t).startswith("deadlock")
    c = sim.find_cycle(t)
    k = c.index(min(c))
    assert c[k:] + c[:k] == [0, 2, 3]  # queue edge 0 -> 2, counters c2: 2 -> 3, c3: 3 -> 0


# ---------------------------------------------------------------- mutant classes
def producers(tasks, c):
    return [i for i, t in enumerate(tasks) if t.signal_counter == c]


def add_or_replace_wait(t, c, count, rng):
    """Append the wait (c, count) to task t, or overwrite a random one of its
    wait slots when all AMK_MAX_WAITS are in use."""
    k = t.n_wait if t.n_wait < amk.AMK_MAX_WAITS else rng.randrange(amk.AMK_MAX_WAITS)
    t.wait_counter[k] = c
    t.wait_count[k] = count
    t.n_wait = max(t.n_wait, k + 1)


def mutate(kind, tasks, nc, rng):
    """One single-injection mutant of class `kind` (paper Table "Validator
    soundness"), or None if this schedule offers no site for it."""
    m = clone(tasks)
    queued = [i for i, t in enumerate(m) if t.cu != amk.AMK_CU_INLINE]
    if kind == "cycle":
        # a task waits on a counter signalled by a task later on its own queue
        cand = [i for i in queued if any(m[j].cu == m[i].cu and m[j].seq > m[i].seq and m[j].signal_counter >= 0
                                          for j in queued)]
        i = rng.choice(cand)
        later = [j for j in queued if m[j].cu == m[i].cu and m[j].seq > m[i].seq and m[j].signal_counter >= 0]
        c = m[rng.choice(later)].signal_counter
        add_or_replace_wait(m[i], c, len(producers(m, c)), rng)
    elif kind == "drop_wait":
        cand = [i for i in queued if m[i].n_wait > 0]
        i = rng.choice(cand)
        m[i].n_wait = 0
    elif kind == "kv_before_append":
        # a task reading the KV cache no longer waits for this step's append:
        # queued attention splits / tiny-schedule O tasks drop their wait; the
        # short schedule's inline attention of group g is run after another
        # group's QKV tasks instead of its own
        cand = [i for i, t in enumerate(m) if t.cu != amk.AMK_CU_INLINE and t.n_wait > 0 and
                (t.op == amk.AMK_OP_ATTN or (t.op == amk.AMK_OP_O and t.aux == 1))]
        inl = [i for i, t in enumerate(m) if t.cu == amk.AMK_CU_INLINE and t.op == amk.AMK_OP_ATTN]
        if cand:
            m[rng.choice(cand)].n_wait = 0
        elif inl:
            i = rng.choice(inl)
            others = [j for j in inl if m[j].layer == m[i].layer and m[j].aux != m[i].aux]
            if not others:
                return None
            m[i].wait_counter[0] = m[rng.choice(others)].wait_counter[0]
        else:
            return None
    elif kind == "self_wait":
        cand = [i for i in queued if m[i].signal_counter >= 0]
        i = rng.choice(cand)
        add_or_replace_wait(m[i], m[i].signal_counter, len(producers(m, m[i].signal_counter)), rng)
    elif kind == "oob_counter":
        i = rng.choice(queued)
        if m[i].n_wait > 0 and rng.random() < 0.5:
            m[i].wait_counter[0] = nc + rng.randrange(1, 100)
        else:
            m[i].signal_counter = nc + rng.randrange(0, 100)
    elif kind == "oob_buffer":
        cand = [i for i in queued if m[i].op != amk.AMK_OP_ATTN]
        i = rng.choice(cand)
        m[i].end += rng.randrange(1, 5000)
    elif kind == "capacity_overflow":
        i = rng.choice(queued)
        if rng.random() < 0.5:
            m[i].n_wait = amk.AMK_MAX_WAITS + rng.randrange(1, 50)
        else:
            m[i].end = m[i].begin + 1025
    elif kind == "partial_shared":
        # a wait that counts fewer producers than the counter has
        cand = [(i, w) for i in queued for w in range(m[i].n_wait) if m[i].wait_count[w] > 1]
        if not cand:
            return None
        i, w = rng.choice(cand)
        m[i].wait_count[w] = 1 if rng.random() < 0.5 else rng.randrange(1, m[i].wait_count[w])
    return m


CLASSES = ["cycle", "drop_wait", "kv_before_append", "self_wait", "oob_counter", "oob_buffer",
           "capacity_overflow", "partial_shared"]


MUTANTS_PER_CLASS = 64
MIN_UNSAFE = 50


@pytest.mark.parametrize("variant", VARIANTS)
def test_no_false_accepts_on_mutants(lib, variant):
    """Every class yields at least MIN_UNSAFE mutants the oracle finds unsafe
    in every schedule variant, and the checker rejects each of them."""
    cfg = cfg_of("tiny")
    tasks, nc = amk.amk_schedule_export(cfg, N_CU, variant=variant)
    s = shape_of("tiny", tasks)
    rng = random.Random(1234 + variant)
    table = {}
    for kind in CLASSES:
        unsafe = rejected = false_accept = 0
        for k in range(MUTANTS_PER_CLASS):
            m = mutate(kind, tasks, nc, rng)
            if m is None:
                continue
            why = sim.label(s, sim.from_descriptors(m), N_CU, nc, runs=16, seed=k)
            acc = checker_accepts(cfg, m, nc)
            if why is not None:
                unsafe += 1
                rejected += not acc
                false_accept += acc
        table[kind] = (unsafe, rejected, false_accept)
        assert false_accept == 0, (kind, table[kind])
    print(f"\nvariant {variant}: class -> (oracle unsafe, rejected, false accepts): {table}")
    for kind, (unsafe, rejected, _) in table.items():
        assert unsafe >= MIN_UNSAFE and rejected == unsafe, (kind, table[kind])


def test_no_false_accepts_on_random_mutations(lib):
    """Several random field changes at once (the random-graph population)."""
    cfg = cfg_of("tiny")
    fields = ["begin", "end", "aux", "n_wait", "signal_counter", "chain_counter", "seq", "cu", "layer", "op"]
    unsafe = accepted_safe = 0
    for variant in VARIANTS:
        tasks, nc = amk.amk_schedule_export(cfg, N_CU, variant=variant)
        s = shape_of("tiny", tasks)
        rng = random.Random(99 + variant)
        for k in range(25):
            m = clone(tasks)
            for _ in range(rng.randrange(1, 4)):
                t = m[rng.randrange(len(m))]
                f = rng.choice(fields)
                setattr(t, f, getattr(t, f) + rng.choice([-2, -1, 1, 2]))
            why = sim.label(s, sim.from_descriptors(m), N_CU, nc, runs=16, seed=k)
            acc = checker_accepts(cfg, m, nc)
            if why is not None:
                unsafe += 1
                assert not acc, f"false accept: {why}"
            elif acc:
                accepted_safe += 1
    assert unsafe > 0


# ---------------------------------------------------------------- random task graphs
# The micro decoder (hidden 64, 2 layers, 2 query heads on 1 KV head, head
# dim 64, SwiGLU 64, vocab 64): a lowering has 28 to 69 tasks, small enough to
# check thousands of random graphs built from it.
MICRO_CFG = dict(hidden=64, n_layers=2, n_heads=2, n_kv_heads=1, head_dim=64, intermediate=64, vocab=64,
                 max_seq=16, rope_theta=10000.0)


def micro_cfg():
    return amk.make_config(**MICRO_CFG)


def micro_shape(tasks, n_cu):
    splits = [t for t in tasks if t.op == amk.AMK_OP_ATTN and t.cu != amk.AMK_CU_INLINE]
    nsplit = splits[0].end if splits else max(1, min(64, n_cu))
    npg = sum(1 for t in tasks if t.op == amk.AMK_OP_QKV and t.layer == 0 and t.aux == 0)
    return sim.Shape(64, 2, 2, 1, 64, 64, 64, nsplit, 1024, npg)


def random_graph(tasks, nc, rng, n_queues):
    """A random task graph over the tasks of a real lowering: a random order
    consistent with the counter edges, dealt onto n_queues queues at random;
    then, at random, adjacent tasks of a queue swapped and extra all-join waits
    added, either of which may close a cycle."""
    m = clone(tasks)
    n = len(m)
    prod = {}
    for i, t in enumerate(m):
        if t.signal_counter >= 0:
            prod.setdefault(t.signal_counter, []).append(i)
    need = [sum(len(prod.get(t.wait_counter[w], [])) for w in range(t.n_wait)) for t in m]
    succ = [[] for _ in range(n)]
    for i, t in enumerate(m):
        for w in range(t.n_wait):
            for p in prod.get(t.wait_counter[w], []):
                succ[p].append(i)
    ready = [i for i in range(n) if need[i] == 0]
    order = []
    while ready:
        i = ready.pop(rng.randrange(len(ready)))
        order.append(i)
        for j in succ[i]:
            need[j] -= 1
            if need[j] == 0:
                ready.append(j)
    assert len(order) == n
    queues = [[] for _ in range(n_queues)]
    for i in order:
        if m[i].cu != amk.AMK_CU_INLINE:
            queues[rng.randrange(n_queues)].append(i)
    perturb = rng.random() < 0.5  # half the graphs stay in a consistent order
    for _ in range(rng.choice([1, 1, 2]) if perturb else 0):
        q = rng.choice(queues)
        if len(q) > 1:
            k = rng.randrange(len(q) - 1)
            q[k], q[k + 1] = q[k + 1], q[k]
    for c, q in enumerate(queues):
        for k, i in enumerate(q):
            m[i].cu, m[i].seq = c, k
    for _ in range(rng.choice([0, 1]) if perturb else 0):
        i = rng.randrange(n)
        if m[i].cu == amk.AMK_CU_INLINE or m[i].n_wait >= amk.AMK_MAX_WAITS:
            continue
        c = rng.choice(sorted(prod))
        m[i].wait_counter[m[i].n_wait] = c
        m[i].wait_count[m[i].n_wait] = len(prod[c])
        m[i].n_wait += 1
    return m


def test_random_graphs_kahn_dfs_and_oracle_agree(lib):
    """Several thousand random graphs: the library's Kahn-based acyclicity
    check and the oracle's depth-first search agree on every graph; a cyclic
    graph deadlocks in the oracle's execution and is rejected; an acyclic one
    is accepted and safe; nothing the oracle finds unsafe is accepted."""
    cfg = micro_cfg()
    rng = random.Random(2024)
    seen = {"cyclic": 0, "acyclic": 0}
    n_graphs = 0
    for variant in VARIANTS:
        for n_queues in (3, 4, 5, 6):
            tasks, nc = amk.amk_schedule_export(cfg, n_queues, variant=variant)
            s = micro_shape(tasks, n_queues)
            for k in range(250):
                m = random_graph(tasks, nc, rng, n_queues)
                rep = amk.amk_schedule_check(cfg, n_queues, m, nc)
                ts = sim.from_descriptors(m)
                cyc = sim.find_cycle(ts)
                why = sim.label(s, ts, n_queues, nc, runs=2, seed=k)
                n_graphs += 1
                if cyc is not None:
                    seen["cyclic"] += 1
                    assert rep.ok == 0 and rep.rule in (amk.AMK_CHECK_ACYCLIC, amk.AMK_CHECK_QUEUE_ORDER), \
                        (variant, n_queues, k, rep.rule, rep.message)
                    assert why is not None and why.startswith("deadlock"), why
                else:
                    seen["acyclic"] += 1
                    assert rep.ok == 1, (variant, n_queues, k, rep.rule, rep.message)
                    assert why is None, why
    print(f"\n{n_graphs} random graphs: {seen}")
    assert n_graphs >= 3000 and min(seen.values()) >= 500
