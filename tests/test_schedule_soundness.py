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
def test_real_lowerings_safe_and_accepted(lib, name, variant, n_cu):
    cfg = cfg_of(name)
    tasks, nc = amk.amk_schedule_export(cfg, n_cu, variant=variant)
    s = shape_of(name, tasks)
    s.nsplit = max(1, min(64, n_cu // synth.get(name).n_kv_heads))
    assert sim.label(s, sim.from_descriptors(tasks), n_cu, nc, runs=4) is None
    assert checker_accepts(cfg, tasks, nc, n_cu)


# ---------------------------------------------------------------- mutant classes
def producers(tasks, c):
    return [i for i, t in enumerate(tasks) if t.signal_counter == c]


def mutate(kind, tasks, nc, rng):
    """One single-injection mutant of class `kind` (paper Table "Validator
    soundness"), or None if this schedule offers no site for it."""
    m = clone(tasks)
    queued = [i for i, t in enumerate(m) if t.cu != amk.AMK_CU_INLINE]
    if kind == "cycle":
        # a task waits on a counter signalled only by tasks later on its own queue
        i = rng.choice(queued)
        later = [j for j in queued if m[j].cu == m[i].cu and m[j].seq > m[i].seq and m[j].signal_counter >= 0]
        if not later or m[i].n_wait >= amk.AMK_MAX_WAITS:
            return None
        c = m[rng.choice(later)].signal_counter
        m[i].wait_counter[m[i].n_wait] = c
        m[i].wait_count[m[i].n_wait] = len(producers(m, c))
        m[i].n_wait += 1
    elif kind == "drop_wait":
        cand = [i for i in queued if m[i].n_wait > 0]
        i = rng.choice(cand)
        m[i].n_wait = 0
    elif kind == "kv_before_append":
        cand = [i for i, t in enumerate(m) if t.cu != amk.AMK_CU_INLINE and t.n_wait > 0 and
                (t.op == amk.AMK_OP_ATTN or (t.op == amk.AMK_OP_O and t.aux == 1))]
        if not cand:
            return None
        m[rng.choice(cand)].n_wait = 0
    elif kind == "self_wait":
        cand = [i for i in queued if m[i].signal_counter >= 0 and m[i].n_wait < amk.AMK_MAX_WAITS]
        i = rng.choice(cand)
        m[i].wait_counter[m[i].n_wait] = m[i].signal_counter
        m[i].wait_count[m[i].n_wait] = len(producers(m, m[i].signal_counter))
        m[i].n_wait += 1
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
        cand = [i for i in queued if m[i].n_wait > 0 and m[i].wait_count[0] > 1]
        if not cand:
            return None
        i = rng.choice(cand)
        m[i].wait_count[0] = rng.randrange(1, m[i].wait_count[0])
    return m


CLASSES = ["cycle", "drop_wait", "kv_before_append", "self_wait", "oob_counter", "oob_buffer",
           "capacity_overflow", "partial_shared"]


@pytest.mark.parametrize("variant", VARIANTS)
def test_no_false_accepts_on_mutants(lib, variant):
    cfg = cfg_of("tiny")
    tasks, nc = amk.amk_schedule_export(cfg, N_CU, variant=variant)
    s = shape_of("tiny", tasks)
    rng = random.Random(1234 + variant)
    table = {}
    for kind in CLASSES:
        unsafe = rejected = false_accept = 0
        for k in range(12):
            m = mutate(kind, tasks, nc, rng)
            if m is None:
                continue
            why = sim.label(s, sim.from_descriptors(m), N_CU, nc, runs=4, seed=k)
            acc = checker_accepts(cfg, m, nc)
            if why is not None:
                unsafe += 1
                rejected += not acc
                false_accept += acc
        table[kind] = (unsafe, rejected, false_accept)
        assert false_accept == 0, (kind, table[kind])
    print(f"\nvariant {variant}: class -> (oracle unsafe, rejected, false accepts): {table}")
    # the structural classes are always unsafe and always caught
    for kind in ("oob_counter", "oob_buffer", "capacity_overflow"):
        assert table[kind][0] == table[kind][1] > 0


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
            why = sim.label(s, sim.from_descriptors(m), N_CU, nc, runs=4, seed=k)
            acc = checker_accepts(cfg, m, nc)
            if why is not None:
                unsafe += 1
                assert not acc, f"false accept: {why}"
            elif acc:
                accepted_safe += 1
    assert unsafe > 0
