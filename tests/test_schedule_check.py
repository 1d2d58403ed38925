"""The static schedule check (paper §4, Table tab:checks) on real lowerings and
on single-injection mutants of the unsafe classes the paper's soundness study
uses (Table tab:soundness), plus a cross-queue deadlock that per-queue order
checks alone would miss.  CPU only."""
import ctypes
import random

import pytest

import synth
from paper_2606_09682_amd import amk


@pytest.fixture(scope="module")
def lib():
    import os
    if not os.path.exists(amk.LIB_PATH):
        from paper_2606_09682_amd import build
        build.build()
    return amk.load()


def cfg_of(name, fmt="bf16"):
    c = synth.get(name)
    return amk.make_config(c.hidden, c.n_layers, c.n_heads, c.n_kv_heads, c.head_dim, c.intermediate, c.vocab,
                           c.seq_capacity, c.rope_theta, c.rms_eps, c.tied_embeddings, fmt)


N_CU = 16


@pytest.fixture(scope="module")
def tiny_sched(lib):
    cfg = cfg_of("tiny")
    tasks, nc = amk.amk_schedule_export(cfg, N_CU)
    return cfg, tasks, nc


def clone(tasks):
    arr = (amk.amk_task_t * len(tasks))()
    ctypes.memmove(arr, tasks, ctypes.sizeof(arr))
    return arr


def check(cfg, tasks, nc, n_cu=N_CU):
    return amk.amk_schedule_check(cfg, n_cu, tasks, nc)


def find(tasks, op, layer=None, pred=None):
    for i, t in enumerate(tasks):
        if t.op == op and (layer is None or t.layer == layer) and (pred is None or pred(t)):
            return i
    raise LookupError


def producers(tasks, c):
    return [i for i, t in enumerate(tasks) if t.signal_counter == c]


@pytest.mark.parametrize("name", list(synth.CONFIGS))
@pytest.mark.parametrize("n_cu", [256, 13])
@pytest.mark.parametrize("variant", [amk.AMK_SCHEDULE_SHORT, amk.AMK_SCHEDULE_LONG, amk.AMK_SCHEDULE_TINY])
def test_real_lowering_accepted(lib, name, n_cu, variant):
    cfg = cfg_of(name, "w8a16")
    tasks, nc = amk.amk_schedule_export(cfg, n_cu, variant=variant)
    rep = check(cfg, tasks, nc, n_cu)
    assert rep.ok == 1, rep.message
    # one queue per CU, every queue used, seq contiguous; inline tasks sit on no queue
    seen = {}
    for t in tasks:
        if t.cu == amk.AMK_CU_INLINE:
            assert variant != amk.AMK_SCHEDULE_TINY
            assert t.op == (amk.AMK_OP_ATTN if variant == amk.AMK_SCHEDULE_SHORT else amk.AMK_OP_COMBINE)
            continue
        seen.setdefault(t.cu, []).append(t.seq)
    assert sorted(seen) == list(range(n_cu))
    for c, seqs in seen.items():
        assert sorted(seqs) == list(range(len(seqs)))
    # each schedule runs on a kernel that carries only its own attention code:
    # the tiny one has no attention tasks, merges or chained inline tasks and
    # computes the attention in every O task (aux 1); the other one in none
    tiny = variant == amk.AMK_SCHEDULE_TINY
    for t in tasks:
        if tiny:
            assert t.op not in (amk.AMK_OP_ATTN, amk.AMK_OP_COMBINE) and t.chain_counter == -1
        if t.op == amk.AMK_OP_O:
            assert t.aux == (1 if tiny else 0)


def test_schedule_shape_8b(lib):
    cfg = cfg_of("llama3_8b")
    tasks, nc = amk.amk_schedule_export(cfg, 256)
    ops = [t.op for t in tasks]
    L = 32
    assert ops.count(amk.AMK_OP_QKV) == 256 * L
    assert ops.count(amk.AMK_OP_ATTN) == 8 * 32 * L
    assert ops.count(amk.AMK_OP_O) == 256 * L
    assert ops.count(amk.AMK_OP_GATEUP) == 256 * L
    assert ops.count(amk.AMK_OP_DOWN) == 256 * L
    assert ops.count(amk.AMK_OP_LMHEAD) == 256
    assert ops.count(amk.AMK_OP_ARGMAX) == 1
    # one inline combine per (layer, KV head), fed by that head's 32 splits
    comb = [t for t in tasks if t.op == amk.AMK_OP_COMBINE]
    assert len(comb) == 8 * L and all(t.cu == amk.AMK_CU_INLINE for t in comb)
    assert all(t.wait_count[0] == 32 for t in comb)
    # every QKV task owns whole RoPE row pairs: 48 heads * 64 pairs / 256 = 12 units each,
    # 32 tasks per KV group of (4 + 2) heads * 64 pairs
    qkv = [t for t in tasks if t.op == amk.AMK_OP_QKV]
    assert {t.end - t.begin for t in qkv} == {12}
    assert all(t.begin // 384 == t.aux == (t.end - 1) // 384 for t in qkv)
    assert all(t.chain_counter == -1 for t in qkv)


def test_schedule_shape_8b_short(lib):
    cfg = cfg_of("llama3_8b")
    tasks, nc = amk.amk_schedule_export(cfg, 256, variant=amk.AMK_SCHEDULE_SHORT)
    assert check(cfg, tasks, nc, 256).ok
    L = 32
    queued_attn = [t for t in tasks if t.op == amk.AMK_OP_ATTN and t.cu != amk.AMK_CU_INLINE]
    inline_attn = [t for t in tasks if t.op == amk.AMK_OP_ATTN and t.cu == amk.AMK_CU_INLINE]
    assert not queued_attn and not [t for t in tasks if t.op == amk.AMK_OP_COMBINE]
    assert len(inline_attn) == 8 * L
    assert all(t.wait_count[0] == 32 and (t.begin, t.end) == (0, 1) for t in inline_attn)
    # each QKV task chains to its layer's attention-output counter, which O waits on
    qkv = [t for t in tasks if t.op == amk.AMK_OP_QKV]
    assert len(qkv) == 256 * L
    for t in qkv:
        assert t.chain_counter >= 0
        group_inline = [a for a in inline_attn if a.layer == t.layer and a.aux == t.aux]
        assert len(group_inline) == 1 and group_inline[0].signal_counter == t.chain_counter
        assert group_inline[0].wait_counter[0] == t.signal_counter
    o = [t for t in tasks if t.op == amk.AMK_OP_O and t.layer == 5]
    assert {t.wait_counter[0] for t in o} == {a.signal_counter for a in inline_attn if a.layer == 5}
    assert all(t.wait_count[0] == 8 for t in o)
    # one queue per CU: four GEMV tasks per layer on every CU, nothing else
    per_cu = {}
    for t in tasks:
        if t.cu != amk.AMK_CU_INLINE and t.op in (amk.AMK_OP_QKV, amk.AMK_OP_O, amk.AMK_OP_GATEUP, amk.AMK_OP_DOWN):
            per_cu[t.cu] = per_cu.get(t.cu, 0) + 1
    assert set(per_cu.values()) == {4 * L}


# ------------------------------------------------------------------ mutants
def test_cycle_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_QKV, 0)
    j = find(m, amk.AMK_OP_DOWN, 1)
    c = m[j].signal_counter
    t = m[i]
    t.wait_counter[t.n_wait] = c
    t.wait_count[t.n_wait] = len(producers(m, c))
    t.n_wait += 1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule in (amk.AMK_CHECK_ACYCLIC, amk.AMK_CHECK_QUEUE_ORDER), rep.message


def test_drop_wait_race_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_O, 1)
    m[i].n_wait = 0
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_RACE, rep.message


def test_kv_read_before_append_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_ATTN, 2)
    m[i].n_wait = 0
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_KV_ORDER, rep.message


def test_self_wait_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_O, 0)  # a task with a free wait slot
    t = m[i]
    assert t.n_wait < amk.AMK_MAX_WAITS
    c = t.signal_counter
    t.wait_counter[t.n_wait] = c
    t.wait_count[t.n_wait] = len(producers(m, c))
    t.n_wait += 1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_QUEUE_ORDER, rep.message


def test_oob_counter_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    m[find(m, amk.AMK_OP_DOWN, 0)].wait_counter[0] = nc
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_WELL_FORMED, rep.message


def test_oob_buffer_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_O, 0, lambda t: t.end == 256)
    m[i].end = 257
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_WELL_FORMED, rep.message


def test_capacity_overflow_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    m[find(m, amk.AMK_OP_QKV, 1)].n_wait = 5
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_CAPACITY, rep.message


def test_partial_shared_wait_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_GATEUP, 1)
    assert m[i].wait_count[0] > 2
    m[i].wait_count[0] -= 1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_ALL_JOIN, rep.message


def test_unsatisfiable_waits_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_DOWN, 0)
    m[i].wait_count[0] += 1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_WAIT_SATISFIABLE
    m = clone(tasks)
    m[i].wait_count[0] = 0
    assert check(cfg, m, nc).rule == amk.AMK_CHECK_WAIT_SATISFIABLE
    # a counter nobody signals: retarget its only producers' signals
    m = clone(tasks)
    c = m[i].wait_counter[0]
    for p in producers(m, c):
        m[p].signal_counter = -1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_WAIT_SATISFIABLE


def test_cross_queue_deadlock_rejected(lib):
    """A deadlock that no single queue shows: the argmax task (queue x) gets a
    fresh signal counter, and an early task A on the other queue y waits on it.
    Argmax waits on every LM-head task, including those queued on y after A.
    Every wait is satisfiable, A's producer sits on another queue (so the
    per-queue order rule passes), yet the queues block each other."""
    cfg = cfg_of("tiny")
    tasks, nc = amk.amk_schedule_export(cfg, 2)
    m = clone(tasks)
    g = find(m, amk.AMK_OP_ARGMAX)
    x = m[g].cu
    y = 1 - x
    a = find(m, amk.AMK_OP_QKV, 0, lambda t: t.cu == y)
    assert any(t.op == amk.AMK_OP_LMHEAD and t.cu == y and t.seq > m[a].seq for t in m)
    m[g].signal_counter = nc
    t = m[a]
    t.wait_counter[t.n_wait] = nc
    t.wait_count[t.n_wait] = 1
    t.n_wait += 1
    rep = check(cfg, m, nc + 1, 2)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_ACYCLIC, rep.message
    assert "deadlock" in rep.message.decode()


def test_duplicate_and_missing_output_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_DOWN, 2, lambda t: t.begin > 0)
    m[i].begin -= 1  # overlaps its neighbour
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_OUTPUT, rep.message
    m = clone(tasks)
    m[i].begin += 1  # leaves a row unwritten
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_OUTPUT, rep.message


def test_queue_position_duplicates_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    m[1].seq = m[0].seq
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_WELL_FORMED


def test_random_single_mutations_never_crash(tiny_sched):
    cfg, tasks, nc = tiny_sched
    rng = random.Random(7)
    fields = ["begin", "end", "aux", "n_wait", "signal_counter", "seq", "cu", "layer", "op"]
    for _ in range(300):
        m = clone(tasks)
        i = rng.randrange(len(m))
        f = rng.choice(fields)
        setattr(m[i], f, getattr(m[i], f) + rng.choice([-3, -1, 1, 2, 1000]))
        rep = check(cfg, m, nc)
        assert rep.ok in (0, 1)


# ------------------------------------------------------------------ inline combine
def test_inline_task_with_two_waits_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_COMBINE, 1)
    t = m[i]
    t.wait_counter[1] = t.wait_counter[0]
    t.wait_count[1] = t.wait_count[0]
    t.n_wait = 2
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_INLINE, rep.message


def test_chain_to_wrong_counter_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_ATTN, 0, lambda t: t.begin == 3)
    m[i].chain_counter = m[find(m, amk.AMK_OP_O, 0)].signal_counter
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_INLINE, rep.message


def test_split_without_chain_rejected(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_ATTN, 2, lambda t: t.begin == 5)
    m[i].chain_counter = -1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_INLINE, rep.message


def test_inline_task_only_for_combine(tiny_sched):
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    i = find(m, amk.AMK_OP_ARGMAX)
    m[i].cu = amk.AMK_CU_INLINE
    m[i].seq = 0
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule in (amk.AMK_CHECK_INLINE, amk.AMK_CHECK_WELL_FORMED), rep.message


def test_o_reading_before_combine_rejected(tiny_sched):
    """O waiting on the attention splits' head counter instead of the combine
    output: it would read the attention output before the combine wrote it."""
    cfg, tasks, nc = tiny_sched
    m = clone(tasks)
    comb = find(m, amk.AMK_OP_COMBINE, 1)
    i = find(m, amk.AMK_OP_O, 1)
    m[i].wait_counter[0] = m[comb].wait_counter[0]
    m[i].wait_count[0] = m[comb].wait_count[0]
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule in (amk.AMK_CHECK_RACE, amk.AMK_CHECK_INLINE), rep.message


# ------------------------------------------------------------------ short schedule (inline attention)
@pytest.fixture(scope="module")
def tiny_short(lib):
    cfg = cfg_of("tiny")
    tasks, nc = amk.amk_schedule_export(cfg, N_CU, variant=amk.AMK_SCHEDULE_SHORT)
    assert check(cfg, tasks, nc).ok
    return cfg, tasks, nc


def test_short_qkv_without_chain_rejected(tiny_short):
    cfg, tasks, nc = tiny_short
    m = clone(tasks)
    m[find(m, amk.AMK_OP_QKV, 1)].chain_counter = -1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_INLINE, rep.message


def test_short_inline_attention_of_other_group_rejected(tiny_short):
    """The device runs the chaining task's own group: an inline attention
    labelled with another group does not pair up."""
    cfg, tasks, nc = tiny_short
    m = clone(tasks)
    i = find(m, amk.AMK_OP_ATTN, 2, lambda t: t.aux == 0)
    m[i].aux = 1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule in (amk.AMK_CHECK_INLINE, amk.AMK_CHECK_OUTPUT), rep.message


def test_short_qkv_task_across_groups_rejected(tiny_short):
    cfg, tasks, nc = tiny_short
    m = clone(tasks)
    # widen the last task of group 0 into group 1 and shrink its neighbour
    i = find(m, amk.AMK_OP_QKV, 0, lambda t: t.aux == 0 and t.end % 128 == 0 and t.end > 0)
    j = find(m, amk.AMK_OP_QKV, 0, lambda t: t.begin == m[i].end)
    m[i].end += 1
    m[j].begin += 1
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_WELL_FORMED, rep.message


def test_short_o_waiting_on_qkv_counter_rejected(tiny_short):
    """O waiting on one group's QKV counter instead of the attention output:
    it would read attention outputs nobody has ordered before it."""
    cfg, tasks, nc = tiny_short
    m = clone(tasks)
    a = find(m, amk.AMK_OP_ATTN, 1)
    i = find(m, amk.AMK_OP_O, 1)
    m[i].wait_counter[0] = m[a].wait_counter[0]
    m[i].wait_count[0] = m[a].wait_count[0]
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_RACE, rep.message


def test_short_producer_count_mismatch_rejected(tiny_short):
    """A QKV task of group 1 relabelled to signal group 0's counter: every
    wait count is fixed up to stay an all-join, but the chaining tasks of
    group 0 would count one producer more than the device expects."""
    cfg, tasks, nc = tiny_short
    m = clone(tasks)
    g0 = find(m, amk.AMK_OP_ATTN, 0, lambda t: t.aux == 0)
    g1 = find(m, amk.AMK_OP_ATTN, 0, lambda t: t.aux == 1)
    i = find(m, amk.AMK_OP_QKV, 0, lambda t: t.aux == 1)
    m[i].signal_counter = m[g0].wait_counter[0]
    m[g0].wait_count[0] += 1
    m[g1].wait_count[0] -= 1
    rep = check(cfg, m, nc)
    assert not rep.ok, rep.message


# ------------------------------------------------------------------ tiny schedule (attention in the O tasks)
def test_schedule_shape_8b_tiny(lib):
    cfg = cfg_of("llama3_8b")
    tasks, nc = amk.amk_schedule_export(cfg, 256, variant=amk.AMK_SCHEDULE_TINY)
    assert check(cfg, tasks, nc, 256).ok
    assert not [t for t in tasks if t.op in (amk.AMK_OP_ATTN, amk.AMK_OP_COMBINE) or t.cu == amk.AMK_CU_INLINE]
    qkv = [t for t in tasks if t.op == amk.AMK_OP_QKV and t.layer == 7]
    o = [t for t in tasks if t.op == amk.AMK_OP_O and t.layer == 7]
    # the QKV stage signals four counters (task i counter i mod 4); every O task
    # waits on each of them for exactly its producers
    sigs = {}
    for t in qkv:
        sigs[t.signal_counter] = sigs.get(t.signal_counter, 0) + 1
    assert len(sigs) == 4 and sum(sigs.values()) == len(qkv) and all(t.chain_counter == -1 for t in qkv)
    for t in o:
        assert t.aux == 1 and t.n_wait == 4
        assert {(t.wait_counter[k], t.wait_count[k]) for k in range(t.n_wait)} == set(sigs.items())


@pytest.fixture(scope="module")
def tiny_tiny(lib):
    cfg = cfg_of("tiny")
    tasks, nc = amk.amk_schedule_export(cfg, N_CU, variant=amk.AMK_SCHEDULE_TINY)
    assert check(cfg, tasks, nc).ok
    return cfg, tasks, nc


def test_tiny_o_without_wait_rejected(tiny_tiny):
    """An O task that computes attention from q and the KV cache must be
    ordered after every QKV task: without its wait it reads the new K/V row
    before it is appended."""
    cfg, tasks, nc = tiny_tiny
    m = clone(tasks)
    m[find(m, amk.AMK_OP_O, 2)].n_wait = 0
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule in (amk.AMK_CHECK_KV_ORDER, amk.AMK_CHECK_RACE), rep.message


def test_tiny_o_reading_unwritten_output_rejected(tiny_tiny):
    """In the tiny schedule nobody writes the attention output buffer: an O
    task that reads it (aux 0) reads a region no task writes."""
    cfg, tasks, nc = tiny_tiny
    m = clone(tasks)
    m[find(m, amk.AMK_OP_O, 1)].aux = 0
    rep = check(cfg, m, nc)
    assert not rep.ok and rep.rule == amk.AMK_CHECK_OUTPUT, rep.message


# ---------------------------------------------------------------- LPT queue assignment
def lpt_tuning():
    t = amk.amk_tuning_t()
    t.queue_assign = amk.AMK_ASSIGN_LPT
    return t


@pytest.mark.parametrize("name", list(synth.CONFIGS))
@pytest.mark.parametrize("n_cu", [256, 13])
@pytest.mark.parametrize("variant", [amk.AMK_SCHEDULE_SHORT, amk.AMK_SCHEDULE_LONG, amk.AMK_SCHEDULE_TINY])
def test_lpt_lowering_accepted(lib, name, n_cu, variant):
    """The longest-processing-time assignment (paper §4 ScheduleConfig
    sm_assignment 'load_balance') lowers every config to a schedule the
    checker accepts, with the same tasks as round robin on other queues."""
    cfg = cfg_of(name, "w8a16")
    t = lpt_tuning()
    tasks, nc = amk.amk_schedule_export(cfg, n_cu, t, variant=variant)
    rep = amk.amk_schedule_check(cfg, n_cu, tasks, nc, t)
    assert rep.ok == 1, rep.message
    rr, nc_rr = amk.amk_schedule_export(cfg, n_cu, variant=variant)
    assert nc == nc_rr
    key = lambda x: (x.op, x.layer, x.begin, x.end, x.aux)  # noqa: E731
    assert sorted(map(key, tasks)) == sorted(map(key, rr))
    assert amk.amk_check_config(cfg, n_cu) == amk.AMK_OK


def _queue_loads(tasks, cfg, n_cu):
    """Estimated work per queue: weight bytes of each GEMV task plus 64 KiB
    per task (the cost model the LPT assignment is documented with)."""
    wb = {amk.AMK_WEIGHTS_BF16: 2.0, amk.AMK_WEIGHTS_W8A16: 1.0}[cfg.weight_format]
    H, I, qd = cfg.hidden, cfg.intermediate, cfg.n_heads * cfg.head_dim
    load = [0.0] * n_cu
    for t in tasks:
        if t.cu == amk.AMK_CU_INLINE or t.op not in (amk.AMK_OP_QKV, amk.AMK_OP_O, amk.AMK_OP_GATEUP,
                                                      amk.AMK_OP_DOWN, amk.AMK_OP_LMHEAD):
            continue
        rows = (t.end - t.begin) * (2 if t.op in (amk.AMK_OP_QKV, amk.AMK_OP_GATEUP) else 1)
        k = qd if t.op == amk.AMK_OP_O else I if t.op == amk.AMK_OP_DOWN else H
        b = 2.0 if (t.op == amk.AMK_OP_LMHEAD and cfg.tied_embeddings) else wb
        load[t.cu] += rows * k * b + 65536
    return load


@pytest.mark.parametrize("name", ["tiny", "smollm2_135m", "tinyllama_1b"])
def test_lpt_balances_at_least_as_well(lib, name):
    """On 13 queues, where the stages do not divide evenly, the most loaded
    queue carries no more estimated GEMV work under LPT than under round
    robin."""
    cfg = cfg_of(name)
    lpt, _ = amk.amk_schedule_export(cfg, 13, lpt_tuning(), variant=amk.AMK_SCHEDULE_TINY)
    rr, _ = amk.amk_schedule_export(cfg, 13, variant=amk.AMK_SCHEDULE_TINY)
    assert max(_queue_loads(lpt, cfg, 13)) <= max(_queue_loads(rr, cfg, 13))


def test_unknown_queue_assign_rejected(lib):
    t = amk.amk_tuning_t()
    t.queue_assign = 7
    with pytest.raises(amk.AmkError) as e:
        amk.amk_schedule_export(cfg_of("tiny"), 16, t)
    assert e.value.status == amk.AMK_ERR_INVALID_ARGUMENT
