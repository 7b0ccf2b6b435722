"""Per-stage KV reservation and admission (CPU).

The plain model (oracle/admission.py) is pinned by hand-computed cases and
invariants; the native scheduler (ps_sched_*) must then take exactly the
model's decisions, step by step, on seeded heavy-tailed request traces:
the same admitted sequence ids, the same preemptions in the same order, the
same chunk size after every completion. Everything here is integer work, so
the comparison is exact. No GPU: the scheduler touches only host metadata.
"""
import numpy as np
import pytest

from oracle.admission import AdmissionModel
from paper_2608_21719_amd import binding as B
from synth import gen
from synth.configs import CONFIGS

FAKE_POOL = 0x10000


# ------------------------------------------------------------ model pins
def test_chunk_size_follows_the_observed_mean_rounded_to_a_page():
    m = AdmissionModel(100, 8, 64, window=3, cs_initial=512, cs_min=32, cs_max=1024)
    assert m.chunk_size() == 512
    for s, L in zip([m.admit(0) for _ in range(2)], [100, 200]):
        m.finish(s, L)
    assert m.chunk_size() == 160          # mean 150 -> 10 pages
    for L in (1000, 1000):
        m.finish(m.admit(0), L)
    assert m.chunk_size() == 736          # window 3: (200 + 1000 + 1000) / 3 = 733.3 -> 46 pages
    m.finish(m.admit(0), 5000)
    assert m.chunk_size() == 1024         # clamped to cs_max
    for _ in range(3):
        m.finish(m.admit(0), 1)
    assert m.chunk_size() == 32           # mean 1 -> one page, clamped up to cs_min


def test_admission_count_is_pool_pages_over_chunk_pages():
    """Memory-limited concurrency: with CS fixed at 64 tokens (4 pages) and
    no context, exactly floor(pages / 4) requests are admitted."""
    for pages in (40, 41, 43, 7):
        m = AdmissionModel(pages, 100, 64, window=4, cs_initial=64, cs_min=64, cs_max=64)
        n = 0
        while m.admit(0) is not None:
            n += 1
        assert n == pages // 4


def test_growth_takes_whole_chunks_and_preempts_the_newest():
    m = AdmissionModel(12, 8, 64, window=4, cs_initial=64, cs_min=64, cs_max=64)
    a, b, c = m.admit(0), m.admit(0), m.admit(0)     # 3 x 4 pages: pool full
    assert (a, b, c) == (0, 1, 2) and m.free == 0
    m.commit(a, 64)
    assert m.reserve_step([a], [1]) == [c]            # a needs 4 more pages: c (newest) goes
    assert m.pages[a] == 8 and m.free == 0 and c not in m.pages
    m.commit(b, 64)
    assert m.reserve_step([b], [1]) == [b]            # b is now the newest: it preempts itself
    assert m.free == 4 and list(m.pages) == [a]
    assert m.admit(16) is None                        # 16 + 64 tokens = 5 pages > 4 free
    assert m.admit(0) == 1 and m.free == 0            # the lowest free slot, 4 pages


def test_random_traces_keep_page_accounting_exact():
    arr, ctx, L = gen.request_trace(1, 300, rate=0.8)
    m = AdmissionModel(900, 64, 400, window=16, cs_initial=512, cs_min=64, cs_max=4096)
    log = replay(ModelDriver(m), arr, ctx, L, steps=200000)
    assert log["finished"] == 300
    assert m.free == 900 and not m.pages


# ------------------------------------------------------------ replay
class ModelDriver:
    def __init__(self, m):
        self.m = m
        self.n_pages = m.free

    def cs(self):
        return self.m.chunk_size()

    def admit(self, ctx):
        return self.m.admit(ctx)

    def reserve(self, seqs):
        return self.m.reserve_step(seqs, [1] * len(seqs))

    def commit(self, seqs):
        for s in seqs:
            self.m.commit(s, 1)

    def finish(self, s, n):
        self.m.finish(s, n)

    def check(self):
        assert self.m.free >= 0
        assert self.m.free + sum(self.m.pages.values()) == self.n_pages
        for s, p in self.m.pages.items():
            assert self.m.length[s] <= 16 * p


class NativeDriver:
    def __init__(self, n_pages, max_seqs, max_pages, window, cs0, lo, hi):
        cfg = B.make_cfg(CONFIGS["llama8b_think"].shape)
        self.kv = B.KV(cfg, 1, n_pages, max_seqs, max_pages, FAKE_POOL, 7)
        self.s = B.Sched(self.kv, window, cs0, lo, hi)
        self.max_seqs = max_seqs

    def cs(self):
        return self.s.chunk_size()

    def admit(self, ctx):
        return self.s.admit(ctx)

    def reserve(self, seqs):
        return self.s.reserve_step(seqs, [1] * len(seqs), self.max_seqs)

    def commit(self, seqs):
        if seqs:
            self.kv.commit(seqs, [1] * len(seqs))

    def finish(self, s, n):
        self.s.finish(s, n)

    def check(self):
        pass


def replay(drv, arrival, ctx, length, steps):
    """One stage pool serving a trace: arrivals queue in order; each step
    admits from the head while requests fit, reserves one more token for
    every running sequence (preempted requests go back to the head of the
    queue and start their stage over), commits it, and finishes the
    sequences that reached their stage length. Returns the decision log."""
    waiting, running, gen_tok = [], {}, {}
    nxt, log = 0, {"events": [], "finished": 0, "preempted": 0, "admitted": 0, "max_running": 0}
    for step in range(steps):
        while nxt < len(arrival) and arrival[nxt] <= step:
            waiting.append(nxt)
            nxt += 1
        while waiting:
            r = waiting[0]
            s = drv.admit(int(ctx[r]))
            if s is None:
                break
            waiting.pop(0)
            running[s] = r
            gen_tok[s] = 0
            log["admitted"] += 1
            log["events"].append(("admit", step, r, s))
        seqs = sorted(running, key=lambda q: (gen_tok[q], q))
        pre = drv.reserve(seqs)
        for s in pre:
            log["events"].append(("preempt", step, running[s], s))
            waiting.insert(0, running.pop(s))
            del gen_tok[s]
        log["preempted"] += len(pre)
        live = [s for s in seqs if s in running]
        drv.commit(live)
        for s in live:
            gen_tok[s] += 1
        log["max_running"] = max(log["max_running"], len(running))
        for s in sorted(running):
            if gen_tok[s] == length[running[s]]:
                drv.finish(s, int(length[running[s]]))
                log["events"].append(("finish", step, running[s], s, drv.cs()))
                del running[s], gen_tok[s]
                log["finished"] += 1
        drv.check()
        if log["finished"] == len(arrival):
            break
    return log


@pytest.mark.parametrize("seed,rate,pages,cs0,lo,hi", [
    (1, 0.8, 900, 512, 64, 4096),      # heavy tail, roomy pool
    (2, 1.5, 600, 1024, 16, 2048),     # overloaded: frequent preemption
    (3, 0.3, 300, 16, 16, 512),        # small initial chunk, low cap
])
def test_native_scheduler_takes_the_models_decisions(seed, rate, pages, cs0, lo, hi):
    arr, ctx, L = gen.request_trace(seed, 250, rate=rate)
    L = np.minimum(L, 16 * 300 - 600)   # every request fits a sequence
    args = (pages, 64, 300, 8, cs0, lo, hi)
    want = replay(ModelDriver(AdmissionModel(*args)), arr, ctx, L, steps=200000)
    got = replay(NativeDriver(*args), arr, ctx, L, steps=200000)
    assert want["finished"] == 250
    assert got["events"] == want["events"]
    assert want["admitted"] > 250 or want["preempted"] == 0


def test_adaptive_chunk_admits_by_observation_and_thrashes_less_than_a_fixed_small_chunk():
    """The paper's motivation for observed-length admission, on a heavy-tailed
    trace: a fixed small chunk admits many requests that later outgrow the
    pool and get preempted; the chunk that follows observed lengths admits
    fewer at a time and preempts less."""
    arr, ctx, L = gen.request_trace(5, 400, rate=1.0)
    L = np.minimum(L, 16 * 300 - 600)
    runs = {}
    for name, (cs0, lo, hi) in {"fixed_64": (64, 64, 64), "adaptive": (64, 64, 4096)}.items():
        runs[name] = replay(ModelDriver(AdmissionModel(800, 96, 300, 16, cs0, lo, hi)), arr, ctx, L, steps=200000)
        assert runs[name]["finished"] == 400
    assert runs["adaptive"]["preempted"] < runs["fixed_64"]["preempted"]


def test_scheduler_rejects_bad_use_without_changing_anything():
    d = NativeDriver(64, 4, 16, 4, 64, 16, 128)
    s = d.admit(16)
    assert s == 0
    with pytest.raises(B.PsError) as e:
        d.s.reserve_step([3], [1], 4)                 # not admitted here
    assert e.value.code == B.PS_E_INVALID
    with pytest.raises(B.PsError) as e:
        d.s.reserve_step([s], [1000], 4)              # beyond max_pages_per_seq
    assert e.value.code == B.PS_E_CAPACITY
    with pytest.raises(B.PsError):
        d.s.reserve_step([s], [1], 2)                 # preempted buffer smaller than max_seqs
    with pytest.raises(B.PsError) as e:
        d.admit(16 * 16)                              # a request no sequence can hold
    assert e.value.code == B.PS_E_CAPACITY
    assert d.kv.capacity(s) == 80 and d.kv.free_pages() == 59 and d.s.running() == 1
    with pytest.raises(B.PsError):
        B.Sched(d.kv, 0, 64, 16, 128)
    with pytest.raises(B.PsError):
        B.Sched(d.kv, 4, 60, 16, 128)
