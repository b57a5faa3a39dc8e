"""The host block manager and the Alg. 1 scheduler (Sec. 5.2, Sec. 4.2), on the
CPU.

The manager is pinned by a simulation that carries token identities instead
of K/V values: a pool of [block][slot] identities, a host store for
checkpointed tokens, and random arrivals, growth (RT prefill chunks and
decode tokens, BE decode tokens), restores and releases. After every step
each request's every position must be found where the manager says it is --
in its slot (through its table and direction) or in the host store -- and the
batch of requests that ran must pass the library's checker and the oracle's
slot-ownership count. A lost victim, a wrong slot, a move that drops a token
or a restore to the wrong place breaks one of these. Victims are also checked
against the oracle's statement of which peer tokens a write overwrites.
"""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import manager as M

bros = pytest.importorskip("paper_2504_09590_amd.bros", reason="libbros_attn.so not built")

RT, BE = 0, 1


def ident(req, pos):
    return req * 1_000_000 + pos


class Sim:
    def __init__(self, num_blocks, seed):
        self.m = M.BlockManager(num_blocks)
        self.nb = num_blocks
        self.pool = np.full((num_blocks, 16), -1, dtype=np.int64)
        self.host = {}
        self.cls = {}
        self.rng = np.random.default_rng(seed)
        self.next_id = 1
        self.stats = {"victims": 0, "moves": 0, "restores": 0, "nomem": 0}

    def add(self, cls):
        rid = self.next_id
        self.next_id += 1
        self.m.add(rid, cls)
        self.cls[rid] = cls
        return rid

    def release(self, rid):
        self.m.release(rid)
        del self.cls[rid]
        for k in [k for k in self.host if k[0] == rid]:
            del self.host[k]

    def slot_of(self, rid, pos):
        tab = self.m.table(rid)
        off = pos % 16
        return int(tab[pos // 16]), off if self.cls[rid] == RT else 15 - off

    def apply(self, rid, plan):
        # the device order: victims gathered, moves, restores, then the new tokens
        for r, p, b, s in plan.victims:
            assert self.pool[b, s] == ident(r, p), "victim is not the peer's token"
            self.host[(int(r), int(p))] = int(self.pool[b, s])
        if len(plan.move_src):
            vals = self.pool.reshape(-1)[plan.move_src].copy()
            self.pool.reshape(-1)[plan.move_dst] = vals
        for p, sid in zip(plan.restore_pos, plan.restore_dst):
            self.pool.reshape(-1)[sid] = self.host.pop((rid, int(p)))
        for p, sid in zip(plan.written_pos, plan.written_slot):
            self.pool.reshape(-1)[sid] = ident(rid, int(p))
        self.stats["victims"] += len(plan.victims)
        self.stats["moves"] += len(plan.move_src)
        self.stats["restores"] += len(plan.restore_pos)

    def tables_for(self, ids):
        tabs = [self.m.table(r) for r in ids]
        maxb = max([len(t) for t in tabs] + [1])
        out = np.zeros((len(ids), maxb), dtype=np.int32)
        for i, t in enumerate(tabs):
            out[i, :len(t)] = t
        dirs = np.array([1 if self.cls[r] == RT else -1 for r in ids], dtype=np.int8)
        ctx = np.array([self.m.query(r)[0] for r in ids], dtype=np.int32)
        return out, dirs, ctx

    def check_all(self):
        for rid in self.cls:
            ctx, _, ck = self.m.query(rid)
            n_host = 0
            for p in range(ctx):
                if (rid, p) in self.host:
                    n_host += 1
                    continue
                b, s = self.slot_of(rid, p)
                assert self.pool[b, s] == ident(rid, p), f"request {rid} position {p} lost (block {b} slot {s})"
            assert n_host == ck, (rid, n_host, ck)


def run_sim(num_blocks, steps, seed, rt_frac=0.4):
    sim = Sim(num_blocks, seed)
    rng = sim.rng
    for step in range(steps):
        # arrivals and completions
        for _ in range(rng.integers(0, 4)):
            sim.add(RT if rng.random() < rt_frac else BE)
        for rid in list(sim.cls):
            if rng.random() < 0.05:
                sim.release(rid)
        ids = list(sim.cls)
        if not ids:
            continue
        run = [r for r in ids if rng.random() < 0.6]
        run.sort(key=lambda r: sim.cls[r])           # RT first, then BE
        ran = []
        for rid in run:
            ctx, _, ck = sim.m.query(rid)
            n_new = int(rng.integers(16, 80)) if (sim.cls[rid] == RT and ctx < 200 and rng.random() < 0.5) else 1
            try:
                if ck:
                    sim.apply(rid, sim.m.restore(rid))
                tab_before, dir_before, ctx_before = sim.tables_for(list(sim.cls))
                plan = sim.m.grow(rid, n_new)
            except bros.BrosError as e:
                assert e.status == -8        # BROS_E_NOMEM: out of blocks
                sim.apply(rid, e.plan)       # what was done before the failure stays done
                sim.stats["nomem"] += 1
                sim.release(rid)
                continue
            # victims = the oracle's overwritten peer tokens, among tokens still on the GPU
            all_ids = list(sim.cls)
            w = all_ids.index(rid)
            if len(plan.written_pos) and not any(sim.m.query(r)[2] for r in all_ids if r != rid) \
                    and tab_before.shape[1] * 16 >= ctx_before[w] + n_new:
                tb, db, cb = tab_before.copy(), dir_before, ctx_before
                new_tab, _, _ = sim.tables_for([rid])
                tb2 = np.zeros((len(all_ids), max(tb.shape[1], new_tab.shape[1])), dtype=np.int32)
                tb2[:, :tb.shape[1]] = tb
                tb2[w, :new_tab.shape[1]] = new_tab[0]
                expect = oracle.overwritten_peer_tokens(tb2, db, cb, w, plan.written_pos)
                got = sorted((all_ids.index(int(r)), int(p), int(b), int(s)) for r, p, b, s in plan.victims)
                if not len(plan.move_src):
                    assert got == sorted(expect)
            sim.apply(rid, plan)
            ran.append(rid)
        sim.check_all()
        sim.m.validate()
        # the requests that ran this step form a consistent batch
        batch = [r for r in ran if r in sim.cls and sim.m.query(r)[2] == 0]
        if batch:
            t, d, c = sim.tables_for(batch)
            bros.bros_check_batch(t, d, None, c, num_blocks)
            assert oracle.slot_owner_counts(t, d, c, num_blocks).max() <= 1
        pt = sim.m.preemption_table()
        for b, rt, be in pt:
            assert rt >= 0 and be >= 0
    return sim


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_simulation_keeps_every_token(seed):
    sim = run_sim(num_blocks=60, steps=120, seed=seed)
    # the scenario space was exercised: lazy checkpoints, relocations and restores happened
    assert sim.stats["victims"] > 0 and sim.stats["restores"] > 0 and sim.stats["moves"] > 0, sim.stats


def test_simulation_under_heavy_pressure():
    sim = run_sim(num_blocks=24, steps=150, seed=9, rt_frac=0.6)
    assert sim.stats["nomem"] > 0


def test_lazy_checkpoint_scenario_from_the_fixture():
    """The hand-enumerated Sec. 5.2 scenario (tests/golden/lazy_checkpoint.json),
    driven through the manager: BE a holds 12 tokens, RT B 20 (its tail of 4
    in a's block), B grows by 4 and checkpoints a's positions 8..11."""
    m = M.BlockManager(2)
    m.add(1, BE)                  # a
    m.grow(1, 12)                 # block 0 (first free), slots 15..4
    m.add(2, RT)                  # B
    p = m.grow(2, 16)             # block 1 (the only free one)
    assert m.table(2).tolist() == [1]
    p = m.grow(2, 4)              # no free block: FindPreemptBlock takes a's block, slots 0..3
    assert m.table(2).tolist() == [1, 0] and len(p.victims) == 0
    p = m.grow(2, 4)              # slots 4..7 hold a's positions 11..8
    assert sorted(map(tuple, p.victims.tolist())) == [(1, 8, 0, 7), (1, 9, 0, 6), (1, 10, 0, 5), (1, 11, 0, 4)]
    assert m.query(1) == (12, 1, 4)
    assert m.preemption_table().tolist() == [[0, 2, 1]]
    with pytest.raises(bros.BrosError):
        m.grow(1, 1)              # a must be restored first
    with pytest.raises(bros.BrosError):
        m.restore(1)              # no block to move a's entry to (NOMEM)
    m.release(2)                  # B finishes: a can come back in place
    r = m.restore(1)
    assert len(r.move_src) == 0 and r.restore_pos.tolist() == [8, 9, 10, 11]
    assert r.restore_dst.tolist() == [7, 6, 5, 4]
    assert m.query(1) == (12, 1, 0)


# --- Alg. 1 and adaptive batch sizing ------------------------------------------

COEF = ((0.01, 0.0, 10.0), (0.05, 0.0, 20.0))     # prefill, decode: a0 * Ln + b (us)


def _rt(i, rem, n=1, ctx=100, prefill=0):
    return dict(id=i, prefill=prefill, n_new=n, ctx_after=ctx, remaining_us=rem)


def _be(i, mcpu, n=1, ctx=100):
    return dict(id=i, prefill=0, n_new=n, ctx_after=ctx, m_cpu=mcpu)


def test_schedule_orders_rt_by_remaining_time_and_caps_the_batch():
    m = M.BlockManager(1000)
    rt = [_rt(1, 500.0), _rt(2, 100.0), _rt(3, 300.0)]
    got_rt, got_be, over = M.schedule(m, rt, [], 2, COEF)
    assert got_rt == [2, 3] and got_be == [] and not over


def test_schedule_stops_at_the_time_budget():
    m = M.BlockManager(1000)
    # decode cost of k requests: 0.05 * k + 20 us; budget = most urgent remaining time
    rt = [_rt(i, 20.12) for i in range(1, 6)]
    got_rt, _, over = M.schedule(m, rt, [], 10, COEF)
    assert got_rt == [1, 2] and over        # 20.10 fits, 20.15 does not


def test_schedule_packs_be_by_checkpointed_slots_then_replaces_rt():
    m = M.BlockManager(1000)
    rt = [_rt(1, 1000.0), _rt(2, 2000.0)]
    be = [_be(10, 5), _be(11, 0), _be(12, 9)]
    got_rt, got_be, over = M.schedule(m, rt, be, 4, COEF)
    # least m_cpu first: 11 and 10 are packed; 12 no longer fits and replaces the least urgent RT (2)
    assert got_rt == [1] and got_be == [11, 10, 12] and not over
    got_rt, got_be, _ = M.schedule(m, rt, be, 2, COEF)
    # full batch: BE 11 replaces RT 2, BE 10 replaces RT 1, BE 12 finds no RT left to replace
    assert got_rt == [] and got_be == [11, 10]


def test_schedule_respects_blocks():
    m = M.BlockManager(4)
    rt = [_rt(1, 1e6, n=40, ctx=40), _rt(2, 2e6, n=40, ctx=40)]   # 3 blocks each
    got_rt, _, _ = M.schedule(m, rt, [], 8, COEF)
    assert got_rt == [1]                    # FindPreemptBlock fails for the second


def test_adaptive_batch_size():
    assert M.next_batch_size(128, 128, 1024, False) == 256
    assert M.next_batch_size(1024, 128, 1024, False) == 1024
    assert M.next_batch_size(512, 128, 1024, True) == 128


def _populated(seed, num_blocks=400, n=60):
    """A manager with RT and BE requests of random lengths, some of them with
    checkpointed tokens (RT growth over shared BE tails)."""
    rng = np.random.default_rng(seed)
    m = M.BlockManager(num_blocks)
    cls = {}
    for rid in range(1, n + 1):
        c = RT if rng.random() < 0.4 else BE
        m.add(rid, c)
        cls[rid] = c
        try:
            m.grow(rid, int(rng.integers(1, 90)))
        except bros.BrosError:
            m.release(rid)
            del cls[rid]
    return m, cls, rng


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_grow_batch_equals_one_call_per_request(seed):
    # Two identical managers: one grows each request by its own restore and
    # grow calls, the other by one batched call. Same plans (concatenated in
    # request order), same tables, same statuses.
    a, cls, rng = _populated(seed)
    b, _, _ = _populated(seed)
    ids = sorted(cls)
    pick = [int(r) for r in rng.choice(ids, size=min(40, len(ids)), replace=False)]
    n_new = [int(rng.integers(1, 40)) if cls[r] == RT and rng.random() < 0.3 else 1 for r in pick]
    parts, status = [], []
    for r, k in zip(pick, n_new):
        got = []
        try:
            if a.query(r)[2]:
                got.append(a.restore(r))
            got.append(a.grow(r, k))
            status.append(0)
        except bros.BrosError as e:
            got.append(e.plan)
            status.append(e.status)
        parts.append(got)
    plan, ends, st = b.grow_batch(pick, n_new, restore_first=True)
    assert st.tolist() == status
    for k, field in enumerate(("victims", "move_src", "restore_pos", "written_pos")):
        lens = [sum(len(getattr(p, field)) for p in got) for got in parts]
        assert ends[:, k].tolist() == np.cumsum(lens).tolist(), field
    for field in ("victims", "move_src", "move_dst", "restore_pos", "restore_dst", "written_pos", "written_slot"):
        want = [getattr(p, field) for got in parts for p in got]
        want = np.concatenate(want) if want else np.zeros(0)
        assert np.array_equal(getattr(plan, field).reshape(want.shape), want), field
    for r in ids:
        assert np.array_equal(a.table(r), b.table(r)) and a.query(r) == b.query(r)
    b.validate()


def test_grow_batch_without_restore_reports_the_checkpointed_request():
    m = M.BlockManager(1)
    m.add(1, BE)
    m.grow(1, 10)                     # BE tokens in slots 15..6 of the only block
    m.add(2, RT)
    m.grow(2, 16)                     # RT fills the block from the left: 10 BE tokens checkpointed
    assert m.query(1)[2] > 0
    plan, ends, st = m.grow_batch([2, 1], [1, 1], restore_first=False)
    assert st.tolist()[1] == -7 and st.tolist()[0] in (0, -8)
    with pytest.raises(bros.BrosError):
        m.grow_batch([99], [1])       # unknown request: nothing changes


def _queue(rng, ids, rt):
    q = np.zeros(len(ids), dtype=M.SCHED_DTYPE)
    q["id"] = ids
    q["prefill"] = rng.random(len(ids)) < 0.3
    q["n_new"] = np.where(q["prefill"], rng.integers(16, 200, len(ids)), 1)
    q["ctx_after"] = rng.integers(20, 3000, len(ids))
    if rt:
        q["remaining_us"] = np.round(rng.uniform(50.0, 5000.0, len(ids)), 0)   # ties happen
    else:
        q["m_cpu"] = rng.integers(0, 30, len(ids))
    return q


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_request_pulling_equals_the_full_sort(seed):
    # Sec. 4.2: with the waiting queue in ascending remaining time, sorting
    # only (the reachable part of) the pending queue and polling the two
    # queue heads gives Alg. 1 the same RT order as sorting both together.
    rng = np.random.default_rng(seed)
    m, cls, _ = _populated(seed, num_blocks=3000, n=200)
    ids = sorted(cls)
    rt_ids = [r for r in ids if cls[r] == RT]
    be_ids = [r for r in ids if cls[r] == BE]
    pending = _queue(rng, rt_ids[: len(rt_ids) // 2], True)
    waiting = _queue(rng, rt_ids[len(rt_ids) // 2:], True)
    waiting = waiting[np.argsort(waiting["remaining_us"], kind="stable")]
    be = _queue(rng, be_ids, False)
    for batch in (1, 4, 16, 64, 1000):
        for coef in (COEF, ((0.0, 0.0, 1.0), (0.0, 0.0, 1.0))):
            full = M.schedule(m, np.concatenate([pending, waiting]), be, batch, coef)
            pulled = M.schedule_pulled(m, pending, waiting, be, batch, coef)
            assert pulled == full, (batch, coef)
