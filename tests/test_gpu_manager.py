"""The host block manager driving the kernels, step after step (Sec. 5.2 with
Sec. 6's kernels): real block tables and directions from the manager, its
plans (lazy checkpoints, relocations, restores) carried out on the device by
PlanExecutor, the new tokens written by bros_kv_write and attended by
bros_attn_prefill_chunk / bros_attn_decode. A host mirror does the same with
the oracle's functions. After every step the device pool must equal the
mirror bit for bit and every attention output must match the oracle."""

import numpy as np
import pytest

import oracle
from paper_2504_09590_amd import manager as M
from tests.gpu_helpers import announce, compare, require_gpu

pytestmark = pytest.mark.gpu

RT, BE = 0, 1


def _bf16(rng, shape):
    x = rng.standard_normal(shape).astype(np.float32)
    return ((x.view(np.uint32) + 0x7FFF + ((x.view(np.uint32) >> 16) & 1)) >> 16).astype(np.uint16)


def _dev(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _host(t):
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def test_manager_drives_the_kernels():
    torch = require_gpu()
    from paper_2504_09590_amd import bros
    from paper_2504_09590_amd.swap import PlanExecutor
    rng = np.random.default_rng(2024)
    nb, hkv, hq, d = 40, 8, 32, 128
    kp, vp = _bf16(rng, (nb, hkv, 16, d)), _bf16(rng, (nb, hkv, 16, d))
    k_dev, v_dev = _dev(torch, kp), _dev(torch, vp)
    mgr = M.BlockManager(nb)
    ex = PlanExecutor(k_dev, v_dev, max_rows=256)
    store = {}                       # the mirror's checkpointed rows
    cls, started = {}, set()
    stats = {"victims": 0, "moves": 0, "restores": 0, "prefill": 0, "decode": 0}
    next_id = 1

    def mirror(req, plan):
        nonlocal kp, vp
        for r, p, b, s in plan.victims:
            store[(int(r), int(p))] = (kp[b, :, s].copy(), vp[b, :, s].copy())
        if len(plan.move_src):
            rk, rv = oracle.kv_gather(kp, plan.move_src), oracle.kv_gather(vp, plan.move_src)
            kp, vp = oracle.kv_scatter(kp, rk, plan.move_dst), oracle.kv_scatter(vp, rv, plan.move_dst)
        if len(plan.restore_pos):
            rows = [store.pop((req, int(p))) for p in plan.restore_pos]
            kp = oracle.kv_scatter(kp, np.stack([r[0] for r in rows]), plan.restore_dst)
            vp = oracle.kv_scatter(vp, np.stack([r[1] for r in rows]), plan.restore_dst)
        stats["victims"] += len(plan.victims)
        stats["moves"] += len(plan.move_src)
        stats["restores"] += len(plan.restore_pos)

    for step in range(14):
        for _ in range(rng.integers(1, 4)):
            cls[next_id] = RT if rng.random() < 0.5 else BE
            mgr.add(next_id, cls[next_id])
            next_id += 1
        for r in list(cls):
            if r in started and rng.random() < 0.08:
                mgr.release(r)
                ex.drop(r)
                for key in [k for k in store if k[0] == r]:
                    del store[key]
                del cls[r]
        run = sorted((r for r in cls if rng.random() < 0.7), key=lambda r: cls[r])   # RT first
        ran = []                     # (request, first new position, count)
        for r in run:
            n_new = int(rng.integers(20, 90)) if r not in started else 1
            try:
                if mgr.query(r)[2]:
                    plan = mgr.restore(r)
                    ex.execute(r, plan)
                    mirror(r, plan)
                p0 = mgr.query(r)[0]
                plan = mgr.grow(r, n_new)
            except bros.BrosError as e:
                if getattr(e, "plan", None) is not None:
                    ex.execute(r, e.plan)
                    mirror(r, e.plan)
                mgr.release(r)
                ex.drop(r)
                for key in [k for k in store if k[0] == r]:
                    del store[key]
                del cls[r]
                continue
            ex.execute(r, plan)
            mirror(r, plan)
            started.add(r)
            ran.append((r, p0, n_new))
        ran = [x for x in ran if x[0] in cls and mgr.query(x[0])[2] == 0]
        if not ran:
            continue
        # the step's batch, from the manager: prefill chunks first, decode rows after
        ran.sort(key=lambda x: x[2] == 1)
        ids = [x[0] for x in ran]
        tabs = [mgr.table(r) for r in ids]
        maxb = max(len(t) for t in tabs)
        tables = np.zeros((len(ids), maxb), dtype=np.int32)
        for i, t in enumerate(tabs):
            tables[i, :len(t)] = t
        dirs = np.array([1 if cls[r] == RT else -1 for r in ids], dtype=np.int8)
        ctx = np.array([mgr.query(r)[0] for r in ids], dtype=np.int32)
        counts = np.array([x[2] for x in ran])
        pos0 = np.array([x[1] for x in ran], dtype=np.int32)
        cu_new = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
        bros.bros_check_batch(tables, dirs, None, ctx, nb)
        k_new, v_new = _bf16(rng, (int(cu_new[-1]), hkv, d)), _bf16(rng, (int(cu_new[-1]), hkv, d))
        announce(f"manager step {step}: {len(ids)} sequences, {int(cu_new[-1])} new tokens, "
                 f"{sum(counts > 1)} prefill chunks")
        td, dd, cd = (torch.from_numpy(x).cuda() for x in (tables, dirs, ctx))
        bros.bros_kv_write(_dev(torch, k_new), _dev(torch, v_new), k_dev, v_dev, td, dd, None,
                           torch.from_numpy(pos0).cuda(), torch.from_numpy(cu_new).cuda())
        kp, vp = oracle.kv_write(kp, vp, k_new, v_new, tables, dirs, pos0, cu_new)
        torch.cuda.synchronize()
        assert np.array_equal(_host(k_dev), kp) and np.array_equal(_host(v_dev), vp), f"pool differs at step {step}"
        P = int(np.sum(counts > 1))
        if P:
            cu_q = cu_new[:P + 1].copy()
            q = _bf16(rng, (int(cu_q[-1]), hq, d))
            out = torch.empty((int(cu_q[-1]), hq, d), dtype=torch.bfloat16, device="cuda")
            bros.bros_attn_prefill_chunk(out, _dev(torch, q), torch.from_numpy(cu_q).cuda(), int(counts[:P].max()),
                                         k_dev, v_dev, td[:P], dd[:P], None, cd[:P], int(ctx[:P].max()))
            torch.cuda.synchronize()
            compare(_host(out), oracle.prefill_chunk(q, cu_q, kp, vp, tables[:P], dirs[:P], ctx[:P], "bf16"),
                    "bf16", f"prefill step {step}")
            stats["prefill"] += P
        if len(ids) > P:
            q = _bf16(rng, (len(ids) - P, hq, d))
            out = torch.empty((len(ids) - P, hq, d), dtype=torch.bfloat16, device="cuda")
            mc = int(ctx[P:].max())
            ws = torch.empty(max(16, bros.bros_attn_workspace_size(0, 1, len(ids) - P, hq, d, mc)), dtype=torch.uint8,
                             device="cuda")
            bros.bros_attn_decode(out, _dev(torch, q), k_dev, v_dev, td[P:], dd[P:], None, cd[P:], mc, workspace=ws)
            torch.cuda.synchronize()
            compare(_host(out), oracle.decode(q, kp, vp, tables[P:], dirs[P:], ctx[P:], "bf16"), "bf16",
                    f"decode step {step}")
            stats["decode"] += len(ids) - P
        mgr.validate()
    print("manager-driven steps:", stats)
    assert stats["victims"] > 0 and stats["restores"] > 0 and stats["prefill"] > 0 and stats["decode"] > 0, stats
