"""A serving loop driven by the library's fidelity controller (Alg. 1) on
the GPU.  Each step every sequence first grows by one 16-token block (the
step's demand D_t), so the pool runs short; the controller demotes ahead
of the shortage and, once growth stops, promotes within its reserve-aware
budget (two requests finish and return their blocks when growth stops).
On the other side the oracle runs the same loop with its own
controller and transitions.  Checked every step: the controller's lists,
shortage, surplus, reserve and budget; device pool blocks, block table,
tags, host mirror and free FIFO bit for bit; decode of every sequence
within the attention tolerance."""

import numpy as np

from oracle import attention as oatt
from oracle import control as oc
from oracle import lowering as olow
from oracle import transitions as otr
from paper_2609_33536_amd import ekv, kvpool, workloads
from tests.gpu_util import check_attention, default_scale, require_gpu, words_to_tensor

import pytest

pytestmark = pytest.mark.gpu

PAGE = 16


def test_controller_driven_growth_loop():
    torch = require_gpu()
    bsz, hq, hkv, grow_steps, steps = 8, 8, 2, 9, 16
    rng = np.random.default_rng(21)
    lens = (rng.integers(20, 40, size=bsz) * PAGE + rng.integers(0, PAGE, size=bsz)).astype(np.int32)
    max_blocks = 2 * (int(lens.max()) // (2 * PAGE) + grow_steps + 2)
    case = workloads.make_decode_case(lens, hq, hkv, seed=21, spare_blocks=3, max_blocks=max_blocks)
    kv = kvpool.PagedKV(case["pool"], case["block_table"], lens, case["free"], hkv)
    host_pool = case["pool"].copy()
    obt, otg, olens = case["block_table"].copy(), case["tags"].copy(), lens.copy()
    ofifo = otr.FreeFifo(case["free"])
    kw = dict(min_batch=16, decay=2, sink_pairs=1, recent_pairs=2)
    cfg, cst = ekv.ctrl_config(**kw), ekv.CtrlState()
    octl = oc.Controller(oc.Config(**kw))
    lo_dev, lo_host = {}, {}
    promoted_total = demoted_total = 0
    for step in range(steps):
        if step == grow_steps:
            # the two longest requests finish: their blocks (a packed pair's once) return to the pool
            for s in np.argsort(-olens, kind="stable")[:2]:
                blocks = list(dict.fromkeys(int(b) for b in obt[s, :-(-int(olens[s]) // PAGE)]))
                ofifo.commit_freed(blocks)
                kv.mirror.commit_freed(blocks)
                olens[s] = 0
                otg[s, :] = 0
                obt[s, :] = 0
                for key in [key for key in lo_dev if key[0] == s]:
                    del lo_dev[key], lo_host[key]
            kv.mirror.bt[:] = obt
            kv.mirror.tags[:] = otg
            kv.mirror.seq_lens[:] = olens
            kv.bt.copy_(torch.from_numpy(obt.copy()))
            kv.tags.copy_(torch.from_numpy(otg.copy()))
            kv.seq_lens.copy_(torch.from_numpy(olens.copy()))
        grow = step < grow_steps
        nblk = -(-olens // PAGE)
        demand = int(((-(-(olens + PAGE) // PAGE)) - nblk).sum()) if grow else 0
        free = len(ofifo)
        assert free == len(kv.mirror.free)
        # ---- demotion ahead of the shortage ----
        dp = ekv.ctrl_demotion(cfg, cst, demand, free, kv.mirror.tags, kv.mirror.seq_lens)
        odp = octl.demotion(demand, free, otg, olens)
        assert dp.tolist() == odp.tolist()
        assert (cst.shortage, cst.surplus) == (octl.shortage, octl.surplus)
        print(f"step {step}: D={demand} F={free} demote {len(dp)}", flush=True)
        if len(dp):
            freed, lo, _ = kv.demote(dp)
            host_pool, obt, otg, ofreed, olo = otr.demote(host_pool, obt, otg, dp, olens)
            torch.cuda.synchronize()
            assert np.array_equal(freed.cpu().numpy(), ofreed)
            for i, (s, j) in enumerate(dp):
                lo_dev[(int(s), int(j))] = lo[i]
                lo_host[(int(s), int(j))] = olo[i]
            kv.commit()
            ofifo.commit_freed(ofreed)
            demoted_total += len(dp)
        # ---- the step's growth: one new block per sequence, 16 new tokens ----
        if grow:
            new_blocks = ofifo.acquire(demand)
            assert [kv.mirror.free.popleft() for _ in range(demand)] == new_blocks.tolist()
            k = 0
            slot_list = []
            for s in range(bsz):
                old = int(olens[s])
                first_new = -(-old // PAGE)
                if -(-(old + PAGE) // PAGE) > first_new:
                    obt[s, first_new] = new_blocks[k]
                    k += 1
                for t in range(old, old + PAGE):
                    slot_list.append(int(obt[s, t // PAGE]) * PAGE + t % PAGE)
            slots = np.array(slot_list, dtype=np.int32)
            knew = workloads.to_words(rng.standard_normal((len(slots), hkv, 128), dtype=np.float32), "bf16")
            vnew = workloads.to_words(rng.standard_normal((len(slots), hkv, 128), dtype=np.float32), "bf16")
            host_pool = otr.append(host_pool, slots, knew, vnew)
            olens = olens + PAGE
            kv.mirror.bt[:] = obt
            kv.mirror.seq_lens[:] = olens
            kv.bt.copy_(torch.from_numpy(obt.copy()))
            kv.seq_lens.copy_(torch.from_numpy(olens.copy()))
            assert (slots // PAGE < host_pool.shape[0]).all()
            kv.append(torch.from_numpy(slots).cuda(), words_to_tensor(knew, torch, "bf16"),
                      words_to_tensor(vnew, torch, "bf16"))
        # ---- promotion within the budget ----
        free_post = len(ofifo)
        pp = ekv.ctrl_promotion(cfg, cst, free_post, 4, kv.mirror.tags, kv.mirror.seq_lens)
        opp = octl.promotion(free_post, 4, otg, olens)
        assert pp.tolist() == opp.tolist()
        assert (cst.reserve, cst.budget) == (octl.reserve, octl.budget)
        if len(pp):
            lo_in = torch.stack([lo_dev.pop((int(s), int(j))) for s, j in pp])
            new = kv.refine(pp, lo_in)
            onew = ofifo.acquire(len(pp))
            assert np.array_equal(new, onew)
            olo_in = np.stack([lo_host.pop((int(s), int(j))) for s, j in pp])
            host_pool, obt, otg = otr.refine(host_pool, obt, otg, pp, onew, olo_in, olens)
            promoted_total += len(pp)
        print(f"  F_post={free_post} R={cst.reserve} P={cst.budget} promote {len(pp)}", flush=True)
        # ---- bookkeeping and pool, bit for bit ----
        torch.cuda.synchronize()
        assert np.array_equal(kv.bt.cpu().numpy(), obt)
        assert np.array_equal(kv.tags.cpu().numpy(), otg)
        assert np.array_equal(kv.mirror.bt, obt) and np.array_equal(kv.mirror.tags, otg)
        assert np.array_equal(np.array(kv.mirror.free, dtype=np.int32), ofifo.snapshot())
        live = sorted({int(b) for s in range(bsz) for b in obt[s, :-(-int(olens[s]) // PAGE)]})
        got = kv.kv.view(-1, 2, hkv, PAGE, 128)[live].cpu().numpy().view(np.uint16)
        assert np.array_equal(got, host_pool[live])
        # ---- decode ----
        mode = kv.relower()
        omode, obounds = olow.lower(otg, olens, PAGE)
        assert mode == omode and np.array_equal(kv.bounds.cpu().numpy(), obounds)
        assert mode != olow.GENERAL          # the rank orders keep BASE runs structured
        q = workloads.to_words(rng.standard_normal((bsz, hq, 128), dtype=np.float32), "bf16")
        batch = kv.batch(hq)
        ws = ekv.decode_workspace(kv.pool, batch)
        out = torch.empty((bsz, hq, 128), dtype=torch.float32, device="cuda")
        ekv.attn_decode(kv.pool, batch, words_to_tensor(q, torch, "bf16"), out, default_scale(), ws)
        torch.cuda.synchronize()
        ref = oatt.decode(q, host_pool, obt, otg, olens)
        check_attention(out.cpu().numpy(), ref, True)
    assert demoted_total > 0 and promoted_total > 0
