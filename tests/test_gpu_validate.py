"""GPU parity of the device-side metadata checks (ekv_validate_batch,
ekv_validate_transition) against oracle/validate.py: every count and every
first index, exactly.  Inputs are valid pools (which must report nothing)
and seeded mutations of them: table entries moved outside the pool, tag
values and mixed pairs, lengths out of range, boundaries that disagree with
the tags; transition lists with repeated, out-of-range, wrong-state and
partial pairs and bad new blocks.  The checks only read the arrays; no
other kernel runs on a mutated input.

With EKV_DEBUG=1 the attention and transition calls run the checks first:
an invalid call raises before anything is enqueued (pool, table, tags and
output unchanged), a valid one still matches the oracle."""

import os

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import lowering as olow
from oracle import transitions as otr
from oracle import validate as ov
from paper_2609_33536_amd import ekv, workloads
from tests.gpu_util import check_attention, default_scale, require_gpu, words_to_tensor

pytestmark = pytest.mark.gpu

PAGE = 16
MODES = {"native": ov.NATIVE, "structured": ov.STRUCTURED, "general": ov.GENERAL}


def _device_report(rep):
    counts = np.array([rep[name][0] for name in ekv.VIOLATIONS])
    first = np.array([rep[name][1] for name in ekv.VIOLATIONS])
    return counts, first


def _assert_same(got, want, what):
    gc, gf = got
    wc, wf = want
    assert np.array_equal(gc, wc), f"{what}: counts {gc.tolist()} != {wc.tolist()}"
    assert np.array_equal(gf, wf), f"{what}: first {gf.tolist()} != {wf.tolist()}"


def _case(seed):
    c = workloads.make_decode_case([64, 300, 1024, 77, 512, 0, 33], 8, 2, seed=seed, base_fraction=0.5,
                                   spare_blocks=8)
    pool, bt, tg, _, _ = otr.demote(c["pool"], c["block_table"], c["tags"], c["pairs"], c["seq_lens"])
    return c, pool, bt, tg


def _batch_check(torch, pool_words, hkv, lens, bt, tags, bounds, mode, max_seq_len=0):
    dev = [torch.from_numpy(np.ascontiguousarray(x)).cuda() if x is not None else None
           for x in (lens, bt, tags, bounds)]
    kvt = torch.empty(pool_words.shape[0] * 2 * hkv * PAGE * 128, dtype=torch.int16, device="cuda")
    pool = ekv.make_pool(kvt, hkv, "bf16")
    batch = ekv.make_batch(dev[0], dev[1], dev[2], dev[3], 4 * hkv, mode, max_seq_len)
    return _device_report(ekv.validate_batch(pool, batch))


def test_valid_batches_report_nothing():
    torch = require_gpu()
    c, pool, bt, tg = _case(5)
    mode, bounds = olow.lower(tg, c["seq_lens"], PAGE)
    assert mode == olow.GENERAL
    none = (np.zeros(ov.KINDS, dtype=np.int64), np.full(ov.KINDS, ov.NONE, dtype=np.int64))
    print("validate: valid general / structured / native batches", flush=True)
    _assert_same(_batch_check(torch, pool, 2, c["seq_lens"], bt, tg, None, ov.GENERAL), none, "general")
    c2 = workloads.make_decode_case([64, 300, 1024, 77, 512], 8, 2, seed=6, base_fraction=0.5,
                                    placement="oldest", spare_blocks=8)
    p2, bt2, tg2, _, _ = otr.demote(c2["pool"], c2["block_table"], c2["tags"], c2["pairs"], c2["seq_lens"])
    mode2, bounds2 = olow.lower(tg2, c2["seq_lens"], PAGE)
    assert mode2 == olow.STRUCTURED
    _assert_same(_batch_check(torch, p2, 2, c2["seq_lens"], bt2, tg2, bounds2, ov.STRUCTURED), none, "structured")
    _assert_same(_batch_check(torch, p2, 2, c2["seq_lens"], bt2, None, bounds2, ov.STRUCTURED), none,
                 "structured, no tags")
    _assert_same(_batch_check(torch, c["pool"], 2, c["seq_lens"], c["block_table"], c["tags"], None, ov.NATIVE),
                 none, "native")


def _mutate(rng, lens, bt, tags, bounds, nb):
    lens, bt, tags, bounds = lens.copy(), bt.copy(), tags.copy(), bounds.copy()
    bsz, max_blocks = bt.shape
    for _ in range(int(rng.integers(1, 6))):
        what = int(rng.integers(0, 4))
        s = int(rng.integers(0, bsz))
        # mostly a visible block (one past the end now and then)
        i = min(max_blocks - 1, int(rng.integers(0, max(1, -(-int(max(lens[s], 0)) // PAGE)) + 1)))
        if what == 0:
            bt[s, i] = [-2, -1, nb, nb + 7, int(rng.integers(0, nb))][int(rng.integers(0, 5))]
        elif what == 1:
            tags[s, i] = int(rng.integers(0, 3))
        elif what == 2:
            lens[s] = [-3, max_blocks * PAGE + int(rng.integers(1, 40)),
                       int(rng.integers(0, max_blocks * PAGE + 1))][int(rng.integers(0, 3))]
        else:
            bounds[s] = rng.integers(-2, max_blocks // 2 + 2, size=2)
    return lens, bt, tags, bounds


@pytest.mark.parametrize("seed", range(6))
def test_mutated_batches_match_oracle(seed):
    torch = require_gpu()
    c, pool, bt, tg = _case(10 + seed)
    nb = pool.shape[0]
    _, bounds = olow.lower(tg, c["seq_lens"], PAGE)
    rng = np.random.default_rng(100 + seed)
    for trial in range(4):
        lens_m, bt_m, tg_m, bounds_m = _mutate(rng, c["seq_lens"], bt, tg, bounds, nb)
        for name, mode in MODES.items():
            for with_tags in (True, False) if mode == ov.STRUCTURED else (True,):
                tags_arg = tg_m if with_tags else None
                bnd = bounds_m if mode == ov.STRUCTURED else None
                max_seq = int(rng.integers(0, bt.shape[1] * PAGE + 1)) if trial == 3 else 0
                print(f"validate batch: seed {seed} trial {trial} mode {name} tags {with_tags} "
                      f"max_seq_len {max_seq}", flush=True)
                got = _batch_check(torch, pool, 2, lens_m, bt_m, tags_arg, bnd, mode, max_seq)
                want = ov.batch_violations(lens_m, bt_m, tags_arg, bnd, mode, nb, max_seq)
                _assert_same(got, want, f"seed {seed} trial {trial} {name}")


@pytest.mark.parametrize("seed", range(6))
def test_transition_lists_match_oracle(seed):
    torch = require_gpu()
    c, pool, bt, tg = _case(20 + seed)
    nb = pool.shape[0]
    bsz, max_blocks = bt.shape
    rng = np.random.default_rng(200 + seed)
    kvt = torch.empty(nb * 2 * 2 * PAGE * 128, dtype=torch.int16, device="cuda")
    dpool = ekv.make_pool(kvt, 2, "bf16")
    bt_d, tg_d = torch.from_numpy(bt).cuda(), torch.from_numpy(tg).cuda()
    lens_d = torch.from_numpy(c["seq_lens"]).cuda()
    used = set(int(b) for s in range(bsz) for b in bt[s, :-(-int(c["seq_lens"][s]) // PAGE)])
    spare = np.array(sorted(set(range(nb)) - used), dtype=np.int32)
    for kind in (0, 1):
        state = 0 if kind == 0 else 1
        ok_pairs = [(s, j) for s in range(bsz) for j in range(int(c["seq_lens"][s]) // (2 * PAGE))
                    if tg[s, 2 * j] == state]
        for trial in range(4):
            k = min(len(ok_pairs), int(rng.integers(1, 12)))
            pick = rng.choice(len(ok_pairs), size=k, replace=False)
            pairs = np.array([ok_pairs[i] for i in pick], dtype=np.int32).reshape(-1, 2)
            new = spare[rng.choice(len(spare), size=len(pairs), replace=False)].copy()
            if trial > 0:   # plant mistakes: repeats, random pairs, bad new blocks
                for _ in range(int(rng.integers(1, 4))):
                    i = int(rng.integers(0, len(pairs)))
                    r = int(rng.integers(0, 3))
                    if r == 0:
                        pairs[i] = pairs[int(rng.integers(0, len(pairs)))]
                    elif r == 1:
                        pairs[i] = (int(rng.integers(-1, bsz + 1)), int(rng.integers(-1, max_blocks // 2 + 1)))
                    else:
                        new[i] = int(rng.integers(-2, nb + 2))
            pairs_d, new_d = torch.from_numpy(pairs).cuda(), torch.from_numpy(new).cuda()
            for with_lens in (True, False):
                print(f"validate list: seed {seed} kind {kind} trial {trial} n {len(pairs)} lens {with_lens}",
                      flush=True)
                rep = ekv.validate_transition(dpool, kind, pairs_d, bt_d, tg_d, lens_d if with_lens else None,
                                              new_d if kind else None)
                want = ov.list_violations(kind, pairs, bt, tg, nb, c["seq_lens"] if with_lens else None,
                                          new if kind else None)
                _assert_same(_device_report(rep), want, f"seed {seed} kind {kind} trial {trial}")
                if trial == 0:
                    assert _device_report(rep)[0].sum() == 0


@pytest.fixture
def debug_env():
    old = os.environ.get("EKV_DEBUG")
    os.environ["EKV_DEBUG"] = "1"
    yield
    if old is None:
        del os.environ["EKV_DEBUG"]
    else:
        os.environ["EKV_DEBUG"] = old


def test_debug_mode_refuses_invalid_calls(debug_env):
    torch = require_gpu()
    c = workloads.make_decode_case([64, 300, 1024, 77], 8, 2, seed=31, base_fraction=0.5, spare_blocks=8)
    dev = torch.from_numpy(c["pool"].view(np.int16).copy()).cuda()
    pool = ekv.make_pool(dev, 2, "bf16")
    bt = torch.from_numpy(c["block_table"].copy()).cuda()
    tags = torch.from_numpy(c["tags"].copy()).cuda()
    lens = torch.from_numpy(c["seq_lens"].copy()).cuda()
    pairs = c["pairs"]
    assert len(pairs) >= 2
    freed = torch.empty(len(pairs) + 1, dtype=torch.int32, device="cuda")
    # a repeated pair: refused, nothing changes
    bad = torch.from_numpy(np.concatenate([pairs, pairs[:1]]).astype(np.int32)).cuda()
    print("EKV_DEBUG: demote with a repeated pair", flush=True)
    with pytest.raises(ekv.EkvError, match="listed twice"):
        ekv.demote(pool, bad, bt, tags, freed)
    torch.cuda.synchronize()
    assert np.array_equal(dev.cpu().numpy().view(np.uint16), c["pool"])
    assert np.array_equal(bt.cpu().numpy(), c["block_table"]) and np.array_equal(tags.cpu().numpy(), c["tags"])
    # the valid list goes through and matches the oracle bit for bit
    print("EKV_DEBUG: valid demote", flush=True)
    ekv.demote(pool, torch.from_numpy(pairs.copy()).cuda(), bt, tags, freed[:len(pairs)])
    torch.cuda.synchronize()
    opool, obt, otg, ofreed, _ = otr.demote(c["pool"], c["block_table"], c["tags"], pairs, c["seq_lens"])
    assert np.array_equal(dev.cpu().numpy().view(np.uint16), opool)
    assert np.array_equal(freed[:len(pairs)].cpu().numpy(), ofreed)
    # demoting the same pairs again: they are BASE now
    print("EKV_DEBUG: demote of BASE pairs", flush=True)
    with pytest.raises(ekv.EkvError, match="wrong state"):
        ekv.demote(pool, torch.from_numpy(pairs.copy()).cuda(), bt, tags, freed[:len(pairs)])
    # decode: valid in general mode, then with a table entry outside the pool
    q = workloads.to_words(np.random.default_rng(32).standard_normal((4, 8, 128), dtype=np.float32), "bf16")
    out = torch.full((4, 8, 128), float("nan"), dtype=torch.float32, device="cuda")
    batch = ekv.make_batch(lens, bt, tags, None, 8, ekv.MODE_GENERAL)
    ws = ekv.decode_workspace(pool, batch)
    print("EKV_DEBUG: valid decode", flush=True)
    ekv.attn_decode(pool, batch, words_to_tensor(q, torch, "bf16"), out, default_scale(), ws)
    torch.cuda.synchronize()
    check_attention(out.cpu().numpy(), oatt.decode(q, opool, obt, otg, c["seq_lens"]), True)
    bt_bad = bt.clone()
    bt_bad[2, 3] = c["pool"].shape[0]
    out.fill_(float("nan"))
    batch_bad = ekv.make_batch(lens, bt_bad, tags, None, 8, ekv.MODE_GENERAL)
    print("EKV_DEBUG: decode with a table entry outside the pool", flush=True)
    with pytest.raises(ekv.EkvError, match="outside the pool"):
        ekv.attn_decode(pool, batch_bad, words_to_tensor(q, torch, "bf16"), out, default_scale(), ws)
    torch.cuda.synchronize()
    assert torch.isnan(out).all()
